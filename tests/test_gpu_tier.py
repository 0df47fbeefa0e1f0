"""The host tier on the GPU, through the C ABI: residency plan, copies from a
pinned host mirror into the GPU reserve, and attention over the reserve.

- The plan (slot of every kept chunk, copy list, slot owners) equals the
  oracle's plan exactly, firing after firing, from a cold reserve on.
- After the copies every kept chunk's reserve blocks equal its mirror blocks
  byte for byte, and slots that received no copy are untouched.
- Attention over the reserve equals the attention over the full cache for the
  same kept chunks bit for bit, and the oracle's attention within tolerance.
- Asynchronous recall: the plan and copies of firing t run on a second stream
  while decode reads the previous kept set on the first; every decode output
  equals the full-cache attention over the set it read.
- The attention over the reserve replays from a captured graph with new slot
  lists between replays, each replay equal to the eager call.
- The DMA-engine copies from a host copy of the list (packed and padded mirror
  layouts, merged runs of adjacent chunks) fill the reserve the same way.
- lsa_tier_step (Level 2 over the resident set, then attention over the chosen
  slots) chooses the oracle's chunks, up to the float32 band of the k2-th
  native score, and attends over them bit for bit like the full-cache path.
- All of the above once more at the benchmark's 1M-token size.
"""
from __future__ import annotations

import numpy as np
import pytest

import lsa_synth as synth
import oracle
import parity
from gpu_case import log

pytestmark = pytest.mark.gpu


def _kept_sets(n, keep, firings, rng):
    """Ascending kept sets of one sequence for consecutive firings: a cold set,
    the same set again, small and large churn, a smaller set, an empty one and
    a full one."""
    def pick(k, base=None, churn=1.0):
        if base is None or len(base) == 0:
            return np.sort(rng.choice(n, size=k, replace=False))
        keep_n = min(len(base), int(round(k * (1.0 - churn))))
        kept = rng.choice(base, size=keep_n, replace=False) if keep_n else np.zeros(0, np.int64)
        rest = np.setdiff1d(np.arange(n), kept)
        new = rng.choice(rest, size=k - keep_n, replace=False)
        return np.sort(np.concatenate([kept, new]))
    out = [pick(keep)]
    patterns = [(keep, 0.0), (keep, 0.1), (keep, 1.0), (max(keep // 2, 1), 0.3), (0, 1.0), (keep, 0.5)]
    for i in range(firings - 1):
        k, churn = patterns[i % len(patterns)]
        out.append(pick(k, out[-1], churn) if k else np.zeros(0, np.int64))
    return out


class TierCase:
    """Device state of one host-tier problem: pinned mirror, reserve, owner table."""

    def __init__(self, prob, seed, slots):
        import torch
        import paper_2606_09079_amd as L
        self.prob, self.seed = prob, seed
        self.dev = synth.device_inputs(prob, seed)
        self.host_k = torch.empty(self.dev["k"].shape, dtype=torch.int16, pin_memory=True)
        self.host_v = torch.empty(self.dev["v"].shape, dtype=torch.int16, pin_memory=True)
        self.host_k.copy_(self.dev["k"])
        self.host_v.copy_(self.dev["v"])
        self.P, self.T = L.Problem.from_synth(prob), L.Tier(slots)
        self.pitch, self.total, self.ws_bytes = L.lsa_tier_sizes(self.P, self.T)
        self.slots = list(slots)
        self.slot_off = np.concatenate([[0], np.cumsum(slots)]).astype(np.int64)
        blk = prob.n_kv_heads * prob.chunk * prob.head_dim
        self.res_k = torch.full((self.total * blk,), 0x5A5A, dtype=torch.int16, device="cuda")
        self.res_v = torch.full((self.total * blk,), 0x3C3C, dtype=torch.int16, device="cuda")
        self.owner = torch.empty(self.total, dtype=torch.int32, device="cuda")
        L.lsa_tier_reset(self.P, self.T, self.owner)
        self.ws = torch.zeros(max(self.ws_bytes, 256), dtype=torch.uint8, device="cuda")
        B = prob.batch
        self.fetch = torch.full((B, self.pitch, 2), -7, dtype=torch.int32, device="cuda")
        self.fetch_count = torch.full((B,), -7, dtype=torch.int32, device="cuda")

    def kept_tensors(self, sets):
        import torch
        B = self.prob.batch
        kept = np.full((B, self.pitch), -1, dtype=np.int32)
        cnt = np.zeros(B, dtype=np.int32)
        for b, s in enumerate(sets):
            kept[b, :len(s)] = s
            cnt[b] = len(s)
        return torch.from_numpy(kept).cuda(), torch.from_numpy(cnt).cuda()

    def blocks(self, t, ids):
        """[len(ids)][Hkv][C * 128] blocks of a chunk-paged buffer at global ids."""
        import torch
        v = t.view(-1, self.prob.n_kv_heads, self.prob.chunk * self.prob.head_dim)
        return v[torch.as_tensor(np.asarray(ids, dtype=np.int64), device=t.device)]


def _plan_and_check(tc, L, sets, prev, oracle_state, stream=None):
    """One firing: plan on the GPU, compare with the oracle, return the slot list tensor."""
    import torch
    prob = tc.prob
    kept, cnt = tc.kept_tensors(sets)
    slot_idx = torch.full((prob.batch, tc.pitch), -9, dtype=torch.int32, device="cuda")
    prev_slots, prev_cnt = prev if prev is not None else (None, None)
    L.lsa_tier_plan(tc.P, tc.T, kept, cnt, prev_slots, prev_cnt, tc.owner, slot_idx, tc.fetch, tc.fetch_count,
                    stream)
    torch.cuda.synchronize()
    g_owner, g_slots = tc.owner.cpu().numpy(), slot_idx.cpu().numpy()
    g_fetch, g_fc = tc.fetch.cpu().numpy(), tc.fetch_count.cpu().numpy()
    copies = []
    for b, s in enumerate(sets):
        o_owner, o_old = oracle_state[b]
        new_owner, new_slots, fetch = oracle.tier_plan(o_owner, o_old, [int(c) for c in s])
        lo, hi = tc.slot_off[b], tc.slot_off[b + 1]
        assert g_owner[lo:hi].tolist() == new_owner, f"seq {b}: owner table differs from the oracle"
        assert g_slots[b, :len(s)].tolist() == new_slots, f"seq {b}: slots differ from the oracle"
        assert int(g_fc[b]) == len(fetch), f"seq {b}: {g_fc[b]} copies, oracle {len(fetch)}"
        assert [tuple(x) for x in g_fetch[b, :len(fetch)].tolist()] == fetch, f"seq {b}: copy list differs"
        oracle_state[b] = (new_owner, new_slots)
        copies.append(fetch)
    return kept, cnt, slot_idx, copies


def _check_reserve(tc, sets, slot_lists):
    """Every kept chunk's reserve blocks equal its mirror blocks."""
    for b, s in enumerate(sets):
        if len(s) == 0:
            continue
        glob_c = np.asarray(s, dtype=np.int64) + tc.prob.chunk_offsets[b]
        glob_s = np.asarray(slot_lists[b], dtype=np.int64) + tc.slot_off[b]
        for which, res in (("k", tc.res_k), ("v", tc.res_v)):
            got = tc.blocks(res, glob_s)
            want = tc.blocks(tc.dev[which], glob_c)
            assert bool((got == want).all()), f"seq {b}: reserve {which} blocks differ from the mirror"


def _direct_attention(tc, L, kept, cnt):
    import torch
    prob = tc.prob
    P = L.Problem.from_synth(prob)
    ws_bytes = L.lsa_workspace_size(P)
    ws = torch.zeros(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    shp = (prob.batch, prob.n_qtok, prob.n_q_heads, prob.head_dim)
    out = torch.empty(shp, dtype=torch.float32, device="cuda")
    lse = torch.empty(shp[:3], dtype=torch.float32, device="cuda")
    L.lsa_sparse_decode_attn(P, tc.dev["q"], tc.dev["k"], tc.dev["v"], kept, cnt, 0.0, out, lse, ws, ws_bytes)
    return out, lse


def _tier_attention(tc, L, slot_idx, cnt, stream=None):
    import torch
    prob = tc.prob
    shp = (prob.batch, prob.n_qtok, prob.n_q_heads, prob.head_dim)
    out = torch.full(shp, float("nan"), dtype=torch.float32, device="cuda")
    lse = torch.full(shp[:3], float("nan"), dtype=torch.float32, device="cuda")
    L.lsa_tier_attend(tc.P, tc.T, tc.dev["q"], tc.res_k, tc.res_v, slot_idx, cnt, 0.0, out, lse, tc.ws, tc.ws_bytes,
                      stream)
    return out, lse


def _oracle_rows(tc, b, kept, out, lse, rows):
    prob, host = tc.prob, tc.dev["host"]
    toks = oracle.kept_tokens(kept, prob.chunk, prob.ctx_tokens[b])
    by_g = {}
    for (t, h) in rows:
        by_g.setdefault(h // prob.group, []).append((t, h))
    for g, rs in sorted(by_g.items()):
        Kh = synth.kv_head_sparse(prob, tc.seed, "k", b, g, kept)
        Vh = synth.kv_head_sparse(prob, tc.seed, "v", b, g, kept)
        qr = np.stack([host["q"][b, t, h] for (t, h) in rs])
        r_out, r_lse = oracle.attention_tokens(qr, Kh, Vh, toks)
        parity.check_attention(np.stack([out[b, t, h] for (t, h) in rs]), [lse[b, t, h] for (t, h) in rs], r_out,
                               r_lse, f"tier seq {b} g {g}")


CASES = [
    ("ragged3", [64 * 300, 64 * 1000, 64 * 77], 64, [40, 100, 77], [80, 250, 154], 8, 2),
    ("c128_one", [128 * 500], 128, [60], [121], 16, 4),
    # the largest sequence the residency plan takes (LSA_MAX_TIER_CHUNKS) with
    # the largest reserve (LSA_MAX_TIER_SLOTS slots)
    ("max_chunks_slots", [64 * 131072], 64, [300], [65536], 1, 1),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: c[0])
def test_tier_firings_match_oracle(case):
    import torch
    import paper_2606_09079_amd as L
    name, ctx, C, keep, slots, hq, hkv = case
    prob = synth.Problem(f"tier_{name}", ctx, C, keep, hq, hkv)
    log(f"[tier] {name} ctx={ctx} C={C} keep={keep} slots={slots}")
    tc = TierCase(prob, 11, slots)
    rng = np.random.default_rng(5)
    per_seq = [_kept_sets(prob.n_chunks[b], keep[b], 7, rng) for b in range(prob.batch)]
    state = [([-1] * slots[b], []) for b in range(prob.batch)]
    prev = None
    for f in range(7):
        sets = [per_seq[b][f] for b in range(prob.batch)]
        kept, cnt, slot_idx, copies = _plan_and_check(tc, L, sets, prev, state)
        L.lsa_tier_fetch(tc.P, tc.T, tc.host_k, tc.host_v, tc.fetch, tc.fetch_count, tc.res_k, tc.res_v)
        torch.cuda.synchronize()
        if f == 0:  # cold start: every kept chunk is copied; untouched slots keep their fill
            for b in range(prob.batch):
                assert len(copies[b]) == len(sets[b])
                unused = np.setdiff1d(np.arange(slots[b]), [s for _, s in copies[b]]) + tc.slot_off[b]
                if len(unused):
                    assert bool((tc.blocks(tc.res_k, unused) == 0x5A5A).all())
        _check_reserve(tc, sets, [state[b][1] for b in range(prob.batch)])
        t_out, t_lse = _tier_attention(tc, L, slot_idx, cnt)
        d_out, d_lse = _direct_attention(tc, L, kept, cnt)
        torch.cuda.synchronize()
        assert torch.equal(t_out, d_out) and torch.equal(t_lse, d_lse), \
            f"firing {f}: reserve attention differs from the full-cache attention"
        if f in (0, 2):
            rows = [(0, h) for h in range(0, prob.n_q_heads, max(prob.group // 2, 1))]
            o, s = t_out.cpu().numpy(), t_lse.cpu().numpy()
            for b in range(prob.batch):
                if len(sets[b]):
                    _oracle_rows(tc, b, sets[b], o, s, rows)
        prev = (slot_idx, cnt)
        log(f"[tier] firing {f}: kept {[len(s) for s in sets]}, copies {[len(c) for c in copies]}")


def test_tier_async_recall_two_streams():
    """Firing t plans and copies on a side stream while decode reads the set of
    firing t - 1 on the main stream; decode t + 1 reads the new set."""
    import torch
    import paper_2606_09079_amd as L
    prob = synth.Problem("tier_async", [64 * 2000, 64 * 600], 64, [200, 60], 8, 2)
    slots = [400, 130]
    tc = TierCase(prob, 12, slots)
    rng = np.random.default_rng(9)
    F = 8
    per_seq = [_kept_sets(prob.n_chunks[b], prob.keep[b], F, rng) for b in range(prob.batch)]
    firings = [tc.kept_tensors([per_seq[b][f] for b in range(prob.batch)]) for f in range(F)]
    slot_buf = [torch.full((prob.batch, tc.pitch), -1, dtype=torch.int32, device="cuda") for _ in range(2)]
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    L.lsa_tier_plan(tc.P, tc.T, firings[0][0], firings[0][1], None, None, tc.owner, slot_buf[0], tc.fetch,
                    tc.fetch_count)
    L.lsa_tier_fetch(tc.P, tc.T, tc.host_k, tc.host_v, tc.fetch, tc.fetch_count, tc.res_k, tc.res_v)
    outs = []
    for t in range(1, F):
        cur, nxt = (t - 1) % 2, t % 2
        side.wait_stream(main)  # decode t - 1 has finished reading slot_buf[nxt]
        L.lsa_tier_plan(tc.P, tc.T, firings[t][0], firings[t][1], slot_buf[cur], firings[t - 1][1], tc.owner,
                        slot_buf[nxt], tc.fetch, tc.fetch_count, side)
        L.lsa_tier_fetch(tc.P, tc.T, tc.host_k, tc.host_v, tc.fetch, tc.fetch_count, tc.res_k, tc.res_v, side)
        outs.append(_tier_attention(tc, L, slot_buf[cur], firings[t - 1][1], main))
        main.wait_stream(side)
    outs.append(_tier_attention(tc, L, slot_buf[(F - 1) % 2], firings[F - 1][1], main))
    torch.cuda.synchronize()
    for t in range(F):
        d_out, d_lse = _direct_attention(tc, L, *firings[t])
        torch.cuda.synchronize()
        assert torch.equal(outs[t][0], d_out) and torch.equal(outs[t][1], d_lse), \
            f"decode over the set of firing {t} differs from the full-cache attention"
    log(f"[tier] async: {F} firings, kept {[int(x) for x in firings[-1][1].cpu()]}")


def test_tier_attention_graph_replay():
    """The attention over the reserve captured once, replayed with new slot lists."""
    import torch
    import paper_2606_09079_amd as L
    prob = synth.Problem("tier_graph", [64 * 900], 64, [90], 32, 8)
    tc = TierCase(prob, 13, [180])
    rng = np.random.default_rng(4)
    sets = _kept_sets(prob.n_chunks[0], 90, 5, rng)
    state = [([-1] * 180, [])]
    slot_g = torch.full((1, tc.pitch), 0, dtype=torch.int32, device="cuda")
    cnt_g = torch.zeros(1, dtype=torch.int32, device="cuda")
    shp = (1, 1, prob.n_q_heads, prob.head_dim)
    out_g = torch.empty(shp, dtype=torch.float32, device="cuda")
    lse_g = torch.empty(shp[:3], dtype=torch.float32, device="cuda")

    def attend():
        L.lsa_tier_attend(tc.P, tc.T, tc.dev["q"], tc.res_k, tc.res_v, slot_g, cnt_g, 0.0, out_g, lse_g, tc.ws,
                          tc.ws_bytes)

    prev = None
    kept, cnt, slot_idx, _ = _plan_and_check(tc, L, [sets[0]], prev, state)
    L.lsa_tier_fetch(tc.P, tc.T, tc.host_k, tc.host_v, tc.fetch, tc.fetch_count, tc.res_k, tc.res_v)
    slot_g.copy_(slot_idx)
    cnt_g.copy_(cnt)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        attend()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        attend()
    torch.cuda.synchronize()
    prev = (slot_idx, cnt)
    for f in range(1, 5):
        kept, cnt, slot_idx, _ = _plan_and_check(tc, L, [sets[f]], prev, state)
        L.lsa_tier_fetch(tc.P, tc.T, tc.host_k, tc.host_v, tc.fetch, tc.fetch_count, tc.res_k, tc.res_v)
        slot_g.copy_(slot_idx)
        cnt_g.copy_(cnt)
        for rep in range(2):
            out_g.fill_(float("nan"))
            g.replay()
            torch.cuda.synchronize()
            e_out, e_lse = _tier_attention(tc, L, slot_idx, cnt)
            torch.cuda.synchronize()
            assert torch.equal(out_g, e_out) and torch.equal(lse_g, e_lse), f"firing {f} replay {rep} differs"
        prev = (slot_idx, cnt)
    log("[tier] graph replays match the eager calls")


def test_tier_fetch_rejects_pageable_mirror():
    """A mirror in ordinary (pageable) host memory is refused before any launch."""
    import torch
    import paper_2606_09079_amd as L
    prob = synth.Problem("tier_pageable", [64 * 40], 64, [8], 8, 2)
    P, T = L.Problem.from_synth(prob), L.Tier([16])
    pitch, total, _ = L.lsa_tier_sizes(P, T)
    n = prob.kv_elems()
    pageable = np.zeros(n + 8, dtype=np.int16)
    base = pageable.ctypes.data
    aligned = base + (-base % 16)
    fetch = torch.zeros((1, pitch, 2), dtype=torch.int32, device="cuda")
    fc = torch.zeros(1, dtype=torch.int32, device="cuda")
    res = torch.zeros(total * 2 * 64 * 128, dtype=torch.int16, device="cuda")
    with pytest.raises(L.LsaError) as e:
        L.lsa_tier_fetch(P, T, aligned, aligned, fetch, fc, res, res)
    assert e.value.status == 1
    pinned = torch.empty(n, dtype=torch.int16, pin_memory=True)
    L.lsa_tier_fetch(P, T, pinned, pinned, fetch, fc, res, res)  # no copies (count 0), accepted
    torch.cuda.synchronize()


def _strided_cache(prob, seed, cs, hs):
    """K and V of prob in a device cache with chunk stride cs and head stride hs (elements)."""
    import torch
    n = (prob.total_chunks - 1) * cs + (prob.n_kv_heads - 1) * hs + prob.chunk * prob.head_dim
    table = torch.from_numpy(synth.normal_table_bf16().view(np.int16)).cuda()
    out = []
    for which in ("k", "v"):
        t = torch.zeros(n, dtype=torch.int16, device="cuda")
        synth.fill_kv_device(prob, seed, which, t.data_ptr(), table.data_ptr(),
                             torch.cuda.current_stream().cuda_stream, chunk_stride=cs, head_stride=hs)
        out.append(t)
    return out


@pytest.mark.parametrize("layout", ["packed", "padded_heads"])
def test_tier_dma_copies(layout):
    """lsa_tier_fetch_dma from the host copy of a plan's list: the reserve holds
    the mirror's blocks, and attention over it equals the full-cache attention."""
    import torch
    import paper_2606_09079_amd as L
    prob = synth.Problem(f"tier_dma_{layout}", [64 * 700, 64 * 90], 64, [70, 30], 16, 4)
    C, d, H = prob.chunk, prob.head_dim, prob.n_kv_heads
    hs = C * d if layout == "packed" else C * d + 64
    cs = H * hs
    k_dev, v_dev = _strided_cache(prob, 14, cs, hs)
    host_k = torch.empty(k_dev.shape, dtype=torch.int16, pin_memory=True)
    host_v = torch.empty(v_dev.shape, dtype=torch.int16, pin_memory=True)
    host_k.copy_(k_dev)
    host_v.copy_(v_dev)
    P = L.Problem.from_synth(prob, kv_chunk_stride=cs, kv_head_stride=hs)
    T = L.Tier([140, 60])
    pitch, total, ws_bytes = L.lsa_tier_sizes(P, T)
    slot_off = [0, 140]
    res_k = torch.full((total * H * C * d,), 0x1111, dtype=torch.int16, device="cuda")
    res_v = torch.full_like(res_k, 0x2222)
    owner = torch.empty(total, dtype=torch.int32, device="cuda")
    L.lsa_tier_reset(P, T, owner)
    rng = np.random.default_rng(2)
    # firing 0: a run of adjacent chunks (merged copies) plus scattered ones; then churn
    sets0 = [np.sort(np.concatenate([np.arange(100, 140), rng.choice(np.arange(200, 700), 30, replace=False)])),
             np.arange(0, 30)]
    sets1 = [np.sort(np.concatenate([sets0[0][::2], rng.choice(np.setdiff1d(np.arange(700), sets0[0]), 35,
                                                                replace=False)])),
             np.sort(rng.choice(90, 30, replace=False))]
    side = torch.cuda.Stream()
    prev = None
    ws = torch.zeros(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    q = torch.from_numpy(synth.host_inputs(prob, 14)["q"].view(np.int16)).cuda()
    for f, sets in enumerate((sets0, sets1)):
        kept = np.full((2, pitch), -1, dtype=np.int32)
        cnt = np.zeros(2, dtype=np.int32)
        for b, s in enumerate(sets):
            kept[b, :len(s)] = s
            cnt[b] = len(s)
        kept_d, cnt_d = torch.from_numpy(kept).cuda(), torch.from_numpy(cnt).cuda()
        slot_idx = torch.empty(2, pitch, dtype=torch.int32, device="cuda")
        fetch = torch.empty(2, pitch, 2, dtype=torch.int32, device="cuda")
        fc = torch.empty(2, dtype=torch.int32, device="cuda")
        L.lsa_tier_plan(P, T, kept_d, cnt_d, prev[0] if prev else None, prev[1] if prev else None, owner, slot_idx,
                        fetch, fc)
        torch.cuda.synchronize()
        h_fetch, h_fc = fetch.cpu().numpy(), fc.cpu().numpy()
        L.lsa_tier_fetch_dma(P, T, host_k, host_v, h_fetch, h_fc, res_k, res_v, side)
        torch.cuda.synchronize()
        slots = slot_idx.cpu().numpy()
        for b, s in enumerate(sets):
            for which, dev_t, res in (("k", k_dev, res_k), ("v", v_dev, res_v)):
                for i, c in enumerate(s):
                    g_off = (prob.chunk_offsets[b] + int(c)) * cs
                    want = torch.as_strided(dev_t, (H, C * d), (hs, 1), g_off)
                    got = res.view(-1, H, C * d)[slot_off[b] + int(slots[b, i])]
                    assert torch.equal(got, want), f"firing {f} seq {b} chunk {c} {which}: reserve != mirror"
        shp = (2, 1, 16, d)
        t_out, t_lse = torch.empty(shp, device="cuda"), torch.empty(shp[:3], device="cuda")
        L.lsa_tier_attend(P, T, q, res_k, res_v, slot_idx, cnt_d, 0.0, t_out, t_lse, ws, ws_bytes)
        d_ws = torch.zeros(max(L.lsa_workspace_size(P), 256), dtype=torch.uint8, device="cuda")
        d_out, d_lse = torch.empty(shp, device="cuda"), torch.empty(shp[:3], device="cuda")
        L.lsa_sparse_decode_attn(P, q, k_dev, v_dev, kept_d, cnt_d, 0.0, d_out, d_lse, d_ws, d_ws.numel())
        torch.cuda.synchronize()
        assert torch.equal(t_out, d_out) and torch.equal(t_lse, d_lse)
        prev = (slot_idx, cnt_d)
        log(f"[tier] DMA {layout} firing {f}: copies {h_fc.tolist()}")


STEP_CASES = [
    # name, ctx tokens, C, K_max, slots, core_keep (k2), native heads, key width
    ("ragged3", [64 * 900, 64 * 400, 64 * 130], 64, [120, 60, 40], [240, 125, 80], [30, 100, 1], 32, 128),
    ("c128_n16_c64", [128 * 700], 128, [90], [180], [25], 16, 64),
]


@pytest.mark.parametrize("case", STEP_CASES, ids=lambda c: c[0])
def test_tier_step_matches_oracle(case):
    """lsa_tier_step after every firing: the chunks behind its slot list equal
    the oracle's Level-2 top-k2 of the native score inside the kept set (or
    differ only inside the float32 band of the k2-th score), and its attention
    equals lsa_tier_attend over the same slots and the full-cache attention over
    the same chunks bit for bit, and the oracle's attention within tolerance."""
    import torch
    import paper_2606_09079_amd as L
    name, ctx, C, keep, slots, k2, nat_heads, dim = case
    prob = synth.Problem(f"tier_step_{name}", ctx, C, keep, 8, 2, idx_layers=1, idx_dim=dim, core_keep=list(k2),
                         nat_heads=nat_heads)
    log(f"[tier-step] {name} ctx={ctx} C={C} keep={keep} slots={slots} k2={k2} native={nat_heads}x{dim}")
    tc = TierCase(prob, 21, slots)
    host, dev = tc.dev["host"], tc.dev
    nat = L.Indexer(1, nat_heads, dim)
    rng = np.random.default_rng(8)
    F = 7
    per_seq = [_kept_sets(prob.n_chunks[b], keep[b], F, rng) for b in range(prob.batch)]
    state = [([-1] * slots[b], []) for b in range(prob.batch)]
    native = [oracle.index_score(host["nat_q"][b], host["nat_w"][b],
                                 host["nat_k"][prob.chunk_offsets[b]:prob.chunk_offsets[b + 1]])
              for b in range(prob.batch)]
    tol = [parity.index_score_tolerance(host["nat_q"][b], host["nat_w"][b],
                                        host["nat_k"][prob.chunk_offsets[b]:prob.chunk_offsets[b + 1]])
           for b in range(prob.batch)]
    shp = (prob.batch, 1, prob.n_q_heads, prob.head_dim)
    prev = None
    modes = set()
    for f in range(F):
        sets = [per_seq[b][f] for b in range(prob.batch)]
        kept, cnt, slot_idx, _ = _plan_and_check(tc, L, sets, prev, state)
        L.lsa_tier_fetch(tc.P, tc.T, tc.host_k, tc.host_v, tc.fetch, tc.fetch_count, tc.res_k, tc.res_v)
        sel = torch.full((prob.batch, tc.pitch), -5, dtype=torch.int32, device="cuda")
        sc = torch.full((prob.batch,), -5, dtype=torch.int32, device="cuda")
        out = torch.full(shp, float("nan"), dtype=torch.float32, device="cuda")
        lse = torch.full(shp[:3], float("nan"), dtype=torch.float32, device="cuda")
        L.lsa_tier_step(tc.P, tc.T, nat, k2, dev["nat_q"], dev["nat_w"], dev["nat_k"], kept, cnt, slot_idx,
                        dev["q"], tc.res_k, tc.res_v, 0.0, out, lse, sel, sc, tc.ws, tc.ws_bytes)
        torch.cuda.synchronize()
        g_sel, g_cnt, g_slot = sel.cpu().numpy(), sc.cpu().numpy(), slot_idx.cpu().numpy()
        chosen_all = np.full((prob.batch, tc.pitch), -1, dtype=np.int32)
        for b, s in enumerate(sets):
            c = int(g_cnt[b])
            assert c == min(len(s), k2[b]), f"firing {f} seq {b}: {c} slots selected"
            slot_to_chunk = {int(g_slot[b, i]): int(s[i]) for i in range(len(s))}
            chosen = np.array([slot_to_chunk[int(x)] for x in g_sel[b, :c]], dtype=np.int64)
            assert np.all(np.diff(chosen) > 0), f"firing {f} seq {b}: slots not in ascending chunk order"
            ref = oracle.two_level(np.asarray(s, dtype=np.int32), native[b], k2[b], prob.n_chunks[b],
                                   prob.n_chunks[b])
            if np.array_equal(chosen, ref):
                modes.add("exact")
            else:
                ns = np.sort(native[b][np.asarray(s, dtype=np.int64)])[::-1]
                kth = ns[k2[b] - 1]
                diff = sorted(set(chosen.tolist()) ^ set(ref.tolist()))
                assert all(abs(native[b][d] - kth) <= 2 * tol[b][d] for d in diff), \
                    f"firing {f} seq {b}: Level-2 set differs outside the band at {diff[:10]}"
                modes.add("band")
            chosen_all[b, :c] = chosen
        a_out, a_lse = _tier_attention(tc, L, sel, sc)
        d_out, d_lse = _direct_attention(tc, L, torch.from_numpy(chosen_all).cuda(), sc)
        torch.cuda.synchronize()
        assert torch.equal(out, a_out) and torch.equal(lse, a_lse), f"firing {f}: step != attend over its slots"
        assert torch.equal(out, d_out) and torch.equal(lse, d_lse), f"firing {f}: step != full-cache attention"
        o, s_ = out.cpu().numpy(), lse.cpu().numpy()
        for b in range(prob.batch):
            c = int(g_cnt[b])
            if c == 0:
                assert np.all(o[b] == 0.0) and np.all(np.isneginf(s_[b])), f"firing {f} seq {b}: empty set"
            elif f in (0, 2):
                rows = [(0, h) for h in range(0, prob.n_q_heads, 3)]
                _oracle_rows(tc, b, chosen_all[b, :c], o, s_, rows)
        prev = (slot_idx, cnt)
        log(f"[tier-step] firing {f}: kept {[len(s) for s in sets]} -> {g_cnt.tolist()}")
    log(f"[tier-step] {name}: Level-2 sets {sorted(modes)}")


def test_tier_step_graph_replay():
    """lsa_tier_step captured once and replayed after every firing with the new
    kept list and slots copied into its buffers; every replay equals the eager
    call."""
    import torch
    import paper_2606_09079_amd as L
    prob = synth.Problem("tier_step_graph", [64 * 800, 64 * 300], 64, [80, 40], 32, 8, idx_layers=1, idx_dim=128,
                         core_keep=[20, 12], nat_heads=64)
    slots = [160, 90]
    tc = TierCase(prob, 23, slots)
    dev = tc.dev
    nat = L.Indexer(1, 64, 128)
    k2 = [20, 12]
    rng = np.random.default_rng(6)
    per_seq = [_kept_sets(prob.n_chunks[b], prob.keep[b], 5, rng) for b in range(prob.batch)]
    state = [([-1] * slots[b], []) for b in range(prob.batch)]
    B, shp = prob.batch, (prob.batch, 1, prob.n_q_heads, prob.head_dim)
    kept_g = torch.zeros((B, tc.pitch), dtype=torch.int32, device="cuda")
    cnt_g = torch.zeros(B, dtype=torch.int32, device="cuda")
    slot_g = torch.zeros((B, tc.pitch), dtype=torch.int32, device="cuda")
    sel_g = torch.zeros((B, tc.pitch), dtype=torch.int32, device="cuda")
    sc_g = torch.zeros(B, dtype=torch.int32, device="cuda")
    out_g = torch.empty(shp, dtype=torch.float32, device="cuda")
    lse_g = torch.empty(shp[:3], dtype=torch.float32, device="cuda")

    def step(kept, cnt, slot_idx, sel, sc, out, lse):
        L.lsa_tier_step(tc.P, tc.T, nat, k2, dev["nat_q"], dev["nat_w"], dev["nat_k"], kept, cnt, slot_idx,
                        dev["q"], tc.res_k, tc.res_v, 0.0, out, lse, sel, sc, tc.ws, tc.ws_bytes)

    prev = None
    kept, cnt, slot_idx, _ = _plan_and_check(tc, L, [per_seq[b][0] for b in range(B)], prev, state)
    L.lsa_tier_fetch(tc.P, tc.T, tc.host_k, tc.host_v, tc.fetch, tc.fetch_count, tc.res_k, tc.res_v)
    for dst, src in ((kept_g, kept), (cnt_g, cnt), (slot_g, slot_idx)):
        dst.copy_(src)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step(kept_g, cnt_g, slot_g, sel_g, sc_g, out_g, lse_g)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(kept_g, cnt_g, slot_g, sel_g, sc_g, out_g, lse_g)
    torch.cuda.synchronize()
    prev = (slot_idx, cnt)
    for f in range(1, 5):
        kept, cnt, slot_idx, _ = _plan_and_check(tc, L, [per_seq[b][f] for b in range(B)], prev, state)
        L.lsa_tier_fetch(tc.P, tc.T, tc.host_k, tc.host_v, tc.fetch, tc.fetch_count, tc.res_k, tc.res_v)
        for dst, src in ((kept_g, kept), (cnt_g, cnt), (slot_g, slot_idx)):
            dst.copy_(src)
        sel_e = torch.full_like(sel_g, -3)
        sc_e = torch.full_like(sc_g, -3)
        out_e, lse_e = torch.empty_like(out_g), torch.empty_like(lse_g)
        step(kept, cnt, slot_idx, sel_e, sc_e, out_e, lse_e)
        torch.cuda.synchronize()
        for rep in range(2):
            out_g.fill_(float("nan"))
            sc_g.fill_(-1)
            g.replay()
            torch.cuda.synchronize()
            c = sc_e.cpu().numpy()
            assert torch.equal(sc_g, sc_e), f"firing {f} replay {rep}: counts differ"
            for b in range(B):
                assert torch.equal(sel_g[b, :int(c[b])], sel_e[b, :int(c[b])]), f"firing {f} replay {rep}: slots"
            assert torch.equal(out_g, out_e) and torch.equal(lse_g, lse_e), f"firing {f} replay {rep}: attention"
        prev = (slot_idx, cnt)
    log("[tier-step] graph replays match the eager calls")


def test_tier_step_ties_go_to_the_lower_chunk():
    """Native index keys repeated so that many resident chunks score exactly
    alike: the chunks Level 2 keeps at the cut are the lowest ids among the
    equal ones, as in the oracle (no band: equal keys give equal scores on both
    sides)."""
    import torch
    import paper_2606_09079_amd as L
    prob = synth.Problem("tier_step_ties", [64 * 600], 64, [100], 8, 2, idx_layers=1, idx_dim=128, core_keep=[37],
                         nat_heads=32)
    tc = TierCase(prob, 31, [200])
    host = tc.dev["host"]
    nat_k = host["nat_k"].copy()
    nat_k[:] = nat_k[np.arange(prob.total_chunks) % 5]  # five distinct keys
    nat_k_d = torch.from_numpy(nat_k.view(np.int16)).cuda()
    native = oracle.index_score(host["nat_q"][0], host["nat_w"][0], nat_k)
    assert len(np.unique(native)) <= 5
    rng = np.random.default_rng(12)
    kept_set = np.sort(rng.choice(prob.n_chunks[0], 100, replace=False))
    state = [([-1] * 200, [])]
    kept, cnt, slot_idx, _ = _plan_and_check(tc, L, [kept_set], None, state)
    L.lsa_tier_fetch(tc.P, tc.T, tc.host_k, tc.host_v, tc.fetch, tc.fetch_count, tc.res_k, tc.res_v)
    sel = torch.full((1, tc.pitch), -5, dtype=torch.int32, device="cuda")
    sc = torch.full((1,), -5, dtype=torch.int32, device="cuda")
    out = torch.empty((1, 1, prob.n_q_heads, prob.head_dim), dtype=torch.float32, device="cuda")
    for k2 in (1, 37, 99, 100, 150):
        L.lsa_tier_step(tc.P, tc.T, L.Indexer(1, 32, 128), [k2], tc.dev["nat_q"], tc.dev["nat_w"], nat_k_d, kept, cnt,
                        slot_idx, tc.dev["q"], tc.res_k, tc.res_v, 0.0, out, None, sel, sc, tc.ws, tc.ws_bytes)
        torch.cuda.synchronize()
        c = int(sc.cpu()[0])
        g_slot, g_sel = slot_idx.cpu().numpy()[0], sel.cpu().numpy()[0, :c]
        slot_to_chunk = {int(g_slot[i]): int(kept_set[i]) for i in range(len(kept_set))}
        chosen = np.array([slot_to_chunk[int(x)] for x in g_sel], dtype=np.int64)
        ref = oracle.two_level(kept_set.astype(np.int32), native, k2, prob.n_chunks[0], prob.n_chunks[0])
        assert np.array_equal(chosen, ref), f"k2 = {k2}: chunks {chosen[:8]} vs oracle {ref[:8]}"
    log("[tier-step] ties resolved to the lower chunk ids")


def test_tier_full_size_1m():
    """The host tier at its benchmark size (1,048,576 tokens, K_max 1,638,
    reserve 3,276 slots, Level 2 keeping 1,024 with 64 native heads), in the
    launch configuration the benchmark times: two firings of the GPU recall,
    each planned (equal to the oracle's plan), copied by the copy kernel and
    attended over the reserve (bitwise equal to the full-cache attention), and
    lsa_tier_step over the second firing's resident set (the oracle's Level-2
    set up to the float32 band, every query head against the oracle's
    attention); every kept chunk's reserve blocks equal the mirror's."""
    import dataclasses
    import math
    import torch
    import paper_2606_09079_amd as L
    prob = dataclasses.replace(synth.make_problem("recall1m", 0), name="tier_full_1m", core_keep=[1024],
                               nat_heads=64)
    K = prob.keep[0]
    slots = [2 * K]
    log(f"[tier-1m] ctx={prob.ctx_tokens} K_max={K} slots={slots} k2=1024")
    tc = TierCase(prob, 0, slots)
    host, dev = tc.dev["host"], tc.dev
    P, ix = tc.P, L.Indexer.from_synth(prob)
    scores = torch.empty(prob.idx_layers * prob.total_chunks, dtype=torch.float32, device="cuda")
    kept = [torch.full((1, tc.pitch), -1, dtype=torch.int32, device="cuda") for _ in range(2)]
    cnt = [torch.zeros(1, dtype=torch.int32, device="cuda") for _ in range(2)]
    slot_idx = [torch.full((1, tc.pitch), -1, dtype=torch.int32, device="cuda") for _ in range(2)]
    # firing 1 uses drifted indexer queries, as the benchmark's firings do
    rng = np.random.default_rng(77)
    qf = synth.bf16_bits_to_f64(host["idx_q"])
    q1 = synth.f64_to_bf16_bits(math.sqrt(0.99) * qf + math.sqrt(0.01) * rng.standard_normal(qf.shape))
    idx_qs = [dev["idx_q"], torch.from_numpy(q1.view(np.int16)).cuda()]
    state_owner, state_slots = [-1] * slots[0], []
    sets = []
    for f in range(2):
        L.lsa_recall_scores(P, ix, idx_qs[f], dev["idx_w"], dev["idx_k"], scores)
        L.lsa_recall_select(P, ix, scores, kept[f], cnt[f])
        prev = (slot_idx[f - 1], cnt[f - 1]) if f else (None, None)
        L.lsa_tier_plan(P, tc.T, kept[f], cnt[f], prev[0], prev[1], tc.owner, slot_idx[f], tc.fetch, tc.fetch_count)
        L.lsa_tier_fetch(P, tc.T, tc.host_k, tc.host_v, tc.fetch, tc.fetch_count, tc.res_k, tc.res_v)
        torch.cuda.synchronize()
        c = int(cnt[f].cpu()[0])
        s_f = kept[f].cpu().numpy()[0, :c].astype(np.int64)
        sets.append(s_f)
        new_owner, new_slots, fetch = oracle.tier_plan(state_owner, state_slots, s_f.tolist())
        assert tc.owner.cpu().numpy().tolist() == new_owner, f"firing {f}: owner table differs from the oracle"
        assert slot_idx[f].cpu().numpy()[0, :c].tolist() == new_slots, f"firing {f}: slots differ from the oracle"
        assert int(tc.fetch_count.cpu()[0]) == len(fetch), f"firing {f}: copy count differs from the oracle"
        state_owner, state_slots = new_owner, new_slots
        for which, res in (("k", tc.res_k), ("v", tc.res_v)):
            got = tc.blocks(res, np.asarray(new_slots))
            want = tc.blocks(tc.dev[which], s_f)
            assert bool((got == want).all()), f"firing {f}: reserve {which} blocks differ from the mirror"
        t_out, t_lse = _tier_attention(tc, L, slot_idx[f], cnt[f])
        d_out, d_lse = _direct_attention(tc, L, kept[f], cnt[f])
        torch.cuda.synchronize()
        assert torch.equal(t_out, d_out) and torch.equal(t_lse, d_lse), f"firing {f}: reserve != full-cache attention"
        log(f"[tier-1m] firing {f}: kept {c}, copies {len(fetch)}; plan, reserve and attention match")
    # Level 2 over the resident set of firing 1
    s1 = sets[1]
    sel = torch.full((1, tc.pitch), -5, dtype=torch.int32, device="cuda")
    sc = torch.full((1,), -5, dtype=torch.int32, device="cuda")
    shp = (1, 1, prob.n_q_heads, prob.head_dim)
    out = torch.empty(shp, dtype=torch.float32, device="cuda")
    lse = torch.empty(shp[:3], dtype=torch.float32, device="cuda")
    L.lsa_tier_step(P, tc.T, L.Indexer(1, 64, prob.idx_dim), [1024], dev["nat_q"], dev["nat_w"], dev["nat_k"],
                    kept[1], cnt[1], slot_idx[1], dev["q"], tc.res_k, tc.res_v, 0.0, out, lse, sel, sc, tc.ws,
                    tc.ws_bytes)
    torch.cuda.synchronize()
    c = int(sc.cpu()[0])
    assert c == min(len(s1), 1024)
    slot_to_chunk = dict(zip(state_slots, s1.tolist()))
    chosen = np.array([slot_to_chunk[int(x)] for x in sel.cpu().numpy()[0, :c]], dtype=np.int64)
    assert np.all(np.diff(chosen) > 0), "chosen chunks not ascending"
    native = oracle.index_score(host["nat_q"][0], host["nat_w"][0], host["nat_k"])
    ref = oracle.two_level(s1.astype(np.int32), native, 1024, prob.n_chunks[0], prob.n_chunks[0])
    if not np.array_equal(chosen, ref):
        tol = parity.index_score_tolerance(host["nat_q"][0], host["nat_w"][0], host["nat_k"])
        kth = np.sort(native[s1])[::-1][1023]
        diff = sorted(set(chosen.tolist()) ^ set(ref.tolist()))
        assert all(abs(native[d] - kth) <= 2 * tol[d] for d in diff), f"Level-2 set differs outside the band {diff[:8]}"
    chosen_t = torch.full((1, tc.pitch), -1, dtype=torch.int32, device="cuda")
    chosen_t[0, :c] = torch.from_numpy(chosen.astype(np.int32)).cuda()
    d_out, d_lse = _direct_attention(tc, L, chosen_t, sc)
    torch.cuda.synchronize()
    assert torch.equal(out, d_out) and torch.equal(lse, d_lse), "tier step != full-cache attention over its chunks"
    _oracle_rows(tc, 0, chosen, out.cpu().numpy(), lse.cpu().numpy(), [(0, h) for h in range(prob.n_q_heads)])
    log(f"[tier-1m] Level 2 kept {c} of {len(s1)}; attention matches the full cache and the oracle")
