"""One parity run of the HIP path against the oracle on a seeded problem.

Everything goes through the C ABI (``paper_2606_09079_amd``): score, top-k and
attention called one by one, then the fused step.  The oracle sees only the
generator's host bytes; the only thing taken from the GPU side is the output
under test.  Where the oracle's k-th and (k+1)-th scores sit inside the 1e-4
band, the GPU's kept set is first checked to be one of the valid answers; the
attention of the fused step is then compared with the oracle's attention over
that same valid set (several results are correct there).
"""
from __future__ import annotations

import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

import lsa_synth as synth
import oracle
import parity


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def _rows_all(prob) -> List[Tuple[int, int]]:
    return [(t, h) for t in range(prob.n_qtok) for h in range(prob.n_q_heads)]


# The oracle runs one (sequence, KV head) per thread; its C calls release the
# interpreter lock.  At most 16 threads, so that the oracle never oversubscribes the host.
WORKERS = max(1, min(16, os.cpu_count() or 1))


def oracle_rows(prob, host, seed: int, kept: Dict[int, np.ndarray], seqs: Sequence[int],
                rows: Sequence[Tuple[int, int]]) -> Dict[int, Dict]:
    """Oracle attention {b: {(t, h): (out, lse)}} of the given rows of each
    sequence over its kept chunks, one task per (sequence, KV head)."""
    synth.host_lib()
    oracle.lib()
    G = prob.group
    tasks = []
    for b in seqs:
        by_g: Dict[int, List] = {}
        for (t, h) in rows:
            by_g.setdefault(h // G, []).append((t, h))
        tasks += [(b, rs) for _, rs in sorted(by_g.items())]

    def run(task):
        b, rs = task
        kv = lambda which, bb, g, ch: synth.kv_head_sparse(prob, seed, which, bb, g, ch)
        return b, oracle.attend_rows(prob, host, b, kept[b], rs, kv)

    res: Dict[int, Dict] = {b: {} for b in seqs}
    with ThreadPoolExecutor(WORKERS) as ex:
        for b, r in ex.map(run, tasks):
            res[b].update(r)
    return res


def run_case(prob, seed: int, seqs: Optional[Sequence[int]] = None,
             rows: Optional[Sequence[Tuple[int, int]]] = None, fused: bool = True) -> Dict[str, object]:
    import torch
    import paper_2606_09079_amd as L

    log(f"[case] {prob.name} seed={seed} B={prob.batch} ctx={prob.ctx_tokens[:4]} C={prob.chunk} "
        f"keep={prob.keep[:4]} Hq={prob.n_q_heads} Hkv={prob.n_kv_heads} Q={prob.n_lookahead} Tq={prob.n_qtok} "
        f"D={prob.emb_dim} {prob.emb_dtype}")
    t0 = time.time()
    host = synth.host_inputs(prob, seed)
    dev = synth.device_inputs(prob, seed, host=host)
    P = L.Problem.from_synth(prob)
    B, Q, i8 = prob.batch, prob.n_lookahead, prob.emb_dtype == "i8"
    ws_bytes = L.lsa_workspace_size(P)
    ws = torch.zeros(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    offs = prob.chunk_offsets
    max_sel, max_keep = L.lsa_max_sel(P), L.lsa_max_keep(P)

    scores = torch.empty(Q * prob.total_chunks, dtype=torch.int32 if i8 else torch.float32, device="cuda")
    L.lsa_score_chunks(P, dev["qe"], dev["E"], scores)
    sel = torch.full((B, max_sel), -1, dtype=torch.int32, device="cuda")
    cnt = torch.zeros(B, dtype=torch.int32, device="cuda")
    pq = torch.full((B, Q, max_keep), -1, dtype=torch.int32, device="cuda") if Q > 1 else None
    L.lsa_topk_chunks(P, scores, sel, cnt, pq, ws, ws_bytes)
    torch.cuda.synchronize()
    g_scores, g_sel, g_cnt = scores.cpu().numpy(), sel.cpu().numpy(), cnt.cpu().numpy()
    g_pq = pq.cpu().numpy() if pq is not None else None
    log(f"[case] gpu score+topk done ({time.time() - t0:.1f}s)")

    seqs = list(range(B)) if seqs is None else list(seqs)
    ref_kept: Dict[int, np.ndarray] = {}
    modes: Dict[int, str] = {}
    worst_score = 0.0
    for b in range(B):
        r_scores, r_lists, r_kept = oracle.select_for_sequence(prob, host, b)
        n, k = prob.n_chunks[b], prob.keep[b]
        blk = g_scores[Q * offs[b]: Q * offs[b] + Q * n].reshape(Q, n)
        for j in range(Q):
            worst_score = max(worst_score, parity.check_scores(
                blk[j], r_scores[j], host["qe"][b, j], host["E"][offs[b]:offs[b + 1]], prob.emb_dtype,
                f"{prob.name} seq {b} query {j}"))
        if Q == 1:
            assert g_cnt[b] == k, f"seq {b}: sel_count {g_cnt[b]} != {k}"
            modes[b] = parity.check_kept(g_sel[b, :k], r_scores[0], k, i8, f"{prob.name} seq {b}")
        else:
            per = []
            for j in range(Q):
                per.append(parity.check_kept(g_pq[b, j, :k], r_scores[j], k, i8, f"{prob.name} seq {b} q {j}"))
            gu = sorted(set(g_pq[b, :, :k].reshape(-1).tolist()))
            assert g_cnt[b] == len(gu), f"seq {b}: union count {g_cnt[b]} != {len(gu)}"
            assert g_sel[b, :g_cnt[b]].tolist() == gu, f"seq {b}: union of the GPU per-query sets differs"
            modes[b] = "exact" if all(m == "exact" for m in per) else "band"
            if modes[b] == "exact":
                assert np.array_equal(g_sel[b, :g_cnt[b]], r_kept), f"seq {b}: union differs from the oracle"
        ref_kept[b] = r_kept
    log(f"[case] scores/top-k parity ok (worst score err {worst_score:.2e}, modes {sorted(set(modes.values()))}) "
        f"({time.time() - t0:.1f}s)")

    # Attention alone, fed the oracle's kept sets.
    sel_in = torch.zeros((B, max_sel), dtype=torch.int32)
    cnt_in = torch.zeros(B, dtype=torch.int32)
    for b in range(B):
        sel_in[b, :len(ref_kept[b])] = torch.from_numpy(ref_kept[b])
        cnt_in[b] = len(ref_kept[b])
    sel_in, cnt_in = sel_in.cuda(), cnt_in.cuda()
    shp = (B, prob.n_qtok, prob.n_q_heads, prob.head_dim)
    out = torch.full(shp, float("nan"), dtype=torch.float32, device="cuda")
    lse = torch.full(shp[:3], float("nan"), dtype=torch.float32, device="cuda")
    L.lsa_sparse_decode_attn(P, dev["q"], dev["k"], dev["v"], sel_in, cnt_in, 0.0, out, lse, ws, ws_bytes)
    torch.cuda.synchronize()
    g_out, g_lse = out.cpu().numpy(), lse.cpu().numpy()

    rows = _rows_all(prob) if rows is None else list(rows)
    worst_attn = 0.0
    ref_attn = oracle_rows(prob, host, seed, ref_kept, seqs, rows)
    log(f"[case] oracle attention of {len(rows)} rows x {len(seqs)} sequences ({time.time() - t0:.1f}s)")
    for b in seqs:
        res = ref_attn[b]
        keys = list(res.keys())
        worst_attn = max(worst_attn, parity.check_attention(
            np.stack([g_out[b, t, h] for (t, h) in keys]), [g_lse[b, t, h] for (t, h) in keys],
            np.stack([res[k_][0] for k_ in keys]), [res[k_][1] for k_ in keys], f"{prob.name} attn seq {b}"))
    log(f"[case] attention parity ok (worst rel err {worst_attn:.2e}) ({time.time() - t0:.1f}s)")

    worst_fused = 0.0
    if fused:
        out2 = torch.full(shp, float("nan"), dtype=torch.float32, device="cuda")
        lse2 = torch.full(shp[:3], float("nan"), dtype=torch.float32, device="cuda")
        sel2 = torch.full((B, max_sel), -1, dtype=torch.int32, device="cuda")
        cnt2 = torch.zeros(B, dtype=torch.int32, device="cuda")
        L.lsa_decode_step(P, dev["qe"], dev["E"], dev["q"], dev["k"], dev["v"], 0.0, out2, lse2, sel2, cnt2, ws,
                          ws_bytes)
        torch.cuda.synchronize()
        f_out, f_lse, f_sel, f_cnt = out2.cpu().numpy(), lse2.cpu().numpy(), sel2.cpu().numpy(), cnt2.cpu().numpy()
        assert np.array_equal(f_cnt, g_cnt), "fused step kept counts differ from lsa_topk_chunks"
        for b in range(B):
            assert np.array_equal(f_sel[b, :f_cnt[b]], g_sel[b, :g_cnt[b]]), f"fused kept set differs, seq {b}"
        band = [b for b in seqs if modes[b] != "exact" and not np.array_equal(f_sel[b, :f_cnt[b]], ref_kept[b])]
        # kept sets in the band were verified above to be valid ones
        band_attn = oracle_rows(prob, host, seed, {b: f_sel[b, :f_cnt[b]].astype(np.int64) for b in band}, band,
                                rows) if band else {}
        for b in seqs:
            kept = f_sel[b, :f_cnt[b]].astype(np.int64)
            if modes[b] == "exact":
                assert np.array_equal(kept, ref_kept[b])
            if np.array_equal(kept, ref_kept[b]):
                # same kept set as the attention call above: the fused step merges its splits in
                # the attention kernel, in the combine's order, so the bits are the same
                assert np.array_equal(f_out[b].view(np.uint32), g_out[b].view(np.uint32)), \
                    f"{prob.name} seq {b}: fused output differs from lsa_sparse_decode_attn"
                assert np.array_equal(f_lse[b].view(np.uint32), g_lse[b].view(np.uint32)), \
                    f"{prob.name} seq {b}: fused lse differs from lsa_sparse_decode_attn"
            res = band_attn[b] if b in band_attn else ref_attn[b]
            keys = list(res.keys())
            worst_fused = max(worst_fused, parity.check_attention(
                np.stack([f_out[b, t, h] for (t, h) in keys]), [f_lse[b, t, h] for (t, h) in keys],
                np.stack([res[k_][0] for k_ in keys]), [res[k_][1] for k_ in keys], f"{prob.name} fused seq {b}"))
        log(f"[case] fused step parity ok (worst rel err {worst_fused:.2e}) ({time.time() - t0:.1f}s)")
    return {"modes": modes, "worst_score": worst_score, "worst_attn": worst_attn, "worst_fused": worst_fused,
            "sel": g_sel, "cnt": g_cnt}
