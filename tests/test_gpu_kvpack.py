"""lsa_kv_pack: token-major K/V rows re-laid into the chunk-paged blocks the
attention reads.  The result must equal, bit for bit, the paged fill of the
same seeded values; positions outside the written range keep their bytes,
and the slots past the context end of a partial last chunk become zero.
Also: the attention ignores whatever bits (NaN included) those slots hold."""
import numpy as np
import pytest

import lsa_synth as synth

pytestmark = pytest.mark.gpu

SENTINEL = 0x7FC1  # a NaN bit pattern that no packed position may keep


def _layout_positions(prob, b, lo, hi, which, chunk_stride, head_stride):
    """Flat cache offsets of tokens [lo, hi) of sequence b, every KV head and dim."""
    if hi <= lo:
        return np.zeros(0, dtype=np.int64)
    C, d = prob.chunk, prob.head_dim
    tok = np.arange(lo, hi, dtype=np.int64)
    c = prob.chunk_offsets[b] + tok // C
    e = np.arange(d, dtype=np.int64)
    inner = synth.block_offset(which, (tok % C)[:, None], e[None, :])  # [tokens][d]
    g = np.arange(prob.n_kv_heads, dtype=np.int64)
    pos = (c[:, None, None] * chunk_stride + g[None, :, None] * head_stride + inner[:, None, :])
    return pos.reshape(-1)


def _setup(prob, seed, row_gap, tok_pad, head_pad):
    import torch
    H, d = prob.n_kv_heads, prob.head_dim
    hs = d + head_pad
    ts = H * hs + tok_pad
    row_off, r = [], 0
    for Lb in prob.ctx_tokens:
        r += row_gap
        row_off.append(r)
        r += Lb
    n_rows = r + row_gap
    table = torch.from_numpy(synth.normal_table_bf16().view(np.int16)).cuda()
    tau = torch.from_numpy(synth.token_rows(prob, row_off, n_rows)).cuda()
    src = {}
    for w in "kv":
        src[w] = torch.zeros(n_rows * ts, dtype=torch.int16, device="cuda")
        synth.fill_kv_tokens_device(prob, seed, w, src[w].data_ptr(), table.data_ptr(), tau.data_ptr(), n_rows,
                                    tok_stride=ts, head_stride=hs)
    offs = torch.tensor(row_off, dtype=torch.int64, device="cuda")
    return table, src, offs, ts, hs, row_off


def _expected(prob, seed, table, cs, hs_dst, n_elems):
    import torch
    out = {}
    for w in "kv":
        t = torch.full((n_elems,), SENTINEL, dtype=torch.int16, device="cuda")
        synth.fill_kv_device(prob, seed, w, t.data_ptr(), table.data_ptr(), 0, chunk_stride=cs, head_stride=hs_dst)
        out[w] = t.cpu().numpy().view(np.uint16)
    return out


CASES = [
    # name, chunk, contexts, Hkv, destination padding (chunk, head), source padding (row gap, token, head)
    ("c64_ragged", 64, [200, 64, 1005], 8, (0, 0), (0, 0, 0)),
    ("c64_padded", 64, [77, 130, 64 * 9], 2, (64, 16), (3, 24, 8)),
    ("c128_ragged", 128, [300, 129, 128, 5], 4, (0, 0), (1, 8, 0)),
    ("c128_one_token", 128, [1], 8, (0, 0), (0, 0, 0)),
]


@pytest.mark.parametrize("name,C,ctx,H,dpad,spad", CASES, ids=[c[0] for c in CASES])
def test_pack_whole_context_equals_paged_fill(name, C, ctx, H, dpad, spad):
    import torch
    import paper_2606_09079_amd as L
    prob = synth.Problem(name, ctx, C, [1] * len(ctx), 2 * H, H)
    seed = 21
    hs_dst = C * 128 + dpad[1]
    cs = H * hs_dst + dpad[0]
    P = L.Problem(ctx, C, [1] * len(ctx), 2 * H, H, kv_chunk_stride=cs, kv_head_stride=hs_dst)
    table, src, offs, ts, hs, _ = _setup(prob, seed, *spad)
    n_elems = prob.total_chunks * cs
    dst = {w: torch.full((n_elems,), SENTINEL, dtype=torch.int16, device="cuda") for w in "kv"}
    L.lsa_kv_pack(P, src["k"], src["v"], offs, dst["k"], dst["v"], tok_stride=ts, tok_head_stride=hs)
    torch.cuda.synchronize()
    exp = _expected(prob, seed, table, cs, hs_dst, n_elems)
    for w in "kv":
        got = dst[w].cpu().numpy().view(np.uint16)
        written = np.zeros(n_elems, dtype=bool)
        for b, Lb in enumerate(ctx):
            pos = _layout_positions(prob, b, 0, Lb, w, cs, hs_dst)
            assert np.array_equal(got[pos], exp[w][pos]), f"{name} {w}: sequence {b} differs"
            written[pos] = True
            tail = _layout_positions(prob, b, Lb, prob.n_chunks[b] * C, w, cs, hs_dst)
            assert np.all(got[tail] == 0), f"{name} {w}: sequence {b}: slots past the end are not zero"
            written[tail] = True
        assert np.all(got[~written] == SENTINEL), f"{name} {w}: a position outside every block changed"


@pytest.mark.parametrize("C,ctx,back", [(64, [200, 64 * 3 + 10, 1005], [5, 0, 40]),
                                        (128, [300, 129, 256], [43, 0, 127])])
def test_pack_in_steps_equals_one_pack(C, ctx, back):
    """Prefill up to ctx - back, then append the last `back` tokens from a
    buffer that holds only the new rows (token offsets below zero), then one
    more call with nothing to write: the caches equal a single whole pack."""
    import torch
    import paper_2606_09079_amd as L
    H = 4
    prob = synth.Problem("steps", ctx, C, [1] * len(ctx), 8, H)
    seed = 5
    table, src, offs, ts, hs, row_off = _setup(prob, seed, 0, 0, 0)
    n_elems = prob.kv_elems()
    one = {w: torch.full((n_elems,), SENTINEL, dtype=torch.int16, device="cuda") for w in "kv"}
    P = L.Problem(ctx, C, [1] * len(ctx), 8, H)
    L.lsa_kv_pack(P, src["k"], src["v"], offs, one["k"], one["v"])
    steps = {w: torch.full((n_elems,), SENTINEL, dtype=torch.int16, device="cuda") for w in "kv"}
    pre = [Lb - r for Lb, r in zip(ctx, back)]
    assert all((p + C - 1) // C == (Lb + C - 1) // C for p, Lb in zip(pre, ctx)), "chunk counts must not change"
    P_pre = L.Problem(pre, C, [1] * len(ctx), 8, H)
    L.lsa_kv_pack(P_pre, src["k"], src["v"], offs, steps["k"], steps["v"])
    # the new rows only, back to back
    new = {}
    rows = np.concatenate([np.arange(row_off[b] + pre[b], row_off[b] + ctx[b]) for b in range(len(ctx))])
    rows_t = torch.from_numpy(rows).cuda()
    for w in "kv":
        new[w] = src[w].view(-1, ts)[rows_t].reshape(-1).contiguous()
    first_row = np.concatenate([[0], np.cumsum(back)[:-1]])
    new_offs = torch.tensor([int(first_row[b]) - pre[b] for b in range(len(ctx))], dtype=torch.int64,
                            device="cuda")
    L.lsa_kv_pack(P, new["k"], new["v"], new_offs, steps["k"], steps["v"], first_token=pre)
    L.lsa_kv_pack(P, new["k"], new["v"], new_offs, steps["k"], steps["v"], first_token=ctx)
    torch.cuda.synchronize()
    for w in "kv":
        assert torch.equal(one[w], steps[w]), f"{w}: prefill + append differs from one pack"


@pytest.mark.parametrize("preset", ["paper1m", "int8"])
def test_pack_full_size(preset):
    """The whole paper-scale context (and the 4-sequence int8 batch) packed from
    token-major rows equals the paged fill, on the device."""
    import torch
    import paper_2606_09079_amd as L
    prob = synth.make_problem(preset, 0)
    P = L.Problem.from_synth(prob)
    H, d = prob.n_kv_heads, prob.head_dim
    n_rows = sum(prob.ctx_tokens)
    row_off = np.concatenate([[0], np.cumsum(prob.ctx_tokens)[:-1]]).tolist()
    table = torch.from_numpy(synth.normal_table_bf16().view(np.int16)).cuda()
    tau = torch.from_numpy(synth.token_rows(prob, row_off, n_rows)).cuda()
    offs = torch.tensor(row_off, dtype=torch.int64, device="cuda")
    n = prob.kv_elems()
    for w in "kv":
        src = torch.empty(n_rows * H * d, dtype=torch.int16, device="cuda")
        synth.fill_kv_tokens_device(prob, 0, w, src.data_ptr(), table.data_ptr(), tau.data_ptr(), n_rows)
        dst = torch.empty(n, dtype=torch.int16, device="cuda")
        # the same rows for K and V: only the `w` cache is checked
        other = torch.empty(n, dtype=torch.int16, device="cuda")
        if w == "k":
            L.lsa_kv_pack(P, src, src, offs, dst, other)
        else:
            L.lsa_kv_pack(P, src, src, offs, other, dst)
        ref = torch.empty(n, dtype=torch.int16, device="cuda")
        synth.fill_kv_device(prob, 0, w, ref.data_ptr(), table.data_ptr(), 0)
        torch.cuda.synchronize()
        assert torch.equal(dst, ref), f"{preset}: packed {w.upper()} differs from the paged fill"
        del src, dst, other, ref


def poison_tail_slots(prob, k, v, value=0x7FC0):
    """Write `value` (a NaN by default) into the K and V slots past the context
    end of every sequence's partial last chunk (default strides)."""
    import torch
    C = prob.chunk
    cs, hs = prob.n_kv_heads * C * prob.head_dim, C * prob.head_dim
    for w, t in (("k", k), ("v", v)):
        pos = [_layout_positions(prob, b, Lb, prob.n_chunks[b] * C, w, cs, hs) for b, Lb in enumerate(prob.ctx_tokens)]
        pos = np.concatenate(pos)
        if len(pos):
            t[torch.from_numpy(pos).cuda()] = value - 65536 if value >= 32768 else value


@pytest.mark.parametrize("C,tail,Hq,Hkv,Tq", [(64, 1, 8, 2, 1), (64, 37, 32, 8, 1), (128, 100, 16, 4, 4),
                                              (64, 33, 64, 8, 16), (128, 1, 64, 8, 16)])
def test_attention_ignores_nan_in_slots_past_the_end(C, tail, Hq, Hkv, Tq):
    """Slots past the context end may hold any bits: NaN there leaves the
    output bit for bit as with finite values (split kernel at <= 16 rows per
    KV head, many-rows kernel above)."""
    import torch
    import paper_2606_09079_amd as L
    prob = synth.Problem("nan_tail", [C * 30 + tail], C, [8], Hq, Hkv, n_qtok=Tq)
    dev = synth.device_inputs(prob, 3)
    n = prob.n_chunks[0]
    kept = np.array([0, 4, 9, n - 2, n - 1], dtype=np.int32)
    P = L.Problem(prob.ctx_tokens, C, [len(kept)], Hq, Hkv, n_qtok=Tq)
    ws_bytes = L.lsa_workspace_size(L.Problem([C * n], C, [len(kept)], Hq, Hkv, n_qtok=Tq))
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    sel = torch.from_numpy(kept[None, :].copy()).cuda()
    cnt = torch.tensor([len(kept)], dtype=torch.int32, device="cuda")
    outs = []
    for poison in (False, True):
        if poison:
            poison_tail_slots(prob, dev["k"], dev["v"])
        out = torch.empty(1, Tq, Hq, 128, device="cuda")
        lse = torch.empty(1, Tq, Hq, device="cuda")
        L.lsa_sparse_decode_attn(P, dev["q"], dev["k"], dev["v"], sel, cnt, 0.0, out, lse, ws, ws_bytes)
        torch.cuda.synchronize()
        outs.append((out.cpu(), lse.cpu()))
    assert torch.isfinite(outs[1][0]).all() and torch.isfinite(outs[1][1]).all()
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
