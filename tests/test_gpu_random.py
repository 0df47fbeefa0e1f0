"""Seeded random shapes through the C ABI, against the CPU oracle.

Every case draws its shape from a fixed seed, so a run is reproducible: batch,
chunk size, KV heads and GQA group, query tokens, lookahead queries, embedding
dtype and width, context lengths and keep budgets.  The fused-step cases run
the whole path (each entry point, then lsa_decode_step) as the other parity
tests do.  The attention cases give lsa_sparse_decode_attn contexts that end
anywhere inside a chunk and random ascending kept lists, with and without the
partial last chunk, and compare every query row of two KV heads per sequence
token by token.
"""
import numpy as np
import pytest

import lsa_synth as synth
from gpu_case import log, run_case

pytestmark = pytest.mark.gpu

N_FUSED = 24
N_ATTN = 16


def _heads(rng):
    """(Hq, Hkv, Tq) with G * Tq <= 128 rows per KV head."""
    hkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.choice([1, 2, 4, 8]))
    tq = int(rng.choice([t for t in (1, 2, 4, 8, 16) if g * t <= 128]))
    return g * hkv, hkv, tq


def fused_problem(i: int) -> synth.Problem:
    rng = np.random.default_rng(7100 + i)
    B = int(rng.integers(1, 9))
    C = int(rng.choice([64, 128]))
    hq, hkv, tq = _heads(rng)
    Q = int(rng.choice([1, 1, 2, 4]))
    dtype = str(rng.choice(["f32", "bf16", "i8"]))
    D = int(rng.choice([64, 128, 256, 512]))
    n = [int(x) for x in rng.integers(1, 300, size=B)]
    keep = [int(rng.integers(1, nb + 1)) for nb in n]
    return synth.Problem(f"rand_fused_{i}", [nb * C for nb in n], C, keep, hq, hkv, emb_dim=D, emb_dtype=dtype,
                         n_lookahead=Q, n_qtok=tq)


@pytest.mark.parametrize("i", range(N_FUSED))
def test_random_fused_step(i):
    prob = fused_problem(i)
    r = run_case(prob, seed=300 + i)
    assert r["worst_attn"] <= 2e-3


@pytest.mark.parametrize("i", range(N_ATTN))
def test_random_partial_attention(i):
    import torch
    import oracle
    import parity
    import paper_2606_09079_amd as L
    rng = np.random.default_rng(9100 + i)
    B = int(rng.integers(1, 5))
    C = int(rng.choice([64, 128]))
    hq, hkv, tq = _heads(rng)
    G = hq // hkv
    ctx = [int(rng.integers(1, 200 * C)) for _ in range(B)]
    prob = synth.Problem(f"rand_attn_{i}", ctx, C, [1] * B, hq, hkv, n_qtok=tq)
    host = synth.host_inputs(prob, 500 + i)
    dev = synth.device_inputs(prob, 500 + i, host=host)
    kept = []
    for nb in prob.n_chunks:
        m = int(rng.integers(1, min(nb, 96) + 1))
        ids = np.sort(rng.choice(nb, size=m, replace=False)).astype(np.int32)
        if rng.random() < 0.7 and ids[-1] != nb - 1:
            ids[-1] = nb - 1  # the partial last chunk kept
        kept.append(np.unique(ids).astype(np.int32))
    ks = [len(k) for k in kept]
    P = L.Problem(ctx, C, ks, hq, hkv, n_qtok=tq)
    ws_bytes = L.lsa_workspace_size(L.Problem([C * nb for nb in prob.n_chunks], C, ks, hq, hkv, n_qtok=tq))
    ws = torch.zeros(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    sel_h = np.full((B, max(ks)), -1, dtype=np.int32)
    for b, k in enumerate(kept):
        sel_h[b, :len(k)] = k
    sel = torch.from_numpy(sel_h).cuda()
    cnt = torch.tensor(ks, dtype=torch.int32, device="cuda")
    out = torch.full((B, tq, hq, 128), float("nan"), device="cuda")
    lse = torch.full((B, tq, hq), float("nan"), device="cuda")
    log(f"[rand attn {i}] B={B} C={C} Hq={hq} Hkv={hkv} Tq={tq} ctx={ctx} kept={ks}")
    L.lsa_sparse_decode_attn(P, dev["q"], dev["k"], dev["v"], sel, cnt, 0.0, out, lse, ws, ws_bytes)
    torch.cuda.synchronize()
    g_out, g_lse = out.cpu().numpy(), lse.cpu().numpy()
    for b in range(B):
        toks = oracle.kept_tokens(kept[b], C, ctx[b])
        for g in sorted({0, hkv - 1}):
            Kh = synth.kv_head_sparse(prob, 500 + i, "k", b, g, kept[b])
            Vh = synth.kv_head_sparse(prob, 500 + i, "v", b, g, kept[b])
            rows = [(t, g * G + j) for t in range(tq) for j in range(G)]
            qr = np.stack([host["q"][b, t, h] for (t, h) in rows])
            r_out, r_lse = oracle.attention_tokens(qr, Kh, Vh, toks)
            parity.check_attention(np.stack([g_out[b, t, h] for (t, h) in rows]),
                                   [g_lse[b, t, h] for (t, h) in rows], r_out, r_lse,
                                   f"rand attn {i}: sequence {b} (ctx {ctx[b]}, {ks[b]} kept), KV head {g}")
