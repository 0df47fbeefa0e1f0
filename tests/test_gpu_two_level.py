"""Parity of the two-level path (Level-1 recall over the history, Level-2
native top-k inside the recalled set, always-resident window, partial last
chunk, attention) with the CPU oracle, on the GPU, through the C ABI."""
import numpy as np
import pytest

import lsa_synth as synth
from gpu_case import log
from two_level_case import run_two_level_case

pytestmark = pytest.mark.gpu


def T(name, ctx, kmax, k2, window, hq=8, hkv=2, layers=2, heads=32, native=32, dim=128, rate=0.1, Tq=1, chunk=64):
    return synth.Problem(name, list(ctx), chunk, list(kmax), hq, hkv, n_qtok=Tq, idx_layers=layers, idx_heads=heads,
                         idx_dim=dim, idx_rate=rate, core_keep=list(k2), nat_heads=native, window_tokens=list(window))


SMALL = [
    T("partial_tail", [64 * 100 + 13], [30], [8], [640]),
    T("tail_one_token", [64 * 80 + 1], [20], [5], [100], layers=3, heads=16, native=16, dim=64),
    T("no_window_full_chunks", [64 * 120], [25], [7], [0], layers=1, heads=64, native=64),
    T("no_window_partial", [64 * 90 + 40], [25], [7], [0]),
    T("window_covers_all", [64 * 10 + 5], [4], [2], [100000]),
    T("k2_above_recall", [64 * 70 + 9], [40], [500], [256], rate=0.05),
    T("kmax_cuts", [64 * 300 + 50], [10], [6], [1000], rate=0.2),
    T("ragged_batch", [64 * 50 + 3, 64 * 200, 7, 64 * 33 + 63], [10, 30, 1, 8], [4, 9, 1, 8], [200, 0, 64, 5000],
      layers=4, heads=16, native=64, dim=64),
    T("c128_partial", [128 * 60 + 100], [12], [5], [512], chunk=128, hq=16, hkv=4, Tq=4),
    T("history_beyond_lds", [64 * 20000 + 17], [1800], [600], [8192], layers=2, heads=16, native=16, dim=64,
      rate=0.05),
]


@pytest.mark.parametrize("prob", SMALL, ids=lambda p: p.name)
def test_two_level_small(prob):
    r = run_two_level_case(prob, seed=31)
    assert r["worst_attn"] <= 2e-3


def test_two_level_nothing_recalled_no_window():
    """Nothing recalled and no window over full chunks: the kept set is empty and
    the attention is out = 0, lse = -inf."""
    prob = T("empty", [64 * 40, 64 * 30], [10, 10], [4, 4], [0, 0], layers=1, heads=16, native=16, dim=64)
    host = synth.host_inputs(prob, 6)
    q = host["idx_q"]
    q[:, :, 1::2, :] = q[:, :, 0::2, :] ^ np.uint16(0x8000)
    host["idx_w"][:] = -1.0
    r = run_two_level_case(prob, seed=6, host=host)
    assert r["cnt"].tolist() == [0, 0]


def test_two_level_rows_above_16_partial_chunk():
    """More than 16 query rows per KV head (the many-rows attention kernel), with
    full chunks and with a context that ends inside its last chunk, whose
    missing tokens get no weight."""
    run_two_level_case(T("rows32_full", [64 * 40], [10], [4], [256], hq=16, hkv=2, Tq=4), seed=7)
    run_two_level_case(T("rows32_partial", [64 * 40 + 3], [10], [4], [256], hq=16, hkv=2, Tq=4), seed=7)
    run_two_level_case(T("rows128_partial_c128", [128 * 50 + 77, 128 * 20 + 1], [12, 6], [5, 3], [300, 0],
                         chunk=128, hq=64, hkv=8, Tq=16), seed=9, rows=[(t, h) for t in (0, 7, 15) for h in range(64)])


def test_preset_two_level_tiny():
    for seed in range(4):
        run_two_level_case(synth.make_problem("twolevel_tiny", seed), seed)


def test_preset_two_level_1m():
    """The 1M-token two-level workload in the benchmark's launch configuration,
    every query row."""
    prob = synth.make_problem("twolevel1m", 0)
    r = run_two_level_case(prob, 0)
    log(f"[twolevel1m] kept {r['cnt'].tolist()} chunks of {prob.n_chunks[0]}")


@pytest.mark.parametrize("chunk,tail", [(64, 1), (64, 32), (64, 33), (64, 63), (128, 1), (128, 64), (128, 65),
                                        (128, 127)])
def test_attention_alone_partial_context_many_rows(chunk, tail):
    """The lookahead head shape (64 query heads on 8 KV heads, 16 query tokens:
    128 rows per KV head) on a context that ends inside its last chunk, through
    lsa_sparse_decode_attn, token by token against the oracle; the partial
    chunk sits last, in the middle of a split and alone."""
    import torch
    import oracle
    import parity
    import paper_2606_09079_amd as L
    Hq, Hkv, Tq = 64, 8, 16
    prob = synth.Problem("partial_rows", [chunk * 40 + tail], chunk, [8], Hq, Hkv, n_qtok=Tq)
    host = synth.host_inputs(prob, 12)
    dev = synth.device_inputs(prob, 12, host=host)
    n = prob.n_chunks[0]
    G = Hq // Hkv
    for kept in (np.array([0, 5, 17, 33, n - 3, n - 1], dtype=np.int32), np.array([n - 1], dtype=np.int32)):
        P = L.Problem(prob.ctx_tokens, chunk, [len(kept)], Hq, Hkv, n_qtok=Tq)
        ws_bytes = L.lsa_workspace_size(L.Problem([chunk * n], chunk, [len(kept)], Hq, Hkv, n_qtok=Tq))
        ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
        sel = torch.from_numpy(kept[None, :].copy()).cuda()
        cnt = torch.tensor([len(kept)], dtype=torch.int32, device="cuda")
        out = torch.full((1, Tq, Hq, 128), float("nan"), device="cuda")
        lse = torch.full((1, Tq, Hq), float("nan"), device="cuda")
        L.lsa_sparse_decode_attn(P, dev["q"], dev["k"], dev["v"], sel, cnt, 0.0, out, lse, ws, ws_bytes)
        torch.cuda.synchronize()
        g_out, g_lse = out.cpu().numpy(), lse.cpu().numpy()
        toks = oracle.kept_tokens(kept, chunk, prob.ctx_tokens[0])
        for g in (0, 3, 7):
            Kh = synth.kv_head_sparse(prob, 12, "k", 0, g, kept)
            Vh = synth.kv_head_sparse(prob, 12, "v", 0, g, kept)
            rows = [(t, g * G + j) for t in range(Tq) for j in range(G)]
            qr = np.stack([host["q"][0, t, h] for (t, h) in rows])
            r_out, r_lse = oracle.attention_tokens(qr, Kh, Vh, toks)
            parity.check_attention(np.stack([g_out[0, t, h] for (t, h) in rows]), [g_lse[0, t, h] for (t, h) in rows],
                                   r_out, r_lse, f"partial context C={chunk}, tail {tail}, {len(kept)} kept, KV head {g}")


@pytest.mark.parametrize("chunk,nfull,tail", [(64, 400, 13), (128, 200, 1), (128, 200, 127)])
def test_attention_alone_partial_context_many_rows_long(chunk, nfull, tail):
    """The lookahead head shape on a context that ends inside its last chunk,
    with long kept lists (every chunk, and every third chunk plus the last):
    each split streams many full tiles before the partial chunk, which comes
    last.  Token by token against the oracle for KV heads 0, 3 and 7."""
    import torch
    import oracle
    import parity
    import paper_2606_09079_amd as L
    Hq, Hkv, Tq = 64, 8, 16
    prob = synth.Problem("partial_rows_long", [chunk * nfull + tail], chunk, [8], Hq, Hkv, n_qtok=Tq)
    host = synth.host_inputs(prob, 21)
    dev = synth.device_inputs(prob, 21, host=host)
    n = prob.n_chunks[0]
    G = Hq // Hkv
    every = np.arange(n, dtype=np.int32)
    third = np.union1d(np.arange(0, n, 3, dtype=np.int32), [n - 1]).astype(np.int32)
    for kept in (every, third):
        P = L.Problem(prob.ctx_tokens, chunk, [len(kept)], Hq, Hkv, n_qtok=Tq)
        ws_bytes = L.lsa_workspace_size(L.Problem([chunk * n], chunk, [len(kept)], Hq, Hkv, n_qtok=Tq))
        ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
        sel = torch.from_numpy(kept[None, :].copy()).cuda()
        cnt = torch.tensor([len(kept)], dtype=torch.int32, device="cuda")
        out = torch.full((1, Tq, Hq, 128), float("nan"), device="cuda")
        lse = torch.full((1, Tq, Hq), float("nan"), device="cuda")
        L.lsa_sparse_decode_attn(P, dev["q"], dev["k"], dev["v"], sel, cnt, 0.0, out, lse, ws, ws_bytes)
        torch.cuda.synchronize()
        g_out, g_lse = out.cpu().numpy(), lse.cpu().numpy()
        toks = oracle.kept_tokens(kept, chunk, prob.ctx_tokens[0])
        for g in (0, 3, 7):
            Kh = synth.kv_head_sparse(prob, 21, "k", 0, g, kept)
            Vh = synth.kv_head_sparse(prob, 21, "v", 0, g, kept)
            rows = [(t, g * G + j) for t in range(Tq) for j in range(G)]
            qr = np.stack([host["q"][0, t, h] for (t, h) in rows])
            r_out, r_lse = oracle.attention_tokens(qr, Kh, Vh, toks)
            parity.check_attention(np.stack([g_out[0, t, h] for (t, h) in rows]), [g_lse[0, t, h] for (t, h) in rows],
                                   r_out, r_lse, f"partial context C={chunk}, tail {tail}, {len(kept)} kept, KV head {g}")
        log(f"[partial long] C={chunk} tail {tail}: {len(kept)} kept chunks, 3 KV heads x 128 rows")


@pytest.mark.parametrize("tail", [1, 31, 32, 33, 63])
def test_attention_alone_partial_context(tail):
    """lsa_sparse_decode_attn on a context that ends inside its last chunk:
    tokens past the end get no weight (compared token by token)."""
    import torch
    import oracle
    import parity
    import paper_2606_09079_amd as L
    prob = synth.Problem("partial_attn", [64 * 30 + tail], 64, [8], 8, 2)
    host = synth.host_inputs(prob, 8)
    dev = synth.device_inputs(prob, 8, host=host)
    P = L.Problem.from_synth(prob)
    n = prob.n_chunks[0]
    kept = np.array([0, 3, 11, 20, n - 2, n - 1], dtype=np.int32)
    P = L.Problem(prob.ctx_tokens, 64, [len(kept)], 8, 2)
    ws_bytes = L.lsa_workspace_size(L.Problem([64 * n], 64, [len(kept)], 8, 2))
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    sel = torch.from_numpy(kept[None, :].copy()).cuda()
    cnt = torch.tensor([len(kept)], dtype=torch.int32, device="cuda")
    out = torch.empty(1, 1, 8, 128, device="cuda")
    lse = torch.empty(1, 1, 8, device="cuda")
    L.lsa_sparse_decode_attn(P, dev["q"], dev["k"], dev["v"], sel, cnt, 0.0, out, lse, ws, ws_bytes)
    torch.cuda.synchronize()
    toks = oracle.kept_tokens(kept, 64, prob.ctx_tokens[0])
    for g in range(2):
        Kh = synth.kv_head_sparse(prob, 8, "k", 0, g, kept)
        Vh = synth.kv_head_sparse(prob, 8, "v", 0, g, kept)
        qr = np.stack([host["q"][0, 0, 4 * g + j] for j in range(4)])
        r_out, r_lse = oracle.attention_tokens(qr, Kh, Vh, toks)
        parity.check_attention(out.cpu().numpy()[0, 0, 4 * g:4 * g + 4], lse.cpu().numpy()[0, 0, 4 * g:4 * g + 4],
                               r_out, r_lse, f"partial context, tail {tail}, KV head {g}")
