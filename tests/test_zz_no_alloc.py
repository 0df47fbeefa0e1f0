"""The allocation-free decode step through the C ABI.

lsa_decode_step_noalloc runs lsa_decode_step on the library's per-GPU device
scratch instead of a caller workspace.  Two calls in a row -- the 1M-token
benchmark step, then a smaller ragged problem -- must each equal, bit for bit,
lsa_decode_step on the same inputs with a fresh caller workspace (the same
kernels on the same plan), so nothing the first call left in the scratch
reaches the second.  The small problem is also checked against the oracle.
"""
from __future__ import annotations

import numpy as np
import pytest

import lsa_synth as synth
import oracle
import parity
from gpu_case import log

pytestmark = pytest.mark.gpu


def _run(L, prob, dev, noalloc: bool, with_sel: bool):
    import torch
    P = L.Problem.from_synth(prob)
    B, Tq, Hq = prob.batch, prob.n_qtok, prob.n_q_heads
    out = torch.full((B, Tq, Hq, 128), float("nan"), dtype=torch.float32, device="cuda")
    lse = torch.full((B, Tq, Hq), float("nan"), dtype=torch.float32, device="cuda")
    sel = torch.full((B, L.lsa_max_sel(P)), -1, dtype=torch.int32, device="cuda") if with_sel else None
    cnt = torch.full((B,), -1, dtype=torch.int32, device="cuda") if with_sel else None
    if noalloc:
        L.lsa_decode_step_noalloc(P, dev["qe"], dev["E"], dev["q"], dev["k"], dev["v"], 0.0, out, lse, sel, cnt)
    else:
        wsb = L.lsa_workspace_size(P)
        ws = torch.zeros(max(wsb, 256), dtype=torch.uint8, device="cuda")
        L.lsa_decode_step(P, dev["qe"], dev["E"], dev["q"], dev["k"], dev["v"], 0.0, out, lse, sel, cnt, ws, wsb)
    torch.cuda.synchronize()
    res = [out.cpu().numpy(), lse.cpu().numpy()]
    if with_sel:
        res += [sel.cpu().numpy(), cnt.cpu().numpy()]
    return res


def _same(a, b, what):
    for x, y in zip(a, b):
        assert x.shape == y.shape and np.array_equal(x.view(np.uint32) if x.dtype == np.float32 else x,
                                                     y.view(np.uint32) if y.dtype == np.float32 else y), what


def test_noalloc_two_calls_match_the_workspace_step():
    import torch
    import paper_2606_09079_amd as L
    torch.cuda.set_device(0)
    big = synth.make_problem("paper1m", 0)
    dev = synth.device_inputs(big, 0)
    log("[noalloc] call 1: paper1m (1,048,576 tokens, keep 1,638)")
    got = _run(L, big, dev, True, True)
    want = _run(L, big, dev, False, True)
    assert not np.isnan(got[0]).any()
    _same(got, want, "paper1m: the allocation-free step differs from the workspace step")
    del dev
    torch.cuda.empty_cache()

    small = synth.Problem("noalloc_small", [64 * 300, 64 * 77, 64 * 1000], 64, [40, 9, 100], 32, 8, planted=4)
    host = synth.host_inputs(small, 5)
    dev = synth.device_inputs(small, 5, host=host)
    log("[noalloc] call 2: 3 ragged sequences (300, 77, 1000 chunks), kept ids left in the scratch")
    got = _run(L, small, dev, True, False)
    want = _run(L, small, dev, False, True)
    assert not np.isnan(got[0]).any()
    _same(got, want[:2], "small: the allocation-free step differs from the workspace step")
    # and against the oracle: the kept sets by the band rule, the attention over the GPU's kept set
    g_sel, g_cnt = want[2], want[3]
    for b in range(small.batch):
        scores, _, _ = oracle.select_for_sequence(small, host, b)
        kept = g_sel[b, :g_cnt[b]]
        parity.check_kept(kept, scores[0], small.keep[b], False, f"noalloc small seq {b}")
        kv = lambda which, bb, g, ch: synth.kv_head_sparse(small, 5, which, bb, g, ch)
        ref = oracle.attend_rows(small, host, b, kept, [(0, h) for h in range(small.n_q_heads)], kv)
        for h in range(small.n_q_heads):
            r_out, r_lse = ref[(0, h)]
            parity.check_attention(got[0][b, 0, h][None], [got[1][b, 0, h]], r_out[None], [r_lse],
                                   f"noalloc small seq {b} head {h}")
    log("[noalloc] both calls equal the workspace step bit for bit")
