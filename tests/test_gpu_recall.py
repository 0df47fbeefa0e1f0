"""Parity of the recall path (full Memory Indexer -> sigmoid threshold -> OR over
layers -> K_max bound -> attention) with the CPU oracle, on the GPU, through the
C ABI.

Small problems cover every kernel shape (1 to 4 layers, 16/32/64 heads, key
widths 64 and 128), ragged batches, the bound both cutting and not cutting,
more than 16,384 entries (the streaming selection), the empty recall and the
all-recalled extremes.  The full-size recall workloads run as the benchmark
times them, with every attention row checked.
"""
import numpy as np
import pytest

import lsa_synth as synth
from gpu_case import log
from recall_case import run_recall_case

pytestmark = pytest.mark.gpu


def R(name, ctx, chunk, kmax, hq, hkv, layers, heads, dim, rate=0.05, Tq=1):
    return synth.Problem(name, list(ctx), chunk, list(kmax), hq, hkv, n_qtok=Tq, idx_layers=layers,
                         idx_heads=heads, idx_dim=dim, idx_rate=rate)


SMALL = [
    R("one_layer_h16_c64", [64 * 200], 64, [200], 8, 8, 1, 16, 64, rate=0.1),
    R("two_layers_cut", [64 * 300], 64, [20], 8, 2, 2, 32, 128, rate=0.1),
    R("four_layers_h64", [128 * 90, 128 * 17], 128, [30, 17], 16, 4, 4, 64, 128, rate=0.08, Tq=2),
    R("three_layers_ragged", [64 * 5, 64 * 130, 64, 64 * 77], 64, [5, 9, 1, 77], 8, 2, 3, 16, 128, rate=0.15),
    R("h32_c64_rows16", [64 * 160], 64, [40], 32, 2, 3, 32, 64, rate=0.05),
    R("beyond_lds_entries", [64 * 20000], 64, [1500], 8, 8, 2, 16, 64, rate=0.05),
]


@pytest.mark.parametrize("prob", SMALL, ids=lambda p: p.name)
def test_recall_small(prob):
    r = run_recall_case(prob, seed=21)
    assert r["worst_attn"] <= 2e-3


def _with_gates(prob, seed, gates):
    """Host inputs of prob with every gate weight replaced by gates(b, l, h)."""
    host = synth.host_inputs(prob, seed)
    w = host["idx_w"]
    for b in range(w.shape[0]):
        for l in range(w.shape[1]):
            for h in range(w.shape[2]):
                w[b, l, h] = gates(b, l, h)
    return host


def test_recall_nothing_recalled():
    """Heads in pairs q and -q with negative gates: every score is below 0, no
    entry is recalled, and the attention of the empty set is out = 0, lse = -inf."""
    prob = R("empty", [64 * 50, 64 * 20], 64, [10, 5], 8, 4, 2, 16, 64)
    host = synth.host_inputs(prob, 3)
    q = host["idx_q"]
    q[:, :, 1::2, :] = q[:, :, 0::2, :] ^ np.uint16(0x8000)
    host["idx_w"][:] = -1.0
    r = run_recall_case(prob, seed=3, host=host)
    assert r["cnt"].tolist() == [0, 0]


def test_recall_everything_below_bound_and_cut():
    """Non-negative gates recall every entry (sigmoid >= 1/2 everywhere): with
    K_max = n all entries come back; with a smaller K_max the bound keeps the
    entries with the largest scores."""
    prob = R("all_gates_pos", [64 * 40, 64 * 60], 64, [40, 25], 8, 8, 2, 16, 64)
    host = _with_gates(prob, 4, lambda b, l, h: 0.25 + 0.01 * h)
    r = run_recall_case(prob, seed=4, host=host)
    assert r["cnt"].tolist() == [40, 25]
    assert r["sel"][0, :40].tolist() == list(range(40))


def test_recall_step_is_deterministic():
    import torch
    import paper_2606_09079_amd as L
    prob = R("det", [64 * 500, 64 * 300], 64, [60, 40], 32, 8, 3, 64, 128)
    dev = synth.device_inputs(prob, 5)
    P, ix = L.Problem.from_synth(prob), L.Indexer.from_synth(prob)
    ws_bytes = L.lsa_workspace_size(P)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    outs = []
    for _ in range(3):
        out = torch.empty(2, 1, 32, 128, device="cuda")
        lse = torch.empty(2, 1, 32, device="cuda")
        L.lsa_recall_step(P, ix, dev["idx_q"], dev["idx_w"], dev["idx_k"], dev["q"], dev["k"], dev["v"], 0.0, out,
                          lse, None, None, ws, ws_bytes)
        torch.cuda.synchronize()
        outs.append((out.cpu().numpy(), lse.cpu().numpy()))
    for o, s in outs[1:]:
        assert np.array_equal(o, outs[0][0]) and np.array_equal(s, outs[0][1])


def test_preset_recall_tiny():
    for seed in range(4):
        run_recall_case(synth.make_problem("recall_tiny", seed), seed)


def test_preset_recall_batch():
    prob = synth.make_problem("recall_batch", 0)
    run_recall_case(prob, 0)


def test_preset_recall1m():
    """The 1M-token recall workload in the benchmark's launch configuration,
    every query row."""
    prob = synth.make_problem("recall1m", 0)
    r = run_recall_case(prob, 0)
    log(f"[recall1m] recalled {r['cnt'].tolist()} of {prob.n_chunks[0]} (K_max {prob.keep[0]})")
