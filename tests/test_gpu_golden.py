"""The golden-label pipeline on the GPU against the oracle, through the C ABI.

The oracle takes the softmax of Eq. 7 in float64 and its top-p set (Eq. 8) as
the shortest prefix, in (logit desc, index asc) order, whose mass reaches p.
The kernel takes the same integer decision from float32 weights held as whole
multiples of 2^-40 of the largest.  Per row, the comparison reads the GPU's
membership bitmap from the workspace and derives the band inside which the
two may differ: each kernel weight is within (|x| + 3) 2^-24 w + 2^-40 of the
exact w = exp(x), x = S - max S (the float32 rounding of x, the float32
exponential within 3 ulp, the floor to 2^-40), so with E the sum of those
bounds over the row and Z the sum of weights, the kernel's mass fraction of
any prefix is within beta = 2 E / (Z - E) of the exact one.  The GPU's set must
then be a prefix of the oracle's order whose length lies between the first
prefix reaching p - beta and the first reaching p + beta; where those agree
(nearly every row) it is exactly the oracle's set.  The top-p set sizes, the
votes, the golden sets and the labels must follow exactly from the GPU's own
rows, and equal the oracle's wherever no row of the window fell in a band.

Cases: the seeded workloads (the full 512K-token window included), rows whose
lengths are not multiples of the 32-entry bitmap words, p from 1/1000 to 1,
theta from 1 to above L, many equal logits at the top-p boundary (the lower
indices must be taken), -0.0 against +0.0, and rows whose boundary bin holds
more entries than the kernel stages in LDS.
"""
from __future__ import annotations

import time

import numpy as np
import pytest

import lsa_synth as synth
import oracle
from gpu_case import log

pytestmark = pytest.mark.gpu


def run_golden(logits_per_seq, tau, L, theta, p_num, p_den):
    """GPU labels for host logits, one [tau][L][n_b] float32 array per sequence,
    compared with the oracle sequence by sequence."""
    import torch
    import paper_2606_09079_amd as L_
    ns = [x.shape[2] for x in logits_per_seq]
    g = L_.Golden(ns, tau, L, theta, p_num, p_den)
    ws_bytes = L_.lsa_golden_sizes(g)
    packed = torch.from_numpy(np.concatenate([x.reshape(-1) for x in logits_per_seq])).cuda()
    return _compare(g, packed, ns, tau, L, theta, p_num, p_den, ws_bytes,
                    lambda b: logits_per_seq[b])


def _kernel_band(S: np.ndarray) -> float:
    """beta of one row: the bound on the kernel's mass fraction error."""
    x = S.astype(np.float64) - float(S.max())
    w = np.exp(x)
    E = float(np.sum(w * (np.abs(x) + 3.0) * 2.0 ** -24 * (1.0 + 2.0 ** -20) + 2.0 ** -40))
    Z = float(np.sum(w))
    return 2.0 * E / (Z - E) + 1e-9


def _check_row(S, gpu_mark, p_num, p_den, where):
    """The GPU row against the oracle's order and prefix masses; returns the
    oracle's marks and whether the row fell in a band."""
    mark, size, order, cum = oracle.top_p(S, p_num, p_den, detail=True)
    p = p_num / p_den
    beta = _kernel_band(S)
    n = len(S)
    k_lo = int(np.searchsorted(cum, p - beta, side="left")) + 1
    k_hi = min(int(np.searchsorted(cum, p + beta, side="left")) + 1, n)
    k_lo = min(k_lo, k_hi)
    assert k_lo <= size <= k_hi, f"{where}: oracle size {size} outside its own band [{k_lo}, {k_hi}]"
    k = int(gpu_mark.sum())
    assert k_lo <= k <= k_hi, f"{where}: GPU set of {k} entries, band [{k_lo}, {k_hi}] (oracle {size})"
    assert np.all(gpu_mark[order[:k]] == 1), f"{where}: the GPU set is not the first {k} entries of the oracle's order"
    return mark, k_lo != k_hi


def _compare(g, packed, ns, tau, L, theta, p_num, p_den, ws_bytes, host_logits, seqs=None):
    import torch
    import paper_2606_09079_amd as L_
    B = len(ns)
    ws = torch.zeros(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    labels = torch.full((sum(ns),), -1, dtype=torch.int32, device="cuda")
    count = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    sizes = torch.full((B, tau, L), -1, dtype=torch.int32, device="cuda")
    golden = torch.full((B, tau), -1, dtype=torch.int32, device="cuda")
    L_.lsa_golden_labels(g, packed, labels, count, sizes, golden, ws, ws_bytes)
    torch.cuda.synchronize()
    g_lab, g_cnt, g_sizes, g_gold = labels.cpu().numpy(), count.cpu().numpy(), sizes.cpu().numpy(), golden.cpu().numpy()
    g_ws = ws.cpu().numpy()
    off = np.concatenate([[0], np.cumsum(ns)])
    bit_off = 0  # bytes: the row bitmaps of sequence b follow those of b - 1, [tau][L][ceil(n_b / 32)] words
    band_rows = 0
    for b in range(B):
        words = (ns[b] + 31) // 32
        nbytes = tau * L * words * 4
        bits = g_ws[bit_off:bit_off + nbytes].reshape(tau, L, words * 4)
        bit_off += nbytes
        if seqs is not None and b not in seqs:
            continue
        x = host_logits(b)
        n = ns[b]
        gpu_rows = np.unpackbits(bits, axis=2, bitorder="little")[:, :, :n]
        orc_rows = np.zeros_like(gpu_rows)
        banded = False
        for i in range(tau):
            for l in range(L):
                orc_rows[i, l], in_band = _check_row(x[i, l], gpu_rows[i, l], p_num, p_den, f"seq {b} row ({i}, {l})")
                band_rows += in_band
                banded |= in_band and not np.array_equal(orc_rows[i, l], gpu_rows[i, l])
        # sizes, votes (Eq. 9), golden sets (Eq. 10) and labels (Eq. 11) follow from the GPU's own rows
        assert np.array_equal(g_sizes[b], gpu_rows.sum(axis=2)), f"seq {b}: top-p set sizes differ from the bitmaps"
        votes = gpu_rows.astype(np.int64).sum(axis=1)
        A = votes >= theta
        assert np.array_equal(g_gold[b], A.sum(axis=1)), f"seq {b}: golden-set sizes differ from the GPU's rows"
        want = np.nonzero(A.any(axis=0))[0]
        got = g_lab[off[b]:off[b] + g_cnt[b]]
        assert g_cnt[b] == len(want) and np.array_equal(got, want), \
            f"seq {b}: labels differ from the GPU's rows; first differences {sorted(set(got) ^ set(want))[:8]}"
        if not banded:  # every row equals the oracle's: the labels are the oracle's
            A_o = orc_rows.astype(np.int64).sum(axis=1) >= theta
            assert np.array_equal(got, np.nonzero(A_o.any(axis=0))[0]), f"seq {b}: labels differ from the oracle's"
            assert np.array_equal(g_gold[b], A_o.sum(axis=1)), f"seq {b}: golden-set sizes differ from the oracle's"
    if band_rows:
        log(f"[golden] {band_rows} row(s) with a cut inside the float32 band")
    return g_lab, g_cnt, g_sizes, g_gold


def _rows(rng, tau, L, n, kind):
    if kind == "gauss":
        return (rng.standard_normal((tau, L, n)) * 2.0).astype(np.float32)
    if kind == "peaked":
        x = rng.standard_normal((tau, L, n)).astype(np.float32)
        hot = rng.choice(n, size=max(1, n // 50), replace=False)
        x[:, :, hot] += np.float32(6.0)
        return x
    if kind == "ties":  # values on a coarse grid: many equal logits at every boundary
        return (np.round(rng.standard_normal((tau, L, n)) * 2.0) / 2.0).astype(np.float32)
    if kind == "equal":  # every logit equal, half of them -0.0
        x = np.zeros((tau, L, n), np.float32)
        x[..., ::2] = np.float32(-0.0)
        return x
    raise KeyError(kind)


@pytest.mark.parametrize("n", [1, 7, 31, 63, 65, 1000, 5003])
@pytest.mark.parametrize("kind", ["gauss", "peaked", "ties", "equal"])
def test_golden_small(n, kind):
    rng = np.random.default_rng(n * 7 + len(kind))
    x = _rows(rng, 3, 5, n, kind)
    run_golden([x], 3, 5, 3, 3, 5)


@pytest.mark.parametrize("p", [(1, 1000), (1, 2), (9, 10), (1, 1)])
@pytest.mark.parametrize("theta", [1, 2, 5, 6, 64])
def test_golden_p_and_theta(p, theta):
    rng = np.random.default_rng(theta * 100 + p[0])
    x = _rows(rng, 4, 5, 777, "peaked")
    run_golden([x], 4, 5, theta, p[0], p[1])


def test_golden_ragged_batch():
    rng = np.random.default_rng(5)
    xs = [_rows(rng, 2, 7, n, k) for n, k in ((100, "gauss"), (4097, "ties"), (33, "equal"), (20000, "peaked"))]
    run_golden(xs, 2, 7, 3, 3, 5)


@pytest.mark.parametrize("kind", ["narrow", "narrow_ties"])
def test_golden_boundary_bin_beyond_lds(kind):
    """Every logit in one 12-bit key bin (more entries than the kernel stages):
    the threshold is refined by passes over the row."""
    rng = np.random.default_rng(9)
    n = 20000
    x = (np.float32(1.0) + rng.random((2, 3, n)).astype(np.float32) * np.float32(0.1)).astype(np.float32)
    if kind == "narrow_ties":
        x = (np.round(x * 64.0) / 64.0).astype(np.float32)
    run_golden([x], 2, 3, 2, 3, 5)


def test_golden_largest_row():
    """A sequence of LSA_MAX_GOLDEN_ENTRIES entries (two rows of 4,194,304
    logits)."""
    rng = np.random.default_rng(17)
    run_golden([_rows(rng, 1, 2, 4194304, "gauss")], 1, 2, 1, 3, 5)


@pytest.mark.parametrize("theta", [1, 32, 63])
def test_golden_most_layers(theta):
    """LSA_MAX_GOLDEN_LAYERS layers voting, with vote thresholds from one layer
    to all of them."""
    rng = np.random.default_rng(23 + theta)
    run_golden([_rows(rng, 2, 63, 500, "peaked")], 2, 63, theta, 3, 5)


def test_golden_tiny_presets():
    import torch
    import paper_2606_09079_amd as L_
    gp = synth.make_golden_problem("golden_tiny")
    for seed in range(3):
        g = L_.Golden.from_synth(gp)
        dev = synth.golden_logits_device(gp, seed)
        _compare(g, dev, gp.n_entries, gp.tau, gp.layers, gp.theta, gp.p_num, gp.p_den, L_.lsa_golden_sizes(g),
                 lambda b: synth.golden_logits(gp, seed, b))
        host = np.concatenate([synth.golden_logits(gp, seed, b).reshape(-1) for b in range(gp.batch)])
        assert np.array_equal(dev.cpu().numpy(), host), "device and host logits differ"


def test_golden_512k_window():
    """The full window of the 512K-token workload (131,072 entries, 64 steps,
    21 layers) in the benchmark's launch configuration."""
    import torch
    import paper_2606_09079_amd as L_
    gp = synth.make_golden_problem("golden512k")
    g = L_.Golden.from_synth(gp)
    t0 = time.time()
    dev = synth.golden_logits_device(gp, 0)
    host = synth.golden_logits(gp, 0, 0)
    assert np.array_equal(dev[:host.size].cpu().numpy(), host.reshape(-1)), "device and host logits differ"
    log(f"[golden] logits ready ({time.time() - t0:.1f}s)")
    g_lab, g_cnt, g_sizes, g_gold = _compare(g, dev, gp.n_entries, gp.tau, gp.layers, gp.theta, gp.p_num, gp.p_den,
                                             L_.lsa_golden_sizes(g), lambda b: host)
    log(f"[golden] 512k: {int(g_cnt[0])} labels, top-p sets {int(g_sizes.min())}..{int(g_sizes.max())}, "
        f"golden sets {int(g_gold.min())}..{int(g_gold.max())} ({time.time() - t0:.1f}s)")


def test_golden_deterministic():
    import torch
    import paper_2606_09079_amd as L_
    rng = np.random.default_rng(3)
    x = torch.from_numpy(_rows(rng, 4, 6, 3000, "ties").reshape(-1)).cuda()
    g = L_.Golden([3000], 4, 6, 2, 1, 2)
    wsb = L_.lsa_golden_sizes(g)
    outs = []
    for _ in range(3):
        ws = torch.zeros(wsb, dtype=torch.uint8, device="cuda")
        lab = torch.empty(3000, dtype=torch.int32, device="cuda")
        cnt = torch.empty(1, dtype=torch.int32, device="cuda")
        sz = torch.empty(4, 6, dtype=torch.int32, device="cuda")
        L_.lsa_golden_labels(g, x, lab, cnt, sz, None, ws, wsb)
        torch.cuda.synchronize()
        c = int(cnt.cpu()[0])
        outs.append((lab.cpu().numpy()[:c].copy(), sz.cpu().numpy().copy()))
    for a, s in outs[1:]:
        assert np.array_equal(a, outs[0][0]) and np.array_equal(s, outs[0][1])
