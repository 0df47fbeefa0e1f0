"""Comparators between the HIP path and the CPU oracle.

Tolerances (written here, derived in the design notes):
* int8 scores and every chunk-id set of the int8 workload: bit-exact;
* fp32 scores: |gpu - oracle| <= 2 * D * 2**-24 * sum_i |qe_i E_ci| + 1e-30, the
  standard bound for a length-D float32 dot product of exactly representable
  products;
* kept sets for float scores: identical unless the oracle's k-th and (k+1)-th
  scores differ by less than 1e-4 relative; inside that band the GPU set must
  contain every chunk scoring above the band, lie inside the band's closure and
  have k members;
* recall index scores x_l[s] = sum_h w_h ReLU(q_h . K_s):
  |gpu - oracle| <= (c + n_h + 4) * 2**-24 * sum_h |w_h| sum_i |q_hi K_si|, the
  float32 bound for c-term dot products of exact products, the ReLU (which
  cannot grow an error), one product with the gate and an n_h-term sum;
* recalled sets: identical to the oracle's unless an entry's max-over-layers
  score lies within that bound of the threshold 0 or, when the K_max bound
  cuts, of the cut; otherwise the GPU set must hold every entry surely
  recalled (up to the bound), no entry that cannot be recalled, and must never
  leave out an entry clearly above one it kept;
* attention: max relative error 2e-3 per (b, t, h) row, normwise
  (max_e |o - r| / max_e |r|), bf16 inputs with fp32 accumulation; lse within
  2e-3 absolute.
"""
from __future__ import annotations

import numpy as np

TOPK_REL_BAND = 1e-4
ATTN_REL_TOL = 2e-3
LSE_ABS_TOL = 2e-3


def score_tolerance(qe: np.ndarray, E: np.ndarray, emb_dtype: str) -> np.ndarray:
    import lsa_synth
    if emb_dtype == "bf16":
        q64, E64 = lsa_synth.bf16_bits_to_f64(qe), lsa_synth.bf16_bits_to_f64(E)
    else:
        q64, E64 = qe.astype(np.float64), E.astype(np.float64)
    D = E.shape[1]
    return 2.0 * D * 2.0 ** -24 * (np.abs(E64) @ np.abs(q64)) + 1e-30


def check_scores(gpu: np.ndarray, ref: np.ndarray, qe, E, emb_dtype: str, what: str) -> float:
    if emb_dtype == "i8":
        bad = np.nonzero(gpu.astype(np.int64) != ref)[0]
        assert len(bad) == 0, f"{what}: int8 scores differ at {bad[:10]} (gpu {gpu[bad[:5]]}, oracle {ref[bad[:5]]})"
        return 0.0
    tol = score_tolerance(qe, E, emb_dtype)
    err = np.abs(gpu.astype(np.float64) - ref)
    bad = np.nonzero(err > tol)[0]
    assert len(bad) == 0, f"{what}: scores off at {bad[:10]} err {err[bad[:5]]} tol {tol[bad[:5]]}"
    return float(err.max())


def kth_gap(ref: np.ndarray, k: int):
    n = len(ref)
    order = np.lexsort((np.arange(n), -ref))
    sk = ref[order[k - 1]]
    sk1 = ref[order[k]] if k < n else -np.inf
    return sk, sk1, order


def check_kept(gpu_sel: np.ndarray, ref: np.ndarray, k: int, exact: bool, what: str):
    """Band rule for one (sequence, query); returns 'exact' or 'band'."""
    gpu_sel = np.asarray(gpu_sel, dtype=np.int64)
    assert len(gpu_sel) == k, f"{what}: {len(gpu_sel)} kept, want {k}"
    assert np.all(np.diff(gpu_sel) > 0), f"{what}: kept ids not strictly ascending"
    sk, sk1, order = kth_gap(ref, k)
    oracle_set = np.sort(order[:k])
    in_band = bool(np.isfinite(sk1)) and (sk - sk1 < TOPK_REL_BAND * max(abs(sk), abs(sk1)))
    if exact or not in_band:
        same = np.array_equal(gpu_sel, oracle_set)
        if not same:
            diff = sorted(set(gpu_sel.tolist()) ^ set(oracle_set.tolist()))
            raise AssertionError(f"{what}: kept set differs from the oracle at chunks {diff[:10]}")
        return "exact"
    delta = TOPK_REL_BAND * max(abs(sk), abs(sk1))
    must = set(np.nonzero(ref > sk + delta)[0].tolist())
    band = set(np.nonzero(np.abs(ref - sk) <= delta)[0].tolist())
    G = set(gpu_sel.tolist())
    assert must <= G, f"{what}: chunks {sorted(must - G)[:10]} above the band missing"
    assert G <= (must | band), f"{what}: chunks {sorted(G - must - band)[:10]} outside the band"
    return "band"


def rowwise_rel_err(gpu: np.ndarray, ref: np.ndarray) -> float:
    return float(np.max(np.abs(gpu.astype(np.float64) - ref)) / max(np.max(np.abs(ref)), 1e-30))


def check_attention(gpu_out: np.ndarray, gpu_lse, ref_out: np.ndarray, ref_lse, what: str) -> float:
    worst = 0.0
    for i in range(ref_out.shape[0]):
        e = rowwise_rel_err(gpu_out[i], ref_out[i])
        worst = max(worst, e)
        assert e <= ATTN_REL_TOL, f"{what}: row {i} relative error {e:.3e} > {ATTN_REL_TOL}"
        if gpu_lse is not None:
            d = abs(float(gpu_lse[i]) - float(ref_lse[i]))
            assert d <= LSE_ABS_TOL, f"{what}: row {i} lse error {d:.3e}"
    return worst


def index_score_tolerance(q: np.ndarray, w: np.ndarray, K: np.ndarray) -> np.ndarray:
    """Bound on |gpu - oracle| of one layer's recall scores; q [n_h][c] and K
    [n][c] are bf16 bit patterns, w [n_h] float32."""
    import lsa_synth
    q64, K64 = np.abs(lsa_synth.bf16_bits_to_f64(q)), np.abs(lsa_synth.bf16_bits_to_f64(K))
    n_h, c = q.shape
    return (c + n_h + 4) * 2.0 ** -24 * ((K64 @ q64.T) @ np.abs(w.astype(np.float64))) + 1e-30


def check_index_scores(gpu: np.ndarray, ref: np.ndarray, tol: np.ndarray, what: str) -> float:
    err = np.abs(gpu.astype(np.float64) - ref)
    bad = np.nonzero(err > tol)[0]
    assert len(bad) == 0, f"{what}: recall scores off at {bad[:10]} err {err[bad[:5]]} tol {tol[bad[:5]]}"
    return float(err.max()) if len(err) else 0.0


def check_recall(gpu_sel: np.ndarray, ref_x: np.ndarray, tol: np.ndarray, kmax: int, what: str) -> str:
    """Band rule for a recalled set.  ref_x, tol: [L][n] oracle scores and their
    bounds.  Returns 'exact' when the GPU set equals the oracle's."""
    import oracle
    gpu_sel = np.asarray(gpu_sel, dtype=np.int64)
    n = ref_x.shape[1]
    assert len(gpu_sel) <= kmax, f"{what}: {len(gpu_sel)} recalled > K_max {kmax}"
    assert np.all(np.diff(gpu_sel) > 0), f"{what}: recalled ids not strictly ascending"
    assert len(gpu_sel) == 0 or (gpu_sel[0] >= 0 and gpu_sel[-1] < n), f"{what}: recalled id out of range"
    want = oracle.recall(ref_x, kmax)
    if np.array_equal(gpu_sel, want):
        return "exact"
    hi = (ref_x + tol).max(axis=0)    # largest score each entry could have on the GPU
    lo = (ref_x - tol).max(axis=0)    # smallest
    G = set(gpu_sel.tolist())
    possible = set(np.nonzero(hi >= 0)[0].tolist())
    sure = set(np.nonzero(lo > 0)[0].tolist())
    assert G <= possible, f"{what}: entries {sorted(G - possible)[:10]} cannot be recalled"
    assert len(G) >= min(kmax, len(sure)), f"{what}: {len(G)} recalled, {len(sure)} surely recalled"
    if len(G) < kmax:
        assert sure <= G, f"{what}: surely recalled entries {sorted(sure - G)[:10]} missing"
    out = sorted(possible - G)
    if G and out:
        weakest_in = min(hi[g] for g in G)
        clearly = [s for s in out if lo[s] > weakest_in]
        assert not clearly, f"{what}: entries {clearly[:10]} left out but surely above a kept one"
    return "band"
