"""The fused step where the split kernel merges its own splits (at most 16
query rows per KV head, at most 8 sequences, at most 16 splits per (sequence,
KV head)): its last workgroup of each (b, g) reads every split's partials and
runs the few-split merge instead of a combine launch.

The cases span the shapes that path has to handle: 1 to 16 rows per KV head
(at 12 and 16 rows a thread merges two row slices), one sequence with 16 KV
heads, eight sequences, one split for a short sequence next to a dozen for
long ones, 64- and 128-token chunks, and bf16 and int8 embeddings.  Each runs the
whole parity case: scores and kept ids against the oracle, attention against
the oracle, and the fused step's output and lse equal to the separate
attention call bit for bit (gpu_case.run_case).
"""
import pytest

import lsa_synth as synth
from gpu_case import run_case

pytestmark = pytest.mark.gpu


def _merges_in_split(prob: synth.Problem) -> bool:
    """The host plan's rule (one resident round of 256 workgroups for at most
    8 sequences, splits in proportion to the kept chunks) restated, so that a
    change to it shows up here rather than as lost coverage."""
    B, C, hkv = prob.batch, prob.chunk, prob.n_kv_heads
    rows = (prob.n_q_heads // hkv) * prob.n_qtok
    n = [-(-L // C) for L in prob.ctx_tokens]
    msel = [min(prob.n_lookahead * k, nb) for k, nb in zip(prob.keep, n)]
    total = sum(msel)
    ns = [max(1, min(round(256 * m / (hkv * total)), 256, m * (C // 32))) for m in msel]
    return rows <= 16 and B <= 8 and max(ns) <= 16


CASES = [
    # 16 rows per KV head (G = 2, Tq = 8): two row slices per thread in the merge
    synth.Problem("merge_rows16", [64 * 300, 64 * 280], 64, [40, 38], 16, 8, n_qtok=8),
    # 12 rows per KV head (G = 3, Tq = 4)
    synth.Problem("merge_rows12", [64 * 260, 64 * 240], 64, [30, 30], 24, 8, n_qtok=4),
    # one sequence, 16 KV heads, 128-token chunks
    synth.Problem("merge_one_seq", [128 * 400], 128, [48], 32, 16),
    # eight sequences of 4 KV heads, 16 rows each (G = 8, Tq = 2)
    synth.Problem("merge_eight_seq", [64 * (120 + 37 * b) for b in range(8)], 64, [20 + 3 * b for b in range(8)],
                  32, 4, n_qtok=2),
    # a short sequence with a single split next to long ones
    synth.Problem("merge_one_split", [64 * 8, 64 * 500, 64 * 450, 64 * 300], 64, [1, 60, 55, 40], 16, 8, n_qtok=2),
    # int8 embeddings (integer scores, exact selection)
    synth.Problem("merge_int8", [64 * 512, 64 * 384, 64 * 256], 64, [48, 40, 32], 32, 8, emb_dtype="i8"),
]


@pytest.mark.parametrize("prob", CASES, ids=[p.name for p in CASES])
def test_fused_step_with_split_kernel_merge(prob):
    assert _merges_in_split(prob), f"{prob.name} no longer takes the split kernel's own merge"
    r = run_case(prob, seed=11)
    assert r["worst_fused"] <= 2e-3
