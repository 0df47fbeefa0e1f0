"""Pins that tie the CPU oracle to the paper and to mathematics, not to itself.

Each ``pin_*`` function raises AssertionError when the oracle disagrees with
an independent fact: a hand-worked example, a closed form, brute force over all
subsets, a library routine that computes the same definition by another route,
or an invariant the paper states (all chunks kept == dense attention, Sec. 2.5
cold start).  ``test_oracle.py`` runs them on the real oracle and
``test_oracle_mutants.py`` checks that planted mistakes in the oracle's C
source make at least one of them fail.
"""
from __future__ import annotations

import itertools
import json
import math
import os

import numpy as np
import scipy.special
import torch

import lsa_synth as synth
import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _bf16(x) -> np.ndarray:
    return synth.f64_to_bf16_bits(np.asarray(x, dtype=np.float64))


def _f64(bits) -> np.ndarray:
    return synth.bf16_bits_to_f64(bits)


# ------------------------------------------------------------------ scores
def pin_score_library_matmul():
    """O1 for f32 and bf16 equals a float64 matrix-vector product (numpy)."""
    rng = np.random.default_rng(1)
    for D in (64, 256):
        E = rng.standard_normal((37, D)).astype(np.float32)
        qe = rng.standard_normal(D).astype(np.float32)
        ref = E.astype(np.float64) @ qe.astype(np.float64)
        got = oracle.score(qe, E, "f32")
        assert np.allclose(got, ref, rtol=1e-12, atol=1e-12), "f32 score != E @ qe"
        Eb, qb = _bf16(E), _bf16(qe)
        ref = _f64(Eb) @ _f64(qb)
        got = oracle.score(qb, Eb, "bf16")
        assert np.allclose(got, ref, rtol=1e-12, atol=1e-12), "bf16 score != E @ qe"


def pin_score_int8_exact():
    """O1 for int8 is the exact integer dot product (Python integers)."""
    rng = np.random.default_rng(2)
    E = rng.integers(-127, 128, size=(23, 256)).astype(np.int8)
    qe = rng.integers(-127, 128, size=256).astype(np.int8)
    got = oracle.score(qe, E, "i8")
    for c in range(E.shape[0]):
        exact = sum(int(a) * int(b) for a, b in zip(qe.tolist(), E[c].tolist()))
        assert int(got[c]) == exact, f"int8 score of chunk {c}"


def pin_score_closed_forms():
    """One-hot chunk rows read out one query component; the sign-aligned
    planted row scores 127 * sum |qe_i|; scaling qe by 2 doubles every score."""
    D = 16
    qe = np.arange(1, D + 1, dtype=np.float64) * np.array([(-1) ** i for i in range(D)])
    E = np.eye(D, dtype=np.float32)
    got = oracle.score(qe.astype(np.float32), E, "f32")
    assert np.array_equal(got, qe), "one-hot rows must return the query components"
    q8 = np.array([5, -3, 0, 127, -127, 1, -1, 2] * 32, dtype=np.int8)
    row = np.where(q8 >= 0, 127, -127).astype(np.int8)[None, :]
    s = oracle.score(q8, row, "i8")
    assert int(s[0]) == 127 * int(np.abs(q8.astype(np.int64)).sum()), "sign-aligned planted score"
    rng = np.random.default_rng(3)
    E = rng.standard_normal((9, 32)).astype(np.float32)
    q = rng.standard_normal(32).astype(np.float32)
    assert np.array_equal(oracle.score(2 * q, E, "f32"), 2 * oracle.score(q, E, "f32")), "homogeneity"


# -------------------------------------------------------------------- top-k
def pin_topk_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "topk_worked.json")))
    s = np.array(g["scores"], dtype=np.float64)
    for case in g["cases"]:
        got = oracle.topk(s, case["k"])
        assert got.tolist() == case["kept"], f"worked top-k, k={case['k']}"
        got_i = oracle.topk(s.astype(np.int64), case["k"])
        assert got_i.tolist() == case["kept"], f"worked int top-k, k={case['k']}"
    u = g["union"]
    assert oracle.union(np.array(u["lists"]), u["n"]).tolist() == u["kept"], "worked union"


def pin_topk_bruteforce():
    """Over all C(n, k) subsets: the kept set has the largest score sum and,
    among those, the lexicographically smallest ascending id list."""
    rng = np.random.default_rng(4)
    for trial in range(60):
        n = int(rng.integers(1, 11))
        k = int(rng.integers(1, n + 1))
        s = rng.integers(-3, 4, size=n).astype(np.float64)  # many ties
        best, best_sum = None, -math.inf
        for comb in itertools.combinations(range(n), k):  # lexicographic order
            tot = s[list(comb)].sum()
            if tot > best_sum:
                best, best_sum = list(comb), tot
        assert oracle.topk(s, k).tolist() == best, f"brute force n={n} k={k} s={s.tolist()}"
        assert oracle.topk(s.astype(np.int64), k).tolist() == best, "brute force (int)"


def pin_topk_library_sort():
    """Agrees with numpy's lexsort on (score desc, id asc); k=1 is numpy's
    first argmax; k=n keeps everything; -0.0 ties +0.0."""
    rng = np.random.default_rng(5)
    for n, k in ((1000, 100), (2048, 256), (777, 1)):
        s = np.round(rng.standard_normal(n), 2)  # ties
        order = np.lexsort((np.arange(n), -s))
        assert oracle.topk(s, k).tolist() == sorted(order[:k].tolist()), f"lexsort n={n} k={k}"
        assert oracle.topk(s, 1).tolist() == [int(np.argmax(s))], "first argmax"
        assert oracle.topk(s, n).tolist() == list(range(n)), "k = n"
    s = np.array([0.0, -0.0, 0.0, -1.0, -0.0])
    assert oracle.topk(s, 2).tolist() == [0, 1], "-0.0 and +0.0 tie"
    assert oracle.topk(s, 4).tolist() == [0, 1, 2, 4], "-0.0 and +0.0 tie"


def pin_union_bruteforce():
    """Union of per-query top-k sets equals the Python set union of brute-force
    sets, and obeys max|S_j| <= |U| <= min(sum |S_j|, n)."""
    rng = np.random.default_rng(6)
    for _ in range(20):
        n, Q = int(rng.integers(4, 12)), int(rng.integers(2, 5))
        k = int(rng.integers(1, n + 1))
        lists = []
        for _ in range(Q):
            s = rng.integers(-2, 3, size=n).astype(np.float64)
            lists.append(sorted(np.lexsort((np.arange(n), -s))[:k].tolist()))
        u = oracle.union(np.array(lists), n).tolist()
        assert u == sorted(set().union(*map(set, lists))), "union"
        assert k <= len(u) <= min(Q * k, n)


def pin_planted_selected(name: str, seeds=(0,)):
    """Planted high-similarity chunks are always in the kept set."""
    for seed in seeds:
        prob = synth.make_problem(name, seed)
        inp = synth.host_inputs(prob, seed)
        for b in range(prob.batch):
            _, _, kept = oracle.select_for_sequence(prob, inp, b)
            missing = set(inp["planted"][b].tolist()) - set(kept.tolist())
            assert not missing, f"{name} seed {seed} seq {b}: planted chunks {sorted(missing)} not kept"


# ---------------------------------------------------------------- attention
def pin_attention_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "attention_worked.json")))
    out, lse = oracle.attention(_bf16(g["q"]), _bf16(g["K"]), _bf16(g["V"]), np.array(g["kept"]), g["chunk"],
                                g["scale"])
    assert np.allclose(out, g["out"], rtol=1e-14, atol=0), "worked attention output"
    assert np.allclose(lse, g["lse"], rtol=1e-14, atol=0), "worked attention lse"


def _rand_head(rng, n_tok, d, scale_k=1.0):
    return _bf16(rng.standard_normal((n_tok, d)) * scale_k), _bf16(rng.standard_normal((n_tok, d)))


def pin_keep_all_is_dense():
    """With every chunk kept the result is plain dense attention (the paper's
    cold start keeps all chunks resident and matches the baseline exactly),
    computed here with scipy's softmax and a numpy matmul."""
    rng = np.random.default_rng(7)
    for (n_chunks, C, d, R) in ((6, 4, 16, 3), (3, 64, 128, 2)):
        K, V = _rand_head(rng, n_chunks * C, d, 0.5)
        q = _bf16(rng.standard_normal((R, d)))
        scale = 1.0 / math.sqrt(d)
        out, lse = oracle.attention(q, K, V, np.arange(n_chunks), C, scale)
        logits = (_f64(q) @ _f64(K).T) * scale
        ref = scipy.special.softmax(logits, axis=1) @ _f64(V)
        assert np.allclose(out, ref, rtol=1e-12, atol=1e-14), "keep-all != dense"
        assert np.allclose(lse, scipy.special.logsumexp(logits, axis=1), rtol=1e-13), "keep-all lse"


def pin_masked_dense_sdpa():
    """Kept-chunk attention equals PyTorch's float64 scaled_dot_product_attention
    with a boolean mask that hides the tokens of the dropped chunks."""
    rng = np.random.default_rng(8)
    n_chunks, C, d, R = 10, 8, 32, 4
    K, V = _rand_head(rng, n_chunks * C, d, 1.5)  # sharp softmax
    q = _bf16(rng.standard_normal((R, d)))
    kept = np.array([1, 4, 5, 9])
    out, _ = oracle.attention(q, K, V, kept, C, None)
    mask = torch.zeros(R, n_chunks * C, dtype=torch.bool)
    for c in kept:
        mask[:, c * C:(c + 1) * C] = True
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(_f64(q))[None], torch.from_numpy(_f64(K))[None], torch.from_numpy(_f64(V))[None],
        attn_mask=mask[None])[0].numpy()
    assert np.allclose(out, ref, rtol=1e-12, atol=1e-14), "masked dense"


def pin_attention_closed_forms():
    """Constant V returns that constant; q = 0 returns the mean of the kept V
    rows and lse = log(#kept tokens); identical keys do the same for any q;
    a single kept token returns its own V row."""
    rng = np.random.default_rng(9)
    n_chunks, C, d = 7, 4, 16
    K, V = _rand_head(rng, n_chunks * C, d)
    kept = np.array([0, 3, 6])
    toks = np.concatenate([np.arange(c * C, (c + 1) * C) for c in kept])
    const = _bf16(np.full((n_chunks * C, d), 0.375))
    out, _ = oracle.attention(_bf16(rng.standard_normal((2, d))), K, const, kept, C)
    assert np.allclose(out, 0.375, rtol=1e-14), "constant V"
    out, lse = oracle.attention(_bf16(np.zeros((1, d))), K, V, kept, C)
    assert np.allclose(out[0], _f64(V)[toks].mean(axis=0), rtol=1e-12, atol=1e-14), "q = 0 mean"
    assert abs(lse[0] - math.log(len(toks))) < 1e-13, "q = 0 lse"
    Ksame = np.tile(K[:1], (n_chunks * C, 1))
    out, _ = oracle.attention(_bf16(rng.standard_normal((1, d))), Ksame, V, kept, C)
    assert np.allclose(out[0], _f64(V)[toks].mean(axis=0), rtol=1e-12, atol=1e-14), "equal keys mean"
    out, lse = oracle.attention(_bf16(rng.standard_normal((1, d))), K, V, np.array([5]), 1)
    assert np.array_equal(out[0], _f64(V)[5]), "single token"


def pin_gqa_mapping():
    """Query head h reads KV head floor(h / G): KV head g holds constant V = g + 1."""
    prob = synth.Problem("gqa", [256], 64, [2], n_q_heads=8, n_kv_heads=2, head_dim=32, emb_dim=64,
                         emb_dtype="f32")
    rng = np.random.default_rng(10)
    inp = {"q": _bf16(rng.standard_normal((1, 1, 8, 32))).reshape(1, 1, 8, 32)}

    def kv(which, b, g, chunks):
        if which == "v":
            return _bf16(np.full((256, 32), g + 1.0))
        return _bf16(rng.standard_normal((256, 32)))

    res = oracle.attend_rows(prob, inp, 0, np.array([0, 3]), [(0, h) for h in range(8)], kv)
    for h in range(8):
        assert np.allclose(res[(0, h)][0], h // 4 + 1.0), f"head {h} must read KV head {h // 4}"


def pin_attention_empty_set():
    """An empty kept set (only the recall path can produce one) gives the empty
    sum: out = 0 and lse = -inf."""
    rng = np.random.default_rng(11)
    K, V = _rand_head(rng, 16, 8)
    out, lse = oracle.attention(_bf16(rng.standard_normal((3, 8))), K, V, np.array([], dtype=np.int32), 4)
    assert np.array_equal(out, np.zeros((3, 8))), "empty set output"
    assert np.all(np.isneginf(lse)), "empty set lse"


# ------------------------------------------------------------------- recall
def pin_recall_worked_example():
    """Hand-worked two-layer example: scores, the threshold at exactly 0, the OR
    over layers and the K_max bound."""
    g = json.load(open(os.path.join(GOLDEN, "recall_worked.json")))
    q, K = _bf16(g["q"]), _bf16(g["K"])
    x = np.stack([oracle.index_score(q, np.array(w, dtype=np.float32), K) for w in g["w"]])
    assert np.array_equal(x, np.array(g["x"])), "worked index scores"
    for case in g["cases"]:
        got = oracle.recall(x[case["layers"]], case["kmax"])
        assert got.tolist() == case["kept"], f"worked recall {case}"


def pin_index_score_single_head():
    """One head with unit gate is ReLU of the dual-encoder dot product (the
    already pinned O1 score); a gate w scales it by w."""
    rng = np.random.default_rng(12)
    K = _bf16(rng.standard_normal((40, 64)))
    q = _bf16(rng.standard_normal((1, 64)))
    dot = oracle.score(q[0], K, "bf16")
    for w in (1.0, -0.75, 2.5):
        x = oracle.index_score(q, np.array([w], dtype=np.float32), K)
        assert np.array_equal(x, w * np.maximum(dot, 0.0)), f"single head, w = {w}"


def pin_index_score_relu_identities():
    """ReLU(a) - ReLU(-a) = a and ReLU(a) + ReLU(-a) = |a| turn the score into
    plain matrix products: x(q) - x(-q) = K (w Q) and x(q) + x(-q) = |K Q^T| w
    (numpy, float64, on the widened bf16 values)."""
    rng = np.random.default_rng(13)
    for n_h, c in ((16, 64), (64, 128), (3, 8)):
        Q = _bf16(rng.standard_normal((n_h, c)))
        K = _bf16(rng.standard_normal((50, c)))
        w = rng.standard_normal(n_h).astype(np.float32)
        xp = oracle.index_score(Q, w, K)
        xm = oracle.index_score(Q ^ np.uint16(0x8000), w, K)  # -q: flip the bf16 sign bits
        Qf, Kf, wf = _f64(Q), _f64(K), w.astype(np.float64)
        assert np.allclose(xp - xm, Kf @ (wf @ Qf), rtol=1e-10, atol=1e-10), f"x(q) - x(-q), n_h={n_h}"
        assert np.allclose(xp + xm, np.abs(Kf @ Qf.T) @ wf, rtol=1e-10, atol=1e-10), f"x(q) + x(-q), n_h={n_h}"


def pin_index_score_head_permutation():
    """Heads are a sum: permuting (q_h, w_h) pairs together leaves x unchanged."""
    rng = np.random.default_rng(14)
    Q = _bf16(rng.standard_normal((32, 64)))
    K = _bf16(rng.standard_normal((30, 64)))
    w = rng.standard_normal(32).astype(np.float32)
    perm = rng.permutation(32)
    a = oracle.index_score(Q, w, K)
    b = oracle.index_score(Q[perm], w[perm], K)
    assert np.allclose(a, b, rtol=1e-12, atol=1e-12), "head permutation"


def pin_recall_sigmoid_threshold():
    """One layer, no bound: the recalled set is {s : sigmoid(x_s) >= 1/2}
    (scipy's expit), including x = +0.0 and -0.0."""
    rng = np.random.default_rng(15)
    x = rng.standard_normal(500)
    x[np.abs(x) < 1e-6] = 1e-3
    x[::37] = 0.0
    x[5::41] = -0.0
    want = np.nonzero(scipy.special.expit(x) >= 0.5)[0]
    assert oracle.recall(x[None, :], len(x)).tolist() == want.tolist(), "sigmoid threshold"


def pin_recall_or_bruteforce():
    """OR over layers is the Python set union of the per-layer recalls; with a
    bound, brute force over all subsets of the union: the kept set has the
    largest sum of max_l x and, among those, the smallest ascending id list."""
    rng = np.random.default_rng(16)
    for _ in range(80):
        L, n = int(rng.integers(1, 5)), int(rng.integers(1, 11))
        x = rng.integers(-3, 3, size=(L, n)).astype(np.float64)
        union = sorted(set().union(*[{s for s in range(n) if x[l, s] >= 0} for l in range(L)]))
        assert oracle.recall(x, n).tolist() == union, f"OR over layers, x={x.tolist()}"
        r = x.max(axis=0)
        for kmax in range(1, n + 1):
            if len(union) <= kmax:
                want = union
            else:
                want, best = None, -math.inf
                for comb in itertools.combinations(union, kmax):
                    tot = r[list(comb)].sum()
                    if tot > best:
                        want, best = list(comb), tot
            assert oracle.recall(x, kmax).tolist() == want, f"bound {kmax}, x={x.tolist()}"


def pin_recall_boundaries():
    """Cases the paper's threshold fixes: with every gate >= 0 every entry is
    recalled; when every head's ReLU is 0 the score is exactly 0 and the entry
    is recalled (sigmoid(0) = 1/2); with heads q and -q and negative gates every
    score is < 0 and nothing is recalled."""
    rng = np.random.default_rng(17)
    Q = _bf16(rng.standard_normal((8, 32)))
    K = _bf16(rng.standard_normal((25, 32)))
    x = oracle.index_score(Q, np.abs(rng.standard_normal(8)).astype(np.float32), K)
    assert oracle.recall(x[None, :], 25).tolist() == list(range(25)), "non-negative gates recall all"
    Kneg = _bf16(-np.abs(rng.standard_normal((25, 32))))
    Qpos = _bf16(np.abs(rng.standard_normal((8, 32))))
    x = oracle.index_score(Qpos, rng.standard_normal(8).astype(np.float32), Kneg)
    assert np.array_equal(x, np.zeros(25)), "all ReLUs zero"
    assert oracle.recall(x[None, :], 25).tolist() == list(range(25)), "score 0 is on the threshold"
    q0 = rng.standard_normal((1, 32))
    Qpm = _bf16(np.concatenate([q0, -q0]))
    x = oracle.index_score(Qpm, np.array([-1.0, -1.0], dtype=np.float32), K)
    assert np.all(x < 0), "q and -q with negative gates"
    assert oracle.recall(x[None, :], 25).tolist() == [], "nothing recalled"


# ---------------------------------------------------------------- two-level
def pin_attention_tokens_reduces_to_chunks():
    """Token-list attention equals the pinned chunk attention: with whole chunks
    on the chunk list, and token by token as chunks of one token; a single token
    returns its V row; the empty list is the empty sum."""
    rng = np.random.default_rng(18)
    n_chunks, C, d = 6, 8, 16
    K, V = _rand_head(rng, n_chunks * C, d)
    q = _bf16(rng.standard_normal((3, d)))
    kept = np.array([0, 2, 5])
    toks = np.concatenate([np.arange(c * C, (c + 1) * C) for c in kept])
    a, la = oracle.attention_tokens(q, K, V, toks)
    b, lb = oracle.attention(q, K, V, kept, C)
    assert np.array_equal(a, b) and np.array_equal(la, lb), "whole chunks"
    part = np.concatenate([toks, np.arange(3 * C, 3 * C + 5)])  # a partial chunk of 5 tokens
    a, la = oracle.attention_tokens(q, K, V, part)
    b, lb = oracle.attention(q, K, V, part.astype(np.int32), 1)
    assert np.array_equal(a, b) and np.array_equal(la, lb), "token by token"
    a, _ = oracle.attention_tokens(q, K, V, np.array([11]))
    assert np.array_equal(a, np.tile(_f64(V)[11], (3, 1))), "single token"
    a, la = oracle.attention_tokens(q, K, V, np.zeros(0, dtype=np.int64))
    assert np.array_equal(a, np.zeros((3, d))) and np.all(np.isneginf(la)), "empty list"


def pin_two_level_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "two_level_worked.json")))
    for case in g["cases"]:
        got = oracle.two_level(np.array(g["recalled"]), np.array(g["native"], dtype=np.float64), case["k2"], g["w0"],
                               g["n_total"])
        assert got.tolist() == case["kept"], f"worked two-level, k2={case['k2']}"


def pin_two_level_bruteforce():
    """Level 2 keeps, among all k2-subsets of the recalled ids, the one with the
    largest native-score sum and, among those, the smallest ascending id list
    (all recalled ids when there are at most k2); the window chunks are always
    appended; nothing recalled leaves the window alone."""
    rng = np.random.default_rng(19)
    for _ in range(80):
        n_hist = int(rng.integers(0, 9))
        n_total = n_hist + int(rng.integers(0, 4))
        native = rng.integers(-2, 3, size=n_hist).astype(np.float64)
        rec = sorted(rng.choice(n_hist, size=int(rng.integers(0, n_hist + 1)), replace=False).tolist()) \
            if n_hist else []
        k2 = int(rng.integers(1, 6))
        if len(rec) <= k2:
            core = rec
        else:
            core, best = None, -math.inf
            for comb in itertools.combinations(rec, k2):
                tot = native[list(comb)].sum()
                if tot > best:
                    core, best = list(comb), tot
        want = core + list(range(n_hist, n_total))
        got = oracle.two_level(np.array(rec, dtype=np.int32), native, k2, n_hist, n_total).tolist()
        assert got == want, f"two-level brute force rec={rec} native={native.tolist()} k2={k2}"


def pin_window_worked_example():
    """The hand-worked windows of tests/golden/window_worked.json (tails of 1 to
    63 tokens, windows of 0, 1, 64, 65 tokens and wider than the context, both
    chunk sizes, the 1M-token two-level workload)."""
    g = json.load(open(os.path.join(GOLDEN, "window_worked.json")))
    for case in g["cases"]:
        got = oracle.window(case["ctx"], case["window"], case["chunk"])
        assert got == (case["w0"], case["n_total"], case["tail"]), (case, got)


def pin_window_token_count():
    """On random shapes: the window and the history partition the chunks; the
    window holds every one of the last window_tokens tokens and every token of
    a partial last chunk; the history's chunks are all complete, and its last
    one holds no recent token."""
    rng = np.random.default_rng(23)
    for _ in range(300):
        C = int(rng.choice([64, 128]))
        ctx = int(rng.integers(1, 40 * C))
        W = int(rng.choice([0, rng.integers(0, 3 * C), rng.integers(0, 50 * C)]))
        w0, n_total, tail = oracle.window(ctx, W, C)
        assert n_total * C >= ctx > (n_total - 1) * C and tail == ctx - (n_total - 1) * C
        assert 0 <= w0 <= n_total
        assert w0 * C <= max(ctx - W, 0) or w0 == 0, "a history chunk holds a recent token"
        if w0 < n_total:
            assert (w0 + 1) * C > ctx - W or (tail < C and w0 == n_total - 1), "the first window chunk is needed"
        assert w0 * C <= ctx and (w0 < n_total or ctx % C == 0), "a partial chunk is in the history"


# ---------------------------------------------------------------- host tier
def pin_tier_plan_invariants():
    """What the reserve must guarantee, checked on random firings: every kept
    chunk ends up in exactly one slot; a chunk already resident is not copied
    again; no slot the previous kept set reads is given to another chunk; the
    copies are exactly the kept chunks that were not resident; an empty reserve
    fills its slots in ascending order."""
    rng = np.random.default_rng(20)
    for trial in range(60):
        n, kmax = int(rng.integers(1, 40)), int(rng.integers(1, 8))
        n_slots = 2 * min(kmax, n) + int(rng.integers(0, 3))
        owner = [-1] * n_slots
        old = []
        for firing in range(6):
            kept = sorted(rng.choice(n, size=int(rng.integers(0, min(kmax, n) + 1)), replace=False).tolist())
            before = list(owner)
            owner, slots, fetch = oracle.tier_plan(owner, old, kept)
            assert len(slots) == len(kept) and len(set(slots)) == len(slots), "one slot per kept chunk"
            assert all(owner[s] == c for c, s in zip(kept, slots)), "the slot holds its chunk"
            assert sorted(c for c in owner if c >= 0) == sorted(set(c for c in owner if c >= 0)), "no chunk twice"
            resident = {c for c in before if c >= 0}
            assert [c for c, _ in fetch] == [c for c in kept if c not in resident], "copies = kept, not resident"
            for s in old:
                assert owner[s] == before[s], "a slot the previous set reads was reassigned"
            for c, s in zip(kept, slots):
                if c in resident:
                    assert before[s] == c, "a resident chunk moved"
            if firing == 0 and trial % 2 == 0:
                assert slots == list(range(len(kept))), "empty reserve fills from slot 0"
            old = slots
    # too small a reserve is an error
    try:
        oracle.tier_plan([-1], [0], [3])
        raise AssertionError("no free slot must raise")
    except ValueError:
        pass


def pin_tier_plan_worked_example():
    """The hand-worked firings of tests/golden/tier_plan_worked.json: resident
    chunks keep their slots, slots of the previous set stay protected, free
    slots go out in ascending order after reuse, a reserve too small raises."""
    g = json.load(open(os.path.join(GOLDEN, "tier_plan_worked.json")))
    owner, old = [-1] * g["slots"], []
    for f in g["firings"]:
        if f.get("too_small"):
            try:
                oracle.tier_plan(owner, old, f["kept"])
            except ValueError:
                continue
            raise AssertionError("a reserve too small must raise")
        owner, slots, fetch = oracle.tier_plan(owner, old, f["kept"])
        assert owner == f["owner"] and slots == f["slot_idx"], (f, owner, slots)
        assert [list(x) for x in fetch] == f["fetch"], (f, fetch)
        old = slots


def pin_tier_plan_bruteforce():
    """After a few random firings (so the reserve is partly full): among every
    assignment of the missing kept chunks (ascending) to distinct slots that
    neither hold a kept chunk nor are read by the previous set, the plan makes
    the lexicographically smallest one; resident chunks keep their slots."""
    rng = np.random.default_rng(29)
    checked = 0
    for trial in range(120):
        n, n_slots = int(rng.integers(2, 12)), int(rng.integers(2, 8))
        owner, old = [-1] * n_slots, []
        for firing in range(4):
            kept = sorted(rng.choice(n, size=int(rng.integers(0, min(n, n_slots // 2) + 1)), replace=False).tolist())
            where = {c: s for s, c in enumerate(owner) if c >= 0}
            taken = set(old) | {where[c] for c in kept if c in where}
            missing = [c for c in kept if c not in where]
            cands = [s for s in range(n_slots) if s not in taken]
            best = min(itertools.permutations(cands, len(missing)), default=None)
            try:
                new_owner, slots, fetch = oracle.tier_plan(owner, old, kept)
            except ValueError:
                assert best is None, "a plan exists but the oracle raised"
                break
            assert best is not None
            assert [s for _, s in fetch] == list(best) and [c for c, _ in fetch] == missing
            assert all(slots[i] == where[c] for i, c in enumerate(kept) if c in where)
            owner, old = new_owner, slots
            checked += firing > 0
    assert checked > 100


# ------------------------------------------------------------ golden labels
def _golden_logits(weights) -> np.ndarray:
    return np.log(np.asarray(weights, dtype=np.float64)).astype(np.float32)


def pin_golden_worked_example():
    """The hand-worked window of tests/golden/golden_labels_worked.json."""
    g = json.load(open(os.path.join(GOLDEN, "golden_labels_worked.json")))
    logits = _golden_logits(g["weights"])
    for case in g["cases"]:
        labels, sizes, golden = oracle.golden_labels(logits, g["p_num"], g["p_den"], case["theta"])
        assert labels.tolist() == case["labels"], (case, labels)
        assert sizes.tolist() == g["nucleus_size"], sizes
        assert golden.tolist() == case["golden_count"], golden


def _numpy_nucleus(S: np.ndarray, p: float):
    """Top-p set from numpy: float64 softmax, stable sort by (logit desc, index
    asc), cumulative mass; returns (set, cumulative masses in that order)."""
    P = scipy.special.softmax(S.astype(np.float64))
    order = np.lexsort((np.arange(len(S)), -S.astype(np.float64)))
    cum = np.cumsum(P[order])
    size = int(np.searchsorted(cum, p - 0.0, side="left")) + 1
    size = min(size, len(S))
    return set(order[:size].tolist()), cum


def pin_top_p_library_softmax():
    """Random rows against scipy's softmax, numpy's stable sort and cumulative
    sum.  The two may differ only where numpy's cumulative mass sits within
    1e-12 of p at the cut (float64 rounding of the two sums)."""
    rng = np.random.default_rng(41)
    for trial in range(300):
        n = int(rng.integers(1, 3000))
        scale = float(rng.choice([0.05, 0.5, 1.0, 3.0, 10.0, 30.0]))
        S = (rng.standard_normal(n) * scale).astype(np.float32)
        if trial % 5 == 0:  # many exact ties
            S = np.round(S * 2.0).astype(np.float32) / np.float32(2.0)
        num, den = [(3, 5), (1, 2), (9, 10), (1, 100), (99, 100), (1, 1)][trial % 6]
        mark, size = oracle.top_p(S, num, den)
        want, cum = _numpy_nucleus(S, num / den)
        got = set(np.nonzero(mark)[0].tolist())
        assert size == len(got)
        if got != want:
            k = len(want)
            near = abs(cum[k - 1] - num / den) <= 1e-12 or (k >= 2 and abs(cum[k - 2] - num / den) <= 1e-12)
            assert near, (trial, n, scale, len(got), len(want))


def pin_top_p_bruteforce():
    """Tiny rows: over all subsets whose probability mass reaches p, the
    smallest ones; among those the most probable; among equals the
    lexicographically smallest index list -- the top-p set by its own
    definition, in exact rational arithmetic over the float64 weights
    exp(S - max S).  Rows where some subset's mass lies within 1e-12 of p
    (but not on it) are skipped: there float64 sums may round either way."""
    from fractions import Fraction
    rng = np.random.default_rng(43)
    checked = 0
    for trial in range(400):
        n = int(rng.integers(1, 8))
        if trial % 3 == 0:  # a coarse grid of logits: ties, masses that are exact multiples
            S = (rng.integers(-4, 3, size=n) * 0.5).astype(np.float32)
        else:
            S = (rng.standard_normal(n) * float(rng.choice([0.3, 1.0, 3.0]))).astype(np.float32)
        num, den = [(3, 5), (1, 2), (2, 3), (1, 7), (6, 7), (1, 1)][trial % 6]
        p = Fraction(num, den)
        m = max(float(x) for x in S)
        wts = [Fraction(math.exp(float(x) - m)) for x in S]
        tot = sum(wts)
        masses = {}
        best = None
        for mask in range(1, 1 << n):
            idx = [s for s in range(n) if mask >> s & 1]
            mass = sum(wts[s] for s in idx) / tot
            masses[mask] = mass
            if mass < p:
                continue
            key = (len(idx), -mass, idx)
            if best is None or key < best[0]:
                best = (key, idx)
        if any(0 < abs(float(x - p)) < 1e-12 for x in masses.values()):
            continue
        mark, size = oracle.top_p(S, num, den)
        assert np.nonzero(mark)[0].tolist() == best[1], (S.tolist(), num, den, best[1])
        assert size == len(best[1])
        checked += 1
    assert checked > 200


def pin_top_p_boundaries():
    """Equal logits make every mass exact: a set that reaches p exactly is
    enough (3 of 5 equal entries at p = 3/5, the lower indices); the most
    probable entry alone when it exceeds p; at p = 1 every entry, however small
    its weight; the first maximum alone for a tiny p; and the order of the
    prefix with its mass fractions."""
    mark, size = oracle.top_p(np.zeros(5, np.float32), 3, 5)
    assert mark.tolist() == [1, 1, 1, 0, 0] and size == 3
    mark, size = oracle.top_p(np.zeros(5, np.float32), 61, 100)
    assert size == 4
    mark, size = oracle.top_p(np.array([0.0, 5.0, 1.0], np.float32), 3, 5)
    assert mark.tolist() == [0, 1, 0]
    S = np.array([0.0, -40.0, -1.0, 0.0], np.float32)
    mark, size = oracle.top_p(S, 1, 1)  # every weight is positive: p = 1 needs them all
    assert mark.tolist() == [1, 1, 1, 1] and size == 4
    mark, size = oracle.top_p(np.array([2.0, 3.0, 3.0, -0.0, 0.0], np.float32), 1, 1 << 30)
    assert mark.tolist() == [0, 1, 0, 0, 0]
    # order (logit desc, index asc; -0.0 equal to +0.0) and prefix masses
    mark, size, order, cum = oracle.top_p(np.array([0.0, 1.0, -0.0, 1.0], np.float32), 1, 2, detail=True)
    assert order.tolist() == [1, 3, 0, 2]
    e = math.e
    assert np.allclose(cum, [e / (2 * e + 2), 2 * e / (2 * e + 2), (2 * e + 1) / (2 * e + 2), 1.0], rtol=1e-15)
    assert size == 2 and mark.tolist() == [0, 1, 0, 1]  # 2e / (2e + 2) = 0.731 >= 1/2, e / (2e + 2) < 1/2


def pin_golden_votes_and_union():
    """Eqs. 9-11 as indicator-matrix arithmetic over the oracle's own top-p sets
    (themselves pinned above): votes are column sums over layers, the golden
    set is votes >= theta, the label set the OR over steps; theta = 1 gives the
    union of every set, theta > L the empty set."""
    rng = np.random.default_rng(47)
    for trial in range(40):
        tau, L, n = int(rng.integers(1, 5)), int(rng.integers(1, 7)), int(rng.integers(1, 300))
        logits = (rng.standard_normal((tau, L, n)) * rng.choice([0.5, 2.0, 6.0])).astype(np.float32)
        num, den = (3, 5) if trial % 2 else (1, 3)
        M = np.stack([np.stack([oracle.top_p(logits[i, l], num, den)[0] for l in range(L)]) for i in range(tau)])
        votes = M.astype(np.int64).sum(axis=1)                      # [tau][n]
        for theta in (1, 2, 3, L, L + 1):
            labels, sizes, golden = oracle.golden_labels(logits, num, den, theta)
            A = votes >= theta
            assert labels.tolist() == np.nonzero(A.any(axis=0))[0].tolist()
            assert golden.tolist() == A.sum(axis=1).tolist()
            assert sizes.tolist() == M.sum(axis=2).tolist()
            if theta == 1:
                assert labels.tolist() == np.nonzero(M.any(axis=(0, 1)))[0].tolist()
            if theta > L:
                assert len(labels) == 0


ALL_PINS = [
    pin_score_library_matmul, pin_score_int8_exact, pin_score_closed_forms,
    pin_topk_worked_example, pin_topk_bruteforce, pin_topk_library_sort, pin_union_bruteforce,
    pin_attention_worked_example, pin_keep_all_is_dense, pin_masked_dense_sdpa, pin_attention_closed_forms,
    pin_gqa_mapping, pin_attention_empty_set,
    pin_recall_worked_example, pin_index_score_single_head, pin_index_score_relu_identities,
    pin_index_score_head_permutation, pin_recall_sigmoid_threshold, pin_recall_or_bruteforce,
    pin_recall_boundaries, pin_attention_tokens_reduces_to_chunks, pin_two_level_worked_example,
    pin_two_level_bruteforce, pin_window_worked_example, pin_window_token_count, pin_tier_plan_invariants,
    pin_tier_plan_worked_example, pin_tier_plan_bruteforce,
    pin_golden_worked_example, pin_top_p_library_softmax, pin_top_p_bruteforce,
    pin_top_p_boundaries, pin_golden_votes_and_union,
]
