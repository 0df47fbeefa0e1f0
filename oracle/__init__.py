"""CPU oracle for the LSA decode hot path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline leg
may import this package.  It wraps ``lsa_oracle.c`` (float64 / int64, plain
loops) and composes its three functions in the paper's order for one decode
step:

* O1 score -- Memory Indexer score, Sec. 2.1 Eq. 4, read as the dual-encoder dot
  product (one head, unit gate);
* O2 select -- top-k with lowest-index tie-break, ascending output; union of the
  per-query sets for several lookahead queries (Sec. 2.1 Eq. 6 and
  Sec. 2.4 Eq. 13; K_max of Sec. 2.5 is the keep budget);
* O3 attend -- softmax(q K^T * scale) V over the tokens of the kept chunks
  (an empty kept set gives out = 0, lse = -inf).

and the golden-label pipeline of Sec. 2.2 (softmax, top-p set, vote over
layers, golden set, union over the window; Eqs. 7-11), and, for the recall
path, the full Memory Indexer in the paper's order:

* R1 index score -- x = sum_h w_h ReLU(q_h . K_s) per indexer layer (the
  argument of the sigmoid of Sec. 2.1 Eq. 4);
* R2 recall -- sigmoid(x) >= 1/2 per layer (Eq. 5), OR over the layers
  (Eq. 13), at most K_max entries (Sec. 2.5), then O3 over the recalled set.

It shares no code with the HIP library; the only common input is the seeded
generator in ``lsa_synth``.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# LSA_ORACLE_SO points the tests at another build of the same source (the
# sanitised one); by default the in-tree library is used.
_SO = os.environ.get("LSA_ORACLE_SO") or os.path.join(_HERE, "liblsa_oracle.so")
_lib: Optional[ctypes.CDLL] = None

_P = ctypes.c_void_p
_I32, _I64, _F64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double


def build() -> None:
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fno-fast-math",
                           os.path.join(_HERE, "lsa_oracle.c"), "-o", os.path.join(_HERE, "liblsa_oracle.so"),
                           "-lm"])


def bind(path: str) -> ctypes.CDLL:
    """Load an oracle shared object and declare its signatures."""
    L = ctypes.CDLL(path)
    L.oracle_score_f32.argtypes = [_P, _P, _I64, _I32, _P]
    L.oracle_score_bf16.argtypes = [_P, _P, _I64, _I32, _P]
    L.oracle_score_i8.argtypes = [_P, _P, _I64, _I32, _P]
    for f in (L.oracle_score_f32, L.oracle_score_bf16, L.oracle_score_i8):
        f.restype = None
    L.oracle_topk_f64.argtypes = [_P, _I64, _I64, _P]
    L.oracle_topk_f64.restype = _I64
    L.oracle_topk_i64.argtypes = [_P, _I64, _I64, _P]
    L.oracle_topk_i64.restype = _I64
    L.oracle_union.argtypes = [_P, _I32, _I64, _I64, _P]
    L.oracle_union.restype = _I64
    L.oracle_attention.argtypes = [_P, _I32, _P, _P, _I64, _I32, _I32, _P, _I64, _F64, _P, _P]
    L.oracle_attention.restype = ctypes.c_int
    L.oracle_index_score_bf16.argtypes = [_P, _P, _P, _I64, _I32, _I32, _P]
    L.oracle_index_score_bf16.restype = None
    L.oracle_recall.argtypes = [_P, _I32, _I64, _I64, _P]
    L.oracle_recall.restype = _I64
    L.oracle_attention_tokens.argtypes = [_P, _I32, _P, _P, _I64, _I32, _P, _I64, _F64, _P, _P]
    L.oracle_attention_tokens.restype = ctypes.c_int
    L.oracle_two_level.argtypes = [_P, _I64, _P, _I64, _I64, _I64, _I64, _P]
    L.oracle_two_level.restype = _I64
    L.oracle_top_p.argtypes = [_P, _I64, _I64, _I64, _P, _P, _P]
    L.oracle_top_p.restype = _I64
    L.oracle_golden_labels.argtypes = [_P, _I32, _I32, _I64, _I64, _I64, _I32, _P, _P, _P]
    L.oracle_golden_labels.restype = _I64
    return L


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        _lib = bind(_SO)
    return _lib


def _c(a: np.ndarray, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


# ------------------------------------------------------------------ O1 score
def score(qe: np.ndarray, E: np.ndarray, emb_dtype: str) -> np.ndarray:
    """Scores of one query embedding qe [D] against chunk embeddings E [n][D].

    float64 for 'f32' / 'bf16' (bf16 given as uint16 bit patterns), int64 for 'i8'.
    """
    n, D = E.shape
    if emb_dtype == "i8":
        out = np.empty(n, dtype=np.int64)
        qe, E = _c(qe, np.int8), _c(E, np.int8)
        lib().oracle_score_i8(qe.ctypes.data, E.ctypes.data, n, D, out.ctypes.data)
        return out
    out = np.empty(n, dtype=np.float64)
    if emb_dtype == "f32":
        qe, E = _c(qe, np.float32), _c(E, np.float32)
        lib().oracle_score_f32(qe.ctypes.data, E.ctypes.data, n, D, out.ctypes.data)
    elif emb_dtype == "bf16":
        qe, E = _c(qe, np.uint16), _c(E, np.uint16)
        lib().oracle_score_bf16(qe.ctypes.data, E.ctypes.data, n, D, out.ctypes.data)
    else:
        raise ValueError(emb_dtype)
    return out


# ----------------------------------------------------------------- O2 select
def topk(s: np.ndarray, k: int) -> np.ndarray:
    """The k chunk ids with the largest scores (lower id wins ties), ascending."""
    n = len(s)
    out = np.empty(k, dtype=np.int32)
    if s.dtype == np.int64:
        s = _c(s, np.int64)
        r = lib().oracle_topk_i64(s.ctypes.data, n, k, out.ctypes.data)
    else:
        s = _c(s, np.float64)
        r = lib().oracle_topk_f64(s.ctypes.data, n, k, out.ctypes.data)
    if r != k:
        raise ValueError(f"oracle_topk rejected n={n} k={k}")
    return out


def union(lists: np.ndarray, n: int) -> np.ndarray:
    """Ascending union of the rows of ``lists`` [n_lists][k]."""
    lists = _c(lists, np.int32)
    out = np.empty(n, dtype=np.int32)
    u = lib().oracle_union(lists.ctypes.data, lists.shape[0], lists.shape[1], n, out.ctypes.data)
    if u < 0:
        raise ValueError("oracle_union rejected its input")
    return out[:u].copy()


# ------------------------------------------------------------------ O3 attend
def attention(q_rows: np.ndarray, Kh: np.ndarray, Vh: np.ndarray, sel: np.ndarray, chunk: int,
              scale: Optional[float] = None):
    """Attention of q_rows [R][d] over the tokens of chunks ``sel`` of one KV head.

    Kh, Vh are logical token-major [n_tok][d] bf16 bit patterns.  Returns
    (out [R][d] float64, lse [R] float64).
    """
    R, d = q_rows.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    q_rows, Kh, Vh = _c(q_rows, np.uint16), _c(Kh, np.uint16), _c(Vh, np.uint16)
    sel = _c(sel, np.int32)
    out = np.empty((R, d), dtype=np.float64)
    lse = np.empty(R, dtype=np.float64)
    rc = lib().oracle_attention(q_rows.ctypes.data, R, Kh.ctypes.data, Vh.ctypes.data, Kh.shape[0], d, chunk,
                                sel.ctypes.data, len(sel), float(scale), out.ctypes.data, lse.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_attention rejected its input")
    return out, lse


# ------------------------------------------------------------ R1 / R2 recall
def index_score(q: np.ndarray, w: np.ndarray, K: np.ndarray) -> np.ndarray:
    """x[s] = sum_h w[h] ReLU(q[h] . K[s]) in float64 (Sec. 2.1 Eq. 4 before the
    sigmoid).  q [n_h][c] and K [n][c] are bf16 bit patterns, w [n_h] float32."""
    n_h, c = q.shape
    n = K.shape[0]
    q, K, w = _c(q, np.uint16), _c(K, np.uint16), _c(w, np.float32)
    out = np.empty(n, dtype=np.float64)
    lib().oracle_index_score_bf16(q.ctypes.data, w.ctypes.data, K.ctypes.data, n, n_h, c, out.ctypes.data)
    return out


def recall(x: np.ndarray, kmax: int) -> np.ndarray:
    """Recalled entry ids, ascending, from the sigmoid arguments x [L][n]
    (threshold 1/2 per layer, OR over layers, at most kmax entries)."""
    x = _c(np.atleast_2d(x), np.float64)
    L, n = x.shape
    out = np.empty(n, dtype=np.int32)
    m = lib().oracle_recall(x.ctypes.data, L, n, kmax, out.ctypes.data)
    if m < 0:
        raise ValueError(f"oracle_recall rejected L={L} n={n} kmax={kmax}")
    return out[:m].copy()


def recall_for_sequence(prob, inputs: Dict[str, object], b: int):
    """R1 then R2 for sequence b: returns (x [L][n_b], recalled ascending ids)."""
    lo, hi = prob.chunk_offsets[b], prob.chunk_offsets[b + 1]
    L = prob.idx_layers
    x = np.stack([index_score(inputs["idx_q"][b, l], inputs["idx_w"][b, l], inputs["idx_k"][l, lo:hi])
                  for l in range(L)])
    return x, recall(x, prob.keep[b])


def attention_tokens(q_rows: np.ndarray, Kh: np.ndarray, Vh: np.ndarray, toks: np.ndarray,
                     scale: Optional[float] = None):
    """Attention of q_rows [R][d] over the explicit token list ``toks`` of one KV
    head (Kh, Vh logical token-major bf16 bit patterns).  Returns (out, lse)."""
    R, d = q_rows.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    q_rows, Kh, Vh = _c(q_rows, np.uint16), _c(Kh, np.uint16), _c(Vh, np.uint16)
    toks = _c(toks, np.int64)
    out = np.empty((R, d), dtype=np.float64)
    lse = np.empty(R, dtype=np.float64)
    rc = lib().oracle_attention_tokens(q_rows.ctypes.data, R, Kh.ctypes.data, Vh.ctypes.data, Kh.shape[0], d,
                                       toks.ctypes.data, len(toks), float(scale), out.ctypes.data, lse.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_attention_tokens rejected its input")
    return out, lse


def two_level(recalled: np.ndarray, native: np.ndarray, k2: int, w0: int, n_total: int) -> np.ndarray:
    """Level 2 (top-k2 of the native score within the recalled history ids) plus
    the window chunks w0 .. n_total - 1; ascending ids."""
    recalled, native = _c(recalled, np.int32), _c(native, np.float64)
    out = np.empty(len(recalled) + max(n_total - w0, 0) + 1, dtype=np.int32)
    m = lib().oracle_two_level(recalled.ctypes.data, len(recalled), native.ctypes.data, len(native), k2, w0,
                               n_total, out.ctypes.data)
    if m < 0:
        raise ValueError("oracle_two_level rejected its input")
    return out[:m].copy()


def window(ctx_tokens: int, window_tokens: int, chunk: int):
    """The always-resident window and the history of one sequence.

    Sec. 2.5 keeps the last window_tokens context tokens (and the decoded tail)
    resident, and Sec. 2.1 scores only complete compressed entries.  Read per
    chunk: chunk c covers tokens [c C, min((c + 1) C, ctx)); it belongs to the
    window when it holds one of the last window_tokens tokens or when it is
    partial (the context ends inside it).  The window is then a run of chunks
    at the end, w0 .. n_total - 1, and the history is the complete chunks
    0 .. w0 - 1 before it.  Returns (w0, n_total, tail), tail = tokens in the
    last chunk."""
    n_total = (ctx_tokens + chunk - 1) // chunk
    in_window = []
    for c in range(n_total):
        lo, hi = c * chunk, min((c + 1) * chunk, ctx_tokens)
        holds_recent = hi > ctx_tokens - window_tokens
        partial = hi - lo < chunk
        in_window.append(holds_recent or partial)
    w0 = in_window.index(True) if True in in_window else n_total
    if not all(in_window[w0:]):
        raise ValueError("the window is not a run of chunks at the end")
    return w0, n_total, ctx_tokens - (n_total - 1) * chunk


def two_level_for_sequence(prob, inputs: Dict[str, object], b: int):
    """Level 1 (recall over the history before the window), Level 2 and the
    window for sequence b.  Returns (x [L][n_hist], recalled, native [n_hist],
    kept ascending chunk ids, token count of the last chunk)."""
    lo = prob.chunk_offsets[b]
    w0, n_total, tail = window(prob.ctx_tokens[b], prob.window_tokens[b] if prob.window_tokens else 0, prob.chunk)
    n_hist = w0
    L = prob.idx_layers
    x = np.stack([index_score(inputs["idx_q"][b, l], inputs["idx_w"][b, l], inputs["idx_k"][l, lo:lo + n_hist])
                  for l in range(L)]) if n_hist > 0 else np.zeros((L, 0))
    recalled = recall(x, prob.keep[b]) if n_hist > 0 else np.zeros(0, dtype=np.int32)
    native = (index_score(inputs["nat_q"][b], inputs["nat_w"][b], inputs["nat_k"][lo:lo + n_hist])
              if n_hist > 0 else np.zeros(0))
    kept = two_level(recalled, native, prob.core_keep[b], w0, n_total)
    return x, recalled, native, kept, tail


def kept_tokens(kept: np.ndarray, chunk: int, ctx_tokens: int) -> np.ndarray:
    """Token list of the kept chunks, ascending, the last chunk cut at the context end."""
    return np.concatenate([np.arange(c * chunk, min((c + 1) * chunk, ctx_tokens)) for c in kept]) \
        if len(kept) else np.zeros(0, dtype=np.int64)


# ------------------------------------------------------------- host tier
def tier_plan(owner: Sequence[int], old_slots: Sequence[int], kept: Sequence[int]):
    """Residency plan of one sequence's GPU reserve (Sec. 2.5: the recalled set
    is materialised from the host cold mirror into a GPU reserve of slots).

    owner[s] is the chunk slot s holds (-1: empty); old_slots are the slots the
    previous kept set is read from (they must survive this step, so that the
    previous set stays readable while the new one is copied in); kept are the
    new kept chunk ids, ascending.  A kept chunk that some slot already holds
    keeps that slot; the others take the free slots -- neither protected by
    old_slots nor holding a kept chunk -- in ascending order.  Returns
    (new_owner, slot of every kept chunk in kept order, [(chunk, slot)] to copy
    in), or raises when the slots do not suffice."""
    owner = list(owner)
    where = {}
    for s, c in enumerate(owner):
        if c >= 0:
            where[c] = s
    protected = set(old_slots) | {where[c] for c in kept if c in where}
    free = [s for s in range(len(owner)) if s not in protected]
    missing = [c for c in kept if c not in where]
    if len(missing) > len(free):
        raise ValueError("reserve too small")
    fetch = list(zip(missing, free))
    for c, s in fetch:
        owner[s] = c
    slot_of = {c: where[c] for c in kept if c in where}
    slot_of.update({c: s for c, s in fetch})
    return owner, [slot_of[c] for c in kept], fetch


# ---------------------------------------------------------------- O4 step
def top_p(S: np.ndarray, p_num: int, p_den: int, detail: bool = False):
    """Top-p set of one row of float32 logits (Eqs. 7-8): (0/1 marks [n], set
    size), plus, with ``detail``, the entry order (logit desc, index asc) and
    the float64 mass fraction of every prefix of it."""
    S = _c(S, np.float32)
    n = len(S)
    mark = np.zeros(n, dtype=np.uint8)
    order = np.empty(n, dtype=np.int64) if detail else None
    cum = np.empty(n, dtype=np.float64) if detail else None
    size = lib().oracle_top_p(S.ctypes.data, n, p_num, p_den, mark.ctypes.data,
                              order.ctypes.data if detail else None, cum.ctypes.data if detail else None)
    if size < 0:
        raise ValueError("oracle_top_p rejected its arguments")
    return (mark, int(size), order, cum) if detail else (mark, int(size))


def golden_labels(logits: np.ndarray, p_num: int, p_den: int, theta: int):
    """Label set of one window (Eqs. 7-11) from float32 logits [tau][L][n]:
    (ascending entry ids of Y, top-p set sizes [tau][L], golden-set sizes [tau])."""
    logits = _c(logits, np.float32)
    tau, L, n = logits.shape
    label = np.zeros(n, dtype=np.uint8)
    sizes = np.zeros((tau, L), dtype=np.int32)
    golden = np.zeros(tau, dtype=np.int32)
    cnt = lib().oracle_golden_labels(logits.ctypes.data, tau, L, n, p_num, p_den, theta, label.ctypes.data,
                                     sizes.ctypes.data, golden.ctypes.data)
    if cnt < 0:
        raise ValueError("oracle_golden_labels rejected its arguments")
    return np.nonzero(label)[0].astype(np.int32), sizes, golden


def select_for_sequence(prob, inputs: Dict[str, object], b: int):
    """O1 then O2 for sequence b.

    Returns (scores [Q][n_b], per-query lists [Q][k_b], kept ascending chunk ids).
    """
    Q = prob.n_lookahead
    lo, hi = prob.chunk_offsets[b], prob.chunk_offsets[b + 1]
    E_b = inputs["E"][lo:hi]
    scores = np.stack([score(inputs["qe"][b, j], E_b, prob.emb_dtype) for j in range(Q)])
    lists = np.stack([topk(scores[j], prob.keep[b]) for j in range(Q)])
    kept = lists[0].copy() if Q == 1 else union(lists, prob.n_chunks[b])
    return scores, lists, kept


def attend_rows(prob, inputs: Dict[str, object], b: int, kept: np.ndarray, rows: Sequence,
                kv: Callable[[str, int, int, np.ndarray], np.ndarray], scale: Optional[float] = None):
    """O3 for the (t, h) query rows of sequence b over the kept chunks.

    ``kv(which, b, g, chunks)`` supplies the logical K or V of KV head g as
    [ctx_tokens][d] (only the kept chunks need to be filled).  Returns
    {(t, h): (out [d], lse)}.
    """
    G = prob.group
    by_g: Dict[int, List] = {}
    for (t, h) in rows:
        by_g.setdefault(h // G, []).append((t, h))
    res = {}
    for g, rs in sorted(by_g.items()):
        Kh, Vh = kv("k", b, g, kept), kv("v", b, g, kept)
        qr = np.stack([inputs["q"][b, t, h] for (t, h) in rs])
        out, lse = attention(qr, Kh, Vh, kept, prob.chunk, scale)
        for j, key in enumerate(rs):
            res[key] = (out[j], lse[j])
    return res
