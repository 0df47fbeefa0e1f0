"""ctypes binding of ``liblsa.so`` (the C ABI in ``include/lsa.h``).

Argument marshalling only: every step of the decode path runs in the HIP
kernels of the shared library.  Device buffers are passed as torch tensors (or
raw integer addresses); PyTorch provides device memory and streams, nothing
else.  There is no fallback: if the library cannot be loaded, importing this
module raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

from . import _build

_P = ctypes.c_void_p


class LsaError(RuntimeError):
    def __init__(self, status: int, fn: str, msg: str):
        super().__init__(f"{fn} failed with status {status} ({STATUS_NAMES.get(status, '?')}): {msg}")
        self.status = status


LSA_OK, LSA_ERR_INVALID_ARG, LSA_ERR_UNSUPPORTED, LSA_ERR_WORKSPACE, LSA_ERR_HIP = 0, 1, 2, 3, 4
STATUS_NAMES = {0: "LSA_OK", 1: "LSA_ERR_INVALID_ARG", 2: "LSA_ERR_UNSUPPORTED", 3: "LSA_ERR_WORKSPACE",
                4: "LSA_ERR_HIP"}
DTYPES = {"f32": 0, "bf16": 1, "i8": 2}

EXPORTS = ("lsa_abi_version", "lsa_status_string", "lsa_last_error", "lsa_validate", "lsa_max_sel",
           "lsa_max_keep", "lsa_workspace_size", "lsa_workspace_init", "lsa_score_chunks", "lsa_topk_chunks",
           "lsa_sparse_decode_attn", "lsa_decode_step", "lsa_recall_scores", "lsa_recall_select",
           "lsa_recall_step", "lsa_two_level_sizes", "lsa_two_level_step", "lsa_tier_sizes", "lsa_tier_reset",
           "lsa_tier_plan", "lsa_tier_fetch", "lsa_tier_fetch_dma", "lsa_tier_attend", "lsa_tier_step",
           "lsa_golden_sizes", "lsa_golden_labels", "lsa_decode_step_noalloc", "lsa_kv_pack")


class lsa_problem(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("chunk_size", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("emb_dim", ctypes.c_int32),
        ("n_lookahead", ctypes.c_int32), ("n_qtok", ctypes.c_int32), ("emb_dtype", ctypes.c_int32),
        ("reserved", ctypes.c_int32), ("ctx_tokens", ctypes.POINTER(ctypes.c_int64)),
        ("keep", ctypes.POINTER(ctypes.c_int32)), ("kv_chunk_stride", ctypes.c_int64),
        ("kv_head_stride", ctypes.c_int64),
    ]


class lsa_indexer(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("key_dim", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class lsa_two_level(ctypes.Structure):
    _fields_ = [("native_heads", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("core_keep", ctypes.POINTER(ctypes.c_int32)), ("window_tokens", ctypes.POINTER(ctypes.c_int64))]


class lsa_tier(ctypes.Structure):
    _fields_ = [("slots", ctypes.POINTER(ctypes.c_int32)), ("reserved", ctypes.c_int32),
                ("fetch_workgroups", ctypes.c_int32)]


class lsa_golden(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_steps", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("theta", ctypes.c_int32), ("p_num", ctypes.c_int32), ("p_den", ctypes.c_int32),
                ("n_entries", ctypes.POINTER(ctypes.c_int64))]


def _load() -> ctypes.CDLL:
    # torch ships its own HIP runtime with the same soname as the system one.
    # Loading torch first makes liblsa.so bind to that already-loaded runtime,
    # so torch's allocations and streams and this library's launches share one
    # HIP runtime instance in the process.
    import torch  # noqa: F401
    path = _build.LIB_PATH
    if not os.path.exists(path):
        _build.build()
    lib = ctypes.CDLL(path)
    lib.lsa_abi_version.restype = ctypes.c_int
    lib.lsa_status_string.restype = ctypes.c_char_p
    lib.lsa_status_string.argtypes = [ctypes.c_int]
    lib.lsa_last_error.restype = ctypes.c_char_p
    pp = ctypes.POINTER(lsa_problem)
    lib.lsa_validate.argtypes = [pp]
    lib.lsa_max_sel.argtypes = [pp, ctypes.POINTER(ctypes.c_int32)]
    lib.lsa_max_keep.argtypes = [pp, ctypes.POINTER(ctypes.c_int32)]
    lib.lsa_workspace_size.argtypes = [pp, ctypes.POINTER(ctypes.c_size_t)]
    lib.lsa_workspace_init.argtypes = [_P, ctypes.c_size_t, _P]
    lib.lsa_score_chunks.argtypes = [pp, _P, _P, _P, _P]
    lib.lsa_topk_chunks.argtypes = [pp, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]
    lib.lsa_sparse_decode_attn.argtypes = [pp, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, ctypes.c_size_t, _P]
    lib.lsa_kv_pack.argtypes = [pp, _P, _P, _P, ctypes.c_int64, ctypes.c_int64, _P, _P, _P, _P]
    lib.lsa_decode_step.argtypes = [pp, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]
    ip = ctypes.POINTER(lsa_indexer)
    lib.lsa_recall_scores.argtypes = [pp, ip, _P, _P, _P, _P, _P]
    lib.lsa_recall_select.argtypes = [pp, ip, _P, _P, _P, _P]
    lib.lsa_recall_step.argtypes = [pp, ip, _P, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, _P, _P,
                                    ctypes.c_size_t, _P]
    tp = ctypes.POINTER(lsa_two_level)
    lib.lsa_two_level_sizes.argtypes = [pp, tp, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_size_t)]
    lib.lsa_two_level_step.argtypes = [pp, ip, tp, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P,
                                       _P, _P, ctypes.c_size_t, _P]
    rp = ctypes.POINTER(lsa_tier)
    lib.lsa_tier_sizes.argtypes = [pp, rp, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int64),
                                   ctypes.POINTER(ctypes.c_size_t)]
    lib.lsa_tier_reset.argtypes = [pp, rp, _P, _P]
    lib.lsa_tier_plan.argtypes = [pp, rp, _P, _P, _P, _P, _P, _P, _P, _P, _P]
    lib.lsa_tier_fetch.argtypes = [pp, rp, _P, _P, _P, _P, _P, _P, _P]
    lib.lsa_tier_fetch_dma.argtypes = [pp, rp, _P, _P, _P, _P, _P, _P, _P]
    lib.lsa_tier_step.argtypes = [pp, rp, ip, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P,
                                  _P, _P, ctypes.c_size_t, _P]
    lib.lsa_tier_attend.argtypes = [pp, rp, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, ctypes.c_size_t, _P]
    lib.lsa_decode_step_noalloc.argtypes = [pp, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, _P, _P]
    gp = ctypes.POINTER(lsa_golden)
    lib.lsa_golden_sizes.argtypes = [gp, ctypes.POINTER(ctypes.c_size_t)]
    lib.lsa_golden_labels.argtypes = [gp, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]
    for name in EXPORTS[3:]:
        getattr(lib, name).restype = ctypes.c_int
    if lib.lsa_abi_version() != 1:
        raise RuntimeError(f"liblsa ABI version {lib.lsa_abi_version()} != 1")
    return lib


LIB = _load()


class Problem:
    """Shape of one decode step (mirrors ``lsa_problem``; keeps its host arrays alive)."""

    def __init__(self, ctx_tokens: Sequence[int], chunk_size: int, keep: Sequence[int], n_q_heads: int,
                 n_kv_heads: int, head_dim: int = 128, emb_dim: int = 256, n_lookahead: int = 1,
                 n_qtok: int = 1, emb_dtype: str = "bf16", kv_chunk_stride: int = 0, kv_head_stride: int = 0):
        B = len(ctx_tokens)
        self._ctx = (ctypes.c_int64 * max(B, 1))(*ctx_tokens)
        self._keep = (ctypes.c_int32 * max(len(keep), 1))(*keep)
        self.c = lsa_problem(B, chunk_size, n_q_heads, n_kv_heads, head_dim, emb_dim, n_lookahead, n_qtok,
                             DTYPES[emb_dtype] if isinstance(emb_dtype, str) else int(emb_dtype), 0,
                             ctypes.cast(self._ctx, ctypes.POINTER(ctypes.c_int64)),
                             ctypes.cast(self._keep, ctypes.POINTER(ctypes.c_int32)), kv_chunk_stride,
                             kv_head_stride)

    @classmethod
    def from_synth(cls, prob, **kw) -> "Problem":
        return cls(prob.ctx_tokens, prob.chunk, prob.keep, prob.n_q_heads, prob.n_kv_heads, prob.head_dim,
                   prob.emb_dim, prob.n_lookahead, prob.n_qtok, prob.emb_dtype, **kw)

    @property
    def ref(self):
        return ctypes.byref(self.c)


class Indexer:
    """Memory Indexer of the recall path (mirrors ``lsa_indexer``)."""

    def __init__(self, n_layers: int, n_heads: int, key_dim: int):
        self.c = lsa_indexer(n_layers, n_heads, key_dim, 0)

    @classmethod
    def from_synth(cls, prob) -> "Indexer":
        return cls(prob.idx_layers, prob.idx_heads, prob.idx_dim)

    @property
    def ref(self):
        return ctypes.byref(self.c)


class TwoLevel:
    """Two-level selection (mirrors ``lsa_two_level``; keeps its host arrays alive)."""

    def __init__(self, native_heads: int, core_keep: Sequence[int], window_tokens: Sequence[int]):
        self._core = (ctypes.c_int32 * max(len(core_keep), 1))(*core_keep)
        self._win = (ctypes.c_int64 * max(len(window_tokens), 1))(*window_tokens)
        self.c = lsa_two_level(native_heads, 0, ctypes.cast(self._core, ctypes.POINTER(ctypes.c_int32)),
                               ctypes.cast(self._win, ctypes.POINTER(ctypes.c_int64)))

    @classmethod
    def from_synth(cls, prob) -> "TwoLevel":
        return cls(prob.nat_heads, prob.core_keep, prob.window_tokens)

    @property
    def ref(self):
        return ctypes.byref(self.c)


class Tier:
    """Host tier: reserve slots per sequence (mirrors ``lsa_tier``; keeps its host array alive)."""

    def __init__(self, slots: Sequence[int], fetch_workgroups: int = 0):
        self._slots = (ctypes.c_int32 * max(len(slots), 1))(*slots)
        self.c = lsa_tier(ctypes.cast(self._slots, ctypes.POINTER(ctypes.c_int32)), 0, fetch_workgroups)

    @property
    def ref(self):
        return ctypes.byref(self.c)


class Golden:
    """Golden-label pipeline shape (mirrors ``lsa_golden``; keeps its host array alive)."""

    def __init__(self, n_entries: Sequence[int], n_steps: int, n_layers: int, theta: int = 3, p_num: int = 3,
                 p_den: int = 5):
        self._n = (ctypes.c_int64 * max(len(n_entries), 1))(*n_entries)
        self.c = lsa_golden(len(n_entries), n_steps, n_layers, theta, p_num, p_den,
                            ctypes.cast(self._n, ctypes.POINTER(ctypes.c_int64)))

    @classmethod
    def from_synth(cls, gp, **kw) -> "Golden":
        args = dict(theta=gp.theta, p_num=gp.p_num, p_den=gp.p_den)
        args.update(kw)
        return cls(gp.n_entries, gp.tau, gp.layers, **args)

    @property
    def ref(self):
        return ctypes.byref(self.c)


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _host_ptr(x) -> Optional[int]:
    """Address of a host buffer: a numpy array (C-contiguous), a CPU tensor or an integer."""
    if x is None or isinstance(x, int):
        return x
    if hasattr(x, "ctypes"):
        if not x.flags["C_CONTIGUOUS"]:
            raise ValueError("host array must be C-contiguous")
        return x.ctypes.data
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(rc: int, fn: str) -> None:
    if rc != LSA_OK:
        raise LsaError(rc, fn, LIB.lsa_last_error().decode())


def last_error() -> str:
    return LIB.lsa_last_error().decode()


def lsa_validate(p: Problem) -> int:
    return LIB.lsa_validate(p.ref)


def lsa_max_sel(p: Problem) -> int:
    v = ctypes.c_int32()
    _check(LIB.lsa_max_sel(p.ref, ctypes.byref(v)), "lsa_max_sel")
    return v.value


def lsa_max_keep(p: Problem) -> int:
    v = ctypes.c_int32()
    _check(LIB.lsa_max_keep(p.ref, ctypes.byref(v)), "lsa_max_keep")
    return v.value


def lsa_workspace_size(p: Problem) -> int:
    v = ctypes.c_size_t()
    _check(LIB.lsa_workspace_size(p.ref, ctypes.byref(v)), "lsa_workspace_size")
    return v.value


def lsa_workspace_init(ws, nbytes: int, stream=None) -> None:
    _check(LIB.lsa_workspace_init(_ptr(ws), nbytes, _stream(stream)), "lsa_workspace_init")


def lsa_score_chunks(p: Problem, query_emb, chunk_emb, scores, stream=None) -> None:
    _check(LIB.lsa_score_chunks(p.ref, _ptr(query_emb), _ptr(chunk_emb), _ptr(scores), _stream(stream)),
           "lsa_score_chunks")


def lsa_topk_chunks(p: Problem, scores, sel_idx, sel_count, per_query_idx=None, ws=None, ws_bytes: int = 0,
                    stream=None) -> None:
    _check(LIB.lsa_topk_chunks(p.ref, _ptr(scores), _ptr(sel_idx), _ptr(sel_count), _ptr(per_query_idx), _ptr(ws),
                               ws_bytes, _stream(stream)), "lsa_topk_chunks")


def lsa_kv_pack(p: Problem, k_tok, v_tok, token_offsets, k_cache, v_cache, first_token=None, tok_stride: int = 0,
                tok_head_stride: int = 0, stream=None) -> None:
    """Write tokens first_token[b] .. ctx_tokens[b] - 1 of token-major K/V rows into the paged caches.

    first_token: host sequence of per-sequence first tokens, or None for 0.
    """
    if first_token is None:
        ft = None
    else:
        ft = (ctypes.c_int64 * max(len(first_token), 1))(*[int(x) for x in first_token])
    _check(LIB.lsa_kv_pack(p.ref, _ptr(k_tok), _ptr(v_tok), _ptr(token_offsets), int(tok_stride),
                           int(tok_head_stride), None if ft is None else ctypes.cast(ft, ctypes.c_void_p),
                           _ptr(k_cache), _ptr(v_cache), _stream(stream)), "lsa_kv_pack")


def lsa_sparse_decode_attn(p: Problem, q, k_cache, v_cache, sel_idx, sel_count, softmax_scale: float, out,
                           lse=None, ws=None, ws_bytes: int = 0, stream=None) -> None:
    _check(LIB.lsa_sparse_decode_attn(p.ref, _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(sel_idx),
                                      _ptr(sel_count), float(softmax_scale), _ptr(out), _ptr(lse), _ptr(ws),
                                      ws_bytes, _stream(stream)), "lsa_sparse_decode_attn")


def lsa_decode_step(p: Problem, query_emb, chunk_emb, q, k_cache, v_cache, softmax_scale: float, out, lse=None,
                    sel_idx=None, sel_count=None, ws=None, ws_bytes: int = 0, stream=None) -> None:
    _check(LIB.lsa_decode_step(p.ref, _ptr(query_emb), _ptr(chunk_emb), _ptr(q), _ptr(k_cache), _ptr(v_cache),
                               float(softmax_scale), _ptr(out), _ptr(lse), _ptr(sel_idx), _ptr(sel_count), _ptr(ws),
                               ws_bytes, _stream(stream)), "lsa_decode_step")


def lsa_decode_step_noalloc(p: Problem, query_emb, chunk_emb, q, k_cache, v_cache, softmax_scale: float, out,
                            lse=None, sel_idx=None, sel_count=None, stream=None) -> None:
    _check(LIB.lsa_decode_step_noalloc(p.ref, _ptr(query_emb), _ptr(chunk_emb), _ptr(q), _ptr(k_cache),
                                       _ptr(v_cache), float(softmax_scale), _ptr(out), _ptr(lse), _ptr(sel_idx),
                                       _ptr(sel_count), _stream(stream)), "lsa_decode_step_noalloc")


def lsa_recall_scores(p: Problem, ix: Indexer, idx_q, idx_w, idx_k, scores, stream=None) -> None:
    _check(LIB.lsa_recall_scores(p.ref, ix.ref, _ptr(idx_q), _ptr(idx_w), _ptr(idx_k), _ptr(scores),
                                 _stream(stream)), "lsa_recall_scores")


def lsa_recall_select(p: Problem, ix: Indexer, scores, sel_idx, sel_count, stream=None) -> None:
    _check(LIB.lsa_recall_select(p.ref, ix.ref, _ptr(scores), _ptr(sel_idx), _ptr(sel_count), _stream(stream)),
           "lsa_recall_select")


def lsa_recall_step(p: Problem, ix: Indexer, idx_q, idx_w, idx_k, q, k_cache, v_cache, softmax_scale: float, out,
                    lse=None, sel_idx=None, sel_count=None, ws=None, ws_bytes: int = 0, stream=None) -> None:
    _check(LIB.lsa_recall_step(p.ref, ix.ref, _ptr(idx_q), _ptr(idx_w), _ptr(idx_k), _ptr(q), _ptr(k_cache),
                               _ptr(v_cache), float(softmax_scale), _ptr(out), _ptr(lse), _ptr(sel_idx),
                               _ptr(sel_count), _ptr(ws), ws_bytes, _stream(stream)), "lsa_recall_step")


def lsa_two_level_sizes(p: Problem, tl: TwoLevel):
    """(row pitch of sel_idx, workspace bytes) of lsa_two_level_step."""
    m, w = ctypes.c_int32(), ctypes.c_size_t()
    _check(LIB.lsa_two_level_sizes(p.ref, tl.ref, ctypes.byref(m), ctypes.byref(w)), "lsa_two_level_sizes")
    return m.value, w.value


def lsa_two_level_step(p: Problem, ix: Indexer, tl: TwoLevel, idx_q, idx_w, idx_k, nat_q, nat_w, nat_k, q, k_cache,
                       v_cache, softmax_scale: float, out, lse=None, sel_idx=None, sel_count=None, ws=None,
                       ws_bytes: int = 0, stream=None) -> None:
    _check(LIB.lsa_two_level_step(p.ref, ix.ref, tl.ref, _ptr(idx_q), _ptr(idx_w), _ptr(idx_k), _ptr(nat_q),
                                  _ptr(nat_w), _ptr(nat_k), _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                  float(softmax_scale), _ptr(out), _ptr(lse), _ptr(sel_idx), _ptr(sel_count), _ptr(ws),
                                  ws_bytes, _stream(stream)), "lsa_two_level_step")


def lsa_tier_sizes(p: Problem, tr: Tier):
    """(pitch of the kept, slot and copy lists, reserve slots in total, workspace bytes of lsa_tier_attend)."""
    m, n, w = ctypes.c_int32(), ctypes.c_int64(), ctypes.c_size_t()
    _check(LIB.lsa_tier_sizes(p.ref, tr.ref, ctypes.byref(m), ctypes.byref(n), ctypes.byref(w)), "lsa_tier_sizes")
    return m.value, n.value, w.value


def lsa_tier_reset(p: Problem, tr: Tier, owner, stream=None) -> None:
    _check(LIB.lsa_tier_reset(p.ref, tr.ref, _ptr(owner), _stream(stream)), "lsa_tier_reset")


def lsa_tier_plan(p: Problem, tr: Tier, kept_idx, kept_count, prev_slots, prev_count, owner, slot_idx, fetch,
                  fetch_count, stream=None) -> None:
    _check(LIB.lsa_tier_plan(p.ref, tr.ref, _ptr(kept_idx), _ptr(kept_count), _ptr(prev_slots), _ptr(prev_count),
                             _ptr(owner), _ptr(slot_idx), _ptr(fetch), _ptr(fetch_count), _stream(stream)),
           "lsa_tier_plan")


def lsa_tier_fetch(p: Problem, tr: Tier, host_k, host_v, fetch, fetch_count, res_k, res_v, stream=None) -> None:
    _check(LIB.lsa_tier_fetch(p.ref, tr.ref, _ptr(host_k), _ptr(host_v), _ptr(fetch), _ptr(fetch_count),
                              _ptr(res_k), _ptr(res_v), _stream(stream)), "lsa_tier_fetch")


def lsa_tier_fetch_dma(p: Problem, tr: Tier, host_k, host_v, h_fetch, h_fetch_count, res_k, res_v,
                       stream=None) -> None:
    """h_fetch / h_fetch_count: host int32 buffers (numpy arrays or CPU tensors) holding a plan's copy list."""
    _check(LIB.lsa_tier_fetch_dma(p.ref, tr.ref, _ptr(host_k), _ptr(host_v), _host_ptr(h_fetch),
                                  _host_ptr(h_fetch_count), _ptr(res_k), _ptr(res_v), _stream(stream)),
           "lsa_tier_fetch_dma")


def lsa_tier_step(p: Problem, tr: Tier, nat: Indexer, core_keep, nat_q, nat_w, nat_k, kept_idx, kept_count, slot_idx,
                  q, res_k, res_v, softmax_scale: float, out, lse, sel_slots, sel_count, ws=None, ws_bytes: int = 0,
                  stream=None) -> None:
    ck = (ctypes.c_int32 * len(core_keep))(*[int(x) for x in core_keep])
    _check(LIB.lsa_tier_step(p.ref, tr.ref, nat.ref, ctypes.cast(ck, ctypes.c_void_p), _ptr(nat_q), _ptr(nat_w),
                             _ptr(nat_k), _ptr(kept_idx), _ptr(kept_count), _ptr(slot_idx), _ptr(q), _ptr(res_k),
                             _ptr(res_v), float(softmax_scale), _ptr(out), _ptr(lse), _ptr(sel_slots), _ptr(sel_count),
                             _ptr(ws), ws_bytes, _stream(stream)), "lsa_tier_step")


def lsa_tier_attend(p: Problem, tr: Tier, q, res_k, res_v, slot_idx, slot_count, softmax_scale: float, out, lse=None,
                    ws=None, ws_bytes: int = 0, stream=None) -> None:
    _check(LIB.lsa_tier_attend(p.ref, tr.ref, _ptr(q), _ptr(res_k), _ptr(res_v), _ptr(slot_idx), _ptr(slot_count),
                               float(softmax_scale), _ptr(out), _ptr(lse), _ptr(ws), ws_bytes, _stream(stream)),
           "lsa_tier_attend")


def lsa_golden_sizes(g: Golden) -> int:
    """Workspace bytes of lsa_golden_labels."""
    w = ctypes.c_size_t()
    _check(LIB.lsa_golden_sizes(g.ref, ctypes.byref(w)), "lsa_golden_sizes")
    return w.value


def lsa_golden_labels(g: Golden, logits, labels, label_count, nucleus_size=None, golden_count=None, ws=None,
                      ws_bytes: int = 0, stream=None) -> None:
    _check(LIB.lsa_golden_labels(g.ref, _ptr(logits), _ptr(labels), _ptr(label_count), _ptr(nucleus_size),
                                 _ptr(golden_count), _ptr(ws), ws_bytes, _stream(stream)), "lsa_golden_labels")
