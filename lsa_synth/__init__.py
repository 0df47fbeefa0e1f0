"""Seeded synthetic inputs for the LSA decode hot path.

Test and benchmark infrastructure.  This module produces the bytes that both
the GPU path and the CPU oracle consume, and holds none of the method's
arithmetic: no scoring, no selection, no attention.  It only draws random
numbers, rounds them to the storage dtypes and lays them out in memory.

Random numbers come from SplitMix64 evaluated as a counter-based generator
(``draw(key, i) = mix64(key + (i + 1) * GAMMA)``), keyed per (seed, stream), so
every tensor element can be regenerated independently of thread count or
device.  Normal draws map the top 16 bits of a draw through a 65536-entry
inverse-normal-CDF table (bin midpoints), which lets host C code and the HIP
device fill produce bit-identical bf16 K/V without transcendental functions on
either side.

Workload shapes follow the paper's decode-time setting (Memory Indexer over
64- or 128-token compressed chunks, Sec. 2.1; 1M-token serving, Sec. 2.5) and
the five presets below.
"""
from __future__ import annotations

import ctypes
import math
import os
import statistics
import subprocess
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_HOST_SO = os.path.join(_HERE, "libsynth.so")
_DEV_SO = os.path.join(_HERE, "libsynth_dev.so")

GAMMA = 0x9E3779B97F4A7C15
STREAM_K, STREAM_V, STREAM_Q, STREAM_E, STREAM_QE, STREAM_LEN, STREAM_QE_NOISE = 1, 2, 3, 4, 5, 6, 7
STREAM_IDX_Q, STREAM_IDX_K, STREAM_IDX_W = 8, 9, 10
STREAM_NAT_Q, STREAM_NAT_K, STREAM_NAT_W = 11, 12, 13
STREAM_GOLD_NOISE, STREAM_GOLD_REL, STREAM_GOLD_BOOST = 14, 15, 16
M64 = (1 << 64) - 1


# --------------------------------------------------------------------------- RNG
def _mix64_int(z: int) -> int:
    z &= M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def stream_key(seed: int, stream: int) -> int:
    """Key of one (seed, stream) pair."""
    return _mix64_int((seed * GAMMA + stream * 0xD1B54A32D192ED03 + 1) & M64)


def _mix64(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))


def draws(key: int, start: int, n: int) -> np.ndarray:
    """Raw 64-bit draws at counters [start, start + n)."""
    with np.errstate(over="ignore"):
        i = np.arange(start, start + n, dtype=np.uint64) + np.uint64(1)
        return _mix64(np.uint64(key) + i * np.uint64(GAMMA))


def uniform53(key: int, start: int, n: int) -> np.ndarray:
    return (draws(key, start, n) >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


# ----------------------------------------------------------------- rounding
def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even from float64 straight to bf16 (no double rounding)."""
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)                      # x = m * 2**e, 0.5 <= |m| < 1
    e = np.maximum(e, -125)                 # below the normal range the quantum stays 2**-133
    q = np.rint(np.ldexp(x, 8 - e))         # significand on an 8-bit grid, ties to even
    r = np.ldexp(q, e - 8).astype(np.float32)  # exact in float32
    return (r.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


# ------------------------------------------------------------- normal table
_TABLES: Dict[str, np.ndarray] = {}


def normal_table_f64() -> np.ndarray:
    """inv_cdf((u + 0.5) / 65536) for u in [0, 65536)."""
    if "f64" not in _TABLES:
        nd = statistics.NormalDist()
        _TABLES["f64"] = np.array([nd.inv_cdf((u + 0.5) / 65536.0) for u in range(65536)], dtype=np.float64)
    return _TABLES["f64"]


def normal_table_bf16() -> np.ndarray:
    if "bf16" not in _TABLES:
        _TABLES["bf16"] = f64_to_bf16_bits(normal_table_f64())
    return _TABLES["bf16"]


def normal_f64(key: int, start: int, n: int) -> np.ndarray:
    return normal_table_f64()[(draws(key, start, n) >> np.uint64(48)).astype(np.int64)]


def normal_bf16(key: int, start: int, n: int) -> np.ndarray:
    return normal_table_bf16()[(draws(key, start, n) >> np.uint64(48)).astype(np.int64)]


def int8_uniform(key: int, start: int, n: int) -> np.ndarray:
    """Uniform integers in [-127, 127] (multiply-shift range reduction)."""
    hi = draws(key, start, n) >> np.uint64(32)
    return ((hi * np.uint64(255)) >> np.uint64(32)).astype(np.int64) - 127


# ---------------------------------------------------------------- problems
@dataclass
class Problem:
    """Shape of one decode step.

    ``keep`` is the per-sequence keep budget k_b (per lookahead query when
    ``n_lookahead > 1``; the retained set is then the union of the per-query
    top-k sets).
    """
    name: str
    ctx_tokens: List[int]
    chunk: int
    keep: List[int]
    n_q_heads: int
    n_kv_heads: int
    head_dim: int = 128
    emb_dim: int = 256
    n_lookahead: int = 1
    n_qtok: int = 1
    emb_dtype: str = "bf16"          # 'f32' | 'bf16' | 'i8'
    planted: int = 0                 # planted relevant chunks per sequence
    q_scale: float = 1.0             # multiplier applied to q before rounding to bf16
    qe_rho: float = 0.95             # correlation of lookahead query embeddings
    # recall path (full Memory Indexer): layers OR-ed together (0 = not used),
    # indexer heads per layer, index-key width, and the fraction of entries each
    # layer's gate weights are drawn to recall; keep[b] is then the bound K_max
    idx_layers: int = 0
    idx_heads: int = 64
    idx_dim: int = 128
    idx_rate: float = 0.05
    # two-level path: Level-2 budget k2 per sequence (empty = not used), native
    # indexer heads, the always-resident window in tokens per sequence, and the
    # fraction of entries the native gates are drawn to favour
    core_keep: List[int] = field(default_factory=list)
    nat_heads: int = 64
    window_tokens: List[int] = field(default_factory=list)
    nat_rate: float = 0.5
    meta: Dict[str, object] = field(default_factory=dict)

    @property
    def batch(self) -> int:
        return len(self.ctx_tokens)

    @property
    def n_chunks(self) -> List[int]:
        """Chunks of every sequence, a partial last chunk included."""
        return [(L + self.chunk - 1) // self.chunk for L in self.ctx_tokens]

    @property
    def chunk_offsets(self) -> List[int]:
        off = [0]
        for n in self.n_chunks:
            off.append(off[-1] + n)
        return off

    @property
    def total_chunks(self) -> int:
        return self.chunk_offsets[-1]

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def max_sel_b(self, b: int) -> int:
        return min(self.n_lookahead * self.keep[b], self.n_chunks[b])

    @property
    def max_sel(self) -> int:
        return max(self.max_sel_b(b) for b in range(self.batch))

    def kv_elems(self) -> int:
        """Elements of one of K or V (whole cache)."""
        return self.total_chunks * self.n_kv_heads * self.chunk * self.head_dim


def planted_positions(n: int, p: int) -> np.ndarray:
    """p positions spread evenly over n chunks: floor((2i + 1) n / (2p))."""
    i = np.arange(p, dtype=np.int64)
    return ((2 * i + 1) * n) // (2 * p)


def make_problem(name: str, seed: int = 0) -> Problem:
    """The five workload presets of the decode hot path."""
    if name == "tiny":
        return Problem("tiny", [4096], 64, [8], 8, 8, emb_dtype="f32", planted=3,
                       q_scale=1.0 / math.sqrt(128.0))
    if name == "int8":
        return Problem("int8", [131072] * 4, 64, [256] * 4, 32, 8, emb_dtype="i8", planted=16)
    if name == "paper1m":
        n = 1048576 // 64
        return Problem("paper1m", [1048576], 64, [int(0.10 * n)], 32, 8, emb_dtype="bf16", planted=64)
    if name == "batch32":
        u = uniform53(stream_key(seed, STREAM_LEN), 0, 32)
        lo, hi = math.log(32768.0), math.log(524288.0)
        lens = [64 * int(math.exp(lo + (hi - lo) * float(x)) // 64) for x in u]
        keep = [max(1, int(0.135 * (L // 64))) for L in lens]
        return Problem("batch32", lens, 64, keep, 32, 8, emb_dtype="bf16", planted=16)
    if name == "lookahead":
        return Problem("lookahead", [1048576] * 8, 128, [512] * 8, 64, 8, emb_dtype="bf16",
                       n_lookahead=16, n_qtok=16, planted=0)
    if name == "recall_tiny":
        return Problem("recall_tiny", [4096], 64, [12], 8, 8, emb_dtype="bf16", idx_layers=3, idx_heads=16,
                       idx_dim=64, idx_rate=0.05)
    if name == "recall_batch":
        return Problem("recall_batch", [131072] * 4, 64, [2048] * 4, 32, 8, emb_dtype="bf16", idx_layers=2,
                       idx_heads=32, idx_dim=128, idx_rate=0.08)
    if name == "recall1m":
        n = 1048576 // 64
        return Problem("recall1m", [1048576], 64, [int(0.10 * n)], 32, 8, emb_dtype="bf16", idx_layers=3,
                       idx_heads=64, idx_dim=128, idx_rate=0.05)
    if name == "twolevel_tiny":
        return Problem("twolevel_tiny", [4096 + 37], 64, [24], 8, 8, emb_dtype="bf16", idx_layers=3, idx_heads=16,
                       idx_dim=64, idx_rate=0.1, core_keep=[6], nat_heads=16, window_tokens=[512])
    if name == "twolevel1m":
        # a 1M-token context with a partial last chunk: Level 1 recalls at most
        # 2,048 history chunks, Level 2 keeps 1,024 of them, plus the window of
        # the last 8,192 tokens (129 chunks with the partial one)
        return Problem("twolevel1m", [1048576 + 37], 64, [2048], 32, 8, emb_dtype="bf16", idx_layers=3,
                       idx_heads=64, idx_dim=128, idx_rate=0.05, core_keep=[1024], nat_heads=64,
                       window_tokens=[8192])
    raise KeyError(name)


PRESETS = ("tiny", "int8", "paper1m", "batch32", "lookahead")
RECALL_PRESETS = ("recall_tiny", "recall_batch", "recall1m")
TWO_LEVEL_PRESETS = ("twolevel_tiny", "twolevel1m")


# ------------------------------------------------------------ host inputs
def _unit_rows(x: np.ndarray) -> np.ndarray:
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _store(x64: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return x64.astype(np.float32)
    if dtype == "bf16":
        return f64_to_bf16_bits(x64)
    raise ValueError(dtype)


def _gate_shift(g: np.ndarray, sig: np.ndarray, rate: float) -> float:
    """Shift beta of gate weights w_h = g_h - beta such that, for random unit
    index keys, sum_h w_h ReLU(z_h) with independent z_h ~ N(0, sig_h^2) is >= 0
    with probability about ``rate`` (normal approximation of the sum; the
    realised recall is whatever the drawn keys give)."""
    z = statistics.NormalDist().inv_cdf(1.0 - rate)
    mean_relu = sig / math.sqrt(2.0 * math.pi)
    var_relu = sig * sig * (0.5 - 1.0 / (2.0 * math.pi))

    def f(beta: float) -> float:
        w = g - beta
        return float((w * mean_relu).sum()) + z * math.sqrt(float((w * w * var_relu).sum()))

    lo, hi = -100.0, 100.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if f(mid) > 0.0:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def _recall_inputs(prob: Problem, seed: int) -> Dict[str, np.ndarray]:
    """Indexer queries [B][L][n_h][c] (bf16 bits, N(0, 1)), gate weights
    [B][L][n_h] (float32) and unit-norm index keys [L][sum n_b][c] (bf16 bits)."""
    B, L, H, c = prob.batch, prob.idx_layers, prob.idx_heads, prob.idx_dim
    n = prob.total_chunks
    q = normal_bf16(stream_key(seed, STREAM_IDX_Q), 0, B * L * H * c).reshape(B, L, H, c)
    K = f64_to_bf16_bits(_unit_rows(normal_f64(stream_key(seed, STREAM_IDX_K), 0, L * n * c).reshape(L * n, c)))
    g = normal_f64(stream_key(seed, STREAM_IDX_W), 0, B * L * H).reshape(B, L, H)
    qf = bf16_bits_to_f64(q)
    w = np.empty((B, L, H), dtype=np.float32)
    for b in range(B):
        for l in range(L):
            sig = np.linalg.norm(qf[b, l], axis=-1) / math.sqrt(c)
            w[b, l] = (g[b, l] - _gate_shift(g[b, l], sig, prob.idx_rate)).astype(np.float32)
    out = {"idx_q": q, "idx_w": w, "idx_k": K.reshape(L, n, c)}
    if prob.core_keep:
        # native indexer of Level 2: its own queries, gates and index keys
        Hn = prob.nat_heads
        nq = normal_bf16(stream_key(seed, STREAM_NAT_Q), 0, B * Hn * c).reshape(B, Hn, c)
        nK = f64_to_bf16_bits(_unit_rows(normal_f64(stream_key(seed, STREAM_NAT_K), 0, n * c).reshape(n, c)))
        ng = normal_f64(stream_key(seed, STREAM_NAT_W), 0, B * Hn).reshape(B, Hn)
        nqf = bf16_bits_to_f64(nq)
        nw = np.empty((B, Hn), dtype=np.float32)
        for b in range(B):
            sig = np.linalg.norm(nqf[b], axis=-1) / math.sqrt(c)
            nw[b] = (ng[b] - _gate_shift(ng[b], sig, prob.nat_rate)).astype(np.float32)
        out.update({"nat_q": nq, "nat_w": nw, "nat_k": nK})
    return out


def host_inputs(prob: Problem, seed: int) -> Dict[str, object]:
    """Small tensors of one step, generated on the host.

    Returns ``qe`` [B][Q][D], ``E`` [sum n_b][D] (float32, bf16 bits as uint16,
    or int8), ``q`` [B][Tq][Hq][d] bf16 bits and ``planted`` (list of global-
    per-sequence chunk ids); with ``idx_layers > 0`` also the recall inputs
    ``idx_q``, ``idx_w`` and ``idx_k`` of :func:`_recall_inputs`.
    """
    B, Q, D = prob.batch, prob.n_lookahead, prob.emb_dim
    offs = prob.chunk_offsets
    kE, kQE, kN = stream_key(seed, STREAM_E), stream_key(seed, STREAM_QE), stream_key(seed, STREAM_QE_NOISE)
    planted = [planted_positions(n, prob.planted) for n in prob.n_chunks]
    if prob.emb_dtype == "i8":
        E = int8_uniform(kE, 0, offs[-1] * D).reshape(offs[-1], D)
        qe = int8_uniform(kQE, 0, B * Q * D).reshape(B, Q, D)
        for b in range(B):
            sign = np.where(qe[b, 0] >= 0, 127, -127)
            for c in planted[b]:
                E[offs[b] + c] = sign
        E, qe = E.astype(np.int8), qe.astype(np.int8)
    else:
        E64 = _unit_rows(normal_f64(kE, 0, offs[-1] * D).reshape(offs[-1], D))
        base = _unit_rows(normal_f64(kQE, 0, B * D).reshape(B, D))
        if Q == 1:
            qe64 = base[:, None, :]
        else:
            g = _unit_rows(normal_f64(kN, 0, B * Q * D).reshape(B, Q, D))
            rho = prob.qe_rho
            qe64 = _unit_rows(math.sqrt(rho) * base[:, None, :] + math.sqrt(1.0 - rho) * g)
        for b in range(B):
            rows = offs[b] + planted[b]
            E64[rows] = _unit_rows(E64[rows] + 0.5 * base[b][None, :])
        E, qe = _store(E64, prob.emb_dtype), _store(qe64, prob.emb_dtype)
    nq = B * prob.n_qtok * prob.n_q_heads * prob.head_dim
    q = normal_bf16(stream_key(seed, STREAM_Q), 0, nq)
    if prob.q_scale != 1.0:
        q = f64_to_bf16_bits(bf16_bits_to_f64(q) * prob.q_scale)
    q = q.reshape(B, prob.n_qtok, prob.n_q_heads, prob.head_dim)
    out = {"qe": qe, "E": E, "q": q, "planted": planted}
    if prob.idx_layers > 0:
        out.update(_recall_inputs(prob, seed))
    return out


# ------------------------------------------------------------ K/V on host
def _so(path: str, builder) -> ctypes.CDLL:
    if not os.path.exists(path):
        builder()
    return ctypes.CDLL(path)


_host_lib: Optional[ctypes.CDLL] = None


def host_lib() -> ctypes.CDLL:
    global _host_lib
    if _host_lib is None:
        lib = _so(_HOST_SO, build_host)
        lib.synth_kv_chunks.argtypes = [ctypes.c_uint64, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                                        ctypes.c_void_p]
        lib.synth_kv_chunks.restype = None
        lib.synth_draws.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p]
        lib.synth_golden_logits.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p,
                                            ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                            ctypes.c_float, ctypes.c_float, ctypes.c_uint32, ctypes.c_uint32,
                                            ctypes.c_void_p]
        lib.synth_golden_logits.restype = None
        lib.synth_stream_key.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        lib.synth_stream_key.restype = ctypes.c_uint64
        _host_lib = lib
    return _host_lib


def kv_chunks(prob: Problem, seed: int, which: str, b: int, h: int, chunks) -> np.ndarray:
    """K or V of sequence b, KV head h, for the listed (per-sequence) chunk ids.

    Returns bf16 bits shaped [len(chunks)][chunk][head_dim], token-major.
    """
    stream = STREAM_K if which == "k" else STREAM_V
    chunks = np.ascontiguousarray(np.asarray(chunks, dtype=np.int64) + prob.chunk_offsets[b])
    out = np.empty((len(chunks), prob.chunk, prob.head_dim), dtype=np.uint16)
    tab = np.ascontiguousarray(normal_table_bf16())
    host_lib().synth_kv_chunks(stream_key(seed, stream), tab.ctypes.data, prob.n_kv_heads, h, prob.head_dim,
                               prob.chunk, chunks.ctypes.data, len(chunks), out.ctypes.data)
    return out


def kv_head_sparse(prob: Problem, seed: int, which: str, b: int, h: int, chunks) -> np.ndarray:
    """Logical token-major K or V of one (sequence, KV head): [n_chunks * chunk][head_dim]
    (the slots past the context end of a partial last chunk hold values too).

    Only the listed chunks are filled; every other token is zero.
    """
    C = prob.chunk
    full = np.zeros((prob.n_chunks[b] * C, prob.head_dim), dtype=np.uint16)
    chunks = np.asarray(chunks, dtype=np.int64)
    if len(chunks):
        vals = kv_chunks(prob, seed, which, b, h, chunks)
        full.reshape(-1, C, prob.head_dim)[chunks] = vals
    return full


# ------------------------------------------------------- K/V on the device
_dev_lib: Optional[ctypes.CDLL] = None


def dev_lib() -> ctypes.CDLL:
    global _dev_lib
    if _dev_lib is None:
        import torch  # noqa: F401  (bind to the HIP runtime torch already loaded)
        lib = _so(_DEV_SO, build_device)
        lib.synth_fill_kv_device.argtypes = [ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                             ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                             ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p]
        lib.synth_fill_kv_device.restype = ctypes.c_int
        lib.synth_fill_kv_tokens_device.argtypes = [ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                                    ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                                    ctypes.c_int64, ctypes.c_void_p]
        lib.synth_fill_kv_tokens_device.restype = ctypes.c_int
        lib.synth_copy_device.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
        lib.synth_copy_device.restype = ctypes.c_int
        lib.synth_read_device.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
        lib.synth_read_device.restype = ctypes.c_int
        lib.synth_read_sink_words.restype = ctypes.c_int
        lib.synth_fill_golden_device.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p,
                                                 ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                                 ctypes.c_float, ctypes.c_float, ctypes.c_uint32, ctypes.c_uint32,
                                                 ctypes.c_void_p, ctypes.c_void_p]
        lib.synth_fill_golden_device.restype = ctypes.c_int
        _dev_lib = lib
    return _dev_lib


def fill_kv_device(prob: Problem, seed: int, which: str, out_ptr: int, table_ptr: int, stream_ptr: int,
                   chunk_stride: Optional[int] = None, head_stride: Optional[int] = None) -> None:
    """Fill a device K or V cache in the library's chunk-paged, MFMA-ordered block layout.

    ``table_ptr`` is a device copy of :func:`normal_table_bf16`.  See
    :func:`block_offset` for where token t, dim e of a block lands.
    """
    C, d, H = prob.chunk, prob.head_dim, prob.n_kv_heads
    hs = C * d if head_stride is None else head_stride
    cs = H * C * d if chunk_stride is None else chunk_stride
    stream = STREAM_K if which == "k" else STREAM_V
    rc = dev_lib().synth_fill_kv_device(stream_key(seed, stream), table_ptr, out_ptr, prob.total_chunks, H, C, d,
                                        cs, hs, 0 if which == "k" else 1, stream_ptr)
    if rc != 0:
        raise RuntimeError(f"synth_fill_kv_device failed with code {rc}")


def token_rows(prob: Problem, row_off: Sequence[int], n_rows: int) -> np.ndarray:
    """Global token of each row of a token-major cache whose sequence b starts
    at row row_off[b] and holds its ctx_tokens[b] tokens; other rows get -1.

    The global token of token i of sequence b is chunk_offsets[b] * chunk + i,
    the token whose values the paged fill puts at that position."""
    tau = np.full(n_rows, -1, dtype=np.int64)
    for b, L in enumerate(prob.ctx_tokens):
        r0 = int(row_off[b])
        tau[r0:r0 + int(L)] = prob.chunk_offsets[b] * prob.chunk + np.arange(int(L), dtype=np.int64)
    return tau


def fill_kv_tokens_device(prob: Problem, seed: int, which: str, out_ptr: int, table_ptr: int, tau_ptr: int,
                          n_rows: int, tok_stride: Optional[int] = None, head_stride: Optional[int] = None,
                          stream_ptr: int = 0) -> None:
    """Fill a device token-major K or V cache: row r holds global token tau[r]
    (:func:`token_rows`), KV head h at r * tok_stride + h * head_stride."""
    d, H = prob.head_dim, prob.n_kv_heads
    hs = d if head_stride is None else head_stride
    ts = H * hs if tok_stride is None else tok_stride
    stream = STREAM_K if which == "k" else STREAM_V
    rc = dev_lib().synth_fill_kv_tokens_device(stream_key(seed, stream), table_ptr, out_ptr, tau_ptr, n_rows, H, d,
                                               ts, hs, stream_ptr)
    if rc != 0:
        raise RuntimeError(f"synth_fill_kv_tokens_device failed with code {rc}")


def block_offset(which: str, t, e):
    """Element offset of (token t, dim e) inside one (chunk, KV head) block of the
    K (``which='k'``) or V cache, head_dim 128.  Works on numpy arrays."""
    t = np.asarray(t, dtype=np.int64)
    e = np.asarray(e, dtype=np.int64)
    if which == "k":
        return ((((t // 32 * 2 + t // 4 % 2) * 4 + e // 32) * 4 + e // 8 % 4) * 16 + t % 32 // 8 * 4 + t % 4) * 8 + e % 8
    return (((t // 32 * 8 + e // 16) * 4 + t % 32 // 8) * 16 + e % 16) * 8 + t % 8


def copy_device(src_ptr: int, dst_ptr: int, nbytes: int, stream_ptr: int) -> None:
    """A plain device copy of known size (for calibrating byte counters)."""
    rc = dev_lib().synth_copy_device(src_ptr, dst_ptr, nbytes, stream_ptr)
    if rc != 0:
        raise RuntimeError(f"synth_copy_device failed with code {rc}")


def read_device(src_ptr: int, nbytes: int, sink_ptr: int, stream_ptr: int) -> None:
    """A plain streaming read of known size (for the read-bandwidth ceiling);
    ``sink`` holds :func:`read_sink_words` uint32 words of device memory."""
    rc = dev_lib().synth_read_device(src_ptr, nbytes, sink_ptr, stream_ptr)
    if rc != 0:
        raise RuntimeError(f"synth_read_device failed with code {rc}")


def read_sink_words() -> int:
    return int(dev_lib().synth_read_sink_words())


def device_inputs(prob: Problem, seed: int, device: str = "cuda", host: Optional[Dict[str, object]] = None):
    """All step inputs resident in device memory (torch tensors).

    Small tensors come from :func:`host_inputs`; K and V are filled in place on
    the device.  bf16 tensors are carried as int16 bit patterns.
    """
    import torch
    h = host if host is not None else host_inputs(prob, seed)

    def up(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            a = a.view(np.int16)
        return torch.from_numpy(a).to(device)

    table = up(normal_table_bf16())
    n = prob.kv_elems()
    k = torch.empty(n, dtype=torch.int16, device=device)
    v = torch.empty(n, dtype=torch.int16, device=device)
    stream = torch.cuda.current_stream(device).cuda_stream
    fill_kv_device(prob, seed, "k", k.data_ptr(), table.data_ptr(), stream)
    fill_kv_device(prob, seed, "v", v.data_ptr(), table.data_ptr(), stream)
    out = {"qe": up(h["qe"]), "E": up(h["E"]), "q": up(h["q"]), "k": k, "v": v, "table": table, "host": h}
    for name in ("idx_q", "idx_w", "idx_k", "nat_q", "nat_w", "nat_k"):
        if name in h:
            out[name] = up(h[name])
    return out


# ------------------------------------------------------ golden-label inputs
@dataclass
class GoldenProblem:
    """One window of the golden-label pipeline per sequence: tau decoding steps x
    L layers x n_b entries of raw indexer logits.  The logits are N(0, 1)
    noise scaled by 2^sigma_log2; a fraction rel_rate of each sequence's
    entries is relevant, and a relevant entry gets +beta in a fraction
    boost_rate of the (step, layer) rows."""
    name: str
    n_entries: List[int]
    tau: int
    layers: int
    p_num: int = 3
    p_den: int = 5
    theta: int = 3
    sigma_log2: int = 0
    beta: float = 8.5
    rel_rate: float = 1.0 / 256.0
    boost_rate: float = 0.5

    @property
    def batch(self) -> int:
        return len(self.n_entries)

    @property
    def entry_offsets(self) -> List[int]:
        out, acc = [], 0
        for n in self.n_entries:
            out.append(acc)
            acc += n
        return out + [acc]

    def logit_offset(self, b: int) -> int:
        """First element of sequence b's block [tau][L][n_b] in the packed logits."""
        return self.tau * self.layers * self.entry_offsets[b]

    @property
    def total_logits(self) -> int:
        return self.tau * self.layers * self.entry_offsets[-1]


def make_golden_problem(name: str) -> GoldenProblem:
    """Golden-label presets.  Entries are compressed KV entries (4 tokens each):
    the paper's training documents run from 16K to 512K tokens, so 4,096 to
    131,072 entries, with tau = 64 steps and the 21 layers of its backbone."""
    if name == "golden_tiny":
        return GoldenProblem("golden_tiny", [1000], 4, 5, rel_rate=1.0 / 16.0, beta=5.0)
    if name == "golden512k":
        return GoldenProblem("golden512k", [131072], 64, 21)
    if name == "golden_batch":
        u = uniform53(stream_key(0, STREAM_LEN), 100, 8)
        lo, hi = math.log(4096.0), math.log(131072.0)
        return GoldenProblem("golden_batch", [int(math.exp(lo + (hi - lo) * float(x))) for x in u], 64, 21)
    raise KeyError(name)


GOLDEN_PRESETS = ("golden_tiny", "golden512k", "golden_batch")


def _golden_args(gp: GoldenProblem, seed: int, b: int):
    return (stream_key(seed, STREAM_GOLD_NOISE), stream_key(seed, STREAM_GOLD_REL), stream_key(seed, STREAM_GOLD_BOOST),
            float(2.0 ** gp.sigma_log2), float(np.float32(gp.beta)), min(int(gp.rel_rate * 2 ** 32), 2 ** 32 - 1),
            min(int(gp.boost_rate * 2 ** 32), 2 ** 32 - 1))


def golden_table_f32() -> np.ndarray:
    return np.ascontiguousarray(normal_table_f64().astype(np.float32))


def golden_logits(gp: GoldenProblem, seed: int, b: int, steps: Optional[Sequence[int]] = None) -> np.ndarray:
    """Host logits of sequence b, [len(steps)][L][n_b] float32 (all tau steps by default)."""
    kn, kr, kb, sigma, beta, rel, boost = _golden_args(gp, seed, b)
    n, L = gp.n_entries[b], gp.layers
    steps = list(range(gp.tau)) if steps is None else list(steps)
    tab = golden_table_f32()
    out = np.empty((len(steps), L, n), dtype=np.float32)
    for j, i in enumerate(steps):
        start = gp.logit_offset(b) + i * L * n
        host_lib().synth_golden_logits(kn, kr, kb, tab.ctypes.data, start, L, n, b, sigma, beta, rel, boost,
                                       out[j].ctypes.data)
    return out


def golden_logits_device(gp: GoldenProblem, seed: int, device: str = "cuda"):
    """All logits of the problem on the device, packed [B]{[tau][L][n_b]} float32."""
    import torch
    tab = torch.from_numpy(golden_table_f32()).to(device)
    out = torch.empty(gp.total_logits, dtype=torch.float32, device=device)
    stream = torch.cuda.current_stream(device).cuda_stream
    for b in range(gp.batch):
        kn, kr, kb, sigma, beta, rel, boost = _golden_args(gp, seed, b)
        off = gp.logit_offset(b)
        rc = dev_lib().synth_fill_golden_device(kn, kr, kb, tab.data_ptr(), off, gp.tau * gp.layers,
                                                gp.n_entries[b], b, sigma, beta, rel, boost,
                                                out.data_ptr() + 4 * off, stream)
        if rc != 0:
            raise RuntimeError(f"synth_fill_golden_device failed with code {rc}")
    torch.cuda.synchronize()
    return out


# ------------------------------------------------------------------ build
def build_host() -> None:
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", os.path.join(_HERE, "synth.c"),
                           "-o", _HOST_SO])


def build_device() -> None:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    subprocess.check_call([hipcc, "--offload-arch=gfx950", "-O3", "-fPIC", "-shared", "-std=c++17",
                           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                           os.path.join(_HERE, "synth_dev.hip"), "-o", _DEV_SO],
                          stderr=subprocess.DEVNULL if os.environ.get("LSA_QUIET_BUILD") else None)


def build() -> None:
    build_host()
    build_device()
