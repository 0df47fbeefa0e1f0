"""The C ABI on the CPU: every symbol that include/lsa.h declares is exported,
and argument validation rejects bad problems and buffers before any launch."""
import ctypes
import os
import re

import pytest

import paper_2606_09079_amd as L
from paper_2606_09079_amd import lsa as B

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "lsa.h")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_ ]*?[\s\*]+(lsa_[a-z_]+)\s*\(", text, re.M)))


def test_header_declares_the_four_steps():
    names = declared_functions()
    for n in ("lsa_score_chunks", "lsa_topk_chunks", "lsa_sparse_decode_attn", "lsa_decode_step"):
        assert n in names


def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(B._build.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} declared in lsa.h but not exported"
    assert set(declared_functions()) == set(B.EXPORTS)


def test_abi_version_and_status_strings():
    assert L.LIB.lsa_abi_version() == 1
    assert L.LIB.lsa_status_string(0) == b"LSA_OK"
    assert L.LIB.lsa_status_string(3) == b"LSA_ERR_WORKSPACE"


def good(**kw):
    args = dict(ctx_tokens=[64 * 100, 64 * 10], chunk_size=64, keep=[10, 3], n_q_heads=8, n_kv_heads=2)
    args.update(kw)
    return L.Problem(**args)


@pytest.mark.parametrize("kw,status", [
    (dict(ctx_tokens=[]), B.LSA_ERR_INVALID_ARG),
    (dict(ctx_tokens=[64] * 65, keep=[1] * 65), B.LSA_ERR_INVALID_ARG),
    (dict(chunk_size=32, ctx_tokens=[3200, 640]), B.LSA_ERR_UNSUPPORTED),
    (dict(ctx_tokens=[6401, 640]), B.LSA_ERR_INVALID_ARG),
    (dict(ctx_tokens=[0, 640]), B.LSA_ERR_INVALID_ARG),
    (dict(keep=[0, 3]), B.LSA_ERR_INVALID_ARG),
    (dict(keep=[101, 3]), B.LSA_ERR_INVALID_ARG),
    (dict(n_q_heads=9), B.LSA_ERR_INVALID_ARG),
    (dict(head_dim=64), B.LSA_ERR_UNSUPPORTED),
    (dict(emb_dim=100), B.LSA_ERR_UNSUPPORTED),
    (dict(n_lookahead=17), B.LSA_ERR_INVALID_ARG),
    (dict(n_qtok=0), B.LSA_ERR_INVALID_ARG),
    (dict(n_q_heads=64, n_kv_heads=1, n_qtok=4), B.LSA_ERR_UNSUPPORTED),
    (dict(emb_dtype=7), B.LSA_ERR_INVALID_ARG),
    (dict(kv_head_stride=64 * 128, kv_chunk_stride=64 * 128), B.LSA_ERR_INVALID_ARG),
    (dict(kv_head_stride=100), B.LSA_ERR_INVALID_ARG),
    (dict(n_lookahead=2, ctx_tokens=[64 * 300000, 64], keep=[1, 1]), B.LSA_ERR_UNSUPPORTED),
])
def test_validation_rejects(kw, status):
    p = good(**kw)
    assert L.lsa_validate(p) == status
    assert L.last_error() != ""


def test_validation_accepts_presets_and_head_major_strides():
    import lsa_synth
    for name in lsa_synth.PRESETS:
        assert L.lsa_validate(L.Problem.from_synth(lsa_synth.make_problem(name, 0))) == 0
    total = 110
    p = good(kv_head_stride=total * 64 * 128, kv_chunk_stride=64 * 128)
    assert L.lsa_validate(p) == 0


def test_sizes():
    p = good()
    assert L.lsa_max_sel(p) == 10
    assert L.lsa_max_keep(p) == 10
    q = good(n_lookahead=4)
    assert L.lsa_max_sel(q) == 40 and L.lsa_max_keep(q) == 10
    assert L.lsa_workspace_size(q) > L.lsa_workspace_size(p) > 0


FAKE = 1 << 20          # 16-byte aligned, never dereferenced: calls fail validation first
MISALIGNED = FAKE + 4


def _rc(fn, *args):
    return fn(*args)


def test_entry_points_reject_bad_buffers_without_launching():
    p = good()
    ws = L.lsa_workspace_size(p)
    lib = L.LIB
    assert lib.lsa_score_chunks(p.ref, None, FAKE, FAKE, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_score_chunks(p.ref, MISALIGNED, FAKE, FAKE, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_topk_chunks(p.ref, FAKE, None, FAKE, None, FAKE, ws, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_sparse_decode_attn(p.ref, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None, FAKE, ws - 1,
                                      None) == B.LSA_ERR_WORKSPACE
    assert lib.lsa_sparse_decode_attn(p.ref, FAKE, FAKE, FAKE, FAKE, FAKE, float("nan"), FAKE, None, FAKE, ws,
                                      None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_sparse_decode_attn(p.ref, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None, None, ws,
                                      None) == B.LSA_ERR_WORKSPACE
    assert lib.lsa_decode_step(p.ref, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None, FAKE, None, FAKE, ws,
                               None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_decode_step(p.ref, FAKE, FAKE, FAKE, FAKE, MISALIGNED, 0.0, FAKE, None, None, None, FAKE,
                               ws, None) == B.LSA_ERR_INVALID_ARG
    q = good(n_lookahead=3)
    assert lib.lsa_topk_chunks(q.ref, FAKE, FAKE, FAKE, None, FAKE, 16, None) == B.LSA_ERR_WORKSPACE
    with pytest.raises(L.LsaError):
        L.lsa_score_chunks(p, None, FAKE, FAKE, stream=0)


@pytest.mark.parametrize("ix,pkw,status", [
    ((0, 64, 128), {}, B.LSA_ERR_INVALID_ARG),
    ((5, 64, 128), {}, B.LSA_ERR_INVALID_ARG),
    ((3, 48, 128), {}, B.LSA_ERR_UNSUPPORTED),
    ((3, 64, 96), {}, B.LSA_ERR_UNSUPPORTED),
    ((3, 64, 128), dict(n_lookahead=2), B.LSA_ERR_INVALID_ARG),
])
def test_recall_validation_rejects(ix, pkw, status):
    p = good(**pkw)
    idx = L.Indexer(*ix)
    lib = L.LIB
    assert lib.lsa_recall_scores(p.ref, idx.ref, FAKE, FAKE, FAKE, FAKE, None) == status
    assert lib.lsa_recall_select(p.ref, idx.ref, FAKE, FAKE, FAKE, None) == status
    assert L.last_error() != ""


def test_recall_entry_points_reject_bad_buffers_without_launching():
    p = good()
    ws = L.lsa_workspace_size(p)
    idx = L.Indexer(3, 64, 128)
    lib = L.LIB
    assert lib.lsa_recall_scores(p.ref, None, FAKE, FAKE, FAKE, FAKE, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_recall_scores(p.ref, idx.ref, FAKE, MISALIGNED, FAKE, FAKE, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_recall_select(p.ref, idx.ref, FAKE, None, FAKE, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_recall_step(p.ref, idx.ref, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None, None, None,
                               FAKE, ws - 1, None) == B.LSA_ERR_WORKSPACE
    assert lib.lsa_recall_step(p.ref, idx.ref, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None, FAKE, None,
                               FAKE, ws, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_recall_step(p.ref, idx.ref, None, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None, None, None,
                               FAKE, ws, None) == B.LSA_ERR_INVALID_ARG


def test_recall_presets_validate():
    import lsa_synth
    for name in lsa_synth.RECALL_PRESETS:
        prob = lsa_synth.make_problem(name, 0)
        p, idx = L.Problem.from_synth(prob), L.Indexer.from_synth(prob)
        assert L.lsa_validate(p) == 0
        assert L.LIB.lsa_recall_select(p.ref, idx.ref, None, FAKE, FAKE, None) == B.LSA_ERR_INVALID_ARG


def test_two_level_sizes_and_validation():
    ix = L.Indexer(2, 32, 128)
    p = L.Problem([64 * 100 + 13, 64 * 50], 64, [30, 10], 8, 2)     # contexts may end inside a chunk here
    tl = L.TwoLevel(32, [8, 4], [640, 0])
    max_sel, ws = L.lsa_two_level_sizes(p, tl)
    # sequence 0: 101 chunks, window 90 .. 100 (11 chunks), core <= 8; sequence 1: no window, core <= 4
    assert max_sel == 8 + 11 and ws > 0
    assert L.lsa_validate(p) == B.LSA_ERR_INVALID_ARG                # the other paths need whole chunks
    lib = L.LIB
    bad = [L.TwoLevel(48, [8, 4], [640, 0]), L.TwoLevel(32, [0, 4], [640, 0]), L.TwoLevel(32, [8, 4], [-1, 0])]
    for t in bad:
        assert lib.lsa_two_level_sizes(p.ref, t.ref, None, None) != 0
    assert lib.lsa_two_level_sizes(p.ref, None, None, None) == B.LSA_ERR_INVALID_ARG
    q = L.Problem([64 * 100], 64, [30], 8, 2, n_lookahead=2)
    assert lib.lsa_two_level_sizes(q.ref, L.TwoLevel(32, [8], [0]).ref, None, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_two_level_step(p.ref, ix.ref, tl.ref, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0,
                                  FAKE, None, None, None, FAKE, ws, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_two_level_step(p.ref, ix.ref, tl.ref, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0,
                                  FAKE, None, None, None, FAKE, ws - 1, None) == B.LSA_ERR_WORKSPACE


def test_two_level_presets_size():
    import lsa_synth
    import oracle
    for name in lsa_synth.TWO_LEVEL_PRESETS:
        prob = lsa_synth.make_problem(name, 0)
        ms, ws = L.lsa_two_level_sizes(L.Problem.from_synth(prob), L.TwoLevel.from_synth(prob))
        want = 0
        for b in range(prob.batch):
            w0, n_total, _ = oracle.window(prob.ctx_tokens[b], prob.window_tokens[b], prob.chunk)
            want = max(want, min(prob.core_keep[b], prob.keep[b], w0) + n_total - w0)
        assert ms == want


def test_tier_sizes_and_validation():
    p = L.Problem([64 * 300, 64 * 1000], 64, [40, 100], 8, 2)
    T = L.Tier([80, 200])
    pitch, total, ws = L.lsa_tier_sizes(p, T)
    assert (pitch, total) == (100, 280) and ws > 0
    # the reserve plan has the context plan's split-K layout, so its workspace
    # differs from the context's only in the per-chunk score region
    assert ws <= L.lsa_workspace_size(p)
    lib = L.LIB
    for slots in ([79, 200], [80, 199], [80, 65537]):
        assert lib.lsa_tier_sizes(p.ref, L.Tier(slots).ref, None, None, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_tier_sizes(p.ref, None, None, None, None) == B.LSA_ERR_INVALID_ARG
    bad = L.Tier([80, 200])
    bad.c.reserved = 1
    assert lib.lsa_tier_sizes(p.ref, bad.ref, None, None, None) == B.LSA_ERR_INVALID_ARG
    for wgs, status in ((-1, B.LSA_ERR_INVALID_ARG), (1025, B.LSA_ERR_INVALID_ARG), (1024, 0), (4, 0)):
        assert lib.lsa_tier_sizes(p.ref, L.Tier([80, 200], fetch_workgroups=wgs).ref, None, None, None) == status
    la = L.Problem([64 * 300], 64, [40], 8, 2, n_lookahead=2)
    assert lib.lsa_tier_sizes(la.ref, L.Tier([80]).ref, None, None, None) == B.LSA_ERR_INVALID_ARG
    part = L.Problem([64 * 300 + 5], 64, [40], 8, 2)
    assert lib.lsa_tier_sizes(part.ref, L.Tier([80]).ref, None, None, None) == B.LSA_ERR_INVALID_ARG
    big = L.Problem([64 * (131072 + 1)], 64, [40], 8, 2)
    assert lib.lsa_tier_sizes(big.ref, L.Tier([80]).ref, None, None, None) == B.LSA_ERR_UNSUPPORTED
    ok = L.Problem([64 * 131072], 64, [40], 8, 2)
    assert lib.lsa_tier_sizes(ok.ref, L.Tier([80]).ref, None, None, None) == 0


def test_tier_entry_points_reject_bad_buffers_without_launching():
    p = L.Problem([64 * 300, 64 * 1000], 64, [40, 100], 8, 2)
    T = L.Tier([80, 200])
    _, _, ws = L.lsa_tier_sizes(p, T)
    lib = L.LIB
    F2 = FAKE + 4096
    assert lib.lsa_tier_reset(p.ref, T.ref, None, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_tier_plan(p.ref, T.ref, None, FAKE, None, None, FAKE, F2, FAKE, FAKE, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_tier_plan(p.ref, T.ref, FAKE, FAKE, FAKE, None, FAKE, F2, FAKE, FAKE, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_tier_plan(p.ref, T.ref, FAKE, FAKE, None, None, FAKE, FAKE, FAKE, FAKE, None) \
        == B.LSA_ERR_INVALID_ARG  # slot_idx aliases kept_idx
    assert lib.lsa_tier_plan(p.ref, T.ref, FAKE + 1, FAKE, None, None, FAKE, F2, FAKE, FAKE, None) \
        == B.LSA_ERR_INVALID_ARG  # misaligned
    assert lib.lsa_tier_fetch(p.ref, T.ref, None, FAKE, FAKE, FAKE, FAKE, FAKE, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_tier_fetch(p.ref, T.ref, FAKE, FAKE, FAKE, FAKE, None, FAKE, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_tier_attend(p.ref, T.ref, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None, FAKE, ws - 1, None) \
        == B.LSA_ERR_WORKSPACE
    assert lib.lsa_tier_attend(p.ref, T.ref, FAKE, FAKE, FAKE, FAKE, FAKE, float("nan"), FAKE, None, FAKE, ws,
                               None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_tier_attend(p.ref, T.ref, FAKE, None, FAKE, FAKE, FAKE, 0.0, FAKE, None, FAKE, ws, None) \
        == B.LSA_ERR_INVALID_ARG


def test_tier_step_rejects_bad_arguments_without_launching():
    import ctypes
    p = L.Problem([64 * 300, 64 * 1000], 64, [40, 100], 8, 2)
    T = L.Tier([80, 200])
    _, _, ws = L.lsa_tier_sizes(p, T)
    lib = L.LIB
    k2 = (ctypes.c_int32 * 2)(10, 20)
    k2_bad = (ctypes.c_int32 * 2)(10, 0)
    nat = L.Indexer(1, 32, 128)

    def call(nat_=nat, core=k2, ptrs=(FAKE,) * 10, scale=0.0, ws_bytes=ws, ws_ptr=FAKE):
        return lib.lsa_tier_step(p.ref, T.ref, nat_.ref if nat_ is not None else None,
                                 ctypes.cast(core, ctypes.c_void_p) if core is not None else None, *ptrs[:3],
                                 *ptrs[3:6], *ptrs[6:9], scale, ptrs[9], None, FAKE + 12288, FAKE + 4096, ws_ptr, ws_bytes,
                                 None)

    assert call(nat_=None) == B.LSA_ERR_INVALID_ARG
    assert call(nat_=L.Indexer(2, 32, 128)) == B.LSA_ERR_INVALID_ARG   # one native layer
    assert call(nat_=L.Indexer(1, 48, 128)) == B.LSA_ERR_UNSUPPORTED   # head count
    assert call(nat_=L.Indexer(1, 32, 96)) == B.LSA_ERR_UNSUPPORTED    # key width
    assert call(core=None) == B.LSA_ERR_INVALID_ARG
    assert call(core=k2_bad) == B.LSA_ERR_INVALID_ARG                  # k2 >= 1
    assert call(ptrs=(FAKE,) * 3 + (None,) + (FAKE,) * 6) == B.LSA_ERR_INVALID_ARG
    assert call(scale=float("inf")) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_tier_step(p.ref, T.ref, nat.ref, ctypes.cast(k2, ctypes.c_void_p), *(FAKE,) * 5, F2 := FAKE + 8192,
                             *(FAKE,) * 3, 0.0, FAKE, None, F2, FAKE + 4096, FAKE, ws, None) \
        == B.LSA_ERR_INVALID_ARG  # sel_slots aliases slot_idx
    assert call(ws_bytes=ws - 1) == B.LSA_ERR_WORKSPACE
    assert call(ws_ptr=FAKE + 8) == B.LSA_ERR_WORKSPACE
    assert call(ws_ptr=None) == B.LSA_ERR_WORKSPACE
    la = L.Problem([64 * 300], 64, [40], 8, 2, n_lookahead=2)
    assert lib.lsa_tier_step(la.ref, L.Tier([80]).ref, nat.ref, ctypes.cast(k2, ctypes.c_void_p), *(FAKE,) * 9,
                             0.0, FAKE, None, FAKE + 12288, FAKE + 4096, FAKE, ws, None) == B.LSA_ERR_INVALID_ARG


def test_tier_dma_validates_the_host_copy_list_before_copying():
    import numpy as np
    p = L.Problem([64 * 300, 64 * 1000], 64, [40, 100], 8, 2)
    T = L.Tier([80, 200])
    pitch, _, _ = L.lsa_tier_sizes(p, T)
    lib = L.LIB
    fl = np.zeros((2, pitch, 2), dtype=np.int32)
    for counts, entry, what in (([-1, 0], None, "negative count"), ([0, pitch + 1], None, "count above pitch"),
                                ([1, 0], (0, 0, 300, 0), "chunk beyond n_b"), ([1, 0], (0, 0, 5, 80), "slot beyond slots"),
                                ([0, 2], (1, 1, -1, 3), "negative chunk")):
        f = fl.copy()
        if entry is not None:
            b, i, c, s = entry
            f[b, i] = (c, s)
        cnt = np.asarray(counts, dtype=np.int32)
        rc = lib.lsa_tier_fetch_dma(p.ref, T.ref, FAKE, FAKE, f.ctypes.data, cnt.ctypes.data, FAKE, FAKE, None)
        assert rc == B.LSA_ERR_INVALID_ARG, what
    cnt = np.zeros(2, dtype=np.int32)
    assert lib.lsa_tier_fetch_dma(p.ref, T.ref, FAKE, FAKE, None, cnt.ctypes.data, FAKE, FAKE, None) \
        == B.LSA_ERR_INVALID_ARG


def test_golden_sizes_and_validation():
    g = L.Golden([1000, 70], 4, 21)
    ws = L.lsa_golden_sizes(g)
    rows = 4 * 21
    bits = rows * (32 + 3) * 4
    assert ws == (bits + 255) // 256 * 256 + ((32 + 3) * 4 + 255) // 256 * 256
    lib = L.LIB
    bad = [dict(n_entries=[0], n_steps=4, n_layers=21), dict(n_entries=[4194305], n_steps=4, n_layers=21),
           dict(n_entries=[10], n_steps=0, n_layers=21), dict(n_entries=[10], n_steps=4, n_layers=0),
           dict(n_entries=[10], n_steps=4, n_layers=64), dict(n_entries=[10], n_steps=4, n_layers=21, theta=0),
           dict(n_entries=[10], n_steps=4, n_layers=21, theta=65),
           dict(n_entries=[10], n_steps=4, n_layers=21, p_num=0, p_den=5),
           dict(n_entries=[10], n_steps=4, n_layers=21, p_num=6, p_den=5),
           dict(n_entries=[10], n_steps=4, n_layers=21, p_num=1, p_den=(1 << 30) + 1),
           dict(n_entries=[], n_steps=4, n_layers=21)]
    for kw in bad:
        gb = L.Golden(**kw)
        assert lib.lsa_golden_sizes(gb.ref, None) == B.LSA_ERR_INVALID_ARG, kw
    assert lib.lsa_golden_sizes(None, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_golden_labels(g.ref, None, FAKE, FAKE, None, None, FAKE, ws, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_golden_labels(g.ref, FAKE, FAKE, FAKE, FAKE + 4, None, FAKE, ws, None) == B.LSA_ERR_INVALID_ARG
    assert lib.lsa_golden_labels(g.ref, FAKE, FAKE, FAKE, None, None, FAKE, ws - 1, None) == B.LSA_ERR_WORKSPACE
    assert lib.lsa_golden_labels(g.ref, FAKE, FAKE, FAKE, None, None, None, ws, None) == B.LSA_ERR_WORKSPACE


def test_noalloc_rejects_a_step_beyond_its_scratch():
    """lsa_decode_step_noalloc refuses, before any launch, a problem whose
    workspace would not fit LSA_SCRATCH_BYTES (64 MiB), and names both sizes."""
    big = L.Problem([64 * 262144] * 64, 64, [1000] * 64, 8, 8)
    assert L.lsa_workspace_size(big) > 64 << 20
    rc = L.LIB.lsa_decode_step_noalloc(big.ref, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None, None, None, None)
    assert rc == B.LSA_ERR_WORKSPACE
    assert b"67108864" in L.LIB.lsa_last_error()
    # a bad problem is still reported as such, ahead of the size
    bad = L.Problem([100], 64, [1], 8, 8)
    assert L.LIB.lsa_decode_step_noalloc(bad.ref, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None, None, None,
                                         None) == B.LSA_ERR_INVALID_ARG


def test_kv_pack_rejects_bad_arguments_without_launching():
    """lsa_kv_pack validates on the host: first tokens outside [0, ctx], strides
    that are not non-negative multiples of 8 elements, missing or misaligned
    buffers, and a problem the attention would refuse."""
    lib = L.LIB
    p = good(ctx_tokens=[64 * 100 + 5, 64 * 10])  # a partial last chunk is accepted here
    i64 = lambda *v: ctypes.cast((ctypes.c_int64 * len(v))(*v), ctypes.c_void_p)
    ok_first = i64(6400, 0)
    call = lambda first=ok_first, ts=0, hs=0, ptrs=(FAKE,) * 5: lib.lsa_kv_pack(
        p.ref, ptrs[0], ptrs[1], ptrs[2], ts, hs, first, ptrs[3], ptrs[4], None)
    assert call(first=i64(-1, 0)) == B.LSA_ERR_INVALID_ARG
    assert call(first=i64(6406, 0)) == B.LSA_ERR_INVALID_ARG
    assert call(first=i64(0, 641)) == B.LSA_ERR_INVALID_ARG
    for ts, hs in ((-8, 0), (12, 0), (0, 4), (0, -128)):
        assert call(ts=ts, hs=hs) == B.LSA_ERR_INVALID_ARG, (ts, hs)
    for i in range(5):
        ptrs = [FAKE] * 5
        ptrs[i] = None
        assert call(ptrs=tuple(ptrs)) == B.LSA_ERR_INVALID_ARG, i
        ptrs[i] = MISALIGNED
        assert call(ptrs=tuple(ptrs)) == B.LSA_ERR_INVALID_ARG, i
    assert lib.lsa_kv_pack(good(chunk_size=32).ref, FAKE, FAKE, FAKE, 0, 0, None, FAKE, FAKE, None) \
        == B.LSA_ERR_UNSUPPORTED
    # nothing to write (every first token at the context end): accepted with no launch at all
    assert call(first=i64(6405, 640)) == B.LSA_OK


def _no_device():
    import torch
    return torch.cuda.device_count() == 0


@pytest.mark.skipif(not _no_device(), reason="forces the HIP failure by calling where no device exists")
def test_hip_failure_is_reported_as_lsa_err_hip():
    # With no device the HIP runtime refuses every launch on the host, so a
    # call that passes validation must come back as LSA_ERR_HIP with the
    # runtime's message, and the Python binding must raise with that status.
    # The pointers are never dereferenced: the launch itself is refused.
    p = good()
    ws = L.lsa_workspace_size(p)
    lib = L.LIB
    assert lib.lsa_workspace_init(FAKE, 4096, None) == B.LSA_ERR_HIP
    assert "zero-fill launch" in B.last_error()
    assert lib.lsa_score_chunks(p.ref, FAKE, FAKE, FAKE, None) == B.LSA_ERR_HIP
    assert "score launch" in B.last_error()
    assert lib.lsa_decode_step(p.ref, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None, None, None, FAKE, ws,
                               None) == B.LSA_ERR_HIP
    with pytest.raises(L.LsaError) as e:
        L.lsa_score_chunks(p, FAKE, FAKE, FAKE, stream=0)
    assert e.value.status == B.LSA_ERR_HIP
