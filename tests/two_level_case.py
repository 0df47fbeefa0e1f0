"""One parity run of the two-level path against the oracle on a seeded problem.

Through the C ABI: lsa_two_level_step (Level-1 recall over the history,
Level-2 native top-k inside the recalled set, the always-resident window with a
partial last chunk, attention).  The kept set must equal the oracle's; where it
differs, every differing chunk must sit inside the float32 band of a decision
(the recall threshold, the K_max cut or the Level-2 cut), and the attention is
then compared with the oracle's attention over the GPU's set.  Attention is
compared token by token, the last chunk cut at the context end.
"""
from __future__ import annotations

import time
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

import lsa_synth as synth
import oracle
import parity
from gpu_case import log


def _explained(diff, x, tol_x, native, tol_n, recalled, kmax, k2) -> bool:
    """Every chunk in which the GPU and the oracle disagree sits in the band of
    one of the three decisions."""
    r = x.max(axis=0) if x.shape[1] else np.zeros(0)
    tr = tol_x.max(axis=0) if x.shape[1] else np.zeros(0)
    rec = set(recalled.tolist())
    cut1 = np.sort(r[r >= 0])[::-1]
    kth1 = cut1[kmax - 1] if len(cut1) > kmax else None   # Level-1 bound active
    nat_rec = np.sort(native[list(rec)])[::-1] if rec else np.zeros(0)
    kth2 = nat_rec[k2 - 1] if len(nat_rec) > k2 else None  # Level-2 cut active
    for s in diff:
        ok = abs(r[s]) <= tr[s]
        ok = ok or (kth1 is not None and abs(r[s] - kth1) <= 2 * tr[s] + 1e-30)
        ok = ok or (kth2 is not None and abs(native[s] - kth2) <= 2 * tol_n[s] + 1e-30)
        if not ok:
            return False
    return True


def run_two_level_case(prob, seed: int, rows: Optional[Sequence[Tuple[int, int]]] = None,
                       host: Optional[Dict[str, object]] = None) -> Dict[str, object]:
    import torch
    import paper_2606_09079_amd as L

    log(f"[two-level] {prob.name} seed={seed} B={prob.batch} ctx={prob.ctx_tokens[:4]} C={prob.chunk} "
        f"kmax={prob.keep[:4]} k2={prob.core_keep[:4]} window={prob.window_tokens[:4]} L={prob.idx_layers} "
        f"n_h={prob.idx_heads} native={prob.nat_heads} c={prob.idx_dim} Hq={prob.n_q_heads} Hkv={prob.n_kv_heads} "
        f"Tq={prob.n_qtok}")
    t0 = time.time()
    host = synth.host_inputs(prob, seed) if host is None else host
    dev = synth.device_inputs(prob, seed, host=host)
    P, ix, tl = L.Problem.from_synth(prob), L.Indexer.from_synth(prob), L.TwoLevel.from_synth(prob)
    max_sel, ws_bytes = L.lsa_two_level_sizes(P, tl)
    B = prob.batch
    ws = torch.zeros(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    shp = (B, prob.n_qtok, prob.n_q_heads, prob.head_dim)
    out = torch.full(shp, float("nan"), dtype=torch.float32, device="cuda")
    lse = torch.full(shp[:3], float("nan"), dtype=torch.float32, device="cuda")
    sel = torch.full((B, max_sel), -1, dtype=torch.int32, device="cuda")
    cnt = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    L.lsa_two_level_step(P, ix, tl, dev["idx_q"], dev["idx_w"], dev["idx_k"], dev["nat_q"], dev["nat_w"],
                         dev["nat_k"], dev["q"], dev["k"], dev["v"], 0.0, out, lse, sel, cnt, ws, ws_bytes)
    torch.cuda.synchronize()
    g_out, g_lse, g_sel, g_cnt = out.cpu().numpy(), lse.cpu().numpy(), sel.cpu().numpy(), cnt.cpu().numpy()
    log(f"[two-level] gpu step done ({time.time() - t0:.1f}s), kept {g_cnt.tolist()[:8]}")

    rows = [(t, h) for t in range(prob.n_qtok) for h in range(prob.n_q_heads)] if rows is None else list(rows)
    modes: Dict[int, str] = {}
    worst = 0.0
    for b in range(B):
        lo = prob.chunk_offsets[b]
        x, recalled, native, kept, _ = oracle.two_level_for_sequence(prob, host, b)
        c = int(g_cnt[b])
        assert 0 <= c <= max_sel, f"seq {b}: kept count {c}"
        got = g_sel[b, :c].astype(np.int64)
        assert np.all(np.diff(got) > 0), f"seq {b}: kept ids not strictly ascending"
        w0, n_total, _ = oracle.window(prob.ctx_tokens[b], prob.window_tokens[b] if prob.window_tokens else 0,
                                       prob.chunk)
        assert np.array_equal(got[got >= w0], np.arange(w0, n_total)), f"seq {b}: window chunks differ"
        if np.array_equal(got, kept):
            modes[b] = "exact"
        else:
            n_hist = w0
            tol_x = np.stack([parity.index_score_tolerance(host["idx_q"][b, l], host["idx_w"][b, l],
                                                           host["idx_k"][l, lo:lo + n_hist])
                              for l in range(prob.idx_layers)])
            tol_n = parity.index_score_tolerance(host["nat_q"][b], host["nat_w"][b], host["nat_k"][lo:lo + n_hist])
            diff = sorted(set(got.tolist()) ^ set(kept.tolist()))
            assert _explained(diff, x, tol_x, native, tol_n, recalled, prob.keep[b], prob.core_keep[b]), \
                f"seq {b}: kept set differs from the oracle at chunks {diff[:10]} outside every band"
            modes[b] = "band"
        toks = oracle.kept_tokens(got, prob.chunk, prob.ctx_tokens[b])
        G = prob.group
        by_g: Dict[int, list] = {}
        for (t, h) in rows:
            by_g.setdefault(h // G, []).append((t, h))
        for g, rs in sorted(by_g.items()):
            Kh = synth.kv_head_sparse(prob, seed, "k", b, g, got)
            Vh = synth.kv_head_sparse(prob, seed, "v", b, g, got)
            qr = np.stack([host["q"][b, t, h] for (t, h) in rs])
            r_out, r_lse = oracle.attention_tokens(qr, Kh, Vh, toks)
            go = np.stack([g_out[b, t, h] for (t, h) in rs])
            gl = [g_lse[b, t, h] for (t, h) in rs]
            if len(toks) == 0:
                assert np.all(go == 0.0) and np.all(np.isneginf(gl)), f"seq {b}: empty set must give 0 / -inf"
                continue
            worst = max(worst, parity.check_attention(go, gl, r_out, r_lse, f"{prob.name} two-level seq {b} g {g}"))
    log(f"[two-level] parity ok (modes {sorted(set(modes.values()))}, worst rel err {worst:.2e}) "
        f"({time.time() - t0:.1f}s)")
    return {"modes": modes, "worst_attn": worst, "cnt": g_cnt, "sel": g_sel}
