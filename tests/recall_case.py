"""One parity run of the recall path against the oracle on a seeded problem.

Through the C ABI: the per-layer index scores (lsa_recall_scores), the recall
from those scores (lsa_recall_select), the recall from the oracle's own scores
rounded to float32 (both sides then decide on the same values, so the sets must
be identical), and the fused lsa_recall_step, whose recalled set must equal the
one selected from the GPU's scores and whose attention is compared with the
oracle's attention over that (validated) set.
"""
from __future__ import annotations

import time
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

import lsa_synth as synth
import oracle
import parity
from gpu_case import log


def run_recall_case(prob, seed: int, rows: Optional[Sequence[Tuple[int, int]]] = None,
                    host: Optional[Dict[str, object]] = None) -> Dict[str, object]:
    import torch
    import paper_2606_09079_amd as L

    log(f"[recall] {prob.name} seed={seed} B={prob.batch} ctx={prob.ctx_tokens[:4]} C={prob.chunk} "
        f"kmax={prob.keep[:4]} L={prob.idx_layers} n_h={prob.idx_heads} c={prob.idx_dim} "
        f"Hq={prob.n_q_heads} Hkv={prob.n_kv_heads} Tq={prob.n_qtok}")
    t0 = time.time()
    host = synth.host_inputs(prob, seed) if host is None else host
    dev = synth.device_inputs(prob, seed, host=host)
    P, ix = L.Problem.from_synth(prob), L.Indexer.from_synth(prob)
    B, Lay, total = prob.batch, prob.idx_layers, prob.total_chunks
    offs = prob.chunk_offsets
    ws_bytes = L.lsa_workspace_size(P)
    ws = torch.zeros(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    max_sel = L.lsa_max_sel(P)

    x = torch.full((Lay, total), float("nan"), dtype=torch.float32, device="cuda")
    L.lsa_recall_scores(P, ix, dev["idx_q"], dev["idx_w"], dev["idx_k"], x)
    sel = torch.full((B, max_sel), -1, dtype=torch.int32, device="cuda")
    cnt = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    L.lsa_recall_select(P, ix, x, sel, cnt)
    torch.cuda.synchronize()
    g_x, g_sel, g_cnt = x.cpu().numpy(), sel.cpu().numpy(), cnt.cpu().numpy()
    log(f"[recall] gpu scores + select done ({time.time() - t0:.1f}s)")

    ref_x: List[np.ndarray] = []
    modes: Dict[int, str] = {}
    worst = 0.0
    for b in range(B):
        lo, hi = offs[b], offs[b + 1]
        xb, _ = oracle.recall_for_sequence(prob, host, b)
        tol = np.stack([parity.index_score_tolerance(host["idx_q"][b, l], host["idx_w"][b, l],
                                                     host["idx_k"][l, lo:hi]) for l in range(Lay)])
        for l in range(Lay):
            worst = max(worst, parity.check_index_scores(g_x[l, lo:hi], xb[l], tol[l],
                                                         f"{prob.name} seq {b} layer {l}"))
        c = int(g_cnt[b])
        assert 0 <= c <= prob.keep[b], f"seq {b}: recalled count {c}"
        modes[b] = parity.check_recall(g_sel[b, :c], xb, tol, prob.keep[b], f"{prob.name} seq {b}")
        ref_x.append(xb)
    log(f"[recall] scores + recall parity ok (worst score err {worst:.2e}, modes {sorted(set(modes.values()))}) "
        f"({time.time() - t0:.1f}s)")

    # the same decision on the same float32 values: identical sets
    x32 = np.zeros((Lay, total), dtype=np.float32)
    for b in range(B):
        x32[:, offs[b]:offs[b + 1]] = ref_x[b].astype(np.float32)
    sel3 = torch.full((B, max_sel), -1, dtype=torch.int32, device="cuda")
    cnt3 = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    L.lsa_recall_select(P, ix, torch.from_numpy(x32).cuda(), sel3, cnt3)
    torch.cuda.synchronize()
    e_sel, e_cnt = sel3.cpu().numpy(), cnt3.cpu().numpy()
    for b in range(B):
        want = oracle.recall(x32[:, offs[b]:offs[b + 1]].astype(np.float64), prob.keep[b])
        got = e_sel[b, :e_cnt[b]]
        assert e_cnt[b] == len(want) and np.array_equal(got, want), \
            f"seq {b}: recall on identical float32 scores differs ({e_cnt[b]} vs {len(want)})"
    log(f"[recall] exact recall on identical scores ok ({time.time() - t0:.1f}s)")

    # fused step
    shp = (B, prob.n_qtok, prob.n_q_heads, prob.head_dim)
    out = torch.full(shp, float("nan"), dtype=torch.float32, device="cuda")
    lse = torch.full(shp[:3], float("nan"), dtype=torch.float32, device="cuda")
    sel2 = torch.full((B, max_sel), -1, dtype=torch.int32, device="cuda")
    cnt2 = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    L.lsa_recall_step(P, ix, dev["idx_q"], dev["idx_w"], dev["idx_k"], dev["q"], dev["k"], dev["v"], 0.0, out, lse,
                      sel2, cnt2, ws, ws_bytes)
    torch.cuda.synchronize()
    f_out, f_lse, f_sel, f_cnt = out.cpu().numpy(), lse.cpu().numpy(), sel2.cpu().numpy(), cnt2.cpu().numpy()
    assert np.array_equal(f_cnt, g_cnt), f"fused recalled counts {f_cnt} differ from lsa_recall_select {g_cnt}"
    rows = [(t, h) for t in range(prob.n_qtok) for h in range(prob.n_q_heads)] if rows is None else list(rows)
    worst_attn = 0.0
    for b in range(B):
        kept = f_sel[b, :f_cnt[b]].astype(np.int64)
        assert np.array_equal(kept, g_sel[b, :g_cnt[b]]), f"fused recalled set differs, seq {b}"
        if len(kept) == 0:
            for (t, h) in rows:
                assert np.all(f_out[b, t, h] == 0.0), f"seq {b} ({t}, {h}): empty recall must give out = 0"
                assert np.isneginf(f_lse[b, t, h]), f"seq {b} ({t}, {h}): empty recall must give lse = -inf"
            continue
        kv = lambda which, bb, g, ch: synth.kv_head_sparse(prob, seed, which, bb, g, ch)
        res = oracle.attend_rows(prob, host, b, kept, rows, kv)
        keys = list(res.keys())
        worst_attn = max(worst_attn, parity.check_attention(
            np.stack([f_out[b, t, h] for (t, h) in keys]), [f_lse[b, t, h] for (t, h) in keys],
            np.stack([res[k_][0] for k_ in keys]), [res[k_][1] for k_ in keys], f"{prob.name} recall attn seq {b}"))
    log(f"[recall] fused step parity ok (worst rel err {worst_attn:.2e}, recalled {f_cnt.tolist()[:8]}) "
        f"({time.time() - t0:.1f}s)")
    return {"modes": modes, "worst_score": worst, "worst_attn": worst_attn, "cnt": f_cnt, "sel": f_sel,
            "out": f_out, "lse": f_lse}
