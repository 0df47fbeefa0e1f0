"""Benchmark of the LSA decode hot path on one MI355X.

One step = the whole hot path -- score every chunk, keep the top-k, sparse
decode attention over the kept chunks -- as one ``lsa_decode_step`` call on
inputs already resident in HBM.  Workload: the paper-scale single sequence, a
1,048,576-token context in 16,384 chunks of 64 tokens, keep 1,638 chunks (10%),
32 query heads over 8 KV heads of dim 128, bf16 K/V, bf16 indexer embeddings of
dim 256.  Four query sets (query embedding and attention query) rotate from
step to step so that each step keeps a different chunk set and the 256 MB
Infinity Cache cannot serve a previous step's bytes.

The other workloads (``--workload``) use the same loop, for profiling.

Prints one JSON line: steps/s, plus a ``roofline`` object for the dominant
kernel (sparse attention: algorithmic bytes = kept K/V + q + out, divided by
its HIP-event-timed average launch duration on the launch stream) and a
``cpu_baseline`` object (the CPU oracle on a bounded sample of the same
workload, on the host cores of this run).
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode steps/sec for score+top-k+sparse attn at 1M ctx; achieved HBM GB/s"
HBM_PEAK_GBS = 8000.0
WORKLOADS = {
    "paper1m": "paper1m: 1,048,576-token context, 64-token chunks (16,384), keep 1,638 (10%), "
               "32 query / 8 KV heads, head_dim 128, bf16 K/V, bf16 indexer dim 256, batch 1",
    "lookahead": "lookahead: 8 sequences x 1,048,576 tokens, 128-token chunks (8,192 each), 16 lookahead "
                 "query embeddings, union of per-query top-512, 16 query tokens, 64 query / 8 KV heads, "
                 "head_dim 128, bf16 K/V, bf16 indexer dim 256",
    "batch32": "batch32: 32 sequences, log-uniform 32K-512K tokens, 64-token chunks, keep 13.5%, "
               "32 query / 8 KV heads, head_dim 128, bf16 K/V, bf16 indexer dim 256",
    "int8": "int8: 4 sequences x 131,072 tokens, 64-token chunks (2,048 each), keep 256, 32 query / 8 KV heads, "
            "head_dim 128, bf16 K/V, int8 indexer dim 256",
    "tiny": "tiny: 4,096 tokens, 64-token chunks (64), keep 8, 8 query / 8 KV heads, head_dim 128, bf16 K/V, "
            "fp32 indexer dim 256",
    "recall1m": "recall1m: 1,048,576-token context, 64-token chunks (16,384), full Memory Indexer of 3 layers x 64 "
                "heads x 128-wide bf16 index keys, sigmoid threshold 1/2, OR over layers, K_max 1,638 (10%), "
                "32 query / 8 KV heads, head_dim 128, bf16 K/V, batch 1",
    "recall_batch": "recall_batch: 4 sequences x 131,072 tokens, 64-token chunks (2,048 each), Memory Indexer of "
                    "2 layers x 32 heads x 128, no K_max cut, 32 query / 8 KV heads, head_dim 128, bf16 K/V",
    "recall_tiny": "recall_tiny: 4,096 tokens, 64-token chunks (64), Memory Indexer of 3 layers x 16 heads x 64, "
                   "K_max 12, 8 query / 8 KV heads, head_dim 128, bf16 K/V",
    "twolevel1m": "twolevel1m: 1,048,613-token context (16,385 64-token chunks, the last one 37 tokens), Level 1: "
                  "Memory Indexer of 3 layers x 64 heads x 128 over the history, K_max 2,048; Level 2: native "
                  "indexer of 64 heads keeps 1,024; plus the window of the last 8,192 tokens; 32 query / 8 KV heads, "
                  "head_dim 128, bf16 K/V, batch 1",
    "tier1m": "tier1m: the recall1m context and Memory Indexer with the host tier: K/V in a pinned host mirror, a "
              "GPU reserve of 2 x K_max chunk slots; every 64 decode steps the indexer fires (recall, residency plan, "
              "copies of the missing chunks by a copy kernel reading the mirror over PCIe) on a second stream, and "
              "the new set is read from the next step on; each decode step attends over the reserve",
    "tier2l1m": "tier2l1m: tier1m with Level 2 inside the resident set: every decode step scores the resident kept "
                "chunks with a native indexer of 64 heads x 128, keeps the 1,024 best and attends over their reserve "
                "slots (lsa_tier_step); firings and copies as tier1m",
    "golden512k": "golden512k: golden-label window of a 512K-token context, 131,072 compressed entries x 64 decoding "
                  "steps x 21 layers of float32 indexer logits (704 MB), top-p 0.6, votes >= 3, union over the window",
    "golden_batch": "golden_batch: 8 golden-label windows of 4,096-131,072 entries (log-uniform), 64 steps x 21 layers",
    "kvpack1m": "kvpack1m: re-layout of the paper1m context's token-major K/V ([1,048,576 tokens][8 KV heads][128] "
                "bf16 each) into the chunk-paged blocks the attention reads (lsa_kv_pack, every token), plus the "
                "per-step append of one decoded token to paper1m and to each of the 32 batch32 sequences",
    "twolevel_tiny": "twolevel_tiny: 4,133 tokens (65 chunks, the last one 37 tokens), Level 1 3 x 16 x 64 with "
                     "K_max 24, Level 2 keeps 6, window 512 tokens, 8 query / 8 KV heads, head_dim 128, bf16 K/V",
}
EMB_BYTES = {"f32": 4, "bf16": 2, "i8": 1}
PMC_SUMMARY = os.path.join(ROOT, "profiles", "attn_kernel_paper1m_traffic.md")
PACK_SUMMARY = os.path.join(ROOT, "profiles", "kvpack_kernel_kvpack1m.md")


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def code_sha(name: str) -> str:
    """sha256[:16] of a kernel source with comments and blank lines removed, so
    that counter summaries stay valid across edits that touch only comments."""
    with open(os.path.join(ROOT, "paper_2606_09079_amd", "csrc", name)) as f:
        text = f.read()
    text = re.sub(r"//[^\n]*", "", text)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = "\n".join(line.rstrip() for line in text.splitlines() if line.strip())
    return hashlib.sha256(text.encode()).hexdigest()[:16]


def calibration_copy(args, stream) -> None:
    """Profiling aid: one plain 16-byte copy of a known size, whose counter
    readings calibrate the traffic counters of the same run."""
    if not args.copy_calibration_mib:
        return
    import torch

    import lsa_synth as synth
    nbytes = args.copy_calibration_mib << 20
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    synth.copy_device(src.data_ptr(), dst.data_ptr(), nbytes, stream.cuda_stream)
    torch.cuda.synchronize()
    log(f"[bench] calibration copy of {nbytes} bytes done")


def part_times(L, prob, P, ix, dev, rot, max_sel, stream, attn_us: float, n: int):
    """Average microseconds of the step's parts, each entry point launched on
    its own between HIP events on the launch stream: scoring, selection (with
    the union for several lookahead queries), attention (split + combine,
    measured with the roofline).  Recall workloads score with lsa_recall_scores
    and select with lsa_recall_select."""
    import torch
    B, Q = prob.batch, prob.n_lookahead
    recall = prob.idx_layers > 0
    if recall:
        scores = torch.empty(prob.idx_layers * prob.total_chunks, dtype=torch.float32, device="cuda")
    else:
        scores = torch.empty(Q * prob.total_chunks, dtype=torch.int32 if prob.emb_dtype == "i8" else torch.float32,
                             device="cuda")
    sel = torch.empty(B, max_sel, dtype=torch.int32, device="cuda")
    cnt = torch.empty(B, dtype=torch.int32, device="cuda")
    pq = torch.empty(B, Q, L.lsa_max_keep(P), dtype=torch.int32, device="cuda") if Q > 1 else None

    def score(i):
        r = rot[i % len(rot)]
        if recall:
            L.lsa_recall_scores(P, ix, r["idx_q"], r["idx_w"], dev["idx_k"], scores, stream)
        else:
            L.lsa_score_chunks(P, r["qe"], dev["E"], scores, stream)

    def select(i):
        if recall:
            L.lsa_recall_select(P, ix, scores, sel, cnt, stream)
        else:
            L.lsa_topk_chunks(P, scores, sel, cnt, pq, stream=stream)

    res = {}
    for name, fn in (("score", score), ("select", select)):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        for i in range(n):
            if name == "select":
                score(i)
            evs[i][0].record(stream)
            fn(i)
            evs[i][1].record(stream)
        torch.cuda.synchronize()
        res[name] = round(1e3 * sum(a.elapsed_time(b) for a, b in evs) / n, 2)
    res["attention"] = round(attn_us, 2)
    res["how"] = ("each entry point on its own between HIP events (score: lsa_score_chunks / lsa_recall_scores, "
                  "which write scores where the fused step writes order keys; select: lsa_topk_chunks / "
                  "lsa_recall_select; attention: lsa_sparse_decode_attn, split kernel + combine)")
    return res


def trace_kernels(workload: str):
    """Per-kernel average durations (us) from the committed rocprofv3 trace of
    this workload, or None when there is none or it was taken on other kernel
    source (every source file it names must still hash the same)."""
    path = os.path.join(ROOT, "profiles", f"step_kernels_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    for src, digest in re.findall(r"(\w+\.hip)[: ]+([0-9a-f]{16})", text):
        if code_sha(src) != digest:
            return None
    rows = re.findall(r"^\| `([^`]+)` \| (\d+) \| ([0-9.]+) \|", text, flags=re.M)
    if not rows:
        return None
    return {"source": os.path.relpath(path, ROOT), "average_us": {k: float(a) for k, _, a in rows}}


def history_chunks(prob, b: int) -> int:
    """Complete chunks before the always-resident window of sequence b (the
    Level-1 index keys a two-level step reads), for the byte count."""
    W = prob.window_tokens[b] if prob.window_tokens else 0
    L = prob.ctx_tokens[b]
    return min(max(L - W, 0) // prob.chunk, L // prob.chunk)


def measured_traffic(summary: str = PMC_SUMMARY, source: str = "attn.hip"):
    """HBM bytes per launch of the dominant kernel from a committed rocprofv3
    counter summary, or None when the summary is missing or was taken on other
    kernel source."""
    if not os.path.exists(summary):
        return None
    text = open(summary).read()
    m = re.search(re.escape(source) + r" code sha256\[:16\]:\s*([0-9a-f]{16})", text)
    t = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m or not t or m.group(1) != code_sha(source):
        return None
    return float(t.group(1))


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="paper1m", choices=sorted(WORKLOADS))
    ap.add_argument("--rotations", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="bound on the oracle sample's CPU time")
    ap.add_argument("--only", choices=["step", "attn"], default=None,
                    help="profiling aid: launch only this entry point in the timed loop")
    ap.add_argument("--read-ceiling-mib", type=int, default=2048,
                    help="size of the plain streaming read that measures the read-bandwidth ceiling "
                         "(a multiple of 32; 0: skip)")
    ap.add_argument("--flush-mib", type=int, default=None,
                    help="untimed streaming read between the per-step samples of the step-time distribution, "
                         "so that the 256 MB Infinity Cache cannot serve a previous step's bytes "
                         "(a multiple of 32; default: 1024 for workloads below 1 GB per step, else 0)")
    ap.add_argument("--tier-fetch-wgs", type=int, default=8, choices=(4, 8, 16, 32),
                    help="tier1m / tier2l1m: workgroups of the copy kernel in the steady-state side band")
    ap.add_argument("--tier-lag", type=int, default=48,
                    help="tier1m: decode steps from a firing until its kept set is read (1 .. 63)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="profiling aid: also run one plain copy of this many MiB (known bytes)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures the decode hot path on exactly one GPU; --gpus {args.gpus} is not "
              f"supported (the kernels run on one GPU's share; sharding is a design note only)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import lsa_synth as synth
    import paper_2606_09079_amd as L

    torch.cuda.set_device(0)
    if args.workload in ("tier1m", "tier2l1m"):
        return bench_tier(args)
    if args.workload.startswith("golden"):
        return bench_golden(args)
    if args.workload == "kvpack1m":
        return bench_kvpack(args)
    stream = torch.cuda.current_stream()
    prob = synth.make_problem(args.workload, 0)
    t_setup = time.time()
    host0 = synth.host_inputs(prob, 0)
    dev = synth.device_inputs(prob, 0, host=host0)
    recall = prob.idx_layers > 0
    two_level = bool(prob.core_keep)

    def up(a):
        a = np.ascontiguousarray(a)
        return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).cuda()

    rot = []
    for r in range(args.rotations):
        h = host0 if r == 0 else synth.host_inputs(prob, 1000 + r)
        # the query side changes from step to step; embeddings, index keys and K/V stay
        rot.append({"qe": up(h["qe"]), "q": up(h["q"]),
                    **({"idx_q": up(h["idx_q"]), "idx_w": up(h["idx_w"])} if recall else {}),
                    **({"nat_q": up(h["nat_q"]), "nat_w": up(h["nat_w"])} if two_level else {})})
    P = L.Problem.from_synth(prob)
    ix = L.Indexer.from_synth(prob) if recall else None
    tl = L.TwoLevel.from_synth(prob) if two_level else None
    B, Tq, Hq, d = prob.batch, prob.n_qtok, prob.n_q_heads, prob.head_dim
    if two_level:
        max_sel, ws_bytes = L.lsa_two_level_sizes(P, tl)
    else:
        ws_bytes, max_sel = L.lsa_workspace_size(P), L.lsa_max_sel(P)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    out = torch.empty(B, Tq, Hq, d, dtype=torch.float32, device="cuda")
    lse = torch.empty(B, Tq, Hq, dtype=torch.float32, device="cuda")
    sels = [torch.empty(B, max_sel, dtype=torch.int32, device="cuda") for _ in rot]
    cnts = [torch.empty(B, dtype=torch.int32, device="cuda") for _ in rot]
    torch.cuda.synchronize()
    log(f"[bench] setup {time.time() - t_setup:.1f}s, workspace {ws_bytes / 2**20:.1f} MiB")

    def step(i: int) -> None:
        r = rot[i % len(rot)]
        if two_level:
            L.lsa_two_level_step(P, ix, tl, r["idx_q"], r["idx_w"], dev["idx_k"], r["nat_q"], r["nat_w"],
                                 dev["nat_k"], r["q"], dev["k"], dev["v"], 0.0, out, lse, sels[i % len(rot)],
                                 cnts[i % len(rot)], ws, ws_bytes, stream)
        elif recall:
            L.lsa_recall_step(P, ix, r["idx_q"], r["idx_w"], dev["idx_k"], r["q"], dev["k"], dev["v"], 0.0, out,
                              lse, sels[i % len(rot)], cnts[i % len(rot)], ws, ws_bytes, stream)
        else:
            L.lsa_decode_step(P, r["qe"], dev["E"], r["q"], dev["k"], dev["v"], 0.0, out, lse, sels[i % len(rot)],
                              cnts[i % len(rot)], ws, ws_bytes, stream)

    # attention alone over the kept sets of the steps; the two-level kept sets
    # have the row pitch of a problem whose keep budget is that pitch
    PA = L.Problem(prob.ctx_tokens, prob.chunk, [max_sel] * B, prob.n_q_heads, prob.n_kv_heads, prob.head_dim,
                   prob.emb_dim, prob.n_lookahead, prob.n_qtok, prob.emb_dtype) if two_level else P

    def attn(i: int) -> None:
        L.lsa_sparse_decode_attn(PA, rot[i % len(rot)]["q"], dev["k"], dev["v"], sels[i % len(rot)],
                                 cnts[i % len(rot)], 0.0, out, lse, ws, ws_bytes, stream)

    # every rotation's kept set exists before any attention-only launch
    for i in range(len(rot)):
        step(i)
    torch.cuda.synchronize()

    calibration_copy(args, stream)

    fn = attn if args.only == "attn" else step
    for i in range(args.warmup):
        fn(i)
    torch.cuda.synchronize()

    # ---- timed region: exactly K steps, synchronised on both sides
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        fn(i)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = ev0.elapsed_time(ev1)
    ms_per_step = ms_total / args.steps
    log(f"[bench] timed {args.steps} x {fn.__name__}: {ms_per_step * 1e3:.2f} us/step (wall {wall:.3f}s)")

    # ---- distribution of single-step times (HIP events around each step, outside
    # the timed region), with an optional untimed cache flush between samples
    flush_mib = args.flush_mib
    sink = torch.empty(synth.read_sink_words(), dtype=torch.int32, device="cuda")
    n_dist = max(args.steps, 100)
    dist_bufs = None
    step_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n_dist)]

    def flush() -> None:
        if dist_bufs is not None:
            synth.read_device(dist_bufs.data_ptr(), dist_bufs.numel(), sink.data_ptr(), stream.cuda_stream)

    # ---- dominant kernel: per-launch HIP events around the attention launch
    n_att = max(args.steps, 20)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n_att)]
    for i in range(n_att):
        evs[i][0].record(stream)
        attn(i)
        evs[i][1].record(stream)
    torch.cuda.synchronize()
    att_ms = [a.elapsed_time(b) for a, b in evs]
    att_avg_us = 1e3 * sum(att_ms) / len(att_ms)

    # ---- the step's parts, each entry point on its own with HIP events around
    # it (the fused step runs the same kernels back to back)
    parts_us = part_times(L, prob, P, ix, dev, rot, max_sel, stream, attn_us=att_avg_us,
                          n=max(20, min(args.steps, 200))) if not two_level else None

    counts = [int(c.cpu().sum()) for c in cnts]
    C_, Hkv_ = prob.chunk, prob.n_kv_heads
    approx_step_bytes = sum(counts) / len(counts) * C_ * Hkv_ * d * 4
    if flush_mib is None:
        flush_mib = 1024 if approx_step_bytes < 1e9 else 0
    if flush_mib:
        dist_bufs = torch.empty(flush_mib << 20, dtype=torch.uint8, device="cuda")
    fn_dist = attn if args.only == "attn" else step
    for i in range(n_dist):
        flush()
        step_ev[i][0].record(stream)
        fn_dist(i)
        step_ev[i][1].record(stream)
    torch.cuda.synchronize()
    step_us = sorted(1e3 * a.elapsed_time(b) for a, b in step_ev)

    def pct(p: float) -> float:
        return round(step_us[min(len(step_us) - 1, int(p * len(step_us)))], 2)

    dist_bufs = None

    # ---- read-bandwidth ceiling of this device: a plain streaming read
    read_gbs = None
    if args.read_ceiling_mib:
        rbuf = torch.ones(args.read_ceiling_mib << 20, dtype=torch.uint8, device="cuda")
        rev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(6)]
        for a_, b_ in rev:
            a_.record(stream)
            synth.read_device(rbuf.data_ptr(), rbuf.numel(), sink.data_ptr(), stream.cuda_stream)
            b_.record(stream)
        torch.cuda.synchronize()
        best_ms = min(a_.elapsed_time(b_) for a_, b_ in rev[1:])
        read_gbs = rbuf.numel() / (best_ms * 1e-3) / 1e9
        del rbuf
    C, Hkv = prob.chunk, prob.n_kv_heads
    kv_bytes = [n * C * Hkv * d * 2 * 2 for n in counts]
    attn_bytes = sum(kv_bytes) / len(kv_bytes) + B * Tq * Hq * d * (2 + 4) + B * Tq * Hq * 4 + max(counts) * 4
    if two_level:  # Level-1 keys of the history, native keys of (at most) K_max recalled chunks, queries, gates
        Lay, nh, c = prob.idx_layers, prob.idx_heads, prob.idx_dim
        hist = sum(history_chunks(prob, b) for b in range(B))
        rec = sum(min(prob.keep[b], history_chunks(prob, b)) for b in range(B))
        emb_bytes = (Lay * hist + rec) * c * 2 + B * (Lay * nh + prob.nat_heads) * (c * 2 + 4)
    elif recall:  # index keys of every layer, plus the indexer queries and gates
        Lay, nh, c = prob.idx_layers, prob.idx_heads, prob.idx_dim
        emb_bytes = Lay * prob.total_chunks * c * 2 + B * Lay * nh * (c * 2 + 4)
    else:
        emb_bytes = (prob.total_chunks + B * prob.n_lookahead) * prob.emb_dim * EMB_BYTES[prob.emb_dtype]
    step_bytes = attn_bytes + emb_bytes
    achieved = attn_bytes / (att_avg_us * 1e-6) / 1e9
    traffic = measured_traffic() if args.workload == "paper1m" else None

    result = {
        "metric": METRIC,
        "value": round(1e3 / ms_per_step, 2) if args.only in (None, "step") else None,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOADS[args.workload], "global_batch": B, "seq_len": prob.ctx_tokens[0],
                   "parallelism": "single GPU", "kept_chunks_per_step": counts[0], "rotations": len(rot)},
        # the whole fused step against the HBM roofline: chunk embeddings (or
        # index keys) + kept K/V + q, out, lse and ids over the timed step time
        "step_roofline": {"bound": "hbm", "achieved": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
                          "peak": HBM_PEAK_GBS, "unit": "GB/s",
                          "frac": round(step_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                          "algorithmic_bytes_per_step": int(step_bytes), "us_per_step": round(ms_per_step * 1e3, 2),
                          "us_per_step_at_70pct": round(step_bytes / (0.7 * HBM_PEAK_GBS * 1e9) * 1e6, 2)},
        "step_gbs": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
        "step_roofline_frac": round(step_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "parts_us": parts_us,
        "kernels_us_trace": trace_kernels(args.workload),
        "step_us": {"p10": pct(0.10), "median": pct(0.50), "p90": pct(0.90), "samples": n_dist,
                    "flush_mib_between_samples": flush_mib},
        "step_gbs_at_median": round(step_bytes / (pct(0.50) * 1e-6) / 1e9, 1),
        "read_ceiling_gbs": round(read_gbs, 1) if read_gbs else None,
        "step_frac_of_read_ceiling": round(step_bytes / (ms_per_step * 1e-3) / 1e9 / read_gbs, 4) if read_gbs else None,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "kernel": "attention: split kernel + combine (one lsa_sparse_decode_attn call)",
                     "avg_launch_us": round(att_avg_us, 2),
                     "algorithmic_bytes_per_launch": int(attn_bytes),
                     "frac_of_read_ceiling": round(achieved / read_gbs, 4) if read_gbs else None},
    }

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(prob, host0, args.cpu_seconds)

    print(json.dumps(result), flush=True)
    return 0


TIER_TAU = 64        # decode steps between firings of the indexer
TIER_RHO = 0.99      # correlation of the indexer queries of consecutive firings
TIER_K2 = 1024       # tier2l1m: chunks Level 2 keeps out of the resident kept set
TIER_AHEAD = 24      # decode steps the host may enqueue ahead of the GPU


def bench_tier(args) -> int:
    """Decode over the host tier at 1M context (the tier1m and tier2l1m workloads).

    Firings: the indexer queries of firing f are bf16(sqrt(rho) q_{f-1} +
    sqrt(1 - rho) g_f) with fresh N(0, 1) draws g_f and the gates of firing 0,
    so that consecutive kept sets overlap as a slowly moving decode state would
    (about 11% of the set changes per firing at rho = 0.99).  A step is one
    decode step: the attention over the reserve, plus 1/64 of a firing (index
    scores of 3 layers over the full history, recall selection, residency plan
    and the copies of the missing chunks over PCIe) run on a second stream.
    The reported value is the copy kernel's side band with the new set read
    at the next step (the materialisation at t + 1): the copy list never
    leaves the GPU.  For comparison the same loop runs with the new set read 16
    steps later, and with DMA-engine copies issued by the host from a host copy
    of the list, the new set read --tier-lag steps after the firing.  The host
    stays at most TIER_AHEAD steps ahead of the GPU.  Decode steps are
    launched directly: replaying them from a HIP graph measured about 5 us
    slower per step here.
    tier2l1m adds Level 2 to every decode step: lsa_tier_step scores the
    resident kept chunks with the native indexer, keeps TIER_K2 of them and
    attends over their slots."""
    import dataclasses

    import numpy as np
    import torch

    import lsa_synth as synth
    import paper_2606_09079_amd as L

    if not 1 <= args.tier_lag < TIER_TAU:
        raise SystemExit(f"--tier-lag must be in 1 .. {TIER_TAU - 1}")
    if args.warmup % TIER_TAU:
        args.warmup += TIER_TAU - args.warmup % TIER_TAU  # the timed region starts at a firing
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()  # default priority
    level2 = args.workload == "tier2l1m"
    prob = synth.make_problem("recall1m", 0)
    if level2:
        prob = dataclasses.replace(prob, name="tier2l1m", core_keep=[TIER_K2], nat_heads=64)
    t_setup = time.time()
    host0 = synth.host_inputs(prob, 0)
    dev = synth.device_inputs(prob, 0, host=host0)
    host_k = torch.empty(dev["k"].shape, dtype=torch.int16, pin_memory=True)
    host_v = torch.empty(dev["v"].shape, dtype=torch.int16, pin_memory=True)
    host_k.copy_(dev["k"])
    host_v.copy_(dev["v"])
    cache_bytes = 2 * dev["k"].numel() * 2
    del dev["k"], dev["v"]  # from here on the GPU holds the reserve only
    torch.cuda.empty_cache()

    def up(a):
        a = np.ascontiguousarray(a)
        return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).cuda()

    n_fire = 3 * ((args.warmup + args.steps) // TIER_TAU + 1) + 2  # three steady-state runs
    rng = np.random.default_rng(2024)
    qf = synth.bf16_bits_to_f64(host0["idx_q"])
    idx_q = []
    for f in range(n_fire):
        if f > 0:
            qf = math.sqrt(TIER_RHO) * qf + math.sqrt(1.0 - TIER_RHO) * rng.standard_normal(qf.shape)
        idx_q.append(up(synth.f64_to_bf16_bits(qf)))
    # unrelated queries: a full change of the kept set
    fresh_qs = [up(synth.f64_to_bf16_bits(rng.standard_normal(qf.shape))) for _ in range(5)]
    rot = [synth.host_inputs(prob, 1000 + r) for r in range(1, 4)]
    qs = [dev["q"]] + [up(h["q"]) for h in rot]
    nat_qs = [dev["nat_q"]] + [up(h["nat_q"]) for h in rot] if level2 else []
    del rot

    B, K, C, Hkv, d = prob.batch, prob.keep[0], prob.chunk, prob.n_kv_heads, prob.head_dim
    P, ix, T = L.Problem.from_synth(prob), L.Indexer.from_synth(prob), L.Tier([2 * K] * B)
    pitch, total, ws_bytes = L.lsa_tier_sizes(P, T)
    slot_bytes = Hkv * C * d * 2
    res_k = torch.empty(total * slot_bytes // 2, dtype=torch.int16, device="cuda")
    res_v = torch.empty_like(res_k)
    owner = torch.empty(total, dtype=torch.int32, device="cuda")
    L.lsa_tier_reset(P, T, owner)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    scores = torch.empty(prob.idx_layers * prob.total_chunks, dtype=torch.float32, device="cuda")
    kept = [torch.empty(B, pitch, dtype=torch.int32, device="cuda") for _ in range(2)]
    cnt = [torch.zeros(B, dtype=torch.int32, device="cuda") for _ in range(2)]
    slots = [torch.empty(B, pitch, dtype=torch.int32, device="cuda") for _ in range(2)]
    fetch = torch.empty(B, pitch, 2, dtype=torch.int32, device="cuda")
    fcount = torch.zeros(B, dtype=torch.int32, device="cuda")
    out = torch.empty(B, 1, prob.n_q_heads, d, dtype=torch.float32, device="cuda")
    lse = torch.empty(B, 1, prob.n_q_heads, dtype=torch.float32, device="cuda")
    sel = torch.empty(B, pitch, dtype=torch.int32, device="cuda")
    sel_cnt = torch.zeros(B, dtype=torch.int32, device="cuda")
    nat = L.Indexer(1, prob.nat_heads, prob.idx_dim)

    def select_and_plan(q_idx, prev, new, s):
        L.lsa_recall_scores(P, ix, q_idx, dev["idx_w"], dev["idx_k"], scores, s)
        L.lsa_recall_select(P, ix, scores, kept[new], cnt[new], s)
        L.lsa_tier_plan(P, T, kept[new], cnt[new], slots[prev] if prev is not None else None,
                        cnt[prev] if prev is not None else None, owner, slots[new], fetch, fcount, s)

    # the copy kernel beside decode runs on fewer workgroups than the cold fill
    T_side = {w: L.Tier([2 * K] * B, fetch_workgroups=w) for w in (4, 8, 16, 32)}

    def fire(q_idx, prev, new, s, wgs=None):
        select_and_plan(q_idx, prev, new, s)
        L.lsa_tier_fetch(P, T_side[wgs or args.tier_fetch_wgs], host_k, host_v, fetch, fcount, res_k, res_v, s)

    def decode(buf, i, s):
        if level2:
            L.lsa_tier_step(P, T, nat, prob.core_keep, nat_qs[i % len(nat_qs)], dev["nat_w"], dev["nat_k"],
                            kept[buf], cnt[buf], slots[buf], qs[i % len(qs)], res_k, res_v, 0.0, out, lse, sel,
                            sel_cnt, ws, ws_bytes, s)
        else:
            L.lsa_tier_attend(P, T, qs[i % len(qs)], res_k, res_v, slots[buf], cnt[buf], 0.0, out, lse, ws, ws_bytes,
                              s)

    def ev():
        return torch.cuda.Event(enable_timing=True)

    # The host enqueues at most TIER_AHEAD decode steps ahead of the GPU, as a
    # serving loop would: an unbounded lead fills the device queue, and the
    # side band's copies then wait behind launches that cannot be queued.  The
    # wait polls a ring of reused events rather than blocking in the runtime,
    # which the side-band thread's copy calls would otherwise queue behind.
    ring = [torch.cuda.Event() for _ in range(TIER_AHEAD)]
    n_paced = [0]

    def pace():
        e_ = ring[n_paced[0] % TIER_AHEAD]
        if n_paced[0] >= TIER_AHEAD:
            while not e_.query():
                time.sleep(0)
        e_.record(main)
        n_paced[0] += 1

    # ---- cold start: everything kept is copied in
    e = [ev() for _ in range(3)]
    e[0].record(main)
    select_and_plan(idx_q[0], None, 0, main)
    e[1].record(main)
    L.lsa_tier_fetch(P, T, host_k, host_v, fetch, fcount, res_k, res_v, main)
    e[2].record(main)
    torch.cuda.synchronize()
    cold_n = int(fcount.cpu()[0])
    cold_ms = e[1].elapsed_time(e[2])
    log(f"[tier] setup {time.time() - t_setup:.1f}s; cold fetch of {cold_n} chunks in {cold_ms:.2f} ms "
        f"({cold_n * 2 * slot_bytes / (cold_ms * 1e-3) / 1e9:.1f} GB/s); select+plan {e[0].elapsed_time(e[1]):.3f} ms")

    # ---- decode alone (HIP events per launch on the launch stream)
    n_dec = 50
    for i in range(20):
        decode(0, i, main)
    de = [(ev(), ev()) for _ in range(n_dec)]
    for i in range(n_dec):
        de[i][0].record(main)
        decode(0, i, main)
        de[i][1].record(main)
    torch.cuda.synchronize()
    dec_us = 1e3 * sum(a.elapsed_time(b) for a, b in de) / n_dec
    # host cost of enqueueing one decode step (binding, validation, launches):
    # the median over single calls, each into an idle queue, so that one stall
    # of the host process does not stand for the cost of every call
    host_t = []
    for i in range(n_dec):
        torch.cuda.synchronize()
        th = time.perf_counter()
        decode(0, i, main)
        host_t.append(time.perf_counter() - th)
    torch.cuda.synchronize()
    host_us = float(np.median(host_t)) * 1e6

    # the copy list on the host, for the DMA engines
    h_fetch = torch.empty(B, pitch, 2, dtype=torch.int32, pin_memory=True)
    h_fcount = torch.empty(B, dtype=torch.int32, pin_memory=True)


    def fire_dma(q_idx, prev, new, s):
        """Selection, plan and the copy of the list to the host on stream s;
        then the DMA copies from the host copy of the list, also on s."""
        select_and_plan(q_idx, prev, new, s)
        with torch.cuda.stream(s):
            h_fetch.copy_(fetch, non_blocking=True)
            h_fcount.copy_(fcount, non_blocking=True)
        listed = ev()
        listed.record(s)
        t_sub = time.perf_counter()
        # the host waits for the list here, while the GPU works through the
        # decode steps already queued (at most TIER_AHEAD of them)
        listed.synchronize()
        t_list = time.perf_counter()
        L.lsa_tier_fetch_dma(P, T, host_k, host_v, h_fetch, h_fcount, res_k, res_v, s)
        # host ms from the firing: list on the host, copies issued
        return round(1e3 * (t_list - t_sub), 3), round(1e3 * (time.perf_counter() - t_sub), 3)

    # ---- a full change of the kept set, copied on the side stream while decode
    # goes on over the old set, by the copy kernel and by the DMA engines
    full = {}
    for mode, q_full in zip([f"kernel_{w}wg" for w in (4, 8, 16, 32)] + ["dma"], fresh_qs):
        n_during = 700
        dd = [(ev(), ev()) for _ in range(n_during)]
        fe = [ev(), ev()]
        # every event exists in the runtime before the copies start, so that no
        # first use of one inside the loop can hold up the decode launches
        for a_, b_ in dd + [tuple(fe)]:
            a_.record(main)
            b_.record(main)
        torch.cuda.synchronize()
        side.wait_stream(main)
        fe[0].record(side)
        if mode == "dma":
            fire_dma(q_full, 0, 1, side)
        else:
            fire(q_full, 0, 1, side, wgs=int(mode.split("_")[1][:-2]))
        fe[1].record(side)
        for i in range(n_during):
            dd[i][0].record(main)
            decode(0, i, main)
            dd[i][1].record(main)
            pace()
        torch.cuda.synchronize()
        n_full = int(fcount.cpu()[0])
        ms_full = fe[0].elapsed_time(fe[1])
        during = [1e3 * a_.elapsed_time(b_) for a_, b_ in dd
                  if fe[0].elapsed_time(a_) >= 0 and fe[0].elapsed_time(b_) <= ms_full]
        full[mode] = {"copies": n_full, "ms": round(ms_full, 3),
                      "gbs": round(n_full * 2 * slot_bytes / (ms_full * 1e-3) / 1e9, 2),
                      "decode_us_during_copies": round(float(np.median(during)), 2) if during else None,
                      "decode_steps_during_copies": len(during)}
        log(f"[tier] full change by {mode}: {full[mode]}")
        # back to the firing-0 set
        side.wait_stream(main)
        fire(idx_q[0], 1, 0, side)
        main.wait_stream(side)
        torch.cuda.synchronize()

    # ---- steady state: a firing every TIER_TAU steps on the side stream; steps
    # t .. t + lag - 1 read the previous set, steps from t + lag on the new one.
    # The side band waits only for the switch to the previous set (the decodes
    # of the set before it have finished then), never for the latest decode.
    state = {"cur": 0, "f": 1}

    def steady(mode, lag):
        cur, f = state["cur"], state["f"]
        fire_ev, copies, new = [], [], None
        side_host = []
        switched = ev()
        switched.record(main)
        e0, e1 = ev(), ev()
        t0 = 0.0
        for i in range(args.warmup + args.steps):
            if i == args.warmup:
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                e0.record(main)
            if i % TIER_TAU == 0:
                new = 1 - cur
                side.wait_event(switched)
                a_, b_ = ev(), ev()
                a_.record(side)
                h = (fire if mode == "kernel" else fire_dma)(idx_q[f], cur, new, side)
                b_.record(side)
                if h is not None:
                    side_host.append(h)
                fire_ev.append((a_, b_, i >= args.warmup))
                f += 1
            if i % TIER_TAU == lag:
                main.wait_stream(side)
                cur = new
                switched = ev()
                switched.record(main)
                copies.append(fcount.clone())
            decode(cur, i, main)
            pace()
        main.wait_stream(side)
        e1.record(main)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        state["cur"], state["f"] = (new if new is not None else cur), f
        ms = e0.elapsed_time(e1) / args.steps
        fire_ms = [a.elapsed_time(b) for a, b, timed in fire_ev if timed]
        n_copies = [int(c.cpu()[0]) for c in copies]
        log(f"[tier] {mode} copies, lag {lag}: {args.steps} steps, {ms * 1e3:.2f} us/step (wall {wall:.3f}s); "
            f"firings {[round(x, 3) for x in fire_ms]} ms; copies {n_copies}; side-band host ms {side_host[-len(fire_ms):] if fire_ms else side_host}")
        return {"us_per_step": round(ms * 1e3, 2), "lag_steps": lag, "firings_timed": len(fire_ms),
                "firing_ms": round(sum(fire_ms) / len(fire_ms), 3) if fire_ms else None,
                "copies_per_firing": n_copies[-len(fire_ms):] if fire_ms else [],
                "side_band_host_ms": side_host[-len(fire_ms):] if side_host and fire_ms else None}

    runs = {"kernel_lag1": steady("kernel", 1), "kernel_lag16": steady("kernel", 16),
            "dma": steady("dma", args.tier_lag)}
    ms_per_step = runs["kernel_lag1"]["us_per_step"] * 1e-3
    cur = state["cur"]

    kept_n = int(cnt[cur].cpu()[0])
    attn_n, attn_us = kept_n, dec_us
    level2_info = None
    if level2:
        # the dominant kernel alone: attention over the slots Level 2 chose
        decode(cur, 0, main)
        torch.cuda.synchronize()
        attn_n = int(sel_cnt.cpu()[0])

        def attend(i):
            L.lsa_tier_attend(P, T, qs[i % len(qs)], res_k, res_v, sel, sel_cnt, 0.0, out, lse, ws, ws_bytes, main)

        for i in range(20):
            attend(i)
        ae = [(ev(), ev()) for _ in range(n_dec)]
        for i in range(n_dec):
            ae[i][0].record(main)
            attend(i)
            ae[i][1].record(main)
        torch.cuda.synchronize()
        attn_us = 1e3 * sum(a.elapsed_time(b) for a, b in ae) / n_dec
        nat_bytes = kept_n * (prob.idx_dim * 2 + 4 + 4) + B * prob.nat_heads * (prob.idx_dim * 2 + 4)
        level2_info = {"core_keep": TIER_K2, "native_heads": prob.nat_heads, "resident_kept": kept_n,
                       "attended_chunks": attn_n, "native_score_bytes": nat_bytes,
                       "attention_us_alone": round(attn_us, 2), "level2_us": round(dec_us - attn_us, 2)}
    attn_bytes = attn_n * 2 * slot_bytes + B * prob.n_q_heads * d * (2 + 4) + B * prob.n_q_heads * 4 + attn_n * 4
    achieved = attn_bytes / (attn_us * 1e-6) / 1e9
    reserve_bytes = 2 * total * slot_bytes
    result = {
        "metric": METRIC,
        "value": round(1e3 / ms_per_step, 2),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOADS[args.workload], "global_batch": B, "seq_len": prob.ctx_tokens[0],
                   "parallelism": "single GPU", "tau": TIER_TAU, "query_correlation_per_firing": TIER_RHO,
                   "k_max": K, "reserve_slots": total},
        "tier": {
            "cache_bytes": cache_bytes, "reserve_bytes": reserve_bytes,
            "cold_fetch": {"chunks": cold_n, "ms": round(cold_ms, 3),
                           "pcie_gbs": round(cold_n * 2 * slot_bytes / (cold_ms * 1e-3) / 1e9, 2)},
            "decode_us_alone": round(dec_us, 2),
            "host_us_per_decode_enqueue": round(host_us, 2),
            "full_change": full,
            "steady_state": runs,
            "kept_chunks": kept_n,
            "level2": level2_info,
        },
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "attn_kernel (lsa_tier_attend)", "avg_launch_us": round(attn_us, 2),
                     "algorithmic_bytes_per_launch": int(attn_bytes)},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(prob, host0, args.cpu_seconds)
    print(json.dumps(result), flush=True)
    return 0


def bench_kvpack(args) -> int:
    """Tokens per second of the re-layout of a token-major cache into the paged
    blocks (lsa_kv_pack over the whole paper1m context, K and V), and the time
    of the per-step append of one decoded token per sequence."""
    import numpy as np
    import torch

    import lsa_synth as synth
    import paper_2606_09079_amd as L

    main = torch.cuda.current_stream()
    sp = main.cuda_stream
    calibration_copy(args, main)
    prob = synth.make_problem("paper1m", 0)
    P = L.Problem.from_synth(prob)
    T, H, d = prob.ctx_tokens[0], prob.n_kv_heads, prob.head_dim
    t_setup = time.time()
    table = torch.from_numpy(synth.normal_table_bf16().view(np.int16)).cuda()
    tau = torch.from_numpy(synth.token_rows(prob, [0], T)).cuda()
    src = {w: torch.empty(T * H * d, dtype=torch.int16, device="cuda") for w in "kv"}
    for w in "kv":
        synth.fill_kv_tokens_device(prob, 0, w, src[w].data_ptr(), table.data_ptr(), tau.data_ptr(), T,
                                    stream_ptr=sp)
    del tau
    n = prob.kv_elems()
    dst = {w: torch.empty(n, dtype=torch.int16, device="cuda") for w in "kv"}
    offs = torch.zeros(1, dtype=torch.int64, device="cuda")

    def pack():
        L.lsa_kv_pack(P, src["k"], src["v"], offs, dst["k"], dst["v"], stream=main)

    pack()
    for w in "kv":  # the packed cache is the paged fill's, byte for byte
        ref = torch.empty(n, dtype=torch.int16, device="cuda")
        synth.fill_kv_device(prob, 0, w, ref.data_ptr(), table.data_ptr(), sp)
        if not torch.equal(ref, dst[w]):
            raise RuntimeError(f"lsa_kv_pack: packed {w.upper()} differs from the paged fill")
        del ref
    log(f"[kvpack] setup and check {time.time() - t_setup:.1f}s")
    for _ in range(args.warmup):
        pack()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(main)
    for _ in range(args.steps):
        pack()
    e1.record(main)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / args.steps
    call_bytes = 2 * 2 * T * H * d * 2  # K and V, each read once and written once

    def append_us(p_, first, src_rows, offsets, k_cache, v_cache, reps=100):
        # one small launch per call: replayed from a HIP graph of `reps` calls,
        # so that the host's time per call does not count
        def call(st):
            L.lsa_kv_pack(p_, src_rows, src_rows, offsets, k_cache, v_cache, first_token=first, stream=st)
        call(main)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            cs = torch.cuda.current_stream()
            for _ in range(reps):
                call(cs)
        graph.replay()
        torch.cuda.synchronize()
        a_, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a_.record(main)
        for _ in range(5):
            graph.replay()
        b_.record(main)
        torch.cuda.synchronize()
        return round(1e3 * a_.elapsed_time(b_) / (5 * reps), 2)

    # one decoded token: its K/V rows sit in a buffer of the new rows only
    new1 = torch.zeros(H * d, dtype=torch.int16, device="cuda")
    ap1 = append_us(P, [T - 1], new1, torch.tensor([-(T - 1)], dtype=torch.int64, device="cuda"), dst["k"], dst["v"])
    del src
    b32 = synth.make_problem("batch32", 0)
    P32 = L.Problem.from_synth(b32)
    new32 = torch.zeros(b32.batch * H * d, dtype=torch.int16, device="cuda")
    first32 = [Lb - 1 for Lb in b32.ctx_tokens]
    offs32 = torch.tensor([b - f for b, f in enumerate(first32)], dtype=torch.int64, device="cuda")
    del dst
    k32 = torch.empty(b32.kv_elems(), dtype=torch.int16, device="cuda")
    v32 = torch.empty(b32.kv_elems(), dtype=torch.int16, device="cuda")
    ap32 = append_us(P32, first32, new32, offs32, k32, v32)
    achieved = call_bytes / (ms * 1e-3) / 1e9
    log(f"[kvpack] {args.steps} packs: {ms * 1e3:.1f} us each (wall {wall:.3f}s), {achieved:.0f} GB/s; "
        f"append {ap1} us (1 sequence), {ap32} us (32 sequences)")
    result = {
        "metric": "tokens/s re-laid from a token-major cache into the paged blocks (K and V, 8 KV heads)",
        "value": round(T / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 (bit copy)",
        "data": "synthetic",
        "config": {"workload": WORKLOADS[args.workload], "global_batch": 1, "seq_len": T, "parallelism": "single GPU"},
        "append_us": {"paper1m_one_token": ap1, "batch32_one_token_each": ap32},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(PACK_SUMMARY, "kvpack.hip"),
                     "kernel": "kv_pack_kernel (one lsa_kv_pack call over the whole context)",
                     "avg_launch_us": round(ms * 1e3, 2), "algorithmic_bytes_per_launch": int(call_bytes)},
    }
    print(json.dumps(result), flush=True)
    return 0


def bench_golden(args) -> int:
    """Label windows per second of the golden-label pipeline (softmax, top-p
    sets, votes across layers, golden sets, union over the window), one
    lsa_golden_labels call per window on logits resident in HBM."""
    import numpy as np
    import torch

    import lsa_synth as synth
    import paper_2606_09079_amd as L

    main = torch.cuda.current_stream()
    calibration_copy(args, main)
    gp = synth.make_golden_problem(args.workload)
    t_setup = time.time()
    logits = synth.golden_logits_device(gp, 0)
    g = L.Golden.from_synth(gp)
    ws_bytes = L.lsa_golden_sizes(g)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    B, tau, Ly = gp.batch, gp.tau, gp.layers
    labels = torch.empty(sum(gp.n_entries), dtype=torch.int32, device="cuda")
    count = torch.empty(B, dtype=torch.int32, device="cuda")
    sizes = torch.empty(B, tau, Ly, dtype=torch.int32, device="cuda")
    golden = torch.empty(B, tau, dtype=torch.int32, device="cuda")
    log(f"[golden] setup {time.time() - t_setup:.1f}s, logits {logits.numel() * 4 / 1e6:.0f} MB")

    def step():
        L.lsa_golden_labels(g, logits, labels, count, sizes, golden, ws, ws_bytes, main)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(main)
    for _ in range(args.steps):
        step()
    e1.record(main)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = e0.elapsed_time(e1) / args.steps
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(20)]
    for a_, b_ in evs:
        a_.record(main)
        step()
        b_.record(main)
    torch.cuda.synchronize()
    call_us = 1e3 * sum(a_.elapsed_time(b_) for a_, b_ in evs) / len(evs)
    n_lab = count.cpu().numpy().tolist()
    sz = sizes.cpu().numpy()
    words = sum((n + 31) // 32 for n in gp.n_entries)
    # logits read once; row bitmaps written, then read by the vote; label bitmap, labels
    call_bytes = gp.total_logits * 4 + 2 * tau * Ly * words * 4 + 2 * words * 4 + 4 * sum(n_lab)
    achieved = call_bytes / (call_us * 1e-6) / 1e9
    log(f"[golden] {args.steps} windows: {ms_per_step * 1e3:.1f} us each (wall {wall:.3f}s); labels {n_lab}")
    result = {
        "metric": METRIC,
        "value": round(1e3 / ms_per_step, 2),
        "unit": "windows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 logits, f64 weights, integer masses",
        "data": "synthetic",
        "config": {"workload": WORKLOADS[args.workload], "global_batch": B, "entries": gp.n_entries, "tau": tau,
                   "layers": Ly, "top_p": f"{gp.p_num}/{gp.p_den}", "theta": gp.theta, "parallelism": "single GPU"},
        "golden": {"labels": n_lab, "top_p_set_size": {"min": int(sz.min()), "mean": round(float(sz.mean()), 1),
                                                      "max": int(sz.max())},
                   "golden_set_size_mean": round(float(golden.float().mean().cpu()), 1)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "lsa_golden_labels (row, vote, compact kernels)", "avg_launch_us": round(call_us, 2),
                     "algorithmic_bytes_per_launch": int(call_bytes)},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = golden_cpu_baseline(gp, args.cpu_seconds)
    print(json.dumps(result), flush=True)
    return 0


def golden_cpu_baseline(gp, budget_s: float):
    """The oracle on whole decoding steps of sequence 0's window (all layers),
    as many as the time bound allows, scaled to windows per second."""
    import lsa_synth as synth
    import oracle

    steps, el = 0, 0.0
    t0 = time.perf_counter()
    while el < budget_s and steps < gp.tau:
        x = synth.golden_logits(gp, 0, 0, steps=[steps])
        t1 = time.perf_counter()
        oracle.golden_labels(x, gp.p_num, gp.p_den, gp.theta)
        el += time.perf_counter() - t1
        steps += 1
    per_window = el / steps * gp.tau * sum(gp.n_entries) / gp.n_entries[0]
    return {"value": round(1.0 / per_window, 5), "unit": "windows/s", "cores": 1, "kind": "oracle",
            "sample": f"{steps} of the {gp.tau} steps of sequence 0 ({gp.layers} layers x {gp.n_entries[0]:,} "
                      f"entries each) in {el:.1f}s of oracle time (logit generation excluded), scaled to a whole "
                      f"window of all {gp.batch} sequence(s); one thread"}


def cpu_baseline(prob, host, budget_s: float):
    """The CPU oracle, as it stands, on one full step of the same workload
    (score all chunks, top-k, attention for every query head), repeated while
    the time bound allows.  The attention of each KV-head group runs as token
    ranges on parallel threads, one task per (group, range) and as many tasks
    as the process has cores; the ranges' outputs merge through their
    log-sum-exps, out = sum_r exp(lse_r - lse) out_r with lse the logsumexp of
    the lse_r."""
    import numpy as np

    import lsa_synth as synth
    import oracle

    def select():
        if prob.core_keep:
            return oracle.two_level_for_sequence(prob, host, 0)[3]
        if prob.idx_layers > 0:
            return oracle.recall_for_sequence(prob, host, 0)[1]
        return oracle.select_for_sequence(prob, host, 0)[2]

    t_prep = time.time()
    kept = select()
    Hkv, G = prob.n_kv_heads, prob.group
    kv = {(w, g): synth.kv_head_sparse(prob, 0, w, 0, g, kept) for g in range(Hkv) for w in ("k", "v")}
    log(f"[bench] cpu baseline inputs prepared in {time.time() - t_prep:.1f}s")
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    ranges = max(1, -(-cores // Hkv))
    threads = min(cores, Hkv * ranges)

    def one_step():
        kept_s = select()
        toks = oracle.kept_tokens(kept_s, prob.chunk, prob.ctx_tokens[0])
        cuts = [len(toks) * r // ranges for r in range(ranges + 1)]

        def part(task):
            g, r = divmod(task, ranges)
            qr = np.stack([host["q"][0, 0, g * G + j] for j in range(G)])
            return oracle.attention_tokens(qr, kv[("k", g)], kv[("v", g)], toks[cuts[r]:cuts[r + 1]])

        with cf.ThreadPoolExecutor(threads) as ex:
            res = list(ex.map(part, range(Hkv * ranges)))
        for g in range(Hkv):
            outs = np.stack([res[g * ranges + r][0] for r in range(ranges)])
            lses = np.stack([res[g * ranges + r][1] for r in range(ranges)])
            lse = np.logaddexp.reduce(lses, axis=0)
            w = np.exp(lses - lse[None, :])
            w[~np.isfinite(w)] = 0.0
            (w[:, :, None] * outs).sum(axis=0)

    reps, t0 = 0, time.perf_counter()
    while True:
        one_step()
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or el / reps * (reps + 1) > 3 * budget_s:
            break
    # the same step on one thread (KV-head groups in turn), once
    t1 = time.perf_counter()
    kept_1 = select()
    toks_1 = oracle.kept_tokens(kept_1, prob.chunk, prob.ctx_tokens[0])
    for g in range(Hkv):
        qr = np.stack([host["q"][0, 0, g * G + j] for j in range(G)])
        oracle.attention_tokens(qr, kv[("k", g)], kv[("v", g)], toks_1)
    one_thread_s = time.perf_counter() - t1
    full = prob.batch == 1 and prob.n_qtok == 1
    what = ("full step(s) of the same workload" if full else
            "step(s) of sequence 0 of the same workload, attention for its first query token only")
    if prob.core_keep:
        sel_what = (f"{prob.idx_layers}-layer x {prob.idx_heads}-head index scores of {history_chunks(prob, 0):,} "
                    f"history chunks, recall bounded by {prob.keep[0]:,}, native top-{prob.core_keep[0]:,}, "
                    f"window of {prob.n_chunks[0] - history_chunks(prob, 0)} chunks")
    elif prob.idx_layers > 0:
        sel_what = (f"{prob.idx_layers}-layer x {prob.idx_heads}-head index scores of {prob.n_chunks[0]:,} chunks, "
                    f"recall bounded by {prob.keep[0]:,}")
    else:
        sel_what = f"score {prob.n_chunks[0]:,} chunks, top-{prob.keep[0]:,}"
    return {"value": round(reps / el, 4), "unit": "steps/s", "cores": threads, "kind": "oracle",
            "sample": f"{reps} {what} ({sel_what}, fp64 attention for {prob.n_q_heads} query heads) in {el:.1f}s; "
                      f"{Hkv} KV-head groups x {ranges} token ranges on {threads} threads (cores available "
                      f"{cores}, os.cpu_count() = {os.cpu_count()}, OMP_NUM_THREADS = "
                      f"{os.environ.get('OMP_NUM_THREADS', 'unset')}); selection on one thread",
            "one_thread": {"value": round(1.0 / one_thread_s, 4), "unit": "steps/s",
                           "sample": "one more step with the KV-head groups in turn on one thread"}}


if __name__ == "__main__":
    sys.exit(main())
