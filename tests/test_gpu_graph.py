"""The fused decode step replayed from a HIP graph, as a serving loop runs it.

One capture of lsa_decode_step (with a caller workspace, and as
lsa_decode_step_noalloc on the library's scratch); then, for several seeds, new query embeddings
and queries are copied into the captured input buffers and the graph is
replayed twice, with eager work and a synchronisation between the replays.
Every replay must equal, bit for bit, the eager call on the same inputs
(outputs, lse, kept ids and counts).  The step launches only kernels (no
memory fills), so nothing in it depends on being recorded once: the arrival
counters of the split kernel's own merge are zeroed by the scoring kernel of
the same replay.
"""
import pytest

import lsa_synth as synth
from gpu_case import log

pytestmark = pytest.mark.gpu

CASES = [
    # ragged bf16 batch, 2 query tokens (split kernel, more than 16 splits per head)
    synth.Problem("graph_ragged", [64 * 300, 64 * 77, 64 * 1030], 64, [40, 77, 100], 16, 4, n_qtok=2),
    # 4 lookahead queries (per-query top-k and union), 16 rows per KV head
    synth.Problem("graph_lookahead", [128 * 200, 128 * 90], 128, [12, 9], 16, 4, n_lookahead=4, n_qtok=4),
    # int8 embeddings, 32 rows per KV head (many-rows kernel)
    synth.Problem("graph_int8_rows", [64 * 256, 64 * 128], 64, [32, 16], 32, 4, emb_dtype="i8", n_qtok=4),
    # four sequences, at most 16 splits each: the split kernel's last workgroups merge the splits
    # on arrival counters that the scoring kernel zeroes in every replay
    synth.Problem("graph_split_merge", [64 * 300, 64 * 200, 64 * 250, 64 * 100], 64, [30, 20, 25, 10], 32, 8),
]


@pytest.mark.parametrize("noalloc", [False, True], ids=["workspace", "noalloc"])
@pytest.mark.parametrize("prob", CASES, ids=[p.name for p in CASES])
def test_fused_step_graph_replays_equal_eager(prob, noalloc):
    import torch
    import paper_2606_09079_amd as L
    P = L.Problem.from_synth(prob)
    dev = synth.device_inputs(prob, 0)
    B, Tq, Hq = prob.batch, prob.n_qtok, prob.n_q_heads
    wsb = L.lsa_workspace_size(P)
    max_sel = L.lsa_max_sel(P)

    def buffers():
        return (torch.empty(B, Tq, Hq, 128, dtype=torch.float32, device="cuda"),
                torch.empty(B, Tq, Hq, dtype=torch.float32, device="cuda"),
                torch.empty(B, max_sel, dtype=torch.int32, device="cuda"),
                torch.empty(B, dtype=torch.int32, device="cuda"),
                torch.zeros(max(wsb, 256), dtype=torch.uint8, device="cuda"))

    qe_g, q_g = dev["qe"].clone(), dev["q"].clone()
    out_g, lse_g, sel_g, cnt_g, ws_g = buffers()

    def step(qe, q, out, lse, sel, cnt, ws):
        if noalloc:  # the step on the library's own scratch (its address is looked up by the first, eager call)
            L.lsa_decode_step_noalloc(P, qe, dev["E"], q, dev["k"], dev["v"], 0.0, out, lse, sel, cnt)
        else:
            L.lsa_decode_step(P, qe, dev["E"], q, dev["k"], dev["v"], 0.0, out, lse, sel, cnt, ws, wsb)

    # warm up on a side stream, then capture
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step(qe_g, q_g, out_g, lse_g, sel_g, cnt_g, ws_g)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(qe_g, q_g, out_g, lse_g, sel_g, cnt_g, ws_g)
    torch.cuda.synchronize()

    out_e, lse_e, sel_e, cnt_e, ws_e = buffers()
    for seed in (1, 2, 3):
        new = synth.device_inputs(prob, seed)
        qe_g.copy_(new["qe"])
        q_g.copy_(new["q"])
        torch.cuda.synchronize()
        step(qe_g, q_g, out_e, lse_e, sel_e, cnt_e, ws_e)  # eager, same inputs
        torch.cuda.synchronize()
        for rep in range(2):
            out_g.fill_(float("nan"))
            sel_g.fill_(-7)
            graph.replay()
            torch.cuda.synchronize()
            for name, a, b in (("out", out_g, out_e), ("lse", lse_g, lse_e), ("sel_count", cnt_g, cnt_e)):
                assert torch.equal(a, b), f"{prob.name} seed {seed} replay {rep}: {name} differs from the eager step"
            for bb in range(B):
                n = int(cnt_e[bb])
                assert torch.equal(sel_g[bb, :n], sel_e[bb, :n]), f"{prob.name} seed {seed} replay {rep}: kept ids"
        del new
    log(f"[graph] {prob.name} ({'noalloc' if noalloc else 'workspace'}): 3 input sets x 2 replays equal the eager step")


RECALL = synth.Problem("graph_recall", [64 * 300, 64 * 120], 64, [40, 30], 16, 4, n_qtok=2, idx_layers=2,
                       idx_heads=32, idx_dim=128, idx_rate=0.08)
TWO_LEVEL = synth.Problem("graph_two_level", [64 * 200 + 17, 64 * 90], 64, [30, 20], 32, 8, n_qtok=4, idx_layers=2,
                          idx_heads=16, idx_dim=64, idx_rate=0.1, core_keep=[12, 9], nat_heads=32,
                          window_tokens=[300, 100])


def _replays_equal_eager(name, step, inputs, fresh, outs_g, outs_e):
    """Capture step(bufs) once with the captured inputs, then for each fresh
    input set replay twice and compare the outputs with an eager call: out,
    lse and the counts bit for bit, and the written kept ids of each row."""
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step(inputs, outs_g)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(inputs, outs_g)
    torch.cuda.synchronize()
    for k, new in enumerate(fresh):
        for key, t in new.items():
            inputs[key].copy_(t)
        torch.cuda.synchronize()
        step(inputs, outs_e)
        torch.cuda.synchronize()
        for rep in range(2):
            for t in outs_g.values():
                t.fill_(-7 if t.dtype == torch.int32 else float("nan"))
            graph.replay()
            torch.cuda.synchronize()
            for key in ("out", "lse", "cnt"):
                assert torch.equal(outs_g[key], outs_e[key]), f"{name} input set {k} replay {rep}: {key} differs"
            # the kept ids: the first cnt[b] entries of each row are written
            for b in range(outs_e["cnt"].numel()):
                c = int(outs_e["cnt"][b])
                assert torch.equal(outs_g["sel"][b, :c], outs_e["sel"][b, :c]), \
                    f"{name} input set {k} replay {rep}: kept ids of sequence {b} differ"
    log(f"[graph] {name}: {len(fresh)} input sets x 2 replays equal the eager step")


def test_recall_step_graph_replays_equal_eager():
    import torch
    import paper_2606_09079_amd as L
    prob = RECALL
    P, ix = L.Problem.from_synth(prob), L.Indexer.from_synth(prob)
    dev = synth.device_inputs(prob, 0)
    B, Tq, Hq = prob.batch, prob.n_qtok, prob.n_q_heads
    wsb, max_sel = L.lsa_workspace_size(P), L.lsa_max_sel(P)
    ws = {"g": torch.zeros(max(wsb, 256), dtype=torch.uint8, device="cuda"),
          "e": torch.zeros(max(wsb, 256), dtype=torch.uint8, device="cuda")}

    def outs():
        return {"out": torch.empty(B, Tq, Hq, 128, dtype=torch.float32, device="cuda"),
                "lse": torch.empty(B, Tq, Hq, dtype=torch.float32, device="cuda"),
                "sel": torch.full((B, max_sel), -1, dtype=torch.int32, device="cuda"),
                "cnt": torch.empty(B, dtype=torch.int32, device="cuda")}

    og, oe = outs(), outs()
    inputs = {"idx_q": dev["idx_q"].clone(), "q": dev["q"].clone()}

    def step(i, o):
        w = ws["g"] if o is og else ws["e"]
        L.lsa_recall_step(P, ix, i["idx_q"], dev["idx_w"], dev["idx_k"], i["q"], dev["k"], dev["v"], 0.0, o["out"],
                          o["lse"], o["sel"], o["cnt"], w, wsb)

    fresh = []
    for seed in (1, 2, 3):
        d = synth.device_inputs(prob, seed)
        fresh.append({"idx_q": d["idx_q"], "q": d["q"]})
    _replays_equal_eager("recall", step, inputs, fresh, og, oe)


def test_two_level_step_graph_replays_equal_eager():
    import torch
    import paper_2606_09079_amd as L
    prob = TWO_LEVEL
    P, ix, tl = L.Problem.from_synth(prob), L.Indexer.from_synth(prob), L.TwoLevel.from_synth(prob)
    dev = synth.device_inputs(prob, 0)
    B, Tq, Hq = prob.batch, prob.n_qtok, prob.n_q_heads
    max_sel, wsb = L.lsa_two_level_sizes(P, tl)
    ws = {"g": torch.zeros(max(wsb, 256), dtype=torch.uint8, device="cuda"),
          "e": torch.zeros(max(wsb, 256), dtype=torch.uint8, device="cuda")}

    def outs():
        return {"out": torch.empty(B, Tq, Hq, 128, dtype=torch.float32, device="cuda"),
                "lse": torch.empty(B, Tq, Hq, dtype=torch.float32, device="cuda"),
                "sel": torch.full((B, max_sel), -1, dtype=torch.int32, device="cuda"),
                "cnt": torch.empty(B, dtype=torch.int32, device="cuda")}

    og, oe = outs(), outs()
    inputs = {"idx_q": dev["idx_q"].clone(), "nat_q": dev["nat_q"].clone(), "q": dev["q"].clone()}

    def step(i, o):
        w = ws["g"] if o is og else ws["e"]
        L.lsa_two_level_step(P, ix, tl, i["idx_q"], dev["idx_w"], dev["idx_k"], i["nat_q"], dev["nat_w"], dev["nat_k"],
                             i["q"], dev["k"], dev["v"], 0.0, o["out"], o["lse"], o["sel"], o["cnt"], w, wsb)

    fresh = []
    for seed in (1, 2, 3):
        d = synth.device_inputs(prob, seed)
        fresh.append({"idx_q": d["idx_q"], "nat_q": d["nat_q"], "q": d["q"]})
    _replays_equal_eager("two-level", step, inputs, fresh, og, oe)
