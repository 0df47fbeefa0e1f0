"""The fused decode step replayed from a HIP graph, as a serving loop runs it.

One capture of lsa_decode_step (with a caller workspace, and as
lsa_decode_step_noalloc on the library's scratch); then, for several seeds, new query embeddings
and queries are copied into the captured input buffers and the graph is
replayed twice, with eager work and a synchronisation between the replays.
Every replay must equal, bit for bit, the eager call on the same inputs
(outputs, lse, kept ids and counts).  The step launches only kernels (no
memory fills), so nothing in it depends on being recorded once.
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
