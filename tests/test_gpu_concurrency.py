"""Two decode steps in flight at once, from two host threads on two streams,
each with its own workspace and outputs: the library keeps no state between
calls other than a per-thread error message, so each result must equal, bit
for bit, the same step run alone."""
import threading

import pytest

import lsa_synth as synth
from gpu_case import log

pytestmark = pytest.mark.gpu

A = synth.Problem("conc_a", [64 * 900, 64 * 300], 64, [90, 30], 32, 8)                    # split kernel + combine
# split kernel with at most 16 splits per (b, g): its last workgroups merge them on arrival counters
M = synth.Problem("conc_m", [64 * 300, 64 * 200, 64 * 250, 64 * 100], 64, [30, 20, 25, 10], 32, 8)
B = synth.Problem("conc_b", [128 * 200, 128 * 80], 128, [12, 9], 64, 8, n_lookahead=4, n_qtok=16)  # union + many rows


class Case:
    def __init__(self, prob, seed):
        import paper_2606_09079_amd as L
        self.prob, self.L = prob, L
        self.P = L.Problem.from_synth(prob)
        self.dev = synth.device_inputs(prob, seed)
        self.wsb = L.lsa_workspace_size(self.P)
        self.max_sel = L.lsa_max_sel(self.P)

    def buffers(self):
        import torch
        p = self.prob
        return {"out": torch.full((p.batch, p.n_qtok, p.n_q_heads, 128), float("nan"), device="cuda"),
                "lse": torch.full((p.batch, p.n_qtok, p.n_q_heads), float("nan"), device="cuda"),
                "sel": torch.full((p.batch, self.max_sel), -1, dtype=torch.int32, device="cuda"),
                "cnt": torch.full((p.batch,), -1, dtype=torch.int32, device="cuda"),
                "ws": torch.zeros(max(self.wsb, 256), dtype=torch.uint8, device="cuda")}

    def step(self, o, stream, reps=1):
        d = self.dev
        for _ in range(reps):
            self.L.lsa_decode_step(self.P, d["qe"], d["E"], d["q"], d["k"], d["v"], 0.0, o["out"], o["lse"], o["sel"],
                                   o["cnt"], o["ws"], self.wsb, stream)


@pytest.mark.parametrize("first", [A, M], ids=["split_combine", "split_merge"])
def test_two_threads_two_streams_equal_each_step_alone(first):
    import torch
    a, b = Case(first, 4), Case(B, 5)
    ref = {}
    for name, c in (("a", a), ("b", b)):
        o = c.buffers()
        c.step(o, torch.cuda.current_stream())
        torch.cuda.synchronize()
        ref[name] = o
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    oa, ob = a.buffers(), b.buffers()
    errors = []

    def run(c, o, s):
        try:
            c.step(o, s, reps=20)  # many launches, interleaved with the other thread's
        except Exception as e:  # surfaced below
            errors.append(e)

    torch.cuda.synchronize()
    threads = [threading.Thread(target=run, args=(a, oa, sa)), threading.Thread(target=run, args=(b, ob, sb))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for name, o in (("a", oa), ("b", ob)):
        r = ref[name]
        for key in ("out", "lse", "cnt"):
            assert torch.equal(o[key], r[key]), f"step {name}: {key} differs from the step run alone"
        for bb in range(r["cnt"].numel()):
            n = int(r["cnt"][bb])
            assert torch.equal(o["sel"][bb, :n], r["sel"][bb, :n]), f"step {name}: kept ids of sequence {bb} differ"
    log(f"[concurrency] {first.name} and {B.name} on two threads and streams: both equal the steps run alone")
