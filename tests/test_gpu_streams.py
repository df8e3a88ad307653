"""Calls on several streams and from several host threads: the library owns no
stream and keeps no per-call device state outside the caller's workspace, so

* calls made at the same time from two host threads, each on its own stream
  and workspace, give bitwise the outputs of the same calls made one after
  the other;
* a replay backward captured into a HIP graph gives, on every replay, bitwise
  the gradients of the eager call, and so does the training pass that saves
  the pre-activations in its forward."""
import threading

import pytest

import workloads as W
from tests.parity import to_dev

pytestmark = pytest.mark.gpu

SHAPE = W.LayerShape("streams", T=3000, d=512, N=32, k=4, m=256, r=8, act="bf16", skew="hot8")


class Problem:
    """One layer's inputs, outputs and workspaces on the device."""

    def __init__(self, seed):
        import torch
        from paper_2606_00395_amd import binding as B
        s = SHAPE
        L = W.layer_inputs(s, seed)
        self.x = to_dev(L["x"], "bf16")
        self.Wr, self.br, self.A, self.Bm = (to_dev(L[n]) for n in ("W_r", "beta", "A", "B"))
        self.Wg, self.Wu, self.Wd = (to_dev(L[n], "bf16") for n in ("W_gate", "W_up", "W_down"))
        self.dy = to_dev(W.upstream_grad(s, seed), "bf16")
        self.idx = torch.empty((s.T, s.k), dtype=torch.int32, device="cuda")
        B.route_predict(self.x, self.Wr, self.br, self.A, self.Bm, s.k, self.idx)
        self.y = torch.empty_like(self.x)
        self.gate = torch.empty((s.T, s.k), device="cuda")
        self.grads = [torch.empty_like(self.x), torch.empty_like(self.Wr), torch.empty_like(self.br),
                      torch.empty(self.Wg.shape, device="cuda"), torch.empty(self.Wu.shape, device="cuda"),
                      torch.empty(self.Wd.shape, device="cuda")]
        self.ws_f = B.replay_workspace(self.x, self.idx, self.Wr, self.Wg)
        self.ws_b = B.backward_workspace(self.x, self.idx, self.Wr, self.Wg)
        torch.cuda.synchronize()

    def forward(self, st):
        from paper_2606_00395_amd import binding as B
        B.moe_replay_forward(self.x, self.idx, self.Wr, self.br, self.Wg, self.Wu, self.Wd, self.y,
                             self.gate, ws=self.ws_f, stream=st)

    def backward(self, st):
        from paper_2606_00395_amd import binding as B
        B.moe_replay_backward(self.x, self.idx, self.Wr, self.br, self.Wg, self.Wu, self.Wd,
                              self.dy, *self.grads, ws=self.ws_b, stream=st)

    def outputs(self):
        return [t.clone() for t in [self.y, self.gate] + self.grads]


def same(a, b):
    import torch
    return all(torch.equal(u, v) for u, v in zip(a, b))


def test_concurrent_calls_from_two_threads_match_serial_calls():
    import torch
    probs = [Problem(21), Problem(22)]
    st = torch.cuda.current_stream()
    ref = []
    for p in probs:
        p.forward(st)
        p.backward(st)
        torch.cuda.synchronize()
        ref.append(p.outputs())
    errors = []
    streams = [torch.cuda.Stream() for _ in probs]

    def run(i):
        try:
            p, s = probs[i], streams[i]
            for it in range(6):
                p.forward(s)
                p.backward(s)
                s.synchronize()
                if not same(p.outputs(), ref[i]):
                    errors.append(f"thread {i} iteration {it}: outputs differ")
        except Exception as e:  # reported below
            errors.append(f"thread {i}: {e!r}")

    threads = [threading.Thread(target=run, args=(i,)) for i in range(len(probs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors


def test_backward_graph_replays_match_eager_call():
    import torch
    p = Problem(23)
    st = torch.cuda.current_stream()
    p.backward(st)
    torch.cuda.synchronize()
    eager = p.outputs()[2:]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        p.backward(torch.cuda.current_stream())
    for rep in range(3):
        for g in p.grads:
            g.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert same(p.outputs()[2:], eager), f"replay {rep}"
        p.forward(st)             # eager work between replays
        torch.cuda.synchronize()


def test_training_pass_with_saved_preactivations_graph_replays_match_eager():
    """pr2_moe_replay_forward_save then pr2_moe_replay_backward_saved, captured
    into one HIP graph: every replay gives bitwise the eager outputs and
    gradients (with other eager work between the replays)."""
    import torch
    from paper_2606_00395_amd import binding as B
    p = Problem(24)
    s = SHAPE
    au = torch.empty((s.T * s.k, 2 * s.m), dtype=torch.bfloat16, device="cuda")

    def step(st):
        B.moe_replay_forward_save(p.x, p.idx, p.Wr, p.br, p.Wg, p.Wu, p.Wd, p.y, au, p.gate,
                                  ws=p.ws_f, stream=st)
        B.moe_replay_backward_saved(p.x, p.idx, p.Wr, p.br, p.Wg, p.Wu, p.Wd, au, p.dy, *p.grads,
                                    ws=p.ws_b, stream=st)

    st = torch.cuda.current_stream()
    step(st)
    torch.cuda.synchronize()
    eager = p.outputs()
    # the recomputing calls give the same outputs and gradients
    p.forward(st)
    p.backward(st)
    torch.cuda.synchronize()
    assert same(p.outputs(), eager), "saved and recomputing passes differ"
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(torch.cuda.current_stream())
    for rep in range(3):
        for t in [p.y, p.gate] + p.grads:
            t.fill_(float("nan"))
        au.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert same(p.outputs(), eager), f"replay {rep}"
        p.forward(st)             # eager work between replays
        torch.cuda.synchronize()
