"""The route + replay-forward step captured into a HIP graph (as bench.py times
it) gives, on every replay, bitwise the outputs of the same calls launched
eagerly: no call on the path records a memset or other state that a replay
would not reproduce.  The replays are interleaved with eager work and
synchronisations, and each replay is checked."""
import pytest

import workloads as W
from tests.parity import to_dev

pytestmark = pytest.mark.gpu


def test_graph_replays_match_eager_step():
    import torch
    from paper_2606_00395_amd import binding as B
    s = W.LayerShape("graph", T=3000, d=512, N=32, k=4, m=256, r=8, act="bf16", skew="hot8")
    L = W.layer_inputs(s, 12)
    x = to_dev(L["x"], "bf16")
    Wr, br, A, Bm = (to_dev(L[n]) for n in ("W_r", "beta", "A", "B"))
    Wg, Wu, Wd = (to_dev(L[n], "bf16") for n in ("W_gate", "W_up", "W_down"))
    idx = torch.empty((s.T, s.k), dtype=torch.int32, device="cuda")
    g1 = torch.empty((s.T, s.k), device="cuda")
    g2 = torch.empty((s.T, s.k), device="cuda")
    y = torch.empty_like(x)
    ws = B.replay_workspace(x, idx, Wr, Wg)
    ws_r = B.route_workspace(x, Wr, A, s.k)

    def step(st):
        B.route_predict(x, Wr, br, A, Bm, s.k, idx, g1, ws=ws_r, stream=st)
        B.moe_replay_forward(x, idx, Wr, br, Wg, Wu, Wd, y, g2, ws=ws, stream=st)

    step(torch.cuda.current_stream())
    torch.cuda.synchronize()
    eager = [t.clone() for t in (idx, g1, g2, y)]

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(torch.cuda.current_stream())
    for rep in range(3):
        for t in (idx, g1, g2, y):
            t.fill_(-7 if t.dtype == torch.int32 else float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, a, b in zip(("idx", "gate_route", "gate_replay", "y"), (idx, g1, g2, y), eager):
            assert torch.equal(a, b), f"replay {rep}: {name} differs from the eager step"
        # eager work between replays: a different input through the same workspaces
        x2 = torch.roll(x, 1, dims=0)
        B.moe_replay_forward(x2, idx, Wr, br, Wg, Wu, Wd, torch.empty_like(x), ws=ws)
        torch.cuda.synchronize()
