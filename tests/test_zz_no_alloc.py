"""pr2_route_predict_noalloc against pr2_route_predict: the same route through
the C ABI with the library's own device scratch in place of a caller
workspace.  Two calls in a row on each shape, the second with a smaller batch
(the scratch keeps the first call's contents); ids bit-exact, weights within
1e-5 relative, router logits equal.  Also captured into a HIP graph and
replayed several times, each replay checked against the eager call."""
import numpy as np
import pytest

import workloads as W
from tests.parity import GATE_RTOL, to_dev

pytestmark = pytest.mark.gpu


def inputs(shape, seed, T):
    L = W.layer_inputs(shape.with_(T=T), seed, experts=False)
    return (to_dev(L["x"], shape.act), to_dev(L["W_r"]),
            to_dev(L["beta"]) if L["beta"] is not None else None, to_dev(L["A"]), to_dev(L["B"]))


def both(x, Wr, br, A, Bm, k, logits):
    import torch
    from paper_2606_00395_amd import binding as B
    T, N = x.shape[0], Wr.shape[1]
    out = []
    for fn in (B.route_predict, B.route_predict_noalloc):
        idx = torch.full((T, k), -1, dtype=torch.int32, device="cuda")
        gate = torch.full((T, k), float("nan"), device="cuda")
        lg = torch.full((T, N), float("nan"), device="cuda") if logits else None
        fn(x, Wr, br, A, Bm, k, idx, gate, lg)
        out.append((idx, gate, lg))
    torch.cuda.synchronize()
    return out


def check(ref, got, where):
    import torch
    (i0, g0, l0), (i1, g1, l1) = ref, got
    assert torch.equal(i0, i1), f"{where}: ids differ"
    rel = ((g1.double() - g0.double()).abs() / g0.double().abs()).max().item()
    assert rel <= GATE_RTOL, f"{where}: gate rel err {rel:.3e}"
    if l0 is not None:
        assert torch.equal(l0, l1), f"{where}: logits differ"


SHAPES = [
    # (layer shape, first T, second T, logits wanted)
    (W.WORKLOADS["qwen3_30b_T16384"], 4096, 1000, False),      # folded predictor, MFMA router
    (W.WORKLOADS["qwen3_30b_T16384"], 2048, 256, True),        # [W_r | A] split, logits out
    (W.WORKLOADS["qwen3_235b_T32768"], 3000, 64, False),       # d 4096: 3 MiB of split
    (W.WORKLOADS["tiny_fp32_T256"], 256, 100, True),           # fp64 vector path: no scratch
]


@pytest.mark.parametrize("case", SHAPES, ids=["30b_folded", "30b_logits", "235b_folded", "tiny_fp32"])
def test_noalloc_matches_route_predict_twice(case):
    shape, T1, T2, logits = case
    for i, T in enumerate((T1, T2)):
        x, Wr, br, A, Bm = inputs(shape, 20 + i, T)
        ref, got = both(x, Wr, br, A, Bm, shape.k, logits)
        check(ref, got, f"{shape.name} T={T}")


def test_noalloc_in_a_graph_replays():
    import torch
    from paper_2606_00395_amd import binding as B
    s = W.WORKLOADS["qwen3_30b_T16384"]
    x, Wr, br, A, Bm = inputs(s, 31, 512)
    k = s.k
    ref = both(x, Wr, br, A, Bm, k, False)[0]
    idx = torch.full((512, k), -1, dtype=torch.int32, device="cuda")
    gate = torch.empty((512, k), device="cuda")
    B.route_predict_noalloc(x, Wr, br, A, Bm, k, idx, gate)     # first call on the device: eager
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        B.route_predict_noalloc(x, Wr, br, A, Bm, k, idx, gate)
    other_x = inputs(s, 32, 512)[0]
    for rep in range(4):
        idx.fill_(-1)
        gate.fill_(float("nan"))
        # eager work on the same scratch between replays
        junk = torch.empty_like(idx)
        B.route_predict_noalloc(other_x, Wr, br, A, Bm, k, junk)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        check(ref, (idx, gate, None), f"graph replay {rep}")
