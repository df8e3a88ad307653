"""GPU parity of pr2_moe_rollout_forward (Eq. pr2_old_output; Alg. 2): the
predicted route is recorded exactly as by pr2_route_predict and the layer
output uses the predictive weights, renormalised (renorm = 1) or the
softmax over all N experts as printed (renorm = 0).

Checks against the float64 oracle: ids and gates under the margin rule,
output rows within 2e-2 (bf16) / 1e-5 (fp32) relative, on tokens outside the
margin; with a zero predictor the rollout output equals the replay output of
the same recorded route (Pr^2 at initialisation is routing replay)."""
import numpy as np
import pytest

from oracle import pr2_oracle as O
import workloads as W
from tests.parity import MARGIN_EPS, compare_route, compare_rows, to_dev

pytestmark = pytest.mark.gpu


def run_rollout(L, s, renorm=True, idx_dtype="int32", ldi_pad=0, logits=False):
    import torch
    from paper_2606_00395_amd import binding as B
    x = to_dev(L["x"], s.act)
    Wr = to_dev(L["W_r"])
    br = to_dev(L["beta"]) if L["beta"] is not None else None
    A = to_dev(L["A"]) if s.r > 0 else None
    Bm = to_dev(L["B"]) if s.r > 0 else None
    Wg, Wu, Wd = (to_dev(L[n], s.act) for n in ("W_gate", "W_up", "W_down"))
    T, k, N = s.T, s.k, s.N
    dt = torch.int16 if idx_dtype == "int16" else torch.int32
    buf = torch.full((T, k + ldi_pad), -3, dtype=dt, device="cuda")
    gate = torch.empty((T, k), device="cuda")
    lg = torch.empty((T, N), device="cuda") if logits else None
    y = torch.empty_like(x)
    B.moe_rollout_forward(x, Wr, br, A, Bm, Wg, Wu, Wd, k, buf[:, :k], y, gate, lg, renorm=renorm)
    torch.cuda.synchronize()
    out = {"idx": buf[:, :k].cpu().numpy(), "gate": gate.cpu().numpy(),
           "y": y.float().cpu().numpy(), "buf": buf.cpu().numpy()}
    if logits:
        out["logits"] = lg.cpu().numpy()
    return out


def check(L, s, g, renorm, where):
    y_ref, ref = O.rollout_forward(L["x"], L["W_r"], L["beta"], L["A"] if s.r else None,
                                   L["B"] if s.r else None, s.k, L["W_gate"], L["W_up"],
                                   L["W_down"], renorm)
    excl = compare_route(g["idx"], g["gate"], ref, s.k, where)
    keep = ref["margin"] >= MARGIN_EPS
    err = compare_rows(g["y"][keep], y_ref[keep], s.act, where)
    print(f"\n{where}: {excl} tokens under the margin, worst row rel err {err:.2e}")
    return ref


def test_rollout_tiny_fp32_both_weightings():
    s = W.WORKLOADS["tiny_fp32_T256"]
    L = W.layer_inputs(s, 0)
    for renorm in (True, False):
        g = run_rollout(L, s, renorm, logits=True)
        ref = check(L, s, g, renorm, f"tiny renorm={renorm}")
        np.testing.assert_allclose(g["logits"], ref["p"], rtol=0, atol=1e-6)


CASES = [
    # (T, d, N, k, m, r, act, skew, idx_dtype, ldi_pad, renorm, logits)
    (1000, 256, 16, 4, 256, 8, "bf16", "hot8", "int32", 0, True, False),
    (777, 512, 64, 6, 128, 5, "bf16", "zipf", "int16", 2, False, True),
    (300, 192, 8, 2, 96, 3, "bf16", "none", "int32", 0, True, True),      # generic GEMMs
    (129, 64, 32, 8, 48, 4, "f32", "hot8", "int32", 0, False, False),
    # more than 32 tiles of 64 tokens: the route kernel forms the permutation's
    # counts (folded and unfolded predictor), ragged last tile
    (4100, 256, 64, 16, 128, 8, "bf16", "zipf", "int16", 3, True, False),
    (2177, 128, 128, 32, 128, 4, "bf16", "hot8", "int32", 0, False, True),
]


@pytest.mark.parametrize("case", CASES, ids=[f"T{c[0]}_d{c[1]}_N{c[2]}_k{c[3]}_m{c[4]}_r{c[5]}"
                                              f"_{c[6]}_renorm{int(c[10])}" for c in CASES])
def test_rollout_shapes(case):
    T, d, N, k, m, r, act, skew, idt, pad, renorm, logits = case
    s = W.LayerShape("case", T=T, d=d, N=N, k=k, m=m, r=r, act=act, skew=skew)
    L = W.layer_inputs(s, 4)
    g = run_rollout(L, s, renorm, idt, pad, logits)
    check(L, s, g, renorm, str(case))
    if pad:
        assert np.all(g["buf"][:, k:] == -3), "padding beyond k was written"


def test_rollout_zero_predictor_equals_replay_of_its_route():
    import torch
    from paper_2606_00395_amd import binding as B
    s = W.LayerShape("zp", T=2000, d=256, N=32, k=4, m=256, r=6, act="bf16", skew="hot8")
    L = W.layer_inputs(s, 6)
    L["A"] = np.zeros_like(L["A"])
    g = run_rollout(L, s)
    x = to_dev(L["x"], "bf16")
    idx = torch.from_numpy(g["idx"]).to("cuda")
    y = torch.empty_like(x)
    B.moe_replay_forward(x, idx, to_dev(L["W_r"]), to_dev(L["beta"]),
                         *(to_dev(L[n], "bf16") for n in ("W_gate", "W_up", "W_down")), y)
    torch.cuda.synchronize()
    compare_rows(g["y"], y.float().cpu().numpy().astype(np.float64), "bf16", "rollout vs replay")
    # the recorded route is the current router's top-k (the predictor is zero)
    ref = O.route_predict(L["x"], L["W_r"], L["beta"], None, None, s.k)
    compare_route(g["idx"], g["gate"], ref, s.k, "zero predictor")


def test_rollout_qwen3_30b_full():
    """Every token of the Qwen3-30B-A3B-shaped rollout forward: the predicted
    route (margin rule), its predictive weights and the layer output (per-row
    rule, tokens outside the margin)."""
    s = W.WORKLOADS["qwen3_30b_T16384"]
    L = W.layer_inputs(s, 0)
    g = run_rollout(L, s)
    y_ref, ref = O.rollout_forward(L["x"], L["W_r"], L["beta"], L["A"], L["B"], s.k,
                                   L["W_gate"], L["W_up"], L["W_down"])
    n_excl = compare_route(g["idx"], g["gate"], ref, s.k, s.name)
    keep = ref["margin"] >= MARGIN_EPS
    err = compare_rows(g["y"][keep], y_ref[keep], "bf16", s.name)
    print(f"\n{s.name}: rollout forward worst row rel err {err:.2e} over {keep.sum()} rows "
          f"({n_excl} under the margin)")
