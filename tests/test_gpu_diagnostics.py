"""GPU parity of pr2_route_diagnostics (Sec. 5.4: top-k agreement, routing
deviation distribution and route KL of the recorded route against the
current router) with the float64 oracle.

The recorded route is the oracle's predictive route (router + rank-r
predictor), so it differs from the current router's top-k on some tokens; the
reference logits for the route KL are the oracle's predictive logits z.  The
same checks run on the diagnostics that pr2_moe_replay_forward_diag forms
inside the replay forward, whose output and weights must equal those of
pr2_moe_replay_forward bit for bit.  The current
top-k follows the margin rule on the current logits; overlaps, the deviation
histogram (exact integer counts) and the per-token KL (fp64 from the fp32
logits) are compared on every token outside it."""
import numpy as np
import pytest

from oracle import pr2_oracle as O
import workloads as W
from tests.parity import MARGIN_EPS, to_dev

pytestmark = pytest.mark.gpu


def run(L, s, idx_np, z_ref, idx_dtype="int32", ldi_pad=0):
    import torch
    from paper_2606_00395_amd import binding as B
    x = to_dev(L["x"], s.act)
    Wr = to_dev(L["W_r"])
    br = to_dev(L["beta"]) if L["beta"] is not None else None
    T, k = idx_np.shape
    dt = torch.int16 if idx_dtype == "int16" else torch.int32
    buf = torch.full((T, k + ldi_pad), -1, dtype=dt, device="cuda")
    buf[:, :k] = torch.from_numpy(idx_np.astype(np.int64)).to(dt).to("cuda")
    cur = torch.full((T, k), -5, dtype=dt, device="cuda")
    ov = torch.full((T,), -5, dtype=torch.int32, device="cuda")
    kl = torch.full((T,), float("nan"), device="cuda")
    hist = torch.full((k + 1,), 12345, dtype=torch.int64, device="cuda")
    B.route_diagnostics(x, buf[:, :k], Wr, br, to_dev(z_ref), cur, ov, kl, hist)
    torch.cuda.synchronize()
    return {"cur": cur.cpu().numpy().astype(np.int64), "overlap": ov.cpu().numpy(),
            "kl": kl.cpu().numpy(), "hist": hist.cpu().numpy()}


def oracle_route(L, s):
    """The recorded ids: the oracle's predictive route (never the HIP path's)."""
    return O.route_predict(L["x"], L["W_r"], L["beta"], L["A"], L["B"], s.k)["idx"]


def check(L, s, idx, g, z_ref, where):
    p = O.router_logits(L["x"], L["W_r"], L["beta"])
    cur = O.topk_ids(p, s.k)
    ok = O.topk_margin(p, s.k) >= MARGIN_EPS
    bad = np.nonzero(ok & np.any(g["cur"] != cur, axis=1))[0]
    assert len(bad) == 0, f"{where}: current top-k differs on tokens {bad[:5]}"
    ov = O.route_overlap(idx, cur)
    np.testing.assert_array_equal(g["overlap"][ok], ov[ok])
    hist = O.route_deviation_histogram(idx, cur)
    n_excl = int((~ok).sum())
    assert np.abs(g["hist"] - hist).sum() <= 2 * n_excl, (g["hist"], hist)
    if n_excl == 0:
        np.testing.assert_array_equal(g["hist"], hist)
    assert g["hist"].sum() == s.T
    kl = O.route_kl(p, z_ref)
    np.testing.assert_allclose(g["kl"], kl, rtol=1e-4, atol=1e-7)
    print(f"\n{where}: agreement {g['overlap'].mean() / s.k:.4f}, hist {g['hist'].tolist()}, "
          f"mean KL {g['kl'].mean():.3e}, {n_excl} tokens under the margin")


def predictive_logits(L):
    return (O.router_logits(L["x"], L["W_r"], L["beta"])
            + O.predictor_bias(L["x"], L["A"], L["B"])).astype(np.float32)


def test_diagnostics_tiny_fp32():
    s = W.WORKLOADS["tiny_fp32_T256"]
    L = W.layer_inputs(s, 0, experts=False)
    idx = oracle_route(L, s)
    z = predictive_logits(L)
    check(L, s, idx, run(L, s, idx, z), z, "tiny")


@pytest.mark.parametrize("case", [
    (3000, 256, 64, 6, 8, "bf16", "hot8", "int32", 0),
    (1000, 512, 128, 8, 16, "bf16", "zipf", "int16", 2),
    (777, 96, 16, 3, 4, "bf16", "none", "int32", 0),
])
def test_diagnostics_shapes(case):
    T, d, N, k, r, act, skew, idt, pad = case
    s = W.LayerShape("case", T=T, d=d, N=N, k=k, m=8, r=r, act=act, skew=skew)
    L = W.layer_inputs(s, 9, experts=False)
    L["A"] = L["A"] * 20.0            # a predictor strong enough to move some routes
    idx = oracle_route(L, s)
    z = predictive_logits(L)
    check(L, s, idx, run(L, s, idx, z, idt, pad), z, str(case))


def test_diagnostics_identical_route_and_reference():
    """Recorded route = current top-k and z_ref = p: every token has deviation
    0 and route KL 0."""
    s = W.LayerShape("same", T=1500, d=256, N=32, k=4, m=8, r=0, act="bf16", skew="hot8")
    L = W.layer_inputs(s, 10, experts=False)
    p = O.router_logits(L["x"], L["W_r"], L["beta"])
    idx = O.topk_ids(p, s.k)
    ok = O.topk_margin(p, s.k) >= MARGIN_EPS
    g = run(L, s, idx, p.astype(np.float32))
    assert np.all(g["overlap"][ok] == s.k)
    assert g["hist"][0] >= ok.sum() and g["hist"].sum() == s.T
    assert np.abs(g["kl"]).max() < 1e-6


def test_diagnostics_qwen3_30b_full():
    s = W.WORKLOADS["qwen3_30b_T16384"]
    L = W.layer_inputs(s, 0, experts=False)
    idx = oracle_route(L, s)
    z = predictive_logits(L)
    check(L, s, idx, run(L, s, idx, z), z, s.name)


def run_fused(L, s, idx_np, z_ref, idx_dtype="int32", ldi_pad=0):
    """pr2_moe_replay_forward_diag and, on the same inputs, pr2_moe_replay_forward
    and pr2_route_diagnostics."""
    import torch
    from paper_2606_00395_amd import binding as B
    x = to_dev(L["x"], s.act)
    Wr = to_dev(L["W_r"])
    br = to_dev(L["beta"]) if L["beta"] is not None else None
    Wg, Wu, Wd = (to_dev(L[n], s.act) for n in ("W_gate", "W_up", "W_down"))
    T, k = idx_np.shape
    dt = torch.int16 if idx_dtype == "int16" else torch.int32
    buf = torch.full((T, k + ldi_pad), -1, dtype=dt, device="cuda")
    buf[:, :k] = torch.from_numpy(idx_np.astype(np.int64)).to(dt).to("cuda")
    idx = buf[:, :k]
    zr = to_dev(z_ref)
    cur = torch.full((T, k), -5, dtype=dt, device="cuda")
    ov = torch.full((T,), -5, dtype=torch.int32, device="cuda")
    kl = torch.full((T,), float("nan"), device="cuda")
    hist = torch.full((k + 1,), 12345, dtype=torch.int64, device="cuda")
    y = torch.empty_like(x)
    gate = torch.empty((T, k), dtype=torch.float32, device="cuda")
    B.moe_replay_forward_diag(x, idx, Wr, br, Wg, Wu, Wd, y, gate, zr, cur, ov, kl, hist)
    y0 = torch.empty_like(x)
    gate0 = torch.empty_like(gate)
    B.moe_replay_forward(x, idx, Wr, br, Wg, Wu, Wd, y0, gate0)
    cur1, ov1, kl1, hist1 = (torch.empty_like(t) for t in (cur, ov, kl, hist))
    B.route_diagnostics(x, idx, Wr, br, zr, cur1, ov1, kl1, hist1)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16) if y.dtype == torch.bfloat16 else y,
                       y0.view(torch.int16) if y0.dtype == torch.bfloat16 else y0), \
        "fused replay output differs from pr2_moe_replay_forward"
    assert torch.equal(gate, gate0)
    for a, b in ((cur, cur1), (ov, ov1), (hist, hist1)):
        assert torch.equal(a, b), "fused diagnostics differ from pr2_route_diagnostics"
    assert torch.equal(kl.view(torch.int32), kl1.view(torch.int32))
    return {"cur": cur.cpu().numpy().astype(np.int64), "overlap": ov.cpu().numpy(),
            "kl": kl.cpu().numpy(), "hist": hist.cpu().numpy()}


@pytest.mark.parametrize("case", [
    (3000, 256, 64, 6, 8, 128, "bf16", "hot8", "int32", 0),
    (1000, 512, 128, 8, 16, 256, "bf16", "zipf", "int16", 2),
    (300, 64, 8, 2, 4, 40, "f32", "none", "int32", 1),
])
def test_replay_forward_fused_diagnostics(case):
    T, d, N, k, r, m, act, skew, idt, pad = case
    s = W.LayerShape("fused", T=T, d=d, N=N, k=k, m=m, r=r, act=act, skew=skew)
    L = W.layer_inputs(s, 12)
    L["A"] = L["A"] * 20.0            # a predictor strong enough to move some routes
    idx = oracle_route(L, s)
    z = predictive_logits(L)
    check(L, s, idx, run_fused(L, s, idx, z, idt, pad), z, "fused " + str(case))


def test_replay_forward_fused_diagnostics_qwen3_30b():
    s = W.WORKLOADS["qwen3_30b_T16384"]
    L = W.layer_inputs(s, 0)
    idx = oracle_route(L, s)
    z = predictive_logits(L)
    check(L, s, idx, run_fused(L, s, idx, z), z, "fused " + s.name)


def test_replay_forward_fused_diagnostics_empty_batch():
    import torch
    from paper_2606_00395_amd import binding as B
    d, N, m, k = 256, 8, 128, 2
    x = torch.empty((0, d), dtype=torch.bfloat16, device="cuda")
    idx = torch.empty((0, k), dtype=torch.int32, device="cuda")
    Wr = torch.zeros((d, N), device="cuda")
    Wg = torch.zeros((N, m, d), dtype=torch.bfloat16, device="cuda")
    Wd = torch.zeros((N, d, m), dtype=torch.bfloat16, device="cuda")
    hist = torch.full((k + 1,), 7, dtype=torch.int64, device="cuda")
    B.moe_replay_forward_diag(x, idx, Wr, None, Wg, Wg, Wd, torch.empty_like(x), hist_out=hist)
    torch.cuda.synchronize()
    assert torch.all(hist == 0)
