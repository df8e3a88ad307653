"""GPU parity of the predictor-training path against the float64 oracle:

* the fused feature-cache write (Alg. 2, caching step): for the positions the
  stratified sampler retains, h_cache holds the exact input rows and p_cache
  the router logits (fp32 rounding of the oracle's), while the recorded
  route follows the usual margin rule;
* the predictive loss and its gradients (Sec. 4.2, Eq. pr2_loss; Alg. 3) and
  the delta-matching variant (Appendix G), from a feature cache against a
  drifted current router: per-token KL, mean loss, dA and dB within 1e-5
  (Frobenius ratio) of the oracle; zeros at mini-step 1.

The drift is synthetic: the current router is W_r plus N(0, 0.002) noise and
the current hidden states are the cached ones plus N(0, 0.05) noise (bf16)."""
import numpy as np
import pytest

from oracle import pr2_oracle as O
import workloads as W
from tests.parity import compare_route, to_dev

pytestmark = pytest.mark.gpu

RTOL = 1e-5


def frob(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def cache_features(L, s, Tc, seed=5):
    import torch
    from paper_2606_00395_amd import binding as B
    pos = B.feature_cache_positions(s.T, Tc, seed)
    np.testing.assert_array_equal(pos, O.feature_cache_positions(s.T, Tc, seed))
    row = np.full(s.T, -1, dtype=np.int32)
    row[pos] = np.arange(len(pos), dtype=np.int32)
    x = to_dev(L["x"], s.act)
    dt = torch.bfloat16 if s.act == "bf16" else torch.float32
    h_cache = torch.full((len(pos), s.d), float("nan"), dtype=dt, device="cuda")
    p_cache = torch.full((len(pos), s.N), float("nan"), device="cuda")
    idx = torch.empty((s.T, s.k), dtype=torch.int32, device="cuda")
    gate = torch.empty((s.T, s.k), device="cuda")
    B.route_predict_cached(x, to_dev(L["W_r"]), to_dev(L["beta"]) if L["beta"] is not None else None,
                           to_dev(L["A"]), to_dev(L["B"]), s.k, idx,
                           torch.from_numpy(row).to("cuda"), h_cache, p_cache, gate)
    torch.cuda.synchronize()
    return pos, idx.cpu().numpy(), gate.cpu().numpy(), h_cache, p_cache


@pytest.mark.parametrize("name,Tc", [("tiny_fp32_T256", 64), ("qwen3_30b_T16384", 2048),
                                     ("tiny_fp32_T256", 300)])
def test_feature_cache_write(name, Tc):
    s = W.WORKLOADS[name]
    L = W.layer_inputs(s, 0, experts=False)
    pos, idx, gate, h_cache, p_cache = cache_features(L, s, Tc)
    ref = O.route_predict(L["x"], L["W_r"], L["beta"], L["A"], L["B"], s.k)
    compare_route(idx, gate, ref, s.k, name + " cached route")
    np.testing.assert_array_equal(h_cache.float().cpu().numpy(), L["x"][pos])
    np.testing.assert_allclose(p_cache.cpu().numpy(), ref["p"][pos], rtol=0,
                               atol=4e-6 * max(1.0, np.abs(ref["p"]).max()))


def drifted(L, s, seed=1):
    rng = np.random.default_rng([seed, 501])
    W_cur = (L["W_r"] + 0.002 * rng.standard_normal(L["W_r"].shape)).astype(np.float32)
    noise = 0.05 * rng.standard_normal(L["x"].shape)
    h_cur = W.round_to_bf16((L["x"] + noise).astype(np.float32)) if s.act == "bf16" else \
        (L["x"] + noise).astype(np.float32)
    return W_cur, h_cur


def run_loss(L, s, Tc, kind, identity=False, mini_step=2):
    """The loss on a feature cache built from the oracle (never from the HIP
    path): h_old = the cached positions' input rows, p_old = the oracle's router
    logits there rounded to fp32 (the precision the cache stores)."""
    import torch
    from paper_2606_00395_amd import binding as B
    pos = O.feature_cache_positions(s.T, Tc, 5)
    p_old = O.router_logits(L["x"][pos], L["W_r"], L["beta"]).astype(np.float32)
    h_cache = to_dev(L["x"][pos], s.act)
    p_cache = to_dev(p_old)
    W_cur, h_cur = drifted(L, s)
    A = L["A"]
    Bm = None if identity else L["B"]
    r = A.shape[1]
    loss = torch.full((1,), float("nan"), device="cuda")
    dA = torch.full((s.d, r), float("nan"), device="cuda")
    dB = None if identity else torch.full((r, s.N), float("nan"), device="cuda")
    kl = torch.full((len(pos),), float("nan"), device="cuda")
    B.predictor_loss(to_dev(h_cur[pos], s.act), to_dev(W_cur),
                     to_dev(L["beta"]) if L["beta"] is not None else None, h_cache, p_cache,
                     to_dev(A), to_dev(Bm), loss, dA, dB, kl, loss_kind=kind, mini_step=mini_step)
    torch.cuda.synchronize()
    g = {"loss": loss.cpu().numpy()[0], "dA": dA.cpu().numpy(), "kl": kl.cpu().numpy(),
         "dB": None if identity else dB.cpu().numpy()}
    p_cur = O.router_logits(h_cur[pos], W_cur, L["beta"])
    fn = O.predictive_kl if kind == 0 else O.delta_matching_kl
    kl_ref, dA_ref, dB_ref = fn(p_cur, L["x"][pos], p_old, A, Bm)
    return g, (kl_ref, dA_ref, dB_ref)


@pytest.mark.parametrize("name,Tc,kind", [("tiny_fp32_T256", 256, 0), ("tiny_fp32_T256", 100, 1),
                                          ("qwen3_30b_T16384", 2048, 0),
                                          ("qwen3_30b_T16384", 2048, 1),
                                          ("qwen3_30b_T16384", 1000, 0)])
def test_predictor_loss_matches_oracle(name, Tc, kind):
    s = W.WORKLOADS[name]
    L = W.layer_inputs(s, 0, experts=False)
    g, (kl_ref, dA_ref, dB_ref) = run_loss(L, s, Tc, kind)
    errs = {"kl": frob(g["kl"], kl_ref), "loss": abs(g["loss"] - kl_ref.mean()) / kl_ref.mean(),
            "dA": frob(g["dA"], dA_ref), "dB": frob(g["dB"], dB_ref)}
    print(f"\n{name} Tc={Tc} kind={kind}: loss {g['loss']:.4e} " +
          ", ".join(f"{k} {v:.1e}" for k, v in errs.items()))
    assert max(errs.values()) <= RTOL, errs


def test_predictor_loss_full_rank_identity():
    s = W.LayerShape("fr", T=600, d=256, N=32, k=4, m=8, r=32, act="bf16", skew="hot8")
    L = W.layer_inputs(s, 2, experts=False)
    g, (kl_ref, dA_ref, _) = run_loss(L, s, 200, 0, identity=True)
    assert frob(g["kl"], kl_ref) <= RTOL and frob(g["dA"], dA_ref) <= RTOL


def test_predictor_loss_skipped_at_first_mini_step():
    s = W.WORKLOADS["tiny_fp32_T256"]
    L = W.layer_inputs(s, 0, experts=False)
    g, _ = run_loss(L, s, 128, 0, mini_step=1)
    assert g["loss"] == 0.0 and np.all(g["dA"] == 0.0) and np.all(g["dB"] == 0.0)
    assert np.all(g["kl"] == 0.0)
