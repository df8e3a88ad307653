"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test ties one oracle function to something other than itself: brute
force over all k-subsets, closed forms on one-hot inputs, library routines
on special cases (scipy softmax/expit, torch's silu MLP), the paper's
Lemma B.2 (Appendix B.2), central finite differences, and the numbers printed
in Table 3 (Appendix E.2).  The last group plants mistakes in copies of the
oracle and checks that these pins catch them.
"""
import itertools
import json
import os

import numpy as np
import pytest
import scipy.special
import torch

from oracle import pr2_oracle as O
from paper_2606_00395_amd import costmodel
import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))


def rand(rng, *shape, std=1.0):
    return rng.standard_normal(shape) * std


# ------------------------------------------------------------ top-k (P2) ---

def brute_topk(z, k):
    """Among all k-subsets maximising the summed score, the lexicographically
    smallest sorted id tuple (ties to the lower id)."""
    best, best_key = None, None
    N = len(z)
    for S in itertools.combinations(range(N), k):
        key = (sum(z[j] for j in S), tuple(-j for j in S))
        if best_key is None or key > best_key:
            best, best_key = S, key
    return np.array(best)


@pytest.mark.parametrize("N,k", [(8, 2), (8, 1), (8, 8), (6, 3), (10, 4)])
def test_topk_matches_brute_force_random(N, k):
    rng = np.random.default_rng(11)
    z = rand(rng, 200, N)
    got = O.topk_ids(z, k)
    for t in range(z.shape[0]):
        np.testing.assert_array_equal(got[t], brute_topk(z[t].astype(np.float32).tolist(), k))


@pytest.mark.parametrize("N,k", [(8, 2), (8, 3), (7, 4), (5, 5)])
def test_topk_ties_go_to_lower_id(N, k):
    # integer-valued logits: sums are exact and ties are frequent
    rng = np.random.default_rng(3)
    z = rng.integers(-2, 3, size=(300, N)).astype(np.float64)
    got = O.topk_ids(z, k)
    for t in range(z.shape[0]):
        np.testing.assert_array_equal(got[t], brute_topk(z[t].tolist(), k))


def test_topk_signed_zero_is_a_tie():
    z = np.array([[-0.0, 0.0, -1.0, -1.0], [0.0, -0.0, -1.0, -1.0]])
    np.testing.assert_array_equal(O.topk_ids(z, 1), [[0], [0]])
    np.testing.assert_array_equal(O.topk_ids(z, 3), [[0, 1, 2], [0, 1, 2]])


def test_topk_decides_in_fp32():
    # two logits equal in fp32 but not in fp64: the fp32 decision makes them a tie
    a = 1.0
    b = 1.0 + 2.0 ** -30
    z = np.array([[a, b, 0.0]])
    assert np.float32(a) == np.float32(b)
    np.testing.assert_array_equal(O.topk_ids(z, 1), [[0]])
    np.testing.assert_array_equal(O.topk_ids(z, 1, decide_dtype=np.float64), [[1]])


def test_topk_margin_closed_form():
    z = np.array([[3.0, 1.0, 2.0, 0.5]])
    np.testing.assert_allclose(O.topk_margin(z, 1), [1.0])
    np.testing.assert_allclose(O.topk_margin(z, 2), [1.0])
    np.testing.assert_allclose(O.topk_margin(z, 3), [0.5])
    assert np.isinf(O.topk_margin(z, 4)[0])


# ------------------------------------------------- Lemma B.2 invariant (P4) --

def test_lemma_b2_topk_mass_regret():
    """Appendix B.2, Lemma B.2: p(S*) - p(S_hat) <= sqrt(2 KL(p || p_hat)), and the
    top-k sets agree when KL < margin^2 / 2.  Checked on random distributions."""
    rng = np.random.default_rng(5)
    checked_equal = 0
    for trial in range(3000):
        N = int(rng.integers(3, 12))
        k = int(rng.integers(1, N))
        zp = rand(rng, 1, N, std=float(rng.uniform(0.3, 3.0)))
        zq = zp + rand(rng, 1, N, std=float(rng.choice([1e-3, 1e-2, 0.1, 1.0])))
        p, q = scipy.special.softmax(zp, axis=1)[0], scipy.special.softmax(zq, axis=1)[0]
        S = O.topk_ids(np.log(p)[None], k, decide_dtype=np.float64)[0]
        Sh = O.topk_ids(np.log(q)[None], k, decide_dtype=np.float64)[0]
        kl = float(np.sum(p * (np.log(p) - np.log(q))))
        assert p[S].sum() - p[Sh].sum() <= np.sqrt(2 * kl) + 1e-12
        # S must carry the most p-mass of any k-subset
        assert p[S].sum() >= np.sort(p)[::-1][:k].sum() - 1e-12
        ps = np.sort(p)[::-1]
        margin = ps[k - 1] - ps[k]
        if margin > 0 and kl < margin ** 2 / 2:
            np.testing.assert_array_equal(S, Sh)
            checked_equal += 1
    assert checked_equal > 100


# --------------------------------------------------------- gates (P3, P5) ---

def test_gates_closed_forms():
    rng = np.random.default_rng(7)
    z = rand(rng, 50, 8, std=2.0)
    # k = N: the renormalised gates are the full softmax (library routine)
    idx = O.topk_ids(z, 8)
    np.testing.assert_allclose(O.gates_on_route(z, idx, True),
                               np.take_along_axis(scipy.special.softmax(z, axis=1), idx, 1),
                               rtol=1e-13)
    # k = 1: the single gate is 1
    idx1 = O.topk_ids(z, 1)
    np.testing.assert_allclose(O.gates_on_route(z, idx1, True), 1.0, rtol=0, atol=1e-15)
    # k = 2: the pair of renormalised gates is (expit(z_a - z_b), expit(z_b - z_a))
    idx2 = O.topk_ids(z, 2)
    g2 = O.gates_on_route(z, idx2, True)
    za = np.take_along_axis(z, idx2, 1)
    np.testing.assert_allclose(g2[:, 0], scipy.special.expit(za[:, 0] - za[:, 1]), rtol=1e-13)
    # literal (no renorm): rho_j from the softmax over all N
    idx3 = O.topk_ids(z, 3)
    np.testing.assert_allclose(O.gates_on_route(z, idx3, False),
                               np.take_along_axis(scipy.special.softmax(z, axis=1), idx3, 1),
                               rtol=1e-13)


def test_renormalised_gates_sum_to_one_and_shift_invariant():
    rng = np.random.default_rng(8)
    z = rand(rng, 400, 16, std=3.0)
    for k in (1, 2, 5, 16):
        idx = O.topk_ids(z, k)
        g = O.gates_on_route(z, idx, True)
        assert np.all(np.abs(g.sum(1) - 1.0) <= 1e-12)
        g_shift = O.gates_on_route(z + 123.25, idx, True)
        np.testing.assert_allclose(g, g_shift, rtol=1e-12)
        # literal weights sum to the route's probability mass, below 1 unless k = N
        gl = O.gates_on_route(z, idx, False)
        assert np.all(gl.sum(1) <= 1 + 1e-12)


# ------------------------------------------------- router and predictor ----

def test_router_logits_one_hot_rows():
    """p = h W + beta: a one-hot router input e_i selects row i of W plus beta."""
    rng = np.random.default_rng(9)
    d, N = 6, 4
    Wr = rand(rng, d, N)
    beta = rand(rng, N)
    h = np.eye(d)
    np.testing.assert_array_equal(O.router_logits(h, Wr, beta), Wr + beta[None])
    np.testing.assert_array_equal(O.router_logits(h, Wr, None), Wr)


def test_predictor_bias_one_hot_and_full_rank():
    """b = h A B: one-hot h gives A[i] B; a full-rank predictor W_p is A with B = identity."""
    rng = np.random.default_rng(10)
    d, r, N = 5, 3, 4
    A, B = rand(rng, d, r), rand(rng, r, N)
    h = np.eye(d)
    np.testing.assert_allclose(O.predictor_bias(h, A, B), np.stack([A[i] @ B for i in range(d)]),
                               rtol=1e-14)
    Wp = rand(rng, d, N)
    np.testing.assert_array_equal(O.predictor_bias(h, Wp, None), Wp)
    np.testing.assert_array_equal(O.predictor_bias(h, Wp, np.eye(N)), Wp)


def test_zero_predictor_is_routing_replay():
    """The predictor is zero-initialised (Sec. 4.1), so Pr^2 at init records the
    old router's own top-k: the vanilla routing-replay route (Sec. 3.2)."""
    rng = np.random.default_rng(12)
    T, d, N, k, r = 300, 16, 8, 2, 4
    h, Wr, beta = rand(rng, T, d), rand(rng, d, N, std=0.3), rand(rng, N)
    A0 = np.zeros((d, r))
    B = rand(rng, r, N)
    rt = O.route_predict(h, Wr, beta, A0, B, k)
    rt_none = O.route_predict(h, Wr, beta, None, None, k)
    np.testing.assert_array_equal(rt["idx"], rt_none["idx"])
    # brute force on the router logits alone
    p = h @ Wr + beta
    for t in range(T):
        np.testing.assert_array_equal(rt["idx"][t], brute_topk(p[t].astype(np.float32).tolist(), k))


def test_replay_reproduces_rollout_with_zero_predictor():
    """With a zero predictor and unchanged router, replaying the recorded ids
    gives the rollout gates and the rollout output exactly (Sec. 4.1)."""
    rng = np.random.default_rng(13)
    T, d, N, k, m, r = 64, 16, 8, 3, 12, 2
    h, Wr = rand(rng, T, d), rand(rng, d, N, std=0.4)
    Wg, Wu, Wd = rand(rng, N, m, d, std=0.2), rand(rng, N, m, d, std=0.2), rand(rng, N, d, m, std=0.2)
    y_roll, rt = O.rollout_forward(h, Wr, None, np.zeros((d, r)), rand(rng, r, N), k, Wg, Wu, Wd)
    y_rep, g_rep = O.replay_forward(h, rt["idx"], Wr, None, Wg, Wu, Wd)
    np.testing.assert_array_equal(g_rep, rt["gate"])
    np.testing.assert_array_equal(y_rep, y_roll)


def test_replay_bypasses_predictor():
    """Replay weights come from the current router only (Sec. 4.1): with a
    one-hot input the replay logits are W[i] + beta whatever A, B are."""
    rng = np.random.default_rng(14)
    d, N, k, r = 6, 5, 2, 3
    Wr, beta = rand(rng, d, N), rand(rng, N)
    A, B = rand(rng, d, r, std=5.0), rand(rng, r, N, std=5.0)
    h = np.eye(d)
    rt = O.route_predict(h, Wr, beta, A, B, k)
    g, p = O.replay_gates(h, Wr, beta, rt["idx"])
    np.testing.assert_array_equal(p, Wr + beta[None])
    sel = np.take_along_axis(Wr + beta[None], rt["idx"], 1)
    np.testing.assert_allclose(g, scipy.special.softmax(sel, axis=1), rtol=1e-13)
    # the rollout gates use the predictive logits instead, which differ here
    zsel = np.take_along_axis(Wr + beta[None] + A @ B, rt["idx"], 1)
    np.testing.assert_allclose(rt["gate"], scipy.special.softmax(zsel, axis=1), rtol=1e-13)
    assert not np.allclose(rt["gate"], g)


# ----------------------------------------------------------- experts (P6) ---

def torch_swiglu(h, Wg, Wu, Wd):
    h, Wg, Wu, Wd = (torch.from_numpy(np.asarray(a, dtype=np.float64)) for a in (h, Wg, Wu, Wd))
    return (torch.nn.functional.silu(torch.nn.functional.linear(h, Wg))
            * torch.nn.functional.linear(h, Wu)) @ Wd.T


def test_single_expert_is_dense_swiglu_mlp():
    """N = 1, k = 1: the MoE layer is one dense SwiGLU MLP (gate 1)."""
    rng = np.random.default_rng(15)
    T, d, m = 40, 12, 20
    h = rand(rng, T, d)
    Wr = rand(rng, d, 1)
    Wg, Wu, Wd = rand(rng, 1, m, d, std=0.3), rand(rng, 1, m, d, std=0.3), rand(rng, 1, d, m, std=0.3)
    idx = np.zeros((T, 1), dtype=np.int64)
    y, g = O.replay_forward(h, idx, Wr, None, Wg, Wu, Wd)
    np.testing.assert_array_equal(g, 1.0)
    np.testing.assert_allclose(y, torch_swiglu(h, Wg[0], Wu[0], Wd[0]).numpy(), rtol=1e-12, atol=1e-14)
    # the expert function alone against the library silu
    np.testing.assert_allclose(O.expert_ffn(h, Wg[0], Wu[0], Wd[0]),
                               torch_swiglu(h, Wg[0], Wu[0], Wd[0]).numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(O.silu(np.linspace(-8, 8, 33)),
                               np.linspace(-8, 8, 33) * scipy.special.expit(np.linspace(-8, 8, 33)),
                               rtol=1e-14)


def small_layer(seed=16, T=96, d=16, N=8, k=3, m=24):
    rng = np.random.default_rng(seed)
    return dict(h=rand(rng, T, d), Wr=rand(rng, d, N, std=0.4), beta=rand(rng, N),
                Wg=rand(rng, N, m, d, std=0.2), Wu=rand(rng, N, m, d, std=0.2),
                Wd=rand(rng, N, d, m, std=0.2), k=k)


def test_zero_down_projection_gives_zero_output():
    L = small_layer()
    idx = O.topk_ids(O.router_logits(L["h"], L["Wr"], L["beta"]), L["k"])
    y, _ = O.replay_forward(L["h"], idx, L["Wr"], L["beta"], L["Wg"], L["Wu"], np.zeros_like(L["Wd"]))
    assert np.all(y == 0)


def test_dense_all_experts_then_mask_matches_masked_per_expert():
    """The per-expert masked combine equals evaluating every expert on every
    token with torch's silu MLP and weighting by a dense [T, N] gate matrix."""
    L = small_layer()
    p = O.router_logits(L["h"], L["Wr"], L["beta"])
    idx = O.topk_ids(p, L["k"])
    y, g = O.replay_forward(L["h"], idx, L["Wr"], L["beta"], L["Wg"], L["Wu"], L["Wd"])
    T, N = p.shape
    G = np.zeros((T, N))
    np.put_along_axis(G, idx, g, axis=1)
    dense = np.stack([torch_swiglu(L["h"], L["Wg"][e], L["Wu"][e], L["Wd"][e]).numpy()
                      for e in range(N)], axis=1)  # [T, N, d]
    np.testing.assert_allclose(y, (G[:, :, None] * dense).sum(1), rtol=1e-12, atol=1e-13)
    # and the one-token-at-a-time path agrees too
    rows = np.arange(0, T, 7)
    yr, gr = O.replay_forward_rows(rows, L["h"][rows], idx[rows], L["Wr"], L["beta"],
                                   L["Wg"], L["Wu"], L["Wd"])
    np.testing.assert_allclose(yr, y[rows], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(gr, g[rows], rtol=1e-14)


def test_expert_relabelling_and_token_permutation():
    L = small_layer(seed=17)
    N = L["Wr"].shape[1]
    A = np.random.default_rng(1).standard_normal((L["h"].shape[1], 2))
    B = np.random.default_rng(2).standard_normal((2, N))
    y, rt = O.rollout_forward(L["h"], L["Wr"], L["beta"], A, B, L["k"], L["Wg"], L["Wu"], L["Wd"])
    pi = np.random.default_rng(3).permutation(N)     # new expert j is old expert pi[j]
    y2, rt2 = O.rollout_forward(L["h"], L["Wr"][:, pi], L["beta"][pi], A, B[:, pi], L["k"],
                                L["Wg"][pi], L["Wu"][pi], L["Wd"][pi])
    np.testing.assert_allclose(y2, y, rtol=1e-12, atol=1e-13)
    assert all(set(pi[rt2["idx"][t]].tolist()) == set(rt["idx"][t].tolist())
               for t in range(len(y)))
    sigma = np.random.default_rng(4).permutation(len(y))
    y3, _ = O.rollout_forward(L["h"][sigma], L["Wr"], L["beta"], A, B, L["k"], L["Wg"], L["Wu"], L["Wd"])
    np.testing.assert_allclose(y3, y[sigma], rtol=1e-12, atol=1e-13)


# -------------------------------------------------------------- backward ---

def _loss(h, Wr, beta, Wg, Wu, Wd, dy, idx, renorm):
    y, _ = O.replay_forward(h, idx, Wr, beta, Wg, Wu, Wd, renorm)
    return float((y * dy).sum())


@pytest.mark.parametrize("renorm", [True, False])
def test_backward_matches_central_differences(renorm):
    rng = np.random.default_rng(18)
    T, d, N, k, m = 10, 6, 5, 2, 7
    h, Wr, beta = rand(rng, T, d), rand(rng, d, N, std=0.5), rand(rng, N)
    Wg, Wu, Wd = rand(rng, N, m, d, std=0.4), rand(rng, N, m, d, std=0.4), rand(rng, N, d, m, std=0.4)
    dy = rand(rng, T, d)
    idx = O.topk_ids(O.router_logits(h, Wr, beta), k)
    g = O.replay_backward(h, idx, Wr, beta, Wg, Wu, Wd, dy, renorm)
    args = dict(h=h, Wr=Wr, beta=beta, Wg=Wg, Wu=Wu, Wd=Wd)
    names = dict(h="dx", Wr="dW_r", beta="dbeta", Wg="dW_gate", Wu="dW_up", Wd="dW_down")
    eps = 1e-6
    for key, gname in names.items():
        a = args[key]
        fd = np.zeros_like(a)
        for i in range(a.size):
            orig = a.flat[i]
            a.flat[i] = orig + eps
            lp = _loss(dy=dy, idx=idx, renorm=renorm, **args)
            a.flat[i] = orig - eps
            lm = _loss(dy=dy, idx=idx, renorm=renorm, **args)
            a.flat[i] = orig
            fd.flat[i] = (lp - lm) / (2 * eps)
        np.testing.assert_allclose(g[gname], fd, rtol=1e-6, atol=1e-8, err_msg=gname)
    if renorm:
        # the route's logits gradient sums to zero per token (softmax shift invariance)
        assert np.allclose(g["dbeta"].sum(), 0.0, atol=1e-10)


# --------------------------------------------------- predictive KL loss -----

def test_predictive_kl_zero_when_predictor_matches_and_gradients():
    rng = np.random.default_rng(19)
    T, d, N, r = 20, 6, 5, 3
    h_old, p_old = rand(rng, T, d), rand(rng, T, N)
    A, B = rand(rng, d, r, std=0.3), rand(rng, r, N, std=0.3)
    # current logits equal to the predictive logits (up to a per-token shift): KL = 0
    p_cur = p_old + h_old @ A @ B + rand(rng, T, 1)
    kl, dA, dB = O.predictive_kl(p_cur, h_old, p_old, A, B)
    np.testing.assert_allclose(kl, 0.0, atol=1e-12)
    np.testing.assert_allclose(dA, 0.0, atol=1e-12)
    # KL against scipy's relative entropy on an unrelated target
    p_cur = rand(rng, T, N)
    kl, dA, dB = O.predictive_kl(p_cur, h_old, p_old, A, B)
    ref = scipy.special.rel_entr(scipy.special.softmax(p_cur, 1),
                                 scipy.special.softmax(p_old + h_old @ A @ B, 1)).sum(1)
    np.testing.assert_allclose(kl, ref, rtol=1e-10)
    eps = 1e-6
    for M, G in ((A, dA), (B, dB)):
        fd = np.zeros_like(M)
        for i in range(M.size):
            o = M.flat[i]
            M.flat[i] = o + eps
            lp = O.predictive_kl(p_cur, h_old, p_old, A, B)[0].mean()
            M.flat[i] = o - eps
            lm = O.predictive_kl(p_cur, h_old, p_old, A, B)[0].mean()
            M.flat[i] = o
            fd.flat[i] = (lp - lm) / (2 * eps)
        np.testing.assert_allclose(G, fd, rtol=1e-6, atol=1e-9)


def _fd_mean(fn, M, eps=1e-6):
    fd = np.zeros_like(M)
    for i in range(M.size):
        o = M.flat[i]
        M.flat[i] = o + eps
        lp = fn()[0].mean()
        M.flat[i] = o - eps
        lm = fn()[0].mean()
        M.flat[i] = o
        fd.flat[i] = (lp - lm) / (2 * eps)
    return fd


def test_predictive_kl_full_rank_identity():
    """B = None (W_p = A, r = N) equals passing the identity matrix."""
    rng = np.random.default_rng(20)
    T, d, N = 15, 5, 6
    h_old, p_old, p_cur = rand(rng, T, d), rand(rng, T, N), rand(rng, T, N)
    A = rand(rng, d, N, std=0.3)
    kl, dA, dB = O.predictive_kl(p_cur, h_old, p_old, A, None)
    kl2, dA2, _ = O.predictive_kl(p_cur, h_old, p_old, A, np.eye(N))
    np.testing.assert_allclose(kl, kl2, rtol=1e-12)
    np.testing.assert_allclose(dA, dA2, rtol=1e-12, atol=1e-15)
    assert dB is None
    np.testing.assert_allclose(dA, _fd_mean(lambda: O.predictive_kl(p_cur, h_old, p_old, A, None), A),
                               rtol=1e-6, atol=1e-9)


def test_delta_matching_kl_closed_forms_and_gradients():
    rng = np.random.default_rng(21)
    T, d, N, r = 20, 6, 5, 3
    h_old, p_old = rand(rng, T, d), rand(rng, T, N)
    A, B = rand(rng, d, r, std=0.3), rand(rng, r, N, std=0.3)
    # the current logits moved by exactly the predicted residual: zero loss and gradient
    p_cur = p_old + h_old @ A @ B + rand(rng, T, 1)
    kl, dA, dB = O.delta_matching_kl(p_cur, h_old, p_old, A, B)
    np.testing.assert_allclose(kl, 0.0, atol=1e-12)
    np.testing.assert_allclose(dB, 0.0, atol=1e-12)
    p_cur = rand(rng, T, N)
    kl, dA, dB = O.delta_matching_kl(p_cur, h_old, p_old, A, B)
    ref = scipy.special.rel_entr(scipy.special.softmax(p_cur - p_old, 1),
                                 scipy.special.softmax(h_old @ A @ B, 1)).sum(1)
    np.testing.assert_allclose(kl, ref, rtol=1e-10)
    # it differs from the standard objective (which keeps p_old inside rho_hat)
    assert not np.allclose(kl, O.predictive_kl(p_cur, h_old, p_old, A, B)[0])
    fn = lambda: O.delta_matching_kl(p_cur, h_old, p_old, A, B)
    np.testing.assert_allclose(dA, _fd_mean(fn, A), rtol=1e-6, atol=1e-9)
    np.testing.assert_allclose(dB, _fd_mean(fn, B), rtol=1e-6, atol=1e-9)


# ------------------------------------------------- Table 3 cost formulas ----

def test_table3_overheads_reproduce():
    with open(os.path.join(HERE, "golden", "table3_overheads.json")) as f:
        rows = json.load(f)["rows"]
    for r in rows:
        idx_mb = costmodel.index_cache_bytes(r["T"], r["L"], r["k"]) / 1e6
        feat_mb = costmodel.feature_cache_bytes(r["Tc"], r["L"], r["d"], r["N"]) / 1e6
        flops_m = costmodel.predictor_flops_per_token(r["L"], r["d"], r["N"]) / 1e6
        ratio = 100 * costmodel.ffn_ratio(r["L"], r["d"], r["N"], r["k"], r["s"], r["m"])
        # each value rounds to the digits the table prints
        for got, key in ((idx_mb, "index_cache_MB"), (feat_mb, "feature_cache_MB"),
                         (flops_m, "flops_M"), (ratio, "ffn_ratio_pct")):
            printed = r[key]
            txt = repr(printed)
            decimals = len(txt.split(".")[1]) if "." in txt else 0
            assert round(got, decimals) == printed, (r["model"], key, got, printed)


# ------------------------------------------------------ input generators ----

def test_bf16_rounding_is_nearest_even_and_exact():
    a = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5e-3], dtype=np.float32)
    r = W.round_to_bf16(a.copy())
    t = torch.from_numpy(a.copy()).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(r, t)
    rng = np.random.default_rng(0)
    b = rng.standard_normal(100000).astype(np.float32)
    np.testing.assert_array_equal(W.round_to_bf16(b.copy()),
                                  torch.from_numpy(b).to(torch.bfloat16).to(torch.float32).numpy())


def test_workload_generators_are_deterministic_and_row_addressable():
    s = W.WORKLOADS["tiny_fp32_T256"]
    a = W.layer_inputs(s, 0)
    b = W.layer_inputs(s, 0)
    for key in a:
        if a[key] is None:
            assert b[key] is None
        else:
            np.testing.assert_array_equal(a[key], b[key])
    rows = np.array([0, 5, 255, 17])
    np.testing.assert_array_equal(W.hidden_states(s, 0, rows), a["x"][rows])
    big = W.WORKLOADS["qwen3_30b_T16384"].with_(T=3000, d=32, N=16, m=8)
    xb = W.hidden_states(big, 1)
    rows = np.array([2999, 0, 1024, 2047])
    np.testing.assert_array_equal(W.hidden_states(big, 1, rows), xb[rows])
    # bf16 activations are exactly representable
    np.testing.assert_array_equal(W.round_to_bf16(xb.copy()), xb)
    beta = W.router_bias(big, 0)
    assert (beta == 1.0).sum() == 8 and (beta == 0).sum() == 8
    z = W.router_bias(W.WORKLOADS["qwen3_235b_T32768"], 0)
    np.testing.assert_allclose(np.sort(np.exp(-z / 1.1)), np.arange(1, 129), rtol=1e-5)
    fl = W.flip_tokens(W.WORKLOADS["qwen3_30b_bwd_T16384"], 0)
    assert len(fl) == 819 and len(np.unique(fl)) == 819


def test_flip_route_recipe_differs_in_exactly_one_slot():
    """The backward workload's recorded route: the current top-k of the replay
    router, with the k-th ranked expert swapped for the (k+1)-th on 5 % of the
    tokens.  Checked with brute force: flipped tokens overlap the current top-k
    in k-1 ids and hold the (k+1)-th ranked one, the others equal it."""
    s = W.LayerShape("flip", T=400, d=32, N=12, k=3, m=8, r=0, act="f32", skew="hot8",
                     flip_frac=0.05)
    L = W.layer_inputs(s, 3, experts=False)
    p = O.router_logits(L["x"], L["W_r"], L["beta"])
    ranked = np.argsort(-p.astype(np.float32), axis=1, kind="stable")[:, :s.k + 1]
    fl = W.flip_tokens(s, 3)
    assert len(fl) == 20
    idx = W.flip_route(ranked, fl, s.k)
    cur = O.topk_ids(p, s.k)
    ov = O.route_overlap(idx, cur)
    flipped = np.zeros(s.T, dtype=bool)
    flipped[fl] = True
    assert np.all(ov[flipped] == s.k - 1) and np.all(ov[~flipped] == s.k)
    np.testing.assert_array_equal(idx[~flipped], cur[~flipped])
    for t in fl:
        order = sorted(range(s.N), key=lambda j: (-np.float32(p[t, j]), j))
        assert order[s.k] in idx[t] and order[s.k - 1] not in idx[t]
    assert np.all(np.diff(idx, axis=1) > 0)


# ------------------------------------------------ route metrics (Sec. 5.4) ---

def test_route_overlap_agreement_and_deviation_brute_force():
    rng = np.random.default_rng(31)
    T, N, k = 200, 9, 3
    a = np.sort(np.array([rng.choice(N, k, replace=False) for _ in range(T)]), axis=1)
    b = np.sort(np.array([rng.choice(N, k, replace=False) for _ in range(T)]), axis=1)
    inter = np.array([sum(int(x == y) for x in a[t] for y in b[t]) for t in range(T)])
    np.testing.assert_array_equal(O.route_overlap(a, b), inter)
    np.testing.assert_allclose(O.route_agreement(a, b), inter / k)
    hist = O.route_deviation_histogram(a, b)
    assert hist.shape == (k + 1,) and hist.sum() == T
    np.testing.assert_array_equal(hist, [(k - inter == dv).sum() for dv in range(k + 1)])
    # identical routes: all mass at zero deviation; disjoint: all at k
    np.testing.assert_array_equal(O.route_deviation_histogram(a, a), [T] + [0] * k)
    c = np.tile(np.arange(k), (T, 1))
    dd = np.tile(np.arange(k, 2 * k), (T, 1))
    np.testing.assert_array_equal(O.route_deviation_histogram(c, dd), [0] * k + [T])
    # order of ids within a row does not matter
    np.testing.assert_array_equal(O.route_overlap(a[:, ::-1], b), inter)


def test_route_kl_closed_forms():
    rng = np.random.default_rng(32)
    p = rand(rng, 50, 7)
    np.testing.assert_allclose(O.route_kl(p, p), 0.0, atol=1e-13)
    z = rand(rng, 50, 7)
    kl = O.route_kl(p, z)
    assert np.all(kl > 0)
    # invariant to a per-token shift of either logit vector
    np.testing.assert_allclose(O.route_kl(p + 3.0, z - 1.5), kl, rtol=1e-10)
    # two experts: the binary KL of the two sigmoids
    a, b = rand(rng, 40), rand(rng, 40)
    s, t = scipy.special.expit(a), scipy.special.expit(b)
    bern = s * np.log(s / t) + (1 - s) * np.log((1 - s) / (1 - t))
    np.testing.assert_allclose(O.route_kl(np.stack([a, 0 * a], 1), np.stack([b, 0 * b], 1)), bern,
                               rtol=1e-10)
    # scipy's relative entropy of the two softmax vectors
    ref = scipy.special.rel_entr(scipy.special.softmax(p, axis=1),
                                 scipy.special.softmax(z, axis=1)).sum(axis=1)
    np.testing.assert_allclose(kl, ref, rtol=1e-10)


def test_route_kl_small_enough_keeps_the_top_k():
    """Lemma B.2: KL(p || p_hat) < margin^2 / 2 implies TopK(p_hat) = TopK(p),
    with p, p_hat the two distributions and the margin taken on p."""
    rng = np.random.default_rng(33)
    N, k = 12, 4
    hits = 0
    for _ in range(400):
        p = rand(rng, 1, N) * 2.0
        z = p + rand(rng, 1, N) * 0.02
        rho = O.softmax(p)[0]
        srt = np.sort(rho)[::-1]
        margin = srt[k - 1] - srt[k]
        if O.route_kl(p, z)[0] < margin ** 2 / 2:
            hits += 1
            assert set(O.topk_ids(p, k)[0]) == set(O.topk_ids(z, k)[0])
    assert hits > 20


# ------------------------------------------------ feature cache (App. E.2) ---

def test_splitmix64_published_sequence():
    """The first outputs of SplitMix64 seeded with 0, as published with the
    generator's reference implementation."""
    outs = [O.splitmix64((i + 1) * 0x9E3779B97F4A7C15) for i in range(3)]
    assert outs == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_feature_cache_positions_stratified_uniform():
    T, Tc = 16384, 2048
    pos = O.feature_cache_positions(T, Tc, 7)
    assert pos.shape == (Tc,) and np.all(np.diff(pos) > 0) and pos[0] >= 0 and pos[-1] < T
    # exactly one retained position per stratum of T / Tc tokens
    np.testing.assert_array_equal(pos // (T // Tc), np.arange(Tc))
    np.testing.assert_array_equal(pos, O.feature_cache_positions(T, Tc, 7))
    assert not np.array_equal(pos, O.feature_cache_positions(T, Tc, 8))
    # uneven strata still cover [0, T) with one draw each
    pos2 = O.feature_cache_positions(1000, 7, 1)
    bounds = [(i * 1000) // 7 for i in range(8)]
    assert all(bounds[i] <= pos2[i] < bounds[i + 1] for i in range(7))
    # offsets within a stratum are uniform: chi-square over many seeds
    off = np.concatenate([O.feature_cache_positions(800, 100, sd) % 8 for sd in range(60)])
    counts = np.bincount(off, minlength=8)
    chi2 = ((counts - off.size / 8) ** 2 / (off.size / 8)).sum()
    assert chi2 < 24.3   # 7 degrees of freedom, p = 0.001
    np.testing.assert_array_equal(O.feature_cache_positions(50, 64, 3), np.arange(50))


# ------------------------------------------------- planted mistakes ----------

def test_pins_catch_planted_mistakes(monkeypatch):
    """A copy of the oracle with one plausible mistake fails at least one pin."""
    import types

    def fails(fn):
        try:
            fn()
        except AssertionError:
            return True
        return False

    # ties to the higher id
    bad = types.SimpleNamespace(**vars(O))
    monkeypatch.setattr(O, "topk_ids", lambda z, k, decide_dtype=np.float32: np.sort(
        (z.shape[-1] - 1 - np.argsort(-np.asarray(z)[:, ::-1].astype(decide_dtype), axis=-1,
                                      kind="stable"))[:, :k], axis=-1))
    assert fails(lambda: test_topk_ties_go_to_lower_id(8, 3))
    monkeypatch.setattr(O, "topk_ids", bad.topk_ids)

    # router bias dropped
    monkeypatch.setattr(O, "router_logits", lambda h, W_r, beta=None: np.asarray(h) @ np.asarray(W_r))
    assert fails(test_router_logits_one_hot_rows)
    monkeypatch.setattr(O, "router_logits", bad.router_logits)

    # gate and up projections swapped
    monkeypatch.setattr(O, "expert_ffn", lambda h, Wg, Wu, Wd: (O.silu(h @ np.asarray(Wu).T) *
                                                                (h @ np.asarray(Wg).T)) @ np.asarray(Wd).T)
    assert fails(test_single_expert_is_dense_swiglu_mlp)
    monkeypatch.setattr(O, "expert_ffn", bad.expert_ffn)

    # predictor left on during replay
    def replay_with_predictor(h, W_r, beta, idx, renorm=True):
        rng = np.random.default_rng(0)
        p = O.router_logits(h, W_r, beta) + 0.5 * rng.standard_normal((np.asarray(h).shape[0],
                                                                       np.asarray(W_r).shape[1]))
        return O.gates_on_route(p, idx, renorm), p
    monkeypatch.setattr(O, "replay_gates", replay_with_predictor)
    assert fails(test_replay_bypasses_predictor)
    monkeypatch.setattr(O, "replay_gates", bad.replay_gates)

    # renormalisation forgotten
    monkeypatch.setattr(O, "gates_on_route", lambda z, idx, renorm=True: bad.gates_on_route(z, idx, False))
    assert fails(test_renormalised_gates_sum_to_one_and_shift_invariant)
    monkeypatch.setattr(O, "gates_on_route", bad.gates_on_route)

    # a sign error in the SwiGLU derivative
    def bad_backward(*a, **kw):
        out = bad.replay_backward(*a, **kw)
        out["dW_gate"] = -out["dW_gate"]
        return out
    monkeypatch.setattr(O, "replay_backward", bad_backward)
    assert fails(lambda: test_backward_matches_central_differences(True))
    monkeypatch.setattr(O, "replay_backward", bad.replay_backward)

    # route KL taken in the reverse direction
    monkeypatch.setattr(O, "route_kl", lambda p, z: bad.route_kl(z, p))
    assert fails(test_route_kl_closed_forms)
    monkeypatch.setattr(O, "route_kl", bad.route_kl)

    # stratum draw off by one (position may land in the next stratum)
    monkeypatch.setattr(O, "feature_cache_positions", lambda T, Tc, seed: np.minimum(
        bad.feature_cache_positions(T, Tc, seed) + 1, T - 1))
    assert fails(test_feature_cache_positions_stratified_uniform)
    monkeypatch.setattr(O, "feature_cache_positions", bad.feature_cache_positions)

    # delta-matching target without the old logits subtracted
    monkeypatch.setattr(O, "delta_matching_kl", lambda p_cur, h_old, p_old, A, B:
                        bad.delta_matching_kl(p_cur, h_old, 0 * p_old, A, B))
    assert fails(test_delta_matching_kl_closed_forms_and_gradients)
    monkeypatch.setattr(O, "delta_matching_kl", bad.delta_matching_kl)
