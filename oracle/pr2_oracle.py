"""Plain float64 CPU oracle of the Pr^2 MoE-layer hot path.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
load this module: only the test suite, the package smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code with the HIP
library.

Everything here is the plain definition written out in numpy float64 from
the exact input values (bf16 inputs upcast exactly), with no blocking,
fusion or permutation beyond what the definitions state.  Citations name
the paper's sections, equations and algorithms:

* router logits   p = h W                      (Sec. 4.1, route prediction)
* predictor bias  b = h W_p,  W_p = A B         (Sec. 4.1; rank-r factor)
* predictive dist rho_hat = Softmax(p + b)      (Eq. pr2_predict)
* predicted route I_hat = TopK(rho_hat, k)      (Eq. pr2_route)
* rollout output  sum_{j in I_hat} rho_hat_j E_j(h)   (Eq. pr2_old_output)
* replay          rho = Softmax(h W), o = sum_{j in I_hat} rho_j E_j(h),
                  predictor bypassed           (Sec. 4.1 replay, Eq. pr2_output)
* predictive loss KL(<rho> || rho_hat)          (Sec. 4.2, Eq. pr2_loss;
                  Alg. 3 in Appendix D)
* route metrics   agreement |I_hat ∩ I| / k, deviation k - |I_hat ∩ I|,
                  route KL                      (Sec. 5.4)
* feature cache   Tc positions by uniform sub-sampling (Appendix E.2)
* expert E_j      gated MLP: W_down (silu(W_gate h) * W_up h)
                                               (Appendix E.2, FFN-ratio paragraph)

Readings where the paper is silent (each is listed in the design notes):
* the router may carry a bias ``beta`` [N]; it belongs to the router, so it
  is added to p in both phases and is never seen by the predictor;
* TopK selects on the logits (softmax is strictly increasing, so the set is
  the same), ties go to the lower expert id, and the decision is taken on
  the logits rounded to fp32 -- the precision the paper gives router logits
  (Table 3 caption, FP32 router logits); ids are stored ascending;
* ``renorm=True`` (default) weights the k experts by the softmax restricted
  to them (gates sum to 1); ``renorm=False`` is the paper-literal weight
  rho_j taken from the softmax over all N experts;
* expert ids are 0-based.

Pins: every function here is checked by tests marked "not gpu" against
brute force, closed forms, library routines on special cases, the paper's
Lemma B.2, finite differences and the values printed in Table 3.
"""
from __future__ import annotations

import numpy as np

F64 = np.float64


def _f64(a):
    return None if a is None else np.asarray(a, dtype=F64)


# ---------------------------------------------------------------- routing --

def router_logits(h, W_r, beta=None):
    """p = h W (+ beta).  Sec. 4.1, route prediction: p_old = h_old W_old."""
    p = _f64(h) @ _f64(W_r)
    if beta is not None:
        p = p + _f64(beta)[None, :]
    return p


def predictor_bias(h, A, B):
    """b = h W_p with the predictor factored as W_p = A B (Sec. 4.1).

    ``B is None`` means the identity, i.e. a full-rank W_p = A (r == N)."""
    u = _f64(h) @ _f64(A)
    return u if B is None else u @ _f64(B)


def softmax(z):
    """Softmax over the last axis, max-shifted."""
    z = _f64(z)
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def topk_ids(z, k, decide_dtype=np.float32):
    """TopK of Eq. pr2_route on logits z [T, N]: the k largest entries, ties to
    the lower expert id, returned ascending by id as int64 [T, k].

    The comparison is made on z rounded to ``decide_dtype`` (fp32 by default);
    -0.0 and +0.0 compare equal, as numbers do."""
    zd = np.asarray(z).astype(decide_dtype).astype(F64)
    order = np.argsort(-zd, axis=-1, kind="stable")  # stable: equal keys keep id order
    return np.sort(order[:, :k], axis=-1)


def topk_margin(z, k):
    """Gap between the k-th and (k+1)-th largest logits, in float64; +inf if k == N."""
    z = _f64(z)
    if k >= z.shape[-1]:
        return np.full(z.shape[0], np.inf)
    s = -np.sort(-z, axis=-1)
    return s[:, k - 1] - s[:, k]


def gates_on_route(z, idx, renorm=True):
    """Expert weights of a route from logits z [T, N] and ids idx [T, k].

    renorm=True: rho_j / sum_{i in I} rho_i (gates sum to one).
    renorm=False: rho_j itself, rho = Softmax(z) over all N (Eq. pr2_old_output,
    Eq. pr2_output as printed)."""
    rho = softmax(z)
    g = np.take_along_axis(rho, np.asarray(idx, dtype=np.int64), axis=-1)
    if renorm:
        g = g / g.sum(axis=-1, keepdims=True)
    return g


def route_predict(h, W_r, beta, A, B, k, renorm=True):
    """Route prediction during rollout (Sec. 4.1; Alg. 1 rollout half; Alg. 2).

    Returns dict with the predicted ids ``idx`` [T, k] (ascending), their
    ``gate`` [T, k], the router logits ``p`` (feature-cache p_old), the
    predictive logits ``z`` = p + b and the top-k ``margin`` of z."""
    p = router_logits(h, W_r, beta)
    z = p if A is None else p + predictor_bias(h, A, B)
    idx = topk_ids(z, k)
    return {"idx": idx, "gate": gates_on_route(z, idx, renorm), "p": p, "z": z,
            "margin": topk_margin(z, k)}


def replay_gates(h, W_r, beta, idx, renorm=True):
    """Replay weights (Sec. 4.1 replay; Alg. 3): rho = Softmax(h W) from the
    current router with the predictor bypassed, restricted to the cached ids."""
    p = router_logits(h, W_r, beta)
    return gates_on_route(p, idx, renorm), p


# ---------------------------------------------------------------- experts --

def silu(a):
    return a / (1.0 + np.exp(-a))


def expert_ffn(h, Wg, Wu, Wd):
    """Gated-MLP expert E(h) = W_down (silu(W_gate h) * (W_up h)) on rows of h.

    Wg, Wu: [m, d]; Wd: [d, m] (output-by-input, as linear-layer weights)."""
    h = _f64(h)
    a = h @ _f64(Wg).T
    u = h @ _f64(Wu).T
    return (silu(a) * u) @ _f64(Wd).T


def moe_combine(h, idx, gate, W_gate, W_up, W_down):
    """o_t = sum_{j in I_t} g_{t,j} E_j(h_t)  (Eq. pr2_output / pr2_old_output).

    Computed expert by expert through a boolean mask over tokens: for each
    expert, the rows routed to it go through a dense float64 expert FFN and
    are added into the output with their weights."""
    h = _f64(h)
    idx = np.asarray(idx, dtype=np.int64)
    gate = _f64(gate)
    T, _ = h.shape
    d_out = np.asarray(W_down).shape[1]
    y = np.zeros((T, d_out))
    for e in np.unique(idx):
        hit = idx == e                      # [T, k]
        rows = np.nonzero(hit.any(axis=1))[0]
        w = (gate * hit).sum(axis=1)[rows]  # an expert appears at most once per row
        y[rows] += w[:, None] * expert_ffn(h[rows], W_gate[e], W_up[e], W_down[e])
    return y


def replay_forward(h, idx, W_r, beta, W_gate, W_up, W_down, renorm=True):
    """Training-phase replay forward (Sec. 4.1 replay; Eq. pr2_output; Alg. 3).

    Returns (y [T, d], gate [T, k])."""
    g, _ = replay_gates(h, W_r, beta, idx, renorm)
    return moe_combine(h, idx, g, W_gate, W_up, W_down), g


def rollout_forward(h, W_r, beta, A, B, k, W_gate, W_up, W_down, renorm=True):
    """Route-recording output o_old with predictive weights (Eq. pr2_old_output;
    Alg. 2).  Returns (y, route dict)."""
    rt = route_predict(h, W_r, beta, A, B, k, renorm)
    return moe_combine(h, rt["idx"], rt["gate"], W_gate, W_up, W_down), rt


def replay_forward_rows(rows, h_rows, idx_rows, W_r, beta, W_gate, W_up, W_down,
                        renorm=True):
    """Replay forward for selected tokens only (their rows of h and of the
    recorded ids): the same masked per-expert combine restricted to them, so
    each expert's weights are read once however many tokens are sampled."""
    del rows
    g, _ = replay_gates(h_rows, W_r, beta, idx_rows, renorm)
    return moe_combine(h_rows, idx_rows, g, W_gate, W_up, W_down), g


# --------------------------------------------------------------- backward --

def replay_backward(h, idx, W_r, beta, W_gate, W_up, W_down, dy, renorm=True):
    """Gradients of L = <dy, y> for the replay forward with the recorded ids
    held fixed (Sec. 4.1: gradients flow through the current router's weights
    on the cached index and through the current experts; the predictor is
    bypassed, so it receives none).

    Returns dict dx [T,d], dW_r [d,N], dbeta [N], dW_gate, dW_up [N,m,d],
    dW_down [N,d,m]."""
    h = _f64(h)
    dy = _f64(dy)
    idx = np.asarray(idx, dtype=np.int64)
    T, d = h.shape
    N = np.asarray(W_r).shape[1]
    p = router_logits(h, W_r, beta)
    rho = softmax(p)
    g = gates_on_route(p, idx, renorm)

    dx = np.zeros_like(h)
    dWg = np.zeros(np.asarray(W_gate).shape)
    dWu = np.zeros(np.asarray(W_up).shape)
    dWd = np.zeros(np.asarray(W_down).shape)
    dg = np.zeros(idx.shape)
    for e in np.unique(idx):
        hit = idx == e
        rows, slots = np.nonzero(hit)
        Wg, Wu, Wd = _f64(W_gate[e]), _f64(W_up[e]), _f64(W_down[e])
        X = h[rows]
        a = X @ Wg.T
        u = X @ Wu.T
        sig = 1.0 / (1.0 + np.exp(-a))
        s = a * sig                       # silu(a)
        H = s * u
        E = H @ Wd.T                      # expert output before weighting
        dg[rows, slots] = (dy[rows] * E).sum(axis=1)
        dE = g[rows, slots][:, None] * dy[rows]
        dWd[e] = dE.T @ H
        dH = dE @ Wd
        du = dH * s
        ds = dH * u
        da = ds * sig * (1.0 + a * (1.0 - sig))   # d silu / da
        dWg[e] = da.T @ X
        dWu[e] = du.T @ X
        np.add.at(dx, rows, da @ Wg + du @ Wu)

    dp = np.zeros((T, N))
    if renorm:
        # g = softmax restricted to the route: dp_j = g_j (dg_j - sum_i g_i dg_i) on the route
        inner = (g * dg).sum(axis=1, keepdims=True)
        np.put_along_axis(dp, idx, g * (dg - inner), axis=1)
    else:
        # g_j = rho_j, rho = softmax over all N: dp_i = rho_i ([i in I] dg_i - sum_j rho_j dg_j)
        full = np.zeros((T, N))
        np.put_along_axis(full, idx, dg, axis=1)
        inner = (rho * full).sum(axis=1, keepdims=True)
        dp = rho * (full - inner)
    dW_r = h.T @ dp
    dbeta = dp.sum(axis=0)
    dx += dp @ _f64(W_r).T
    return {"dx": dx, "dW_r": dW_r, "dbeta": dbeta, "dW_gate": dWg, "dW_up": dWu,
            "dW_down": dWd, "dgate": dg, "gate": g}


# ------------------------------------------------------- predictor loss ----

def predictive_kl(p_cur, h_old, p_old, A, B):
    """Per-token KL(<rho> || rho_hat) of Eq. pr2_loss (Sec. 4.2; Alg. 3), with
    rho = Softmax(p_cur) under stop-gradient and
    rho_hat = Softmax(p_old + h_old A B) rebuilt from the feature cache.

    B = None means the identity (a full-rank predictor W_p = A, r = N).
    Returns (kl [T], dA, dB) where dA, dB are gradients of mean_t kl (dB is
    None for the identity)."""
    u = _f64(h_old) @ _f64(A)
    zhat = _f64(p_old) + (u if B is None else u @ _f64(B))
    return _kl_and_grads(softmax(p_cur), zhat, u, h_old, B)


def delta_matching_kl(p_cur, h_old, p_old, A, B):
    """The delta-matching alternative of the predictive loss (Appendix G,
    predictive-objective ablation): per-token
    KL(Softmax(<p_cur - p_old>) || Softmax(h_old W_p)), W_p = A B (B = None:
    identity).  Returns (kl [T], dA, dB) like predictive_kl."""
    u = _f64(h_old) @ _f64(A)
    b = u if B is None else u @ _f64(B)
    return _kl_and_grads(softmax(_f64(p_cur) - _f64(p_old)), b, u, h_old, B)


def _kl_and_grads(target, zhat, u, h_old, B):
    """KL(target || Softmax(zhat)) per token and the gradients of its mean
    through zhat = const + u B, u = h_old A."""
    rho_hat = softmax(zhat)
    log_t = np.log(np.where(target > 0, target, 1.0))
    log_rho_hat = zhat - zhat.max(axis=1, keepdims=True)
    log_rho_hat = log_rho_hat - np.log(np.exp(log_rho_hat).sum(axis=1, keepdims=True))
    kl = (target * (log_t - log_rho_hat)).sum(axis=1)
    T = zhat.shape[0]
    dz = (rho_hat - target) / T       # d mean KL / d zhat
    if B is None:
        return kl, _f64(h_old).T @ dz, None
    dB = u.T @ dz
    dA = _f64(h_old).T @ (dz @ _f64(B).T)
    return kl, dA, dB


# ------------------------------------------------------ route diagnostics --

def route_overlap(idx_cached, idx_current):
    """|I_hat ∩ I| per token: how many recorded ids the current top-k also
    picks (Sec. 5.4, top-k agreement and routing deviation)."""
    a = np.asarray(idx_cached)
    b = np.asarray(idx_current)
    return np.array([len(set(a[t].tolist()) & set(b[t].tolist())) for t in range(a.shape[0])],
                    dtype=np.int64)


def route_agreement(idx_cached, idx_current):
    """|I_hat ∩ I| / k per token (the agreement metric of Sec. 5.4)."""
    k = np.asarray(idx_cached).shape[1]
    return route_overlap(idx_cached, idx_current) / k


def route_deviation_histogram(idx_cached, idx_current):
    """Counts of the deviation k - |I_hat ∩ I| over tokens, for deviations
    0..k (the routing deviation distribution of Sec. 5.4)."""
    k = np.asarray(idx_cached).shape[1]
    dev = k - route_overlap(idx_cached, idx_current)
    return np.bincount(dev, minlength=k + 1)


def route_kl(p_cur, z_ref):
    """Per-token KL(Softmax(p_cur) || Softmax(z_ref)): the route KL between the
    current router's distribution and a reference distribution given by its
    logits (Sec. 5.4; with z_ref = p_old + h_old W_p it is the summand of
    Eq. pr2_loss)."""
    rho = softmax(p_cur)
    zc = _f64(p_cur) - _f64(p_cur).max(axis=1, keepdims=True)
    log_rho = zc - np.log(np.exp(zc).sum(axis=1, keepdims=True))
    zr = _f64(z_ref) - _f64(z_ref).max(axis=1, keepdims=True)
    log_ref = zr - np.log(np.exp(zr).sum(axis=1, keepdims=True))
    return (rho * (log_rho - log_ref)).sum(axis=1)


# -------------------------------------------------------- feature cache ----

_GOLDEN = 0x9E3779B97F4A7C15
_M64 = (1 << 64) - 1


def splitmix64(state):
    """The SplitMix64 output function of Steele, Lea and Flood (OOPSLA 2014)
    applied to a 64-bit state: the counter-based generator both sides use to
    draw feature-cache positions."""
    z = state & _M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M64
    return z ^ (z >> 31)


def feature_cache_positions(T, Tc, seed):
    """Positions retained by a feature cache of length Tc over a rollout of T
    tokens, drawn by uniform sub-sampling along the rollout (Appendix E.2,
    feature-cache paragraph): the rollout is cut into Tc strata of (nearly)
    equal length and one position is drawn uniformly inside stratum i with
    the i-th SplitMix64 output for the seed.  Tc >= T keeps every position."""
    if Tc >= T:
        return np.arange(T, dtype=np.int64)
    pos = np.empty(Tc, dtype=np.int64)
    for i in range(Tc):
        lo = (i * T) // Tc
        hi = ((i + 1) * T) // Tc
        r = splitmix64(seed + (i + 1) * _GOLDEN)
        pos[i] = lo + r % (hi - lo)
    return pos
