"""Algorithmic cost model of the Pr^2 MoE-layer hot path.

Two parts:

* the paper's own overhead formulas (Appendix E.2, Table 3 and its caption):
  index cache 4*T*L*k bytes per response (int32 ids), feature cache
  T_c*L*(2d + 4N) bytes per response (bf16 hidden features, fp32 router
  logits), predictor projection 2*L*d*N extra FLOPs per token, and the FFN
  ratio 2*L*d*N / (6*L*(k+s)*d*m);
* the per-kernel algorithmic FLOPs and minimum HBM bytes of this library's
  kernels, used to express measured times as a fraction of the MI355X roofline.

All byte counts are algorithmic (each input read once, each output written
once); they are not counter readings.
"""
from __future__ import annotations

# MI355X published peaks
PEAK_BF16_FLOPS = 2.5e15        # dense bf16 MFMA
PEAK_FP32_FLOPS = 157.3e12      # fp32 vector / matrix
PEAK_HBM_BYTES = 8.0e12         # HBM3E


# ------------------------------------------------ paper, Table 3 formulas ---

def index_cache_bytes(T, L, k, id_bytes=4):
    """Replay-index cache per response: id_bytes * T * L * k (int32: 4TLk)."""
    return id_bytes * T * L * k


def feature_cache_bytes(Tc, L, d, N):
    """Feature cache per response: T_c * L * (2d + 4N) (bf16 h_old, fp32 p_old)."""
    return Tc * L * (2 * d + 4 * N)


def predictor_flops_per_token(L, d, N):
    """Extra route-recording FLOPs per generated token from a full-rank predictor."""
    return 2 * L * d * N


def ffn_ratio(L, d, N, k, s, m):
    """Predictor FLOPs over active-expert FLOPs, 2LdN / (6L(k+s)dm)."""
    return (2 * L * d * N) / (6 * L * (k + s) * d * m)


# ------------------------------------------------- this library's kernels ---

def route_flops(T, d, N, r):
    """Router + rank-r predictor projection: 2*T*d*(N + r) + 2*T*r*N."""
    return 2 * T * d * (N + r) + 2 * T * r * N


def route_bytes(T, d, N, r, k, act_bytes=2, id_bytes=4, logits=False):
    """x read once, W_r/A/B/beta read once, ids and gates written once."""
    b = T * d * act_bytes + 4 * (d * N + d * r + r * N + N) + T * k * (id_bytes + 4)
    if logits:
        b += 4 * T * N
    return b


def replay_gate_bytes(T, d, N, k, act_bytes=2, id_bytes=4):
    return T * d * act_bytes + 4 * (d * N + N) + T * k * (id_bytes + 4)


def expert_flops(T, d, k, m):
    """gate+up and down projections of every routed (token, expert) pair: 6*T*k*d*m."""
    return 6 * T * k * d * m


def gemm1_flops(T, d, k, m):
    return 4 * T * k * d * m


def gemm2_flops(T, d, k, m):
    return 2 * T * k * d * m


def combine_bytes(T, d, k, o_bytes=2, act_bytes=2):
    """Combine reads the k weighted expert outputs of every token and writes y."""
    return T * k * d * o_bytes + T * d * act_bytes + T * k * 4


def replay_forward_min_bytes(T, d, N, k, m, act_bytes=2, id_bytes=4):
    """Whole replay forward, every tensor touched once: weights, x, y, ids, gates."""
    return (3 * N * m * d * act_bytes + 2 * T * d * act_bytes + 4 * (d * N + N)
            + T * k * (id_bytes + 4))
