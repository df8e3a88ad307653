"""Seeded synthetic inputs for one Pr^2 MoE layer.

This module is shared by the CPU oracle's tests and by the GPU path's tests
and benchmark.  It draws random numbers and rounds them to the storage
precision of each tensor; it holds none of the method's arithmetic (no router
logits, no softmax, no top-k, no expert math).

Every tensor comes from its own ``numpy.random.default_rng([seed, tag, ...])``
stream, so any tensor (or one expert's weights) can be regenerated alone and
in parallel.  Values are returned as float32 arrays; tensors whose storage
type is bf16 hold values that are exactly representable in bf16 (rounded to
nearest-even), so the GPU side converts them losslessly and the oracle
upcasts them exactly to float64.

Shapes follow the paper's Qwen3-30B-A3B layer (d=2048, N=128, k=8, m=768;
Table 3 in Appendix E.2) and a Qwen3-235B-A22B-shaped layer; the paper's
rollouts on math-reasoning prompts are replaced by these synthetic hidden
states, since neither the trained models nor the datasets are available.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace

import numpy as np

# stream tags: one per tensor kind
TAG_X, TAG_WR, TAG_A, TAG_B, TAG_WG, TAG_WU, TAG_WD, TAG_BETA, TAG_DY, TAG_FLIP, TAG_XSTEP = range(1, 12)

WEIGHT_STD = 0.02


@dataclass(frozen=True)
class LayerShape:
    """One MoE layer workload.

    T tokens, d hidden, N experts, k routed experts per token, m expert
    intermediate size, r predictor rank.  ``act`` is the storage type of the
    activations and expert weights ("f32" or "bf16"); the router W_r, the
    predictor factors A, B and the router bias are always fp32.
    ``skew`` selects the router-bias recipe: "none" (no bias), "hot8"
    (+1.0 on 8 random experts), "zipf" (a Zipf(1.1) prior over experts).
    """
    name: str
    T: int
    d: int
    N: int
    k: int
    m: int
    r: int
    act: str = "bf16"
    skew: str = "none"
    idx_dtype: str = "int32"
    flip_frac: float = 0.0

    def with_(self, **kw) -> "LayerShape":
        return replace(self, **kw)


WORKLOADS = {
    # tiny fp32 layer that the oracle finishes in well under a second
    "tiny_fp32_T256": LayerShape("tiny_fp32_T256", T=256, d=64, N=8, k=2, m=128, r=4,
                                 act="f32", skew="none"),
    # Qwen3-30B-A3B-shaped layer, rollout batch 8 x 2048 tokens
    "qwen3_30b_T16384": LayerShape("qwen3_30b_T16384", T=16384, d=2048, N=128, k=8, m=768,
                                   r=16, act="bf16", skew="hot8"),
    # the same layer in decode style: 256 sequences x 2048 positions, int16 route record,
    # replayed in micro-batches of 32768 tokens
    "qwen3_30b_decode_256x2048": LayerShape("qwen3_30b_decode_256x2048", T=32768, d=2048,
                                            N=128, k=8, m=768, r=16, act="bf16",
                                            skew="hot8", idx_dtype="int16"),
    # Qwen3-235B-A22B-shaped layer with Zipf(1.1) expert load
    "qwen3_235b_T32768": LayerShape("qwen3_235b_T32768", T=32768, d=4096, N=128, k=8,
                                    m=1536, r=32, act="bf16", skew="zipf"),
    # Qwen3-30B-A3B-shaped layer for the replay backward: 5% of routes differ from the
    # current router's top-8
    "qwen3_30b_bwd_T16384": LayerShape("qwen3_30b_bwd_T16384", T=16384, d=2048, N=128, k=8,
                                       m=768, r=16, act="bf16", skew="hot8", flip_frac=0.05),
}

DECODE_SEQS = 256
DECODE_STEPS = 2048
DECODE_MICROBATCH = 32768


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round a float32 array in place to the nearest bf16 value (ties to even)."""
    assert a.dtype == np.float32
    u = a.view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    u += bias
    u &= np.uint32(0xFFFF0000)
    return a


def _normal(seed_seq, shape, std, bf16, out=None):
    rng = np.random.default_rng(seed_seq)
    a = out if out is not None else np.empty(shape, dtype=np.float32)
    rng.standard_normal(out=a.reshape(-1), dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    if bf16:
        round_to_bf16(a.reshape(-1))
    return a


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def expert_weights(shape: LayerShape, seed: int, which: str, experts=None) -> np.ndarray:
    """W_gate / W_up ([N, m, d]) or W_down ([N, d, m]) for all or some experts."""
    tag = {"gate": TAG_WG, "up": TAG_WU, "down": TAG_WD}[which]
    per = (shape.m, shape.d) if which != "down" else (shape.d, shape.m)
    ids = list(range(shape.N)) if experts is None else list(experts)
    out = np.empty((len(ids),) + per, dtype=np.float32)
    bf16 = shape.act == "bf16"

    def fill(i):
        _normal([seed, tag, ids[i]], per, WEIGHT_STD, bf16, out=out[i])

    if len(ids) > 1:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(len(ids))))
    else:
        for i in range(len(ids)):
            fill(i)
    return out


def router_bias(shape: LayerShape, seed: int):
    """The router bias beta [N] (fp32) of the load-skew recipe, or None."""
    rng = np.random.default_rng([seed, TAG_BETA])
    if shape.skew == "none":
        return None
    beta = np.zeros(shape.N, dtype=np.float32)
    if shape.skew == "hot8":
        beta[rng.choice(shape.N, 8, replace=False)] = 1.0
    elif shape.skew == "zipf":
        rank = 1 + rng.permutation(shape.N)
        beta[:] = (-1.1 * np.log(rank.astype(np.float64))).astype(np.float32)
    else:
        raise ValueError(shape.skew)
    return beta


def hidden_states(shape: LayerShape, seed: int, rows=None) -> np.ndarray:
    """x [T, d] ~ N(0, 1), rounded to the activation storage type.

    Rows are drawn in blocks of 1024 tokens from their own streams, so a
    subset of rows can be regenerated without drawing the rest."""
    bf16 = shape.act == "bf16"
    blk = 1024
    nblk = (shape.T + blk - 1) // blk
    if rows is None:
        x = np.empty((shape.T, shape.d), dtype=np.float32)

        def fill(b):
            lo, hi = b * blk, min(shape.T, (b + 1) * blk)
            _normal([seed, TAG_X, b], (hi - lo, shape.d), 1.0, bf16, out=x[lo:hi])

        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(nblk)))
        return x
    rows = np.asarray(rows)
    out = np.empty((len(rows), shape.d), dtype=np.float32)
    for b in np.unique(rows // blk):
        lo, hi = b * blk, min(shape.T, (b + 1) * blk)
        xb = _normal([seed, TAG_X, int(b)], (hi - lo, shape.d), 1.0, bf16)
        sel = np.nonzero(rows // blk == b)[0]
        out[sel] = xb[rows[sel] - lo]
    return out


def decode_step_states(shape: LayerShape, seed: int, step: int) -> np.ndarray:
    """Hidden states of decode step ``step``: [DECODE_SEQS, d], one row per sequence."""
    return _normal([seed, TAG_XSTEP, step], (DECODE_SEQS, shape.d), 1.0, shape.act == "bf16")


def decode_all_states(shape: LayerShape, seed: int, steps: int = DECODE_STEPS) -> np.ndarray:
    """All decode hidden states laid out [seq, pos, d] (sequence-major, as replayed)."""
    out = np.empty((DECODE_SEQS, steps, shape.d), dtype=np.float32)

    def fill(s):
        out[:, s, :] = decode_step_states(shape, seed, s)

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(fill, range(steps)))
    return out


def upstream_grad(shape: LayerShape, seed: int) -> np.ndarray:
    """dy [T, d] ~ N(0, 1) for the backward workload."""
    return _normal([seed, TAG_DY], (shape.T, shape.d), 1.0, shape.act == "bf16")


def flip_tokens(shape: LayerShape, seed: int) -> np.ndarray:
    """Sorted token ids whose recorded route differs in one slot from the current top-k."""
    n = int(round(shape.flip_frac * shape.T))
    rng = np.random.default_rng([seed, TAG_FLIP])
    return np.sort(rng.choice(shape.T, n, replace=False))


def flip_route(ranked: np.ndarray, tokens: np.ndarray, k: int) -> np.ndarray:
    """The recorded route of the backward workload from a ranking computed elsewhere.

    ``ranked`` [T, k+1] holds each token's k+1 highest-ranked expert ids, best
    first.  Every token records its first k ids; each token in ``tokens`` records
    the (k+1)-th instead of the k-th (a one-slot difference from the current
    top-k).  Rows are returned sorted ascending, int64 [T, k].  Index work only."""
    ranked = np.asarray(ranked, dtype=np.int64)
    assert ranked.ndim == 2 and ranked.shape[1] == k + 1
    idx = ranked[:, :k].copy()
    idx[tokens, k - 1] = ranked[tokens, k]
    return np.sort(idx, axis=1)


def layer_inputs(shape: LayerShape, seed: int = 0, experts: bool = True) -> dict:
    """All inputs of one layer as float32 numpy arrays (beta may be None).

    Keys: x [T,d], W_r [d,N], A [d,r], B [r,N], beta [N] | None and, if
    ``experts``, W_gate [N,m,d], W_up [N,m,d], W_down [N,d,m]."""
    out = {
        "x": hidden_states(shape, seed),
        "W_r": _normal([seed, TAG_WR], (shape.d, shape.N), WEIGHT_STD, False),
        "A": _normal([seed, TAG_A], (shape.d, shape.r), WEIGHT_STD, False),
        "B": _normal([seed, TAG_B], (shape.r, shape.N), WEIGHT_STD, False),
        "beta": router_bias(shape, seed),
    }
    if experts:
        out["W_gate"] = expert_weights(shape, seed, "gate")
        out["W_up"] = expert_weights(shape, seed, "up")
        out["W_down"] = expert_weights(shape, seed, "down")
    return out
