"""GPU parity of pr2_moe_replay_forward against the float64 oracle (Sec. 4.1
replay, Eq. pr2_output; Alg. 3): gate recompute from the current router with
the predictor bypassed, permutation, grouped SwiGLU expert GEMMs and combine.

The recorded ids fed to both sides always come from the oracle's own route
(or from the seeded generator), never from the HIP path."""
import os

import numpy as np
import pytest

from oracle import pr2_oracle as O
import workloads as W
from tests.parity import compare_gates, compare_rows, to_dev

pytestmark = pytest.mark.gpu


def torch_mod():
    import torch
    return torch


def dev_layer(L, act):
    return {"x": to_dev(L["x"], act), "W_r": to_dev(L["W_r"]),
            "beta": to_dev(L["beta"]) if L["beta"] is not None else None,
            "W_gate": to_dev(L["W_gate"], act), "W_up": to_dev(L["W_up"], act),
            "W_down": to_dev(L["W_down"], act)}


def run_replay(D, idx_np, renorm=True, idx_dtype="int32", ldi_pad=0, ws=None, x=None):
    torch = torch_mod()
    from paper_2606_00395_amd import binding as B
    x = D["x"] if x is None else x
    T, d = x.shape
    k = idx_np.shape[1]
    dt = torch.int16 if idx_dtype == "int16" else torch.int32
    buf = torch.zeros((T, k + ldi_pad), dtype=dt, device="cuda")
    buf[:, :k] = torch.from_numpy(np.ascontiguousarray(idx_np)).to(dt)
    idx = buf[:, :k]
    y = torch.empty((T, d), dtype=x.dtype, device="cuda")
    gate = torch.empty((T, k), dtype=torch.float32, device="cuda")
    B.moe_replay_forward(x, idx, D["W_r"], D["beta"], D["W_gate"], D["W_up"], D["W_down"], y,
                         gate, ws=ws, renorm=renorm)
    torch.cuda.synchronize()
    return y.float().cpu().numpy(), gate.cpu().numpy()


def oracle_ids(L, k):
    """Rollout route of the oracle with the layer's predictor (the recorded ids)."""
    return O.route_predict(L["x"], L["W_r"], L["beta"], L["A"], L["B"], k)["idx"]


def test_replay_tiny_fp32():
    s = W.WORKLOADS["tiny_fp32_T256"]
    L = W.layer_inputs(s, 0)
    idx = oracle_ids(L, s.k)
    y, g = run_replay(dev_layer(L, s.act), idx)
    y_ref, g_ref = O.replay_forward(L["x"], idx, L["W_r"], L["beta"], L["W_gate"], L["W_up"],
                                    L["W_down"])
    compare_gates(g, g_ref, "tiny")
    compare_rows(y, y_ref, "f32", "tiny")


CASES = [
    # (T, d, N, k, m, act, skew, renorm, idx_dtype, ldi_pad, name)
    (1000, 256, 16, 4, 128, "bf16", "hot8", True, "int32", 0, "mfma_ragged"),
    (517, 512, 8, 2, 256, "bf16", "zipf", False, "int16", 5, "mfma_literal_i16"),
    (300, 96, 12, 3, 80, "bf16", "hot8", True, "int32", 0, "generic_bf16"),
    (200, 72, 6, 6, 40, "f32", "none", True, "int32", 2, "generic_f32_k_eq_N"),
    (130, 256, 1, 1, 128, "bf16", "none", True, "int32", 0, "single_expert"),
    (70, 256, 128, 8, 128, "bf16", "hot8", True, "int32", 0, "few_tokens_many_experts"),
    (40, 256, 512, 256, 128, "bf16", "none", True, "int32", 0, "k256_N512_max_route"),
    (33, 64, 1024, 96, 32, "f32", "zipf", False, "int16", 1, "N1024_literal_generic"),
    # m a multiple of 192: the gate/up GEMM with 384-row panels (one and two
    # panels per tile, ragged tiles)
    (1300, 256, 16, 4, 192, "bf16", "hot8", True, "int32", 0, "wide_panel_m192"),
    (900, 512, 8, 2, 384, "bf16", "zipf", False, "int16", 2, "wide_panel_m384"),
    (70, 256, 128, 8, 576, "bf16", "hot8", True, "int32", 0, "wide_panel_few_rows_per_expert"),
    # more than 32 tiles of 64 tokens: the replay-weight pass forms the
    # permutation's counts (k = 8, 16, 32, 64), ragged last tile
    (4100, 256, 64, 16, 128, "bf16", "zipf", True, "int16", 3, "fused_counts_k16"),
    (2113, 256, 64, 32, 128, "bf16", "hot8", False, "int32", 0, "fused_counts_k32"),
    (2177, 128, 128, 64, 128, "bf16", "none", True, "int32", 1, "fused_counts_k64"),
]


@pytest.mark.parametrize("case", CASES, ids=[c[-1] for c in CASES])
def test_replay_shapes(case):
    T, d, N, k, m, act, skew, renorm, idt, pad, name = case
    s = W.LayerShape(name, T=T, d=d, N=N, k=k, m=m, r=4, act=act, skew=skew)
    L = W.layer_inputs(s, 7)
    idx = oracle_ids(L, k)
    # replay accepts ids in any order within a row
    idx = idx[:, ::-1].copy()
    y, g = run_replay(dev_layer(L, act), idx, renorm=renorm, idx_dtype=idt, ldi_pad=pad)
    y_ref, g_ref = O.replay_forward(L["x"], idx, L["W_r"], L["beta"], L["W_gate"], L["W_up"],
                                    L["W_down"], renorm)
    compare_gates(g, g_ref, name)
    compare_rows(y, y_ref, act, name)


def test_replay_ids_differ_from_current_router():
    """Recorded ids chosen away from the current router's top-k (the replay
    case the method exists for): weights still come from the current router
    restricted to the recorded ids."""
    s = W.LayerShape("stale", T=600, d=256, N=32, k=4, m=128, r=4, act="bf16", skew="hot8")
    L = W.layer_inputs(s, 9)
    rng = np.random.default_rng(0)
    idx = np.sort(np.stack([rng.choice(s.N, s.k, replace=False) for _ in range(s.T)]), axis=1)
    y, g = run_replay(dev_layer(L, s.act), idx)
    y_ref, g_ref = O.replay_forward(L["x"], idx, L["W_r"], L["beta"], L["W_gate"], L["W_up"],
                                    L["W_down"])
    compare_gates(g, g_ref, "stale")
    compare_rows(y, y_ref, "bf16", "stale")


@pytest.fixture(scope="module")
def qwen30b():
    s = W.WORKLOADS["qwen3_30b_T16384"]
    L = W.layer_inputs(s, 0)
    idx = oracle_ids(L, s.k)
    return s, L, idx, dev_layer(L, s.act)


def test_replay_qwen3_30b_full(qwen30b):
    """Every token's replay weights and output row at the Qwen3-30B-A3B shape
    (16384 tokens, 131072 routes over 582 row tiles), per-row rule."""
    s, L, idx, D = qwen30b
    y, g = run_replay(D, idx)
    y_ref, g_ref = O.replay_forward(L["x"], idx, L["W_r"], L["beta"], L["W_gate"], L["W_up"],
                                    L["W_down"])
    compare_gates(g, g_ref, s.name)
    err = compare_rows(y, y_ref, "bf16", s.name)
    print(f"\n{s.name}: worst row rel err {err:.2e} over all {s.T} rows")
    # determinism
    y2, g2 = run_replay(D, idx)
    np.testing.assert_array_equal(y, y2)
    np.testing.assert_array_equal(g, g2)
    # the combine sums exactly k expert rows per token: no row of y is zero
    assert np.all(np.abs(y).sum(axis=1) > 0)


def test_replay_validate_flags_bad_routes(qwen30b):
    """PR2_VALIDATE=1 reports out-of-range and repeated ids (kernels skip
    out-of-range ids and keep every access in bounds)."""
    from paper_2606_00395_amd import binding as B
    s, L, idx, D = qwen30b
    n = 256
    bad = idx[:n].copy()
    bad[3, 2] = s.N + 5
    bad[7, 1] = -1
    dup = idx[:n].copy()
    dup[11, 1] = dup[11, 0]
    x = D["x"][:n]
    os.environ["PR2_VALIDATE"] = "1"
    try:
        run_replay(D, idx[:n], x=x)     # valid route passes
        for r, what in ((bad, "2 out-of-range and 0 repeated"),
                        (dup, "0 out-of-range and 1 repeated")):
            with pytest.raises(B.Pr2Error) as ei:
                run_replay(D, r, x=x)
            assert ei.value.status == 7 and what in str(ei.value), str(ei.value)
        # 4096 tokens: the counts (and the out-of-range count) come from the
        # replay-weight pass, which must count each bad id once
        n = 4096
        bad = idx[:n].copy()
        bad[3, 2] = s.N + 5
        bad[3000, 1] = -1
        bad[4095, 7] = 1 << 20
        with pytest.raises(B.Pr2Error) as ei:
            run_replay(D, bad, x=D["x"][:n])
        assert ei.value.status == 7 and "3 out-of-range and 0 repeated" in str(ei.value), \
            str(ei.value)
    finally:
        del os.environ["PR2_VALIDATE"]


def test_replay_qwen3_235b_full():
    """Every token at the Qwen3-235B-A22B shape (32768 tokens, d 4096, m 1536,
    Zipf(1.1) expert load), per-row rule."""
    s = W.WORKLOADS["qwen3_235b_T32768"]
    L = W.layer_inputs(s, 0)
    idx = oracle_ids(L, s.k)
    D = dev_layer(L, s.act)
    y, g = run_replay(D, idx)
    del D
    y_ref, g_ref = O.replay_forward(L["x"], idx, L["W_r"], L["beta"], L["W_gate"], L["W_up"],
                                    L["W_down"])
    compare_gates(g, g_ref, s.name)
    err = compare_rows(y, y_ref, "bf16", s.name)
    counts = np.bincount(idx.ravel(), minlength=s.N)
    print(f"\n{s.name}: worst row rel err {err:.2e} over all {s.T} rows; expert load "
          f"max/mean {counts.max() / counts.mean():.1f}, min {counts.min()}")
