"""GPU parity of pr2_route_predict against the float64 oracle (Sec. 4.1,
Eq. pr2_predict / pr2_route): ids bit-exact outside the 1e-6 margin rule,
gates within 1e-5 relative, router logits (feature-cache p_old) within fp32
rounding, on seeded inputs from tiny to the full Qwen3-30B-A3B-shaped layer."""
import numpy as np
import pytest

from oracle import pr2_oracle as O
import workloads as W
from tests.parity import compare_route, to_dev

pytestmark = pytest.mark.gpu


def torch_mod():
    import torch
    return torch


def run_route(L, shape, k, renorm=True, idx_dtype="int32", ldi_pad=0, predictor=True,
              full_rank=False, logits=False):
    torch = torch_mod()
    from paper_2606_00395_amd import binding as B
    x = to_dev(L["x"], shape.act)
    Wr = to_dev(L["W_r"])
    br = to_dev(L["beta"]) if L["beta"] is not None else None
    A = to_dev(L["A"]) if predictor else None
    Bm = None if (full_rank or not predictor) else to_dev(L["B"])
    T = L["x"].shape[0]
    dt = torch.int16 if idx_dtype == "int16" else torch.int32
    buf = torch.full((T, k + ldi_pad), -7, dtype=dt, device="cuda")
    idx = buf[:, :k]
    gate = torch.empty((T, k), dtype=torch.float32, device="cuda")
    lg = torch.empty((T, L["W_r"].shape[1]), dtype=torch.float32, device="cuda") if logits else None
    B.route_predict(x, Wr, br, A, Bm, k, idx, gate, lg, renorm=renorm)
    torch.cuda.synchronize()
    out = {"idx": idx.cpu().numpy(), "gate": gate.cpu().numpy(), "buf": buf.cpu().numpy()}
    if logits:
        out["logits"] = lg.cpu().numpy()
    return out


def oracle_route(L, k, renorm=True, predictor=True, full_rank=False):
    A = L["A"] if predictor else None
    Bm = None if (full_rank or not predictor) else L["B"]
    return O.route_predict(L["x"], L["W_r"], L["beta"], A, Bm, k, renorm)


def test_route_tiny_fp32():
    s = W.WORKLOADS["tiny_fp32_T256"]
    L = W.layer_inputs(s, 0, experts=False)
    g = run_route(L, s, s.k, logits=True)
    ref = oracle_route(L, s.k)
    assert compare_route(g["idx"], g["gate"], ref, s.k, "tiny") == 0
    np.testing.assert_allclose(g["logits"], ref["p"], rtol=0, atol=1e-6)


CASES = [
    # (T, d, N, k, r, act, skew, idx_dtype, ldi_pad, renorm, full_rank)
    (1000, 256, 16, 4, 8, "bf16", "hot8", "int32", 0, True, False),
    (777, 200, 60, 6, 5, "bf16", "zipf", "int16", 3, True, False),
    (513, 64, 128, 8, 16, "f32", "none", "int32", 8, False, False),
    (300, 128, 256, 16, 0, "bf16", "hot8", "int32", 0, True, False),
    (129, 96, 1024, 8, 32, "bf16", "zipf", "int16", 0, True, False),
    (64, 128, 32, 32, 4, "f32", "none", "int32", 0, True, False),       # k = N
    (250, 64, 1, 1, 0, "f32", "none", "int32", 0, True, False),         # N = 1
    (200, 64, 64, 2, 64, "bf16", "none", "int32", 0, True, True),       # full-rank W_p = A
    (33, 1024, 128, 8, 256, "bf16", "hot8", "int32", 0, False, False),  # NC > 256, literal
    (40, 64, 512, 256, 4, "bf16", "none", "int32", 0, True, False),     # k = 256 (maximum)
    (17, 128, 1024, 256, 0, "f32", "none", "int16", 0, True, False),    # N = 1024, k = 256
]


@pytest.mark.parametrize("case", CASES, ids=[f"T{c[0]}_d{c[1]}_N{c[2]}_k{c[3]}_r{c[4]}_{c[5]}"
                                              for c in CASES])
def test_route_shapes(case):
    T, d, N, k, r, act, skew, idt, pad, renorm, full = case
    s = W.LayerShape("case", T=T, d=d, N=N, k=k, m=8, r=r, act=act, skew=skew)
    L = W.layer_inputs(s, 3, experts=False)
    ref = oracle_route(L, k, renorm=renorm, predictor=r > 0, full_rank=full)
    # with router logits requested the projection is [W_r | A]; without, the predictor is
    # folded into the router weights first: both must meet the same bar
    for want_logits in (True, False):
        g = run_route(L, s, k, renorm=renorm, idx_dtype=idt, ldi_pad=pad, predictor=r > 0,
                      full_rank=full, logits=want_logits)
        compare_route(g["idx"], g["gate"], ref, k, f"{case} logits={want_logits}")
        if pad:
            assert np.all(g["buf"][:, k:] == -7), "padding beyond k was written"
        if want_logits:
            np.testing.assert_allclose(g["logits"], ref["p"], rtol=0,
                                       atol=2e-6 * max(1.0, np.abs(ref["p"]).max()))


def test_route_exact_ties_go_to_lower_id():
    """One-hot router inputs make every logit an exact small integer, so ties
    are exact and the lower id must win (no margin exclusion)."""
    rng = np.random.default_rng(21)
    T, d, N, k = 512, 64, 16, 5
    x = np.zeros((T, d), dtype=np.float32)
    x[np.arange(T), np.arange(T) % d] = 1.0
    Wr = rng.integers(-2, 3, size=(d, N)).astype(np.float32)
    L = {"x": x, "W_r": Wr, "beta": None, "A": None, "B": None}
    s = W.LayerShape("ties", T=T, d=d, N=N, k=k, m=8, r=0, act="bf16")
    g = run_route(L, s, k, predictor=False)
    ref = O.route_predict(x, Wr, None, None, None, k)
    np.testing.assert_array_equal(g["idx"], ref["idx"])
    np.testing.assert_allclose(g["gate"], ref["gate"], rtol=1e-6)
    # signed zeros tie too
    x2 = np.zeros((2, d), dtype=np.float32)
    x2[:, 0] = [1.0, -1.0]
    Wz = np.zeros((d, N), dtype=np.float32)   # logits are +0.0 and -0.0
    L2 = {"x": x2, "W_r": Wz, "beta": None, "A": None, "B": None}
    g2 = run_route(L2, s.with_(T=2), k, predictor=False)
    np.testing.assert_array_equal(g2["idx"], np.tile(np.arange(k), (2, 1)))


def test_route_zero_predictor_equals_router_only():
    s = W.LayerShape("zp", T=700, d=256, N=64, k=6, m=8, r=8, act="bf16", skew="hot8")
    L = W.layer_inputs(s, 5, experts=False)
    L0 = dict(L, A=np.zeros_like(L["A"]))
    g0 = run_route(L0, s, s.k)
    gn = run_route(L, s.with_(r=0), s.k, predictor=False)
    np.testing.assert_array_equal(g0["idx"], gn["idx"])
    np.testing.assert_array_equal(g0["gate"], gn["gate"])


def test_route_qwen3_30b_full():
    s = W.WORKLOADS["qwen3_30b_T16384"]
    L = W.layer_inputs(s, 0, experts=False)
    ref = oracle_route(L, s.k)
    g = run_route(L, s, s.k, logits=True)
    excl = compare_route(g["idx"], g["gate"], ref, s.k, s.name + " with logits")
    print(f"\n{s.name}: {excl} of {s.T} tokens under the 1e-6 margin")
    np.testing.assert_allclose(g["logits"], ref["p"], rtol=0, atol=4e-6)
    # the folded projection (no logits requested), twice: parity and bitwise determinism
    g1 = run_route(L, s, s.k)
    compare_route(g1["idx"], g1["gate"], ref, s.k, s.name + " folded")
    g2 = run_route(L, s, s.k)
    np.testing.assert_array_equal(g1["idx"], g2["idx"])
    np.testing.assert_array_equal(g1["gate"], g2["gate"])


def test_route_empty_batch():
    torch = torch_mod()
    from paper_2606_00395_amd import binding as B
    x = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    Wr = torch.zeros((64, 8), device="cuda")
    idx = torch.empty((0, 2), dtype=torch.int32, device="cuda")
    B.route_predict(x, Wr, None, None, None, 2, idx)


def test_route_is_batch_invariant():
    """A token's logits, route and weights do not depend on the batch it is
    routed in: batches small enough for the split-K path (2048, 1000, 256 and
    a single token) give bitwise the results of the same tokens inside a
    4096-token batch, which takes the fused path, in the
    rollout (with and without logits, i.e. with the predictor as separate
    columns or folded into the router weights) and in the replay router
    (current top-k and route KL of the diagnostics)."""
    torch = torch_mod()
    from paper_2606_00395_amd import binding as B
    s = W.WORKLOADS["qwen3_30b_T16384"].with_(T=4096)
    L = W.layer_inputs(s, 7, experts=False)
    for T_small in (2048, 256, 1000, 1):
        Ls = {n: (v[:T_small] if n == "x" else v) for n, v in L.items()}
        for want_logits in (True, False):
            big = run_route(L, s, s.k, logits=want_logits)
            small = run_route(Ls, s.with_(T=T_small), s.k, logits=want_logits)
            for n in ("idx", "gate") + (("logits",) if want_logits else ()):
                np.testing.assert_array_equal(small[n], big[n][:T_small],
                                              err_msg=f"T={T_small} {n} logits={want_logits}")
        # the replay router: current top-k and route KL against given reference logits
        x = to_dev(L["x"], s.act)
        Wr, br = to_dev(L["W_r"]), to_dev(L["beta"])
        idx = torch.from_numpy(big["idx"]).to("cuda")
        zref = torch.from_numpy(np.ascontiguousarray(O.router_logits(L["x"], L["W_r"], L["beta"]),
                                                     dtype=np.float32)).to("cuda")
        outs = []
        for T in (s.T, T_small):
            cur = torch.empty((T, s.k), dtype=torch.int32, device="cuda")
            kl = torch.empty((T,), dtype=torch.float32, device="cuda")
            B.route_diagnostics(x[:T], idx[:T], Wr, br, zref[:T], cur_idx_out=cur, kl_out=kl)
            torch.cuda.synchronize()
            outs.append((cur.cpu().numpy(), kl.cpu().numpy()))
        np.testing.assert_array_equal(outs[1][0], outs[0][0][:T_small])
        np.testing.assert_array_equal(outs[1][1], outs[0][1][:T_small])


@pytest.mark.parametrize("logits,act", [(False, "bf16"), (True, "bf16"), (False, "f32")],
                         ids=["folded", "with_logits", "fp32_vector_path"])
def test_route_reuse_split_matches_fresh_calls(logits, act):
    """Decode-style steps: the first call splits the weights, the later ones
    (pr2_route_predict_reuse) read that split.  Every step's ids, gates (and
    logits) equal those of a fresh pr2_route_predict on the same tokens, bit
    for bit, and the ids match the oracle's; covers both split layouts (the
    predictor folded into the weights, and kept apart when logits are wanted),
    a batch size that changes between steps, and fp32 activations (the fp64
    vector path, which keeps no split)."""
    torch = torch_mod()
    from paper_2606_00395_amd import binding as B
    s = W.LayerShape("reuse", T=384, d=512, N=64, k=4, m=8, r=16, act=act, skew="hot8")
    L = W.layer_inputs(s, 21, experts=False)
    Wr, br, A, Bm = to_dev(L["W_r"]), to_dev(L["beta"]), to_dev(L["A"]), to_dev(L["B"])
    x_all = to_dev(L["x"], s.act)
    ws = B.route_workspace(x_all, Wr, A, s.k)
    steps = [(0, 256), (256, 384), (0, 100), (100, 356)]   # token ranges of four steps
    for n, (a, b) in enumerate(steps):
        T = b - a
        outs = []
        for reuse in (n > 0, False):
            idx = torch.full((T, s.k), -1, dtype=torch.int32, device="cuda")
            gate = torch.empty((T, s.k), dtype=torch.float32, device="cuda")
            lg = torch.empty((T, s.N), dtype=torch.float32, device="cuda") if logits else None
            if reuse or n == 0:
                B.route_predict(x_all[a:b], Wr, br, A, Bm, s.k, idx, gate, lg, ws=ws,
                                reuse_split=reuse)
            else:
                B.route_predict(x_all[a:b], Wr, br, A, Bm, s.k, idx, gate, lg)   # own workspace
            torch.cuda.synchronize()
            outs.append((idx.cpu(), gate.cpu(), None if lg is None else lg.cpu()))
        (i0, g0, l0), (i1, g1, l1) = outs
        assert torch.equal(i0, i1) and torch.equal(g0, g1), f"step {n}"
        if logits:
            assert torch.equal(l0, l1), f"step {n} logits"
        Ls = dict(L, x=L["x"][a:b])
        ref = oracle_route(Ls, s.k)
        assert compare_route(i0.numpy(), g0.numpy(), ref, s.k, f"reuse step {n}") == 0


def test_reuse_checks_the_recorded_split():
    """pr2_route_predict_reuse reads the split a route call formed in the same
    workspace and refuses one formed from other weights, in the other layout, or
    dropped by another call that used the workspace."""
    torch = torch_mod()
    from paper_2606_00395_amd import binding as B
    s = W.LayerShape("reuse", T=300, d=256, N=16, k=4, m=128, r=4, act="bf16", skew="hot8")
    L = W.layer_inputs(s, 4)
    x = to_dev(L["x"], "bf16")
    Wr, br, A, Bm = (to_dev(L[n]) for n in ("W_r", "beta", "A", "B"))
    rw = B.workspace_bytes(B.make_desc(s.T, s.d, s.N, s.k, s.m, s.r), B.OP_ROUTE)
    fw = B.workspace_bytes(B.make_desc(s.T, s.d, s.N, s.k, s.m, 0), B.OP_REPLAY_FWD)
    ws = torch.empty(max(rw, fw), dtype=torch.uint8, device="cuda")
    idx = torch.empty((s.T, s.k), dtype=torch.int32, device="cuda")
    idx2 = torch.empty_like(idx)
    B.route_predict(x, Wr, br, A, Bm, s.k, idx, ws=ws)
    B.route_predict(x, Wr, br, A, Bm, s.k, idx2, ws=ws, reuse_split=True)
    torch.cuda.synchronize()
    assert torch.equal(idx, idx2)
    ref = oracle_route(L, s.k)
    compare_route(idx2.cpu().numpy(), None, ref, s.k, "reuse")
    for kw in (dict(W=Wr.clone()), dict(A=A.clone()), dict(Bm=Bm.clone()),
               dict(logits=torch.empty((s.T, s.N), device="cuda"))):
        with pytest.raises(B.Pr2Error) as ei:
            B.route_predict(x, kw.get("W", Wr), br, kw.get("A", A), kw.get("Bm", Bm), s.k, idx2,
                            logits_out=kw.get("logits"), ws=ws, reuse_split=True)
        assert ei.value.status == 5, str(ei.value)
    # a replay forward writes its own scratch into the workspace: the split is gone
    y = torch.empty_like(x)
    B.moe_replay_forward(x, idx, Wr, br, to_dev(L["W_gate"], "bf16"), to_dev(L["W_up"], "bf16"),
                         to_dev(L["W_down"], "bf16"), y, ws=ws)
    with pytest.raises(B.Pr2Error) as ei:
        B.route_predict(x, Wr, br, A, Bm, s.k, idx2, ws=ws, reuse_split=True)
    assert ei.value.status == 5
    # forming it again makes the reuse valid again
    B.route_predict(x, Wr, br, A, Bm, s.k, idx2, ws=ws)
    B.route_predict(x, Wr, br, A, Bm, s.k, idx2, ws=ws, reuse_split=True)
    torch.cuda.synchronize()
    assert torch.equal(idx, idx2)
