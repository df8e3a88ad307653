"""Decode-style route recording and replay on the Qwen3-30B-A3B-shaped layer:
256 sequences x 2048 decode steps, each step's route written into one
index-stable int16 buffer [seq, pos, k] (Sec. 4.1: the predicted ids are
cached for replay; Alg. 2, caching step), then replayed in micro-batches of
16 whole sequences = 32768 tokens (Sec. 4.1 replay; Alg. 3).

Oracle checks: the routes of sampled steps against the float64 oracle (margin
rule); all 16 micro-batches (the whole 524288-route record) are replayed, and
in each the first and last rows and 32 random ones are checked against the
oracle's replay forward on the oracle's own route of those tokens (only where
it equals the recorded one)."""
import numpy as np
import pytest

from oracle import pr2_oracle as O
import workloads as W
from tests.parity import MARGIN_EPS, compare_rows, to_dev

pytestmark = pytest.mark.gpu


def test_decode_record_then_replay():
    import torch
    from paper_2606_00395_amd import binding as B

    s = W.WORKLOADS["qwen3_30b_decode_256x2048"]
    S, P, k = W.DECODE_SEQS, W.DECODE_STEPS, s.k
    L = W.layer_inputs(s.with_(T=S), 0)           # weights (x is drawn per step below)
    X = W.decode_all_states(s, 0)                 # [S, P, d] float32 (bf16 values)
    dev = torch.device("cuda", 0)
    Xd = torch.from_numpy(X).to(torch.bfloat16).to(dev)           # [S, P, d]
    Xsteps = Xd.permute(1, 0, 2).contiguous()                     # [P, S, d]
    Wr, br, A, Bm = (to_dev(L[n]) for n in ("W_r", "beta", "A", "B"))
    buf = torch.full((S, P, k), -1, dtype=torch.int16, device=dev)
    ws = B.route_workspace(Xsteps[0], Wr, A, k, B.PR2_I16)
    # as a rollout runs it: the first step splits the weights, the others reuse the split
    for pos in range(P):
        # the step writes row s of its [S, k] view at buf[s, pos, :] (row stride P*k)
        B.route_predict(Xsteps[pos], Wr, br, A, Bm, k, buf[:, pos, :], ws=ws, reuse_split=pos > 0)
    torch.cuda.synchronize()
    rec = buf.cpu().numpy()
    assert rec.min() >= 0 and rec.max() < s.N, "some route slot was never written"

    # index stability: a step recorded into a contiguous buffer gives the same rows
    # (each such call forms the split afresh, so this also checks the reused split)
    for pos in (0, 777, P - 1):
        one = torch.empty((S, k), dtype=torch.int16, device=dev)
        B.route_predict(Xsteps[pos], Wr, br, A, Bm, k, one, ws=ws)
        np.testing.assert_array_equal(one.cpu().numpy(), rec[:, pos, :])

    # oracle parity of sampled steps
    steps = list(range(0, P, 64)) + [P - 1]
    excluded = 0
    for pos in steps:
        ref = O.route_predict(X[:, pos, :], L["W_r"], L["beta"], L["A"], L["B"], k)
        ok = ref["margin"] >= MARGIN_EPS
        excluded += int((~ok).sum())
        bad = np.nonzero(ok & np.any(rec[:, pos, :].astype(np.int64) != ref["idx"], axis=1))[0]
        assert len(bad) == 0, f"step {pos}: sequences {bad[:5]} differ"
    print(f"\ndecode: {len(steps)} steps checked, {excluded} tokens under the margin")

    # replay every micro-batch (16 whole sequences = 32768 tokens each)
    Wg, Wu, Wd = (to_dev(L[n], "bf16") for n in ("W_gate", "W_up", "W_down"))
    Xseq = Xd.reshape(S * P, s.d)                                 # rows (seq, pos), seq-major
    mbt = W.DECODE_MICROBATCH
    nseq = mbt // P
    n_mb = S // nseq
    assert n_mb == 16
    ys = torch.empty((S * P, s.d), dtype=torch.bfloat16, device=dev)
    ws_r = B.replay_workspace(Xseq[:mbt], buf[:nseq].reshape(mbt, k), Wr, Wg)
    for mb in range(n_mb):
        lo = mb * mbt
        B.moe_replay_forward(Xseq[lo:lo + mbt], buf[mb * nseq:(mb + 1) * nseq].reshape(mbt, k),
                             Wr, br, Wg, Wu, Wd, ys[lo:lo + mbt], ws=ws_r)
    torch.cuda.synchronize()
    Y = ys.float().cpu().numpy()
    rng = np.random.default_rng(5)
    # sampled rows of every micro-batch, checked in one oracle pass
    rows = np.concatenate([mb * mbt + np.unique(np.concatenate(
        [[0, mbt - 1], rng.choice(mbt, 32, replace=False)])) for mb in range(n_mb)])
    seq, pos = rows // P, rows % P
    xr = X[seq, pos, :]
    ref = O.route_predict(xr, L["W_r"], L["beta"], L["A"], L["B"], k)
    same = (ref["margin"] >= MARGIN_EPS) & np.all(rec[seq, pos, :] == ref["idx"], axis=1)
    assert same.sum() >= len(rows) - 4
    for mb in range(n_mb):
        got = (rows // mbt == mb) & same
        assert got.sum() >= 30, f"micro-batch {mb}: too few rows to check"
    y_ref, _ = O.replay_forward_rows(rows[same], xr[same], ref["idx"][same], L["W_r"], L["beta"],
                                     L["W_gate"], L["W_up"], L["W_down"])
    err = compare_rows(Y[rows[same]], y_ref, "bf16", "decode micro-batches")
    print(f"decode replay: {n_mb} micro-batches, {same.sum()} sampled rows, worst rel err {err:.2e}")
