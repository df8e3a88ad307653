"""Decode-style route recording and replay on the Qwen3-30B-A3B-shaped layer:
256 sequences x 2048 decode steps, each step's route written into one
index-stable int16 buffer [seq, pos, k] (Sec. 4.1: the predicted ids are
cached for replay; Alg. 2, caching step), then replayed in micro-batches of
16 whole sequences = 32768 tokens (Sec. 4.1 replay; Alg. 3).

Oracle checks: the routes of sampled steps against the float64 oracle (margin
rule), and sampled replayed rows against the oracle's replay forward on the
oracle's own route of those tokens (only where it equals the recorded one)."""
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

    # replay micro-batches 0 and 15 (16 whole sequences = 32768 tokens each)
    Wg, Wu, Wd = (to_dev(L[n], "bf16") for n in ("W_gate", "W_up", "W_down"))
    Xseq = Xd.reshape(S * P, s.d)                                 # rows (seq, pos), seq-major
    rng = np.random.default_rng(5)
    for mb in (0, 15):
        lo = mb * 16 * P
        x_mb = Xseq[lo:lo + 16 * P]
        idx_mb = buf[mb * 16:(mb + 1) * 16].reshape(16 * P, k)
        y = torch.empty_like(x_mb)
        B.moe_replay_forward(x_mb, idx_mb, Wr, br, Wg, Wu, Wd, y)
        torch.cuda.synchronize()
        rows = np.unique(np.concatenate([[0, 16 * P - 1], rng.choice(16 * P, 96, replace=False)]))
        seq, pos = mb * 16 + rows // P, rows % P
        xr = X[seq, pos, :]
        ref = O.route_predict(xr, L["W_r"], L["beta"], L["A"], L["B"], k)
        same = (ref["margin"] >= MARGIN_EPS) & np.all(rec[seq, pos, :] == ref["idx"], axis=1)
        assert same.sum() >= len(rows) - 2
        keep = rows[same]
        y_ref, _ = O.replay_forward_rows(keep, xr[same], ref["idx"][same], L["W_r"], L["beta"],
                                         L["W_gate"], L["W_up"], L["W_down"])
        compare_rows(y.float().cpu().numpy()[keep], y_ref, "bf16", f"micro-batch {mb}")
