"""C ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects invalid arguments on the host before any HIP call
(outputs untouched, documented status).  A valid call on a machine without a
GPU must report PR2_ERR_DEVICE rather than crash."""
import ctypes
import os
import re
from ctypes import byref, c_void_p

import pytest

from paper_2606_00395_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.skipif(not os.path.exists(B.LIB_PATH), reason="libpr2.so not built")

FAKE = 0x10000   # a 64 KiB-aligned fake device address: never dereferenced by these tests


def header_symbols():
    with open(os.path.join(ROOT, "include", "pr2.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(pr2_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    L = B.lib()
    syms = header_symbols()
    assert set(syms) == set(B.EXPORTS), syms
    for s in syms:
        assert hasattr(L, s), s
    assert L.pr2_version().decode().startswith("pr2")


def test_status_strings():
    L = B.lib()
    for code, name in enumerate(B.STATUS):
        assert L.pr2_status_string(code).decode() == name
    assert L.pr2_status_string(99).decode() == "PR2_ERR_UNKNOWN"


def desc(**kw):
    base = dict(T=64, d=64, N=8, k=2, m=32, r=4, act=B.PR2_BF16, idx=B.PR2_I32, renorm=True)
    base.update(kw)
    return B.make_desc(**base)


def route(d, x=FAKE, W=FAKE, b=None, A=FAKE, Bm=FAKE, idx=FAKE, ldi=None, gate=None, logits=None,
          ws=FAKE, ws_bytes=None):
    L = B.lib()
    ldi = d.k if ldi is None else ldi
    if ws_bytes is None:
        ws_bytes = B.workspace_bytes(d, B.OP_ROUTE)
    st = L.pr2_route_predict(byref(d), c_void_p(x), c_void_p(W), c_void_p(b), c_void_p(A),
                             c_void_p(Bm), c_void_p(idx), ldi, c_void_p(gate), c_void_p(logits),
                             c_void_p(ws), ws_bytes, None)
    return st, L.pr2_last_error().decode()


def replay(d, x=FAKE, idx=FAKE, ldi=None, W=FAKE, b=None, Wg=FAKE, Wu=FAKE, Wd=FAKE, y=FAKE,
           gate=None, ws=FAKE, ws_bytes=None):
    L = B.lib()
    ldi = d.k if ldi is None else ldi
    if ws_bytes is None:
        ws_bytes = B.workspace_bytes(d, B.OP_REPLAY_FWD)
    st = L.pr2_moe_replay_forward(byref(d), c_void_p(x), c_void_p(idx), ldi, c_void_p(W),
                                  c_void_p(b), c_void_p(Wg), c_void_p(Wu), c_void_p(Wd),
                                  c_void_p(y), c_void_p(gate), c_void_p(ws), ws_bytes, None)
    return st, L.pr2_last_error().decode()


def backward(d, x=FAKE, idx=FAKE, ldi=None, W=FAKE, b=None, Wg=FAKE, Wu=FAKE, Wd=FAKE, dy=FAKE,
             dx=FAKE, dW=FAKE, db=None, dWg=FAKE, dWu=FAKE, dWd=FAKE, ws=FAKE, ws_bytes=None):
    L = B.lib()
    ldi = d.k if ldi is None else ldi
    if ws_bytes is None:
        ws_bytes = B.workspace_bytes(d, B.OP_REPLAY_BWD)
    st = L.pr2_moe_replay_backward(byref(d), c_void_p(x), c_void_p(idx), ldi, c_void_p(W),
                                   c_void_p(b), c_void_p(Wg), c_void_p(Wu), c_void_p(Wd),
                                   c_void_p(dy), c_void_p(dx), c_void_p(dW), c_void_p(db),
                                   c_void_p(dWg), c_void_p(dWu), c_void_p(dWd), c_void_p(ws),
                                   ws_bytes, None)
    return st, L.pr2_last_error().decode()


@pytest.mark.parametrize("kw,status", [
    (dict(k=0), "PR2_ERR_SHAPE"),
    (dict(k=9), "PR2_ERR_SHAPE"),
    (dict(d=0), "PR2_ERR_SHAPE"),
    (dict(N=0, k=1), "PR2_ERR_SHAPE"),
    (dict(T=-1), "PR2_ERR_SHAPE"),
    (dict(r=-1), "PR2_ERR_SHAPE"),
    (dict(act=7), "PR2_ERR_DTYPE"),
    (dict(idx=5), "PR2_ERR_DTYPE"),
    (dict(N=2048, k=8), "PR2_ERR_UNSUPPORTED"),
    (dict(r=300), "PR2_ERR_UNSUPPORTED"),
])
def test_route_rejects_bad_descriptor(kw, status):
    st, msg = route(desc(**kw))
    assert B.STATUS[st] == status, msg
    assert msg


def test_route_rejects_bad_pointers_and_strides():
    d = desc()
    assert B.STATUS[route(d, x=0)[0]] == "PR2_ERR_NULL"
    assert B.STATUS[route(d, W=0)[0]] == "PR2_ERR_NULL"
    assert B.STATUS[route(d, idx=0)[0]] == "PR2_ERR_NULL"
    assert B.STATUS[route(d, A=0)[0]] == "PR2_ERR_NULL"          # r > 0 needs A
    assert B.STATUS[route(d, Bm=0)[0]] == "PR2_ERR_NULL"         # r != N needs B
    assert B.STATUS[route(d, ldi=1)[0]] == "PR2_ERR_SHAPE"       # ldi < k
    assert B.STATUS[route(d, x=FAKE + 2)[0]] == "PR2_ERR_ALIGN"
    assert B.STATUS[route(d, W=FAKE + 2)[0]] == "PR2_ERR_ALIGN"
    assert B.STATUS[route(d, idx=FAKE + 2)[0]] == "PR2_ERR_ALIGN"
    d16 = desc(idx=B.PR2_I16)
    # int16 ids only need 2-byte alignment (a decode step writes at buf + pos*k)
    st, msg = route(d16, idx=FAKE + 2)
    assert B.STATUS[st] in ("PR2_ERR_DEVICE", "PR2_OK"), msg


def test_route_workspace():
    d = desc()
    need = B.workspace_bytes(d, B.OP_ROUTE)
    # bf16 x with d % 32 == 0 and N + r <= 160 takes the MFMA router: 3 bf16 parts of [W_r | A]
    assert need >= 3 * 32 * 64 * 2
    assert B.STATUS[route(d, ws_bytes=need - 1)[0]] == "PR2_ERR_WORKSPACE"
    assert B.STATUS[route(d, ws=0)[0]] == "PR2_ERR_NULL"
    # fp32 x takes the fp64 vector path: no workspace
    assert B.workspace_bytes(desc(act=B.PR2_F32), B.OP_ROUTE) == 0
    st, msg = route(desc(act=B.PR2_F32), ws=0, ws_bytes=0)
    assert B.STATUS[st] in ("PR2_ERR_DEVICE", "PR2_OK"), msg


def test_route_noop_and_device_status():
    # T == 0 is a no-op even with null tensors
    assert route(desc(T=0), x=0, W=0, idx=0, A=0, Bm=0)[0] == 0
    # no predictor: A and B may be null
    st, msg = route(desc(r=0), A=0, Bm=0)
    assert B.STATUS[st] in ("PR2_ERR_DEVICE", "PR2_OK"), msg
    # full-rank predictor: B = NULL means identity when r == N
    st, msg = route(desc(r=8), Bm=0)
    assert B.STATUS[st] in ("PR2_ERR_DEVICE", "PR2_OK"), msg


def test_replay_rejects_bad_arguments():
    d = desc()
    need = B.workspace_bytes(d, B.OP_REPLAY_FWD)
    assert need > 0
    assert B.STATUS[replay(d, ws_bytes=need - 1)[0]] == "PR2_ERR_WORKSPACE"
    assert B.STATUS[replay(d, ws=0)[0]] == "PR2_ERR_NULL"
    assert B.STATUS[replay(d, y=0)[0]] == "PR2_ERR_NULL"
    assert B.STATUS[replay(d, Wd=0)[0]] == "PR2_ERR_NULL"
    assert B.STATUS[replay(d, idx=0)[0]] == "PR2_ERR_NULL"
    assert B.STATUS[replay(d, y=FAKE + 8)[0]] == "PR2_ERR_ALIGN"
    assert B.STATUS[replay(d, ldi=1)[0]] == "PR2_ERR_SHAPE"
    assert B.STATUS[replay(desc(m=0))[0]] == "PR2_ERR_SHAPE"
    assert replay(desc(T=0), x=0, idx=0, W=0, Wg=0, Wu=0, Wd=0, y=0, ws=0, ws_bytes=0)[0] == 0
    assert B.workspace_bytes(desc(k=0), B.OP_REPLAY_FWD) == 0
    assert B.workspace_bytes(desc(k=0), B.OP_ROUTE) == 0


def test_backward_rejects_bad_arguments():
    d = desc()
    need = B.workspace_bytes(d, B.OP_REPLAY_BWD)
    assert need > B.workspace_bytes(d, B.OP_REPLAY_FWD) > 0
    assert B.STATUS[backward(d, ws_bytes=need - 1)[0]] == "PR2_ERR_WORKSPACE"
    assert B.STATUS[backward(d, ws=0)[0]] == "PR2_ERR_NULL"
    for arg in ("x", "idx", "W", "Wg", "Wu", "Wd", "dy", "dx", "dW", "dWg", "dWu", "dWd"):
        st, msg = backward(d, **{arg: 0})
        assert B.STATUS[st] == "PR2_ERR_NULL", (arg, msg)
    assert B.STATUS[backward(d, dx=FAKE + 8)[0]] == "PR2_ERR_ALIGN"
    assert B.STATUS[backward(d, dWd=FAKE + 4)[0]] == "PR2_ERR_ALIGN"
    assert B.STATUS[backward(d, db=FAKE + 2)[0]] == "PR2_ERR_ALIGN"
    assert B.STATUS[backward(d, ldi=1)[0]] == "PR2_ERR_SHAPE"
    # the paper-literal weights: accepted for k <= 64 (this host has no GPU), refused above
    st, msg = backward(desc(renorm=False))
    assert B.STATUS[st] in ("PR2_ERR_DEVICE", "PR2_OK"), msg
    dk = desc(renorm=False, N=128, k=65)
    st, msg = backward(dk)
    assert B.STATUS[st] == "PR2_ERR_UNSUPPORTED" and "k <= 64" in msg
    # its workspace holds the dense logits and logit gradients too
    assert B.workspace_bytes(desc(renorm=False), B.OP_REPLAY_BWD) > \
        B.workspace_bytes(desc(), B.OP_REPLAY_BWD)
    # T = 0 still has weight gradients to zero: those pointers stay required
    st, _ = backward(desc(T=0), x=0, idx=0, dy=0, dx=0, ws=0, ws_bytes=0, dWg=0)
    assert B.STATUS[st] == "PR2_ERR_NULL"
    assert B.workspace_bytes(desc(k=0), B.OP_REPLAY_BWD) == 0


def test_saved_activation_entry_points_reject_bad_arguments():
    L = B.lib()
    d = desc()

    def fwd_save(dd=d, au=FAKE, y=FAKE):
        ws = B.workspace_bytes(dd, B.OP_REPLAY_FWD)
        st = L.pr2_moe_replay_forward_save(byref(dd), c_void_p(FAKE), c_void_p(FAKE), dd.k,
                                           c_void_p(FAKE), None, c_void_p(FAKE), c_void_p(FAKE),
                                           c_void_p(FAKE), c_void_p(y), None, c_void_p(au),
                                           c_void_p(FAKE), ws, None)
        return B.STATUS[st], L.pr2_last_error().decode()

    def bwd_saved(dd=d, au=FAKE, dx=FAKE):
        ws = B.workspace_bytes(dd, B.OP_REPLAY_BWD)
        st = L.pr2_moe_replay_backward_saved(byref(dd), c_void_p(FAKE), c_void_p(FAKE), dd.k,
                                             c_void_p(FAKE), None, c_void_p(FAKE),
                                             c_void_p(FAKE), c_void_p(FAKE), c_void_p(au),
                                             c_void_p(FAKE), c_void_p(dx), c_void_p(FAKE), None,
                                             c_void_p(FAKE), c_void_p(FAKE), c_void_p(FAKE),
                                             c_void_p(FAKE), ws, None)
        return B.STATUS[st], L.pr2_last_error().decode()

    assert fwd_save(au=0)[0] == "PR2_ERR_NULL"
    assert fwd_save(au=FAKE + 8)[0] == "PR2_ERR_ALIGN"
    assert fwd_save(y=0)[0] == "PR2_ERR_NULL"             # the forward's own checks still run
    assert bwd_saved(au=0)[0] == "PR2_ERR_NULL"
    assert bwd_saved(au=FAKE + 8)[0] == "PR2_ERR_ALIGN"
    assert bwd_saved(dx=0)[0] == "PR2_ERR_NULL"
    assert bwd_saved(desc(renorm=False, N=128, k=65))[0] == "PR2_ERR_UNSUPPORTED"
    assert fwd_save(desc(act=7))[0] == "PR2_ERR_DTYPE"
    for st, msg in (fwd_save(), bwd_saved()):
        assert st in ("PR2_ERR_DEVICE", "PR2_OK"), msg


def test_valid_call_without_gpu_reports_device():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    st, msg = route(desc())
    assert B.STATUS[st] == "PR2_ERR_DEVICE", msg
    st, msg = replay(desc())
    assert B.STATUS[st] == "PR2_ERR_DEVICE", msg
    st, msg = backward(desc())
    assert B.STATUS[st] == "PR2_ERR_DEVICE", msg
    st, msg = backward(desc(T=0), x=0, idx=0, dy=0, dx=0, ws=0, ws_bytes=0)
    assert B.STATUS[st] == "PR2_ERR_DEVICE", msg


def test_workspace_grows_with_tokens():
    a = B.workspace_bytes(desc(T=1000), B.OP_REPLAY_FWD)
    b = B.workspace_bytes(desc(T=2000), B.OP_REPLAY_FWD)
    assert b > a > 0
    # H [T*k, m] and O [T*k, d] in bf16 dominate
    d = desc(T=16384, d=2048, N=128, k=8, m=768)
    assert B.workspace_bytes(d, B.OP_REPLAY_FWD) >= 16384 * 8 * (768 + 2048) * 2


# ------------------------------------------------ feature cache (host) ----

@pytest.mark.parametrize("T,Tc,seed", [(16384, 2048, 0), (16384, 2048, 12345), (1000, 7, 1),
                                       (1000, 999, 2**64 - 1), (50, 64, 3), (1, 1, 9),
                                       (2**20 + 3, 4096, 2**63 + 11)])
def test_feature_cache_positions_match_oracle(T, Tc, seed):
    """The library's sampler (host C) and the oracle's (Python integers) draw
    the same positions: both implement the same stratified rule with
    SplitMix64."""
    import numpy as np
    from oracle import pr2_oracle as O
    got = B.feature_cache_positions(T, Tc, seed)
    np.testing.assert_array_equal(got, O.feature_cache_positions(T, Tc, seed))


def test_feature_cache_positions_rejects_bad_arguments():
    L = B.lib()
    assert L.pr2_feature_cache_positions(-1, 4, 0, None) == -1
    assert L.pr2_feature_cache_positions(10, 0, 0, None) == -1
    assert L.pr2_feature_cache_positions(10, 4, 0, None) == -1
    assert "NULL" in L.pr2_last_error().decode()
    assert L.pr2_feature_cache_positions(0, 4, 0, None) == 0


def test_cached_route_and_predictor_loss_reject_bad_arguments():
    L = B.lib()
    d = desc()
    ws = B.workspace_bytes(d, B.OP_ROUTE)

    def cached(dd=d, row=FAKE, h=FAKE, p=FAKE, rows=16, x=FAKE):
        st = L.pr2_route_predict_cached(byref(dd), c_void_p(x), c_void_p(FAKE), None,
                                        c_void_p(FAKE), c_void_p(FAKE), c_void_p(FAKE), dd.k, None,
                                        c_void_p(row), c_void_p(h), c_void_p(p), rows,
                                        c_void_p(FAKE), ws, None)
        return B.STATUS[st]
    assert cached(row=0) == "PR2_ERR_NULL"
    assert cached(h=0) == "PR2_ERR_NULL"
    assert cached(h=FAKE + 4) == "PR2_ERR_ALIGN"
    assert cached(rows=-1) == "PR2_ERR_SHAPE"
    assert cached(x=0) == "PR2_ERR_NULL"

    def loss(dd=d, kind=0, step=2, A=FAKE, Bm=FAKE, dB=FAKE, loss_out=FAKE, h=FAKE, ws_bytes=None):
        wb = B.workspace_bytes(dd, B.OP_PREDICTOR_LOSS) if ws_bytes is None else ws_bytes
        st = L.pr2_predictor_loss(byref(dd), c_void_p(h), c_void_p(FAKE), None, c_void_p(FAKE),
                                  c_void_p(FAKE), c_void_p(A), c_void_p(Bm), kind, step, None,
                                  c_void_p(loss_out), c_void_p(FAKE), c_void_p(dB),
                                  c_void_p(FAKE), wb, None)
        return B.STATUS[st]
    assert B.workspace_bytes(d, B.OP_PREDICTOR_LOSS) > 0
    assert B.workspace_bytes(desc(r=0), B.OP_PREDICTOR_LOSS) == 0
    assert loss(desc(r=0)) == "PR2_ERR_SHAPE"
    assert loss(kind=2) == "PR2_ERR_SHAPE"
    assert loss(step=0) == "PR2_ERR_SHAPE"
    assert loss(A=0) == "PR2_ERR_NULL"
    assert loss(Bm=0) == "PR2_ERR_NULL"            # r != N: B required
    assert loss(dB=0) == "PR2_ERR_NULL"
    assert loss(loss_out=0) == "PR2_ERR_NULL"
    assert loss(h=0) == "PR2_ERR_NULL"
    assert loss(ws_bytes=1) == "PR2_ERR_WORKSPACE"
    assert loss(desc(r=8), Bm=0, dB=0) in ("PR2_ERR_DEVICE", "PR2_OK")   # identity, r == N


def test_workspace_bytes_do_not_decrease_with_batch():
    """A workspace sized for a batch also serves every smaller batch of the
    same layer (decode loops shrink their batch as sequences finish)."""
    from paper_2606_00395_amd import binding as B
    for op in (B.OP_ROUTE, B.OP_REPLAY_FWD, B.OP_ROLLOUT_FWD, B.OP_REPLAY_BWD, B.OP_ROUTE_DIAG,
               B.OP_PREDICTOR_LOSS):
        prev = 0
        for T in (1, 63, 64, 65, 256, 1000, 1024, 1025, 2048, 16384):
            desc = B.make_desc(T, 2048, 128, 8, 768, 16, B.PR2_BF16, B.PR2_I32, 1)
            n = B.workspace_bytes(desc, op)
            assert n >= prev, (op, T, n, prev)
            prev = n


@pytest.mark.parametrize("k", list(range(1, 65)) + [96, 128, 255])
def test_token_division_by_multiply_high(k):
    """The backward GEMMs turn a route entry n = t k + s into its token t as
    mulhi(n, ceil(2^32 / k)) (k = 1: the constant is 0 and t = n); the host
    keeps T k * k below 2^32, so every entry is below 2^32 / k.  Checked here
    against integer division at the ends of that range, at multiples of k and
    their neighbours, and at random entries."""
    import numpy as np
    kmul = 0 if k == 1 else (0xFFFFFFFF // k + 1)
    top = (1 << 32) // k - (1 if (1 << 32) % k == 0 else 0)   # largest n with n k < 2^32
    rng = np.random.default_rng(k)
    q = np.arange(0, top // k + 1, max(1, (top // k) // 4096), dtype=np.uint64)
    n = np.concatenate([q * k, q * k + (k - 1), q * k + 1,
                        rng.integers(0, top + 1, 20000, dtype=np.uint64),
                        np.arange(max(0, top - 4096), top + 1, dtype=np.uint64)])
    n = n[n <= top]
    t = ((n * np.uint64(kmul)) >> np.uint64(32)) + (n if kmul == 0 else np.uint64(0))
    assert np.array_equal(t, n // np.uint64(k))


def test_route_reuse_rejects_bad_arguments():
    """pr2_route_predict_reuse runs pr2_route_predict's checks before anything else."""
    L = B.lib()
    d = desc()
    ws_bytes = B.workspace_bytes(d, B.OP_ROUTE)

    def reuse(x=FAKE, idx=FAKE, ldi=d.k, ws=FAKE, nbytes=ws_bytes):
        st = L.pr2_route_predict_reuse(byref(d), c_void_p(x), c_void_p(FAKE), None,
                                       c_void_p(FAKE), c_void_p(FAKE), c_void_p(idx), ldi, None,
                                       None, c_void_p(ws), nbytes, None)
        return B.STATUS[st], L.pr2_last_error().decode()

    assert reuse(x=0)[0] == "PR2_ERR_NULL"
    assert reuse(idx=0)[0] == "PR2_ERR_NULL"
    assert reuse(ldi=1)[0] == "PR2_ERR_SHAPE"
    assert reuse(x=FAKE + 2)[0] == "PR2_ERR_ALIGN"
    assert reuse(nbytes=ws_bytes - 1)[0] == "PR2_ERR_WORKSPACE"


def route_reuse(d, x=FAKE, W=FAKE, b=None, A=FAKE, Bm=FAKE, idx=FAKE, logits=None, ws=FAKE):
    L = B.lib()
    st = L.pr2_route_predict_reuse(byref(d), c_void_p(x), c_void_p(W), c_void_p(b), c_void_p(A),
                                   c_void_p(Bm), c_void_p(idx), d.k, None, c_void_p(logits),
                                   c_void_p(ws), B.workspace_bytes(d, B.OP_ROUTE), None)
    return st, L.pr2_last_error().decode()


def test_reuse_needs_a_recorded_split():
    """pr2_route_predict_reuse refuses a workspace that holds no split formed by a
    route call (checked on the host, before any HIP call)."""
    d = desc()                                    # bf16, d % 32 == 0: the MFMA router's split
    assert B.workspace_bytes(d, B.OP_ROUTE) > 0
    st, msg = route_reuse(d, ws=FAKE + 0x100000)
    assert B.STATUS[st] == "PR2_ERR_WORKSPACE", msg
    assert "no router split" in msg
    # with logits wanted (the unfolded layout) the same
    st, msg = route_reuse(d, ws=FAKE + 0x200000, logits=FAKE)
    assert B.STATUS[st] == "PR2_ERR_WORKSPACE", msg
    # the fp64 vector path keeps no split: nothing to check, the call goes on
    st, msg = route_reuse(desc(act=B.PR2_F32))
    assert B.STATUS[st] in ("PR2_ERR_DEVICE", "PR2_OK"), msg


def test_noalloc_rejects_a_split_beyond_its_scratch():
    """pr2_route_predict_noalloc keeps the weight split in a 6 MiB device array: a
    shape whose split is larger is refused on the host, before any HIP call."""
    L = B.lib()

    def call(d, logits=None):
        st = L.pr2_route_predict_noalloc(byref(d), c_void_p(FAKE), c_void_p(FAKE), None,
                                         c_void_p(FAKE), c_void_p(FAKE), c_void_p(FAKE), d.k,
                                         None, c_void_p(logits), None)
        return B.STATUS[st], L.pr2_last_error().decode()
    # d 8192, N 128 folded: 3 x 2 x 8192 x 128 = 6 MiB fits exactly
    st, msg = call(desc(d=8192, N=128, k=8, r=16))
    assert st in ("PR2_ERR_DEVICE", "PR2_OK"), msg
    # with logits wanted the split is [W_r | A]: 192 columns, 9 MiB
    st, msg = call(desc(d=8192, N=128, k=8, r=16), logits=FAKE)
    assert st == "PR2_ERR_UNSUPPORTED" and "scratch" in msg, msg
    # the usual argument checks still come first
    st, msg = call(desc(k=0))
    assert st == "PR2_ERR_SHAPE", msg
