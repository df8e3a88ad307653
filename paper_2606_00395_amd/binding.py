"""ctypes binding of libpr2.so: argument marshalling only.

Every computation runs in the library's HIP kernels; this module only reads
shapes, dtypes, strides and device pointers off torch tensors and passes them
through the C ABI declared in include/pr2.h.  Importing it needs no GPU; the
library itself is loaded on first use and a missing build raises at once.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import (POINTER, byref, c_char_p, c_double, c_int, c_int32, c_int64, c_size_t,
                    c_uint64, c_void_p)

HERE = os.path.dirname(os.path.abspath(__file__))
# PR2_LIBRARY names another build of the same library (the host-sanitizer build
# of build_sanitized.py, for the CPU checks)
LIB_PATH = os.environ.get("PR2_LIBRARY") or os.path.join(HERE, "libpr2.so")

PR2_F32, PR2_BF16 = 0, 1
PR2_I32, PR2_I16 = 0, 1
OP_ROUTE, OP_REPLAY_FWD, OP_REPLAY_BWD, OP_ROLLOUT_FWD, OP_ROUTE_DIAG, OP_PREDICTOR_LOSS = range(6)

STATUS = ["PR2_OK", "PR2_ERR_NULL", "PR2_ERR_SHAPE", "PR2_ERR_DTYPE", "PR2_ERR_ALIGN",
          "PR2_ERR_WORKSPACE", "PR2_ERR_UNSUPPORTED", "PR2_ERR_ROUTE", "PR2_ERR_DEVICE",
          "PR2_ERR_HIP"]

# every symbol include/pr2.h declares
EXPORTS = ["pr2_workspace_bytes", "pr2_route_predict", "pr2_route_predict_reuse",
           "pr2_route_predict_noalloc",
           "pr2_moe_replay_forward", "pr2_moe_replay_forward_diag",
           "pr2_moe_replay_forward_save", "pr2_moe_replay_backward_saved",
           "pr2_moe_replay_backward", "pr2_moe_rollout_forward", "pr2_route_diagnostics",
           "pr2_feature_cache_positions", "pr2_route_predict_cached", "pr2_predictor_loss",
           "pr2_status_string",
           "pr2_last_error", "pr2_version", "pr2_profile_enable",
           "pr2_profile_reset", "pr2_profile_collect"]


class Pr2Error(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        name = STATUS[status] if 0 <= status < len(STATUS) else str(status)
        super().__init__(f"{name}: {detail}")


class MoeDesc(ctypes.Structure):
    _fields_ = [("T", c_int64), ("d", c_int32), ("N", c_int32), ("k", c_int32), ("m", c_int32),
                ("r", c_int32), ("act_dtype", c_int32), ("idx_dtype", c_int32),
                ("renorm", c_int32)]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it first "
                           "(python -c 'import __graft_entry__ as g; g.build()')")
    L = ctypes.CDLL(LIB_PATH)
    P = c_void_p
    L.pr2_workspace_bytes.argtypes = [POINTER(MoeDesc), c_int]
    L.pr2_workspace_bytes.restype = c_size_t
    L.pr2_route_predict.argtypes = [POINTER(MoeDesc), P, P, P, P, P, P, c_int64, P, P, P,
                                    c_size_t, P]
    L.pr2_route_predict.restype = c_int
    L.pr2_route_predict_reuse.argtypes = L.pr2_route_predict.argtypes
    L.pr2_route_predict_reuse.restype = c_int
    L.pr2_route_predict_noalloc.argtypes = [POINTER(MoeDesc), P, P, P, P, P, P, c_int64, P, P, P]
    L.pr2_route_predict_noalloc.restype = c_int
    L.pr2_moe_replay_forward.argtypes = [POINTER(MoeDesc), P, P, c_int64, P, P, P, P, P, P, P,
                                         P, c_size_t, P]
    L.pr2_moe_replay_forward.restype = c_int
    L.pr2_moe_replay_forward_diag.argtypes = [POINTER(MoeDesc), P, P, c_int64, P, P, P, P, P, P,
                                              P, P, P, P, P, P, P, c_size_t, P]
    L.pr2_moe_replay_forward_diag.restype = c_int
    L.pr2_moe_replay_backward.argtypes = [POINTER(MoeDesc), P, P, c_int64, P, P, P, P, P, P, P,
                                          P, P, P, P, P, P, c_size_t, P]
    L.pr2_moe_replay_backward.restype = c_int
    L.pr2_moe_replay_forward_save.argtypes = [POINTER(MoeDesc), P, P, c_int64, P, P, P, P, P, P,
                                              P, P, P, c_size_t, P]
    L.pr2_moe_replay_forward_save.restype = c_int
    L.pr2_moe_replay_backward_saved.argtypes = [POINTER(MoeDesc), P, P, c_int64, P, P, P, P, P, P,
                                                P, P, P, P, P, P, P, P, c_size_t, P]
    L.pr2_moe_replay_backward_saved.restype = c_int
    L.pr2_moe_rollout_forward.argtypes = [POINTER(MoeDesc), P, P, P, P, P, P, P, P, P, c_int64, P,
                                          P, P, P, c_size_t, P]
    L.pr2_moe_rollout_forward.restype = c_int
    L.pr2_route_diagnostics.argtypes = [POINTER(MoeDesc), P, P, c_int64, P, P, P, P, P, P, P, P,
                                        c_size_t, P]
    L.pr2_route_diagnostics.restype = c_int
    L.pr2_feature_cache_positions.argtypes = [c_int64, c_int64, c_uint64, P]
    L.pr2_feature_cache_positions.restype = c_int64
    L.pr2_route_predict_cached.argtypes = [POINTER(MoeDesc), P, P, P, P, P, P, c_int64, P, P, P, P,
                                           c_int64, P, c_size_t, P]
    L.pr2_route_predict_cached.restype = c_int
    L.pr2_predictor_loss.argtypes = [POINTER(MoeDesc), P, P, P, P, P, P, P, c_int, c_int, P, P, P,
                                     P, P, c_size_t, P]
    L.pr2_predictor_loss.restype = c_int
    L.pr2_status_string.argtypes = [c_int]
    L.pr2_status_string.restype = c_char_p
    L.pr2_last_error.argtypes = []
    L.pr2_last_error.restype = c_char_p
    L.pr2_version.argtypes = []
    L.pr2_version.restype = c_char_p
    L.pr2_profile_enable.argtypes = [c_int]
    L.pr2_profile_enable.restype = None
    L.pr2_profile_reset.argtypes = []
    L.pr2_profile_reset.restype = None
    L.pr2_profile_collect.argtypes = [POINTER(c_char_p), POINTER(c_double), POINTER(c_int64), c_int]
    L.pr2_profile_collect.restype = c_int
    _lib = L
    return L


def check(status: int):
    if status != 0:
        raise Pr2Error(status, lib().pr2_last_error().decode())


# ----------------------------------------------------------- torch glue ----

def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else c_void_p(t.data_ptr())


def _act_code(t):
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return PR2_BF16
    if t.dtype == torch.float32:
        return PR2_F32
    raise TypeError(f"activations must be bfloat16 or float32, got {t.dtype}")


def _idx_code(t):
    torch = _torch()
    if t.dtype == torch.int16:
        return PR2_I16
    if t.dtype == torch.int32:
        return PR2_I32
    raise TypeError(f"expert ids must be int16 or int32, got {t.dtype}")


def _stream(stream):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return c_void_p(stream.cuda_stream)


def _row_stride(idx):
    if idx.dim() != 2 or idx.stride(1) != 1:
        raise ValueError("ids must be a 2-D view [T, k] with unit stride along k")
    if idx.shape[0] > 1 and idx.stride(0) < idx.shape[1]:
        raise ValueError("id rows overlap: row stride below k")
    return idx.stride(0)


def _need(t, name, shape, dtype=None, device=None, optional=False):
    """Checks that tensor ``t`` is what the C ABI will read or write through its
    pointer: the given shape, dtype and device, row-major and contiguous."""
    torch = _torch()
    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous (row-major)")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")


def _need_ids(idx, name, T, k, device):
    torch = _torch()
    if tuple(idx.shape) != (T, k):
        raise ValueError(f"{name} has shape {tuple(idx.shape)}, expected {(T, k)}")
    if idx.dtype not in (torch.int16, torch.int32):
        raise TypeError(f"{name} must be int16 or int32, got {idx.dtype}")
    if idx.device != device:
        raise ValueError(f"{name} is on {idx.device}, expected {device}")
    return _row_stride(idx)


def _need_act(x, name="x"):
    torch = _torch()
    if x.dim() != 2:
        raise ValueError(f"{name} must be 2-D [T, d]")
    _act_code(x)
    if not x.is_contiguous():
        raise ValueError(f"{name} must be contiguous (row-major)")
    if x.device.type != "cuda":
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    return x.shape[0], x.shape[1], x.dtype, x.device


def _need_ws(ws, device):
    torch = _torch()
    if ws is None:
        return
    if ws.dtype != torch.uint8 or not ws.is_contiguous() or ws.device != device:
        raise ValueError("ws must be a contiguous uint8 tensor on the inputs' device")


def _new_ws(nbytes, device, stream):
    """A workspace of nbytes; allocated on ``stream`` when one is given, so that
    the caching allocator does not hand its memory to another stream while the
    call may still be using it."""
    torch = _torch()
    if stream is None:
        return torch.empty(max(1, nbytes), dtype=torch.uint8, device=device)
    with torch.cuda.stream(stream):
        return torch.empty(max(1, nbytes), dtype=torch.uint8, device=device)


def _experts(W_gate, W_up, W_down, N, d, dtype, device):
    if W_gate.dim() != 3:
        raise ValueError("W_gate must be [N, m, d]")
    m = W_gate.shape[1]
    _need(W_gate, "W_gate", (N, m, d), dtype, device)
    _need(W_up, "W_up", (N, m, d), dtype, device)
    _need(W_down, "W_down", (N, d, m), dtype, device)
    return m


def _router(W_r, b_r, d, device):
    torch = _torch()
    if W_r.dim() != 2 or W_r.shape[0] != d:
        raise ValueError(f"W_r must be [d={d}, N]")
    N = W_r.shape[1]
    _need(W_r, "W_r", (d, N), torch.float32, device)
    _need(b_r, "b_r", (N,), torch.float32, device, optional=True)
    return N


def _predictor(A, B, d, N, device):
    torch = _torch()
    if A is None:
        if B is not None:
            raise ValueError("B given without A")
        return 0
    if A.dim() != 2 or A.shape[0] != d:
        raise ValueError(f"A must be [d={d}, r]")
    r = A.shape[1]
    _need(A, "A", (d, r), torch.float32, device)
    if B is None and r != N:
        raise ValueError("B may be omitted only for a full-rank predictor (r == N)")
    _need(B, "B", (r, N), torch.float32, device, optional=True)
    return r


def make_desc(T, d, N, k, m=0, r=0, act=PR2_BF16, idx=PR2_I32, renorm=True) -> MoeDesc:
    return MoeDesc(T, d, N, k, m, r, act, idx, 1 if renorm else 0)


def workspace_bytes(desc: MoeDesc, op: int) -> int:
    return int(lib().pr2_workspace_bytes(byref(desc), op))


def route_workspace(x, W_r, A, k, idx_dtype_code=PR2_I32, stream=None):
    T, d = x.shape
    r = 0 if A is None else A.shape[1]
    desc = make_desc(T, d, W_r.shape[1], k, 0, r, _act_code(x), idx_dtype_code)
    return _new_ws(workspace_bytes(desc, OP_ROUTE), x.device, stream)


def route_predict(x, W_r, b_r, A, B, k, idx_out, gate_out=None, logits_out=None, renorm=True,
                  ws=None, stream=None, reuse_split=False):
    """pr2_route_predict on torch tensors.  ``idx_out`` is a [T, k] view (any row stride)
    of int16/int32; A/B may be None (no predictor); B None with A given means identity.
    ``reuse_split`` calls pr2_route_predict_reuse: ``ws`` must hold the weight split of the
    previous call with the same weights (see include/pr2.h)."""
    torch = _torch()
    if reuse_split and ws is None:
        raise ValueError("reuse_split needs the workspace of the previous call")
    T, d, _, dev = _need_act(x)
    N = _router(W_r, b_r, d, dev)
    r = _predictor(A, B, d, N, dev)
    ldi = _need_ids(idx_out, "idx_out", T, k, dev)
    _need(gate_out, "gate_out", (T, k), torch.float32, dev, optional=True)
    _need(logits_out, "logits_out", (T, N), torch.float32, dev, optional=True)
    _need_ws(ws, dev)
    desc = make_desc(T, d, N, k, 0, r, _act_code(x), _idx_code(idx_out), renorm)
    if ws is None:
        ws = route_workspace(x, W_r, A, k, _idx_code(idx_out), stream)
    fn = lib().pr2_route_predict_reuse if reuse_split else lib().pr2_route_predict
    check(fn(byref(desc), _ptr(x), _ptr(W_r), _ptr(b_r), _ptr(A), _ptr(B), _ptr(idx_out),
             ldi, _ptr(gate_out), _ptr(logits_out), _ptr(ws), ws.numel(), _stream(stream)))


def route_predict_noalloc(x, W_r, b_r, A, B, k, idx_out, gate_out=None, logits_out=None,
                          renorm=True, stream=None):
    """pr2_route_predict_noalloc on torch tensors: pr2_route_predict with the library's
    own device scratch instead of a workspace (nothing is allocated)."""
    torch = _torch()
    T, d, _, dev = _need_act(x)
    N = _router(W_r, b_r, d, dev)
    r = _predictor(A, B, d, N, dev)
    ldi = _need_ids(idx_out, "idx_out", T, k, dev)
    _need(gate_out, "gate_out", (T, k), torch.float32, dev, optional=True)
    _need(logits_out, "logits_out", (T, N), torch.float32, dev, optional=True)
    desc = make_desc(T, d, N, k, 0, r, _act_code(x), _idx_code(idx_out), renorm)
    check(lib().pr2_route_predict_noalloc(byref(desc), _ptr(x), _ptr(W_r), _ptr(b_r), _ptr(A),
                                          _ptr(B), _ptr(idx_out), ldi, _ptr(gate_out),
                                          _ptr(logits_out), _stream(stream)))


def replay_workspace(x, idx, W_r, W_gate, renorm=True, stream=None):
    T, d = x.shape
    desc = make_desc(T, d, W_r.shape[1], idx.shape[1], W_gate.shape[1], 0, _act_code(x),
                     _idx_code(idx), renorm)
    return _new_ws(workspace_bytes(desc, OP_REPLAY_FWD), x.device, stream)


def moe_replay_forward(x, idx, W_r, b_r, W_gate, W_up, W_down, y, gate_out=None, ws=None,
                       renorm=True, stream=None):
    """pr2_moe_replay_forward on torch tensors.  ``idx`` is a [T, k] view (any row stride)."""
    torch = _torch()
    T, d, adt, dev = _need_act(x)
    N = _router(W_r, b_r, d, dev)
    k = idx.shape[1] if idx.dim() == 2 else -1
    ldi = _need_ids(idx, "idx", T, k, dev)
    m = _experts(W_gate, W_up, W_down, N, d, adt, dev)
    _need(y, "y", (T, d), adt, dev)
    _need(gate_out, "gate_out", (T, k), torch.float32, dev, optional=True)
    _need_ws(ws, dev)
    desc = make_desc(T, d, N, k, m, 0, _act_code(x), _idx_code(idx), renorm)
    if ws is None:
        ws = replay_workspace(x, idx, W_r, W_gate, renorm, stream)
    check(lib().pr2_moe_replay_forward(byref(desc), _ptr(x), _ptr(idx), ldi,
                                       _ptr(W_r), _ptr(b_r), _ptr(W_gate), _ptr(W_up),
                                       _ptr(W_down), _ptr(y), _ptr(gate_out), _ptr(ws),
                                       ws.numel(), _stream(stream)))


def moe_replay_forward_save(x, idx, W_r, b_r, W_gate, W_up, W_down, y, au_out, gate_out=None,
                            ws=None, renorm=True, stream=None):
    """pr2_moe_replay_forward_save: the replay forward, also writing the experts'
    pre-activations to ``au_out`` ([T*k, 2m], the activation dtype) for
    moe_replay_backward_saved."""
    torch = _torch()
    T, d, adt, dev = _need_act(x)
    N = _router(W_r, b_r, d, dev)
    k = idx.shape[1] if idx.dim() == 2 else -1
    ldi = _need_ids(idx, "idx", T, k, dev)
    m = _experts(W_gate, W_up, W_down, N, d, adt, dev)
    _need(y, "y", (T, d), adt, dev)
    _need(au_out, "au_out", (T * k, 2 * m), adt, dev)
    _need(gate_out, "gate_out", (T, k), torch.float32, dev, optional=True)
    _need_ws(ws, dev)
    desc = make_desc(T, d, N, k, m, 0, _act_code(x), _idx_code(idx), renorm)
    if ws is None:
        ws = replay_workspace(x, idx, W_r, W_gate, renorm, stream)
    check(lib().pr2_moe_replay_forward_save(byref(desc), _ptr(x), _ptr(idx), ldi, _ptr(W_r),
                                            _ptr(b_r), _ptr(W_gate), _ptr(W_up), _ptr(W_down),
                                            _ptr(y), _ptr(gate_out), _ptr(au_out), _ptr(ws),
                                            ws.numel(), _stream(stream)))


def moe_replay_forward_diag(x, idx, W_r, b_r, W_gate, W_up, W_down, y, gate_out=None,
                            z_ref=None, cur_idx_out=None, overlap_out=None, kl_out=None,
                            hist_out=None, ws=None, renorm=True, stream=None):
    """pr2_moe_replay_forward_diag: the replay forward plus the route diagnostics
    (current top-k, overlap, route KL against ``z_ref``, deviation histogram)."""
    torch = _torch()
    T, d, adt, dev = _need_act(x)
    N = _router(W_r, b_r, d, dev)
    k = idx.shape[1] if idx.dim() == 2 else -1
    ldi = _need_ids(idx, "idx", T, k, dev)
    m = _experts(W_gate, W_up, W_down, N, d, adt, dev)
    _need(y, "y", (T, d), adt, dev)
    _need(gate_out, "gate_out", (T, k), torch.float32, dev, optional=True)
    _need(z_ref, "z_ref", (T, N), torch.float32, dev, optional=True)
    if cur_idx_out is not None:
        _need(cur_idx_out, "cur_idx_out", (T, k), idx.dtype, dev)
    _need(overlap_out, "overlap_out", (T,), torch.int32, dev, optional=True)
    _need(kl_out, "kl_out", (T,), torch.float32, dev, optional=True)
    if hist_out is not None:
        _need(hist_out, "hist_out", (k + 1,), None, dev)
        if hist_out.dtype not in (torch.int64, torch.uint64):
            raise TypeError("hist_out must be int64 or uint64")
    _need_ws(ws, dev)
    desc = make_desc(T, d, N, k, m, 0, _act_code(x), _idx_code(idx), renorm)
    if ws is None:
        ws = replay_workspace(x, idx, W_r, W_gate, renorm, stream)
    check(lib().pr2_moe_replay_forward_diag(byref(desc), _ptr(x), _ptr(idx), ldi, _ptr(W_r),
                                            _ptr(b_r), _ptr(W_gate), _ptr(W_up), _ptr(W_down),
                                            _ptr(y), _ptr(gate_out), _ptr(z_ref),
                                            _ptr(cur_idx_out), _ptr(overlap_out), _ptr(kl_out),
                                            _ptr(hist_out), _ptr(ws), ws.numel(),
                                            _stream(stream)))


def rollout_workspace(x, W_r, A, W_gate, k, idx_dtype_code=PR2_I32, renorm=True, stream=None):
    T, d = x.shape
    r = 0 if A is None else A.shape[1]
    desc = make_desc(T, d, W_r.shape[1], k, W_gate.shape[1], r, _act_code(x), idx_dtype_code,
                     renorm)
    return _new_ws(workspace_bytes(desc, OP_ROLLOUT_FWD), x.device, stream)


def moe_rollout_forward(x, W_r, b_r, A, B, W_gate, W_up, W_down, k, idx_out, y, gate_out=None,
                        logits_out=None, renorm=True, ws=None, stream=None):
    """pr2_moe_rollout_forward on torch tensors: records the predicted route into ``idx_out``
    (a [T, k] view, any row stride) and writes the layer output under the predictive weights."""
    torch = _torch()
    T, d, adt, dev = _need_act(x)
    N = _router(W_r, b_r, d, dev)
    r = _predictor(A, B, d, N, dev)
    ldi = _need_ids(idx_out, "idx_out", T, k, dev)
    m = _experts(W_gate, W_up, W_down, N, d, adt, dev)
    _need(y, "y", (T, d), adt, dev)
    _need(gate_out, "gate_out", (T, k), torch.float32, dev, optional=True)
    _need(logits_out, "logits_out", (T, N), torch.float32, dev, optional=True)
    _need_ws(ws, dev)
    desc = make_desc(T, d, N, k, m, r, _act_code(x), _idx_code(idx_out), renorm)
    if ws is None:
        ws = rollout_workspace(x, W_r, A, W_gate, k, _idx_code(idx_out), renorm, stream)
    check(lib().pr2_moe_rollout_forward(byref(desc), _ptr(x), _ptr(W_r), _ptr(b_r), _ptr(A),
                                        _ptr(B), _ptr(W_gate), _ptr(W_up), _ptr(W_down),
                                        _ptr(idx_out), ldi, _ptr(gate_out),
                                        _ptr(logits_out), _ptr(y), _ptr(ws), ws.numel(),
                                        _stream(stream)))


def route_diagnostics(x, idx, W_r, b_r, z_ref=None, cur_idx_out=None, overlap_out=None,
                      kl_out=None, hist_out=None, ws=None, stream=None):
    """pr2_route_diagnostics on torch tensors; ``hist_out`` is an int64/uint64 tensor of k+1."""
    torch = _torch()
    T, d, _, dev = _need_act(x)
    N = _router(W_r, b_r, d, dev)
    k = idx.shape[1] if idx.dim() == 2 else -1
    ldi = _need_ids(idx, "idx", T, k, dev)
    _need(z_ref, "z_ref", (T, N), torch.float32, dev, optional=True)
    if cur_idx_out is not None:
        _need(cur_idx_out, "cur_idx_out", (T, k), idx.dtype, dev)
    _need(overlap_out, "overlap_out", (T,), torch.int32, dev, optional=True)
    _need(kl_out, "kl_out", (T,), torch.float32, dev, optional=True)
    if hist_out is not None:
        _need(hist_out, "hist_out", (k + 1,), None, dev)
        if hist_out.dtype not in (torch.int64, torch.uint64):
            raise TypeError("hist_out must be int64 or uint64")
    _need_ws(ws, dev)
    desc = make_desc(T, d, N, k, 0, 0, _act_code(x), _idx_code(idx))
    if ws is None:
        ws = _new_ws(workspace_bytes(desc, OP_ROUTE_DIAG), dev, stream)
    check(lib().pr2_route_diagnostics(byref(desc), _ptr(x), _ptr(idx), ldi,
                                      _ptr(W_r), _ptr(b_r), _ptr(z_ref), _ptr(cur_idx_out),
                                      _ptr(overlap_out), _ptr(kl_out), _ptr(hist_out), _ptr(ws),
                                      ws.numel(), _stream(stream)))


def feature_cache_positions(T: int, Tc: int, seed: int):
    """pr2_feature_cache_positions: the retained positions as a numpy int64 array."""
    import numpy as np
    n = min(T, Tc)
    out = np.empty(max(n, 1), dtype=np.int64)
    got = lib().pr2_feature_cache_positions(T, Tc, seed & ((1 << 64) - 1),
                                            out.ctypes.data_as(c_void_p))
    if got < 0:
        raise Pr2Error(lib().pr2_last_error().decode())
    return out[:got]


def route_predict_cached(x, W_r, b_r, A, B, k, idx_out, cache_row, h_cache, p_cache,
                         gate_out=None, renorm=True, ws=None, stream=None):
    """pr2_route_predict_cached on torch tensors: ``cache_row`` int32 [T] on the device."""
    torch = _torch()
    T, d, adt, dev = _need_act(x)
    N = _router(W_r, b_r, d, dev)
    r = _predictor(A, B, d, N, dev)
    ldi = _need_ids(idx_out, "idx_out", T, k, dev)
    _need(gate_out, "gate_out", (T, k), torch.float32, dev, optional=True)
    _need(cache_row, "cache_row", (T,), torch.int32, dev)
    rows = h_cache.shape[0]
    _need(h_cache, "h_cache", (rows, d), adt, dev)
    _need(p_cache, "p_cache", (rows, N), torch.float32, dev)
    _need_ws(ws, dev)
    desc = make_desc(T, d, N, k, 0, r, _act_code(x), _idx_code(idx_out), renorm)
    if ws is None:
        ws = route_workspace(x, W_r, A, k, _idx_code(idx_out), stream)
    check(lib().pr2_route_predict_cached(byref(desc), _ptr(x), _ptr(W_r), _ptr(b_r), _ptr(A),
                                         _ptr(B), _ptr(idx_out), ldi,
                                         _ptr(gate_out), _ptr(cache_row), _ptr(h_cache),
                                         _ptr(p_cache), h_cache.shape[0], _ptr(ws), ws.numel(),
                                         _stream(stream)))


def predictor_loss(h, W_r, b_r, h_old, p_old, A, B, loss_out, dA, dB=None, kl_out=None,
                   loss_kind=0, mini_step=2, ws=None, stream=None):
    """pr2_predictor_loss on torch tensors (h, h_old [Tc, d]; p_old [Tc, N])."""
    torch = _torch()
    T, d, adt, dev = _need_act(h_old, "h_old")
    N = p_old.shape[1] if p_old.dim() == 2 else -1
    _need(p_old, "p_old", (T, N), torch.float32, dev)
    _need(h, "h", (T, d), adt, dev)
    _router(W_r, b_r, d, dev)
    if W_r.shape[1] != N:
        raise ValueError("W_r and p_old disagree on N")
    r = _predictor(A, B, d, N, dev)
    _need(loss_out, "loss_out", (1,), torch.float32, dev)
    _need(dA, "dA", (d, r), torch.float32, dev)
    if B is not None:
        _need(dB, "dB", (r, N), torch.float32, dev)
    _need(kl_out, "kl_out", (T,), torch.float32, dev, optional=True)
    _need_ws(ws, dev)
    desc = make_desc(T, d, N, 1, 0, r, _act_code(h_old))
    if ws is None:
        ws = _new_ws(workspace_bytes(desc, OP_PREDICTOR_LOSS), dev, stream)
    check(lib().pr2_predictor_loss(byref(desc), _ptr(h), _ptr(W_r), _ptr(b_r), _ptr(h_old),
                                   _ptr(p_old), _ptr(A), _ptr(B), loss_kind, mini_step,
                                   _ptr(kl_out), _ptr(loss_out), _ptr(dA), _ptr(dB), _ptr(ws),
                                   ws.numel(), _stream(stream)))


def backward_workspace(x, idx, W_r, W_gate, renorm=True, stream=None):
    T, d = x.shape
    desc = make_desc(T, d, W_r.shape[1], idx.shape[1], W_gate.shape[1], 0, _act_code(x),
                     _idx_code(idx), renorm)
    return _new_ws(workspace_bytes(desc, OP_REPLAY_BWD), x.device, stream)


def moe_replay_backward(x, idx, W_r, b_r, W_gate, W_up, W_down, dy, dx, dW_r, db_r, dW_gate,
                        dW_up, dW_down, ws=None, renorm=True, stream=None):
    """pr2_moe_replay_backward on torch tensors; every gradient tensor is overwritten.
    ``db_r`` may be None."""
    torch = _torch()
    T, d, adt, dev = _need_act(x)
    N = _router(W_r, b_r, d, dev)
    k = idx.shape[1] if idx.dim() == 2 else -1
    ldi = _need_ids(idx, "idx", T, k, dev)
    m = _experts(W_gate, W_up, W_down, N, d, adt, dev)
    _need(dy, "dy", (T, d), adt, dev)
    _need(dx, "dx", (T, d), adt, dev)
    _need(dW_r, "dW_r", (d, N), torch.float32, dev)
    _need(db_r, "db_r", (N,), torch.float32, dev, optional=True)
    _need(dW_gate, "dW_gate", (N, m, d), torch.float32, dev)
    _need(dW_up, "dW_up", (N, m, d), torch.float32, dev)
    _need(dW_down, "dW_down", (N, d, m), torch.float32, dev)
    _need_ws(ws, dev)
    desc = make_desc(T, d, N, k, m, 0, _act_code(x), _idx_code(idx), renorm)
    if ws is None:
        ws = backward_workspace(x, idx, W_r, W_gate, renorm, stream)
    check(lib().pr2_moe_replay_backward(byref(desc), _ptr(x), _ptr(idx), ldi,
                                        _ptr(W_r), _ptr(b_r), _ptr(W_gate), _ptr(W_up),
                                        _ptr(W_down), _ptr(dy), _ptr(dx), _ptr(dW_r), _ptr(db_r),
                                        _ptr(dW_gate), _ptr(dW_up), _ptr(dW_down), _ptr(ws),
                                        ws.numel(), _stream(stream)))


def moe_replay_backward_saved(x, idx, W_r, b_r, W_gate, W_up, W_down, au_saved, dy, dx, dW_r,
                              db_r, dW_gate, dW_up, dW_down, ws=None, renorm=True, stream=None):
    """pr2_moe_replay_backward_saved: the replay backward reading the pre-activations
    that moe_replay_forward_save wrote (``au_saved`` is only read)."""
    torch = _torch()
    T, d, adt, dev = _need_act(x)
    N = _router(W_r, b_r, d, dev)
    k = idx.shape[1] if idx.dim() == 2 else -1
    ldi = _need_ids(idx, "idx", T, k, dev)
    m = _experts(W_gate, W_up, W_down, N, d, adt, dev)
    _need(au_saved, "au_saved", (T * k, 2 * m), adt, dev)
    _need(dy, "dy", (T, d), adt, dev)
    _need(dx, "dx", (T, d), adt, dev)
    _need(dW_r, "dW_r", (d, N), torch.float32, dev)
    _need(db_r, "db_r", (N,), torch.float32, dev, optional=True)
    _need(dW_gate, "dW_gate", (N, m, d), torch.float32, dev)
    _need(dW_up, "dW_up", (N, m, d), torch.float32, dev)
    _need(dW_down, "dW_down", (N, d, m), torch.float32, dev)
    _need_ws(ws, dev)
    desc = make_desc(T, d, N, k, m, 0, _act_code(x), _idx_code(idx), renorm)
    if ws is None:
        ws = backward_workspace(x, idx, W_r, W_gate, renorm, stream)
    check(lib().pr2_moe_replay_backward_saved(byref(desc), _ptr(x), _ptr(idx), ldi, _ptr(W_r),
                                              _ptr(b_r), _ptr(W_gate), _ptr(W_up), _ptr(W_down),
                                              _ptr(au_saved), _ptr(dy), _ptr(dx), _ptr(dW_r),
                                              _ptr(db_r), _ptr(dW_gate), _ptr(dW_up),
                                              _ptr(dW_down), _ptr(ws), ws.numel(),
                                              _stream(stream)))


# ------------------------------------------------------ measurement hooks --

def profile_enable(on: bool = True):
    lib().pr2_profile_enable(1 if on else 0)


def profile_reset():
    lib().pr2_profile_reset()


def profile_collect(cap: int = 64) -> dict:
    """{kernel name: (total ms, launches)} since the last reset."""
    names = (c_char_p * cap)()
    ms = (c_double * cap)()
    n_l = (c_int64 * cap)()
    n = lib().pr2_profile_collect(names, ms, n_l, cap)
    if n < 0:
        raise RuntimeError("pr2_profile_collect failed")
    return {names[i].decode(): (ms[i], int(n_l[i])) for i in range(min(n, cap))}
