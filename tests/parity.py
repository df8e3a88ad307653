"""Shared helpers of the GPU parity tests: device upload and the comparison
rules between the HIP path and the float64 oracle.

Rules (for every test that compares the two):
* route ids: bit-exact, except tokens whose k-th/(k+1)-th predictive-logit
  margin (float64, from the oracle) is below 1e-6; those are counted and
  reported, and excluded from the id and gate checks;
* replayed ids are never re-derived, so anything computed from them is
  compared on every token;
* gates: |g - g_ref| <= 1e-5 * g_ref elementwise (fp32);
* outputs: per-token relative L2 error ||y - y_ref|| / ||y_ref|| <= 2e-2 for
  bf16 activations and <= 1e-5 for fp32 activations.
"""
from __future__ import annotations

import numpy as np

MARGIN_EPS = 1e-6
GATE_RTOL = 1e-5
Y_RTOL = {"bf16": 2e-2, "f32": 1e-5}


def torch_mod():
    import torch
    return torch


def to_dev(a, act="f32"):
    """float32 numpy -> cuda tensor (bf16 values are exactly representable)."""
    torch = torch_mod()
    if a is None:
        return None
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if act == "bf16":
        t = t.to(torch.bfloat16)
    return t.to("cuda")


def compare_route(idx_gpu, gate_gpu, ref, k, where=""):
    """Returns the number of margin-excluded tokens; asserts on the rest."""
    idx_gpu = np.asarray(idx_gpu, dtype=np.int64)
    excl = ref["margin"] < MARGIN_EPS
    ok = ~excl
    bad = np.nonzero(ok & np.any(idx_gpu != ref["idx"], axis=1))[0]
    assert len(bad) == 0, (f"{where}: {len(bad)} token routes differ outside the margin rule; "
                           f"first {bad[:5]}: gpu {idx_gpu[bad[:3]]}, oracle {ref['idx'][bad[:3]]}, "
                           f"margin {ref['margin'][bad[:3]]}")
    if gate_gpu is not None:
        g = np.asarray(gate_gpu, dtype=np.float64)[ok]
        gr = ref["gate"][ok]
        rel = np.abs(g - gr) / gr
        assert rel.max(initial=0.0) <= GATE_RTOL, f"{where}: gate rel err {rel.max():.3e}"
    return int(excl.sum())


def compare_gates(gate_gpu, gate_ref, where=""):
    g = np.asarray(gate_gpu, dtype=np.float64)
    rel = np.abs(g - gate_ref) / np.abs(gate_ref)
    assert rel.max(initial=0.0) <= GATE_RTOL, f"{where}: gate rel err {rel.max():.3e}"


def row_rel_err(y_gpu, y_ref):
    y = np.asarray(y_gpu, dtype=np.float64)
    num = np.linalg.norm(y - y_ref, axis=1)
    den = np.linalg.norm(y_ref, axis=1)
    return num / np.maximum(den, 1e-300)


def compare_rows(y_gpu, y_ref, act, where=""):
    rel = row_rel_err(y_gpu, y_ref)
    tol = Y_RTOL[act]
    worst = int(np.argmax(rel)) if rel.size else 0
    assert rel.max(initial=0.0) <= tol, (f"{where}: worst row {worst} rel err {rel.max():.3e} > "
                                         f"{tol}")
    return float(rel.max(initial=0.0))
