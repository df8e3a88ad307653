"""Benchmark of the Pr^2 MoE-layer hot path on one MI355X.

One step = route prediction (router + rank-r evolution predictor, top-k,
route record) followed by the replay forward of the recorded route (replay
weights, permutation, grouped SwiGLU expert GEMMs, combine) over one batch of
synthetic tokens already resident in HBM.  Prints ONE JSON line.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "MoE-layer tokens/sec (predictive route + replay forward); MFMA util; HBM GB/s"
DOMINANT = "gemm1_gate_up_swiglu"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="qwen3_30b_T16384")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-tokens", type=int, default=0,
                    help="tokens of the oracle's CPU sample (0: whole workload)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="first run a plain device copy of this many MiB (a known-size "
                         "kernel for scaling memory-traffic counters)")
    return ap.parse_args()


def profiled_traffic(workload, kernel="grouped_gemm_mfma<0>"):
    """HBM bytes per launch of the dominant kernel from the committed rocprofv3
    summary (FETCH_SIZE + WRITE_SIZE, copy-calibrated), or None when there is
    no summary for this workload or the kernel source changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"replay_and_route_kernels_{workload}.txt")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"gemm_source_sha256: ([0-9a-f]+)", text)
    src = os.path.join(ROOT, "paper_2606_00395_amd", "csrc", "gemm.hip")
    cur = hashlib.sha256(open(src, "rb").read()).hexdigest()
    if not m or m.group(1) != cur:
        return None
    m = re.search(r"traffic_bytes_per_launch\[" + re.escape(kernel) + r"\]: fetch (\d+) write (\d+)",
                  text)
    return int(m.group(1)) + int(m.group(2)) if m else None


def cpu_baseline(shape, L, n_tok, min_seconds=10.0):
    """The float64 oracle (route + replay forward) on the first n_tok tokens,
    repeated until at least min_seconds of CPU time have been measured."""
    import numpy as np
    from oracle import pr2_oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()
                       if p.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        threads = int(os.environ.get("OMP_NUM_THREADS", "1"))
    x = L["x"][:n_tok]
    reps = 0
    t0 = time.perf_counter()
    while True:
        rt = O.route_predict(x, L["W_r"], L["beta"], L["A"], L["B"], shape.k)
        O.replay_forward(x, rt["idx"], L["W_r"], L["beta"], L["W_gate"], L["W_up"], L["W_down"])
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    del np
    return {"value": reps * n_tok / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{n_tok} of {shape.T} tokens of {shape.name}, float64 route prediction "
                      f"+ replay forward, {reps} pass(es) in {dt:.1f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); this build has no "
              "multi-GPU path", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import workloads as W
    from paper_2606_00395_amd import binding as B
    from paper_2606_00395_amd import costmodel as C

    shape = W.WORKLOADS[args.workload]
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    L = W.layer_inputs(shape, args.seed)
    tdt = torch.bfloat16 if shape.act == "bf16" else torch.float32

    def up(a, act=False):
        if a is None:
            return None
        t = torch.from_numpy(a)
        return (t.to(tdt) if act else t).to(dev)

    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    x = up(L["x"], True)
    Wr, br, A, Bm = up(L["W_r"]), up(L["beta"]), up(L["A"]), up(L["B"])
    Wg, Wu, Wd = up(L["W_gate"], True), up(L["W_up"], True), up(L["W_down"], True)
    T, d, N, k, m, r = shape.T, shape.d, shape.N, shape.k, shape.m, shape.r
    idt = torch.int16 if shape.idx_dtype == "int16" else torch.int32
    idx = torch.empty((T, k), dtype=idt, device=dev)
    gate_roll = torch.empty((T, k), dtype=torch.float32, device=dev)
    gate_rep = torch.empty((T, k), dtype=torch.float32, device=dev)
    y = torch.empty((T, d), dtype=tdt, device=dev)
    ws = B.replay_workspace(x, idx, Wr, Wg)
    stream = torch.cuda.current_stream()

    def step():
        B.route_predict(x, Wr, br, A, Bm, k, idx, gate_roll, stream=stream)
        B.moe_replay_forward(x, idx, Wr, br, Wg, Wu, Wd, y, gate_rep, ws=ws, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K steps, synchronised on both sides
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps

    # the same K steps with every kernel bracketed by events on its own stream
    B.profile_enable(True)
    B.profile_reset()
    torch.cuda.synchronize()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    prof = B.profile_collect()
    B.profile_enable(False)
    kern = {name: tot / n for name, (tot, n) in prof.items()}   # ms per launch

    ab = 2 if shape.act == "bf16" else 4
    ib = 2 if shape.idx_dtype == "int16" else 4
    f_g1 = C.gemm1_flops(T, d, k, m)
    f_g2 = C.gemm2_flops(T, d, k, m)
    t_g1 = kern.get(DOMINANT, float("nan"))
    t_g2 = kern.get("gemm2_down_scale", float("nan"))
    t_route = kern.get("route_predict", float("nan"))
    t_gates = kern.get("replay_gates", float("nan"))
    t_comb = kern.get("combine", float("nan"))
    t_perm = sum(kern.get(n, 0.0) for n in ("perm_count", "perm_scan", "perm_scatter"))
    t_replay = sum(v for n, v in kern.items() if n != "route_predict")
    achieved = f_g1 / (t_g1 * 1e-3) / 1e12
    peak = C.PEAK_BF16_FLOPS / 1e12
    out = {
        "metric": METRIC,
        "value": T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if shape.act == "bf16" else "f32",
        "data": "synthetic (seeded N(0,1) tokens, N(0,0.02) weights; see workloads/)",
        "config": {"workload": shape.name, "tokens": T, "hidden": d, "experts": N, "top_k": k,
                   "expert_intermediate": m, "predictor_rank": r, "router": "fp32",
                   "idx_dtype": shape.idx_dtype, "load_skew": shape.skew},
        "roofline": {"bound": "mfma", "kernel": DOMINANT, "achieved": achieved, "peak": peak,
                     "unit": "TFLOP/s", "frac": achieved / peak,
                     "traffic": profiled_traffic(shape.name)},
        "kernels_ms": {n: round(v, 5) for n, v in kern.items()},
        "replay_forward": {
            "ms": t_replay,
            "mfma_frac_whole_layer": C.expert_flops(T, d, k, m) / (t_replay * 1e-3) / C.PEAK_BF16_FLOPS,
            "mfma_frac_gemm1": f_g1 / (t_g1 * 1e-3) / C.PEAK_BF16_FLOPS,
            "mfma_frac_gemm2": f_g2 / (t_g2 * 1e-3) / C.PEAK_BF16_FLOPS,
        },
        "hbm_gbps": {
            "route_predict": C.route_bytes(T, d, N, r, k, ab, ib) / (t_route * 1e-3) / 1e9,
            "replay_gates": C.replay_gate_bytes(T, d, N, k, ab, ib) / (t_gates * 1e-3) / 1e9,
            "combine": C.combine_bytes(T, d, k, ab, ab) / (t_comb * 1e-3) / 1e9,
            "permute_ms": t_perm,
        },
    }
    if not args.no_cpu_baseline:
        n_tok = args.cpu_sample_tokens if args.cpu_sample_tokens > 0 else T
        out["cpu_baseline"] = cpu_baseline(shape, L, min(n_tok, T))
    del np
    print(json.dumps(out))


if __name__ == "__main__":
    main()
