"""Benchmark of the Pr^2 MoE-layer hot path on one MI355X.

Default (``--mode forward``): one step = route prediction (router + rank-r
evolution predictor, top-k, route record) followed by the replay forward of
the recorded route (replay weights, permutation, grouped SwiGLU expert GEMMs,
combine) over one batch of synthetic tokens already resident in HBM.

``--mode backward``: one step = the replay backward of a recorded route (the
rollout route of the same layer, which differs from the current router's
top-k on some tokens): gradients of x, the experts and the router.

``--mode next``: the method's other per-layer calls on the same layer and
batch, each timed on its own: the rollout-phase layer output under the
predictive gates (the step whose tokens/s is reported), the route with the
feature-cache write of 2048 sub-sampled positions, the predictive KL loss and
its delta-matching variant with dA, dB over those positions, and the route
diagnostics (current top-k, overlap, deviation histogram, route KL).

``--mode decode``: the decode-style rollout of 256 sequences x 2048 steps, each
step's route written into an index-stable int16 record, timed per step both
as separate launches and replayed from one captured HIP graph, then the replay
forward of 32768-token micro-batches of the record (tokens/s is for those).

Prints ONE JSON line.

    python bench.py [--mode forward|backward|decode|next] [--steps K] [--warmup W]
                    [--workload NAME] [--no-cpu-baseline]
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
DEFAULT_WORKLOAD = {"forward": "qwen3_30b_T16384", "backward": "qwen3_30b_bwd_T16384",
                    "decode": "qwen3_30b_decode_256x2048", "next": "qwen3_30b_T16384"}
FEATURE_CACHE_POSITIONS = 2048      # cached positions per 16384-token response (App. E.2)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--mode", choices=("forward", "backward", "decode", "next"), default="forward")
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=50,
                    help="untimed steps first (the clock ramps up over the first ~10 ms)")
    ap.add_argument("--workload", default=None)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="forward mode: skip the other workloads (235B forward, backward, "
                         "decode, the method's other calls) that follow the headline")
    ap.add_argument("--cpu-sample-tokens", type=int, default=0,
                    help="tokens of the oracle's CPU sample (0: the mode's default)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="first run a plain device copy of this many MiB (a known-size "
                         "kernel for scaling memory-traffic counters)")
    return ap.parse_args()


def kernel_source_hash(names):
    """sha256 over the given kernel source files of csrc/, in order."""
    h = hashlib.sha256()
    for name in names:
        h.update(open(os.path.join(ROOT, "paper_2606_00395_amd", "csrc", name), "rb").read())
    return h.hexdigest()


def profiled_traffic(profile, kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 summary
    `profiles/<profile>` (FETCH_SIZE + WRITE_SIZE, copy-calibrated), or None
    when there is no such summary or a source it names changed since it was
    taken."""
    path = os.path.join(ROOT, "profiles", profile)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    srcs = re.search(r"kernel_sources: (.+)", text)
    m = re.search(r"kernel_source_sha256: ([0-9a-f]+)", text)
    if not srcs or not m or m.group(1) != kernel_source_hash(srcs.group(1).split()):
        return None
    m = re.search(r"traffic_bytes_per_launch\[" + re.escape(kernel) + r"\]: fetch (\d+) write (\d+)",
                  text)
    return int(m.group(1)) + int(m.group(2)) if m else None


def gemm1_kernel(m):
    """The gate/up GEMM kernel the library launches for expert width m (its
    name in the rocprofv3 summaries)."""
    return "gemm1_wide" if m % 192 == 0 else "grouped_gemm_mfma<0>"


def profiled_counters(profile, kernel):
    """The SQ counter figures (mfma_busy, lds_conflict_per_inst, ...) that the
    committed summary `profiles/<profile>` holds for `kernel`, or None when the
    summary is missing or its sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", profile)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    srcs = re.search(r"kernel_sources: (.+)", text)
    m = re.search(r"kernel_source_sha256: ([0-9a-f]+)", text)
    if not srcs or not m or m.group(1) != kernel_source_hash(srcs.group(1).split()):
        return None
    m = re.search(r"counters\[" + re.escape(kernel) + r"\]: (.+)", text)
    if not m:
        return None
    vals = m.group(1).split()
    return {vals[i]: float(vals[i + 1]) for i in range(0, len(vals) - 1, 2)}


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([p.get("num_threads", 1) for p in threadpool_info()
                    if p.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        return int(os.environ.get("OMP_NUM_THREADS", "1"))


def host_info():
    """CPU model and the number of CPUs this process may run on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    return {"cpu_model": model, "affinity_cpus": len(os.sched_getaffinity(0))}


def timed_cpu(fn, n_tok, min_seconds):
    reps = 0
    t0 = time.perf_counter()
    while True:
        fn()
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            return reps, dt


def cpu_baseline_forward(shape, L, n_tok, min_seconds=10.0):
    """The float64 oracle (route + replay forward) on the first n_tok tokens,
    repeated until at least min_seconds of CPU time have been measured."""
    from oracle import pr2_oracle as O
    x = L["x"][:n_tok]

    def run():
        rt = O.route_predict(x, L["W_r"], L["beta"], L["A"], L["B"], shape.k)
        O.replay_forward(x, rt["idx"], L["W_r"], L["beta"], L["W_gate"], L["W_up"], L["W_down"])
    reps, dt = timed_cpu(run, n_tok, min_seconds)
    return {"value": reps * n_tok / dt, "unit": "tokens/s", "cores": blas_threads(),
            "kind": "oracle", "host": host_info(),
            "sample": f"{n_tok} of {shape.T} tokens of {shape.name}, float64 route prediction "
                      f"+ replay forward, {reps} pass(es) in {dt:.1f} s"}


def cpu_baseline_backward(shape, L, idx, dy, n_tok, min_seconds=10.0):
    from oracle import pr2_oracle as O
    x = L["x"][:n_tok]

    def run():
        O.replay_backward(x, idx[:n_tok], L["W_r"], L["beta"], L["W_gate"], L["W_up"],
                          L["W_down"], dy[:n_tok])
    reps, dt = timed_cpu(run, n_tok, min_seconds)
    return {"value": reps * n_tok / dt, "unit": "tokens/s", "cores": blas_threads(),
            "kind": "oracle", "host": host_info(),
            "sample": f"{n_tok} of {shape.T} tokens of {shape.name}, float64 replay backward, "
                      f"{reps} pass(es) in {dt:.1f} s"}


def measured_peaks(dev):
    """A plain 1 GiB device copy (GB/s, read + write) and a dense 8192^3 bf16
    library GEMM (TFLOP/s), as this GPU runs them now: context for the
    published peaks the rooflines use."""
    import torch
    n = 1 << 28
    a = torch.ones(n, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    m = 8192
    x = torch.randn(m, m, dtype=torch.bfloat16, device=dev)
    w = torch.randn(m, m, dtype=torch.bfloat16, device=dev)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    out = {}
    for name, fn, work in (("copy_gbps", lambda: b.copy_(a), 2 * 4 * n / 1e9),
                           ("library_gemm_bf16_tflops", lambda: torch.matmul(x, w),
                            2 * m ** 3 / 1e12)):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(10):
            fn()
        e1.record()
        torch.cuda.synchronize()
        out[name] = work / (e0.elapsed_time(e1) / 10 * 1e-3)
    del a, b, x, w
    return out


def cpu_baseline_small_1thread(min_seconds=2.0):
    """The oracle on the 256-token fp32 configuration with one BLAS thread."""
    import workloads as W
    from oracle import pr2_oracle as O
    s = W.WORKLOADS["tiny_fp32_T256"]
    L = W.layer_inputs(s, 0)
    import contextlib
    try:
        from threadpoolctl import threadpool_limits
        ctx = threadpool_limits(limits=1, user_api="blas")
    except ImportError:  # pragma: no cover
        ctx = contextlib.nullcontext()

    def run():
        rt = O.route_predict(L["x"], L["W_r"], L["beta"], L["A"], L["B"], s.k)
        O.replay_forward(L["x"], rt["idx"], L["W_r"], L["beta"], L["W_gate"], L["W_up"],
                         L["W_down"])
    with ctx:
        reps, dt = timed_cpu(run, s.T, min_seconds)
    return {"value": reps * s.T / dt, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"{s.name}: float64 route prediction + replay forward, {reps} pass(es) "
                      f"in {dt:.1f} s"}


def cpu_baseline_rollout(shape, L, n_tok, min_seconds=10.0):
    from oracle import pr2_oracle as O
    x = L["x"][:n_tok]

    def run():
        O.rollout_forward(x, L["W_r"], L["beta"], L["A"], L["B"], shape.k, L["W_gate"],
                          L["W_up"], L["W_down"])
    reps, dt = timed_cpu(run, n_tok, min_seconds)
    return {"value": reps * n_tok / dt, "unit": "tokens/s", "cores": blas_threads(),
            "kind": "oracle", "host": host_info(),
            "sample": f"{n_tok} of {shape.T} tokens of {shape.name}, float64 rollout forward "
                      f"(route prediction + layer output under the predictive gates), {reps} "
                      f"pass(es) in {dt:.1f} s"}


def cpu_baseline_decode(shape, L, min_seconds=10.0):
    from oracle import pr2_oracle as O
    import workloads as W
    xs = [W.decode_step_states(shape, 0, s) for s in range(8)]
    i = [0]

    def run():
        O.route_predict(xs[i[0] % 8], L["W_r"], L["beta"], L["A"], L["B"], shape.k)
        i[0] += 1
    reps, dt = timed_cpu(run, W.DECODE_SEQS, min_seconds)
    return {"value": reps * W.DECODE_SEQS / dt, "unit": "routed tokens/s",
            "cores": blas_threads(), "kind": "oracle", "host": host_info(),
            "sample": f"{reps} decode steps of {W.DECODE_SEQS} tokens, float64 route prediction, "
                      f"in {dt:.1f} s"}


def timed_steps(step, steps, warmup, stream, B):
    """Mean ms per step over `steps` synchronised steps, then the same steps with
    every kernel bracketed by HIP events on its stream (ms per launch by name)."""
    import torch
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    # the same steps each between its own pair of events, for the median
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    for a, b in evs:
        a.record(stream)
        step()
        b.record(stream)
    torch.cuda.synchronize()
    per = sorted(a.elapsed_time(b) for a, b in evs)
    timed_steps.median_ms = per[len(per) // 2] if len(per) % 2 else 0.5 * (
        per[len(per) // 2 - 1] + per[len(per) // 2])
    B.profile_enable(True)
    B.profile_reset()
    torch.cuda.synchronize()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    prof = B.profile_collect()
    B.profile_enable(False)
    return ms, {name: tot / n for name, (tot, n) in prof.items()}


def cold_ms_per_step(step, steps, stream):
    """Mean ms per step when every step follows a 512 MiB device write, which
    evicts the L2s and the 256 MB last-level cache (inputs come from HBM)."""
    import torch
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    total = 0.0
    for _ in range(steps):
        scratch.fill_(1)
        e0.record(stream)
        step()
        e1.record(stream)
        torch.cuda.synchronize()
        total += e0.elapsed_time(e1)
    del scratch
    return total / steps


def graph_ms_per_step(step_on, steps, warmup=20):
    """Mean ms per step when the step's launches are captured once into a HIP
    graph and replayed (no host work or launch gaps between kernels).  The
    first replays after instantiation run slower (measured: 1.565 ms against
    1.478 ms later on the Qwen3-30B step), so the graph is warmed up like the
    eager path before it is timed."""
    import torch
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step_on(torch.cuda.current_stream())
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    st = torch.cuda.current_stream()
    e0.record(st)
    for _ in range(steps):
        graph.replay()
    e1.record(st)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def base_record(args, metric, value, unit, ms, dtype, config):
    return {"metric": metric, "value": value, "unit": unit, "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": dtype,
            "data": "synthetic (seeded N(0,1) tokens, N(0,0.02) weights; see workloads/)",
            "config": config}


def layer_config(shape):
    return {"workload": shape.name, "tokens": shape.T, "hidden": shape.d, "experts": shape.N,
            "top_k": shape.k, "expert_intermediate": shape.m, "predictor_rank": shape.r,
            "router": "fp32", "idx_dtype": shape.idx_dtype, "load_skew": shape.skew}


def upload(L, shape, dev):
    import torch
    tdt = torch.bfloat16 if shape.act == "bf16" else torch.float32

    def up(a, act=False):
        if a is None:
            return None
        t = torch.from_numpy(a)
        return (t.to(tdt) if act else t).to(dev)
    out = {n: up(L[n]) for n in ("W_r", "beta", "A", "B")}
    out["x"] = up(L["x"], True)
    for n in ("W_gate", "W_up", "W_down"):
        if n in L:
            out[n] = up(L[n], True)
    return out, up


def run_forward(args, shape, dev):
    import torch
    import workloads as W
    from paper_2606_00395_amd import binding as B
    from paper_2606_00395_amd import costmodel as C
    L = W.layer_inputs(shape, args.seed)
    G, _ = upload(L, shape, dev)
    T, d, N, k, m, r = shape.T, shape.d, shape.N, shape.k, shape.m, shape.r
    idt = torch.int16 if shape.idx_dtype == "int16" else torch.int32
    idx = torch.empty((T, k), dtype=idt, device=dev)
    gate_roll = torch.empty((T, k), dtype=torch.float32, device=dev)
    gate_rep = torch.empty((T, k), dtype=torch.float32, device=dev)
    y = torch.empty_like(G["x"])
    ws = B.replay_workspace(G["x"], idx, G["W_r"], G["W_gate"])
    ws_r = B.route_workspace(G["x"], G["W_r"], G["A"], k, B.PR2_I16 if shape.idx_dtype == "int16"
                             else B.PR2_I32)
    stream = torch.cuda.current_stream()

    def step_on(st):
        B.route_predict(G["x"], G["W_r"], G["beta"], G["A"], G["B"], k, idx, gate_roll, ws=ws_r,
                        stream=st)
        B.moe_replay_forward(G["x"], idx, G["W_r"], G["beta"], G["W_gate"], G["W_up"],
                             G["W_down"], y, gate_rep, ws=ws, stream=st)

    def step():
        step_on(stream)

    ms, kern = timed_steps(step, args.steps, args.warmup, stream, B)
    median = timed_steps.median_ms
    light = getattr(args, "light", False)
    if not light:
        ms_graph = graph_ms_per_step(step_on, args.steps)
        ms_cold = cold_ms_per_step(step, args.steps, stream)
    ab = 2 if shape.act == "bf16" else 4
    ib = 2 if shape.idx_dtype == "int16" else 4
    dominant = "gemm1_gate_up_swiglu"
    f_g1 = C.gemm1_flops(T, d, k, m)
    f_g2 = C.gemm2_flops(T, d, k, m)
    t_g1 = kern.get(dominant, float("nan"))
    t_g2 = kern.get("gemm2_down_scale", float("nan"))
    t_route = kern.get("route_predict", float("nan"))
    t_gates = kern.get("replay_gates", float("nan"))
    t_comb = kern.get("combine", float("nan"))
    t_perm = sum(kern.get(n, 0.0) for n in ("perm_count", "perm_scan", "perm_scatter"))
    t_replay = sum(v for n, v in kern.items() if n != "route_predict")
    achieved = f_g1 / (t_g1 * 1e-3) / 1e12
    peak = C.PEAK_BF16_FLOPS / 1e12
    out = base_record(args, METRIC, T / (ms * 1e-3), "tokens/s", ms,
                      "bf16" if shape.act == "bf16" else "f32", layer_config(shape))
    out["roofline"] = {"bound": "mfma", "kernel": dominant, "achieved": achieved, "peak": peak,
                       "unit": "TFLOP/s", "frac": achieved / peak,
                       "traffic": profiled_traffic(f"replay_and_route_kernels_{shape.name}.txt",
                                                  gemm1_kernel(shape.m))}
    if not light:
        out["hip_graph"] = {"ms_per_step": ms_graph, "value": T / (ms_graph * 1e-3),
                            "note": "the same step captured once and replayed as a HIP graph"}
        out["cold_cache"] = {"ms_per_step": ms_cold, "value": T / (ms_cold * 1e-3),
                             "note": "each step after a 512 MiB device write that evicts L2 "
                                     "and the 256 MB last-level cache"}
    out["ms_per_step_median"] = median
    out["kernels_ms"] = {n: round(v, 5) for n, v in kern.items()}
    if not light:
        out["measured_peaks"] = mp = measured_peaks(dev)
        # the gate/up GEMM's rate over the library's dense square GEMM, same GPU, same run
        mp["gemm1_over_library_gemm"] = (f_g1 / (t_g1 * 1e-3) / 1e12) / mp["library_gemm_bf16_tflops"]
    out["replay_forward"] = {
        "ms": t_replay,
        "mfma_frac_whole_layer": C.expert_flops(T, d, k, m) / (t_replay * 1e-3) / C.PEAK_BF16_FLOPS,
        "mfma_frac_gemm1": f_g1 / (t_g1 * 1e-3) / C.PEAK_BF16_FLOPS,
        "mfma_frac_gemm2": f_g2 / (t_g2 * 1e-3) / C.PEAK_BF16_FLOPS,
    }
    out["hbm_gbps"] = {
        "route_predict": C.route_bytes(T, d, N, r, k, ab, ib) / (t_route * 1e-3) / 1e9,
        "replay_gates": C.replay_gate_bytes(T, d, N, k, ab, ib) / (t_gates * 1e-3) / 1e9,
        "combine": C.combine_bytes(T, d, k, ab, ab) / (t_comb * 1e-3) / 1e9,
        "permute_ms": t_perm,
        "note": "algorithmic bytes / event-timed duration",
    }
    # the same kernels' HBM bytes as rocprofv3's FETCH_SIZE + WRITE_SIZE counters read
    # them (copy-calibrated, from the committed summary of this source), over the
    # durations measured here
    prof = f"replay_and_route_kernels_{shape.name}.txt"
    cg = {}
    for key, kname, t_ms in (("route_predict", "router_mfma_kernel<2, 0, 0>", t_route),
                             ("replay_gates", "router_mfma_kernel<2, 1, 0>", t_gates),
                             ("perm_count", "perm_count_kernel", kern.get("perm_count")),
                             ("perm_scan", "perm_scan_kernel", kern.get("perm_scan")),
                             ("perm_scatter", "perm_scatter_kernel", kern.get("perm_scatter")),
                             ("combine", "combine_bf16_kernel", t_comb)):
        b = profiled_traffic(prof, kname)
        if b is not None and t_ms:
            cg[key] = {"bytes": b, "gbps": b / (t_ms * 1e-3) / 1e9,
                       "frac_of_8tbs": b / (t_ms * 1e-3) / C.PEAK_HBM_BYTES}
    out["hbm_gbps_counters"] = cg or None
    out["mfma_busy_counters"] = {
        key: (profiled_counters(prof, kname) or {}).get("mfma_busy")
        for key, kname in (("gemm1_gate_up_swiglu", gemm1_kernel(shape.m)),
                           ("gemm2_down_scale", "grouped_gemm_mfma<1>"),
                           ("route_predict", "router_mfma_kernel<2, 0, 0>"))}
    out["mfma_busy_counters"]["note"] = ("SQ_VALU_MFMA_BUSY_CYCLES / (4 SIMDs x SQ_BUSY_CU_CYCLES) "
                                         "from the committed rocprofv3 summary of these sources")
    if not args.no_cpu_baseline:
        n_tok = args.cpu_sample_tokens if args.cpu_sample_tokens > 0 else T
        out["cpu_baseline"] = cpu_baseline_forward(shape, L, min(n_tok, T))
        out["cpu_baseline_small_1thread"] = cpu_baseline_small_1thread()
    return out


def recorded_flip_route(G, shape, seed, dev):
    """The backward workload's recorded route: the current router's top-k (this
    library's router, no predictor) with flip_frac of the tokens recording the
    (k+1)-th ranked expert in place of the k-th (workloads.flip_route).  The
    ranking of each token's k+1 ids is read off the router's fp32 logits."""
    import numpy as np
    import torch
    import workloads as W
    from paper_2606_00395_amd import binding as B
    T, N, k = shape.T, shape.N, shape.k
    top = torch.empty((T, k + 1), dtype=torch.int32, device=dev)
    p = torch.empty((T, N), dtype=torch.float32, device=dev)
    B.route_predict(G["x"], G["W_r"], G["beta"], None, None, k + 1, top, logits_out=p)
    top_np = top.cpu().numpy().astype(np.int64)
    lg = np.take_along_axis(p.cpu().numpy(), top_np, axis=1)
    # best first; equal logits keep the lower id first (the ids are ascending)
    order = np.argsort(-lg, axis=1, kind="stable")
    ranked = np.take_along_axis(top_np, order, axis=1)
    idx = W.flip_route(ranked, W.flip_tokens(shape, seed), k)
    return torch.from_numpy(idx.astype(np.int32)).to(dev)


def run_backward(args, shape, dev):
    import torch
    import workloads as W
    from paper_2606_00395_amd import binding as B
    from paper_2606_00395_amd import costmodel as C
    L = W.layer_inputs(shape, args.seed)
    G, up = upload(L, shape, dev)
    dy_np = W.upstream_grad(shape, args.seed)
    dy = up(dy_np, True)
    T, d, N, k, m = shape.T, shape.d, shape.N, shape.k, shape.m
    idx = recorded_flip_route(G, shape, args.seed, dev)
    dx = torch.empty_like(G["x"])
    dWr = torch.empty_like(G["W_r"])
    dbr = torch.empty_like(G["beta"])
    dWg = torch.empty(G["W_gate"].shape, device=dev)
    dWu = torch.empty(G["W_up"].shape, device=dev)
    dWd = torch.empty(G["W_down"].shape, device=dev)
    ws = B.backward_workspace(G["x"], idx, G["W_r"], G["W_gate"])
    stream = torch.cuda.current_stream()

    def step():
        B.moe_replay_backward(G["x"], idx, G["W_r"], G["beta"], G["W_gate"], G["W_up"],
                              G["W_down"], dy, dx, dWr, dbr, dWg, dWu, dWd, ws=ws, stream=stream)

    ms, kern = timed_steps(step, args.steps, args.warmup, stream, B)
    flops = {"bwd_preact_gate_up": 4, "bwd_dh_swiglu": 2, "bwd_dx_gemm": 4, "bwd_wgrad_down": 2,
             "bwd_wgrad_gate_up": 4}
    unit = T * k * d * m
    dominant = "bwd_wgrad_gate_up"
    achieved = flops[dominant] * unit / (kern[dominant] * 1e-3) / 1e12
    peak = C.PEAK_BF16_FLOPS / 1e12
    out = base_record(args, "MoE-layer tokens/sec (replay backward: dx, expert and router grads)",
                      T / (ms * 1e-3), "tokens/s", ms, "bf16", layer_config(shape))
    out["roofline"] = {"bound": "mfma", "kernel": dominant, "achieved": achieved, "peak": peak,
                       "unit": "TFLOP/s", "frac": achieved / peak,
                       "traffic": profiled_traffic(f"replay_backward_kernels_{shape.name}.txt",
                                                   "bwd_gemm<3>")}
    out["kernels_ms"] = {n: round(v, 5) for n, v in kern.items()}
    out["mfma_frac"] = {n: f * unit / (kern[n] * 1e-3) / C.PEAK_BF16_FLOPS
                        for n, f in flops.items() if n in kern}
    out["mfma_frac_whole_backward"] = 16 * unit / (ms * 1e-3) / C.PEAK_BF16_FLOPS
    out["recorded_route"] = ("the current router's top-k with the k-th ranked expert swapped for "
                             f"the (k+1)-th on {int(round(shape.flip_frac * T))} tokens")
    # the printed weights (rho_j of the softmax over all N): the logit gradient
    # is dense over N, so the router gradient and the router term of dx cover
    # every expert
    ws_lit = B.backward_workspace(G["x"], idx, G["W_r"], G["W_gate"], renorm=False)

    def literal_step():
        B.moe_replay_backward(G["x"], idx, G["W_r"], G["beta"], G["W_gate"], G["W_up"],
                              G["W_down"], dy, dx, dWr, dbr, dWg, dWu, dWd, ws=ws_lit,
                              renorm=False, stream=stream)

    ms_lit, kern_lit = timed_steps(literal_step, args.steps, args.warmup, stream, B)
    del ws_lit
    out["paper_literal_weights"] = {"ms": ms_lit, "value": T / (ms_lit * 1e-3),
                                    "kernels_ms": {n: round(v, 5) for n, v in kern_lit.items()}}
    out["training_pass"] = training_pass(args, G, idx, dy, (dx, dWr, dbr, dWg, dWu, dWd), ws,
                                         step, stream)
    if not args.no_cpu_baseline:
        idx_np = idx.cpu().numpy()
        n_tok = args.cpu_sample_tokens if args.cpu_sample_tokens > 0 else 1024
        out["cpu_baseline"] = cpu_baseline_backward(shape, L, idx_np, dy_np, min(n_tok, T))
    return out


def training_pass(args, G, idx, dy, grads, bws, backward_step, stream):
    """The replay forward followed by its backward (one training pass of the MoE
    layer under the recorded route), two ways: the backward recomputing the
    experts' gate / up pre-activations, and the forward saving them for the
    backward (2 m activation values per route held between the passes)."""
    import torch
    from paper_2606_00395_amd import binding as B
    T, k = idx.shape
    m = G["W_gate"].shape[1]
    x = G["x"]
    y = torch.empty_like(x)
    gate = torch.empty((T, k), dtype=torch.float32, device=x.device)
    au = torch.empty((T * k, 2 * m), dtype=x.dtype, device=x.device)
    fws = B.replay_workspace(x, idx, G["W_r"], G["W_gate"])
    experts = (G["W_gate"], G["W_up"], G["W_down"])

    def recompute():
        B.moe_replay_forward(x, idx, G["W_r"], G["beta"], *experts, y, gate, ws=fws,
                             stream=stream)
        backward_step()

    def saved():
        B.moe_replay_forward_save(x, idx, G["W_r"], G["beta"], *experts, y, au, gate, ws=fws,
                                  stream=stream)
        B.moe_replay_backward_saved(x, idx, G["W_r"], G["beta"], *experts, au, dy, *grads,
                                    ws=bws, stream=stream)

    ms_r, kern_r = timed_steps(recompute, args.steps, args.warmup, stream, B)
    ms_s, kern_s = timed_steps(saved, args.steps, args.warmup, stream, B)
    del au, fws
    return {"forward_then_backward_ms": ms_r, "with_saved_preactivations_ms": ms_s,
            "saved_bytes": T * k * 2 * m * x.element_size(),
            "kernels_ms_recompute": {n: round(v, 5) for n, v in kern_r.items()},
            "kernels_ms_saved": {n: round(v, 5) for n, v in kern_s.items()}}


def run_decode(args, shape, dev):
    import torch
    import workloads as W
    from paper_2606_00395_amd import binding as B
    from paper_2606_00395_amd import costmodel as C
    S, P, k = W.DECODE_SEQS, W.DECODE_STEPS, shape.k
    L = W.layer_inputs(shape.with_(T=S), args.seed)
    G, _ = upload(L, shape.with_(T=S), dev)
    X = torch.from_numpy(W.decode_all_states(shape, args.seed)).to(torch.bfloat16).to(dev)
    Xsteps = X.permute(1, 0, 2).contiguous()                       # [P, S, d]
    buf = torch.full((S, P, k), -1, dtype=torch.int16, device=dev)
    ws = B.route_workspace(Xsteps[0], G["W_r"], G["A"], k, B.PR2_I16)
    stream = torch.cuda.current_stream()

    # the policy's router and predictor are fixed for the whole rollout: the first step
    # splits them, the other steps reuse that split (pr2_route_predict_reuse)
    def record_all(st):
        for pos in range(P):
            B.route_predict(Xsteps[pos], G["W_r"], G["beta"], G["A"], G["B"], k, buf[:, pos, :],
                            ws=ws, stream=st, reuse_split=pos > 0)

    record_all(stream)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    record_all(stream)
    e1.record(stream)
    torch.cuda.synchronize()
    us_launch = e0.elapsed_time(e1) * 1e3 / P
    # the same 2048 steps captured once and replayed as one HIP graph
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        record_all(torch.cuda.current_stream())      # the capture stream
    for _ in range(3):
        graph.replay()
    torch.cuda.synchronize()
    reps = 3
    e0.record(stream)
    for _ in range(reps):
        graph.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    us_graph = e0.elapsed_time(e1) * 1e3 / (P * reps)
    rec_bytes = S * k * 2

    # replay forward of 32768-token micro-batches (16 whole sequences each)
    Xseq = X.reshape(S * P, shape.d)
    mb = W.DECODE_MICROBATCH
    nseq = mb // P
    y = torch.empty((mb, shape.d), dtype=torch.bfloat16, device=dev)
    wsr = B.replay_workspace(Xseq[:mb], buf[:nseq].reshape(mb, k), G["W_r"], G["W_gate"])
    batches = list(range(S // nseq))          # all 16 micro-batches: the whole record

    def step():
        for b in batches:
            B.moe_replay_forward(Xseq[b * mb:(b + 1) * mb], buf[b * nseq:(b + 1) * nseq].reshape(mb, k),
                                 G["W_r"], G["beta"], G["W_gate"], G["W_up"], G["W_down"], y,
                                 ws=wsr, stream=stream)

    ms, kern = timed_steps(step, args.steps, args.warmup, stream, B)
    tok = mb * len(batches)
    dominant = "gemm1_gate_up_swiglu"
    achieved = C.gemm1_flops(mb, shape.d, k, shape.m) / (kern[dominant] * 1e-3) / 1e12
    peak = C.PEAK_BF16_FLOPS / 1e12
    out = base_record(args, "decode-style route record (us/step) and micro-batch replay "
                      "tokens/sec", tok / (ms * 1e-3), "tokens/s", ms, "bf16",
                      dict(layer_config(shape), sequences=S, steps=P, microbatch=mb,
                           microbatches=batches))
    out["roofline"] = {"bound": "mfma", "kernel": dominant, "achieved": achieved, "peak": peak,
                       "unit": "TFLOP/s", "frac": achieved / peak, "traffic": None}
    out["route_record"] = {"us_per_step_launches": us_launch, "us_per_step_hip_graph": us_graph,
                           "record_bytes_per_step": rec_bytes,
                           "record_gbps_graph": rec_bytes / (us_graph * 1e-6) / 1e9}
    out["kernels_ms"] = {n: round(v, 5) for n, v in kern.items()}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_decode(shape, L)
    return out


def run_next(args, shape, dev):
    import numpy as np
    import torch
    import workloads as W
    from paper_2606_00395_amd import binding as B
    from paper_2606_00395_amd import costmodel as C
    L = W.layer_inputs(shape, args.seed)
    G, up = upload(L, shape, dev)
    T, d, N, k, m, r = shape.T, shape.d, shape.N, shape.k, shape.m, shape.r
    ab = 2 if shape.act == "bf16" else 4
    x = G["x"]
    stream = torch.cuda.current_stream()

    def measure(step):
        ms, kern = timed_steps(step, args.steps, args.warmup, stream, B)
        return ms, {n: round(v, 5) for n, v in kern.items()}

    # f2: rollout-phase layer output (route prediction, record, experts under the
    # predictive gates), renormalised and paper-literal
    idx = torch.empty((T, k), dtype=torch.int32, device=dev)
    gate = torch.empty((T, k), dtype=torch.float32, device=dev)
    y = torch.empty_like(x)
    ws_ro = B.rollout_workspace(x, G["W_r"], G["A"], G["W_gate"], k)
    ws_lit = B.rollout_workspace(x, G["W_r"], G["A"], G["W_gate"], k, renorm=False)

    def rollout(renorm, ws):
        def step():
            B.moe_rollout_forward(x, G["W_r"], G["beta"], G["A"], G["B"], G["W_gate"], G["W_up"],
                                  G["W_down"], k, idx, y, gate, renorm=renorm, ws=ws,
                                  stream=stream)
        return step
    ms_lit, kern_lit = measure(rollout(False, ws_lit))
    ms, kern = measure(rollout(True, ws_ro))
    dominant = "gemm1_gate_up_swiglu"
    achieved = C.gemm1_flops(T, d, k, m) / (kern[dominant] * 1e-3) / 1e12
    peak = C.PEAK_BF16_FLOPS / 1e12
    out = base_record(args, "MoE-layer tokens/sec (rollout forward: predictive route, record, "
                      "layer output under the predictive gates)", T / (ms * 1e-3), "tokens/s", ms,
                      "bf16" if shape.act == "bf16" else "f32", layer_config(shape))
    out["roofline"] = {"bound": "mfma", "kernel": dominant, "achieved": achieved, "peak": peak,
                       "unit": "TFLOP/s", "frac": achieved / peak,
                       "traffic": profiled_traffic(f"replay_and_route_kernels_{shape.name}.txt",
                                                  gemm1_kernel(shape.m))}
    out["kernels_ms"] = kern
    out["rollout_paper_literal_gates"] = {"ms": ms_lit, "value": T / (ms_lit * 1e-3),
                                          "kernels_ms": kern_lit}

    # f1: route with the feature-cache write of Tc sub-sampled positions
    Tc = min(FEATURE_CACHE_POSITIONS, T)
    pos = B.feature_cache_positions(T, Tc, args.seed + 5)
    row = np.full(T, -1, dtype=np.int32)
    row[pos] = np.arange(len(pos), dtype=np.int32)
    cache_row = torch.from_numpy(row).to(dev)
    h_cache = torch.empty((len(pos), d), dtype=x.dtype, device=dev)
    p_cache = torch.empty((len(pos), N), dtype=torch.float32, device=dev)
    ws_r = B.route_workspace(x, G["W_r"], G["A"], k)

    def cached():
        B.route_predict_cached(x, G["W_r"], G["beta"], G["A"], G["B"], k, idx, cache_row, h_cache,
                               p_cache, gate, ws=ws_r, stream=stream)
    ms_c, kern_c = measure(cached)
    t_route = kern_c.get("route_predict", float("nan"))
    rbytes = C.route_bytes(T, d, N, r, k, ab, 4) + len(pos) * (d * ab + N * 4)
    out["feature_cache_route"] = {
        "ms": ms_c, "cached_positions": len(pos), "kernels_ms": kern_c,
        "roofline": {"bound": "hbm", "kernel": "route_predict", "achieved": rbytes / (t_route * 1e-3)
                     / 1e9, "peak": C.PEAK_HBM_BYTES / 1e9, "unit": "GB/s",
                     "frac": rbytes / (t_route * 1e-3) / C.PEAK_HBM_BYTES}}

    # f1 / f4: predictor loss over the cached positions, current router drifted from
    # the rollout's, standard and delta-matching forms
    rng = np.random.default_rng([args.seed, 601])
    W_cur = up((L["W_r"] + 0.002 * rng.standard_normal(L["W_r"].shape)).astype(np.float32))
    h_cur = x[torch.from_numpy(pos).to(dev)].contiguous()
    loss = torch.empty((1,), dtype=torch.float32, device=dev)
    dA = torch.empty((d, r), dtype=torch.float32, device=dev)
    dB = torch.empty((r, N), dtype=torch.float32, device=dev)
    kl = torch.empty((len(pos),), dtype=torch.float32, device=dev)
    desc = B.make_desc(len(pos), d, N, 1, 0, r, B._act_code(x))
    ws_p = torch.empty(max(1, B.workspace_bytes(desc, B.OP_PREDICTOR_LOSS)), dtype=torch.uint8,
                       device=dev)
    pflops = 2 * len(pos) * d * N + 4 * len(pos) * d * r + 4 * len(pos) * r * N
    pbytes = len(pos) * (2 * d * ab + N * 4 + 4) + (d * N + 2 * d * r + 2 * r * N) * 4
    for kind, name in ((0, "predictor_loss"), (1, "delta_matching_loss")):
        def loss_step():
            B.predictor_loss(h_cur, W_cur, G["beta"], h_cache, p_cache, G["A"], G["B"], loss, dA,
                             dB, kl, loss_kind=kind, mini_step=2, ws=ws_p, stream=stream)
        ms_p, kern_p = measure(loss_step)
        out[name] = {"ms": ms_p, "cached_positions": len(pos), "kernels_ms": kern_p,
                     "flops": pflops, "algorithmic_bytes": pbytes,
                     "hbm_gbps": pbytes / (ms_p * 1e-3) / 1e9}

    # f3: route diagnostics of the recorded rollout route under the drifted router
    z_ref = torch.empty((T, N), dtype=torch.float32, device=dev)
    B.route_predict(x, G["W_r"], G["beta"], G["A"], G["B"], k, idx, gate, logits_out=z_ref,
                    stream=stream)
    cur = torch.empty((T, k), dtype=torch.int32, device=dev)
    ov = torch.empty((T,), dtype=torch.int32, device=dev)
    kl_t = torch.empty((T,), dtype=torch.float32, device=dev)
    hist = torch.empty((k + 1,), dtype=torch.int64, device=dev)
    desc = B.make_desc(T, d, N, k, 0, 0, B._act_code(x))
    ws_d = torch.empty(max(1, B.workspace_bytes(desc, B.OP_ROUTE_DIAG)), dtype=torch.uint8,
                       device=dev)

    def diag():
        B.route_diagnostics(x, idx, W_cur, G["beta"], z_ref, cur, ov, kl_t, hist, ws=ws_d,
                            stream=stream)
    ms_d, kern_d = measure(diag)
    t_diag = kern_d.get("route_diagnostics", float("nan"))
    dbytes = T * d * ab + T * N * 4 + T * k * 4 * 2 + T * 8 + (k + 1) * 8
    out["route_diagnostics"] = {
        "ms": ms_d, "kernels_ms": kern_d,
        "agreement": float(ov.double().mean().item() / k), "hist": hist.cpu().tolist(),
        "roofline": {"bound": "hbm", "kernel": "route_diagnostics",
                     "achieved": dbytes / (t_diag * 1e-3) / 1e9, "peak": C.PEAK_HBM_BYTES / 1e9,
                     "unit": "GB/s", "frac": dbytes / (t_diag * 1e-3) / C.PEAK_HBM_BYTES}}

    # f3 fused into the replay forward: the same diagnostics from the replay-weight
    # epilogue (pr2_moe_replay_forward_diag) against the plain replay forward,
    # interleaved A/B rounds
    ws_f = B.replay_workspace(x, idx, W_cur, G["W_gate"])
    yb = torch.empty_like(x)
    gr = torch.empty((T, k), dtype=torch.float32, device=dev)

    def plain():
        B.moe_replay_forward(x, idx, W_cur, G["beta"], G["W_gate"], G["W_up"], G["W_down"], yb,
                             gr, ws=ws_f, stream=stream)

    def fused():
        B.moe_replay_forward_diag(x, idx, W_cur, G["beta"], G["W_gate"], G["W_up"], G["W_down"],
                                  yb, gr, z_ref, cur, ov, kl_t, hist, ws=ws_f, stream=stream)
    ab_ms = {"plain": [], "fused": []}
    for _ in range(3):
        for name, fn in (("plain", plain), ("fused", fused)):
            ab_ms[name].append(timed_steps(fn, args.steps, 3, stream, B)[0])
    mp = sorted(ab_ms["plain"])[1]
    mf = sorted(ab_ms["fused"])[1]
    out["replay_forward_fused_diagnostics"] = {
        "ms_plain": mp, "ms_with_diagnostics": mf, "ratio": mf / mp,
        "note": "median of 3 interleaved rounds each; the fused call also writes the current "
                "top-k, overlap, route KL and deviation histogram"}
    if not args.no_cpu_baseline:
        n_tok = args.cpu_sample_tokens if args.cpu_sample_tokens > 0 else 4096
        out["cpu_baseline"] = cpu_baseline_rollout(shape, L, min(n_tok, T))
    return out


def run_extras(args, dev):
    """The other workloads, each on its own (GPU timings only, no CPU legs): the
    Qwen3-235B-A22B-shaped forward, the replay backward, the decode-style record
    and replay of the whole route record, and the method's other calls."""
    import copy
    import torch
    import workloads as W
    out = {}
    a = copy.copy(args)
    a.no_cpu_baseline = True
    a.light = True
    a.steps = min(args.steps, 10)
    a.warmup = min(args.warmup, 10)
    legs = (("qwen3_235b_forward", run_forward, "qwen3_235b_T32768"),
            ("qwen3_30b_backward", run_backward, "qwen3_30b_bwd_T16384"),
            ("qwen3_30b_decode", run_decode, "qwen3_30b_decode_256x2048"),
            ("qwen3_30b_next", run_next, "qwen3_30b_T16384"))
    for name, fn, wl in legs:
        b = copy.copy(a)
        if fn is run_decode:
            b.steps, b.warmup = 3, 1
        rec = fn(b, W.WORKLOADS[wl], dev)
        for key in ("n_gpus", "steps", "warmup", "higher_is_better", "scaling", "vs_baseline",
                    "data"):
            rec.pop(key, None)
        out[name] = rec
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        print(f"bench: extra {name} done", file=sys.stderr, flush=True)
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the library has no "
              "multi-GPU path", file=sys.stderr)
        sys.exit(2)
    import torch
    import workloads as W

    shape = W.WORKLOADS[args.workload or DEFAULT_WORKLOAD[args.mode]]
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b
    run = {"forward": run_forward, "backward": run_backward, "decode": run_decode,
           "next": run_next}[args.mode]
    rec = run(args, shape, dev)
    if args.mode == "forward" and not args.no_extras:
        torch.cuda.empty_cache()
        rec["extras"] = run_extras(args, dev)
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
