// Router kernels: the fused router + evolution-predictor projection with the
// rollout top-k epilogue (Sec. 4.1, Eq. pr2_predict / pr2_route), and the same
// projection with the replay-weight epilogue (Sec. 4.1 replay, Eq. pr2_output).
//
// Projection: each block owns TM tokens and computes their logits against the
// NC = N (+ r) columns of [W_r | A] in column passes.  x and the weight panel
// are staged through LDS in K-slices of KB; each thread accumulates a 4-token x
// 4-column micro-tile in float64, so the logits reach the epilogue with one
// rounding to fp32 and the top-k decision does not depend on the summation
// order over d.
//
// Epilogue: one wavefront per token.  Lane l holds logits l, l+64, ...; the
// top-k is k rounds of a wavefront max over packed (orderable logit, ~id) keys,
// so equal logits resolve to the lower id; the chosen ids are written in
// ascending id order with their gates.
#include "common.h"

namespace pr2 {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxLanesVals = kMaxExperts / 64;

__device__ __forceinline__ uint32_t orderable(float z) {
    if (z == 0.0f) z = 0.0f;                 // -0.0 ties with +0.0
    uint32_t u = __float_as_uint(z);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
        uint32_t olo = __shfl_xor(lo, off, 64), ohi = __shfl_xor(hi, off, 64);
        uint64_t o = ((uint64_t)ohi << 32) | olo;
        v = o > v ? o : v;
    }
    return v;
}

__device__ __forceinline__ float wave_sum_f32(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__device__ __forceinline__ float wave_max_f32(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    return v;
}

__device__ __forceinline__ int wave_sum_i32(int v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

struct ProjArgs {
    const void* x;
    const float* W_r;
    const float* A;   // may be null (no predictor columns)
    int64_t T;
    int d, N, r, NC, TM, KB;   // KB: K slice staged per step
};

// Computes the TM x NC fp32 logit tile of tokens [t0, t0+TM) into lds_logits
// (row stride NC).  Columns < N come from W_r, columns >= N from A.
template <typename XT>
__device__ void project_tile(const ProjArgs& a, int64_t t0, float* xs, float* ws,
                             float* lds_logits) {
    const int tid = threadIdx.x;
    const int tgroups = a.TM / 4;                    // token groups of 4
    const int cgroups = kThreads / tgroups;          // column groups of 4
    const int cols_per_pass = cgroups * 4;
    const int tg = tid / cgroups;
    const int cg = tid % cgroups;

    for (int c0 = 0; c0 < a.NC; c0 += cols_per_pass) {
        double acc[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;

        for (int k0 = 0; k0 < a.d; k0 += a.KB) {
            // stage x[t0 .. t0+TM) x [k0 .. k0+KB) as fp32 (zero outside)
            for (int q = tid; q < a.TM * a.KB; q += kThreads) {
                int tt = q / a.KB, kk = q % a.KB;
                int64_t t = t0 + tt;
                int kg = k0 + kk;
                float v = 0.0f;
                if (t < a.T && kg < a.d)
                    v = Act<XT>::load((const XT*)a.x + t * (int64_t)a.d + kg);
                xs[tt * a.KB + kk] = v;
            }
            // stage the weight panel [k0 .. k0+KB) x [c0 .. c0+cols_per_pass)
            for (int q = tid; q < a.KB * cols_per_pass; q += kThreads) {
                int kk = q / cols_per_pass, cc = q % cols_per_pass;
                int kg = k0 + kk, c = c0 + cc;
                float v = 0.0f;
                if (kg < a.d && c < a.NC)
                    v = c < a.N ? a.W_r[(int64_t)kg * a.N + c]
                                : a.A[(int64_t)kg * a.r + (c - a.N)];
                ws[kk * cols_per_pass + cc] = v;
            }
            __syncthreads();
            if (tg < tgroups) {
#pragma unroll 4
                for (int kk = 0; kk < a.KB; ++kk) {
                    double xv[4], wv[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) xv[i] = (double)xs[(tg * 4 + i) * a.KB + kk];
#pragma unroll
                    for (int j = 0; j < 4; ++j) wv[j] = (double)ws[kk * cols_per_pass + cg * 4 + j];
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int j = 0; j < 4; ++j) acc[i][j] = fma(xv[i], wv[j], acc[i][j]);
                }
            }
            __syncthreads();
        }
        if (tg < tgroups) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    int c = c0 + cg * 4 + j;
                    if (c < a.NC) lds_logits[(tg * 4 + i) * a.NC + c] = (float)acc[i][j];
                }
        }
    }
    __syncthreads();
}

template <typename XT>
__global__ void __launch_bounds__(kThreads)
route_predict_kernel(ProjArgs a, const float* b_r, const float* B, int k, int renorm,
                     void* idx_out, int idx_dtype, int64_t ldi, float* gate_out,
                     float* logits_out) {
    extern __shared__ float smem[];
    float* xs = smem;                                   // TM*KB
    float* ws = xs + a.TM * a.KB;                       // KB*cols_per_pass
    const int cols_per_pass = (kThreads / (a.TM / 4)) * 4;
    float* lg = ws + a.KB * cols_per_pass;              // TM*NC

    const int64_t t0 = (int64_t)blockIdx.x * a.TM;
    project_tile<XT>(a, t0, xs, ws, lg);

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int nv = (a.N + 63) / 64;
    for (int tt = wave; tt < a.TM; tt += kThreads / 64) {
        const int64_t t = t0 + tt;
        if (t >= a.T) break;
        const float* row = lg + tt * a.NC;
        float z[kMaxLanesVals];
        float pz[kMaxLanesVals];
        for (int v = 0; v < nv; ++v) {
            int j = v * 64 + lane;
            z[v] = -INFINITY;
            pz[v] = 0.0f;
            if (j < a.N) {
                // p = xW + beta, then z = p + (xA) B, accumulated in fp64
                double p = (double)row[j] + (b_r ? (double)b_r[j] : 0.0);
                float pf = (float)p;
                pz[v] = pf;
                double zz = p;
                if (a.r > 0) {
                    const float* u = row + a.N;
                    if (B) {
                        for (int q = 0; q < a.r; ++q) zz += (double)u[q] * (double)B[(int64_t)q * a.N + j];
                    } else {
                        zz += (double)u[j];          // B = identity (full-rank predictor)
                    }
                }
                z[v] = (float)zz;
            }
        }
        if (logits_out) {
            for (int v = 0; v < nv; ++v) {
                int j = v * 64 + lane;
                if (j < a.N) logits_out[t * a.N + j] = pz[v];
            }
        }
        // k rounds of a wavefront arg-max; ties go to the lower id
        uint32_t taken = 0;
        float zmax = 0.0f;
        for (int it = 0; it < k; ++it) {
            uint64_t best = 0;
            for (int v = 0; v < nv; ++v) {
                int j = v * 64 + lane;
                if (j < a.N && !((taken >> v) & 1u)) {
                    uint64_t key = ((uint64_t)orderable(z[v]) << 32) | (uint32_t)(0xffffffffu - (uint32_t)j);
                    best = key > best ? key : best;
                }
            }
            best = wave_max_u64(best);
            int jw = (int)(0xffffffffu - (uint32_t)best);
            if (it == 0) {
                // the top-1 logit, recovered from its owner lane
                float zw = 0.0f;
                for (int v = 0; v < nv; ++v)
                    if (v * 64 + lane == jw) zw = z[v];
                zmax = __shfl(zw, jw & 63, 64);
            }
            if ((jw & 63) == lane) taken |= 1u << (jw >> 6);
        }
        // weights
        float e[kMaxLanesVals];
        float s_sel = 0.0f, s_all = 0.0f;
        for (int v = 0; v < nv; ++v) {
            int j = v * 64 + lane;
            e[v] = 0.0f;
            if (j < a.N) {
                e[v] = expf(z[v] - zmax);
                s_all += e[v];
                if ((taken >> v) & 1u) s_sel += e[v];
            }
        }
        const float denom = renorm ? wave_sum_f32(s_sel) : wave_sum_f32(s_all);
        // write ids ascending with their gates
        int before = 0;
        for (int v = 0; v < nv; ++v) {
            bool mine = (taken >> v) & 1u;
            uint64_t bal = __ballot(mine);
            if (mine) {
                uint64_t lt = lane ? (bal & ((~0ull) >> (64 - lane))) : 0ull;
                int rank = before + __popcll(lt);
                int j = v * 64 + lane;
                int64_t pos = t * ldi + rank;
                if (idx_dtype == PR2_I16) ((int16_t*)idx_out)[pos] = (int16_t)j;
                else ((int32_t*)idx_out)[pos] = j;
                if (gate_out) gate_out[t * k + rank] = e[v] / denom;
            }
            before += __popcll(bal);
        }
    }
}

template <typename XT>
__global__ void __launch_bounds__(kThreads)
replay_gates_kernel(ProjArgs a, const float* b_r, int k, int renorm, const void* idx,
                    int idx_dtype, int64_t ldi, float* gate_out, int* err, int validate) {
    extern __shared__ float smem[];
    float* xs = smem;
    float* ws = xs + a.TM * a.KB;
    const int cols_per_pass = (kThreads / (a.TM / 4)) * 4;
    float* lg = ws + a.KB * cols_per_pass;

    const int64_t t0 = (int64_t)blockIdx.x * a.TM;
    project_tile<XT>(a, t0, xs, ws, lg);

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    for (int tt = wave; tt < a.TM; tt += kThreads / 64) {
        const int64_t t = t0 + tt;
        if (t >= a.T) break;
        const float* row = lg + tt * a.NC;
        // current-router logits p = xW + beta (predictor bypassed)
        float pmax_all = -INFINITY;
        for (int j = lane; j < a.N; j += 64) {
            float p = (float)((double)row[j] + (b_r ? (double)b_r[j] : 0.0));
            pmax_all = fmaxf(pmax_all, p);
        }
        pmax_all = wave_max_f32(pmax_all);
        float pmax_sel = -INFINITY;
        int bad = 0;
        for (int s = lane; s < k; s += 64) {
            int id = load_id(idx, idx_dtype, t * ldi + s);
            if (id >= 0 && id < a.N) {
                float p = (float)((double)row[id] + (b_r ? (double)b_r[id] : 0.0));
                pmax_sel = fmaxf(pmax_sel, p);
            } else {
                bad++;
            }
        }
        pmax_sel = wave_max_f32(pmax_sel);
        const float ref = renorm ? pmax_sel : pmax_all;
        float s_sel = 0.0f, s_all = 0.0f;
        for (int s = lane; s < k; s += 64) {
            int id = load_id(idx, idx_dtype, t * ldi + s);
            if (id >= 0 && id < a.N)
                s_sel += expf((float)((double)row[id] + (b_r ? (double)b_r[id] : 0.0)) - ref);
        }
        if (!renorm)
            for (int j = lane; j < a.N; j += 64)
                s_all += expf((float)((double)row[j] + (b_r ? (double)b_r[j] : 0.0)) - ref);
        const float denom = renorm ? wave_sum_f32(s_sel) : wave_sum_f32(s_all);
        for (int s = lane; s < k; s += 64) {
            int id = load_id(idx, idx_dtype, t * ldi + s);
            float g = 0.0f;
            if (id >= 0 && id < a.N)
                g = expf((float)((double)row[id] + (b_r ? (double)b_r[id] : 0.0)) - ref) / denom;
            gate_out[t * k + s] = g;
        }
        if (validate) {
            int dup = 0;
            for (int s = lane; s < k; s += 64) {
                int id = load_id(idx, idx_dtype, t * ldi + s);
                for (int s2 = 0; s2 < s; ++s2)
                    if (load_id(idx, idx_dtype, t * ldi + s2) == id) dup++;
            }
            dup = wave_sum_i32(dup);
            int nbad = wave_sum_i32(bad);
            if (lane == 0) {
                if (nbad) atomicAdd(err + ERR_BAD_ID, nbad);
                if (dup) atomicAdd(err + ERR_DUP_ID, dup);
            }
        }
    }
}

// Token-tile height and K slice keep the block's LDS under 64 KiB for NC <= 1280.
void pick_tile(ProjArgs& a) {
    if (a.NC <= 256) { a.TM = 32; a.KB = 16; }
    else if (a.NC <= 704) { a.TM = 16; a.KB = 16; }
    else { a.TM = 8; a.KB = 8; }
}

size_t router_smem(const ProjArgs& a) {
    int cols_per_pass = (kThreads / (a.TM / 4)) * 4;
    return sizeof(float) * ((size_t)a.TM * a.KB + (size_t)a.KB * cols_per_pass +
                            (size_t)a.TM * a.NC);
}

}  // namespace

hipError_t launch_route_predict(const pr2_moe_desc& d, const void* x, const float* W_r,
                                const float* b_r, const float* A, const float* B, void* idx_out,
                                int64_t ldi, float* gate_out, float* logits_out, hipStream_t s) {
    ProjArgs a;
    a.x = x;
    a.W_r = W_r;
    a.A = d.r > 0 ? A : nullptr;
    a.T = d.T;
    a.d = d.d;
    a.N = d.N;
    a.r = d.r;
    a.NC = d.N + d.r;
    pick_tile(a);
    dim3 grid((unsigned)((d.T + a.TM - 1) / a.TM));
    size_t smem = router_smem(a);
    LaunchScope scope("route_predict", s);
    if (d.act_dtype == PR2_BF16)
        hipLaunchKernelGGL(route_predict_kernel<bf16_t>, grid, dim3(kThreads), smem, s, a, b_r,
                           d.r > 0 ? B : nullptr, d.k, d.renorm, idx_out, d.idx_dtype, ldi,
                           gate_out, logits_out);
    else
        hipLaunchKernelGGL(route_predict_kernel<float>, grid, dim3(kThreads), smem, s, a, b_r,
                           d.r > 0 ? B : nullptr, d.k, d.renorm, idx_out, d.idx_dtype, ldi,
                           gate_out, logits_out);
    return hipGetLastError();
}

hipError_t launch_replay_gates(const pr2_moe_desc& d, const void* x, const void* idx, int64_t ldi,
                               const float* W_r, const float* b_r, float* gate_out, int* err,
                               hipStream_t s) {
    ProjArgs a;
    a.x = x;
    a.W_r = W_r;
    a.A = nullptr;
    a.T = d.T;
    a.d = d.d;
    a.N = d.N;
    a.r = 0;
    a.NC = d.N;
    pick_tile(a);
    dim3 grid((unsigned)((d.T + a.TM - 1) / a.TM));
    size_t smem = router_smem(a);
    const char* v = getenv("PR2_VALIDATE");
    int validate = (v && v[0] == '1') ? 1 : 0;
    LaunchScope scope("replay_gates", s);
    if (d.act_dtype == PR2_BF16)
        hipLaunchKernelGGL(replay_gates_kernel<bf16_t>, grid, dim3(kThreads), smem, s, a, b_r,
                           d.k, d.renorm, idx, d.idx_dtype, ldi, gate_out, err, validate);
    else
        hipLaunchKernelGGL(replay_gates_kernel<float>, grid, dim3(kThreads), smem, s, a, b_r,
                           d.k, d.renorm, idx, d.idx_dtype, ldi, gate_out, err, validate);
    return hipGetLastError();
}

}  // namespace pr2
