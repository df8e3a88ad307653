// Evolution-predictor training on the feature cache (Sec. 4.2, Eq. pr2_loss;
// Alg. 3 in Appendix D, its predictive-loss steps), for the cached tokens t:
//
//   p_t       = h_t W_r + b_r                  current router (the teacher, no gradient)
//   u_t       = h_old,t A,  b_t = u_t B        predictor residual, W_p = A B
//   standard:  KL(softmax(p_t) || softmax(p_old,t + b_t))
//   delta:     KL(softmax(p_t - p_old,t) || softmax(b_t))   (Appendix G ablation)
//   loss = mean_t KL,  dz_t = (softmax(zhat_t) - target_t) / T
//   dB = sum_t u_t^T dz_t,  dA = sum_t h_old,t^T (dz_t B^T)
//
// p comes from the replay router kernels (exact products, one rounding to fp32).
// Everything after it runs in fp64.  The three products u = h_old A,
// dB = u^T dz and dA = h_old^T w go through one tiled kernel: a workgroup forms
// a 64 x 16 output tile over one slice of the summed index, staging both
// operands through LDS as fp64, and a second kernel adds the slices in slice
// order.  The two softmaxes, the KL and dz take one wavefront per token.  The
// sums are deterministic (no atomics).
#include <algorithm>

#include "common.h"

namespace pr2 {
namespace {

constexpr int kMaxVals = kMaxExperts / 64;

__device__ __forceinline__ double wsum(double v) {
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}
__device__ __forceinline__ double wmax(double v) {
    for (int off = 32; off >= 1; off >>= 1) v = fmax(v, __shfl_xor(v, off, 64));
    return v;
}

__device__ __forceinline__ double to_f64(bf16_t v) { return (double)Act<bf16_t>::to_f32(v); }
__device__ __forceinline__ double to_f64(float v) { return (double)v; }
__device__ __forceinline__ double to_f64(double v) { return v; }

constexpr int kPM = 64, kPN = 16, kPK = 32;     // output tile and staged slice of the sum

// C[m][n] = sum_k a(m, k) b(k, n), operands addressed through strides:
// a(m, k) = a[m*a_m + k*a_k], b(k, n) = b[k*b_k + n*b_n].
struct ProdArgs {
    const void* a;
    int64_t a_m, a_k;
    const void* b;
    int64_t b_k, b_n;
    int M, Nc;
    int64_t K, kslice;
    double* part;       // [slices][M][Nc]
};

// workgroup (m tile, n tile, slice); thread (tm, tn) keeps rows 4tm..4tm+3 of column tn
template <typename TA, typename TB>
__global__ void __launch_bounds__(256) prod_f64_kernel(ProdArgs p) {
    __shared__ double sa[kPK][kPM + 1];
    __shared__ double sb[kPK][kPN];
    const int tid = threadIdx.x;
    const int tn = tid & 15, tm = tid >> 4;
    const int m0 = blockIdx.x * kPM, n0 = blockIdx.y * kPN;
    const int64_t k0 = (int64_t)blockIdx.z * p.kslice;
    const int64_t k1 = min(p.K, k0 + p.kslice);
    const TA* a = (const TA*)p.a;
    const TB* b = (const TB*)p.b;
    const bool a_kfast = p.a_k == 1;
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int64_t kc = k0; kc < k1; kc += kPK) {
        for (int e = tid; e < kPM * kPK; e += 256) {
            const int kk = a_kfast ? (e & (kPK - 1)) : e / kPM;
            const int mm = a_kfast ? e / kPK : (e & (kPM - 1));
            const int64_t k = kc + kk;
            const int m = m0 + mm;
            sa[kk][mm] = (m < p.M && k < k1) ? to_f64(a[(int64_t)m * p.a_m + k * p.a_k]) : 0.0;
        }
        for (int e = tid; e < kPN * kPK; e += 256) {
            const int kk = e / kPN, nn = e & (kPN - 1);
            const int64_t k = kc + kk;
            const int n = n0 + nn;
            sb[kk][nn] = (n < p.Nc && k < k1) ? to_f64(b[k * p.b_k + (int64_t)n * p.b_n]) : 0.0;
        }
        __syncthreads();
#pragma unroll 8
        for (int kk = 0; kk < kPK; ++kk) {
            const double bv = sb[kk][tn];
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] = fma(sa[kk][tm * 4 + i], bv, acc[i]);
        }
        __syncthreads();
    }
    const int n = n0 + tn;
    if (n >= p.Nc) return;
    double* out = p.part + (int64_t)blockIdx.z * p.M * p.Nc;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = m0 + tm * 4 + i;
        if (m < p.M) out[(int64_t)m * p.Nc + n] = acc[i];
    }
}

// out[e] = sum over slices of part[s][e], slice order
template <typename OT>
__global__ void __launch_bounds__(256)
sum_slices_kernel(const double* part, int slices, int64_t n, OT* out) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= n) return;
    double acc = 0.0;
    int s = 0;
    for (; s + 8 <= slices; s += 8) {       // eight loads in flight, added in slice order
        double v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = part[(int64_t)(s + i) * n + e];
#pragma unroll
        for (int i = 0; i < 8; ++i) acc += v[i];
    }
    for (; s < slices; ++s) acc += part[(int64_t)s * n + e];
    out[e] = (OT)acc;
}

// slices of the summed index: about 1024 workgroups in all, each slice a whole
// number of staged chunks, at most 64 slices
int64_t prod_kslice(int M, int Nc, int64_t K) {
    const int64_t tiles = (int64_t)((M + kPM - 1) / kPM) * ((Nc + kPN - 1) / kPN);
    const int64_t chunks = (K + kPK - 1) / kPK;
    int64_t s = (1024 + tiles - 1) / tiles;
    s = std::max<int64_t>(1, std::min<int64_t>({s, chunks, 64}));
    return std::max<int64_t>(1, (chunks + s - 1) / s) * kPK;
}

int prod_slices(int M, int Nc, int64_t K) {
    return (int)std::max<int64_t>(1, (K + prod_kslice(M, Nc, K) - 1) / prod_kslice(M, Nc, K));
}

template <typename TA, typename TB, typename OT>
hipError_t launch_prod(const TA* a, int64_t a_m, int64_t a_k, const TB* b, int64_t b_k,
                       int64_t b_n, int M, int Nc, int64_t K, double* part, OT* out,
                       hipStream_t s) {
    if (M <= 0 || Nc <= 0) return hipSuccess;
    ProdArgs p{a, a_m, a_k, b, b_k, b_n, M, Nc, K, prod_kslice(M, Nc, K), part};
    const int slices = prod_slices(M, Nc, K);
    dim3 grid((unsigned)((M + kPM - 1) / kPM), (unsigned)((Nc + kPN - 1) / kPN), (unsigned)slices);
    hipLaunchKernelGGL((prod_f64_kernel<TA, TB>), grid, dim3(256), 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t n = (int64_t)M * Nc;
    hipLaunchKernelGGL(sum_slices_kernel<OT>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       part, slices, n, out);
    return hipGetLastError();
}

struct LossArgs {
    const float* p_cur;     // [T, N]
    const float* p_old;     // [T, N]
    const double* u;        // [T, r]
    const float* B;         // [r, N] or null (identity, r == N)
    int64_t T;
    int N, r, kind;
    float* kl_out;          // [T] or null
    double* kl;             // [T]
    double* dz;             // [T, N]
    double* w;              // [T, r]  dz B^T (unused for the identity)
};

constexpr int kLdsB = 4096;      // B entries staged in LDS (r N <= 4096)

// one wavefront per token; B in LDS and the token's u in lanes when they fit
__global__ void __launch_bounds__(256) pred_loss_kernel(LossArgs a) {
    __shared__ float sB[kLdsB];
    const int N = a.N, r = a.r;
    const bool b_lds = a.B && r * N <= kLdsB;
    if (b_lds) {
        for (int e = threadIdx.x; e < r * N; e += 256) sB[e] = a.B[e];
        __syncthreads();
    }
    const float* Bm = b_lds ? sB : a.B;
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (t >= a.T) return;
    const int nv = (N + 63) / 64;
    const double* ut = a.u + t * r;
    const bool u_lanes = r <= 64;
    const double ul = (u_lanes && lane < r) ? ut[lane] : 0.0;
    double zh[kMaxVals], tl[kMaxVals];
    double mz = -INFINITY, mt = -INFINITY;
    for (int v = 0; v < nv; ++v) {
        const int j = v * 64 + lane;
        const int jc = j < N ? j : N - 1;       // every lane takes part in the shuffles
        double b = 0.0;
        if (a.B) {
            for (int q = 0; q < r; ++q)
                b = fma(u_lanes ? __shfl(ul, q, 64) : ut[q], (double)Bm[(int64_t)q * N + jc], b);
        } else {
            b = ut[jc];
        }
        zh[v] = -INFINITY;
        tl[v] = -INFINITY;
        if (j < N) {
            const double po = (double)a.p_old[t * N + j];
            const double pc = (double)a.p_cur[t * N + j];
            zh[v] = a.kind == 0 ? po + b : b;
            tl[v] = a.kind == 0 ? pc : pc - po;
            mz = fmax(mz, zh[v]);
            mt = fmax(mt, tl[v]);
        }
    }
    mz = wmax(mz);
    mt = wmax(mt);
    double sz = 0.0, st = 0.0;
    for (int v = 0; v < nv; ++v) {
        if (v * 64 + lane < N) {
            sz += exp(zh[v] - mz);
            st += exp(tl[v] - mt);
        }
    }
    sz = wsum(sz);
    st = wsum(st);
    const double lsz = log(sz), lst = log(st);
    double kl = 0.0;
    for (int v = 0; v < nv; ++v) {
        const int j = v * 64 + lane;
        if (j < N) {
            const double lt = tl[v] - mt - lst;         // log target
            const double lh = zh[v] - mz - lsz;         // log rho_hat
            const double tg = exp(lt);
            kl += tg * (lt - lh);
            const double g = (exp(lh) - tg) / (double)a.T;
            a.dz[t * N + j] = g;
            zh[v] = g;                                  // keep dz for the B^T product
        }
    }
    kl = wsum(kl);
    if (lane == 0) {
        a.kl[t] = kl;
        if (a.kl_out) a.kl_out[t] = (float)kl;
    }
    if (a.B) {
        for (int q = 0; q < r; ++q) {
            double part = 0.0;
            for (int v = 0; v < nv; ++v) {
                const int j = v * 64 + lane;
                if (j < N) part = fma(zh[v], (double)Bm[(int64_t)q * N + j], part);
            }
            part = wsum(part);
            if (lane == (q & 63)) a.w[t * r + q] = part;
        }
    }
}

// loss = mean of kl, fixed-order reduction in one block
__global__ void __launch_bounds__(256) mean_kernel(const double* kl, int64_t T, float* out) {
    __shared__ double s[256];
    double acc = 0.0;
    for (int64_t t = threadIdx.x; t < T; t += 256) acc += kl[t];
    s[threadIdx.x] = acc;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) s[threadIdx.x] += s[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[0] = T > 0 ? (float)(s[0] / (double)T) : 0.0f;
}

__global__ void __launch_bounds__(256) fill_f32_kernel(float* p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
        p[i] = 0.0f;
}

hipError_t fill0(float* p, int64_t n, hipStream_t s) {
    if (!p || n <= 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(fill_f32_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n);
    return hipGetLastError();
}

}  // namespace

// Partial sums of the three products.  The u product's slice count falls as
// its row tiles grow, so its part is bounded by a size that does not decrease
// with T (slices <= 1024 / tiles + 1 with tiles >= T ntiles / 64, and
// slices <= min(64, K chunks)): a workspace sized for a batch serves every
// smaller one.
size_t predictor_partial_doubles(const pr2_moe_desc& d) {
    const int64_t T = d.T;
    const int64_t ntiles = (d.r + kPN - 1) / kPN;
    const int64_t su_max = std::min<int64_t>(64, std::max<int64_t>(1, (d.d + kPK - 1) / kPK));
    const size_t pu = (size_t)std::min<int64_t>(su_max * T, 1024 * kPM / ntiles + T) * d.r;
    const size_t pb = (size_t)prod_slices(d.r, d.N, T) * (size_t)d.r * d.N;
    const size_t pa = (size_t)prod_slices(d.d, d.r, T) * (size_t)d.d * d.r;
    return std::max({pu, pb, pa});
}

hipError_t launch_predictor_zero(const pr2_moe_desc& d, float* kl_out, float* loss_out, float* dA,
                                 float* dB, hipStream_t s) {
    LaunchScope scope("predictor_loss_skip", s);
    hipError_t e;
    if ((e = fill0(kl_out, d.T, s)) != hipSuccess) return e;
    if ((e = fill0(loss_out, 1, s)) != hipSuccess) return e;
    if ((e = fill0(dA, (int64_t)d.d * d.r, s)) != hipSuccess) return e;
    return fill0(dB, (int64_t)d.r * d.N, s);
}

hipError_t launch_predictor_loss(const pr2_moe_desc& d, const void* h, const float* W_r,
                                 const float* b_r, const void* h_old, const float* p_old,
                                 const float* A, const float* B, int kind, float* kl_out,
                                 float* loss_out, float* dA, float* dB, const PredLossWs& ws,
                                 hipStream_t s) {
    hipError_t e = launch_router_logits(d, h, W_r, b_r, ws.p_cur, ws.wsplit, s);
    if (e != hipSuccess) return e;
    const bool bf = d.act_dtype == PR2_BF16;
    dim3 tok((unsigned)((d.T + 3) / 4));
    {
        // u = h_old A: (token, column) entries summed over the hidden index
        LaunchScope scope("predictor_proj_u", s);
        e = bf ? launch_prod((const bf16_t*)h_old, d.d, 1, A, d.r, 1, (int)d.T, d.r, d.d, ws.part,
                             ws.u, s)
               : launch_prod((const float*)h_old, d.d, 1, A, d.r, 1, (int)d.T, d.r, d.d, ws.part,
                             ws.u, s);
    }
    if (e != hipSuccess) return e;
    LossArgs a{ws.p_cur, p_old, ws.u, B, d.T, d.N, d.r, kind, kl_out, ws.kl, ws.dz, ws.w};
    {
        LaunchScope scope("predictor_kl", s);
        hipLaunchKernelGGL(pred_loss_kernel, tok, dim3(256), 0, s, a);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    {
        LaunchScope scope("predictor_loss_mean", s);
        hipLaunchKernelGGL(mean_kernel, dim3(1), dim3(256), 0, s, ws.kl, d.T, loss_out);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (B) {
        // dB[q][j] = sum_t u[t][q] dz[t][j]
        LaunchScope scope("predictor_grad_b", s);
        e = launch_prod(ws.u, 1, d.r, ws.dz, d.N, 1, d.r, d.N, d.T, ws.part, dB, s);
        if (e != hipSuccess) return e;
    }
    // dA[i][q] = sum_t h_old[t][i] g[t][q], g = dz B^T (dz itself for the identity)
    const double* g = B ? ws.w : ws.dz;
    LaunchScope scope("predictor_grad_a", s);
    return bf ? launch_prod((const bf16_t*)h_old, 1, d.d, g, d.r, 1, d.d, d.r, d.T, ws.part, dA, s)
              : launch_prod((const float*)h_old, 1, d.d, g, d.r, 1, d.d, d.r, d.T, ws.part, dA, s);
}

}  // namespace pr2
