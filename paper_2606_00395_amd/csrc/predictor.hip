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
// Everything after it runs in fp64: u by an fp64 dot product per (token,
// column), one wavefront per token for the two softmaxes, the KL and dz, and
// one thread per gradient entry summing over the tokens in a fixed order.
// Sizes are those of a feature cache (thousands of tokens), so these are small
// kernels; the sums are deterministic (no atomics).
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

// u[t][q] = sum_i h_old[t][i] A[i][q]; one wavefront per token, lanes over q
template <typename XT>
__global__ void __launch_bounds__(256)
proj_u_kernel(const XT* h, int64_t T, int d, const float* A, int r, double* u) {
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (t >= T) return;
    const XT* hr = h + t * d;
    for (int q = lane; q < r; q += 64) {
        double acc = 0.0;
        for (int i = 0; i < d; ++i)
            acc = fma((double)Act<XT>::to_f32(hr[i]), (double)A[(int64_t)i * r + q], acc);
        u[t * r + q] = acc;
    }
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

// one wavefront per token
__global__ void __launch_bounds__(256) pred_loss_kernel(LossArgs a) {
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (t >= a.T) return;
    const int N = a.N, r = a.r;
    const int nv = (N + 63) / 64;
    const double* ut = a.u + t * r;
    double zh[kMaxVals], tl[kMaxVals];
    double mz = -INFINITY, mt = -INFINITY;
    for (int v = 0; v < nv; ++v) {
        const int j = v * 64 + lane;
        zh[v] = -INFINITY;
        tl[v] = -INFINITY;
        if (j < N) {
            double b = 0.0;
            if (a.B) {
                for (int q = 0; q < r; ++q) b = fma(ut[q], (double)a.B[(int64_t)q * N + j], b);
            } else {
                b = ut[j];
            }
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
                if (j < N) part = fma(zh[v], (double)a.B[(int64_t)q * N + j], part);
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

// dB[q][j] = sum_t u[t][q] dz[t][j]
__global__ void __launch_bounds__(256)
grad_b_kernel(const double* u, const double* dz, int64_t T, int r, int N, float* dB) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= (int64_t)r * N) return;
    const int q = (int)(e / N), j = (int)(e % N);
    double acc = 0.0;
    for (int64_t t = 0; t < T; ++t) acc = fma(u[t * r + q], dz[t * N + j], acc);
    dB[e] = (float)acc;
}

// dA[i][q] = sum_t h_old[t][i] g[t][q], g = dz B^T (or dz for the identity)
template <typename XT>
__global__ void __launch_bounds__(256)
grad_a_kernel(const XT* h, const double* g, int64_t T, int d, int r, float* dA) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= (int64_t)d * r) return;
    const int q = (int)(e / d), i = (int)(e % d);    // i fastest: coalesced reads of h
    double acc = 0.0;
    for (int64_t t = 0; t < T; ++t)
        acc = fma((double)Act<XT>::to_f32(h[t * d + i]), g[t * r + q], acc);
    dA[(int64_t)i * r + q] = (float)acc;
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

dim3 blocks_for(int64_t n) { return dim3((unsigned)((n + 255) / 256)); }

}  // namespace

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
        LaunchScope scope("predictor_proj_u", s);
        if (bf)
            hipLaunchKernelGGL(proj_u_kernel<bf16_t>, tok, dim3(256), 0, s, (const bf16_t*)h_old,
                               d.T, d.d, A, d.r, ws.u);
        else
            hipLaunchKernelGGL(proj_u_kernel<float>, tok, dim3(256), 0, s, (const float*)h_old, d.T,
                               d.d, A, d.r, ws.u);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
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
        LaunchScope scope("predictor_grad_b", s);
        hipLaunchKernelGGL(grad_b_kernel, blocks_for((int64_t)d.r * d.N), dim3(256), 0, s, ws.u,
                           ws.dz, d.T, d.r, d.N, dB);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const double* g = B ? ws.w : ws.dz;
    LaunchScope scope("predictor_grad_a", s);
    if (bf)
        hipLaunchKernelGGL(grad_a_kernel<bf16_t>, blocks_for((int64_t)d.d * d.r), dim3(256), 0, s,
                           (const bf16_t*)h_old, g, d.T, d.d, d.r, dA);
    else
        hipLaunchKernelGGL(grad_a_kernel<float>, blocks_for((int64_t)d.d * d.r), dim3(256), 0, s,
                           (const float*)h_old, g, d.T, d.d, d.r, dA);
    return hipGetLastError();
}

}  // namespace pr2
