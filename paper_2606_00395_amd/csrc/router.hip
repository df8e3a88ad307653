// Router kernels: the fused router + evolution-predictor projection with the
// rollout top-k epilogue (Sec. 4.1, Eq. pr2_predict / pr2_route), and the same
// projection with the replay-weight epilogue (Sec. 4.1 replay, Eq. pr2_output).
//
// MFMA path (bf16 x, d % 32 == 0, at most 192 projection columns).  x is bf16,
// so each fp32 weight is split into three bf16 parts with hi + mid + lo == w
// exactly and every MFMA product is exact; fp32 partial sums over two K-steps
// of 32 are added into fp64 accumulators, and the logits are rounded to fp32
// once.  When the caller does not ask for the router logits p, the predictor is
// folded into the weights first (W_r + A B, formed in fp64 before the split),
// so the projection has N columns; otherwise it has N + r columns [W_r | A]
// and the epilogue forms z = p + u B in fp64.  The split weights are stored
// K-tiled ([K/32][3 * columns][32] bf16) so that every K-step reads one
// contiguous block.  A workgroup of 8 wavefronts owns 64 tokens; each
// wavefront computes 32 tokens x a quarter of the columns with
// v_mfma_f32_16x16x32_bf16.  Token rows and weight rows of a K step are copied
// straight from global memory into LDS (16-byte copies, 64-byte rows with
// XOR-swizzled chunks), three or four steps deep, so the copies of later steps
// are in flight while one step is consumed.
//
// fp64 vector path (fp32 x or other shapes): each thread accumulates a 4-token
// x 4-column micro-tile in fp64 from LDS-staged slices.
//
// Epilogues run one wavefront per token.  Rollout: k rounds of a DPP wavefront
// max over orderable 32-bit logit keys, the lowest id among equal keys taken
// by ballot, ids written ascending with their gates.  Replay: softmax over the
// recorded ids (or over all N for the literal weights) from the current
// router's logits.
#include "common.h"

namespace pr2 {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxLanesVals = kMaxExperts / 64;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t orderable(float z) {
    if (z == 0.0f) z = 0.0f;                 // -0.0 ties with +0.0
    uint32_t u = __float_as_uint(z);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float from_orderable(uint32_t key) {
    return __uint_as_float((key & 0x80000000u) ? (key & 0x7fffffffu) : ~key);
}

// DPP wavefront reductions from the device library (fixed order: deterministic)
extern "C" __device__ __attribute__((const)) float __ockl_wfred_add_f32(float);
extern "C" __device__ __attribute__((const)) float __ockl_wfred_max_f32(float);
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) { return __ockl_wfred_max_u32(v); }
__device__ __forceinline__ float wave_sum_f32(float v) { return __ockl_wfred_add_f32(v); }
__device__ __forceinline__ float wave_max_f32(float v) { return __ockl_wfred_max_f32(v); }
__device__ __forceinline__ int wave_sum_i32(int v) { return __ockl_wfred_add_i32(v); }

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
            for (int q = tid; q < a.TM * a.KB; q += kThreads) {
                int tt = q / a.KB, kk = q % a.KB;
                int64_t t = t0 + tt;
                int kg = k0 + kk;
                float v = 0.0f;
                if (t < a.T && kg < a.d)
                    v = Act<XT>::load((const XT*)a.x + t * (int64_t)a.d + kg);
                xs[tt * a.KB + kk] = v;
            }
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

// ------------------------------------------------------------ epilogues --
struct PredictOut {
    const float* b_r;     // [N] or null
    const float* B;       // [r, N] or null (identity when r == N)
    int k, renorm;
    int folded;           // 1: the row holds x (W_r + A B); 0: [x W_r | x A]
    void* idx_out;
    int idx_dtype;
    int64_t ldi;
    float* gate_out;      // [T, k] or null
    float* logits_out;    // [T, N] or null (only when not folded)
    FeatureCache cache;   // route-recording features of retained tokens (only when not folded)
    const void* x;        // the layer input, for the hidden-feature copy
    int d;
    int act_dtype;
    int* counts;          // the permutation's counts [N][nblk], or null
    int64_t nblk;
    int tb;               // tokens per count block (divides kRTM)
};

// k rounds of a wavefront arg-max over orderable keys (lane l holds ids
// v*64 + l in key[v], v < nv <= MAXV); among equal keys the lower id wins.
// Returns the selection as a per-lane bit mask over v and the largest logit in
// zmax.  MAXV is a compile-time bound so that every loop unrolls and the
// per-lane arrays stay in fixed registers.
template <int MAXV>
__device__ uint32_t select_topk(const uint32_t* key, int nv, int N, int k, float& zmax) {
    const int lane = threadIdx.x & 63;
    uint32_t taken = 0;
    zmax = 0.0f;
    for (int it = 0; it < k; ++it) {
        uint32_t best = 0;
#pragma unroll
        for (int v = 0; v < MAXV; ++v)
            if (v < nv && !((taken >> v) & 1u) && key[v] > best) best = key[v];
        const uint32_t wmax = wave_max_u32(best);
        int jw = -1;
#pragma unroll
        for (int v = 0; v < MAXV; ++v) {
            if (v < nv && jw < 0) {
                const int j = v * 64 + lane;
                const uint64_t m = __ballot(j < N && !((taken >> v) & 1u) && key[v] == wmax);
                if (m) jw = v * 64 + (__ffsll((unsigned long long)m) - 1);
            }
        }
        if (it == 0) zmax = from_orderable(wmax);
        if (jw >= 0 && (jw & 63) == lane) taken |= 1u << (jw >> 6);
    }
    return taken;
}

// Writes the selected ids ascending from idx + pos0 (and, when gate is not
// null, e[v] / denom aligned with them).
template <int MAXV>
__device__ void write_route(uint32_t taken, int nv, void* idx, int idx_dtype, int64_t pos0,
                            float* gate, const float* e, float denom) {
    const int lane = threadIdx.x & 63;
    int before = 0;
#pragma unroll
    for (int v = 0; v < MAXV; ++v) {
        const bool mine = v < nv && ((taken >> v) & 1u);
        const uint64_t bal = __ballot(mine);
        if (mine) {
            uint64_t lt = lane ? (bal & ((~0ull) >> (64 - lane))) : 0ull;
            int rank = before + __popcll(lt);
            int j = v * 64 + lane;
            int64_t pos = pos0 + rank;
            if (idx_dtype == PR2_I16) ((int16_t*)idx)[pos] = (int16_t)j;
            else ((int32_t*)idx)[pos] = j;
            if (gate) gate[rank] = e[v] / denom;
        }
        before += __popcll(bal);
    }
}

// One wavefront: rollout epilogue of token t from its LDS row of logits.
// bias: the router bias (in LDS or global memory) or null.
template <int MAXV>
__device__ void predict_token(const float* row, int64_t t, int N, int r, const PredictOut& o,
                              const float* bias) {
    const int lane = threadIdx.x & 63;
    const int nv = (N + 63) / 64;
    float* lrow = o.logits_out ? o.logits_out + t * N : nullptr;
    if (o.cache.row) {
        // feature cache: p_old and h_old of a retained token go to its cache row
        const int cr = o.cache.row[t];
        if (cr >= 0 && cr < o.cache.rows) {
            lrow = o.cache.p + (int64_t)cr * N;
            const size_t eb = o.act_dtype == PR2_BF16 ? 2 : 4;
            const size_t bytes = (size_t)o.d * eb;
            const unsigned char* src = (const unsigned char*)o.x + (size_t)t * bytes;
            unsigned char* dst = (unsigned char*)o.cache.h + (size_t)cr * bytes;
            if (bytes % 16 == 0) {
                for (size_t c = lane; c < bytes / 16; c += 64)
                    ((u32x4_t*)dst)[c] = ((const u32x4_t*)src)[c];
            } else {
                for (size_t c = lane; c < bytes / eb; c += 64) {
                    if (eb == 2) ((uint16_t*)dst)[c] = ((const uint16_t*)src)[c];
                    else ((uint32_t*)dst)[c] = ((const uint32_t*)src)[c];
                }
            }
        }
    }
    float z[MAXV];
    uint32_t key[MAXV];
#pragma unroll
    for (int v = 0; v < MAXV; ++v) {
        int j = v * 64 + lane;
        z[v] = -INFINITY;
        key[v] = 0;                          // below every real logit's key
        if (j < N) {
            // p = xW + beta and z = p + (xA) B in fp64, one final rounding
            double p = (double)row[j] + (bias ? (double)bias[j] : 0.0);
            double zz = p;
            if (!o.folded && r > 0) {
                const float* u = row + N;
                if (o.B) {
                    for (int q = 0; q < r; ++q) zz += (double)u[q] * (double)o.B[(int64_t)q * N + j];
                } else {
                    zz += (double)u[j];      // B = identity (full-rank predictor)
                }
            }
            if (lrow) lrow[j] = (float)p;
            z[v] = (float)zz;
            key[v] = orderable(z[v]);
        }
    }
    float zmax;
    const uint32_t taken = select_topk<MAXV>(key, nv, N, o.k, zmax);
    float e[MAXV];
    float s_sel = 0.0f, s_all = 0.0f;
#pragma unroll
    for (int v = 0; v < MAXV; ++v) {
        int j = v * 64 + lane;
        e[v] = 0.0f;
        if (j < N) {
            e[v] = expf(z[v] - zmax);
            s_all += e[v];
            if ((taken >> v) & 1u) s_sel += e[v];
        }
    }
    const float denom = o.renorm ? wave_sum_f32(s_sel) : wave_sum_f32(s_all);
    write_route<MAXV>(taken, nv, o.idx_out, o.idx_dtype, t * o.ldi, o.gate_out ? o.gate_out + t * o.k : nullptr,
                e, denom);
}

// Route-tracking diagnostics of the recorded route against the current router.
struct DiagOut {
    const float* z_ref;            // [T, N] reference logits (for the route KL) or null
    void* cur_idx;                 // [T, k] current top-k, ascending, idx dtype, or null
    int* overlap;                  // [T] |recorded ∩ current top-k| or null
    float* kl;                     // [T] KL(softmax(p) || softmax(z_ref)) or null
    unsigned long long* hist;      // [k + 1] tokens per deviation k - overlap, or null
    float* p_out;                  // [T, N] the current logits p, or null
};

struct ReplayOut {
    const float* b_r;
    int k, renorm;
    const void* idx;
    int idx_dtype;
    int64_t ldi;
    float* gate_out;      // [T, k] or null (diagnostics only)
    int* err;
    int validate;
    DiagOut diag;
    int* counts;          // the permutation's counts [N][nblk], or null
    int64_t nblk;
    int tb;               // tokens per count block (divides kRTM)
};

__device__ __forceinline__ double wave_sum_f64(double v) {
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}
__device__ __forceinline__ double wave_max_f64(double v) {
    for (int off = 32; off >= 1; off >>= 1) v = fmax(v, __shfl_xor(v, off, 64));
    return v;
}

// One wavefront: the current top-k of token t (ties to the lower id, decided on
// the fp32 logits), its overlap with the recorded ids, and the route KL.
template <int MAXV>
__device__ void diag_token(const float* row, int64_t t, int N, const ReplayOut& o,
                           const float* bias, const int* ids, unsigned int* lhist) {
    const int lane = threadIdx.x & 63;
    const int nv = (N + 63) / 64;
    const DiagOut& g = o.diag;
    float p[MAXV];
    uint32_t key[MAXV];
#pragma unroll
    for (int v = 0; v < MAXV; ++v) {
        const int j = v * 64 + lane;
        p[v] = -INFINITY;
        key[v] = 0;
        if (j < N) {
            p[v] = (float)((double)row[j] + (bias ? (double)bias[j] : 0.0));
            key[v] = orderable(p[v]);
            if (g.p_out) g.p_out[t * N + j] = p[v];
        }
    }
    if (!(g.cur_idx || g.overlap || g.kl || g.hist)) return;
    // the reference logits are fetched before the top-k so that their latency
    // overlaps the selection
    float zv[MAXV];
#pragma unroll
    for (int v = 0; v < MAXV; ++v) {
        const int j = v * 64 + lane;
        zv[v] = (g.kl && j < N) ? g.z_ref[t * N + j] : 0.0f;
    }
    float pmax;
    const uint32_t taken = select_topk<MAXV>(key, nv, N, o.k, pmax);
    if (g.cur_idx) write_route<MAXV>(taken, nv, g.cur_idx, o.idx_dtype, t * o.k, nullptr, nullptr, 1.0f);
    if (g.overlap || g.hist) {
        int cnt = 0;
        for (int s = 0; s < o.k; ++s) {
            const int id = ids ? ids[s] : load_id(o.idx, o.idx_dtype, t * o.ldi + s);
            if (id >= 0 && id < N && (id & 63) == lane && ((taken >> (id >> 6)) & 1u)) cnt++;
        }
        cnt = wave_sum_i32(cnt);
        if (lane == 0) {
            if (g.overlap) g.overlap[t] = cnt;
            // the workgroup's LDS histogram when there is one (flushed once per
            // bin by the kernel), else the global counters directly
            if (g.hist) {
                if (lhist) atomicAdd(lhist + (o.k - cnt), 1u);
                else atomicAdd(g.hist + (o.k - cnt), 1ull);
            }
        }
    }
    if (g.kl) {
        double mz = -INFINITY;
#pragma unroll
        for (int v = 0; v < MAXV; ++v) {
            const int j = v * 64 + lane;
            if (j < N) mz = fmax(mz, (double)zv[v]);
        }
        mz = wave_max_f64(mz);
        const double mp = (double)pmax;
        // KL = sum_j e_j / sp * ((p_j - z_j) - shift), e_j = exp(p_j - max p)
        double sp = 0.0, sz = 0.0, ep[MAXV];
#pragma unroll
        for (int v = 0; v < MAXV; ++v) {
            const int j = v * 64 + lane;
            ep[v] = 0.0;
            if (j < N) {
                ep[v] = exp((double)p[v] - mp);
                sp += ep[v];
                sz += exp((double)zv[v] - mz);
            }
        }
        sp = wave_sum_f64(sp);
        sz = wave_sum_f64(sz);
        const double shift = (mp + log(sp)) - (mz + log(sz));
        double acc = 0.0;
#pragma unroll
        for (int v = 0; v < MAXV; ++v) {
            const int j = v * 64 + lane;
            if (j < N) acc += ep[v] * (((double)p[v] - (double)zv[v]) - shift);
        }
        acc = wave_sum_f64(acc) / sp;
        if (lane == 0) g.kl[t] = (float)acc;
    }
}

// One wavefront: replay weights of token t over its recorded ids from the LDS
// row of N current-router logits (predictor bypassed).  bias: the router bias
// (LDS or global) or null; ids: the token's recorded ids already staged in LDS,
// or null to read them from the route record.
template <int MAXV>
__device__ void replay_token(const float* row, int64_t t, int N, const ReplayOut& o,
                             const float* bias, const int* ids, unsigned int* lhist = nullptr) {
    if (o.diag.cur_idx || o.diag.overlap || o.diag.kl || o.diag.hist || o.diag.p_out)
        diag_token<MAXV>(row, t, N, o, bias, ids, lhist);
    if (!o.gate_out) return;
    const int lane = threadIdx.x & 63;
    auto logit = [&](int j) {
        return (float)((double)row[j] + (bias ? (double)bias[j] : 0.0));
    };
    auto id_at = [&](int s) { return ids ? ids[s] : load_id(o.idx, o.idx_dtype, t * o.ldi + s); };
    float ref;
    if (o.renorm) {
        float pmax_sel = -INFINITY;
        for (int s = lane; s < o.k; s += 64) {
            int id = id_at(s);
            if (id >= 0 && id < N) pmax_sel = fmaxf(pmax_sel, logit(id));
        }
        ref = wave_max_f32(pmax_sel);
    } else {
        float pmax_all = -INFINITY;
        for (int j = lane; j < N; j += 64) pmax_all = fmaxf(pmax_all, logit(j));
        ref = wave_max_f32(pmax_all);
    }
    float part = 0.0f;
    if (o.renorm) {
        for (int s = lane; s < o.k; s += 64) {
            int id = id_at(s);
            if (id >= 0 && id < N) part += expf(logit(id) - ref);
        }
    } else {
        for (int j = lane; j < N; j += 64) part += expf(logit(j) - ref);
    }
    const float denom = wave_sum_f32(part);
    for (int s = lane; s < o.k; s += 64) {
        int id = id_at(s);
        float g = 0.0f;
        if (id >= 0 && id < N) g = expf(logit(id) - ref) / denom;
        o.gate_out[t * o.k + s] = g;
    }
    // out-of-range ids are counted by the permutation's count pass alone;
    // repeated ids of a row are counted here
    if (o.validate) {
        int dup = 0;
        for (int s = lane; s < o.k; s += 64) {
            int id = id_at(s);
            for (int s2 = 0; s2 < s; ++s2)
                if (id_at(s2) == id) dup++;
        }
        dup = wave_sum_i32(dup);
        if (lane == 0 && dup) atomicAdd(o.err + ERR_DUP_ID, dup);
    }
}

// ------------------------------------------------- fp64 vector-ALU path ----
template <typename XT>
__global__ void __launch_bounds__(kThreads)
route_predict_kernel(ProjArgs a, PredictOut o) {
    extern __shared__ float smem[];
    float* xs = smem;                                   // TM*KB
    float* ws = xs + a.TM * a.KB;                       // KB*cols_per_pass
    const int cols_per_pass = (kThreads / (a.TM / 4)) * 4;
    float* lg = ws + a.KB * cols_per_pass;              // TM*NC
    const int64_t t0 = (int64_t)blockIdx.x * a.TM;
    project_tile<XT>(a, t0, xs, ws, lg);
    for (int tt = threadIdx.x >> 6; tt < a.TM; tt += kThreads / 64) {
        const int64_t t = t0 + tt;
        if (t >= a.T) break;
        predict_token<kMaxLanesVals>(lg + tt * a.NC, t, a.N, a.r, o, o.b_r);
    }
}

template <typename XT>
__global__ void __launch_bounds__(kThreads)
replay_gates_kernel(ProjArgs a, ReplayOut o) {
    extern __shared__ float smem[];
    float* xs = smem;
    float* ws = xs + a.TM * a.KB;
    const int cols_per_pass = (kThreads / (a.TM / 4)) * 4;
    float* lg = ws + a.KB * cols_per_pass;
    const int64_t t0 = (int64_t)blockIdx.x * a.TM;
    project_tile<XT>(a, t0, xs, ws, lg);
    for (int tt = threadIdx.x >> 6; tt < a.TM; tt += kThreads / 64) {
        const int64_t t = t0 + tt;
        if (t >= a.T) break;
        replay_token<kMaxLanesVals>(lg + tt * a.NC, t, a.N, o, o.b_r, nullptr);
    }
}

// ------------------------------------------- 16-lane group epilogues ----
// The MFMA path runs its epilogues four tokens per wavefront: the 16 lanes of
// group g = lane / 16 own one token, lane l16 = lane % 16 holding experts
// j = 16 v + l16 (v < MAXV16).  Reductions inside the group are DPP row
// rotations (by 8, 4, 2, 1); floating-point sums are then taken from the
// group's first lane so that every lane uses the same value.

// row_ror:n of the 16-lane row (DPP): every lane reads lane (l16 + n) % 16 of its row
template <int N_>
__device__ __forceinline__ int row_ror(int v) {
    static_assert(N_ >= 1 && N_ < 16, "row rotate");
    return __builtin_amdgcn_update_dpp(0, v, 0x120 + N_, 0xf, 0xf, false);
}
__device__ __forceinline__ uint32_t gmax_u32(uint32_t v) {
    v = max(v, (uint32_t)row_ror<8>((int)v));
    v = max(v, (uint32_t)row_ror<4>((int)v));
    v = max(v, (uint32_t)row_ror<2>((int)v));
    return max(v, (uint32_t)row_ror<1>((int)v));
}
__device__ __forceinline__ int gmin_i32(int v) {
    v = min(v, row_ror<8>(v));
    v = min(v, row_ror<4>(v));
    v = min(v, row_ror<2>(v));
    return min(v, row_ror<1>(v));
}
__device__ __forceinline__ float gmax_f32(float v) {
    v = fmaxf(v, __int_as_float(row_ror<8>(__float_as_int(v))));
    v = fmaxf(v, __int_as_float(row_ror<4>(__float_as_int(v))));
    v = fmaxf(v, __int_as_float(row_ror<2>(__float_as_int(v))));
    return fmaxf(v, __int_as_float(row_ror<1>(__float_as_int(v))));
}
// each lane adds in its own rotation order; the group's first lane's sum is used by all
__device__ __forceinline__ float gsum_f32(float v) {
    v += __int_as_float(row_ror<8>(__float_as_int(v)));
    v += __int_as_float(row_ror<4>(__float_as_int(v)));
    v += __int_as_float(row_ror<2>(__float_as_int(v)));
    v += __int_as_float(row_ror<1>(__float_as_int(v)));
    return __shfl(v, 0, 16);
}
__device__ __forceinline__ int gsum_i32(int v) {
    v += row_ror<8>(v);
    v += row_ror<4>(v);
    v += row_ror<2>(v);
    return v + row_ror<1>(v);
}

// Rollout epilogue of token t (valid: t < T) by one 16-lane group.
template <int MAXV16>
__device__ void predict_group(const float* row, int64_t t, bool valid, int N, int r,
                              const PredictOut& o, const float* bias, int* lids = nullptr) {
    const int lane = threadIdx.x & 63;
    const int l16 = lane & 15, grp = lane >> 4;
    float* lrow = (valid && o.logits_out) ? o.logits_out + t * N : nullptr;
    if (valid && o.cache.row) {
        const int cr = o.cache.row[t];
        if (cr >= 0 && cr < o.cache.rows) {
            lrow = o.cache.p + (int64_t)cr * N;
            const size_t eb = o.act_dtype == PR2_BF16 ? 2 : 4;
            const size_t bytes = (size_t)o.d * eb;
            const unsigned char* src = (const unsigned char*)o.x + (size_t)t * bytes;
            unsigned char* dst = (unsigned char*)o.cache.h + (size_t)cr * bytes;
            if (bytes % 16 == 0) {
                for (size_t c = l16; c < bytes / 16; c += 16)
                    ((u32x4_t*)dst)[c] = ((const u32x4_t*)src)[c];
            } else {
                for (size_t c = l16; c < bytes / eb; c += 16) {
                    if (eb == 2) ((uint16_t*)dst)[c] = ((const uint16_t*)src)[c];
                    else ((uint32_t*)dst)[c] = ((const uint32_t*)src)[c];
                }
            }
        }
    }
    float z[MAXV16];
    uint32_t key[MAXV16];
#pragma unroll
    for (int v = 0; v < MAXV16; ++v) {
        const int j = v * 16 + l16;
        z[v] = -INFINITY;
        key[v] = 0;
        if (j < N) {
            const double p = (double)row[j] + (bias ? (double)bias[j] : 0.0);
            double zz = p;
            if (!o.folded && r > 0) {
                const float* u = row + N;
                if (o.B) {
                    for (int q = 0; q < r; ++q) zz += (double)u[q] * (double)o.B[(int64_t)q * N + j];
                } else {
                    zz += (double)u[j];
                }
            }
            if (lrow) lrow[j] = (float)p;
            z[v] = (float)zz;
            key[v] = orderable(z[v]);
        }
    }
    // k rounds of a group arg-max; among equal keys the lower id wins
    uint32_t taken = 0;
    float zmax = 0.0f;
    for (int it = 0; it < o.k; ++it) {
        uint32_t best = 0;
#pragma unroll
        for (int v = 0; v < MAXV16; ++v)
            if (!((taken >> v) & 1u) && key[v] > best) best = key[v];
        const uint32_t gm = gmax_u32(best);
        int cand = 0x7fffffff;
#pragma unroll
        for (int v = MAXV16 - 1; v >= 0; --v)
            if (v * 16 + l16 < N && !((taken >> v) & 1u) && key[v] == gm) cand = v * 16 + l16;
        const int win = gmin_i32(cand);
        if (it == 0) zmax = from_orderable(gm);
        if (win < N && (win & 15) == l16) taken |= 1u << (win >> 4);
    }
    float e[MAXV16];
    float s_sel = 0.0f, s_all = 0.0f;
#pragma unroll
    for (int v = 0; v < MAXV16; ++v) {
        e[v] = 0.0f;
        if (v * 16 + l16 < N) {
            e[v] = expf(z[v] - zmax);
            s_all += e[v];
            if ((taken >> v) & 1u) s_sel += e[v];
        }
    }
    const float denom = gsum_f32(o.renorm ? s_sel : s_all);
    // ids ascending (v-major, then lane), gates aligned
    int before = 0;
#pragma unroll
    for (int v = 0; v < MAXV16; ++v) {
        const bool mine = (taken >> v) & 1u;
        const uint32_t gbits = (uint32_t)(__ballot(mine) >> (16 * grp)) & 0xffffu;
        if (mine && valid) {
            const int rank = before + __popc(gbits & ((1u << l16) - 1u));
            const int j = v * 16 + l16;
            const int64_t pos = t * o.ldi + rank;
            if (o.idx_dtype == PR2_I16) ((int16_t*)o.idx_out)[pos] = (int16_t)j;
            else ((int32_t*)o.idx_out)[pos] = j;
            if (o.gate_out) o.gate_out[t * o.k + rank] = e[v] / denom;
            if (lids) lids[rank] = j;
        }
        before += __popc(gbits);
    }
}

// Replay weights of token t over its recorded ids (ids: staged in LDS, or
// null to read the record) by one 16-lane group.
// Diagnostics of token t by one 16-lane group (lane l16 holds experts
// j = 16 v + l16): current top-k (ties to the lower id), overlap with the
// recorded ids, deviation histogram (LDS, lhist) and route KL in fp64.  The
// fp64 sums run over the group as an xor butterfly, which leaves every lane
// with the same bits.
__device__ __forceinline__ double gsum_f64(double v) {
    v += __shfl_xor(v, 8, 64);
    v += __shfl_xor(v, 4, 64);
    v += __shfl_xor(v, 2, 64);
    return v + __shfl_xor(v, 1, 64);
}

template <int MAXV16>
__device__ void diag_group(const float* row, int64_t t, bool valid, int N, const ReplayOut& o,
                           const float* bias, const int* ids, unsigned int* lhist) {
    const int lane = threadIdx.x & 63;
    const int l16 = lane & 15, grp = lane >> 4;
    const DiagOut& g = o.diag;
    float p[MAXV16], zv[MAXV16];
    uint32_t key[MAXV16];
#pragma unroll
    for (int v = 0; v < MAXV16; ++v) {
        const int j = v * 16 + l16;
        p[v] = -INFINITY;
        zv[v] = 0.0f;
        key[v] = 0;
        if (j < N) {
            p[v] = (float)((double)row[j] + (bias ? (double)bias[j] : 0.0));
            key[v] = orderable(p[v]);
            if (valid && g.p_out) g.p_out[t * N + j] = p[v];
            if (valid && g.kl) zv[v] = g.z_ref[t * N + j];
        }
    }
    if (!(g.cur_idx || g.overlap || g.kl || g.hist)) return;
    uint32_t taken = 0;
    float pmax = 0.0f;
    for (int it = 0; it < o.k; ++it) {
        uint32_t best = 0;
#pragma unroll
        for (int v = 0; v < MAXV16; ++v)
            if (!((taken >> v) & 1u) && key[v] > best) best = key[v];
        const uint32_t gm = gmax_u32(best);
        int cand = 0x7fffffff;
#pragma unroll
        for (int v = MAXV16 - 1; v >= 0; --v)
            if (v * 16 + l16 < N && !((taken >> v) & 1u) && key[v] == gm) cand = v * 16 + l16;
        const int win = gmin_i32(cand);
        if (it == 0) pmax = from_orderable(gm);
        if (win < N && (win & 15) == l16) taken |= 1u << (win >> 4);
    }
    if (g.cur_idx) {
        int before = 0;
#pragma unroll
        for (int v = 0; v < MAXV16; ++v) {
            const bool mine = (taken >> v) & 1u;
            const uint32_t gbits = (uint32_t)(__ballot(mine) >> (16 * grp)) & 0xffffu;
            if (mine && valid) {
                const int rank = before + __popc(gbits & ((1u << l16) - 1u));
                const int64_t pos = t * o.k + rank;
                if (o.idx_dtype == PR2_I16) ((int16_t*)g.cur_idx)[pos] = (int16_t)(v * 16 + l16);
                else ((int32_t*)g.cur_idx)[pos] = v * 16 + l16;
            }
            before += __popc(gbits);
        }
    }
    if (g.overlap || g.hist) {
        int cnt = 0;
        if (valid) {
            for (int s = 0; s < o.k; ++s) {
                const int id = ids ? ids[s] : load_id(o.idx, o.idx_dtype, t * o.ldi + s);
                if (id >= 0 && id < N && (id & 15) == l16 && ((taken >> (id >> 4)) & 1u)) cnt++;
            }
        }
        cnt = gsum_i32(cnt);
        if (valid && l16 == 0) {
            if (g.overlap) g.overlap[t] = cnt;
            if (g.hist) {
                if (lhist) atomicAdd(lhist + (o.k - cnt), 1u);
                else atomicAdd(g.hist + (o.k - cnt), 1ull);
            }
        }
    }
    if (g.kl) {
        // KL(softmax(p) || softmax(z_ref)) = sum_j e_j / sp * ((p_j - z_j) - shift)
        float zm = -INFINITY;
#pragma unroll
        for (int v = 0; v < MAXV16; ++v)
            if (v * 16 + l16 < N) zm = fmaxf(zm, zv[v]);
        zm = fmaxf(zm, __shfl_xor(zm, 8, 64));
        zm = fmaxf(zm, __shfl_xor(zm, 4, 64));
        zm = fmaxf(zm, __shfl_xor(zm, 2, 64));
        zm = fmaxf(zm, __shfl_xor(zm, 1, 64));
        const double mz = (double)zm, mp = (double)pmax;
        double sp = 0.0, sz = 0.0, ep[MAXV16];
#pragma unroll
        for (int v = 0; v < MAXV16; ++v) {
            ep[v] = 0.0;
            if (v * 16 + l16 < N) {
                ep[v] = exp((double)p[v] - mp);
                sp += ep[v];
                sz += exp((double)zv[v] - mz);
            }
        }
        sp = gsum_f64(sp);
        sz = gsum_f64(sz);
        const double shift = (mp + log(sp)) - (mz + log(sz));
        double acc = 0.0;
#pragma unroll
        for (int v = 0; v < MAXV16; ++v)
            if (v * 16 + l16 < N) acc += ep[v] * (((double)p[v] - (double)zv[v]) - shift);
        acc = gsum_f64(acc) / sp;
        if (valid && l16 == 0) g.kl[t] = (float)acc;
    }
}

template <int MAXV16>
__device__ void replay_group(const float* row, int64_t t, bool valid, int N, const ReplayOut& o,
                             const float* bias, const int* ids) {
    const int lane = threadIdx.x & 63;
    const int l16 = lane & 15;
    auto logit = [&](int j) {
        return (float)((double)row[j] + (bias ? (double)bias[j] : 0.0));
    };
    auto id_at = [&](int s) {
        if (ids) return ids[s];
        return valid ? load_id(o.idx, o.idx_dtype, t * o.ldi + s) : -1;
    };
    float mx = -INFINITY;
    if (o.renorm) {
        for (int s = l16; s < o.k; s += 16) {
            const int id = id_at(s);
            if (id >= 0 && id < N) mx = fmaxf(mx, logit(id));
        }
    } else {
#pragma unroll
        for (int v = 0; v < MAXV16; ++v)
            if (v * 16 + l16 < N) mx = fmaxf(mx, logit(v * 16 + l16));
    }
    const float ref = gmax_f32(mx);
    float part = 0.0f;
    if (o.renorm) {
        for (int s = l16; s < o.k; s += 16) {
            const int id = id_at(s);
            if (id >= 0 && id < N) part += expf(logit(id) - ref);
        }
    } else {
#pragma unroll
        for (int v = 0; v < MAXV16; ++v)
            if (v * 16 + l16 < N) part += expf(logit(v * 16 + l16) - ref);
    }
    const float denom = gsum_f32(part);
    for (int s = l16; s < o.k; s += 16) {
        const int id = id_at(s);
        float g = 0.0f;
        if (id >= 0 && id < N) g = expf(logit(id) - ref) / denom;
        if (valid) o.gate_out[t * o.k + s] = g;
    }
    // out-of-range ids are counted by the permutation's count pass alone;
    // repeated ids of a row are counted here
    if (o.validate) {
        int dup = 0;
        for (int s = l16; s < o.k; s += 16) {
            const int id = id_at(s);
            for (int s2 = 0; s2 < s; ++s2)
                if (id_at(s2) == id) dup++;
        }
        dup = gsum_i32(dup);
        if (l16 == 0 && valid && dup) atomicAdd(o.err + ERR_DUP_ID, dup);
    }
}

// ---------------------------------------------------------- MFMA path -----
constexpr int kRTM = 64;                  // tokens per workgroup
constexpr int kRBK = 32;                  // K step
constexpr int kRThreads = 512;            // 8 wavefronts: 2 token halves x 4 column quarters
constexpr int kRMaxNTW = 3;               // 16-column tiles per wavefront (<= 192 columns)

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

// Ws[kt][p * NCp + c][kk] = part p of column c at K index kt*32 + kk (zero for c >= NC).
// Columns: folded -> W_r + A B (or W_r + A when B is null); else [W_r | A].
// Workgroup (32 columns, K step kt): each thread forms 4 weights (neighbouring
// threads read neighbouring columns), the parts are transposed through LDS,
// and each part's 32 x 32 block (2 KiB, contiguous in Ws) is stored 8 bytes
// per thread.
__global__ void __launch_bounds__(256)
router_split_kernel(const float* W_r, const float* A, const float* B, int N, int r, int folded,
                    int NCp, bf16_t* Ws) {
    __shared__ bf16_t tile[3][32][kRBK + 1];
    // the predictor factors this workgroup folds in: A rows kt*32.. and B columns c0..
    constexpr int kStageR = 64;
    __shared__ float sA[kRBK][kStageR];
    __shared__ float sB[kStageR][32];
    const int NC = folded ? N : N + r;
    const int c0 = blockIdx.x * 32, kt = blockIdx.y;
    const int cl = threadIdx.x & 31, kq = threadIdx.x >> 5;
    const int c = c0 + cl;
    const bool staged = folded && B && r > 0 && r <= kStageR;
    if (staged) {
        for (int i = threadIdx.x; i < kRBK * r; i += 256)
            sA[i / r][i % r] = A[((int64_t)kt * kRBK + i / r) * r + i % r];
        for (int i = threadIdx.x; i < r * 32; i += 256)
            sB[i / 32][i % 32] = c0 + i % 32 < N ? B[(int64_t)(i / 32) * N + c0 + i % 32] : 0.0f;
        __syncthreads();
    }
#pragma unroll
    for (int e = 0; e < kRBK / 8; ++e) {
        const int kk = kq + 8 * e;
        const int64_t kg = (int64_t)kt * kRBK + kk;
        double w = 0.0;
        if (c < NC) {
            if (c < N) {
                w = (double)W_r[kg * N + c];
                if (folded && r > 0) {
                    if (staged) {
                        for (int j = 0; j < r; ++j) w += (double)sA[kk][j] * (double)sB[j][cl];
                    } else if (B) {
                        for (int j = 0; j < r; ++j)
                            w += (double)A[kg * r + j] * (double)B[(int64_t)j * N + c];
                    } else {
                        w += (double)A[kg * r + c];
                    }
                }
            } else {
                w = (double)A[kg * r + (c - N)];
            }
        }
        // three bf16 parts; for a weight representable in fp32 they sum to it exactly
        const bf16_t hi = f32_to_bf16((float)w);
        const double r1 = w - (double)bf16_to_f32(hi);
        const bf16_t mid = f32_to_bf16((float)r1);
        tile[0][cl][kk] = hi;
        tile[1][cl][kk] = mid;
        tile[2][cl][kk] = f32_to_bf16((float)(r1 - (double)bf16_to_f32(mid)));
    }
    __syncthreads();
    const int row = threadIdx.x >> 3, q4 = (threadIdx.x & 7) * 4;
#pragma unroll
    for (int p = 0; p < 3; ++p) {
        const bf16_t* t = &tile[p][row][q4];
        const uint2 v = make_uint2((uint32_t)t[0] | ((uint32_t)t[1] << 16),
                                   (uint32_t)t[2] | ((uint32_t)t[3] << 16));
        *(uint2*)(Ws + ((int64_t)kt * 3 * NCp + (int64_t)p * NCp + c0 + row) * kRBK + q4) = v;
    }
}

// 16-byte chunk c of a 64-byte LDS row r sits at position c ^ rswz(r): 16
// consecutive rows read at one chunk hit 16 different 16-byte bank groups.
__device__ __forceinline__ int rswz(int r) { return ((r >> 1) ^ (r >> 2)) & 3; }

template <int n>
__device__ __forceinline__ void router_wait_vmcnt() {
    static_assert(n >= 0 && n < 16, "vmcnt field");
    __builtin_amdgcn_s_waitcnt(0x0f70 | n);
}

template <int NTW>
struct RouterTile {
    static constexpr int NCp = 64 * NTW;
    static constexpr int ROWS = kRTM + 3 * NCp;          // x rows, then hi | mid | lo weight rows
    static constexpr int STAGEB = ROWS * 64;             // one K step of 32 bf16 per row
    static constexpr int NSTAGE = NTW <= 2 ? 4 : 3;      // K steps in flight: NSTAGE - 1
    static constexpr int GROUPS = ROWS / 16;             // 1 KiB copies (16 rows) per stage
    static constexpr int GPW = (GROUPS + 7) / 8;         // copies per wavefront (uniform)
};

// Split-K for small token counts: a few 64-token tiles cannot fill the GPU,
// and each of them would stream every weight of the projection through one CU.
// Phase 1 gives workgroup (tile, pair) the two K steps of one K pair and
// stores their fp32 sum as the fused loop forms it, token-major; phase 2 adds
// the pairs of each logit in K order in fp64 and rounds once, as the fused
// loop does, then runs the epilogue, over workgroups of kRTM2 tokens (more
// workgroups share the serial top-k rounds and the pair sums).  The logits
// are bitwise those of the fused kernel.
constexpr int kRTM2 = 8;                  // tokens per phase-2 workgroup

struct SplitK {
    float* part;       // [npairs][rows][NCp]: phase 1 output, token-major
    int64_t rows;      // tiles * kRTM
    int npairs;
};

template <int NTW, int MODE, int PHASE>   // MODE 0: rollout, 1: replay; PHASE 0: fused, 1, 2: split-K
__global__ void __launch_bounds__(kRThreads)
router_mfma_kernel(const bf16_t* x, const bf16_t* Ws, int64_t T, int d, int N, int r, int NC,
                   PredictOut po, ReplayOut ro, SplitK sk) {
    using RT = RouterTile<NTW>;
    constexpr int NCp = RT::NCp;
    constexpr int NSTAGE = RT::NSTAGE;
    constexpr int GPW = RT::GPW;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[NSTAGE * RT::STAGEB];
    static_assert(NSTAGE * RT::STAGEB >=
                      (int)sizeof(float) * (kRTM * NCp + NCp + kRTM * 64 + 257 + 8 * NCp),
                  "logit tile, bias, staged ids, the deviation histogram and the count "
                  "blocks' histograms must fit over the copy stages");
    // tokens this workgroup's epilogue covers
    constexpr int TOK = PHASE == 2 ? kRTM2 : kRTM;
    const int64_t t0 = (int64_t)blockIdx.x * TOK;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar branches
    const int wr = wave >> 2, wc = wave & 3;

    // Copies straight into LDS, 16 bytes per lane: copy slot i of wavefront w
    // moves 16-row group g = w + 8 i (a wavefront whose last slot falls past
    // the end issues one copy fewer per step), lane l row 16 g + l/4 at
    // position l%4.  Rows below kRTM are tokens (past T: the last token, never
    // written out); the rest are the K-tiled split weights of the step.
    const bf16_t* src[GPW];
    int dst[GPW];
#pragma unroll
    for (int i = 0; i < GPW; ++i) {
        int g = wave + 8 * i;
        if (g >= RT::GROUPS) g = RT::GROUPS - 1;     // never copied (see issue)
        const int row = g * 16 + (lane >> 2);
        const int chunk = (lane & 3) ^ rswz(row);
        if (row < kRTM) {
            const int64_t t = t0 + row < T ? t0 + row : T - 1;
            src[i] = x + t * (int64_t)d + chunk * 8;          // + kt * 32 per step
        } else {
            src[i] = Ws + (int64_t)(row - kRTM) * kRBK + chunk * 8;   // + kt * 3 NCp * 32
        }
        dst[i] = g * 1024;
    }
    // copies per step of this wavefront: GPW, or GPW - 1 when its last slot
    // is past the last group (the waits below count them)
    const bool full_slots = wave + 8 * (GPW - 1) < RT::GROUPS;
    auto issue = [&](int stage, int kt) {
#pragma unroll
        for (int i = 0; i < GPW; ++i) {
            if (i == GPW - 1 && !full_slots) continue;
            const int64_t step = dst[i] < kRTM * 64 ? (int64_t)kt * kRBK
                                                     : (int64_t)kt * 3 * NCp * kRBK;
            __builtin_amdgcn_global_load_lds((const void*)(src[i] + step),
                                             (lds_void*)&lds[stage * RT::STAGEB + dst[i]], 16, 0, 0);
        }
    };

    // replay: the recorded ids of the workgroup's tokens are fetched now and
    // parked in LDS after the K loop, so the epilogue never waits on them
    constexpr int kStageK = 64;                       // ids staged when k <= kStageK
    constexpr int kIdsPerThread = kRTM * kStageK / kRThreads;
    const bool stage_ids = MODE == 1 && ro.idx != nullptr && ro.k <= kStageK;
    int pre_ids[kIdsPerThread];
    if (stage_ids) {
#pragma unroll
        for (int i = 0; i < kIdsPerThread; ++i) {
            const int e = tid + kRThreads * i;
            const int tok = e / ro.k, slot = e % ro.k;
            pre_ids[i] = (e < TOK * ro.k && t0 + tok < T)
                             ? load_id(ro.idx, ro.idx_dtype, (t0 + tok) * ro.ldi + slot) : -1;
        }
    }

    f32x4 acc[2][NTW];
    double acc64[2][NTW][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int t = 0; t < NTW; ++t)
#pragma unroll
            for (int v = 0; v < 4; ++v) { acc[i][t][v] = 0.0f; acc64[i][t][v] = 0.0; }

    // MFMA operand reads: lane l reads row (base + l%16), chunk l/16
    const int lrow = lane & 15;
    const int lch = lane >> 4;
    const int nk = d / kRBK;
    // K steps of this workgroup: all (fused), one pair (phase 1), none (phase 2)
    const int kb = PHASE == 1 ? (int)blockIdx.y * 2 : 0;
    const int ke = PHASE == 1 ? min(nk, kb + 2) : (PHASE == 2 ? 0 : nk);
#pragma unroll
    for (int st = 0; st < NSTAGE - 1; ++st)
        if (kb + st < ke) issue(st, kb + st);
    for (int kt = kb; kt < ke; ++kt) {
        // step kt landed (later steps may be in flight) and every wavefront is
        // done with step kt-1, whose stage is refilled next
        if (kt + NSTAGE - 2 < ke) {
            if (full_slots) router_wait_vmcnt<(NSTAGE - 2) * GPW>();
            else router_wait_vmcnt<(NSTAGE - 2) * (GPW - 1)>();
        } else {
            router_wait_vmcnt<0>();
        }
        // a plain barrier: __syncthreads() would also wait for every copy
        // still in flight (vmcnt(0)) and undo the pipelining
        __builtin_amdgcn_s_waitcnt(0xc07f);      // lgkmcnt(0)
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        if (kt + NSTAGE - 1 < ke) issue((kt - kb + NSTAGE - 1) % NSTAGE, kt + NSTAGE - 1);
        const unsigned char* base = lds + ((kt - kb) % NSTAGE) * RT::STAGEB;
        bf16x8 fa[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int row = wr * 32 + i * 16 + lrow;
            fa[i] = __builtin_bit_cast(bf16x8, *(const u32x4*)(base + row * 64 + ((lch ^ rswz(row)) << 4)));
        }
#pragma unroll
        for (int t = 0; t < NTW; ++t) {
#pragma unroll
            for (int p = 0; p < 3; ++p) {
                const int row = kRTM + p * NCp + (wc * NTW + t) * 16 + lrow;
                bf16x8 fb = __builtin_bit_cast(bf16x8, *(const u32x4*)(base + row * 64 + ((lch ^ rswz(row)) << 4)));
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    acc[i][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb, acc[i][t], 0, 0, 0);
            }
        }
        if (PHASE == 0 && ((kt & 1) || kt + 1 == nk)) {
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int t = 0; t < NTW; ++t)
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        acc64[i][t][v] += (double)acc[i][t][v];
                        acc[i][t][v] = 0.0f;
                    }
        }
    }
    if (PHASE == 1) {
        // the pair's sums, token-major (no global store inside the loop: the
        // compiler would then wait for every copy in flight before each LDS read)
        float* pp = sk.part + ((int64_t)blockIdx.y * sk.rows + (int64_t)blockIdx.x * kRTM) * NCp;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int t = 0; t < NTW; ++t)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int tok = wr * 32 + i * 16 + 4 * (lane >> 4) + v;
                    const int col = (wc * NTW + t) * 16 + (lane & 15);
                    pp[tok * NCp + col] = acc[i][t][v];
                }
        return;
    }
    __syncthreads();
    // logits -> LDS [TOK][NC]; 16x16 accumulator element v of lane l is C[4*(l/16)+v][l%16]
    float* lg = (float*)lds;
    if (PHASE == 2) {
        // logit (row wave + 8 a, column lane + 64 b): the fp64 sum over the K
        // pairs, in order, of phase 1's partial sums, rounded once; eight
        // pairs of every element are loaded before any is added (rows up to
        // the last tile's end exist)
        static_assert(TOK % (kRThreads / 64) == 0, "rows per wavefront");
        constexpr int RPW = TOK / (kRThreads / 64);
        const int64_t pstride = sk.rows * NCp;
        const float* src = sk.part + (t0 + wave) * NCp + lane;
        double s[RPW][NTW];
#pragma unroll
        for (int a = 0; a < RPW; ++a)
#pragma unroll
            for (int b = 0; b < NTW; ++b) s[a][b] = 0.0;
        int p0 = 0;
        for (; p0 + 8 <= sk.npairs; p0 += 8) {
            float v[8][RPW][NTW];
#pragma unroll
            for (int q = 0; q < 8; ++q)
#pragma unroll
                for (int a = 0; a < RPW; ++a)
#pragma unroll
                    for (int b = 0; b < NTW; ++b)
                        v[q][a][b] = src[(int64_t)(p0 + q) * pstride + a * (kRThreads / 64) * NCp + b * 64];
#pragma unroll
            for (int q = 0; q < 8; ++q)
#pragma unroll
                for (int a = 0; a < RPW; ++a)
#pragma unroll
                    for (int b = 0; b < NTW; ++b) s[a][b] += (double)v[q][a][b];
        }
        for (; p0 < sk.npairs; ++p0)
#pragma unroll
            for (int a = 0; a < RPW; ++a)
#pragma unroll
                for (int b = 0; b < NTW; ++b)
                    s[a][b] += (double)src[(int64_t)p0 * pstride + a * (kRThreads / 64) * NCp + b * 64];
#pragma unroll
        for (int a = 0; a < RPW; ++a)
#pragma unroll
            for (int b = 0; b < NTW; ++b)
                if (lane + 64 * b < NC)
                    lg[(wave + a * (kRThreads / 64)) * NC + lane + 64 * b] = (float)s[a][b];
    } else {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int t = 0; t < NTW; ++t)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int tok = wr * 32 + i * 16 + 4 * (lane >> 4) + v;
                    const int col = (wc * NTW + t) * 16 + (lane & 15);
                    if (col < NC) lg[tok * NC + col] = (float)acc64[i][t][v];
                }
    }
    // the router bias and (replay) the staged ids go behind the logit tile
    float* sbias = lg + kRTM * NC;
    int* sids = (int*)(sbias + N);
    const float* b_r = MODE == 0 ? po.b_r : ro.b_r;
    for (int j = tid; j < N; j += kRThreads) sbias[j] = b_r ? b_r[j] : 0.0f;
    // diagnostics: the workgroup's deviation histogram (k + 1 <= 257 bins)
    unsigned int* shist = (unsigned int*)(sids + kRTM * 64);
    const bool lds_hist = MODE == 1 && ro.diag.hist != nullptr;
    if (lds_hist)
        for (int i = tid; i <= ro.k; i += kRThreads) shist[i] = 0u;
    // the permutation's expert counts of the count blocks inside this tile
    // (kRTM / tb <= 8 of them), after the deviation histogram: from the staged
    // recorded ids (replay), or from the ids the epilogue selects (rollout)
    const bool fcount = PHASE == 0 && (MODE == 1 ? ro.counts != nullptr && stage_ids
                                                 : po.counts != nullptr);
    int* chist = (int*)(shist + 257);
    const int ctb = MODE == 1 ? ro.tb : po.tb;
    const int nsub = fcount ? kRTM / ctb : 0;
    for (int i = tid; i < nsub * N; i += kRThreads) chist[i] = 0;
    // histogram of ids[tok * k + s] over this tile's tokens, then its global
    // store; every thread calls it (two barriers)
    auto count_blocks = [&](int k, int* counts, int64_t nblk, int* err) {
        int bad = 0;
        for (int e = tid; e < kRTM * k; e += kRThreads) {
            const int tok = e / k;
            if (t0 + tok >= T) break;
            const int id = sids[e];
            if (id >= 0 && id < N) atomicAdd(&chist[(tok / ctb) * N + id], 1);
            else ++bad;
        }
        if (err) {
            bad = wave_sum_i32(bad);
            if (lane == 0 && bad) atomicAdd(err + ERR_BAD_ID, bad);
        }
        __syncthreads();
        const int64_t b0 = (int64_t)blockIdx.x * nsub;
        for (int i = tid; i < nsub * N; i += kRThreads) {
            const int sub = i / N;
            if (b0 + sub < nblk) counts[(int64_t)(i - sub * N) * nblk + b0 + sub] = chist[i];
        }
    };
    if (stage_ids) {
#pragma unroll
        for (int i = 0; i < kIdsPerThread; ++i) {
            const int e = tid + kRThreads * i;
            if (e < TOK * ro.k) sids[e] = pre_ids[i];
        }
    }
    __syncthreads();
    if (MODE == 1 && fcount) count_blocks(ro.k, ro.counts, ro.nblk, ro.err);
    const bool diag = MODE == 1 && (ro.diag.cur_idx || ro.diag.overlap || ro.diag.kl ||
                                    ro.diag.hist || ro.diag.p_out);
    if (diag) {
        // diagnostics: four tokens per wavefront, one per 16-lane group
        for (int base = wave * 4; base < TOK; base += (kRThreads / 64) * 4) {
            if (t0 + base >= T) break;
            const int tt = base + (lane >> 4);
            const int64_t t = t0 + tt;
            const bool valid = t < T;
            const int* tids = stage_ids ? sids + tt * ro.k : nullptr;
            diag_group<4 * NTW>(lg + tt * NC, t, valid, N, ro, sbias, tids,
                                lds_hist ? shist : nullptr);
            if (ro.gate_out) replay_group<4 * NTW>(lg + tt * NC, t, valid, N, ro, sbias, tids);
        }
        if (lds_hist) {
            __syncthreads();
            for (int i = tid; i <= ro.k; i += kRThreads)
                if (shist[i]) atomicAdd(ro.diag.hist + i, (unsigned long long)shist[i]);
        }
        return;
    }
    // four tokens per wavefront, one per 16-lane group
    for (int base = wave * 4; base < TOK; base += (kRThreads / 64) * 4) {
        if (t0 + base >= T) break;
        const int tt = base + (lane >> 4);
        const int64_t t = t0 + tt;
        const bool valid = t < T;
        if (MODE == 0) predict_group<4 * NTW>(lg + tt * NC, t, valid, N, r, po, sbias,
                                              fcount ? sids + tt * po.k : nullptr);
        else replay_group<4 * NTW>(lg + tt * NC, t, valid, N, ro, sbias,
                                   stage_ids ? sids + tt * ro.k : nullptr);
    }
    if (MODE == 0 && fcount) {
        __syncthreads();
        count_blocks(po.k, po.counts, po.nblk, nullptr);
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

int ncp_of(int NC) { return ((NC + 63) / 64) * 64; }


// split-K below this many 64-token tiles, for K loops of at least kSplitMinSteps
constexpr int kSplitMaxTiles = 32;
constexpr int kSplitMinSteps = 8;

bool use_splitk(const pr2_moe_desc& d) {
    const int64_t tiles = (d.T + kRTM - 1) / kRTM;
    return d.T > 0 && tiles <= kSplitMaxTiles && d.d / kRBK >= kSplitMinSteps;
}

size_t split_weight_bytes(int NC, int d) {
    return ((size_t)3 * ncp_of(NC) * d * sizeof(bf16_t) + 255) & ~(size_t)255;
}

template <int MODE>
hipError_t launch_router_mfma(const pr2_moe_desc& d, int NC, int r, const void* x,
                              const bf16_t* Ws, const PredictOut& po, const ReplayOut& ro,
                              hipStream_t s, bool splitk_ok = true) {
    const int NTW = ncp_of(NC) / 64;
    const int64_t tiles = (d.T + kRTM - 1) / kRTM;
    dim3 grid((unsigned)tiles);
    const bf16_t* xb = (const bf16_t*)x;
    SplitK sk{nullptr, 0, 0};
    if (!splitk_ok || !use_splitk(d)) {
        switch (NTW) {
#define PR2_CASE(n) case n: hipLaunchKernelGGL((router_mfma_kernel<n, MODE, 0>), grid, dim3(kRThreads), 0, s, xb, Ws, d.T, d.d, d.N, r, NC, po, ro, sk); break;
            PR2_CASE(1) PR2_CASE(2) PR2_CASE(3)
#undef PR2_CASE
            default: return hipErrorInvalidValue;
        }
        return hipGetLastError();
    }
    const int npairs = (d.d / kRBK + 1) / 2;
    sk.part = (float*)((char*)Ws + split_weight_bytes(NC, d.d));
    sk.rows = tiles * kRTM;
    sk.npairs = npairs;
    dim3 pgrid((unsigned)tiles, (unsigned)npairs);
    switch (NTW) {
#define PR2_CASE(n) case n: hipLaunchKernelGGL((router_mfma_kernel<n, 0, 1>), pgrid, dim3(kRThreads), 0, s, xb, Ws, d.T, d.d, d.N, r, NC, po, ro, sk); break;
        PR2_CASE(1) PR2_CASE(2) PR2_CASE(3)
#undef PR2_CASE
        default: return hipErrorInvalidValue;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 grid2((unsigned)((d.T + kRTM2 - 1) / kRTM2));
    switch (NTW) {
#define PR2_CASE(n) case n: hipLaunchKernelGGL((router_mfma_kernel<n, MODE, 2>), grid2, dim3(kRThreads), 0, s, xb, Ws, d.T, d.d, d.N, r, NC, po, ro, sk); break;
        PR2_CASE(1) PR2_CASE(2) PR2_CASE(3)
#undef PR2_CASE
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_split(const float* W_r, const float* A, const float* B, const pr2_moe_desc& d,
                        int r, int folded, bf16_t* Ws, hipStream_t s) {
    const int NC = folded ? d.N : d.N + r;
    const int NCp = ncp_of(NC);
    LaunchScope scope("router_split", s);
    hipLaunchKernelGGL(router_split_kernel, dim3((unsigned)(NCp / 32), (unsigned)(d.d / kRBK)),
                       dim3(256), 0, s, W_r, A, B, d.N, r, folded, NCp, Ws);
    return hipGetLastError();
}

}  // namespace

// The split-K buffers are reserved for min(T, the split-K limit) tokens at
// every T, so that a workspace sized for some batch also serves any smaller one.
size_t router_split_weight_bytes(int NC, const pr2_moe_desc& d) {
    return split_weight_bytes(NC, d.d);
}

size_t router_split_bytes(int NC, const pr2_moe_desc& d) {
    size_t b = split_weight_bytes(NC, d.d);
    if (d.T > 0 && d.d / kRBK >= kSplitMinSteps) {
        const int64_t tiles = min((d.T + kRTM - 1) / kRTM, (int64_t)kSplitMaxTiles);
        const int64_t n = tiles * kRTM * ncp_of(NC);
        b += ((d.d / kRBK + 1) / 2) * (size_t)n * sizeof(float);       // pair sums
    }
    return b;
}

bool router_mfma_ok(const pr2_moe_desc& d, int NC) {
    return d.act_dtype == PR2_BF16 && d.d % kRBK == 0 && ncp_of(NC) <= 64 * kRMaxNTW;
}

hipError_t launch_route_predict(const pr2_moe_desc& d, const void* x, const float* W_r,
                                const float* b_r, const float* A, const float* B, void* idx_out,
                                int64_t ldi, float* gate_out, float* logits_out, void* split_ws,
                                hipStream_t s, const FeatureCache& cache, bool reuse_split,
                                bool splitk_ok, int* counts, bool* counted) {
    // reuse_split: split_ws already holds this call's split (same weights, same layout)
    const float* Bn = d.r > 0 ? B : nullptr;
    if (counted) *counted = false;
    // the fused MFMA kernel (not its split-K form) also forms the permutation's
    // counts when its 64-token tiles hold whole count blocks
    auto add_counts = [&](PredictOut& o) {
        if (!counts || (splitk_ok && use_splitk(d)) ||
            !(d.k == 8 || d.k == 16 || d.k == 32 || d.k == 64))
            return;
        o.counts = counts;
        o.tb = perm_tokens_per_block(d.k);
        o.nblk = (d.T + o.tb - 1) / o.tb;
        if (counted) *counted = true;
    };
    if (logits_out == nullptr && cache.row == nullptr && router_mfma_ok(d, d.N)) {
        // the router logits are not wanted: fold the predictor into the weights
        PredictOut o{b_r, Bn, d.k, d.renorm, 1, idx_out, d.idx_dtype, ldi, gate_out, nullptr,
                     FeatureCache{}, x, d.d, d.act_dtype, nullptr, 0, 0};
        add_counts(o);
        if (!reuse_split) {
            hipError_t e = launch_split(W_r, A, Bn, d, d.r, 1, (bf16_t*)split_ws, s);
            if (e != hipSuccess) return e;
        }
        LaunchScope scope("route_predict", s);
        return launch_router_mfma<0>(d, d.N, d.r, x, (const bf16_t*)split_ws, o, ReplayOut{}, s,
                                     splitk_ok);
    }
    PredictOut o{b_r, Bn, d.k, d.renorm, 0, idx_out, d.idx_dtype, ldi, gate_out, logits_out, cache,
                 x, d.d, d.act_dtype, nullptr, 0, 0};
    const int NC = d.N + d.r;
    if (router_mfma_ok(d, NC)) {
        add_counts(o);
        if (!reuse_split) {
            hipError_t e = launch_split(W_r, A, Bn, d, d.r, 0, (bf16_t*)split_ws, s);
            if (e != hipSuccess) return e;
        }
        LaunchScope scope("route_predict", s);
        return launch_router_mfma<0>(d, NC, d.r, x, (const bf16_t*)split_ws, o, ReplayOut{}, s,
                                     splitk_ok);
    }
    ProjArgs a;
    a.x = x;
    a.W_r = W_r;
    a.A = d.r > 0 ? A : nullptr;
    a.T = d.T;
    a.d = d.d;
    a.N = d.N;
    a.r = d.r;
    a.NC = NC;
    pick_tile(a);
    dim3 grid((unsigned)((d.T + a.TM - 1) / a.TM));
    size_t smem = router_smem(a);
    LaunchScope scope("route_predict", s);
    if (d.act_dtype == PR2_BF16)
        hipLaunchKernelGGL(route_predict_kernel<bf16_t>, grid, dim3(kThreads), smem, s, a, o);
    else
        hipLaunchKernelGGL(route_predict_kernel<float>, grid, dim3(kThreads), smem, s, a, o);
    return hipGetLastError();
}

namespace {

__global__ void __launch_bounds__(64) zero_u64_kernel(unsigned long long* p, int n) {
    for (int i = threadIdx.x; i < n; i += 64) p[i] = 0ull;
}

hipError_t launch_router_replay(const pr2_moe_desc& d, const void* x, const float* W_r,
                                const ReplayOut& o, void* split_ws, const char* name,
                                hipStream_t s) {
    if (router_mfma_ok(d, d.N)) {
        hipError_t e = launch_split(W_r, nullptr, nullptr, d, 0, 0, (bf16_t*)split_ws, s);
        if (e != hipSuccess) return e;
        LaunchScope scope(name, s);
        return launch_router_mfma<1>(d, d.N, 0, x, (const bf16_t*)split_ws, PredictOut{}, o, s);
    }
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
    LaunchScope scope(name, s);
    if (d.act_dtype == PR2_BF16)
        hipLaunchKernelGGL(replay_gates_kernel<bf16_t>, grid, dim3(kThreads), smem, s, a, o);
    else
        hipLaunchKernelGGL(replay_gates_kernel<float>, grid, dim3(kThreads), smem, s, a, o);
    return hipGetLastError();
}

}  // namespace

bool replay_counts_fused(const pr2_moe_desc& d) {
    return router_mfma_ok(d, d.N) && !use_splitk(d) &&
           (d.k == 8 || d.k == 16 || d.k == 32 || d.k == 64);
}

hipError_t launch_replay_gates(const pr2_moe_desc& d, const void* x, const void* idx, int64_t ldi,
                               const float* W_r, const float* b_r, float* gate_out, int* err,
                               void* split_ws, hipStream_t s, const RouteDiag* diag,
                               int* counts) {
    const char* v = getenv("PR2_VALIDATE");
    DiagOut g{};
    if (diag) {
        // the diagnostics epilogue runs on the same logits, before the weights
        g = DiagOut{diag->z_ref, diag->cur_idx, diag->overlap, diag->kl, diag->hist,
                    diag->p_out};
        if (diag->hist) {
            LaunchScope scope("replay_diagnostics_zero", s);
            hipLaunchKernelGGL(zero_u64_kernel, dim3(1), dim3(64), 0, s, diag->hist, d.k + 1);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
    }
    ReplayOut o{b_r, d.k, d.renorm, idx, d.idx_dtype, ldi, gate_out, err,
                (v && v[0] == '1') ? 1 : 0, g, nullptr, 0, 0};
    if (counts) {
        if (!replay_counts_fused(d)) return hipErrorInvalidValue;
        o.counts = counts;
        o.tb = perm_tokens_per_block(d.k);
        o.nblk = (d.T + o.tb - 1) / o.tb;
    }
    return launch_router_replay(d, x, W_r, o, split_ws, "replay_gates", s);
}

hipError_t launch_router_logits(const pr2_moe_desc& d, const void* x, const float* W_r,
                                const float* b_r, float* p_out, void* split_ws, hipStream_t s) {
    DiagOut g{};
    g.p_out = p_out;
    ReplayOut o{b_r, d.k, 1, nullptr, d.idx_dtype, d.k, nullptr, nullptr, 0, g, nullptr, 0, 0};
    return launch_router_replay(d, x, W_r, o, split_ws, "router_logits", s);
}

hipError_t launch_route_diagnostics(const pr2_moe_desc& d, const void* x, const void* idx,
                                    int64_t ldi, const float* W_r, const float* b_r,
                                    const float* z_ref, void* cur_idx, int* overlap, float* kl,
                                    unsigned long long* hist, void* split_ws, hipStream_t s) {
    if (hist) {
        LaunchScope scope("route_diagnostics_zero", s);
        hipLaunchKernelGGL(zero_u64_kernel, dim3(1), dim3(64), 0, s, hist, d.k + 1);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (d.T == 0) return hipSuccess;
    ReplayOut o{b_r, d.k, 1, idx, d.idx_dtype, ldi, nullptr, nullptr, 0,
                DiagOut{z_ref, cur_idx, overlap, kl, hist, nullptr}, nullptr, 0, 0};
    return launch_router_replay(d, x, W_r, o, split_ws, "route_diagnostics", s);
}

}  // namespace pr2
