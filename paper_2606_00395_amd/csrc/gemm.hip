// Grouped expert GEMMs over the permuted routes (gated-MLP experts, Appendix E.2;
// weighted sum of Eq. pr2_output).
//
//   GEMM1  H[rows_e, m] = silu(X_e W_gate_e^T) * (X_e W_up_e^T)   X_e gathered from x
//   GEMM2  O[rows_e, d] = g * (H_e W_down_e^T)                     g = replay weight
//
// bf16 path (d % 256 == 0, m % 128 == 0): one workgroup computes a 256-row tile
// of one expert against a 256-row panel of weights (GEMM1: 128 gate rows + the
// matching 128 up rows; GEMM2: 256 rows of W_down).  K advances in slices of 64
// (one 128-byte line per row) copied straight from global memory into LDS with
// 16-byte DMA loads (no register staging), two LDS stages deep, 16-byte chunks
// XOR-swizzled per row so the MFMA operand reads are free of bank conflicts.
// Eight wavefronts (two per SIMD) in a 4 x 2 arrangement each own 64 rows x 128
// panel rows as 2 x 4 tiles of v_mfma_f32_32x32x16_bf16 (fp32 accumulation); a
// wavefront whose rows are all past the end of a partial tile skips its MFMAs.
// GEMM1's epilogue applies SwiGLU in registers (gate and up tiles of the same
// columns live in the same lanes) and rounds H to bf16; GEMM2's epilogue scales
// by the route weight and rounds O to bf16.  Workgroups are mapped so that each
// XCD takes a contiguous range of the tile list (same experts, shared L2).
//
// Other shapes and the fp32 path use a plain one-thread-per-output kernel.
#include "common.h"

namespace pr2 {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int BM = kTileM;      // 256 rows per tile
constexpr int BP = 256;         // weight panel rows per tile
constexpr int BK = 64;          // K slice: one 128-byte line per row
constexpr int ROWB = BK * 2;    // bytes per LDS row (unpadded; chunks are swizzled)
constexpr int kGemmThreads = 512;   // 8 wavefronts: 4 row quarters x 2 panel halves
constexpr int kNumXcd = 8;
constexpr int kGroups = (BM + BP) / 8 / (kGemmThreads / 64);   // 8-row DMA groups per wavefront

struct MfmaArgs {
    const bf16_t* A;        // GEMM1: x [T, d]; GEMM2: H [T*k, m]
    const int* perm_src;    // permuted row -> t*k + s
    int k;
    const bf16_t* W0;       // GEMM1: W_gate; GEMM2: W_down
    const bf16_t* W1;       // GEMM1: W_up
    int K;                  // reduction length (d or m)
    int n_out;              // output row length (m or d)
    int ntn;                // panels per expert
    int64_t w_stride;       // elements per expert weight matrix
    const int* tiles;
    const int* tile_count;
    const float* gate;      // GEMM2
    bf16_t* out;
};

__device__ __forceinline__ float silu_f(float a) { return a / (1.0f + __expf(-a)); }

// 16-byte chunk c of LDS row r is stored at position c ^ swz(r): rows 16 apart
// repeat the pattern, and any 16 (or 8) consecutive rows read at the same
// chunk hit disjoint banks.
__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

template <int MODE>
__global__ void __launch_bounds__(kGemmThreads)
grouped_gemm_mfma(MfmaArgs g) {
    __shared__ __attribute__((aligned(1024))) unsigned char lds[2][(BM + BP) * ROWB];

    // XCD-aware mapping: physical block b runs on XCD b % 8; give each XCD a
    // contiguous range of the (tile, panel) work list.
    const int64_t L = (int64_t)(*g.tile_count) * g.ntn;
    const int64_t per_xcd = (L + kNumXcd - 1) / kNumXcd;
    const int64_t local = blockIdx.x / kNumXcd;
    if (local >= per_xcd) return;
    const int64_t logical = (int64_t)(blockIdx.x % kNumXcd) * per_xcd + local;
    if (logical >= L) return;
    const int tile = (int)(logical / g.ntn);
    const int pn = (int)(logical % g.ntn);
    const int expert = g.tiles[3 * tile + 0];
    const int row0 = g.tiles[3 * tile + 1];
    const int rows = g.tiles[3 * tile + 2];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wr = wave >> 1;     // 64-row quarter
    const int wc = wave & 1;      // panel half
    // a wavefront whose 64 rows are all past the tile's end only helps copy
    const bool active = wr * 64 < rows;

    // DMA assignments: wavefront w copies 8-row groups w*kGroups .. of the
    // [A rows | panel rows] tile; lane l moves row 8*grp + l/8, position l%8.
    const bf16_t* src[kGroups];
#pragma unroll
    for (int i = 0; i < kGroups; ++i) {
        const int grp = wave * kGroups + i;
        const int r = grp * 8 + (lane >> 3);          // row in [0, BM + BP)
        const int chunk = (lane & 7) ^ swz(r);
        const bf16_t* rowp;
        if (r < BM) {
            // rows past the tile's end read a valid row; their results are never stored
            const int rr = r < rows ? r : 0;
            if (MODE == 0) rowp = g.A + (int64_t)(g.perm_src[row0 + rr] / g.k) * g.K;
            else rowp = g.A + ((int64_t)row0 + rr) * g.K;
        } else {
            const int pr = r - BM;
            if (MODE == 0)
                rowp = (pr < 128 ? g.W0 : g.W1) + (int64_t)expert * g.w_stride +
                       (int64_t)(pn * 128 + (pr & 127)) * g.K;
            else
                rowp = g.W0 + (int64_t)expert * g.w_stride + (int64_t)(pn * BP + pr) * g.K;
        }
        src[i] = rowp + chunk * 8;
    }
    auto issue = [&](int buf, int k0) {
#pragma unroll
        for (int i = 0; i < kGroups; ++i) {
            const int grp = wave * kGroups + i;
            __builtin_amdgcn_global_load_lds((const void*)(src[i] + k0),
                                             (lds_void*)&lds[buf][grp * 8 * ROWB], 16, 0, 0);
        }
    };

    f32x16 acc[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    // LDS rows each lane reads for its MFMA operands
    const int lrow = lane & 31;
    const int lhalf = lane >> 5;           // 8-element half of the K=16 step
    int a_row[2], b_row[4];
#pragma unroll
    for (int i = 0; i < 2; ++i) a_row[i] = wr * 64 + i * 32 + lrow;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        int prow;
        if (MODE == 0) prow = (j < 2 ? 0 : 128) + wc * 64 + (j & 1) * 32 + lrow;
        else prow = wc * 128 + j * 32 + lrow;
        b_row[j] = BM + prow;
    }

    const int nk = g.K / BK;
    issue(0, 0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < nk) issue(cur ^ 1, (kt + 1) * BK);
        if (active) {
            const unsigned char* base = lds[cur];
#pragma unroll
            for (int ks = 0; ks < BK / 16; ++ks) {
                const int c = 2 * ks + lhalf;
                bf16x8 fa[2], fb[4];
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    fa[i] = __builtin_bit_cast(bf16x8, *(const u32x4*)(base + a_row[i] * ROWB +
                                                                       ((c ^ swz(a_row[i])) << 4)));
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    fb[j] = __builtin_bit_cast(bf16x8, *(const u32x4*)(base + b_row[j] * ROWB +
                                                                       ((c ^ swz(b_row[j])) << 4)));
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j],
                                                                             acc[i][j], 0, 0, 0);
            }
        }
        __builtin_amdgcn_s_waitcnt(0);     // this wavefront's copies of the next slice landed
        __syncthreads();
    }
    if (!active) return;

    // epilogue: 32x32 accumulator element v of lane l is
    // C[8*(v/4) + 4*(l/32) + v%4][l%32]
    const int ccol = lane & 31;
    const int rbase = 4 * (lane >> 5);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int r = wr * 64 + i * 32 + 8 * (v >> 2) + rbase + (v & 3);
            if (r >= rows) continue;
            const int64_t orow = (int64_t)row0 + r;
            if (MODE == 0) {
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const int col = pn * 128 + wc * 64 + j * 32 + ccol;
                    const float h = silu_f(acc[i][j][v]) * acc[i][j + 2][v];
                    g.out[orow * g.n_out + col] = f32_to_bf16(h);
                }
            } else {
                const float gw = g.gate[g.perm_src[orow]];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int col = pn * BP + wc * 128 + j * 32 + ccol;
                    g.out[orow * g.n_out + col] = f32_to_bf16(gw * acc[i][j][v]);
                }
            }
        }
    }
}

// ---------------------------------------------------------------- generic --
template <typename T>
__global__ void __launch_bounds__(256)
gemm1_generic(const T* x, const int* perm_src, int k, const T* Wg, const T* Wu, int d, int m,
              const int* tiles, const int* tile_count, T* H) {
    const int tile = blockIdx.x;
    if (tile >= *tile_count) return;
    const int expert = tiles[3 * tile], row0 = tiles[3 * tile + 1], rows = tiles[3 * tile + 2];
    const int r = threadIdx.x;
    const int col = blockIdx.y;
    if (r >= rows || col >= m) return;
    const int64_t tok = perm_src[row0 + r] / k;
    const T* xr = x + tok * d;
    const T* g = Wg + ((int64_t)expert * m + col) * d;
    const T* u = Wu + ((int64_t)expert * m + col) * d;
    float a = 0.0f, b = 0.0f;
    for (int i = 0; i < d; ++i) {
        float xv = Act<T>::to_f32(xr[i]);
        a = fmaf(xv, Act<T>::to_f32(g[i]), a);
        b = fmaf(xv, Act<T>::to_f32(u[i]), b);
    }
    H[(int64_t)(row0 + r) * m + col] = Act<T>::from_f32(a / (1.0f + expf(-a)) * b);
}

template <typename T>
__global__ void __launch_bounds__(256)
gemm2_generic(const T* H, const int* perm_src, const float* gate, const T* Wd, int d, int m,
              const int* tiles, const int* tile_count, T* O) {
    const int tile = blockIdx.x;
    if (tile >= *tile_count) return;
    const int expert = tiles[3 * tile], row0 = tiles[3 * tile + 1], rows = tiles[3 * tile + 2];
    const int r = threadIdx.x;
    const int col = blockIdx.y;
    if (r >= rows || col >= d) return;
    const T* h = H + (int64_t)(row0 + r) * m;
    const T* w = Wd + ((int64_t)expert * d + col) * m;
    float a = 0.0f;
    for (int i = 0; i < m; ++i) a = fmaf(Act<T>::to_f32(h[i]), Act<T>::to_f32(w[i]), a);
    O[(int64_t)(row0 + r) * d + col] = Act<T>::from_f32(gate[perm_src[row0 + r]] * a);
}

}  // namespace

bool mfma_shape_ok(const pr2_moe_desc& d) {
    return d.act_dtype == PR2_BF16 && d.d % BP == 0 && d.m % 128 == 0 && d.d % BK == 0 &&
           d.m % BK == 0;
}

hipError_t launch_expert_gemms(const pr2_moe_desc& d, const void* x, const void* W_gate,
                               const void* W_up, const void* W_down, const float* gate,
                               const ReplayWs& ws, hipStream_t s) {
    if (mfma_shape_ok(d)) {
        MfmaArgs g1{};
        g1.A = (const bf16_t*)x;
        g1.perm_src = ws.perm_src;
        g1.k = d.k;
        g1.W0 = (const bf16_t*)W_gate;
        g1.W1 = (const bf16_t*)W_up;
        g1.K = d.d;
        g1.n_out = d.m;
        g1.ntn = d.m / 128;
        g1.w_stride = (int64_t)d.m * d.d;
        g1.tiles = ws.tiles;
        g1.tile_count = ws.tile_count;
        g1.gate = gate;
        g1.out = (bf16_t*)ws.H;
        int64_t work = ws.max_tiles * g1.ntn;
        int64_t grid = ((work + kNumXcd - 1) / kNumXcd) * kNumXcd;
        {
            LaunchScope scope("gemm1_gate_up_swiglu", s);
            hipLaunchKernelGGL(grouped_gemm_mfma<0>, dim3((unsigned)grid), dim3(kGemmThreads), 0,
                               s, g1);
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        MfmaArgs g2 = g1;
        g2.A = (const bf16_t*)ws.H;
        g2.W0 = (const bf16_t*)W_down;
        g2.W1 = nullptr;
        g2.K = d.m;
        g2.n_out = d.d;
        g2.ntn = d.d / BP;
        g2.out = (bf16_t*)ws.O;
        work = ws.max_tiles * g2.ntn;
        grid = ((work + kNumXcd - 1) / kNumXcd) * kNumXcd;
        {
            LaunchScope scope("gemm2_down_scale", s);
            hipLaunchKernelGGL(grouped_gemm_mfma<1>, dim3((unsigned)grid), dim3(kGemmThreads), 0,
                               s, g2);
        }
        return hipGetLastError();
    }
    static_assert(BM == 256, "generic kernels map one thread per tile row");
    dim3 grid1((unsigned)ws.max_tiles, (unsigned)d.m);
    dim3 grid2((unsigned)ws.max_tiles, (unsigned)d.d);
    if (d.act_dtype == PR2_BF16) {
        {
            LaunchScope scope("gemm1_generic", s);
            hipLaunchKernelGGL(gemm1_generic<bf16_t>, grid1, dim3(256), 0, s, (const bf16_t*)x,
                               ws.perm_src, d.k, (const bf16_t*)W_gate, (const bf16_t*)W_up, d.d,
                               d.m, ws.tiles, ws.tile_count, (bf16_t*)ws.H);
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        LaunchScope scope("gemm2_generic", s);
        hipLaunchKernelGGL(gemm2_generic<bf16_t>, grid2, dim3(256), 0, s, (const bf16_t*)ws.H,
                           ws.perm_src, gate, (const bf16_t*)W_down, d.d, d.m, ws.tiles,
                           ws.tile_count, (bf16_t*)ws.O);
    } else {
        {
            LaunchScope scope("gemm1_generic", s);
            hipLaunchKernelGGL(gemm1_generic<float>, grid1, dim3(256), 0, s, (const float*)x,
                               ws.perm_src, d.k, (const float*)W_gate, (const float*)W_up, d.d,
                               d.m, ws.tiles, ws.tile_count, (float*)ws.H);
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        LaunchScope scope("gemm2_generic", s);
        hipLaunchKernelGGL(gemm2_generic<float>, grid2, dim3(256), 0, s, (const float*)ws.H,
                           ws.perm_src, gate, (const float*)W_down, d.d, d.m, ws.tiles,
                           ws.tile_count, (float*)ws.O);
    }
    return hipGetLastError();
}

}  // namespace pr2
