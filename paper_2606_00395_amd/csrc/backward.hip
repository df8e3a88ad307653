// Replay backward: gradients of <dy, y> for the replay forward with the
// recorded ids held fixed (Sec. 4.1, replay during training: the experts and
// the current router receive gradients through the replayed set; the
// predictor is bypassed and receives none).  Weights are the renormalised
// replay weights g = softmax of the k recorded logits, or (renorm = 0) the
// paper-literal rho_j of the softmax over all N logits (Eq. pr2_output).
//
// Per route (token t, slot s, expert e, permuted row q), with X = x_t:
//   a = X W_gate_e^T, u = X W_up_e^T, H = silu(a) * u       (recomputed)
//   G = dy_t W_down_e                   [m]   so that   dg = <H, G> = <dy_t, E_e(X)>
//   dH = g G,  du = dH silu(a),  da = dH u silu'(a)
//   dx_t   += da W_gate_e + du W_up_e + sum_j dp_tj W_r[:, j]
//   dW_down_e = sum_q dy_t^T (g H),  dW_gate_e = sum_q da^T X,  dW_up_e = sum_q du^T X
//   dp_ts = g_ts (dg_ts - sum_s' g_ts' dg_ts'),  dW_r[:, e] = sum_q X dp,  db_r[e] = sum_q dp
//
// bf16 path: four grouped GEMMs on v_mfma_f32_32x32x16_bf16 with the tile
// shape of the forward kernels (256 x 256 output tile, K slices of 64, two
// LDS stages, eight wavefronts of 64 x 128), every operand copied global ->
// LDS by 16-byte direct-to-LDS loads.  An operand whose K index runs along
// its rows in memory (the weights in the input-gradient GEMMs, both operands
// of the token-contracted weight-gradient GEMMs) is kept K-major in LDS and
// its MFMA fragments are read with the transposing LDS read of gfx950
// (ds_read_b64_tr_b16), so no operand passes through registers on its way in.
// The router weight gradient is a separate pass over the x rows.
// Every gradient is written exactly once (no atomics): results are
// deterministic and overwrite the outputs.
#include "common.h"

namespace pr2 {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) v4s lds_v4s;

constexpr int BM = 256;         // output tile rows
constexpr int BN = 256;         // output tile columns
constexpr int BK = 64;          // K slice
constexpr int ROWB = BK * 2;    // bytes per LDS row
constexpr int NSTAGE = 2;
constexpr int WM = 64, WN = 128;
constexpr int MI = WM / 32, NJ = WN / 32;
constexpr int NWAVE = 8;
constexpr int kThreads = 64 * NWAVE;
constexpr int kGroups = 8;      // 8-row DMA groups per wavefront (4 wavefronts x 64 rows)
constexpr int STAGEB = (BM + BN) * ROWB;
constexpr int LDSB = NSTAGE * STAGEB;
constexpr int kNumXcd = 8;

enum { DH = 0, DX = 1, WD = 2, WGU = 3 };

struct BwdArgs {
    const int* perm_src;     // permuted row -> t*k + s
    const int* tiles;        // (expert, first permuted row, rows) per 256-row tile
    const int* tile_count;
    const int* offsets;      // [N+1] first permuted row of each expert
    const int* order;        // [N] experts by decreasing route count (ties: lower id)
    int k, N, d, m, Tk;
    uint32_t kmul;           // ceil(2^32 / k), 0 for k = 1 (token of a route entry by multiply-high)
    int ntn;                 // DH, DX: 256-column panels per tile
    const bf16_t* x;
    const bf16_t* dy;
    const bf16_t* Wg;
    const bf16_t* Wu;
    const bf16_t* Wd;
    const float* gate;       // [T*k] replay weights, route order
    const bf16_t* AUin;      // [T*k, 2m]: a | u (DH reads them here; may be AU itself)
    bf16_t* AU;              // [T*k, 2m]: da | du out (and what DX, WGU read)
    bf16_t* Hg;              // [T*k, m]: g * H
    float* dgp;              // [T*k, m/128] partial gate gradients
    bf16_t* dxr;             // [T*k, d] per-route input gradients
    float* dWg;
    float* dWu;
    float* dWd;
};

__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

template <int n>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(n >= 0 && n < 16, "vmcnt field");
    __builtin_amdgcn_s_waitcnt(0x0f70 | n);
}

// Direct global -> LDS copy of 16 bytes per lane: lane l fills dst + 16 l
// (dst is the same for the whole wavefront).  Written as inline assembly:
// issued through the compiler builtin, every later LDS read that carries no
// type-based alias information (the transposing reads do not) is made to wait
// for all copies in flight, which serialises each K slice's copies with the
// slice before.  The K loop waits for its own copies explicitly (vmcnt 0 ahead
// of the barrier that publishes a stage), so nothing relies on that wait.
// M0 takes the LDS base; the nop covers the M0-write -> LDS-DMA hazard.  The
// compiler keeps no value of its own in M0 in these kernels (it sets M0 only
// right before its own LDS-DMA and message instructions, and they use none),
// so the clobber it warns about is harmless here.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void* src, const unsigned char* dst) {
    const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(const lds_void*)dst);
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 1\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(src), "s"(m0)
                 : "memory", "m0");
}
#pragma clang diagnostic pop

// value of lane (l + n) mod 16 of this lane's group of 16 (DPP row rotate)
template <int n>
__device__ __forceinline__ float row_ror_f(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x120 + n, 0xf, 0xf, false));
}

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ uint32_t pack_bf(float lo, float hi) {
    return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

// SwiGLU backward of one element.  H is taken at the precision the forward
// stores it (rounded to bf16 when round_h), so that dg = <H, G> is the
// gradient of the computed output.
__device__ __forceinline__ void swiglu_bwd(float a, float u, float G, float g, bool round_h,
                                           float& da, float& du, float& hg, float& hG) {
    const float sig = __builtin_amdgcn_rcpf(1.0f + __expf(-a));   // as the forward's silu
    const float s = a * sig;
    float H = s * u;
    if (round_h) H = bf16_to_f32(f32_to_bf16(H));
    const float dH = g * G;
    du = dH * s;
    da = dH * u * (sig * (1.0f + a * (1.0f - sig)));
    hg = g * H;
    hG = H * G;
}

// all-zero source row for the copies of K rows past an expert's last route
__device__ __attribute__((aligned(16))) const bf16_t kZeroRow[BN] = {};

template <int MODE>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
bwd_gemm(BwdArgs g) {
    __shared__ __attribute__((aligned(1024))) unsigned char lds[LDSB];
    constexpr bool kRowTiles = (MODE == DH || MODE == DX);   // C rows are permuted routes

    // ---- work item
    int nct = 1;
    int expert, row0 = 0, rows = BM, pn = 0, rt = 0, ct = 0, klen;
    if (kRowTiles) {
        // XCD-aware: XCD b % 8 takes a contiguous range of the (tile, panel) list
        const int64_t L = (int64_t)(*g.tile_count) * g.ntn;
        const int64_t per_xcd = (L + kNumXcd - 1) / kNumXcd;
        const int64_t local = blockIdx.x / kNumXcd;
        if (local >= per_xcd) return;
        const int64_t logical = (int64_t)(blockIdx.x % kNumXcd) * per_xcd + local;
        if (logical >= L) return;
        const int tile = (int)(logical / g.ntn);
        pn = (int)(logical % g.ntn);
        expert = g.tiles[3 * tile + 0];
        row0 = g.tiles[3 * tile + 1];
        rows = g.tiles[3 * tile + 2];
        klen = MODE == DH ? g.d : 2 * g.m;
    } else {
        // Token-contracted: an item's cost grows with its expert's route count.
        // Experts are dealt to the XCDs round-robin in decreasing count order and
        // each XCD runs its experts' output tiles biggest first (the dispatcher
        // starts workgroups in index order), so the busiest experts neither pile
        // up on one XCD nor start last.
        const int nrt = MODE == WD ? g.d / BM : 2 * g.m / BM;
        nct = MODE == WD ? g.m / BN : g.d / BN;
        const int per_e = nrt * nct;
        const int xcd = blockIdx.x % kNumXcd;
        const int local = blockIdx.x / kNumXcd;
        const int slot = local / per_e;
        if (xcd + kNumXcd * slot >= g.N) return;
        expert = g.order[xcd + kNumXcd * slot];
        const int tt = local % per_e;
        rt = tt / nct;
        ct = tt % nct;
        row0 = g.offsets[expert];
        klen = g.offsets[expert + 1] - row0;
    }

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar branches
    const int wr = wave >> 1;            // 64-row block of the output tile
    const int wc = wave & 1;             // 128-column block
    const int half = wave >> 2;          // operand this wavefront loads: 0 rows, 1 columns
    const bool active = wr * WM < rows;

    // ---- operand loading.  Both operands are copied global -> LDS with
    // 16-byte direct-to-LDS loads; wavefronts 0-3 copy the row operand (C
    // rows), 4-7 the column operand.  A K-contiguous operand (the gathered dy
    // rows of DH, the da | du rows of DX) is stored as 256 tile rows of 128
    // bytes (64 K values), 16-byte chunks XOR-swizzled per row.  A K-strided
    // operand (the weights of DH and DX, both operands of WD and WGU) is
    // stored K-major: 64 K rows of 512 bytes (the tile's 256 columns), chunk c
    // of K row kr at position c ^ 4 (kr & 3).  Both forms fill 32 KiB.
    constexpr bool kStridedA = (MODE == WD || MODE == WGU);
    const bool strided = half == 1 || kStridedA;
    const int wq = wave & 3;
    const int64_t ew = (int64_t)expert * g.m * g.d;      // elements per expert matrix

    // K-contiguous rows (DH: gathered dy, DX: da | du): copy group i of this
    // wavefront moves tile rows 8 (8 wq + i) .. +7
    const bf16_t* sbase = MODE == DH ? g.dy : g.AU;
    uint32_t soff[kGroups];
    if (!kStridedA) {
#pragma unroll
        for (int i = 0; i < kGroups; ++i) {
            const int r = wq * (kGroups * 8) + i * 8 + lane / 8;
            const int chunk = (lane % 8) ^ swz(r);
            const int rr = r < rows ? r : 0;
            uint32_t off;
            if (MODE == DH)
                off = (uint32_t)(min(max(g.perm_src[row0 + rr], 0), g.Tk - 1) / g.k) * (uint32_t)g.d;
            else
                off = (uint32_t)(row0 + rr) * (uint32_t)(2 * g.m);
            soff[i] = off + chunk * 8;
        }
    }
    // K-strided: copy instruction i of this wavefront moves K rows
    // k0 + 2 i (lanes 0-31) and k0 + 2 i + 1 (lanes 32-63) of the slice,
    // k0 = 16 wq; lane l lands at chunk position l % 32 and so loads chunk
    // (l % 32) ^ 4 ((2 i + l / 32) & 3) of its K row: one column pattern for
    // even i, one for odd.  Rows at or past klen read zeros.  The two rows of
    // a copy are the same for the whole wavefront, so their addresses are
    // formed on the scalar unit and each lane only adds its own offset.
    const int hi = lane >> 5;
    const int cpat[2] = {8 * ((lane & 31) ^ (4 * hi)), 8 * ((lane & 31) ^ (4 * (hi + 2)))};
    constexpr bool kHasGather = (MODE == WD || MODE == WGU);
    const bool gathered = (MODE == WD && half == 0) || (MODE == WGU && half == 1);
    // plain strided operand: K row 0 at this tile's columns, row stride ld
    const bf16_t* rbase = nullptr;
    int64_t ld = 0;
    if (MODE == DH) { rbase = g.Wd + ew + pn * BN; ld = g.m; }
    if (MODE == DX) { rbase = g.Wg + ew + pn * BN; ld = g.d; }
    if (MODE == WD) { rbase = g.Hg + (int64_t)row0 * g.m + ct * BN; ld = g.m; }
    if (MODE == WGU) { rbase = g.AU + (int64_t)row0 * (2 * g.m) + rt * BM; ld = 2 * g.m; }
    const int64_t loff[2] = {hi * ld + cpat[0], hi * ld + cpat[1]};
    // gathered operand (WD: dy rows, WGU: x rows): lane l holds the route
    // entry of K row 16 wq + l % 16 of the next slice, loaded one slice ahead
    // (rows past klen load the expert's last entry and copy zeros)
    const bf16_t* gbase = MODE == WD ? g.dy + rt * BM : g.x + ct * BN;
    int gent = 0;
    auto fetch_tok = [&](int kt) __attribute__((always_inline)) {
        gent = g.perm_src[row0 + min(kt * BK + 16 * wq + (lane & 15), klen - 1)];
    };
    // token row of a route entry t k + s: multiply-high by kmul = ceil(2^32 / k)
    // is exact for entries below 2^32 / k (checked on the host); k = 1 has kmul 0
    auto tok_of = [&](int e) __attribute__((always_inline)) {
        const uint32_t n = (uint32_t)min(max(e, 0), g.Tk - 1);
        return (int64_t)(__umulhi(n, g.kmul) + (g.kmul == 0u ? n : 0u));
    };
    auto issue_strided = [&](int stage, int kt) __attribute__((always_inline)) {
        unsigned char* dst = lds + stage * STAGEB + (half ? BM * ROWB : 0) + wq * (16 * 512);
        const int k0 = kt * BK + 16 * wq;
        const bool full = kt * BK + BK <= klen;
        if (kHasGather && gathered) {
#pragma unroll
            for (int i = 0; i < kGroups; ++i) {
                const int ka = k0 + 2 * i;
                const bf16_t* pa = ka < klen ? gbase + tok_of(__builtin_amdgcn_readlane(gent, 2 * i)) * g.d : kZeroRow;
                const bf16_t* pb =
                    ka + 1 < klen ? gbase + tok_of(__builtin_amdgcn_readlane(gent, 2 * i + 1)) * g.d : kZeroRow;
                dma16((hi ? pb : pa) + cpat[i & 1], dst + i * 1024);
            }
        } else {
            const bf16_t* rb = rbase;
            int kr = k0;
            if (MODE == DX && kt * BK >= g.m) { rb = g.Wu + ew + pn * BN; kr -= g.m; }
            const bf16_t* p = rb + (int64_t)kr * ld;
            if (kHasGather && !full) {
#pragma unroll
                for (int i = 0; i < kGroups; ++i)
                    dma16(k0 + 2 * i + hi < klen ? p + 2 * i * ld + loff[i & 1] : kZeroRow + cpat[i & 1],
                          dst + i * 1024);
            } else {
#pragma unroll
                for (int i = 0; i < kGroups; ++i) dma16(p + 2 * i * ld + loff[i & 1], dst + i * 1024);
            }
        }
    };
    auto issue = [&](int stage, int kt) __attribute__((always_inline)) {
        if (strided) {
            issue_strided(stage, kt);
            if (kHasGather && gathered && kt + 1 < (klen + BK - 1) / BK) fetch_tok(kt + 1);
        } else {
#pragma unroll
            for (int i = 0; i < kGroups; ++i) {
                const int grp = wq * kGroups + i;
                dma16(sbase + (soff[i] + (uint32_t)(kt * BK)), &lds[stage * STAGEB + grp * 1024]);
            }
        }
    };

    f32x16 acc[MI][NJ];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    // MFMA fragments: lane l supplies K values 8 (l / 32) .. +7 of the K=16
    // step for tile row (or column) l % 32 of a 32-block.
    // K-contiguous: one 16-byte read at the swizzled chunk.
    const int lrow = lane & 31;
    const int sw = swz(lrow);
    int kpos[BK / 16];
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) kpos[ks] = lrow * ROWB + (((2 * ks + (lane >> 5)) ^ sw) << 4);
    // K-strided: two ds_read_b64_tr_b16.  Within each group of 16 lanes, lane
    // s reads 4 values of K row 8 (g/2) + s/4 (+4 for the second read) at
    // columns 16 (g%2) + 4 (s%4) .. +3 of the block; the instruction hands
    // lane s value s%4 of the reads of lanes s/4 + 4j, j = 0..3, so each lane
    // ends up with four consecutive K values of column 16 (g%2) + s.
    const int s16 = lane & 15, g4 = lane >> 4;
    const int nl = 16 * (g4 & 1) + 4 * (s16 & 3);
    const int kl = 8 * (g4 >> 1) + (s16 >> 2);
    const int tsw = (nl >> 3) ^ (4 * (kl & 3));
    auto tr_pos = [&](int cb) { return kl * 512 + ((((cb >> 3) ^ tsw)) << 4) + ((nl & 4) << 1); };
    int a_pos[MI], b_pos[NJ];
#pragma unroll
    for (int i = 0; i < MI; ++i)
        a_pos[i] = kStridedA ? tr_pos(wr * WM + i * 32) : (wr * WM + i * 32) * ROWB;
#pragma unroll
    for (int j = 0; j < NJ; ++j) b_pos[j] = BM * ROWB + tr_pos(wc * WN + j * 32);

    const int nk = (klen + BK - 1) / BK;
    if (nk > 0) {
        if (kHasGather && gathered) fetch_tok(0);
        issue(0, 0);
    }
    for (int kt = 0; kt < nk; ++kt) {
        wait_vmcnt<0>();
        __syncthreads();
        if (kt + 1 < nk) issue((kt + 1) % NSTAGE, kt + 1);
        if (active) {
            const unsigned char* base = lds + (kt % NSTAGE) * STAGEB;
            bf16x8 fa[2][MI], fb[2][NJ];
            auto tr_frag = [&](int pos, int ks) __attribute__((always_inline)) {
                const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_v4s*)(base + pos + ks * (16 * 512)));
                const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_v4s*)(base + pos + ks * (16 * 512) + 4 * 512));
                return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
            };
            auto read_frags = [&](int buf, int ks) __attribute__((always_inline)) {
#pragma unroll
                for (int i = 0; i < MI; ++i)
                    fa[buf][i] = kStridedA ? tr_frag(a_pos[i], ks)
                                           : __builtin_bit_cast(bf16x8, *(const u32x4*)(base + a_pos[i] + kpos[ks]));
#pragma unroll
                for (int j = 0; j < NJ; ++j) fb[buf][j] = tr_frag(b_pos[j], ks);
            };
            read_frags(0, 0);
#pragma unroll
            for (int ks = 0; ks < BK / 16; ++ks) {
                if (ks + 1 < BK / 16) read_frags((ks + 1) & 1, ks + 1);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int i = 0; i < MI; ++i)
#pragma unroll
                    for (int j = 0; j < NJ; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            fb[ks & 1][j], fa[ks & 1][i], acc[i][j], 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
    // ---- epilogues.  Lane l holds output row l%32 of each 32-row block and
    // columns 8*(v/4) + 4*(l/32) + v%4 of each 32-column block.
    const int ncol0 = 4 * (lane >> 5);
    if (MODE != DH) {
        // DX (bf16 rows) and WD / WGU (fp32 rows) are staged through this
        // wavefront's share of the freed LDS stages (16-byte chunks XOR-swizzled
        // by row; for bf16 the 8-byte halves of a chunk are also swapped in rows
        // with bit 3 set, so the 16 rows of one 8-byte write cycle hit distinct
        // banks) and stored 16 bytes per lane along whole row segments,
        // instead of 8- or 16-byte pieces of 32 rows per store
        __syncthreads();
        if (!active) return;
        if (MODE == DX) {
            constexpr int RB = WN * 2, NCH = RB / 16;        // 256-byte staged rows
            unsigned char* sw = lds + wave * (WM * RB);
#pragma unroll
            for (int i = 0; i < MI; ++i) {
                const int row = i * 32 + (lane & 31);
#pragma unroll
                for (int j = 0; j < NJ; ++j)
#pragma unroll
                    for (int a4 = 0; a4 < 4; ++a4) {
                        const int col = j * 32 + 8 * a4 + ncol0;
                        const int v0 = 4 * a4;
                        *(uint2*)(sw + row * RB + ((((col >> 3) ^ (row & (NCH - 1)))) << 4) +
                                  (((col & 4) << 1) ^ (row & 8))) =
                            make_uint2(pack_bf(acc[i][j][v0], acc[i][j][v0 + 1]),
                                       pack_bf(acc[i][j][v0 + 2], acc[i][j][v0 + 3]));
                    }
            }
            __builtin_amdgcn_s_waitcnt(0xc07f);
            __builtin_amdgcn_wave_barrier();
            const int ch = lane % NCH;
#pragma unroll
            for (int p = 0; p < WM / (64 / NCH); ++p) {
                const int row = p * (64 / NCH) + lane / NCH;
                const int r = wr * WM + row;
                u32x4 v = *(const u32x4*)(sw + row * RB + ((ch ^ (row & (NCH - 1))) << 4));
                if (row & 8) v = u32x4{v[2], v[3], v[0], v[1]};
                if (r < rows)
                    *(u32x4*)(g.dxr + ((int64_t)row0 + r) * g.d + pn * BN + wc * WN + ch * 8) = v;
            }
        } else {
            // fp32: 512-byte staged rows, one 32-row block at a time
            constexpr int RB = WN * 4, NCH = RB / 16;
            unsigned char* sw = lds + wave * (32 * RB);
            const int64_t ew = (int64_t)expert * g.m * g.d;
#pragma unroll
            for (int i = 0; i < MI; ++i) {
                const int row = lane & 31;
#pragma unroll
                for (int j = 0; j < NJ; ++j)
#pragma unroll
                    for (int a4 = 0; a4 < 4; ++a4) {
                        const int col = j * 32 + 8 * a4 + ncol0;
                        const int v0 = 4 * a4;
                        *(f32x4*)(sw + row * RB + (((col >> 2) ^ (row & (NCH - 1))) << 4)) =
                            f32x4{acc[i][j][v0], acc[i][j][v0 + 1], acc[i][j][v0 + 2], acc[i][j][v0 + 3]};
                    }
                __builtin_amdgcn_s_waitcnt(0xc07f);
                __builtin_amdgcn_wave_barrier();
                const int ch = lane % NCH;
#pragma unroll
                for (int p = 0; p < 32 / (64 / NCH); ++p) {
                    const int row2 = p * (64 / NCH) + lane / NCH;
                    const int R = rt * BM + wr * WM + i * 32 + row2;
                    float* orow;
                    if (MODE == WD) orow = g.dWd + ew + (int64_t)R * g.m;
                    else orow = (R < g.m ? g.dWg + ew + (int64_t)R * g.d
                                         : g.dWu + ew + (int64_t)(R - g.m) * g.d);
                    *(u32x4*)(orow + ct * BN + wc * WN + ch * 4) =
                        *(const u32x4*)(sw + row2 * RB + ((ch ^ (row2 & (NCH - 1))) << 4));
                }
                // the next block overwrites the region
                __builtin_amdgcn_s_waitcnt(0xc07f);
                __builtin_amdgcn_wave_barrier();
            }
        }
        return;
    }
    // DH, one 32-row block at a time: G (fp32) goes through this wavefront's
    // LDS region (512-byte rows, 16-byte chunks XOR-swizzled by row), then each
    // lane takes 8 consecutive columns of a row, so the loads of a, u and the
    // stores of da, du and g H are 16 bytes per lane along 256-byte row
    // segments (reading and writing each lane's own 8-byte pieces of 32 rows
    // took half the kernel's time).  All of a block's a, u loads go out before
    // its G is staged.
    // route weight of the wavefront row this lane's index names, for __shfl
    const int rl = wr * WM + lane;
    const int ql = row0 + (rl < rows ? rl : 0);
    const float gql = g.gate[min(max(g.perm_src[ql], 0), g.Tk - 1)];
    __syncthreads();
    if (!active) return;
    constexpr int RB = WN * 4;                  // bytes per staged row: 32 chunks of 16
    unsigned char* stg = lds + wave * (32 * RB);
    const int np = g.m / 128;
    const int64_t ldau = 2 * (int64_t)g.m;
    const int cl = lane & 15, rsub = lane >> 4;
    const int col = pn * BN + wc * WN + 8 * cl;            // this lane's first column
    // lanes 4-7 of each group of 8 read their second chunk first, so the 8
    // lanes of one read cycle hit 8 distinct bank groups
    const int h0 = (cl >> 2) & 1;
#pragma unroll
    for (int i = 0; i < MI; ++i) {
        u32x4 av[8], uv[8];
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            const int r = wr * WM + i * 32 + p * 4 + rsub;
            const int64_t q = row0 + (r < rows ? r : 0);
            av[p] = *(const u32x4*)(g.AUin + q * ldau + col);
            uv[p] = *(const u32x4*)(g.AUin + q * ldau + g.m + col);
        }
        {
            const int row = lane & 31;
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int a4 = 0; a4 < 4; ++a4) {
                    const int c = j * 32 + 8 * a4 + ncol0;
                    *(f32x4*)(stg + row * RB + (((c >> 2) ^ row) << 4)) =
                        f32x4{acc[i][j][4 * a4], acc[i][j][4 * a4 + 1], acc[i][j][4 * a4 + 2], acc[i][j][4 * a4 + 3]};
                }
        }
        __builtin_amdgcn_s_waitcnt(0xc07f);
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            const int row = p * 4 + rsub;
            const int r = wr * WM + i * 32 + row;
            const bool ok = r < rows;
            const int64_t q = row0 + (ok ? r : 0);
            const f32x4 x0 = *(const f32x4*)(stg + row * RB + (((2 * cl + h0) ^ row) << 4));
            const f32x4 x1 = *(const f32x4*)(stg + row * RB + (((2 * cl + 1 - h0) ^ row) << 4));
            const f32x4 G0 = h0 ? x1 : x0, G1 = h0 ? x0 : x1;
            const float gq = __shfl(gql, i * 32 + row);
            const float Gv[8] = {G0[0], G0[1], G0[2], G0[3], G1[0], G1[1], G1[2], G1[3]};
            uint32_t dw[4], uw[4], hw[4];
            float part = 0.0f;
#pragma unroll
            for (int e2 = 0; e2 < 4; ++e2) {
                float da[2], du[2], hgv[2];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const float a = h ? bf_hi(av[p][e2]) : bf_lo(av[p][e2]);
                    const float u = h ? bf_hi(uv[p][e2]) : bf_lo(uv[p][e2]);
                    float hG;
                    swiglu_bwd(a, u, Gv[2 * e2 + h], gq, true, da[h], du[h], hgv[h], hG);
                    part += hG;
                }
                dw[e2] = pack_bf(da[0], da[1]);
                uw[e2] = pack_bf(du[0], du[1]);
                hw[e2] = pack_bf(hgv[0], hgv[1]);
            }
            // row sum over the 16 lanes of this row (lane cl = 0 keeps it)
            part += row_ror_f<8>(part);
            part += row_ror_f<4>(part);
            part += row_ror_f<2>(part);
            part += row_ror_f<1>(part);
            if (ok) {
                bf16_t* au = g.AU + q * ldau;
                *(u32x4*)(au + col) = u32x4{dw[0], dw[1], dw[2], dw[3]};
                *(u32x4*)(au + g.m + col) = u32x4{uw[0], uw[1], uw[2], uw[3]};
                *(u32x4*)(g.Hg + q * g.m + col) = u32x4{hw[0], hw[1], hw[2], hw[3]};
                if (cl == 0) g.dgp[q * np + pn * 2 + wc] = part;
            }
        }
        if (i + 1 < MI) {            // the next block overwrites the region
            __builtin_amdgcn_s_waitcnt(0xc07f);
            __builtin_amdgcn_wave_barrier();
        }
    }
}

// Experts by decreasing route count, ties to the lower id (one workgroup).
__global__ void __launch_bounds__(1024) expert_order_kernel(const int* offsets, int N, int* order) {
    __shared__ int cnt[kMaxExperts];
    for (int e = threadIdx.x; e < N; e += blockDim.x) cnt[e] = offsets[e + 1] - offsets[e];
    __syncthreads();
    for (int e = threadIdx.x; e < N; e += blockDim.x) {
        const int c = cnt[e];
        int rank = 0;
        for (int f = 0; f < N; ++f) rank += (cnt[f] > c) || (cnt[f] == c && f < e);
        order[rank] = e;
    }
}

// ------------------------------------------------------------ generic ----
// One thread per output element; any shape, bf16 or fp32.

template <typename T>
__global__ void __launch_bounds__(256)
dh_generic(const T* dy, const int* perm_src, int k, const T* Wd, const float* gate, int d, int m,
           const int* tiles, const int* tile_count, const T* AUin, T* AU, T* Hg, float* dgp) {
    const int tile = blockIdx.x;
    if (tile >= *tile_count) return;
    const int expert = tiles[3 * tile], row0 = tiles[3 * tile + 1], rows = tiles[3 * tile + 2];
    const int r = threadIdx.x;
    const int j = blockIdx.y;
    if (r >= rows || j >= m) return;
    const int64_t q = row0 + r;
    const int src = perm_src[q];
    const T* dyr = dy + (int64_t)(src / k) * d;
    const T* w = Wd + (int64_t)expert * d * m + j;
    float G = 0.0f;
    for (int i = 0; i < d; ++i) G = fmaf(Act<T>::to_f32(dyr[i]), Act<T>::to_f32(w[(int64_t)i * m]), G);
    const T* ain = AUin + q * 2 * m;
    T* au = AU + q * 2 * m;
    float da, du, hg, hG;
    swiglu_bwd(Act<T>::to_f32(ain[j]), Act<T>::to_f32(ain[m + j]), G, gate[src],
               sizeof(T) == 2, da, du, hg, hG);
    au[j] = Act<T>::from_f32(da);
    au[m + j] = Act<T>::from_f32(du);
    Hg[q * m + j] = Act<T>::from_f32(hg);
    dgp[q * m + j] = hG;
}

template <typename T>
__global__ void __launch_bounds__(256)
dx_generic(const T* AU, const T* Wg, const T* Wu, int d, int m, const int* tiles,
           const int* tile_count, T* dxr) {
    const int tile = blockIdx.x;
    if (tile >= *tile_count) return;
    const int expert = tiles[3 * tile], row0 = tiles[3 * tile + 1], rows = tiles[3 * tile + 2];
    const int r = threadIdx.x;
    const int i = blockIdx.y;
    if (r >= rows || i >= d) return;
    const int64_t q = row0 + r;
    const T* au = AU + q * 2 * m;
    const T* wg = Wg + (int64_t)expert * m * d + i;
    const T* wu = Wu + (int64_t)expert * m * d + i;
    float acc = 0.0f;
    for (int j = 0; j < m; ++j) {
        acc = fmaf(Act<T>::to_f32(au[j]), Act<T>::to_f32(wg[(int64_t)j * d]), acc);
        acc = fmaf(Act<T>::to_f32(au[m + j]), Act<T>::to_f32(wu[(int64_t)j * d]), acc);
    }
    dxr[q * d + i] = Act<T>::from_f32(acc);
}

// dW_down[e][i][j] = sum over expert e's routes of dy[t][i] * (g H)[q][j]
template <typename T>
__global__ void __launch_bounds__(256)
wd_generic(const T* dy, const T* Hg, const int* perm_src, const int* offsets, int k, int d, int m,
           float* dWd) {
    const int e = blockIdx.x;
    const int i = blockIdx.y;
    const int q0 = offsets[e], q1 = offsets[e + 1];
    for (int j = threadIdx.x; j < m; j += blockDim.x) {
        float acc = 0.0f;
        for (int q = q0; q < q1; ++q)
            acc = fmaf(Act<T>::to_f32(dy[(int64_t)(perm_src[q] / k) * d + i]),
                       Act<T>::to_f32(Hg[(int64_t)q * m + j]), acc);
        dWd[((int64_t)e * d + i) * m + j] = acc;
    }
}

// dW_gate[e][r][i] (r < m) / dW_up[e][r - m][i] = sum over routes of (da | du)[q][r] * x[t][i]
template <typename T>
__global__ void __launch_bounds__(256)
wgu_generic(const T* x, const T* AU, const int* perm_src, const int* offsets, int k, int d, int m,
            float* dWg, float* dWu) {
    const int e = blockIdx.x;
    const int r = blockIdx.y;
    const int q0 = offsets[e], q1 = offsets[e + 1];
    float* out = r < m ? dWg + ((int64_t)e * m + r) * d : dWu + ((int64_t)e * m + r - m) * d;
    for (int i = threadIdx.x; i < d; i += blockDim.x) {
        float acc = 0.0f;
        for (int q = q0; q < q1; ++q)
            acc = fmaf(Act<T>::to_f32(AU[(int64_t)q * 2 * m + r]),
                       Act<T>::to_f32(x[(int64_t)(perm_src[q] / k) * d + i]), acc);
        out[i] = acc;
    }
}

// ------------------------------------------------------------ router ----

// W_r [d, N] -> [N, d]
__global__ void __launch_bounds__(256)
transpose_wr_kernel(const float* W_r, int d, int N, float* wrt) {
    __shared__ float tile[32][33];
    const int i0 = blockIdx.x * 32, e0 = blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    for (int y = ty; y < 32; y += 8)
        if (i0 + y < d && e0 + tx < N) tile[y][tx] = W_r[(int64_t)(i0 + y) * N + e0 + tx];
    __syncthreads();
    for (int y = ty; y < 32; y += 8)
        if (e0 + y < N && i0 + tx < d) wrt[(int64_t)(e0 + y) * d + i0 + tx] = tile[tx][y];
}

// Per token: dg_s = sum of its partials, then the renormalised-softmax backward
// dp_s = g_s (dg_s - sum_s' g_s' dg_s'), in route and in permuted order.
// One lane per route: the k routes of a token sit in an aligned group of
// 2^kp_log2 >= k lanes of one wavefront (k <= 64), and every lane forms the
// token's inner product from its group by shuffles, in slot order, so the sums
// are those of a serial loop over the slots.
__global__ void __launch_bounds__(256)
gate_grad_lanes_kernel(const float* dgp, int np, const int* inv, const float* gate, int64_t T,
                       int k, int kp_log2, float* dp_route, float* dp_perm) {
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t t = gid >> kp_log2;
    const int s = (int)(gid & ((1 << kp_log2) - 1));
    const bool valid = t < T && s < k;
    float dg = 0.0f, gs = 0.0f;
    int q = -1;
    if (valid) {
        q = inv[t * k + s];
        gs = gate[t * k + s];
        if (q >= 0)
            for (int p = 0; p < np; ++p) dg += dgp[(int64_t)q * np + p];
    }
    const int base = (threadIdx.x & 63) & ~((1 << kp_log2) - 1);
    float inner = 0.0f;
    for (int j = 0; j < k; ++j)
        inner = fmaf(__shfl(gs, base + j, 64), __shfl(dg, base + j, 64), inner);
    if (valid) {
        const float dp = gs * (dg - inner);
        dp_route[t * k + s] = dp;
        if (q >= 0) dp_perm[q] = dp;
    }
}

__global__ void __launch_bounds__(256)
gate_grad_kernel(const float* dgp, int np, const int* inv, const float* gate, int64_t T, int k,
                 float* dp_route, float* dp_perm) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= T) return;
    float inner = 0.0f;
    for (int s = 0; s < k; ++s) {
        const int q = inv[t * k + s];
        float dg = 0.0f;
        if (q >= 0)
            for (int p = 0; p < np; ++p) dg += dgp[(int64_t)q * np + p];
        dp_route[t * k + s] = dg;
        inner = fmaf(gate[t * k + s], dg, inner);
    }
    for (int s = 0; s < k; ++s) {
        const float gs = gate[t * k + s];
        const float dp = gs * (dp_route[t * k + s] - inner);
        dp_route[t * k + s] = dp;
        const int q = inv[t * k + s];
        if (q >= 0) dp_perm[q] = dp;
    }
}

// dW_r[:, e] = sum over expert e's routes of dp * x_t, db_r[e] = sum of dp, in
// two passes so that a heavily loaded expert is spread over many workgroups:
//   partials: workgroup (256-row tile, column chunk of 256) sums the tile's
//             routes (8 row groups of 32 threads, 8 columns per thread, each
//             thread over its rows in order, then the groups in a fixed order);
//   reduce:   each expert's tile partials are added in tile order.
template <typename T>
__global__ void __launch_bounds__(256)
router_wgrad_partial_kernel(const T* x, const int* perm_src, const int* tiles, const int* tile_count,
                            const float* dp_perm, int k, int d, float* part, float* dbpart) {
    __shared__ float red[8][256];
    __shared__ float dbs[8];
    const int tile = blockIdx.x;
    if (tile >= *tile_count) return;
    const int q0 = tiles[3 * tile + 1], q1 = q0 + tiles[3 * tile + 2];
    const int cg = threadIdx.x & 31, rg = threadIdx.x >> 5;
    const int i0 = blockIdx.y * 256 + 8 * cg;
    float acc[8];
#pragma unroll
    for (int v = 0; v < 8; ++v) acc[v] = 0.0f;
    float dbacc = 0.0f;
    // each thread sums routes q0 + rg, q0 + rg + 8, ... in that order; the loads
    // of kRwU consecutive ones are issued together
    constexpr int kRwU = 8;
    for (int qb = q0 + rg; qb < q1; qb += 8 * kRwU) {
        int tok[kRwU];
        float w[kRwU];
#pragma unroll
        for (int u = 0; u < kRwU; ++u) {
            const int q = qb + 8 * u;
            tok[u] = q < q1 ? perm_src[q] / k : -1;
            w[u] = q < q1 ? dp_perm[q] : 0.0f;
        }
        if (sizeof(T) == 2 && i0 + 8 <= d) {
            u32x4 v[kRwU];
#pragma unroll
            for (int u = 0; u < kRwU; ++u)
                v[u] = tok[u] >= 0 ? *(const u32x4*)(x + (int64_t)tok[u] * d + i0) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
            for (int u = 0; u < kRwU; ++u) {
                if (tok[u] < 0) continue;
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    acc[2 * h] = fmaf(w[u], bf_lo(v[u][h]), acc[2 * h]);
                    acc[2 * h + 1] = fmaf(w[u], bf_hi(v[u][h]), acc[2 * h + 1]);
                }
            }
        } else {
#pragma unroll
            for (int u = 0; u < kRwU; ++u) {
                if (tok[u] < 0) continue;
                const T* xr = x + (int64_t)tok[u] * d;
#pragma unroll
                for (int v = 0; v < 8; ++v)
                    if (i0 + v < d) acc[v] = fmaf(w[u], Act<T>::to_f32(xr[i0 + v]), acc[v]);
            }
        }
#pragma unroll
        for (int u = 0; u < kRwU; ++u) dbacc += w[u];
    }
#pragma unroll
    for (int v = 0; v < 8; ++v) red[rg][8 * cg + v] = acc[v];
    if (cg == 0) dbs[rg] = dbacc;
    __syncthreads();
    const int c = threadIdx.x;
    float sum = 0.0f;
#pragma unroll
    for (int g = 0; g < 8; ++g) sum += red[g][c];
    const int i = blockIdx.y * 256 + c;
    if (i < d) part[(int64_t)tile * d + i] = sum;
    if (blockIdx.y == 0 && threadIdx.x == 0) {
        float db = 0.0f;
        for (int g = 0; g < 8; ++g) db += dbs[g];
        dbpart[tile] = db;
    }
}

// dW_r[i][e] = sum of expert e's tile partials in tile order (tiles are expert-major)
__global__ void __launch_bounds__(256)
router_wgrad_reduce_kernel(const int* offsets, const float* part, const float* dbpart, int bm,
                           int d, int N, float* dW_r, float* db_r) {
    const int e = blockIdx.x;
    // first tile of expert e: the tile counts of experts 0 .. e-1, summed by all
    // threads (integer sums, so the order does not matter)
    __shared__ int s_t0;
    if (threadIdx.x == 0) s_t0 = 0;
    __syncthreads();
    int c = 0;
    for (int f = threadIdx.x; f < e; f += blockDim.x) c += (offsets[f + 1] - offsets[f] + bm - 1) / bm;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off, 64);
    if ((threadIdx.x & 63) == 0) atomicAdd(&s_t0, c);
    __syncthreads();
    const int t0 = s_t0;
    const int nt = (offsets[e + 1] - offsets[e] + bm - 1) / bm;
    const int i = blockIdx.y * 256 + threadIdx.x;
    if (i < d) {
        // the expert's tile sums in tile order, eight loads in flight
        float s = 0.0f;
        int t = 0;
        for (; t + 8 <= nt; t += 8) {
            float v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = part[(int64_t)(t0 + t + j) * d + i];
#pragma unroll
            for (int j = 0; j < 8; ++j) s += v[j];
        }
        for (; t < nt; ++t) s += part[(int64_t)(t0 + t) * d + i];
        dW_r[(int64_t)i * N + e] = s;
    }
    if (db_r && blockIdx.y == 0 && threadIdx.x == 0) {
        float s = 0.0f;
        for (int t = 0; t < nt; ++t) s += dbpart[t0 + t];
        db_r[e] = s;
    }
}

// dx_t = sum_s dxr[route (t, s)] + sum_s dp_ts W_r[:, idx_ts], summed in slot order in fp32
template <typename T>
__global__ void __launch_bounds__(256)
dx_combine_kernel(const T* dxr, const int* inv, const float* dp_route, const float* wrt,
                  const void* idx, int idx_dtype, int64_t ldi, int64_t T_, int k, int d, int N,
                  T* dx) {
    const int64_t t = blockIdx.x;
    if (t >= T_) return;
    for (int i = threadIdx.x; i < d; i += blockDim.x) {
        float acc = 0.0f;
        for (int s = 0; s < k; ++s) {
            const int q = inv[t * k + s];
            if (q >= 0) acc += Act<T>::to_f32(dxr[(int64_t)q * d + i]);
        }
        for (int s = 0; s < k; ++s) {
            const int e = load_id(idx, idx_dtype, t * ldi + s);
            if (e >= 0 && e < N) acc = fmaf(dp_route[t * k + s], wrt[(int64_t)e * d + i], acc);
        }
        dx[t * d + i] = Act<T>::from_f32(acc);
    }
}

// bf16, d % 8 == 0: each thread owns 8 consecutive columns of kDxTok tokens;
// per token the k per-route rows are added in slot order, then the router
// terms dp_ts W_r[:, idx_ts] in slot order (fp32)
constexpr int kDxTok = 2;
__global__ void __launch_bounds__(256)
dx_combine_bf16_kernel(const bf16_t* dxr, const int* inv, const float* dp_route, const float* wrt,
                       const void* idx, int idx_dtype, int64_t ldi, int64_t T_, int k, int d, int N,
                       bf16_t* dx) {
    constexpr int kSlots = 8;
    const int64_t step = (int64_t)gridDim.x * kDxTok;
    for (int64_t t0 = (int64_t)blockIdx.x * kDxTok; t0 < T_; t0 += step) {
        for (int c0 = threadIdx.x * 8; c0 < d; c0 += 256 * 8) {
            float acc[kDxTok][8];
#pragma unroll
            for (int u = 0; u < kDxTok; ++u)
#pragma unroll
                for (int v = 0; v < 8; ++v) acc[u][v] = 0.0f;
            for (int s0 = 0; s0 < k; s0 += kSlots) {
                int r[kDxTok][kSlots];
                u32x4 raw[kDxTok][kSlots];
#pragma unroll
                for (int u = 0; u < kDxTok; ++u)
#pragma unroll
                    for (int j = 0; j < kSlots; ++j) {
                        const int64_t t = t0 + u;
                        r[u][j] = (t < T_ && s0 + j < k) ? inv[t * k + s0 + j] : -1;
                    }
#pragma unroll
                for (int u = 0; u < kDxTok; ++u)
#pragma unroll
                    for (int j = 0; j < kSlots; ++j)
                        raw[u][j] = r[u][j] >= 0 ? *(const u32x4*)(dxr + (int64_t)r[u][j] * d + c0)
                                                 : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
                for (int j = 0; j < kSlots; ++j)
#pragma unroll
                    for (int u = 0; u < kDxTok; ++u)
#pragma unroll
                        for (int w = 0; w < 4; ++w) {
                            acc[u][2 * w] += bf_lo(raw[u][j][w]);
                            acc[u][2 * w + 1] += bf_hi(raw[u][j][w]);
                        }
            }
#pragma unroll
            for (int u = 0; u < kDxTok; ++u) {
                const int64_t t = t0 + u;
                if (t >= T_) continue;
                // the router rows of kSlots slots are fetched together, then added in slot order
                for (int s0 = 0; s0 < k; s0 += kSlots) {
                    int es[kSlots];
                    float gs[kSlots];
#pragma unroll
                    for (int j = 0; j < kSlots; ++j) {
                        const int e = s0 + j < k ? load_id(idx, idx_dtype, t * ldi + s0 + j) : -1;
                        es[j] = (e >= 0 && e < N) ? e : -1;
                        gs[j] = es[j] >= 0 ? dp_route[t * k + s0 + j] : 0.0f;
                    }
                    f32x4 w0[kSlots], w1[kSlots];
#pragma unroll
                    for (int j = 0; j < kSlots; ++j) {
                        const float* wr = wrt + (int64_t)(es[j] >= 0 ? es[j] : 0) * d + c0;
                        w0[j] = *(const f32x4*)wr;
                        w1[j] = *(const f32x4*)(wr + 4);
                    }
#pragma unroll
                    for (int j = 0; j < kSlots; ++j) {
                        if (es[j] < 0) continue;
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            acc[u][v] = fmaf(gs[j], w0[j][v], acc[u][v]);
                            acc[u][4 + v] = fmaf(gs[j], w1[j][v], acc[u][4 + v]);
                        }
                    }
                }
                *(uint4*)(dx + t * (int64_t)d + c0) =
                    make_uint4(pack_bf(acc[u][0], acc[u][1]), pack_bf(acc[u][2], acc[u][3]),
                               pack_bf(acc[u][4], acc[u][5]), pack_bf(acc[u][6], acc[u][7]));
            }
        }
    }
}

// ---------------------------------------------- paper-literal weights ----
// With the weight of id j equal to rho_j, the softmax of all N current logits
// (Eq. pr2_output as printed), every logit of a token receives a gradient:
//   dp_ti = rho_ti ([i in route] dg_ti - sum_{j in route} rho_tj dg_tj),
// that is g_s (dg_s - inner) at the route's ids and -rho_i inner elsewhere,
// with inner = sum_s g_s dg_s.  The router gradients become dense over N:
//   dW_r = x^T dp,  db_r = sum_t dp_t,  and dx_t gains dp_t W_r^T.

// One wavefront per token (k <= 64): dg_s = the sum of its partials, inner in
// slot order (as the renormalised kernel forms it), rho from the fp32 logits
// p (max-shifted, fp32, as the forward's weights), the row dpf[t, :] written
// once.  Out-of-range ids (inv = -1) contribute nothing.
__global__ void __launch_bounds__(256)
literal_dp_kernel(const float* dgp, int np, const int* inv, const float* gate, const float* p,
                  const void* idx, int idx_dtype, int64_t ldi, int64_t T, int k, int N,
                  float* dpf) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= T) return;                        // uniform across the wavefront
    float dg = 0.0f, gs = 0.0f;
    int id = -1;
    if (lane < k) {
        const int q = inv[t * k + lane];
        gs = gate[t * k + lane];
        if (q >= 0) {
            for (int pp = 0; pp < np; ++pp) dg += dgp[(int64_t)q * np + pp];
            id = load_id(idx, idx_dtype, t * ldi + lane);
        }
    }
    float inner = 0.0f;
    for (int j = 0; j < k; ++j) inner = fmaf(__shfl(gs, j, 64), __shfl(dg, j, 64), inner);
    const float on_route = gs * (dg - inner);
    const float* pr = p + t * N;
    float mx = -INFINITY;
    for (int i = lane; i < N; i += 64) mx = fmaxf(mx, pr[i]);
    for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    float sum = 0.0f;
    for (int i = lane; i < N; i += 64) sum += expf(pr[i] - mx);
    for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, 64);
    for (int i0 = 0; i0 < N; i0 += 64) {
        const int i = i0 + lane;
        float v = i < N ? -(expf(pr[i] - mx) / sum) * inner : 0.0f;
        for (int j = 0; j < k; ++j) {
            const int idj = __shfl(id, j, 64);
            const float vj = __shfl(on_route, j, 64);
            if (idj == i) v = vj;
        }
        if (i < N) dpf[t * N + i] = v;
    }
}

constexpr int kLitTok = 1024;      // tokens per dW_r partial
constexpr int kLitTile = 64;       // dW_r partial tile: 64 rows of d x 64 logits

// part[c][i][j] = sum over the tokens of chunk c (in order) of x[t][i] dpf[t][j];
// dbpart[c][j] the same of dpf[t][j] (workgroups of the first row block).
template <typename T>
__global__ void __launch_bounds__(256)
literal_wgrad_partial_kernel(const T* x, const float* dpf, int64_t Ttot, int d, int N,
                             float* part, float* dbpart) {
    __shared__ __attribute__((aligned(16))) float xs[32][kLitTile];
    __shared__ __attribute__((aligned(16))) float ps[32][kLitTile];
    const int i0 = blockIdx.x * kLitTile, j0 = blockIdx.y * kLitTile;
    const int64_t c = blockIdx.z;
    const int64_t t0 = c * kLitTok;
    const int64_t t1 = t0 + kLitTok < Ttot ? t0 + kLitTok : Ttot;
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    float acc[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = 0.0f;
    float db = 0.0f;
    for (int64_t tb = t0; tb < t1; tb += 32) {
        for (int e = threadIdx.x; e < 32 * kLitTile; e += 256) {
            const int r = e / kLitTile, q = e % kLitTile;
            const int64_t t = tb + r;
            xs[r][q] = (t < t1 && i0 + q < d) ? Act<T>::to_f32(x[t * d + i0 + q]) : 0.0f;
            ps[r][q] = (t < t1 && j0 + q < N) ? dpf[t * N + j0 + q] : 0.0f;
        }
        __syncthreads();
#pragma unroll 4
        for (int r = 0; r < 32; ++r) {
            // 16-byte reads: four rows of x (a 16-lane broadcast) and four logits
            const f32x4 a = *(const f32x4*)&xs[r][ty * 4];
            const f32x4 b = *(const f32x4*)&ps[r][tx * 4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int v = 0; v < 4; ++v) acc[u][v] = fmaf(a[u], b[v], acc[u][v]);
        }
        if (blockIdx.x == 0 && threadIdx.x < kLitTile)
            for (int r = 0; r < 32; ++r) db += ps[r][threadIdx.x];
        __syncthreads();
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int i = i0 + ty * 4 + u;
        if (i >= d) continue;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int j = j0 + tx * 4 + v;
            if (j < N) part[(c * d + i) * N + j] = acc[u][v];
        }
    }
    if (blockIdx.x == 0 && threadIdx.x < kLitTile && j0 + (int)threadIdx.x < N)
        dbpart[c * N + j0 + threadIdx.x] = db;
}

// dW_r[q] and db_r[j]: the chunk partials added in chunk order
__global__ void __launch_bounds__(256)
literal_wgrad_reduce_kernel(const float* part, const float* dbpart, int nchunk, int64_t n, int N,
                            float* dW_r, float* db_r) {
    for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < n;
         q += (int64_t)gridDim.x * 256) {
        float s = 0.0f;
        for (int c = 0; c < nchunk; ++c) s += part[(int64_t)c * n + q];
        dW_r[q] = s;
        if (db_r && q < N) {
            float b = 0.0f;
            for (int c = 0; c < nchunk; ++c) b += dbpart[(int64_t)c * N + q];
            db_r[q] = b;
        }
    }
}

// dx_t = sum_s dxr[route (t, s)] (slot order) + sum_i dpf[t, i] W_r[:, i]
// (in logit order), fp32: one column per thread, 16 tokens per workgroup.
constexpr int kLitDxTok = 16;
template <typename T>
__global__ void __launch_bounds__(256)
literal_dx_combine_kernel(const T* dxr, const int* inv, const float* dpf, const float* wrt,
                          int64_t Ttot, int k, int d, int N, T* dx) {
    __shared__ __attribute__((aligned(16))) float ps[kLitDxTok][64];
    const int c = blockIdx.x * 256 + threadIdx.x;
    const int64_t t0 = (int64_t)blockIdx.y * kLitDxTok;
    float racc[kLitDxTok];
#pragma unroll
    for (int r = 0; r < kLitDxTok; ++r) racc[r] = 0.0f;
    for (int j0 = 0; j0 < N; j0 += 64) {
        for (int e = threadIdx.x; e < kLitDxTok * 64; e += 256) {
            const int r = e / 64, q = e % 64;
            const int64_t t = t0 + r;
            ps[r][q] = (t < Ttot && j0 + q < N) ? dpf[t * N + j0 + q] : 0.0f;
        }
        __syncthreads();
        if (c < d) {
            // W_r transposed ([N, d]): a wavefront reads 64 consecutive columns
            const float* wcol = wrt + (int64_t)j0 * d + c;
            const int jn = N - j0 < 64 ? N - j0 : 64;
            // four logits per step: one 16-byte (broadcast) LDS read per token
            // for four FMAs, added in the same order as one at a time
            int q = 0;
            for (; q + 4 <= jn; q += 4) {
                const float w0 = wcol[(int64_t)q * d], w1 = wcol[(int64_t)(q + 1) * d],
                            w2 = wcol[(int64_t)(q + 2) * d], w3 = wcol[(int64_t)(q + 3) * d];
#pragma unroll
                for (int r = 0; r < kLitDxTok; ++r) {
                    const f32x4 p = *(const f32x4*)&ps[r][q];
                    racc[r] = fmaf(p[0], w0, racc[r]);
                    racc[r] = fmaf(p[1], w1, racc[r]);
                    racc[r] = fmaf(p[2], w2, racc[r]);
                    racc[r] = fmaf(p[3], w3, racc[r]);
                }
            }
            for (; q < jn; ++q) {
                const float w = wcol[(int64_t)q * d];
#pragma unroll
                for (int r = 0; r < kLitDxTok; ++r) racc[r] = fmaf(ps[r][q], w, racc[r]);
            }
        }
        __syncthreads();
    }
    if (c >= d) return;
#pragma unroll
    for (int r = 0; r < kLitDxTok; ++r) {
        const int64_t t = t0 + r;
        if (t >= Ttot) break;
        float acc = 0.0f;
        for (int s = 0; s < k; ++s) {
            const int q = inv[t * k + s];
            if (q >= 0) acc += Act<T>::to_f32(dxr[(int64_t)q * d + c]);
        }
        dx[t * d + c] = Act<T>::from_f32(acc + racc[r]);
    }
}

// The same with four consecutive columns per thread (d % 4 == 0): each
// broadcast LDS read of four logits feeds 64 FMAs; every output's sums run in
// the same order as above, so the result is bitwise the same.
template <typename T>
__global__ void __launch_bounds__(256)
literal_dx_combine4_kernel(const T* dxr, const int* inv, const float* dpf, const float* wrt,
                           int64_t Ttot, int k, int d, int N, T* dx) {
    __shared__ __attribute__((aligned(16))) float ps[kLitDxTok][64];
    const int c = (blockIdx.x * 256 + threadIdx.x) * 4;
    const int64_t t0 = (int64_t)blockIdx.y * kLitDxTok;
    float racc[kLitDxTok][4];
#pragma unroll
    for (int r = 0; r < kLitDxTok; ++r)
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) racc[r][cc] = 0.0f;
    for (int j0 = 0; j0 < N; j0 += 64) {
        for (int e = threadIdx.x; e < kLitDxTok * 64; e += 256) {
            const int r = e / 64, q = e % 64;
            const int64_t t = t0 + r;
            ps[r][q] = (t < Ttot && j0 + q < N) ? dpf[t * N + j0 + q] : 0.0f;
        }
        __syncthreads();
        if (c < d) {
            const float* wcol = wrt + (int64_t)j0 * d + c;
            const int jn = N - j0 < 64 ? N - j0 : 64;
            int q = 0;
            for (; q + 4 <= jn; q += 4) {
                f32x4 w[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) w[u] = *(const f32x4*)(wcol + (int64_t)(q + u) * d);
#pragma unroll
                for (int r = 0; r < kLitDxTok; ++r) {
                    const f32x4 p = *(const f32x4*)&ps[r][q];
#pragma unroll
                    for (int u = 0; u < 4; ++u)
#pragma unroll
                        for (int cc = 0; cc < 4; ++cc)
                            racc[r][cc] = fmaf(p[u], w[u][cc], racc[r][cc]);
                }
            }
            for (; q < jn; ++q) {
                const f32x4 w = *(const f32x4*)(wcol + (int64_t)q * d);
#pragma unroll
                for (int r = 0; r < kLitDxTok; ++r)
#pragma unroll
                    for (int cc = 0; cc < 4; ++cc) racc[r][cc] = fmaf(ps[r][q], w[cc], racc[r][cc]);
            }
        }
        __syncthreads();
    }
    if (c >= d) return;
#pragma unroll
    for (int r = 0; r < kLitDxTok; ++r) {
        const int64_t t = t0 + r;
        if (t >= Ttot) break;
        float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        for (int s = 0; s < k; ++s) {
            const int q = inv[t * k + s];
            if (q < 0) continue;
            const T* row = dxr + (int64_t)q * d + c;
#pragma unroll
            for (int cc = 0; cc < 4; ++cc) acc[cc] += Act<T>::to_f32(row[cc]);
        }
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) dx[t * d + c + cc] = Act<T>::from_f32(acc[cc] + racc[r][cc]);
    }
}

__global__ void __launch_bounds__(256) fill_zero_kernel(float* p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0.0f;
}

hipError_t zero(float* p, int64_t n, hipStream_t s) {
    if (!p || n <= 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_generic_gemms(const pr2_moe_desc& d, const void* x, const void* Wg,
                                const void* Wu, const void* dy, const BwdWs& ws,
                                const BwdGrads& out, hipStream_t s) {
    // the SwiGLU backward (dh_generic) has already run: AU holds da | du, H holds g H
    const ReplayWs& w = ws.fw;
    hipError_t e;
    {
        LaunchScope scope("bwd_dx_generic", s);
        hipLaunchKernelGGL(dx_generic<T>, dim3((unsigned)w.max_tiles, (unsigned)d.d), dim3(256), 0,
                           s, (const T*)ws.AU, (const T*)Wg, (const T*)Wu, d.d, d.m, w.tiles,
                           w.tile_count, (T*)w.O);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    {
        LaunchScope scope("bwd_wd_generic", s);
        hipLaunchKernelGGL(wd_generic<T>, dim3((unsigned)d.N, (unsigned)d.d), dim3(256), 0, s,
                           (const T*)dy, (const T*)w.H, w.perm_src, w.offsets, d.k, d.d, d.m,
                           out.dW_down);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    LaunchScope scope("bwd_wgu_generic", s);
    hipLaunchKernelGGL(wgu_generic<T>, dim3((unsigned)d.N, (unsigned)(2 * d.m)), dim3(256), 0, s,
                       (const T*)x, (const T*)ws.AU, w.perm_src, w.offsets, d.k, d.d, d.m,
                       out.dW_gate, out.dW_up);
    return hipGetLastError();
}

}  // namespace

bool bwd_mfma_ok(const pr2_moe_desc& d) {
    const int64_t lim = (int64_t)1 << 31;
    const int64_t Tk = d.T * (int64_t)d.k;
    // (route entries below 2^32 / k keep the multiply-high token division exact)
    return mfma_shape_ok(d) && d.m % BN == 0 && d.d % BN == 0 && Tk * 2 * d.m < lim &&
           Tk * (int64_t)d.k < ((int64_t)1 << 32);
}

int bwd_partials(const pr2_moe_desc& d) { return bwd_mfma_ok(d) ? d.m / 128 : d.m; }

hipError_t launch_zero_grads(const pr2_moe_desc& d, const BwdGrads& out, hipStream_t s) {
    LaunchScope scope("bwd_zero_grads", s);
    const int64_t wmd = (int64_t)d.N * d.m * d.d;
    hipError_t e;
    if ((e = zero(out.dW_r, (int64_t)d.d * d.N, s)) != hipSuccess) return e;
    if ((e = zero(out.db_r, d.N, s)) != hipSuccess) return e;
    if ((e = zero(out.dW_gate, wmd, s)) != hipSuccess) return e;
    if ((e = zero(out.dW_up, wmd, s)) != hipSuccess) return e;
    return zero(out.dW_down, wmd, s);
}

hipError_t launch_replay_backward(const pr2_moe_desc& d, const void* x, const void* idx,
                                  int64_t ldi, const float* W_r, const void* W_gate,
                                  const void* W_up, const void* W_down, const void* dy,
                                  const float* gate, const BwdWs& ws, const BwdGrads& out,
                                  hipStream_t s, const void* au_in) {
    const ReplayWs& w = ws.fw;
    const bool bf = d.act_dtype == PR2_BF16;
    const bool mfma = bwd_mfma_ok(d);
    hipError_t e = hipSuccess;
    // the pre-activations: recomputed, or read from the forward's saved copy
    if (!au_in && (e = launch_preact(d, x, W_gate, W_up, w, ws.AU, s)) != hipSuccess) return e;

    BwdArgs g{};
    g.perm_src = w.perm_src;
    g.tiles = w.tiles;
    g.tile_count = w.tile_count;
    g.offsets = w.offsets;
    g.order = ws.order;
    g.k = d.k;
    g.kmul = d.k == 1 ? 0u : (uint32_t)(0xffffffffull / (uint64_t)d.k + 1);
    g.N = d.N;
    g.d = d.d;
    g.m = d.m;
    g.Tk = (int)(d.T * d.k);
    g.x = (const bf16_t*)x;
    g.dy = (const bf16_t*)dy;
    g.Wg = (const bf16_t*)W_gate;
    g.Wu = (const bf16_t*)W_up;
    g.Wd = (const bf16_t*)W_down;
    g.gate = gate;
    g.AU = (bf16_t*)ws.AU;
    g.AUin = au_in ? (const bf16_t*)au_in : g.AU;
    g.Hg = (bf16_t*)w.H;
    g.dgp = ws.dgp;
    g.dxr = (bf16_t*)w.O;
    g.dWg = out.dW_gate;
    g.dWu = out.dW_up;
    g.dWd = out.dW_down;
    auto grid_for = [](int64_t work) {
        return dim3((unsigned)(((work + kNumXcd - 1) / kNumXcd) * kNumXcd));
    };

    // gate gradient partials and the SwiGLU backward
    if (mfma) {
        g.ntn = d.m / BN;
        LaunchScope scope("bwd_dh_swiglu", s);
        hipLaunchKernelGGL(bwd_gemm<DH>, grid_for(w.max_tiles * g.ntn), dim3(kThreads), 0, s, g);
    } else {
        LaunchScope scope("bwd_dh_generic", s);
        if (bf)
            hipLaunchKernelGGL(dh_generic<bf16_t>, dim3((unsigned)w.max_tiles, (unsigned)d.m),
                               dim3(256), 0, s, (const bf16_t*)dy, w.perm_src, d.k,
                               (const bf16_t*)W_down, gate, d.d, d.m, w.tiles, w.tile_count,
                               au_in ? (const bf16_t*)au_in : (const bf16_t*)ws.AU,
                               (bf16_t*)ws.AU, (bf16_t*)w.H, ws.dgp);
        else
            hipLaunchKernelGGL(dh_generic<float>, dim3((unsigned)w.max_tiles, (unsigned)d.m),
                               dim3(256), 0, s, (const float*)dy, w.perm_src, d.k,
                               (const float*)W_down, gate, d.d, d.m, w.tiles, w.tile_count,
                               au_in ? (const float*)au_in : (const float*)ws.AU,
                               (float*)ws.AU, (float*)w.H, ws.dgp);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // router-logit gradients (needed by the router weight gradient below)
    const bool literal = d.renorm == 0;
    if (literal) {
        LaunchScope scope("bwd_gate_grad_literal", s);
        hipLaunchKernelGGL(literal_dp_kernel, dim3((unsigned)((d.T + 3) / 4)), dim3(256), 0, s,
                           ws.dgp, ws.np, w.inv, gate, ws.plog, idx, d.idx_dtype, ldi, d.T, d.k,
                           d.N, ws.dpf);
    } else {
        LaunchScope scope("bwd_gate_grad", s);
        int kp_log2 = 0;
        while ((1 << kp_log2) < d.k) ++kp_log2;
        if (kp_log2 <= 6) {
            const int64_t lanes = d.T << kp_log2;
            hipLaunchKernelGGL(gate_grad_lanes_kernel, dim3((unsigned)((lanes + 255) / 256)), dim3(256),
                               0, s, ws.dgp, ws.np, w.inv, gate, d.T, d.k, kp_log2, ws.dp_route,
                               ws.dp_perm);
        } else {
            hipLaunchKernelGGL(gate_grad_kernel, dim3((unsigned)((d.T + 255) / 256)), dim3(256), 0, s,
                               ws.dgp, ws.np, w.inv, gate, d.T, d.k, ws.dp_route, ws.dp_perm);
        }
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;

    // W_r transposed, [N, d]: rows of the router term
    auto launch_transpose_wr = [&](hipStream_t ts) -> hipError_t {
        LaunchScope scope("bwd_transpose_wr", ts);
        hipLaunchKernelGGL(transpose_wr_kernel,
                           dim3((unsigned)((d.d + 31) / 32), (unsigned)((d.N + 31) / 32)), dim3(256),
                           0, ts, W_r, d.d, d.N, ws.wrt);
        return hipGetLastError();
    };
    // the router weight gradient and the combine of the input gradient
    auto tail = [&](hipStream_t ts) -> hipError_t {
        hipError_t e = hipSuccess;
        if (literal) {
            // dense over all N logits
            {
                LaunchScope scope("bwd_router_wgrad_literal", ts);
                dim3 grid((unsigned)((d.d + kLitTile - 1) / kLitTile),
                          (unsigned)((d.N + kLitTile - 1) / kLitTile), (unsigned)ws.nchunk);
                if (bf)
                    hipLaunchKernelGGL(literal_wgrad_partial_kernel<bf16_t>, grid, dim3(256), 0, ts,
                                       (const bf16_t*)x, ws.dpf, d.T, d.d, d.N, ws.lwpart,
                                       ws.lbpart);
                else
                    hipLaunchKernelGGL(literal_wgrad_partial_kernel<float>, grid, dim3(256), 0, ts,
                                       (const float*)x, ws.dpf, d.T, d.d, d.N, ws.lwpart,
                                       ws.lbpart);
                if ((e = hipGetLastError()) != hipSuccess) return e;
                const int64_t n = (int64_t)d.d * d.N;
                int64_t blocks = (n + 255) / 256;
                if (blocks > 4096) blocks = 4096;
                hipLaunchKernelGGL(literal_wgrad_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0,
                                   ts, ws.lwpart, ws.lbpart, ws.nchunk, n, d.N, out.dW_r, out.db_r);
                if ((e = hipGetLastError()) != hipSuccess) return e;
            }
            if ((e = launch_transpose_wr(ts)) != hipSuccess) return e;
            LaunchScope scope("bwd_dx_combine_literal", ts);
            if (d.d % 4 == 0) {
                dim3 grid4((unsigned)((d.d + 1023) / 1024),
                           (unsigned)((d.T + kLitDxTok - 1) / kLitDxTok));
                if (bf)
                    hipLaunchKernelGGL(literal_dx_combine4_kernel<bf16_t>, grid4, dim3(256), 0, ts,
                                       (const bf16_t*)w.O, w.inv, ws.dpf, ws.wrt, d.T, d.k, d.d, d.N,
                                       (bf16_t*)out.dx);
                else
                    hipLaunchKernelGGL(literal_dx_combine4_kernel<float>, grid4, dim3(256), 0, ts,
                                       (const float*)w.O, w.inv, ws.dpf, ws.wrt, d.T, d.k, d.d, d.N,
                                       (float*)out.dx);
                return hipGetLastError();
            }
            dim3 grid((unsigned)((d.d + 255) / 256), (unsigned)((d.T + kLitDxTok - 1) / kLitDxTok));
            if (bf)
                hipLaunchKernelGGL(literal_dx_combine_kernel<bf16_t>, grid, dim3(256), 0, ts,
                                   (const bf16_t*)w.O, w.inv, ws.dpf, ws.wrt, d.T, d.k, d.d, d.N,
                                   (bf16_t*)out.dx);
            else
                hipLaunchKernelGGL(literal_dx_combine_kernel<float>, grid, dim3(256), 0, ts,
                                   (const float*)w.O, w.inv, ws.dpf, ws.wrt, d.T, d.k, d.d, d.N,
                                   (float*)out.dx);
            return hipGetLastError();
        }
        {
            LaunchScope scope("bwd_router_wgrad", ts);
            dim3 grid((unsigned)w.max_tiles, (unsigned)((d.d + 255) / 256));
            if (bf)
                hipLaunchKernelGGL(router_wgrad_partial_kernel<bf16_t>, grid, dim3(256), 0, ts,
                                   (const bf16_t*)x, w.perm_src, w.tiles, w.tile_count, ws.dp_perm, d.k,
                                   d.d, ws.rwpart, ws.rbpart);
            else
                hipLaunchKernelGGL(router_wgrad_partial_kernel<float>, grid, dim3(256), 0, ts,
                                   (const float*)x, w.perm_src, w.tiles, w.tile_count, ws.dp_perm, d.k,
                                   d.d, ws.rwpart, ws.rbpart);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            hipLaunchKernelGGL(router_wgrad_reduce_kernel, dim3((unsigned)d.N, (unsigned)((d.d + 255) / 256)),
                               dim3(256), 0, ts, w.offsets, ws.rwpart, ws.rbpart, kTileM, d.d, d.N,
                               out.dW_r, out.db_r);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }

        // input gradient: per-route rows plus the router term dp W_r^T
        if ((e = launch_transpose_wr(ts)) != hipSuccess) return e;
        LaunchScope scope("bwd_dx_combine", ts);
        if (bf && d.d % 8 == 0) {
            const int64_t want = (d.T + kDxTok - 1) / kDxTok;
            hipLaunchKernelGGL(dx_combine_bf16_kernel, dim3((unsigned)(want < 8192 ? want : 8192)),
                               dim3(256), 0, ts, (const bf16_t*)w.O, w.inv, ws.dp_route, ws.wrt, idx,
                               d.idx_dtype, ldi, d.T, d.k, d.d, d.N, (bf16_t*)out.dx);
        } else if (bf) {
            hipLaunchKernelGGL(dx_combine_kernel<bf16_t>, dim3((unsigned)d.T), dim3(256), 0, ts,
                               (const bf16_t*)w.O, w.inv, ws.dp_route, ws.wrt, idx, d.idx_dtype, ldi,
                               d.T, d.k, d.d, d.N, (bf16_t*)out.dx);
        } else {
            hipLaunchKernelGGL(dx_combine_kernel<float>, dim3((unsigned)d.T), dim3(256), 0, ts,
                               (const float*)w.O, w.inv, ws.dp_route, ws.wrt, idx, d.idx_dtype, ldi,
                               d.T, d.k, d.d, d.N, (float*)out.dx);
        }
        return hipGetLastError();
    };

    if (mfma) {
        {
            LaunchScope scope("bwd_expert_order", s);
            hipLaunchKernelGGL(expert_order_kernel, dim3(1), dim3(1024), 0, s, w.offsets, d.N,
                               ws.order);
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
        g.ntn = d.d / BN;
        {
            LaunchScope scope("bwd_dx_gemm", s);
            hipLaunchKernelGGL(bwd_gemm<DX>, grid_for(w.max_tiles * g.ntn), dim3(kThreads), 0, s, g);
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
        const int64_t experts_per_xcd = (d.N + kNumXcd - 1) / kNumXcd;
        {
            LaunchScope scope("bwd_wgrad_down", s);
            hipLaunchKernelGGL(bwd_gemm<WD>,
                               dim3((unsigned)(kNumXcd * experts_per_xcd * (d.d / BM) * (d.m / BN))),
                               dim3(kThreads), 0, s, g);
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
        {
            LaunchScope scope("bwd_wgrad_gate_up", s);
            hipLaunchKernelGGL(bwd_gemm<WGU>,
                               dim3((unsigned)(kNumXcd * experts_per_xcd * (2 * d.m / BM) * (d.d / BN))),
                               dim3(kThreads), 0, s, g);
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
        return tail(s);
    }
    e = bf ? launch_generic_gemms<bf16_t>(d, x, W_gate, W_up, dy, ws, out, s)
           : launch_generic_gemms<float>(d, x, W_gate, W_up, dy, ws, out, s);
    if (e != hipSuccess) return e;
    return tail(s);
}

}  // namespace pr2
