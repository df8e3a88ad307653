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
// 16-byte DMA loads (no register staging), two LDS stages deep (the next slice
// in flight while one is consumed), 16-byte chunks XOR-swizzled per row so the
// MFMA operand reads are free of bank conflicts.
// Eight wavefronts (two per SIMD) in a 4 x 2 arrangement each own 64 rows x 128
// panel rows as 4 x 8 tiles of v_mfma_f32_16x16x32_bf16 (fp32 accumulation;
// it issues about 9 % faster than the 32x32x16 form on gfx950 and gives the
// same sums);
// operand fragments are double-buffered in registers so the LDS reads of one
// K=32 step overlap the MFMAs of the previous one; a wavefront whose rows are
// all past the end of a partial tile skips its MFMAs.
// GEMM1's epilogue applies SwiGLU in registers (gate and up tiles of the same
// columns live in the same lanes) and rounds H to bf16; GEMM2's epilogue scales
// by the route weight and rounds O to bf16.  The MFMA operands are given as
// (weights, tokens), so each lane's accumulators hold runs of four consecutive
// output columns of one token row.  GEMM1 stores them 8 bytes at a time
// straight from registers; GEMM2 (and the pre-activation epilogue below)
// stages its outputs through the freed LDS stages so that every store covers
// whole row segments.  Workgroups are mapped so that each XCD takes a
// contiguous range of the tile list (same experts, shared L2).
//
// A third epilogue serves the backward pass: it stores the pre-activations
// a = X_e W_gate_e^T and u = X_e W_up_e^T (bf16) instead of H; a fourth stores
// both (a forward that saves them for the backward).
//
// When m is a multiple of 192, the forward GEMM1 runs a second kernel with a
// 384-row panel (192 gate + 192 up rows; 80 KiB per LDS stage, all 160 KiB of
// LDS in two stages), 17 % fewer copied bytes per flop: each of the eight
// wavefronts owns 64 token rows x 192 panel rows (192 accumulators per lane),
// reads its A fragments once per K=32 step and its B fragments two tiles at a
// time, double-buffered.  Per output the sums run in the same K order as the
// 256-row panel, so H is bitwise the same; measured 2 % faster on both layer
// shapes.
//
// Other shapes and the fp32 path use a plain one-thread-per-output kernel.
#include "common.h"

namespace pr2 {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int BM = kTileM;      // 256 rows per tile
constexpr int BP = 256;         // weight panel rows per tile
constexpr int BK = 64;          // K slice: 128 bytes per row (32 and 64 supported)
constexpr int ROWB = BK * 2;    // bytes per LDS row (unpadded; chunks are swizzled)
constexpr int CHUNKS = ROWB / 16;   // 16-byte chunks per row
constexpr int NSTAGE = 2;       // LDS stages: slices kt+1 .. kt+NSTAGE-1 in flight during slice kt
constexpr int WM = 64;          // token rows per wavefront
constexpr int WN = 128;         // panel rows per wavefront
constexpr int MT = 16;          // MFMA tile edge: 16 (16x16x32, faster here) or 32 (32x32x16)
constexpr int MK = 512 / MT;    // K per MFMA
constexpr int NKS = BK / MK;    // MFMA K sub-steps per slice
constexpr int ACCN = MT * MT / 64;  // accumulators per lane per tile
constexpr int MI = WM / MT;     // MFMA tiles per wavefront, token direction
constexpr int NJ = WN / MT;     // MFMA tiles per wavefront, panel direction
template <int E> struct MfmaOp;
template <> struct MfmaOp<32> {
    typedef f32x16 acc_t;
    __device__ __forceinline__ static acc_t run(bf16x8 a, bf16x8 b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
};
template <> struct MfmaOp<16> {
    typedef f32x4 acc_t;
    __device__ __forceinline__ static acc_t run(bf16x8 a, bf16x8 b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};
typedef MfmaOp<MT>::acc_t accv;
static_assert(sizeof(accv) == ACCN * sizeof(float), "accumulator size");

__device__ __forceinline__ accv mfma_bf16(bf16x8 a, bf16x8 b, accv c) {
    return MfmaOp<MT>::run(a, b, c);
}
// tiles per group of the work order (1: tile-major, every panel of a tile in turn)
constexpr int kGroupGemm1 = 1;
constexpr int kGroupGemm2 = 1;
constexpr int NWAVE = (BM / WM) * (BP / WN);
constexpr int kGemmThreads = 64 * NWAVE;
constexpr int kNumXcd = 8;
constexpr int kRowsPerDma = 1024 / ROWB;                                   // 8 rows / DMA
constexpr int kGroups = (BM + BP) / kRowsPerDma / NWAVE;                    // DMAs / wavefront
constexpr int STAGEB = (BM + BP) * ROWB;                                    // 64 KiB
constexpr int LDSB = NSTAGE * STAGEB;

struct MfmaArgs {
    const bf16_t* A;        // GEMM1: x [T, d]; GEMM2: H [T*k, m]
    const int* perm_src;    // permuted row -> t*k + s
    int k;
    int Tk;                 // routes (perm_src entries)
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
    bf16_t* out2;           // GEMM1 that also saves a | u (MODE 3): [T*k, 2m]
    int group;              // work order: groups of this many tiles, panel-major inside
};

// silu(a) = a / (1 + e^-a) with the hardware reciprocal (about 1 ulp; H is rounded to bf16)
__device__ __forceinline__ float silu_f(float a) {
    return a * __builtin_amdgcn_rcpf(1.0f + __expf(-a));
}

// 16-byte chunk c of LDS row r is stored at position c ^ swz(r): any 16 (or
// 8) consecutive rows read at the same chunk hit disjoint banks.  swz depends
// on r % 16 only.
__device__ __forceinline__ int swz(int r) {
    return CHUNKS == 8 ? (r & 7) ^ ((r >> 3) & 1) : ((r >> 1) ^ (r >> 2)) & 3;
}

// wait until at most n of this wavefront's global loads are outstanding
template <int n>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(n >= 0 && n < 16, "vmcnt field");
    __builtin_amdgcn_s_waitcnt(0x0f70 | n);   // expcnt and lgkmcnt left at their maxima
}

template <int MODE>
__global__ void __launch_bounds__(kGemmThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
grouped_gemm_mfma(MfmaArgs g) {
    __shared__ __attribute__((aligned(1024))) unsigned char lds[LDSB];

    // XCD-aware mapping: physical block b runs on XCD b % 8; give each XCD a
    // contiguous range of the (tile, panel) work list.  The list runs over
    // groups of g.group consecutive tiles (the last group may be smaller); inside
    // a group it is panel-major, so the workgroups that start together share
    // one weight panel and the group's gathered rows stay in that XCD's L2.
    const int ntile = *g.tile_count;
    const int64_t L = (int64_t)ntile * g.ntn;
    const int64_t per_xcd = (L + kNumXcd - 1) / kNumXcd;
    const int64_t local = blockIdx.x / kNumXcd;
    if (local >= per_xcd) return;
    const int64_t logical = (int64_t)(blockIdx.x % kNumXcd) * per_xcd + local;
    if (logical >= L) return;
    const int64_t wgrp = logical / ((int64_t)g.group * g.ntn);
    const int first = (int)(wgrp * g.group);
    const int gsz = min(g.group, ntile - first);
    const int within = (int)(logical - wgrp * g.group * g.ntn);
    const int tile = first + within % gsz;
    const int pn = within / gsz;
    const int expert = g.tiles[3 * tile + 0];
    const int row0 = g.tiles[3 * tile + 1];
    const int rows = g.tiles[3 * tile + 2];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    // uniform across the wavefront; saying so lets the compiler branch on it
    // with scalar branches instead of per-lane masks
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wr = wave / (BP / WN);     // token-row block of WM rows
    const int wc = wave % (BP / WN);     // panel block of WN rows
    // a wavefront whose rows are all past the tile's end only helps copy
    const bool active = wr * WM < rows;
    // each lane's accumulators belong to MI token rows (one per MT-row block);
    // GEMM2's route weights for them are fetched now, long before the epilogue
    // (loads are unconditional, rows clamped into the tile, so that they all
    // go out together rather than one masked branch at a time)
    float gw[MI];
    if (MODE == 1) {
        int src[MI];
#pragma unroll
        for (int i = 0; i < MI; ++i) src[i] = g.perm_src[row0 + min(wr * WM + i * MT + (lane % MT), rows - 1)];
#pragma unroll
        for (int i = 0; i < MI; ++i) gw[i] = g.gate[min(max(src[i], 0), g.Tk - 1)];
#pragma unroll
        for (int i = 0; i < MI; ++i)
            if (wr * WM + i * MT + (lane % MT) >= rows) gw[i] = 0.0f;
    }

    // DMA assignments: wavefront w copies row groups w*kGroups .. of the
    // [A rows | panel rows] tile; lane l moves row grp*kRowsPerDma + l/CHUNKS,
    // position l%CHUNKS.  A wavefront's groups all come from one tensor (the
    // token rows, the gate or up panel, or the down panel), so it keeps one
    // base pointer and a 32-bit element offset per group.
    const int wrow0 = wave * kGroups * kRowsPerDma;
    const bf16_t* sbase;
    if (wrow0 < BM) sbase = g.A;
    else if (MODE != 1) sbase = (wrow0 - BM < 128 ? g.W0 : g.W1) + (int64_t)expert * g.w_stride;
    else sbase = g.W0 + (int64_t)expert * g.w_stride;
    // (wrow0 < BM holds for a whole wavefront: a scalar branch, and the
    // gathered route entries are loaded together before any is used)
    uint32_t soff[kGroups];
    if (wrow0 < BM) {
        // rows past the tile's end read a valid row; their results are never stored
        int rsrc[kGroups];
#pragma unroll
        for (int i = 0; i < kGroups; ++i) {
            const int r = wrow0 + i * kRowsPerDma + lane / CHUNKS;
            const int rr = r < rows ? r : 0;
            rsrc[i] = MODE != 1 ? g.perm_src[row0 + rr] : row0 + rr;
        }
#pragma unroll
        for (int i = 0; i < kGroups; ++i) {
            const int r = wrow0 + i * kRowsPerDma + lane / CHUNKS;
            const int64_t row = MODE != 1 ? (int64_t)(min(max(rsrc[i], 0), g.Tk - 1) / g.k) : rsrc[i];
            soff[i] = (uint32_t)(row * g.K + ((lane % CHUNKS) ^ swz(r)) * 8);
        }
    } else {
#pragma unroll
        for (int i = 0; i < kGroups; ++i) {
            const int r = wrow0 + i * kRowsPerDma + lane / CHUNKS;  // row in [BM, BM + BP)
            const int pr = r - BM;
            const int64_t off = MODE != 1 ? (int64_t)(pn * 128 + (pr & 127)) * g.K
                                          : (int64_t)(pn * BP + pr) * g.K;
            soff[i] = (uint32_t)(off + ((lane % CHUNKS) ^ swz(r)) * 8);
        }
    }
    // A groups of 8 token rows wholly past the end of a partial tile are not
    // copied: no stored output depends on those LDS rows (a wavefront-uniform,
    // scalar test).  The K loop's waits are for all copies in flight (two
    // stages: vmcnt 0), so the count issued does not matter; a deeper pipeline
    // would count copies per stage and must not skip any.
    static_assert(NSTAGE == 2, "the copy skip below assumes vmcnt(0) waits");
    auto issue = [&](int stage, int k0) {
#pragma unroll
        for (int i = 0; i < kGroups; ++i) {
            const int grp = wave * kGroups + i;
            if (wrow0 < BM && wrow0 + i * kRowsPerDma >= rows) continue;
            __builtin_amdgcn_global_load_lds((const void*)(sbase + (soff[i] + (uint32_t)k0)),
                                             (lds_void*)&lds[stage * STAGEB + grp * 1024], 16,
                                             0, 0);
        }
    };

    accv acc[MI][NJ];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int v = 0; v < ACCN; ++v) acc[i][j][v] = 0.0f;

    // LDS reads for the MFMA operands: lane l reads row (block base + l%MT)
    // and the 16 bytes of one 8-wide K chunk, at position chunk ^ swz(row);
    // block bases are multiples of 16 rows, so the swizzle is the same for
    // every fragment.  Which chunk of the sub-step a lane group g = l/MT
    // takes is free (A and B fragments use the same assignment, so each MFMA
    // still sums over the same K values): a ds_read_b128 serves lanes
    // 8q..8q+7 together with lanes 32+8q..32+8q+7, so for 16x16 tiles groups
    // g and g+2 take chunks differing in the lowest bit (0,2,1,3), which keeps
    // the two halves of every LDS cycle in disjoint banks.
    const int lrow = lane % MT;
    const int sw = swz(lrow);
    const int grp = lane / MT;
    const int cperm = MT == 16 ? (((grp & 1) << 1) | (grp >> 1)) : grp;
    int kpos[NKS];
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
        kpos[ks] = lrow * ROWB + ((((MK / 8) * ks + cperm) ^ sw) << 4);
    int a_base[MI], b_base[NJ];
#pragma unroll
    for (int i = 0; i < MI; ++i) a_base[i] = (wr * WM + i * MT) * ROWB;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        int prow;
        if (MODE != 1) prow = (j < NJ / 2 ? 0 : 128) + wc * (WN / 2) + (j % (NJ / 2)) * MT;
        else prow = wc * WN + j * MT;
        b_base[j] = (BM + prow) * ROWB;
    }

    const int nk = g.K / BK;
#pragma unroll
    for (int st = 0; st < NSTAGE - 1; ++st)
        if (st < nk) issue(st, st * BK);
    for (int kt = 0; kt < nk; ++kt) {
        // slice kt landed (the copies of the later slices may still be in
        // flight) and every wavefront is done with slice kt-1, whose stage is
        // refilled next
        if (kt + NSTAGE - 2 < nk) wait_vmcnt<(NSTAGE - 2) * kGroups>();
        else wait_vmcnt<0>();
        __syncthreads();
        if (kt + NSTAGE - 1 < nk) issue((kt + NSTAGE - 1) % NSTAGE, (kt + NSTAGE - 1) * BK);
        if (active) {
            // fragments double-buffered in registers: the reads for sub-step
            // ks+1 are in flight while the MFMAs of sub-step ks run
            const unsigned char* base = lds + (kt % NSTAGE) * STAGEB;
            bf16x8 fa[2][MI], fb[2][NJ];
            auto read_frags = [&](int buf, int ks) {
#pragma unroll
                for (int i = 0; i < MI; ++i)
                    fa[buf][i] = __builtin_bit_cast(bf16x8, *(const u32x4*)(base + a_base[i] + kpos[ks]));
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    fb[buf][j] = __builtin_bit_cast(bf16x8, *(const u32x4*)(base + b_base[j] + kpos[ks]));
            };
            read_frags(0, 0);
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) {
                if (ks + 1 < NKS) read_frags((ks + 1) & 1, ks + 1);
                // keep the scheduler from sinking those reads below the MFMAs
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int i = 0; i < MI; ++i)
#pragma unroll
                    for (int j = 0; j < NJ; ++j)
                        acc[i][j] = mfma_bf16(fb[ks & 1][j], fa[ks & 1][i], acc[i][j]);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
    // Epilogue.  The MFMA computed the transposed tile (weights x tokens), so
    // accumulator element v of lane l is, for 16x16 tiles, column 4*(l/16) + v
    // of token row l%16 of its block (for 32x32 tiles, column
    // 8*(v/4) + 4*(l/32) + v%4 of token row l%32): runs of four consecutive
    // outputs per lane.
    if ((MODE == 0 || MODE == 3) && active) {
        // GEMM1: H = silu(gate) * up, stored straight from registers, one
        // 8-byte write per run (gate and up tiles of the same columns sit in
        // the same lanes)
        const int ncol0 = 4 * (lane / MT);
        constexpr int NA4 = ACCN / 4;           // runs of four per tile
        constexpr int A4STEP = MT == 32 ? 8 : 0;
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            const int r = wr * WM + i * MT + (lane % MT);
            if (r >= rows) continue;
            bf16_t* orow = g.out + ((int64_t)row0 + r) * g.n_out;
#pragma unroll
            for (int j = 0; j < NJ / 2; ++j) {
                const int col = pn * 128 + wc * (WN / 2) + j * MT + ncol0;
#pragma unroll
                for (int a4 = 0; a4 < NA4; ++a4) {
                    uint32_t w[2];
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int v0 = 4 * a4 + 2 * h;
                        const float h0 = silu_f(acc[i][j][v0]) * acc[i][j + NJ / 2][v0];
                        const float h1 = silu_f(acc[i][j][v0 + 1]) * acc[i][j + NJ / 2][v0 + 1];
                        w[h] = (uint32_t)f32_to_bf16(h0) | ((uint32_t)f32_to_bf16(h1) << 16);
                    }
                    *(uint2*)(orow + col + A4STEP * a4) = make_uint2(w[0], w[1]);
                }
            }
        }
    }
    // MODE 3 goes on to save the pre-activations a | u as MODE 2 stores them
    if (MODE == 0) return;

    // GEMM2 (route weight times the output) and the pre-activations (a and u)
    // are staged: the rounded outputs go into this wavefront's LDS region (64
    // rows of CW columns per output block, 16-byte chunks XOR-swizzled by
    // row, the two 8-byte halves of a chunk swapped in rows with bit 3 set so
    // that the 16 rows of one 8-byte write cycle hit 16 distinct bank pairs)
    // and are read back 16 bytes per lane, so that each global store
    // covers whole row segments (256 or 128 contiguous bytes) instead of
    // 8-byte pieces of 16 rows: measured 10 % faster for GEMM2 (and slower
    // for GEMM1, whose outputs are half as wide).
    // Every wavefront must be done with the operand stages first.
    __syncthreads();
    if (!active) return;
    static_assert(MT == 16, "staged epilogue assumes 16x16 MFMA tiles");
    constexpr int CW = MODE == 1 ? WN : WN / 2;          // columns per output block
    constexpr bool kPreact = MODE == 2 || MODE == 3;     // stores a | u
    constexpr int NB = kPreact ? 2 : 1;                   // output blocks per wavefront
    constexpr int RB = CW * 2;                            // bytes per staged row
    constexpr int NCH = RB / 16;                          // 16-byte chunks per row
    unsigned char* stage_w = lds + wave * (NB * WM * RB);
    auto spos = [&](int blk, int row, int col) {          // byte offset of (row, col), col % 4 == 0
        const int ch = (col >> 3) ^ (row & (NCH - 1));
        return blk * WM * RB + row * RB + (ch << 4) + (((col & 4) << 1) ^ (row & 8));
    };
    const int ncol0 = 4 * (lane / MT);
#pragma unroll
    for (int i = 0; i < MI; ++i) {
        const int row = i * MT + (lane % MT);
#pragma unroll
        for (int j = 0; j < (MODE == 1 ? NJ : NJ / 2); ++j) {
            const int col = j * MT + ncol0;
            if (kPreact) {
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    const int jj = j + half * (NJ / 2);
                    const uint32_t w0 = (uint32_t)f32_to_bf16(acc[i][jj][0]) |
                                        ((uint32_t)f32_to_bf16(acc[i][jj][1]) << 16);
                    const uint32_t w1 = (uint32_t)f32_to_bf16(acc[i][jj][2]) |
                                        ((uint32_t)f32_to_bf16(acc[i][jj][3]) << 16);
                    *(uint2*)(stage_w + spos(half, row, col)) = make_uint2(w0, w1);
                }
            } else {
                const uint32_t w0 = (uint32_t)f32_to_bf16(gw[i] * acc[i][j][0]) |
                                    ((uint32_t)f32_to_bf16(gw[i] * acc[i][j][1]) << 16);
                const uint32_t w1 = (uint32_t)f32_to_bf16(gw[i] * acc[i][j][2]) |
                                    ((uint32_t)f32_to_bf16(gw[i] * acc[i][j][3]) << 16);
                *(uint2*)(stage_w + spos(0, row, col)) = make_uint2(w0, w1);
            }
        }
    }
    // the wavefront's own region: LDS operations of one wavefront complete in order
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
    constexpr int RPI = 64 / NCH;                         // rows per 64-lane pass
    const int rsub = lane / NCH, ch = lane % NCH;
    bf16_t* const dst = MODE == 3 ? g.out2 : g.out;
    const int ldo = MODE == 3 ? 2 * g.n_out : g.n_out;   // MODE 3: H rows are m, a | u rows 2m
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) {
        int colbase;
        if (MODE == 1) colbase = pn * BP + wc * WN;
        else colbase = blk * (ldo / 2) + pn * 128 + wc * (WN / 2);
#pragma unroll
        for (int p = 0; p < WM / RPI; ++p) {
            const int row = p * RPI + rsub;
            const int r = wr * WM + row;
            u32x4 v = *(const u32x4*)(stage_w + blk * WM * RB + row * RB + ((ch ^ (row & (NCH - 1))) << 4));
            if (row & 8) v = u32x4{v[2], v[3], v[0], v[1]};
            if (r < rows) *(u32x4*)(dst + ((int64_t)row0 + r) * ldo + colbase + ch * 8) = v;
        }
    }
}

// ---------------------------------------------------------------- generic --
// pre-activations a = x W_gate^T, u = x W_up^T of each permuted row (backward recompute)
template <typename T>
__global__ void __launch_bounds__(256)
preact_generic(const T* x, const int* perm_src, int k, const T* Wg, const T* Wu, int d, int m,
               const int* tiles, const int* tile_count, T* AU) {
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
    T* o = AU + (int64_t)(row0 + r) * 2 * m;
    o[col] = Act<T>::from_f32(a);
    o[m + col] = Act<T>::from_f32(b);
}

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

// ------------------------------------------- GEMM1 with a 384-row panel --
constexpr int BPW = 384;                          // panel rows
constexpr int WNW = 192;                          // panel rows per wavefront (96 gate + 96 up)
constexpr int NJW = WNW / MT;                     // 12
constexpr int STAGEBW = (BM + BPW) * ROWB;        // 80 KiB
constexpr int LDSBW = NSTAGE * STAGEBW;           // 160 KiB
constexpr int kAGroupsW = BM / kRowsPerDma / NWAVE;          // 4 token-row groups per wavefront
constexpr int kWGroupsW = (BPW / 2) / kRowsPerDma / NWAVE;   // 3 gate (and 3 up) groups per wavefront
static_assert(kAGroupsW * kRowsPerDma * NWAVE == BM && kWGroupsW * kRowsPerDma * NWAVE * 2 == BPW,
              "row groups divide evenly");

__global__ void __launch_bounds__(kGemmThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
gemm1_wide(MfmaArgs g) {
    __shared__ __attribute__((aligned(1024))) unsigned char lds[LDSBW];
    const int ntile = *g.tile_count;
    const int64_t L = (int64_t)ntile * g.ntn;
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
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wr = wave / (BPW / WNW);
    const int wc = wave % (BPW / WNW);
    const bool active = wr * WM < rows;

    // copies: wavefront w moves token-row groups 4w..4w+3, gate groups
    // 3w..3w+2 and up groups 3w..3w+2 (8 rows of 128 bytes each)
    const bf16_t* wg = g.W0 + (int64_t)expert * g.w_stride;
    const bf16_t* wu = g.W1 + (int64_t)expert * g.w_stride;
    uint32_t soa[kAGroupsW], sog[kWGroupsW], sou[kWGroupsW];
    {
        int rsrc[kAGroupsW];
#pragma unroll
        for (int i = 0; i < kAGroupsW; ++i) {
            const int r = (wave * kAGroupsW + i) * kRowsPerDma + lane / CHUNKS;
            rsrc[i] = g.perm_src[row0 + (r < rows ? r : 0)];
        }
#pragma unroll
        for (int i = 0; i < kAGroupsW; ++i) {
            const int r = (wave * kAGroupsW + i) * kRowsPerDma + lane / CHUNKS;
            const int64_t row = (int64_t)(min(max(rsrc[i], 0), g.Tk - 1) / g.k);
            soa[i] = (uint32_t)(row * g.K + ((lane % CHUNKS) ^ swz(r)) * 8);
        }
#pragma unroll
        for (int i = 0; i < kWGroupsW; ++i) {
            const int pr = (wave * kWGroupsW + i) * kRowsPerDma + lane / CHUNKS;   // 0..191
            const uint32_t off = (uint32_t)((int64_t)(pn * (BPW / 2) + pr) * g.K);
            sog[i] = off + ((lane % CHUNKS) ^ swz(BM + pr)) * 8;
            sou[i] = off + ((lane % CHUNKS) ^ swz(BM + BPW / 2 + pr)) * 8;
        }
    }
    static_assert(NSTAGE == 2, "the copy skip below assumes vmcnt(0) waits");
    auto issue = [&](int stage, int k0) {
        unsigned char* sb = lds + stage * STAGEBW;
#pragma unroll
        for (int i = 0; i < kAGroupsW; ++i) {
            const int grp = wave * kAGroupsW + i;
            if (grp * kRowsPerDma >= rows) continue;
            __builtin_amdgcn_global_load_lds((const void*)(g.A + (soa[i] + (uint32_t)k0)),
                                             (lds_void*)(sb + grp * 1024), 16, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < kWGroupsW; ++i) {
            const int grp = BM / kRowsPerDma + wave * kWGroupsW + i;
            __builtin_amdgcn_global_load_lds((const void*)(wg + (sog[i] + (uint32_t)k0)),
                                             (lds_void*)(sb + grp * 1024), 16, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < kWGroupsW; ++i) {
            const int grp = (BM + BPW / 2) / kRowsPerDma + wave * kWGroupsW + i;
            __builtin_amdgcn_global_load_lds((const void*)(wu + (sou[i] + (uint32_t)k0)),
                                             (lds_void*)(sb + grp * 1024), 16, 0, 0);
        }
    };

    accv acc[MI][NJW];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJW; ++j)
#pragma unroll
            for (int v = 0; v < ACCN; ++v) acc[i][j][v] = 0.0f;

    const int lrow = lane % MT;
    const int sw = swz(lrow);
    const int grp = lane / MT;
    const int cperm = MT == 16 ? (((grp & 1) << 1) | (grp >> 1)) : grp;
    int kpos[NKS];
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
        kpos[ks] = lrow * ROWB + ((((MK / 8) * ks + cperm) ^ sw) << 4);
    const int a0 = (wr * WM) * ROWB;
    // panel row of fragment j: gate rows for j < NJW/2, the matching up rows after
    const int b0 = (BM + wc * (WNW / 2)) * ROWB;

    const int nk = g.K / BK;
    issue(0, 0);
    for (int kt = 0; kt < nk; ++kt) {
        wait_vmcnt<0>();
        __syncthreads();
        if (kt + 1 < nk) issue((kt + 1) % NSTAGE, (kt + 1) * BK);
        if (active) {
            const unsigned char* base = lds + (kt % NSTAGE) * STAGEBW;
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) {
                bf16x8 fa[MI], fb[2][2];
                auto read_pair = [&](int buf, int jp) {
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int j = 2 * jp + h;
                        const int prow = (j < NJW / 2 ? 0 : BPW / 2) + (j % (NJW / 2)) * MT;
                        fb[buf][h] = __builtin_bit_cast(bf16x8, *(const u32x4*)(base + b0 + prow * ROWB + kpos[ks]));
                    }
                };
#pragma unroll
                for (int i = 0; i < MI; ++i)
                    fa[i] = __builtin_bit_cast(bf16x8, *(const u32x4*)(base + a0 + i * MT * ROWB + kpos[ks]));
                read_pair(0, 0);
#pragma unroll
                for (int jp = 0; jp < NJW / 2; ++jp) {
                    if (jp + 1 < NJW / 2) read_pair((jp + 1) & 1, jp + 1);
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int h = 0; h < 2; ++h)
#pragma unroll
                        for (int i = 0; i < MI; ++i)
                            acc[i][2 * jp + h] = mfma_bf16(fb[jp & 1][h], fa[i], acc[i][2 * jp + h]);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
    }
    if (!active) return;
    // H = silu(gate) * up straight from registers (8-byte runs)
    const int ncol0 = 4 * (lane / MT);
#pragma unroll
    for (int i = 0; i < MI; ++i) {
        const int r = wr * WM + i * MT + (lane % MT);
        if (r >= rows) continue;
        bf16_t* orow = g.out + ((int64_t)row0 + r) * g.n_out;
#pragma unroll
        for (int j = 0; j < NJW / 2; ++j) {
            const int col = pn * (BPW / 2) + wc * (WNW / 2) + j * MT + ncol0;
            uint32_t w[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const float h0 = silu_f(acc[i][j][2 * h]) * acc[i][j + NJW / 2][2 * h];
                const float h1 = silu_f(acc[i][j][2 * h + 1]) * acc[i][j + NJW / 2][2 * h + 1];
                w[h] = (uint32_t)f32_to_bf16(h0) | ((uint32_t)f32_to_bf16(h1) << 16);
            }
            *(uint2*)(orow + col) = make_uint2(w[0], w[1]);
        }
    }
}

}  // namespace

bool mfma_shape_ok(const pr2_moe_desc& d) {
    // copy offsets are 32-bit element offsets from the tensor (or expert) base
    const int64_t lim = (int64_t)1 << 31;
    const int64_t Tk = d.T * (int64_t)d.k;
    return d.act_dtype == PR2_BF16 && d.d % BP == 0 && d.m % 128 == 0 && d.d % BK == 0 &&
           d.m % BK == 0 && d.T * (int64_t)d.d < lim && Tk * d.m < lim &&
           (int64_t)d.m * d.d < lim;
}

hipError_t launch_expert_gemms(const pr2_moe_desc& d, const void* x, const void* W_gate,
                               const void* W_up, const void* W_down, const float* gate,
                               const ReplayWs& ws, hipStream_t s, void* au_out) {
    if (mfma_shape_ok(d)) {
        MfmaArgs g1{};
        g1.A = (const bf16_t*)x;
        g1.perm_src = ws.perm_src;
        g1.k = d.k;
        g1.Tk = (int)(d.T * d.k);
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
        g1.group = kGroupGemm1;
        int64_t work = ws.max_tiles * g1.ntn;
        int64_t grid = ((work + kNumXcd - 1) / kNumXcd) * kNumXcd;
        if (!au_out && d.m % (BPW / 2) == 0) {
            // the 384-row panel: m / 192 panels per tile
            g1.ntn = d.m / (BPW / 2);
            const int64_t wide = ws.max_tiles * g1.ntn;
            const int64_t wgrid = ((wide + kNumXcd - 1) / kNumXcd) * kNumXcd;
            LaunchScope scope("gemm1_gate_up_swiglu", s);
            hipLaunchKernelGGL(gemm1_wide, dim3((unsigned)wgrid), dim3(kGemmThreads), 0, s, g1);
            g1.ntn = d.m / 128;
        } else if (au_out) {
            g1.out2 = (bf16_t*)au_out;
            LaunchScope scope("gemm1_gate_up_swiglu_save", s);
            hipLaunchKernelGGL(grouped_gemm_mfma<3>, dim3((unsigned)grid), dim3(kGemmThreads), 0,
                               s, g1);
        } else {
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
        g2.group = kGroupGemm2;
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
    if (au_out) {
        hipError_t e = launch_preact(d, x, W_gate, W_up, ws, au_out, s);
        if (e != hipSuccess) return e;
    }
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

hipError_t launch_preact(const pr2_moe_desc& d, const void* x, const void* W_gate,
                         const void* W_up, const ReplayWs& ws, void* AU, hipStream_t s) {
    if (mfma_shape_ok(d)) {
        MfmaArgs g{};
        g.A = (const bf16_t*)x;
        g.perm_src = ws.perm_src;
        g.k = d.k;
        g.Tk = (int)(d.T * d.k);
        g.W0 = (const bf16_t*)W_gate;
        g.W1 = (const bf16_t*)W_up;
        g.K = d.d;
        g.n_out = 2 * d.m;
        g.ntn = d.m / 128;
        g.w_stride = (int64_t)d.m * d.d;
        g.tiles = ws.tiles;
        g.tile_count = ws.tile_count;
        g.out = (bf16_t*)AU;
        g.group = kGroupGemm1;
        const int64_t work = ws.max_tiles * g.ntn;
        const int64_t grid = ((work + kNumXcd - 1) / kNumXcd) * kNumXcd;
        LaunchScope scope("bwd_preact_gate_up", s);
        hipLaunchKernelGGL(grouped_gemm_mfma<2>, dim3((unsigned)grid), dim3(kGemmThreads), 0, s, g);
        return hipGetLastError();
    }
    dim3 grid((unsigned)ws.max_tiles, (unsigned)d.m);
    LaunchScope scope("bwd_preact_generic", s);
    if (d.act_dtype == PR2_BF16)
        hipLaunchKernelGGL(preact_generic<bf16_t>, grid, dim3(256), 0, s, (const bf16_t*)x,
                           ws.perm_src, d.k, (const bf16_t*)W_gate, (const bf16_t*)W_up, d.d, d.m,
                           ws.tiles, ws.tile_count, (bf16_t*)AU);
    else
        hipLaunchKernelGGL(preact_generic<float>, grid, dim3(256), 0, s, (const float*)x,
                           ws.perm_src, d.k, (const float*)W_gate, (const float*)W_up, d.d, d.m,
                           ws.tiles, ws.tile_count, (float*)AU);
    return hipGetLastError();
}

}  // namespace pr2
