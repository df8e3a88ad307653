// Token permutation for the grouped expert GEMMs, and the combine.
//
// The recorded route of T tokens is a list of T*k (token, slot) entries.  They
// are sorted by expert, stably in (token, slot) order, in three launches:
//   count   one block per chunk of <= 512 consecutive entries counts its
//           entries per expert (LDS integer atomics) -> counts[e][block];
//   scan    one block turns the expert-major counts into the exclusive prefix
//           over (expert, block), which is each block's first output position
//           per expert; it also writes the expert offsets and the tile list
//           (expert, first row, rows) of kTileM-row (256) grouped-GEMM tiles;
//   scatter one wavefront per chunk walks its entries 64 at a time; lanes with
//           the same expert find each other with ballots over the id bits, so
//           each entry's position is its block base + the entries of the same
//           expert before it.  perm_src[pos] = t*k + s, inv[t*k + s] = pos.
// Out-of-range ids are not dispatched (inv = -1); the count pass is the one
// place that counts them (in the workspace's error words).  The replay forward
// and backward form the counts in their replay-weight pass instead, where that
// pass's workgroups cover whole count blocks (it also counts those ids then).
//
// Combine: y_t = sum over slots s (in slot order) of the weighted expert output
// row O[inv[t*k + s]], accumulated in fp32 (Eq. pr2_output).
#include "common.h"

namespace pr2 {
namespace {

__global__ void __launch_bounds__(64)
perm_count_kernel(const void* idx, int idx_dtype, int64_t ldi, int64_t T, int k, int N,
                  int tb, int64_t nblk, int* counts, int* err) {
    extern __shared__ int cnt[];
    const int lane = threadIdx.x;
    const int64_t b = blockIdx.x;
    for (int e = lane; e < N; e += 64) cnt[e] = 0;
    __syncthreads();
    const int64_t t0 = b * tb;
    const int64_t tend = t0 + tb < T ? t0 + tb : T;
    const int entries = (int)((tend - t0) * k);
    int bad = 0;
    for (int q = lane; q < entries; q += 64) {
        int64_t t = t0 + q / k;
        int s = q % k;
        int e = load_id(idx, idx_dtype, t * ldi + s);
        if (e >= 0 && e < N) atomicAdd(&cnt[e], 1);
        else bad++;
    }
    __syncthreads();
    for (int e = lane; e < N; e += 64) counts[(int64_t)e * nblk + b] = cnt[e];
    for (int off = 32; off >= 1; off >>= 1) bad += __shfl_xor(bad, off, 64);
    if (lane == 0 && bad) atomicAdd(err + ERR_BAD_ID, bad);
}

constexpr int kScanThreads = 1024;

// inclusive prefix sum across the 64 lanes of a wavefront: row_shr 1, 2, 4, 8
// within rows of 16 lanes, then row_bcast 15 and 31 carry the row totals
__device__ __forceinline__ int wave_incl_scan(int x) {
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);
    return x;
}

// Exclusive prefix sum over the workgroup's threads: a DPP scan inside each
// wavefront, then one scan of the wavefront totals (three barriers).  sh needs
// kScanThreads / 64 + 1 ints.
__device__ int block_exclusive_scan(int v, int* sh, int* total) {
    constexpr int kWaves = kScanThreads / 64;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int incl = wave_incl_scan(v);
    if (lane == 63) sh[wave] = incl;
    __syncthreads();
    if (wave == 0) {
        const int w = lane < kWaves ? sh[lane] : 0;
        const int wi = wave_incl_scan(w);
        if (lane < kWaves) sh[lane] = wi - w;
        if (lane == kWaves - 1) sh[kWaves] = wi;
    }
    __syncthreads();
    const int res = sh[wave] + incl - v;
    *total = sh[kWaves];
    __syncthreads();
    return res;
}

// counts: [N * nblk] expert-major; rewritten in place with each block's first
// output position per expert.  One wavefront per expert scans that expert's
// block counts (coalesced, 64 blocks per step); the expert totals are then
// scanned across experts and added back in a second coalesced pass.
__global__ void __launch_bounds__(kScanThreads)
perm_scan_kernel(int* counts, int64_t nblk, int N, int bm, int* offsets, int* tiles,
                 int* tile_count) {
    __shared__ int sh[kScanThreads];
    __shared__ int s_off[kMaxExperts + 1];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    constexpr int kWaves = kScanThreads / 64;
    constexpr int kScanE = 8, kScanC = 8;
    int grand;
    if (N <= kWaves * kScanE && nblk <= 64 * kScanC) {
        // Register-resident path: wavefront w owns experts w, w+16, ...; lane l
        // owns blocks [l*P, l*P + P) of each, so one wavefront scan per expert
        // turns the lanes' totals into their starting offsets.
        const int P = ((int)nblk + 63) / 64;
        // a lane's P block counts are consecutive: when they are 4 or 8
        // 16-byte aligned ints (nblk a multiple of 256 or 512) they move as
        // 16-byte vectors, 8x fewer memory instructions through this one CU
        const bool vec = (P == 4 || P == 8) && nblk == 64 * P;
        int v[kScanE][kScanC];
        int tot[kScanE];
#pragma unroll
        for (int i = 0; i < kScanE; ++i) {
            const int e = wave + kWaves * i;
            if (vec) {
#pragma unroll
                for (int c4 = 0; c4 < kScanC; c4 += 4) {
                    int4 q = make_int4(0, 0, 0, 0);
                    if (e < N && c4 < P) q = *(const int4*)(counts + (int64_t)e * nblk + lane * P + c4);
                    v[i][c4] = q.x; v[i][c4 + 1] = q.y; v[i][c4 + 2] = q.z; v[i][c4 + 3] = q.w;
                }
                continue;
            }
#pragma unroll
            for (int c = 0; c < kScanC; ++c) {
                const int b = lane * P + c;
                const bool ok = e < N && c < P && b < (int)nblk;
                const int val = counts[ok ? (int64_t)e * nblk + b : 0];
                v[i][c] = ok ? val : 0;
            }
        }
#pragma unroll
        for (int i = 0; i < kScanE; ++i) {
            int run = 0;
#pragma unroll
            for (int c = 0; c < kScanC; ++c) {
                const int x = v[i][c];
                v[i][c] = run;                          // exclusive within the lane
                run += x;
            }
            const int incl = wave_incl_scan(run);
            const int lane_start = incl - run;
#pragma unroll
            for (int c = 0; c < kScanC; ++c) v[i][c] += lane_start;
            tot[i] = __shfl(incl, 63, 64);
        }
        if (lane == 0)
#pragma unroll
            for (int i = 0; i < kScanE; ++i)
                if (wave + kWaves * i < N) s_off[wave + kWaves * i] = tot[i];
        __syncthreads();
        const int t = tid < N ? s_off[tid] : 0;
        const int ex = block_exclusive_scan(t, sh, &grand);
        if (tid < N) s_off[tid] = ex;
        if (tid == 0) s_off[N] = grand;
        __syncthreads();
#pragma unroll
        for (int i = 0; i < kScanE; ++i) {
            const int e = wave + kWaves * i;
            if (e >= N) continue;
            const int add = s_off[e];
            if (vec) {
#pragma unroll
                for (int c4 = 0; c4 < kScanC; c4 += 4)
                    if (c4 < P)
                        *(int4*)(counts + (int64_t)e * nblk + lane * P + c4) =
                            make_int4(v[i][c4] + add, v[i][c4 + 1] + add, v[i][c4 + 2] + add, v[i][c4 + 3] + add);
                continue;
            }
#pragma unroll
            for (int c = 0; c < kScanC; ++c) {
                const int b = lane * P + c;
                if (c < P && b < (int)nblk) counts[(int64_t)e * nblk + b] = v[i][c] + add;
            }
        }
    } else {
        // general path: experts in batches, block counts in chunks, in place
        for (int e = wave; e < N; e += kWaves) {
            int* row = counts + (int64_t)e * nblk;
            int carry = 0;
            for (int b0 = 0; b0 < (int)nblk; b0 += 64) {
                const int b = b0 + lane;
                const int c = b < (int)nblk ? row[b] : 0;
                int incl = c;
#pragma unroll
                for (int off = 1; off < 64; off <<= 1) {
                    int y = __shfl_up(incl, off, 64);
                    if (lane >= off) incl += y;
                }
                if (b < (int)nblk) row[b] = carry + incl - c;
                carry += __shfl(incl, 63, 64);
            }
            if (lane == 0) s_off[e] = carry;
        }
        __syncthreads();
        for (int e0 = 0; e0 < N; e0 += kScanThreads) {
            // N <= kMaxExperts == kScanThreads: one round
            const int t = e0 + tid < N ? s_off[e0 + tid] : 0;
            const int ex = block_exclusive_scan(t, sh, &grand);
            if (e0 + tid < N) s_off[e0 + tid] = ex;
        }
        if (tid == 0) s_off[N] = grand;
        __syncthreads();
        for (int e = wave; e < N; e += kWaves) {
            int* row = counts + (int64_t)e * nblk;
            const int add = s_off[e];
            for (int b = lane; b < (int)nblk; b += 64) row[b] += add;
        }
    }
    // tiles per expert, and their exclusive prefix
    int ntile = 0;
    if (tid < N) {
        int n_e = s_off[tid + 1] - s_off[tid];
        ntile = (n_e + bm - 1) / bm;
    }
    int ntot;
    int tstart = block_exclusive_scan(ntile, sh, &ntot);
    if (tid < N) {
        int base = s_off[tid];
        int n_e = s_off[tid + 1] - base;
        for (int j = 0; j < ntile; ++j) {
            int rows = n_e - j * bm;
            tiles[3 * (tstart + j) + 0] = tid;
            tiles[3 * (tstart + j) + 1] = base + j * bm;
            tiles[3 * (tstart + j) + 2] = rows < bm ? rows : bm;
        }
    }
    for (int e = tid; e <= N; e += kScanThreads) offsets[e] = s_off[e];
    if (tid == 0) *tile_count = ntot;
}

__global__ void __launch_bounds__(64)
perm_scatter_kernel(const void* idx, int idx_dtype, int64_t ldi, int64_t T, int k, int N,
                    int tb, int64_t nblk, const int* bases, int* perm_src, int* inv) {
    extern __shared__ int cnt[];
    const int lane = threadIdx.x;
    const int64_t b = blockIdx.x;
    for (int e = lane; e < N; e += 64) cnt[e] = bases[(int64_t)e * nblk + b];
    __syncthreads();
    int nbits = 0;
    while ((1 << nbits) < N) ++nbits;
    const int64_t t0 = b * tb;
    const int64_t tend = t0 + tb < T ? t0 + tb : T;
    const int entries = (int)((tend - t0) * k);
    const uint64_t lt = lane ? ((~0ull) >> (64 - lane)) : 0ull;
    // the ids of up to kPrefetch passes are loaded before the first pass, so
    // the passes (each ending in a barrier) do not wait on global loads
    constexpr int kPrefetch = kEntriesPerPermBlock / 64;
    int pre[kPrefetch];
#pragma unroll
    for (int i = 0; i < kPrefetch; ++i) {
        const int q = i * 64 + lane;
        pre[i] = q < entries ? load_id(idx, idx_dtype, (t0 + q / k) * ldi + q % k) : -1;
    }
    for (int q0 = 0; q0 < entries; q0 += 64) {
        const int q = q0 + lane;
        int e = -1;
        int64_t src = 0;
        if (q < entries) {
            int64_t t = t0 + q / k;
            int s = q % k;
            src = t * k + s;
            int pe = pre[0];
#pragma unroll
            for (int i = 1; i < kPrefetch; ++i)
                if (q0 == i * 64) pe = pre[i];
            e = q0 < kPrefetch * 64 ? pe : load_id(idx, idx_dtype, t * ldi + s);
            if (e < 0 || e >= N) {
                inv[src] = -1;
                e = -1;
            }
        }
        const bool valid = e >= 0;
        uint64_t peers = __ballot(valid);
        for (int bit = 0; bit < nbits; ++bit) {
            uint64_t ones = __ballot(valid && ((e >> bit) & 1));
            peers &= ((e >> bit) & 1) ? ones : ~ones;
        }
        if (valid) {
            int base = cnt[e];
            int pos = base + __popcll(peers & lt);
            if (pos < T * k) {                 // always true for a consistent scan
                perm_src[pos] = (int)src;
                inv[src] = pos;
            } else {
                inv[src] = -1;
            }
            // the highest lane of each peer group advances the expert's cursor
            if ((peers >> lane) == 1ull) cnt[e] = base + __popcll(peers);
        }
        __syncthreads();
    }
}

// bf16, d % 8 == 0: each thread owns 8 consecutive columns of kCombTok tokens
// per iteration and issues the loads of kCombSlots route slots of each before
// summing them, so up to kCombTok * kCombSlots 16-byte loads are in flight
constexpr int kCombTok = 2;
constexpr int kCombSlots = 8;   // route slots whose loads are in flight together
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(256)
combine_bf16_kernel(const bf16_t* O, const int* inv, int64_t ntok, int k, int d, bf16_t* y) {
    const int64_t step = (int64_t)gridDim.x * kCombTok;
    for (int64_t t0 = (int64_t)blockIdx.x * kCombTok; t0 < ntok; t0 += step) {
        for (int c0 = threadIdx.x * 8; c0 < d; c0 += 256 * 8) {
            float acc[kCombTok][8];
#pragma unroll
            for (int u = 0; u < kCombTok; ++u)
#pragma unroll
                for (int v = 0; v < 8; ++v) acc[u][v] = 0.0f;
            // slots in groups of kCombSlots: all their row indices, then all
            // their loads are issued before the first is consumed; the sum
            // still runs in slot order
            for (int s0 = 0; s0 < k; s0 += kCombSlots) {
                int r[kCombTok][kCombSlots];
#pragma unroll
                for (int u = 0; u < kCombTok; ++u)
#pragma unroll
                    for (int j = 0; j < kCombSlots; ++j) {
                        const int64_t t = t0 + u;
                        r[u][j] = (t < ntok && s0 + j < k) ? inv[t * k + s0 + j] : -1;
                    }
                u32x4 raw[kCombTok][kCombSlots];
#pragma unroll
                for (int u = 0; u < kCombTok; ++u)
#pragma unroll
                    for (int j = 0; j < kCombSlots; ++j)
                        raw[u][j] = r[u][j] >= 0
                            ? __builtin_nontemporal_load((const u32x4*)(O + (int64_t)r[u][j] * d + c0))
                            : u32x4{0, 0, 0, 0};
#pragma unroll
                for (int j = 0; j < kCombSlots; ++j)
#pragma unroll
                    for (int u = 0; u < kCombTok; ++u) {
                        if (r[u][j] < 0) continue;
                        const uint32_t w[4] = {raw[u][j][0], raw[u][j][1], raw[u][j][2], raw[u][j][3]};
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            acc[u][2 * v] += __uint_as_float(w[v] << 16);
                            acc[u][2 * v + 1] += __uint_as_float(w[v] & 0xffff0000u);
                        }
                    }
            }
#pragma unroll
            for (int u = 0; u < kCombTok; ++u) {
                const int64_t t = t0 + u;
                if (t >= ntok) continue;
                uint32_t w[4];
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    w[v] = (uint32_t)f32_to_bf16(acc[u][2 * v]) |
                           ((uint32_t)f32_to_bf16(acc[u][2 * v + 1]) << 16);
                *(uint4*)(y + t * (int64_t)d + c0) = make_uint4(w[0], w[1], w[2], w[3]);
            }
        }
    }
}

template <typename T>
__global__ void __launch_bounds__(256)
combine_kernel(const T* O, const int* inv, int64_t ntok, int k, int d, T* y) {
    for (int64_t t = blockIdx.x; t < ntok; t += gridDim.x) {
        for (int c = threadIdx.x; c < d; c += 256) {
            float acc = 0.0f;
            for (int s = 0; s < k; ++s) {
                int r = inv[t * k + s];
                if (r >= 0) acc += Act<T>::to_f32(O[(int64_t)r * d + c]);
            }
            y[t * (int64_t)d + c] = Act<T>::from_f32(acc);
        }
    }
}

}  // namespace

hipError_t launch_permute(const pr2_moe_desc& d, const void* idx, int64_t ldi, const ReplayWs& ws,
                          hipStream_t s, bool counted) {
    const int tb = perm_tokens_per_block(d.k);
    const size_t sm = sizeof(int) * (size_t)d.N;
    if (!counted) {
        LaunchScope scope("perm_count", s);
        hipLaunchKernelGGL(perm_count_kernel, dim3((unsigned)ws.nblk), dim3(64), sm, s, idx,
                           d.idx_dtype, ldi, d.T, d.k, d.N, tb, ws.nblk, ws.bcount, ws.err);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    {
        LaunchScope scope("perm_scan", s);
        hipLaunchKernelGGL(perm_scan_kernel, dim3(1), dim3(kScanThreads), 0, s, ws.bcount,
                           ws.nblk, d.N, kTileM, ws.offsets, ws.tiles, ws.tile_count);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    {
        LaunchScope scope("perm_scatter", s);
        hipLaunchKernelGGL(perm_scatter_kernel, dim3((unsigned)ws.nblk), dim3(64), sm, s, idx,
                           d.idx_dtype, ldi, d.T, d.k, d.N, tb, ws.nblk, ws.bcount, ws.perm_src,
                           ws.inv);
    }
    return hipGetLastError();
}

namespace {
__global__ void __launch_bounds__(64) zero_i32_kernel(int* p, int n) {
    for (int i = threadIdx.x; i < n; i += 64) p[i] = 0;
}
}  // namespace

// A fill kernel rather than hipMemsetAsync, so that a captured HIP graph holds
// no memset node.
hipError_t launch_zero_i32(int* p, int n, hipStream_t s) {
    hipLaunchKernelGGL(zero_i32_kernel, dim3(1), dim3(64), 0, s, p, n);
    return hipGetLastError();
}

hipError_t launch_combine(const pr2_moe_desc& d, const ReplayWs& ws, void* y, hipStream_t s) {
    LaunchScope scope("combine", s);
    if (d.act_dtype == PR2_BF16 && d.d % 8 == 0) {
        const int64_t want = (d.T + kCombTok - 1) / kCombTok;
        dim3 grid((unsigned)(want < 8192 ? want : 8192));
        hipLaunchKernelGGL(combine_bf16_kernel, grid, dim3(256), 0, s, (const bf16_t*)ws.O, ws.inv,
                           d.T, d.k, d.d, (bf16_t*)y);
    } else {
        dim3 grid((unsigned)(d.T < 8192 ? d.T : 8192));
        if (d.act_dtype == PR2_BF16)
            hipLaunchKernelGGL(combine_kernel<bf16_t>, grid, dim3(256), 0, s, (const bf16_t*)ws.O,
                               ws.inv, d.T, d.k, d.d, (bf16_t*)y);
        else
            hipLaunchKernelGGL(combine_kernel<float>, grid, dim3(256), 0, s, (const float*)ws.O,
                               ws.inv, d.T, d.k, d.d, (float*)y);
    }
    return hipGetLastError();
}

}  // namespace pr2
