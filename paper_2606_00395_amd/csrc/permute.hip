// Token permutation for the grouped expert GEMMs, and the combine.
//
// The recorded route of T tokens is a list of T*k (token, slot) entries.  They
// are sorted by expert, stably in (token, slot) order, in three launches:
//   count   one block per chunk of <= 512 consecutive entries counts its
//           entries per expert (LDS integer atomics) -> counts[e][block];
//   scan    one block turns the expert-major counts into the exclusive prefix
//           over (expert, block), which is each block's first output position
//           per expert; it also writes the expert offsets and the tile list
//           (expert, first row, rows) of 128-row grouped-GEMM tiles;
//   scatter one wavefront per chunk walks its entries 64 at a time; lanes with
//           the same expert find each other with ballots over the id bits, so
//           each entry's position is its block base + the entries of the same
//           expert before it.  perm_src[pos] = t*k + s, inv[t*k + s] = pos.
// Out-of-range ids are not dispatched (inv = -1) and are counted.
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

__device__ int block_exclusive_scan(int v, int* sh, int* total) {
    const int tid = threadIdx.x;
    sh[tid] = v;
    __syncthreads();
    for (int off = 1; off < kScanThreads; off <<= 1) {
        int add = tid >= off ? sh[tid - off] : 0;
        __syncthreads();
        sh[tid] += add;
        __syncthreads();
    }
    int incl = sh[tid];
    *total = sh[kScanThreads - 1];
    __syncthreads();
    return incl - v;
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
    for (int e = wave; e < N; e += kScanThreads / 64) {
        int* row = counts + (int64_t)e * nblk;
        int carry = 0;
        for (int64_t b0 = 0; b0 < nblk; b0 += 64) {
            const int64_t b = b0 + lane;
            const int c = b < nblk ? row[b] : 0;
            int incl = c;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                int y = __shfl_up(incl, off, 64);
                if (lane >= off) incl += y;
            }
            if (b < nblk) row[b] = carry + incl - c;
            carry += __shfl(incl, 63, 64);
        }
        if (lane == 0) s_off[e] = carry;
    }
    __syncthreads();
    int grand;
    const int tot = tid < N ? s_off[tid] : 0;
    const int ex = block_exclusive_scan(tot, sh, &grand);
    if (tid < N) s_off[tid] = ex;
    if (tid == 0) s_off[N] = grand;
    __syncthreads();
    const int64_t L = (int64_t)N * nblk;
    for (int64_t q = tid; q < L; q += kScanThreads) counts[q] += s_off[q / nblk];
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
    for (int q0 = 0; q0 < entries; q0 += 64) {
        const int q = q0 + lane;
        int e = -1;
        int64_t src = 0;
        if (q < entries) {
            int64_t t = t0 + q / k;
            int s = q % k;
            src = t * k + s;
            e = load_id(idx, idx_dtype, t * ldi + s);
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
            perm_src[pos] = (int)src;
            inv[src] = pos;
            // the highest lane of each peer group advances the expert's cursor
            if ((peers >> lane) == 1ull) cnt[e] = base + __popcll(peers);
        }
        __syncthreads();
    }
}

template <typename T, int V>
__global__ void __launch_bounds__(256)
combine_kernel(const T* O, const int* inv, int64_t ntok, int k, int d, T* y) {
    for (int64_t t = blockIdx.x; t < ntok; t += gridDim.x) {
        for (int c0 = threadIdx.x * V; c0 < d; c0 += 256 * V) {
            float acc[V];
#pragma unroll
            for (int v = 0; v < V; ++v) acc[v] = 0.0f;
            for (int s = 0; s < k; ++s) {
                int r = inv[t * k + s];
                if (r < 0) continue;
                const T* src = O + (int64_t)r * d + c0;
                if (V == 8 && sizeof(T) == 2) {
                    uint4 u = *(const uint4*)src;
                    uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        acc[2 * v] += __uint_as_float(w[v] << 16);
                        acc[2 * v + 1] += __uint_as_float(w[v] & 0xffff0000u);
                    }
                } else {
#pragma unroll
                    for (int v = 0; v < V; ++v)
                        if (c0 + v < d) acc[v] += Act<T>::to_f32(src[v]);
                }
            }
            T* dst = y + t * (int64_t)d + c0;
            if (V == 8 && sizeof(T) == 2) {
                uint32_t w[4];
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    w[v] = (uint32_t)f32_to_bf16(acc[2 * v]) |
                           ((uint32_t)f32_to_bf16(acc[2 * v + 1]) << 16);
                *(uint4*)dst = make_uint4(w[0], w[1], w[2], w[3]);
            } else {
#pragma unroll
                for (int v = 0; v < V; ++v)
                    if (c0 + v < d) dst[v] = Act<T>::from_f32(acc[v]);
            }
        }
    }
}

}  // namespace

hipError_t launch_permute(const pr2_moe_desc& d, const void* idx, int64_t ldi, const ReplayWs& ws,
                          hipStream_t s) {
    const int tb = perm_tokens_per_block(d.k);
    const size_t sm = sizeof(int) * (size_t)d.N;
    {
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

hipError_t launch_combine(const pr2_moe_desc& d, const ReplayWs& ws, void* y, hipStream_t s) {
    const int64_t grid64 = d.T < 8192 ? d.T : 8192;
    dim3 grid((unsigned)grid64);
    LaunchScope scope("combine", s);
    if (d.act_dtype == PR2_BF16) {
        if (d.d % 8 == 0)
            hipLaunchKernelGGL((combine_kernel<bf16_t, 8>), grid, dim3(256), 0, s,
                               (const bf16_t*)ws.O, ws.inv, d.T, d.k, d.d, (bf16_t*)y);
        else
            hipLaunchKernelGGL((combine_kernel<bf16_t, 1>), grid, dim3(256), 0, s,
                               (const bf16_t*)ws.O, ws.inv, d.T, d.k, d.d, (bf16_t*)y);
    } else {
        hipLaunchKernelGGL((combine_kernel<float, 1>), grid, dim3(256), 0, s, (const float*)ws.O,
                           ws.inv, d.T, d.k, d.d, (float*)y);
    }
    return hipGetLastError();
}

}  // namespace pr2
