// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "../../include/pr2.h"

namespace pr2 {

// ---------------------------------------------------------------- bf16 ----
typedef uint16_t bf16_t;                    // storage of one bf16 value
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf16_to_f32(bf16_t v) {
    return __uint_as_float(((uint32_t)v) << 16);
}

// round to nearest even, NaN stays a (quiet) NaN: gfx950's v_cvt_pk_bf16_f32,
// which gives bitwise the integer rounding u + 0x7fff + ((u >> 16) & 1) for
// every non-NaN pattern and sets the quiet bit of NaNs
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
    return __builtin_bit_cast(bf16_t, (__bf16)f);
}

template <typename T> struct Act;
template <> struct Act<float> {
    __device__ __forceinline__ static float load(const float* p) { return *p; }
    __device__ __forceinline__ static float to_f32(float v) { return v; }
    __device__ __forceinline__ static float from_f32(float v) { return v; }
};
template <> struct Act<bf16_t> {
    __device__ __forceinline__ static float load(const bf16_t* p) { return bf16_to_f32(*p); }
    __device__ __forceinline__ static float to_f32(bf16_t v) { return bf16_to_f32(v); }
    __device__ __forceinline__ static bf16_t from_f32(float v) { return f32_to_bf16(v); }
};

__device__ __forceinline__ int load_id(const void* idx, int idx_dtype, int64_t pos) {
    return idx_dtype == PR2_I16 ? (int)((const int16_t*)idx)[pos] : ((const int32_t*)idx)[pos];
}

// ------------------------------------------------------------ limits -----
constexpr int kMaxExperts = 1024;
constexpr int kEntriesPerPermBlock = 512;   // (token, slot) entries per permutation block
constexpr int kTileM = 256;                 // rows per grouped-GEMM tile (tile list granularity)

inline int perm_tokens_per_block(int k) {
    int tb = kEntriesPerPermBlock / k;
    return tb < 1 ? 1 : tb;
}

// error-word slots in the workspace
enum { ERR_BAD_ID = 0, ERR_DUP_ID = 1, ERR_WORDS = 4 };

// ----------------------------------------------------------- workspace ----
struct ReplayWs {
    float* gate;        // [T*k] (used when the caller passes no gate_out)
    int* err;           // [ERR_WORDS]
    int* bcount;        // [nblk*N]  per-block counts, then per-block bases
    int* offsets;       // [N+1]
    int* tile_count;    // [1]
    int* tiles;         // [max_tiles*3]: expert, first permuted row, rows
    int* perm_src;      // [T*k] permuted row -> t*k + s
    int* inv;           // [T*k] t*k + s -> permuted row (or -1)
    void* H;            // [T*k, m] act
    void* O;            // [T*k, d] act
    void* wsplit;       // router weight split (bf16 x 3)
    int64_t nblk;
    int64_t max_tiles;
    size_t bytes;
};

ReplayWs replay_ws_layout(const pr2_moe_desc& d, void* base);

// the replay segments followed by the backward pass's own
struct BwdWs {
    ReplayWs fw;        // fw.H holds g*H, fw.O the per-route input gradients
    void* AU;           // [T*k, 2m] act: pre-activations a | u, then their gradients
    float* dgp;         // [T*k, np] partial gate gradients
    float* dp_route;    // [T*k] router-logit gradient per (token, slot)
    float* dp_perm;     // [T*k] the same in permuted order
    float* wrt;         // [N, d] W_r transposed
    int* order;         // [N] experts by decreasing route count
    float* rwpart;      // [max_tiles, d] router weight-gradient partials per 256-row tile
    float* rbpart;      // [max_tiles] router bias-gradient partials
    // paper-literal weights (renorm = 0) only: the router gradient is dense over N
    float* plog;        // [T, N] current router logits
    float* dpf;         // [T, N] router-logit gradient
    float* lwpart;      // [nchunk, d, N] dW_r partials per chunk of 1024 tokens
    float* lbpart;      // [nchunk, N] db_r partials
    int nchunk;
    int np;
    size_t bytes;
};

BwdWs bwd_ws_layout(const pr2_moe_desc& d, void* base);

// ------------------------------------------------- host helpers (api.hip) ----
// fail() records a sentence for pr2_last_error and returns s; ok() clears it.
pr2_status fail(pr2_status s, const char* fmt, ...);
pr2_status ok();
pr2_status hip_fail(hipError_t e, const char* what);
// the current device is usable and is a gfx950
pr2_status device_ready();
// argument checks shared by the route calls; *empty is set for T == 0 (a no-op)
pr2_status check_route_args(const pr2_moe_desc* desc, const void* x, const float* W_r,
                            const float* b_r, const float* A, const float* B, void* idx_out,
                            int64_t ldi, float* gate_out, float* logits_out, bool* empty);

// ------------------------------------------------------------ launches ----
// Every launch goes through this so that measurement events can bracket it.
struct LaunchScope {
    LaunchScope(const char* name, hipStream_t s);
    ~LaunchScope();
    const char* name;
    hipStream_t stream;
    int slot;
};

// Route-recording features of the retained tokens (feature cache): token t with
// row[t] in [0, rows) writes its hidden state to h[row[t]] and its router logits
// to p[row[t]].
struct FeatureCache {
    const int* row;     // [T] or null (no feature cache)
    void* h;            // [rows, d] act
    float* p;           // [rows, N]
    int64_t rows;
};

// router.hip
// Scratch for the bf16 three-way split of [W_r | A] used by the MFMA router
// (0 when the shape takes the fp64 vector path).
// router scratch: the split weights and, for small token counts, the split-K
// pair sums and logits
size_t router_split_bytes(int NC, const pr2_moe_desc& d);
// the split weights alone (what the fused, non-split-K router reads)
size_t router_split_weight_bytes(int NC, const pr2_moe_desc& d);
bool router_mfma_ok(const pr2_moe_desc& d, int NC);
// splitk_ok = false keeps every batch size on the fused kernel (same logits
// bit for bit), so split_ws needs only router_split_weight_bytes
hipError_t launch_route_predict(const pr2_moe_desc& d, const void* x, const float* W_r,
                                const float* b_r, const float* A, const float* B, void* idx_out,
                                int64_t ldi, float* gate_out, float* logits_out, void* split_ws,
                                hipStream_t s, const FeatureCache& cache = FeatureCache{},
                                bool reuse_split = false, bool splitk_ok = true,
                                int* counts = nullptr, bool* counted = nullptr);
// (counts, counted: as launch_replay_gates' counts, for the ids this call
// selects; *counted says whether the kernel path taken wrote them)
// current router logits p = x W_r + b_r of every token into p_out [T, N]
hipError_t launch_router_logits(const pr2_moe_desc& d, const void* x, const float* W_r,
                                const float* b_r, float* p_out, void* split_ws, hipStream_t s);
// Route-tracking diagnostics a replay-weight pass can form from the same logits
// (current top-k, overlap with the recorded ids, route KL against z_ref, the
// deviation histogram); any field may be null.
struct RouteDiag {
    const float* z_ref;         // [T, N] reference logits (needed by kl)
    void* cur_idx;              // [T, k] idx_dtype
    int* overlap;               // [T]
    float* kl;                  // [T]
    unsigned long long* hist;   // [k + 1], zeroed by the launch
    float* p_out;               // [T, N] the current logits p
};
// counts (or null): also write the permutation's per-block expert counts
// ([N][nblk], blocks of perm_tokens_per_block(k) tokens) and count the
// out-of-range ids, as the permutation's count pass does; only where
// replay_counts_fused(d) holds
hipError_t launch_replay_gates(const pr2_moe_desc& d, const void* x, const void* idx, int64_t ldi,
                               const float* W_r, const float* b_r, float* gate_out, int* err,
                               void* split_ws, hipStream_t s, const RouteDiag* diag = nullptr,
                               int* counts = nullptr);
// whether the replay-weight pass can form the permutation's counts: the fused
// MFMA router (not its split-K form) with k in {8, 16, 32, 64}, whose count
// blocks (512 / k tokens) tile its 64-token workgroups
bool replay_counts_fused(const pr2_moe_desc& d);

hipError_t launch_route_diagnostics(const pr2_moe_desc& d, const void* x, const void* idx,
                                    int64_t ldi, const float* W_r, const float* b_r,
                                    const float* z_ref, void* cur_idx, int* overlap, float* kl,
                                    unsigned long long* hist, void* split_ws, hipStream_t s);

// permute.hip
// counted: the per-block counts and the out-of-range count are already in the
// workspace (written by the replay-weight pass)
hipError_t launch_permute(const pr2_moe_desc& d, const void* idx, int64_t ldi, const ReplayWs& ws,
                          hipStream_t s, bool counted = false);
hipError_t launch_combine(const pr2_moe_desc& d, const ReplayWs& ws, void* y, hipStream_t s);
// p[0..n) = 0 (one workgroup; for the few error words)
hipError_t launch_zero_i32(int* p, int n, hipStream_t s);

// gemm.hip
// au_out (or null): also store the pre-activations a | u of every permuted row,
// [T*k, 2m] act, as the backward's launch_preact forms them
hipError_t launch_expert_gemms(const pr2_moe_desc& d, const void* x, const void* W_gate,
                               const void* W_up, const void* W_down, const float* gate,
                               const ReplayWs& ws, hipStream_t s, void* au_out = nullptr);
bool mfma_shape_ok(const pr2_moe_desc& d);
hipError_t launch_preact(const pr2_moe_desc& d, const void* x, const void* W_gate,
                         const void* W_up, const ReplayWs& ws, void* AU, hipStream_t s);

// predictor.hip
struct PredLossWs {
    float* p_cur;       // [T, N] current router logits
    double* u;          // [T, r] h_old A
    double* dz;         // [T, N] d loss / d zhat
    double* w;          // [T, r] dz B^T
    double* kl;         // [T]
    double* part;       // per-slice partial products (predictor_partial_doubles)
    void* wsplit;       // router split (N columns)
    size_t bytes;
};
size_t predictor_partial_doubles(const pr2_moe_desc& d);
hipError_t launch_predictor_loss(const pr2_moe_desc& d, const void* h, const float* W_r,
                                 const float* b_r, const void* h_old, const float* p_old,
                                 const float* A, const float* B, int kind, float* kl_out,
                                 float* loss_out, float* dA, float* dB, const PredLossWs& ws,
                                 hipStream_t s);
hipError_t launch_predictor_zero(const pr2_moe_desc& d, float* kl_out, float* loss_out, float* dA,
                                 float* dB, hipStream_t s);

// backward.hip
bool bwd_mfma_ok(const pr2_moe_desc& d);
int bwd_partials(const pr2_moe_desc& d);    // partial gate-gradient sums per route
struct BwdGrads {
    void* dx;
    float* dW_r;
    float* db_r;        // may be null
    float* dW_gate;
    float* dW_up;
    float* dW_down;
};
hipError_t launch_replay_backward(const pr2_moe_desc& d, const void* x, const void* idx,
                                  int64_t ldi, const float* W_r, const void* W_gate,
                                  const void* W_up, const void* W_down, const void* dy,
                                  const float* gate, const BwdWs& ws, const BwdGrads& out,
                                  hipStream_t s, const void* au_in = nullptr);
hipError_t launch_zero_grads(const pr2_moe_desc& d, const BwdGrads& out, hipStream_t s);

}  // namespace pr2
