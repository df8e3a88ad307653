// Host side of the C ABI: argument validation (before any HIP call), workspace
// layout, kernel sequencing and the measurement hooks.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

namespace pr2 {

// ------------------------------------------------------------- errors ----
static thread_local std::string t_err;

pr2_status fail(pr2_status s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    t_err = buf;
    return s;
}

pr2_status ok() {
    t_err.clear();
    return PR2_OK;
}

static bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

static size_t act_bytes(const pr2_moe_desc& d) { return d.act_dtype == PR2_BF16 ? 2 : 4; }

static bool validate_env() {
    const char* v = getenv("PR2_VALIDATE");
    return v && v[0] == '1';
}

// PR2_VALIDATE=1 waits for the stream, which a HIP graph capture forbids
static pr2_status validation_allowed(bool validate, hipStream_t st) {
    if (!validate) return PR2_OK;
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(st, &cs) != hipSuccess) {
        (void)hipGetLastError();
        return fail(PR2_ERR_HIP, "hipStreamIsCapturing failed");
    }
    if (cs != hipStreamCaptureStatusNone)
        return fail(PR2_ERR_UNSUPPORTED, "PR2_VALIDATE=1 synchronises the stream, which is not "
                    "allowed while it is captured into a HIP graph");
    return PR2_OK;
}

// ------------------------------------------------------- device check ----
pr2_status device_ready() {
    static std::mutex mu;
    static std::map<int, int> ok_dev;  // device -> 1 gfx950, 0 not
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
        (void)hipGetLastError();
        return fail(PR2_ERR_DEVICE, "no usable HIP device");
    }
    std::lock_guard<std::mutex> lk(mu);
    auto it = ok_dev.find(dev);
    if (it == ok_dev.end()) {
        hipDeviceProp_t prop;
        if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
            (void)hipGetLastError();
            return fail(PR2_ERR_DEVICE, "hipGetDeviceProperties failed on device %d", dev);
        }
        int good = strncmp(prop.gcnArchName, "gfx950", 6) == 0;
        it = ok_dev.emplace(dev, good).first;
    }
    if (!it->second) return fail(PR2_ERR_DEVICE, "device %d is not gfx950 (MI355X)", dev);
    return PR2_OK;
}

// ------------------------------------------------ weight-split records ----
// pr2_route_predict_reuse reads the bf16 split of the router (and predictor)
// weights that an earlier route call left in the same workspace.  Each route
// call that forms a split records what it was formed from (device, weight
// pointers, layout, shape) under the workspace's address; every other call
// that writes into a workspace drops the records inside it.  The reuse call
// refuses a workspace without a matching record.  (Changed weight values under
// the same pointers stay undetectable: the caller guarantees them.)
struct SplitRecord {
    uintptr_t end;          // ws + ws_bytes of the recording call
    int dev;
    const float* W_r;
    const float* A;
    const float* B;
    int d, N, r;
    bool folded;            // predictor folded into N columns (no logits wanted)
};
static std::mutex g_split_mu;
static std::map<uintptr_t, SplitRecord> g_splits;   // keyed by workspace address

static void drop_split_records(const void* ws, size_t bytes) {
    if (!ws) return;
    const uintptr_t lo = (uintptr_t)ws, hi = lo + (bytes ? bytes : 1);
    std::lock_guard<std::mutex> lk(g_split_mu);
    for (auto it = g_splits.begin(); it != g_splits.end();) {
        if (it->first < hi && lo < it->second.end) it = g_splits.erase(it);
        else ++it;
    }
}

pr2_status hip_fail(hipError_t e, const char* what) {
    return fail(PR2_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// --------------------------------------------------- descriptor checks ----
static pr2_status check_desc(const pr2_moe_desc* d, bool need_m, bool need_idx_dtype) {
    if (!d) return fail(PR2_ERR_NULL, "desc is NULL");
    if (d->act_dtype != PR2_F32 && d->act_dtype != PR2_BF16)
        return fail(PR2_ERR_DTYPE, "act_dtype %d is not PR2_F32 or PR2_BF16", d->act_dtype);
    if (need_idx_dtype && d->idx_dtype != PR2_I32 && d->idx_dtype != PR2_I16)
        return fail(PR2_ERR_DTYPE, "idx_dtype %d is not PR2_I32 or PR2_I16", d->idx_dtype);
    if (d->T < 0) return fail(PR2_ERR_SHAPE, "T = %lld < 0", (long long)d->T);
    if (d->d < 1) return fail(PR2_ERR_SHAPE, "d = %d < 1", d->d);
    if (d->N < 1) return fail(PR2_ERR_SHAPE, "N = %d < 1", d->N);
    if (d->k < 1 || d->k > d->N) return fail(PR2_ERR_SHAPE, "k = %d not in [1, N = %d]", d->k, d->N);
    if (d->r < 0) return fail(PR2_ERR_SHAPE, "r = %d < 0", d->r);
    if (need_m && d->m < 1) return fail(PR2_ERR_SHAPE, "m = %d < 1", d->m);
    if (d->renorm != 0 && d->renorm != 1) return fail(PR2_ERR_SHAPE, "renorm = %d is not 0 or 1", d->renorm);
    if (d->N > kMaxExperts) return fail(PR2_ERR_UNSUPPORTED, "N = %d > %d", d->N, kMaxExperts);
    if (d->k > 256) return fail(PR2_ERR_UNSUPPORTED, "k = %d > 256", d->k);
    if (need_idx_dtype && d->idx_dtype == PR2_I16 && d->N > 32767)
        return fail(PR2_ERR_SHAPE, "int16 ids need N <= 32767");
    if (d->T > 0 && d->T * (int64_t)d->k >= ((int64_t)1 << 31))
        return fail(PR2_ERR_UNSUPPORTED, "T*k = %lld routes exceed 2^31 - 1", (long long)(d->T * d->k));
    return PR2_OK;
}

// ----------------------------------------------------------- workspace ----
static size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }

// Split scratch of the route call: the predictor folded into the router weights (N columns)
// when no logits are wanted, [W_r | A] (N + r columns) otherwise.
static size_t route_split_need(const pr2_moe_desc& d) {
    size_t need = 0;
    if (router_mfma_ok(d, d.N)) need = router_split_bytes(d.N, d);
    if (router_mfma_ok(d, d.N + d.r)) {
        size_t b = router_split_bytes(d.N + d.r, d);
        need = b > need ? b : need;
    }
    return need;
}

static ReplayWs moe_ws_layout(const pr2_moe_desc& d, void* base, size_t split_bytes) {
    ReplayWs w{};
    const int64_t Tk = d.T * (int64_t)d.k;
    const int tb = perm_tokens_per_block(d.k);
    w.nblk = (d.T + tb - 1) / tb;
    w.max_tiles = (Tk + kTileM - 1) / kTileM + d.N;
    const size_t ab = act_bytes(d);
    char* p = (char*)(((uintptr_t)base + 255) & ~(uintptr_t)255);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char* q = p ? p + off : nullptr;
        off += up256(bytes);
        return q;
    };
    w.gate = (float*)take(sizeof(float) * Tk);
    w.err = (int*)take(sizeof(int) * ERR_WORDS);
    w.bcount = (int*)take(sizeof(int) * (size_t)d.N * w.nblk);
    w.offsets = (int*)take(sizeof(int) * (size_t)(d.N + 1));
    w.tile_count = (int*)take(sizeof(int));
    w.tiles = (int*)take(sizeof(int) * 3 * (size_t)w.max_tiles);
    w.perm_src = (int*)take(sizeof(int) * Tk);
    w.inv = (int*)take(sizeof(int) * Tk);
    w.H = take(ab * Tk * (size_t)d.m);
    w.O = take(ab * Tk * (size_t)d.d);
    w.wsplit = take(split_bytes);
    w.bytes = off + 256;   // slack for aligning the caller's base
    return w;
}

ReplayWs replay_ws_layout(const pr2_moe_desc& d, void* base) {
    return moe_ws_layout(d, base, router_mfma_ok(d, d.N) ? router_split_bytes(d.N, d) : 0);
}

static ReplayWs rollout_ws_layout(const pr2_moe_desc& d, void* base) {
    return moe_ws_layout(d, base, route_split_need(d));
}

BwdWs bwd_ws_layout(const pr2_moe_desc& d, void* base) {
    BwdWs b{};
    b.fw = replay_ws_layout(d, base);
    const int64_t Tk = d.T * (int64_t)d.k;
    b.np = bwd_partials(d);
    char* p = base ? (char*)(((uintptr_t)base + 255) & ~(uintptr_t)255) : nullptr;
    size_t off = b.fw.bytes - 256;   // end of the replay segments
    auto take = [&](size_t bytes) {
        char* q = p ? p + off : nullptr;
        off += up256(bytes);
        return q;
    };
    b.AU = take(act_bytes(d) * Tk * 2 * (size_t)d.m);
    b.dgp = (float*)take(sizeof(float) * Tk * (size_t)b.np);
    b.dp_route = (float*)take(sizeof(float) * Tk);
    b.dp_perm = (float*)take(sizeof(float) * Tk);
    b.wrt = (float*)take(sizeof(float) * (size_t)d.N * d.d);
    b.order = (int*)take(sizeof(int) * (size_t)d.N);
    b.rwpart = (float*)take(sizeof(float) * (size_t)b.fw.max_tiles * d.d);
    b.rbpart = (float*)take(sizeof(float) * (size_t)b.fw.max_tiles);
    b.nchunk = 0;
    if (d.renorm == 0) {
        b.nchunk = (int)((d.T + 1023) / 1024);
        b.plog = (float*)take(sizeof(float) * (size_t)d.T * d.N);
        b.dpf = (float*)take(sizeof(float) * (size_t)d.T * d.N);
        b.lwpart = (float*)take(sizeof(float) * (size_t)b.nchunk * d.d * d.N);
        b.lbpart = (float*)take(sizeof(float) * (size_t)b.nchunk * d.N);
    }
    b.bytes = off + 256;
    return b;
}

static size_t diag_ws_bytes(const pr2_moe_desc& d) {
    return router_mfma_ok(d, d.N) ? router_split_bytes(d.N, d) + 256 : 0;
}

static PredLossWs pred_ws_layout(const pr2_moe_desc& d, void* base) {
    PredLossWs w{};
    char* p = base ? (char*)(((uintptr_t)base + 255) & ~(uintptr_t)255) : nullptr;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char* q = p ? p + off : nullptr;
        off += up256(bytes);
        return q;
    };
    const size_t T = (size_t)d.T;
    w.p_cur = (float*)take(sizeof(float) * T * d.N);
    w.u = (double*)take(sizeof(double) * T * d.r);
    w.dz = (double*)take(sizeof(double) * T * d.N);
    w.w = (double*)take(sizeof(double) * T * d.r);
    w.kl = (double*)take(sizeof(double) * T);
    w.part = (double*)take(sizeof(double) * predictor_partial_doubles(d));
    w.wsplit = take(router_mfma_ok(d, d.N) ? router_split_bytes(d.N, d) : 0);
    w.bytes = off + 256;
    return w;
}

static size_t route_ws_bytes(const pr2_moe_desc& d) {
    const size_t need = route_split_need(d);
    return need ? need + 256 : 0;
}

// ---------------------------------------------------- measurement hooks ----
struct ProfState {
    bool on = false;
    std::vector<std::pair<hipEvent_t, hipEvent_t>> pool;
    std::vector<int> free_slots;
    std::vector<std::pair<const char*, int>> pending;
    std::map<std::string, std::pair<double, int64_t>> totals;
    std::vector<std::string> order;
    std::vector<std::string> name_store;
};
static ProfState g_prof;

LaunchScope::LaunchScope(const char* n, hipStream_t s) : name(n), stream(s), slot(-1) {
    if (!g_prof.on) return;
    if (g_prof.free_slots.empty()) {
        hipEvent_t a, b;
        if (hipEventCreate(&a) != hipSuccess) return;
        if (hipEventCreate(&b) != hipSuccess) { (void)hipEventDestroy(a); return; }
        g_prof.pool.push_back({a, b});
        g_prof.free_slots.push_back((int)g_prof.pool.size() - 1);
    }
    slot = g_prof.free_slots.back();
    g_prof.free_slots.pop_back();
    (void)hipEventRecord(g_prof.pool[slot].first, stream);
}

LaunchScope::~LaunchScope() {
    if (slot < 0) return;
    (void)hipEventRecord(g_prof.pool[slot].second, stream);
    g_prof.pending.push_back({name, slot});
}

// Argument checks of the route calls; *empty is set for T == 0 (a no-op).
pr2_status check_route_args(const pr2_moe_desc* desc, const void* x, const float* W_r,
                                   const float* b_r, const float* A, const float* B,
                                   void* idx_out, int64_t ldi, float* gate_out,
                                   float* logits_out, bool* empty) {
    *empty = false;
    pr2_status s = check_desc(desc, false, true);
    if (s != PR2_OK) return s;
    const pr2_moe_desc& d = *desc;
    if (d.r > 256) return fail(PR2_ERR_UNSUPPORTED, "predictor rank r = %d > 256", d.r);
    if (ldi < d.k) return fail(PR2_ERR_SHAPE, "ldi = %lld < k = %d", (long long)ldi, d.k);
    if (d.T == 0) {
        *empty = true;
        return PR2_OK;
    }
    if (!x) return fail(PR2_ERR_NULL, "x is NULL");
    if (!W_r) return fail(PR2_ERR_NULL, "W_r is NULL");
    if (!idx_out) return fail(PR2_ERR_NULL, "idx_out is NULL");
    if (d.r > 0 && !A) return fail(PR2_ERR_NULL, "A is NULL with r = %d > 0", d.r);
    if (d.r > 0 && !B && d.r != d.N)
        return fail(PR2_ERR_NULL, "B is NULL but r = %d != N = %d (identity needs r == N)", d.r, d.N);
    if (!aligned(x, 16)) return fail(PR2_ERR_ALIGN, "x is not 16-byte aligned");
    if (!aligned(W_r, 4) || (b_r && !aligned(b_r, 4)) || (A && !aligned(A, 4)) ||
        (B && !aligned(B, 4)))
        return fail(PR2_ERR_ALIGN, "an fp32 router/predictor tensor is not 4-byte aligned");
    if (!aligned(idx_out, d.idx_dtype == PR2_I16 ? 2 : 4))
        return fail(PR2_ERR_ALIGN, "idx_out is not aligned to its element size");
    if ((gate_out && !aligned(gate_out, 4)) || (logits_out && !aligned(logits_out, 4)))
        return fail(PR2_ERR_ALIGN, "gate_out / logits_out is not 4-byte aligned");
    return PR2_OK;
}

}  // namespace pr2

using namespace pr2;

extern "C" {

const char* pr2_version(void) { return "pr2-mi355x 0.1"; }

const char* pr2_status_string(pr2_status s) {
    // a C caller may pass any int: read the raw value (loading an out-of-range
    // value as the enum type would be undefined behaviour here)
    int v;
    memcpy(&v, &s, sizeof v);
    switch (v) {
        case PR2_OK: return "PR2_OK";
        case PR2_ERR_NULL: return "PR2_ERR_NULL";
        case PR2_ERR_SHAPE: return "PR2_ERR_SHAPE";
        case PR2_ERR_DTYPE: return "PR2_ERR_DTYPE";
        case PR2_ERR_ALIGN: return "PR2_ERR_ALIGN";
        case PR2_ERR_WORKSPACE: return "PR2_ERR_WORKSPACE";
        case PR2_ERR_UNSUPPORTED: return "PR2_ERR_UNSUPPORTED";
        case PR2_ERR_ROUTE: return "PR2_ERR_ROUTE";
        case PR2_ERR_DEVICE: return "PR2_ERR_DEVICE";
        case PR2_ERR_HIP: return "PR2_ERR_HIP";
    }
    return "PR2_ERR_UNKNOWN";
}

const char* pr2_last_error(void) { return t_err.c_str(); }

size_t pr2_workspace_bytes(const pr2_moe_desc* desc, int op) {
    if (!desc) return 0;
    switch (op) {
        case PR2_OP_ROUTE: {
            std::string saved = t_err;
            pr2_status s = check_desc(desc, false, true);
            t_err = saved;
            if (s != PR2_OK || desc->r < 0) return 0;
            return route_ws_bytes(*desc);
        }
        case PR2_OP_REPLAY_FWD: {
            std::string saved = t_err;
            pr2_status s = check_desc(desc, true, true);
            t_err = saved;
            if (s != PR2_OK) return 0;
            return replay_ws_layout(*desc, nullptr).bytes;
        }
        case PR2_OP_ROLLOUT_FWD: {
            std::string saved = t_err;
            pr2_status s = check_desc(desc, true, true);
            t_err = saved;
            if (s != PR2_OK || desc->r < 0) return 0;
            return rollout_ws_layout(*desc, nullptr).bytes;
        }
        case PR2_OP_ROUTE_DIAG: {
            std::string saved = t_err;
            pr2_status s = check_desc(desc, false, true);
            t_err = saved;
            if (s != PR2_OK) return 0;
            return diag_ws_bytes(*desc);
        }
        case PR2_OP_PREDICTOR_LOSS: {
            std::string saved = t_err;
            pr2_status s = check_desc(desc, false, false);
            t_err = saved;
            if (s != PR2_OK || desc->r < 1) return 0;
            return pred_ws_layout(*desc, nullptr).bytes;
        }
        case PR2_OP_REPLAY_BWD: {
            std::string saved = t_err;
            pr2_status s = check_desc(desc, true, true);
            t_err = saved;
            if (s != PR2_OK) return 0;
            return bwd_ws_layout(*desc, nullptr).bytes;
        }
        default:
            return 0;
    }
}

static pr2_status route_predict_impl(const pr2_moe_desc* desc, const void* x, const float* W_r,
                                     const float* b_r, const float* A, const float* B,
                                     void* idx_out, int64_t ldi, float* gate_out,
                                     float* logits_out, void* ws, size_t ws_bytes,
                                     pr2_stream_t stream, bool reuse_split) {
    bool empty = false;
    pr2_status s = check_route_args(desc, x, W_r, b_r, A, B, idx_out, ldi, gate_out, logits_out,
                                    &empty);
    if (s != PR2_OK) return s;
    if (empty) return ok();
    const pr2_moe_desc& d = *desc;
    const size_t need = route_ws_bytes(d);
    if (need && !ws) return fail(PR2_ERR_NULL, "ws is NULL (need %zu bytes)", need);
    if (ws_bytes < need)
        return fail(PR2_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
    // the split this call reads or forms: none on the fp64 vector path
    const bool folded = logits_out == nullptr && router_mfma_ok(d, d.N);
    const bool has_split = folded || router_mfma_ok(d, d.N + d.r);
    const float* A_key = d.r > 0 ? A : nullptr;
    const float* B_key = d.r > 0 ? B : nullptr;
    SplitRecord want{(uintptr_t)ws + ws_bytes, -1, W_r, A_key, B_key, d.d, d.N, d.r, folded};
    if (reuse_split && has_split) {
        std::lock_guard<std::mutex> lk(g_split_mu);
        auto it = g_splits.find((uintptr_t)ws);
        if (it == g_splits.end())
            return fail(PR2_ERR_WORKSPACE, "ws holds no router split: call pr2_route_predict "
                        "with this workspace first");
        const SplitRecord& h = it->second;
        if (h.W_r != W_r || h.A != A_key || h.B != B_key || h.d != d.d || h.N != d.N ||
            h.r != d.r || h.folded != folded)
            return fail(PR2_ERR_WORKSPACE, "ws holds the split of other weights, shape or layout "
                        "(W_r, A, B, d, N, r and the NULL-ness of logits_out must match the "
                        "call that formed it)");
        want.dev = h.dev;
    }
    s = device_ready();
    if (s != PR2_OK) return s;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return fail(PR2_ERR_DEVICE, "no usable HIP device");
    }
    if (reuse_split && has_split && want.dev != dev)
        return fail(PR2_ERR_WORKSPACE, "ws holds a split formed on device %d, not %d", want.dev, dev);
    if (!reuse_split) drop_split_records(ws, ws_bytes);
    void* split = need ? (void*)(((uintptr_t)ws + 255) & ~(uintptr_t)255) : nullptr;
    hipError_t e = launch_route_predict(d, x, W_r, b_r, A, B, idx_out, ldi, gate_out, logits_out,
                                        split, (hipStream_t)stream, FeatureCache{}, reuse_split);
    if (e != hipSuccess) return hip_fail(e, "route_predict launch");
    if (!reuse_split && has_split) {
        want.dev = dev;
        std::lock_guard<std::mutex> lk(g_split_mu);
        g_splits[(uintptr_t)ws] = want;
    }
    return ok();
}

pr2_status pr2_route_predict(const pr2_moe_desc* desc, const void* x, const float* W_r,
                             const float* b_r, const float* A, const float* B, void* idx_out,
                             int64_t ldi, float* gate_out, float* logits_out, void* ws,
                             size_t ws_bytes, pr2_stream_t stream) {
    return route_predict_impl(desc, x, W_r, b_r, A, B, idx_out, ldi, gate_out, logits_out, ws,
                              ws_bytes, stream, false);
}

pr2_status pr2_route_predict_reuse(const pr2_moe_desc* desc, const void* x, const float* W_r,
                                   const float* b_r, const float* A, const float* B,
                                   void* idx_out, int64_t ldi, float* gate_out, float* logits_out,
                                   void* ws, size_t ws_bytes, pr2_stream_t stream) {
    return route_predict_impl(desc, x, W_r, b_r, A, B, idx_out, ldi, gate_out, logits_out, ws,
                              ws_bytes, stream, true);
}

static pr2_status check_diag_outputs(const pr2_moe_desc& d, const float* z_ref,
                                     const void* cur_idx_out, const int32_t* overlap_out,
                                     const float* kl_out, const uint64_t* hist_out) {
    if (kl_out && !z_ref) return fail(PR2_ERR_NULL, "kl_out needs z_ref");
    if (hist_out && !aligned(hist_out, 8)) return fail(PR2_ERR_ALIGN, "hist_out is not 8-byte aligned");
    if ((z_ref && !aligned(z_ref, 4)) || (kl_out && !aligned(kl_out, 4)) ||
        (overlap_out && !aligned(overlap_out, 4)))
        return fail(PR2_ERR_ALIGN, "z_ref, kl_out and overlap_out must be 4-byte aligned");
    if (cur_idx_out && !aligned(cur_idx_out, d.idx_dtype == PR2_I16 ? 2 : 4))
        return fail(PR2_ERR_ALIGN, "cur_idx_out is not aligned to its element size");
    return PR2_OK;
}

static pr2_status replay_forward_impl(const pr2_moe_desc* desc, const void* x, const void* idx,
                                      int64_t ldi, const float* W_r, const float* b_r,
                                      const void* W_gate, const void* W_up, const void* W_down,
                                      void* y, float* gate_out, const RouteDiag* diag, void* ws,
                                      size_t ws_bytes, pr2_stream_t stream,
                                      void* au_out = nullptr) {
    pr2_status s = check_desc(desc, true, true);
    if (s != PR2_OK) return s;
    const pr2_moe_desc& d = *desc;
    if (ldi < d.k) return fail(PR2_ERR_SHAPE, "ldi = %lld < k = %d", (long long)ldi, d.k);
    if (diag && diag->hist && d.T == 0) {
        // the histogram of an empty batch is all zeros
        s = device_ready();
        if (s != PR2_OK) return s;
        hipError_t e = launch_zero_i32((int*)diag->hist, 2 * (d.k + 1), (hipStream_t)stream);
        if (e != hipSuccess) return hip_fail(e, "histogram reset");
        return ok();
    }
    if (d.T == 0) return ok();
    if (!x) return fail(PR2_ERR_NULL, "x is NULL");
    if (!idx) return fail(PR2_ERR_NULL, "idx is NULL");
    if (!W_r) return fail(PR2_ERR_NULL, "W_r is NULL");
    if (!W_gate || !W_up || !W_down) return fail(PR2_ERR_NULL, "an expert weight pointer is NULL");
    if (!y) return fail(PR2_ERR_NULL, "y is NULL");
    if (!aligned(x, 16) || !aligned(y, 16) || !aligned(W_gate, 16) || !aligned(W_up, 16) ||
        !aligned(W_down, 16))
        return fail(PR2_ERR_ALIGN, "x, y and expert weights must be 16-byte aligned");
    if (!aligned(W_r, 4) || (b_r && !aligned(b_r, 4)) || (gate_out && !aligned(gate_out, 4)))
        return fail(PR2_ERR_ALIGN, "an fp32 tensor is not 4-byte aligned");
    if (!aligned(idx, d.idx_dtype == PR2_I16 ? 2 : 4))
        return fail(PR2_ERR_ALIGN, "idx is not aligned to its element size");
    const size_t need = replay_ws_layout(d, nullptr).bytes;
    if (!ws) return fail(PR2_ERR_NULL, "ws is NULL (need %zu bytes)", need);
    if (ws_bytes < need)
        return fail(PR2_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
    s = device_ready();
    if (s != PR2_OK) return s;

    hipStream_t st = (hipStream_t)stream;
    ReplayWs w = replay_ws_layout(d, ws);
    const bool validate = validate_env();
    s = validation_allowed(validate, st);
    if (s != PR2_OK) return s;
    drop_split_records(ws, ws_bytes);
    hipError_t e;
    if (validate) {
        e = launch_zero_i32(w.err, ERR_WORDS, st);
        if (e != hipSuccess) return hip_fail(e, "error-word reset");
    }
    float* gate = gate_out ? gate_out : w.gate;
    const bool counted = replay_counts_fused(d);
    e = launch_replay_gates(d, x, idx, ldi, W_r, b_r, gate, w.err, w.wsplit, st, diag,
                            counted ? w.bcount : nullptr);
    if (e != hipSuccess) return hip_fail(e, "replay_gates launch");
    e = launch_permute(d, idx, ldi, w, st, counted);
    if (e != hipSuccess) return hip_fail(e, "permute launch");
    e = launch_expert_gemms(d, x, W_gate, W_up, W_down, gate, w, st, au_out);
    if (e != hipSuccess) return hip_fail(e, "expert GEMM launch");
    e = launch_combine(d, w, y, st);
    if (e != hipSuccess) return hip_fail(e, "combine launch");
    if (validate) {
        int errs[ERR_WORDS];
        e = hipMemcpyAsync(errs, w.err, sizeof(errs), hipMemcpyDeviceToHost, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
        if (e != hipSuccess) return hip_fail(e, "validation readback");
        if (errs[ERR_BAD_ID] || errs[ERR_DUP_ID])
            return fail(PR2_ERR_ROUTE, "route has %d out-of-range and %d repeated ids",
                        errs[ERR_BAD_ID], errs[ERR_DUP_ID]);
    }
    return ok();
}

pr2_status pr2_moe_replay_forward(const pr2_moe_desc* desc, const void* x, const void* idx,
                                  int64_t ldi, const float* W_r, const float* b_r,
                                  const void* W_gate, const void* W_up, const void* W_down,
                                  void* y, float* gate_out, void* ws, size_t ws_bytes,
                                  pr2_stream_t stream) {
    return replay_forward_impl(desc, x, idx, ldi, W_r, b_r, W_gate, W_up, W_down, y, gate_out,
                               nullptr, ws, ws_bytes, stream);
}

pr2_status pr2_moe_replay_forward_save(const pr2_moe_desc* desc, const void* x, const void* idx,
                                       int64_t ldi, const float* W_r, const float* b_r,
                                       const void* W_gate, const void* W_up, const void* W_down,
                                       void* y, float* gate_out, void* au_out, void* ws,
                                       size_t ws_bytes, pr2_stream_t stream) {
    pr2_status s = check_desc(desc, true, true);
    if (s != PR2_OK) return s;
    if (desc->T > 0 && !au_out) return fail(PR2_ERR_NULL, "au_out is NULL");
    if (!aligned(au_out, 16)) return fail(PR2_ERR_ALIGN, "au_out must be 16-byte aligned");
    return replay_forward_impl(desc, x, idx, ldi, W_r, b_r, W_gate, W_up, W_down, y, gate_out,
                               nullptr, ws, ws_bytes, stream, au_out);
}

pr2_status pr2_moe_replay_forward_diag(const pr2_moe_desc* desc, const void* x, const void* idx,
                                       int64_t ldi, const float* W_r, const float* b_r,
                                       const void* W_gate, const void* W_up, const void* W_down,
                                       void* y, float* gate_out, const float* z_ref,
                                       void* cur_idx_out, int32_t* overlap_out, float* kl_out,
                                       uint64_t* hist_out, void* ws, size_t ws_bytes,
                                       pr2_stream_t stream) {
    pr2_status s = check_desc(desc, true, true);
    if (s != PR2_OK) return s;
    s = check_diag_outputs(*desc, z_ref, cur_idx_out, overlap_out, kl_out, hist_out);
    if (s != PR2_OK) return s;
    const RouteDiag diag{kl_out ? z_ref : nullptr, cur_idx_out, overlap_out, kl_out,
                         (unsigned long long*)hist_out, nullptr};
    const bool any = cur_idx_out || overlap_out || kl_out || hist_out;
    return replay_forward_impl(desc, x, idx, ldi, W_r, b_r, W_gate, W_up, W_down, y, gate_out,
                               any ? &diag : nullptr, ws, ws_bytes, stream);
}

pr2_status pr2_moe_rollout_forward(const pr2_moe_desc* desc, const void* x, const float* W_r,
                                   const float* b_r, const float* A, const float* B,
                                   const void* W_gate, const void* W_up, const void* W_down,
                                   void* idx_out, int64_t ldi, float* gate_out, float* logits_out,
                                   void* y, void* ws, size_t ws_bytes, pr2_stream_t stream) {
    pr2_status s = check_desc(desc, true, true);
    if (s != PR2_OK) return s;
    const pr2_moe_desc& d = *desc;
    if (d.r > 256) return fail(PR2_ERR_UNSUPPORTED, "predictor rank r = %d > 256", d.r);
    if (ldi < d.k) return fail(PR2_ERR_SHAPE, "ldi = %lld < k = %d", (long long)ldi, d.k);
    if (d.T == 0) return ok();
    if (!x) return fail(PR2_ERR_NULL, "x is NULL");
    if (!W_r) return fail(PR2_ERR_NULL, "W_r is NULL");
    if (!idx_out) return fail(PR2_ERR_NULL, "idx_out is NULL");
    if (d.r > 0 && !A) return fail(PR2_ERR_NULL, "A is NULL with r = %d > 0", d.r);
    if (d.r > 0 && !B && d.r != d.N)
        return fail(PR2_ERR_NULL, "B is NULL but r = %d != N = %d (identity needs r == N)", d.r, d.N);
    if (!W_gate || !W_up || !W_down) return fail(PR2_ERR_NULL, "an expert weight pointer is NULL");
    if (!y) return fail(PR2_ERR_NULL, "y is NULL");
    if (!aligned(x, 16) || !aligned(y, 16) || !aligned(W_gate, 16) || !aligned(W_up, 16) ||
        !aligned(W_down, 16))
        return fail(PR2_ERR_ALIGN, "x, y and the expert weights must be 16-byte aligned");
    if (!aligned(W_r, 4) || (b_r && !aligned(b_r, 4)) || (A && !aligned(A, 4)) ||
        (B && !aligned(B, 4)) || (gate_out && !aligned(gate_out, 4)) ||
        (logits_out && !aligned(logits_out, 4)))
        return fail(PR2_ERR_ALIGN, "an fp32 router/predictor/gate/logit tensor is not 4-byte aligned");
    if (!aligned(idx_out, d.idx_dtype == PR2_I16 ? 2 : 4))
        return fail(PR2_ERR_ALIGN, "idx_out is not aligned to its element size");
    const size_t need = rollout_ws_layout(d, nullptr).bytes;
    if (!ws) return fail(PR2_ERR_NULL, "ws is NULL (need %zu bytes)", need);
    if (ws_bytes < need)
        return fail(PR2_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
    s = device_ready();
    if (s != PR2_OK) return s;

    hipStream_t st = (hipStream_t)stream;
    ReplayWs w = rollout_ws_layout(d, ws);
    drop_split_records(ws, ws_bytes);
    float* gate = gate_out ? gate_out : w.gate;
    bool counted = false;
    hipError_t e = launch_route_predict(d, x, W_r, b_r, A, B, idx_out, ldi, gate, logits_out,
                                        w.wsplit, st, FeatureCache{}, false, true, w.bcount,
                                        &counted);
    if (e != hipSuccess) return hip_fail(e, "route_predict launch");
    e = launch_permute(d, idx_out, ldi, w, st, counted);
    if (e != hipSuccess) return hip_fail(e, "permute launch");
    e = launch_expert_gemms(d, x, W_gate, W_up, W_down, gate, w, st);
    if (e != hipSuccess) return hip_fail(e, "expert GEMM launch");
    e = launch_combine(d, w, y, st);
    if (e != hipSuccess) return hip_fail(e, "combine launch");
    return ok();
}

static pr2_status replay_backward_impl(const pr2_moe_desc* desc, const void* x, const void* idx,
                                       int64_t ldi, const float* W_r, const float* b_r,
                                       const void* W_gate, const void* W_up, const void* W_down,
                                       const void* au_saved, const void* dy, void* dx,
                                       float* dW_r, float* db_r, float* dW_gate, float* dW_up,
                                       float* dW_down, void* ws, size_t ws_bytes,
                                       pr2_stream_t stream) {
    pr2_status s = check_desc(desc, true, true);
    if (s != PR2_OK) return s;
    const pr2_moe_desc& d = *desc;
    if (d.renorm == 0 && d.k > 64)
        return fail(PR2_ERR_UNSUPPORTED, "the paper-literal backward (renorm = 0) needs k <= 64");
    if (ldi < d.k) return fail(PR2_ERR_SHAPE, "ldi = %lld < k = %d", (long long)ldi, d.k);
    if (!W_r) return fail(PR2_ERR_NULL, "W_r is NULL");
    if (!W_gate || !W_up || !W_down) return fail(PR2_ERR_NULL, "an expert weight pointer is NULL");
    if (!dW_r || !dW_gate || !dW_up || !dW_down)
        return fail(PR2_ERR_NULL, "a weight-gradient pointer is NULL");
    if (d.T > 0) {
        if (!x) return fail(PR2_ERR_NULL, "x is NULL");
        if (!idx) return fail(PR2_ERR_NULL, "idx is NULL");
        if (!dy) return fail(PR2_ERR_NULL, "dy is NULL");
        if (!dx) return fail(PR2_ERR_NULL, "dx is NULL");
    }
    if (!aligned(x, 16) || !aligned(dy, 16) || !aligned(dx, 16) || !aligned(W_gate, 16) ||
        !aligned(W_up, 16) || !aligned(W_down, 16))
        return fail(PR2_ERR_ALIGN, "x, dy, dx and the expert weights must be 16-byte aligned");
    if (!aligned(dW_gate, 16) || !aligned(dW_up, 16) || !aligned(dW_down, 16))
        return fail(PR2_ERR_ALIGN, "expert weight gradients must be 16-byte aligned");
    if (!aligned(W_r, 4) || !aligned(dW_r, 4) || (b_r && !aligned(b_r, 4)) || (db_r && !aligned(db_r, 4)))
        return fail(PR2_ERR_ALIGN, "router tensors must be 4-byte aligned");
    if (d.T > 0 && !aligned(idx, d.idx_dtype == PR2_I16 ? 2 : 4))
        return fail(PR2_ERR_ALIGN, "idx is not aligned to its element size");
    const BwdGrads out{dx, dW_r, db_r, dW_gate, dW_up, dW_down};
    hipStream_t st = (hipStream_t)stream;
    if (d.T == 0) {
        s = device_ready();
        if (s != PR2_OK) return s;
        hipError_t e = launch_zero_grads(d, out, st);
        if (e != hipSuccess) return hip_fail(e, "zero-gradient launch");
        return ok();
    }
    const size_t need = bwd_ws_layout(d, nullptr).bytes;
    if (!ws) return fail(PR2_ERR_NULL, "ws is NULL (need %zu bytes)", need);
    if (ws_bytes < need)
        return fail(PR2_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
    s = device_ready();
    if (s != PR2_OK) return s;

    BwdWs w = bwd_ws_layout(d, ws);
    const bool validate = validate_env();
    s = validation_allowed(validate, st);
    if (s != PR2_OK) return s;
    drop_split_records(ws, ws_bytes);
    hipError_t e;
    if (validate) {
        e = launch_zero_i32(w.fw.err, ERR_WORDS, st);
        if (e != hipSuccess) return hip_fail(e, "error-word reset");
    }
    // the paper-literal weights also need every token's N logits
    RouteDiag logits{};
    logits.p_out = w.plog;
    const bool counted = replay_counts_fused(d);
    e = launch_replay_gates(d, x, idx, ldi, W_r, b_r, w.fw.gate, w.fw.err, w.fw.wsplit, st,
                            d.renorm == 0 ? &logits : nullptr, counted ? w.fw.bcount : nullptr);
    if (e == hipSuccess) e = launch_permute(d, idx, ldi, w.fw, st, counted);
    if (e != hipSuccess) return hip_fail(e, "replay_gates / permute launch");
    e = launch_replay_backward(d, x, idx, ldi, W_r, W_gate, W_up, W_down, dy, w.fw.gate, w, out,
                               st, au_saved);
    if (e != hipSuccess) return hip_fail(e, "backward launch");
    if (validate) {
        int errs[ERR_WORDS];
        e = hipMemcpyAsync(errs, w.fw.err, sizeof(errs), hipMemcpyDeviceToHost, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
        if (e != hipSuccess) return hip_fail(e, "validation readback");
        if (errs[ERR_BAD_ID] || errs[ERR_DUP_ID])
            return fail(PR2_ERR_ROUTE, "route has %d out-of-range and %d repeated ids",
                        errs[ERR_BAD_ID], errs[ERR_DUP_ID]);
    }
    return ok();
}

pr2_status pr2_moe_replay_backward(const pr2_moe_desc* desc, const void* x, const void* idx,
                                   int64_t ldi, const float* W_r, const float* b_r,
                                   const void* W_gate, const void* W_up, const void* W_down,
                                   const void* dy, void* dx, float* dW_r, float* db_r,
                                   float* dW_gate, float* dW_up, float* dW_down, void* ws,
                                   size_t ws_bytes, pr2_stream_t stream) {
    return replay_backward_impl(desc, x, idx, ldi, W_r, b_r, W_gate, W_up, W_down, nullptr, dy,
                                dx, dW_r, db_r, dW_gate, dW_up, dW_down, ws, ws_bytes, stream);
}

pr2_status pr2_moe_replay_backward_saved(const pr2_moe_desc* desc, const void* x, const void* idx,
                                         int64_t ldi, const float* W_r, const float* b_r,
                                         const void* W_gate, const void* W_up,
                                         const void* W_down, const void* au_saved,
                                         const void* dy, void* dx, float* dW_r, float* db_r,
                                         float* dW_gate, float* dW_up, float* dW_down, void* ws,
                                         size_t ws_bytes, pr2_stream_t stream) {
    pr2_status s = check_desc(desc, true, true);
    if (s != PR2_OK) return s;
    if (desc->T > 0 && !au_saved) return fail(PR2_ERR_NULL, "au_saved is NULL");
    if (!aligned(au_saved, 16)) return fail(PR2_ERR_ALIGN, "au_saved must be 16-byte aligned");
    return replay_backward_impl(desc, x, idx, ldi, W_r, b_r, W_gate, W_up, W_down, au_saved, dy,
                                dx, dW_r, db_r, dW_gate, dW_up, dW_down, ws, ws_bytes, stream);
}

pr2_status pr2_route_diagnostics(const pr2_moe_desc* desc, const void* x, const void* idx,
                                 int64_t ldi, const float* W_r, const float* b_r,
                                 const float* z_ref, void* cur_idx_out, int32_t* overlap_out,
                                 float* kl_out, uint64_t* hist_out, void* ws, size_t ws_bytes,
                                 pr2_stream_t stream) {
    pr2_status s = check_desc(desc, false, true);
    if (s != PR2_OK) return s;
    const pr2_moe_desc& d = *desc;
    if (ldi < d.k) return fail(PR2_ERR_SHAPE, "ldi = %lld < k = %d", (long long)ldi, d.k);
    if (kl_out && !z_ref) return fail(PR2_ERR_NULL, "kl_out needs z_ref");
    if (hist_out && !aligned(hist_out, 8)) return fail(PR2_ERR_ALIGN, "hist_out is not 8-byte aligned");
    if (d.T == 0 && !hist_out) return ok();
    if (d.T > 0) {
        if (!x) return fail(PR2_ERR_NULL, "x is NULL");
        if (!idx) return fail(PR2_ERR_NULL, "idx is NULL");
        if (!W_r) return fail(PR2_ERR_NULL, "W_r is NULL");
        if (!aligned(x, 16)) return fail(PR2_ERR_ALIGN, "x is not 16-byte aligned");
        if (!aligned(W_r, 4) || (b_r && !aligned(b_r, 4)) || (z_ref && !aligned(z_ref, 4)) ||
            (kl_out && !aligned(kl_out, 4)) || (overlap_out && !aligned(overlap_out, 4)))
            return fail(PR2_ERR_ALIGN, "an fp32 / int32 tensor is not 4-byte aligned");
        const size_t ib = d.idx_dtype == PR2_I16 ? 2 : 4;
        if (!aligned(idx, ib) || (cur_idx_out && !aligned(cur_idx_out, ib)))
            return fail(PR2_ERR_ALIGN, "an id buffer is not aligned to its element size");
        const size_t need = diag_ws_bytes(d);
        if (need && !ws) return fail(PR2_ERR_NULL, "ws is NULL (need %zu bytes)", need);
        if (ws_bytes < need)
            return fail(PR2_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
    }
    s = device_ready();
    if (s != PR2_OK) return s;
    drop_split_records(ws, ws_bytes);
    void* split = ws ? (void*)(((uintptr_t)ws + 255) & ~(uintptr_t)255) : nullptr;
    hipError_t e = launch_route_diagnostics(d, x, idx, ldi, W_r, b_r, z_ref, cur_idx_out,
                                            overlap_out, kl_out, (unsigned long long*)hist_out,
                                            split, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "route diagnostics launch");
    return ok();
}

int64_t pr2_feature_cache_positions(int64_t T, int64_t Tc, uint64_t seed, int64_t* pos_out) {
    if (T < 0 || Tc < 1 || T > ((int64_t)1 << 40)) {
        fail(PR2_ERR_SHAPE, "need T >= 0 (at most 2^40) and Tc >= 1");
        return -1;
    }
    const int64_t n = Tc < T ? Tc : T;
    if (n > 0 && !pos_out) {
        fail(PR2_ERR_NULL, "pos_out is NULL");
        return -1;
    }
    if (Tc >= T) {
        for (int64_t t = 0; t < T; ++t) pos_out[t] = t;
        ok();
        return T;
    }
    const uint64_t golden = 0x9E3779B97F4A7C15ull;
    for (int64_t i = 0; i < Tc; ++i) {
        const int64_t lo = (int64_t)(((__int128)i * T) / Tc);
        const int64_t hi = (int64_t)(((__int128)(i + 1) * T) / Tc);
        uint64_t z = seed + (uint64_t)(i + 1) * golden;     // SplitMix64 state of draw i
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        z ^= z >> 31;
        pos_out[i] = lo + (int64_t)(z % (uint64_t)(hi - lo));
    }
    ok();
    return Tc;
}

pr2_status pr2_route_predict_cached(const pr2_moe_desc* desc, const void* x, const float* W_r,
                                    const float* b_r, const float* A, const float* B,
                                    void* idx_out, int64_t ldi, float* gate_out,
                                    const int32_t* cache_row, void* h_cache, float* p_cache,
                                    int64_t cache_rows, void* ws, size_t ws_bytes,
                                    pr2_stream_t stream) {
    pr2_status s = check_desc(desc, false, true);
    if (s != PR2_OK) return s;
    const pr2_moe_desc& d = *desc;
    if (!cache_row || !h_cache || !p_cache)
        return fail(PR2_ERR_NULL, "cache_row, h_cache and p_cache are required");
    if (cache_rows < 0) return fail(PR2_ERR_SHAPE, "cache_rows = %lld < 0", (long long)cache_rows);
    if (!aligned(h_cache, 16) || !aligned(p_cache, 4) || !aligned(cache_row, 4))
        return fail(PR2_ERR_ALIGN, "h_cache must be 16-byte, p_cache and cache_row 4-byte aligned");
    if (d.r > 256) return fail(PR2_ERR_UNSUPPORTED, "predictor rank r = %d > 256", d.r);
    if (ldi < d.k) return fail(PR2_ERR_SHAPE, "ldi = %lld < k = %d", (long long)ldi, d.k);
    if (d.T == 0) return ok();
    if (!x) return fail(PR2_ERR_NULL, "x is NULL");
    if (!W_r) return fail(PR2_ERR_NULL, "W_r is NULL");
    if (!idx_out) return fail(PR2_ERR_NULL, "idx_out is NULL");
    if (d.r > 0 && !A) return fail(PR2_ERR_NULL, "A is NULL with r = %d > 0", d.r);
    if (d.r > 0 && !B && d.r != d.N)
        return fail(PR2_ERR_NULL, "B is NULL but r = %d != N = %d (identity needs r == N)", d.r, d.N);
    if (!aligned(x, 16)) return fail(PR2_ERR_ALIGN, "x is not 16-byte aligned");
    if (!aligned(W_r, 4) || (b_r && !aligned(b_r, 4)) || (A && !aligned(A, 4)) ||
        (B && !aligned(B, 4)) || (gate_out && !aligned(gate_out, 4)))
        return fail(PR2_ERR_ALIGN, "an fp32 router/predictor/gate tensor is not 4-byte aligned");
    if (!aligned(idx_out, d.idx_dtype == PR2_I16 ? 2 : 4))
        return fail(PR2_ERR_ALIGN, "idx_out is not aligned to its element size");
    const size_t need = route_ws_bytes(d);
    if (need && !ws) return fail(PR2_ERR_NULL, "ws is NULL (need %zu bytes)", need);
    if (ws_bytes < need)
        return fail(PR2_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
    s = device_ready();
    if (s != PR2_OK) return s;
    drop_split_records(ws, ws_bytes);
    void* split = need ? (void*)(((uintptr_t)ws + 255) & ~(uintptr_t)255) : nullptr;
    const FeatureCache cache{cache_row, h_cache, p_cache, cache_rows};
    hipError_t e = launch_route_predict(d, x, W_r, b_r, A, B, idx_out, ldi, gate_out, nullptr,
                                        split, (hipStream_t)stream, cache);
    if (e != hipSuccess) return hip_fail(e, "route_predict launch");
    return ok();
}

pr2_status pr2_predictor_loss(const pr2_moe_desc* desc, const void* h, const float* W_r,
                              const float* b_r, const void* h_old, const float* p_old,
                              const float* A, const float* B, int loss_kind, int mini_step,
                              float* kl_out, float* loss_out, float* dA, float* dB, void* ws,
                              size_t ws_bytes, pr2_stream_t stream) {
    pr2_status s = check_desc(desc, false, false);
    if (s != PR2_OK) return s;
    const pr2_moe_desc& d = *desc;
    if (d.r < 1) return fail(PR2_ERR_SHAPE, "the predictor loss needs r >= 1");
    if (loss_kind != 0 && loss_kind != 1)
        return fail(PR2_ERR_SHAPE, "loss_kind = %d is not 0 (KL) or 1 (delta matching)", loss_kind);
    if (mini_step < 1) return fail(PR2_ERR_SHAPE, "mini_step = %d < 1", mini_step);
    if (!A) return fail(PR2_ERR_NULL, "A is NULL");
    if (!B && d.r != d.N)
        return fail(PR2_ERR_NULL, "B is NULL but r = %d != N = %d (identity needs r == N)", d.r, d.N);
    if (!loss_out || !dA) return fail(PR2_ERR_NULL, "loss_out and dA are required");
    if (B && !dB) return fail(PR2_ERR_NULL, "dB is NULL");
    if (!aligned(A, 4) || (B && !aligned(B, 4)) || !aligned(loss_out, 4) || !aligned(dA, 4) ||
        (dB && !aligned(dB, 4)) || (kl_out && !aligned(kl_out, 4)))
        return fail(PR2_ERR_ALIGN, "an fp32 tensor is not 4-byte aligned");
    float* dBo = B ? dB : nullptr;
    hipStream_t st = (hipStream_t)stream;
    if (mini_step == 1 || d.T == 0) {
        // Alg. 3: no predictive loss on the first (on-policy) mini-step
        s = device_ready();
        if (s != PR2_OK) return s;
        hipError_t e = launch_predictor_zero(d, kl_out, loss_out, dA, dBo, st);
        if (e != hipSuccess) return hip_fail(e, "zero fill launch");
        return ok();
    }
    if (!h || !h_old) return fail(PR2_ERR_NULL, "h and h_old are required");
    if (!W_r || !p_old) return fail(PR2_ERR_NULL, "W_r and p_old are required");
    if (!aligned(h, 16) || !aligned(h_old, 16))
        return fail(PR2_ERR_ALIGN, "h and h_old must be 16-byte aligned");
    if (!aligned(W_r, 4) || (b_r && !aligned(b_r, 4)) || !aligned(p_old, 4))
        return fail(PR2_ERR_ALIGN, "W_r, b_r, p_old must be 4-byte aligned");
    const size_t need = pred_ws_layout(d, nullptr).bytes;
    if (!ws) return fail(PR2_ERR_NULL, "ws is NULL (need %zu bytes)", need);
    if (ws_bytes < need)
        return fail(PR2_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
    s = device_ready();
    if (s != PR2_OK) return s;
    drop_split_records(ws, ws_bytes);
    PredLossWs w = pred_ws_layout(d, ws);
    hipError_t e = launch_predictor_loss(d, h, W_r, b_r, h_old, p_old, A, B, loss_kind, kl_out,
                                         loss_out, dA, dBo, w, st);
    if (e != hipSuccess) return hip_fail(e, "predictor loss launch");
    return ok();
}

void pr2_profile_enable(int on) { g_prof.on = on != 0; }

void pr2_profile_reset(void) {
    for (auto& p : g_prof.pending) g_prof.free_slots.push_back(p.second);
    g_prof.pending.clear();
    g_prof.totals.clear();
    g_prof.order.clear();
}

int pr2_profile_collect(const char** names, double* total_ms, int64_t* launches, int cap) {
    for (auto& p : g_prof.pending) {
        auto& ev = g_prof.pool[p.second];
        if (hipEventSynchronize(ev.second) != hipSuccess) return -1;
        float ms = 0.0f;
        if (hipEventElapsedTime(&ms, ev.first, ev.second) != hipSuccess) return -1;
        std::string key(p.first);
        auto it = g_prof.totals.find(key);
        if (it == g_prof.totals.end()) {
            g_prof.totals[key] = {0.0, 0};
            g_prof.order.push_back(key);
        }
        g_prof.totals[key].first += ms;
        g_prof.totals[key].second += 1;
        g_prof.free_slots.push_back(p.second);
    }
    g_prof.pending.clear();
    g_prof.name_store = g_prof.order;
    int n = (int)g_prof.order.size();
    for (int i = 0; i < n && i < cap; ++i) {
        const auto& t = g_prof.totals[g_prof.order[i]];
        if (names) names[i] = g_prof.name_store[i].c_str();
        if (total_ms) total_ms[i] = t.first;
        if (launches) launches[i] = t.second;
    }
    return n;
}

}  // extern "C"
