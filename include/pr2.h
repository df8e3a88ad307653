/*
 * pr2.h -- C ABI of the MI355X (gfx950) Predictive Routing Replay MoE-layer hot path.
 *
 * One MoE layer of a Pr^2 model, in both phases of the method:
 *   rollout:  predictive route  I_hat = TopK(Softmax(h W + h W_p), k)   (Sec. 4.1,
 *             Eq. pr2_predict, Eq. pr2_route; Alg. 2 in Appendix D), recorded into a
 *             caller-owned route buffer;
 *   training: replay of the recorded ids with weights from the current router and the
 *             predictor bypassed, o = sum_{j in I_hat} rho_j E_j(h)  (Sec. 4.1, Eq. pr2_output;
 *             Alg. 3), experts being gated MLPs with gate, up and down projections
 *             (Appendix E.2).
 *
 * Conventions shared by every entry point
 *   - All tensor arguments are DEVICE pointers owned by the caller, row-major.  Alignment:
 *     activations (x, y, dy, dx) and expert weights and their gradients 16 bytes; fp32
 *     router, predictor, gate and logit tensors 4 bytes; id buffers their element size.
 *     The library never allocates, frees or keeps them; scratch memory comes from the
 *     caller's workspace `ws` of at least pr2_workspace_bytes(desc, op) bytes (any
 *     alignment; may be NULL when that size is 0).
 *   - Calls are asynchronous on `stream` (NULL = the null stream of the current device) and
 *     run on the current HIP device.  They return once the kernels are enqueued; every
 *     launch of a call goes on `stream` (the library owns no stream), so a call can be
 *     captured into a HIP graph.  Global state: the per-device gfx950 check and the
 *     workspace split records of pr2_route_predict_reuse, both host-side and guarded by
 *     mutexes, so calls may come from several threads (each with its own workspace).
 *   - Every argument is checked on the host before any HIP call.  On an error nothing is
 *     enqueued, outputs are untouched, the status says what was wrong and pr2_last_error()
 *     (thread-local) gives a sentence naming the argument.
 *   - T == 0 is a no-op returning PR2_OK (the backward then zeroes its weight gradients).
 *   - Expert ids are 0-based.  Results are deterministic: the same inputs on the same device
 *     give bitwise identical outputs (no floating-point atomics anywhere).
 *   - Route contents (0 <= id < N, distinct within a row) are a precondition.  Kernels never
 *     touch memory out of bounds for any id value: an out-of-range id is skipped and counted.
 *     With the environment variable PR2_VALIDATE=1 each call that reads a route also
 *     synchronises its stream and returns PR2_ERR_ROUTE if any id was out of range or
 *     repeated within its row (PR2_ERR_UNSUPPORTED, nothing enqueued, if the stream is
 *     being captured into a HIP graph).
 *   - Inputs must be finite; NaN or Inf give unspecified (but memory-safe) results.
 */
#ifndef PR2_H
#define PR2_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Same type as hipStream_t. */
typedef struct ihipStream_t* pr2_stream_t;

typedef enum {
    PR2_OK = 0,
    PR2_ERR_NULL = 1,        /* a required pointer is NULL                                  */
    PR2_ERR_SHAPE = 2,       /* a size is out of range (k > N, k < 1, d < 1, ldi < k, ...)     */
    PR2_ERR_DTYPE = 3,       /* unknown act_dtype / idx_dtype code                             */
    PR2_ERR_ALIGN = 4,       /* a pointer is not aligned as its argument requires              */
    PR2_ERR_WORKSPACE = 5,   /* workspace smaller than pr2_workspace_bytes(desc, op)           */
    PR2_ERR_UNSUPPORTED = 6, /* valid but not implemented (e.g. N > 1024)                      */
    PR2_ERR_ROUTE = 7,       /* PR2_VALIDATE=1 found an out-of-range or repeated id             */
    PR2_ERR_DEVICE = 8,      /* no usable HIP device, or the device is not gfx950              */
    PR2_ERR_HIP = 9          /* a HIP runtime call or kernel launch failed                     */
} pr2_status;

/* act_dtype: storage type of activations (x, y, dy, dx) and expert weights.
 * The router W_r, its bias, the predictor factors A, B, gates and logits are always fp32. */
enum { PR2_F32 = 0, PR2_BF16 = 1 };
/* idx_dtype: storage type of recorded expert ids. */
enum { PR2_I32 = 0, PR2_I16 = 1 };
/* op codes for pr2_workspace_bytes. */
enum {
    PR2_OP_ROUTE = 0,
    PR2_OP_REPLAY_FWD = 1,
    PR2_OP_REPLAY_BWD = 2,
    PR2_OP_ROLLOUT_FWD = 3,
    PR2_OP_ROUTE_DIAG = 4,
    PR2_OP_PREDICTOR_LOSS = 5
};

/*
 * Layer descriptor.
 *   T tokens (>= 0), d hidden size, N experts (1..1024), k experts per token (1..N),
 *   m expert intermediate size, r predictor rank (>= 0; 0 = no predictor),
 *   act_dtype PR2_F32 | PR2_BF16, idx_dtype PR2_I32 | PR2_I16 (PR2_I16 needs N <= 32767),
 *   renorm: 1 = the k weights are the softmax restricted to the k ids (they sum to one);
 *           0 = the weight of id j is rho_j of the softmax over all N experts, as Eq.
 *               pr2_old_output and Eq. pr2_output print it.
 */
typedef struct {
    int64_t T;
    int32_t d, N, k, m, r;
    int32_t act_dtype;
    int32_t idx_dtype;
    int32_t renorm;
} pr2_moe_desc;

/* Bytes of workspace an op needs for this descriptor (0 if none).  Never fails: an invalid
 * descriptor yields 0 and the call itself then reports the error.  The size does not
 * decrease with T: a workspace sized for a batch also serves any smaller batch of the
 * same layer shape. */
size_t pr2_workspace_bytes(const pr2_moe_desc* desc, int op);

/*
 * Route prediction during rollout (Sec. 4.1 "Route Prediction During Rollout";
 * Eq. pr2_predict, Eq. pr2_route; Alg. 2 in Appendix D, its logits, top-k and caching steps).
 *
 *   p = x W_r + b_r                      router logits (the feature-cache p_old)
 *   z = p + (x A) B                      predictive logits, W_p = A B of rank r
 *   idx = TopK(z, k)                     ties to the lower id, stored ASCENDING by id
 *   gate_j = softmax(z) restricted to idx (renorm = 1) or softmax over all N (renorm = 0)
 *
 *   x          [T, d] act_dtype
 *   W_r        [d, N] fp32;  b_r [N] fp32 or NULL (no router bias)
 *   A          [d, r] fp32;  B [r, N] fp32.  Both ignored when r == 0.  B may be NULL only
 *              when r == N, meaning the identity (a full-rank predictor W_p = A).
 *   idx_out    route record: token t's k ids go to idx_out + t*ldi (elements of idx_dtype),
 *              ldi >= k.  Rows of other tokens and elements beyond k in a row are never
 *              written, so a [seq, pos, k] buffer can be filled one decode step at a time
 *              (pass idx_out = buf + pos*k, ldi = n_pos*k).
 *   gate_out   [T, k] fp32, aligned with idx_out's order; may be NULL.
 *   logits_out [T, N] fp32 router logits p (without the predictor term); may be NULL.
 *   ws         scratch of at least pr2_workspace_bytes(desc, PR2_OP_ROUTE) bytes (the bf16
 *              three-way split of [W_r | A] that the MFMA router reads, and for batches of at
 *              most 2048 tokens the partial logits of its split-K form; 0 bytes when the
 *              shape takes the fp64 vector path).  Reused freely between calls on one stream.
 * Logits are accumulated from exact products (fp32 weights split into three bf16 parts times
 * bf16 x, or fp64 FMA for fp32 x) in fp32 chunks summed in fp64, then rounded once to fp32.
 */
pr2_status pr2_route_predict(const pr2_moe_desc* desc, const void* x, const float* W_r,
                             const float* b_r, const float* A, const float* B, void* idx_out,
                             int64_t ldi, float* gate_out, float* logits_out, void* ws,
                             size_t ws_bytes, pr2_stream_t stream);

/*
 * Route prediction for the later steps of a rollout (Sec. 4.1 "Route Prediction During
 * Rollout": the policy's router and predictor stay fixed while a batch is generated, so one
 * decode step follows another with the same W_r, A, B).  Same arguments, checks and results
 * as pr2_route_predict, except that the bf16 three-way split of the weights is not formed
 * again: the call reads the split that the previous pr2_route_predict (or _reuse) call on
 * this workspace left there.  The library keeps a host-side record per workspace address of
 * the split it holds (device, W_r, A, B pointers, d, N, r and the layout, which depends on the
 * NULL-ness of logits_out); any other call that takes the workspace drops the records inside
 * it.  The call returns PR2_ERR_WORKSPACE, with nothing enqueued, when ws holds no record or
 * one that differs from this call in any of those.  The caller still guarantees that the
 * VALUES of W_r, A and B did not change since the split was formed (only pointers are
 * compared).  Shapes that take the fp64 vector path keep no split and behave exactly as
 * pr2_route_predict.
 */
pr2_status pr2_route_predict_reuse(const pr2_moe_desc* desc, const void* x, const float* W_r,
                                   const float* b_r, const float* A, const float* B,
                                   void* idx_out, int64_t ldi, float* gate_out, float* logits_out,
                                   void* ws, size_t ws_bytes, pr2_stream_t stream);

/*
 * Route prediction that allocates nothing, for callers that cannot allocate device memory:
 * code being captured into a HIP graph, tight serving loops, harnesses that forbid it.
 * Same arguments (minus the workspace), checks and results as pr2_route_predict: the same
 * kernels, always the fused (non-split-K) form, whose logits are bitwise those of the split-K
 * form.  The bf16 split of the weights goes to a file-scope device array of 6 MiB that the
 * library holds on each GPU it runs on until the process ends; a shape whose split needs more
 * (3 x 2 bytes x d x the columns N, or N + r when logits_out is given, rounded up to 64)
 * returns PR2_ERR_UNSUPPORTED with nothing enqueued.  The call allocates and frees nothing;
 * its first call on a device looks up that device's copy of the array (make it outside a
 * capture).  Every call on a GPU shares that GPU's array: calls that overlap on one GPU (two
 * streams, two threads) race and give unspecified routes; order them on one stream.
 */
pr2_status pr2_route_predict_noalloc(const pr2_moe_desc* desc, const void* x, const float* W_r,
                                     const float* b_r, const float* A, const float* B,
                                     void* idx_out, int64_t ldi, float* gate_out,
                                     float* logits_out, pr2_stream_t stream);

/*
 * Replay forward during training (Sec. 4.1 "Replay During Training"; Eq. pr2_output;
 * Alg. 3 in Appendix D, its first two steps).  No fresh top-k: the recorded ids are used as
 * given, in any order; the weights come from the current router with the predictor bypassed:
 *
 *   p = x W_r + b_r,  g_{t,s} = softmax over the k recorded ids (renorm = 1) or rho of the
 *   softmax over all N (renorm = 0),
 *   y_t = sum_s g_{t,s} E_{idx[t,s]}(x_t),  E_j(h) = W_down_j (silu(W_gate_j h) * (W_up_j h)).
 *
 *   x        [T, d] act_dtype;  idx: token t's ids at idx + t*ldi (idx_dtype), ldi >= k
 *   W_r      [d, N] fp32;  b_r [N] fp32 or NULL
 *   W_gate   [N, m, d], W_up [N, m, d], W_down [N, d, m]   act_dtype
 *   y        [T, d] act_dtype (overwritten)
 *   gate_out [T, k] fp32 replay weights in idx's slot order; may be NULL.
 *   ws       >= pr2_workspace_bytes(desc, PR2_OP_REPLAY_FWD)
 * bf16 expert GEMMs use MFMA with fp32 accumulation; the SwiGLU activation is rounded to
 * act_dtype before the down projection and the weighted expert outputs are rounded to
 * act_dtype before the combine, which sums each token's k terms in slot order in fp32.
 */
pr2_status pr2_moe_replay_forward(const pr2_moe_desc* desc, const void* x, const void* idx,
                                  int64_t ldi, const float* W_r, const float* b_r,
                                  const void* W_gate, const void* W_up, const void* W_down,
                                  void* y, float* gate_out, void* ws, size_t ws_bytes,
                                  pr2_stream_t stream);

/*
 * Replay forward that also saves the experts' pre-activations for the backward (Sec. 4.1
 * "Replay During Training", Alg. 3: the training pass runs the replay forward and then its
 * backward under the same recorded routes).  Everything pr2_moe_replay_forward does, plus
 *
 *   au_out  [T*k, 2m] act_dtype, 16-byte aligned: row q holds a = x W_gate_e^T (first m) and
 *           u = x W_up_e^T (last m), rounded to act_dtype, for the q-th route in the
 *           library's expert-sorted order (a stable sort of the routes by expert id, which the
 *           backward forms again from the same ids).  Opaque to the caller: pass it unchanged
 *           to pr2_moe_replay_backward_saved with the same desc, x, idx, W_gate and W_up.
 *
 * y and gate_out are bitwise those of pr2_moe_replay_forward.  The saved rows are bitwise
 * what the backward would otherwise recompute, so the saved backward's gradients are bitwise
 * those of pr2_moe_replay_backward.  Same workspace and checks as pr2_moe_replay_forward, and
 * au_out NULL with T > 0 returns PR2_ERR_NULL, a misaligned au_out PR2_ERR_ALIGN (nothing
 * enqueued).
 */
pr2_status pr2_moe_replay_forward_save(const pr2_moe_desc* desc, const void* x, const void* idx,
                                       int64_t ldi, const float* W_r, const float* b_r,
                                       const void* W_gate, const void* W_up, const void* W_down,
                                       void* y, float* gate_out, void* au_out, void* ws,
                                       size_t ws_bytes, pr2_stream_t stream);

/*
 * Replay forward with the route-tracking diagnostics of Sec. 5.4 (top-k agreement, routing
 * deviation, route KL) formed in the same pass: the replay-weight epilogue already holds all N
 * current router logits of each token, so it also selects their top-k and compares it with the
 * recorded ids.  Everything pr2_moe_replay_forward does, plus (each output may be NULL):
 *
 *   p = x W_r + b_r (the replay router, predictor bypassed),  I = TopK(p, k) (ties to the lower
 *   id, decided on the fp32 logits)
 *   cur_idx_out [T, k] idx_dtype   I, ascending
 *   overlap_out [T] int32          |idx_t ∩ I_t|   (agreement = overlap / k, deviation = k - overlap)
 *   kl_out      [T] fp32           KL(softmax(p_t) || softmax(z_ref_t)), evaluated in fp64
 *   hist_out    [k + 1] uint64     tokens per deviation value, overwritten (8-byte aligned)
 *   z_ref       [T, N] fp32 reference logits (e.g. the rollout's predictive logits); needed only
 *               with kl_out
 * Same workspace, streams and checks as pr2_moe_replay_forward; y and gate_out are bitwise
 * those of pr2_moe_replay_forward, and the diagnostics bitwise those of pr2_route_diagnostics
 * on the same inputs.  T = 0 only zeroes hist_out.
 */
pr2_status pr2_moe_replay_forward_diag(const pr2_moe_desc* desc, const void* x, const void* idx,
                                       int64_t ldi, const float* W_r, const float* b_r,
                                       const void* W_gate, const void* W_up, const void* W_down,
                                       void* y, float* gate_out, const float* z_ref,
                                       void* cur_idx_out, int32_t* overlap_out, float* kl_out,
                                       uint64_t* hist_out, void* ws, size_t ws_bytes,
                                       pr2_stream_t stream);

/*
 * Rollout-phase layer forward (Sec. 4.1 "Route Prediction During Rollout"; Eq. pr2_old_output;
 * Alg. 2 in Appendix D): route prediction exactly as pr2_route_predict, then the layer output
 * under the predictive weights,
 *
 *   o_old,t = sum_s rho_hat_{t,s} E_{idx[t,s]}(x_t)
 *
 * with rho_hat renormalised over the k predicted ids (renorm = 1) or the softmax of the
 * predictive logits over all N (renorm = 0, the printed equation).  Arguments as for
 * pr2_route_predict and pr2_moe_replay_forward; idx_out and gate_out receive the recorded
 * route and its predictive weights (gate_out may be NULL).
 *   ws       >= pr2_workspace_bytes(desc, PR2_OP_ROLLOUT_FWD)
 */
pr2_status pr2_moe_rollout_forward(const pr2_moe_desc* desc, const void* x, const float* W_r,
                                   const float* b_r, const float* A, const float* B,
                                   const void* W_gate, const void* W_up, const void* W_down,
                                   void* idx_out, int64_t ldi, float* gate_out, float* logits_out,
                                   void* y, void* ws, size_t ws_bytes, pr2_stream_t stream);

/*
 * Replay backward (Sec. 4.1 "Replay During Training": the current experts and router are
 * trained through the replayed routes; Alg. 3 in Appendix D, its backward step).  Gradients
 * of L = sum_t <dy_t, y_t> for the replay forward above, with the recorded ids held fixed:
 *
 *   dg_ts = <dy_t, E_j(x_t)>                                        (j = idx[t, s])
 *   renorm = 1 (g = softmax over the k recorded logits):
 *     dp_t,j = g_ts (dg_ts - sum_s' g_ts' dg_ts') at the recorded ids, 0 at the others
 *   renorm = 0 (g_ts = rho_j of the softmax over all N logits, Eq. pr2_output as printed):
 *     dp_t,i = rho_ti ([i recorded] dg_ti - sum_s g_ts dg_ts) for every i < N (k <= 64)
 *   dW_r = sum_t x_t^T dp_t,  db_r = sum_t dp_t
 *   dW_gate_j, dW_up_j, dW_down_j = sums over the routes through expert j of the SwiGLU
 *   expert's weight gradients, each route's output scaled by g_ts
 *   dx_t = sum_s g_ts dE_j/dx(x_t)^T dy_t + dp_t W_r^T
 *
 * The predictor (A, B) is bypassed in replay and gets no gradient.  Arguments as for
 * pr2_moe_replay_forward, plus:
 *   dy       [T, d] act_dtype, gradient of the output y
 *   dx       [T, d] act_dtype (out)
 *   dW_r     [d, N] fp32 (out);  db_r [N] fp32 (out) or NULL when not wanted
 *   dW_gate  [N, m, d], dW_up [N, m, d], dW_down [N, d, m] fp32 (out), 16-byte aligned
 *   ws       >= pr2_workspace_bytes(desc, PR2_OP_REPLAY_BWD)
 * Every gradient is overwritten (not accumulated); an expert no route uses gets zeros, and
 * T = 0 writes zeros to all weight gradients (x, idx, dy, dx, ws may then be NULL).  Results
 * are bitwise deterministic.  With renorm = 0 the router gradients are dense over N (fp32
 * FMA passes over x and the [T, N] logit gradient) and k > 64 returns PR2_ERR_UNSUPPORTED.
 * The pre-activations
 * are recomputed (nothing is saved from the forward call); on the bf16 MFMA path
 * (d % 256 == 0, m % 256 == 0) a, u, their gradients, g H and the per-route input gradients
 * are held in bf16, with fp32 accumulation everywhere.
 */
pr2_status pr2_moe_replay_backward(const pr2_moe_desc* desc, const void* x, const void* idx,
                                   int64_t ldi, const float* W_r, const float* b_r,
                                   const void* W_gate, const void* W_up, const void* W_down,
                                   const void* dy, void* dx, float* dW_r, float* db_r,
                                   float* dW_gate, float* dW_up, float* dW_down, void* ws,
                                   size_t ws_bytes, pr2_stream_t stream);

/*
 * Replay backward from saved pre-activations: pr2_moe_replay_backward with the gate/up
 * pre-activations read from au_saved (written by pr2_moe_replay_forward_save with the same
 * desc, x, idx, W_gate and W_up) instead of recomputed by a grouped GEMM.  au_saved is only
 * read.  Same arguments otherwise, same workspace, bitwise the same gradients; au_saved NULL
 * with T > 0 returns PR2_ERR_NULL, a misaligned one PR2_ERR_ALIGN (nothing enqueued).  A
 * buffer not written by pr2_moe_replay_forward_save for these inputs gives wrong gradients
 * (nothing detects it).
 */
pr2_status pr2_moe_replay_backward_saved(const pr2_moe_desc* desc, const void* x, const void* idx,
                                         int64_t ldi, const float* W_r, const float* b_r,
                                         const void* W_gate, const void* W_up,
                                         const void* W_down, const void* au_saved,
                                         const void* dy, void* dx, float* dW_r, float* db_r,
                                         float* dW_gate, float* dW_up, float* dW_down, void* ws,
                                         size_t ws_bytes, pr2_stream_t stream);

/*
 * Route-tracking diagnostics (Sec. 5.4: top-k agreement, routing deviation and route KL) of a
 * recorded route against the current router, the predictor bypassed as in replay:
 *
 *   p = x W_r + b_r,  I = TopK(p, k)   (ties to the lower id, decided on the fp32 logits)
 *   overlap_t = |idx_t ∩ I_t|           (agreement = overlap / k, deviation = k - overlap)
 *   kl_t = KL(softmax(p_t) || softmax(z_ref_t))
 *   hist[v] = number of tokens whose deviation is v, v = 0..k
 *
 *   x, idx, ldi, W_r, b_r   as for pr2_moe_replay_forward (desc.m, desc.r, desc.renorm unused)
 *   z_ref        [T, N] fp32 reference logits, e.g. the rollout-time predictive logits; may be
 *                NULL when kl_out is NULL
 *   cur_idx_out  [T, k] idx_dtype, the current top-k ascending, or NULL
 *   overlap_out  [T] int32 or NULL;  kl_out [T] fp32 or NULL
 *   hist_out     [k + 1] uint64 (8-byte aligned), overwritten with exact counts, or NULL
 *   ws           >= pr2_workspace_bytes(desc, PR2_OP_ROUTE_DIAG)
 * The logits are the replay router's (exact bf16 x times fp32 W_r, one rounding to fp32); the
 * route KL is evaluated in fp64 from them.  T = 0 only zeroes hist_out.
 */
pr2_status pr2_route_diagnostics(const pr2_moe_desc* desc, const void* x, const void* idx,
                                 int64_t ldi, const float* W_r, const float* b_r,
                                 const float* z_ref, void* cur_idx_out, int32_t* overlap_out,
                                 float* kl_out, uint64_t* hist_out, void* ws, size_t ws_bytes,
                                 pr2_stream_t stream);

/*
 * Feature-cache positions (Appendix E.2, feature-cache paragraph: a fixed number Tc of token
 * positions per response keep their route-recording features, drawn by uniform
 * sub-sampling along the rollout).  HOST function, no device work: fills pos_out[0..n) with
 * n = min(T, Tc) increasing positions in [0, T): Tc >= T keeps every position; otherwise
 * position i is drawn uniformly inside the stratum [floor(i T / Tc), floor((i+1) T / Tc))
 * with the i-th output of SplitMix64 (Steele, Lea and Flood, 2014) for `seed`, so the cache
 * covers the whole rollout evenly.  Returns n, or -1 on a bad argument (pr2_last_error).
 */
int64_t pr2_feature_cache_positions(int64_t T, int64_t Tc, uint64_t seed, int64_t* pos_out);

/*
 * Route prediction with the feature-cache write fused in (Alg. 2 in Appendix D, its caching
 * step: the predicted ids go to the index cache and the retained tokens' route-recording
 * features (h_old, p_old) to the feature cache).  Same as pr2_route_predict with
 * logits_out = NULL, plus: token t with 0 <= cache_row[t] < cache_rows copies its input row
 * x_t to h_cache[cache_row[t]] ([cache_rows, d] act_dtype, 16-byte aligned) and writes its
 * router logits p_t (no predictor term) to p_cache[cache_row[t]] ([cache_rows, N] fp32);
 * tokens with any other cache_row value are not cached.  cache_row is a device int32 [T];
 * rows must be distinct.  ws >= pr2_workspace_bytes(desc, PR2_OP_ROUTE).
 */
pr2_status pr2_route_predict_cached(const pr2_moe_desc* desc, const void* x, const float* W_r,
                                    const float* b_r, const float* A, const float* B,
                                    void* idx_out, int64_t ldi, float* gate_out,
                                    const int32_t* cache_row, void* h_cache, float* p_cache,
                                    int64_t cache_rows, void* ws, size_t ws_bytes,
                                    pr2_stream_t stream);

/*
 * Evolution-predictor loss and gradients on the feature cache (Sec. 4.2, Eq. pr2_loss; Alg. 3
 * in Appendix D, its predictive-loss steps).  desc.T = number of cached tokens; desc.d, N, r
 * as for the layer (r >= 1); desc.k must be valid; m, idx_dtype and renorm are unused.
 *
 *   p_t = h_t W_r + b_r               the current router on the same tokens (teacher)
 *   zhat_t = p_old,t + h_old,t A B    rebuilt predictive logits
 *   loss_kind 0:  kl_t = KL(softmax(p_t) || softmax(zhat_t))                  (Eq. pr2_loss)
 *   loss_kind 1:  kl_t = KL(softmax(p_t - p_old,t) || softmax(h_old,t A B))   (delta matching,
 *                 the objective ablation of Appendix G)
 *   loss = mean_t kl_t;  dA, dB = gradients of loss (the router gets none: stop-gradient)
 *
 *   h, h_old   [T, d] act_dtype (16-byte aligned);  W_r [d, N], b_r [N] or NULL, p_old [T, N],
 *              A [d, r], B [r, N] fp32 (B NULL means the identity, needs r == N; dB unused)
 *   mini_step  1-based index of the update within the batch: mini_step == 1 is the
 *              on-policy first step, where the loss is skipped (zeros written, h, h_old, W_r,
 *              p_old and ws may be NULL)
 *   kl_out [T] fp32 or NULL;  loss_out [1] fp32;  dA [d, r], dB [r, N] fp32 (overwritten)
 *   ws         >= pr2_workspace_bytes(desc, PR2_OP_PREDICTOR_LOSS)
 * p is computed as by the replay router (exact products, one rounding to fp32); everything
 * after it, including the gradient sums over tokens, in fp64 with a fixed summation order.
 */
pr2_status pr2_predictor_loss(const pr2_moe_desc* desc, const void* h, const float* W_r,
                              const float* b_r, const void* h_old, const float* p_old,
                              const float* A, const float* B, int loss_kind, int mini_step,
                              float* kl_out, float* loss_out, float* dA, float* dB, void* ws,
                              size_t ws_bytes, pr2_stream_t stream);

/* Status name ("PR2_OK", ...); never NULL. */
const char* pr2_status_string(pr2_status s);
/* Detail of the last error on this thread ("" if none); valid until the next call. */
const char* pr2_last_error(void);
/* Library version string. */
const char* pr2_version(void);

/*
 * Measurement hooks (not part of the method).  While enabled, every kernel the library
 * enqueues is bracketed by a pair of HIP events recorded on the same stream.
 * pr2_profile_collect waits for the recorded events, adds each kernel's elapsed time to a
 * per-kernel-name total and fills up to `cap` entries of names / total_ms / launches,
 * returning the number of distinct kernel names seen since the last reset (or -1 on a HIP
 * error).  Names are static strings.  Not thread-safe; for single-threaded benchmarking.
 */
void pr2_profile_enable(int on);
void pr2_profile_reset(void);
int pr2_profile_collect(const char** names, double* total_ms, int64_t* launches, int cap);

#ifdef __cplusplus
}
#endif
#endif /* PR2_H */
