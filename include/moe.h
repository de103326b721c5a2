/*
 * moe.h - C ABI of libmoe, an MI355X (gfx950) implementation of one
 * capacity-bounded top-k Mixture-of-Experts layer with dynamic per-expert
 * capacities and a cached-assignment (gate bypass) path, forward and
 * backward.  Method: Kossmann, Jia, Aiken, "Optimizing Mixture of Experts
 * using Dynamic Recompilations" (MLSys 2022): Algorithm 1 (top-k MoE
 * forward), Eq. 1 (weighted sum of expert outputs), Eq. 4 and Section 4.1
 * (expert capacity, drops, dynamic capacity factors), Section 4.2 (sample
 * assignment caching), Eq. 3 (balance term), Eq. 2 and its appendix
 * (specification loss, AggregateSpec), Section 3 with its implementation
 * appendix (metric-driven changes at the launch frontier).
 *
 * Conventions shared by every call
 * --------------------------------
 * - `stream` is a hipStream_t (NULL = the legacy default stream).  Every
 *   call only enqueues work on it and never synchronises; results are
 *   ready when the stream reaches that point.
 * - Pointers are DEVICE pointers unless a parameter is marked [host].  The
 *   caller owns all memory, including scratch `workspace` buffers sized by
 *   the matching *_workspace_bytes query.  The library keeps no state
 *   beyond the capacity-policy objects the caller creates and destroys.
 * - Argument errors (bad sizes, NULL pointers, unsupported combinations,
 *   a workspace that is too small) are reported synchronously through the
 *   returned moe_status and nothing is enqueued.  Errors that depend on
 *   device data (bad cached ids, capacity regions that do not fit) never
 *   abort: the offending assignment is dropped and a bit is OR-ed into the
 *   caller's device `status` word (the caller zeroes it beforehand).
 * - Layer tensors (x, weights, activations, outputs) are row-major in the
 *   layer dtype `dt`: MOE_F32 (float) or MOE_BF16 (bf16 bit patterns,
 *   uint16).  Gate logits, probabilities, combine weights and every weight
 *   gradient are float32.  Accumulation is float32 in both dtypes.
 * - Weights are stored output-features x input-features, the layout of a
 *   linear map y = x W^T: w_g [E,d], w1 [E,f,d], w3 [E,f,d], w2 [E,d,f].
 * - Limits: 1 <= E <= 64, 1 <= k <= min(E, 8), T >= 0 (T = 0 is a valid
 *   empty batch), d, f >= 1 and multiples of 8, T*k and rows_alloc < 2^31.
 *   The expert FFN calls further need d and 2 f times the element size to
 *   stay below 2^23 bytes; larger requests are EINVAL.
 * - Every output is deterministic run to run (no floating-point atomics).
 */
#ifndef MOE_H_
#define MOE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MOE_OK = 0,
  MOE_EINVAL = 1,        /* bad size, NULL pointer or flag */
  MOE_EUNSUPPORTED = 2,  /* valid request the library does not implement */
  MOE_EHIP = 3,          /* a HIP launch failed */
  MOE_EWORKSPACE = 4     /* workspace NULL or smaller than the query said */
} moe_status;

typedef enum { MOE_F32 = 0, MOE_BF16 = 1 } moe_dtype;

typedef enum { MOE_RELU = 0, MOE_GELU_TANH = 1, MOE_SWIGLU = 2 } moe_act;

/* Bits OR-ed into the device status word. */
#define MOE_STATUS_BAD_ID 1 /* a cached expert id outside [0, E) */
#define MOE_STATUS_DUP_ID 2 /* a token names the same expert twice */
#define MOE_STATUS_REGION 4 /* an expert's capacity region does not fit */

/* Human-readable name of a moe_status value. [host] */
const char* moe_status_string(int status);

/* ABI version (incremented on incompatible change). [host] */
int moe_abi_version(void);

/*
 * moe_gate_topk - Algorithm 1, first three steps: score <- G(x),
 * indices <- argmax_k(score), (w_1..w_k) <- normalize(score[indices]),
 * for a linear gate G(x) = x w_g^T + bias.
 *   x       [T,d]  layer dtype
 *   w_g     [E,d]  layer dtype
 *   bias    [E]    float32, or NULL for no bias
 *   logits  [T,E]  float32 out: the gate scores
 *   ids     [T,k]  int32 out: the k largest logits per token, largest first;
 *                  equal logits go to the lower expert index
 *   weights [T,k]  float32 out: p = softmax(logits); renorm != 0 gives
 *                  p[ids]/sum p[ids] (the normalisation of Algorithm 1,
 *                  used for k >= 2); renorm == 0 gives the raw p[ids]
 *                  (Switch-style k = 1).
 */
moe_status moe_gate_topk(void* stream, moe_dtype dt, int T, int d, int E, int k,
                         int renorm, const void* x, const void* w_g,
                         const float* bias, float* logits, int32_t* ids,
                         float* weights);

/*
 * moe_count - the per-expert load that dynamic capacity factors follow
 * (Section 4.1: how many samples the gate assigns to each expert), before
 * any capacity is applied.
 *   ids    [T,k] int32 expert ids (gate output or cached)
 *   counts [E]   int32 out: live assignments per expert.  An id outside
 *                [0,E) is not counted (status bit 1); a repeat of an
 *                expert already named by the token at a lower j is not
 *                counted (status bit 2).
 *   status [1]   int32 in/out, bits OR-ed in.
 */
moe_status moe_count(void* stream, int T, int E, int k, const int32_t* ids,
                     int32_t* counts, int32_t* status);

/*
 * moe_update_capacity - Eq. 4 and Section 4.1: per-expert capacities and
 * the row layout of the grouped expert buffer.
 *   counts == NULL: static capacity factor alpha = num/den,
 *                   C_e = ceil(num*T*k / (den*E)) for every expert;
 *   counts != NULL: dynamic capacity factors, C_e = ceil(num*counts[e]/den)
 *                   (num/den is the margin over the observed load; 1/1 is
 *                   exact capacity).
 * Computed in exact 64-bit integer arithmetic, then clamped to [cap_min, T].
 *   capacity [E]   int32 out
 *   offsets  [E+1] int32 out: the row layout of the grouped buffers.
 *                  offsets[e] = sum over experts e' < e of C_e' rounded up
 *                  to a multiple of row_align, so expert e owns rows
 *                  [offsets[e], offsets[e]+C_e) and every region starts at
 *                  a multiple of row_align; offsets[E] is the rows the
 *                  layout needs (the caller's rows_alloc must be at least
 *                  that: at most sum C_e + E (row_align - 1)).  row_align = 1
 *                  packs the regions; 256 (one GEMM tile of rows) keeps each
 *                  expert's tiles aligned, which the FFN products run faster
 *                  on.  The layout changes where rows live, not which
 *                  assignments are kept.
 * num, den >= 1; cap_min >= 0; 1 <= row_align <= 1024.
 */
moe_status moe_update_capacity(void* stream, int T, int k, int E,
                               const int32_t* counts, int num, int den,
                               int cap_min, int row_align, int32_t* capacity,
                               int32_t* offsets);

/* Workspace bytes of moe_dispatch for these sizes. [host] */
size_t moe_dispatch_workspace_bytes(int T, int E, int k);

/*
 * moe_dispatch - GroupBy with the capacity/drop rule of Section 4.1: each
 * expert's tensor is filled from its first entry, assignments beyond the
 * expert's capacity are dropped.  Priority: all first choices in token
 * order, then all second choices, and so on.
 *   x         [T,d]          layer dtype
 *   ids       [T,k]          int32 expert ids (gate output or cached ids:
 *                            the gate-bypass path of Section 4.2)
 *   capacity  [E], offsets [E+1]  as written by moe_update_capacity
 *   rows_alloc                rows of the grouped buffers
 *   counts    [E]   out: live assignments per expert (as moe_count)
 *   fill      [E]   out: kept assignments per expert, min(counts, C_e)
 *   dest_row  [T,k] out: row of x_disp holding (t,j), or -1 if dropped
 *   src       [rows_alloc] out: t*k+j of the assignment in that row, or -1
 *   x_disp    [rows_alloc,d] out: x_disp[dest_row[t,j]] = x[t] (exact
 *             copy); rows without an assignment are left untouched.
 *   status    [1] in/out: bits 1, 2 as moe_count; bit 4 when an expert's
 *             region [offsets[e], offsets[e]+C_e) overlaps the next one or
 *             runs past rows_alloc (the region is cut to what fits).
 *   workspace moe_dispatch_workspace_bytes(T,E,k) bytes.
 */
moe_status moe_dispatch(void* stream, moe_dtype dt, int T, int d, int E, int k,
                        const void* x, const int32_t* ids,
                        const int32_t* capacity, const int32_t* offsets,
                        int64_t rows_alloc, int32_t* counts, int32_t* fill,
                        int32_t* dest_row, int32_t* src, void* x_disp,
                        int32_t* status, void* workspace,
                        size_t workspace_bytes);

/*
 * moe_dispatch_noalloc - moe_dispatch for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same arguments, results and errors,
 * without the workspace.  Its scratch (the routing histograms) is a fixed
 * device array inside the library, 1 MiB + 256 bytes, one copy per GPU,
 * held until the process ends.  The call allocates nothing.
 *   T*k must not exceed moe_dispatch_noalloc_max_assignments() (2^21);
 *   larger requests return MOE_EWORKSPACE and enqueue nothing.
 *   The stream must belong to the current device (else MOE_EINVAL).
 * Every call on one GPU uses that GPU's array: calls that overlap on one
 * GPU (other streams, other host threads) race and must be ordered by the
 * caller.  Nothing carries over between calls.
 */
moe_status moe_dispatch_noalloc(void* stream, moe_dtype dt, int T, int d, int E, int k,
                                const void* x, const int32_t* ids,
                                const int32_t* capacity, const int32_t* offsets,
                                int64_t rows_alloc, int32_t* counts, int32_t* fill,
                                int32_t* dest_row, int32_t* src, void* x_disp,
                                int32_t* status);

/* Largest T*k moe_dispatch_noalloc accepts. [host] */
size_t moe_dispatch_noalloc_max_assignments(void);

/* Workspace bytes of moe_expert_ffn_fwd / moe_expert_ffn_bwd. [host] */
size_t moe_ffn_fwd_workspace_bytes(moe_dtype dt, moe_act act, int E, int d,
                                   int f, int64_t rows_alloc);
size_t moe_ffn_bwd_workspace_bytes(moe_dtype dt, moe_act act, int E, int d,
                                   int f, int64_t rows_alloc);

/*
 * moe_expert_ffn_fwd - the expert modules E_e(x) of Algorithm 1, run on each
 * expert's own rows only (dynamically sized expert tensors, Section 4.1).
 * For expert e the rows are [offsets[e], offsets[e]+rows[e]) of the grouped
 * buffers; rows[e] is clamped to the expert's region and to rows_alloc.
 *   MOE_RELU / MOE_GELU_TANH: H = X w1_e^T, A = act(H), Y = A w2_e^T
 *   MOE_SWIGLU:  H1 = X w1_e^T, H3 = X w3_e^T, A = silu(H1)*H3, Y = A w2_e^T
 * bf16 layers round H (H1, H3), A and Y to bf16; A is computed from the
 * rounded H.  No bias.
 *   offsets [E+1], rows [E] int32 (rows = fill: the method; rows = capacity:
 *           a padded static-shape baseline)
 *   x_disp  [rows_alloc,d], w1/w3 [E,f,d] (w3 NULL unless SwiGLU), w2 [E,d,f]
 *   h_save  NULL for inference, else out: the planes moe_expert_ffn_bwd
 *           reads, each [rows_alloc,f]: ReLU A [1,rows_alloc,f]
 *           (relu'(H) = [A > 0], so H is not kept), GELU H, A
 *           [2,rows_alloc,f], SwiGLU H1, H3, A [3,rows_alloc,f] (A = act(H)
 *           as the second product consumed it).
 *   y_disp  [rows_alloc,d] out.  Rows outside every expert's rows are left
 *           untouched.
 */
moe_status moe_expert_ffn_fwd(void* stream, moe_dtype dt, moe_act act, int E,
                              int d, int f, const int32_t* offsets,
                              const int32_t* rows, int64_t rows_alloc,
                              const void* x_disp, const void* w1,
                              const void* w3, const void* w2, void* h_save,
                              void* y_disp, void* workspace,
                              size_t workspace_bytes);

/*
 * moe_zero_pad_rows - the padded static-shape baseline that Section 4.1
 * compares against: an expert tensor of fixed capacity whose first entries
 * hold the expert's samples and whose unused entries are zero, so they add
 * nothing to the weight gradients.  Writes zeros to rows
 * [offsets[e] + fill[e], offsets[e] + rows[e]) of buf for every expert,
 * with rows[e] clamped to the expert's region and to rows_alloc as the FFN
 * calls clamp it (fill[e] clamped to [0, rows[e]]).  Call it on x_disp after
 * moe_dispatch and on dy_disp after moe_combine_bwd (or moe_spec_loss)
 * before running the FFN with rows = capacity; the method itself
 * (rows = fill) never reads those rows and does not need it.
 *   offsets [E+1], fill [E], rows [E] int32
 *   buf     [rows_alloc,d] layer dtype, in/out; other rows untouched
 */
moe_status moe_zero_pad_rows(void* stream, moe_dtype dt, int E, int d,
                             const int32_t* offsets, const int32_t* fill,
                             const int32_t* rows, int64_t rows_alloc, void* buf);

/*
 * moe_combine - Aggregate (Algorithm 1's weighted sum, Eq. 1):
 * y[t] = sum over kept j, in order j = 0..k-1, of weights[t,j] *
 * y_disp[dest_row[t,j]], summed in float32 and rounded once.  A token with
 * no kept assignment gets 0 (dropped samples contribute nothing).
 *   y_disp [rows_alloc,d], dest_row [T,k], weights [T,k] f32, y [T,d] out.
 */
moe_status moe_combine(void* stream, moe_dtype dt, int T, int d, int k,
                       int64_t rows_alloc, const void* y_disp,
                       const int32_t* dest_row, const float* weights, void* y);

/*
 * moe_combine_bwd - backward of moe_combine.  Dropped assignments get zero
 * gradient (Section 4.1).
 *   dy       [T,d] upstream gradient
 *   dweights [T,k] f32 out: <dy[t], y_disp[dest_row[t,j]]> if kept, else 0
 *   dy_disp  [rows_alloc,d] out: dy_disp[dest_row[t,j]] = weights[t,j]*dy[t]
 *            (rounded to the layer dtype); other rows untouched.
 */
moe_status moe_combine_bwd(void* stream, moe_dtype dt, int T, int d, int k,
                           int64_t rows_alloc, const void* dy,
                           const void* y_disp, const int32_t* dest_row,
                           const float* weights, void* dy_disp,
                           float* dweights);

/*
 * moe_expert_ffn_bwd - backward of moe_expert_ffn_fwd over the same rows.
 *   dA = dY w2_e;  RELU/GELU: dH = dA * act'(H) (relu'(0) = 0);
 *   SWIGLU: dH1 = dA * H3 * silu'(H1), dH3 = dA * silu(H1)
 *   (bf16 layers round dH, dH1, dH3);
 *   dw2_e = dY^T A,  dw1_e = dH1^T X,  dw3_e = dH3^T X  (float32; an expert
 *   with no rows gets zeros);  dx_disp = dH1 w1_e + dH3 w3_e (one rounding).
 *   h_save   as written by moe_expert_ffn_fwd (A; H and A; or H1, H3 and A)
 *   dy_disp  [rows_alloc,d] (moe_combine_bwd output)
 *   dx_disp  [rows_alloc,d] out (rows outside every expert's rows untouched)
 *   dw1 [E,f,d], dw3 [E,f,d] (NULL unless SwiGLU), dw2 [E,d,f] float32 out,
 *   fully overwritten.
 */
moe_status moe_expert_ffn_bwd(void* stream, moe_dtype dt, moe_act act, int E,
                              int d, int f, const int32_t* offsets,
                              const int32_t* rows, int64_t rows_alloc,
                              const void* x_disp, const void* h_save,
                              const void* w1, const void* w3, const void* w2,
                              const void* dy_disp, void* dx_disp, float* dw1,
                              float* dw3, float* dw2, void* workspace,
                              size_t workspace_bytes);

/* Workspace bytes of moe_gate_bwd. [host] */
size_t moe_gate_bwd_workspace_bytes(int T, int d, int E);

/*
 * moe_gate_bwd - backward of moe_gate_topk through normalize() and the
 * softmax (top-k indices are piecewise constant: no gradient).
 *   raw (renorm = 0): g_j = dweights[t,j]
 *   renorm:           g_j = (dweights_j - sum_i dweights_i w_i) / S,
 *                     S = sum_j p[ids_j], w_j = p[ids_j]/S
 *   dp[t,e] = sum_j [ids[t,j] = e] g_j (+ dprob_coef[e]);
 *   dlogits = p * (dp - <dp, p>)
 *   dw_g[e,i] = sum_t dlogits[t,e] x[t,i]  (float32, fixed summation order)
 *   logits [T,E] (moe_gate_topk output), ids [T,k], dweights [T,k]
 *   dprob_coef [E] float32 or NULL: a gradient with respect to the
 *            probabilities that is the same for every token, such as the
 *            balance term's (moe_balance_fwd)
 *   dlogits [T,E] f32 out, dw_g [E,d] f32 out (fully overwritten).
 */
moe_status moe_gate_bwd(void* stream, moe_dtype dt, int T, int d, int E, int k,
                        int renorm, const void* x, const float* logits,
                        const int32_t* ids, const float* dweights,
                        const float* dprob_coef, float* dlogits, float* dw_g,
                        void* workspace, size_t workspace_bytes);

/*
 * moe_dispatch_bwd - backward of moe_dispatch plus the gate's input term:
 * dx[t] = sum over kept j of dx_disp[dest_row[t,j]]  (+ dlogits[t] . w_g
 * when dlogits and w_g are both non-NULL; both NULL on the cached path),
 * summed in float32, rounded once.  dx [T,d] out, fully overwritten.
 */
moe_status moe_dispatch_bwd(void* stream, moe_dtype dt, int T, int d, int E,
                            int k, int64_t rows_alloc, const void* dx_disp,
                            const int32_t* dest_row, const float* dlogits,
                            const void* w_g, void* dx);

/* ---- loss-side operators ------------------------------------------------ */

/* Workspace bytes of moe_balance_fwd. [host] */
size_t moe_balance_workspace_bytes(int T, int E);

/*
 * moe_balance_fwd - the balance term of Eq. 3, B = lambda * n * sum_i T_i G_i
 * over the n = E experts, with T_i = counts[i] / (T k) (the share of the
 * batch's assignments the gate gives expert i, counted before capacity) and
 * G_i = mean over the T tokens of softmax(logits[t])[i].  T_i comes from an
 * arg-top-k and has no gradient, so dB/dp[t,i] = lambda n T_i / T for every
 * token; pass dprob_coef to moe_gate_bwd to add it to the gate gradient.
 *   lambda     >= 0, finite (the regulariser's weight)
 *   logits     [T,E] float32 (moe_gate_topk output)
 *   counts     [E] int32 (moe_count / moe_dispatch output)
 *   loss       [1] float32 out: B (0 for T = 0)
 *   dprob_coef [E] float32 out: lambda n T_i / T
 * Sums run in a fixed order (per-256-token partials in the workspace, then
 * float64), so both outputs are deterministic.
 */
moe_status moe_balance_fwd(void* stream, int T, int E, int k, float lambda,
                           const float* logits, const int32_t* counts,
                           float* loss, float* dprob_coef, void* workspace,
                           size_t workspace_bytes);

/*
 * moe_aggregate_spec - the AggregateSpec operator of the specification-loss
 * appendix: the prediction of every (token, choice) pair, concatenated.
 *   out [T*k, d] layer dtype: row t*k + j = y_disp[dest_row[t,j]] when that
 *       assignment was kept, zeros when it was dropped (fully overwritten).
 */
moe_status moe_aggregate_spec(void* stream, moe_dtype dt, int T, int d, int k,
                              const void* y_disp, const int32_t* dest_row,
                              int64_t rows_alloc, void* out);

/* Workspace bytes of moe_spec_loss. [host] */
size_t moe_spec_loss_workspace_bytes(int T);

/*
 * moe_spec_loss - the specification loss of Eq. 2 with the squared error as
 * the task loss, L(y, o) = (1/d) sum_c (o_c - y_c)^2, averaged over tokens,
 * and both of its gradients, in one pass over the expert rows:
 *   loss          = (1/T) sum_t sum_{j kept} w[t,j] L(target[t], O[t,j])
 *   dweights[t,j] = L(target[t], O[t,j]) / T   (0 for a dropped assignment)
 *   dy_disp[r]    = w[t,j] * 2 (O[t,j] - target[t]) / (T d)   for r = dest_row[t,j]
 * with O[t,j] = y_disp[dest_row[t,j]].  A dropped assignment has no
 * prediction and takes no part.  dy_disp feeds moe_expert_ffn_bwd and
 * dweights feeds moe_gate_bwd, in place of moe_combine_bwd's outputs.
 *   target   [T,d] layer dtype;  weights [T,k] float32 (the combine weights)
 *   dy_disp  [rows_alloc,d] out: kept rows written, other rows untouched
 *   dweights [T,k] float32 out;  loss [1] float32 out (0 for T = 0)
 */
moe_status moe_spec_loss(void* stream, moe_dtype dt, int T, int d, int k,
                         const void* y_disp, const int32_t* dest_row,
                         const float* weights, const void* target,
                         int64_t rows_alloc, void* dy_disp, float* dweights,
                         float* loss, void* workspace, size_t workspace_bytes);

/* ---- sample assignment caching (Section 4.2) ------------------------------ */

/*
 * moe_cache_update - the Cache operator on one mini-batch: counts the
 * samples whose set of picked experts in fresh_ids equals the set cached for
 * them (order within a row does not matter), adds that number to
 * *unchanged, and writes fresh_ids to cache_out for the next epoch.
 *   fresh_ids [T,k] int32 (moe_gate_topk output)
 *   cached    [T,k] int32: the previous epoch's picks of these samples
 *   cache_out [T,k] int32 out: may be `cached` itself (in place); a separate
 *             buffer (one per epoch parity) lets the cached picks stay
 *             readable by the dispatch and the gate backward of the same
 *             iteration without ordering this call after them
 *   unchanged [1] int32 device counter, accumulated (the caller zeroes it at
 *             the start of an epoch); an integer sum, so deterministic
 */
moe_status moe_cache_update(void* stream, int T, int k, const int32_t* fresh_ids,
                            const int32_t* cached, int32_t* cache_out,
                            int32_t* unchanged);

/*
 * moe_cached_weights - combine weights for cached picks from the gate's
 * fresh scores: weights[t,j] = p[t, ids[t,j]], renorm != 0 divides by the
 * sum over the row's picks, p = softmax(logits[t]).  Evaluated exactly as
 * moe_gate_topk evaluates its weights, so picks equal to the gate's give
 * bit-identical weights.  An id outside [0,E) gets weight 0.
 *   logits [T,E] float32;  ids [T,k] int32;  weights [T,k] float32 out
 */
moe_status moe_cached_weights(void* stream, int T, int E, int k, int renorm,
                              const float* logits, const int32_t* ids,
                              float* weights);

/*
 * moe_caching_decision - the caching switch with hysteresis of Section 5.3:
 * off -> on when unchanged/samples >= on_num/on_den and epoch >= min_epoch;
 * on -> off when unchanged/samples < off_num/off_den (exact integer
 * comparison).  The paper's setting is 96/100, 90/100, epoch 10.  Returns
 * the new state (0 or 1), the old one for samples = 0, or -1 for invalid
 * arguments (a denominator <= 0, negative values, unchanged > samples).
 * [host]
 */
int moe_caching_decision(int enabled, int64_t unchanged, int64_t samples,
                         int epoch, int on_num, int on_den, int off_num,
                         int off_den, int min_epoch);

/* ---- capacity policy at the launch frontier (Section 3, Section 4.1) ------ */

/*
 * A host object that turns the per-expert assignment counts of past
 * iterations (the model metric) into per-expert capacities for the next
 * launch, without stalling the device.  Owned by the caller: create,
 * then per iteration moe_policy_begin before the launches that read the
 * capacities and moe_policy_end after the launch that produces the counts;
 * destroy at the end.  Not thread-safe; one stream per object.  It issues
 * host-device copies, so keep it out of HIP graph capture.
 *
 * Trigger (run on the host): with the counts c of iteration i - 1 - delta,
 * recompile when some c_e exceeds its capacity (drops) or some capacity
 * exceeds ceil(shrink c_e) clamped to [cap_min, T]; a recompile sets every
 * C_e = ceil(grow c_e) clamped to [cap_min, T].  Iterations 0..delta run
 * with init_cap.
 *
 * moe_policy_create: delta_launch in [0, 64] (iterations launched ahead of
 *   the metric the trigger sees); grow = grow_num/grow_den <= shrink =
 *   shrink_num/shrink_den, all in [1, 10^6]; row_align in [1, 1024] (the
 *   region alignment of moe_update_capacity); init_cap [host] [E] >= 0.
 *   Allocates pinned host memory and events.  *out = NULL on error.
 * moe_policy_begin: waits (host) until at most delta_launch iterations are
 *   outstanding, runs the trigger on each metric consumed, and enqueues on
 *   `stream` the upload of capacity [E] and offsets [E+1] (laid out as
 *   moe_update_capacity lays them out with row_align) when they changed or
 *   the buffers differ from the last call.  *rows_needed [host, optional] =
 *   offsets[E] (the rows the dispatch needs); *recompiled [host, optional] =
 *   1 if the capacities changed.  EINVAL when called twice without
 *   moe_policy_end.
 * moe_policy_end: enqueues on `stream` the copy of counts [E] (device) into
 *   the pinned ring and the event that marks it done.
 * moe_policy_state [host]: current capacities cap [E] (optional), iterations
 *   launched and consumed, recompiles so far.
 */
typedef struct moe_capacity_policy moe_capacity_policy;

/* The trigger alone, as the policy runs it: updates cap [host] [E] in place
 * from counts [host] [E]; returns 1 if it recompiled, 0 if not, -1 for
 * invalid arguments. [host] */
int moe_capacity_trigger(int T, int E, const int32_t* counts, int32_t* cap,
                         int grow_num, int grow_den, int shrink_num,
                         int shrink_den, int cap_min);

moe_status moe_policy_create(int T, int k, int E, int delta_launch, int grow_num,
                             int grow_den, int shrink_num, int shrink_den,
                             int cap_min, int row_align, const int32_t* init_cap,
                             moe_capacity_policy** out);
void moe_policy_destroy(moe_capacity_policy* p);
moe_status moe_policy_begin(moe_capacity_policy* p, void* stream, int32_t* capacity,
                            int32_t* offsets, int64_t* rows_needed, int* recompiled);
moe_status moe_policy_end(moe_capacity_policy* p, void* stream, const int32_t* counts);
moe_status moe_policy_state(const moe_capacity_policy* p, int32_t* cap,
                            int64_t* launched, int64_t* consumed,
                            int64_t* recompiles);

/*
 * Kernel timing (instrumentation; not part of the method).  While enabled,
 * every kernel the library launches is bracketed by two HIP events recorded
 * on the stream it is launched on.  moe_timing_report waits for the recorded
 * events, writes one line "name launches total_ms" per kernel name (in first
 * launch order) into buf [host, len bytes, NUL-terminated, truncated to fit],
 * clears the records and returns the number of names.  Off by default; leave
 * it off under HIP graph capture.  [host]
 */
moe_status moe_timing_enable(int on);
int moe_timing_report(char* buf, size_t len);

/*
 * Tile shape of the expert products (a tuning and testing aid; not part of
 * the method).  mode 0 (default): the library picks per product.  bf16: from
 * N, K, the row budget and E, between 256x256 tiles (one workgroup per CU)
 * and 128x128 tiles (two workgroups per CU) -- the latter for products with
 * few tiles per CU; both kernels add every output's products in the same
 * order, so results are identical bit for bit in every mode.  float32: the
 * forward products of small layers (at most 4096 blocks of 32x32 outputs
 * for the row budget) run one wavefront per 32x32 block, the others on
 * 256x256 tiles (the two add in different orders).  1: 256x256 only (both
 * dtypes); 2: 128x128 only (bf16; float32 as in mode 0).  Process-wide; read
 * when a product is launched.  Returns MOE_EINVAL for other modes. [host]
 */
moe_status moe_set_gemm_tiles(int mode);

/*
 * Operand layout of the bf16 dX product of moe_expert_ffn_bwd (a tuning and
 * testing aid; not part of the method).  dX contracts over f, the row index
 * of w1/w3, so it reads them K-major; it can instead read a transposed copy
 * that the call makes first in its workspace ([E, d, F] with F = 2f under
 * SwiGLU, bf16).  mode 0 (default): the copy when the row budget holds at
 * least 8192 rows per expert (rows_alloc >= 8192 E), where the faster
 * product outweighs the copy; 1: never; 2: always.  The products are
 * identical bit for bit either way.  moe_ffn_bwd_workspace_bytes includes
 * the copy's E*d*F*2 bytes when the current mode would make it; a call
 * whose workspace lacks them reads the weights K-major.  Process-wide; read
 * when moe_expert_ffn_bwd (or the workspace query) is called.  Returns
 * MOE_EINVAL for other modes. [host]
 */
moe_status moe_set_dx_weight_copy(int mode);

#ifdef __cplusplus
}
#endif

#endif /* MOE_H_ */
