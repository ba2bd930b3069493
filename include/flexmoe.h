/*
 * flexmoe.h -- C ABI of the FlexMoE masked MoE-layer forward for MI355X (gfx950).
 *
 * The library computes one MoE layer in which every routed expert e runs only
 * the first k_e channels of its importance-ranked intermediate dimension
 * (FlexMoE, Sec. 3.1, Eq. 4).  Ranking is a one-time channel permutation of
 * the expert weights (Eq. 3); a budget is the per-expert keep-count array
 * k[E] (the hardened action mask of Eqs. 9-10 expressed as channel counts).
 * Switching budgets rewrites only that array: no weight is moved, which is the
 * online clipping mode of Sec. 4.4 (Table 3).  Around that forward: the
 * offline-clipped mode (Table 2), the bucketed kernel design of App. C.3 as an
 * ablation, the channel saliency of Eq. 2 on the device, and one
 * action-learning step (Eqs. 5-8): sampled widths, the masked layer's
 * training forward and backward, and the action-logit gradient.
 *
 * General rules for every entry point
 *   - All pointers except the descriptor, the host keep table of
 *     flexmoe_set_budget and the debug-output struct are DEVICE pointers of the
 *     current HIP device.  The caller owns and allocates every buffer,
 *     including the forward workspace; the library allocates no device memory
 *     and keeps no device data between calls, except the static scratch array
 *     of flexmoe_layer_forward_noalloc (below).
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *     work is ordered after the work already queued on it, and later work
 *     queued on it is ordered after the call's work; no call synchronises the
 *     host.  A forward of a layer with a shared expert may run that expert's
 *     two GEMMs on a second stream of the same device (forked from `stream` by
 *     an event before routing, joined by an event before the combine): it does
 *     so for T <= 64 and while the shared expert's gate/up GEMM has fewer than
 *     1024 tiles (the training forwards and flexmoe_layer_forward_noalloc
 *     never do).  That stream, its two events and a mutex guarding the fork
 *     and join are process-wide state of the library: created on first use
 *     per device (default priority) and kept for the life of the process.
 *     Forwards on one device share them, so concurrent forwards on one device
 *     serialise their shared-expert GEMMs, and a graph capture of such a
 *     forward needs one eager call first (to create the stream).
 *   - Return value 0 = success, otherwise one of the negative FLEXMOE_E* codes;
 *     flexmoe_last_error() then returns a message (thread-local).  Argument
 *     checks happen on the host before any device work: a call that returns
 *     an argument error has enqueued nothing.  Device-resident data (logits,
 *     keep counts) is not inspected by the host; keep counts read on the device
 *     are clamped to [0, I] so that no access leaves its buffer.
 *   - No call allocates, frees, synchronises or sets memory with a memset:
 *     the calls can be captured into a HIP graph (the side stream joins the
 *     capture through its fork and join events; create it with one eager call
 *     before capturing).
 *   - x, weights and y must be 16-byte aligned; logits and keep arrays 4-byte
 *     aligned (FLEXMOE_EINVAL otherwise); the workspace 256-byte aligned.
 *
 * Element types: dtype FLEXMOE_F32 (x, weights and y in fp32) or FLEXMOE_BF16
 * (x, weights and y in bf16).  Router logits are always fp32.  Accumulation is
 * fp32; in bf16 mode the SwiGLU activations and each expert's down-projection
 * output are rounded to bf16, the weighted combine sums in fp32 and y is
 * rounded once at the end (round to nearest even throughout).
 *
 * Shape rules (FLEXMOE_ESHAPE otherwise): d, I and I_shared are multiples of
 * 8; 1 <= E <= 256; 1 <= top_k <= min(E, 16); E * I < 2^31; 0 <= T <=
 * max_tokens; max_tokens * (top_k + 1) <= 2^30.  In bf16 mode every operand block one
 * GEMM tile addresses stays below 2^30 elements: max_tokens * d,
 * max_tokens * I, max_tokens * I_shared, I * d and I_shared * d (the prefill
 * kernels reach their operands through 32-bit buffer offsets).
 */
#ifndef FLEXMOE_H
#define FLEXMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    FLEXMOE_OK = 0,
    FLEXMOE_EINVAL = -1,     /* null pointer, negative count, bad flag value   */
    FLEXMOE_ESHAPE = -2,     /* dimension rule broken, T > max_tokens           */
    FLEXMOE_EKEEP = -3,      /* a host keep count outside [0, I]                */
    FLEXMOE_EWORKSPACE = -4, /* workspace missing or smaller than required      */
    FLEXMOE_EDTYPE = -5,     /* dtype is neither FLEXMOE_F32 nor FLEXMOE_BF16   */
    FLEXMOE_EHIP = -6        /* a HIP call or kernel launch failed              */
};

typedef enum { FLEXMOE_F32 = 0, FLEXMOE_BF16 = 1 } flexmoe_dtype;

/* Static description of one MoE layer. */
typedef struct flexmoe_layer_desc {
    int32_t d;          /* hidden size                                          */
    int32_t E;          /* routed experts                                       */
    int32_t I;          /* intermediate channels per routed expert (d_ff)       */
    int32_t top_k;      /* experts per token                                    */
    int32_t I_shared;   /* channels of the one unpruned shared expert, 0 = none */
    int32_t dtype;      /* flexmoe_dtype of x, weights and y                    */
    int32_t norm_topk;  /* 1: router weights renormalised over the top-k;
                           0: raw softmax probabilities                         */
    int32_t max_tokens; /* largest T a forward will be called with              */
} flexmoe_layer_desc;

/* Optional copies of the routing and dispatch results (device pointers; any
 * field may be NULL).  They are written on `stream` at the end of a forward.
 *   topk_idx [T][top_k] int32  expert ids, slot j = j-th largest logit
 *   topk_w   [T][top_k] fp32   router weights
 *   counts   [E]        int32  tokens routed to each expert (k_e = 0 included)
 *   offsets  [E+1]      int32  segment starts of the active experts (k_e > 0)
 *                              in perm; offsets[E] = P
 *   perm     [T*top_k]  int32  assignment ids a = t*top_k + j grouped by
 *                              expert, ascending a inside an expert; entries
 *                              at and past P are unspecified
 *   pos      [T*top_k]  int32  slot of assignment a in perm, -1 if k_e = 0 */
typedef struct flexmoe_route_out {
    int32_t *topk_idx;
    float *topk_w;
    int32_t *counts;
    int32_t *offsets;
    int32_t *perm;
    int32_t *pos;
} flexmoe_route_out;

/* Bytes of device workspace flexmoe_layer_forward needs for T tokens
 * (T <= desc->max_tokens).  Returns 0 and sets the last error when the
 * descriptor or T is invalid.  A workspace sized for max_tokens serves every
 * smaller T. */
size_t flexmoe_workspace_bytes(const flexmoe_layer_desc *desc, int32_t T);

/* One-time channel ranking and reorder (Sec. 3.1, Eq. 3).
 *   scores  [E][I] fp32   channel saliency (Eq. 2); larger = more important
 *   w_gate, w_up [E][I][d]  original weights, rows = channels
 *   w_down  [E][d][I]       original weights, columns = channels
 *   w_gate_r, w_up_r [E][I][d], w_down_r [E][d][I]  ranked outputs (must not
 *                           overlap the inputs)
 *   perm    [E][I] int32  output: ranked channel c holds original channel
 *                         perm[e][c]
 * The order is a stable descending sort of the scores: equal scores keep the
 * lower original index first; NaN scores order after every number.  The same
 * permutation is applied to gate rows, up rows and down columns, so the
 * unpruned expert function is unchanged.  Uses desc->d, E, I and dtype. */
int flexmoe_rank_reorder(const flexmoe_layer_desc *desc, const float *scores,
                         const void *w_gate, const void *w_up, const void *w_down,
                         void *w_gate_r, void *w_up_r, void *w_down_r, int32_t *perm,
                         void *stream);

/* ---- Channel saliency on the device (Sec. 3.1, Eq. 2) --------------------
 * The first-order Taylor saliency of every hidden channel of every routed
 * expert, for one calibration batch, added into a running score table:
 *   scores[e][j] += scale * sum over theta in {W_gate[e][j][:], W_up[e][j][:],
 *                                              W_down[e][:][j]} of (theta * dL/dtheta)^2
 * The loss is the layer-level L = 1/2 sum_t ||Y_t - y_target_t||^2 of the
 * UNPRUNED layer (every k_e = I) on this batch; the paper's language-model
 * loss needs a whole model and is out of this library's scope.  Router
 * weights come from the logits (not trained); the shared expert contributes
 * to Y but is not scored.  With scale = 1/|B_rank| over the calibration
 * batches, scores ends as Eq. 2's mean; flexmoe_rank_reorder then sorts it.
 *   x [T][d], weights (original order) as for flexmoe_rank_reorder, shared
 *   weights as for the forward (or NULL iff I_shared == 0), logits [T][E] fp32,
 *   y_target [T][d] fp32 (16-byte aligned), scores [E][I] fp32 (4-byte
 *   aligned; read and written, on `stream`).
 * bf16 layers only (FLEXMOE_EDTYPE otherwise).  Arithmetic: fp32 accumulation
 * in every GEMM; g, u, h, dO = w*dY, dG and dU are rounded to bf16 as MFMA
 * operands; Y and dY stay fp32; the squares and their sums are fp32, summed in
 * a fixed order (repeated calls give identical bits).
 * w_down_t: W_down^T [E][I][d] as written by flexmoe_transpose_weights, or
 * NULL, in which case every call writes that copy into its workspace (a
 * ranking set of several batches makes it once and passes it).
 * Workspace: flexmoe_saliency_workspace_bytes(desc, T), 256-byte aligned; it
 * holds room for that copy (E*I*d bf16) besides per-token buffers.
 * Shapes: the bf16 rules of the forward, and
 * max(d, I) * (T*top_k + 7*E rounded up to 8) < 2^30 (FLEXMOE_ESHAPE). */
size_t flexmoe_saliency_workspace_bytes(const flexmoe_layer_desc *desc, int32_t T);
int flexmoe_channel_saliency(const flexmoe_layer_desc *desc, int32_t T, const void *x,
                             const float *logits, const void *w_gate, const void *w_up,
                             const void *w_down, const void *w_down_t, const void *ws_gate,
                             const void *ws_up, const void *ws_down, const float *y_target,
                             float scale, float *scores, void *workspace,
                             size_t workspace_bytes, void *stream);

/* ---- Action learning on the device (Sec. 3.2, Eqs. 5-8) ------------------
 * One training step of the per-expert width actions of a layer:
 *   1. flexmoe_sample_actions: the hard straight-through Gumbel-softmax
 *      sample (Eq. 5) of one action per expert, written as a device keep
 *      table (no host round trip);
 *   2. flexmoe_train_forward: the sampled subnet's forward (the masked layer
 *      at that keep table), keeping what the backward needs in the workspace;
 *   3. flexmoe_train_backward: for an upstream gradient dY, the input
 *      gradient dx, the router-logit gradient and the mask gradient
 *      dM[e][c] = dL/dM_{e,c} of the prefix mask (every channel c < I);
 *   4. flexmoe_action_grad: the action-logit gradient through the
 *      straight-through estimator (Eq. 6) plus lambda_cost times the
 *      load-weighted cost of Eq. 7 minus beta times the entropy of the clean
 *      action distribution, with the cost and entropy values.
 * The weights are frozen (only the action logits learn), so their gradients
 * are not formed; the transposed copies the backward reads are made once by
 * flexmoe_transpose_weights.  bf16 layers only (FLEXMOE_EDTYPE otherwise).
 *
 * Actions: K <= FLEXMOE_MAX_ACTIONS retention ratios r_k in (0, 1]
 * (FLEXMOE_EINVAL otherwise); action k keeps ceil(r_k I) channels
 * (flexmoe_keep_from_ratio), at least one.  alpha, gumbel [E][K] fp32 on the
 * device; gumbel holds the caller's Gumbel(0, 1) draws.  The hard sample is
 * argmax_k (alpha + gumbel) in fp32, the first index on ties (the softmax of
 * Eq. 5 is monotone in its argument). */
#define FLEXMOE_MAX_ACTIONS 16
typedef struct flexmoe_action_set {
    int32_t K;
    double ratio[FLEXMOE_MAX_ACTIONS];   /* fp64, so that the widths ceil(r I)
                                            are those of the decimal ratios */
} flexmoe_action_set;

/* Transposed weight copies: w_gate_t, w_up_t [E][d][I]; w_down_t [E][I][d];
 * ws_gate_t, ws_up_t [d][I_s]; ws_down_t [I_s][d].  Each (input, output) pair
 * is given or NULL together (the training backward needs all of them; the
 * saliency only the down one); shared pairs only if I_s > 0.  Outputs must not
 * overlap inputs. */
int flexmoe_transpose_weights(const flexmoe_layer_desc *desc, const void *w_gate, const void *w_up,
                              const void *w_down, const void *ws_gate, const void *ws_up,
                              const void *ws_down, void *w_gate_t, void *w_up_t, void *w_down_t,
                              void *ws_gate_t, void *ws_up_t, void *ws_down_t, void *stream);

/* Eq. 5: keep_dev[e] = ceil(r_{k*} I) with k* = argmax_k (alpha + gumbel);
 * action_dev [E] int32 receives k* (may be NULL). */
int flexmoe_sample_actions(const flexmoe_layer_desc *desc, const flexmoe_action_set *actions,
                           const float *alpha, const float *gumbel, int32_t *keep_dev,
                           int32_t *action_dev, void *stream);

/* Workspace of flexmoe_train_forward/backward/action_grad for T tokens.  The
 * forward writes it and the other two read it: keep it, and T and logits,
 * unchanged between the calls of one step. */
size_t flexmoe_train_workspace_bytes(const flexmoe_layer_desc *desc, int32_t T);

/* The masked layer's forward at keep_dev (any 0 <= k_e <= I; an expert at 0
 * is skipped and gets no mask gradient), y [T][d] bf16 as from
 * flexmoe_layer_forward.  The gate/up GEMM computes every channel (the mask
 * gradient needs g and u past the prefix); the down GEMM only the kept ones. */
int flexmoe_train_forward(const flexmoe_layer_desc *desc, int32_t T, const void *x,
                          const float *logits, const void *w_gate, const void *w_up,
                          const void *w_down, const int32_t *keep_dev, const void *ws_gate,
                          const void *ws_up, const void *ws_down, void *y, void *workspace,
                          size_t workspace_bytes, void *stream);

/* Backward of the forward above for dy [T][d] fp32 = dL/dY:
 *   dx [T][d] fp32        dL/dx through the routed experts (kept channels)
 *                         and the shared expert;
 *   dlogits [T][E] fp32   dL/dlogits through the router weights (softmax over
 *                         all E, then the top-k renormalisation if norm_topk);
 *   dmask [E][I] fp32     dL/dM_{e,c} = sum over e's tokens of
 *                         dh'_c silu(g_c) u_c, dh' = w dY W_down (every c).
 * Arithmetic: fp32 accumulation; dO = w*dY, dY (shared), g, u, dG, dU are
 * rounded to bf16 as MFMA operands; fixed summation orders. */
int flexmoe_train_backward(const flexmoe_layer_desc *desc, int32_t T, const float *logits,
                           const float *dy, const void *w_gate_t, const void *w_up_t,
                           const void *w_down_t, const void *ws_gate_t, const void *ws_up_t,
                           const void *ws_down_t, float *dx, float *dlogits, float *dmask,
                           void *workspace, size_t workspace_bytes, void *stream);

/* Eqs. 6-8 for this layer: dalpha [E][K] fp32 = (1/tau) z (dz - <z, dz>)
 * with z = softmax((alpha + gumbel) / tau) and dz_k = sum_{c < ceil(r_k I)}
 * dmask[e][c], plus lambda_cost q_e p_k (r_k - <p, r>) and
 * beta p_k (log p_k + H_e) / E, where p = softmax(alpha),
 * H_e = -<p, log p> and q_e = n_e / (T top_k) from the forward's routing.
 * stats (may be NULL) [2] fp32 receives C = sum_e q_e <p_e, r> and
 * H = mean_e H_e.  tau > 0 (FLEXMOE_EINVAL otherwise).  The workspace is the
 * step's training workspace: its routing counts are read and a small region
 * of it is written. */
int flexmoe_action_grad(const flexmoe_layer_desc *desc, int32_t T, const flexmoe_action_set *actions,
                        const float *alpha, const float *gumbel, float tau, float lambda_cost,
                        float beta, const float *dmask, float *dalpha, float *stats,
                        void *workspace, size_t workspace_bytes, void *stream);

/* Budget switch (online clipping, Sec. 4.4 and Table 3: a new budget is a new
 * per-expert width table, the hardened action mask of Eqs. 9-10 as channel
 * counts, applied without moving any weight).
 * Validates 0 <= keep_host[e] <= I for every e on the host, then
 * writes the E counts into keep_dev [E] on `stream` (one small kernel whose
 * arguments carry the table, so keep_host may be reused as soon as the call
 * returns).  A forward queued later on the same stream sees the new budget.
 * Holding several device keep tables and passing a different keep_dev pointer
 * to the forward is an equally valid zero-copy switch. */
int flexmoe_set_budget(const flexmoe_layer_desc *desc, int32_t *keep_dev,
                       const int32_t *keep_host, void *stream);

/* Masked MoE-layer forward (Eq. 4 inside a top-k MoE layer; App. C.3).
 *   x        [T][d]            hidden states (dtype)
 *   logits   [T][E] fp32       router logits
 *   w_gate_r, w_up_r [E][I][d] ranked weights; channel c of expert e is used
 *                              iff c < keep_dev[e]
 *   w_down_r [E][d][I]         ranked down projection (columns = channels)
 *   keep_dev [E] int32         keep counts k_e (k_e = 0: the expert is skipped
 *                              and contributes exactly 0)
 *   ws_gate, ws_up [I_shared][d], ws_down [d][I_shared]  shared expert
 *                              (NULL iff I_shared = 0), added with weight 1
 *   y        [T][d]            output (dtype)
 *   workspace / workspace_bytes  device scratch of at least
 *                              flexmoe_workspace_bytes(desc, T) bytes, 256-byte
 *                              aligned; its contents are clobbered
 *   dbg                        optional routing/dispatch copies (may be NULL)
 * Routing: softmax over all E logits; the top_k experts by (logit descending,
 * expert id ascending; NaN last) are selected; with norm_topk their weights are
 * divided by their sum.  y[t] = sum_j w[t][j] * FFN_{e_j}^{(k_e)}(x[t]) + shared.
 * T = 0 is a valid no-op.  Deterministic: the same inputs give the same bits. */
int flexmoe_layer_forward(const flexmoe_layer_desc *desc, int32_t T, const void *x,
                          const float *logits, const void *w_gate_r, const void *w_up_r,
                          const void *w_down_r, const int32_t *keep_dev, const void *ws_gate,
                          const void *ws_up, const void *ws_down, void *y, void *workspace,
                          size_t workspace_bytes, const flexmoe_route_out *dbg, void *stream);

/* No-allocation forward, for callers that cannot allocate device memory or
 * pass a workspace: code under HIP graph capture, tight serving loops, and
 * harnesses that forbid allocation.  Arguments, results, rules and errors are
 * those of flexmoe_layer_forward, without the workspace: the workspace
 * regions live in a static device array of the library (64 MiB per device,
 * held by every device the library runs on until the process ends), so T is
 * limited to what fits there (flexmoe_workspace_bytes(desc, T) up to about
 * 64 MiB: every T <= 64 of the shapes this library is measured on, and a
 * few hundred to a thousand tokens of them).  A larger T returns
 * FLEXMOE_EWORKSPACE with nothing enqueued.  The array's device address is
 * looked up on the first call on each device; after that the call allocates
 * nothing, creates no stream or event (unless per-kernel timing is on) and
 * issues no memset.  Every launch goes to `stream`: the shared expert's GEMMs
 * run in the same launches as the routed experts' (no second stream), so the
 * bits of y may differ from flexmoe_layer_forward's by the summation order of
 * the shared expert (routing and dispatch outputs are identical).  All calls
 * on one device share the one array, which keeps the last call's contents
 * (nothing in it needs to start at zero): calls that overlap on one device,
 * on different streams or threads, race and give wrong results; order them. */
int flexmoe_layer_forward_noalloc(const flexmoe_layer_desc *desc, int32_t T, const void *x,
                                  const float *logits, const void *w_gate_r, const void *w_up_r,
                                  const void *w_down_r, const int32_t *keep_dev, const void *ws_gate,
                                  const void *ws_up, const void *ws_down, void *y,
                                  const flexmoe_route_out *dbg, void *stream);

/* ---- Offline clipping (Sec. 4.4, Table 2): one budget exported as a
 * standalone compact subnetwork, run by the same kernels.
 *
 * Clipped layout of a budget k[E]: expert e keeps kp_e = ceil8(k_e) channels
 * (k_e rounded up to a multiple of 8, so every packed row is 16-byte
 * aligned), and the experts' blocks follow one another in expert order:
 *   w_gate_c, w_up_c  expert e's block [kp_e][d]: row c < k_e = ranked row c,
 *                     rows k_e .. kp_e-1 are zero
 *   w_down_c          expert e's block [d][kp_e]: column c < k_e = ranked
 *                     column c, the other columns are zero
 * Expert e's blocks start at element ch0_e * d of each buffer, ch0_e =
 * sum_{e' < e} kp_e'.  Each buffer holds P * d elements of dtype, P =
 * flexmoe_clipped_channels(desc, k).  Experts with k_e = 0 hold nothing.
 *
 * flexmoe_clipped_channels: P for the keep table keep_host [E] (host array);
 *   FLEXMOE_EKEEP if some k_e is outside [0, I], another negative code for
 *   a bad descriptor or NULL table.
 * flexmoe_export_clipped: packs the ranked weights (layouts of
 *   flexmoe_layer_forward) into caller-allocated buffers of P * d elements
 *   each, on `stream`.  keep_host is validated on the host and may be reused
 *   when the call returns.  The ranked buffers are only read.
 * flexmoe_layer_forward_clipped: flexmoe_layer_forward over the packed
 *   weights.  keep_dev must hold the exported budget; packed_channels = P.
 *   Results equal those of flexmoe_layer_forward on the ranked weights with
 *   the same keep counts, bit for bit.  Device keep counts are not trusted
 *   for addressing: an expert whose packed block would end past
 *   packed_channels is skipped (as if k_e = 0), so a wrong table yields a
 *   wrong result but never an access outside the buffers.
 *   FLEXMOE_EINVAL if packed_channels is outside [0, E * ceil8(I)]; every
 *   other rule and error of flexmoe_layer_forward applies. */
int64_t flexmoe_clipped_channels(const flexmoe_layer_desc *desc, const int32_t *keep_host);
int flexmoe_export_clipped(const flexmoe_layer_desc *desc, const int32_t *keep_host,
                           const void *w_gate_r, const void *w_up_r, const void *w_down_r,
                           void *w_gate_c, void *w_up_c, void *w_down_c, void *stream);
int flexmoe_layer_forward_clipped(const flexmoe_layer_desc *desc, int32_t T, const void *x,
                                  const float *logits, const void *w_gate_c, const void *w_up_c,
                                  const void *w_down_c, const int32_t *keep_dev,
                                  int64_t packed_channels, const void *ws_gate, const void *ws_up,
                                  const void *ws_down, void *y, void *workspace,
                                  size_t workspace_bytes, const flexmoe_route_out *dbg,
                                  void *stream);

/* Bucketed forward (App. C.3, Alg. 2), kept as an ablation of the ragged
 * design of flexmoe_layer_forward: the routed experts are grouped by retained
 * width k_e (widest group first), and each group's gate/up and down GEMMs run
 * as their own launch pair over AlignUp(k_e, k_align) channels (capped at I):
 * the extra channels are computed with the ranked weights and their
 * activations zeroed before the down projection, as the paper does.  The
 * widths are read from keep_host [E] (a host array, validated on the host:
 * FLEXMOE_EKEEP outside [0, I]); k_align >= 1 (FLEXMOE_EINVAL otherwise).
 * The workspace of flexmoe_workspace_bytes serves this call too.  Results
 * equal those of flexmoe_layer_forward with keep_dev = keep_host (the padded
 * channels contribute exact zeros); every other argument, rule and error is
 * that of flexmoe_layer_forward. */
int flexmoe_layer_forward_bucketed(const flexmoe_layer_desc *desc, int32_t T, const void *x,
                                   const float *logits, const void *w_gate_r, const void *w_up_r,
                                   const void *w_down_r, const int32_t *keep_host, int32_t k_align,
                                   const void *ws_gate, const void *ws_up, const void *ws_down,
                                   void *y, void *workspace, size_t workspace_bytes,
                                   const flexmoe_route_out *dbg, void *stream);

/* k = ceil(r * I) for a retention ratio r in [0, 1] (Sec. 3.1).  A slack of
 * 1e-9 absorbs the binary representation error of decimal ratios (0.7 * 1000
 * gives 700).  Returns -1 for r outside [0, 1], NaN, or I < 1. */
int flexmoe_keep_from_ratio(double r, int32_t I);

/* Per-kernel timing, a measurement aid for benchmarks.  flexmoe_timing_enable(1)
 * clears the accumulators and makes every later forward record a HIP event
 * pair around each of its kernels, on the forward's stream;
 * flexmoe_timing_enable(0) stops recording.  flexmoe_timing_read waits for
 * every recorded event, writes the summed durations (milliseconds) and launch
 * counts per kernel into *out (indexed by FLEXMOE_K_*) and clears the
 * accumulators.  Recording costs two event records per kernel; it creates
 * events (host-side HIP objects) on first use and reuses them afterwards. */
enum {
    FLEXMOE_K_ROUTE = 0,          /* top-k routing + chunk histograms          */
    FLEXMOE_K_DISPATCH_SCAN = 1,  /* per-expert scan of the histograms         */
    FLEXMOE_K_DISPATCH_SCATTER = 2, /* stable permutation, segment/tile tables */
    FLEXMOE_K_GATE_UP = 3,        /* gate/up GEMM with fused SwiGLU            */
    FLEXMOE_K_DOWN = 4,           /* down GEMM                                 */
    FLEXMOE_K_COMBINE = 5,        /* weighted combine + shared add             */
    FLEXMOE_K_GATE_UP_SHARED = 6, /* gate/up GEMM of the shared expert         */
    FLEXMOE_K_DOWN_SHARED = 7,    /* down GEMM of the shared expert            */
    FLEXMOE_K_SAL_TRANSPOSE = 8,  /* saliency: transposed down-weight copy     */
    FLEXMOE_K_SAL_PREP = 9,       /* saliency: transposed x and dO copies      */
    FLEXMOE_K_SAL_DGRAD = 10,     /* saliency: dgrad GEMM + SwiGLU backward    */
    FLEXMOE_K_SAL_WGRAD = 11,     /* saliency: wgrad GEMMs + Eq. 2 reduction   */
    FLEXMOE_K_SAL_REDUCE = 12,    /* saliency: sum of the partial scores       */
    FLEXMOE_K_ACT_DGRAD = 13,     /* training: dgrad + SwiGLU bwd + mask grad  */
    FLEXMOE_K_ACT_DX = 14,        /* training: input-gradient GEMMs            */
    FLEXMOE_K_ACT_OTHER = 15,     /* training: sampling, prep, combine bwd,
                                     mask sums, action gradient              */
    FLEXMOE_K_COUNT = 16
};
typedef struct flexmoe_kernel_times {
    double ms[FLEXMOE_K_COUNT];
    int64_t launches[FLEXMOE_K_COUNT];
} flexmoe_kernel_times;
int flexmoe_timing_enable(int on);
int flexmoe_timing_read(flexmoe_kernel_times *out);

/* Message for the last non-zero return on this thread ("" if none). */
const char *flexmoe_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* FLEXMOE_H */
