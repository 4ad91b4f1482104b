/*
 * dmoe.h -- C ABI of libdmoe.so: one Decentralized Mixture-of-Experts layer
 * (Ryabinin & Gusev, arXiv 2002.04013), forward and backward, on one gfx950 GPU.
 *
 * The layer (Sec. 3.1, Sec. 3.2, Eq. 1):
 *   experts sit on a d-dimensional grid, expert f has uid (u_0 .. u_{d-1}), u_i in [0, M);
 *   the gate is d linear layers g_i : R^D -> R^M and scores expert f by
 *       g(x, f) = sum_i g_i(x)[u_i];
 *   TopK(x) are the k experts with the highest g (ties: lower flat index);
 *   DMoE(x) = sum_{f in TopK(x)} f(x) exp(g(x,f)) / sum_{f' in TopK(x)} exp(g(x,f')),
 *   with experts that do not respond excluded and the remaining weights
 *   renormalised to sum to 1 (Sec. 3.2).
 * Each expert is the feed-forward block f(x) = W2 act(W1 x + b1) + b2 (Sec. 4.1), or the
 * block with layer normalisation of the dmoe_expert_ffblock_* entry points below.
 *
 * Conventions shared by every entry point
 *   - Every array pointer is a DEVICE pointer, row-major, owned by the caller.
 *     The library allocates nothing, frees nothing and never synchronises; all
 *     work is enqueued on `stream` (a hipStream_t passed as void*; NULL = the
 *     default stream).  Results are ready when the stream reaches them.
 *   - Flat expert index: flat = sum_i u_i * M^(d-1-i) (u_0 most significant).
 *     N = M^d experts; gate column c = i*M + u belongs to grid dimension i.
 *   - dtype DMOE_BF16: x, gate and expert weights/biases, activations, outputs
 *     and their gradients are bf16 (uint16 bit patterns); all arithmetic
 *     accumulates in fp32 (gate scores in fp64).  DMOE_F32: all of those are fp32.
 *     w, dw, dg, g and scores are always fp32; indices are int32; alive is uint8.
 *   - "pairs": pair p = t*k + j is token t's j-th chosen expert.  P_max = T*k.
 *   - Buffers are sized for P_max rows; the number of rows actually used,
 *     offsets[N], stays on the device (no host synchronisation on the path).
 *   - Results are bitwise reproducible from run to run (no floating-point atomics).
 *   - Workspace contents need no initialisation: an entry point reads only workspace
 *     memory it has written itself (counters are cleared by kernels, not memsets).
 *   - The calls can be recorded into a HIP graph by stream capture and replayed (no
 *     allocation, synchronisation or memset node); a replay computes what the eager
 *     calls compute, bit for bit.
 *   - Process state: the library keeps three things beyond the call.  (1) Per device,
 *     its compute-unit count and, per kernel, the blocks per compute unit the occupancy
 *     query reports; both are looked up on first use and cached in atomics (concurrent
 *     first calls may both look up; they store the same value), so entry points may be
 *     called from several host threads.  (2) The launch trace below, per host thread.
 *     (3) The 131328-byte device array of dmoe_expert_ffn_fwd_noalloc, per device.
 *   - Supported: 1 <= d <= 4, 1 <= M, d*M <= 128, 1 <= k <= min(N, 8),
 *     N <= 16384, T >= 0 and T*k < 2^30, D and H multiples of 64 and at most 2^22,
 *     pointers 16-byte aligned.  Dims outside these give DMOE_EINVAL where they make no
 *     sense (T < 0, D or H or d or M or k < 1, k > N, unknown dtype, act or flag bits)
 *     and DMOE_EUNSUPPORTED where they are only beyond the supported set.
 *
 * Return codes: DMOE_OK (0); DMOE_EINVAL (-1) null required pointer or bad
 * dims; DMOE_EUNSUPPORTED (-2) shape/alignment outside the supported set;
 * DMOE_EHIP (-3) a launch failed (hipGetLastError).  Device faults surface at
 * the caller's next synchronisation, as HIP reports them.
 */
#ifndef DMOE_H
#define DMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { DMOE_OK = 0, DMOE_EINVAL = -1, DMOE_EUNSUPPORTED = -2, DMOE_EHIP = -3 };
enum { DMOE_F32 = 0, DMOE_BF16 = 1 };          /* dmoe_dims.dtype */
enum { DMOE_RELU = 0, DMOE_GELU = 1 };         /* dmoe_dims.act; GELU is the erf form */

typedef struct {
  int64_t T;      /* tokens */
  int64_t D;      /* d_model */
  int64_t H;      /* expert hidden size */
  int32_t d;      /* grid dimensions */
  int32_t M;      /* indices per grid dimension */
  int32_t k;      /* experts chosen per token */
  int32_t dtype;  /* DMOE_F32 or DMOE_BF16 */
  int32_t act;    /* DMOE_RELU or DMOE_GELU */
  int32_t flags;  /* 0, or DMOE_FLAG_* bits */
} dmoe_dims;

/* dmoe_dims.flags: DMOE_FLAG_GATE_EXACT makes dmoe_gate_topk compute every token's
 * bf16 gate scores with exact fp64 accumulation (the path it otherwise takes only
 * for tokens whose MFMA-computed decision is not certified).  Results are the same;
 * only the speed differs. */
/* DMOE_FLAG_ALIVE_TOPK makes TopK choose among the alive experts only (the partially
 * populated grid of App. C, where Algorithm 1 extends prefixes by active suffixes
 * only): cells are ranked by (alive first, g descending, lower flat index) and the k
 * first chosen, so dead experts are taken only when fewer than k are alive (they get
 * weight 0).  Without it, TopK ranks every expert and dead chosen ones get weight 0.
 * The decision is exact either way: a token whose alive-first choice the fast path
 * cannot certify is recomputed with exact fp64 scores over every cell. */
enum { DMOE_FLAG_GATE_EXACT = 1, DMOE_FLAG_ALIVE_TOPK = 2 };

/* Bytes of device workspace every entry point below needs for these dims
 * (one buffer of this size serves all of them; it may be reused between calls
 * on the same stream).  Returns 0 for invalid dims. */
size_t dmoe_workspace_bytes(const dmoe_dims* dims);

/* Static text for a return code. */
const char* dmoe_strerror(int code);

/* Launch trace, a measurement aid (it implements no part of the layer).  After
 * dmoe_trace_begin(events, names, capacity) on a host thread, each kernel that an entry
 * point called from that thread enqueues is followed, on the same stream, by
 * hipEventRecord(events[i]) for the i-th such kernel (i < capacity; later ones are
 * counted but not recorded), and names[i] is set to a static string naming the kernel.
 *   events  [capacity]  hipEvent_t handles (as void*), created and owned by the caller
 *   names   [capacity]  host array the library fills
 * The device time of kernel i is the time from events[i-1] (for i = 0: an event the
 * caller records on the stream before its first traced call) to events[i]; on one
 * stream kernels run in order, so these intervals partition the traced calls.
 * dmoe_trace_end() stops the trace and returns the number of kernels enqueued while
 * it was active (which may exceed capacity).  Without an active trace nothing is
 * recorded.  The trace state is per host thread; it is the caller's job not to combine
 * a trace with HIP graph capture.  Returns DMOE_EINVAL for capacity < 0 or, with
 * capacity > 0, NULL arrays. */
int dmoe_trace_begin(void* const* events, const char** names, int capacity);
int dmoe_trace_end(void);

/* Gate scores, exact TopK over the grid and Eq. 1 weights (Sec. 3.2; Eq. 1; App. C).
 *   x      [T, D]      layer input
 *   Wg     [d*M, D]    rows i*M .. i*M+M-1 are the weight of g_i (nn.Linear layout)
 *   bg     [d*M]       gate bias, or NULL for none
 *   alive  [N] uint8   1 = the expert responds; NULL = all respond
 * outputs
 *   idx    [T, k] int32  chosen flat expert ids, best first: by g descending,
 *                        ties to the lower flat index
 *   w      [T, k] fp32   Eq. 1 weights over the chosen experts that are alive,
 *                        renormalised to sum to 1; 0 for dead ones; all 0 if
 *                        every chosen expert is dead
 *   g      [T, k] fp32   chosen totals g(x, f), or NULL
 *   scores [T, d*M] fp32 per-dimension decision scores g_i(x), or NULL
 * Selection compares the fp32 rounding of each exact score g_i(x)[u] and adds the d
 * fp32 values of a cell in fp64 in dim order.  bf16: scores are computed on MFMA
 * with a per-token error bound; a token whose TopK order is within the bound of a
 * tie is recomputed with exact fp64 accumulation, so the selection equals the one
 * of the exact scores; the returned scores, g and w carry the (bounded) MFMA error.
 * fp32, and bf16 with d*M > 96: exact fp64 accumulation for every token.
 * Inputs are expected to be finite: with NaN or infinite scores the choice is
 * unspecified (every returned index is still a valid expert id) and w may be NaN.
 * Uses workspace: bf16 with d*M <= 96, and DMOE_FLAG_ALIVE_TOPK with either dtype
 * (the queue of tokens to recompute; ws must not be NULL, else DMOE_EINVAL);
 * otherwise no. */
int dmoe_gate_topk(const dmoe_dims* dims, const void* x, const void* Wg, const void* bg,
                   const uint8_t* alive, int32_t* idx, float* w, float* g, float* scores,
                   void* ws, void* stream);

/* Group the alive pairs by expert: the per-expert batches a Runtime forms from
 * incoming requests (Sec. 3.3), and the input each chosen expert receives (Sec. 3.2).
 * Rows of one expert are contiguous and in token order.
 *   x [T, D], idx [T, k], alive [N] or NULL
 * outputs
 *   counts    [N]       alive pairs per expert
 *   offsets   [N+1]     exclusive prefix sum of counts (offsets[N] = rows used)
 *   row_token [P_max]   token of each row (entries >= offsets[N] untouched)
 *   pos       [T, k]    row of each pair, -1 if its expert is dead
 *   x_perm    [P_max, D] x_perm[r] = x[row_token[r]] (rows >= offsets[N] untouched)
 * Uses workspace. */
int dmoe_dispatch(const dmoe_dims* dims, const void* x, const int32_t* idx,
                  const uint8_t* alive, int32_t* counts, int32_t* offsets, int32_t* row_token,
                  int32_t* pos, void* x_perm, void* ws, void* stream);

/* Expert feed-forward blocks on the grouped rows (the Runtime Forward, Sec. 3.3):
 * for rows r of expert e,  h = x_perm W1_e^T + b1_e,  a = act(h),  y = a W2_e^T + b2_e.
 *   offsets [N+1] (from dmoe_dispatch), x_perm [P_max, D]
 *   W1 [N, H, D], b1 [N, H], W2 [N, D, H], b2 [N, D]
 * outputs (rows < offsets[N] written)
 *   h [P_max, H] pre-activation, a [P_max, H] activation, y_perm [P_max, D]
 * Uses workspace. */
int dmoe_expert_ffn_fwd(const dmoe_dims* dims, const int32_t* offsets, const void* x_perm,
                        const void* W1, const void* b1, const void* W2, const void* b2,
                        void* h, void* a, void* y_perm, void* ws, void* stream);

/* dmoe_expert_ffn_fwd without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, results and kernels as dmoe_expert_ffn_fwd, bit
 * for bit; its only scratch, the tile plan (2 (N + 1) int32, at most 131328 bytes for
 * N <= 16384), lives in a static device array of the library that each GPU holds until
 * the process ends.  It calls no allocating routine.  Every call on one GPU uses that
 * GPU's copy of the array, so calls that overlap on one GPU (different streams, or other
 * host threads) race and must not be issued; calls in sequence on one stream are fine.
 * Returns DMOE_EUNSUPPORTED if the tile plan would exceed the array, DMOE_EHIP if its
 * device address cannot be obtained. */
int dmoe_expert_ffn_fwd_noalloc(const dmoe_dims* dims, const int32_t* offsets, const void* x_perm,
                                const void* W1, const void* b1, const void* W2, const void* b2,
                                void* h, void* a, void* y_perm, void* stream);

/* Weighted average of Eq. 1:  y[t] = sum_j w[t,j] y_perm[pos[t,j]] over pairs with
 * pos >= 0, in slot order, fp32 accumulation.  y [T, D] written (zeros for tokens
 * with no alive expert).  Uses workspace: no. */
int dmoe_combine(const dmoe_dims* dims, const void* y_perm, const int32_t* pos,
                 const float* w, void* y, void* stream);

/* Backward of the weighted average (derivative of Eq. 1 in w and in f(x)):
 *   dy_perm[pos[t,j]] = w[t,j] dy[t]          (rows of alive pairs)
 *   dw[t,j] = <dy[t], y_perm[pos[t,j]]>        (0 for dead pairs), fp32
 * Uses workspace: no. */
int dmoe_combine_bwd(const dmoe_dims* dims, const void* dy, const void* y_perm,
                     const int32_t* pos, const float* w, void* dy_perm, float* dw,
                     void* stream);

/* Backward of the Eq. 1 weights and of the gate layers (Sec. 3.2).  TopK is
 * piecewise constant; the gradient reaches the gate through the softmax over
 * the chosen alive experts only:
 *   dg[t,j] = w[t,j] (dw[t,j] - sum_l w[t,l] dw[t,l])   (0 for dead pairs)
 *   ds[t, i*M + u_i(idx[t,j])] += dg[t,j]  for every dimension i
 *   dWg = ds^T x   [d*M, D]  (dtype of Wg),   dbg = sum_t ds  [d*M] (dtype of Wg)
 * The gate's share of dx (ds Wg) is added by dmoe_dispatch_bwd.
 *   x [T, D], idx [T, k], w [T, k], dw [T, k], alive [N] or NULL
 * outputs: dg [T, k] fp32, dWg, dbg (dbg may be NULL).  Uses workspace. */
int dmoe_gate_topk_bwd(const dmoe_dims* dims, const void* x, const int32_t* idx,
                       const float* w, const float* dw, const uint8_t* alive, float* dg,
                       void* dWg, void* dbg, void* ws, void* stream);

/* Backward of the expert blocks (the Runtime Backward, Sec. 3.3, which returns
 * input gradients; the parameter update is left to the caller):
 *   dh = (dy_perm W2_e) * act'(h)       [P_max, H]  (may alias h: h is then overwritten)
 *   dx_perm = dh W1_e                   [P_max, D]
 *   dW2_e = dy_perm_e^T a_e,  db2_e = sum of dy_perm_e rows
 *   dW1_e = dh_e^T x_perm_e,  db1_e = sum of dh_e rows
 * dW1 [N,H,D], db1 [N,H], dW2 [N,D,H], db2 [N,D]: written only for experts with
 * counts[e] > 0 (an expert with no rows has zero gradient; its slots are not touched).
 * Uses workspace. */
int dmoe_expert_ffn_bwd(const dmoe_dims* dims, const int32_t* offsets, const int32_t* counts,
                        const void* x_perm, const void* h, const void* a, const void* dy_perm,
                        const void* W1, const void* W2, void* dh, void* dx_perm, void* dW1,
                        void* db1, void* dW2, void* db2, void* ws, void* stream);

/* The same backward with the forward's activations recomputed instead of kept
 * (gradient checkpointing, as the Runtime's Backward does, Sec. 3.3 and App. D: it
 * runs the expert's forward again when the gradient arrives; about one third more
 * expert arithmetic, and h and a need not survive from the forward call):
 *   h, a = x_perm W1_e^T + b1_e, act(.)   recomputed into the scratch h and a [P_max, H]
 *   then exactly dmoe_expert_ffn_bwd with dh written over h.
 * Outputs are bit-identical to dmoe_expert_ffn_bwd given the forward's h and a.
 * h and a are caller-owned scratch (overwritten); b1 [N,H] is the up-projection bias.
 * Uses workspace. */
int dmoe_expert_ffn_bwd_recompute(const dmoe_dims* dims, const int32_t* offsets, const int32_t* counts,
                                  const void* x_perm, const void* W1, const void* b1, const void* W2,
                                  const void* dy_perm, void* h, void* a, void* dx_perm, void* dW1,
                                  void* db1, void* dW2, void* db2, void* ws, void* stream);

/* The backward with the expert parameters updated by gradient descent in place
 * (the Runtime's Backward updates its expert's parameters, Sec. 3.3):
 *   W2_e <- W2_e - lr dy_perm_e^T a_e      b2_e <- b2_e - lr (sum of dy_perm_e rows)
 *   W1_e <- W1_e - lr dh_e^T x_perm_e      b1_e <- b1_e - lr (sum of dh_e rows)
 * with dh and dx_perm as in dmoe_expert_ffn_bwd, computed from the parameters as they
 * were on entry.  The gradients are never stored: each update is applied from the
 * fp32 accumulation and rounded once to the parameter dtype.  Experts with no rows
 * keep their parameters.  dh may alias h.  lr must not be NaN.  Uses workspace. */
int dmoe_expert_ffn_bwd_sgd(const dmoe_dims* dims, const int32_t* offsets, const int32_t* counts,
                            const void* x_perm, const void* h, const void* a, const void* dy_perm,
                            void* W1, void* b1, void* W2, void* b2, float lr, void* dh,
                            void* dx_perm, void* ws, void* stream);

/* Input gradient of the layer (derivative of Eq. 1 with respect to x).  x reaches
 * the output along two routes: through each chosen alive expert f(x) (the Trainer
 * sends x to those experts and their Backward returns input gradients, Sec. 3.3), and
 * through the gate scores g(x, f) = sum_i g_i(x)[u_i] of the Sec. 3.2 gate.  So
 *   dx[t] = sum_j dx_perm[pos[t,j]]                       (alive pairs, slot order)
 *         + sum_j dg[t,j] sum_i Wg[i*M + u_i(idx[t,j])]   (when idx, dg, Wg are non-NULL)
 * with dg from dmoe_gate_topk_bwd.  The gate's share is added here rather than in
 * dmoe_gate_topk_bwd so that dx is written once, in one pass over its T*D elements.
 * fp32 accumulation, one rounding.  dx [T, D] written.  Uses workspace: no. */
int dmoe_dispatch_bwd(const dmoe_dims* dims, const void* dx_perm, const int32_t* pos,
                      const int32_t* idx, const float* dg, const void* Wg, void* dx,
                      void* stream);

/* ------------------------------------------------------------------------------
 * The feed-forward block expert of Sec. 4.1: linear layers of widths D -> F -> F -> D
 * with layer normalisation and the activation between them,
 *   h1 = x W1^T + b1,  a1 = act(LN(h1; g1, be1)),
 *   h2 = a1 W2^T + b2, a2 = act(LN(h2; g2, be2)),
 *   y  = a2 W3^T + b3,
 * LN(h; g, b) = g (h - mean(h)) / sqrt(var(h) + 1e-5) + b over the F features of a row
 * (biased variance).  F = dims->H, D = dims->D, act = dims->act; F is at most 4096
 * for bf16 and 2048 for fp32.  These entry points replace dmoe_expert_ffn_fwd/bwd
 * for a layer whose experts are such blocks; gate, dispatch and combine are shared.
 * ------------------------------------------------------------------------------ */

/* The parameters of every expert, stacked over the N experts, in the layer dtype,
 * row-major: W1 [N,F,D], b1 [N,F], g1 and be1 [N,F] (scale and shift of the first
 * normalisation), W2 [N,F,F], b2 [N,F], g2 and be2 [N,F], W3 [N,D,F], b3 [N,D].
 * The same struct carries their gradients (same shapes). */
typedef struct {
  void* W1; void* b1; void* g1; void* be1;
  void* W2; void* b2; void* g2; void* be2;
  void* W3; void* b3;
} dmoe_ffblock_params;

/* Per-row tensors the forward keeps for the backward (P_max rows each, in expert
 * row order like x_perm): h1, a1, h2, a2 [P_max, F] in the layer dtype; st1, st2
 * [P_max, 2] fp32 holding each row's (mean, 1/sqrt(var + 1e-5)) of h1 and h2. */
typedef struct {
  void* h1; void* a1; float* st1;
  void* h2; void* a2; float* st2;
} dmoe_ffblock_acts;

/* Forward of the block experts on the expert-grouped rows (the Runtime's batched
 * Forward, Sec. 3.3; the block of Sec. 4.1).  x_perm [P_max, D] and offsets [N+1]
 * come from dmoe_dispatch; writes every buffer of *acts and y_perm [P_max, D] for
 * the rows [0, offsets[N]).  Uses workspace. */
int dmoe_expert_ffblock_fwd(const dmoe_dims* dims, const int32_t* offsets, const void* x_perm,
                            const dmoe_ffblock_params* params, const dmoe_ffblock_acts* acts,
                            void* y_perm, void* ws, void* stream);

/* Backward of the block experts (the Runtime's Backward, Sec. 3.3): from dy_perm
 * [P_max, D] (dmoe_combine_bwd) and the forward's *acts,
 *   dW3 = dy^T a2, db3 = sum dy, da2 = dy W3,  g2 <- da2, then dh2 in place,
 *   dg2, dbe2 and dh2 = the normalisation backward at h2,
 *   dW2 = dh2^T a1, db2 = sum dh2, da1 = dh2 W2, g1 <- da1, then dh1 in place,
 *   dW1 = dh1^T x_perm, db1 = sum dh1, dx_perm = dh1 W1,
 * per expert over its rows.  g1 and g2 are caller-owned [P_max, F] buffers in the
 * layer dtype that end holding dh1 and dh2.  grads receives every parameter gradient;
 * experts with no rows keep the caller's contents.  No output may alias an input.
 * Uses workspace. */
int dmoe_expert_ffblock_bwd(const dmoe_dims* dims, const int32_t* offsets, const void* x_perm,
                            const dmoe_ffblock_params* params, const dmoe_ffblock_acts* acts,
                            const void* dy_perm, void* g1, void* g2, void* dx_perm,
                            const dmoe_ffblock_params* grads, void* ws, void* stream);

/* One normalisation step of the block on its own (Sec. 4.1): for each row r of h
 * [P_max, F] (rows [0, offsets[N]), F = dims->H) owned by expert e,
 *   stats[r] = (mean, rstd) fp32, a[r] = act(gamma[e] (h[r] - mean) rstd + beta[e]),
 * gamma and beta [N, F].  No workspace. */
int dmoe_ln_act_fwd(const dmoe_dims* dims, const int32_t* offsets, const void* h, const void* gamma,
                    const void* beta, void* a, float* stats, void* stream);

/* Backward of dmoe_ln_act_fwd given da [P_max, F] and the forward's stats:
 *   n = (h - mean) rstd, dz = da act'(gamma n + beta), dn = dz gamma,
 *   dh = rstd (dn - mean_f(dn) - n mean_f(dn n)),
 *   dgamma[e] = sum over e's rows of dz n, dbeta[e] = sum over e's rows of dz.
 * dh may alias da (the scale and shift gradients are taken before dh is written);
 * experts with no rows keep the caller's dgamma, dbeta.  No workspace. */
int dmoe_ln_act_bwd(const dmoe_dims* dims, const int32_t* offsets, const void* h, const float* stats,
                    const void* gamma, const void* beta, const void* da, void* dh, void* dgamma,
                    void* dbeta, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DMOE_H */
