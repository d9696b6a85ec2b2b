/*
 * vmoe.h -- C ABI of libvmoe: one sparse Vision-MoE layer, forward and
 * backward, on an AMD Instinct MI355X (gfx950).
 *
 * The operation. The paper co-adapts V-MoE vision backbones whose blocks
 * route every token to a few experts out of a shared pool (Sec. 1, Sec. 2.1:
 * sparse expert routing over expertised MLP blocks; Sec. 2.2: experts of
 * several models pooled as one parallel expert set, each model keeping its
 * own router), under per-expert capacity limits (Sec. 2.3), and adapts the
 * experts by back-propagation (Sec. 3.1-3.2: V-MoE retraining). The paper
 * does not write the layer out; this library implements V-MoE's definition
 * as read for this project:
 *
 *   logits = x W_r[g]^T (+ bias) (+ noise)       noisy gate, one router per group g
 *   p      = softmax(logits)                     exact-order fp32, see vmoe_route
 *   e_1..k = top-k experts of each token         ties to the lower expert index
 *   priority = p[e_1]; each group's tokens are walked by priority (desc),
 *   first choices of all tokens before second choices, and an assignment is
 *   kept while its expert has fewer than C tokens of that group
 *   (batch-prioritized routing); kept gates are p[e_j], not renormalised
 *   xe     = kept tokens packed into per-expert buffers
 *   ye     = W2_e gelu(W1_e xe + b1_e) + b2_e   per expert (exact-erf GELU)
 *   y[t]   = sum_j gate[t,j] ye[row(t,j)]        dropped tokens give 0
 * and the gradients of y w.r.t. x, the router and every expert parameter.
 *
 * Conventions shared by every entry point
 * - All tensor pointers are DEVICE pointers owned by the caller, row-major and
 *   contiguous, 16-byte aligned. The library allocates no device memory,
 *   never synchronises and never reads device data on the host. Its only
 *   state is per GPU: the static scratch of vmoe_route_noalloc, and a side
 *   stream with two events that the bf16 expert-MLP backward creates on its
 *   first call (kept until the process ends).
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream). Work
 *   is enqueued asynchronously on it, in call order (a call that also uses
 *   the side stream forks it from `stream` and joins it back before
 *   returning, so its work still starts after, and completes before, the
 *   neighbouring work on `stream`).
 * - Activations and weights use shape.dtype (VMOE_F32 or VMOE_BF16; bf16 is
 *   stored as raw 16-bit patterns). Gating tensors (logits, probs, gate,
 *   dgate, noise, bias) and all weight / router / input gradients are f32.
 * - Sizes: N tokens in G equal routing groups (N_g = N / G), model width d,
 *   expert hidden width f, E experts, top-k, capacity C per (group, expert)
 *   from vmoe_capacity. Expert buffers are [E, G*C, width]; expert e's kept
 *   rows are packed at the front, group by group: rows [0, n_e) with
 *   n_e = sum_g counts[g, e]. Rows at or beyond n_e are never read.
 *   row(t, j) = e*G*C + row_base[g, e] + slot[t, j]  for e = expert_idx[t, j].
 * - Every call overwrites its outputs, except vmoe_route_bwd's dx (+=).
 * - Errors are status codes, checked before anything is enqueued: a NULL
 *   required pointer, N % G != 0, k outside [1, E], E > 64, d or f not a
 *   multiple of 8, a non-positive capacity factor, an unknown dtype or
 *   misaligned pointer -> VMOE_ERR_INVALID_ARG; a shape beyond the kernels'
 *   32-bit addressing (one expert's [G*C, d or f] operand or [f, d] weight of
 *   2 GiB or more, 2^31 or more elements in the pooled expert buffers or
 *   the token-major tensors, or d >= 2^22, where 128 f32 rows of width d
 *   reach 2 GiB) -> VMOE_ERR_UNSUPPORTED (vmoe_capacity returns
 *   -1 for it); a too-small workspace -> VMOE_ERR_WORKSPACE; a failed kernel
 *   launch -> VMOE_ERR_HIP. Required
 *   pointers are checked whatever the sizes: with N = 0 they still point to
 *   an allocation (nothing is read from it). Nothing
 *   throws across the ABI. All entry points are thread-safe (stateless).
 */
#ifndef VMOE_H
#define VMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define VMOE_ABI_VERSION 1

typedef enum {
    VMOE_OK = 0,
    VMOE_ERR_INVALID_ARG = 1,
    VMOE_ERR_UNSUPPORTED = 2,
    VMOE_ERR_WORKSPACE = 3,
    VMOE_ERR_HIP = 4
} vmoe_status;

typedef enum { VMOE_F32 = 0, VMOE_BF16 = 1 } vmoe_dtype;

/* vmoe_route flags */
#define VMOE_ROUTE_LOGITS_IN 1 /* skip the router product; `logits` is an input */

typedef struct vmoe_shape {
    int32_t n_tokens;          /* N >= 0                                        */
    int32_t n_groups;          /* G >= 1, divides N                             */
    int32_t d_model;           /* d, multiple of 8                              */
    int32_t d_ff;              /* f, multiple of 8                              */
    int32_t n_experts;         /* E in [1, 64]                                  */
    int32_t k;                 /* top-k in [1, E]                               */
    double capacity_factor;    /* c > 0                                         */
    int32_t capacity_rounding; /* 0: round half away from zero, 1: ceil         */
    int32_t capacity_override; /* > 0: use this C instead of the formula        */
    int32_t dtype;             /* vmoe_dtype                                    */
    int32_t reserved;          /* must be 0                                     */
} vmoe_shape;

/* ABI version of the loaded library (VMOE_ABI_VERSION). */
int32_t vmoe_abi_version(void);

/* Static description of a status code. */
const char* vmoe_status_string(int32_t status);

/* Capacity per (group, expert): C = round(k * N_g * c / E), at least 1, the
 * buffer size of V-MoE's capacity limit (capacity limits, paper Sec. 2.3).
 * Returns -1 if the shape is invalid. */
int32_t vmoe_capacity(const vmoe_shape* shape);

/* Bytes of scratch that vmoe_route needs (0 on an invalid shape). */
size_t vmoe_route_workspace_bytes(const vmoe_shape* shape);

/* Bytes of scratch that vmoe_route_bwd needs (0 on an invalid shape). */
size_t vmoe_route_bwd_workspace_bytes(const vmoe_shape* shape);

/* Noisy top-k gating with capacity and batch-prioritized routing
 * (sparse expert routing, paper Sec. 1 and Sec. 2.1; capacity, Sec. 2.3).
 *   x          [N, d] dtype         tokens (unused with LOGITS_IN)
 *   w_router   [G, E, d] dtype      router of each group (unused with LOGITS_IN)
 *   logit_bias [E] f32 or NULL      constant logit offset
 *   noise      [N, E] f32 or NULL   gating noise drawn by the caller
 *   logits     [N, E] f32           out: sum_i x[t,i] w_router[g,e,i], summed in
 *                                   double in increasing i and rounded once to f32
 *                                   (in with LOGITS_IN)
 *   probs      [N, E] f32           out: softmax of z = (logits + bias) + noise,
 *                                   exp by Cody-Waite reduction and a degree-7
 *                                   polynomial, sum in expert order, IEEE divide
 *   expert_idx [N, k] i32           out: top-k experts by z, ties to lower index
 *   slot       [N, k] i32           out: slot in the expert's group buffer, -1 = dropped
 *   gate       [N, k] f32           out: probs[t, expert_idx[t,j]] if kept, else 0
 *   order      [N] i32              out: each group's tokens by priority p[e_1]
 *                                   descending, token index ascending
 *   counts     [G, E] i32           out: kept assignments per (group, expert) (<= C)
 *   row_base   [G, E] i32           out: sum_{g' < g} counts[g', e]
 *   workspace  device scratch of vmoe_route_workspace_bytes(shape) bytes
 * Given the same fp32 logits, every integer output and probs/gate are
 * bit-for-bit deterministic. */
vmoe_status vmoe_route(const vmoe_shape* shape, const void* x, const void* w_router,
                       const float* logit_bias, const float* noise, int32_t flags, float* logits,
                       float* probs, int32_t* expert_idx, int32_t* slot, float* gate,
                       int32_t* order, int32_t* counts, int32_t* row_base, void* workspace,
                       size_t workspace_bytes, void* stream);

/* Scratch held by vmoe_route_noalloc on each GPU it runs on (16 MiB). */
#define VMOE_ROUTE_NOALLOC_SCRATCH_BYTES (16u << 20)

/* vmoe_route for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same routing with the same outputs, bit for bit, but no workspace
 * argument. Its scratch is a static device array of
 * VMOE_ROUTE_NOALLOC_SCRATCH_BYTES on each GPU, placed when the library's
 * code is loaded there and held until the process ends; the call allocates
 * and frees nothing. Shapes whose vmoe_route_workspace_bytes exceeds that size
 * get VMOE_ERR_WORKSPACE (before anything is enqueued); VMOE_ERR_HIP if the
 * array's device address cannot be looked up. Every call on one GPU shares
 * that GPU's array: calls that overlap on one GPU (on any streams, from any
 * threads) race on it, and the caller must serialise them. Other arguments
 * and errors as vmoe_route. */
vmoe_status vmoe_route_noalloc(const vmoe_shape* shape, const void* x, const void* w_router,
                               const float* logit_bias, const float* noise, int32_t flags,
                               float* logits, float* probs, int32_t* expert_idx, int32_t* slot,
                               float* gate, int32_t* order, int32_t* counts, int32_t* row_base,
                               void* stream);

/* Dispatch of kept tokens into per-expert buffers (sparse routing sends each
 * token to its chosen experts, paper Sec. 2.1; a token past an expert's
 * capacity is dropped, Sec. 2.3): xe[row(t, j), :] = x[t, :] for every kept
 * (t, j), row(t, j) = e * G*C + row_base[g, e] + slot[t, j] with
 * e = expert_idx[t, j]. x [N, d], xe [E, G*C, d] (dtype, caller-owned; rows
 * at or past an expert's n_e are not written). Device pointers, each non-null
 * and 16-byte aligned; VMOE_ERR_INVALID_ARG otherwise or on a bad shape. */
vmoe_status vmoe_dispatch(const vmoe_shape* shape, const void* x, const int32_t* expert_idx,
                          const int32_t* slot, const int32_t* row_base, void* xe, void* stream);

/* Expert MLP forward over each expert's n_e packed rows (expertised MLP
 * blocks, paper Sec. 2.1): H = xe W1_e^T + b1_e, A = gelu(H), ye = A W2_e^T + b2_e,
 * with the exact-erf GELU gelu(h) = h Phi(h).
 *   xe [E, G*C, d], counts [G, E] (device; n_e = sum_g counts[g, e])
 *   w1 [E, f, d], b1 [E, f], w2 [E, d, f], b2 [E, d]     (dtype)
 *   act      [E, G*C, f] out: A = gelu(H)       } saved for the backward;
 *   act_grad [E, G*C, f] out: gelu'(H)          } H itself is not stored
 *   ye       [E, G*C, d] out.
 * bf16 runs on bf16 matrix cores with f32 accumulation (GELU evaluated in f32
 * to ~1e-7 absolute, then rounded to bf16); f32 accumulates in f32. */
vmoe_status vmoe_expert_ffn_fwd(const vmoe_shape* shape, const void* xe, const int32_t* counts,
                                const void* w1, const void* b1, const void* w2, const void* b2,
                                void* act, void* act_grad, void* ye, void* stream);

/* Gate-weighted combine of the experts' outputs (the sparse layer's output
 * is the gate-weighted sum over the chosen experts, paper Sec. 2.1; dropped
 * assignments contribute nothing, Sec. 2.3): y[t] = sum over kept j (in j
 * order, f32 accumulation) of gate[t,j] * ye[row(t,j)]; 0 for a token with no
 * kept assignment. ye [E, G*C, d], gate [N, k] f32, y [N, d] (dtype,
 * overwritten). Device pointers; VMOE_ERR_INVALID_ARG on a bad shape. */
vmoe_status vmoe_combine_fwd(const vmoe_shape* shape, const void* ye, const int32_t* expert_idx,
                             const int32_t* slot, const int32_t* row_base, const float* gate,
                             void* y, void* stream);

/* Backward of the combine (back-propagation through the layer, paper
 * Sec. 3.1-3.2): dye[row(t,j)] = gate[t,j] * dy[t];
 * dgate[t,j] = <dy[t], ye[row(t,j)]> (f32) for kept j, 0 for dropped j.
 * dy [N, d], dye [E, G*C, d] (dtype; rows of kept assignments written),
 * dgate [N, k] f32 (overwritten). Device pointers; VMOE_ERR_INVALID_ARG on a
 * bad shape. */
vmoe_status vmoe_combine_bwd(const vmoe_shape* shape, const void* dy, const void* ye,
                             const int32_t* expert_idx, const int32_t* slot,
                             const int32_t* row_base, const float* gate, void* dye, float* dgate,
                             void* stream);

/* Backward of the expert MLP (adaptation by back-propagation, paper Sec. 3):
 *   dH  = (dye W2_e) * act_grad          dh  [E, G*C, f] out (dtype)
 *   dxe = dH W1_e                        dxe [E, G*C, d] out (dtype)
 *   dW2 = dye^T act, db2 = sum_rows dye  dw2 [E, d, f], db2 [E, d]  f32 out
 *   dW1 = dH^T xe,  db1 = sum_rows dH    dw1 [E, f, d], db1 [E, f]  f32 out
 * act and act_grad are the forward's saved tensors. Experts with n_e = 0 get
 * zero weight gradients. With 16 or more bf16 experts, dxe runs on the
 * library's side stream beside the weight gradients (forked after dH and
 * joined before the call returns); concurrent calls on one GPU from several
 * host threads serialise their dxe launches on that stream. */
vmoe_status vmoe_expert_ffn_bwd(const vmoe_shape* shape, const void* xe, const int32_t* counts,
                                const void* w1, const void* w2, const void* act,
                                const void* act_grad, const void* dye, void* dh, void* dxe,
                                float* dw1, float* db1, float* dw2, float* db2, void* stream);

/* The dispatch fused into the expert MLP's operand loads (bf16 layers): the
 * up-projection reads each expert row straight from the token's row of x
 * (buffer loads with per-row offsets), so xe is neither written nor read.
 *   vmoe_dispatch_ffn_fwd = vmoe_dispatch + vmoe_expert_ffn_fwd without xe:
 *     row_token [E, G*C] i32 out: the token of each kept expert row
 *     (row_token[row(t, j)] = t; rows at or beyond n_e unspecified), for the
 *     backward; act, act_grad, ye as vmoe_expert_ffn_fwd.
 *   vmoe_expert_ffn_bwd_gather = vmoe_expert_ffn_bwd with dW1 = dH^T xe
 *     reading xe's rows from x through row_token.
 * Bit-identical to the unfused calls (the same bf16 values reach the same
 * products). VMOE_ERR_UNSUPPORTED for f32 layers, for N * d * 2 > 2^31 - 16
 * bytes of x, and (backward) for G * C > 6144 rows per expert. */
vmoe_status vmoe_dispatch_ffn_fwd(const vmoe_shape* shape, const void* x,
                                  const int32_t* expert_idx, const int32_t* slot,
                                  const int32_t* row_base, const int32_t* counts, const void* w1,
                                  const void* b1, const void* w2, const void* b2,
                                  int32_t* row_token, void* act, void* act_grad, void* ye,
                                  void* stream);
vmoe_status vmoe_expert_ffn_bwd_gather(const vmoe_shape* shape, const void* x,
                                       const int32_t* row_token, const int32_t* counts,
                                       const void* w1, const void* w2, const void* act,
                                       const void* act_grad, const void* dye, void* dh, void* dxe,
                                       float* dw1, float* db1, float* dw2, float* db2,
                                       void* stream);

/* vmoe_expert_ffn_fwd and vmoe_expert_ffn_bwd with a device-side tile
 * scheduler (the lifespan-aware aligning of paper Sec. 3.2.2 applied to the
 * experts of one grouped GEMM): each GEMM runs as many persistent workgroups
 * as the GPU holds at once, and every workgroup first computes, from the
 * device row counts, the fill-clamp-refill split of those workgroups among
 * the experts (minimum one for an expert with tiles, saturation its tile
 * count, work coefficient its tiles times a per-tile cost model of its rows);
 * expert e then owns a contiguous range of units_e workgroups, each taking
 * every units_e-th tile of e. Same arguments, same results as the two calls
 * (each output tile is computed by the same code); bf16 layers only (f32
 * layers run the calls above). */
vmoe_status vmoe_expert_ffn_fwd_quota(const vmoe_shape* shape, const void* xe,
                                      const int32_t* counts, const void* w1, const void* b1,
                                      const void* w2, const void* b2, void* act, void* act_grad,
                                      void* ye, void* stream);
vmoe_status vmoe_expert_ffn_bwd_quota(const vmoe_shape* shape, const void* xe,
                                      const int32_t* counts, const void* w1, const void* w2,
                                      const void* act, const void* act_grad, const void* dye,
                                      void* dh, void* dxe, float* dw1, float* db1, float* dw2,
                                      float* db2, void* stream);

/* The device implementation of vmoe_fill_clamp_refill's whole-unit shares
 * (paper Sec. 3.2.2) that the quota-scheduled GEMMs run, on one wavefront:
 * n <= 64 experts, min_units, sat_units [n] i32, coef [n] f64, budget
 * units -> alloc_units [n] i32 (device memory, asynchronous on stream).
 * Every sum is taken in ascending expert order with the host routine's
 * operations, so for valid inputs the units equal vmoe_fill_clamp_refill's
 * alloc_units. VMOE_ERR_INVALID_ARG for n outside [0, 64], a negative
 * budget or a missing pointer; inputs are not otherwise validated. */
vmoe_status vmoe_fill_clamp_refill_device(int32_t n, const int32_t* min_units,
                                          const int32_t* sat_units, const double* coef,
                                          int32_t budget, int32_t* alloc_units, void* stream);

/* Backward of the dispatch (paper Sec. 2.1 routing, back-propagated as in
 * Sec. 3.1-3.2): dx[t] = sum over kept j of dxe[row(t,j)] (j ascending, f32,
 * overwritten; 0 for a token with no kept assignment). dxe [E, G*C, d]
 * (dtype), dx [N, d] f32. Device pointers; VMOE_ERR_INVALID_ARG on a bad
 * shape. */
vmoe_status vmoe_dispatch_bwd(const vmoe_shape* shape, const void* dxe,
                              const int32_t* expert_idx, const int32_t* slot,
                              const int32_t* row_base, float* dx, void* stream);

/* Backward through the gate into the router (the router is part of the
 * adapted layer, paper Sec. 3.1-3.2; the top-k choice of Sec. 2.1 and the
 * capacity and priority order of Sec. 2.3 are piecewise constant and pass
 * no gradient):
 *   dp[t,e]  = sum of dgate[t,j] over kept j with expert_idx[t,j] = e
 *   dz[t,e]  = probs[t,e] * (dp[t,e] - sum_e' probs[t,e'] dp[t,e'])
 *   dx[t,:] += sum_e dz[t,e] w_router[g,e,:]                    (accumulates)
 *   dw_router[g,e,:] = sum_{t in g} dz[t,e] x[t,:]  f32 [G,E,d], overwritten;
 *                      NULL skips it (frozen routers)
 * workspace: vmoe_route_bwd_workspace_bytes(shape) bytes of device memory
 * (the per-chunk router-gradient partials), required with or without
 * dw_router; VMOE_ERR_WORKSPACE if it is smaller or not device memory. */
vmoe_status vmoe_route_bwd(const vmoe_shape* shape, const void* x, const void* w_router,
                           const float* probs, const int32_t* expert_idx, const int32_t* slot,
                           const float* dgate, float* dx, float* dw_router, void* workspace,
                           size_t workspace_bytes, void* stream);

/* vmoe_dispatch_bwd followed by vmoe_route_bwd in one pass over the tokens:
 *   dx[t,:] = sum over kept j of dxe[row(t,j),:] (j ascending, from 0)
 *             + sum_e dz[t,e] w_router[g,e,:]        dx [N, d] f32, overwritten
 *   dw_router as in vmoe_route_bwd (NULL skips it).
 * Bit-identical to the two calls in sequence; it reads dxe where they would
 * write and re-read dx. Arguments and workspace as in those two calls. */
vmoe_status vmoe_dispatch_route_bwd(const vmoe_shape* shape, const void* dxe,
                                    const int32_t* row_base, const void* x, const void* w_router,
                                    const float* probs, const int32_t* expert_idx,
                                    const int32_t* slot, const float* dgate, float* dx,
                                    float* dw_router, void* workspace, size_t workspace_bytes,
                                    void* stream);

/* vmoe_dispatch_route_bwd with an extra gradient with respect to the router
 * logits added before the router products (chain rule: the logits also feed
 * an auxiliary loss, e.g. the dlogits of vmoe_balance_loss):
 *   dz[t,e] = probs[t,e] (dp[t,e] - <p, dp>) + dlogits[t,e]
 *   dx, dw_router from that dz as in vmoe_dispatch_route_bwd.
 * dlogits [N, E] f32 (required). Other arguments and workspace as there. */
vmoe_status vmoe_dispatch_route_bwd_dlogits(const vmoe_shape* shape, const void* dxe,
                                            const int32_t* row_base, const void* x,
                                            const void* w_router, const float* probs,
                                            const int32_t* expert_idx, const int32_t* slot,
                                            const float* dgate, const float* dlogits, float* dx,
                                            float* dw_router, void* workspace,
                                            size_t workspace_bytes, void* stream);

/* Bytes of scratch that vmoe_balance_loss needs (0 on an invalid shape). */
size_t vmoe_balance_loss_workspace_bytes(const vmoe_shape* shape);

/* Auxiliary balance losses on the gate, per routing group, and their gradient
 * with respect to the router logits. The paper cites such losses (Sec. 1,
 * Sec. 2.3) as the alternative to capacity limits without defining them;
 * this is the published noisy top-k gating form:
 *   importance[g,e] = sum over the group's tokens of probs[t,e]
 *   load[g,e]       = sum over tokens of Phi((l[t,e] - thr[t,e]) / noise_std),
 *                     l = logits + bias, thr = the k-th largest noisy logit
 *                     z = (logits + bias) + noise among the OTHER experts
 *                     (ties: lower index first; -inf if fewer than k): the
 *                     chance that e stays in the top-k when only its own
 *                     noise is drawn again (Phi: standard normal CDF)
 *   losses[g,0|1]   = CV^2 = var / mean^2 over the experts of importance[g]
 *                     and load[g] (population variance; 0 for a zero sum)
 *   dlogits[t,e]    = d/dlogits of sum_g w_importance losses[g,0]
 *                     + w_load losses[g,1]; pass it to
 *                     vmoe_dispatch_route_bwd_dlogits
 *   logits, probs   [N, E] f32   vmoe_route's outputs (z is rebuilt in f32
 *                                 exactly as vmoe_route forms it)
 *   logit_bias [E], noise [N, E] f32 or NULL, as given to vmoe_route
 *   noise_std  > 0, the standard deviation the noise was drawn with
 *   losses [G, 2], dlogits [N, E] f32 out; importance, load [G, E] f32 out
 *   or NULL; workspace: vmoe_balance_loss_workspace_bytes(shape) bytes.
 * Sums over tokens are f32 within a chunk of tokens and double across chunks
 * in chunk order (deterministic); the chunk is 256 tokens for E <= 8, 64 for
 * E <= 16, 32 for E <= 32 and 16 for E <= 64. VMOE_ERR_INVALID_ARG for a
 * non-positive or non-finite noise_std or non-finite weights. */
vmoe_status vmoe_balance_loss(const vmoe_shape* shape, const float* logits,
                              const float* logit_bias, const float* noise, const float* probs,
                              float noise_std, float w_importance, float w_load, float* losses,
                              float* importance, float* load, float* dlogits, void* workspace,
                              size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Cross-task expert grouping (paper Sec. 3.2.1). HOST routines: every pointer
 * below is host memory, nothing runs on the GPU.
 * ------------------------------------------------------------------------- */

/* Temporary DRAM of one expert: M_tmp = B_p (theta1 T d_k + theta2 T^2) + m_f
 * bytes for T = tokens routed to it (m_c, the compute-dependent buffers, plus
 * m_f, the profiled per-call overhead). Evaluated as written, left to right. */
double vmoe_expert_mtmp(int64_t tokens, int32_t d_k, double bytes_per_elem, double theta1,
                        double theta2, double m_f);

/* Host scratch bytes for vmoe_group_experts (0 on invalid arguments). */
size_t vmoe_group_experts_workspace_bytes(int32_t n, double mem_budget, double mem_static,
                                          double unit_bytes);

/* Ordered time slices of n experts under a DRAM budget: slice s is the 0/1
 * knapsack optimum over the experts not in slices 0..s-1, with weight
 * w_i = ceil(mtmp[i] / unit_bytes), value v_i = mtmp[i] / mem_budget -
 * eta * lifespan[i], capacity floor((mem_budget - mem_static) / unit_bytes),
 * by dp[i][j] = max(dp[i-1][j], dp[i-1][j - w_i] + v_i) over the remaining
 * experts in index order (an expert enters only if strictly better; the set
 * is read back from full capacity). A slice with no gain takes the remaining
 * expert of shortest lifespan (lower index on ties), so every expert is placed.
 *   mtmp, lifespan [n] f64 (>= 0)   in
 *   slice_of       [n] i32          out: slice of each expert, 0-based
 *   n_slices       i32              out
 *   workspace      host memory of vmoe_group_experts_workspace_bytes(...)
 * VMOE_ERR_INVALID_ARG: n outside [0, 65536], unit_bytes <= 0, mem_budget <=
 * mem_static, a capacity above 2^24 units, a negative input, or an expert
 * whose weight alone exceeds the capacity; VMOE_ERR_WORKSPACE: too small. */
vmoe_status vmoe_group_experts(int32_t n, const double* mtmp, const double* lifespan,
                               double mem_budget, double mem_static, double eta,
                               double unit_bytes, int32_t* slice_of, int32_t* n_slices,
                               void* workspace, size_t workspace_bytes);

/* Lifespan aligning within a slice (paper Sec. 3.2.2): fill-clamp-refill
 * allocation of `budget` whole compute units (or workgroup slots) among n
 * experts. Every expert starts from min_units[i]; the rest is split among the
 * experts below saturation in proportion to coef[i] (>= 0; an expert with
 * coef 0 keeps its minimum); an expert pushed past sat_units[i] is clamped
 * there and its excess is split again among the others, until nothing is
 * returned (at most n rounds). Budget beyond the saturations stays unused.
 *   alloc [n] f64        out: the real shares; they equal
 *                        min(sat_i, min_i + lambda coef_i) with one lambda
 *   alloc_units [n] i32  out: largest-remainder rounding of alloc to
 *                        floor(sum alloc) units (each share rounded down or
 *                        up, ties to the lower index)
 *   n_rounds             out: share-clamp rounds taken
 *   workspace            host memory of at least 4 n bytes
 * HOST routine. VMOE_ERR_INVALID_ARG for n outside [0, 65536], a negative
 * minimum, sat < min, a negative or non-finite coefficient or a budget below
 * the sum of the minima; VMOE_ERR_WORKSPACE for a small workspace. */
vmoe_status vmoe_fill_clamp_refill(int32_t n, const int32_t* min_units, const int32_t* sat_units,
                                   const double* coef, int64_t budget, double* alloc,
                                   int32_t* alloc_units, int32_t* n_rounds, void* workspace,
                                   size_t workspace_bytes);

#ifdef __cplusplus
}
#endif

#endif /* VMOE_H */
