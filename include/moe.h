/*
 * moe.h -- C ABI of one GPU's share of a Mixture-of-Experts layer on MI355X
 * (gfx950): router, dispatch plan, routed + shared SwiGLU experts, combine,
 * and the backward pass.
 *
 * The layer is the one of "Mixture-of-Kittens: MoE Megakernel for NVL72s",
 * §2.1 (equation of MoE(x, s)):
 *
 *     Y[t] = f_shared(x_t) + sum_{e in S_t} w[t,e] * f_e(x_t),
 *     f_e(x) = (silu(x W_gate[e]) * (x W_up[e])) W_down[e],
 *
 * with S_t the k largest router logits Z[t,:] = x_t W_r + bias and w the
 * softmax of Z[t,:] renormalised over S_t.  Weights use row-vector
 * orientation: W_gate[e] is [d, f], the transpose of the paper's
 * column-vector matrix in R^{I x D}.
 *
 * Conventions shared by every entry point
 * ----------------------------------------
 * - Every tensor pointer is a DEVICE pointer to row-major, densely packed
 *   memory owned by the caller.  The library allocates nothing, keeps no
 *   global state, never synchronises the stream and never copies device
 *   data to the host, so every call can be captured in a HIP graph.
 * - bf16 tensors hold raw bf16 bit patterns (moe_bf16).  All conversions to
 *   bf16 round to nearest even.
 * - Every pointer must be 16-byte aligned.
 * - Arguments are validated on the host before anything is launched; on a
 *   validation error nothing is launched and outputs are untouched.
 * - Outputs are overwritten, never accumulated into.
 * - Work is enqueued on `stream` (a hipStream_t; NULL = null stream).  A
 *   return of MOE_OK means the launches were accepted; kernel faults surface
 *   through the HIP runtime at the caller's next synchronisation.
 * - Results are bitwise deterministic: no floating-point atomics, every
 *   reduction runs in a fixed order (§3.4 "Determinism").
 * - Route ids are token-major: route j = t*k + slot, and a token's slots
 *   list its selected experts in ascending expert id.
 *
 * Limits (MOE_EUNSUPPORTED outside them): d % 256 == 0, f % 256 == 0,
 * f_shared % 256 == 0, 1 <= k <= 16, k <= E <= 256, T*k < 2^31.
 */
#ifndef MOE_H
#define MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t moe_bf16;   /* bf16 bit pattern */
typedef void *moe_stream;    /* a hipStream_t */

/* Layer shape.  T tokens of width d, E local routed experts, top-k routing,
 * routed intermediate size f, shared-expert intermediate size f_shared
 * (0 = no shared expert). */
typedef struct {
    int64_t T, d, E, k, f, f_shared;
} moe_shape;

typedef enum {
    MOE_OK = 0,
    MOE_EINVAL = 1,        /* null/misaligned pointer, bad dimension, k > E */
    MOE_EUNSUPPORTED = 2,  /* valid but outside the limits above */
    MOE_ENOSPACE = 3,      /* workspace smaller than moe_workspace_bytes() */
    MOE_EHIP = 4           /* a HIP launch was rejected */
} moe_status;

/* Expert weights (all bf16, caller-owned, read-only). */
typedef struct {
    const moe_bf16 *W_gate;  /* [E, d, f] */
    const moe_bf16 *W_up;    /* [E, d, f] */
    const moe_bf16 *W_down;  /* [E, f, d] */
    const moe_bf16 *Wg_s;    /* [d, f_shared], NULL iff f_shared == 0 */
    const moe_bf16 *Wu_s;    /* [d, f_shared], NULL iff f_shared == 0 */
    const moe_bf16 *Wd_s;    /* [f_shared, d], NULL iff f_shared == 0 */
} moe_weights;

/* Dispatch plan (§3.1, Algorithm 1 with one source rank).  Written by
 * moe_plan, read by moe_dispatch / moe_forward / moe_backward. */
typedef struct {
    int32_t *counts;     /* [E]   routes per expert                        */
    int32_t *offsets;    /* [E+1] exclusive prefix of counts; [E] = T*k    */
    int32_t *perm;       /* [T*k] buffer position p -> route j             */
    int32_t *route_pos;  /* [T*k] route j -> buffer position p             */
} moe_plan_bufs;

/* Gradients written by moe_backward (fp32, overwritten). */
typedef struct {
    float *dW_gate;  /* [E, d, f] */
    float *dW_up;    /* [E, d, f] */
    float *dW_down;  /* [E, f, d] */
    float *dW_r;     /* [d, E]    */
    float *dZ;       /* [T, E] gradient wrt the router logits (zero for
                        unselected experts); may be NULL (kept internally) */
    float *dWg_s;    /* [d, f_shared], NULL iff f_shared == 0 */
    float *dWu_s;    /* [d, f_shared], NULL iff f_shared == 0 */
    float *dWd_s;    /* [f_shared, d], NULL iff f_shared == 0 */
} moe_grads;

/* Named regions of the workspace, for inspection after a synchronisation.
 * With dense routing (k == E: every token routes to every local expert)
 * moe_forward and moe_forward_fused keep w * h in MOE_WS_H and write neither
 * MOE_WS_YEXP nor MOE_WS_YSH, and moe_backward does not write MOE_WS_DXPERM:
 * the combines are folded into the down and dX products (see moe_forward). */
typedef enum {
    MOE_WS_ERROR = 0,   /* int32[1], reset by moe_plan.  Bit 0: moe_plan
                           saw an expert id outside [0, E) (such routes are
                           left unplaced).  Bit 1: a dependency wait of
                           moe_forward_fused gave up (results invalid). */
    MOE_WS_A = 1,       /* bf16 [T*k, f]  x W_gate[e] in plan order         */
    MOE_WS_B = 2,       /* bf16 [T*k, f]  x W_up[e]                         */
    MOE_WS_H = 3,       /* bf16 [T*k, f]  silu(A) * B                       */
    MOE_WS_YEXP = 4,    /* bf16 [T*k, d]  f_e(x) per route, plan order      */
    MOE_WS_YSH = 5,     /* bf16 [T, d]    shared-expert output              */
    MOE_WS_DG = 6,      /* fp32 [T*k]     <dY, f_e(x)> per route, plan order*/
    MOE_WS_DA = 7,      /* bf16 [T*k, f]  gradient wrt A                    */
    MOE_WS_DB = 8,      /* bf16 [T*k, f]  gradient wrt B                    */
    MOE_WS_DXPERM = 9,  /* bf16 [T*k, d]  routed dX terms, plan order       */
    /* MXFP8 forward only (moe_mx_workspace_region): */
    MOE_WS_XQ = 10,     /* E4M3 [T, d]    X, one scale per 32 of d          */
    MOE_WS_XS = 11,     /* E8M0 [T, d/32] scales of MOE_WS_XQ               */
    MOE_WS_HQ = 12,     /* E4M3 [T*k, f]  gated activation, plan order      */
    MOE_WS_HS = 13,     /* E8M0 [T*k, f/32] scales of MOE_WS_HQ             */
    /* MXFP8 backward only (moe_mx_workspace_region): */
    MOE_WS_DYQ = 14,    /* E4M3 [T, d]    dY, one scale per 32 of d         */
    MOE_WS_DYS = 15,    /* E8M0 [T, d/32] scales of MOE_WS_DYQ              */
    MOE_WS_DAQ = 16,    /* E4M3 [T*k, f]  gradient wrt A, plan order        */
    MOE_WS_DAS = 17,    /* E8M0 [T*k, f/32]                                 */
    MOE_WS_DBQ = 18,    /* E4M3 [T*k, f]  gradient wrt B                    */
    MOE_WS_DBS = 19,    /* E8M0 [T*k, f/32]                                 */
    /* MXFP8 weight gradients only (moe_backward_mx with wgrad_mxfp8 = 1).
     * Expert e's plan rows sit at padded positions [poff[e], poff[e] + count)
     * of a token axis of P = roundup(T*k + 128 E, 128) positions; poff[e] is
     * a multiple of 128, and positions past an expert's rows hold zeros.
     * With dense routing (k = E) every expert's rows are tokens 0 .. T-1 in
     * order, so X^T and dY^T are written for expert 0's range only, which
     * every expert's weight-gradient product reads. */
    MOE_WS_POFF = 20,   /* int32 [E+1]    padded expert offsets             */
    MOE_WS_XTQ = 21,    /* E4M3 [d, P]    X^T by token, 32-blocks along P   */
    MOE_WS_XTS = 22,    /* E8M0 [d, P/32]                                   */
    MOE_WS_DYTQ = 23,   /* E4M3 [d, P]    dY^T likewise                     */
    MOE_WS_DYTS = 24,   /* E8M0 [d, P/32]                                   */
    /* Backward (either layout): */
    MOE_WS_HW = 25,     /* bf16 [T*k, f]  gate weight times silu(A) * B     */
    /* MXFP8 only (moe_mx_workspace_region).  Values a quantiser reads are
     * kept at the precision they were produced in (fp32): */
    MOE_WS_AF = 26,     /* fp32 [T*k, f]  routed gate pre-activation A,
                           kept by moe_forward_mx (save_for_backward = 1)   */
    MOE_WS_BF = 27,     /* fp32 [T*k, f]  routed up pre-activation B        */
    MOE_WS_DAF = 28,    /* fp32 [T*k, f]  dA (moe_backward_mx, wgrad_mxfp8 = 1) */
    MOE_WS_DBF = 29,    /* fp32 [T*k, f]  dB (same)                          */
    MOE_WS_HWF = 30,    /* fp32 [T*k, f]  gate weight times h (same)         */
    MOE_WS_COUNT = 31
} moe_ws_tensor;

/* MXFP8 routed-expert weights (§3.4 "MXFP8 Support"), written once by
 * moe_mx_quantize_weights and read by moe_forward_mx.  Codes are OCP FP8
 * E4M3; each scale byte b stands for 2^(b - 127) and covers 32 consecutive
 * elements along the contraction axis of the GEMM that reads the weight.
 * Both are stored K-contiguous, i.e. transposed from the bf16 layout:
 *   Wg_q, Wu_q [E, f, d] codes: row n is column n of W_gate[e] / W_up[e]
 *   Wg_s, Wu_s [E, f, d/32] scales
 *   Wd_q       [E, d, f] codes: row n is column n of W_down[e]
 *   Wd_s       [E, d, f/32] scales
 * Quantisation of a block with largest magnitude amax: scale exponent
 * s = floor(log2(amax)) - 8, clamped to [-127, 127] (-127 for an all-zero
 * block); each element is x * 2^-s clamped to +-448 and rounded to the
 * nearest E4M3 value, ties to even (a negative value that rounds to zero
 * keeps its sign). */
typedef struct {
    uint8_t *Wg_q, *Wu_q, *Wd_q;
    uint8_t *Wg_s, *Wu_s, *Wd_s;
} moe_mx_weights;

/* Optional per-stage timing.  When a moe_stage_events pointer is passed to
 * moe_forward / moe_backward, ev[i] (a hipEvent_t, or NULL to skip) is
 * recorded on the stream just before stage i is enqueued and ev[n] after the
 * last stage, so the elapsed time between ev[i] and ev[i+1] is stage i.
 * Stages that do not apply (no shared expert) still record their events.
 *   forward  (n = 6): 0 plan-order prologue, 1 routed up/gate + SwiGLU,
 *                     2 shared up/gate + SwiGLU, 3 routed down, 4 shared down,
 *                     5 combine.
 *   backward (n = 11): 0 prologue, 1 routed dgrad + SwiGLU backward,
 *                     2 softmax backward, 3 routed dX GEMM, 4 routed dW_gate
 *                     and dW_up, 5 routed dW_down, 6 shared dgrad, 7 shared
 *                     dX GEMM, 8 shared weight gradients, 9 dW_r,
 *                     10 reverse combine. */
#define MOE_MAX_STAGE_EVENTS 16
typedef struct {
    void *ev[MOE_MAX_STAGE_EVENTS];
} moe_stage_events;

/* Workspace bytes needed by moe_route/moe_plan/moe_forward (with_backward=0)
 * or additionally moe_backward (with_backward=1).  Pure host function;
 * returns 0 for an invalid or unsupported shape. */
size_t moe_workspace_bytes(const moe_shape *shape, int with_backward);

/* Byte offset and size of a named workspace region (host only). */
moe_status moe_workspace_region(const moe_shape *shape, int with_backward,
                                moe_ws_tensor which, size_t *offset, size_t *bytes);

/* Router (§2.1: the router projection selects the top-k experts and assigns
 * each a weight).
 *   X [T, d] bf16, W_r [d, E] bf16, bias [E] fp32 or NULL.
 *   logits  [T, E] fp32 out: Z = X W_r + bias (fp32 accumulation).
 *   topk_idx [T, k] int32 out: the k largest logits, ties to the lower
 *            expert id, listed in ascending expert id.
 *   topk_w  [T, k] fp32 out: exp(Z_te) / sum_{e' in S_t} exp(Z_te').
 * Uses the workspace for a transposed copy of W_r and, with 128 or more
 * experts, for fp32 partial logits of slices of the d axis (added in slice
 * order, so the logits are deterministic). */
moe_status moe_route(const moe_shape *shape, const moe_bf16 *X, const moe_bf16 *W_r,
                     const float *bias, float *logits, int32_t *topk_idx, float *topk_w,
                     void *ws, size_t ws_bytes, moe_stream stream);

/* Dispatch plan (§3.1, Algorithm 1 for one source rank: a stable counting
 * sort of the routes by expert; no host readback).
 *   topk_idx [T, k] int32 in.  plan: counts, offsets, perm, route_pos out.
 * An expert id outside [0, E) sets the MOE_WS_ERROR word; that route gets
 * no position (perm/route_pos entries are then unspecified and the later
 * steps bound-check every index they read). */
moe_status moe_plan(const moe_shape *shape, const int32_t *topk_idx,
                    const moe_plan_bufs *plan, void *ws, size_t ws_bytes,
                    moe_stream stream);

/* The dispatch plan of moe_plan for callers that cannot allocate device
 * memory or pass a workspace (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation).  Same inputs and plan outputs as
 * moe_plan; its scratch (per-chunk histograms, bases and flags) lives in a
 * device array of MOE_PLAN_NOALLOC_SCRATCH_BYTES that the library holds on
 * each GPU it runs on until the process ends.  The call allocates nothing
 * (no hipMalloc, hipFree or allocating library routine).
 *   error_word [1] int32 out (device): 1 if some expert id lies outside
 *              [0, E) (that route is left unplaced, as in moe_plan), else 0.
 * The plan needs 8 * ceil(T*k / 1024) * E bytes of scratch (each of its
 * regions rounded up to 256 bytes) plus 4 * ceil(T*k / 1024): shapes needing
 * more than MOE_PLAN_NOALLOC_SCRATCH_BYTES return MOE_EUNSUPPORTED before
 * anything is launched (at E = 256 that admits T*k up to about 2 million
 * routes).  All calls on one GPU share its array: calls that overlap on one
 * GPU (on different streams, or from different threads) race and must be
 * serialised by the caller.  Other errors as moe_plan; MOE_EHIP also when
 * the array's device address cannot be obtained. */
#define MOE_PLAN_NOALLOC_SCRATCH_BYTES (4u << 20)
moe_status moe_plan_noalloc(const moe_shape *shape, const int32_t *topk_idx,
                            const moe_plan_bufs *plan, int32_t *error_word, moe_stream stream);

/* Pull-based dispatch schedule for R source ranks (§3.1, Algorithm 1, and
 * its sort-key statement in "Scheduling").  Each of R ranks holds N tokens
 * with K routes each; A is the all-gathered route table and the schedule is
 * the one rank c builds for its L local experts (global ids c*L .. c*L+L-1).
 *   A   [R, NK] int32 in: A[r*NK + j] = global expert id of route j of
 *       source rank r, in [0, R*L).
 *   M   [R, L] int32 out: M[r*L + l] = routes of rank r to local expert l.
 *   S   [L+1] int32 out: S[l] = start of local expert l's region
 *       (sum of M over all ranks and all experts before l); S[L] = P, the
 *       number of routes this rank receives.
 *   phi [phi_rows, 2] int32 out: row p < P holds (source rank r, route j):
 *       buffer position p receives route j of rank r.  Within a region the
 *       rows are ordered by (o, r), o = number of earlier routes of row r to
 *       the same expert, so source ranks interleave round-robin.  Rows >= P
 *       are not written.
 * Error word (the first int32 of ws, readable after a synchronisation):
 * bit 0 = some id outside [0, R*L) (such routes are never scheduled, the
 * counts ignore them); bit 1 = P > phi_rows (rows past phi_rows are
 * dropped).  Work per local route is O(R).  With R = 1 and c = 0 the
 * schedule equals moe_plan's perm.
 * Limits: 1 <= R <= 1024, 1 <= L <= 256, 0 <= c < R, 0 <= NK, R*NK < 2^31,
 * L * (R rounded up to a multiple of 4) <= 8192; otherwise MOE_EINVAL
 * (R, L < 1, NK < 0, c outside [0, R), phi_rows < 0, null or misaligned
 * pointer), MOE_EUNSUPPORTED (outside the limits) or MOE_ENOSPACE (ws_bytes
 * below moe_schedule_workspace_bytes, a pure host function that returns 0
 * for invalid or unsupported dimensions). */
size_t moe_schedule_workspace_bytes(int64_t R, int64_t NK, int64_t L);
moe_status moe_schedule(int64_t R, int64_t NK, int64_t L, int64_t c, const int32_t *A,
                        int32_t *M, int32_t *S, int32_t *phi, int64_t phi_rows, void *ws,
                        size_t ws_bytes, moe_stream stream);

/* MXFP8 weight pre-quantisation (§3.4 "MXFP8 Support": weights are
 * quantised ahead of time by a dedicated kernel).  Reads W_gate, W_up,
 * W_down of `weights` (the shared-expert pointers are ignored) and writes
 * every array of `mx` (layouts above; caller-owned device memory).  Extra
 * limits: T*d, T*k*f and E*f*d below 2^32 (MOE_EUNSUPPORTED). */
moe_status moe_mx_quantize_weights(const moe_shape *shape, const moe_weights *weights,
                                   const moe_mx_weights *mx, moe_stream stream);

/* Workspace bytes of moe_forward_mx (with_backward = 0; it also serves
 * moe_route and moe_plan), of moe_forward_mx with save_for_backward = 1
 * followed by moe_backward_mx (with_backward = 1), or of the same with the
 * MXFP8 weight gradients (with_backward = 2; adds the token-axis operands,
 * (2 d + 3 f) P bytes of codes and 1/32 of that of scales, P as for
 * MOE_WS_POFF, and their fp32 sources, 12 T k f bytes); 0 for an invalid or
 * unsupported shape.  Pure host function. */
size_t moe_mx_workspace_bytes(const moe_shape *shape, int with_backward);

/* Byte offset and size of a region of the MXFP8 workspace: the MXFP8 regions
 * MOE_WS_XQ .. MOE_WS_DYTS, or any region of moe_workspace_region's
 * backward layout (the MXFP8 paths use it for the rest). */
moe_status moe_mx_workspace_region(const moe_shape *shape, moe_ws_tensor which, size_t *offset,
                                   size_t *bytes);

/* MXFP8 weights for the backward (§3.4 "MXFP8 Support"), written by
 * moe_mx_quantize_weights_bwd.  Each weight row is quantised along the axis
 * its backward product contracts, which is its contiguous axis, so the
 * layouts are those of the bf16 weights:
 *   Wg_q, Wu_q [E, d, f] codes, blocks along f; Wg_s, Wu_s [E, d, f/32]
 *   Wd_q       [E, f, d] codes, blocks along d; Wd_s       [E, f, d/32]
 * (same quantisation rule as moe_mx_weights). */
typedef struct {
    uint8_t *Wg_q, *Wu_q, *Wd_q;
    uint8_t *Wg_s, *Wu_s, *Wd_s;
} moe_mx_bwd_weights;

/* Pre-quantises the routed weights for moe_backward_mx (once per weight
 * update).  Reads W_gate, W_up, W_down of `weights`; writes every array of
 * `mx`.  Limits as moe_mx_quantize_weights. */
moe_status moe_mx_quantize_weights_bwd(const moe_shape *shape, const moe_weights *weights,
                                       const moe_mx_bwd_weights *mx, moe_stream stream);

/* Forward of the layer with MXFP8 routed experts and a BF16 shared expert
 * (§3.4 "MXFP8 Support").  As moe_forward, except:
 *   - X is quantised once per token (32-blocks along d) before the routed
 *     up/gate GEMM reads it through the plan;
 *   - the routed GEMMs run on E4M3 x E4M3 block-scaled matrix cores with
 *     fp32 accumulation, on the weights in `mx`;
 *   - the gated activation H is quantised along f (32-blocks) straight from
 *     fp32 in the up/gate epilogue, and Yexp is rounded to bf16;
 *   - `weights` supplies only the shared expert (its routed pointers are
 *     ignored and may be NULL);
 *   - save_for_backward = 1 keeps the routed pre-activations A, B in fp32
 *     (the accumulators of the MXFP8 products; the backward's dA, dB
 *     quantisation reads values computed from them) and the shared
 *     expert's in bf16, for moe_backward_mx.
 * Y [T, d] bf16 out.  ws: at least moe_mx_workspace_bytes(shape,
 * save_for_backward) bytes. */
moe_status moe_forward_mx(const moe_shape *shape, const moe_bf16 *X, const moe_weights *weights,
                          const moe_mx_weights *mx, const int32_t *topk_idx, const float *topk_w,
                          const moe_plan_bufs *plan, moe_bf16 *Y, int save_for_backward, void *ws,
                          size_t ws_bytes, moe_stream stream,
                          const moe_stage_events *events /* NULL = no timing */);

/* Backward of the layer with MXFP8 routed experts (§3.4 "MXFP8 Support":
 * activation quantisation fused into the dispatch, the grouped GEMMs and the
 * gated activation).  As moe_backward, except:
 *   - dY is quantised once per token along d, and dh' = Q(dY) Q(W_down)^T
 *     runs on the block-scaled matrix cores with the weights in `mx`;
 *   - the gated-activation backward in that GEMM's epilogue (on the fp32
 *     A, B the forward kept) quantises dA, dB along f from their fp32
 *     values, and dXperm = Q(dA) Q(W_gate)^T + Q(dB) Q(W_up)^T runs in MXFP8;
 *   - the weight gradients contract over each expert's ragged token set;
 *     with wgrad_mxfp8 = 0 they stay BF16 on X, dY and dA, dB, w h stored
 *     in bf16 (MOE_WS_DA, MOE_WS_DB, MOE_WS_HW); with wgrad_mxfp8 = 1 dA,
 *     dB, w h are stored in fp32 instead (MOE_WS_DAF .. MOE_WS_HWF) and
 *     every operand is quantised along the token axis (blocks of 32 plan
 *     rows from each expert's first row; the quantisation the
 *     expert-grouped GEMMs need for a contraction over tokens), and
 *     dW_gate = Q_t(X_e)^T Q_t(dA_e), dW_up = Q_t(X_e)^T Q_t(dB_e),
 *     dW_down = Q_t(w h)^T Q_t(dY_e) run on the block-scaled matrix cores;
 *   - the shared expert, the router gradient and dX's router term are those
 *     of moe_backward.
 * Needs the ws of a preceding moe_forward_mx with save_for_backward = 1 (at
 * least moe_mx_workspace_bytes(shape, 1 + wgrad_mxfp8) bytes) and the same
 * inputs.  `weights` as for moe_backward.  wgrad_mxfp8 is 0 or 1 (else
 * MOE_EINVAL); with 1, d*P and f*P must stay below 2^32 (P as for
 * MOE_WS_POFF; else MOE_EUNSUPPORTED). */
moe_status moe_backward_mx(const moe_shape *shape, const moe_bf16 *dY, const moe_bf16 *X,
                           const moe_bf16 *W_r, const moe_weights *weights,
                           const moe_mx_bwd_weights *mx, const int32_t *topk_idx,
                           const float *topk_w, const moe_plan_bufs *plan, moe_bf16 *dX,
                           const moe_grads *grads, int wgrad_mxfp8, void *ws, size_t ws_bytes,
                           moe_stream stream);

/* Materialised dispatch (§3.1 "Scheduling", local part): Xperm[p] =
 * X[perm[p] / k] for p < T*k.  moe_forward does not need it (its GEMMs read
 * token rows through the plan); it exists for callers that want the
 * expert-contiguous buffer itself.  Xperm [T*k, d] bf16 out. */
moe_status moe_dispatch(const moe_shape *shape, const moe_bf16 *X,
                        const moe_plan_bufs *plan, moe_bf16 *Xperm, moe_stream stream);

/* Forward of the layer (§2.1 equation).
 *   X [T, d], weights, topk_idx/topk_w from moe_route, plan from moe_plan.
 *   Y [T, d] bf16 out: Ysh[t] + sum over the token's experts in ascending
 *   id of w * f_e(x_t), accumulated in fp32 and rounded once.
 *   save_for_backward: keep A and B (gate/up pre-activations) in ws.
 * Dense routing (k == E; each token's k ids are then 0 .. E-1): the token's
 * route to expert e is plan row offsets[e] + t, so the combine is one
 * contraction over the experts' intermediate columns in ascending expert id
 * followed by the shared expert's: Y[t] = sum_e (w h_e[t]) W_down[e] +
 * h_s[t] Wd_s in one fp32 accumulator (w h rounded to bf16), rounded once.
 * The same holds for dX in moe_backward (routed terms in ascending expert
 * id, then the shared expert, then dZ[t] W_r^T, one fp32 accumulator). */
moe_status moe_forward(const moe_shape *shape, const moe_bf16 *X, const moe_weights *weights,
                       const int32_t *topk_idx, const float *topk_w,
                       const moe_plan_bufs *plan, moe_bf16 *Y, int save_for_backward,
                       void *ws, size_t ws_bytes, moe_stream stream,
                       const moe_stage_events *events /* NULL = no timing */);

/* Forward of the layer as one persistent launch (§3.2: all of the layer's
 * computation fused into one kernel; §3.4 "Shared Expert": the shared
 * expert's tiles are scheduled first).  One workgroup per compute unit takes
 * work items from per-XCD queues in a fixed order: shared up/gate tiles,
 * routed up/gate tiles, shared down tiles, routed down tiles, then the
 * combine of blocks of 16 tokens.  A down tile starts when every up/gate tile
 * of its rows is done; a token block's combine starts when the down tiles
 * holding all of its routes are done, so the combine overlaps the last down
 * tiles instead of following them.
 * Same arguments, workspace and results as moe_forward, bitwise (each tile
 * runs the same code, the combine adds in the same order); A and B are kept
 * when save_for_backward = 1, so moe_backward can follow.  Every wait is
 * bounded: if one gives up, bit 1 of the MOE_WS_ERROR word is set and the
 * launch still ends (the outputs are then invalid). */
moe_status moe_forward_fused(const moe_shape *shape, const moe_bf16 *X, const moe_weights *weights,
                             const int32_t *topk_idx, const float *topk_w,
                             const moe_plan_bufs *plan, moe_bf16 *Y, int save_for_backward,
                             void *ws, size_t ws_bytes, moe_stream stream);

/* Backward of the layer for upstream gradient dY [T, d] bf16, with the
 * selection held fixed.  Needs the same ws as a preceding moe_forward with
 * save_for_backward = 1 and the same inputs.  The router-weight gradient
 * uses <dY, f_e(x)> = <dY W_down[e]^T, h> (§3.4 "Router Weight Gradient
 * Computation"), fused into the gated-activation backward.
 *   dX [T, d] bf16 out; grads out (fp32). */
moe_status moe_backward(const moe_shape *shape, const moe_bf16 *dY, const moe_bf16 *X,
                        const moe_bf16 *W_r, const moe_weights *weights,
                        const int32_t *topk_idx, const float *topk_w,
                        const moe_plan_bufs *plan, moe_bf16 *dX, const moe_grads *grads,
                        void *ws, size_t ws_bytes, moe_stream stream,
                        const moe_stage_events *events /* NULL = no timing */);

/* Bounded-memory execution (§3.3 "macrobatch" ring buffer and "Ring-Aware
 * Forward Replay").  The per-route activations (A, B, H, Yexp and their
 * gradients) live in a ring of ring_rows rows instead of T*k rows; the plan
 * positions are processed in windows [m C, min((m+1) C, T*k)), C = ring_rows.
 *
 *   moe_forward_ring  runs the windows in descending order (reverse
 *                     macrobatch order) after the shared expert, so the
 *                     ring ends holding window 0 in full.  Per window: the
 *                     routed up/gate + SwiGLU and down GEMMs, then each
 *                     token's routes that fall in the window are added, in
 *                     ascending slot order and weighted, to an fp32
 *                     per-token accumulator seeded with the shared-expert
 *                     output; the last window rounds it into Y.
 *   moe_backward_ring runs the windows in ascending order: window 0 uses the
 *                     activations the forward left in the ring; the gate/up
 *                     pre-activations of every later window are recomputed
 *                     (A, B only: the down projection and H are not
 *                     replayed), in the same launch as the previous window's
 *                     weight gradients.  Weight gradients of a window are
 *                     added to the previous windows' in fp32; the routed dX
 *                     terms are summed per token across windows as in the
 *                     forward.
 *
 * Results are deterministic.  With one window (ring_rows >= T*k) they are
 * bitwise those of moe_forward / moe_backward; with several, Y, dX and the
 * routed weight gradients differ only by fp32 summation order, and dZ and
 * dW_r are bitwise those of moe_backward.
 *   ring_rows >= 1 (MOE_EINVAL otherwise), < 2^31.
 *   ws: at least moe_ring_workspace_bytes(shape, ring_rows, with_backward)
 *   bytes; the region layout differs from moe_workspace_region's, so the
 *   ring entry points and moe_forward / moe_backward must not share a ws
 *   between a forward and its backward.  moe_route and moe_plan accept a
 *   ring workspace.  moe_backward_ring needs the ws of a preceding
 *   moe_forward_ring with save_for_backward = 1, the same ring_rows and the
 *   same inputs.  Other arguments as moe_forward / moe_backward. */
size_t moe_ring_workspace_bytes(const moe_shape *shape, int64_t ring_rows, int with_backward);

moe_status moe_forward_ring(const moe_shape *shape, const moe_bf16 *X, const moe_weights *weights,
                            const int32_t *topk_idx, const float *topk_w,
                            const moe_plan_bufs *plan, moe_bf16 *Y, int64_t ring_rows,
                            int save_for_backward, void *ws, size_t ws_bytes, moe_stream stream);

moe_status moe_backward_ring(const moe_shape *shape, const moe_bf16 *dY, const moe_bf16 *X,
                             const moe_bf16 *W_r, const moe_weights *weights,
                             const int32_t *topk_idx, const float *topk_w,
                             const moe_plan_bufs *plan, moe_bf16 *dX, const moe_grads *grads,
                             int64_t ring_rows, void *ws, size_t ws_bytes, moe_stream stream);

/* Static strings; never NULL. */
const char *moe_status_string(moe_status status);
const char *moe_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MOE_H */
