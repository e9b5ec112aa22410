/*
 * moe_vie.h - C ABI of the MI355X (gfx950) forward pass of one fine-grained
 * Mixture-of-Experts MLP layer of a ViT encoder (MoE-ViE).
 *
 * The layer, per token x in R^d (paper Sec. 3.1 Eq. (1)-(3), Sec. 3.2
 * Eq. (4)-(7)):
 *   s      = W_r x                                   router logits, E routed experts
 *   sel    = top-K of Sigmoid(s) + b                 b only selects experts
 *   g'_e   = Sigmoid(s_e) / sum_{i in sel} Sigmoid(s_i)     for e in sel
 *   y      = sum_{e in sel} g'_e E_e(x) + lambda * E_shared(x)
 *   E(x)   = W2 GELU(W1 x)                           fc1 -> GELU -> fc2
 * or, with MOE_FLAG_SWIGLU, SwiGLU experts (appendix "MoE Kernel",
 * Algorithm 1, Phase 2, and the SwiGLU MLPs of appendix "Implementation
 * Details"):
 *   E(x)   = W2 (SiLU(W1 x) * (W3 x)),  SiLU(v) = v / (1 + exp(-v))
 * GELU(v) = v Phi(v): fp32 layers evaluate the erf form with the device erff;
 * bf16 layers use v times the sigmoid of a clamped odd quintic in v, within
 * 2.6e-5 (absolute) of the erf form (see moe_grouped_mlp).
 * The stages (route, permute, grouped expert MLP, combine) are exposed
 * separately and fused in moe_layer_forward.
 *
 * Conventions shared by every entry point
 *  - All tensors are row-major and live in device memory of the current HIP
 *    device; the caller allocates and owns every buffer, the library
 *    allocates nothing and keeps no state between calls (the one exception
 *    is the device scratch of moe_layer_forward_noalloc, below).
 *  - "Layer dtype" (desc->dtype) is the element type of x, all weights,
 *    expert outputs and y: MOE_F32 (fp32) or MOE_BF16 (bf16 bit patterns,
 *    round-to-nearest-even). Biases and gates are fp32, indices int32.
 *  - Weights use the nn.Linear layout [out, in]: W_r [E, d], W1 [E, h, d],
 *    W2 [E, d, h], shared W1s [h_s, d], W2s [d, h_s].
 *  - SwiGLU experts (MOE_FLAG_SWIGLU) pass the gate and up projections
 *    stacked, "w13" [E, 2h, d]: rows 0..h-1 are W1 (gate), rows h..2h-1 are
 *    W3 (up); the shared expert likewise [2 h_s, d]. The second layer is
 *    stored with its rows padded to ldh = h rounded up to a multiple of 64:
 *    W2 [E, d, ldh] and W2s [d, ldh_s]; columns h..ldh-1 may hold any finite
 *    values (they multiply activation columns that are exactly zero). h and
 *    h_s may then be any value in [1, 8192].
 *  - A "slot" is one (token, choice) pair, slot id n = t*K + j, j < K.
 *  - Every call is asynchronous on `stream` (a hipStream_t; NULL is the
 *    default stream) and never synchronises with the host.
 *  - Arguments are validated on the host before anything is enqueued; a call
 *    that returns an error has enqueued nothing. Inputs must be finite.
 *  - Pointers must be 16-byte aligned; d must be a multiple of 64, and so
 *    must h and h_s for GELU experts.
 *  - Calls on one stream are ordered; calls that share output or workspace
 *    buffers must not overlap on different streams.
 */
#ifndef MOE_VIE_H
#define MOE_VIE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MOE_OK = 0,
    MOE_ERR_INVALID_ARG = 1, /* null pointer, bad size, misaligned pointer   */
    MOE_ERR_UNSUPPORTED = 2, /* dtype or shape outside what is implemented  */
    MOE_ERR_WORKSPACE = 3,   /* workspace smaller than moe_workspace_size   */
    MOE_ERR_HIP = 4          /* a HIP runtime call or kernel launch failed  */
} moe_status_t;

typedef enum { MOE_F32 = 0, MOE_BF16 = 1 } moe_dtype_t;

/* Flags of moe_desc_t.flags. */
#define MOE_FLAG_EXACT_ROUTER 1 /* compute every router logit by the exact chain
                                   (no MFMA pre-pass); the routing result is the
                                   same bit for bit, only the work differs */
#define MOE_FLAG_SWIGLU 2       /* SwiGLU experts (bf16 layers only): see below */

/* Layer descriptor. Limits: 1 <= T, T*K < 2^31; 1 <= K <= 16; K <= E <= 1024;
 * 64 <= d <= 8192 a multiple of 64; h and h_shared (0 = no shared expert)
 * at most 8192 and, for GELU experts, multiples of 64 and >= 64; x
 * (T*d elements), the expert activations (T*K*ldh) and the shared
 * activations (T*ldh_s) each below 4 GiB in bytes of the layer dtype (ldh = h
 * for GELU experts); flags a combination of MOE_FLAG_* bits (MOE_FLAG_SWIGLU
 * needs dtype MOE_BF16). */
typedef struct {
    int32_t T;        /* tokens                                   */
    int32_t d;        /* model width                              */
    int32_t E;        /* routed experts                           */
    int32_t K;        /* experts chosen per token                 */
    int32_t h;        /* hidden width of one routed expert        */
    int32_t h_shared; /* hidden width of the shared expert, or 0  */
    float lambda;     /* weight of the shared expert (paper: 1)   */
    int32_t dtype;    /* moe_dtype_t                              */
    int32_t flags;    /* MOE_FLAG_* bits, 0 by default            */
} moe_desc_t;

/* Human-readable name of a status code (static string). */
const char *moe_status_string(moe_status_t status);

/* Details of the last error returned on the calling host thread (static,
 * thread-local buffer; "" if none). */
const char *moe_last_error(void);

/* Bytes of device workspace that every entry point below needs for `desc`
 * (one size serves all of them). Writes *bytes; validates desc. */
moe_status_t moe_workspace_size(const moe_desc_t *desc, size_t *bytes);

/* Stages 1+2: router and gating (Eq. (1), Eqs. (4)-(5), Eq. (7)).
 *   x         [T, d] layer dtype          w_router [E, d] layer dtype
 *   bias      [E] fp32 or NULL (= 0): added to the sigmoid score for
 *             selection only
 *   topk_idx  [T, K] int32 out: chosen experts, in descending selection key
 *             (Sigmoid(s_e) + b_e); equal keys go to the lower expert index
 *   topk_gate [T, K] fp32 out: Sigmoid(s_e) / sum of Sigmoid over the chosen
 * Arithmetic is fp32 and reproducible bit for bit: each logit is one fused
 * multiply-add chain over i = 0..d-1 in ascending order starting from +0;
 * the sigmoid is 1/(1 + exp(-s)) with -s clamped to [-87, 87]
 * and evaluated by Cody-Waite reduction with ln2 = 22713*2^-15 + fl32(ln2 -
 * 22713*2^-15) and a degree-7 Taylor polynomial in Horner form; the gate
 * denominator is summed in slot order. For bf16 layers the logits are first
 * computed with bf16 MFMA; every expert whose key
 * could still reach the top K under a proven bound on the difference is then
 * recomputed with the exact chain, so the result is the exact one.
 * Uses the workspace. */
moe_status_t moe_route(const moe_desc_t *desc, const void *x, const void *w_router,
                       const float *bias, int32_t *topk_idx, float *topk_gate, void *workspace,
                       size_t workspace_bytes, void *stream);

/* Stage 3: group slots by expert (Algorithm 1, Phase 1: sort by expert id,
 * bincount, cumulative sum).
 *   topk_idx     [T, K] int32 in, every entry in [0, E)
 *   counts       [E] int32 out: slots routed to each expert
 *   offsets      [E+1] int32 out: exclusive prefix sum of counts
 *   sorted_slots [T*K] int32 out: slot ids grouped by expert; within an
 *                expert in ascending slot id (a stable sort)
 * Deterministic; uses the workspace. */
moe_status_t moe_permute(const moe_desc_t *desc, const int32_t *topk_idx, int32_t *counts,
                         int32_t *offsets, int32_t *sorted_slots, void *workspace,
                         size_t workspace_bytes, void *stream);

/* Stage 4: grouped expert MLPs (Algorithm 1, Phases 2-3, with fc1 -> GELU ->
 * fc2 experts and no routing weight applied).
 *   x            [T, d] layer dtype: token rows, gathered via slot / K
 *   sorted_slots [T*K], offsets [E+1]: as produced by moe_permute
 *   w1 [E, h, d], w2 [E, d, h] layer dtype (SwiGLU: w1 = w13 [E, 2h, d],
 *                w2 [E, d, ldh], see the conventions above)
 *   expert_out   [T*K, d] layer dtype out, row n = W2[e] GELU(W1[e] x_t) for
 *                slot n = t*K + j routed to expert e (SwiGLU:
 *                W2[e] (SiLU(W1[e] x_t) * (W3[e] x_t)))
 * For bf16 the activation (GELU(W1 x), or SiLU(W1 x) * W3 x with both
 * projections accumulated in fp32 in the same kernel) is rounded to bf16
 * before fc2; accumulation is fp32. bf16 layers evaluate GELU within 2.6e-5
 * (absolute) of the erf form, fp32 layers with the device erff. The shared expert can be run through this call with
 * a descriptor {E = 1, K = 1, h = h_s}, sorted_slots = 0..T-1, offsets =
 * {0, T}. Uses the workspace. */
moe_status_t moe_grouped_mlp(const moe_desc_t *desc, const void *x, const int32_t *sorted_slots,
                             const int32_t *offsets, const void *w1, const void *w2,
                             void *expert_out, void *workspace, size_t workspace_bytes,
                             void *stream);

/* Stage 5: gate-weighted combine back to token order (Eq. (6)).
 *   expert_out [T*K, d] layer dtype, topk_gate [T, K] fp32
 *   shared_out [T, d] layer dtype or NULL: added with weight desc->lambda
 *   y          [T, d] layer dtype out
 * y[t] = sum_j topk_gate[t, j] * expert_out[t*K + j] + lambda * shared_out[t],
 * accumulated in fp32 in that order (deterministic, no atomics). */
moe_status_t moe_combine(const moe_desc_t *desc, const void *expert_out, const float *topk_gate,
                         const void *shared_out, void *y, void *stream);

/* The whole layer (Eq. (6) with routing by Eq. (7)): route, permute, grouped
 * routed experts, shared expert (if desc->h_shared > 0) and combine, enqueued
 * back to back on `stream` with no host synchronisation.
 *   x [T, d], w_router [E, d], bias [E] fp32 or NULL, w1 [E, h, d],
 *   w2 [E, d, h], w1s [h_s, d] and w2s [d, h_s] (ignored when h_s == 0);
 *   SwiGLU: w1 [E, 2h, d], w2 [E, d, ldh], w1s [2 h_s, d], w2s [d, ldh_s]
 *   y [T, d] layer dtype out
 *   topk_idx_out [T, K] int32 and topk_gate_out [T, K] fp32: optional
 *   copies of the routing (NULL = not returned)
 *   events: NULL, or three hipEvent_t slots (events created by the caller)
 *   recorded on `stream` right before the routed fc1 launch, between fc1 and
 *   fc2, and right after fc2: a timing hook for the grouped expert GEMMs
 *   inside the layer. The middle slot may be NULL (not recorded): each
 *   recorded event leaves a gap of a few microseconds in the queue, so the
 *   pair is timed best from the outer two alone. The first and the last must
 *   be events (MOE_ERR_INVALID_ARG otherwise)
 * The shared expert's output stays fp32 until the combine. */
moe_status_t moe_layer_forward(const moe_desc_t *desc, const void *x, const void *w_router,
                               const float *bias, const void *w1, const void *w2,
                               const void *w1s, const void *w2s, void *y, int32_t *topk_idx_out,
                               float *topk_gate_out, void *workspace, size_t workspace_bytes,
                               void *const *events, void *stream);

/* Bytes of device scratch that moe_layer_forward_noalloc holds on each GPU
 * it runs on: 64 MiB, enough for the single-image ViT-G layer (1025 tokens,
 * d = 1536, 256 experts, K = 8, h = 768, h_s = 1536 needs about 46 MiB). */
#define MOE_NOALLOC_SCRATCH_BYTES (64u << 20)

/* moe_layer_forward for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same layer, the same kernels and the same results bit for
 * bit, with no workspace argument and no timing events. Its scratch is a
 * device array of MOE_NOALLOC_SCRATCH_BYTES inside the library, one per GPU,
 * held from the first call on that GPU until the process ends; the call
 * allocates nothing (no hipMalloc, hipFree or allocating library routine).
 *   Arguments as for moe_layer_forward.
 * Errors: MOE_ERR_WORKSPACE (nothing enqueued) when the layer's workspace
 * (moe_workspace_size) exceeds MOE_NOALLOC_SCRATCH_BYTES; MOE_ERR_HIP if the
 * scratch's device address cannot be found. Every call on one GPU uses that
 * GPU's single scratch array, so calls that overlap on one GPU (different
 * streams, or different host threads without ordering) race and give
 * undefined results; calls ordered on one stream are safe. */
moe_status_t moe_layer_forward_noalloc(const moe_desc_t *desc, const void *x, const void *w_router,
                                       const float *bias, const void *w1, const void *w2,
                                       const void *w1s, const void *w2s, void *y, int32_t *topk_idx_out,
                                       float *topk_gate_out, void *stream);

/* Bytes of device workspace that moe_grouped_mlp_backward needs for `desc`
 * (bf16 layers). Writes *bytes; validates desc. */
moe_status_t moe_backward_workspace_size(const moe_desc_t *desc, size_t *bytes);

/* Backward of stage 4 for training (the grouped GEMMs of the paper's training
 * kernel, with the activation as its own step: App. "MoE Kernel", the
 * paragraph after Algorithm 1). For every slot n = t*K + j routed to expert
 * e, with G_n = grad_expert_out[n] (the gradient of expert_out[n]) and
 * p_n = W1[e] x_t:
 *   dx[t]  = sum over j of W1[e]^T dH_n      dH_n = (W2[e]^T G_n) * GELU'(p_n)
 *   dw1[e] = sum over the slots of e of dH_n x_t^T
 *   dw2[e] = sum over the slots of e of G_n GELU(p_n)^T
 *   x [T, d], w1 [E, h, d], w2 [E, d, h], grad_expert_out [T*K, d] (slot
 *   order): layer dtype (bf16); sorted_slots, offsets: as from moe_permute
 *   dx  [T, d] bf16 out: the K slot gradients summed in fp32 in slot order,
 *       rounded once
 *   dw1 [E, h, d] and dw2 [E, d, h] fp32 out; experts with no slots get 0
 * SwiGLU experts (MOE_FLAG_SWIGLU; w1 = w13 [E, 2h, d], w2 [E, d, ldh]): with
 * g_n = W1[e] x_t, u_n = W3[e] x_t and dA_n = W2[e]^T G_n,
 *   dG_n = dA_n * u_n * SiLU'(g_n),  dU_n = dA_n * SiLU(g_n)
 *   dx[t]   = sum over j of W1[e]^T dG_n + W3[e]^T dU_n
 *   dw1[e]  = [E, 2h, d] fp32: rows 0..h-1 sum dG_n x_t^T, rows h..2h-1 dU_n x_t^T
 *   dw2[e]  = [E, d, ldh] fp32, the layout of w2: columns < h sum G_n a_n^T
 *             (a_n = SiLU(g_n) * u_n), padding columns 0
 * As in the forward, the activation is rounded to bf16 (dw2 uses that
 * value); the pre-activation gradient (dH, or dG and dU) is rounded to bf16,
 * the operand of the dx and dw1 products; every product accumulates in fp32.
 * bf16 layers only (fp32 layers: MOE_ERR_UNSUPPORTED). Deterministic: no
 * atomics. Uses its own workspace (moe_backward_workspace_size), 256-byte
 * aligned. */
moe_status_t moe_grouped_mlp_backward(const moe_desc_t *desc, const void *x, const int32_t *sorted_slots,
                                      const int32_t *offsets, const void *w1, const void *w2,
                                      const void *grad_expert_out, void *dx, float *dw1, float *dw2,
                                      void *workspace, size_t workspace_bytes, void *stream);

/* Rules of moe_bias_update. */
typedef enum { MOE_BIAS_SIGN = 0, MOE_BIAS_ZSCORE = 1 } moe_bias_rule_t;

/* Loss-free load balancing (Sec. 3.2 "Load Balancing"): update the selection
 * bias in place from one iteration's token counts.
 *   counts [E] int32 in: tokens routed to each expert (as moe_permute
 *          produces them; non-negative)
 *   bias   [E] fp32 in/out
 *   alpha  step size, finite and >= 0
 *   rule   MOE_BIAS_SIGN:   b_e <- b_e - alpha * sign(t_e - mu)      (Eq. (8))
 *          MOE_BIAS_ZSCORE: b_e <- b_e - alpha * (t_e - mu) / sigma  (Eq. (9))
 * mu is the mean of the E counts and sigma their standard deviation over the
 * E experts (divided by E). sign(0) = 0; sigma = 0 (all counts equal) leaves
 * the bias unchanged. The sign is decided exactly (E t_e against the sum of
 * the counts) and applied as one fp32 add of -alpha or +alpha. The z-score
 * rule is evaluated in double precision in a fixed order - mu = sum / E;
 * variance = (sum over e = 0..E-1 of (t_e - mu)^2, each square and each add
 * rounded) / E; sigma = correctly rounded sqrt; z = (t_e - mu) / sigma;
 * b_e - alpha z - and rounded to fp32 once, so it is reproducible bit for bit.
 * Only desc->E is used (desc must still be valid). No workspace. */
moe_status_t moe_bias_update(const moe_desc_t *desc, const int32_t *counts, float *bias, float alpha,
                             int32_t rule, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* MOE_VIE_H */
