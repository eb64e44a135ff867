/*
 * prunepath.h -- C ABI of the MI355X (gfx950) PrunePath sparse-FFN forward.
 *
 * What is computed (PrunePath, Sec. 3.1, on the MoEfied FFN of Sec. 2.2):
 * a bias-free SwiGLU FFN (Eq. ffn) whose d_ff intermediate neurons are split
 * into E contiguous experts of de = d_ff/E = 128 neurons (Eq. moefication_decomp,
 * optionally after a neuron permutation, Eq. permuted_weights).  For every
 * token x a linear router gives logits g = W_r x (Eq. routing_logits), their
 * softmax p (Eq. softmax_prob) is ordered descending, and a prefix of that
 * order is kept according to the cumulative-mass budget tau
 * (Eq. tau_thresh_activate).  Only the kept experts' gate/up/down slices are
 * evaluated and their outputs summed (Eq. moefication_decomp restricted to the
 * kept set; Eq. moe_output with PP_AGG_SIGMOID).
 *
 * Conventions shared by every entry point
 *  - All array arguments are DEVICE pointers on the current HIP device, unless
 *    stated otherwise.  bf16 values are passed as their uint16_t bit patterns.
 *  - Row-major layouts with the API's [out, in] orientation: W_r [E, d],
 *    W_gate/W_up [d_ff, d], W_down [d, d_ff] (the paper's matrices are the
 *    transposes), x [T, d], y [T, d].
 *  - `hip_stream` is a hipStream_t (NULL = the default stream).  Every call
 *    except create/destroy only enqueues work on that stream and returns; the
 *    results are valid once the stream has reached that point.
 *  - A handle owns internal scratch, so one handle must not be used by two
 *    calls that can run concurrently (for example on two streams).
 *  - Errors: a call that returns anything but PP_OK has enqueued no work and
 *    left every output untouched, except PP_EHIP, which reports a failure of
 *    the HIP runtime (outputs then undefined), and PP_ENOTCONVERGED (see
 *    prunepath_balanced_kmeans).  No exception or abort crosses this
 *    interface.
 */
#ifndef PRUNEPATH_H
#define PRUNEPATH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Opaque layer handle: the repacked expert weights plus scratch. */
typedef struct pp_layer pp_layer;

typedef enum {
    PP_OK = 0,
    PP_EINVAL = 1,        /* bad argument (NULL pointer, size, tau, permutation) */
    PP_ENOMEM = 2,        /* device allocation failed */
    PP_EHIP = 3,          /* HIP runtime error */
    PP_EUNSUPPORTED = 4,  /* valid but unsupported shape (see create) */
    PP_ENOTCONVERGED = 5  /* iteration limit reached (balanced k-means assignment) */
} pp_status;

/* Selection rule (Eq. tau_thresh_activate; pi = experts by descending p,
 * C_i = p_pi1 + ... + p_pii; ties in p are ordered by ascending expert index):
 *  PP_SELECT_NUCLEUS: keep the smallest prefix pi_1..pi_k with C_k >= tau (the
 *    top-p reading named next to the equation); tau >= 1 keeps all E experts,
 *    tau = 0 keeps pi_1.
 *  PP_SELECT_STRICT: the printed rule {pi_1} U {pi_i : C_i < tau}, C_E = 1.
 * Two comparison rules run on the same kernels, the call's `tau` argument
 * then carrying their parameter:
 *  PP_SELECT_TOPK: the k experts ranked first by the router, pi_1..pi_k, with
 *    k = tau rounded to the nearest integer and clamped to [1, E] (the forced
 *    top-k budget of the paper's reconstruction analysis, Sec. 4.3.2 "Top-k
 *    Reconstruction Analysis").
 *  PP_SELECT_LTE: the independent threshold of Eq. (lte_hard_set),
 *    {e : sigmoid(g_e) > delta} with delta = tau; a token may keep no expert
 *    (count 0, y row 0).  The kept experts are still listed in pi order.
 * At most one PP_SELECT_* bit may be set. */
#define PP_SELECT_NUCLEUS 0u
#define PP_SELECT_STRICT 1u
#define PP_SELECT_TOPK 4u
#define PP_SELECT_LTE 8u
/* Aggregation: PP_AGG_SUM = plain sum of the kept experts' outputs (the
 * all-expert case is the dense FFN, Eq. moefication_decomp);
 * PP_AGG_SIGMOID = each kept expert scaled by sigmoid(g_e), Eq. moe_output. */
#define PP_AGG_SUM 0u
#define PP_AGG_SIGMOID 2u

/* prunepath_create -- build a layer (Sec. 2.2 expert split, Sec. 3.1 router).
 *   out        : receives the handle (host pointer to a host variable).
 *   d          : model width; a positive multiple of 64, at most 8192
 *                (PP_EUNSUPPORTED otherwise).
 *   d_ff, E    : intermediate width and expert count; d_ff must equal 128*E
 *                (PP_EUNSUPPORTED otherwise) and 1 <= E <= 256.
 *   max_tokens : largest T any later call will pass (1 .. 65536); scratch is
 *                sized for it.
 *   W_r        : [E, d] bf16 router weights (paper's W_r transposed).
 *   W_gate,
 *   W_up       : [d_ff, d] bf16, row n = intermediate neuron n.
 *   W_down     : [d, d_ff] bf16, column n = intermediate neuron n.
 *   perm       : [d_ff] int32 neuron permutation Pi (expert e owns neurons
 *                perm[128e .. 128e+127]), or NULL for the identity; it must be
 *                a permutation of 0..d_ff-1 (PP_EINVAL otherwise).
 *   router_bias: [E] fp32 added to the logits (g = W_r x + b), or NULL.
 *   flags      : one PP_SELECT_* rule | PP_AGG_* (PP_EINVAL for unknown bits or
 *                two selection rules).
 * The weights are copied and repacked into library-owned device memory; the
 * call synchronises `hip_stream` before returning, after which the caller may
 * free its arrays.  On failure *out is set to NULL. */
pp_status prunepath_create(pp_layer **out, int32_t d, int32_t d_ff, int32_t E,
                           int32_t max_tokens, const uint16_t *W_r, const uint16_t *W_gate,
                           const uint16_t *W_up, const uint16_t *W_down, const int32_t *perm,
                           const float *router_bias, uint32_t flags, void *hip_stream);

/* prunepath_create_mlp -- a layer whose FFN is the non-gated GELU MLP of
 * GPT-2 (the paper's GPT-2 Medium target, Sec. 4.2.2 and Sec. 4.5; Sec. 2.1
 * notes that the expert decomposition holds for any FFN whose intermediate
 * neurons are separable):
 *   FFN(x) = GELU(x W_fc + b_fc) W_proj + b_proj,
 * GELU in GPT-2's tanh form 0.5 a (1 + tanh(sqrt(2/pi) (a + 0.044715 a^3))).
 * Expert e owns neurons perm[128e .. 128e+127] of W_fc, b_fc and W_proj; a
 * kept expert contributes GELU(x W_fc^(e) + b_fc^(e)) W_proj^(e) [* sigmoid(g_e)]
 * and b_proj is added once per token whatever is kept (a token that keeps no
 * expert gets y = b_proj).
 *   W_fc   : [d_ff, d] bf16, row n = intermediate neuron n (GPT-2's c_fc
 *            weight transposed).
 *   b_fc   : [d_ff] fp32 or NULL (zero).
 *   W_proj : [d, d_ff] bf16, column n = intermediate neuron n.
 *   b_proj : [d] fp32 or NULL (zero).
 * Every other argument, the limits and the error behaviour are those of
 * prunepath_create; the handle works with every call below. */
pp_status prunepath_create_mlp(pp_layer **out, int32_t d, int32_t d_ff, int32_t E,
                               int32_t max_tokens, const uint16_t *W_r, const uint16_t *W_fc,
                               const float *b_fc, const uint16_t *W_proj, const float *b_proj,
                               const int32_t *perm, const float *router_bias, uint32_t flags,
                               void *hip_stream);

/* prunepath_route -- routing only (Eqs. routing_logits, softmax_prob,
 * tau_thresh_activate).
 *   x          : [T, d] bf16 tokens, 1 <= T <= max_tokens.
 *   tau        : budget, >= 0 (NaN or negative: PP_EINVAL): the cumulative
 *                mass (nucleus, strict), k (top-k) or delta (LTE).
 *   inv_temp   : [T] fp32 per-token inverse temperature, or NULL (= 1):
 *                g = (W_r x + b) * inv_temp[t].
 *   expert_idx : [T, E] int32 out; row t holds the kept experts pi_1..pi_k in
 *                descending-logit order, then -1.
 *   count      : [T] int32 out; k for each token (>= 1 except with LTE).
 *   gate_w     : [T, E] fp32 out or NULL; weight applied to the expert in the
 *                same slot of expert_idx (sigmoid(g_e) with PP_AGG_SIGMOID,
 *                else 1), 0 in unused slots. */
pp_status prunepath_route(pp_layer *L, const uint16_t *x, int32_t T, float tau,
                          const float *inv_temp, int32_t *expert_idx, int32_t *count,
                          float *gate_w, void *hip_stream);

/* prunepath_ffn_decode -- routing plus the sparse FFN output, tuned for small
 * token batches (decode).  Batches larger than 64 tokens are processed in
 * slices of 64.
 *   x, T, tau, inv_temp : as for prunepath_route.
 *   y          : [T, d] fp32 out, overwritten: sum over kept experts of
 *                FFN_e(x) (times sigmoid(g_e) with PP_AGG_SIGMOID).
 *   expert_idx, count   : as for prunepath_route, or both NULL to skip them. */
pp_status prunepath_ffn_decode(pp_layer *L, const uint16_t *x, int32_t T, float tau,
                               const float *inv_temp, float *y, int32_t *expert_idx,
                               int32_t *count, void *hip_stream);

/* prunepath_ffn_prefill -- same result as prunepath_ffn_decode (up to fp32
 * summation order), organised for long token batches: tokens are bucketed per
 * kept expert and each expert's bucket runs as a grouped bf16 MFMA GEMM
 * (the multi-token dispatch described in Sec. 4.5).  Deterministic: no
 * floating-point atomics; each token's expert contributions are added to the
 * output (bias) in ascending expert order. */
pp_status prunepath_ffn_prefill(pp_layer *L, const uint16_t *x, int32_t T, float tau,
                                const float *inv_temp, float *y, int32_t *expert_idx,
                                int32_t *count, void *hip_stream);

/* prunepath_residual_rmsnorm -- the wiring between stacked FFN layers (not
 * part of the paper's method; its stacked-layer decode workload chains layers
 * with pre-norm residuals, x_{l+1} = x_l + FFN_l(u_l), u_l = RMSNorm(x_l)):
 *   x_out[t, :] = x[t, :] + y[t, :]            (y NULL: x_out = x)
 *   u[t, :]     = bf16(x_out[t, :] / sqrt(mean_j x_out[t, j]^2 + eps))
 * with norm weight 1 and round-to-nearest-even to bf16 (u NULL: residual add
 * only).  x, y, x_out: [T, d] fp32; u: [T, d] bf16 bits; all device pointers,
 * owned by the caller; x, y and x_out may be the same array.  The sum of
 * squares is fp32 in a fixed order that does not depend on T.
 * PP_EINVAL: NULL x or x_out, T outside [1, 65536], d not a multiple of 4 or
 * outside [4, 2^20], eps NaN or negative (when u is given), x/y/x_out not
 * 16-byte aligned or u not 8-byte aligned. */
pp_status prunepath_residual_rmsnorm(const float *x, const float *y, float *x_out, int32_t T,
                                     int32_t d, float eps, uint16_t *u, void *hip_stream);

/* prunepath_router_loss -- the routing regularisers of the training
 * objective and their gradient, over a batch of B router-logit rows
 * (Sec. 3.2, Eqs. (entropy_loss), (load_balance_loss), (train_loss); the
 * gate-magnitude term of Sec. 4.2.3):
 *   p_ij   = softmax_j(g_i)                                 Eq. (softmax_prob)
 *   L_ent  = -(1/B) sum_ij p_ij log(p_ij + eps)
 *   L_bal  = E sum_j m_j^2,  m_j = (1/B) sum_i p_ij
 *   L_gate = (1/(B E)) sum_ij sigmoid(g_ij)
 *   losses = [L_ent, L_bal, L_gate, eta L_ent + lambda L_bal + gamma L_gate]
 *   dg     = d losses[3] / d g                 (skipped when dg is NULL)
 * The task loss is not included; a term with p_ij = 0 counts as 0.  Does not
 * need a handle.
 *   g         : [B, E] fp32 logits, row-major (device, caller-owned)
 *   losses    : 4 fp32 (device)
 *   dg        : [B, E] fp32 (device) or NULL; may not alias g
 *   workspace : prunepath_router_loss_workspace(B, E) bytes of device memory,
 *               no initial contents required; overwritten
 * Every sum is taken in an order fixed by (B, E): repeated calls give
 * identical bits.  Enqueued on hip_stream (NULL: the null stream).
 * PP_EINVAL: NULL g, losses or workspace; dg == g; B outside [1, 2^22]; E outside
 * [1, 256]; eps negative, NaN or infinite; eta, lambda or gamma not finite;
 * g or dg not 16-byte aligned, losses or workspace not 4-byte aligned. */
size_t prunepath_router_loss_workspace(int32_t B, int32_t E); /* 0 for bad sizes */
pp_status prunepath_router_loss(const float *g, int32_t B, int32_t E, float eps, float eta,
                                float lambda, float gamma, float *losses, float *dg,
                                void *workspace, void *hip_stream);

/* prunepath_router_loss_noalloc -- prunepath_router_loss for callers that
 * cannot allocate device memory: code under HIP graph capture, tight training
 * or serving loops, harnesses that forbid hipMalloc.  Same arguments, results
 * and bits as prunepath_router_loss, minus `workspace`: the partial sums live
 * in a device array inside the library, PP_ROUTER_LOSS_NOALLOC_SCRATCH_BYTES
 * (4 MiB) per GPU, held until the process ends.  Calls no allocator.
 *  - Sizes: prunepath_router_loss_workspace(B, E) must not exceed the array
 *    (ceil(B / 64) * (E + 2) * 4 bytes: B up to 588672 rows at E = 112,
 *    260096 at E = 256); larger sizes return PP_EUNSUPPORTED, enqueue nothing.
 *  - The first call on each device looks up that device's copy of the array
 *    (hipGetSymbolAddress); make it outside any graph capture.
 *  - Every call on one GPU shares its array: calls that can overlap on one GPU
 *    (two streams, two threads, two captured graphs replayed concurrently)
 *    race and give undefined results.  The array needs no clearing: each call
 *    overwrites the partials it reads.
 * Other errors as for prunepath_router_loss. */
#define PP_ROUTER_LOSS_NOALLOC_SCRATCH_BYTES (4u << 20)
pp_status prunepath_router_loss_noalloc(const float *g, int32_t B, int32_t E, float eps,
                                        float eta, float lambda, float gamma, float *losses,
                                        float *dg, void *hip_stream);

/* prunepath_balanced_kmeans -- MoEfication's neuron clustering (Sec. 2.2):
 * balanced k-means of the n rows of F into k clusters of exactly m = n / k
 * rows (the constrained k-means the paper cites), which gives the
 * permutation Pi of Eq. (permuted_weights) that prunepath_create takes as
 * `perm` (n = d_ff, k = E, F = one feature row per intermediate neuron, e.g.
 * the rows of W_gate or of W_fc).  Each of `iters` Lloyd iterations:
 *   assignment  minimise sum_i ||F_i - mu_a(i)||^2 subject to the balance,
 *               exactly (an auction on k cluster prices whose final argmax
 *               assignment is balanced, hence optimal by LP duality);
 *   update      mu_j = mean of cluster j's rows.
 *   F              : [n, D] bf16, 16-byte aligned (device)
 *   init_centroids : [k, D] fp32 (device); may equal `centroids`
 *   iters          : 1 .. 1000
 *   assign         : [n] int32 out (device): cluster of each row, last iteration
 *   perm           : [n] int32 out (device): Pi, cluster 0's rows ascending,
 *                    then cluster 1's, ...
 *   centroids      : [k, D] fp32 out (device): the means of the last assignment
 *   objective      : [iters] fp32 out (device) or NULL: the assignment cost of
 *                    each iteration with the centroids it used
 *   prices         : [k] fp32 out (device) or NULL: the last step's prices
 *                    (row i's cluster maximises -||mu_j||^2 + 2 F_i.mu_j -
 *                    price_j over j, in the kernels' fp32 arithmetic)
 *   rounds         : [iters] int32 out (HOST memory) or NULL: auction rounds
 *                    each assignment took (-1: did not converge)
 *   workspace      : prunepath_kmeans_workspace(n, D, k) bytes (device),
 *                    16-byte aligned, no initial contents required
 * Limits: 1 <= k <= 256, k <= n <= 65536, n % k == 0, 64 <= D <= 16384,
 * D % 64 == 0 (PP_EINVAL otherwise; the workspace query returns 0).  The
 * call blocks: it synchronises hip_stream to follow the auction.
 * PP_ENOTCONVERGED when an assignment needs more than 32768 auction rounds
 * (possible when rows are exact duplicates of each other); outputs then hold
 * the last unbalanced state. */
size_t prunepath_kmeans_workspace(int32_t n, int32_t D, int32_t k); /* 0 for bad sizes */
pp_status prunepath_balanced_kmeans(const uint16_t *F, int32_t n, int32_t D, int32_t k,
                                    const float *init_centroids, int32_t iters, int32_t *assign,
                                    int32_t *perm, float *centroids, float *objective,
                                    float *prices, int32_t *rounds, void *workspace,
                                    void *hip_stream);

/* Kernel kinds reported by prunepath_profile_end. */
#define PP_KERNEL_ROUTE 0     /* router: logits, softmax, sort, cut */
#define PP_KERNEL_DISPATCH 1  /* prefill token bucketing */
#define PP_KERNEL_GATEUP 2    /* gate/up projections + SiLU product */
#define PP_KERNEL_DOWN 3      /* down projection + per-token sum */
#define PP_KERNEL_COUNT 4

/* prunepath_profile_begin -- benchmarking aid (not part of the method):
 * from now on every kernel this handle launches is bracketed by two HIP
 * events recorded on the call's stream, for at most `capacity` launches
 * (1 .. 1<<20).  Creates the events, so call it outside any timed or
 * captured region.  PP_EINVAL if already recording. */
pp_status prunepath_profile_begin(pp_layer *L, int32_t capacity);

/* prunepath_profile_end -- stop recording, wait for the recorded events and
 * return, per kernel kind k < PP_KERNEL_COUNT, the summed device time in
 * milliseconds (ms[k], host array) and the number of launches recorded
 * (launches[k], host array).  Either array may be NULL.  PP_EINVAL if not
 * recording. */
pp_status prunepath_profile_end(pp_layer *L, double *ms, int32_t *launches);

/* prunepath_destroy -- free a handle and its device memory.  NULL is a no-op.
 * The caller must ensure no enqueued work still uses the handle. */
void prunepath_destroy(pp_layer *L);

/* prunepath_status_string -- static text for a status code (never NULL). */
const char *prunepath_status_string(pp_status s);

#ifdef __cplusplus
}
#endif

#endif /* PRUNEPATH_H */
