/*
 * groupmask.h -- C ABI of the group-masked linear layer of GroupMask
 * (layer-adaptive group-wise sparsity with frozen weights, Sec. 2).
 *
 * One target linear layer holds a frozen weight W [d_out, d_in], cut into
 * g_out x g groups (Sec. 2.1): group (u, v) covers W[u*g_out : (u+1)*g_out,
 * v*g : (v+1)*g], u < G_out = d_out / g_out, v < G_in = d_in / g.  Eq. 1
 * expands the selector matrix B [G_out, G_in] to the full-resolution mask by a
 * Kronecker product with a g_out x g block of ones.  Shapes built: row groups
 * 1 x g with g in {64, 128, 256, 512} (g_out = 1) and square groups
 * g x g with g in {16, 32, 64, 128} (g_out = g).
 *
 * Conventions shared by every call:
 *   - bf16 tensors are passed as uint16_t bit patterns; fp32 as float.
 *   - All tensors are dense, row-major, contiguous, in the nn.Linear
 *     convention: X [T, d_in], W [d_out, d_in], Y / dY [T, d_out],
 *     mask / dgate [G_out, G_in].
 *   - Every pointer argument is a DEVICE pointer unless stated otherwise, and
 *     must be 16-byte aligned unless stated otherwise (the per-layer arrays of
 *     the budget calls need only their element alignment).  The caller owns
 *     every buffer; the library never
 *     allocates or frees device memory.  Scratch space is passed in as a
 *     caller-owned workspace sized by gm_workspace_size().
 *   - Every call validates its arguments before launching anything and returns
 *     a gm_status; nothing aborts and no exception crosses the ABI.  On an
 *     error return no kernel has been launched and no output was touched.
 *   - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL is the
 *     null stream).  No call synchronises the host.  Calls that share a
 *     workspace must be ordered on one stream.
 *   - Only gfx950 (MI355X) devices are supported; any other device returns
 *     GM_ERR_DEVICE.
 */
#ifndef GROUPMASK_H
#define GROUPMASK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GM_ABI_VERSION 3

/* Same object as a hipStream_t, declared here so that callers need no HIP headers. */
typedef struct ihipStream_t* gm_stream_t;

/* Status codes.  In C++ the enumeration has int as its fixed underlying type,
 * so that every int a C caller passes (gm_status_string(99) included) is a
 * valid value of it. */
typedef enum gm_status
#ifdef __cplusplus
    : int
#endif
{
  GM_OK = 0,
  GM_ERR_NULL = 1,      /* a required pointer is NULL */
  GM_ERR_SHAPE = 2,     /* a size is out of range or inconsistent */
  GM_ERR_VALUE = 3,     /* a scalar argument is out of range (tau, hard) */
  GM_ERR_ALIGN = 4,     /* a pointer is not 16-byte aligned */
  GM_ERR_WORKSPACE = 5, /* workspace missing or smaller than gm_workspace_size() */
  GM_ERR_DEVICE = 6     /* not a gfx950 device, or a HIP launch error */
} gm_status;

/* Operation codes for gm_workspace_size(). */
enum { GM_OP_FWD = 0, GM_OP_BWD = 1 };

/* Returns GM_ABI_VERSION of the built library. */
int gm_abi_version(void);

/* Static, NUL-terminated description of a status code (host memory, never freed). */
const char* gm_status_string(gm_status status);

/*
 * gm_gate -- Gumbel-Sigmoid gate with straight-through forward (Sec. 2.2;
 * evaluation-time thresholding, Sec. 2.2 and Appendix F).
 *
 * For each of the n groups (a flat array, so the selectors of many layers can
 * go through one call):
 *   z    = logits[j] + (noise ? ln(noise[j]) - ln(1 - noise[j]) : 0)
 *   y    = 1 / (1 + exp(-z / tau))
 *   mask_out[j] = hard ? (z > 0 ? 1 : 0) : y       (z > 0 is exactly y > 1/2)
 *   soft_out[j] = y                                  (only if soft_out != NULL)
 * noise holds one uniform variate per group in the open interval (0, 1); NULL
 * selects evaluation mode (noise removed).  Precondition, not checked: noise
 * values lie in (0, 1).
 *   logits   [n] fp32, required
 *   noise    [n] fp32 or NULL
 *   n        >= 0 (n == 0 is a no-op)
 *   tau      > 0 and finite
 *   hard     0 or 1
 *   mask_out [n] fp32, required
 *   soft_out [n] fp32 or NULL; keep it for the backward (gm_gate_bwd)
 */
gm_status gm_gate(const float* logits, const float* noise, int64_t n, float tau, int hard,
                  float* mask_out, float* soft_out, gm_stream_t stream);

/*
 * gm_gate_bwd -- straight-through backward of the gate (Sec. 2.2): the
 * gradient passes through the continuous relaxation,
 *   dlogits[j] = dmask[j] * y[j] * (1 - y[j]) / tau,
 * where y = soft_out of the forward and dmask the gradient of the selector
 * (dgate of gm_masked_linear_bwd).
 *   dmask, soft, dlogits: [n] fp32, required; n >= 0; tau > 0 and finite.
 *   dlogits may alias dmask.
 */
gm_status gm_gate_bwd(const float* dmask, const float* soft, int64_t n, float tau, float* dlogits,
                      gm_stream_t stream);

/*
 * gm_budget_loss -- sparsity-budget regulariser (Sec. 2.3) of L layers on
 * their discrete selectors, with Eq. 2's layer-wise and parameter-weighted
 * sparsity.  The selectors of all layers lie back to back in one flat array
 * (the layout gm_gate accepts): layer l owns mask[offsets[l] .. offsets[l+1]).
 *   kept[l] = number of selectors of layer l with mask != 0 (exact)
 *   s^l = 1 - kept[l] / G^l (G^l = offsets[l+1] - offsets[l]),
 *   s   = sum_l s^l params[l] / sum_l params[l]
 *   uniform == 0:  loss = lambda |log(s / s_target)|
 *                  coeff[l] = lambda sgn(log(s/s_target)) / s * (-(params[l] / G^l) / sum_k params[k])
 *   uniform == 1:  loss = sum_l lambda |log(s^l / s_target)|
 *                  coeff[l] = lambda sgn(log(s^l/s_target)) / s^l * (-1 / G^l)
 * coeff[l] is d loss / d selector for every selector of layer l (sgn(0) = 0);
 * gm_gate_bwd_budget folds it into the logit gradient.  A sparsity of 0
 * makes the loss and coefficient infinite.  loss and the sums are fp64.
 *   mask    [n] fp32 (device), n >= 1, 16-byte aligned
 *   offsets [L + 1] int64 (device, 8-byte aligned): offsets[0] = 0, strictly
 *           increasing, offsets[L] = n (not checked: wrong offsets give wrong
 *           sums, never an access outside mask)
 *   params  [L] int64 (device, 8-byte aligned): weights per layer, d_out * d_in, >= 1
 *   L >= 1; 0 < s_target < 1; lambda >= 0 and finite; uniform in {0, 1}
 *   kept  [L] uint64 (device, 8-byte aligned, output; cleared by the call)
 *   loss  [1] fp64 (device, 8-byte aligned, output)
 *   coeff [L] fp32 (device, 4-byte aligned, output)
 * Three launches on `stream`: clear kept, count (HBM bound, 4 bytes per
 * selector), finalize (one block).
 */
gm_status gm_budget_loss(const float* mask, int64_t n, const int64_t* offsets, const int64_t* params, int32_t L,
                         float s_target, float lambda, int uniform, uint64_t* kept, double* loss, float* coeff,
                         gm_stream_t stream);

/*
 * gm_gate_bwd_budget -- gm_gate_bwd with the regulariser's gradient added to
 * the selector gradient (Sec. 2.2 and 2.3):
 *   dlogits[j] = (dgate[j] + coeff[l(j)]) * y[j] * (1 - y[j]) / tau,
 * with l(j) the layer owning selector j under `offsets` (as in gm_budget_loss).
 *   dgate, soft, dlogits: [n] fp32 (device), 16-byte aligned, n >= 1;
 *   dlogits may alias dgate.  offsets [L + 1] int64 (device, 8-byte aligned),
 *   coeff [L] fp32 (device, 4-byte aligned).
 *   L >= 1; tau > 0 and finite.
 */
gm_status gm_gate_bwd_budget(const float* dgate, const float* soft, int64_t n, float tau, const int64_t* offsets,
                             int32_t L, const float* coeff, float* dlogits, gm_stream_t stream);

/*
 * gm_workspace_size -- host-only query of the workspace (bytes) that
 * gm_masked_linear_fwd (op = GM_OP_FWD) or gm_masked_linear_bwd
 * (op = GM_OP_BWD) needs for the given shape.  No device work.  The forward
 * needs one only for launches of few output tiles (at most 128 tiles of
 * 256 x 256, e.g. T = 512 with d_out = 5120), where it splits K: then
 * ksplit * T * d_out fp32 for the partial tiles (ksplit <= 8); otherwise 0.
 *   bytes: HOST pointer, required.
 */
gm_status gm_workspace_size(int op, int64_t T, int64_t d_in, int64_t d_out, int32_t g, int32_t g_out,
                            size_t* bytes);

/*
 * gm_masked_linear_fwd -- student forward of one target linear (Eq. 1):
 *   Y = X (W (.) (mask (x) 1_{g_out x g}))^T,
 *   Y[t, o] = sum_v mask[o / g_out, v] * sum_{i in group v} X[t, i] W[o, i].
 * A group with mask == 0 is skipped (its weights are never read); any other
 * value scales the group (1.0 for a hard selector).  bf16 inputs, fp32
 * accumulation, Y rounded to bf16 (round to nearest even).
 *   X    [T, d_in]  bf16       W [d_out, d_in] bf16
 *   mask [d_out / g_out, d_in / g] fp32
 *   Y    [T, d_out] bf16, written in full
 *   T >= 1; d_in, d_out >= 1 and multiples of 8; (g_out, g) one of the
 *   built shapes; d_in a multiple of max(g, 64) and at most 512 * max(g, 32);
 *   d_out a multiple of g_out; each of X, W, Y (T rounded up to a multiple
 *   of 8) below 2^30 - 2^22 elements.  Mask values must be finite and >= 0
 *   (not checked).
 *   ws / ws_bytes: optional workspace (16-byte aligned).  NULL: the GEMM
 *   runs unsplit.  Otherwise at least gm_workspace_size(GM_OP_FWD, ...) bytes
 *   (GM_ERR_WORKSPACE if smaller), and shapes with few output tiles split K
 *   over several blocks whose fp32 partial tiles are added in a fixed order
 *   before the one rounding to bf16 (the same Y up to fp32 summation order;
 *   deterministic for a given shape).  The workspace is scratch: its contents
 *   are not used across calls.
 */
gm_status gm_masked_linear_fwd(const uint16_t* X, const uint16_t* W, const float* mask, int64_t T,
                               int64_t d_in, int64_t d_out, int32_t g, int32_t g_out, uint16_t* Y,
                               void* ws, size_t ws_bytes, gm_stream_t stream);

/*
 * gm_masked_linear_bwd -- backward of one target linear with frozen W
 * (Sec. 2.2 STE, Sec. 2.4 frozen weights):
 *   dX = dY (W (.) expand(mask))                       [T, d_in]   bf16
 *   dgate[u, v] = sum_{(o, i) in group (u, v)} W[o, i] (dY^T X)[o, i]   [G_out, G_in] fp32
 * dgate is produced for every group, kept or pruned, and does not depend on
 * the mask; the weight gradient is never formed.  Either output may be NULL to
 * skip it (both NULL is a no-op); mask may be NULL only when dX is NULL.
 *   Shapes and constraints as gm_masked_linear_fwd; dY [T, d_out] bf16.
 *   ws / ws_bytes: at least gm_workspace_size(GM_OP_BWD, ...) bytes.
 */
gm_status gm_masked_linear_bwd(const uint16_t* dY, const uint16_t* X, const uint16_t* W,
                               const float* mask, int64_t T, int64_t d_in, int64_t d_out, int32_t g,
                               int32_t g_out, uint16_t* dX, float* dgate, void* ws, size_t ws_bytes,
                               gm_stream_t stream);

/*
 * gm_masked_linear_bwd_noalloc -- gm_masked_linear_bwd for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation.  Same arguments without the workspace,
 * same kernels, same results bit for bit.
 *
 * Its workspace is a fixed scratch array of GM_NOALLOC_SCRATCH_BYTES (96 MiB)
 * that the library keeps on every device it runs on until the process ends
 * (the array's device address is looked up once per device, on the first
 * call there).  A shape whose backward workspace (gm_workspace_size with
 * GM_OP_BWD) exceeds it returns GM_ERR_WORKSPACE before any launch; the
 * backward of every LLaMA-2-7B linear at 4096 tokens fits.  Nothing in the
 * scratch needs to start at zero: each call rewrites what it reads.  Every
 * call on one device shares that device's scratch, so calls that overlap on
 * one GPU (different streams, or host threads without ordering between them)
 * race and give wrong results: order them on one stream.  The call allocates
 * and frees nothing.  A dgate-only call (dX == NULL) uses no scratch.
 */
#define GM_NOALLOC_SCRATCH_BYTES ((size_t)96 << 20)
gm_status gm_masked_linear_bwd_noalloc(const uint16_t* dY, const uint16_t* X, const uint16_t* W, const float* mask,
                                       int64_t T, int64_t d_in, int64_t d_out, int32_t g, int32_t g_out,
                                       uint16_t* dX, float* dgate, gm_stream_t stream);

/*
 * gm_pack_rows -- export of a learned mask (Appendix F): copies the retained
 * groups of W, row by row, into a packed buffer for the pruned model.  A
 * g_out x g group is stored as its g_out row pieces of g weights, so the
 * export of every group shape is the same row-wise format.
 *   rowptr [d_out + 1] int32: rowptr[o] = number of kept groups in rows < o;
 *                             rowptr[d_out] = total kept groups k.
 *   Wp     [capacity, g] bf16: kept group number j of the matrix at Wp[j*g];
 *   chunk  [capacity] int32:  its group column v;
 *   scale  [capacity] fp32:   its mask value (1.0 for a hard selector).
 * Groups with mask == 0 are dropped.  Row pieces beyond `capacity` are not
 * written: the caller checks rowptr[d_out] <= capacity (capacity = d_out *
 * d_in / g is always enough).  Shape constraints as gm_masked_linear_fwd.
 */
gm_status gm_pack_rows(const uint16_t* W, const float* mask, int64_t d_in, int64_t d_out, int32_t g,
                       int32_t g_out, int64_t capacity, uint16_t* Wp, int32_t* chunk, float* scale,
                       int32_t* rowptr, gm_stream_t stream);

/*
 * gm_packed_linear_fwd -- forward of a pruned linear from its packed export
 * (the inference path of the pruned model): the same Y as gm_masked_linear_fwd
 * with the mask that gm_pack_rows consumed.  Built for decode-sized T (reads
 * every kept weight once per 16 tokens); any T >= 1 is accepted.
 *   X [T, d_in] bf16; Wp, chunk, scale, rowptr as written by gm_pack_rows,
 *   which must have held every kept group (rowptr[d_out] <= its capacity);
 *   g is the width of the exported pieces (the group width; a square export
 *   with g < 64 also needs d_out a multiple of g);
 *   Y [T, d_out] bf16, written in full.
 */
gm_status gm_packed_linear_fwd(const uint16_t* X, const uint16_t* Wp, const int32_t* chunk,
                               const float* scale, const int32_t* rowptr, int64_t T, int64_t d_in,
                               int64_t d_out, int32_t g, uint16_t* Y, gm_stream_t stream);

/*
 * Self-distillation loss through the frozen LM head (Sec. 2.4, Eq. 4).
 * The teacher pass (all selectors 1) and the student pass (the learned
 * selectors) end in final hidden states H_T, H_S [N, d] (bf16), and share
 * the LM head W [V, d] (bf16, row v = vocabulary entry v).  With
 * z = H W^T, p = softmax over the vocabulary, and N_valid the number of
 * tokens whose `valid` flag is nonzero (all N when valid is NULL):
 *   L = -(1/N_valid) sum_{valid t} sum_v p_T(t, v) log p_S(t, v)
 * (the forward KL from teacher to student plus the teacher entropy, which
 * does not depend on the student).  Gradients go to H_S only (the teacher is
 * detached, the LM head frozen):
 *   dH_S = dz_S W,  dz_S(t, v) = (p_S(t, v) - p_T(t, v)) / N_valid for valid t, 0 otherwise.
 * With no valid token, L = 0 and dH_S = 0.
 * Shapes: N >= 1; d a multiple of 32 in [32, 65536]; V a multiple of 8 in
 * [8, 2^20]; V d, N d and N ceil32(V) each below 2^30 - 2^22 elements.
 * Logits are accumulated in fp32 from the bf16 inputs; softmax statistics
 * and the token sums in fp32/fp64; dz_S is rounded to bf16 before the
 * product with W.
 *
 * gm_distill_workspace_size -- host-only query of the workspace both calls
 * below need (bytes; about 8 N V + 2 N V bytes: the fp32 logits of both passes
 * and the bf16 dz_S).  bytes: HOST pointer, required.
 */
gm_status gm_distill_workspace_size(int64_t N, int64_t d, int64_t V, size_t* bytes);

/*
 * gm_distill_fwd -- the loss.
 *   Ht, Hs [N, d] bf16; W [V, d] bf16; valid [N] uint8 or NULL;
 *   loss: one fp32 (device), written; ce [N] fp32 or NULL: each token's
 *   cross-entropy -sum_v p_T log p_S (for every token, valid or not).
 *   ws / ws_bytes: caller-owned workspace of gm_distill_workspace_size bytes;
 *   it receives both passes' logits and per-token statistics, which
 *   gm_distill_bwd reads.  loss and ce need 4-byte alignment.
 */
gm_status gm_distill_fwd(const uint16_t* Ht, const uint16_t* Hs, const uint16_t* W, const uint8_t* valid,
                         int64_t N, int64_t d, int64_t V, float* loss, float* ce, void* ws, size_t ws_bytes,
                         gm_stream_t stream);

/*
 * gm_distill_bwd -- dH_S [N, d] bf16 (written in full) from the workspace
 * that the last gm_distill_fwd on the same stream filled for the same W, N,
 * d and V (the workspace must not change in between; the valid flags of that
 * call apply).
 */
gm_status gm_distill_bwd(const uint16_t* W, int64_t N, int64_t d, int64_t V, uint16_t* dHs, void* ws,
                         size_t ws_bytes, gm_stream_t stream);

/*
 * Hypernetwork that generates the selector logits (Sec. 2.2, Eq. 3), trained
 * with AdamW (Table 5).  The paper prints no sizes; this library builds:
 *   z [L, D] fp32: the fixed random input, one D-vector per target layer;
 *   a bidirectional GRU with H in {32, 64, 128} units per direction (standard
 *   GRU cell: reset, update and candidate gates, the reset gate scaling the
 *   recurrent candidate term W_hn h + b_hn, zero initial state); its output
 *   for layer l is o_l = [forward; backward] (2H values);
 *   layer-specific affine heads: logits[e] = A[e, :] . o_l + c[e] for the
 *   selectors e in [offsets[l], offsets[l+1]) of layer l, with the heads of
 *   all layers stacked in A [G_total, 2H] fp32 and c [G_total] fp32, in the
 *   order of the flat selector array of the gate and the budget regulariser.
 *   gru [2 P] fp32, P = 3H (D + H + 2): per direction (forward, then
 *   backward) W_ih [3H, D], W_hh [3H, H], b_ih [3H], b_hh [3H], row-major,
 *   gate rows in the order reset, update, candidate.
 *   offsets [L + 1] int64 (device): nondecreasing, offsets[0] = 0,
 *   offsets[L] = G_total (not checked).
 * Limits: 1 <= L <= 65536, 1 <= D <= 4096, G_total >= 1.  A and its AdamW
 * moments need 16-byte alignment, the other arrays 4 (offsets 8).
 *
 * gm_hyper_workspace_size -- host-only query of the workspace both calls need.
 */
gm_status gm_hyper_workspace_size(int64_t L, int64_t D, int64_t H, int64_t G_total, size_t* bytes);

/*
 * gm_hyper_fwd -- logits [G_total] fp32 (written in full).  The workspace
 * keeps the GRU states and the row chunking of the heads for gm_hyper_bwd.
 */
gm_status gm_hyper_fwd(const float* z, const float* gru, const float* A, const float* c,
                       const int64_t* offsets, int64_t L, int64_t D, int64_t H, int64_t G_total,
                       float* logits, void* ws, size_t ws_bytes, gm_stream_t stream);

/*
 * gm_hyper_bwd -- backward of gm_hyper_fwd for the gradient dlogits
 * [G_total] fp32 (the logit gradient of the gate backward), and one AdamW
 * step on the heads, in place: with g the gradient of an element,
 *   p <- p (1 - lr weight_decay);  m <- beta1 m + (1 - beta1) g;  v <- beta2 v + (1 - beta2) g^2;
 *   p <- p - lr (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps)
 * for A (moments mA, vA [G_total, 2H]) and c (mc, vc [G_total]); the GRU
 * gradient goes to dgru [2 P] (apply gm_adamw to gru with it).  The GRU
 * gradient uses the heads before this update.  Reads the workspace that the
 * last gm_hyper_fwd on the same stream filled for the same z, gru, A, c and
 * shapes.  lr >= 0, beta in [0, 1), eps > 0, weight_decay >= 0, step >= 1
 * (else GM_ERR_VALUE).  The hyperparameters are taken in fp64; the update
 * coefficients (1 - beta, the bias corrections, 1 - lr weight_decay) are
 * formed in fp64 and rounded once to fp32.
 */
gm_status gm_hyper_bwd(const float* dlogits, const float* z, const float* gru, float* A, float* c,
                       float* mA, float* vA, float* mc, float* vc, int64_t L, int64_t D, int64_t H,
                       int64_t G_total, double lr, double beta1, double beta2, double eps,
                       double weight_decay, int32_t step, float* dgru, void* ws, size_t ws_bytes,
                       gm_stream_t stream);

/*
 * gm_adamw -- one AdamW step (as above) on n fp32 parameters p with gradient
 * g and moments m, v, in place.  n = 0 is a no-op.
 */
gm_status gm_adamw(float* p, const float* g, float* m, float* v, int64_t n, double lr, double beta1,
                   double beta2, double eps, double weight_decay, int32_t step, gm_stream_t stream);

#ifdef __cplusplus
} /* extern "C" */
#endif

#endif /* GROUPMASK_H */
