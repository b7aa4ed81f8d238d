/*
 * mpx.h — C ABI of the MI355X (gfx950) mixed-precision training hot path.
 *
 * The calls follow MPX (Gräfe & Trimpe, "MPX: Mixed Precision Training for
 * JAX", arXiv 2507.03312):
 *   §3.1  cast_to_half_precision         -> mpx_cast_to_half
 *   §3.1  cast_to_float32                -> mpx_cast_to_float
 *   §2, §3.4 half forward/backward       -> mpx_linear_fwd, mpx_linear_bwd,
 *                                            mpx_gemm_batched (+ support ops)
 *   §3.3  DynamicLossScaling.unscale      -> mpx_unscale_check (with the
 *         and the finite check of §3.4       all-finite reduction)
 *   §3.3  DynamicLossScaling.adjust       -> mpx_scale_update
 *   §3.5  optimizer_update (skip when     -> mpx_adamw_masked
 *         gradients are not finite)
 *
 * Conventions shared by every call:
 *  - Pointers named d_* and every tensor pointer are DEVICE pointers; the
 *    caller allocates and owns them.  Pointers to hyperparameter structs are
 *    host pointers, read during the call.
 *  - "half" means IEEE binary16 (MPX_F16) or bfloat16 (MPX_BF16), stored as
 *    16-bit values.  Every rounding to half is round-to-nearest-even; overflow
 *    gives +-inf; subnormals are kept; NaN stays NaN.
 *  - Matrices are row-major.  A linear layer's weight W is [N, K] (out, in), so
 *    the layer computes Y[M, N] = X[M, K] W^T + b.
 *  - Every call is asynchronous on `stream` (a hipStream_t, NULL = the null
 *    stream) and never synchronises the host.  Calls on one stream run in
 *    order; results are visible to later calls on the same stream.
 *  - Full precision (MPX's use_mixed_precision switched off, the baseline of
 *    §4): mpx_linear_fwd/bwd, mpx_gemm_batched, mpx_layernorm_fwd/bwd,
 *    mpx_softmax_fwd/bwd, mpx_cross_entropy, mpx_mse, mpx_patchify_cast and
 *    mpx_embed_assemble(_bwd) also accept dt == MPX_F32: every tensor named
 *    "half" in their description is then float32 and half() is the identity
 *    (d_nonfinite must be NULL).
 *  - Return value: MPX_OK (0) or a negative code; mpx_last_error() gives a
 *    message (per host thread).  Invalid arguments are detected before
 *    anything is launched.  Non-finite DATA is never an error: it is reported
 *    through the non-finite count (MPX §2.1: overflow makes the step skip).
 *  - The calls that write parameter gradients (mpx_linear_bwd's dW and db,
 *    mpx_layernorm_bwd's and mpx_classifier_head's dgamma and dbeta,
 *    mpx_embed_assemble_bwd's dcls and dpos) take a nullable int32 device
 *    counter d_nonfinite: when set, the number of those half results whose
 *    exponent bits are all ones (+-inf or NaN) is ADDED to it atomically.
 *    That is the finite check of MPX §3.4 done where the gradients are
 *    written: a step that zeroes the counter (mpx_zero), passes it to every
 *    gradient-writing call and then hands it to mpx_adamw_masked and
 *    mpx_scale_update gets the same count as mpx_unscale_check over the
 *    gradient list, without reading the gradients again.  Activation
 *    cotangents (dX) are never counted.
 *  - The library keeps no state between calls except tensor-list objects
 *    (and their small device tables), which the caller creates and destroys,
 *    and the static scratch array of mpx_linear_bwd_noalloc (one per GPU).
 */
#ifndef MPX_H
#define MPX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { MPX_F32 = 0, MPX_F16 = 1, MPX_BF16 = 2 } mpx_dtype;

enum {
  MPX_OK = 0,
  MPX_ERR_INVALID = -1,     /* null pointer, bad size, bad dtype, mismatched lists */
  MPX_ERR_UNSUPPORTED = -2, /* a valid request the library does not implement */
  MPX_ERR_HIP = -3,         /* a HIP runtime call or kernel launch failed */
  MPX_ERR_WORKSPACE = -4    /* workspace missing or smaller than required */
};

/* Dynamic loss-scale state (MPX §3.3), resident in device memory.
 * scale: current factor (a power of two in practice); counter: consecutive
 * finite steps since the last change; period: finite steps needed to grow;
 * factor: growth/shrink factor (2); min_scale/max_scale: clamps. */
typedef struct {
  float scale;
  int32_t counter;
  int32_t period;
  float factor;
  float min_scale;
  float max_scale;
} mpx_scale_state;

/* AdamW hyperparameters (decoupled weight decay), given in float64 on the
 * host.  Derived constants (1 - beta, bias corrections) are computed from
 * these in float64 and rounded to float32 once. */
typedef struct {
  double lr;
  double beta1;
  double beta2;
  double eps;
  double weight_decay;
} mpx_adamw_hp;

/* An immutable list of device tensors (the float leaves of a parameter
 * tree, MPX §3.1), described once so a whole tree is swept by a single
 * multi-tensor launch.  ptrs[i] points to numels[i] elements (numels[i] >= 0);
 * the element type is given per call.  The library copies the descriptors to
 * device memory (a synchronous upload: create lists at set-up, not inside a
 * captured region) and owns that copy; the caller keeps owning the tensors and
 * must keep them alive while the list is used. */
typedef struct mpx_tlist_s* mpx_tlist;

int mpx_tlist_create(const void* const* ptrs, const int64_t* numels, int32_t n,
                     mpx_tlist* out);
int mpx_tlist_destroy(mpx_tlist list);
int64_t mpx_tlist_numel(mpx_tlist list);

/* MPX §3.1 (cast_to_half_precision / cast_to_float16 / cast_to_bfloat16):
 * dst[i][j] = half(src[i][j]) for every tensor i of the float32 list `src`,
 * in one multi-tensor launch.  `dst` must have the same numels as `src`;
 * `half` is MPX_F16 or MPX_BF16. */
int mpx_cast_to_half(mpx_tlist src_f32, mpx_tlist dst_half, mpx_dtype half, void* stream);

/* MPX §3.1 cast_to_float32, the other direction: dst[i][j] = float32(src[i][j])
 * for every tensor i of the half list `src` (dtype `half`), exact, in one
 * multi-tensor launch.  `dst` (float32) must have the same numels as `src`.
 * With mpx_cast_to_half it carries the PyTree casts of §3.1 and the
 * function casts of §3.2 (cast_function, force_full_precision), which the
 * Python layer composes. */
int mpx_cast_to_float(mpx_tlist src_half, mpx_tlist dst_f32, mpx_dtype half, void* stream);

/* MPX §3.3 unscale and the finite check of §3.4 (the "convert to float32,
 * divide by the scale, check for overflow" steps of the recipe in §2.1).
 * Over every element g of the half list `grads` (dtype `gdt`):
 *   *d_nonfinite = number of elements whose exponent bits are all ones
 *                  (+-inf or NaN); 0 means the gradients are finite;
 *   if out_f32 != NULL: out_f32[i][j] = float32(g) / d_state->scale
 *                  (widen first, then divide; exact for a power-of-two scale).
 * The count is exact (integer); *d_nonfinite is overwritten, not added to
 * (it is zeroed first, then workgroups that find non-finite values add their
 * counts, so two calls sharing d_nonfinite must not overlap). */
int mpx_unscale_check(mpx_tlist grads, mpx_dtype gdt, const mpx_scale_state* d_state,
                      int32_t* d_nonfinite, mpx_tlist out_f32, void* stream);

/* MPX §3.3 adjust(grads_finite), the dynamic rule of §2.1, on device state:
 *   if *d_nonfinite == 0: counter += 1; if counter == period:
 *                         scale = min(scale * factor, max_scale), counter = 0
 *   else:                 scale = max(scale / factor, min_scale), counter = 0
 * One thread; stream-ordered after the unscale check and the optimizer. */
int mpx_scale_update(mpx_scale_state* d_state, const int32_t* d_nonfinite, void* stream);

/* MPX §3.5 optimizer_update: AdamW on float32 masters, applied only when the
 * gradients are finite (*d_nonfinite == 0).  On a skipped step nothing is
 * written at all: p, m, v, *d_step and half_copy keep their bit patterns.
 * On an applied step, with t = *d_step + 1 and g = float32(grad) / scale:
 *   m = b1 m + (1 - b1) g;  v = b2 v + (1 - b2) g^2
 *   p = p - lr (m / (1 - b1^t) / (sqrt(v / (1 - b2^t)) + eps) + wd p)
 *   *d_step = t;  half_copy (if not NULL) = half(p) in dtype `half`.
 * grads has dtype `gdt` (MPX_F16, MPX_BF16 or MPX_F32 for already-unscaled
 * gradients, in which case the scale is not applied).  The scale is read from
 * d_state, so call this before mpx_scale_update.  All lists must have equal
 * numels; hp is read on the host during the call. */
int mpx_adamw_masked(mpx_tlist p32, mpx_tlist m32, mpx_tlist v32, mpx_tlist grads,
                     mpx_dtype gdt, const mpx_adamw_hp* hp, int32_t* d_step,
                     const mpx_scale_state* d_state, const int32_t* d_nonfinite,
                     mpx_tlist half_copy, mpx_dtype half, void* stream);

/* Activation codes. */
enum { MPX_ACT_NONE = 0, MPX_ACT_GELU_TANH = 1 };

/* Half-precision linear layer forward (MPX §2: forward pass in half
 * precision; products accumulated in float32).  X [M,K], W [N,K], b [N]
 * (nullable), R [M,N] (nullable residual), Y [M,N], Ypre [M,N]; all `dt`.
 *   pre = half(sum_k X[m,k] W[n,k] + b[n])        (one rounding)
 *   act == MPX_ACT_NONE:      out = pre
 *   act == MPX_ACT_GELU_TANH: Ypre = pre (required), out = half(gelu(pre))
 *   Y = R ? half(out + R) : out
 * M, N, K >= 1.  Rows are dense (leading dimension = row length).
 * dt == MPX_F32 is full-precision training (MPX's use_mixed_precision
 * switched off, the baseline of §4): every operand and result is float32,
 * the products run on the float32 matrix cores and half() above is the
 * identity. */
int mpx_linear_fwd(const void* X, const void* W, const void* b, const void* R, void* Y,
                   void* Ypre, int64_t M, int64_t N, int64_t K, mpx_dtype dt, int32_t act,
                   void* stream);

/* Half-precision linear layer backward (MPX §2.1: gradients of the scaled
 * loss, in half precision).  For Y = X W^T + b and the half cotangent dY:
 *   dX = half(dY W)            [M,K] (skipped when dX is NULL; needs W)
 *   dW = half(dY^T X)          [N,K] (skipped when dW is NULL; needs X)
 *   db = half(sum_m dY[m,:])   [N]   (skipped when db is NULL)
 * At least one of dX, dW, db.  If x_act == MPX_ACT_GELU_TANH, X was produced
 * as X = gelu(Xpre) and dX is returned for Xpre instead:
 * dX = half(half(dY W) * gelu'(Xpre)).  Any subset may be requested, so dX
 * (on the critical path) and dW / db can run on different streams.
 * `workspace` (device, ws_bytes) holds split-K partial sums and column
 * partials; its required size is mpx_linear_bwd_workspace(M, N, K) when dW
 * or db is requested (a dX-only call needs none, a db-only call only the
 * column partials, which that size always covers).  Concurrent calls need
 * separate workspaces.  d_nonfinite (nullable) counts non-finite dW and db
 * elements (MPX §3.4's check, fused into the kernels that write them).
 * dt == MPX_F32: the same products in float32 (full precision, see
 * mpx_linear_fwd; the workspace size is the same); d_nonfinite must be NULL. */
int mpx_linear_bwd(const void* X, const void* W, const void* dY, const void* Xpre,
                   int32_t x_act, void* dX, void* dW, void* db, int64_t M, int64_t N,
                   int64_t K, mpx_dtype dt, void* workspace, size_t ws_bytes,
                   int32_t* d_nonfinite, void* stream);
size_t mpx_linear_bwd_workspace(int64_t M, int64_t N, int64_t K);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * mpx_linear_bwd without a workspace argument.  Same arguments, results
 * (the same kernels, bit for bit) and errors as mpx_linear_bwd; the split-K
 * and column partials live in a static device array of
 * MPX_LINEAR_BWD_NOALLOC_SCRATCH bytes that the library holds on every GPU
 * it runs on until the process ends.  The call allocates nothing (no
 * hipMalloc, hipFree or allocating library routine).  A product whose
 * mpx_linear_bwd_workspace(M, N, K) exceeds that size (column partials only,
 * for a db-only call) is rejected with MPX_ERR_WORKSPACE before anything is
 * launched.  The split-K partials of dW never exceed 32 MiB (at most 512
 * output tiles of 128 x 128 float32 sums); the column partials of db take
 * 4 bytes per output column per row slice, so only layers with more than
 * about 16 million outputs are rejected (every weight gradient of the ViT
 * workloads needs at most about 28 MB).  All calls on one GPU share its array: calls that overlap on that
 * GPU (concurrent streams, or host threads) race and give wrong results;
 * order them on one stream or with events.  The first call on a GPU looks up
 * the array's device address (hipGetSymbolAddress, not a stream operation);
 * make one call outside any graph capture first. */
#define MPX_LINEAR_BWD_NOALLOC_SCRATCH (64u << 20)
int mpx_linear_bwd_noalloc(const void* X, const void* W, const void* dY, const void* Xpre,
                           int32_t x_act, void* dX, void* dW, void* db, int64_t M, int64_t N,
                           int64_t K, mpx_dtype dt, int32_t* d_nonfinite, void* stream);

/* Batched half GEMM with float32 accumulation (attention QK^T, PV and their
 * backward).  For i0 < nb0, i1 < nb1, with offsets o_X = i0*sX0 + i1*sX1
 * (elements):
 *   C[o_C + m*ldc + n] = half(sum_k opA(m,k) opB(k,n))
 *   opA(m,k) = A[o_A + m*lda + k] if trans_a == 0, else A[o_A + k*lda + m]
 *   opB(k,n) = B[o_B + k*ldb + n] if trans_b == 0, else B[o_B + n*ldb + k]
 * M, N, K >= 1. */
int mpx_gemm_batched(int32_t trans_a, int32_t trans_b, int64_t M, int64_t N, int64_t K,
                     int64_t nb0, int64_t nb1, const void* A, int64_t lda, int64_t sA0,
                     int64_t sA1, const void* B, int64_t ldb, int64_t sB0, int64_t sB1,
                     void* C, int64_t ldc, int64_t sC0, int64_t sC1, mpx_dtype dt,
                     void* stream);

/* Tile configuration of the GEMMs above, for tuning and tests: 0 (default)
 * picks per call from the problem shape; 1..11 force one configuration
 * (1: 64x64 register-staged; 2: 128x128 register-staged; 3: 256x256,
 * 4: 256x128, 5: 128x256, 6: 128x128 four-stage, 7: 128x128 two-stage
 * direct-to-LDS; 8: one wave or lane per output, for skinny products with
 * at most bias and residual epilogues; 9: 64x128 direct-to-LDS, A k-major;
 * 10 and 11: 7 and 9 with persistent workgroups that walk the tiles, for
 * products without split-K or batching).
 * A forced configuration that a call's operands do not allow (alignment,
 * k not a multiple of 64, layout, epilogue) falls back to the automatic
 * choice.  Process-wide setting; not synchronised with concurrent calls.
 * Errors: MPX_ERR_INVALID for a value outside [0, 11]. */
int mpx_gemm_set_config(int32_t config);

/* Fused multi-head self-attention core (MPX §2.1 half products with float32
 * accumulation; §3.2 softmax and its backward in full precision), one pass
 * each way:
 *   S = half(Q K^T);  P = half(softmax(S / sqrt(hd))) (float32 math);
 *   O = half(P V).
 * qkv [B*T, 3*H*hd] half, row-major: Q | K | V, head h at columns h*hd of
 * each third.  O [B*T, H*hd].  P [B*H, T, ldP] with ldP = T rounded up to a
 * multiple of 8: the probabilities, kept for the backward pass (columns
 * T..ldP-1 are written as 0).  Buffers are caller-owned device memory.
 * Implemented for hd == 64 and 1 <= T <= 256 (else MPX_ERR_UNSUPPORTED);
 * qkv, O and P 16-byte aligned (else MPX_ERR_INVALID). */
int mpx_attention_fwd(const void* qkv, void* O, void* P, int64_t B, int64_t T, int64_t H,
                      int64_t hd, mpx_dtype dt, void* stream);

/* Backward of mpx_attention_fwd, given the P it wrote and dO [B*T, H*hd]:
 *   dP = half(dO V^T);  dV = half(P^T dO);
 *   dS = half(scale P (dP - rowsum(dP P))) (float32 math, scale = 1/sqrt(hd));
 *   dQ = half(dS K);  dK = half(dS^T Q),
 * written into dqkv [B*T, 3*H*hd] in the layout of qkv.  Same limits as the
 * forward; qkv, dO and dqkv 16-byte aligned, P 8-byte aligned.  One kernel, dS
 * never leaves the chip: workspace and ws_bytes are accepted for
 * compatibility and ignored (workspace may be NULL), and
 * mpx_attention_bwd_workspace returns 0. */
int mpx_attention_bwd(const void* qkv, const void* P, const void* dO, void* dqkv, int64_t B,
                      int64_t T, int64_t H, int64_t hd, mpx_dtype dt, void* workspace,
                      size_t ws_bytes, void* stream);
size_t mpx_attention_bwd_workspace(int64_t B, int64_t T, int64_t H, int64_t hd);

/* ---- Support ops of the half forward/backward (full-precision islands,
 * MPX §3.2 force_full_precision: sums, means, softmax) ---- */

/* Row LayerNorm, eps 1e-5, float32 math on widened half inputs.
 * X [rows, d] with row stride ldx (elements), Y [rows, d] dense, gamma/beta [d]
 * half.  mean_rstd (float32 [rows, 2], nullable) receives (mean, 1/std). */
int mpx_layernorm_fwd(const void* X, int64_t ldx, const void* gamma, const void* beta,
                      void* Y, float* mean_rstd, int64_t rows, int64_t d, mpx_dtype dt,
                      void* stream);

/* The input cast of MPX §3.4 fused with a first LayerNorm (a model whose
 * float32 inputs feed a pre-LayerNorm block): X float32 [rows, d] with row
 * stride ldx; Xh = half(X) [rows, d] dense (round to nearest even), and Y,
 * mean_rstd exactly as mpx_layernorm_fwd(Xh, d, gamma, beta, Y, mean_rstd)
 * gives them: the same bits as mpx_cast_to_half followed by that call, in one
 * pass.  1 <= d <= 2048; half dtypes only. */
int mpx_layernorm_fwd_cast(const float* X, int64_t ldx, const void* gamma, const void* beta,
                           void* Xh, void* Y, float* mean_rstd, int64_t rows, int64_t d,
                           mpx_dtype dt, void* stream);

/* LayerNorm backward.  dX = half(dLN) or, if Rgrad != NULL, dX = half(Rgrad +
 * half(dLN)) (the residual branch's cotangent added after the LN cotangent is
 * rounded).  X has row stride ldx; dX, dY, Rgrad are dense [rows, d] unless
 * ldo (row stride of dX and Rgrad) says otherwise.  dgamma, dbeta [d] half =
 * half(column sums); their partial sums use `workspace` (float32,
 * mpx_layernorm_bwd_workspace bytes).  dX (NULL: skipped) and the pair
 * dgamma / dbeta (both NULL: skipped, no workspace needed) may be requested
 * in separate calls, e.g. on two streams; at least one must be given; the
 * split calls give the same bits as one call computing both.
 * d_nonfinite (nullable) counts non-finite dgamma / dbeta elements. */
int mpx_layernorm_bwd(const void* X, int64_t ldx, const void* gamma, const void* dY,
                      const void* Rgrad, void* dX, int64_t ldo, void* dgamma, void* dbeta,
                      int64_t rows, int64_t d, mpx_dtype dt, void* workspace,
                      size_t ws_bytes, int32_t* d_nonfinite, void* stream);
size_t mpx_layernorm_bwd_workspace(int64_t rows, int64_t d);

/* Row softmax of scale * S (float32 math): P = half(softmax(scale * S)).
 * rows of length n (1 <= n <= 1024) with row stride ld (S and P); columns
 * n..ld-1 of P are set to zero. */
int mpx_softmax_fwd(const void* S, void* P, int64_t rows, int64_t n, int64_t ld, float scale,
                    mpx_dtype dt, void* stream);

/* Softmax backward: dS = half(scale * P * (dP - sum_j dP_j P_j)); same
 * layout as mpx_softmax_fwd, padding columns of dS set to zero. */
int mpx_softmax_bwd(const void* P, const void* dP, void* dS, int64_t rows, int64_t n,
                    int64_t ld, float scale, mpx_dtype dt, void* stream);

/* Workspace (bytes) for the loss calls over n rows (cross-entropy) or n
 * elements (MSE): per-row losses or per-block partial sums, overwritten by
 * every call. */
size_t mpx_loss_workspace(int64_t n);

/* Mean softmax cross-entropy over B rows of C logits (row stride ldz) with
 * int32 labels, and its cotangent seeded with the loss scale (MPX §3.4: the
 * function output is scaled before differentiation):
 *   *d_loss = mean_b(logsumexp(z_b) - z_b[y_b])          (float32)
 *   dZ = half(scale * (softmax(z) - onehot(y)) / B), scale = d_state->scale,
 *   dZ dense [B, C].  The row losses are added in row order (deterministic).
 * A label outside [0, C) makes the loss NaN (never an out-of-range read). */
int mpx_cross_entropy(const void* Z, int64_t ldz, const int32_t* labels, int64_t B,
                      int64_t C, const mpx_scale_state* d_state, float* d_loss, void* dZ,
                      mpx_dtype dt, void* workspace, size_t ws_bytes, void* stream);

/* Workspace (bytes) of mpx_classifier_head for B rows of width d: the row
 * losses and one pair of float32 gamma / beta partial rows per 4 rows,
 * overwritten by every call. */
size_t mpx_classifier_head_workspace(int64_t B, int64_t d);

/* The classifier head of a ViT step, forward and backward, one pass per row
 * (a fusion of mpx_layernorm_fwd, mpx_linear_fwd, mpx_cross_entropy, the dX
 * half of mpx_linear_bwd and mpx_layernorm_bwd for C <= 32 classes; the
 * final LayerNorm and the loss run in full precision, MPX §3.2, and the
 * backward is seeded with the loss scale, §3.4):
 *   Z = half(LayerNorm(X; gamma, beta))                     [B, d] dense
 *   logit = half(Z W^T + b)  (W [C, d], b [C])   (not stored)
 *   *d_loss = mean_b(logsumexp(logit_b) - logit_b[y_b])     (float32)
 *   dlogits = half(scale * (softmax(logit) - onehot(y)) / B) [B, C] dense
 *   dZ = half(dlogits W)  (classes summed in order; not stored)
 *   dX = half(LayerNorm backward of dZ)   rows of stride ldo
 *   dgamma = half(sum_b dZ * xhat), dbeta = half(sum_b dZ)
 * X: B rows of width d with row stride ldx (e.g. the CLS rows of a
 * [B, T, d] activation: ldx = T d); labels: int32 [B]; 1 <= C <= 32,
 * 1 <= d <= 2048, C * d <= 16384 (W is staged in on-chip memory), B <= 2048.  Every result is the same bits as the separate
 * calls give (same arithmetic, summation orders and roundings), except
 * dgamma and dbeta when mpx_layernorm_bwd works in row groups (d = 384 or
 * 768 with 16-byte aligned rows): it adds the same float32 terms over the
 * rows in another grouping, so those two can differ in the last place.  The weight
 * and bias gradients of the linear layer are left to mpx_linear_bwd (from Z
 * and dlogits).  d_nonfinite (nullable) counts non-finite dgamma / dbeta
 * elements.  A label outside [0, C) makes the loss NaN.  Errors:
 * MPX_ERR_INVALID (NULL, sizes, C outside [1, 32], C * d > 16384, B > 2048),
 * MPX_ERR_WORKSPACE. */
int mpx_classifier_head(const void* X, int64_t ldx, const void* gamma, const void* beta,
                        const void* W, const void* b, const int32_t* labels, int64_t B, int64_t d,
                        int64_t C, const mpx_scale_state* d_state, void* Z, float* d_loss,
                        void* dlogits, void* dX, int64_t ldo, void* dgamma, void* dbeta,
                        mpx_dtype dt, void* workspace, size_t ws_bytes, int32_t* d_nonfinite,
                        void* stream);

/* Mean squared error over n elements and its scaled cotangent:
 *   *d_loss = mean((y - t)^2);  dY = half(scale * 2 (y - t) / n).
 * dt == MPX_F32: Y, T and dY are float32 (full precision; half() is the
 * identity; a state with scale 1 gives the unscaled cotangent). */
int mpx_mse(const void* Y, const void* T, int64_t n, const mpx_scale_state* d_state,
            float* d_loss, void* dY, mpx_dtype dt, void* workspace, size_t ws_bytes,
            void* stream);

/* Cast float32 NHWC images [B,H,W,C] to half patch vectors [B*G, p*p*C]
 * (MPX §3.4: inputs cast to half).  Patches row-major over the grid; a
 * patch vector lists pixels row-major, channels fastest. */
int mpx_patchify_cast(const float* images, void* patches, int64_t B, int64_t H, int64_t W,
                      int64_t C, int64_t p, mpx_dtype dt, void* stream);

/* Token assembly of a ViT: X[b,0,:] = half(cls + pos[0]);
 * X[b,1+g,:] = half(E[b*G+g,:] + pos[1+g]) with E the patch embeddings. */
int mpx_embed_assemble(const void* E, const void* cls, const void* pos, void* X, int64_t B,
                       int64_t T, int64_t d, mpx_dtype dt, void* stream);

/* Backward of mpx_embed_assemble: dE[b*G+g,:] = dX[b,1+g,:];
 * dcls = half(sum_b dX[b,0,:]); dpos[t,:] = half(sum_b dX[b,t,:]).
 * d_nonfinite (nullable) counts non-finite dcls and dpos elements. */
int mpx_embed_assemble_bwd(const void* dX, void* dE, void* dcls, void* dpos, int64_t B,
                           int64_t T, int64_t d, mpx_dtype dt, int32_t* d_nonfinite,
                           void* stream);

/* Row gather: dst[r, :] = src[r*stride_rows, :] for r < rows (d columns). */
int mpx_gather_rows(const void* src, int64_t stride_rows, void* dst, int64_t rows, int64_t d,
                    mpx_dtype dt, void* stream);

/* Zero n bytes of device memory with a kernel (usable under graph capture). */
int mpx_zero(void* dst, size_t nbytes, void* stream);

/* Message for the last failing call on this host thread ("" if none). */
const char* mpx_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MPX_H */
