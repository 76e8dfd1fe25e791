/*
 * lcvq.h -- C ABI of the LC-VQ linear layer library (liblcvq.so, gfx950).
 *
 * The layer is the linear-constrained vector-quantised linear layer of
 * LC-QAT (arXiv 2606.10531).  A weight matrix W (m out-features x n
 * in-features) is held as latent proxy weights Z (the paper's W_p), one
 * d x d map A and one offset b of length d shared by the whole matrix
 * (eq. lc_codebook, Sec. 2.2).  The forward pass (Sec. 3.2) is
 *
 *   codes  = clip(round(Z), 0, 3)                     eq. quant_param, b = 2 bits
 *   W_hat[r, g*d + j] = sum_k A[j,k] codes[r, g*d + k] + b[j]   def. forward
 *   Y      = X W_hat^T                                X: N tokens x n
 *
 * and is evaluated in the reformulated order of def. forward_x
 * (Y = (X blockdiag(A)) codes^T + (X b~) 1^T), so the dense W_hat is never
 * written to device memory.  The backward pass uses the straight-through
 * estimator of Sec. 3.3 (round() passes gradients; clip() zeroes them outside
 * its range) and yields dX, dZ, dA and db.
 *
 * Conventions shared by every call
 *  - All tensors are dense, row-major, caller-owned DEVICE pointers; the
 *    library allocates no device memory.  Its only mutable global state is
 *    the kernel timer below (instrumentation, off unless enabled): every
 *    layer call is otherwise a pure function of its arguments.
 *  - A layer call takes at most 2^22 - 256 = 4194048 tokens (N); more returns
 *    LCVQ_EUNSUPPORTED (split the tokens over several calls, accumulating the
 *    weight gradients).
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Every call only enqueues work on it and returns; device-side results are
 *    visible after the caller synchronises that stream.
 *  - round() is IEEE round-half-to-even; clip bounds are inclusive; a NaN
 *    latent gives code 0 and mask 0; +inf / -inf give codes 3 / 0, mask 0.
 *  - Arguments are validated on the host before anything is enqueued; on any
 *    error nothing is enqueued and outputs are untouched.  A zero-sized
 *    problem returns LCVQ_OK without enqueuing work.  Launch failures return
 *    LCVQ_EHIP.  lcvq_last_error() gives a human-readable detail for the
 *    calling thread's last non-OK status.
 *  - Outputs must not alias inputs.  Calls that share a workspace must not
 *    overlap in time (use one stream, or one workspace per stream).
 */
#ifndef LCVQ_H
#define LCVQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LCVQ_OK = 0,
  LCVQ_EINVAL = 1,        /* null required pointer, negative size, bad enum, n % d != 0 */
  LCVQ_EUNSUPPORTED = 2,  /* d not in {4, 8}; bf16 path with m or n not a multiple of 8 */
  LCVQ_EALIGN = 3,        /* a device pointer not 16-byte aligned */
  LCVQ_EWORKSPACE = 4,    /* workspace smaller than lcvq_workspace_bytes() */
  LCVQ_EHIP = 5           /* the HIP runtime refused a launch */
} lcvq_status_t;

/* Element type of Z, X, Y, dY, dX (and of dZ unless dz_dtype says otherwise).
 * A, b, dA and db are always fp32. */
typedef enum { LCVQ_F32 = 0, LCVQ_BF16 = 1 } lcvq_dtype_t;

/* What a code source holds. */
typedef enum {
  LCVQ_SRC_LATENT = 0,    /* latent Z (m x n, fp32 or bf16): codes = clip(round(Z), 0, 3) */
  LCVQ_SRC_CODES_U8 = 1,  /* one byte per code (m x n, values above 3 are taken as 3) */
  LCVQ_SRC_PACKED2 = 2    /* packed 2-bit codes, layout of lcvq_pack2bit */
} lcvq_src_t;

/* Where the straight-through gradient is passed (Sec. 3.3 with the chain rule
 * of clip()). */
typedef enum {
  LCVQ_MASK_ROUNDED = 0,  /* default: 0 <= round(Z) <= 3, i.e. Z in [-0.5, 3.5) */
  LCVQ_MASK_LATENT = 1    /* 0 <= Z <= 3 */
} lcvq_mask_t;

/* Gradient estimator of the latent through round() (Sec. 3.3). */
typedef enum {
  LCVQ_EST_STE = 0,  /* straight-through: slope 1 */
  LCVQ_EST_DGE = 1   /* differentiable gradient estimator (eq. dge), see lcvq_linear_bwd_dge */
} lcvq_estimator_t;

typedef enum { LCVQ_OP_FWD = 0, LCVQ_OP_BWD = 1, LCVQ_OP_FWD_PACKED = 2 } lcvq_op_t;

/*
 * lcvq_pack2bit -- packed 2-bit codes, four per byte.
 * The paper fixes the width only (2-bit codes, Sec. 2.1 / 3.2); this layout is
 * the library's: the code of column c of row r sits at bits 2*(c % 4) and
 * 2*(c % 4) + 1 of byte r*(n/4) + c/4 (least significant first), so a
 * little-endian 32-bit word holds 16 consecutive codes.
 *   src      m x n latent Z (src_kind LATENT, element type src_dtype) or
 *            m x n uint8 codes (src_kind CODES_U8, src_dtype ignored)
 *   packed   m * n / 4 bytes, written
 * Requires n % 4 == 0 (else LCVQ_EINVAL); src and packed 16-byte aligned.
 */
lcvq_status_t lcvq_pack2bit(const void *src, int32_t src_kind, int32_t src_dtype,
                            int64_t m, int64_t n, uint8_t *packed, void *stream);

/*
 * lcvq_dequant -- the dense effective weight W_hat (def. forward, Sec. 3.2):
 *   W_hat[r, g*d + j] = sum_k A[j*d + k] * code[r, g*d + k] + b[j]
 * with codes taken from `src` (lcvq_src_t `src_kind`; element type `src_dtype`
 * for LATENT).  A is d x d row-major fp32, b has d fp32 entries.  W_hat is
 * m x n of element type `out_dtype` (bf16 results are rounded to nearest even
 * from fp32 arithmetic; packed sources sum each group's two 4-code halves from
 * per-map tables, so their fp32 rounding can differ from the plain fma chain's
 * in the last bit).  d in {4, 8}; n % d == 0.  This is a utility for export and
 * inspection: the training calls below never form W_hat.
 */
lcvq_status_t lcvq_dequant(int64_t m, int64_t n, int32_t d, int32_t src_kind, int32_t src_dtype,
                           const void *src, const float *A, const float *b,
                           void *W_hat, int32_t out_dtype, void *stream);

/*
 * lcvq_xavier_quantizer -- the quantiser domain of the Xavier
 * reparameterisation (Sec. 3.4, eq. xavier_preprocess) for an m x n matrix of
 * 2-bit codes: a = sqrt(6 / (m + n)), s' = 2a / 3, t = 3/2, and
 *   *q_scale = 1 / s',  *q_shift = t
 * (computed in double, each rounded to fp32 once), the values to pass to the
 * _ex layer calls so that codes = clip(round(W_p / s' + t), 0, 3).  Host-side
 * only: writes the two floats through host pointers, launches nothing.
 * m, n > 0 and non-NULL outputs (else LCVQ_EINVAL).
 */
lcvq_status_t lcvq_xavier_quantizer(int64_t m, int64_t n, float *q_scale, float *q_shift);

/*
 * lcvq_xavier_init -- initial proxy weights of the Xavier reparameterisation
 * (Sec. 3.4, eq. xavier_preprocess): W_p = s' (W_z - t) for codes W_z, with s'
 * and t as in lcvq_xavier_quantizer, evaluated per element in fp32 as
 * fma(s', code, -s' t) (s' and -s' t rounded to fp32 once), i.e. lcvq_dequant
 * with A = s' I and b = -s' t up to fp32 rounding.
 *   codes     m x n bytes (src_kind LCVQ_SRC_CODES_U8; values above 3 are taken
 *             as 3) or m * n / 4 packed bytes (LCVQ_SRC_PACKED2)
 *   W_p       m x n of element type out_dtype (F32 or BF16), written
 * Requires m, n > 0, n % 4 == 0, both pointers 16-byte aligned.  Round trip:
 * the _ex calls with lcvq_xavier_quantizer's values give these codes back.
 */
lcvq_status_t lcvq_xavier_init(int64_t m, int64_t n, int32_t src_kind, const void *codes, void *W_p,
                               int32_t out_dtype, void *stream);

/*
 * lcvq_encode -- codes of a dense weight W under the map A, b: for group g of
 * row r, v = A^-1 (w_g - b) and code = clip(round(v), 0, 3) (eq. lc_codebook
 * inverted; round() ties to even).  With A = s G, G orthogonal (the form of
 * eq. init_ab), these are the nearest codewords A z + b of eq. vq_assign,
 * because the distance separates over the d coordinates after the rotation; for
 * other invertible A they are the rounding of A^-1 (w_g - b).  The kernel
 * evaluates v in fp32 (A^-1 by Gauss-Jordan elimination with partial
 * pivoting, then a d-term fma chain), so its codes equal those of the exact v
 * except where the exact v lies within that evaluation's rounding error of a
 * decision boundary (0.5, 1.5, 2.5).  Non-finite weights follow the written
 * sum sum_j Ainv[k, j] (w_j - b_j) in IEEE arithmetic (NaN gives code 0).  A
 * map with a zero pivot (singular) gives NaN v, i.e. code 0; the codes of a
 * nearly singular map carry no meaning.
 *   W          m x n, element type w_dtype (F32 or BF16), 16-byte aligned
 *   A, b       d x d and d fp32
 *   codes_out  NULL, or m x n bytes (values 0..3), written
 *   packed_out NULL, or m * n / 4 bytes in the lcvq_pack2bit layout, written
 * d in {4, 8} (else LCVQ_EUNSUPPORTED), n % d == 0; at least one output.
 */
lcvq_status_t lcvq_encode(int64_t m, int64_t n, int32_t d, const void *W, int32_t w_dtype,
                          const float *A, const float *b, uint8_t *codes_out, uint8_t *packed_out,
                          void *stream);

/*
 * lcvq_workspace_bytes -- device workspace needed by lcvq_linear_fwd
 * (op = LCVQ_OP_FWD), lcvq_linear_bwd / lcvq_linear_bwd_dge (op = LCVQ_OP_BWD)
 * or lcvq_linear_fwd_packed (op = LCVQ_OP_FWD_PACKED, dtype LCVQ_BF16; the
 * size does not depend on N) for these sizes and element type.  Returns 0 for invalid arguments.  The workspace holds
 * transient, library-private data (transformed activations, codes in the
 * matrix-core operand layout, per-token sums, partial sums of dA and db); its
 * contents are undefined between calls.
 */
size_t lcvq_workspace_bytes(int32_t op, int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype);

/*
 * lcvq_linear_fwd -- Y = X W_hat^T for one LC-VQ weight matrix, computed as in
 * def. forward_x (Sec. 3.2): X' = X blockdiag(A) and s = X b~ once per call,
 * then Y = X' codes^T + s 1^T with the codes fed to the matrix cores exactly.
 *   N, m, n   tokens, out-features, in-features; d in {4, 8}; n % d == 0
 *   dtype     element type of Z, X and Y (LCVQ_F32 or LCVQ_BF16)
 *   Z         m x n latent proxy weights
 *   A, b      map (d x d, row-major, A[j*d + k]) and offset (d), fp32
 *   X         N x n activations;  Y  N x m output (written)
 *   packed_codes_out  NULL, or m*n/4 bytes that receive the codes of this call
 *             in the lcvq_pack2bit layout
 *   workspace device buffer of at least lcvq_workspace_bytes(LCVQ_OP_FWD, ...)
 * bf16 additionally requires m % 8 == 0 and n % 8 == 0.
 */
lcvq_status_t lcvq_linear_fwd(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype,
                              const void *Z, const float *A, const float *b,
                              const void *X, void *Y, uint8_t *packed_codes_out,
                              void *workspace, size_t workspace_bytes, void *stream);

/*
 * lcvq_linear_fwd_ex -- lcvq_linear_fwd with the latent in another domain:
 * the quantiser rounds the fp32 value fma(Z, q_scale, q_shift) (one rounding),
 *   codes = clip(round(Z * q_scale + q_shift), 0, 3).
 * This is the Xavier reparameterisation of Sec. 3.4 (eq. xavier_preprocess):
 * with proxy weights W_p = s' (W_z - t), s' = 2a / 3, t = 3/2,
 * a = sqrt(6 / (m + n)), pass Z = W_p, q_scale = 1 / s', q_shift = t (as
 * lcvq_xavier_quantizer gives them).  lcvq_xavier_init makes such W_p from codes.
 * q_scale = 1, q_shift = 0 is lcvq_linear_fwd exactly.  q_scale must be finite
 * and nonzero, q_shift finite (else LCVQ_EINVAL).  packed_codes_out receives
 * these codes.  All else as lcvq_linear_fwd.
 */
lcvq_status_t lcvq_linear_fwd_ex(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype,
                                 const void *Z, float q_scale, float q_shift, const float *A, const float *b,
                                 const void *X, void *Y, uint8_t *packed_codes_out,
                                 void *workspace, size_t workspace_bytes, void *stream);

/*
 * lcvq_linear_fwd_packed -- Y = X W_hat^T with the codes read from their packed
 * 2-bit form (lcvq_pack2bit layout): inference with the compressed weight
 * (def. forward_x, Sec. 3.2, evaluated as in the paper's inference kernel of
 * App. A.2 without ever forming W_hat).  For decode-sized batches: tokens are
 * processed 16 at a time, and the packed codes (m * n / 4 bytes, the only
 * large operand) are streamed once per 16 tokens.
 *   N, m, n    tokens, out-features, in-features; d in {4, 8}
 *   packed     m * n / 4 bytes of codes (device, 16-byte aligned)
 *   A, b       map and offset, fp32 (device)
 *   X          N x n bf16 activations;  Y  N x m output of element type y_dtype
 *              (LCVQ_BF16 or LCVQ_F32), written
 *   workspace  at least lcvq_workspace_bytes(LCVQ_OP_FWD_PACKED, N, m, n, d, LCVQ_BF16)
 * Requires n % 64 == 0 and m % 8 == 0 (else LCVQ_EUNSUPPORTED).  X' = X
 * blockdiag(A) is rounded to bf16 as in lcvq_linear_fwd.  Calls that share a
 * workspace must not run concurrently (it holds per-call tile counters).
 */
lcvq_status_t lcvq_linear_fwd_packed(int64_t N, int64_t m, int64_t n, int32_t d, const uint8_t *packed,
                                     const float *A, const float *b, const void *X, void *Y, int32_t y_dtype,
                                     void *workspace, size_t workspace_bytes, void *stream);

/*
 * lcvq_linear_fwd_packed_noalloc -- lcvq_linear_fwd_packed for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): the same kernels and the same
 * results bit for bit, with the workspace replaced by a fixed array of
 * lcvq_packed_scratch_bytes() = 8 MiB that the library holds per device until
 * the process ends.  Nothing is allocated by this call.  The caller still
 * passes inputs and outputs; every other argument is as in
 * lcvq_linear_fwd_packed.
 *   - A shape whose workspace (lcvq_workspace_bytes(LCVQ_OP_FWD_PACKED, ...))
 *     exceeds the array returns LCVQ_EUNSUPPORTED before anything is enqueued
 *     (every m x n up to 16384 x 131072 fits).
 *   - The stream must belong to the current device (the array's address is
 *     looked up for the current device).
 *   - All calls on one device share that device's array: calls that overlap in
 *     time on one device (different streams, or host threads) race and give
 *     wrong results.  What must start at zero is cleared by each call.
 */
lcvq_status_t lcvq_linear_fwd_packed_noalloc(int64_t N, int64_t m, int64_t n, int32_t d, const uint8_t *packed,
                                             const float *A, const float *b, const void *X, void *Y,
                                             int32_t y_dtype, void *stream);
/* Size in bytes of the per-device array of lcvq_linear_fwd_packed_noalloc. */
size_t lcvq_packed_scratch_bytes(void);

/*
 * lcvq_linear_bwd -- straight-through backward of lcvq_linear_fwd (Sec. 3.3):
 *   dX = dY W_hat                                   (N x n, written, type dtype)
 *   dW = dY^T X  (never stored)
 *   dZ[r, g*d + k] = mask[r, g*d + k] * sum_j dW[r, g*d + j] A[j, k]
 *   dA[j, k] = sum_{r,g} dW[r, g*d + j] code[r, g*d + k]
 *   db[j]    = sum_{r,g} dW[r, g*d + j]
 *   mask_mode  lcvq_mask_t
 *   accumulate 0: dZ, dA, db are overwritten; 1: results are added to them
 *              (gradient accumulation).  dX is always overwritten.
 *   dX, dZ, dA, db  each may be NULL to skip it (dA and db are produced
 *              together: both NULL or both non-NULL)
 *   dz_dtype   element type of dZ: LCVQ_F32, or LCVQ_BF16 when dtype is bf16
 * bf16: dA/db are per-block partial sums added in a fixed order, so repeated
 * calls give the same bits.  fp32: they are summed with floating-point
 * atomics, so their last bits may vary from run to run.
 */
lcvq_status_t lcvq_linear_bwd(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype,
                              const void *Z, const float *A, const float *b,
                              const void *X, const void *dY, int32_t mask_mode, int32_t accumulate,
                              void *dX, void *dZ, int32_t dz_dtype, float *dA, float *db,
                              void *workspace, size_t workspace_bytes, void *stream);

/*
 * lcvq_linear_bwd_dge -- lcvq_linear_bwd with the differentiable gradient
 * estimator of Sec. 3.3 (eq. dge) in place of the straight-through one.  round()
 * is stood in for by f(x) = 1/2 (1 + sign(2x - 1) |2x - 1|^(1/k)) on each
 * rounding interval (quantisation interval delta = 1 on the code-domain
 * latent), so the latent's gradient gains the slope f' at Z's position
 * x = Z - floor(Z) within its interval:
 *   dZ[r, c] = mask[r, c] * min(cap, (1/k) |2x - 1|^(1/k - 1)) * sum_j dW[r, g*d + j] A[j, k]
 * f' is unbounded at x = 1/2, hence the cap (the slope there is `cap` for
 * k > 1; k = 1 gives slope 1 everywhere, i.e. the straight-through result).
 * Through clip(f(Z), 0, 3) the chain rule gives the LCVQ_MASK_LATENT mask;
 * mask_mode selects it as in lcvq_linear_bwd.  dX, dA and db are those of
 * lcvq_linear_bwd.  The paper trains with k = 5.
 *   k    finite, >= 1 (else LCVQ_EINVAL)
 *   cap  finite, > 0 (else LCVQ_EINVAL)
 * All other arguments, the workspace size and the error behaviour are those
 * of lcvq_linear_bwd.
 */
lcvq_status_t lcvq_linear_bwd_dge(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype,
                                  const void *Z, const float *A, const float *b,
                                  const void *X, const void *dY, int32_t mask_mode, float k, float cap,
                                  int32_t accumulate, void *dX, void *dZ, int32_t dz_dtype, float *dA, float *db,
                                  void *workspace, size_t workspace_bytes, void *stream);

/*
 * lcvq_linear_bwd_ex -- the general backward: latent domain as in
 * lcvq_linear_fwd_ex (codes and mask taken at v = fma(Z, q_scale, q_shift);
 * the chain rule through v multiplies dZ by q_scale) and the estimator
 * (lcvq_estimator_t; dge_k and dge_cap as k and cap of lcvq_linear_bwd_dge,
 * ignored for LCVQ_EST_STE):
 *   dZ[r, c] = q_scale * mask(v) * slope(v) * sum_j dW[r, g*d + j] A[j, k].
 * dX, dA and db are those of lcvq_linear_bwd for the codes of v.
 * (q_scale, q_shift) = (1, 0) with LCVQ_EST_STE is lcvq_linear_bwd exactly.
 * All else as lcvq_linear_bwd.
 */
lcvq_status_t lcvq_linear_bwd_ex(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype,
                                 const void *Z, float q_scale, float q_shift, const float *A, const float *b,
                                 const void *X, const void *dY, int32_t mask_mode, int32_t estimator,
                                 float dge_k, float dge_cap, int32_t accumulate, void *dX, void *dZ,
                                 int32_t dz_dtype, float *dA, float *db,
                                 void *workspace, size_t workspace_bytes, void *stream);

/*
 * The training pair: lcvq_linear_fwd_train / lcvq_linear_bwd_train.  A
 * training step runs the forward and then the backward of the same layer on
 * the same Z, A, b, X and quantiser.  The backward's prepass would read Z and
 * X again to rebuild the codes in its own operand layout, the straight-through
 * mask and X' = X blockdiag(A) (def. forward_x, Sec. 3.2) in the
 * weight-gradient operand layout; the forward already reads Z and X, so the
 * pair lets it write those once into a caller-owned `saved` buffer, and the
 * backward's prepass then handles dY alone.  Results are those of
 * lcvq_linear_fwd_ex / lcvq_linear_bwd_ex with the same arguments (the same
 * kernels on the same values).
 *
 * lcvq_saved_bytes -- size of `saved` for N tokens and an m x n matrix (bf16;
 * 0 for LCVQ_F32, whose path needs no saved state, and for invalid arguments).
 * At 4096 x 4096 with 4096 tokens it is 44 MB: the codes (4 bits each), X'
 * (bf16) and two one-bit masks.
 */
size_t lcvq_saved_bytes(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype);

/*
 * lcvq_linear_fwd_train -- lcvq_linear_fwd_ex that also writes the saved state
 * for lcvq_linear_bwd_train into `saved` (bf16: at least lcvq_saved_bytes(...)
 * bytes, 16-byte aligned, else LCVQ_EWORKSPACE / LCVQ_EALIGN; fp32: unused and
 * may be NULL).  Both straight-through masks are saved, so the backward may
 * choose either.  All other arguments as lcvq_linear_fwd_ex.
 */
lcvq_status_t lcvq_linear_fwd_train(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype,
                                    const void *Z, float q_scale, float q_shift, const float *A, const float *b,
                                    const void *X, void *Y, uint8_t *packed_codes_out,
                                    void *saved, size_t saved_bytes,
                                    void *workspace, size_t workspace_bytes, void *stream);

/*
 * lcvq_linear_bwd_train -- lcvq_linear_bwd_ex that reads the codes, X' and the
 * mask from `saved`, as the preceding lcvq_linear_fwd_train wrote them.  The
 * caller guarantees that call had the same N, m, n, d, dtype, Z, A, b, X,
 * q_scale and q_shift and that `saved` is unchanged since (the library cannot
 * check device contents; a mismatch gives wrong gradients, not a fault).  Z
 * and X are still read: Z by the differentiable estimator and the fp32 path, X
 * for dA and db.  Same workspace as lcvq_linear_bwd_ex; all other arguments
 * and the error behaviour as lcvq_linear_bwd_ex.
 */
lcvq_status_t lcvq_linear_bwd_train(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype,
                                    const void *Z, float q_scale, float q_shift, const float *A, const float *b,
                                    const void *X, const void *dY, int32_t mask_mode, int32_t estimator,
                                    float dge_k, float dge_cap, int32_t accumulate, void *dX, void *dZ,
                                    int32_t dz_dtype, float *dA, float *db, const void *saved, size_t saved_bytes,
                                    void *workspace, size_t workspace_bytes, void *stream);

/*
 * lcvq_adamw_step -- one AdamW update of a flat fp32 parameter array: the
 * optimiser the paper trains Z, A and b with (Sec. 4.4), with bias correction
 * and decoupled weight decay, all arithmetic in fp32:
 *   m1 = beta1 m1 + (1 - beta1) g;   m2 = beta2 m2 + (1 - beta2) g^2
 *   theta = theta - lr weight_decay theta
 *           - lr (m1 / (1 - beta1^step)) / (sqrt(m2 / (1 - beta2^step)) + eps)
 *   theta, m1, m2  numel fp32 each, updated in place (caller zeroes m1, m2
 *                  before step 1)
 *   grad           numel gradients of element type grad_dtype (F32 or BF16)
 *   shadow         NULL, or numel elements of shadow_dtype (F32 or BF16) that
 *                  receive the updated theta (bf16: rounded to nearest even);
 *                  the latent copy the layer calls read
 *   step           1-based step count (>= 1)
 * Requires beta1, beta2 in [0, 1), eps > 0, lr >= 0; pointers 16-byte aligned;
 * theta, m1, m2, grad and shadow must not overlap.  numel == 0 returns LCVQ_OK.
 */
lcvq_status_t lcvq_adamw_step(float *theta, const void *grad, int32_t grad_dtype, float *m1, float *m2,
                              void *shadow, int32_t shadow_dtype, int64_t numel, float lr, float beta1,
                              float beta2, float eps, float weight_decay, int32_t step, void *stream);

/*
 * Instrumentation: device time of individual kernels, measured with HIP events.
 * This timer is the library's one piece of global mutable state (a process-wide
 * record list guarded by a mutex); it is off until enabled and changes no result.
 * lcvq_timer_enable(mask) makes every later launch of a kernel whose bit
 * (1 << lcvq_kernel_t) is set in `mask`, by any thread, record a start event
 * immediately before and a stop event immediately after it on the launch's
 * stream; mask 0 switches recording off and discards pending records.
 * lcvq_timer_read(kernel, &total_ms, &launches) waits for the recorded launches
 * of `kernel`, returns their summed duration and count, and clears them.  Not
 * for use while the stream is being captured into a graph.
 */
typedef enum {
  LCVQ_K_FWD_PREP = 0,  /* forward prepass: codes in the product's operand layout (+ 2-bit pack)
                           and X' = X blockdiag(A), s = X b~ */
  LCVQ_K_FWD = 1,       /* Y = X' codes^T + s 1^T */
  LCVQ_K_BWD_PREP = 2,  /* backward prepass: codes in the input-gradient operand layout, X' and dY
                           in the weight-gradient operand layout (fp32: row sums of dY) */
  LCVQ_K_DX = 3,        /* dX (with dA, db in bf16 mode) */
  LCVQ_K_DW = 4,        /* dZ = mask * (dY^T X') (with dA, db in fp32 mode) */
  LCVQ_K_PACK = 5,      /* lcvq_pack2bit */
  LCVQ_K_DEQUANT = 6,   /* lcvq_dequant */
  LCVQ_K_FILL = 7,      /* zero fills of degenerate shapes */
  LCVQ_K_ADAM = 8,      /* lcvq_adamw_step */
  LCVQ_K_PACKED_PREP = 9,  /* lcvq_linear_fwd_packed: X' and s of up to 16 tokens */
  LCVQ_K_PACKED = 10,      /* lcvq_linear_fwd_packed: Y from the packed codes */
  LCVQ_K_ENCODE = 11,      /* lcvq_encode */
  LCVQ_K_MAP_SUM = 12,     /* bf16 backward: dA, db, summed over the input-gradient product's blocks */
  LCVQ_K_COUNT = 13
} lcvq_kernel_t;
lcvq_status_t lcvq_timer_enable(uint32_t mask);
lcvq_status_t lcvq_timer_read(int32_t kernel, double *total_ms, int64_t *launches);

/* Static description of a status code. */
const char *lcvq_status_string(lcvq_status_t status);

/* Detail message of the calling thread's most recent non-OK status ("" if none). */
const char *lcvq_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LCVQ_H */
