// Internal launchers of the LC-VQ kernels (host side).
#pragma once

#include "lcvq_common.hpp"

namespace lcvq {

// The bf16 activation transform splits K into at most sixteen chunks and
// writes one partial s per chunk (rows of Np floats); the forward product sums
// them.  A chunk is a whole number of step pairs (the transform takes steps two
// at a time), at least four steps.  Both are at least 1 (ldp may be 0 for an
// empty problem).
constexpr int kMaxActChunks = 16;
inline int act_steps_per_chunk(int64_t ldp) {
  const int64_t spc = (ldp / 64 + kMaxActChunks - 1) / kMaxActChunks;
  return spc <= 4 ? 4 : (int)((spc + 1) / 2 * 2);
}
inline int act_chunks(int64_t ldp) {
  const int64_t c = (ldp / 64 + act_steps_per_chunk(ldp) - 1) / act_steps_per_chunk(ldp);
  return c < 1 ? 1 : (int)c;
}

// streaming kernels (lcvq_prep.hip)
// What the forward of the training pair saves for its backward (bf16): the
// codes in the input-gradient operand layout (as the backward prepass writes
// them), both straight-through masks (rounded, latent) and X' in the
// weight-gradient operand layout.
struct FwdSave {
  uint32_t *frag_t;
  uint64_t *mask_r, *mask_l;
  uint16_t *xt;
};
// bf16 forward prepass: codes (+ 2-bit pack) and X' = X A, partial s, in one
// launch; with `save`, also the backward's operands above from the same reads
hipError_t launch_fwd_prep_bf16(const uint16_t *Z, int64_t m, int64_t n, const Quantizer &qz, uint32_t *frag,
                                uint8_t *packed,
                                const uint16_t *X, int64_t N, int64_t Np, int64_t ldp, int d, const float *A,
                                const float *b, uint16_t *Xp, float *sp, const FwdSave *save, hipStream_t st);
// Tokens of the bf16 backward are padded to whole 256-token tiles of the
// input-gradient product (the weight-gradient operands and row sums use the
// same padding).
inline int64_t bwd_tokens(int64_t N) { return (N + 255) / 256 * 256; }

// The bf16 backward prepass sums each dY row in at most sixteen parts (runs of
// 64-feature sub-tiles of the out-features, padded to 256); the input-gradient
// product adds the parts.  (Sixteen parts: four blocks per CU at 4096 x 4096
// instead of two, 13.7 -> 12.2 us.)
inline int rowsum_subtiles_per_part(int64_t m) {
  const int64_t nfy = (m + 255) / 256 * 4;
  const int64_t spf = (nfy + 15) / 16;
  return spf < 1 ? 1 : (int)spf;
}
inline int rowsum_parts(int64_t m) {
  const int64_t nfy = (m + 255) / 256 * 4;
  const int64_t p = (nfy + rowsum_subtiles_per_part(m) - 1) / rowsum_subtiles_per_part(m);
  return p < 1 ? 1 : (int)p;
}
// Straight-through mask bitmap of an m x n matrix, in tiles of 64 rows x 256
// columns (2 KiB each, row-band-major, mask_col_blocks(n) tiles per band).
// Within a tile, row i holds four 64-bit words (32 bytes), word j for columns
// 64 j .. 64 j + 63 of the tile, bit c % 64 for column c.  Each quantise block
// writes exactly one tile per bitmap.
inline int64_t mask_col_blocks(int64_t n) { return (n + 255) / 256; }
inline int64_t mask_bytes(int64_t m, int64_t n) { return (m + 63) / 64 * mask_col_blocks(n) * 2048; }

// bf16 backward prepass in one launch: codes of the input-gradient product
// (frag, optional; that product reads dY in place), the weight-gradient operands (xt, dyt; skipped when xt is nullptr), the partial
// row sums of dY (rsp: rowsum_parts(m) rows of bwd_tokens(N) floats) and the
// mask bitmap of the straight-through estimator (maskbits, optional; written by
// the quantise blocks, so only together with frag)
hipError_t launch_bwd_prep_bf16(const uint16_t *Z, int64_t m, int64_t n, const Quantizer &qz, uint32_t *frag,
                                const uint16_t *X,
                                const uint16_t *dY, const float *A, int d, int64_t N, uint16_t *xt,
                                uint16_t *dyt, float *rsp, uint64_t *maskbits, int mask_mode, hipStream_t st);
hipError_t launch_act_transform(const void *X, bool bf16, int64_t N, int64_t Np, int64_t n, int d,
                                const float *A, const float *b, void *Xp, int64_t ldp, float *s,
                                hipStream_t st);
hipError_t launch_rowsum(const void *dY, bool bf16, int64_t N, int64_t Np, int64_t m, float *rs, float *dA,
                         float *db, int d, hipStream_t st);
hipError_t launch_pack2bit(const void *src, int kind, bool bf16, int64_t m, int64_t n, uint8_t *packed,
                           const Quantizer &qz, hipStream_t st);
hipError_t launch_dequant(const void *src, int kind, bool z_bf16, int64_t m, int64_t n, int d,
                          const float *A, const float *b, void *W, bool out_bf16, hipStream_t st);
// W[i] = fma(scale, code[i], shift) over `total` codes (kind 1: bytes, 2: packed
// 2-bit; total % 4 == 0): the decode of the diagonal map scale I, shift
hipError_t launch_decode_scalar(const void *src, int kind, int64_t total, float scale, float shift, void *W,
                                bool out_bf16, hipStream_t st);

// layer output from packed 2-bit codes, 16 tokens per pass (lcvq_packed.hip)
struct PackedPlan {
  int64_t nP;     // K padded to whole 256-column steps
  int KT;         // steps
  int row_tiles;  // 64-row tiles
  int nchunks;    // 4096-column chunks of the prepass (partial sums of s)
  int KS, spb;    // K splits over blocks, steps per split
};
PackedPlan packed_plan(int64_t m, int64_t n);
// X' (16 x nP bf16, columns reordered per 16-column group), partial s
// (nchunks x 16 fp32) and zeroed tile counters (row_tiles ints) for tokens
// 0 .. Nc - 1 of X (Nc <= 16)
hipError_t launch_packed_prep(const uint16_t *X, int Nc, int64_t m, int64_t n, int d, const float *A,
                              const float *b, uint16_t *xq, float *sp, int *counters, hipStream_t st);
// Y (Nc x m, bf16 or fp32) = codes X'^T + s; part holds row_tiles * KS * 16 * 64 fp32 split-K partials
hipError_t launch_packed_gemv(const uint8_t *packed, int64_t m, int64_t n, const uint16_t *xq, const float *sp,
                              int Nc, float *part, int *counters, void *Y, bool y_bf16, hipStream_t st);
// Whether the product for Nc tokens runs as one launch that also does the
// prepass (one block per row tile, few tokens, long rows); then
// launch_packed_fused replaces launch_packed_prep + launch_packed_gemv.
bool packed_fused(int64_t m, int64_t n, int Nc);
hipError_t launch_packed_fused(const uint8_t *packed, int64_t m, int64_t n, const uint16_t *X, int Nc, int d,
                               const float *A, const float *b, void *Y, bool y_bf16, hipStream_t st);

// LC encode (lcvq_encode.hip): codes (m x n bytes) and / or packed codes of a dense weight
hipError_t launch_encode(const void *W, bool w_bf16, int64_t m, int64_t n, int d, const float *A, const float *b,
                         uint8_t *codes, uint8_t *packed, hipStream_t st);

// optimiser (lcvq_adam.hip); shadow_kind 0 none, 1 fp32, 2 bf16
hipError_t launch_adamw(float *theta, const void *grad, bool grad_bf16, float *m1, float *m2, void *shadow,
                        int shadow_kind, int64_t numel, float lr, float beta1, float beta2, float eps,
                        float weight_decay, int step, hipStream_t st);

// bf16 matrix-core products (lcvq_gemm.hip)
hipError_t launch_fwd_bf16(const uint32_t *frag, const uint16_t *Xp, int64_t ldp, const float *s,
                           uint16_t *Y, int64_t N, int64_t m, int64_t n, hipStream_t st);
// Map gradients of the input-gradient product: each of its map_rows(N, n)
// blocks stores its partial sums of dA (d x d) and db (d), entry-major (entry
// e of block b at mapp[e * map_rows + b]; every place is written, so mapp
// needs no clearing); launch_map_combine then sums each entry over the blocks
// in a fixed order into dA and db (added to them when accumulating).
int map_rows(int64_t N, int64_t n);
hipError_t launch_dx_bf16(const uint32_t *frag, const uint16_t *dY, const float *rsp, const float *A, const float *b,
                          int d, uint16_t *dX, const uint16_t *X, float *mapp, int64_t N, int64_t m, int64_t n,
                          hipStream_t st);
hipError_t launch_map_combine(const float *mapp, int rows, int d, int accumulate, float *dA, float *db,
                              hipStream_t st);
// maskbits: the straight-through mask; or, with est.dge set, nullptr and the
// mask and slope are taken from Z (bf16, m x n) under mask_mode
hipError_t launch_dw_bf16(const uint16_t *xt, const uint16_t *dyt, const uint64_t *maskbits, const uint16_t *Z,
                          const Quantizer &qz, int mask_mode, const GradEst &est, int accumulate, void *dZ,
                          bool dz_bf16, int64_t N, int64_t m, int64_t n, hipStream_t st);

// fp32 products on the vector ALUs (lcvq_f32.hip)
hipError_t launch_fwd_f32(const float *Z, const Quantizer &qz, const float *Xp, const float *s, float *Y,
                          int64_t N, int64_t m, int64_t n, hipStream_t st);
hipError_t launch_dx_f32(const float *Z, const Quantizer &qz, const float *dY, const float *rs, const float *A,
                         const float *b, int d, float *dX, int64_t N, int64_t m, int64_t n, hipStream_t st);
hipError_t launch_dz_f32(const float *X, const float *dY, const float *Z, const Quantizer &qz, const float *A,
                         int d, int mask_mode, const GradEst &est, int accumulate, float *dZ, float *dA, float *db,
                         int64_t N, int64_t m, int64_t n, hipStream_t st);

}  // namespace lcvq
