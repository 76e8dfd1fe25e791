// Shared device helpers of the LC-VQ kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lcvq {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

typedef __attribute__((address_space(3))) void lds_void;
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr int kMaxCode = 3;  // 2^b - 1 with b = 2 bits

// ---- bf16 <-> fp32 -------------------------------------------------------

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// fp32 -> bf16 bits, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}
typedef float float2_t __attribute__((ext_vector_type(2)));
// Two fp32 -> packed bf16 (round to nearest even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const float2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

// ---- the quantiser of eq. quant_param ------------------------------------
// code = clip(rint(z), 0, 3); rint is round-half-to-even (v_rndne_f32).
// fmaxf(NaN, 0) = 0, so a NaN latent gives code 0.
__device__ __forceinline__ uint32_t quant_code(float z) {
  float u = __builtin_rintf(z);
  return (uint32_t)fminf(fmaxf(u, 0.0f), (float)kMaxCode);
}
// Straight-through mask: mode 0 "rounded" (0 <= rint(z) <= 3), mode 1 "latent".
__device__ __forceinline__ bool ste_pass(float z, int mode) {
  float v = mode == 0 ? __builtin_rintf(z) : z;
  return v >= 0.0f && v <= (float)kMaxCode;
}

// Quantiser domain (Sec. 3.4): the quantiser rounds fp32 fma(w, scale, shift);
// in the code domain (affine = 0) it rounds w itself, bit for bit.  The latent's
// gradient gains the factor `scale` (1 in the code domain).
struct Quantizer {
  int affine;
  float scale, shift;
};
__device__ __forceinline__ float code_value(float w, const Quantizer &q) {
  return q.affine ? fmaf(w, q.scale, q.shift) : w;
}

// Gradient estimator of the latent: straight-through (dge = 0), or the
// differentiable estimator of eq. dge (Sec. 3.3) with delta = 1, slope
// s |2x - 1|^e capped at `cap`, where s = 1/k and e = 1/k - 1.
struct GradEst {
  int dge;
  float e, s, cap;
};
// The slope at the position x = z - floor(z) of z within its rounding
// interval.  At x = 1/2 (w = 0) it is unbounded for k > 1 and 1 for k = 1; the
// hardware log/exp would give NaN there for k = 1, so that point is set
// explicitly.  A NaN or infinite z gives the (finite) cap; the mask is 0 there.
__device__ __forceinline__ float dge_slope(float z, const GradEst &g) {
  const float w = fabsf(2.0f * (z - floorf(z)) - 1.0f);
  float f = g.s * __builtin_amdgcn_exp2f(g.e * __builtin_amdgcn_logf(w));
  if (w == 0.0f) f = g.e < 0.0f ? g.cap : g.s;
  return fminf(f, g.cap);
}

// ---- operand layouts of v_mfma_f32_16x16x32_bf16 -------------------------
// The instruction reads, in lane L, eight K values of A row L % 16 and eight K
// values of B column L % 16 (K group L / 16 of the 32), and leaves rows
// 4 (L / 16) + e, e = 0..3, of output column L % 16 in the lane.  A 32-row slab
// of the weight side is two 16-row MFMA blocks; MFMA row m = 16 rb + i of the
// slab carries weight-side row slab_row(m) = 8 (i / 4) + 4 rb + (i % 4), so that
// lane L ends with weight-side rows 8 (L / 16) .. + 7 of the slab (block 0:
// the first four, block 1: the last four) for one column: whole groups of
// d = 4 or 8, contiguous in memory.
__host__ __device__ __forceinline__ int slab_row(int m) { return 8 * ((m & 15) >> 2) + 4 * (m >> 4) + (m & 3); }

// A 32 x 64 (M x K) slab of codes occupies 1 KiB: lane L owns 16 bytes, dword
// 2 rb + kk2 holding the codes of weight-side row slab_row(16 rb + L % 16) of
// the slab and K = 32 kk2 + 8 (L / 16) + i (nibble i at bits 4i..4i+3): the A
// operands of the slab's two row blocks for the step's two 32-wide K sub-steps.
// Slabs are stored M-slab-major: slab (mb, kb) at byte ((mb * KB) + kb) * 1024.
__device__ __forceinline__ uint32_t frag_dword_index(int mb, int kb, int KB, int lane, int dw) {
  return ((uint32_t)(mb * KB + kb) * 64u + (uint32_t)lane) * 4u + (uint32_t)dw;
}

// Activations in the B-operand layout: a block of 32 tokens x 64 K (4 KiB)
// holds four 1 KiB fragments, fragment 2 th + kk2 for tokens 32 tb + 16 th +
// 0..15 and K 64 kb + 32 kk2 + 0..31, in which lane L owns the 16 bytes of token
// 32 tb + 16 th + L % 16, K = 64 kb + 32 kk2 + 8 (L / 16) + 0..7.  Blocks are
// token-block-major.

// Token-K operand fragments of the weight-gradient product (features f on the
// MFMA M or N axis, tokens t on K): block (f / 32, t / 64) holds four 1 KiB
// fragments, fragment 2 fh + kk2 for features 16 fh .. + 15 of the block (in
// MFMA order) and tokens 64 kb + 32 kk2 + 0..31; in it lane L owns the 16 bytes
// of feature 32 (f / 32) + sel(16 fh + L % 16), tokens 64 kb + 32 kk2 +
// 8 (L / 16) + 0..7, with sel = slab_row on the M side (in-features) and the
// identity on the N side.

// Eight 4-bit codes (0..3) -> eight exact bf16 values via the fp4 (e2m1)
// converter: nibble c encodes c / 2 in e2m1 for c <= 3, and the scale 2 makes
// it exactly c.
__device__ __forceinline__ bf16x8 nibbles_to_bf16x8(uint32_t w) {
  bf16x2 p0 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, 2.0f, 0);
  bf16x2 p1 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, 2.0f, 1);
  bf16x2 p2 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, 2.0f, 2);
  bf16x2 p3 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, 2.0f, 3);
  bf16x8 r;
  r[0] = p0[0]; r[1] = p0[1]; r[2] = p1[0]; r[3] = p1[1];
  r[4] = p2[0]; r[5] = p2[1]; r[6] = p3[0]; r[7] = p3[1];
  return r;
}

// ---- misc ----------------------------------------------------------------
__host__ __device__ __forceinline__ int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
__host__ __device__ __forceinline__ int64_t ceil_div(int64_t x, int64_t m) { return (x + m - 1) / m; }

// ---- buffer resources ----------------------------------------------------
// Raw buffer over [base, base + bytes) (bytes clamped below 2^31).  Loads at an
// offset >= bytes return zero, which zero-pads tiles at ragged edges; lanes
// with nothing to load use kOffNone.
constexpr uint32_t kOffNone = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, int64_t bytes) {
  int64_t b = bytes < 0 ? 0 : (bytes > 0x7fffffffLL ? 0x7fffffffLL : bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)b, 0x00020000);
}
// 16 bytes per lane from the buffer straight into LDS at lds_base + 16 * lane.
__device__ __forceinline__ void buffer_to_lds16(__amdgpu_buffer_rsrc_t r, lds_void *lds_base, uint32_t off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds_base, 16, (int)off, 0, 0, 0);
}

}  // namespace lcvq
