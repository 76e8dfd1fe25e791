// LC encode: the codes of a dense weight under a map A, b (eq. lc_codebook
// inverted).  Per group g of row r, v = A^-1 (w_g - b) and code_k =
// clip(round(v_k), 0, 3).  For A = s G with G orthogonal (the form eq. init_ab
// gives) the distance ||w_g - A z - b|| = s ||v - z|| separates over the d
// coordinates, so these are the nearest codewords of eq. vq_assign; for other
// maps they are the rounding of A^-1 (w_g - b).
//
// v is evaluated in fp32: A^-1 by Gauss-Jordan elimination with partial
// pivoting (largest |pivot|), the pivot row times the reciprocal of the pivot,
// then row_k = fma(-f, pivot_row, row_k) for every other row k; then
// t_j = w_j - b_j and v_k = sum_j Ainv[k, j] t_j as an fma chain.  The codes
// therefore equal those of the exact v except within that evaluation's
// rounding error of a decision boundary.
// Each block inverts A once (one thread, in LDS); HBM-bound otherwise: the
// weight is read once (2 or 4 bytes per element), the codes written once
// (1 byte and / or 2 bits per element).
#include "lcvq_prep.hpp"

namespace lcvq {

template <int D>
__device__ void invert_f32(const float *__restrict__ A, float (*M)[D], float (*I)[D]) {
  for (int i = 0; i < D; ++i)
    for (int j = 0; j < D; ++j) {
      M[i][j] = A[i * D + j];
      I[i][j] = i == j ? 1.0f : 0.0f;
    }
  for (int c = 0; c < D; ++c) {
    int p = c;
    float best = fabsf(M[c][c]);
    for (int r = c + 1; r < D; ++r)
      if (fabsf(M[r][c]) > best) {
        best = fabsf(M[r][c]);
        p = r;
      }
    if (p != c)
      for (int j = 0; j < D; ++j) {
        const float tm = M[c][j], ti = I[c][j];
        M[c][j] = M[p][j];
        I[c][j] = I[p][j];
        M[p][j] = tm;
        I[p][j] = ti;
      }
    const float rcp = __fdiv_rn(1.0f, M[c][c]);
    for (int j = 0; j < D; ++j) {
      M[c][j] = __fmul_rn(M[c][j], rcp);
      I[c][j] = __fmul_rn(I[c][j], rcp);
    }
    for (int k = 0; k < D; ++k) {
      if (k == c) continue;
      const float f = M[k][c];
      for (int j = 0; j < D; ++j) {
        M[k][j] = fmaf(-f, M[c][j], M[k][j]);
        I[k][j] = fmaf(-f, I[c][j], I[k][j]);
      }
    }
  }
}

// One thread per group (grid-stride).  codes: m x n bytes (optional);
// packed: m x n/4 bytes in the lcvq_pack2bit layout (optional).
template <int D, typename WT>
__global__ __launch_bounds__(256) void k_encode(const WT *__restrict__ W, int64_t groups, const float *__restrict__ A,
                                                const float *__restrict__ b, uint8_t *__restrict__ codes,
                                                uint8_t *__restrict__ packed) {
  __shared__ float M[D][D], Ai[D][D];
  if (threadIdx.x == 0) invert_f32<D>(A, M, Ai);
  __syncthreads();
  float inv[D][D], bv[D];
#pragma unroll
  for (int k = 0; k < D; ++k) {
    bv[k] = b[k];
#pragma unroll
    for (int j = 0; j < D; ++j) inv[k][j] = Ai[k][j];
  }
  for (int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x; g < groups; g += (int64_t)gridDim.x * 256) {
    float t[D];
    if constexpr (sizeof(WT) == 2) {
      if constexpr (D == 8) {
        const uint4 u = reinterpret_cast<const uint4 *>(W)[g];
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          t[2 * e] = bf16_lo(w[e]);
          t[2 * e + 1] = bf16_hi(w[e]);
        }
      } else {
        const uint2 u = reinterpret_cast<const uint2 *>(W)[g];
        t[0] = bf16_lo(u.x); t[1] = bf16_hi(u.x); t[2] = bf16_lo(u.y); t[3] = bf16_hi(u.y);
      }
    } else {
#pragma unroll
      for (int e = 0; e < D / 4; ++e) {
        const float4 u = reinterpret_cast<const float4 *>(W)[g * (D / 4) + e];
        t[4 * e] = u.x; t[4 * e + 1] = u.y; t[4 * e + 2] = u.z; t[4 * e + 3] = u.w;
      }
    }
#pragma unroll
    for (int j = 0; j < D; ++j) t[j] = __fsub_rn(t[j], bv[j]);
    uint32_t c[D];
#pragma unroll
    for (int k = 0; k < D; ++k) {
      float v = 0.0f;
#pragma unroll
      for (int j = 0; j < D; ++j) v = fmaf(inv[k][j], t[j], v);
      c[k] = quant_code(v);
    }
    if (codes != nullptr) {
      if constexpr (D == 8) {
        reinterpret_cast<uint2 *>(codes)[g] =
            make_uint2(c[0] | c[1] << 8 | c[2] << 16 | c[3] << 24, c[4] | c[5] << 8 | c[6] << 16 | c[7] << 24);
      } else {
        reinterpret_cast<uint32_t *>(codes)[g] = c[0] | c[1] << 8 | c[2] << 16 | c[3] << 24;
      }
    }
    if (packed != nullptr) {
      uint32_t bits = 0;
#pragma unroll
      for (int k = 0; k < D; ++k) bits |= c[k] << (2 * k);
      if constexpr (D == 8) reinterpret_cast<uint16_t *>(packed)[g] = (uint16_t)bits;
      else packed[g] = (uint8_t)bits;
    }
  }
}

hipError_t launch_encode(const void *W, bool w_bf16, int64_t m, int64_t n, int d, const float *A, const float *b,
                         uint8_t *codes, uint8_t *packed, hipStream_t st) {
  const int64_t groups = m * (n / d);
  int64_t blocks = (groups + 255) / 256;
  if (blocks > 4096) blocks = 4096;  // the grid-stride loop takes the rest
  if (blocks < 1) blocks = 1;
  const unsigned g = (unsigned)blocks;
  if (d == 8) {
    if (w_bf16) k_encode<8, uint16_t><<<g, 256, 0, st>>>((const uint16_t *)W, groups, A, b, codes, packed);
    else k_encode<8, float><<<g, 256, 0, st>>>((const float *)W, groups, A, b, codes, packed);
  } else {
    if (w_bf16) k_encode<4, uint16_t><<<g, 256, 0, st>>>((const uint16_t *)W, groups, A, b, codes, packed);
    else k_encode<4, float><<<g, 256, 0, st>>>((const float *)W, groups, A, b, codes, packed);
  }
  return hipGetLastError();
}

}  // namespace lcvq
