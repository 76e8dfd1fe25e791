// fp32 mode of the LC-VQ layer: the same three products as the bf16 path,
// evaluated in fp32 on the vector ALUs (gfx950 has no reduced-precision fp32
// matrix format that would keep the 1e-5 accuracy of this mode).
//
// Block tile 64 (I) x 64 (J), K step 16; thread -> rows 2*ti, 2*ti + 1 and the
// eight consecutive columns 8*tj .. 8*tj + 7, so a group of d = 8 (or two of
// d = 4) along J is thread-local.
//   mode 0 forward : I = t, J = r, K = c   P = X'[t,c]   Q = code[r,c]
//   mode 1 input   : I = t, J = c, K = r   P = dY[t,r]   Q = code[r,c]
//   mode 2 weight  : I = r, J = c, K = t   P = dY[t,r]   Q = X[t,c]
#include "lcvq_prep.hpp"

namespace lcvq {

constexpr int kF = 64, kFK = 16;

template <int kMode>
__device__ __forceinline__ float load_p(const float *P, int64_t i, int64_t k, int64_t I, int64_t K, int64_t ld) {
  if (i >= I || k >= K) return 0.0f;
  if constexpr (kMode == 2) return P[k * ld + i];  // dY[t][r], i = r, k = t
  else return P[i * ld + k];                       // X'[t][c] / dY[t][r]
}
template <int kMode>
__device__ __forceinline__ float load_q(const float *Q, int64_t k, int64_t j, int64_t K, int64_t J, int64_t ld,
                                       const Quantizer &qz) {
  if (k >= K || j >= J) return 0.0f;
  if constexpr (kMode == 0) return (float)quant_code(code_value(Q[j * ld + k], qz));  // Z[r][c], j = r, k = c
  else if constexpr (kMode == 1) return (float)quant_code(code_value(Q[k * ld + j], qz));  // Z[r][c], k = r, j = c
  else return Q[k * ld + j];  // X[t][c]
}

template <int kMode, int D>
__global__ __launch_bounds__(256) void k_f32(const float *__restrict__ P, int64_t ldp, const float *__restrict__ Q,
                                             int64_t ldq, int64_t I, int64_t J, int64_t K,
                                             const float *__restrict__ vecI, const float *__restrict__ A,
                                             const float *__restrict__ bvec, const float *__restrict__ Z,
                                             Quantizer qz, int mask_mode, GradEst est, int accumulate,
                                             float *__restrict__ out, int64_t ldo, float *__restrict__ dA,
                                             float *__restrict__ db) {
  __shared__ float Ps[kFK][kF + 1];
  __shared__ float Qs[kFK][kF + 4];
  __shared__ float sred[D * D + D];
  const int tid = threadIdx.x, ti = tid >> 3, tj = tid & 7;
  const int64_t i0 = (int64_t)blockIdx.y * kF, j0 = (int64_t)blockIdx.x * kF;
  float acc[2][8];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 8; ++b) acc[a][b] = 0.0f;

  for (int64_t k0 = 0; k0 < K; k0 += kFK) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = tid + 256 * u;
      if constexpr (kMode == 2) {
        const int ii = e & 63, kk = e >> 6;
        Ps[kk][ii] = load_p<kMode>(P, i0 + ii, k0 + kk, I, K, ldp);
      } else {
        const int kk = e & 15, ii = e >> 4;
        Ps[kk][ii] = load_p<kMode>(P, i0 + ii, k0 + kk, I, K, ldp);
      }
      if constexpr (kMode == 0) {
        const int kk = e & 15, jj = e >> 4;
        Qs[kk][jj] = load_q<kMode>(Q, k0 + kk, j0 + jj, K, J, ldq, qz);
      } else {
        const int jj = e & 63, kk = e >> 6;
        Qs[kk][jj] = load_q<kMode>(Q, k0 + kk, j0 + jj, K, J, ldq, qz);
      }
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kFK; ++kk) {
      const float p0 = Ps[kk][2 * ti], p1 = Ps[kk][2 * ti + 1];
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        const float q = Qs[kk][8 * tj + b];
        acc[0][b] = fmaf(p0, q, acc[0][b]);
        acc[1][b] = fmaf(p1, q, acc[1][b]);
      }
    }
    __syncthreads();
  }

  const int64_t jb = j0 + 8 * tj;
  if constexpr (kMode == 0) {
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int64_t i = i0 + 2 * ti + a;
      if (i >= I) continue;
#pragma unroll
      for (int b = 0; b < 8; ++b)
        if (jb + b < J) out[i * ldo + jb + b] = acc[a][b] + vecI[i];
    }
  } else if constexpr (kMode == 1) {
    // dX[t, g*D + j] = sum_k A[j,k] P[t, g*D + k] + rs[t] b[j]
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int64_t i = i0 + 2 * ti + a;
      if (i >= I) continue;
      const float rst = vecI[i];
#pragma unroll
      for (int g = 0; g < 8 / D; ++g)
#pragma unroll
        for (int j = 0; j < D; ++j) {
          float v = rst * bvec[j];
#pragma unroll
          for (int k = 0; k < D; ++k) v = fmaf(A[j * D + k], acc[a][g * D + k], v);
          const int64_t c = jb + g * D + j;
          if (c < J) out[i * ldo + c] = v;
        }
    }
  } else {
    // dW[r, c] = acc; dZ = mask * (dW-group A) (times the estimator's slope);
    // dA, db summed over (r, g)
    float gA[D * D], gb[D];
#pragma unroll
    for (int x = 0; x < D * D; ++x) gA[x] = 0.0f;
#pragma unroll
    for (int x = 0; x < D; ++x) gb[x] = 0.0f;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int64_t r = i0 + 2 * ti + a;
      const bool rv = r < I;
#pragma unroll
      for (int g = 0; g < 8 / D; ++g) {
        const int64_t cg = jb + g * D;
        const bool valid = rv && cg < J;
        float code[D];
#pragma unroll
        for (int k = 0; k < D; ++k) {
          const float z = code_value(valid ? Z[r * ldo + cg + k] : 0.0f, qz);
          code[k] = (float)quant_code(z);
          float v = 0.0f;
#pragma unroll
          for (int j = 0; j < D; ++j) v = fmaf(acc[a][g * D + j], A[j * D + k], v);
          if (valid && out != nullptr) {
            const float gz = ste_pass(z, mask_mode) ? (est.dge ? v * dge_slope(z, est) : v) * qz.scale : 0.0f;
            float *p = out + r * ldo + cg + k;
            *p = accumulate ? *p + gz : gz;
          }
        }
#pragma unroll
        for (int j = 0; j < D; ++j) {
          gb[j] += acc[a][g * D + j];
#pragma unroll
          for (int k = 0; k < D; ++k) gA[j * D + k] = fmaf(acc[a][g * D + j], code[k], gA[j * D + k]);
        }
      }
    }
    if (dA == nullptr) return;
    for (int x = tid; x < D * D + D; x += 256) sred[x] = 0.0f;
    __syncthreads();
#pragma unroll
    for (int x = 0; x < D * D; ++x) atomicAdd(&sred[x], gA[x]);
#pragma unroll
    for (int x = 0; x < D; ++x) atomicAdd(&sred[D * D + x], gb[x]);
    __syncthreads();
    if (tid < D * D) unsafeAtomicAdd(dA + tid, sred[tid]);
    else if (tid < D * D + D) unsafeAtomicAdd(db + tid - D * D, sred[tid]);
  }
}

static inline dim3 grid2(int64_t J, int64_t I) {
  return dim3((unsigned)ceil_div(J, kF), (unsigned)ceil_div(I, kF));
}

hipError_t launch_fwd_f32(const float *Z, const Quantizer &qz, const float *Xp, const float *s, float *Y,
                          int64_t N, int64_t m, int64_t n, hipStream_t st) {
  k_f32<0, 8><<<grid2(m, N), 256, 0, st>>>(Xp, n, Z, n, N, m, n, s, nullptr, nullptr, nullptr, qz, 0, GradEst{},
                                           0, Y, m, nullptr, nullptr);
  return hipGetLastError();
}

hipError_t launch_dx_f32(const float *Z, const Quantizer &qz, const float *dY, const float *rs, const float *A,
                         const float *b, int d, float *dX, int64_t N, int64_t m, int64_t n, hipStream_t st) {
  if (d == 8)
    k_f32<1, 8><<<grid2(n, N), 256, 0, st>>>(dY, m, Z, n, N, n, m, rs, A, b, nullptr, qz, 0, GradEst{}, 0, dX,
                                             n, nullptr, nullptr);
  else
    k_f32<1, 4><<<grid2(n, N), 256, 0, st>>>(dY, m, Z, n, N, n, m, rs, A, b, nullptr, qz, 0, GradEst{}, 0, dX,
                                             n, nullptr, nullptr);
  return hipGetLastError();
}

hipError_t launch_dz_f32(const float *X, const float *dY, const float *Z, const Quantizer &qz, const float *A,
                         int d, int mask_mode, const GradEst &est, int accumulate, float *dZ, float *dA, float *db,
                         int64_t N, int64_t m, int64_t n, hipStream_t st) {
  if (d == 8)
    k_f32<2, 8><<<grid2(n, m), 256, 0, st>>>(dY, m, X, n, m, n, N, nullptr, A, nullptr, Z, qz, mask_mode, est,
                                             accumulate, dZ, n, dA, db);
  else
    k_f32<2, 4><<<grid2(n, m), 256, 0, st>>>(dY, m, X, n, m, n, N, nullptr, A, nullptr, Z, qz, mask_mode, est,
                                             accumulate, dZ, n, dA, db);
  return hipGetLastError();
}

}  // namespace lcvq
