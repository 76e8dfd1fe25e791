// One AdamW step over a flat fp32 parameter array (the optimiser of Sec. 4.4:
// Adam with bias correction and decoupled weight decay), with an optional
// bf16 or fp32 copy of the updated parameters for the layer calls.
//
// Pure streaming work: per element it reads theta, m1, m2 (fp32) and the
// gradient (fp32 or bf16) and writes theta, m1, m2 and the copy, so it is bound
// by HBM bandwidth.  Each lane moves four consecutive elements per trip with
// 16-byte (8-byte for bf16) accesses; the last numel % 4 elements are taken by
// the first lanes of block 0.
#include <cmath>

#include "lcvq_prep.hpp"

namespace lcvq {

struct AdamCoef {
  float lr, b1, b2, eps, decay;  // decay = lr * weight_decay
  float c1, c2;                  // 1 / (1 - b1^step), 1 / (1 - b2^step)
};

__device__ __forceinline__ float adam_one(float &th, float g, float &m1, float &m2, const AdamCoef &c) {
  m1 = fmaf(c.b1, m1, (1.0f - c.b1) * g);
  m2 = fmaf(c.b2, m2, (1.0f - c.b2) * (g * g));
  const float upd = (m1 * c.c1) / (__builtin_sqrtf(m2 * c.c2) + c.eps);
  th = th - c.decay * th - c.lr * upd;
  return th;
}

// kShadow: 0 none, 1 fp32 copy, 2 bf16 copy (round to nearest even).
template <bool kGradBf16, int kShadow>
__global__ __launch_bounds__(256) void k_adamw(float *__restrict__ theta, const void *__restrict__ grad,
                                                float *__restrict__ m1, float *__restrict__ m2,
                                                void *__restrict__ shadow, int64_t numel, AdamCoef c) {
  const int64_t quads = numel >> 2;
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < quads; q += (int64_t)gridDim.x * 256) {
    float4 th = reinterpret_cast<float4 *>(theta)[q];
    float4 a = reinterpret_cast<float4 *>(m1)[q];
    float4 v = reinterpret_cast<float4 *>(m2)[q];
    float g[4];
    if constexpr (kGradBf16) {
      const uint2 w = reinterpret_cast<const uint2 *>(grad)[q];
      g[0] = bf16_lo(w.x); g[1] = bf16_hi(w.x); g[2] = bf16_lo(w.y); g[3] = bf16_hi(w.y);
    } else {
      const float4 w = reinterpret_cast<const float4 *>(grad)[q];
      g[0] = w.x; g[1] = w.y; g[2] = w.z; g[3] = w.w;
    }
    adam_one(th.x, g[0], a.x, v.x, c);
    adam_one(th.y, g[1], a.y, v.y, c);
    adam_one(th.z, g[2], a.z, v.z, c);
    adam_one(th.w, g[3], a.w, v.w, c);
    reinterpret_cast<float4 *>(theta)[q] = th;
    reinterpret_cast<float4 *>(m1)[q] = a;
    reinterpret_cast<float4 *>(m2)[q] = v;
    if constexpr (kShadow == 1) reinterpret_cast<float4 *>(shadow)[q] = th;
    if constexpr (kShadow == 2)
      reinterpret_cast<uint2 *>(shadow)[q] = make_uint2(pack_bf16x2(th.x, th.y), pack_bf16x2(th.z, th.w));
  }
  if (blockIdx.x == 0 && threadIdx.x < (numel & 3)) {
    const int64_t i = quads * 4 + threadIdx.x;
    const float g = kGradBf16 ? bf16_to_f32(reinterpret_cast<const uint16_t *>(grad)[i])
                              : reinterpret_cast<const float *>(grad)[i];
    float t = theta[i], a = m1[i], v = m2[i];
    adam_one(t, g, a, v, c);
    theta[i] = t; m1[i] = a; m2[i] = v;
    if constexpr (kShadow == 1) reinterpret_cast<float *>(shadow)[i] = t;
    if constexpr (kShadow == 2) reinterpret_cast<uint16_t *>(shadow)[i] = (uint16_t)f32_to_bf16(t);
  }
}

template <bool kGradBf16>
static void adamw_dispatch(int shadow_kind, float *theta, const void *grad, float *m1, float *m2, void *shadow,
                           int64_t numel, const AdamCoef &c, int grid, hipStream_t st) {
  if (shadow_kind == 0) k_adamw<kGradBf16, 0><<<grid, 256, 0, st>>>(theta, grad, m1, m2, shadow, numel, c);
  else if (shadow_kind == 1) k_adamw<kGradBf16, 1><<<grid, 256, 0, st>>>(theta, grad, m1, m2, shadow, numel, c);
  else k_adamw<kGradBf16, 2><<<grid, 256, 0, st>>>(theta, grad, m1, m2, shadow, numel, c);
}

hipError_t launch_adamw(float *theta, const void *grad, bool grad_bf16, float *m1, float *m2, void *shadow,
                        int shadow_kind, int64_t numel, float lr, float beta1, float beta2, float eps,
                        float weight_decay, int step, hipStream_t st) {
  AdamCoef c;
  c.lr = lr; c.b1 = beta1; c.b2 = beta2; c.eps = eps;
  c.decay = (float)((double)lr * (double)weight_decay);
  c.c1 = (float)(1.0 / (1.0 - std::pow((double)beta1, (double)step)));
  c.c2 = (float)(1.0 / (1.0 - std::pow((double)beta2, (double)step)));
  int64_t blocks = ((numel >> 2) + 255) / 256;
  // a few waves of blocks per CU are enough to saturate HBM; the loop strides the rest
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  if (grad_bf16) adamw_dispatch<true>(shadow_kind, theta, grad, m1, m2, shadow, numel, c, (int)blocks, st);
  else adamw_dispatch<false>(shadow_kind, theta, grad, m1, m2, shadow, numel, c, (int)blocks, st);
  return hipGetLastError();
}

}  // namespace lcvq
