// C ABI of the LC-VQ linear layer: argument validation, workspace layout and
// the launch sequence of each call.  Every check runs on the host before the
// first launch, so a rejected call enqueues nothing.
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <mutex>
#include <utility>
#include <vector>

#include "lcvq.h"
#include "lcvq_prep.hpp"

namespace {

thread_local char g_err[512];

lcvq_status_t fail(lcvq_status_t s, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}
lcvq_status_t ok() {
  g_err[0] = 0;
  return LCVQ_OK;
}
lcvq_status_t hip_fail(hipError_t e, const char *what) {
  return fail(LCVQ_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }
// quantiser of the code domain: codes = clip(round(Z), 0, 3), gradient factor 1
constexpr lcvq::Quantizer kCodeDomain{0, 1.0f, 0.0f};
size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }

// Largest row length of an operand streamed through the 256-row tiles with
// 32-bit buffer offsets (256 rows * ld * 4 bytes must stay below 2^31).
constexpr int64_t kMaxLd = (int64_t)1 << 21;
// Most tokens of one layer call: the weight-gradient operands of eight 32-row
// slabs take 8 * (tokens / 64) * 4 KiB, which must stay below the 2^31 bytes a
// buffer resource addresses (tokens padded to 256, at most 2^22 - 256).
constexpr int64_t kMaxTokens = ((int64_t)1 << 22) - 256;

struct FwdLayout {
  size_t xp, s, frag, total;
  int64_t Np, ldp;
};
struct BwdLayout {
  size_t rs, frag, xt, dyt, mask, map, total;
};

FwdLayout fwd_layout(int64_t N, int64_t m, int64_t n, bool bf16) {
  FwdLayout L{};
  if (bf16) {
    // K padded to an even number of 64-wide steps (the product loop takes two per trip)
    L.Np = lcvq::round_up(N, 256);
    L.ldp = lcvq::round_up(n, 128);
    // s is held as one partial row of Np floats per K chunk of the transform
    const size_t xp = (size_t)L.Np * L.ldp * 2, s = (size_t)lcvq::act_chunks(L.ldp) * L.Np * 4;
    const size_t frag = (size_t)(lcvq::round_up(m, 256) / 32) * (L.ldp / 64) * 1024;
    L.xp = 0;
    L.s = up256(xp);
    L.frag = L.s + up256(s);
    L.total = L.frag + up256(frag);
  } else {
    L.Np = N;
    L.ldp = n;
    L.xp = 0;
    L.s = up256((size_t)N * n * 4);
    L.frag = L.s + up256((size_t)N * 4);
    L.total = L.frag;
  }
  return L;
}

BwdLayout bwd_layout(int64_t N, int64_t m, int64_t n, bool bf16) {
  BwdLayout L{};
  L.rs = 0;
  if (bf16) {
    // partial row sums of dY; codes in the input-gradient operand layout
    // (K = out-features padded to 128; that product reads dY in place); X' and
    // dY in the token-K fragment layout (features padded to 256); tokens padded
    // to 256 throughout
    const size_t Nt = (size_t)lcvq::bwd_tokens(N);
    const size_t rs = up256((size_t)lcvq::rowsum_parts(m) * Nt * 4);
    const size_t frag = (size_t)(lcvq::round_up(n, 256) / 32) * (lcvq::round_up(m, 128) / 64) * 1024;
    L.frag = rs;
    L.xt = L.frag + up256(frag);
    L.dyt = L.xt + up256((size_t)lcvq::round_up(n, 256) * Nt * 2);
    // straight-through mask of Z, one bit per element (rows of whole 64-bit words)
    L.mask = L.dyt + up256((size_t)lcvq::round_up(m, 256) * Nt * 2);
    // the map gradients' per-block partial sums (d d + d <= 72 entries)
    L.map = L.mask + up256((size_t)lcvq::mask_bytes(m, n));
    L.total = L.map + up256((size_t)lcvq::map_rows(N, n) * 72 * 4);
  } else {
    L.frag = L.xt = L.dyt = L.mask = L.map = L.total = up256((size_t)N * 4);
  }
  return L;
}

// The training pair's saved state (bf16): what the backward prepass would
// otherwise rebuild from Z and X -- the codes in the input-gradient operand
// layout, X' in the weight-gradient operand layout, and both straight-through
// masks -- in the layouts of BwdLayout.
struct SavedLayout {
  size_t frag_t, xt, mask_r, mask_l, total;
};
SavedLayout saved_layout(int64_t N, int64_t m, int64_t n) {
  SavedLayout L{};
  const size_t Nt = (size_t)lcvq::bwd_tokens(N);
  const size_t mask = (size_t)lcvq::mask_bytes(m, n);
  L.frag_t = 0;
  L.xt = up256((size_t)(lcvq::round_up(n, 256) / 32) * (lcvq::round_up(m, 128) / 64) * 1024);
  L.mask_r = L.xt + up256((size_t)lcvq::round_up(n, 256) * Nt * 2);
  L.mask_l = L.mask_r + up256(mask);
  L.total = L.mask_l + up256(mask);
  return L;
}

// Layer output from packed codes: X' of 16 tokens, partial s, split-K
// partials of the product and its tile counters.
struct PackedLayout {
  size_t xq, sp, part, counters, total;
};
PackedLayout packed_layout(int64_t m, int64_t n) {
  const lcvq::PackedPlan p = lcvq::packed_plan(m, n);
  PackedLayout L{};
  L.xq = 0;
  L.sp = up256((size_t)16 * p.nP * 2);
  L.part = L.sp + up256((size_t)p.nchunks * 16 * 4);
  L.counters = L.part + up256(p.KS > 1 ? (size_t)p.row_tiles * p.KS * 16 * 64 * 4 : 0);
  L.total = L.counters + up256((size_t)p.row_tiles * 4);
  return L;
}

// ---- per-kernel event timing (instrumentation, off by default) ------------
struct Timer {
  std::atomic<uint32_t> mask{0};
  std::mutex mu;
  std::vector<hipEvent_t> pool;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> rec[LCVQ_K_COUNT];
  hipEvent_t get() {  // caller holds mu
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    // timing only: no system-scope fence (it would write back and invalidate the
    // caches at every record and slow the launches being timed)
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    return e;
  }
};
Timer g_timer;

// Brackets one launch with start/stop events when its kernel is being timed.
struct Timed {
  int k;
  hipStream_t st;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  Timed(int kernel, hipStream_t s) : k(kernel), st(s) {
    if (!(g_timer.mask.load(std::memory_order_relaxed) & (1u << k))) return;
    std::lock_guard<std::mutex> lock(g_timer.mu);
    e0 = g_timer.get();
    e1 = g_timer.get();
    if (e0 && e1) hipEventRecord(e0, st);
  }
  hipError_t done(hipError_t e) {
    if (e0 && e1) {
      hipEventRecord(e1, st);
      std::lock_guard<std::mutex> lock(g_timer.mu);
      g_timer.rec[k].emplace_back(e0, e1);
    }
    return e;
  }
};

// Zero-fill without hipMemsetAsync (safe to capture in a graph).
__global__ void k_fill_zero(uint32_t *p, int64_t words) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < words; i += (int64_t)gridDim.x * 256) p[i] = 0u;
}
hipError_t fill_zero(void *p, size_t bytes, hipStream_t st) {
  if (p == nullptr || bytes == 0) return hipSuccess;
  const int64_t words = (int64_t)(bytes / 4);
  int64_t g = (words + 255) / 256;
  if (g > 65536) g = 65536;
  if (g < 1) g = 1;
  Timed tm(LCVQ_K_FILL, st);
  k_fill_zero<<<(unsigned)g, 256, 0, st>>>((uint32_t *)p, words);
  return tm.done(hipGetLastError());
}

lcvq_status_t check_common(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype) {
  if (N < 0 || m < 0 || n < 0) return fail(LCVQ_EINVAL, "negative size (N=%lld m=%lld n=%lld)", (long long)N, (long long)m, (long long)n);
  if (d != 4 && d != 8) return fail(LCVQ_EUNSUPPORTED, "group size d=%d (supported: 4, 8)", d);
  if (n % d != 0) return fail(LCVQ_EINVAL, "n=%lld is not a multiple of d=%d", (long long)n, d);
  if (dtype != LCVQ_F32 && dtype != LCVQ_BF16) return fail(LCVQ_EINVAL, "dtype=%d", dtype);
  if (N > kMaxTokens) return fail(LCVQ_EUNSUPPORTED, "N=%lld tokens (at most %lld per call)", (long long)N, (long long)kMaxTokens);
  if (dtype == LCVQ_BF16) {
    if (m % 8 != 0 || n % 8 != 0)
      return fail(LCVQ_EUNSUPPORTED, "bf16 path needs m and n multiples of 8 (m=%lld n=%lld)", (long long)m, (long long)n);
    if (m >= kMaxLd || n >= kMaxLd) return fail(LCVQ_EUNSUPPORTED, "m or n above %lld", (long long)kMaxLd);
  }
  return LCVQ_OK;
}

}  // namespace

extern "C" {

const char *lcvq_status_string(lcvq_status_t s) {
  switch (s) {
    case LCVQ_OK: return "ok";
    case LCVQ_EINVAL: return "invalid argument";
    case LCVQ_EUNSUPPORTED: return "unsupported configuration";
    case LCVQ_EALIGN: return "pointer not 16-byte aligned";
    case LCVQ_EWORKSPACE: return "workspace too small";
    case LCVQ_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char *lcvq_last_error(void) { return g_err; }

lcvq_status_t lcvq_timer_enable(uint32_t mask) {
  if (mask >> LCVQ_K_COUNT) return fail(LCVQ_EINVAL, "timer mask 0x%x has unknown kernel bits", mask);
  g_timer.mask.store(mask);
  if (mask == 0) {
    std::lock_guard<std::mutex> lock(g_timer.mu);
    for (auto &v : g_timer.rec) {
      for (auto &p : v) {
        hipEventSynchronize(p.second);
        g_timer.pool.push_back(p.first);
        g_timer.pool.push_back(p.second);
      }
      v.clear();
    }
  }
  return ok();
}

lcvq_status_t lcvq_timer_read(int32_t kernel, double *total_ms, int64_t *launches) {
  if (kernel < 0 || kernel >= LCVQ_K_COUNT || total_ms == nullptr || launches == nullptr)
    return fail(LCVQ_EINVAL, "timer_read(kernel=%d)", kernel);
  std::vector<std::pair<hipEvent_t, hipEvent_t>> recs;
  {
    std::lock_guard<std::mutex> lock(g_timer.mu);
    recs.swap(g_timer.rec[kernel]);
  }
  double tot = 0.0;
  hipError_t err = hipSuccess;
  for (auto &p : recs) {
    float ms = 0.0f;
    hipError_t e = hipEventSynchronize(p.second);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.first, p.second);
    if (e != hipSuccess && err == hipSuccess) err = e;
    tot += ms;
  }
  {
    std::lock_guard<std::mutex> lock(g_timer.mu);
    for (auto &p : recs) {
      g_timer.pool.push_back(p.first);
      g_timer.pool.push_back(p.second);
    }
  }
  *total_ms = tot;
  *launches = (int64_t)recs.size();
  return err == hipSuccess ? ok() : hip_fail(err, "timer events");
}

size_t lcvq_workspace_bytes(int32_t op, int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype) {
  if (N < 0 || m < 0 || n < 0 || (d != 4 && d != 8) || (dtype != LCVQ_F32 && dtype != LCVQ_BF16)) return 0;
  const bool bf16 = dtype == LCVQ_BF16;
  if (op == LCVQ_OP_FWD) return fwd_layout(N, m, n, bf16).total;
  if (op == LCVQ_OP_BWD) return bwd_layout(N, m, n, bf16).total;
  if (op == LCVQ_OP_FWD_PACKED) return bf16 ? packed_layout(m, n).total : 0;
  return 0;
}

lcvq_status_t lcvq_pack2bit(const void *src, int32_t src_kind, int32_t src_dtype, int64_t m, int64_t n,
                            uint8_t *packed, void *stream) {
  if (m < 0 || n < 0) return fail(LCVQ_EINVAL, "negative size");
  if (n % 4 != 0) return fail(LCVQ_EINVAL, "n=%lld is not a multiple of 4", (long long)n);
  if (src_kind != LCVQ_SRC_LATENT && src_kind != LCVQ_SRC_CODES_U8)
    return fail(LCVQ_EINVAL, "src_kind=%d (pack takes LATENT or CODES_U8)", src_kind);
  if (src_kind == LCVQ_SRC_LATENT && src_dtype != LCVQ_F32 && src_dtype != LCVQ_BF16)
    return fail(LCVQ_EINVAL, "src_dtype=%d", src_dtype);
  if (m == 0 || n == 0) return ok();
  if (src == nullptr || packed == nullptr) return fail(LCVQ_EINVAL, "null pointer");
  if (!aligned16(src) || !aligned16(packed)) return fail(LCVQ_EALIGN, "src/packed must be 16-byte aligned");
  Timed tm(LCVQ_K_PACK, (hipStream_t)stream);
  hipError_t e = tm.done(lcvq::launch_pack2bit(src, src_kind, src_dtype == LCVQ_BF16, m, n, packed, kCodeDomain,
                                               (hipStream_t)stream));
  return e == hipSuccess ? ok() : hip_fail(e, "pack2bit launch");
}

lcvq_status_t lcvq_adamw_step(float *theta, const void *grad, int32_t grad_dtype, float *m1, float *m2,
                              void *shadow, int32_t shadow_dtype, int64_t numel, float lr, float beta1,
                              float beta2, float eps, float weight_decay, int32_t step, void *stream) {
  if (numel < 0) return fail(LCVQ_EINVAL, "negative numel");
  if (grad_dtype != LCVQ_F32 && grad_dtype != LCVQ_BF16) return fail(LCVQ_EINVAL, "grad_dtype=%d", grad_dtype);
  if (shadow != nullptr && shadow_dtype != LCVQ_F32 && shadow_dtype != LCVQ_BF16)
    return fail(LCVQ_EINVAL, "shadow_dtype=%d", shadow_dtype);
  if (step < 1) return fail(LCVQ_EINVAL, "step=%d (1-based)", step);
  if (!(beta1 >= 0.0f && beta1 < 1.0f) || !(beta2 >= 0.0f && beta2 < 1.0f) || !(eps > 0.0f) || !(lr >= 0.0f) ||
      !(weight_decay >= 0.0f))
    return fail(LCVQ_EINVAL, "hyper-parameters out of range");
  if (numel == 0) return ok();
  if (theta == nullptr || grad == nullptr || m1 == nullptr || m2 == nullptr) return fail(LCVQ_EINVAL, "null pointer");
  if (!aligned16(theta) || !aligned16(grad) || !aligned16(m1) || !aligned16(m2) || (shadow && !aligned16(shadow)))
    return fail(LCVQ_EALIGN, "theta/grad/m1/m2/shadow must be 16-byte aligned");
  const int shadow_kind = shadow == nullptr ? 0 : (shadow_dtype == LCVQ_F32 ? 1 : 2);
  Timed tm(LCVQ_K_ADAM, (hipStream_t)stream);
  hipError_t e = tm.done(lcvq::launch_adamw(theta, grad, grad_dtype == LCVQ_BF16, m1, m2, shadow, shadow_kind, numel,
                                            lr, beta1, beta2, eps, weight_decay, step, (hipStream_t)stream));
  return e == hipSuccess ? ok() : hip_fail(e, "adamw launch");
}

lcvq_status_t lcvq_encode(int64_t m, int64_t n, int32_t d, const void *W, int32_t w_dtype, const float *A,
                          const float *b, uint8_t *codes_out, uint8_t *packed_out, void *stream) {
  if (m < 0 || n < 0) return fail(LCVQ_EINVAL, "negative size");
  if (d != 4 && d != 8) return fail(LCVQ_EUNSUPPORTED, "d=%d (4 or 8)", d);
  if (n % d != 0) return fail(LCVQ_EINVAL, "n=%lld is not a multiple of d=%d", (long long)n, d);
  if (w_dtype != LCVQ_F32 && w_dtype != LCVQ_BF16) return fail(LCVQ_EINVAL, "w_dtype=%d", w_dtype);
  if (codes_out == nullptr && packed_out == nullptr) return fail(LCVQ_EINVAL, "no output requested");
  if (m == 0 || n == 0) return ok();
  if (W == nullptr || A == nullptr || b == nullptr) return fail(LCVQ_EINVAL, "null required pointer (W, A, b)");
  if (!aligned16(W) || (codes_out && !aligned16(codes_out)) || (packed_out && !aligned16(packed_out)))
    return fail(LCVQ_EALIGN, "W, codes_out and packed_out must be 16-byte aligned");
  Timed tm(LCVQ_K_ENCODE, (hipStream_t)stream);
  hipError_t e = tm.done(lcvq::launch_encode(W, w_dtype == LCVQ_BF16, m, n, d, A, b, codes_out, packed_out,
                                             (hipStream_t)stream));
  return e == hipSuccess ? ok() : hip_fail(e, "encode launch");
}

lcvq_status_t lcvq_dequant(int64_t m, int64_t n, int32_t d, int32_t src_kind, int32_t src_dtype,
                           const void *src, const float *A, const float *b, void *W_hat, int32_t out_dtype,
                           void *stream) {
  if (m < 0 || n < 0) return fail(LCVQ_EINVAL, "negative size");
  if (d != 4 && d != 8) return fail(LCVQ_EUNSUPPORTED, "group size d=%d (supported: 4, 8)", d);
  if (n % d != 0) return fail(LCVQ_EINVAL, "n=%lld is not a multiple of d=%d", (long long)n, d);
  if (src_kind < LCVQ_SRC_LATENT || src_kind > LCVQ_SRC_PACKED2) return fail(LCVQ_EINVAL, "src_kind=%d", src_kind);
  if (src_kind == LCVQ_SRC_LATENT && src_dtype != LCVQ_F32 && src_dtype != LCVQ_BF16)
    return fail(LCVQ_EINVAL, "src_dtype=%d", src_dtype);
  if (out_dtype != LCVQ_F32 && out_dtype != LCVQ_BF16) return fail(LCVQ_EINVAL, "out_dtype=%d", out_dtype);
  if (m == 0 || n == 0) return ok();
  if (src == nullptr || A == nullptr || b == nullptr || W_hat == nullptr) return fail(LCVQ_EINVAL, "null pointer");
  if (!aligned16(src) || !aligned16(W_hat)) return fail(LCVQ_EALIGN, "src/W_hat must be 16-byte aligned");
  Timed tm(LCVQ_K_DEQUANT, (hipStream_t)stream);
  hipError_t e = tm.done(lcvq::launch_dequant(src, src_kind, src_dtype == LCVQ_BF16, m, n, d, A, b, W_hat,
                                              out_dtype == LCVQ_BF16, (hipStream_t)stream));
  return e == hipSuccess ? ok() : hip_fail(e, "dequant launch");
}

// eq. xavier_preprocess (Sec. 3.4) for b = 2 bits: a = sqrt(6 / (m + n)),
// s' = 2a / (2^b - 1), t = (2^b - 1) / 2; evaluated in double, rounded to fp32 once.
static bool xavier_scale(int64_t m, int64_t n, double *sp, double *t) {
  if (m <= 0 || n <= 0) return false;
  const double a = std::sqrt(6.0 / ((double)m + (double)n));
  *sp = 2.0 * a / (double)lcvq::kMaxCode;
  *t = (double)lcvq::kMaxCode / 2.0;
  return true;
}

lcvq_status_t lcvq_xavier_quantizer(int64_t m, int64_t n, float *q_scale, float *q_shift) {
  double sp, t;
  if (!xavier_scale(m, n, &sp, &t)) return fail(LCVQ_EINVAL, "m=%lld n=%lld (need m, n > 0)", (long long)m, (long long)n);
  if (q_scale == nullptr || q_shift == nullptr) return fail(LCVQ_EINVAL, "null output pointer");
  *q_scale = (float)(1.0 / sp);
  *q_shift = (float)t;
  return ok();
}

lcvq_status_t lcvq_xavier_init(int64_t m, int64_t n, int32_t src_kind, const void *codes, void *W_p,
                               int32_t out_dtype, void *stream) {
  double sp, t;
  if (!xavier_scale(m, n, &sp, &t)) return fail(LCVQ_EINVAL, "m=%lld n=%lld (need m, n > 0)", (long long)m, (long long)n);
  if (src_kind != LCVQ_SRC_CODES_U8 && src_kind != LCVQ_SRC_PACKED2)
    return fail(LCVQ_EINVAL, "src_kind=%d (CODES_U8 or PACKED2)", src_kind);
  if (n % 4 != 0) return fail(LCVQ_EINVAL, "n=%lld is not a multiple of 4", (long long)n);
  if (out_dtype != LCVQ_F32 && out_dtype != LCVQ_BF16) return fail(LCVQ_EINVAL, "out_dtype=%d", out_dtype);
  if (codes == nullptr || W_p == nullptr) return fail(LCVQ_EINVAL, "null pointer");
  if (!aligned16(codes) || !aligned16(W_p)) return fail(LCVQ_EALIGN, "codes/W_p must be 16-byte aligned");
  Timed tm(LCVQ_K_DEQUANT, (hipStream_t)stream);
  hipError_t e = tm.done(lcvq::launch_decode_scalar(codes, src_kind, m * n, (float)sp, (float)(-sp * t), W_p,
                                                    out_dtype == LCVQ_BF16, (hipStream_t)stream));
  return e == hipSuccess ? ok() : hip_fail(e, "xavier init launch");
}

}  // extern "C"

// Both forward entry points: `qz` is the quantiser domain (Sec. 3.4).
static lcvq_status_t linear_fwd(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype, const void *Z,
                                const lcvq::Quantizer &qz, const float *A, const float *b, const void *X, void *Y,
                                uint8_t *packed_codes_out, void *workspace, size_t workspace_bytes, void *stream,
                                void *saved = nullptr, size_t saved_bytes = 0, bool want_saved = false) {
  lcvq_status_t s = check_common(N, m, n, d, dtype);
  if (s != LCVQ_OK) return s;
  const bool bf16 = dtype == LCVQ_BF16;
  const size_t es = bf16 ? 2 : 4;
  hipStream_t st = (hipStream_t)stream;
  if (N == 0 || m == 0 || n == 0) {
    // Y = X W_hat^T is an N x m matrix of zeros when n == 0; codes exist only if m*n > 0.
    if (N > 0 && m > 0) {
      if (Y == nullptr) return fail(LCVQ_EINVAL, "null Y");
      if (!aligned16(Y)) return fail(LCVQ_EALIGN, "Y must be 16-byte aligned");
      hipError_t e = fill_zero(Y, (size_t)N * m * es, st);
      if (e != hipSuccess) return hip_fail(e, "zero fill");
    }
    if (m > 0 && n > 0 && packed_codes_out != nullptr) {
      if (Z == nullptr) return fail(LCVQ_EINVAL, "null Z");
      if (!aligned16(Z) || !aligned16(packed_codes_out)) return fail(LCVQ_EALIGN, "Z and packed_codes_out must be 16-byte aligned");
      Timed tm(LCVQ_K_PACK, st);
      hipError_t e = tm.done(lcvq::launch_pack2bit(Z, LCVQ_SRC_LATENT, bf16, m, n, packed_codes_out, qz, st));
      if (e != hipSuccess) return hip_fail(e, "pack launch");
    }
    return ok();
  }
  if (Z == nullptr || A == nullptr || b == nullptr || X == nullptr || Y == nullptr)
    return fail(LCVQ_EINVAL, "null required pointer (Z, A, b, X, Y)");
  if (!aligned16(Z) || !aligned16(X) || !aligned16(Y) || (packed_codes_out && !aligned16(packed_codes_out)) ||
      !aligned16(workspace))
    return fail(LCVQ_EALIGN, "Z, X, Y, packed_codes_out and workspace must be 16-byte aligned");
  const FwdLayout L = fwd_layout(N, m, n, bf16);
  if (workspace == nullptr || workspace_bytes < L.total)
    return fail(LCVQ_EWORKSPACE, "workspace %zu bytes, need %zu", workspace_bytes, L.total);
  lcvq::FwdSave save{};
  if (want_saved && bf16) {
    const SavedLayout S = saved_layout(N, m, n);
    if (saved == nullptr || saved_bytes < S.total)
      return fail(LCVQ_EWORKSPACE, "saved state %zu bytes, need %zu", saved_bytes, S.total);
    if (!aligned16(saved)) return fail(LCVQ_EALIGN, "saved state must be 16-byte aligned");
    char *sv = (char *)saved;
    save = lcvq::FwdSave{(uint32_t *)(sv + S.frag_t), (uint64_t *)(sv + S.mask_r), (uint64_t *)(sv + S.mask_l),
                         (uint16_t *)(sv + S.xt)};
  }
  char *ws = (char *)workspace;
  float *svec = (float *)(ws + L.s);
  hipError_t e;
  if (bf16) {
    uint32_t *frag = (uint32_t *)(ws + L.frag);
    {
      Timed tm(LCVQ_K_FWD_PREP, st);
      e = tm.done(lcvq::launch_fwd_prep_bf16((const uint16_t *)Z, m, n, qz, frag, packed_codes_out, (const uint16_t *)X,
                                             N, L.Np, L.ldp, d, A, b, (uint16_t *)(ws + L.xp), svec,
                                             want_saved ? &save : nullptr, st));
    }
    if (e != hipSuccess) return hip_fail(e, "forward prepass launch");
    { Timed tm(LCVQ_K_FWD, st); e = tm.done(lcvq::launch_fwd_bf16(frag, (const uint16_t *)(ws + L.xp), L.ldp, svec, (uint16_t *)Y, N, m, n, st)); }
    if (e != hipSuccess) return hip_fail(e, "forward product launch");
  } else {
    { Timed tm(LCVQ_K_FWD_PREP, st); e = tm.done(lcvq::launch_act_transform(X, false, N, N, n, d, A, b, ws + L.xp, n, svec, st)); }
    if (e != hipSuccess) return hip_fail(e, "activation transform launch");
    {
      Timed tm(LCVQ_K_FWD, st);
      e = tm.done(lcvq::launch_fwd_f32((const float *)Z, qz, (const float *)(ws + L.xp), svec, (float *)Y, N, m, n, st));
    }
    if (e != hipSuccess) return hip_fail(e, "forward product launch");
    if (packed_codes_out != nullptr) {
      Timed tm(LCVQ_K_PACK, st);
      e = tm.done(lcvq::launch_pack2bit(Z, LCVQ_SRC_LATENT, false, m, n, packed_codes_out, qz, st));
      if (e != hipSuccess) return hip_fail(e, "pack launch");
    }
  }
  return ok();
}

// The quantiser of the `_ex` entry points: (1, 0) is the code domain itself.
static lcvq_status_t make_quantizer(float q_scale, float q_shift, lcvq::Quantizer *qz) {
  if (!std::isfinite(q_scale) || !std::isfinite(q_shift) || q_scale == 0.0f)
    return fail(LCVQ_EINVAL, "quantiser scale=%g shift=%g (need finite values, scale != 0)", (double)q_scale,
                (double)q_shift);
  *qz = (q_scale == 1.0f && q_shift == 0.0f) ? kCodeDomain : lcvq::Quantizer{1, q_scale, q_shift};
  return LCVQ_OK;
}

extern "C" {

lcvq_status_t lcvq_linear_fwd(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype, const void *Z,
                              const float *A, const float *b, const void *X, void *Y, uint8_t *packed_codes_out,
                              void *workspace, size_t workspace_bytes, void *stream) {
  return linear_fwd(N, m, n, d, dtype, Z, kCodeDomain, A, b, X, Y, packed_codes_out, workspace, workspace_bytes,
                    stream);
}

lcvq_status_t lcvq_linear_fwd_ex(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype, const void *Z,
                                 float q_scale, float q_shift, const float *A, const float *b, const void *X, void *Y,
                                 uint8_t *packed_codes_out, void *workspace, size_t workspace_bytes, void *stream) {
  lcvq::Quantizer qz;
  const lcvq_status_t s = make_quantizer(q_scale, q_shift, &qz);
  if (s != LCVQ_OK) return s;
  return linear_fwd(N, m, n, d, dtype, Z, qz, A, b, X, Y, packed_codes_out, workspace, workspace_bytes, stream);
}

lcvq_status_t lcvq_linear_fwd_packed(int64_t N, int64_t m, int64_t n, int32_t d, const uint8_t *packed,
                                     const float *A, const float *b, const void *X, void *Y, int32_t y_dtype,
                                     void *workspace, size_t workspace_bytes, void *stream) {
  lcvq_status_t s = check_common(N, m, n, d, LCVQ_BF16);
  if (s != LCVQ_OK) return s;
  if (n % 64 != 0) return fail(LCVQ_EUNSUPPORTED, "packed forward needs n %% 64 == 0 (n=%lld)", (long long)n);
  if (y_dtype != LCVQ_F32 && y_dtype != LCVQ_BF16) return fail(LCVQ_EINVAL, "y_dtype=%d", y_dtype);
  const size_t ys = y_dtype == LCVQ_BF16 ? 2 : 4;
  hipStream_t st = (hipStream_t)stream;
  hipError_t e;
  if (N == 0 || m == 0) return ok();
  if (Y == nullptr) return fail(LCVQ_EINVAL, "null Y");
  if (!aligned16(Y)) return fail(LCVQ_EALIGN, "Y must be 16-byte aligned");
  if (n == 0) {  // empty sums: Y = 0
    if ((e = fill_zero(Y, (size_t)N * m * ys, st)) != hipSuccess) return hip_fail(e, "zero fill");
    return ok();
  }
  if (packed == nullptr || A == nullptr || b == nullptr || X == nullptr)
    return fail(LCVQ_EINVAL, "null required pointer (packed, A, b, X)");
  if (!aligned16(packed) || !aligned16(X) || !aligned16(workspace))
    return fail(LCVQ_EALIGN, "packed, X and workspace must be 16-byte aligned");
  const PackedLayout L = packed_layout(m, n);
  if (workspace == nullptr || workspace_bytes < L.total)
    return fail(LCVQ_EWORKSPACE, "workspace %zu bytes, need %zu", workspace_bytes, L.total);
  char *ws = (char *)workspace;
  uint16_t *xq = (uint16_t *)(ws + L.xq);
  float *sp = (float *)(ws + L.sp), *part = (float *)(ws + L.part);
  int *counters = (int *)(ws + L.counters);
  for (int64_t t0 = 0; t0 < N; t0 += 16) {
    const int Nc = (int)std::min<int64_t>(16, N - t0);
    if (lcvq::packed_fused(m, n, Nc)) {  // the product block computes its own X'' and s
      Timed tm(LCVQ_K_PACKED, st);
      e = tm.done(lcvq::launch_packed_fused(packed, m, n, (const uint16_t *)X + t0 * n, Nc, d, A, b,
                                            (char *)Y + t0 * m * ys, y_dtype == LCVQ_BF16, st));
      if (e != hipSuccess) return hip_fail(e, "packed product launch");
      continue;
    }
    {
      Timed tm(LCVQ_K_PACKED_PREP, st);
      e = tm.done(lcvq::launch_packed_prep((const uint16_t *)X + t0 * n, Nc, m, n, d, A, b, xq, sp, counters, st));
      if (e != hipSuccess) return hip_fail(e, "packed prepass launch");
    }
    Timed tm(LCVQ_K_PACKED, st);
    e = tm.done(lcvq::launch_packed_gemv(packed, m, n, xq, sp, Nc, part, counters, (char *)Y + t0 * m * ys,
                                         y_dtype == LCVQ_BF16, st));
    if (e != hipSuccess) return hip_fail(e, "packed product launch");
  }
  return ok();
}

}  // extern "C"

// ---- scratch of the allocation-free packed forward --------------------------
// A fixed device array takes the place of the workspace argument: X'' of 16
// tokens, the partial sums of s, the split-K partial tiles and the tile
// counters (which the prepass zeroes on every call).  Each device that runs the
// call holds its own copy until the process ends; in host code `scratch` is
// only a stand-in for the symbol, so its device address is looked up once per
// device (hipGetSymbolAddress, with that device current) and only that address
// is ever passed to kernels.
static constexpr size_t kScratchBytes = (size_t)8 << 20;
static __device__ __align__(256) char scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the current device.
lcvq_status_t scratch_of_current_device(void **ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(LCVQ_EUNSUPPORTED, "device %d (at most %d devices)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (p == nullptr || ((uintptr_t)p & 255u) != 0) return fail(LCVQ_EHIP, "scratch address %p", p);
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return LCVQ_OK;
}
}  // namespace

extern "C" {

size_t lcvq_packed_scratch_bytes(void) { return kScratchBytes; }

lcvq_status_t lcvq_linear_fwd_packed_noalloc(int64_t N, int64_t m, int64_t n, int32_t d, const uint8_t *packed,
                                             const float *A, const float *b, const void *X, void *Y,
                                             int32_t y_dtype, void *stream) {
  // the size check needs no device: reject before touching the runtime
  if (m > 0 && n > 0 && m < kMaxLd && n < kMaxLd && n % 64 == 0 && packed_layout(m, n).total > kScratchBytes)
    return fail(LCVQ_EUNSUPPORTED, "m=%lld n=%lld needs %zu bytes of scratch, the static array holds %zu",
                (long long)m, (long long)n, packed_layout(m, n).total, kScratchBytes);
  void *ws = nullptr;
  if (N > 0 && m > 0 && n > 0) {
    const lcvq_status_t s = scratch_of_current_device(&ws);
    if (s != LCVQ_OK) return s;
  }
  return lcvq_linear_fwd_packed(N, m, n, d, packed, A, b, X, Y, y_dtype, ws, ws ? kScratchBytes : 0, stream);
}

}  // extern "C"

// Both backward entry points: `est` selects the estimator of the latent's gradient.
static lcvq_status_t linear_bwd(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype, const void *Z,
                                const lcvq::Quantizer &qz, const float *A, const float *b, const void *X,
                                const void *dY, int32_t mask_mode,
                                const lcvq::GradEst &est, int32_t accumulate, void *dX, void *dZ, int32_t dz_dtype,
                                float *dA, float *db, void *workspace, size_t workspace_bytes, void *stream,
                                const void *saved = nullptr, size_t saved_bytes = 0, bool use_saved = false) {
  lcvq_status_t s = check_common(N, m, n, d, dtype);
  if (s != LCVQ_OK) return s;
  if (mask_mode != LCVQ_MASK_ROUNDED && mask_mode != LCVQ_MASK_LATENT) return fail(LCVQ_EINVAL, "mask_mode=%d", mask_mode);
  if (accumulate != 0 && accumulate != 1) return fail(LCVQ_EINVAL, "accumulate=%d", accumulate);
  if ((dA == nullptr) != (db == nullptr)) return fail(LCVQ_EINVAL, "dA and db must both be given or both be NULL");
  const bool bf16 = dtype == LCVQ_BF16;
  if (dz_dtype != LCVQ_F32 && !(dz_dtype == LCVQ_BF16 && bf16))
    return fail(LCVQ_EINVAL, "dz_dtype=%d with dtype=%d", dz_dtype, dtype);
  const size_t es = bf16 ? 2 : 4, dzs = dz_dtype == LCVQ_BF16 ? 2 : 4;
  hipStream_t st = (hipStream_t)stream;
  hipError_t e;
  if (N == 0 || m == 0 || n == 0) {
    // Every product has an empty sum: dX = 0, dZ = 0, dA = db = 0 (or left as they are when accumulating).
    if (dX != nullptr && N > 0 && n > 0) {
      if (!aligned16(dX)) return fail(LCVQ_EALIGN, "dX must be 16-byte aligned");
      if ((e = fill_zero(dX, (size_t)N * n * es, st)) != hipSuccess) return hip_fail(e, "zero fill");
    }
    if (!accumulate) {
      if (dZ != nullptr && m > 0 && n > 0) {
        if (!aligned16(dZ)) return fail(LCVQ_EALIGN, "dZ must be 16-byte aligned");
        if ((e = fill_zero(dZ, (size_t)m * n * dzs, st)) != hipSuccess) return hip_fail(e, "zero fill");
      }
      if (dA != nullptr) {
        if ((e = fill_zero(dA, (size_t)d * d * 4, st)) != hipSuccess) return hip_fail(e, "zero fill");
        if ((e = fill_zero(db, (size_t)d * 4, st)) != hipSuccess) return hip_fail(e, "zero fill");
      }
    }
    return ok();
  }
  if (Z == nullptr || A == nullptr || b == nullptr || X == nullptr || dY == nullptr)
    return fail(LCVQ_EINVAL, "null required pointer (Z, A, b, X, dY)");
  if (!aligned16(Z) || !aligned16(X) || !aligned16(dY) || (dX && !aligned16(dX)) || (dZ && !aligned16(dZ)) ||
      !aligned16(workspace))
    return fail(LCVQ_EALIGN, "Z, X, dY, dX, dZ and workspace must be 16-byte aligned");
  const BwdLayout L = bwd_layout(N, m, n, bf16);
  if (workspace == nullptr || workspace_bytes < L.total)
    return fail(LCVQ_EWORKSPACE, "workspace %zu bytes, need %zu", workspace_bytes, L.total);
  char *ws = (char *)workspace;
  float *rs = (float *)(ws + L.rs);
  const bool want_map = dA != nullptr;
  const bool clear_map = want_map && !accumulate;

  if (bf16) {
    // 1. one prepass launch: codes in the input-gradient operand layout (when
    //    dX or dA/db are wanted), X' = X blockdiag(A) and dY in the
    //    weight-gradient fragments (when dZ is wanted), and the partial row sums
    //    of dY
    // 2. dZ = mask * dY^T X'    3. dX = (dY codes) A-map + rowsum(dY) b (+ the
    //    per-block partial sums of dA, db)    4. their sum into dA, db
    //    (the two products are independent; in this order the step measured
    //    slightly shorter)
    const bool run_dx = dX != nullptr || want_map;
    float *mapp = want_map ? (float *)(ws + L.map) : nullptr;
    uint32_t *frag = (uint32_t *)(ws + L.frag);
    uint16_t *xt = (uint16_t *)(ws + L.xt), *dyt = (uint16_t *)(ws + L.dyt);
    // the straight-through mask as a bitmap (the differentiable estimator reads Z itself)
    uint64_t *maskbits = dZ != nullptr && !est.dge ? (uint64_t *)(ws + L.mask) : nullptr;
    if (use_saved) {
      // codes, X' and the masks come from the forward of the training pair: the
      // prepass handles dY alone
      const SavedLayout S = saved_layout(N, m, n);
      if (saved == nullptr || saved_bytes < S.total)
        return fail(LCVQ_EWORKSPACE, "saved state %zu bytes, need %zu", saved_bytes, S.total);
      if (!aligned16(saved)) return fail(LCVQ_EALIGN, "saved state must be 16-byte aligned");
      const char *sv = (const char *)saved;
      frag = (uint32_t *)(sv + S.frag_t);
      xt = (uint16_t *)(sv + S.xt);
      if (maskbits != nullptr) maskbits = (uint64_t *)(sv + (mask_mode == LCVQ_MASK_ROUNDED ? S.mask_r : S.mask_l));
    }
    {
      // the quantise blocks run when the input-gradient product or the bitmap
      // needs them and nothing was saved
      Timed tm(LCVQ_K_BWD_PREP, st);
      e = tm.done(lcvq::launch_bwd_prep_bf16((const uint16_t *)Z, m, n, qz,
                                             !use_saved && (run_dx || maskbits) ? frag : nullptr,
                                             (const uint16_t *)X, (const uint16_t *)dY, A, d, N,
                                             dZ != nullptr && !use_saved ? xt : nullptr,
                                             dZ != nullptr ? dyt : nullptr, rs, use_saved ? nullptr : maskbits, mask_mode,
                                             st));
      if (e != hipSuccess) return hip_fail(e, "backward prepass launch");
    }
    if (dZ != nullptr) {
      Timed tm(LCVQ_K_DW, st);
      e = tm.done(lcvq::launch_dw_bf16(xt, dyt, maskbits, (const uint16_t *)Z, qz, mask_mode, est, accumulate, dZ,
                                       dz_dtype == LCVQ_BF16, N, m, n, st));
      if (e != hipSuccess) return hip_fail(e, "weight-gradient launch");
    }
    if (run_dx) {
      Timed tm(LCVQ_K_DX, st);
      e = tm.done(lcvq::launch_dx_bf16(frag, (const uint16_t *)dY, rs, A, b, d, (uint16_t *)dX, (const uint16_t *)X,
                                       mapp, N, m, n, st));
      if (e != hipSuccess) return hip_fail(e, "input-gradient launch");
    }
    if (want_map) {
      Timed tm(LCVQ_K_MAP_SUM, st);
      e = tm.done(lcvq::launch_map_combine(mapp, lcvq::map_rows(N, n), d, accumulate, dA, db, st));
      if (e != hipSuccess) return hip_fail(e, "map-gradient sum launch");
    }
    return ok();
  }

  // fp32 mode
  float *zA = clear_map ? dA : nullptr;
  float *zb = clear_map ? db : nullptr;
  if (dX != nullptr) {
    { Timed tm(LCVQ_K_BWD_PREP, st); e = tm.done(lcvq::launch_rowsum(dY, false, N, N, m, rs, zA, zb, d, st)); }
    if (e != hipSuccess) return hip_fail(e, "row-sum launch");
    zA = zb = nullptr;  // cleared by the row-sum launch
    Timed tm(LCVQ_K_DX, st);
    e = tm.done(lcvq::launch_dx_f32((const float *)Z, qz, (const float *)dY, rs, A, b, d, (float *)dX, N, m, n, st));
    if (e != hipSuccess) return hip_fail(e, "input-gradient launch");
  }
  if (zA != nullptr) {
    if ((e = fill_zero(zA, (size_t)d * d * 4, st)) != hipSuccess) return hip_fail(e, "zero fill");
    if ((e = fill_zero(zb, (size_t)d * 4, st)) != hipSuccess) return hip_fail(e, "zero fill");
  }
  if (dZ != nullptr || want_map) {
    Timed tm(LCVQ_K_DW, st);
    e = tm.done(lcvq::launch_dz_f32((const float *)X, (const float *)dY, (const float *)Z, qz, A, d, mask_mode, est,
                                    accumulate, (float *)dZ, dA, db, N, m, n, st));
    if (e != hipSuccess) return hip_fail(e, "weight-gradient launch");
  }
  return ok();
}

extern "C" {

lcvq_status_t lcvq_linear_bwd(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype, const void *Z,
                              const float *A, const float *b, const void *X, const void *dY, int32_t mask_mode,
                              int32_t accumulate, void *dX, void *dZ, int32_t dz_dtype, float *dA, float *db,
                              void *workspace, size_t workspace_bytes, void *stream) {
  return linear_bwd(N, m, n, d, dtype, Z, kCodeDomain, A, b, X, dY, mask_mode, lcvq::GradEst{0, 0.0f, 1.0f, 1.0f},
                    accumulate, dX, dZ, dz_dtype, dA, db, workspace, workspace_bytes, stream);
}

}  // extern "C"

static lcvq_status_t make_estimator(int32_t estimator, float k, float cap, lcvq::GradEst *est) {
  if (estimator == LCVQ_EST_STE) {
    *est = lcvq::GradEst{0, 0.0f, 1.0f, 1.0f};
    return LCVQ_OK;
  }
  if (estimator != LCVQ_EST_DGE) return fail(LCVQ_EINVAL, "estimator=%d", estimator);
  if (!(k >= 1.0f) || !std::isfinite(k)) return fail(LCVQ_EINVAL, "dge k=%g (need a finite k >= 1)", (double)k);
  if (!(cap > 0.0f) || !std::isfinite(cap)) return fail(LCVQ_EINVAL, "dge cap=%g (need a finite cap > 0)", (double)cap);
  *est = lcvq::GradEst{1, (float)(1.0 / (double)k - 1.0), (float)(1.0 / (double)k), cap};
  return LCVQ_OK;
}

extern "C" {

lcvq_status_t lcvq_linear_bwd_dge(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype, const void *Z,
                                  const float *A, const float *b, const void *X, const void *dY, int32_t mask_mode,
                                  float k, float cap, int32_t accumulate, void *dX, void *dZ, int32_t dz_dtype,
                                  float *dA, float *db, void *workspace, size_t workspace_bytes, void *stream) {
  lcvq::GradEst est;
  const lcvq_status_t s = make_estimator(LCVQ_EST_DGE, k, cap, &est);
  if (s != LCVQ_OK) return s;
  return linear_bwd(N, m, n, d, dtype, Z, kCodeDomain, A, b, X, dY, mask_mode, est, accumulate, dX, dZ, dz_dtype,
                    dA, db, workspace, workspace_bytes, stream);
}

size_t lcvq_saved_bytes(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype) {
  if (N < 0 || m < 0 || n < 0 || (d != 4 && d != 8) || dtype != LCVQ_BF16) return 0;
  return saved_layout(N, m, n).total;
}

lcvq_status_t lcvq_linear_fwd_train(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype, const void *Z,
                                    float q_scale, float q_shift, const float *A, const float *b, const void *X,
                                    void *Y, uint8_t *packed_codes_out, void *saved, size_t saved_bytes,
                                    void *workspace, size_t workspace_bytes, void *stream) {
  lcvq::Quantizer qz;
  const lcvq_status_t s = make_quantizer(q_scale, q_shift, &qz);
  if (s != LCVQ_OK) return s;
  return linear_fwd(N, m, n, d, dtype, Z, qz, A, b, X, Y, packed_codes_out, workspace, workspace_bytes, stream, saved,
                    saved_bytes, N > 0 && m > 0 && n > 0);
}

lcvq_status_t lcvq_linear_bwd_train(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype, const void *Z,
                                    float q_scale, float q_shift, const float *A, const float *b, const void *X,
                                    const void *dY, int32_t mask_mode, int32_t estimator, float dge_k, float dge_cap,
                                    int32_t accumulate, void *dX, void *dZ, int32_t dz_dtype, float *dA, float *db,
                                    const void *saved, size_t saved_bytes, void *workspace, size_t workspace_bytes,
                                    void *stream) {
  lcvq::Quantizer qz;
  lcvq::GradEst est;
  lcvq_status_t s = make_quantizer(q_scale, q_shift, &qz);
  if (s == LCVQ_OK) s = make_estimator(estimator, dge_k, dge_cap, &est);
  if (s != LCVQ_OK) return s;
  return linear_bwd(N, m, n, d, dtype, Z, qz, A, b, X, dY, mask_mode, est, accumulate, dX, dZ, dz_dtype, dA, db,
                    workspace, workspace_bytes, stream, saved, saved_bytes, dtype == LCVQ_BF16);
}

lcvq_status_t lcvq_linear_bwd_ex(int64_t N, int64_t m, int64_t n, int32_t d, int32_t dtype, const void *Z,
                                 float q_scale, float q_shift, const float *A, const float *b, const void *X,
                                 const void *dY, int32_t mask_mode, int32_t estimator, float dge_k, float dge_cap,
                                 int32_t accumulate, void *dX, void *dZ, int32_t dz_dtype, float *dA, float *db,
                                 void *workspace, size_t workspace_bytes, void *stream) {
  lcvq::Quantizer qz;
  lcvq::GradEst est;
  lcvq_status_t s = make_quantizer(q_scale, q_shift, &qz);
  if (s == LCVQ_OK) s = make_estimator(estimator, dge_k, dge_cap, &est);
  if (s != LCVQ_OK) return s;
  return linear_bwd(N, m, n, d, dtype, Z, qz, A, b, X, dY, mask_mode, est, accumulate, dX, dZ, dz_dtype, dA, db,
                    workspace, workspace_bytes, stream);
}

}  // extern "C"
