// Layer output straight from packed 2-bit codes, for inference with the
// compressed weight (def. forward_x, Sec. 3.2; the paper's inference kernel,
// App. A.2, fuses decode, dot products and reduction in the same spirit).
// One pass handles up to 16 tokens:
//
//   prepass : X' = X blockdiag(A) rounded to bf16, s = X b~, and the tile
//             counters of the product zeroed.  X' is stored in the product's
//             B-operand order, each value scaled by the power of two its code
//             position needs (below), and the prepass also sums those scaled
//             values per token (the offset the product subtracts).  Operand
//             fragment (j, i) of step j, sub-step i is 64 lanes x 16 bytes, so
//             each operand load of a wave reads 1 KiB of contiguous memory.
//   product : Y[t, r] = sum_c code[r, c] X'[t, c] + s[t] on the matrix cores,
//             v_mfma_f32_16x16x32_bf16 with 16 weight rows on M and 16 tokens
//             on N.  The packed codes (0.25 byte per weight) are the only
//             large stream; they are read once per pass, 16 bytes per lane.
//
// For few tokens and long rows the X' rows of a block's steps are held in LDS;
// where one block covers a whole row tile (no K split) it also computes them
// (and its share of s) from X itself, so that pass is a single launch with no
// prepass.
//
// Decoding without conversions: a 32-bit word w holds 16 codes, code i at bits
// 2i, 2i + 1.  A bf16 whose exponent field reads 1.0 and whose mantissa holds a
// code c at bits p, p + 1 has the value 1 + c 2^(p - 7); the low and high halves
// of (w & mask) | 0x3F803F80 are such values for the codes under the mask.
// Masks 0x00030003, 0x000C000C, 0x00300030 applied to w, w >> 6 and w >> 12
// reach all 16 codes at p in {0, 2, 4} (two shifts and eight and-or per word).
// With X'' = X' 2^(7 - p) (exact), sum (1 + c 2^(p-7)) X'' = sum X'' + sum c X',
// so the product subtracts the per-token sum of X''.
//
// Order of the 16 codes of a word in the two MFMA operands it feeds
// (element e of operand E / O; p = bit position):
//   E: codes 0, 8, 1, 9, 2, 10, 3, 11   p = 0, 0, 2, 2, 4, 4, 0, 0
//   O: codes 4, 12, 5, 13, 6, 14, 7, 15 p = 2, 2, 4, 4, 0, 0, 2, 2
#include "lcvq_prep.hpp"

namespace lcvq {

constexpr int kPkChunk = 4096;  // prepass columns per block (16 per thread)
constexpr int kPkRows = 64;     // product rows per block (16 per MFMA row block, four row blocks)
constexpr int kPkStep = 256;    // K columns per product step (64 bytes of codes per row)
constexpr int kMaxPairs = 6;    // fused product: (token, 256-group run) pairs per thread in the X'' fill
constexpr int kPrePairs = 2;    // .. of which loaded ahead of the first codes
constexpr int kPreChunks = 8;   // X'' chunks per thread loaded ahead of the first codes (copied product)

// ---------------------------------------------------------------- prepass --
// grid (ceil(nP / 4096), 16): block (chunk, t) transforms columns
// [4096 chunk, 4096 chunk + 4096) of token t; tokens t >= Nc and columns
// c >= n are written as zeros up to nP (a multiple of 256).  Thread tid takes
// the 16 columns c0 = 4096 chunk + 16 tid .., i.e. step j = c0 / 256, lane
// group q = (c0 / 64) % 4 and dword kk = (c0 / 16) % 4 of the product.
// One 16-column group of one token: X'[g D + k] = sum_j X[g D + j] A[j, k] is
// rounded to bf16 and scaled exactly by 2^(7 - p) for the mantissa position p
// its code takes in the product (the two operand dwords ev / od, in element
// order); s gains sum_j X[g D + j] b[j] and loses sum X'', the offset of the
// 1.0 bits of the decoded codes.
template <int D>
__device__ __forceinline__ void xpp_group(const float (&x)[16], const float *__restrict__ A,
                                          const float *__restrict__ b, float &s, u32x4 &ev, u32x4 &od) {
  float xp[16];
#pragma unroll
  for (int g = 0; g < 16 / D; ++g)
#pragma unroll
    for (int k = 0; k < D; ++k) {
      float v = 0.0f;
#pragma unroll
      for (int j = 0; j < D; ++j) v = fmaf(x[g * D + j], A[j * D + k], v);
      xp[g * D + k] = v;
      s = fmaf(x[g * D + k], b[k], s);
    }
  constexpr int kCode[16] = {0, 8, 1, 9, 2, 10, 3, 11, 4, 12, 5, 13, 6, 14, 7, 15};
  constexpr float kScale[16] = {128.f, 128.f, 32.f, 32.f, 8.f, 8.f, 128.f, 128.f,
                                32.f, 32.f, 8.f, 8.f, 128.f, 128.f, 32.f, 32.f};
  uint32_t h[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    h[e] = f32_to_bf16(xp[kCode[e]]);                           // X' rounded to bf16 ..
    const float sc = __uint_as_float(h[e] << 16) * kScale[e];   // .. then scaled exactly
    h[e] = __float_as_uint(sc) >> 16;
    s -= sc;
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    ev[e] = h[2 * e] | h[2 * e + 1] << 16;
    od[e] = h[8 + 2 * e] | h[8 + 2 * e + 1] << 16;
  }
}

// Loads the 16 columns c0 .. c0 + 15 of one token row (zeros when c0 >= n;
// n is a multiple of 64, so a group is whole or absent).
__device__ __forceinline__ void load_x16(const uint16_t *__restrict__ row, int64_t c0, int64_t n, float (&x)[16]) {
  if (c0 < n) {
    const uint4 *src = reinterpret_cast<const uint4 *>(row + c0);
    const uint4 u0 = src[0], u1 = src[1];
    const uint32_t w[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      x[2 * e] = bf16_lo(w[e]);
      x[2 * e + 1] = bf16_hi(w[e]);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 16; ++e) x[e] = 0.0f;
  }
}

template <int D>
__global__ __launch_bounds__(256) void k_packed_prep(const uint16_t *__restrict__ X, int Nc, int64_t n, int64_t nP,
                                                     const float *__restrict__ A, const float *__restrict__ b,
                                                     uint16_t *__restrict__ xq, float *__restrict__ sp,
                                                     int *__restrict__ counters, int ncounters) {
  const int tid = threadIdx.x, t = blockIdx.y;
  const int64_t c0 = (int64_t)blockIdx.x * kPkChunk + 16 * tid;
  if (blockIdx.x == 0 && blockIdx.y == 0)
    for (int i = tid; i < ncounters; i += 256) counters[i] = 0;
  float x[16];
  load_x16(X + (int64_t)t * n, t < Nc ? c0 : n, n, x);  // absent tokens: zeros
  float s = 0.0f;
  if (c0 < nP) {
    u32x4 ev, od;
    xpp_group<D>(x, A, b, s, ev, od);
    const int64_t j = c0 / kPkStep;
    const int qq = (int)((c0 / 64) % 4), kk = (int)((c0 / 16) % 4);
    u32x4 *dst = reinterpret_cast<u32x4 *>(xq);
    dst[(j * 8 + 2 * kk) * 64 + qq * 16 + t] = ev;
    dst[(j * 8 + 2 * kk + 1) * 64 + qq * 16 + t] = od;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
  __shared__ float red[4];
  if ((tid & 63) == 0) red[tid >> 6] = s;
  __syncthreads();
  if (tid == 0) sp[blockIdx.x * 16 + t] = red[0] + red[1] + red[2] + red[3];
}

// ---------------------------------------------------------------- product --
// Block (rt, ks) of KS K-splits: weight rows [64 rt, 64 rt + 64), product
// steps [ks spb, min(KT, ks spb + spb)).  Wave w takes the steps j with
// j = w mod 4, so the four waves read 256 contiguous bytes of every row
// together.  Each wave holds the four 16-row blocks of the tile, so every
// X' fragment it loads feeds four MFMAs.  The waves' partial tiles are summed
// in LDS; with KS > 1 each block stores its tile (fp32) and the last block of
// the row tile to finish (a counter the prepass zeroed) adds them up.
//
// MFMA operands (16x16x32): lane L (row or token L % 16, K group q = L / 16)
// holds, for step j and sub-step i = 2 kk + (E: 0, O: 1), eight of the codes of
// dword kk of its 16 bytes (columns 256 j + 64 q + 16 kk .. + 15, in the order
// above) and the matching eight X'' values, fragment (j, i) of the prepass.
//
// kXL (few tokens): the X'' rows of the Nc tokens for the block's steps sit
// in LDS (dynamic, 512 Nc bytes per step plus a zero chunk) and each step reads
// its fragments from there, instead of every wave loading eight mostly idle
// 1 KiB fragments per step from the L2.  kXL = 1 copies them from the prepass
// output; kXL = 2 (one block per row tile, KS = 1) computes them from X in the
// block, with the partial sums of s, so that no prepass launch is needed.
template <int kXL, int D>
__global__ __launch_bounds__(256) void k_packed_gemv(const uint8_t *__restrict__ packed, int64_t m, int64_t n, int KT,
                                                     int KS, int spb, const uint16_t *__restrict__ xq, int64_t nP,
                                                     const float *__restrict__ sp, int nchunks, int Nc,
                                                     float *__restrict__ part, int *__restrict__ counters,
                                                     void *__restrict__ Y, int y_bf16, const uint16_t *__restrict__ X,
                                                     const float *__restrict__ A, const float *__restrict__ b) {
  extern __shared__ u32x4 xl[];
  __shared__ float s_red[4][16];  // kXL = 2: offsets s per wave and token
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q = lane >> 4, tl = lane & 15;
  const int rt = (int)blockIdx.x / KS, ks = (int)blockIdx.x % KS;
  const int j0 = ks * spb, j1 = min(KT, j0 + spb);
  const int64_t ldb = n / 4;  // bytes per packed row
  const int64_t r0 = (int64_t)rt * kPkRows;
  // rows past m lie beyond the buffer: their loads give zero codes
  const __amdgpu_buffer_rsrc_t rP = make_rsrc(packed + r0 * ldb, (m - r0) * ldb);
  const __amdgpu_buffer_rsrc_t rX = make_rsrc(xq, 16 * nP * 2);

  floatx4 acc[4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) acc[rb] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
  u32x4 cw[2][4], xf[2][8];
  const int nch = (j1 - j0) * 32 * Nc;  // kXL: 16-byte chunks in LDS; chunk nch is zero
  // chunk c = ((jj * 8 + i) * 4 + q) * Nc + t holds fragment (j0 + jj, i), lane 16 q + t
  auto codes_load = [&](int buf, int j) {
    const bool live = j < j1;
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
      cw[buf][rb] = __builtin_amdgcn_raw_buffer_load_b128(
          rP, live ? (uint32_t)((16 * rb + tl) * ldb + 64 * j + 16 * q) : kOffNone, 0, 0);
  };
  auto x_load = [&](int buf, int j) {
    const bool xlive = j < j1 && tl < Nc;  // X' rows of absent tokens are zero: not loaded
    if constexpr (kXL > 0) {
      const int base = xlive ? ((j - j0) * 32 + q) * Nc + tl : nch;
      const int stride = xlive ? 4 * Nc : 0;
#pragma unroll
      for (int i = 0; i < 8; ++i) xf[buf][i] = xl[base + i * stride];
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        xf[buf][i] = __builtin_amdgcn_raw_buffer_load_b128(
            rX, xlive ? (uint32_t)(((j * 8 + i) * 64 + lane) * 16) : kOffNone, 0, 0);
    }
  };
  auto load = [&](int buf, int j) {
    codes_load(buf, j);
    x_load(buf, j);
  };
  // With X'' in LDS, the codes of the wave's first two steps are loaded before
  // the block fills those rows (after the fill's own first loads), so that
  // their latency passes during the fill; the barrier after the fill waits for
  // LDS only, not for those loads.
  int j = j0 + wave;
  if constexpr (kXL == 1) {
    auto xoff = [&](int c) {
      const int t = c % Nc, fq = c / Nc;
      return c < nch ? (uint32_t)(((j0 * 8 + (fq >> 2)) * 64 + (fq & 3) * 16 + t) * 16) : kOffNone;
    };
    u32x4 xc[kPreChunks];
#pragma unroll
    for (int ci = 0; ci < kPreChunks; ++ci)
      xc[ci] = __builtin_amdgcn_raw_buffer_load_b128(rX, xoff(tid + 256 * ci), 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    codes_load(0, j);
    codes_load(1, j + 4);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ci = 0; ci < kPreChunks; ++ci)
      if (tid + 256 * ci < nch) xl[tid + 256 * ci] = xc[ci];
    for (int c = tid + 256 * kPreChunks; c < nch; c += 256)  // (these wait behind the codes)
      xl[c] = __builtin_amdgcn_raw_buffer_load_b128(rX, xoff(c), 0, 0);
  } else if constexpr (kXL == 2) {
    // token by token, thread tid takes the 16-column groups g16 = tid + 256 k
    // (k < G) of the block's steps (step j0 + g16 / 16, lane group (g16 / 4) %
    // 4, dword g16 % 4): pair p = t G + k, at most kMaxPairs (the rows fit in
    // 48 KiB); the offsets s are summed in a fixed order (per thread, across
    // the wave, then across the four waves in the epilogue), so the result
    // does not depend on scheduling
    const int ng = (j1 - j0) * 16, G = (ng + 255) >> 8, P = Nc * G;
    const __amdgpu_buffer_rsrc_t rXr = make_rsrc(X, (int64_t)Nc * n * 2);
    auto xload = [&](int p, u32x4 (&w)[2]) {
      const int t = p < P ? p / G : 0, g16 = tid + 256 * (p - t * G);
      const int64_t c0 = (int64_t)j0 * kPkStep + 16 * g16;
      const bool in = p < P && g16 < ng && c0 < n;
      const uint32_t off = in ? (uint32_t)(((int64_t)t * n + c0) * 2) : kOffNone;
      w[0] = __builtin_amdgcn_raw_buffer_load_b128(rXr, off, 0, 0);
      w[1] = __builtin_amdgcn_raw_buffer_load_b128(rXr, in ? off + 16u : kOffNone, 0, 0);
    };
    u32x4 xr[kPrePairs][2];
#pragma unroll
    for (int p = 0; p < kPrePairs; ++p) xload(p, xr[p]);
    __builtin_amdgcn_sched_barrier(0);
    codes_load(0, j);
    codes_load(1, j + 4);
    __builtin_amdgcn_sched_barrier(0);
    float s = 0.0f;
#pragma unroll
    for (int p = 0; p < kMaxPairs; ++p) {
      if (p < P) {
        const int t = p / G, k = p - t * G, g16 = tid + 256 * k;
        u32x4 w[2];
        if (p < kPrePairs) {
          w[0] = xr[p < kPrePairs ? p : 0][0];
          w[1] = xr[p < kPrePairs ? p : 0][1];
        } else {
          xload(p, w);  // (waits behind the codes)
        }
        if (g16 < ng) {
          float x[16];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const uint32_t wd = e < 4 ? w[0][e] : w[1][e - 4];
            x[2 * e] = bf16_lo(wd);
            x[2 * e + 1] = bf16_hi(wd);
          }
          u32x4 ev, od;
          xpp_group<D>(x, A, b, s, ev, od);
          const int jj = g16 >> 4, qq = (g16 >> 2) & 3, kk = g16 & 3;
          xl[((jj * 8 + 2 * kk) * 4 + qq) * Nc + t] = ev;
          xl[((jj * 8 + 2 * kk + 1) * 4 + qq) * Nc + t] = od;
        }
        if (k == G - 1) {
#pragma unroll
          for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
          if (lane == 0) s_red[wave][t] = s;
          s = 0.0f;
        }
      }
    }
  }
  if constexpr (kXL > 0) {
    if (tid == 0) xl[nch] = u32x4{0u, 0u, 0u, 0u};
    // barrier over the LDS fill only (no wait for the codes in flight)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4));  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    x_load(0, j);
    x_load(1, j + 4);
  } else {
    load(0, j);
    __builtin_amdgcn_sched_barrier(0);
    load(1, j + 4);
  }
  __builtin_amdgcn_sched_barrier(0);
  // bf16 1.0 in both halves, held in a vector register: with the mask from a
  // scalar register each operand dword is then one v_and_or_b32 (a literal
  // would not fit that instruction and costs a separate and + or)
  uint32_t one;
  asm volatile("v_mov_b32 %0, 0x3f803f80" : "=v"(one));
  auto compute = [&](int buf) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      bf16x8 ae[4], ao[4];
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        const uint32_t w0 = cw[buf][rb][kk], w6 = w0 >> 6, w12 = w0 >> 12;
        u32x4 e, o;
        e[0] = (w0 & 0x00030003u) | one;
        e[1] = (w0 & 0x000C000Cu) | one;
        e[2] = (w0 & 0x00300030u) | one;
        e[3] = (w6 & 0x00030003u) | one;
        o[0] = (w6 & 0x000C000Cu) | one;
        o[1] = (w6 & 0x00300030u) | one;
        o[2] = (w12 & 0x00030003u) | one;
        o[3] = (w12 & 0x000C000Cu) | one;
        ae[rb] = __builtin_bit_cast(bf16x8, e);
        ao[rb] = __builtin_bit_cast(bf16x8, o);
      }
      // the four row blocks in turn, so dependent MFMAs are four apart
#pragma unroll
      for (int rb = 0; rb < 4; ++rb)
        acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ae[rb], __builtin_bit_cast(bf16x8, xf[buf][2 * kk]),
                                                          acc[rb], 0, 0, 0);
#pragma unroll
      for (int rb = 0; rb < 4; ++rb)
        acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ao[rb], __builtin_bit_cast(bf16x8, xf[buf][2 * kk + 1]),
                                                          acc[rb], 0, 0, 0);
    }
  };
  // two register buffers, the loads of a wave's step after next issued once
  // the current step's MFMAs are (the first two steps' loads are issued above)
  // (the scheduling fences keep each buffer's loads together, so the wait
  // before a step covers that step's loads only)
  for (; j < j1; j += 8) {
    compute(0);
    __builtin_amdgcn_sched_barrier(0);
    load(0, j + 8);
    __builtin_amdgcn_sched_barrier(0);
    compute(1);
    __builtin_amdgcn_sched_barrier(0);
    load(1, j + 12);
    __builtin_amdgcn_sched_barrier(0);
  }

  // ------------------------------------------------------------ epilogue
  // lane L of wave w holds rows 16 rb + 4 q + (0..3) of token tl in acc[rb]
  __shared__ floatx4 red[4][4][64];
  __shared__ int last;
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) red[wave][rb][lane] = acc[rb];
  __syncthreads();
  // thread (rb = wave, lane): rows 16 rb + 4 q + (0..3), token tl
  const int rb = wave;
  floatx4 v = red[0][rb][lane] + red[1][rb][lane] + red[2][rb][lane] + red[3][rb][lane];
  const int64_t row = r0 + 16 * rb + 4 * q;  // m is a multiple of 8: the four rows are all in or all out
  if (KS > 1) {
    // The blocks of a row tile may run on different XCDs (separate L2s).  The
    // partials are written and read with device-scope atomics, so each one is
    // performed at device scope.  Ordering: the block's partial stores precede
    // the barrier, the barrier precedes thread 0's arrival increment, which is a
    // device-scope release; the block that arrives last acquires at device
    // scope (fence by thread 0, then the barrier) before any of its threads
    // reads the partials.  Only that block pays for the acquire.
    float *pp = part + (((int64_t)rt * KS + ks) * 16 + tl) * kPkRows + 16 * rb + 4 * q;
    if (tl < Nc) {
#pragma unroll
      for (int e = 0; e < 4; ++e) __hip_atomic_store(pp + e, v[e], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __builtin_amdgcn_s_waitcnt(0);  // this wave's partial stores have completed
    __syncthreads();
    if (tid == 0) {
      last = __hip_atomic_fetch_add(counters + rt, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT) == KS - 1;
      if (last) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    __syncthreads();
    if (!last) return;
    if (tl < Nc) {
      v = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
      for (int k2 = 0; k2 < KS; ++k2) {
        const float *src = part + (((int64_t)rt * KS + k2) * 16 + tl) * kPkRows + 16 * rb + 4 * q;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] += __hip_atomic_load(src + e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
  if (tl >= Nc || row >= m) return;
  float s = 0.0f;
  if constexpr (kXL == 2) s = (s_red[0][tl] + s_red[1][tl]) + (s_red[2][tl] + s_red[3][tl]);
  else
    for (int c = 0; c < nchunks; ++c) s += sp[c * 16 + tl];
  const int64_t o = (int64_t)tl * m + row;
  if (y_bf16) {
    uint2 w;
    w.x = pack_bf16x2(v[0] + s, v[1] + s);
    w.y = pack_bf16x2(v[2] + s, v[3] + s);
    *reinterpret_cast<uint2 *>(reinterpret_cast<uint16_t *>(Y) + o) = w;
  } else {
    *reinterpret_cast<floatx4 *>(reinterpret_cast<float *>(Y) + o) = v + s;
  }
}

// ---------------------------------------------------------------- launch ---
PackedPlan packed_plan(int64_t m, int64_t n) {
  PackedPlan p{};
  p.nP = round_up(n, kPkStep);
  p.KT = (int)(p.nP / kPkStep);
  p.row_tiles = (int)ceil_div(m, kPkRows);
  p.nchunks = (int)ceil_div(p.nP, kPkChunk);
  // Split K over blocks only until about 192 blocks run (four or more steps
  // per block, one per wave): the split costs every block a write-through of
  // its partial tile and a counter round trip, which measured dearer than the
  // idle CUs of a smaller grid once the grid passes about 200 blocks.
  int ks = (int)ceil_div(192, p.row_tiles > 0 ? p.row_tiles : 1);
  const int ks_max = p.KT / 4 > 1 ? p.KT / 4 : 1;
  ks = ks < 1 ? 1 : (ks > ks_max ? ks_max : ks);
  p.spb = p.KT > 0 ? (int)ceil_div(p.KT, ks) : 1;  // n = 0: no steps, one split
  p.KS = p.KT > 0 ? (int)ceil_div(p.KT, p.spb) : 1;
  return p;
}

hipError_t launch_packed_prep(const uint16_t *X, int Nc, int64_t m, int64_t n, int d, const float *A,
                              const float *b, uint16_t *xq, float *sp, int *counters, hipStream_t st) {
  const PackedPlan p = packed_plan(m, n);
  const dim3 g((unsigned)p.nchunks, 16);
  if (d == 8)
    k_packed_prep<8><<<g, 256, 0, st>>>(X, Nc, n, p.nP, A, b, xq, sp, counters, p.row_tiles);
  else
    k_packed_prep<4><<<g, 256, 0, st>>>(X, Nc, n, p.nP, A, b, xq, sp, counters, p.row_tiles);
  return hipGetLastError();
}

// X'' of a block's steps in LDS when it fits in 48 KiB (few tokens) and the
// block has enough steps to repay the copy and its barrier (on short K ranges
// the product is latency-bound and the copy only adds to it).
static bool packed_xl(const PackedPlan &p, int Nc) {
  // (the 48 KiB bound with spb >= 24 also keeps the fused fill's pairs within kMaxPairs)
  return ((size_t)p.spb * 32 * Nc + 1) * 16 <= 48 * 1024 && p.spb >= 24 && Nc * ((p.spb + 15) / 16) <= kMaxPairs;
}

bool packed_fused(int64_t m, int64_t n, int Nc) {
  const PackedPlan p = packed_plan(m, n);
  return p.KS == 1 && p.KT > 0 && packed_xl(p, Nc);
}

hipError_t launch_packed_gemv(const uint8_t *packed, int64_t m, int64_t n, const uint16_t *xq, const float *sp,
                              int Nc, float *part, int *counters, void *Y, bool y_bf16, hipStream_t st) {
  const PackedPlan p = packed_plan(m, n);
  const size_t xl_bytes = ((size_t)p.spb * 32 * Nc + 1) * 16;
  if (packed_xl(p, Nc))
    k_packed_gemv<1, 8><<<p.row_tiles * p.KS, 256, xl_bytes, st>>>(
        packed, m, n, p.KT, p.KS, p.spb, xq, p.nP, sp, p.nchunks, Nc, part, counters, Y, y_bf16 ? 1 : 0, nullptr,
        nullptr, nullptr);
  else
    k_packed_gemv<0, 8><<<p.row_tiles * p.KS, 256, 0, st>>>(packed, m, n, p.KT, p.KS, p.spb, xq, p.nP, sp,
                                                            p.nchunks, Nc, part, counters, Y, y_bf16 ? 1 : 0,
                                                            nullptr, nullptr, nullptr);
  return hipGetLastError();
}

hipError_t launch_packed_fused(const uint8_t *packed, int64_t m, int64_t n, const uint16_t *X, int Nc, int d,
                               const float *A, const float *b, void *Y, bool y_bf16, hipStream_t st) {
  const PackedPlan p = packed_plan(m, n);
  if (!(p.KS == 1 && p.KT > 0 && packed_xl(p, Nc))) return hipErrorInvalidValue;
  const size_t xl_bytes = ((size_t)p.spb * 32 * Nc + 1) * 16;
  if (d == 8)
    k_packed_gemv<2, 8><<<p.row_tiles, 256, xl_bytes, st>>>(packed, m, n, p.KT, 1, p.spb, nullptr, p.nP, nullptr,
                                                            p.nchunks, Nc, nullptr, nullptr, Y, y_bf16 ? 1 : 0, X,
                                                            A, b);
  else
    k_packed_gemv<2, 4><<<p.row_tiles, 256, xl_bytes, st>>>(packed, m, n, p.KT, 1, p.spb, nullptr, p.nP, nullptr,
                                                            p.nchunks, Nc, nullptr, nullptr, Y, y_bf16 ? 1 : 0, X,
                                                            A, b);
  return hipGetLastError();
}

}  // namespace lcvq
