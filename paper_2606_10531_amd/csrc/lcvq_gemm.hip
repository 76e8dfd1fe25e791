// bf16 matrix-core (MFMA) products of the LC-VQ layer, gfx950.
//
// All three products put the weight-side axis (out-features r or in-features
// c) on the MFMA M axis and tokens (or out-features for dW) on N.  The M rows
// of every 32-row block are permuted (perm32) so that accumulator register i
// of lane L holds weight-side index 16 (L / 32) + i: each lane owns sixteen
// consecutive weight-side columns of one token row, i.e. whole groups.
//
//   forward : D[r, t] = sum_c code[r, c] X'[t, c]          Y[t, r] = D + s[t]
//   input   : D[c, t] = sum_r code[r, c] dY[t, r]          dX[t, c] = (D-group) A^T + rs[t] b
//   weight  : D[c, r] = sum_t X[t, c] dY[t, r]  (= dW[r,c]) dZ = mask * (dW-group) A, dA, db
//
// Codes reach the matrix cores exactly: the operand layout holds them as 4-bit
// nibbles and the fp4 -> bf16 converter turns them into bf16 values 0..3 in
// registers, so the dense W_hat never exists anywhere.
#include "lcvq_prep.hpp"

namespace lcvq {

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr int kTile = 256;   // block tile (M and N)
constexpr int kKStep = 64;   // K per main-loop step

// s_waitcnt with every counter at zero.
#define LCVQ_WAIT_ALL() __builtin_amdgcn_s_waitcnt(0)

// Blocks are dispatched round-robin over the eight XCDs.  Give each XCD a
// contiguous run of tile ids, and walk tiles in bands of four M-tiles, so the
// blocks sharing an XCD's L2 share operand tiles.
__device__ __forceinline__ void tile_of_block(int tiles_m, int tiles_n, int &tm, int &tn) {
  const int nblocks = (int)gridDim.x;
  int id = (int)blockIdx.x;
  if (nblocks % 8 == 0) id = (id % 8) * (nblocks / 8) + id / 8;
  constexpr int GM = 4;
  const int band = id / (GM * tiles_n);
  const int first = band * GM;
  const int gm = min(tiles_m - first, GM);
  const int in = id - band * GM * tiles_n;
  tm = first + in % gm;
  tn = in / gm;
}

__device__ __forceinline__ float as_f(uint32_t u) { return __uint_as_float(u); }
__device__ __forceinline__ uint32_t as_u(float f) { return __float_as_uint(f); }

// ============================================================================
// Products with codes as the A operand (forward, input gradient).
// B operand tile in LDS: 256 token rows x 64 K (bf16), 128 B per row; 16-byte
// chunk q of row r lives at physical chunk q ^ ((r >> 1) & 7).
// ============================================================================

__device__ __forceinline__ uint32_t btile_off(int row, int chunk) {
  return (uint32_t)(row * 128 + ((chunk ^ ((row >> 1) & 7)) << 4));
}

template <int kMode, int D, bool kMaskK>  // kMode 0: forward, 1: input gradient
__global__ __launch_bounds__(256, 1) void k_gemm_codes(
    const uint32_t *__restrict__ frag, int KB, const uint16_t *__restrict__ Bsrc, int ldb,
    int64_t brows, int kvalid, int tiles_m, int tiles_n, const float *__restrict__ vecT,
    const float *__restrict__ A, const float *__restrict__ bvec, uint16_t *__restrict__ out,
    int64_t ldo, int64_t Mvalid, int64_t Tvalid) {
  __shared__ __attribute__((aligned(1024))) char lds[2 * kTile * 128];  // two stages

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  int tm, tn;
  tile_of_block(tiles_m, tiles_n, tm, tn);
  const int64_t tok0 = (int64_t)tn * kTile;

  // B tile loads: instruction j of wave w fills rows 32 j + 8 w .. + 7; the
  // lane part of the byte offset is fixed, the K step moves the buffer base.
  const int brow0 = 8 * wave + (lane >> 3);
  const int bchunk = (lane & 7) ^ ((brow0 >> 1) & 7);
  const uint32_t boff0 = (uint32_t)(brow0 * ldb + bchunk * 8) * 2u;
  const uint32_t bstep = (uint32_t)ldb * 64u;  // 32 rows
  const uint16_t *Bt = Bsrc + tok0 * ldb;
  const int64_t bbytes = (brows - tok0) * (int64_t)ldb * 2;

  // codes: this wave's four 32-row slabs, 1 KiB per (slab, K step)
  const uint32_t *fw = frag + (size_t)(tm * 8 + wm * 4) * KB * 256;
  const __amdgpu_buffer_rsrc_t rsA = make_rsrc(fw, (int64_t)4 * KB * 1024);

  // B fragment reads: row wn*128 + ni*32 + lane%32, logical chunk 2 kk + h
  const int bx = ((lane & 31) >> 1) & 7;
  const uint32_t brow = (uint32_t)(wn * 128 + (lane & 31)) * 128u;
  uint32_t brd[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) brd[kk] = brow + ((uint32_t)((2 * kk + h) ^ bx) << 4);

  floatx16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx16{};

  auto issue_b = [&](char *stage, int kb) {
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(Bt + kb * kKStep, bbytes - (int64_t)kb * 128);
    uint32_t base = boff0;
    if constexpr (kMaskK) base = (kb * kKStep + bchunk * 8 < kvalid) ? boff0 : kOffNone;
#pragma unroll
    for (int j = 0; j < 8; ++j)
      buffer_to_lds16(rs, (lds_void *)(stage + (j * 4 + wave) * 1024), base + (uint32_t)j * bstep);
  };
  auto load_a = [&](u32x4 *dst, int kb) {
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
      dst[mi] = __builtin_amdgcn_raw_buffer_load_b128(rsA, lane * 16, (mi * KB + kb) * 1024, 0);
  };
  auto compute = [&](const char *stage, const u32x4 *ca) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      bf16x8 a[4], b[4];
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) b[ni] = *reinterpret_cast<const bf16x8 *>(stage + brd[kk] + ni * 4096);
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) a[mi] = nibbles_to_bf16x8(ca[mi][kk]);
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
    }
  };

  u32x4 ca[4], cn[4];
  issue_b(lds, 0);
  load_a(cn, 0);
  for (int kb = 0; kb < KB; ++kb) {
    LCVQ_WAIT_ALL();
    __syncthreads();
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) ca[mi] = cn[mi];
    if (kb + 1 < KB) {
      issue_b(lds + ((kb + 1) & 1) * (kTile * 128), kb + 1);
      load_a(cn, kb + 1);
    }
    compute(lds + (kb & 1) * (kTile * 128), ca);
  }

  // ---------------------------------------------------------------- epilogue
  // Lane L holds, for each (mi, ni), the 16 consecutive weight-side columns
  // cb .. cb + 15 of token row t.  Branch-free: rows beyond the tensor fall
  // outside the buffer (loads give 0, stores are dropped) and columns beyond it
  // get an out-of-range offset.
  const __amdgpu_buffer_rsrc_t ro = make_rsrc(out + tok0 * ldo, (Tvalid - tok0) * ldo * 2);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vecT + tok0, (Tvalid - tok0) * 4);
  const int64_t cb0 = (int64_t)tm * kTile + wm * 128 + 16 * h;
  float am[D][D], bm[D];
  if constexpr (kMode == 1) {
#pragma unroll
    for (int j = 0; j < D; ++j) {
      bm[j] = bvec[j];
#pragma unroll
      for (int k = 0; k < D; ++k) am[j][k] = A[j * D + k];
    }
  }
#pragma unroll
  for (int ni = 0; ni < 4; ++ni) {
    const int tl = wn * 128 + ni * 32 + (lane & 31);
    const float vt = as_f(__builtin_amdgcn_raw_buffer_load_b32(rv, tl * 4, 0, 0));
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
      float y[16];
      if constexpr (kMode == 0) {
        // forward: Y[t, r] = D + s[t]
#pragma unroll
        for (int i = 0; i < 16; ++i) y[i] = acc[mi][ni][i] + vt;
      } else {
        // input gradient: dX[t, g*D + j] = sum_k A[j, k] P[t, g*D + k] + rs[t] b[j]
#pragma unroll
        for (int g = 0; g < 16 / D; ++g)
#pragma unroll
          for (int j = 0; j < D; ++j) {
            float v = vt * bm[j];
#pragma unroll
            for (int k = 0; k < D; ++k) v = fmaf(am[j][k], acc[mi][ni][g * D + k], v);
            y[g * D + j] = v;
          }
      }
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int64_t c = cb0 + mi * 32 + 8 * half;
        const uint32_t off = c < Mvalid ? (uint32_t)(tl * ldo + c) * 2u : kOffNone;
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(y[8 * half + 2 * e], y[8 * half + 2 * e + 1]);
        __builtin_amdgcn_raw_buffer_store_b128(w, ro, off, 0, 0);
      }
    }
  }
}

// ============================================================================
// Weight-gradient product with the straight-through epilogue.
// Both operands are K(token)-major in memory; tiles of 64 token rows x 256
// columns (512 B per row) go to LDS, and ds_read_b64_tr_b16 hands each lane
// eight consecutive tokens of one column.  16-byte chunk q of row t lives at
// physical chunk q ^ (4 * (t & 3)).
// ============================================================================

template <int D>
__global__ __launch_bounds__(256, 1) void k_gemm_dz(
    const uint16_t *__restrict__ X, const uint16_t *__restrict__ dY, const uint16_t *__restrict__ Z,
    const float *__restrict__ A, int mask_mode, int accumulate, void *__restrict__ dZ, int dz_bf16,
    float *__restrict__ dA, float *__restrict__ db, int64_t N, int m, int n, int tiles_m,
    int tiles_n, int KB) {
  // two stages, each an X tile then a dY tile of 64 token rows x 512 B
  __shared__ __attribute__((aligned(1024))) char lds[4 * 64 * 512];
  __shared__ float red[4][D * D + D];

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  int tm, tn;
  tile_of_block(tiles_m, tiles_n, tm, tn);
  const int c0 = tm * kTile, r0 = tn * kTile;

  // tile loads: instruction j of wave w fills token rows 8 j + 2 w + {0, 1};
  // columns outside the tensor get an out-of-range offset (zero fill).
  const int lrow = 2 * wave + h;
  const int lchunk = (lane & 31) ^ (4 * (lrow & 3));
  const uint32_t xoff0 = c0 + lchunk * 8 < n ? (uint32_t)(lrow * n + lchunk * 8) * 2u : kOffNone;
  const uint32_t yoff0 = r0 + lchunk * 8 < m ? (uint32_t)(lrow * m + lchunk * 8) * 2u : kOffNone;
  const uint32_t xstep = (uint32_t)n * 16u, ystep = (uint32_t)m * 16u;  // 8 rows

  // transposed fragment reads: per-lane offsets for the four 32-column blocks
  const int g = lane >> 4, s = lane & 15;
  const int trow = 8 * (g >> 1) + (s >> 2), tsw = 4 * (trow & 3);
  // A operand rows follow perm32: source lane s of group g reads the four
  // columns perm32(16 (g & 1) + 4 (s & 3)) .. + 3.
  uint32_t ra[4], rb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ca = wm * 128 + i * 32 + perm32(16 * (g & 1) + 4 * (s & 3));
    const int cb = wn * 128 + i * 32 + 16 * (g & 1) + 4 * (s & 3);
    ra[i] = (uint32_t)(trow * 512 + (((ca >> 3) ^ tsw) << 4) + (ca & 7) * 2);
    rb[i] = (uint32_t)(trow * 512 + (((cb >> 3) ^ tsw) << 4) + (cb & 7) * 2);
  }

  floatx16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx16{};

  auto issue = [&](char *sx, char *sy, int kb) {
    const int64_t t0 = (int64_t)kb * 64;
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(X + t0 * n + c0, (N - t0) * n * 2 - (int64_t)c0 * 2);
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(dY + t0 * m + r0, (N - t0) * m * 2 - (int64_t)r0 * 2);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      buffer_to_lds16(rx, (lds_void *)(sx + (j * 4 + wave) * 1024), xoff0 + (uint32_t)j * xstep);
      buffer_to_lds16(ry, (lds_void *)(sy + (j * 4 + wave) * 1024), yoff0 + (uint32_t)j * ystep);
    }
  };
  auto frag_tr = [&](const char *tile, uint32_t off) {
    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(tile + off));
    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(tile + off + 2048));
    return (bf16x8)__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  };
  auto compute = [&](const char *sx, const char *sy) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      bf16x8 a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = frag_tr(sx + kk * 8192, ra[i]);
#pragma unroll
      for (int i = 0; i < 4; ++i) b[i] = frag_tr(sy + kk * 8192, rb[i]);
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
    }
  };

  constexpr int kStage = 2 * 64 * 512;
  issue(lds, lds + 64 * 512, 0);
  for (int kb = 0; kb < KB; ++kb) {
    LCVQ_WAIT_ALL();
    __syncthreads();
    if (kb + 1 < KB) {
      char *nx = lds + ((kb + 1) & 1) * kStage;
      issue(nx, nx + 64 * 512, kb + 1);
    }
    const char *cx = lds + (kb & 1) * kStage;
    compute(cx, cx + 64 * 512);
  }

  // ------------------------------------------------ straight-through epilogue
  // Lane L holds dW[r, cb .. cb + 15] for each (mi, ni): whole groups, so the
  // map A (uniform, in scalar registers) applies lane-locally.
  float am[D][D];
#pragma unroll
  for (int j = 0; j < D; ++j)
#pragma unroll
    for (int k = 0; k < D; ++k) am[j][k] = A[j * D + k];
  float gA[D][D], gb[D];
#pragma unroll
  for (int j = 0; j < D; ++j) {
    gb[j] = 0.0f;
#pragma unroll
    for (int k = 0; k < D; ++k) gA[j][k] = 0.0f;
  }

  // rows r >= m fall outside these buffers; columns c >= n get an out-of-range index
  const __amdgpu_buffer_rsrc_t rz = make_rsrc(Z + (int64_t)r0 * n, (int64_t)(m - r0) * n * 2);
  const int es = dz_bf16 ? 2 : 4;
  const __amdgpu_buffer_rsrc_t rg =
      make_rsrc((char *)dZ + (int64_t)r0 * n * es, dZ == nullptr ? 0 : (int64_t)(m - r0) * n * es);
#pragma unroll
  for (int ni = 0; ni < 4; ++ni) {
    const int rl = wn * 128 + ni * 32 + (lane & 31);
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int c = c0 + wm * 128 + mi * 32 + 16 * h + 8 * half;
        const bool cv = c < n;
        const uint32_t e2 = cv ? (uint32_t)(rl * n + c) * 2u : kOffNone;  // byte offsets, bf16
        const uint32_t e4 = cv ? (uint32_t)(rl * n + c) * 4u : kOffNone;  // and fp32
        const u32x4 zw = __builtin_amdgcn_raw_buffer_load_b128(rz, e2, 0, 0);
        float z[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          z[2 * e] = bf16_lo(zw[e]);
          z[2 * e + 1] = bf16_hi(zw[e]);
        }
        float gz[8];
#pragma unroll
        for (int g = 0; g < 8 / D; ++g) {
          float w[D], code[D];
#pragma unroll
          for (int j = 0; j < D; ++j) {
            w[j] = acc[mi][ni][8 * half + g * D + j];
            code[j] = (float)quant_code(z[g * D + j]);
            gb[j] += w[j];
          }
#pragma unroll
          for (int k = 0; k < D; ++k) {
            float v = 0.0f;
#pragma unroll
            for (int j = 0; j < D; ++j) {
              v = fmaf(w[j], am[j][k], v);
              gA[j][k] = fmaf(w[j], code[k], gA[j][k]);
            }
            gz[g * D + k] = ste_pass(z[g * D + k], mask_mode) ? v : 0.0f;
          }
        }
        if (dz_bf16) {
          if (accumulate) {
            const u32x4 o = __builtin_amdgcn_raw_buffer_load_b128(rg, e2, 0, 0);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              gz[2 * e] += bf16_lo(o[e]);
              gz[2 * e + 1] += bf16_hi(o[e]);
            }
          }
          u32x4 wv;
#pragma unroll
          for (int e = 0; e < 4; ++e) wv[e] = pack_bf16x2(gz[2 * e], gz[2 * e + 1]);
          __builtin_amdgcn_raw_buffer_store_b128(wv, rg, e2, 0, 0);
        } else {
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            u32x4 wv;
            if (accumulate) {
              const u32x4 o = __builtin_amdgcn_raw_buffer_load_b128(rg, e4 + 16u * q, 0, 0);
#pragma unroll
              for (int e = 0; e < 4; ++e) gz[4 * q + e] += as_f(o[e]);
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) wv[e] = as_u(gz[4 * q + e]);
            __builtin_amdgcn_raw_buffer_store_b128(wv, rg, e4 + 16u * q, 0, 0);
          }
        }
        // keep the scheduler from hoisting every block's loads (register pressure)
        __builtin_amdgcn_sched_barrier(0);
      }
  }

  // reduce the map gradients: lanes -> wave (shuffles), waves -> block (LDS),
  // then one atomic per block per entry.
#pragma unroll
  for (int j = 0; j < D; ++j) {
#pragma unroll
    for (int k = 0; k < D; ++k)
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) gA[j][k] += __shfl_xor(gA[j][k], o, 64);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) gb[j] += __shfl_xor(gb[j], o, 64);
  }
  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < D; ++j) {
      red[wave][D * D + j] = gb[j];
#pragma unroll
      for (int k = 0; k < D; ++k) red[wave][j * D + k] = gA[j][k];
    }
  }
  __syncthreads();
  if (tid < D * D + D) {
    const float v = red[0][tid] + red[1][tid] + red[2][tid] + red[3][tid];
    if (tid < D * D) unsafeAtomicAdd(dA + tid, v);
    else unsafeAtomicAdd(db + (tid - D * D), v);
  }
}

// ---- launchers -------------------------------------------------------------

hipError_t launch_fwd_bf16(const uint32_t *frag, const uint16_t *Xp, int64_t ldp, const float *s,
                           uint16_t *Y, int64_t N, int64_t m, int64_t n, hipStream_t st) {
  (void)n;
  const int tiles_m = (int)ceil_div(m, kTile), tiles_n = (int)ceil_div(N, kTile);
  const int KB = (int)(ldp / kKStep);
  const int64_t Np = (int64_t)tiles_n * kTile;
  k_gemm_codes<0, 8, false><<<tiles_m * tiles_n, 256, 0, st>>>(frag, KB, Xp, (int)ldp, Np, (int)ldp, tiles_m,
                                                               tiles_n, s, nullptr, nullptr, Y, m, m, N);
  return hipGetLastError();
}

hipError_t launch_dx_bf16(const uint32_t *frag, const uint16_t *dY, const float *rs, const float *A,
                          const float *b, int d, uint16_t *dX, int64_t N, int64_t m, int64_t n,
                          hipStream_t st) {
  const int tiles_m = (int)ceil_div(n, kTile), tiles_n = (int)ceil_div(N, kTile);
  const int KB = (int)ceil_div(m, kKStep);
  if (d == 8)
    k_gemm_codes<1, 8, true><<<tiles_m * tiles_n, 256, 0, st>>>(frag, KB, dY, (int)m, N, (int)m, tiles_m,
                                                                tiles_n, rs, A, b, dX, n, n, N);
  else
    k_gemm_codes<1, 4, true><<<tiles_m * tiles_n, 256, 0, st>>>(frag, KB, dY, (int)m, N, (int)m, tiles_m,
                                                                tiles_n, rs, A, b, dX, n, n, N);
  return hipGetLastError();
}

hipError_t launch_dz_bf16(const uint16_t *X, const uint16_t *dY, const uint16_t *Z, const float *A, int d,
                          int mask_mode, int accumulate, void *dZ, bool dz_bf16, float *dA, float *db,
                          int64_t N, int64_t m, int64_t n, hipStream_t st) {
  const int tiles_m = (int)ceil_div(n, kTile), tiles_n = (int)ceil_div(m, kTile);
  const int KB = (int)ceil_div(N, 64);
  if (d == 8)
    k_gemm_dz<8><<<tiles_m * tiles_n, 256, 0, st>>>(X, dY, Z, A, mask_mode, accumulate, dZ, dz_bf16 ? 1 : 0,
                                                    dA, db, N, (int)m, (int)n, tiles_m, tiles_n, KB);
  else
    k_gemm_dz<4><<<tiles_m * tiles_n, 256, 0, st>>>(X, dY, Z, A, mask_mode, accumulate, dZ, dz_bf16 ? 1 : 0,
                                                    dA, db, N, (int)m, (int)n, tiles_m, tiles_n, KB);
  return hipGetLastError();
}

}  // namespace lcvq
