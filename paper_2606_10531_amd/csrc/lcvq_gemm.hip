// bf16 matrix-core (MFMA) products of the LC-VQ layer, gfx950.
//
// All three products put the weight-side axis (out-features r or in-features
// c) on the MFMA M axis and tokens (or out-features for dW) on N, and use the
// 16x16x32 instruction: on this chip it sustains about a fifth more throughput
// than 32x32x16 on real-valued operands (the clock is power-limited, and the
// smaller shape draws less per flop).  The M rows of every 32-row slab are
// permuted (slab_row) so that each lane ends with eight consecutive
// weight-side indices of one token (or out-feature), i.e. whole groups.
//
//   forward : D[r, t] = sum_c code[r, c] X'[t, c]          Y[t, r] = D + s[t]
//   input   : D[c, t] = sum_r code[r, c] dY[t, r]          dX[t, c] = (D-group) A^T + rs[t] b,
//                                                           dA, db from D and X
//   weight  : D[c, r] = sum_t X'[t, c] dY[t, r]             dZ[r, c] = mask * D  (D = dW blockdiag(A))
//
// Codes reach the matrix cores exactly: the operand layout holds them as 4-bit
// nibbles and the fp4 -> bf16 converter turns them into bf16 values 0..3 in
// registers, so the dense W_hat never exists anywhere.
//
// The main loops issue the instructions from inline assembly with the
// accumulators bound to AGPRs: the compiler's own selection of this
// instruction moves the accumulators between registers around every loop
// trip.  The compiler cannot see hazards inside such statements, so the code
// provides the wait states itself: after the zeroing of the accumulators
// (acc_fence), before an MFMA that reads a just-converted codes operand
// (mfma16_valu_a; only the first of a step: the other conversions are
// themselves inline assembly placed two MFMAs ahead of their consumer), and
// after the loop (mfma_drain).  All other operands come from loads, which the
// compiler's waits cover.  The input gradient's epilogue products (the A-map
// and the map gradient) use the compiler's builtin, whose hazards it handles.
#include "lcvq_prep.hpp"

namespace lcvq {

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr int kTile = 256;   // block tile (M and N)
constexpr int kKStep = 64;   // K per main-loop step

// s_waitcnt with every counter at zero.
#define LCVQ_WAIT_ALL() __builtin_amdgcn_s_waitcnt(0)
// s_waitcnt vmcnt(N) lgkmcnt(0) (gfx9 encoding; expcnt left at its maximum).
#define LCVQ_WAIT_VM_LGKM0(N) __builtin_amdgcn_s_waitcnt(((N) & 15) | (((N) >> 4) << 14) | (7 << 4))
// s_waitcnt vmcnt(N) only (lgkmcnt and expcnt left at their maximum).
#define LCVQ_WAIT_VM(N) __builtin_amdgcn_s_waitcnt(((N) & 15) | (((N) >> 4) << 14) | (7 << 4) | (15 << 8))
// s_waitcnt lgkmcnt(0) only.
#define LCVQ_WAIT_LGKM0() __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4))
// Workgroup barrier without the release fence of __syncthreads() (which would
// drain the prefetch loads); the asm statements keep the compiler from moving
// memory operations across it.  LDS visibility is ensured by the waits above.
#define LCVQ_BARRIER()                   \
  do {                                   \
    asm volatile("" ::: "memory");       \
    __builtin_amdgcn_s_barrier();        \
    asm volatile("" ::: "memory");       \
  } while (0)

// Blocks are dispatched round-robin over the eight XCDs.  Give each XCD a
// contiguous run of tile ids, and walk tiles in bands of eight M-tiles, so the
// blocks sharing an XCD's L2 share operand tiles (with 256 tiles: 8 M-tiles x
// 4 token tiles per XCD, the fewest operand bytes per L2 for these products).
__device__ __forceinline__ void tile_of_block(int tiles_m, int tiles_n, int &tm, int &tn) {
  const int nblocks = (int)gridDim.x;
  int id = (int)blockIdx.x;
  if (nblocks % 8 == 0) id = (id % 8) * (nblocks / 8) + id / 8;
  constexpr int GM = 8;
  const int band = id / (GM * tiles_n);
  const int first = band * GM;
  const int gm = min(tiles_m - first, GM);
  const int in = id - band * GM * tiles_n;
  tm = first + in % gm;
  tn = in / gm;
}

// acc = A * B + acc, operands loaded (no VALU producer): issued in program order.
__device__ __forceinline__ void mfma16(floatx4 &acc, const bf16x8 &a, const bf16x8 &b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// The same with A produced by VALU instructions: the leading s_nop covers the
// VALU-write to matrix-core-read wait states.
__device__ __forceinline__ void mfma16_valu_a(floatx4 &acc, const bf16x8 &a, const bf16x8 &b) {
  asm volatile("s_nop 2\n\tv_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// Wait states between the zeroing of the accumulators (vector writes) and the
// first matrix-core read of them, R x C accumulators.  Each statement passes
// four accumulators through itself, so every zeroing write precedes the whole
// chain and every MFMA follows it: at least R C / 4 statements and a final
// s_nop 4 lie between a write and a read.
template <int R, int C>
__device__ __forceinline__ void acc_fence(floatx4 (&acc)[R][C]) {
  static_assert(C % 4 == 0, "four accumulators per statement");
#pragma unroll
  for (int i = 0; i < R; ++i)
#pragma unroll
    for (int j = 0; j < C; j += 4) {
      if (i + 1 < R || j + 4 < C)
        asm volatile("s_nop 0" : "+a"(acc[i][j]), "+a"(acc[i][j + 1]), "+a"(acc[i][j + 2]), "+a"(acc[i][j + 3]));
      else
        asm volatile("s_nop 4" : "+a"(acc[i][j]), "+a"(acc[i][j + 1]), "+a"(acc[i][j + 2]), "+a"(acc[i][j + 3]));
    }
}
// Wait states between the last matrix-core write of an accumulator and the
// epilogue's vector reads of it.  The statement is a scheduling boundary with
// a memory clobber; the reads are copies the compiler places at their uses,
// which all lie in the epilogue after it.
__device__ __forceinline__ void mfma_drain() { asm volatile("s_nop 15\n\ts_nop 15" ::: "memory"); }

// The codes conversion as ordered inline assembly: it stays where it is written
// (between two MFMAs of the previous operand), so the two MFMAs that follow it
// supply the wait states its consumer needs.
__device__ __forceinline__ bf16x8 nibbles_to_bf16x8_ordered(uint32_t w) {
  uint32_t p0, p1, p2, p3;
  asm volatile("v_cvt_scalef32_pk_bf16_fp4 %0, %1, 2.0" : "=v"(p0) : "v"(w));
  asm volatile("v_cvt_scalef32_pk_bf16_fp4 %0, %1, 2.0 op_sel:[1,0,0]" : "=v"(p1) : "v"(w));
  asm volatile("v_cvt_scalef32_pk_bf16_fp4 %0, %1, 2.0 op_sel:[0,1,0]" : "=v"(p2) : "v"(w));
  asm volatile("v_cvt_scalef32_pk_bf16_fp4 %0, %1, 2.0 op_sel:[1,1,0]" : "=v"(p3) : "v"(w));
  return __builtin_bit_cast(bf16x8, u32x4{p0, p1, p2, p3});
}

__device__ __forceinline__ float as_f(uint32_t u) { return __uint_as_float(u); }
// Copy a (uniform) value into a vector register.
__device__ __forceinline__ float to_vgpr(float x) {
  float v;
  asm volatile("v_mov_b32 %0, %1" : "=v"(v) : "s"(x));
  return v;
}
__device__ __forceinline__ uint32_t as_u(float f) { return __float_as_uint(f); }

// ============================================================================
// Products with codes as the A operand (forward, input gradient).
// Each wave owns 256 weight-side rows x 64 tokens (where those sit in the
// block tile is set at the top of the kernel) and streams both operands
// straight into registers, with no LDS stage: the codes of its eight 32-row
// slabs (operand layout; waves on the same rows share them through the L1)
// and its activations: for the forward X' in the matrix-core B layout, as the
// activation transform writes it; for the input gradient dY itself,
// row-major, read in place (a lane's B operand, eight consecutive
// out-features of one token, is 16 contiguous bytes of dY, and the 16 token
// rows a load touches are each read in whole 128-byte lines by its two K
// halves).  K is padded to an even number of 64-wide steps; out-features >=
// ldB read as zero.  LDS holds only the input gradient's X tile and map-
// gradient staging (below).
// ============================================================================

// Input-gradient mode also forms the map gradients from the same accumulator
// P = dY codes: dA[j, k] = sum_{t,g} X[t, g*D + j] P[t, g*D + k] and
// db[j] = sum_{t,g} X[t, g*D + j] rs[t] (the chain rule through X' = X blockdiag(A)
// and s = X b~): dA on the matrix cores, db on the vector units, reduced
// lanes -> wave -> block; entry e of block b is stored (no atomics) at
// mapp[e * gridDim.x + b], and a later launch sums each entry over the blocks
// in a fixed order, so dA and db come out the same bit for bit on every call.
// X is N x Mvalid row-major; mapp == nullptr skips this.
template <int kMode, int D>  // kMode 0: forward (B = X' fragments), 1: input gradient (B = dY, row length ldB)
__global__ __launch_bounds__(256, 1) void k_gemm_codes(
    const uint32_t *__restrict__ frag, int KB, const uint16_t *__restrict__ Bsrc, int64_t ldB,
    int tiles_m, int tiles_n, const float *__restrict__ vecT, int vparts,
    int64_t vstride, const float *__restrict__ A, const float *__restrict__ bvec, uint16_t *__restrict__ out,
    int64_t ldo, int64_t Mvalid, int64_t Tvalid, const uint16_t *__restrict__ X,
    float *__restrict__ mapp) {
  const int tid = threadIdx.x, lane = tid & 63, q = lane >> 4, c16 = lane & 15;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // The wave's 256 weight-side rows (256-row tile tm) and 64 tokens from tw.
  // Forward: block tile 512 rows x 128 tokens, wave w on rows 256 (w % 2) and
  // tokens 64 (w / 2) of it, so two waves share each codes slab and two each
  // token block through the L1 (a fifth less L2 traffic per step than 256 x
  // 256; measured 2.5 us shorter at 4096^3).  Input gradient: 256 x 256, wave
  // w on tokens 64 w (the 2 x 2 arrangement measured 2.8 us longer there).
  int tm;
  int64_t tw;
  {
    int bm, bn;
    tile_of_block(tiles_m, tiles_n, bm, bn);
    if constexpr (kMode == 0) {
      tm = 2 * bm + (wave & 1);
      tw = (int64_t)bn * 128 + 64 * (wave >> 1);
    } else {
      tm = bm;
      tw = (int64_t)bn * kTile + 64 * wave;
    }
  }

  // codes: slabs tm * 8 + mi, 1 KiB per (slab, step), lane owns 16 bytes (none
  // for a wave past the weight side)
  const __amdgpu_buffer_rsrc_t rsA =
      make_rsrc(frag + (size_t)(tm * 8) * KB * 256, (int64_t)tm * kTile < Mvalid ? (int64_t)8 * KB * 1024 : 0);
  // B operand of tokens tw .. tw + 63: X' in the B-operand fragment layout
  // with KB K steps (forward), or rows tw .. tw + 63 of dY (input gradient;
  // rows past Tvalid lie beyond the buffer and read as zero).  Fragment
  // 2 th + kk2 of 32-token block ni holds tokens 32 ni + 16 th + L % 16 and
  // K = 32 kk2 + 8 (L / 16) + 0..7 of each step.
  const __amdgpu_buffer_rsrc_t rsB =
      kMode == 0 ? make_rsrc(Bsrc + (tw >> 5) * (int64_t)KB * 2048, (int64_t)2 * KB * 4096)
                 : make_rsrc(Bsrc + tw * ldB, (Tvalid - tw < 64 ? Tvalid - tw : 64) * ldB * 2);
  uint32_t boff[2][4];  // per (32-token block, fragment): byte offset of this lane's 16 bytes at step 0
#pragma unroll
  for (int ni = 0; ni < 2; ++ni)
#pragma unroll
    for (int fr = 0; fr < 4; ++fr)
      boff[ni][fr] = kMode == 0 ? (uint32_t)((ni * KB * 4 + fr) * 1024 + lane * 16)
                                : (uint32_t)(((ni * 32 + (fr >> 1) * 16 + c16) * ldB + (fr & 1) * 32 + 8 * q) * 2);
  // bytes per K step; input gradient: the last out-feature chunk a lane may read
  const uint32_t bstep = kMode == 0 ? 4096u : 128u;
  const int kB_last = kMode == 0 ? KB * 64 : (int)ldB - 8;

  // Input gradient with map gradients: the wave's X tile (its 64 tokens x the
  // block's 256 columns) is copied to LDS during the main loop, one 1 KiB pair
  // (16-token block tb, slab mi) per K step, in the order the epilogue reads
  // it: lane L of pair p = 8 tb + mi holds X[t, c .. c + 7] with t = tw + 16 tb
  // + L % 16 and c = 256 tm + 32 mi + 8 (L / 16).  The epilogue then finds X
  // in LDS instead of waiting on HBM latency once per pair.
  constexpr int kXPairs = 32;
  __shared__ __attribute__((aligned(1024))) char xs[kMode == 1 ? 4 * kXPairs * 1024 : 16];
  const bool want_map = kMode == 1 && mapp != nullptr;
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(X + tw * Mvalid, want_map ? (Tvalid - tw) * Mvalid * 2 : 0);
  if (want_map && (tw + 64 > Tvalid || (int64_t)tm * kTile + kTile > Mvalid)) {
    // a tile reaching past the tensor: the pairs start as zeros, so rows and
    // columns outside it read as zero whatever the out-of-range copies leave
#pragma unroll
    for (int p = 0; p < kXPairs; ++p)
      *reinterpret_cast<u32x4 *>(xs + (wave * kXPairs + p) * 1024 + lane * 16) = u32x4{0u, 0u, 0u, 0u};
    LCVQ_WAIT_LGKM0();
    asm volatile("" ::: "memory");
  }
  // this lane's offset for pair 0 and its columns inside the tensor from there
  const int64_t xcol0 = (int64_t)tm * kTile + 8 * q;
  const uint32_t xoff0 = (uint32_t)(c16 * Mvalid + xcol0) * 2u;
  const int xcols = (int)(Mvalid - xcol0 < 256 ? Mvalid - xcol0 : 256);
  auto xprefetch = [&](int p) {
    if constexpr (kMode == 1) {
      const int tb = p >> 3, mi = p & 7;
      const uint32_t off = 32 * mi < xcols ? xoff0 + (uint32_t)(tb * 16 * Mvalid + mi * 32) * 2u : kOffNone;
      buffer_to_lds16(rx, (lds_void *)(xs + (wave * kXPairs + p) * 1024), off);
    }
  };

  floatx4 acc[16][4];  // [row block 2 mi + rb][16-token block tb]
#pragma unroll
  for (int i = 0; i < 16; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
  acc_fence(acc);

  // Two register buffers of one 64-wide step each; the loads of step k + 2 are
  // issued as soon as step k's MFMAs have been issued.
  u32x4 ca[2][8], cb[2][2][4];
  auto load = [&](int buf, int kb) {
    const bool live = kb < KB;
#pragma unroll
    for (int mi = 0; mi < 8; ++mi)
      ca[buf][mi] = __builtin_amdgcn_raw_buffer_load_b128(rsA, live ? lane * 16 : (int)kOffNone,
                                                          (mi * KB + kb) * 1024, 0);
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int fr = 0; fr < 4; ++fr) {
        // input gradient: K chunks at or past ldB (the last, padded steps) are not read
        const bool kin = kMode == 0 || kb * 64 + (fr & 1) * 32 + 8 * q <= kB_last;
        cb[buf][ni][fr] = __builtin_amdgcn_raw_buffer_load_b128(
            rsB, live && kin ? (int)(boff[ni][fr] + (uint32_t)kb * bstep) : (int)kOffNone, 0, 0);
      }
    if (want_map && kb < kXPairs) xprefetch(kb);
  };
  // 32 A operands per step (sub-step kk2, row block 2 mi + rb), each used by
  // four MFMAs; the conversion of the next one is placed between the second
  // and third of them, so the converter works while the matrix core does.
  auto compute = [&](int buf) {
    auto conv = [&](int s2) {  // s2 = 16 kk2 + 2 mi + rb
      return nibbles_to_bf16x8_ordered(ca[buf][(s2 & 15) >> 1][2 * (s2 & 1) + (s2 >> 4)]);
    };
    bf16x8 an = conv(0);
#pragma unroll
    for (int s2 = 0; s2 < 32; ++s2) {
      const int kk2 = s2 >> 4, p = s2 & 15;
      const bf16x8 a = an;
      const bf16x8 b0 = __builtin_bit_cast(bf16x8, cb[buf][0][kk2]), b1 = __builtin_bit_cast(bf16x8, cb[buf][0][2 + kk2]);
      const bf16x8 b2 = __builtin_bit_cast(bf16x8, cb[buf][1][kk2]), b3 = __builtin_bit_cast(bf16x8, cb[buf][1][2 + kk2]);
      if (s2 == 0) mfma16_valu_a(acc[p][0], a, b0); else mfma16(acc[p][0], a, b0);
      mfma16(acc[p][1], a, b1);
      if (s2 + 1 < 32) an = conv(s2 + 1);
      mfma16(acc[p][2], a, b2);
      mfma16(acc[p][3], a, b3);
    }
  };

  // The scheduling fences keep every load of buffer 0 ahead of every load of
  // buffer 1, so the compiler can wait for one buffer while the other is still
  // in flight (without them it sinks both groups to the end of the trip and
  // waits for all loads before the next MFMA).
  load(0, 0);
  __builtin_amdgcn_sched_barrier(0);
  load(1, 1);
  __builtin_amdgcn_sched_barrier(0);
  for (int kb = 0; kb < KB; kb += 2) {
    compute(0);
    __builtin_amdgcn_sched_barrier(0);
    load(0, kb + 2);
    __builtin_amdgcn_sched_barrier(0);
    compute(1);
    __builtin_amdgcn_sched_barrier(0);
    load(1, kb + 3);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (want_map)  // K shorter than the pair count: the rest of the X tile
    for (int p = KB + 2; p < kXPairs; ++p) xprefetch(p);
  mfma_drain();

  // ---------------------------------------------------------------- epilogue
  // Lane L holds, for each (slab mi, token block tb), the 8 consecutive
  // weight-side columns c .. c + 7 (c = 256 tm + 32 mi + 8 (L / 16);
  // acc[2 mi][tb] the first four, acc[2 mi + 1][tb] the last four) of token
  // t = tw + 16 tb + L % 16.  Branch-free: rows beyond the tensor fall outside
  // the buffer (loads give 0, stores are dropped) and columns beyond it get an
  // out-of-range offset.  Every load is issued before the first store: the
  // store and load counters are shared, so a load behind stores would wait for
  // all of them.
  const __amdgpu_buffer_rsrc_t ro = make_rsrc(out + tw * ldo, out == nullptr ? 0 : (Tvalid - tw) * ldo * 2);
  const int64_t cb0 = (int64_t)tm * kTile + 8 * q;
  // Per-token term, held as up to kMaxParts partial rows vstride apart and
  // summed here: s of the forward, rowsum(dY) of the input gradient.  The
  // four lanes of a token (L % 16 + 16 q) split the parts (lane q adds parts
  // q, q + 4, ..., in that order) and then exchange their sums: (q0 + q1) +
  // (q2 + q3) in every one of them, the same bits in all four.
  constexpr int kMaxParts = kMaxActChunks;  // s and rowsum(dY) have at most this many parts
  static_assert(kMaxParts % 4 == 0, "whole parts per lane");
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vecT + tw, ((int64_t)(vparts - 1) * vstride + Tvalid - tw) * 4);
  float vp[kMaxParts / 4][4], vt[4];
#pragma unroll
  for (int i = 0; i < kMaxParts / 4; ++i)
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      const int p = 4 * i + q;
      vp[i][tb] = p < vparts ? as_f(__builtin_amdgcn_raw_buffer_load_b32(rv, (int)((p * vstride + tb * 16 + c16) * 4),
                                                                        0, 0))
                             : 0.0f;
    }
#pragma unroll
  for (int tb = 0; tb < 4; ++tb) {
    float v = vp[0][tb];
#pragma unroll
    for (int i = 1; i < kMaxParts / 4; ++i) v += vp[i][tb];
    const float h = v + __shfl_xor(v, 16, 64);
    vt[tb] = h + __shfl_xor(h, 32, 64);
  }
  // Each accumulator is read out of its AGPR at its use, one ordered statement
  // per value (the drain's wait states cover them).  Left to the compiler, the
  // copies cluster at the loop exit: in the input gradient they then exceed
  // the register file with the epilogue's other values and spill to scratch;
  // ordered, the forward is 2.5 us and the input gradient 2 us shorter at
  // 4096^3.
  auto d8 = [&](int mi, int tb, int i) -> float {
    float r;
    asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(r) : "a"(i < 4 ? acc[2 * mi][tb][i] : acc[2 * mi + 1][tb][i - 4]));
    return r;
  };
  if constexpr (kMode == 0) {
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      const int tl = tb * 16 + c16;
#pragma unroll
      for (int mi = 0; mi < 8; ++mi) {
        const int64_t c = cb0 + mi * 32;
        const uint32_t off = c < Mvalid ? (uint32_t)(tl * ldo + c) * 2u : kOffNone;
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(d8(mi, tb, 2 * e) + vt[tb], d8(mi, tb, 2 * e + 1) + vt[tb]);
        __builtin_amdgcn_raw_buffer_store_b128(w, ro, off, 0, 0);
      }
    }
  } else {
    // X pairs in LDS (complete once this wave's loads are; the empty statement
    // keeps the compiler from moving the LDS reads above the wait)
    LCVQ_WAIT_VM_LGKM0(0);
    asm volatile("" ::: "memory");
    // The A^T map on the matrix cores: per slab and 16-token block, dX^T =
    // blockdiag(A) P^T, with M = output column c' (rows in slab_row order, so
    // lane L ends with c' = 8 (L / 16) + 0..7 of token L % 16, one 16-byte
    // store), N = token, K = the slab's 32 input columns c.  The B operand,
    // eight consecutive c of token L % 16 in lane L, is exactly what the lane
    // holds of P, so P never moves between lanes.  The A operand is the
    // constant block-diagonal map: lane L supplies row c' = slab_row(16 mb +
    // L % 16) at c = 8 (L / 16) + i, i.e. A[c' % D, c % D] when c' and c share
    // a group and 0 otherwise.  P and the map are each split into bf16 high
    // and low parts (x = hi + lo to 16 significant bits), and hi*hi + lo*hi +
    // hi*lo is summed in fp32 by the matrix core: dX is exact to about 2^-16
    // before its own bf16 rounding.  The accumulator starts at rs[t] b[c' % D].
    bf16x8 amh[2], aml[2];
    float bsel[2][4];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      const int cp = slab_row(16 * mb + c16);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int c = 8 * q + i;
        const float v = cp / D == c / D ? A[(cp % D) * D + (c % D)] : 0.0f;
        const __bf16 h = (__bf16)v;
        amh[mb][i] = h;
        aml[mb][i] = (__bf16)(v - (float)h);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) bsel[mb][e] = to_vgpr(bvec[(4 * mb + e) % D]);
    }
    // The map gradient on the matrix cores: dA[j, k] = sum over samples (t, g)
    // of X[t, g D + j] P[t, g D + k], a product with the samples as K.  Both
    // operands need a pair's samples along each lane's eight K values, i.e. the
    // pair tile transposed: X from its LDS pair, P (split into bf16 high and
    // low parts as for dX) after a pass through a two-pair LDS ring, both read
    // with the transposing LDS load.  Operand row r (M for X, N for P) holds,
    // at K = 8 G + i (G = lane / 16), element r % 8 of the 16-byte row of the
    // pair's lane 16 (2 (r / 8) + G / 2) + 8 (G % 2) + i.  For D = 8 that is
    // column r % 8 of the lane's group, so rows r < 8 and r >= 8 form two slots
    // of 32 samples each; for D = 4 it is column r % 4 of the lane's group
    // (r / 4) % 2: four slots.  One 16x16x32 instruction per pair and part, of
    // which the diagonal slot blocks (r / D == r' / D) are kept.  (Transposing
    // read: in each 16-lane group G, lane 4 e + u addresses row 16 (2 (u / 2)
    // + G / 2) + 8 (G % 2) + e, + 4 for the second read, at column 4 (u % 2);
    // output lane 4 u + w gets column 4 (u % 2) + w of the eight rows.)
    // db[j] = sum X[t, g D + j] rs[t] stays on the vector units.
    __shared__ __attribute__((aligned(1024))) char pst[kMode == 1 ? 4 * 2 * 2048 : 16];
    const int tq = c16 & 3, te = c16 >> 2;
    const int toff = 16 * (16 * (2 * (tq >> 1) + (q >> 1)) + 8 * (q & 1) + te) + 8 * (tq & 1);
    auto tr8 = [&](const char *base) {
      const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(base + toff));
      const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(base + toff + 64));
      return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    };
    floatx4 dah = floatx4{0.0f, 0.0f, 0.0f, 0.0f}, dal = dah;
    float gb[D];
#pragma unroll
    for (int j = 0; j < D; ++j) gb[j] = 0.0f;
#pragma unroll
    for (int p = 0; p < 32; ++p) {
      const int tb = p >> 3, mi = p & 7, tl = tb * 16 + c16;
      const char *xp = xs + (wave * kXPairs + p) * 1024;
      float y[8], pv8[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) pv8[i] = d8(mi, tb, i);
      u32x4 ph, pl;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ph[e] = pack_bf16x2(pv8[2 * e], pv8[2 * e + 1]);
        pl[e] = pack_bf16x2(pv8[2 * e] - bf16_lo(ph[e]), pv8[2 * e + 1] - bf16_hi(ph[e]));
      }
      const bf16x8 bh = __builtin_bit_cast(bf16x8, ph), bl = __builtin_bit_cast(bf16x8, pl);
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        floatx4 cacc;
#pragma unroll
        for (int e = 0; e < 4; ++e) cacc[e] = vt[tb] * bsel[mb][e];
        cacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(amh[mb], bh, cacc, 0, 0, 0);
        cacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aml[mb], bh, cacc, 0, 0, 0);
        cacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(amh[mb], bl, cacc, 0, 0, 0);
#pragma unroll
        for (int e = 0; e < 4; ++e) y[4 * mb + e] = cacc[e];
      }
      if (want_map) {
        char *pp = pst + (wave * 2 + (p & 1)) * 2048;
        *reinterpret_cast<u32x4 *>(pp + lane * 16) = ph;
        *reinterpret_cast<u32x4 *>(pp + 1024 + lane * 16) = pl;
        const bf16x8 xa = tr8(xp), pbh = tr8(pp), pbl = tr8(pp + 1024);
        dah = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa, pbh, dah, 0, 0, 0);
        dal = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa, pbl, dal, 0, 0, 0);
        const u32x4 xv = *reinterpret_cast<const u32x4 *>(xp + lane * 16);
#pragma unroll
        for (int e = 0; e < 8; ++e)
          gb[e % D] = fmaf((e & 1) ? bf16_hi(xv[e >> 1]) : bf16_lo(xv[e >> 1]), vt[tb], gb[e % D]);
      }
      const int64_t c = cb0 + mi * 32;
      const uint32_t off = c < Mvalid ? (uint32_t)(tl * ldo + c) * 2u : kOffNone;
      u32x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(y[2 * e], y[2 * e + 1]);
      __builtin_amdgcn_raw_buffer_store_b128(w, ro, off, 0, 0);
    }
    if (want_map) {
      // lane L holds rows 4 (L / 16) + 0..3 of column L % 16; slot blocks on the
      // diagonal go to LDS per wave and slot, db by shuffles; then the block's
      // sum of each entry, in a fixed order, to its place in mapp
      constexpr int kSlots = 16 / D;
      __shared__ float red[4][kSlots * D * D + D];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int mrow = 4 * q + e;
        if (mrow / D == c16 / D) red[wave][(mrow / D) * D * D + (mrow % D) * D + c16 % D] = dah[e] + dal[e];
      }
#pragma unroll
      for (int j = 0; j < D; ++j)
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) gb[j] += __shfl_xor(gb[j], o, 64);
      if (lane == 0) {
#pragma unroll
        for (int j = 0; j < D; ++j) red[wave][kSlots * D * D + j] = gb[j];
      }
      __syncthreads();
      if (tid < D * D + D) {
        float v = 0.0f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          if (tid < D * D) {
#pragma unroll
            for (int sl = 0; sl < kSlots; ++sl) v += red[w][sl * D * D + tid];
          } else {
            v += red[w][kSlots * D * D + tid - D * D];
          }
        }
        mapp[(int64_t)tid * gridDim.x + blockIdx.x] = v;
      }
    }
  }
}

// ============================================================================
// Weight-gradient product with the gradient-estimator epilogue:
//   D[c, r] = sum_t X'[t, c] dY[t, r] = (dW blockdiag(A))[r, c],  dZ = mask * D
// (straight-through), or dZ = mask * slope(Z) * D with mask and slope taken
// from Z (differentiable estimator of eq. dge, kDge)
// (X' = X blockdiag(A), so the map is already applied).  Both operands come
// pre-transposed in the token-K fragment layout.  16x16x32 matrix-core
// instructions.  Wave w owns in-features [64 w, 64 w + 64) of the block tile
// (two 32-row slabs, four 16-row blocks mb, A operand, streamed straight into
// registers) against all 256 out-features (sixteen 16-column blocks nb, B
// operand, shared by the four waves through four LDS stages filled by
// direct-to-LDS loads; each half-step's sixteen B reads are spread between the
// previous half-step's MFMAs, so the matrix core does not wait on LDS
// latency: 113 -> 104 us at 4096^3).  The slab rows are permuted (slab_row) so that lane L
// ends with in-features 8 (L / 16) .. + 7 of each slab for out-feature L % 16
// of each column block: whole groups, and 16 contiguous bytes of dZ.
// ============================================================================

template <bool kDge>
__global__ __launch_bounds__(256, 1) void k_gemm_dw(const uint16_t *__restrict__ xt, const uint16_t *__restrict__ dyt,
                                                    int KBt, const uint64_t *__restrict__ maskbits, int64_t nbc,
                                                    const uint16_t *__restrict__ Zb, Quantizer qz, int mask_mode,
                                                    GradEst est,
                                                    int accumulate, void *__restrict__ dZ, int dz_bf16, int m, int n,
                                                    int tiles_m, int tiles_n) {
  constexpr int kStage = 32 * 1024;  // eight 4 KiB B blocks
  __shared__ __attribute__((aligned(1024))) char lds[4 * kStage];

  const int tid = threadIdx.x, lane = tid & 63, q = lane >> 4, c16 = lane & 15;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int tm, tn;
  tile_of_block(tiles_m, tiles_n, tm, tn);
  const int c0 = tm * kTile, r0 = tn * kTile;

  // A: slabs tm * 8 + 2 * wave + mi; 4 KiB per (slab, step)
  const __amdgpu_buffer_rsrc_t rsA =
      make_rsrc(xt + (size_t)(tm * 8 + 2 * wave) * KBt * 2048, (int64_t)2 * KBt * 4096);
  // B: blocks tn * 8 + j; wave w copies blocks 2w, 2w + 1 (4 KiB each per step)
  const __amdgpu_buffer_rsrc_t rsB = make_rsrc(dyt + (size_t)(tn * 8) * KBt * 2048, (int64_t)8 * KBt * 4096);

  floatx4 acc[4][16];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[i][j] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
  acc_fence(acc);

  // Loads past the last step (the prefetch runs two or three steps ahead)
  // read the next slab's data or, past the buffer, zeros; the stages and
  // registers they fill are never used.  Unconditional loads keep the loop
  // free of branches, so the compiler's own waits stay pipelined.
  auto issue = [&](int st, int kb) {  // 8 direct-to-LDS loads per wave
    char *stage = lds + st * kStage;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int blk = 2 * wave + j;
#pragma unroll
      for (int ph = 0; ph < 4; ++ph)
        buffer_to_lds16(rsB, (lds_void *)(stage + (blk * 4 + ph) * 1024),
                        (uint32_t)(((blk * KBt + kb) * 4 + ph) * 1024 + lane * 16));
    }
  };
  // A fragments per (buffer, half-step kk2, slab mi, fh): fragment 2 fh + kk2
  // of the step.  Each half-step's four are reloaded as soon as its MFMAs have
  // been issued.
  u32x4 ca[2][2][2][2];
  auto load_a = [&](int buf, int kk2, int kb) {  // 4 loads per wave
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int fh = 0; fh < 2; ++fh)
        ca[buf][kk2][mi][fh] = __builtin_amdgcn_raw_buffer_load_b128(
            rsA, (int)(((mi * KBt + kb) * 4 + 2 * fh + kk2) * 1024 + lane * 16), 0, 0);
  };
  // B operands of one half-step, 16 column blocks; the reads of the next
  // half-step's operands are spread between this one's MFMAs.
  bf16x8 b0[16], b1[16];
  auto rd = [&](bf16x8 &dst, int st, int nb, int kk2) {
    dst = *reinterpret_cast<const bf16x8 *>(lds + st * kStage + ((nb >> 1) * 4 + 2 * (nb & 1) + kk2) * 1024 + lane * 16);
  };
  auto half = [&](int buf, int kk2, bf16x8 (&b)[16], bf16x8 (&nxt)[16], int rst, int rkk2) {
#pragma unroll
    for (int nb = 0; nb < 16; ++nb) {
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
        mfma16(acc[mb][nb], __builtin_bit_cast(bf16x8, ca[buf][kk2][mb >> 1][mb & 1]), b[nb]);
      rd(nxt[nb], rst, nb, rkk2);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Four LDS stages; B of step k in stage k % 4.  Per step k:
  //   first half-step's MFMAs (B read during the previous half-step), the
  //     reads of the second half-step's B between them; A loads of k + 2, kk2 0;
  //   wait (B of k + 1, own loads) + barrier (everyone's);
  //   B loads of k + 3 into the stage of step k - 1, which every wave has
  //     finished reading by then;
  //   second half-step's MFMAs, the reads of step k + 1's first B between them;
  //     A loads of k + 2, kk2 1.
  // The explicit waits count loads in this issue order, which the scheduling
  // fences keep inside the branch-free loop; the compiler may still sink the
  // prologue's A loads (used only in the loop) past the prologue's barrier, so
  // that wait does not rely on them.  The wait before a step's barrier lets the loads issued after
  // B of k + 1 stay in flight: A of k, kk2 1 and of k + 1, kk2 0, B of k + 2,
  // A of k + 1, kk2 1 and of k + 2, kk2 0 (24), less the four of A of k, kk2 1,
  // which the second half-step needs anyway; the same count covers steps 0 and
  // 1 after the prologue.  The prologue's wait (16) holds B of step 0 complete
  // wherever the A loads end up.
  // The loop runs from the barrier of one step to the wait of the next (the
  // last step's second half-step is peeled).  Its head thus comes before the
  // MFMAs that read A loaded a step earlier: at a loop head the compiler's own
  // waits do not count the previous trip's direct-to-LDS loads, and MFMAs
  // right after the head would wait for those too.
  issue(0, 0);
  load_a(0, 0, 0);
  load_a(0, 1, 0);
  __builtin_amdgcn_sched_barrier(0);
  issue(1, 1);
  load_a(1, 0, 1);
  load_a(1, 1, 1);
  __builtin_amdgcn_sched_barrier(0);
  issue(2, 2);
  __builtin_amdgcn_sched_barrier(0);
  LCVQ_WAIT_VM_LGKM0(16);
  LCVQ_BARRIER();
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int nb = 0; nb < 16; ++nb) rd(b0[nb], 0, nb, 0);
  __builtin_amdgcn_sched_barrier(0);
  half(0, 0, b0, b1, 0, 1);
  load_a(0, 0, 2);
  __builtin_amdgcn_sched_barrier(0);
  LCVQ_WAIT_VM(20);
  // from the barrier of step k to the wait of step k + 1 (u = k % 4)
  auto tail = [&](int u, int k, bool next) {
    LCVQ_BARRIER();
    __builtin_amdgcn_sched_barrier(0);
    issue((u + 3) & 3, k + 3);
    __builtin_amdgcn_sched_barrier(0);
    half(u & 1, 1, b1, b0, (u + 1) & 3, 0);
    load_a(u & 1, 1, k + 2);
    __builtin_amdgcn_sched_barrier(0);
    if (next) {
      half((u + 1) & 1, 0, b0, b1, (u + 1) & 3, 1);
      load_a((u + 1) & 1, 0, k + 3);
      __builtin_amdgcn_sched_barrier(0);
      LCVQ_WAIT_VM(20);
    }
  };
  int kb = 0;
  for (; kb + 4 < KBt; kb += 4) {
#pragma unroll
    for (int u = 0; u < 4; ++u) tail(u, kb + u, true);
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) tail(u, kb + u, u < 3);
  LCVQ_WAIT_VM_LGKM0(0);
  mfma_drain();

  // ------------------------------------------------ gradient-estimator epilogue
  // Lane L holds, for column block nb and slab mi, D[c .. c + 7, r] with
  // r = r0 + 16 nb + L % 16 and c = c0 + 64 w + 32 mi + 8 (L / 16):
  // acc[2 mi][nb] the first four, acc[2 mi + 1][nb] the last four.  dZ[r, c ..
  // c + 7] = mask * D, the mask read from the bitmap the backward prepass wrote
  // (one 64-bit word per row and wave: columns c0 + 64 w .. + 63; byte 4 mi +
  // L / 16 holds these eight); with kDge, mask and slope come from Z[r, c ..
  // c + 7] instead.  Rows r >= m fall outside the buffers; columns c >= n get
  // an out-of-range offset.  Every load (mask words or Z, and old dZ when
  // accumulating) of a column block is issued before the stores of the
  // previous one: loads and stores share one counter.
  // the bitmap tiles of rows r0 .. r0 + 255 (four 64-row bands of nbc tiles)
  const __amdgpu_buffer_rsrc_t rmk = make_rsrc((const char *)maskbits + (int64_t)(r0 / 64) * nbc * 2048,
                                               kDge ? 0 : ((int64_t)(m + 63) / 64 - r0 / 64) * nbc * 2048);
  const __amdgpu_buffer_rsrc_t rz = make_rsrc(Zb + (int64_t)r0 * n, kDge ? (int64_t)(m - r0) * n * 2 : 0);
  // this wave's 64 columns are word `wave` of each row of column block tm
  const int es = dz_bf16 ? 2 : 4;
  const __amdgpu_buffer_rsrc_t rg = make_rsrc((char *)dZ + (int64_t)r0 * n * es, (int64_t)(m - r0) * n * es);
  u32x2 mk[2];        // mask word of the row, per buffer
  u32x4 ov[2][2][2];  // old dZ per (buffer, mi, 16-byte half)
  u32x4 zv[2][2];     // kDge: Z[r, c .. c + 7] per (buffer, mi)
  auto eload = [&](int buf, int nb) {
    const int rl = nb * 16 + c16;
    if constexpr (kDge) {
#pragma unroll
      for (int mi = 0; mi < 2; ++mi) {
        const int c = c0 + 64 * wave + 32 * mi + 8 * q;
        zv[buf][mi] = __builtin_amdgcn_raw_buffer_load_b128(rz, c < n ? (uint32_t)(rl * n + c) * 2u : kOffNone, 0, 0);
      }
    } else {
      mk[buf] = __builtin_amdgcn_raw_buffer_load_b64(
          rmk, r0 + rl < m ? (int)((((rl >> 6) * nbc + tm) * 64 + (rl & 63)) * 32 + wave * 8) : (int)kOffNone, 0, 0);
    }
    if (!accumulate) return;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi) {
      const int c = c0 + 64 * wave + 32 * mi + 8 * q;
      const bool cv = c < n;
      const uint32_t e = (uint32_t)(rl * n + c);
      if (dz_bf16) {
        ov[buf][mi][0] = __builtin_amdgcn_raw_buffer_load_b128(rg, cv ? e * 2u : kOffNone, 0, 0);
      } else {
        ov[buf][mi][0] = __builtin_amdgcn_raw_buffer_load_b128(rg, cv ? e * 4u : kOffNone, 0, 0);
        ov[buf][mi][1] = __builtin_amdgcn_raw_buffer_load_b128(rg, cv ? e * 4u + 16u : kOffNone, 0, 0);
      }
    }
  };
  eload(0, 0);
#pragma unroll
  for (int nb = 0; nb < 16; ++nb) {
    const int buf = nb & 1;
    if (nb + 1 < 16) eload(buf ^ 1, nb + 1);
    const int rl = nb * 16 + c16;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi) {
      const int c = c0 + 64 * wave + 32 * mi + 8 * q;
      const bool cv = c < n;
      const uint32_t e = (uint32_t)(rl * n + c);
      float d8[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        d8[i] = acc[2 * mi][nb][i];
        d8[4 + i] = acc[2 * mi + 1][nb][i];
      }
      // (times the quantiser scale: the chain rule through the code-domain value)
      float g[8];
      if constexpr (kDge) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const uint32_t zw = zv[buf][mi][i >> 1];
          const float z = code_value((i & 1) ? bf16_hi(zw) : bf16_lo(zw), qz);
          g[i] = ste_pass(z, mask_mode) ? d8[i] * dge_slope(z, est) * qz.scale : 0.0f;
        }
      } else {
        const uint32_t mb = mk[buf][mi] >> (8 * q);
#pragma unroll
        for (int i = 0; i < 8; ++i) g[i] = ((mb >> i) & 1u) ? d8[i] * qz.scale : 0.0f;
      }
      if (dz_bf16) {
        if (accumulate) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            g[2 * i] += bf16_lo(ov[buf][mi][0][i]);
            g[2 * i + 1] += bf16_hi(ov[buf][mi][0][i]);
          }
        }
        u32x4 w;
#pragma unroll
        for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2(g[2 * i], g[2 * i + 1]);
        __builtin_amdgcn_raw_buffer_store_b128(w, rg, cv ? e * 2u : kOffNone, 0, 0);
      } else {
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          u32x4 w;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float v = g[4 * p + i];
            if (accumulate) v += as_f(ov[buf][mi][p][i]);
            w[i] = as_u(v);
          }
          __builtin_amdgcn_raw_buffer_store_b128(w, rg, cv ? e * 4u + 16u * p : kOffNone, 0, 0);
        }
      }
    }
  }
}

// ---- launchers -------------------------------------------------------------

hipError_t launch_fwd_bf16(const uint32_t *frag, const uint16_t *Xp, int64_t ldp, const float *s,
                           uint16_t *Y, int64_t N, int64_t m, int64_t n, hipStream_t st) {
  (void)n;
  const int tiles_m = (int)ceil_div(m, 2 * kTile), tiles_n = (int)ceil_div(N, kTile / 2);  // 512 x 128 tiles
  const int KB = (int)(ldp / kKStep);  // even: ldp is a multiple of 128
  const int64_t Np = round_up(N, kTile);  // row stride of the partial sums of s
  k_gemm_codes<0, 8><<<tiles_m * tiles_n, 256, 0, st>>>(frag, KB, Xp, 0, tiles_m, tiles_n, s,
                                                        act_chunks(ldp), Np, nullptr, nullptr, Y, m, m, N, nullptr, nullptr);
  return hipGetLastError();
}

hipError_t launch_dx_bf16(const uint32_t *frag, const uint16_t *dY, const float *rsp, const float *A, const float *b,
                          int d, uint16_t *dX, const uint16_t *X, float *mapp, int64_t N, int64_t m, int64_t n,
                          hipStream_t st) {
  const int parts = rowsum_parts(m);
  const int64_t Nt = bwd_tokens(N);  // row stride of the partial row sums
  const int tiles_m = (int)ceil_div(n, kTile), tiles_n = (int)ceil_div(N, kTile);
  const int KB = (int)(round_up(m, 128) / kKStep);  // even, matches the operand layout
  // dX == nullptr: the product still runs for dA/db; its stores are dropped.
  if (d == 8)
    k_gemm_codes<1, 8><<<tiles_m * tiles_n, 256, 0, st>>>(frag, KB, dY, m, tiles_m, tiles_n, rsp,
                                                          parts, Nt, A, b, dX, n, n, N, X, mapp);
  else
    k_gemm_codes<1, 4><<<tiles_m * tiles_n, 256, 0, st>>>(frag, KB, dY, m, tiles_m, tiles_n, rsp,
                                                          parts, Nt, A, b, dX, n, n, N, X, mapp);
  return hipGetLastError();
}

int map_rows(int64_t N, int64_t n) { return (int)(ceil_div(n, kTile) * ceil_div(N, kTile)); }

// Entry blockIdx.x of dA (< D D) or db: the sum of its `rows` per-block
// partial sums in a fixed order (thread i: rows i, i + 256, ...; then a
// butterfly over each wave and the four wave totals in order), plus the old
// value when accumulating.
__global__ __launch_bounds__(256) void k_map_combine(const float *__restrict__ mapp, int rows, int D, int accumulate,
                                                     float *__restrict__ dA, float *__restrict__ db) {
  __shared__ float part[4];
  const int e = blockIdx.x, tid = threadIdx.x;
  const float *src = mapp + (int64_t)e * rows;
  float v = 0.0f;
  for (int r = tid; r < rows; r += 256) v += src[r];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  if ((tid & 63) == 0) part[tid >> 6] = v;
  __syncthreads();
  if (tid == 0) {
    float *o = e < D * D ? dA + e : db + (e - D * D);
    const float t = (part[0] + part[1]) + (part[2] + part[3]);
    *o = (accumulate ? *o : 0.0f) + t;
  }
}

hipError_t launch_map_combine(const float *mapp, int rows, int d, int accumulate, float *dA, float *db,
                              hipStream_t st) {
  k_map_combine<<<d * d + d, 256, 0, st>>>(mapp, rows, d, accumulate, dA, db);
  return hipGetLastError();
}

hipError_t launch_dw_bf16(const uint16_t *xt, const uint16_t *dyt, const uint64_t *maskbits, const uint16_t *Z,
                          const Quantizer &qz, int mask_mode, const GradEst &est, int accumulate, void *dZ,
                          bool dz_bf16, int64_t N, int64_t m, int64_t n, hipStream_t st) {
  const int tiles_m = (int)ceil_div(n, kTile), tiles_n = (int)ceil_div(m, kTile);
  const int KBt = (int)(bwd_tokens(N) / 64);  // even
  if (est.dge)
    k_gemm_dw<true><<<tiles_m * tiles_n, 256, 0, st>>>(xt, dyt, KBt, nullptr, mask_col_blocks(n), Z, qz,
                                                       mask_mode, est, accumulate, dZ, dz_bf16 ? 1 : 0, (int)m, (int)n, tiles_m,
                                                       tiles_n);
  else
    k_gemm_dw<false><<<tiles_m * tiles_n, 256, 0, st>>>(xt, dyt, KBt, maskbits, mask_col_blocks(n), nullptr,
                                                        qz, mask_mode, est, accumulate, dZ, dz_bf16 ? 1 : 0, (int)m,
                                                        (int)n, tiles_m, tiles_n);
  return hipGetLastError();
}
}  // namespace lcvq
