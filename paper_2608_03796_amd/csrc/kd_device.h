// Device-side building blocks for gfx950 (CDNA4): vector types, buffer
// resources, the XCD-aware tile order, and the 256x256 MFMA GEMM main loop
// shared by the logits, logit-recompute, dH and dW kernels.
//
// GEMM convention: C[M, N] = A[M, K] * B[N, K]^T with both operands stored
// row-major with K contiguous ("NT"). Every contraction on the hot path is
// issued in this form; the operands that are not naturally K-contiguous (W for
// dH, the chunk's hidden rows and dZ for dW) are supplied as transposed copies.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kd {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4_t;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2_t;

constexpr int kTile = 256;                       // BM = BN
constexpr int kThreads = 256;                    // 4 waves of 64, 2 x 2
constexpr int kRowBytes = 128;                   // one tile row per K step
constexpr int kStageBytes = kTile * kRowBytes;   // 32 KiB per operand
constexpr int kLdsMain = 4 * kStageBytes;        // A, B x 2 stages = 128 KiB
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// gfx9 buffer resource word 3 for raw (untyped) loads and stores.
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           kRsrcWord3);
}

// 16-byte slot swizzle of the main-loop tiles (8 slots per 128-byte row):
// conflict-free for the row-parallel LDS writes and the MFMA fragment reads.
__device__ __forceinline__ int swz8(int row) { return (row ^ (row >> 3)) & 7; }

// Workgroups are dispatched round-robin over the 8 XCDs (pid % 8). Give each
// XCD a contiguous range of the linear tile order, so the ~32 tiles an XCD runs
// at once are neighbours and share operand rows in that XCD's L2; inside the
// order, tiles are grouped gm at a time along M.
__device__ __forceinline__ void tile_coords(int pid, int TM, int TN, int gm, int& mt, int& nt) {
  const int T = TM * TN;
  const int q = T >> 3, r = T & 7;
  const int x = pid & 7, k = pid >> 3;
  const int L = x * q + (x < r ? x : r) + k;
  const int per_group = gm * TN;
  const int g = L / per_group;
  const int first_m = g * gm;
  const int gs = (TM - first_m) < gm ? (TM - first_m) : gm;
  const int rem = L - g * per_group;
  mt = first_m + rem % gs;
  nt = rem / gs;
}

template <typename T>
struct Elt;
template <>
struct Elt<__bf16> {
  static constexpr int bytes = 2;
};
template <>
struct Elt<float> {
  static constexpr int bytes = 4;
};

// MFMA step on one 16-byte K slot of A (rows m) and B (rows n). The K order
// inside a slot only has to agree between A and B, which it does by
// construction: both fragments come from the same logical slot.
__device__ __forceinline__ f32x16_t mfma_slot(u32x4_t a, u32x4_t b, f32x16_t c, __bf16*) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x16_t mfma_slot(u32x4_t a, u32x4_t b, f32x16_t c, float*) {
  f32x4_t fa = __builtin_bit_cast(f32x4_t, a);
  f32x4_t fb = __builtin_bit_cast(f32x4_t, b);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[0], fb[0], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[1], fb[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[2], fb[2], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[3], fb[3], c, 0, 0, 0);
  return c;
}

// Accumulator layout of one wave (wm, wn) after gemm_tile: acc[i][j][r] is
// C[m][n] with
//   m = wm*128 + 32*i + 8*(r>>2) + 4*(lane>>5) + (r&3)
//   n = wn*128 + 32*j + (lane&31)
// (the 32x32 MFMA output layout: lane holds column lane&31, 4 groups of 4 rows).
struct AccTile {
  f32x16_t v[4][4];
};

// One 256x256 output tile: acc = A[m0:m0+256, k-range] * B[n0:n0+256, k-range]^T.
// ra / rb are buffer resources based at the tile's first row, sized so rows
// outside the operand read as zero (hardware range check). K steps are 128
// bytes of a row (64 bf16 or 32 fp32). Double-buffered LDS, one barrier per
// K step; the caller's LDS must hold kLdsMain bytes. Ends with a barrier, so
// the caller may reuse the LDS.
template <typename T>
__device__ __forceinline__ void gemm_tile(__amdgpu_buffer_rsrc_t ra, int lda_bytes,
                                          __amdgpu_buffer_rsrc_t rb, int ldb_bytes, int ks_begin,
                                          int ks_end, char* lds, AccTile& acc) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc.v[i][j][r] = 0.0f;

  if (ks_end <= ks_begin) {
    __syncthreads();
    return;
  }

  // global -> LDS: thread loads slot (tid&7) of rows (tid>>3) + 32*i
  const int lrow = tid >> 3;
  const int lslot = tid & 7;
  // byte offsets are unsigned 32-bit (the buffer instruction's offset type)
  const uint32_t voffA = (uint32_t)lrow * (uint32_t)lda_bytes + lslot * 16u;
  const uint32_t voffB = (uint32_t)lrow * (uint32_t)ldb_bytes + lslot * 16u;
  int ldsw[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int row = lrow + 32 * i;
    ldsw[i] = row * kRowBytes + ((lslot ^ swz8(row)) << 4);
  }
  // fragment reads: A row m = wm*128 + 32*i + (lane&31), logical slot
  // 4*(lane>>5) + s for K sub-step s.
  int rdA[4], rdB[4], fxA[4], fxB[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ma = wm * 128 + 32 * i + (lane & 31);
    const int nb = wn * 128 + 32 * i + (lane & 31);
    rdA[i] = ma * kRowBytes;
    rdB[i] = nb * kRowBytes;
    fxA[i] = (4 * (lane >> 5)) ^ swz8(ma);
    fxB[i] = (4 * (lane >> 5)) ^ swz8(nb);
  }

  u32x4_t sa[8], sb[8];
  auto gload = [&](int ks) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      // all offsets in the VGPR offset (soffset = 0) so the hardware range
      // check sees the full offset and returns zeros past the operand's rows
      const uint32_t ka = voffA + 32u * i * (uint32_t)lda_bytes + (uint32_t)ks * kRowBytes;
      const uint32_t kb = voffB + 32u * i * (uint32_t)ldb_bytes + (uint32_t)ks * kRowBytes;
      sa[i] = __builtin_amdgcn_raw_buffer_load_b128(ra, (int)ka, 0, 0);
      sb[i] = __builtin_amdgcn_raw_buffer_load_b128(rb, (int)kb, 0, 0);
    }
  };
  auto lstore = [&](int stage) {
    char* a = lds + stage * (2 * kStageBytes);
    char* b = a + kStageBytes;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      *reinterpret_cast<u32x4_t*>(a + ldsw[i]) = sa[i];
      *reinterpret_cast<u32x4_t*>(b + ldsw[i]) = sb[i];
    }
  };
  auto compute = [&](int stage) {
    const char* a = lds + stage * (2 * kStageBytes);
    const char* b = a + kStageBytes;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      u32x4_t fa[4], fb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        fa[i] = *reinterpret_cast<const u32x4_t*>(a + rdA[i] + ((fxA[i] ^ s) << 4));
        fb[i] = *reinterpret_cast<const u32x4_t*>(b + rdB[i] + ((fxB[i] ^ s) << 4));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc.v[i][j] = mfma_slot(fa[i], fb[j], acc.v[i][j], (T*)nullptr);
    }
  };

  gload(ks_begin);
  lstore(0);
  __syncthreads();
  for (int ks = ks_begin; ks < ks_end; ++ks) {
    const int stage = (ks - ks_begin) & 1;
    const bool more = ks + 1 < ks_end;
    if (more) gload(ks + 1);
    compute(stage);
    if (more) lstore(stage ^ 1);
    __syncthreads();
  }
}

// ---------------------------------------------------------------- wave ops --
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  return x;
}
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// round-to-nearest-even fp32 -> bf16 bits
__device__ __forceinline__ uint32_t bf16_bits(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  if ((u & 0x7f800000u) == 0x7f800000u) return (u >> 16) | ((u & 0xffffu) ? 0x40u : 0u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return bf16_bits(lo) | (bf16_bits(hi) << 16);
}

}  // namespace kd
