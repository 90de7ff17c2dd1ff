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
constexpr int kThreads = 512;                    // 8 waves of 64: 2 (M) x 4 (N)
constexpr int kRowB = 128;                       // bytes of a tile row per K step
constexpr int kStages = 2;                       // LDS stages of the main loop
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// gfx9 buffer resource word 3 for raw (untyped) loads and stores.
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           kRsrcWord3);
}

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

// MFMA step on one 16-byte K slot of A (rows m) and B (rows n), 16x16 output
// block. The K order inside a slot only has to agree between A and B, which
// it does by construction: both fragments come from the same logical slot.
__device__ __forceinline__ f32x4_t mfma_slot(u32x4_t a, u32x4_t b, f32x4_t c, __bf16*) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mfma_slot(u32x4_t a, u32x4_t b, f32x4_t c, float*) {
  f32x4_t fa = __builtin_bit_cast(f32x4_t, a);
  f32x4_t fb = __builtin_bit_cast(f32x4_t, b);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[0], fb[0], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[1], fb[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[2], fb[2], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[3], fb[3], c, 0, 0, 0);
  return c;
}

// Accumulator layout of wave w (wm = w >> 2 in 0..1, wn = w & 3 in 0..3)
// after gemm_tile: acc.v[i][j][r] (i < 8, j < 4, r < 4) is C[m][n] with
//   m = wm*128 + 16*i + 4*(lane>>4) + r
//   n = wn*64 + 16*j + (lane&15)
// (the 16x16 MFMA output layout: lane holds column lane&15 of 4 rows).
struct AccTile {
  f32x4_t v[8][4];
};
__device__ __forceinline__ int acc_m(int wm, int i, int lane, int r) {
  return wm * 128 + 16 * i + 4 * (lane >> 4) + r;
}
__device__ __forceinline__ int acc_n(int wn, int j, int lane) { return wn * 64 + 16 * j + (lane & 15); }

// One 256x256 output tile: acc = A[m0:m0+256, k-range] * B[n0:n0+256, k-range]^T.
//
// ra / rb are buffer resources based at the tile's first row, sized so rows
// outside the operand read as zero (hardware range check). A K step is ROWB
// bytes of every row (ROWB = 64: 32 bf16 / 16 fp32). Operands go straight from
// memory into LDS (buffer loads with the LDS-DMA bit: no VGPR staging, no
// ds_write) through S stages, so S-1 K steps of operand data are in flight
// while one is consumed; one barrier per K step. The MFMA fragments of the
// next K sub-step are read while the current sub-step's MFMAs run. The
// caller's LDS must hold gemm_lds_bytes<ROWB, S>() bytes. Ends with a barrier,
// so the caller may reuse the LDS.
typedef __attribute__((address_space(3))) void lds_void_t;

template <int ROWB, int S>
constexpr int gemm_lds_bytes() { return S * 2 * kTile * ROWB; }
constexpr int kLdsMain = gemm_lds_bytes<kRowB, kStages>();  // 160 KiB

// 16-byte slot swizzle of a ROWB-byte tile row: conflict-free for the DMA
// rows and for 8- or 16-lane groups of MFMA fragment reads.
template <int ROWB>
__device__ __forceinline__ int slot_swz(int row) {
  if constexpr (ROWB == 128) return (row ^ (row >> 3)) & 7;
  else return ((row >> 1) ^ (row >> 3)) & 3;
}

// s_waitcnt vmcnt(n) for a compile-time n; expcnt/lgkmcnt are not waited.
#define KD_VMCNT(n) __builtin_amdgcn_s_waitcnt((0x0f70 & ~0x000f) | ((n) & 0xf) | (((n) >> 4) << 14))
template <typename T, int ROWB = kRowB, int S = kStages>
__device__ __forceinline__ void gemm_tile(__amdgpu_buffer_rsrc_t ra, int lda_bytes,
                                          __amdgpu_buffer_rsrc_t rb, int ldb_bytes, int ks_begin,
                                          int ks_end, char* lds, AccTile& acc) {
  constexpr int SL = ROWB / 16;           // 16-byte slots per row
  constexpr int SUB = SL / 4;             // MFMA sub-steps (64-byte K slices) per K step
  constexpr int OPB = kTile * ROWB;       // one operand's stage
  constexpr int STB = 2 * OPB;            // one stage (A and B)
  constexpr int RPI = 1024 / ROWB;        // rows per 1 KiB DMA instruction
  constexpr int NDMA = kTile / RPI / 8;   // DMA instructions per operand per wave
  constexpr int NI = 2 * NDMA;            // per K step per wave (vmcnt units)
  static_assert(SUB >= 2, "two or more sub-steps per K step");
  static_assert((S - 1) * NI <= 63, "vmcnt range of the in-flight DMA steps");
  static_assert(NDMA <= 8, "DMA offsets array");
  // (arrays captured by the lambdas below have literal bounds: clang's host
  // pass rejects a second instantiation when the bound is a dependent local)

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;

#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc.v[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int nsteps = ks_end - ks_begin;
  if (nsteps <= 0) {
    __syncthreads();
    return;
  }

  // DMA instruction q (= wave*NDMA + i) fills rows [RPI*q, RPI*(q+1)) of an
  // operand stage, 1 KiB contiguous: lane l lands at row RPI*q + l/SL,
  // physical slot l%SL, so it fetches logical slot (l%SL) ^ swz(row).
  uint32_t voffA[8], voffB[8];  // NDMA <= 8 used (fixed bound: see above)
#pragma unroll
  for (int i = 0; i < NDMA; ++i) {
    const int row = (wave * NDMA + i) * RPI + lane / SL;
    const uint32_t slot = (uint32_t)((lane % SL) ^ slot_swz<ROWB>(row));
    voffA[i] = (uint32_t)row * (uint32_t)lda_bytes + slot * 16u;
    voffB[i] = (uint32_t)row * (uint32_t)ldb_bytes + slot * 16u;
  }
  // fragment reads: 16x16 blocks; lane group g = lane>>4 reads logical slot
  // 4*s + g of row (block base + lane&15) in sub-step s.
  int rdA[8], fxA[8], rdB[4], fxB[4];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int ma = wm * 128 + 16 * i + (lane & 15);
    rdA[i] = ma * ROWB;
    fxA[i] = (lane >> 4) ^ slot_swz<ROWB>(ma);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int nb = wn * 64 + 16 * j + (lane & 15);
    rdB[j] = nb * ROWB;
    fxB[j] = (lane >> 4) ^ slot_swz<ROWB>(nb);
  }

  // DMA of K step ks into `stage`; past the last step the offset is made
  // out of range, so the hardware fills zeros without touching memory (the
  // schedule stays branch-free; those stages are never read).
  auto dma = [&](int ks, int stage) {
    char* a = lds + stage * STB;
    char* b = a + OPB;
    const uint32_t k0 = ks < ks_end ? (uint32_t)ks * ROWB : 0x80000000u;
#pragma unroll
    for (int i = 0; i < NDMA; ++i) {
      const int q = wave * NDMA + i;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void_t*)(a + q * 1024), 16,
                                               voffA[i] + k0, 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void_t*)(b + q * 1024), 16,
                                               voffB[i] + k0, 0, 0, 0);
    }
  };
  auto frag = [&](int stage, int s, u32x4_t (&fa)[8], u32x4_t (&fb)[4]) {
    const char* a = lds + stage * STB;
    const char* b = a + OPB;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      fa[i] = *reinterpret_cast<const u32x4_t*>(a + rdA[i] + ((fxA[i] ^ (4 * s)) << 4));
#pragma unroll
    for (int j = 0; j < 4; ++j)
      fb[j] = *reinterpret_cast<const u32x4_t*>(b + rdB[j] + ((fxB[j] ^ (4 * s)) << 4));
  };
  auto mfma32 = [&](const u32x4_t (&fa)[8], const u32x4_t (&fb)[4]) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc.v[i][j] = mfma_slot(fa[i], fb[j], acc.v[i][j], (T*)nullptr);
  };

  // Step j lives in stage j % S; S steps of DMA are always in flight. In
  // step j, each of the first SUB-1 sub-steps issues the next sub-step's 12
  // fragment reads interleaved with its 32 MFMAs. Then the wave waits for its
  // reads and for step j+1's DMA, the barrier publishes every wave's DMA and
  // retires stage j % S, and the last sub-step's MFMAs run interleaved with
  // the DMA of step j+S into that stage and the fragment reads of step j+1's
  // sub-step 0. Two waves per SIMD fill each other's waits.
#pragma unroll
  for (int p = 0; p < S; ++p) dma(ks_begin + p, p);
  KD_VMCNT((S - 1) * NI);
  __syncthreads();
  u32x4_t fa[2][8], fb[2][4];
  frag(0, 0, fa[0], fb[0]);
  int st = 0;
  for (int j = 0; j < nsteps; ++j) {
#pragma unroll
    for (int s = 0; s < SUB - 1; ++s) {
      frag(st, s + 1, fa[(s + 1) & 1], fb[(s + 1) & 1]);
      mfma32(fa[s & 1], fb[s & 1]);
#pragma unroll
      for (int q = 0; q < 12; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f & ~0x0f00);  // lgkmcnt(0)
    KD_VMCNT((S - 2) * NI);
    __syncthreads();
    const int nst = st + 1 == S ? 0 : st + 1;
    dma(ks_begin + j + S, st);
    frag(nst, 0, fa[SUB & 1], fb[SUB & 1]);
    mfma32(fa[(SUB - 1) & 1], fb[(SUB - 1) & 1]);
#pragma unroll
    for (int q = 0; q < 12; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMA
      if (q < NI) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read (DMA)
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    __builtin_amdgcn_sched_barrier(0);
    st = nst;
    if constexpr ((SUB & 1) != 0) {
      // odd sub-step count: next step's sub-step 0 landed in buffer 1
#pragma unroll
      for (int i = 0; i < 8; ++i) fa[0][i] = fa[1][i];
#pragma unroll
      for (int i = 0; i < 4; ++i) fb[0][i] = fb[1][i];
    }
  }
  KD_VMCNT(0);
  __syncthreads();
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
