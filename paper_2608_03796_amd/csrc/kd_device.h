// Device-side building blocks for gfx950 (CDNA4): vector types, buffer
// resources, the XCD-aware tile order, and the 256x256 MFMA GEMM main loop
// shared by the logits, logit-recompute, dH and dW kernels.
//
// GEMM convention: C[M, N] = A[M, K] * B[N, K]^T. Each operand is read where it
// lives, either with K contiguous along its rows (W and the hidden rows for the
// logits, dZ for dH) or with K along its columns (W for dH, dZ and the hidden
// rows for dW); no operand is copied or transposed in memory.
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
typedef __attribute__((ext_vector_type(4))) int i32x4_t;  // buffer resource in 4 SGPRs

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

// Index of the calling wave in its workgroup, as a wave-uniform (scalar) value:
// loops and branches on it stay scalar instead of running under an exec mask.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
}

// Workgroups are dispatched round-robin over the 8 XCDs (pid % 8). Give each
// XCD a contiguous range of the linear tile order, so the ~32 tiles an XCD runs
// at once are neighbours and share operand rows in that XCD's L2; inside the
// order, tiles are grouped gm at a time along M.
// tile_order_xcd maps pid < n to a position in [0, n) of that order; tile_at
// maps a position to the tile (mt, nt).
__device__ __forceinline__ int tile_order_xcd(int pid, int n) {
  const int q = n >> 3, r = n & 7;
  const int x = pid & 7, k = pid >> 3;
  return x * q + (x < r ? x : r) + k;
}
__device__ __forceinline__ void tile_at(int L, int TM, int TN, int gm, int& mt, int& nt) {
  const int per_group = gm * TN;
  const int g = L / per_group;
  const int first_m = g * gm;
  const int gs = (TM - first_m) < gm ? (TM - first_m) : gm;
  const int rem = L - g * per_group;
  mt = first_m + rem % gs;
  nt = rem / gs;
}
__device__ __forceinline__ void tile_coords(int pid, int TM, int TN, int gm, int& mt, int& nt) {
  tile_at(tile_order_xcd(pid, TM * TN), TM, TN, gm, mt, nt);
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

// A 256x256 tile is computed by NW waves: 8 waves in a 2 (M) x 4 (N) grid,
// each 128x64, or 4 waves in a 2 x 2 grid, each 128x128 (its accumulators
// then live in the AGPR half of the register file). Accumulator layout of wave
// w (wm = w / (NW/2), wn = w % (NW/2)) after gemm_tile: acc.v[i][j][r]
// (i < 8, j < NJ, r < 4) is C[m][n] with
//   m = wm*128 + 16*i + 4*(lane>>4) + r
//   n = wn*16*NJ + 16*j + (lane&15)
// (the 16x16 MFMA output layout: lane holds column lane&15 of 4 rows).
template <int NW>
struct WaveGrid {
  static_assert(NW == 8 || NW == 4, "8 or 4 waves per 256x256 tile");
  static constexpr int NJ = 32 / NW;         // 16-column blocks per wave
  static constexpr int NPW = 32 / NW;        // DMA instructions per wave per operand step
  __device__ static int wm(int wave) { return wave >> (NW == 8 ? 2 : 1); }
  __device__ static int wn(int wave) { return wave & (NW / 2 - 1); }
};
template <int NJ>
struct AccTileT {
  f32x4_t v[8][NJ];
};
typedef AccTileT<4> AccTile;  // 8-wave tiles
__device__ __forceinline__ int acc_m(int wm, int i, int lane, int r) {
  return wm * 128 + 16 * i + 4 * (lane >> 4) + r;
}
template <int NJ = 4>
__device__ __forceinline__ int acc_n(int wn, int j, int lane) {
  return wn * 16 * NJ + 16 * j + (lane & 15);
}

// One 256x256 output tile: acc = A[m0:m0+256, k-range] * B[n0:n0+256, k-range]^T.
//
// Each operand is stored in one of two layouts:
//  * K-contiguous (KcOp): rows are the tile's 256 M (or N) indices, K runs
//    along the row; a K step is 128 bytes of each row. `base` points at the
//    tile's first row and `bytes` covers only the rows that exist, so missing
//    rows read as zeros (hardware range check).
//  * K-major (KmOp): rows are K indices and the tile's 256 M (or N) indices run
//    along the row; a K step is 128/sizeof(T) rows of 256 elements. `base`
//    points at the tile's first column of K row 0 and `bytes` counts the bytes
//    from there to the end of the last K row that exists; the resource is
//    re-based every K step, so K rows past the end read as zeros and offsets
//    stay 32-bit for any operand size. The MFMA fragments are read with
//    transposing LDS reads (ds_read_b64_tr_b16: inside a 16-lane group, lane i
//    gets element i%4 of the 8 bytes addressed by lane 4k + i/4 as its value
//    k), so W, dZ and the hidden rows are consumed where they are.
// Operands go straight from memory into LDS (buffer loads with the LDS-DMA
// bit) through stages of 32 KiB per operand (two per operand, or three for A
// and two for B); one barrier per K step; the next sub-step's fragments are
// read while the current sub-step's MFMAs run. The caller's LDS must hold
// kLdsMain bytes (kLdsA3 with SA = 3); ends with a barrier.
//
// The DMA loads are issued from inline assembly, so the compiler does not
// track them: it would otherwise make every transposing LDS read wait for all
// DMA in flight (those reads carry no alias information), which serialises the
// prefetch of step j+2 with the reads of step j+1. Completion is ordered by
// hand instead: s_waitcnt vmcnt before each barrier that publishes a stage.
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short s16x4_t;
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

constexpr int kLdsMain = kStages * 2 * kTile * kRowB;  // 128 KiB
constexpr int kLdsA3 = 5 * kTile * kRowB;              // 160 KiB: 3 A stages + 2 B stages

struct KcOp {
  const char* base;
  uint32_t bytes;
  int ld;  // row pitch in bytes
};
struct KmOp {
  const char* base;
  int64_t bytes;
  int ld;  // row pitch in bytes
};

// 16-byte slot swizzles of the LDS stages. The DMA writes whole 1 KiB runs
// (conflict-free for any permutation); the swizzles make the fragment reads
// conflict-free. The K-contiguous pattern was chosen by measurement
// (SQ_LDS_BANK_CONFLICT and read throughput of the exact fragment-read
// pattern): XOR of the slot with row % 8 reads at full rate, while
// (row ^ row/8) % 8, which a 16-consecutive-lane bank model also predicts to
// be conflict-free, measured 2-way.
// K-contiguous rows: 128 bytes, 8 slots.
__device__ __forceinline__ int swz_kc(int row) { return row & 7; }
// K-major bf16 rows (512 bytes, 32 slots): a transposing read covers slot
// pairs of rows r..r+3 and r+8..r+11, which get 8 distinct even XOR values.
__device__ __forceinline__ int swz_km16(int row) {
  return ((row & 3) | (((row >> 3) & 1) << 2)) << 1;
}
// K-major fp32 rows (1 KiB, 64 slots): a 32-bit read covers 4 slots of rows
// r, r+4, r+8, r+12, which get the XOR values 0, 4, 8, 12.
__device__ __forceinline__ int swz_km32(int row) { return ((row >> 2) & 3) << 2; }

// s_waitcnt vmcnt(n) for a compile-time n; expcnt/lgkmcnt are not waited.
#define KD_VMCNT(n) __builtin_amdgcn_s_waitcnt((0x0f70 & ~0x000f) | ((n) & 0xf) | (((n) >> 4) << 14))

constexpr uint32_t kOobOffset = 0xfffffff0u;  // past every resource: DMA writes zeros

// Raw buffer resource (stride 0, 32-bit range) in scalar registers.
__device__ __forceinline__ i32x4_t rsrc_words(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  return i32x4_t{__builtin_amdgcn_readfirstlane((int)(uint32_t)a),
                 __builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32)),
                 __builtin_amdgcn_readfirstlane((int)bytes), kRsrcWord3};
}

// One wave-wide 16-byte-per-lane LDS-DMA load: lane i's 16 bytes at voffset
// land at LDS byte address lds_addr + 16 i. M0 is set in the same statement;
// an LDS-DMA instruction must not directly follow an SALU write of M0 (one
// wait state), hence the s_nop.
__device__ __forceinline__ void dma_b128(i32x4_t r, uint32_t lds_addr, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds_addr), "v"(voff), "s"(r)
               : "memory");
}
// 4-byte-per-lane LDS-DMA load: lane i's dword at voffset lands at lds_addr + 4 i.
__device__ __forceinline__ void dma_b32(i32x4_t r, uint32_t lds_addr, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds"
               :
               : "s"(lds_addr), "v"(voff), "s"(r)
               : "memory");
}
__device__ __forceinline__ uint32_t lds_addr(const char* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)p;
}

// DMA of one operand's K step: 4 instructions of 1 KiB per wave. prep()
// computes the step's resource, LDS address and offsets; one(i) issues
// instruction i.
template <int NPW>
struct DmaStep {
  i32x4_t r;
  uint32_t la;
  uint32_t off[NPW];
  __device__ __forceinline__ void one(int i) const { dma_b128(r, la + i * 1024, off[i]); }
};

// An operand's 32 KiB stage is 32 instructions of 1 KiB; wave w issues
// instructions w*NPW .. w*NPW + NPW - 1.
template <typename T, typename Op, int NPW>
struct OpDma;

template <typename T, int NPW>
struct OpDma<T, KcOp, NPW> {
  uint32_t voff[NPW];
  i32x4_t r;
  __device__ __forceinline__ void init(const KcOp& op, int wave, int lane) {
    r = rsrc_words(op.base, op.bytes);
    // 8 rows of 128 bytes per instruction: lane -> row 8q + lane/8, slot lane%8
#pragma unroll
    for (int i = 0; i < NPW; ++i) {
      const int row = (wave * NPW + i) * 8 + (lane >> 3);
      voff[i] = (uint32_t)row * (uint32_t)op.ld + (uint32_t)(((lane & 7) ^ swz_kc(row)) << 4);
    }
  }
  __device__ __forceinline__ DmaStep<NPW> prep(const KcOp&, char* stage, int wave, int ks,
                                               bool live) const {
    DmaStep<NPW> d;
    d.r = r;
    d.la = __builtin_amdgcn_readfirstlane(lds_addr(stage) + wave * NPW * 1024);
#pragma unroll
    for (int i = 0; i < NPW; ++i)
      d.off[i] = live ? voff[i] + (uint32_t)ks * (uint32_t)kRowB : kOobOffset;
    return d;
  }
};

template <typename T, int NPW>
struct OpDma<T, KmOp, NPW> {
  static constexpr int KS = kRowB / (int)sizeof(T);  // K rows per step
  uint32_t voff[NPW];
  __device__ __forceinline__ void init(const KmOp& op, int wave, int lane) {
#pragma unroll
    for (int i = 0; i < NPW; ++i) {
      if constexpr (sizeof(T) == 2) {
        // 2 K rows of 512 bytes per instruction: lane -> row 2q + lane/32, slot lane%32
        const int row = (wave * NPW + i) * 2 + (lane >> 5);
        voff[i] = (uint32_t)row * (uint32_t)op.ld + (uint32_t)(((lane & 31) ^ swz_km16(row)) << 4);
      } else {
        // 1 K row of 1 KiB per instruction: lane -> slot lane
        const int row = wave * NPW + i;
        voff[i] = (uint32_t)row * (uint32_t)op.ld + (uint32_t)((lane ^ swz_km32(row)) << 4);
      }
    }
  }
  __device__ __forceinline__ DmaStep<NPW> prep(const KmOp& op, char* stage, int wave, int ks,
                                               bool live) const {
    const int64_t step0 = (int64_t)ks * KS * op.ld;
    int64_t left = op.bytes - step0;
    left = left < 0 ? 0 : (left > 0x7fffffff ? 0x7fffffff : left);
    DmaStep<NPW> d;
    d.r = rsrc_words(op.base + step0, (uint32_t)left);
    d.la = __builtin_amdgcn_readfirstlane(lds_addr(stage) + wave * NPW * 1024);
#pragma unroll
    for (int i = 0; i < NPW; ++i) d.off[i] = live ? voff[i] : kOobOffset;
    return d;
  }
};

// Fragment reads of NB blocks of 16 rows (M or N) from `base` within the tile.
// Sub-step s of a K step covers K elements [s*KS/2, (s+1)*KS/2) of the step;
// lane (g = lane/16, j = lane%16) holds row base + 16b + j with K elements
// s*KS/2 + 8g + 0..7 (bf16) or s*KS/2 + 4g + 0..3 (fp32), in both layouts.
template <typename T, typename Op, int NB>
struct OpFrag;

template <typename T, int NB>
struct OpFrag<T, KcOp, NB> {
  static constexpr int kReads = NB;
  int rd[NB], fx[NB];
  __device__ __forceinline__ void init(int base, int lane) {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int m = base + 16 * b + (lane & 15);
      rd[b] = m * kRowB;
      fx[b] = (lane >> 4) ^ swz_kc(m);
    }
  }
  __device__ __forceinline__ u32x4_t one(const char* op, int s, int b) const {
    return *reinterpret_cast<const u32x4_t*>(op + rd[b] + ((fx[b] ^ (4 * s)) << 4));
  }
};

template <int NB>
struct OpFrag<__bf16, KmOp, NB> {
  static constexpr int kReads = 2 * NB;
  static constexpr int kRow = kTile * 2;  // bytes of a K row in LDS
  int off[NB];                            // byte offset at sub-step 0, h = 0
  __device__ __forceinline__ void init(int base, int lane) {
    // lane j of group g points at K row 8g + j/4 (+ 32s + 4h), columns
    // base + 16b + 4(j%4) .. +3, so lane i receives columns base + 16b + i
    const int g = lane >> 4, j = lane & 15;
    const int row = 8 * g + (j >> 2);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int col = base + 16 * b + 4 * (j & 3);
      off[b] = row * kRow + (((col >> 3) ^ swz_km16(row)) << 4) + ((col & 4) << 1);
    }
  }
  __device__ __forceinline__ u32x4_t one(const char* op, int s, int b) const {
    u32x2_t h0 = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                                 (lds_s16x4_t*)(op + off[b] + 32 * s * kRow)));
    u32x2_t h1 = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                                 (lds_s16x4_t*)(op + off[b] + (32 * s + 4) * kRow)));
    return u32x4_t{h0[0], h0[1], h1[0], h1[1]};
  }
};

template <int NB>
struct OpFrag<float, KmOp, NB> {
  static constexpr int kReads = 4 * NB;
  static constexpr int kRow = kTile * 4;
  int off[NB];  // byte offset of K row 4g, sub-step 0
  __device__ __forceinline__ void init(int base, int lane) {
    const int g = lane >> 4, j = lane & 15;
    const int row = 4 * g;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int col = base + 16 * b + j;
      off[b] = row * kRow + (((col >> 2) ^ swz_km32(row)) << 4) + ((col & 3) << 2);
    }
  }
  __device__ __forceinline__ u32x4_t one(const char* op, int s, int b) const {
    // K rows 16s + 4g + e share row 4g's swizzle (it depends on (row/4) % 4 only)
    uint32_t v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      v[e] = *reinterpret_cast<const uint32_t*>(op + off[b] + (16 * s + e) * kRow);
    return u32x4_t{v[0], v[1], v[2], v[3]};
  }
};

// SPREAD selects the fragment-read placement: false puts sub-step 1's reads
// under the compiler's MFMA/read interleave (by hand, one per pair, with
// SA = 3) and sub-step 0's reads on the first pairs of the second half; true
// places both by hand, fragment f with pair f * NP / (8 + NJ). Which one is
// faster depends on the operand layouts (measured per kernel). SA is the
// number of A stages: 2 (all DMA of a step in its second half) or 3 (the DMA
// split between the halves; 160 KiB of LDS).
template <typename T, typename OA, typename OB, int NW = 8, bool SPREAD = false, int SA = 2>
__device__ __forceinline__ void gemm_tile(const OA& opa, const OB& opb, int ks_begin, int ks_end,
                                          char* lds, AccTileT<WaveGrid<NW>::NJ>& acc) {
  typedef WaveGrid<NW> WG;
  constexpr int NJ = WG::NJ, NPW = WG::NPW;
  constexpr int S = kStages;
  constexpr int OPB = kTile * kRowB;  // one operand's stage (32 KiB)
  constexpr int STB = 2 * OPB;        // one stage (A and B)
  constexpr int NI = 2 * NPW;         // DMA instructions per K step per wave
  constexpr int NP = 4 * NJ;          // MFMA pairs per sub-step
  constexpr int RD = OpFrag<T, OA, 8>::kReads + OpFrag<T, OB, NJ>::kReads;
  constexpr int RQ = (RD + NP - 1) / NP;  // LDS reads per MFMA pair in sub-step 0
  static_assert((S - 1) * NI <= 63, "vmcnt range of the in-flight DMA steps");
  static_assert(2 * NI == NP, "one DMA instruction on every other MFMA pair");

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = wave_id();
  const int wm = WG::wm(wave), wn = WG::wn(wave);

#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc.v[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int nsteps = ks_end - ks_begin;
  if (nsteps <= 0) {
    __syncthreads();
    return;
  }

  OpDma<T, OA, NPW> da;
  OpDma<T, OB, NPW> db;
  da.init(opa, wave, lane);
  db.init(opb, wave, lane);
  OpFrag<T, OA, 8> fra;
  OpFrag<T, OB, NJ> frb;
  fra.init(wm * 128, lane);
  frb.init(wn * 16 * NJ, lane);

  auto frag = [&](int stage, int s, u32x4_t (&fa)[8], u32x4_t (&fb)[NJ]) {
    const char* a = lds + stage * STB;
#pragma unroll
    for (int b = 0; b < 8; ++b) fa[b] = fra.one(a, s, b);
#pragma unroll
    for (int b = 0; b < NJ; ++b) fb[b] = frb.one(a + OPB, s, b);
  };
  // pair q: row block i = q / (NJ/2), two column blocks, in a snake order (odd
  // rows right to left) so that consecutive MFMAs change one operand only
  // (the fewest operand changes; measured ~0.8% faster per step than
  // restarting every row at column 0)
  auto mfma2 = [&](int q, const u32x4_t (&fa)[8], const u32x4_t (&fb)[NJ]) {
    const int i = q / (NJ / 2), jj = 2 * (q % (NJ / 2));
    const int j0 = (i & 1) ? NJ - 1 - jj : jj, j1 = (i & 1) ? NJ - 2 - jj : jj + 1;
    acc.v[i][j0] = mfma_slot(fa[i], fb[j0], acc.v[i][j0], (T*)nullptr);
    acc.v[i][j1] = mfma_slot(fa[i], fb[j1], acc.v[i][j1], (T*)nullptr);
  };

  if constexpr (SA == 3) {
    // Three A stages and two B stages (160 KiB): step k's A operand lives in
    // A stage k % 3 and its B operand in B stage k % 2. Step j+2's A DMA goes
    // out during step j's first half (into the A stage retired at barrier
    // j-1), its B DMA during step j's second half (into the B stage retired at
    // barrier j), so each half issues half of the step's DMA (the per-CU
    // DMA issue rate is what limited the half that carried all of it) and the
    // A half has ~1.4 steps to land; both are waited for at barrier j+1. The
    // instructions go on every fourth MFMA pair, A's on pairs 3, 7, 11, 15 and
    // B's on pairs 0, 4, 8, 12 (measured best of the placements tried).
    constexpr int DS = NP / NPW;  // pairs per DMA instruction
    char* const lb = lds + 3 * OPB;
    auto aS = [&](int k3) { return lds + k3 * OPB; };
    auto bS = [&](int k2) { return lb + k2 * OPB; };
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const bool live = ks_begin + p < ks_end;
      const DmaStep<NPW> sa = da.prep(opa, aS(p), wave, ks_begin + p, live);
      const DmaStep<NPW> sb = db.prep(opb, bS(p), wave, ks_begin + p, live);
#pragma unroll
      for (int i = 0; i < NPW; ++i) sa.one(i);
#pragma unroll
      for (int i = 0; i < NPW; ++i) sb.one(i);
    }
    KD_VMCNT(NI);
    __syncthreads();
    u32x4_t fa[2][8], fb[2][NJ];
#pragma unroll
    for (int b = 0; b < 8; ++b) fa[0][b] = fra.one(aS(0), 0, b);
#pragma unroll
    for (int b = 0; b < NJ; ++b) fb[0][b] = frb.one(bS(0), 0, b);
    constexpr int NF3 = 8 + NJ;
    auto read3 = [&](int q, const char* a, const char* b, int s, u32x4_t (&xa)[8],
                     u32x4_t (&xb)[NJ]) {
#pragma unroll
      for (int f = 0; f < NF3; ++f)
        if ((SPREAD ? (f * NP) / NF3 : f) == q) {
          if (f < 8) xa[f] = fra.one(a, s, f);
          else xb[f - 8] = frb.one(b, s, f - 8);
        }
    };
    int ca = 0, cb = 0;  // A and B stages of step j
    for (int j = 0; j < nsteps; ++j) {
      const int ks = ks_begin + j + 2;
      {
        const DmaStep<NPW> sa = da.prep(opa, aS(ca == 0 ? 2 : ca - 1), wave, ks, ks < ks_end);
        const char* a = aS(ca);
        const char* b = bS(cb);
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          if (q % DS == DS - 1) sa.one(q / DS);
          mfma2(q, fa[0], fb[0]);
          read3(q, a, b, 1, fa[1], fb[1]);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      __builtin_amdgcn_s_waitcnt(0xc07f & ~0x0f00);  // lgkmcnt(0)
      KD_VMCNT(NPW);  // step j+1 landed; step j+2's A DMA may still fly
      __syncthreads();
      const int na = ca == 2 ? 0 : ca + 1, nb = cb ^ 1;
      {
        const DmaStep<NPW> sb = db.prep(opb, bS(cb), wave, ks, ks < ks_end);
        const char* a = aS(na);
        const char* b = bS(nb);
        // the second half runs at wave priority 1, the first half, the waits
        // and the barrier at 0: a wave still in its second half is issued
        // before its SIMD partner that has moved on (measured: projection
        // 4.5% and dH 1.5% faster; priority in the first half, or in both,
        // was slower)
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          if (q % DS == 0) sb.one(q / DS);
          mfma2(q, fa[1], fb[1]);
          read3(q, a, b, 0, fa[0], fb[0]);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      __builtin_amdgcn_s_setprio(0);
      ca = na;
      cb = nb;
    }
    KD_VMCNT(0);
    __syncthreads();
    return;
  }

  // Step j lives in stage j % S; S steps of DMA are always in flight. Sub-step
  // 0's MFMAs run interleaved with the reads of sub-step 1's fragments; then
  // the wave waits for its reads and for step j+1's DMA, the barrier
  // publishes every wave's DMA and retires stage j % S, and sub-step 1's MFMAs
  // run in pairs: every other pair is issued with one DMA instruction of step
  // j+S (into the retired stage; spreading them keeps the LDS writes from
  // bunching up against the fragment reads), and the fragments of step j+1's
  // sub-step 0 are read alongside (placement per SPREAD).
#pragma unroll
  for (int p = 0; p < S; ++p) {
    char* a = lds + p * STB;
    const bool live = ks_begin + p < ks_end;
    const DmaStep<NPW> sa = da.prep(opa, a, wave, ks_begin + p, live);
    const DmaStep<NPW> sb = db.prep(opb, a + OPB, wave, ks_begin + p, live);
#pragma unroll
    for (int i = 0; i < NPW; ++i) sa.one(i);
#pragma unroll
    for (int i = 0; i < NPW; ++i) sb.one(i);
  }
  KD_VMCNT((S - 1) * NI);
  __syncthreads();
  u32x4_t fa[2][8], fb[2][NJ];
  frag(0, 0, fa[0], fb[0]);
  int st = 0;
  constexpr int NF = 8 + NJ;  // fragments per sub-step
  auto read_at = [&](int q, const char* a, int s, u32x4_t (&xa)[8], u32x4_t (&xb)[NJ]) {
#pragma unroll
    for (int f = 0; f < NF; ++f)
      if ((SPREAD ? (f * NP) / NF : f) == q) {
        if (f < 8) xa[f] = fra.one(a, s, f);
        else xb[f - 8] = frb.one(a + OPB, s, f - 8);
      }
  };
  for (int j = 0; j < nsteps; ++j) {
    if constexpr (SPREAD) {
      const char* c = lds + st * STB;
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        mfma2(q, fa[0], fb[0]);
        read_at(q, c, 1, fa[1], fb[1]);
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
      frag(st, 1, fa[1], fb[1]);
#pragma unroll
      for (int q = 0; q < NP; ++q) mfma2(q, fa[0], fb[0]);
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);   // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, RQ, 0);  // LDS read
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f & ~0x0f00);  // lgkmcnt(0)
    KD_VMCNT((S - 2) * NI);
    __syncthreads();
    const int nst = st + 1 == S ? 0 : st + 1;
    {
      char* a = lds + st * STB;
      const char* n = lds + nst * STB;
      const int ks = ks_begin + j + S;
      const DmaStep<NPW> sa = da.prep(opa, a, wave, ks, ks < ks_end);
      const DmaStep<NPW> sb = db.prep(opb, a + OPB, wave, ks, ks < ks_end);
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        if ((q & 1) == 0) {
          if (q < 2 * NPW) sa.one(q >> 1);
          else sb.one((q - 2 * NPW) >> 1);
        }
        mfma2(q, fa[1], fb[1]);
        if constexpr (SPREAD) {
          read_at(q, n, 0, fa[0], fb[0]);
        } else {
          if (q < 8) fa[0][q] = fra.one(n, 0, q);
          else if (q < 8 + NJ) fb[0][q - 8] = frb.one(n + OPB, 0, q - 8);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    st = nst;
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

// Sum / max over each row of 16 lanes, result in all 16 lanes, by DPP lane
// moves: swap neighbours (quad_perm 1,0,3,2), swap pairs (quad_perm 2,3,0,1),
// mirror within 8 (row_half_mirror), mirror within 16 (row_mirror).
__device__ __forceinline__ float dpp_f(float x, int ctrl_id) {
  const int v = __builtin_bit_cast(int, x);
  int r;
  switch (ctrl_id) {
    case 0: r = __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false); break;
    case 1: r = __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false); break;
    case 2: r = __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, false); break;
    default: r = __builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, false); break;
  }
  return __builtin_bit_cast(float, r);
}
__device__ __forceinline__ float row16_sum(float x) {
#pragma unroll
  for (int c = 0; c < 4; ++c) x += dpp_f(x, c);
  return x;
}
__device__ __forceinline__ float row16_max(float x) {
#pragma unroll
  for (int c = 0; c < 4; ++c) x = fmaxf(x, dpp_f(x, c));
  return x;
}

// inclusive prefix sum over the 64 lanes of a wave
__device__ __forceinline__ int wave_incl_scan(int x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  return x;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// two fp32 -> packed bf16 (v_cvt_pk_bf16_f32, round to nearest even)
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}


}  // namespace kd
