// HIP kernels (gfx950) of the fused chunked top-K KL loss and their launchers.
//
// Per call:    count_valid
// Per group of chunks, with a mask:
//              compact_scan, compact_rows -> the group's tokens that are not
//                                   ignored (row map, count, their hidden rows);
//                                   the kernels below then skip the rows past them
// Per chunk:   teacher_prologue  -> p, M, H, g/tau                 (§3.2, Eq. 2 terms)
//              bucket            -> teacher entries grouped by vocabulary tile
//   loss and gradients together (one projection per chunk):
//              ref_logit         -> per-token reference logit R
//              logits_dz         -> (reference, sum-exp) partials per (token, vocab
//                                   tile), z at the teacher entries, dZ'' = 2^(y - R)
//              row_finish        -> log Z, the row factor (g/tau) M 2^(R - log2 Z),
//                                   fallback rows, teacher cells (Eq. 3) / factor,
//                                   l_t = H - C/tau + M log Z       (Eq. 2)
//   forward only:  logits_lse (with z at the teacher entries), lse_merge, row_loss
//   backward only: dz            -> recomputed logits, dZ = g/tau (M q - p)
//              dh (+ split reduce): dH = dZ W (per chunk or per group; rows scaled
//                                   by the factor in the one-projection schedule)
// Per group of chunks: transpose_rows, dw -> grad_W (+)= dZ^T H (fp32 accumulate)
// Per call:    finalize_loss     -> mean over non-ignored tokens
#include "kd_device.h"
#include <type_traits>
#include "kd_launch.h"

#include <string.h>

namespace kd {

// ------------------------------------------------------------------ small --
// N_valid = tokens not ignored, and 1/N_valid (0 if none). One workgroup:
// 4 mask bytes per load when the mask is 4-byte aligned.
constexpr int kCountThreads = 1024;
__global__ __launch_bounds__(kCountThreads) void k_count_valid(const uint8_t* ignore, int64_t N,
                                                               int* nvalid, float* inv_nvalid) {
  __shared__ int red[kCountThreads / 64];
  const int tid = threadIdx.x;
  int c = 0;
  if (ignore == nullptr) {
    c = tid == 0 ? (int)N : 0;
  } else {
    int64_t i0 = 0;
    if (((uintptr_t)ignore & 3u) == 0u) {
      const uint32_t* w = reinterpret_cast<const uint32_t*>(ignore);
      const int64_t nw = N >> 2;
      for (int64_t i = tid; i < nw; i += kCountThreads) {
        const uint32_t v = w[i];
        c += ((v & 0xffu) == 0u) + (((v >> 8) & 0xffu) == 0u) + (((v >> 16) & 0xffu) == 0u) +
             ((v >> 24) == 0u);
      }
      i0 = nw << 2;
    }
    for (int64_t i = i0 + tid; i < N; i += kCountThreads) c += ignore[i] == 0 ? 1 : 0;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) c += __shfl_xor(c, o);
  if ((tid & 63) == 0) red[tid >> 6] = c;
  __syncthreads();
  if (tid == 0) {
    int n = 0;
    for (int w = 0; w < kCountThreads / 64; ++w) n += red[w];
    nvalid[0] = n;
    inv_nvalid[0] = n > 0 ? 1.0f / (float)n : 0.0f;
  }
}

__global__ void k_fill_f32(float* p, int64_t n, float v) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) p[i] = v;
}

// Teacher distribution over the K cached entries of each chunk row (§3.2):
// p = softmax(teacher_logit / tau), or p = exp(value) as given for cached
// log-probabilities (partial mass); M = sum p, H = sum p log p (0 log 0 = 0).
// Row weight coef = g/tau, g = 1/N_valid times the upstream gradient of the
// mean (gscale, default 1), or the upstream gradient of the token's own loss
// (gtok); 0 for ignored rows. With a saved log-normaliser (backward only) the
// row's log2 Z is set from it. One wave per row. With a rowmap, row r is
// token rowmap[r], and a row without a token (-1) gets p = 0, index -1 and
// weight 0.
//
// The support is a set; a row that repeats an index is read as the dense
// teacher row that sums the repeated entries (scatter-add): the first
// occurrence carries the sum of their probabilities (in entry order), H takes
// P log P of that sum, and the later occurrences get p = 0 and the index -1 in
// tidx_out, the row's copy of its indices that every later kernel reads (an
// index outside [0, V) is skipped everywhere). Rows without repeats are
// unchanged. Repeats are found with a hash set of the row's indices in LDS
// (an insertion that meets its own index); only a wave in which some row
// repeats an index compares the row's entries pairwise, in entry order.
// LDS hash set of the row's valid indices (power-of-two slots, at least K):
// size in ints for K entries
__host__ __device__ constexpr int prologue_hash_slots(int K) {
  int t = 64;
  while (t < 2 * K && t < 4096) t *= 2;
  return t;
}

__global__ __launch_bounds__(64) void k_teacher_prologue(
    const int32_t* __restrict__ tidx, int32_t* __restrict__ tidx_out, const float* tlogit,
    const uint8_t* ignore, int64_t row0, const int* __restrict__ rowmap, int rows, int K, int V,
    float inv_tau, int logprobs, const float* inv_nvalid, const float* gscale, const float* gtok,
    const float* logz_in, float* p_out, float* rowM, float* rowH, float* rowCoef,
    float* rowCoefM, float* rowL2) {
  extern __shared__ __attribute__((aligned(16))) char psm[];
  const int T = prologue_hash_slots(K);
  int* hset = reinterpret_cast<int*>(psm);
  int* sidx = hset + T;
  float* sp = reinterpret_cast<float*>(sidx + K);
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x;
  if (r >= rows) return;
  const int64_t t = rowmap != nullptr ? (int64_t)rowmap[r] : row0 + r;
  if (t < 0) {
    for (int k = lane; k < K; k += 64) {
      p_out[(int64_t)r * K + k] = 0.f;
      tidx_out[(int64_t)r * K + k] = -1;
    }
    if (lane == 0) {
      rowM[r] = 0.f;
      rowH[r] = 0.f;
      rowCoef[r] = 0.f;
      rowCoefM[r] = 0.f;
      if (logz_in != nullptr) rowL2[r] = 0.f;
    }
    return;
  }
  const float* u = tlogit + t * (int64_t)K;
  const int32_t* ix = tidx + t * (int64_t)K;
  for (int i = lane; i < T; i += 64) hset[i] = -1;
  float mx = 0.f, logs = 0.f, scale = 1.f;
  if (!logprobs) {
    mx = -INFINITY;
    for (int k = lane; k < K; k += 64) mx = fmaxf(mx, u[k] * inv_tau);
    mx = wave_max(mx);
    float s = 0.f;
    for (int k = lane; k < K; k += 64) s += expf(u[k] * inv_tau - mx);
    s = wave_sum(s);
    logs = logf(s);
    scale = inv_tau;
  }
  __syncthreads();  // the cleared hash set
  // p, and the row's indices into the hash set: an insertion that finds its
  // own index already there has seen a repeat (invalid indices are skipped
  // by every kernel and take no part)
  float m = 0.f;
  bool seen = false;
  for (int k = lane; k < K; k += 64) {
    const float pk = expf(u[k] * scale - mx - logs);
    const int v = ix[k];
    sidx[k] = v;
    sp[k] = pk;
    m += pk;
    if ((unsigned)v < (unsigned)V) {
      uint32_t h = ((uint32_t)v * 2654435761u) >> 7;
      for (int probe = 0; probe < T; ++probe, ++h) {
        const int prev = atomicCAS(&hset[h & (T - 1)], -1, v);
        if (prev == -1) break;
        if (prev == v) {
          seen = true;
          break;
        }
      }
    }
  }
  const bool any_repeat = __builtin_amdgcn_ballot_w64(seen) != 0ull;
  __syncthreads();  // sidx and sp of the whole row
  float h = 0.f;
  for (int k = lane; k < K; k += 64) {
    const int v = sidx[k];
    const float pk = sp[k];
    bool dup = false;
    float acc = pk;
    if (any_repeat) {
      // rare: an entry repeats an earlier index (p = 0, index -1) or is the
      // first of repeats (their probabilities summed in entry order)
      if ((unsigned)v < (unsigned)V) {
        for (int j = 0; j < K; ++j) {
          if (j != k && sidx[j] == v) {
            if (j < k) dup = true;
            else acc += sp[j];
          }
        }
      }
    }
    const float lp = u[k] * scale - mx - logs;
    float pe = pk, term = pk > 0.f ? pk * lp : 0.f;
    if (dup) {
      pe = 0.f;
      term = 0.f;
    } else if (acc != pk) {
      pe = acc;
      term = acc > 0.f ? acc * logf(acc) : 0.f;
    }
    p_out[(int64_t)r * K + k] = pe;
    tidx_out[(int64_t)r * K + k] = dup ? -1 : v;
    h += term;
  }
  m = wave_sum(m);
  h = wave_sum(h);
  if (lane == 0) {
    const bool valid = ignore == nullptr || ignore[t] == 0;
    const float g = gtok != nullptr ? gtok[t] : inv_nvalid[0] * (gscale != nullptr ? gscale[0] : 1.f);
    const float coef = valid ? inv_tau * g : 0.f;
    rowM[r] = m;
    rowH[r] = h;
    rowCoef[r] = coef;
    rowCoefM[r] = coef * m;
    if (logz_in != nullptr) rowL2[r] = logz_in[t] * kLog2e;
  }
}

// ------------------------------------------------- logits + online LSE -----
// Tile of z^T = W H_c^T (M = vocabulary, N = chunk tokens). Each lane holds 32
// vocabulary values of 4 tokens; the per-token max and sum of 2^(y - max) of
// y = z log2(e)/tau are reduced in registers, across the four lane groups of
// the wave, and across the two waves sharing the tokens through LDS. Output per (token,
// vocabulary tile): (max, sum) in base-2 units.
//
// With zhit set (forward-only calls, which have no logit recompute), the tile
// also records z at its teacher entries for C = sum_k p z (Eq. 2), in O(1)
// per entry: the entries of the tile's bucket mark a 256 x 256 bit map of
// cells (token, column) in LDS; an exclusive prefix sum of the words' bit
// counts numbers the marked cells; the lane holding a marked cell stores its
// z at that number in an LDS array; then every entry reads the z of its cell.
// A tile with more marked cells than the array holds (a teacher whose
// entries crowd one vocabulary tile) has the holders of the excess cells
// search the bucket for their entries instead.
constexpr int kZhBits = 0;                      // LDS: 256 tokens x 8 words
constexpr int kZhPre = 8192;                    // exclusive prefix per word
constexpr int kZhWs = 16384;                    // per-wave totals of the scan
constexpr int kZhVal = 16384 + 64;              // z of the marked cells
constexpr int kZhCap = (kLdsMain - kZhVal) / 4; // 28656 cells

template <typename T>
__global__ __launch_bounds__(kThreads, 1) void k_logits_lse(const T* __restrict__ W,
                                                            const T* __restrict__ Hc, int D,
                                                            int V, int rows, int TM, int TN,
                                                            float k2, float* part_m,
                                                            float* part_s, int nVT,
                                                            const uint32_t* __restrict__ hits,
                                                            const int* __restrict__ hoff, int K,
                                                            float* zhit,
                                                            const int* __restrict__ nrow,
                                                            int nrow_base) {
  __shared__ __attribute__((aligned(16))) char lds[kLdsA3];
  int mt, nt;
  tile_coords(blockIdx.x, TM, TN, 4, mt, nt);
  const int m0 = mt * kTile, n0 = nt * kTile;
  const int eb = Elt<T>::bytes;
  const int ld = D * eb;
  // with ignored tokens left out only the first *nrow - nrow_base rows hold
  // tokens (as in k_logits_dz)
  int trows = rows;
  if (nrow != nullptr) {
    trows = min(rows, __builtin_amdgcn_readfirstlane(*nrow) - nrow_base);
    if (n0 >= trows) return;
  }
  const int mrows = min(kTile, V - m0), nrows = min(kTile, trows - n0);
  AccTile acc;
  gemm_tile<T, KcOp, KcOp, 8, false, 3>(
      KcOp{reinterpret_cast<const char*>(W + (int64_t)m0 * D), (uint32_t)(mrows * ld), ld},
      KcOp{reinterpret_cast<const char*>(Hc + (int64_t)n0 * D), (uint32_t)(nrows * ld), ld}, 0,
      ld / kRowB, lds, acc);

  const int lane = threadIdx.x & 63, wave = wave_id();
  const int wm = wave >> 2, wn = wave & 3;
  const bool full = m0 + kTile <= V;
  if (zhit != nullptr) {
    const int tid = threadIdx.x;
    const int64_t seg = (int64_t)nt * kTile * K;
    const int* ho = hoff + (int64_t)nt * (nVT + 1) + mt;
    const int hb = ho[0], cnt = ho[1] - hb;
    const uint32_t* hl = hits + seg + hb;
    uint32_t* bits = reinterpret_cast<uint32_t*>(lds + kZhBits);
    int* pre = reinterpret_cast<int*>(lds + kZhPre);
    int* wsum = reinterpret_cast<int*>(lds + kZhWs);
    float* zval = reinterpret_cast<float*>(lds + kZhVal);
    *reinterpret_cast<u32x4_t*>(bits + 4 * tid) = u32x4_t{0u, 0u, 0u, 0u};
    __syncthreads();
    for (int q = tid; q < cnt; q += kThreads) {
      const uint32_t e = hl[q];
      const int tl = (int)(e & 255u), vl = (int)((e >> 8) & 255u);
      atomicOr(&bits[tl * 8 + (vl >> 5)], 1u << (vl & 31));
    }
    __syncthreads();
    // exclusive prefix of the 2048 word counts: thread tid owns words 4 tid .. 4 tid + 3
    {
      const u32x4_t wd = *reinterpret_cast<const u32x4_t*>(bits + 4 * tid);
      const int c0 = __builtin_popcount(wd[0]), c1 = __builtin_popcount(wd[1]);
      const int c2 = __builtin_popcount(wd[2]), c3 = __builtin_popcount(wd[3]);
      const int run = c0 + c1 + c2 + c3;
      const int incl = wave_incl_scan(run);
      if (lane == 63) wsum[wave] = incl;
      __syncthreads();
      int base = incl - run;
      for (int w = 0; w < wave; ++w) base += wsum[w];
      *reinterpret_cast<i32x4_t*>(pre + 4 * tid) =
          i32x4_t{base, base + c0, base + c0 + c1, base + c0 + c1 + c2};
    }
    __syncthreads();
    const int g = lane >> 4;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = acc_n(wn, j, lane);  // token in the tile
      const u32x4_t wd = *reinterpret_cast<const u32x4_t*>(bits + n * 8 + wm * 4);
      const i32x4_t wp = *reinterpret_cast<const i32x4_t*>(pre + n * 8 + wm * 4);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int sh = 16 * (i & 1) + 4 * g;  // bit of the cell's first column in its word
        const uint32_t nib = (wd[i >> 1] >> sh) & 15u;
        if (nib == 0u) continue;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          if (((nib >> r) & 1u) == 0u) continue;
          const int rank = wp[i >> 1] + __builtin_popcount(wd[i >> 1] & ((1u << (sh + r)) - 1u));
          if (rank < kZhCap) {
            zval[rank] = acc.v[i][j][r];
          } else {
            const uint32_t cell = (uint32_t)n | ((uint32_t)acc_m(wm, i, lane, r) << 8);
            for (int q = 0; q < cnt; ++q) {
              const uint32_t e = hl[q];
              if ((e & 0xffffu) == cell) zhit[(int64_t)(n0 + n) * K + (e >> 16)] = acc.v[i][j][r];
            }
          }
        }
      }
    }
    __syncthreads();
    for (int q = tid; q < cnt; q += kThreads) {
      const uint32_t e = hl[q];
      const int tl = (int)(e & 255u), vl = (int)((e >> 8) & 255u);
      const int w = tl * 8 + (vl >> 5);
      const int rank = pre[w] + __builtin_popcount(bits[w] & ((1u << (vl & 31)) - 1u));
      if (rank < kZhCap) zhit[(int64_t)(n0 + tl) * K + (e >> 16)] = zval[rank];
    }
    __syncthreads();
  }
  float* xch = reinterpret_cast<float*>(lds);  // [wn][j][16 lanes][max, sum]
  float rm[4], rs[4];
  // Per token: the max is taken over z itself (k2 > 0), then sum 2^(z k2 - max)
  // (one fma, one exp2 and one add per element). Only the last vocabulary
  // tile of a V that is not a multiple of 256 tests its columns.
  auto lse = [&](auto full_tile) {
    constexpr bool kFull = decltype(full_tile)::value;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float za = -INFINITY;
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (kFull || m0 + acc_m(wm, i, lane, r) < V) za = fmaxf(za, acc.v[i][j][r]);
      // the four lane groups (lane>>4) hold the other rows of the same token
      za = fmaxf(za, __shfl_xor(za, 16));
      za = fmaxf(za, __shfl_xor(za, 32));
      const float mx = za * k2;
      float s = 0.f;
      if (mx != -INFINITY) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float e = fast_exp2(acc.v[i][j][r] * k2 - mx);
            if (kFull || m0 + acc_m(wm, i, lane, r) < V) s += e;
          }
      }
      s += __shfl_xor(s, 16);
      s += __shfl_xor(s, 32);
      rm[j] = mx;
      rs[j] = s;
      if (wm == 1 && lane < 16) {
        xch[((wn * 4 + j) * 16 + lane) * 2 + 0] = mx;
        xch[((wn * 4 + j) * 16 + lane) * 2 + 1] = s;
      }
    }
  };
  if (full)
    lse(std::integral_constant<bool, true>());
  else
    lse(std::integral_constant<bool, false>());
  __syncthreads();
  if (wm == 0 && lane < 16) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int t = n0 + acc_n(wn, j, lane);
      const float m1 = rm[j], s1 = rs[j];
      const float m2 = xch[((wn * 4 + j) * 16 + lane) * 2 + 0];
      const float s2 = xch[((wn * 4 + j) * 16 + lane) * 2 + 1];
      const float mm = fmaxf(m1, m2);
      float ss = 0.f;
      if (mm != -INFINITY) ss = s1 * fast_exp2(m1 - mm) + s2 * fast_exp2(m2 - mm);
      if (t < rows) {
        part_m[(int64_t)t * nVT + mt] = mm;
        part_s[(int64_t)t * nVT + mt] = ss;
      }
    }
  }
}

// log2 of the normaliser per token from the vocabulary-tile partials (fixed
// order, one wave per token). L2 = log2 sum_v 2^(z_v log2(e)/tau); a partial
// is the tile max and the sum of 2^(y - max) over the tile's columns.
__global__ void k_lse_merge(const float* part_m, const float* part_s, int rows, int nVT,
                            float* rowL2, const int* __restrict__ rowmap) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + wave_id();
  if (r >= rows) return;
  if (rowmap != nullptr && rowmap[r] < 0) {
    // a row without a token: its partials were never written
    if (lane == 0) rowL2[r] = 0.f;
    return;
  }
  const float* pm = part_m + (int64_t)r * nVT;
  const float* ps = part_s + (int64_t)r * nVT;
  float mx = -INFINITY;
  for (int j = lane; j < nVT; j += 64) mx = fmaxf(mx, pm[j]);
  mx = wave_max(mx);
  float s = 0.f;
  for (int j = lane; j < nVT; j += 64) {
    const float m = pm[j];
    if (m != -INFINITY) s += ps[j] * fast_exp2(m - mx);
  }
  s = wave_sum(s);
  if (lane == 0) rowL2[r] = mx + log2f(s);
}

// ------------------------------------------------ teacher entry buckets ----
// The K cached entries of each token are folded into the dZ tile that holds
// their vocabulary column (§3.2). One workgroup per 256-token tile groups the
// tile's entries by vocabulary tile with a counting sort in LDS: segment nt of
// `hits` (capacity 256 K) lists, for vocabulary tile b, the entries
// [hoff[nt][b], hoff[nt][b+1]) as (token in tile | column in tile << 8 | k << 16)
// with their teacher probability in `hitp`. An index outside [0, V) gets no
// slot and a zero z (it contributes nothing to C or dZ).
constexpr int kBucketThreads = 1024;
constexpr int kBucketBatch = 8;  // entries per thread whose loads are in flight together
constexpr int kMaxVT = 4096;     // vocabulary tiles (V <= 2^20)

__global__ __launch_bounds__(kBucketThreads) void k_bucket(const int32_t* __restrict__ tidx,
                                                           const float* __restrict__ p, int rows,
                                                           int K, int V, int nVT, uint32_t* hits,
                                                           float* hitp, int* hoff, float* zhit) {
  __shared__ int cnt[kMaxVT];
  __shared__ int cur[kMaxVT];
  __shared__ int wsum[kBucketThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
  const int t0 = blockIdx.x * kTile;
  const int total = min(kTile, rows - t0) * K;
  const int64_t seg = (int64_t)blockIdx.x * kTile * K;
  // entry e of the tile is element t0 K + e of the row-major [rows, K] arrays
  const int32_t* ti = tidx + (int64_t)t0 * K;
  const float invK = 1.0f / (float)K;
  for (int b = tid; b < nVT; b += kBucketThreads) cnt[b] = 0;
  __syncthreads();
  for (int base = 0; base < total; base += kBucketThreads * kBucketBatch) {
    int v[kBucketBatch];
#pragma unroll
    for (int u = 0; u < kBucketBatch; ++u) {
      const int e = base + u * kBucketThreads + tid;
      v[u] = e < total ? ti[e] : 0;
    }
#pragma unroll
    for (int u = 0; u < kBucketBatch; ++u) {
      const int e = base + u * kBucketThreads + tid;
      if (e >= total) continue;
      if ((unsigned)v[u] < (unsigned)V)
        atomicAdd(&cnt[v[u] >> 8], 1);
      else
        zhit[(int64_t)t0 * K + e] = 0.f;
    }
  }
  __syncthreads();
  // exclusive scan: thread tid owns bins [tid R, tid R + R)
  const int R = (nVT + kBucketThreads - 1) / kBucketThreads;
  int run = 0;
  for (int q = 0; q < R; ++q) {
    const int b = tid * R + q;
    if (b < nVT) run += cnt[b];
  }
  const int incl = wave_incl_scan(run);
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    const int x = lane < kBucketThreads / 64 ? wsum[lane] : 0;
    const int y = wave_incl_scan(x);
    if (lane < kBucketThreads / 64) wsum[lane] = y - x;
  }
  __syncthreads();
  int off = wsum[wave] + incl - run;
  int* ho = hoff + (int64_t)blockIdx.x * (nVT + 1);
  for (int q = 0; q < R; ++q) {
    const int b = tid * R + q;
    if (b < nVT) {
      cur[b] = off;
      ho[b] = off;
      off += cnt[b];
    }
  }
  if (tid == kBucketThreads - 1) ho[nVT] = off;
  __syncthreads();
  for (int base = 0; base < total; base += kBucketThreads * kBucketBatch) {
    int v[kBucketBatch];
    float pv[kBucketBatch];
#pragma unroll
    for (int u = 0; u < kBucketBatch; ++u) {
      const int e = base + u * kBucketThreads + tid;
      v[u] = e < total ? ti[e] : -1;
      pv[u] = e < total ? p[(int64_t)t0 * K + e] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kBucketBatch; ++u) {
      const int e = base + u * kBucketThreads + tid;
      if (e >= total || (unsigned)v[u] >= (unsigned)V) continue;
      // token = e / K (exact: e < 2^20, and (e + 0.5) / K stays >= 1/(2K)
      // away from an integer while the float product errs by < 2^-12)
      const int tl = (int)(((float)e + 0.5f) * invK);
      const int k = e - tl * K;
      const int pos = atomicAdd(&cur[v[u] >> 8], 1);
      hits[seg + pos] = (uint32_t)tl | ((uint32_t)(v[u] & 255) << 8) | ((uint32_t)k << 16);
      hitp[seg + pos] = pv[u];
    }
  }
}

// --------------------------------------- logit recompute + dZ epilogue -----
// Same tile as k_logits_lse (bitwise identical z). Before the main loop the
// tile's per-token scalars (g/tau M, g/tau, log2 Z) and its teacher entries
// (one per thread) are loaded into registers, so the epilogue issues no
// global loads (a load waited for after a store would also wait for that
// store); after the loop the scalars go to LDS beside the staging area.
// The fp32 tile is staged 128 tokens at a time as [token][vocab] with a
// 16-byte-slot swizzle; each teacher entry of the half is patched in place to
// its final value (g/tau)(M q - p), its z is recorded for C, and a bitmap marks
// it; then one wave per token row forms G = (g/tau) M 2^(y - L2) elsewhere and
// stores the row of dZ[rows, Vp] (columns V..Vp as zeros).
__device__ __forceinline__ int hsw16(int n) { return (n ^ (n >> 3)) & 15; }

// largest exponent (base 2) of the sum of a tile row's stored provisional
// gradients 2^(y - R), and so of each of them
constexpr float kRefGap = 40.f;
constexpr float kRefGapScale = 1099511627776.f;  // 2^kRefGap
// R is the reference logit plus this many (base 2): stored values are then
// smaller, which the dH and dW contractions run about 1% faster on (MFMA power
// depends on the operands); terms below 2^-126 relative to R + kRefShift,
// i.e. 2^-102 below the reference logit, flush to zero
constexpr float kRefShift = 24.f;

// epilogue LDS (the main loop's stages are free by then): staging [0, 128 KiB)
constexpr int kDzBits = kLdsMain;              // 128 x 256-bit hit map of one half
constexpr int kDzRows = kDzBits + 4 * 1024;    // 3 x 256 floats: g/tau M, g/tau, log2 Z
static_assert(kDzRows + 3 * 1024 <= kLdsA3, "dZ epilogue LDS");

template <typename T>
__global__ __launch_bounds__(kThreads, 1) void k_dz(
    const T* __restrict__ W, const T* __restrict__ Hc, int D, int V, int rows, int TM, int TN,
    float k2, const float* __restrict__ rowL2, const float* __restrict__ rowCoef,
    const float* __restrict__ rowCoefM, const uint32_t* __restrict__ hits,
    const float* __restrict__ hitp, const int* __restrict__ hoff, int K, int nVT, T* dZ,
    int64_t ldz, float* zhit, const int* __restrict__ nrow, int nrow_base) {
  __shared__ __attribute__((aligned(16))) char lds[kLdsA3];
  int mt, nt;
  tile_coords(blockIdx.x, TM, TN, 4, mt, nt);
  const int m0 = mt * kTile, n0 = nt * kTile;
  const int eb = Elt<T>::bytes;
  const int ld = D * eb;
  // with ignored tokens left out only the first *nrow - nrow_base rows hold
  // tokens (as in k_logits_dz; the rows past them have weight 0)
  int trows = rows;
  if (nrow != nullptr) {
    trows = min(rows, __builtin_amdgcn_readfirstlane(*nrow) - nrow_base);
    if (n0 >= trows) return;
  }
  const int mrows = min(kTile, V - m0), nrows = min(kTile, trows - n0);
  const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
  const int wm = wave >> 2, wn = wave & 3;

  // this tile's bucket of teacher entries
  const int64_t seg = (int64_t)nt * kTile * K;
  const int* ho = hoff + (int64_t)nt * (nVT + 1) + mt;
  const int hb = ho[0], cnt = ho[1] - hb;
  // wave w holds the scalars of tokens [32 w, 32 w + 32): lane l has token
  // 32 w + (l & 31), g/tau M and g/tau (l < 32) or log2 Z (l >= 32, in rv0)
  float rv0, rv1 = 0.f;
  {
    const int t = n0 + 32 * wave + (lane & 31);
    const bool ok = t < rows;
    rv0 = ok ? (lane < 32 ? rowCoefM[t] : rowL2[t]) : 0.f;
    if (lane < 32) rv1 = ok ? rowCoef[t] : 0.f;
  }
  uint32_t fe = 0u;  // this thread's teacher entry (entry tid of the bucket) and its p
  float fpk = 0.f;
  if (tid < cnt) {
    fe = hits[seg + hb + tid];
    fpk = hitp[seg + hb + tid];
  }

  AccTile acc;
  gemm_tile<T, KcOp, KcOp, 8, false, 3>(
      KcOp{reinterpret_cast<const char*>(W + (int64_t)m0 * D), (uint32_t)(mrows * ld), ld},
      KcOp{reinterpret_cast<const char*>(Hc + (int64_t)n0 * D), (uint32_t)(nrows * ld), ld}, 0,
      ld / kRowB, lds, acc);
  {
    float* rs = reinterpret_cast<float*>(lds + kDzRows);
    const int t = 32 * wave + (lane & 31);
    if (lane < 32) {
      rs[t] = rv0;
      rs[256 + t] = rv1;
    } else {
      rs[512 + t] = rv0;
    }
  }

  float* st = reinterpret_cast<float*>(lds);
  const float* rs_cm = reinterpret_cast<const float*>(lds + kDzRows);
  const float* rs_cf = rs_cm + 256;
  const float* rs_l2 = rs_cm + 512;
  uint32_t* hbits = reinterpret_cast<uint32_t*>(lds + kDzBits);
  const int vl0 = 4 * lane;  // this lane's 4 vocabulary columns in the row pass

  // unrolled: a loop header here would make the compiler wait for the first
  // half's dZ stores before staging the second half
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if ((wn >> 1) == h) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = (wn & 1) * 64 + 16 * j + (lane & 15);  // token row of the half
          const int vl = acc_m(wm, i, lane, 0);                 // 4 consecutive vocab
          const int slot = (vl >> 2) ^ hsw16(n);
          *reinterpret_cast<f32x4_t*>(st + n * 256 + slot * 4) = acc.v[i][j];
        }
    }
    hbits[tid] = 0u;
    hbits[tid + kThreads] = 0u;
    __syncthreads();

    // Teacher entries of this half: dZ = (g/tau) M q - (g/tau) p in place,
    // z kept for C = sum_k p z (Eq. 2). Thread tid has entry tid of the
    // bucket in registers; a skewed teacher with more entries in one tile
    // than threads reads the rest from memory.
    auto fold = [&](uint32_t e, float pk) {
      const int tl = (int)(e & 255u);
      if ((tl >> 7) != h) return;
      const int n = tl & 127, v = (int)((e >> 8) & 255u), k = (int)(e >> 16);
      float* cell = st + n * 256 + ((((v >> 2) ^ hsw16(n)) << 2) | (v & 3));
      const float z = *cell;
      if (zhit != nullptr) zhit[(int64_t)(n0 + tl) * K + k] = z;
      *cell = rs_cm[tl] * fast_exp2(z * k2 - rs_l2[tl]) - rs_cf[tl] * pk;
      atomicOr(&hbits[n * 8 + (v >> 5)], 1u << (v & 31));
    };
    if (tid < cnt) fold(fe, fpk);
    // a bucket with more entries than threads: the rest from memory
    for (int q = kThreads + tid; q < cnt; q += kThreads) fold(hits[seg + hb + q], hitp[seg + hb + q]);
    __syncthreads();

    if (dZ != nullptr) {
      // The wave's 16 rows go in two batches of 8 whose LDS reads are all
      // issued before their arithmetic. The row pass is VALU-bound (every
      // element costs an exp2), so it carries no per-element selects: a row's
      // teacher cells (about one row in five has any) are substituted behind
      // a wave-uniform test, and columns past V get no mask (their z is
      // exactly 0, as W's rows past V read as zeros, so they hold finite
      // values that only ever meet those zero rows).
      const int rb = wave * 16;                                      // first row in the half
      const int nrow = max(0, min(16, rows - (n0 + 128 * h + rb)));  // rows that exist
      {
#pragma unroll
        for (int b8 = 0; b8 < 16; b8 += 8) {
          f32x4_t zr[8];
          uint32_t mk[8];
#pragma unroll
          for (int rr = 0; rr < 8; ++rr) {
            const int n = rb + b8 + rr;
            zr[rr] = *reinterpret_cast<const f32x4_t*>(st + n * 256 + ((lane ^ hsw16(n)) << 2));
            mk[rr] = (hbits[n * 8 + (lane >> 3)] >> ((lane & 7) * 4)) & 15u;
          }
          f32x4_t cmv[2], l2v[2];  // the rows' g/tau M and log2 Z (16-byte aligned runs)
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            cmv[u] = *reinterpret_cast<const f32x4_t*>(rs_cm + 128 * h + rb + b8 + 4 * u);
            l2v[u] = *reinterpret_cast<const f32x4_t*>(rs_l2 + 128 * h + rb + b8 + 4 * u);
          }
#pragma unroll
          for (int rr = 0; rr < 8; ++rr) {
            const float cm = cmv[rr >> 2][rr & 3], L2 = l2v[rr >> 2][rr & 3];
            f32x4_t G;
#pragma unroll
            for (int e = 0; e < 4; ++e) G[e] = cm * fast_exp2(zr[rr][e] * k2 - L2);
            if (__builtin_amdgcn_ballot_w64(mk[rr] != 0u) != 0ull) {
              // teacher cells hold their final value (patched by the fold)
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if ((mk[rr] >> e) & 1u) G[e] = zr[rr][e];
            }
            if (b8 + rr < nrow) {
              T* dst = dZ + (int64_t)(n0 + 128 * h + rb + b8 + rr) * ldz + m0 + vl0;
              if constexpr (sizeof(T) == 2) {
                u32x2_t pk2 = {pack_bf16x2(G[0], G[1]), pack_bf16x2(G[2], G[3])};
                *reinterpret_cast<u32x2_t*>(dst) = pk2;
              } else {
                *reinterpret_cast<f32x4_t*>(dst) = G;
              }
            }
          }
        }
      }
    }
    __syncthreads();
  }
}

// ------------------------------------ one projection per chunk (fused call) --
// A call that wants the loss and its gradients together has each chunk's
// normaliser complete as soon as that chunk's projection has run, so the
// chunk is projected once instead of once for log Z and again for dZ: the
// tile records per token z at its teacher entries, the provisional gradient
// dZ'' = 2^(y - R) with y = z log2(e) / tau in the dZ buffer (0 past V), R
// being the token's reference logit from k_ref_logit, and the partials (R,
// sum of 2^(y - R)) of log Z (a reference and a sum relative to it, like
// the (max, sum) partials of k_logits_lse).
// Once log Z is merged, the row factor (g/tau) M 2^(R - log2 Z) turns dZ''
// into (g/tau) M q; it is applied to the rows of dH and, through the
// transposed hidden rows, to dW, so dZ'' is never rewritten, except the
// teacher cells (k_row_finish writes (g/tau)(M q - p) / factor, Eq. 3) and the
// rare rows where a tile's sum of 2^(y - R) exceeded 2^kRefGap (k_row_finish
// rescales them).
// The [c, V] buffer is the same transient chunk the recompute schedule holds;
// nothing grows with N. Staging and teacher bookkeeping are those of k_dz.
template <typename T>
__global__ __launch_bounds__(kThreads, 1) void k_logits_dz(
    const T* __restrict__ W, const T* __restrict__ Hc, int D, int V, int rows, int TM, int TN,
    float k2, float* __restrict__ part_m, float* __restrict__ part_s, int nVT,
    const uint32_t* __restrict__ hits, const int* __restrict__ hoff, int K, T* dZ, int64_t ldz,
    float* zhit, const float* __restrict__ rowR, int* rowFlag, const int* __restrict__ nrow,
    int nrow_base) {
  __shared__ __attribute__((aligned(16))) char lds[kLdsA3];
  int mt, nt;
  tile_coords(blockIdx.x, TM, TN, 4, mt, nt);
  const int m0 = mt * kTile, n0 = nt * kTile;
  const int eb = Elt<T>::bytes;
  const int ld = D * eb;
  // with ignored tokens left out only the first *nrow - nrow_base rows hold
  // tokens: a tile of rows past them has nothing to compute, and rows past
  // them in the last tile read hidden rows of zeros (stored like the others,
  // with a row factor of 0)
  int trows = rows;
  if (nrow != nullptr) {
    trows = min(rows, __builtin_amdgcn_readfirstlane(*nrow) - nrow_base);
    if (n0 >= trows) return;
  }
  const int mrows = min(kTile, V - m0), nrows = min(kTile, trows - n0);
  const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
  const int wm = wave >> 2, wn = wave & 3;

  const int64_t seg = (int64_t)nt * kTile * K;
  const int* ho = hoff + (int64_t)nt * (nVT + 1) + mt;
  const int hb = ho[0], cnt = ho[1] - hb;
  const uint32_t fe = tid < cnt ? hits[seg + hb + tid] : 0u;
  // the tile's reference logits, loaded before the main loop: a load issued
  // in the epilogue would wait for every store issued before it (loads and
  // stores complete in order), serialising the row pass on its stores
  const float rref = (tid < kTile && n0 + tid < rows) ? rowR[n0 + tid] : 0.f;

  AccTile acc;
  gemm_tile<T, KcOp, KcOp, 8, false, 3>(
      KcOp{reinterpret_cast<const char*>(W + (int64_t)m0 * D), (uint32_t)(mrows * ld), ld},
      KcOp{reinterpret_cast<const char*>(Hc + (int64_t)n0 * D), (uint32_t)(nrows * ld), ld}, 0,
      ld / kRowB, lds, acc);
  const bool full = m0 + kTile <= V;

  float* st = reinterpret_cast<float*>(lds);
  // past the staging area: R of the tile's 256 tokens (0 past the chunk)
  float* rs_r = reinterpret_cast<float*>(lds + kLdsMain);
  if (tid < kTile) rs_r[tid] = rref;
  const int rho = lane >> 4, lam = lane & 15;  // row pass: 4 token rows per wave, 16 lanes each
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if ((wn >> 1) == h) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = (wn & 1) * 64 + 16 * j + (lane & 15);  // token row of the half
          const int vl = acc_m(wm, i, lane, 0);                 // 4 consecutive vocab
          const int slot = (vl >> 2) ^ hsw16(n);
          *reinterpret_cast<f32x4_t*>(st + n * 256 + slot * 4) = acc.v[i][j];
        }
    }
    __syncthreads();
    // z at the teacher entries of this half, for C = sum_k p z (Eq. 2)
    auto rec = [&](uint32_t e) {
      const int tl = (int)(e & 255u);
      if ((tl >> 7) != h) return;
      const int n = tl & 127, v = (int)((e >> 8) & 255u);
      zhit[(int64_t)(n0 + tl) * K + (e >> 16)] =
          st[n * 256 + ((((v >> 2) ^ hsw16(n)) << 2) | (v & 3))];
    };
    if (tid < cnt) rec(fe);
    for (int q = kThreads + tid; q < cnt; q += kThreads) rec(hits[seg + hb + q]);

    // 16 lanes per token row, lane lam holding columns 4 lam + 64 k + (0..3).
    // The row's run of dZ'' is 2^(y - R) against the token's reference R; the
    // partials are (R, sum of 2^(y - R)) with the sum reduced within the 16
    // lanes (DPP). A run whose sum exceeds 2^kRefGap (so its values could
    // too) is stored against the run's own max m instead, with partials
    // (m, sum of 2^(y - m)), and its token is flagged for a row rescale.
    // Columns past V give 0 and count for neither.
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      const int n = wave * 16 + 4 * gq + rho;  // token row of the half
      const int t = n0 + 128 * h + n;
      f32x4_t zr[4];
#pragma unroll
      for (int k = 0; k < 4; ++k)
        zr[k] = *reinterpret_cast<const f32x4_t*>(st + n * 256 + (((lam + 16 * k) ^ hsw16(n)) << 2));
      // rows past the chunk use a finite reference (nothing of them is stored)
      float ref = rs_r[128 * h + n];
      f32x4_t G[4];
#pragma unroll
      for (int k = 0; k < 4; ++k)
        G[k] = f32x4_t{fast_exp2(zr[k][0] * k2 - ref), fast_exp2(zr[k][1] * k2 - ref),
                       fast_exp2(zr[k][2] * k2 - ref), fast_exp2(zr[k][3] * k2 - ref)};
      // the column mask only on the last vocabulary tile (a wave-uniform
      // branch instead of per-element selects on every tile)
      if (!full) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int c = m0 + 4 * lam + 64 * k;
          G[k] = f32x4_t{c < V ? G[k][0] : 0.f, c + 1 < V ? G[k][1] : 0.f,
                         c + 2 < V ? G[k][2] : 0.f, c + 3 < V ? G[k][3] : 0.f};
        }
      }
      float sum = 0.f;
#pragma unroll
      for (int k = 0; k < 4; ++k) sum += (G[k][0] + G[k][1]) + (G[k][2] + G[k][3]);
      sum = row16_sum(sum);
      const bool own = !(sum <= kRefGapScale);
      if (__builtin_amdgcn_ballot_w64(own) != 0ull) {
        // rare: some row of the wave falls back to its own max (formed for
        // every row so that the 16-lane reductions run on a full wave)
        float mx = -INFINITY;
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (full || m0 + 4 * lam + 64 * k + e < V) mx = fmaxf(mx, zr[k][e]);
        const float m = row16_max(mx) * k2;
        float s2 = 0.f;
        f32x4_t G2[4];
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float ev = fast_exp2(zr[k][e] * k2 - m);
            if (!full && m0 + 4 * lam + 64 * k + e >= V) ev = 0.f;
            G2[k][e] = ev;
            s2 += ev;
          }
        s2 = row16_sum(s2);
        if (own) {
          ref = m;
          sum = s2;
#pragma unroll
          for (int k = 0; k < 4; ++k) G[k] = G2[k];
        }
      }
      if (t < rows) {
        T* dst = dZ + (int64_t)t * ldz + m0 + 4 * lam;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if constexpr (sizeof(T) == 2) {
            const u32x2_t pk2 = {pack_bf16x2(G[k][0], G[k][1]), pack_bf16x2(G[k][2], G[k][3])};
            *reinterpret_cast<u32x2_t*>(dst + 64 * k) = pk2;
          } else {
            *reinterpret_cast<f32x4_t*>(dst + 64 * k) = G[k];
          }
        }
        if (lam == 0) {
          part_m[(int64_t)t * nVT + mt] = ref;
          part_s[(int64_t)t * nVT + mt] = sum;
          if (own) rowFlag[t] = 1;
        }
      }
    }
    __syncthreads();
  }
}

// The reference logit of each token for k_logits_dz: R = z log2(e)/tau at the
// teacher entry with the largest teacher logit (a valid index), plus
// kRefShift, one wave per token; -inf when the row has no valid index. The
// logit part never exceeds the row's max y beyond rounding, so 2^(y - R)
// keeps every term that matters; a tile whose sum of 2^(y - R) exceeds
// 2^kRefGap falls back to its own max. Also clears the row's fallback flag.
// Row r is token row0 + r, or rowmap[r] (a row without a token has no valid
// index after the prologue).
template <typename T>
__global__ void k_ref_logit(const T* __restrict__ H, const T* __restrict__ W, int D,
                            const int32_t* __restrict__ tidx, const float* __restrict__ tlogit,
                            int64_t row0, const int* __restrict__ rowmap, int rows, int K, int V,
                            float k2, float* rowR, int* rowFlag) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + wave_id();
  if (r >= rows) return;
  const int64_t t = rowmap != nullptr ? (int64_t)rowmap[r] : row0 + r;
  const int32_t* ix = tidx + (int64_t)r * K;
  const float* tl = tlogit + (t < 0 ? 0 : t) * (int64_t)K;
  float best = -INFINITY;
  int bk = K;
  for (int k = lane; k < K; k += 64) {
    const int v = ix[k];
    if ((unsigned)v < (unsigned)V && (tl[k] > best || (tl[k] == best && k < bk))) {
      best = tl[k];
      bk = k;
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float ob = __shfl_xor(best, o);
    const int ok = __shfl_xor(bk, o);
    if (ob > best || (ob == best && ok < bk)) {
      best = ob;
      bk = ok;
    }
  }
  float z = 0.f;
  if (bk < K) {
    // 16-byte pieces of both rows (D is a multiple of 64, rows 16-byte aligned)
    constexpr int VPT = 16 / (int)sizeof(T);
    const T* h = H + t * D;
    const T* w = W + (int64_t)ix[bk] * D;
    for (int d = lane * VPT; d < D; d += 64 * VPT) {
      const u32x4_t hv = *reinterpret_cast<const u32x4_t*>(h + d);
      const u32x4_t wv = *reinterpret_cast<const u32x4_t*>(w + d);
      T he[VPT], we[VPT];
      __builtin_memcpy(he, &hv, 16);
      __builtin_memcpy(we, &wv, 16);
#pragma unroll
      for (int x = 0; x < VPT; ++x) z += (float)he[x] * (float)we[x];
    }
    z = wave_sum(z);
  }
  if (lane == 0) {
    rowR[r] = bk < K ? z * k2 + kRefShift : -INFINITY;
    rowFlag[r] = 0;
  }
}

// l_t = H_t - C_t / tau + M_t log Z_t (Eq. 2) with C_t = sum_k p_k z_{t, idx_k},
// 0 on ignored rows; one wave per row and a partial sum per block of
// kLossRows rows in a fixed order, for the deterministic mean.
__global__ void k_row_loss(const float* zhit, const float* p, int K, const float* rowL2,
                           const float* rowM, const float* rowH, const uint8_t* ignore,
                           int64_t row0, const int* __restrict__ rowmap, int rows, float inv_tau,
                           float* loss_per_token, float* logz_out, float* block_partial) {
  __shared__ float red[kLossRows];
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int r = blockIdx.x * kLossRows + wave;
  float l = 0.f;
  // with a rowmap, row r is token rowmap[r] (loss_per_token and logz_out
  // indexed by token), and a row without a token (-1) has a loss of 0
  const int tok = (rowmap != nullptr && r < rows) ? rowmap[r] : 0;
  if (r < rows && tok >= 0) {
    float c = 0.f;
    for (int k = lane; k < K; k += 64) c += p[(int64_t)r * K + k] * zhit[(int64_t)r * K + k];
    c = wave_sum(c);
    const bool valid = rowmap != nullptr || ignore == nullptr || ignore[row0 + r] == 0;
    l = valid ? rowH[r] - c * inv_tau + rowM[r] * rowL2[r] * kLn2 : 0.f;
    if (lane == 0) {
      if (loss_per_token) loss_per_token[rowmap != nullptr ? (int64_t)tok : r] = l;
      if (logz_out) logz_out[rowmap != nullptr ? (int64_t)tok : r] = rowL2[r] * kLn2;
    }
  }
  if (lane == 0) red[wave] = l;
  __syncthreads();
  if (threadIdx.x == 0) block_partial[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

// The end of a chunk in the single-projection schedule, one wave per token
// (one pass instead of four launches): log2 Z merged from the tile partials
// (each a reference and a sum relative to it), the row factor that turns the
// stored 2^(y - mx) into (g/tau) M q, mx being the largest reference of the
// row's tiles (the token's reference logit unless a tile fell back to its own
// max); for a row with such a tile, every run brought to mx; the teacher
// cells (g/tau)(M q - p) (Eq. 3) in the row's stored scale (0 where the
// factor is 0, i.e. on ignored rows); and the token's loss (Eq. 2) with a
// partial per block of kLossRows rows as k_row_loss forms it. With a rowmap,
// row r is token rowmap[r] (loss_per_token is then indexed by token), and a
// row without a token (-1) only gets a row factor of 0 and a loss of 0.
template <typename T>
__global__ __launch_bounds__(256) void k_row_finish(
    const float* __restrict__ part_m, const float* __restrict__ part_s, int nVT,
    const int* __restrict__ rowFlag, T* dZ, int64_t ldz, const int32_t* __restrict__ tidx,
    const float* __restrict__ p, const float* __restrict__ zhit, int K, int V, float k2,
    const float* __restrict__ rowM, const float* __restrict__ rowH,
    const float* __restrict__ rowCoef, const float* __restrict__ rowCoefM,
    const uint8_t* __restrict__ ignore, int64_t row0, const int* __restrict__ rowmap, int rows,
    float inv_tau, float* rowL2, float* rowFactor, float* loss_per_token, float* block_partial) {
  __shared__ float red[kLossRows];
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int r = blockIdx.x * kLossRows + wave;
  float l = 0.f;
  const int tok = (rowmap != nullptr && r < rows) ? rowmap[r] : 0;
  if (r < rows && tok < 0) {
    if (lane == 0) {
      rowL2[r] = 0.f;
      rowFactor[r] = 0.f;
    }
  } else if (r < rows) {
    const float* pm = part_m + (int64_t)r * nVT;
    const float* ps = part_s + (int64_t)r * nVT;
    // up to 512 vocabulary tiles: the row's partials are loaded into registers
    // in one batch, with the row scalars, before any arithmetic (one round of
    // memory latency instead of one per pass); the sums keep the same order
    constexpr int kRF = 8;
    const bool in_regs = nVT <= 64 * kRF;
    float pmv[kRF], psv[kRF];
    if (in_regs) {
#pragma unroll
      for (int i = 0; i < kRF; ++i) {
        const int j = lane + 64 * i;
        pmv[i] = j < nVT ? pm[j] : -INFINITY;
        psv[i] = j < nVT ? ps[j] : 0.f;
      }
    }
    const float cm = rowCoefM[r], cf = rowCoef[r];
    float mx = -INFINITY;
    if (in_regs) {
#pragma unroll
      for (int i = 0; i < kRF; ++i) mx = fmaxf(mx, pmv[i]);
    } else {
      for (int j = lane; j < nVT; j += 64) mx = fmaxf(mx, pm[j]);
    }
    mx = wave_max(mx);
    float s = 0.f;
    if (in_regs) {
#pragma unroll
      for (int i = 0; i < kRF; ++i)
        if (pmv[i] != -INFINITY) s += psv[i] * fast_exp2(pmv[i] - mx);
    } else {
      for (int j = lane; j < nVT; j += 64) {
        const float m = pm[j];
        if (m != -INFINITY) s += ps[j] * fast_exp2(m - mx);
      }
    }
    s = wave_sum(s);
    const float L2 = mx + log2f(s);
    const float f = cm * fast_exp2(mx - L2);
    if (lane == 0) {
      rowL2[r] = L2;
      rowFactor[r] = f;
    }
    T* row = dZ + (int64_t)r * ldz;
    if (rowFlag[r] != 0) {
      // rare: runs stored against different references
      constexpr int VPT = 16 / (int)sizeof(T);
      for (int64_t c0 = (int64_t)lane * VPT; c0 < ldz; c0 += 64 * VPT) {
        const float fr = fast_exp2(pm[c0 >> 8] - mx);
        u32x4_t* q = reinterpret_cast<u32x4_t*>(row + c0);
        const u32x4_t v = *q;
        // built as a new vector (in-place element updates were miscompiled)
        if constexpr (sizeof(T) == 2) {
          uint32_t o[4];
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const uint32_t x = v[w];
            o[w] = pack_bf16x2(__builtin_bit_cast(float, x << 16) * fr,
                               __builtin_bit_cast(float, x & 0xffff0000u) * fr);
          }
          *q = u32x4_t{o[0], o[1], o[2], o[3]};
        } else {
          *q = __builtin_bit_cast(u32x4_t, __builtin_bit_cast(f32x4_t, v) * fr);
        }
      }
      // the teacher cells below overwrite some of these elements: the wave's
      // rescale stores complete first (a workgroup-scope fence emits no wait
      // here, so the wait is explicit; the clobber keeps the compiler from
      // moving memory accesses across it)
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    float c = 0.f;
    for (int k = lane; k < K; k += 64) {
      const int64_t e = (int64_t)r * K + k;
      const float pk = p[e], z = zhit[e];
      c += pk * z;
      const int v = tidx[e];
      if ((unsigned)v < (unsigned)V) {
        const float g = cm * fast_exp2(z * k2 - L2) - cf * pk;
        row[v] = (T)(f != 0.f ? g / f : 0.f);
      }
    }
    c = wave_sum(c);
    const bool valid = rowmap != nullptr || ignore == nullptr || ignore[row0 + r] == 0;
    l = valid ? rowH[r] - c * inv_tau + rowM[r] * L2 * kLn2 : 0.f;
    if (lane == 0 && loss_per_token) loss_per_token[rowmap != nullptr ? (int64_t)tok : r] = l;
  }
  if (lane == 0) red[wave] = l;
  __syncthreads();
  if (threadIdx.x == 0) block_partial[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

// loss = (sum of the loss partials) / N_valid, in a fixed order: thread i sums
// partials i, i + 1024, ..., then a tree over the threads.
constexpr int kFinThreads = 1024;
__global__ __launch_bounds__(kFinThreads) void k_finalize_loss(const float* partials, int n,
                                                               const float* inv_nvalid,
                                                               float* loss) {
  __shared__ float red[kFinThreads];
  float s = 0.f;
  for (int i = threadIdx.x; i < n; i += kFinThreads) s += partials[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int o = kFinThreads / 2; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) loss[0] = red[0] * inv_nvalid[0];
}

// -------------------------------------------------------------------- dH ----
// dH_c[t, d] = sum_v dZ[t, v] W[v, d]: A = dZ (K = vocabulary contiguous),
// B = W read K-major (rows v, columns d); rows of W past V read as zeros. With
// split > 1 each split covers a K range and writes fp32 partials. With a
// rowmap, dZ row t is grad_hidden row rowmap[t] (-1: none), and only the
// first *nrow - nrow_base rows hold tokens (tiles past them are skipped).
template <typename T>
__global__ __launch_bounds__(kThreads, 1) void k_dh(const T* __restrict__ dZ, int64_t ldz,
                                                    const T* __restrict__ W, int V, int rows,
                                                    int D, int TM, int TN, int ks_total,
                                                    int split, void* gH, int gh_f32,
                                                    float* partial,
                                                    const float* __restrict__ rowscale,
                                                    const int* __restrict__ rowmap,
                                                    const int* __restrict__ nrow, int nrow_base) {
  __shared__ __attribute__((aligned(16))) char lds[kLdsA3];
  const int tiles = TM * TN;
  const int sidx = blockIdx.x / tiles;
  int mt, nt;
  tile_coords(blockIdx.x - sidx * tiles, TM, TN, 4, mt, nt);
  const int m0 = mt * kTile, n0 = nt * kTile;
  if (rowmap != nullptr && m0 >= __builtin_amdgcn_readfirstlane(*nrow) - nrow_base) return;
  const int eb = Elt<T>::bytes;
  const int lda = (int)(ldz * eb), ldb = D * eb;
  const int per = (ks_total + split - 1) / split;
  const int kb = sidx * per, ke = min(ks_total, kb + per);
  AccTile acc;
  const int mrows = min(kTile, rows - m0);
  // the row factors of the tile's 256 rows, loaded before the main loop and
  // kept in LDS for the epilogue: a load there would wait for every store
  // issued before it (loads and stores complete in order)
  const int tid = threadIdx.x;
  const float rsv =
      (rowscale != nullptr && split == 1 && tid < kTile && m0 + tid < rows) ? rowscale[m0 + tid]
                                                                           : 1.f;
  gemm_tile<T, KcOp, KmOp, 8, true, 3>(
      KcOp{reinterpret_cast<const char*>(dZ + (int64_t)m0 * ldz), (uint32_t)(mrows * lda), lda},
               KmOp{reinterpret_cast<const char*>(W + n0),
                    (int64_t)V * ldb - (int64_t)n0 * eb, ldb},
               kb, ke, lds, acc);
  const int lane = tid & 63, wave = wave_id();
  const int wm = wave >> 2, wn = wave & 3;
  float* rsl = reinterpret_cast<float*>(lds);
  int* rml = reinterpret_cast<int*>(lds) + kTile;
  if (tid < kTile) {
    rsl[tid] = rsv;
    // the output row of each of the tile's rows (loaded here: nothing of the
    // unmasked call is kept live through the main loop for it)
    rml[tid] = (rowmap != nullptr && split == 1 && m0 + tid < rows) ? rowmap[m0 + tid] : m0 + tid;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const f32x4_t sc = *reinterpret_cast<const f32x4_t*>(rsl + acc_m(wm, i, lane, 0));
    const i32x4_t om = *reinterpret_cast<const i32x4_t*>(rml + acc_m(wm, i, lane, 0));
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int d = n0 + acc_n(wn, j, lane);
      if (d >= D) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = m0 + acc_m(wm, i, lane, r);
        if (t < rows) {
          if (split == 1) {
            const float v = acc.v[i][j][r] * sc[r];
            const int64_t o = om[r];  // the grad_hidden row
            if (o < 0) continue;
            if (gh_f32)
              static_cast<float*>(gH)[o * D + d] = v;
            else
              static_cast<T*>(gH)[o * D + d] = (T)v;
          } else
            partial[((int64_t)sidx * rows + t) * D + d] = acc.v[i][j][r];
        }
      }
    }
  }
}

template <typename T>
__global__ void k_dh_reduce(const float* partial, int split, int64_t n, int D,
                            const float* __restrict__ rowscale, void* gH, int gh_f32,
                            const int* __restrict__ rowmap) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) {
    const int64_t t = i / D;
    // with a rowmap: the grad_hidden row of dZ row t (rows without a token,
    // whose partials were never written, are skipped)
    const int64_t o = rowmap != nullptr ? (int64_t)rowmap[t] * D + (i - t * D) : i;
    if (o < 0) continue;
    float s = 0.f;
    for (int k = 0; k < split; ++k) s += partial[(int64_t)k * n + i];
    const float v = rowscale ? s * rowscale[t] : s;
    if (gh_f32)
      static_cast<float*>(gH)[o] = v;
    else
      static_cast<T*>(gH)[o] = (T)v;
  }
}

// -------------------------------------------------------------------- dW ----
// The group's hidden rows transposed: Ht[d, t] = H[t, d] for t < tokens and 0
// for tokens <= t < ldt (ldt a multiple of 64), so that the dW contraction
// reads them with the tokens (its K dimension) contiguous. One 64 x 64 block
// per workgroup, 16-byte loads and stores on both sides. With a rowmap,
// column t is hidden row rowmap[t] (-1: zeros).
template <typename T>
__global__ __launch_bounds__(256) void k_transpose_rows(const T* __restrict__ H, int tokens,
                                                         int D, T* __restrict__ Ht, int ldt,
                                                         const float* __restrict__ rowscale,
                                                         const int* __restrict__ rowmap) {
  constexpr int VPT = 16 / (int)sizeof(T);      // elements per 16-byte piece
  constexpr int PAD = 4 / (int)sizeof(T);       // one dword of padding per LDS row
  __shared__ T tile[64][64 + PAD];              // [token][feature]
  const int t0 = blockIdx.x * 64, d0 = blockIdx.y * 64;
  const int tid = threadIdx.x;
#pragma unroll
  for (int u = 0; u < 64 * 64 / VPT / 256; ++u) {
    const int q = tid + 256 * u;
    const int row = q / (64 / VPT), c = (q % (64 / VPT)) * VPT;
    u32x4_t v = u32x4_t{0u, 0u, 0u, 0u};
    const int64_t src = t0 + row >= tokens ? -1 : rowmap != nullptr ? rowmap[t0 + row] : t0 + row;
    if (src >= 0) v = *reinterpret_cast<const u32x4_t*>(H + src * D + d0 + c);
    T e[VPT];
    __builtin_memcpy(e, &v, 16);
    // a per-token factor of the gradient rows is applied to the hidden rows
    // here, so that dW = sum_t (factor_t H_t)^T dZ''_t
    const float f = (rowscale != nullptr && t0 + row < tokens) ? rowscale[t0 + row] : 1.f;
#pragma unroll
    for (int x = 0; x < VPT; ++x) tile[row][c + x] = rowscale ? (T)((float)e[x] * f) : e[x];
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < 64 * 64 / VPT / 256; ++u) {
    const int q = tid + 256 * u;
    const int d = q / (64 / VPT), c = (q % (64 / VPT)) * VPT;
    T e[VPT];
#pragma unroll
    for (int x = 0; x < VPT; ++x) e[x] = tile[c + x][d];
    u32x4_t v;
    __builtin_memcpy(&v, e, 16);
    *reinterpret_cast<u32x4_t*>(Ht + (int64_t)(d0 + d) * ldt + t0 + c) = v;
  }
}

// grad_W[v, d] (+)= sum_t dZ[t, v] H[t, d] over the tokens of a group of
// chunks, computed as the tile C[d, v] = Ht[d, :] dZ[:, v]: A = the transposed
// hidden rows (K = tokens contiguous, zero past the group), B = dZ read
// K-major (rows = tokens; rows past the group read as zeros). Lane (g, c) of
// a wave holds C at four consecutive d of one v for each block, i.e. 16
// contiguous bytes of a grad_W row, so the tile goes to memory straight from
// the accumulators: with beta = 1 one half of the tile's old values is loaded,
// added, and the other half's loads are issued before the first half's stores
// (loads and stores complete in issue order, so waiting for those loads does
// not wait for the stores).
//
// SPLIT (for a tile count that leaves the last round of the 256 compute units
// partly filled): blocks [0, nfull) compute the whole tiles of the full
// rounds (in the XCD-aware order over those), and the tail tiles are split
// into `split` token ranges, block nfull + split q + s taking range s of tail
// tile nfull + q and storing its fp32 partial tile (pitch 256) at partial
// slot split q + s; k_dw_fixup then adds the parts to grad_W in a fixed
// order, so the last round is split times shorter. Without SPLIT every block
// computes a whole tile (nfull, split and partial unused).
//
// With nrow (ignored tokens left out), only the group's first *nrow dZ rows
// hold tokens: the K range stops there, and the dZ rows past it read as
// zeros.
template <typename T, bool SPLIT>
__global__ __launch_bounds__(kThreads, 1) void k_dw(const T* __restrict__ Ht, int ldt,
                                                    const T* __restrict__ dZ, int64_t ldz,
                                                    int tokens, int V, int D, int TM, int TN,
                                                    int beta, float* __restrict__ gW, int nfull,
                                                    int split, float* __restrict__ partial,
                                                    const int* __restrict__ nrow) {
  __shared__ __attribute__((aligned(16))) char lds[kLdsA3];
  constexpr int KS = kRowB / (int)sizeof(T);
  if (nrow != nullptr) tokens = min(tokens, __builtin_amdgcn_readfirstlane(*nrow));
  const int nks = min(ldt / KS, (tokens + KS - 1) / KS);
  const int pid = blockIdx.x;
  int L, ks0 = 0, ks1 = nks, slot = -1;
  if (!SPLIT) {
    L = tile_order_xcd(pid, TM * TN);
  } else if (pid < nfull) {
    L = tile_order_xcd(pid, nfull);
  } else {
    const int q = (pid - nfull) / split, s = (pid - nfull) - q * split;
    L = nfull + q;
    slot = q * split + s;
    ks0 = (int)((int64_t)nks * s / split);
    ks1 = (int)((int64_t)nks * (s + 1) / split);
  }
  int mt, nt;
  tile_at(L, TM, TN, 4, mt, nt);
  const int m0 = mt * kTile, n0 = nt * kTile;  // m: feature d, n: vocabulary v
  const int eb = Elt<T>::bytes;
  const int lda = ldt * eb, ldb = (int)(ldz * eb);
  const int mrows = min(kTile, D - m0);
  AccTile acc;
  gemm_tile<T, KcOp, KmOp, 8, true, 3>(
      KcOp{reinterpret_cast<const char*>(Ht + (int64_t)m0 * ldt), (uint32_t)(mrows * lda), lda},
      KmOp{reinterpret_cast<const char*>(dZ + n0), (int64_t)tokens * ldb - (int64_t)n0 * eb, ldb},
      ks0, ks1, lds, acc);
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int wm = wave >> 2, wn = wave & 3;
  // the tile's rows of grad_W (or of its partial slot, pitch 256) as one
  // resource: rows past V are out of range (loads give 0, stores are
  // dropped), features past D get an out-of-range offset
  const bool part = SPLIT && slot >= 0;
  const int pitch = part ? kTile : D;
  const int vrows = __builtin_amdgcn_readfirstlane(part ? kTile : min(kTile, V - n0));
  const __amdgpu_buffer_rsrc_t ro =
      part ? make_rsrc(partial + (int64_t)slot * kTile * kTile, (uint32_t)kTile * kTile * 4u)
           : make_rsrc(gW + (int64_t)n0 * D, (uint32_t)vrows * (uint32_t)D * 4u);
  // block (i, j) sits at byte offset obase + 64 i (16 features) + 64 pitch j
  // (16 rows): the per-lane part is one register, 64 i goes into the
  // instruction's immediate offset and 64 pitch j into its scalar offset. D
  // is a multiple of 64, so whether block i's features exist is the same for
  // the whole wave.
  const int dw0 = (part ? 0 : m0) + wm * 128;
  const uint32_t obase =
      ((uint32_t)acc_n(wn, 0, lane) * (uint32_t)pitch + (uint32_t)(dw0 + 4 * (lane >> 4))) * 4u;
  const uint32_t jstep = 64u * (uint32_t)pitch;
  auto ld = [&](int i, int j) {
    return __builtin_bit_cast(
        f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(ro, obase + 64u * i, jstep * j, 0));
  };
  auto st = [&](int i, int j, f32x4_t v) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), ro, obase + 64u * i,
                                           jstep * j, 0);
  };
  auto live = [&](int i) { return part || dw0 + 16 * i < D; };
  if (beta && !part) {
    f32x4_t old[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (live(i))
#pragma unroll
        for (int j = 0; j < 4; ++j) old[i][j] = ld(i, j);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (live(i))
#pragma unroll
        for (int j = 0; j < 4; ++j) acc.v[i][j] += old[i][j];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (live(4 + i))
#pragma unroll
        for (int j = 0; j < 4; ++j) old[i][j] = ld(4 + i, j);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (live(i))
#pragma unroll
        for (int j = 0; j < 4; ++j) st(i, j, acc.v[i][j]);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (live(4 + i))
#pragma unroll
        for (int j = 0; j < 4; ++j) st(4 + i, j, acc.v[4 + i][j] + old[i][j]);
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (live(i))
#pragma unroll
        for (int j = 0; j < 4; ++j) st(i, j, acc.v[i][j]);
  }
}

// The split tail tiles of k_dw: grad_W = (beta ? grad_W : 0) + part 0 + part 1
// + ... in this order. One thread per 4 features of a vocabulary row of a tail
// tile (grid: tail tiles x 256 rows x 64 threads).
__global__ __launch_bounds__(256) void k_dw_fixup(const float* __restrict__ partial, int split,
                                                  int nfull, int TM, int TN, int V, int D,
                                                  int beta, float* __restrict__ gW) {
  const int q = blockIdx.x;                      // tail tile
  const int row = blockIdx.y * 4 + (threadIdx.x >> 6);
  const int c4 = (threadIdx.x & 63) * 4;         // first of 4 features in the tile
  int mt, nt;
  tile_at(nfull + q, TM, TN, 4, mt, nt);
  const int v = nt * kTile + row, d = mt * kTile + c4;
  if (v >= V || d >= D) return;
  f32x4_t sum = beta ? *reinterpret_cast<const f32x4_t*>(gW + (int64_t)v * D + d)
                     : f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < split; ++s)
    sum += *reinterpret_cast<const f32x4_t*>(partial + ((int64_t)(q * split + s) * kTile + row) *
                                                           kTile + c4);
  *reinterpret_cast<f32x4_t*>(gW + (int64_t)v * D + d) = sum;
}

// ------------------------------------------------- ignored tokens left out --
// The tokens of a dW group [row0, row0 + rows) that are not ignored, in
// order: rowmap[j] = the j-th of them, -1 for j >= their count, *nrow = the
// count. One workgroup: thread i counts a contiguous run of the mask, an
// exclusive scan of the counts over the threads gives each run its first
// slot.
constexpr int kScanThreads = 1024;
__global__ __launch_bounds__(kScanThreads) void k_compact_scan(const uint8_t* __restrict__ ignore,
                                                               int64_t row0, int rows,
                                                               int* __restrict__ rowmap,
                                                               int* __restrict__ nrow) {
  __shared__ int sc[kScanThreads];
  const int tid = threadIdx.x;
  const int per = (rows + kScanThreads - 1) / kScanThreads;
  const int b = min(rows, tid * per), e = min(rows, b + per);
  const uint8_t* m = ignore + row0;
  int c = 0;
  for (int i = b; i < e; ++i) c += m[i] == 0 ? 1 : 0;
  sc[tid] = c;
  __syncthreads();
  // inclusive scan (Hillis-Steele) of the counts
  for (int o = 1; o < kScanThreads; o <<= 1) {
    const int add = tid >= o ? sc[tid - o] : 0;
    __syncthreads();
    sc[tid] += add;
    __syncthreads();
  }
  int pos = sc[tid] - c;
  const int total = sc[kScanThreads - 1];
  for (int i = b; i < e; ++i)
    if (m[i] == 0) rowmap[pos++] = (int)(row0 + i);
  for (int j = total + tid; j < rows; j += kScanThreads) rowmap[j] = -1;
  if (tid == 0) nrow[0] = total;
}

// Row j of the group: hidden row rowmap[j] copied to hcomp row j (j < *nrow);
// if token row0 + j is ignored, its grad_hidden row, per-token loss and saved
// log Z are set to 0 (the rest of the call never writes them). One workgroup per row,
// 16 bytes per thread and step.
__global__ __launch_bounds__(256) void k_compact_rows(const char* __restrict__ hidden,
                                                      int64_t row_bytes, int64_t row0,
                                                      const uint8_t* __restrict__ ignore,
                                                      const int* __restrict__ rowmap,
                                                      const int* __restrict__ nrow,
                                                      char* __restrict__ hcomp, char* gH,
                                                      int64_t gh_row_bytes, float* lpt,
                                                      float* logz) {
  const int j = blockIdx.x;
  const int tid = threadIdx.x;
  if (j < nrow[0]) {
    const u32x4_t* src = reinterpret_cast<const u32x4_t*>(hidden + (int64_t)rowmap[j] * row_bytes);
    u32x4_t* dst = reinterpret_cast<u32x4_t*>(hcomp + (int64_t)j * row_bytes);
    for (int64_t q = tid; q < row_bytes / 16; q += 256) dst[q] = src[q];
  }
  const int64_t t = row0 + j;
  if (ignore[t] != 0) {
    if (gH != nullptr) {
      u32x4_t* z = reinterpret_cast<u32x4_t*>(gH + t * gh_row_bytes);
      for (int64_t q = tid; q < gh_row_bytes / 16; q += 256) z[q] = u32x4_t{0u, 0u, 0u, 0u};
    }
    if (tid == 0) {
      if (lpt != nullptr) lpt[t] = 0.f;
      if (logz != nullptr) logz[t] = 0.f;
    }
  }
}

// ------------------------------------------------------------ index check --
// flag |= 1 if an index is outside [0, V); |= 2 if a row repeats an index.
__global__ void k_check_indices(const int32_t* idx, int64_t N, int K, int64_t V, int* flag) {
  const int64_t r = (int64_t)blockIdx.x * 4 + wave_id();
  const int lane = threadIdx.x & 63;
  if (r >= N) return;
  const int32_t* row = idx + r * K;
  int bad = 0;
  for (int k = lane; k < K; k += 64) {
    const int32_t v = row[k];
    if (v < 0 || (int64_t)v >= V) bad |= 1;
    for (int k2 = k + 1; k2 < K; ++k2)
      if (row[k2] == v) bad |= 2;
  }
  if (bad) atomicOr(flag, bad);
}


// ------------------------------------------------- upstream-gradient scale --
// y = g x elementwise, g a device scalar: the gradients of the mean loss
// times the upstream gradient of that mean (Algorithm 1's backward scales G
// by g; the loss is linear in g, so scaling the finished gradients is the
// same function). fp32 in; out in fp32 or bf16 (one rounding); in place when
// x and y are the same fp32 buffer. Each thread handles 8 elements, 16-byte
// accesses where the 8 are in range (the buffers are 16-byte aligned).
template <typename TO>
__global__ void k_scale_f32(const float* x, TO* y, int64_t n, const float* __restrict__ g) {
  const float s = g[0];
  const int64_t stride = (int64_t)gridDim.x * blockDim.x * 8;
  for (int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 8; i < n; i += stride) {
    if (i + 8 <= n) {
      const f32x4_t a = *reinterpret_cast<const f32x4_t*>(x + i) * s;
      const f32x4_t b = *reinterpret_cast<const f32x4_t*>(x + i + 4) * s;
      if constexpr (sizeof(TO) == 2) {
        *reinterpret_cast<u32x4_t*>(y + i) =
            u32x4_t{pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]), pack_bf16x2(b[0], b[1]),
                    pack_bf16x2(b[2], b[3])};
      } else {
        *reinterpret_cast<f32x4_t*>(y + i) = a;
        *reinterpret_cast<f32x4_t*>(y + i + 4) = b;
      }
    } else {
      for (int64_t k = i; k < n; ++k) y[k] = (TO)(x[k] * s);
    }
  }
}

}  // namespace kd

// ================================================================ launchers ==
using namespace kd;

#include <atomic>
#include <mutex>
#include <vector>

#include "../../include/kdtopk.h"

static inline int cdiv(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// ------------------------------------------------- event instrumentation ----
namespace {
enum ProfKind {
  P_COUNT_VALID, P_PROLOGUE, P_BUCKET, P_LOGITS, P_MERGE, P_DZ, P_ROW_LOSS, P_DH, P_DH_REDUCE,
  P_DW, P_FINALIZE, P_FILL, P_TRANSPOSE, P_LOGITS_DZ, P_REF, P_ROW_FINISH, P_DW_FIXUP,
  P_COMPACT, P_NKINDS
};
const char* const kProfNames[P_NKINDS] = {
    "count_valid", "teacher_prologue", "bucket", "logits_lse", "lse_merge", "dz", "row_loss",
    "dh", "dh_reduce", "dw", "finalize_loss", "fill", "transpose_rows", "logits_dz", "ref_logit",
    "row_finish", "dw_fixup", "compact"};
struct ProfRec {
  int kind;
  hipEvent_t a, b;
  double flops;
};
std::atomic<int> g_prof_mode{0};  // 0 off, 1 every kernel, 2 contractions only
// set while the allocation-free entry point enqueues: no events are created
thread_local bool t_prof_suppressed = false;
std::mutex g_prof_mu;
std::vector<ProfRec> g_prof_recs;
std::vector<hipEvent_t> g_prof_pool;

hipEvent_t prof_event() {
  if (!g_prof_pool.empty()) {
    hipEvent_t e = g_prof_pool.back();
    g_prof_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Records an event pair around the launches in its scope when enabled.
struct ProfScope {
  int kind;
  double flops;
  hipStream_t s;
  hipEvent_t a = nullptr;
  ProfScope(int k, double f, hipStream_t st) : kind(k), flops(f), s(st) {
    const int mode = g_prof_mode.load(std::memory_order_relaxed);
    if (mode == 0 || (mode == 2 && f == 0.0) || t_prof_suppressed) return;
    std::lock_guard<std::mutex> g(g_prof_mu);
    a = prof_event();
    if (a) (void)hipEventRecord(a, s);
  }
  ~ProfScope() {
    if (!a) return;
    std::lock_guard<std::mutex> g(g_prof_mu);
    hipEvent_t b = prof_event();
    if (!b) {
      g_prof_pool.push_back(a);  // no pair: drop this record, keep the event
      return;
    }
    (void)hipEventRecord(b, s);
    g_prof_recs.push_back({kind, a, b, flops});
  }
};
}  // namespace

extern "C" kd_status kd_profile_enable(int mode) {
  if (mode < 0 || mode > 2) return KD_ERR_BAD_ARG;
  g_prof_mode.store(mode);
  return KD_OK;
}

extern "C" int kd_profile_read(kd_kernel_time* out, int max) {
  std::lock_guard<std::mutex> g(g_prof_mu);
  double ms[P_NKINDS] = {0}, fl[P_NKINDS] = {0};
  int64_t n[P_NKINDS] = {0};
  int rc = 0;
  for (const ProfRec& r : g_prof_recs) {
    float t = 0.f;
    if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&t, r.a, r.b) != hipSuccess)
      rc = -1;
    ms[r.kind] += t;
    fl[r.kind] += r.flops;
    n[r.kind] += 1;
    g_prof_pool.push_back(r.a);
    g_prof_pool.push_back(r.b);
  }
  g_prof_recs.clear();
  if (rc != 0) return rc;
  int w = 0;
  for (int k = 0; k < P_NKINDS && w < max; ++k) {
    if (n[k] == 0) continue;
    kd_kernel_time& o = out[w++];
    memset(o.name, 0, sizeof(o.name));
    strncpy(o.name, kProfNames[k], sizeof(o.name) - 1);
    o.launches = n[k];
    o.total_ms = ms[k];
    o.flops = fl[k];
  }
  return w;
}

template <typename T>
static int launch_chunk_impl(const KdChunkArgs& a, hipStream_t s) {
  const T* W = static_cast<const T*>(a.W);
  const T* Hc = static_cast<const T*>(a.Hc);
  const int TMv = cdiv(a.V, kTile), TNt = cdiv(a.rows, kTile);
  const float k2 = kLog2e * a.inv_tau;
  const double gemm_flops = 2.0 * (double)a.rows * (double)a.D * (double)a.V;

  const bool fwd = a.mode != KD_MODE_BWD, bwd = a.mode != KD_MODE_FWD;
  if (a.stages & KD_STAGE_PREP) {
    {
      ProfScope ps_(P_PROLOGUE, 0.0, s);
      hipLaunchKernelGGL(k_teacher_prologue, dim3(a.rows), dim3(64),
                         (size_t)4 * prologue_hash_slots(a.K) + (size_t)8 * a.K, s, a.tidx_in,
                         a.tidx, a.tlogit, a.ignore, a.row0, a.rowmap, a.rows, a.K, (int)a.V,
                         a.inv_tau,
                         a.teacher_logprobs, a.inv_nvalid, a.gscale, a.gtok,
                         fwd ? nullptr : a.logz_in, a.p, a.rowM, a.rowH, a.rowCoef, a.rowCoefM,
                         a.rowL2);
    }
    {
      ProfScope ps_(P_BUCKET, 0.0, s);
      hipLaunchKernelGGL(k_bucket, dim3(TNt), dim3(kBucketThreads), 0, s, a.tidx, a.p, a.rows,
                         a.K, (int)a.V, a.nVT, a.hits, a.hitp, a.hoff, a.zhit);
    }
    if (a.one_projection) {
      ProfScope ps_(P_REF, 0.0, s);
      hipLaunchKernelGGL(k_ref_logit<T>, dim3(cdiv(a.rows, 4)), dim3(256), 0, s,
                         static_cast<const T*>(a.hidden), W, (int)a.D, a.tidx, a.tlogit, a.row0,
                         a.rowmap, a.rows, a.K, (int)a.V, k2, a.rowR, a.rowFlag);
    }
  }
  if (!(a.stages & KD_STAGE_CHUNK)) return (int)hipGetLastError();
  if (a.one_projection) {
    // loss and gradients together: one projection per chunk (k_logits_dz)
    // against the reference logit, then the merge of log Z with the row
    // factors, the fallback rows, the teacher cells and the row losses
    {
      ProfScope ps_(P_LOGITS_DZ, gemm_flops, s);
      hipLaunchKernelGGL(k_logits_dz<T>, dim3(TMv * TNt), dim3(kThreads), 0, s, W, Hc, (int)a.D,
                         (int)a.V, a.rows, TMv, TNt, k2, a.part_m, a.part_s, a.nVT, a.hits,
                         a.hoff, a.K, static_cast<T*>(a.dZ), a.ldz, a.zhit, a.rowR, a.rowFlag,
                         a.nrow, a.nrow_base);
    }
    {
      ProfScope ps_(P_ROW_FINISH, 0.0, s);
      hipLaunchKernelGGL(k_row_finish<T>, dim3(cdiv(a.rows, kLossRows)), dim3(64 * kLossRows), 0,
                         s, a.part_m, a.part_s, a.nVT, a.rowFlag, static_cast<T*>(a.dZ), a.ldz,
                         a.tidx, a.p, a.zhit, a.K, (int)a.V, k2, a.rowM, a.rowH, a.rowCoef,
                         a.rowCoefM, a.ignore, a.row0, a.rowmap, a.rows, a.inv_tau, a.rowL2,
                         a.rowFactor, a.loss_per_token, a.block_partial);
    }
  } else {
    if (fwd) {
      {
        ProfScope ps_(P_LOGITS, gemm_flops, s);
        // no recompute follows (forward only, or a fused call that wants no
        // gradients): z at the teacher entries comes from this GEMM
        hipLaunchKernelGGL(k_logits_lse<T>, dim3(TMv * TNt), dim3(kThreads), 0, s, W, Hc,
                           (int)a.D, (int)a.V, a.rows, TMv, TNt, k2, a.part_m, a.part_s, a.nVT,
                           a.hits, a.hoff, a.K, a.zhit, a.nrow, a.nrow_base);
      }
      {
        ProfScope ps_(P_MERGE, 0.0, s);
        hipLaunchKernelGGL(k_lse_merge, dim3(cdiv(a.rows, 4)), dim3(256), 0, s, a.part_m,
                           a.part_s, a.rows, a.nVT, a.rowL2, a.rowmap);
      }
    }
    if (bwd && !fwd) {
      // the backward of the split entry points: the logit recompute from the
      // saved log Z (Algorithm 1's backward)
      ProfScope ps_(P_DZ, gemm_flops, s);
      hipLaunchKernelGGL(k_dz<T>, dim3(TMv * TNt), dim3(kThreads), 0, s, W, Hc, (int)a.D,
                         (int)a.V, a.rows, TMv, TNt, k2, a.rowL2, a.rowCoef, a.rowCoefM, a.hits,
                         a.hitp, a.hoff, a.K, a.nVT, static_cast<T*>(a.dZ), a.ldz,
                         (float*)nullptr, a.nrow, a.nrow_base);
    }
    if (fwd) {
      ProfScope ps_(P_ROW_LOSS, 0.0, s);
      hipLaunchKernelGGL(k_row_loss, dim3(cdiv(a.rows, kLossRows)), dim3(64 * kLossRows), 0, s,
                         a.zhit, a.p, a.K, a.rowL2, a.rowM, a.rowH, a.ignore, a.row0, a.rowmap,
                         a.rows, a.inv_tau, a.loss_per_token, a.logz_out, a.block_partial);
    }
  }
  return (int)hipGetLastError();
}

extern "C" int kd_launch_chunk(const KdChunkArgs* a, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  return a->dtype == 1 ? launch_chunk_impl<__bf16>(*a, s) : launch_chunk_impl<float>(*a, s);
}

template <typename T>
static int launch_dh_impl(const KdDhArgs& a, hipStream_t s) {
  const int rows = (int)a.tokens;
  const int TM = cdiv(rows, kTile), TN = cdiv(a.D, kTile);
  const int ks = (int)(a.ldz * sizeof(T) / kRowB);
  {
    ProfScope ps_(P_DH, 2.0 * (double)a.tokens * (double)a.D * (double)a.V, s);
    hipLaunchKernelGGL(k_dh<T>, dim3(TM * TN * a.split), dim3(kThreads), 0, s,
                       static_cast<const T*>(a.dZ), a.ldz, static_cast<const T*>(a.W), (int)a.V,
                       rows, (int)a.D, TM, TN, ks, a.split, a.gH, a.gh_f32, a.partial,
                       a.rowscale, a.rowmap, a.nrow, a.nrow_base);
  }
  if (a.split > 1) {
    const int64_t n = (int64_t)rows * a.D;
    ProfScope ps_(P_DH_REDUCE, 0.0, s);
    hipLaunchKernelGGL(k_dh_reduce<T>, dim3(std::min<int64_t>(cdiv(n, 256), 8192)), dim3(256), 0,
                       s, a.partial, a.split, n, (int)a.D, a.rowscale, a.gH, a.gh_f32, a.rowmap);
  }
  return (int)hipGetLastError();
}

extern "C" int kd_launch_dh(const KdDhArgs* a, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  return a->dtype == 1 ? launch_dh_impl<__bf16>(*a, s) : launch_dh_impl<float>(*a, s);
}

template <typename T>
static int launch_dw_impl(const KdDwArgs& a, hipStream_t s) {
  const int ldt = (int)(((a.tokens + 63) / 64) * 64);
  T* Ht = static_cast<T*>(a.Ht);
  {
    ProfScope ps_(P_TRANSPOSE, 0.0, s);
    hipLaunchKernelGGL(k_transpose_rows<T>, dim3(ldt / 64, (int)(a.D / 64)), dim3(256), 0, s,
                       static_cast<const T*>(a.Hg), (int)a.tokens, (int)a.D, Ht, ldt,
                       a.rowscale, a.rowmap);
  }
  const int TM = cdiv(a.D, kTile), TN = cdiv(a.V, kTile);
  const int tiles = TM * TN;
  // a partly filled last round of the 256 compute units is split along the
  // tokens when the host provides the partial tiles' workspace
  int nfull = tiles, split = 1;
  const int nks = ldt * (int)sizeof(T) / kRowB;
  if (a.partial != nullptr && tiles > kDwUnits && tiles % kDwUnits != 0) {
    const int tail = tiles % kDwUnits;
    split = std::min(kDwMaxSplit, std::min(kDwUnits / tail, nks));
    if (split >= 2) nfull = tiles - tail;
    else split = 1;
  }
  {
    ProfScope ps_(P_DW, 2.0 * (double)a.tokens * (double)a.D * (double)a.V, s);
    if (nfull < tiles)
      hipLaunchKernelGGL((k_dw<T, true>), dim3(nfull + (tiles - nfull) * split), dim3(kThreads),
                         0, s, static_cast<const T*>(Ht), ldt, static_cast<const T*>(a.dZ), a.ldz,
                         (int)a.tokens, (int)a.V, (int)a.D, TM, TN, a.beta, a.gW, nfull, split,
                         a.partial, a.nrow);
    else
      hipLaunchKernelGGL((k_dw<T, false>), dim3(tiles), dim3(kThreads), 0, s,
                         static_cast<const T*>(Ht), ldt, static_cast<const T*>(a.dZ), a.ldz,
                         (int)a.tokens, (int)a.V, (int)a.D, TM, TN, a.beta, a.gW, tiles, 1,
                         (float*)nullptr, a.nrow);
  }
  if (nfull < tiles) {
    ProfScope ps_(P_DW_FIXUP, 0.0, s);
    hipLaunchKernelGGL(k_dw_fixup, dim3(tiles - nfull, kTile / 4), dim3(256), 0, s, a.partial,
                       split, nfull, TM, TN, (int)a.V, (int)a.D, a.beta, a.gW);
  }
  return (int)hipGetLastError();
}

extern "C" int kd_launch_dw(const KdDwArgs* a, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  return a->dtype == 1 ? launch_dw_impl<__bf16>(*a, s) : launch_dw_impl<float>(*a, s);
}

extern "C" int kd_launch_compact(const KdCompactArgs* a, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (a->rows <= 0) return 0;
  const int64_t eb = a->dtype == 1 ? 2 : 4;
  {
    ProfScope ps_(P_COMPACT, 0.0, s);
    hipLaunchKernelGGL(k_compact_scan, dim3(1), dim3(kScanThreads), 0, s, a->ignore, a->row0,
                       a->rows, a->rowmap, a->nrow);
    hipLaunchKernelGGL(k_compact_rows, dim3(a->rows), dim3(256), 0, s,
                       static_cast<const char*>(a->hidden), a->D * eb, a->row0, a->ignore,
                       a->rowmap, a->nrow, static_cast<char*>(a->hcomp),
                       static_cast<char*>(a->grad_hidden), a->D * (a->gh_f32 ? 4 : eb),
                       a->loss_per_token, a->logz_out);
  }
  return (int)hipGetLastError();
}

extern "C" int kd_launch_prepare(const KdPrepareArgs* a, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  {
    ProfScope ps_(P_COUNT_VALID, 0.0, s);
    hipLaunchKernelGGL(k_count_valid, dim3(1), dim3(kCountThreads), 0, s, a->ignore, a->N,
                       a->nvalid, a->inv_nvalid);
  }
  if (a->zero_gW != nullptr) {
    const int64_t n = a->V * a->D;
    ProfScope ps_(P_FILL, 0.0, s);
    hipLaunchKernelGGL(k_fill_f32, dim3(std::min<int64_t>(cdiv(n, 256), 16384)), dim3(256), 0, s,
                       a->zero_gW, n, 0.0f);
  }
  return (int)hipGetLastError();
}

extern "C" int kd_launch_finalize(const float* partials, int n, const float* inv_nvalid,
                                  float* loss, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  {
    ProfScope ps_(P_FINALIZE, 0.0, s);
    hipLaunchKernelGGL(k_finalize_loss, dim3(1), dim3(kFinThreads), 0, s, partials, n, inv_nvalid,
                       loss);
  }
  return (int)hipGetLastError();
}

extern "C" int kd_launch_check_indices(const int32_t* idx, int64_t N, int K, int64_t V,
                                       int* flag, int* host_flag, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipMemsetAsync(flag, 0, sizeof(int), s);
  if (e != hipSuccess) return (int)e;
  if (N > 0)
    hipLaunchKernelGGL(k_check_indices, dim3(cdiv(N, 4)), dim3(256), 0, s, idx, N, K, V, flag);
  e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  e = hipMemcpyAsync(host_flag, flag, sizeof(int), hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return (int)e;
  return (int)hipStreamSynchronize(s);
}

// y = g x for the gradients (see k_scale_f32): x fp32, y fp32 (out_bf16 = 0)
// or bf16 (out_bf16 = 1)
extern "C" int kd_launch_scale(int out_bf16, const float* x, void* y, int64_t n, const float* g,
                               void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (n <= 0) return 0;
  const int64_t blocks = std::min<int64_t>((n + 2047) / 2048, 8192);
  if (out_bf16)
    hipLaunchKernelGGL(k_scale_f32<__bf16>, dim3((int)blocks), dim3(256), 0, s, x,
                       static_cast<__bf16*>(y), n, g);
  else
    hipLaunchKernelGGL(k_scale_f32<float>, dim3((int)blocks), dim3(256), 0, s, x,
                       static_cast<float*>(y), n, g);
  return (int)hipGetLastError();
}

// ------------------------------------------------------ static scratch ------
// The workspace of the allocation-free entry point: one file-scope array per
// device, held until the process ends. In host code the array's name denotes
// a host-side stand-in, not device memory, so host code never uses it as an
// address: the device address comes from hipGetSymbolAddress, once per
// device with that device current, and only that address is passed to
// kernels. Every call on a device shares its array.
static __device__ __align__(256) char scratch[kd_scratch_bytes_max];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};
}  // namespace

extern "C" int kd_scratch_get(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return (int)e;
  if (dev < 0 || dev >= kMaxDevices) return (int)hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return (int)e;
    if (p == nullptr) return (int)hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *ptr = g_scratch[dev];
  return 0;
}

extern "C" void kd_launch_suppress_profiling(int on) { t_prof_suppressed = on != 0; }
