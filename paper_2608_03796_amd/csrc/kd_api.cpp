// C ABI of the fused chunked top-K KL loss: argument checks, workspace plan
// and the chunk schedule of Algorithm 1 (§3.2.3). Plain C++: every device
// operation goes through the launchers of kd_kernels.hip.
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>

#include "../../include/kdtopk.h"
#include "kd_launch.h"

static_assert(KD_SCRATCH_BYTES == kd_scratch_bytes_max, "scratch size in the header");

namespace {

constexpr int64_t kTile = 256;
constexpr int64_t kMaxN = (int64_t)1 << 31;     // N < 2^31
constexpr int64_t kMaxV = (int64_t)1 << 20;     // keeps 32-bit buffer offsets in range
constexpr int64_t kMaxD = 65536;
constexpr int64_t kMaxChunk = (int64_t)1 << 20; // rows per chunk actually used
// teacher entries per token: a 256-token tile's 256 K entries are numbered in
// 20 bits by the bucket pass, and k is packed in 16
constexpr int64_t kMaxK = 4096;

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t rup(int64_t a, int64_t b) { return cdiv(a, b) * b; }
inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct Plan {
  int64_t N, D, V, K;
  int eb;              // element bytes of hidden / W / dZ
  int64_t c;           // rows per chunk
  int64_t cp;          // c rounded up to the 256-row tile
  int64_t Vp;          // V rounded up to the 256-column tile
  int64_t nVT;         // vocabulary tiles
  int64_t nchunks;
  int64_t nblk;        // loss partials of a full chunk (one per kLossRows rows)
  int64_t G;           // chunks whose dZ rows are gathered before one dH and one dW GEMM
  int64_t merged;      // caller's chunks per chunk of the plan (1 or the group size)
  int64_t ngroups;
  bool dh_per_group;   // dH once per group (a chunk alone has too few tiles) or per chunk
  bool prep_per_group; // rows prepared once per group (chunks of whole 256-token tiles)
  int64_t ng;          // rows of the per-row arrays: the group's, or one chunk's (padded)
  int64_t td, ksteps;  // dH column tiles and K steps (for its vocabulary split)
  size_t off_misc, off_p, off_tidx, off_rows, off_pm, off_ps, off_hits, off_hitp, off_hoff, off_zhit,
      off_lossp, off_dz, off_fac, off_ht, off_rowmap, off_dhs, off_dwp, total;
};

kd_status check_problem(const kd_problem* p) {
  if (p == nullptr) return KD_ERR_NULL_PTR;
  if ((p->flags & ~(KD_FLAG_TEACHER_LOGPROBS | KD_FLAG_GRAD_HIDDEN_F32)) != 0) return KD_ERR_BAD_ARG;
  if (p->dtype != KD_F32 && p->dtype != KD_BF16) return KD_ERR_UNSUPPORTED;
  if (p->N < 0 || p->N >= kMaxN) return KD_ERR_BAD_SHAPE;
  if (p->D < 64 || p->D > kMaxD) return KD_ERR_BAD_SHAPE;
  if (p->V < 1 || p->V > kMaxV) return KD_ERR_BAD_SHAPE;
  if (p->K < 1 || (int64_t)p->K > p->V || p->K > kMaxK) return KD_ERR_BAD_SHAPE;
  if (p->chunk < 1) return KD_ERR_BAD_ARG;
  if (!(isfinite(p->temperature) && p->temperature > 0.0f)) return KD_ERR_BAD_ARG;
  if (p->D % 64 != 0) return KD_ERR_UNSUPPORTED;
  return KD_OK;
}

// Split of the dH GEMM's K range (the vocabulary) so that the number of
// workgroups fills whole waves of the 256 compute units.
int choose_dh_split(int64_t tiles, int64_t ksteps) {
  int best = 1;
  double best_eff = (double)tiles / (double)(cdiv(tiles, 256) * 256);
  for (int s = 2; s <= 16; ++s) {
    if (ksteps / s < 8) break;
    const double eff = (double)(tiles * s) / (double)(cdiv(tiles * s, 256) * 256);
    if (eff > best_eff + 0.05) {
      best = s;
      best_eff = eff;
    }
  }
  return best;
}

// g_max > 0 caps the chunks per dW group (see plan_within).
Plan make_plan(const kd_problem* p, int64_t g_max = 0) {
  Plan pl{};
  pl.N = p->N;
  pl.D = p->D;
  pl.V = p->V;
  pl.K = p->K;
  pl.eb = p->dtype == KD_BF16 ? 2 : 4;
  pl.c = std::min<int64_t>(std::min<int64_t>(p->chunk, std::max<int64_t>(p->N, 1)), kMaxChunk);
  pl.cp = rup(pl.c, kTile);
  pl.Vp = rup(pl.V, kTile);
  pl.nVT = pl.Vp / kTile;
  pl.nchunks = cdiv(pl.N, pl.c);
  pl.nblk = cdiv(pl.c, kLossRows);
  // dW is accumulated in fp32 in place: each dW GEMM reads and writes all of
  // grad_W once, so gather the dZ rows of up to ~16384 tokens (and at most
  // 4 GiB of dZ) per GEMM
  pl.G = std::max<int64_t>(1, std::min<int64_t>(16384 / pl.c, std::max<int64_t>(pl.nchunks, 1)));
  pl.G = std::max<int64_t>(
      1, std::min<int64_t>(pl.G, ((int64_t)4 << 30) / std::max<int64_t>(pl.c * pl.Vp * pl.eb, 1)));
  if (g_max > 0) pl.G = std::min<int64_t>(pl.G, g_max);
  // Chunks of whole 256-token tiles that share a dW group are processed as one
  // chunk of the group's rows when a chunk's projection leaves its last round
  // of tiles partly filled (its tiles are not a multiple of the 256 compute
  // units) and dH runs per group anyway: the same transient (the group's dZ
  // rows) and the same arithmetic per token and per grad_W contraction, with
  // one projection launch (and one teacher bucketing) per group, so the
  // partly filled round comes once per group. When a chunk's tiles fill whole
  // rounds, each chunk's dH right after its own projection measured faster
  // than one dH over the group.
  pl.merged = 1;
  const int64_t proj_tiles = cdiv(pl.c, kTile) * (pl.Vp / kTile);
  const bool dh_grouped =
      choose_dh_split(cdiv(pl.c, kTile) * cdiv(pl.D, kTile), pl.Vp * pl.eb / 128) > 1;
  if (pl.G > 1 && pl.c % kTile == 0 && proj_tiles % 256 != 0 && dh_grouped) {
    pl.merged = pl.G;
    pl.c *= pl.G;
    pl.cp = pl.c;
    pl.nchunks = cdiv(pl.N, pl.c);
    pl.nblk = cdiv(pl.c, kLossRows);
    pl.G = 1;
  }
  // dH runs per chunk when a chunk's tiles fill the chip, else once per group
  // of G chunks (G times the tiles, dW's grouping); its vocabulary range is
  // split only when the rows it covers still have too few tiles
  pl.ngroups = cdiv(pl.nchunks, pl.G);
  // the teacher prologue, bucketing and reference logits run once per group
  // when every chunk starts on a 256-token tile of the group (the buckets are
  // per tile), else once per chunk
  pl.prep_per_group = pl.G > 1 && pl.c % kTile == 0;
  pl.ng = pl.prep_per_group ? pl.G * pl.c : pl.cp;
  pl.td = cdiv(pl.D, kTile);
  pl.ksteps = pl.Vp * pl.eb / 128;
  pl.dh_per_group = choose_dh_split(cdiv(pl.c, kTile) * pl.td, pl.ksteps) > 1;
  int64_t dh_rows[2];  // the row counts dH runs on: full and last chunk or group
  if (pl.dh_per_group) {
    dh_rows[0] = std::min<int64_t>(pl.G * pl.c, pl.N);
    dh_rows[1] = pl.N - (pl.ngroups - 1) * pl.G * pl.c;
  } else {
    dh_rows[0] = pl.c;
    dh_rows[1] = pl.N - (pl.nchunks - 1) * pl.c;
  }
  size_t t = 0;
  auto take = [&](size_t bytes) {
    const size_t o = align256(t);
    t = o + bytes;
    return o;
  };
  pl.off_misc = take(256);
  pl.off_p = take((size_t)pl.ng * pl.K * 4);
  pl.off_tidx = take((size_t)pl.ng * pl.K * 4);
  pl.off_rows = take((size_t)7 * pl.ng * 4);
  pl.off_pm = take((size_t)pl.cp * pl.nVT * 4);
  pl.off_ps = take((size_t)pl.cp * pl.nVT * 4);
  pl.off_hits = take((size_t)pl.ng * pl.K * 4);
  pl.off_hitp = take((size_t)pl.ng * pl.K * 4);
  pl.off_hoff = take((size_t)(pl.ng / kTile) * (pl.nVT + 1) * 4);
  pl.off_zhit = take((size_t)pl.ng * pl.K * 4);
  pl.off_lossp = take((size_t)std::max<int64_t>(pl.nchunks, 1) * pl.nblk * 4);
  pl.off_dz = take((size_t)pl.G * pl.c * pl.Vp * pl.eb);
  // factor of each dZ row of the group in the single-projection schedule
  pl.off_fac = take((size_t)pl.G * pl.c * 4);
  // the hidden rows of one dW group, transposed (tokens padded to 64); until
  // the group's dW it holds the group's tokens that are not ignored, as rows
  pl.off_ht = take((size_t)pl.D * rup(pl.G * pl.c, 64) * pl.eb);
  // the token of each of those rows
  pl.off_rowmap = take((size_t)pl.G * pl.c * 4);
  {
    int64_t part = 0;
    for (int64_t r : dh_rows) {
      if (r <= 0) continue;
      const int sp = choose_dh_split(cdiv(r, kTile) * pl.td, pl.ksteps);
      if (sp > 1) part = std::max<int64_t>(part, sp * r);
    }
    pl.off_dhs = part > 0 ? take((size_t)part * pl.D * 4) : 0;
  }
  // partial tiles of the dW contraction's split last round (when its tiles
  // leave the last round of the compute units partly filled)
  {
    const int64_t tiles = cdiv(pl.D, kTile) * pl.nVT;
    pl.off_dwp = (tiles > kDwUnits && tiles % kDwUnits != 0)
                     ? take((size_t)kDwUnits * kTile * kTile * 4)
                     : 0;
  }
  pl.total = align256(t);
  return pl;
}

// The plan of make_plan, with fewer chunks per dW group if its workspace
// exceeds `cap` bytes (the same plan when it fits); false if the workspace of
// one chunk per group does not fit.
bool plan_within(const kd_problem* p, size_t cap, Plan* out) {
  Plan pl = make_plan(p);
  int64_t g = pl.G * pl.merged;  // the caller's chunks per dW group
  while (pl.total > cap && g > 1) pl = make_plan(p, --g);
  if (pl.total > cap) return false;
  *out = pl;
  return true;
}

inline bool aligned16(const void* q) { return ((uintptr_t)q & 15u) == 0; }

// KD_DEBUG_CHECK=1: every entry point validates the teacher indices first.
bool debug_index_check() {
  const char* e = getenv("KD_DEBUG_CHECK");
  return e != nullptr && e[0] == '1' && e[1] == '\0';
}

}  // namespace

extern "C" {

int kd_abi_version(void) { return KDTOPK_ABI_VERSION; }

const char* kd_status_string(int s) {
  switch (s) {
    case KD_OK: return "KD_OK: success";
    case KD_ERR_NULL_PTR: return "KD_ERR_NULL_PTR: a required pointer is NULL";
    case KD_ERR_BAD_SHAPE: return "KD_ERR_BAD_SHAPE: invalid N, D, V or K, or a size limit";
    case KD_ERR_BAD_ARG: return "KD_ERR_BAD_ARG: invalid chunk, temperature, flags or mode";
    case KD_ERR_UNSUPPORTED: return "KD_ERR_UNSUPPORTED: dtype, D % 64 != 0 or misaligned pointer";
    case KD_ERR_WORKSPACE_TOO_SMALL: return "KD_ERR_WORKSPACE_TOO_SMALL: workspace below the required size";
    case KD_ERR_BAD_INDEX: return "KD_ERR_BAD_INDEX: teacher index outside [0, V) or repeated in a row";
    case KD_ERR_DEVICE: return "KD_ERR_DEVICE: HIP launch or runtime error";
    default: return "unknown kd_status";
  }
}

kd_status kd_topk_kl_workspace_size(const kd_problem* p, size_t* bytes) {
  if (p == nullptr || bytes == nullptr) return KD_ERR_NULL_PTR;
  const kd_status st = check_problem(p);
  if (st != KD_OK) return st;
  *bytes = make_plan(p).total;
  return KD_OK;
}

}  // extern "C"

namespace {

// Arguments shared by the three entry points once they are validated.
struct Call {
  int mode;
  const void* hidden;
  const void* W;
  const int32_t* idx;
  const float* tlogit;
  const uint8_t* ignore;
  float* loss;              // forward modes
  float* lpt;
  float* logz_out;          // forward only
  const float* logz_in;     // backward only
  const float* gscale;
  const float* gtok;
  void* grad_hidden;        // backward modes
  float* grad_W;
  int accumulate;
  void* ws;
  size_t ws_bytes;
  void* stream;
};

// Common checks: problem, pointers every mode needs, alignment, workspace
// (unless the workspace is the library's own scratch).
kd_status validate(const kd_problem* p, const Call& c, const Plan& pl, bool own_ws = false) {
  if (!own_ws && c.ws == nullptr) return KD_ERR_NULL_PTR;
  if (p->N > 0 && (c.hidden == nullptr || c.W == nullptr || c.idx == nullptr ||
                   c.tlogit == nullptr))
    return KD_ERR_NULL_PTR;
  if (c.accumulate != 0 && c.accumulate != 1) return KD_ERR_BAD_ARG;
  if (!aligned16(c.hidden) || !aligned16(c.W) || !aligned16(c.grad_hidden) ||
      !aligned16(c.grad_W) || !aligned16(c.ws))
    return KD_ERR_UNSUPPORTED;
  if (!own_ws && c.ws_bytes < pl.total) return KD_ERR_WORKSPACE_TOO_SMALL;
  return KD_OK;
}

// Enqueues Algorithm 1 for one call: the host chunk schedule (§3.2.3).
kd_status enqueue(const kd_problem* p, const Plan& pl, const Call& c) {
  const bool fwd = c.mode != KD_MODE_BWD, bwd = c.mode != KD_MODE_FWD;
  char* ws = static_cast<char*>(c.ws);
  int* nvalid = reinterpret_cast<int*>(ws + pl.off_misc);
  float* inv_nvalid = reinterpret_cast<float*>(ws + pl.off_misc + 4);
  float* lossp = reinterpret_cast<float*>(ws + pl.off_lossp);
  const bool want_dh = bwd && c.grad_hidden != nullptr && pl.N > 0;
  const bool want_dw = bwd && c.grad_W != nullptr && pl.N > 0;

  KdPrepareArgs pa{};
  pa.dtype = p->dtype;
  pa.N = pl.N;
  pa.D = pl.D;
  pa.V = pl.V;
  pa.ignore = c.ignore;
  pa.nvalid = nvalid;
  pa.inv_nvalid = inv_nvalid;
  pa.zero_gW = (bwd && c.grad_W != nullptr && pl.N == 0 && !c.accumulate) ? c.grad_W : nullptr;
  if (kd_launch_prepare(&pa, c.stream) != 0) return KD_ERR_DEVICE;

  float* rows = reinterpret_cast<float*>(ws + pl.off_rows);
  float* fac = reinterpret_cast<float*>(ws + pl.off_fac);
  // the single-projection schedule stores dZ up to a factor per row, which
  // dH applies to its rows and dW to the hidden rows
  const bool scaled = fwd && bwd && (want_dh || want_dw);
  // With a mask, every entry point leaves the ignored tokens out (their loss
  // and gradient rows are 0): each dW group's other tokens are gathered
  // first, and the group's rows are those tokens in order, then rows without
  // a token, whose tiles the contractions skip (their count is on the
  // device).
  const bool compact = c.ignore != nullptr && pl.N > 0;
  int* rowmap = reinterpret_cast<int*>(ws + pl.off_rowmap);
  int* gnrow = reinterpret_cast<int*>(ws + pl.off_misc + 16);
  char* hcomp = ws + pl.off_ht;
  int64_t n_partials = 0;
  int64_t group_tokens = 0;
  bool dw_done = false;
  // the per-row arrays from row `o` of the prepared rows; `g` = the row of
  // the chunk within its dW group
  auto chunk_args = [&](int64_t row0, int rcount, int64_t o, int64_t g, int stages) {
    KdChunkArgs a{};
    a.dtype = p->dtype;
    a.mode = c.mode;
    a.stages = stages;
    a.one_projection = scaled ? 1 : 0;
    a.teacher_logprobs = (p->flags & KD_FLAG_TEACHER_LOGPROBS) ? 1 : 0;
    a.gscale = c.gscale;
    a.gtok = c.gtok;
    a.logz_in = c.logz_in;
    a.logz_out = c.logz_out ? (compact ? c.logz_out : c.logz_out + row0) : nullptr;
    a.D = pl.D;
    a.V = pl.V;
    a.K = (int)pl.K;
    a.row0 = row0;
    a.rows = rcount;
    a.inv_tau = 1.0f / p->temperature;
    a.W = c.W;
    a.Hc = compact ? hcomp + g * pl.D * pl.eb
                   : static_cast<const char*>(c.hidden) + row0 * pl.D * pl.eb;
    a.hidden = c.hidden;
    a.tidx_in = c.idx;
    a.tidx = reinterpret_cast<int32_t*>(ws + pl.off_tidx) + o * pl.K;
    a.tlogit = c.tlogit;
    a.ignore = c.ignore;
    a.inv_nvalid = inv_nvalid;
    a.rowmap = compact ? rowmap + g : nullptr;
    a.nrow = compact ? gnrow : nullptr;
    a.nrow_base = (int)g;
    a.p = reinterpret_cast<float*>(ws + pl.off_p) + o * pl.K;
    a.rowM = rows + o;
    a.rowH = rows + pl.ng + o;
    a.rowCoef = rows + 2 * pl.ng + o;
    a.rowCoefM = rows + 3 * pl.ng + o;
    a.rowL2 = rows + 4 * pl.ng + o;
    a.rowR = rows + 5 * pl.ng + o;
    a.rowFlag = reinterpret_cast<int*>(rows + 6 * pl.ng) + o;
    a.part_m = reinterpret_cast<float*>(ws + pl.off_pm);
    a.part_s = reinterpret_cast<float*>(ws + pl.off_ps);
    a.hits = reinterpret_cast<uint32_t*>(ws + pl.off_hits) + o * pl.K;
    a.hitp = reinterpret_cast<float*>(ws + pl.off_hitp) + o * pl.K;
    a.hoff = reinterpret_cast<int*>(ws + pl.off_hoff) + (o / kTile) * (pl.nVT + 1);
    a.zhit = reinterpret_cast<float*>(ws + pl.off_zhit) + o * pl.K;
    a.nVT = (int)pl.nVT;
    return a;
  };
  for (int64_t ci = 0; ci < pl.nchunks; ++ci) {
    const int64_t row0 = ci * pl.c;
    const int rcount = (int)std::min<int64_t>(pl.c, pl.N - row0);
    const int64_t slot = ci % pl.G;
    if (compact && slot == 0) {
      KdCompactArgs k{};
      k.dtype = p->dtype;
      k.D = pl.D;
      k.ignore = c.ignore;
      k.row0 = row0;
      k.rows = (int)std::min<int64_t>(pl.G * pl.c, pl.N - row0);
      k.hidden = c.hidden;
      k.hcomp = hcomp;
      k.rowmap = rowmap;
      k.nrow = gnrow;
      k.grad_hidden = want_dh ? c.grad_hidden : nullptr;
      k.gh_f32 = (p->flags & KD_FLAG_GRAD_HIDDEN_F32) ? 1 : 0;
      k.loss_per_token = c.lpt;
      k.logz_out = c.logz_out;
      if (kd_launch_compact(&k, c.stream) != 0) return KD_ERR_DEVICE;
    }
    if (pl.prep_per_group && slot == 0) {
      const int grows = (int)std::min<int64_t>(pl.G * pl.c, pl.N - row0);
      KdChunkArgs g = chunk_args(row0, grows, 0, 0, KD_STAGE_PREP);
      if (kd_launch_chunk(&g, c.stream) != 0) return KD_ERR_DEVICE;
    }
    KdChunkArgs a = chunk_args(row0, rcount, pl.prep_per_group ? slot * pl.c : 0, slot * pl.c,
                               pl.prep_per_group ? KD_STAGE_CHUNK
                                                 : (KD_STAGE_PREP | KD_STAGE_CHUNK));
    a.rowFactor = fac + slot * pl.c;
    a.dZ = (want_dh || want_dw) ? ws + pl.off_dz + slot * pl.c * pl.Vp * pl.eb : nullptr;
    a.ldz = pl.Vp;
    a.loss_per_token = c.lpt ? (compact ? c.lpt : c.lpt + row0) : nullptr;
    a.block_partial = lossp + n_partials;
    if (kd_launch_chunk(&a, c.stream) != 0) return KD_ERR_DEVICE;
    n_partials += cdiv(rcount, kLossRows);
    group_tokens += rcount;
    // dH over rows [r0, r0 + n) of the dZ buffer (from its row `zrow`)
    auto dh = [&](int64_t r0, int64_t n, int64_t zrow) -> bool {
      KdDhArgs h{};
      h.dtype = p->dtype;
      h.D = pl.D;
      h.V = pl.V;
      h.dZ = ws + pl.off_dz + zrow * pl.Vp * pl.eb;
      h.ldz = pl.Vp;
      h.W = c.W;
      h.tokens = n;
      h.split = choose_dh_split(cdiv(n, kTile) * pl.td, pl.ksteps);
      h.partial = h.split > 1 ? reinterpret_cast<float*>(ws + pl.off_dhs) : nullptr;
      h.gh_f32 = (p->flags & KD_FLAG_GRAD_HIDDEN_F32) ? 1 : 0;
      h.gH = compact ? c.grad_hidden
                     : static_cast<char*>(c.grad_hidden) + r0 * pl.D * (h.gh_f32 ? 4 : pl.eb);
      h.rowscale = scaled ? fac + zrow : nullptr;
      h.rowmap = compact ? rowmap + zrow : nullptr;
      h.nrow = compact ? gnrow : nullptr;
      h.nrow_base = (int)zrow;
      return kd_launch_dh(&h, c.stream) == 0;
    };
    if (want_dh && !pl.dh_per_group && !dh(row0, rcount, slot * pl.c)) return KD_ERR_DEVICE;
    if (!(want_dh || want_dw) || !(slot == pl.G - 1 || ci == pl.nchunks - 1)) continue;
    // the group's dH (when it runs per group) and dW over the G chunks' dZ rows
    const int64_t row_first = row0 + rcount - group_tokens;
    if (want_dh && pl.dh_per_group && !dh(row_first, group_tokens, 0)) return KD_ERR_DEVICE;
    if (want_dw) {
      KdDwArgs d{};
      d.dtype = p->dtype;
      d.D = pl.D;
      d.V = pl.V;
      d.dZ = ws + pl.off_dz;
      d.ldz = pl.Vp;
      d.Hg = compact ? c.hidden : static_cast<const char*>(c.hidden) + row_first * pl.D * pl.eb;
      d.tokens = group_tokens;
      d.Ht = ws + pl.off_ht;
      d.beta = (dw_done || c.accumulate) ? 1 : 0;
      d.gW = c.grad_W;
      d.rowscale = scaled ? fac : nullptr;
      d.partial = pl.off_dwp ? reinterpret_cast<float*>(ws + pl.off_dwp) : nullptr;
      d.rowmap = compact ? rowmap : nullptr;
      d.nrow = compact ? gnrow : nullptr;
      if (kd_launch_dw(&d, c.stream) != 0) return KD_ERR_DEVICE;
      dw_done = true;
    }
    group_tokens = 0;
  }
  if (fwd && kd_launch_finalize(lossp, (int)n_partials, inv_nvalid, c.loss, c.stream) != 0)
    return KD_ERR_DEVICE;
  return KD_OK;
}

}  // namespace

extern "C" {

kd_status kd_topk_kl_fwd_bwd(const kd_problem* p, const void* hidden, const void* W,
                             const int32_t* teacher_idx, const float* teacher_logit,
                             const uint8_t* ignore, float* loss, float* loss_per_token,
                             void* grad_hidden, float* grad_W, int accumulate_grad_W,
                             void* workspace, size_t workspace_bytes, void* hip_stream) {
  kd_status st = check_problem(p);
  if (st != KD_OK) return st;
  if (loss == nullptr) return KD_ERR_NULL_PTR;
  const Call c{KD_MODE_FWD_BWD, hidden, W, teacher_idx, teacher_logit, ignore, loss,
               loss_per_token, nullptr, nullptr, nullptr, nullptr, grad_hidden, grad_W,
               accumulate_grad_W, workspace, workspace_bytes, hip_stream};
  const Plan pl = make_plan(p);
  st = validate(p, c, pl);
  if (st != KD_OK) return st;
  if (debug_index_check() && p->N > 0) {
    st = kd_topk_kl_check_indices(p, teacher_idx, workspace, workspace_bytes, hip_stream);
    if (st != KD_OK) return st;
  }
  return enqueue(p, pl, c);
}

kd_status kd_topk_kl_fwd(const kd_problem* p, const void* hidden, const void* W,
                         const int32_t* teacher_idx, const float* teacher_logit,
                         const uint8_t* ignore, float* loss, float* loss_per_token,
                         float* saved_logz, void* workspace, size_t workspace_bytes,
                         void* hip_stream) {
  kd_status st = check_problem(p);
  if (st != KD_OK) return st;
  if (loss == nullptr || (p->N > 0 && saved_logz == nullptr)) return KD_ERR_NULL_PTR;
  const Call c{KD_MODE_FWD, hidden, W, teacher_idx, teacher_logit, ignore, loss,
               loss_per_token, saved_logz, nullptr, nullptr, nullptr, nullptr, nullptr, 0,
               workspace, workspace_bytes, hip_stream};
  const Plan pl = make_plan(p);
  st = validate(p, c, pl);
  if (st != KD_OK) return st;
  if (debug_index_check() && p->N > 0) {
    st = kd_topk_kl_check_indices(p, teacher_idx, workspace, workspace_bytes, hip_stream);
    if (st != KD_OK) return st;
  }
  return enqueue(p, pl, c);
}

kd_status kd_topk_kl_bwd(const kd_problem* p, const void* hidden, const void* W,
                         const int32_t* teacher_idx, const float* teacher_logit,
                         const uint8_t* ignore, const float* saved_logz,
                         const float* grad_loss, const float* grad_loss_per_token,
                         void* grad_hidden, float* grad_W, int accumulate_grad_W,
                         void* workspace, size_t workspace_bytes, void* hip_stream) {
  kd_status st = check_problem(p);
  if (st != KD_OK) return st;
  if (p->N > 0 && saved_logz == nullptr) return KD_ERR_NULL_PTR;
  const Call c{KD_MODE_BWD, hidden, W, teacher_idx, teacher_logit, ignore, nullptr, nullptr,
               nullptr, saved_logz, grad_loss, grad_loss_per_token, grad_hidden, grad_W,
               accumulate_grad_W, workspace, workspace_bytes, hip_stream};
  const Plan pl = make_plan(p);
  st = validate(p, c, pl);
  if (st != KD_OK) return st;
  if (debug_index_check() && p->N > 0) {
    st = kd_topk_kl_check_indices(p, teacher_idx, workspace, workspace_bytes, hip_stream);
    if (st != KD_OK) return st;
  }
  return enqueue(p, pl, c);
}

kd_status kd_topk_kl_check_indices(const kd_problem* p, const int32_t* teacher_idx,
                                   void* workspace, size_t workspace_bytes, void* hip_stream) {
  kd_status st = check_problem(p);
  if (st != KD_OK) return st;
  if (workspace == nullptr || (p->N > 0 && teacher_idx == nullptr)) return KD_ERR_NULL_PTR;
  if (!aligned16(workspace)) return KD_ERR_UNSUPPORTED;
  const Plan pl = make_plan(p);
  if (workspace_bytes < pl.total) return KD_ERR_WORKSPACE_TOO_SMALL;
  int* flag = reinterpret_cast<int*>(static_cast<char*>(workspace) + pl.off_misc + 8);
  int host_flag = 0;
  if (kd_launch_check_indices(teacher_idx, p->N, p->K, p->V, flag, &host_flag, hip_stream) != 0)
    return KD_ERR_DEVICE;
  return host_flag ? KD_ERR_BAD_INDEX : KD_OK;
}

// Checks one gradient of kd_scale_grads: in [n] fp32 -> out [n] dtype.
static kd_status scale_one(const float* g, const float* in, int32_t dtype, void* out, int64_t n,
                    void* stream) {
  if ((in == nullptr) != (out == nullptr)) return KD_ERR_NULL_PTR;
  if (n < 0) return KD_ERR_BAD_SHAPE;
  if (in == nullptr || n == 0) return KD_OK;
  if (dtype != KD_F32 && dtype != KD_BF16) return KD_ERR_UNSUPPORTED;
  if (!aligned16(in) || !aligned16(out)) return KD_ERR_UNSUPPORTED;
  // fp32 output: in place or disjoint; bf16 output: disjoint from the input
  const uintptr_t a0 = (uintptr_t)in, a1 = a0 + (uintptr_t)n * 4;
  const uintptr_t b0 = (uintptr_t)out, b1 = b0 + (uintptr_t)n * (dtype == KD_F32 ? 4 : 2);
  if (a0 < b1 && b0 < a1 && !(dtype == KD_F32 && a0 == b0)) return KD_ERR_BAD_ARG;
  return KD_OK;
}

kd_status kd_scale_grads(const float* grad_loss, const float* grad_hidden_f32,
                         int32_t hidden_dtype, void* grad_hidden_out, int64_t n_hidden,
                         const float* grad_W_f32, int32_t w_dtype, void* grad_W_out, int64_t n_W,
                         void* hip_stream) {
  if (grad_loss == nullptr) return KD_ERR_NULL_PTR;
  kd_status st = scale_one(grad_loss, grad_hidden_f32, hidden_dtype, grad_hidden_out, n_hidden,
                           hip_stream);
  if (st != KD_OK) return st;
  st = scale_one(grad_loss, grad_W_f32, w_dtype, grad_W_out, n_W, hip_stream);
  if (st != KD_OK) return st;
  if (grad_hidden_f32 != nullptr && n_hidden > 0 &&
      kd_launch_scale(hidden_dtype == KD_BF16, grad_hidden_f32, grad_hidden_out, n_hidden,
                      grad_loss, hip_stream) != 0)
    return KD_ERR_DEVICE;
  if (grad_W_f32 != nullptr && n_W > 0 &&
      kd_launch_scale(w_dtype == KD_BF16, grad_W_f32, grad_W_out, n_W, grad_loss, hip_stream) != 0)
    return KD_ERR_DEVICE;
  return KD_OK;
}

kd_status kd_topk_kl_fwd_bwd_noalloc(const kd_problem* p, const void* hidden, const void* W,
                                     const int32_t* teacher_idx, const float* teacher_logit,
                                     const uint8_t* ignore, float* loss, float* loss_per_token,
                                     void* grad_hidden, float* grad_W, int accumulate_grad_W,
                                     void* hip_stream) {
  kd_status st = check_problem(p);
  if (st != KD_OK) return st;
  if (loss == nullptr) return KD_ERR_NULL_PTR;
  Call c{KD_MODE_FWD_BWD, hidden, W, teacher_idx, teacher_logit, ignore, loss,
         loss_per_token, nullptr, nullptr, nullptr, nullptr, grad_hidden, grad_W,
         accumulate_grad_W, nullptr, 0, hip_stream};
  Plan pl;
  if (!plan_within(p, kd_scratch_bytes_max, &pl)) return KD_ERR_WORKSPACE_TOO_SMALL;
  st = validate(p, c, pl, true);
  if (st != KD_OK) return st;
  // the device's scratch array (its address is looked up once per device)
  void* ws = nullptr;
  if (kd_scratch_get(&ws) != 0 || ws == nullptr) return KD_ERR_DEVICE;
  c.ws = ws;
  c.ws_bytes = kd_scratch_bytes_max;
  if (debug_index_check() && p->N > 0) {
    int* flag = reinterpret_cast<int*>(static_cast<char*>(ws) + pl.off_misc + 8);
    int host_flag = 0;
    if (kd_launch_check_indices(teacher_idx, p->N, p->K, p->V, flag, &host_flag, hip_stream) != 0)
      return KD_ERR_DEVICE;
    if (host_flag) return KD_ERR_BAD_INDEX;
  }
  kd_launch_suppress_profiling(1);
  st = enqueue(p, pl, c);
  kd_launch_suppress_profiling(0);
  return st;
}

}  // extern "C"
