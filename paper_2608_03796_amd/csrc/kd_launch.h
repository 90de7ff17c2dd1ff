// Internal interface between the host scheduler (kd_api.cpp, plain C++) and
// the HIP launchers (kd_kernels.hip). No HIP types: streams travel as void*.
#pragma once

#include <stddef.h>
#include <stdint.h>

struct KdPrepareArgs {
  int dtype;                // 0 fp32, 1 bf16
  int64_t N, D, V;
  const uint8_t* ignore;    // [N] or null
  int* nvalid;              // device int
  float* inv_nvalid;        // device float: 1/N_valid or 0
  float* zero_gW;           // grad_W to clear, or null
};

enum { KD_MODE_FWD_BWD = 0, KD_MODE_FWD = 1, KD_MODE_BWD = 2 };

// bytes of the allocation-free entry point's static per-device scratch
constexpr size_t kd_scratch_bytes_max = (size_t)256 << 20;

// tokens per loss partial (one block of the row-loss kernels, a wave per token)
constexpr int kLossRows = 4;

// Stages of kd_launch_chunk: preparing rows (teacher prologue, bucketing,
// and in the one-projection schedule the reference logits) and the chunk's
// projection and what follows it. The host prepares the rows of a whole dW
// group at once when chunks align with 256-token tiles, else each chunk.
enum { KD_STAGE_PREP = 1, KD_STAGE_CHUNK = 2 };

struct KdChunkArgs {
  int dtype;
  int mode;                 // KD_MODE_*: which half of Algorithm 1 runs
  int stages;               // KD_STAGE_* bits
  int one_projection;       // loss and gradients together (k_logits_dz schedule)
  int teacher_logprobs;     // cached log-probabilities (partial mass) instead of logits
  const float* gscale;      // upstream gradient of the mean (device scalar) or null = 1
  const float* gtok;        // full [N] upstream per-token gradients or null
  const float* logz_in;     // full [N] saved log Z (backward only) or null
  float* logz_out;          // this chunk's rows of the saved log Z (forward; full [N]
                            // with a rowmap) or null
  int64_t D, V;
  int K;
  int64_t row0;             // first token of the chunk (of the prepared rows)
  int rows;                 // tokens in the chunk (prepared rows)
  float inv_tau;
  const void* W;            // [V, D]
  const void* Hc;           // hidden + row0 * D (the projection's token rows)
  const void* hidden;       // full [N, D] (the reference logits read rows by token)
  const int32_t* tidx_in;   // full [N, K] (the caller's)
  int32_t* tidx;            // [rows, K] the prologue's copy (repeats -1), read by the rest
  const float* tlogit;      // full [N, K] (prologue indexes with row0)
  const uint8_t* ignore;    // full [N] or null
  const float* inv_nvalid;
  // ignored tokens left out (one-projection schedule): row r of the prepared
  // rows is token rowmap[r] (-1: no token; such rows come after every token),
  // and *nrow - nrow_base of the rows hold tokens. Null: row r is token row0 + r.
  const int* rowmap;
  const int* nrow;
  int nrow_base;
  // per-chunk workspace
  float* p;                 // [rows, K]
  float *rowM, *rowH, *rowCoef, *rowCoefM, *rowL2;   // [rows]
  float* rowR;              // [rows] reference logit of the single projection
  int* rowFlag;             // [rows] a tile fell back to its own max
  float* rowFactor;         // [rows] factor of the row's stored gradient (this
                            // chunk's rows of the group's factor array)
  float *part_m, *part_s;                            // [rows, nVT]
  int nVT;
  uint32_t* hits;           // [cdiv(rows, 256) * 256 * K] teacher entries by vocab tile
  float* hitp;              // their p
  int* hoff;                // [cdiv(rows, 256), nVT + 1] bucket offsets
  float* zhit;              // [rows, K] student logit at each teacher entry
  void* dZ;                 // this chunk's rows of the group's dZ [rows, ldz]
  int64_t ldz;              // = padded vocabulary (columns V..ldz: finite, z = 0 there)
  // outputs
  float* loss_per_token;    // + row0 (full [N] with a rowmap), or null
  float* block_partial;     // this chunk's cdiv(rows, kLossRows) partial sums
};

// dH GEMM over the chunks of one group: grad_hidden[rows] = dZ[rows] W
struct KdDhArgs {
  int dtype;
  int64_t D, V;
  const void* dZ;           // the group's dZ rows [tokens, ldz]
  int64_t ldz;
  const void* W;            // [V, D]
  int64_t tokens;           // tokens in the group
  int split;                // split of the vocabulary (K) range, >= 1
  float* partial;           // [split, tokens, D] when split > 1
  void* gH;                 // grad_hidden + the group's first row * D (full with a rowmap)
  int gh_f32;               // grad_hidden is fp32 (else the operands' dtype)
  const float* rowscale;    // [tokens] factor of each dZ row, or null (= 1)
  const int* rowmap;        // [tokens] grad_hidden row of each dZ row (-1: none), or null
  const int* nrow;          // with rowmap: *nrow - nrow_base dZ rows hold tokens
  int nrow_base;
};

// dW tiles per full round (the compute units) and the largest split of the
// tail tiles' token range; the partial tiles' workspace holds
// kDwUnits * 256 * 256 floats (64 MiB)
constexpr int kDwUnits = 256;
constexpr int kDwMaxSplit = 4;

// dW GEMM over the chunks of one group: grad_W (+)= dZ[:tokens]^T H[:tokens]
struct KdDwArgs {
  int dtype;
  int64_t D, V;
  const void* dZ;           // the group's dZ rows [tokens, ldz]
  int64_t ldz;
  const void* Hg;           // the group's hidden rows [tokens, D] (full with a rowmap)
  int64_t tokens;           // tokens in the group
  void* Ht;                 // workspace for Hg transposed: [D, tokens rounded up to 64]
  int beta;                 // 0 overwrite, 1 accumulate
  float* gW;
  const float* rowscale;    // [tokens] factor of each dZ row (applied to the
                            // hidden rows), or null (= 1)
  float* partial;           // workspace of the split tail tiles, or null (no split)
  const int* rowmap;        // [tokens] hidden row of each dZ row (-1: none), or null
  const int* nrow;          // with rowmap: the dZ rows [0, *nrow) hold tokens
};

// Ignored tokens of one dW group [row0, row0 + rows) left out: rowmap[j] =
// the j-th token not ignored (then -1), *nrow = their count, their hidden
// rows copied to hcomp [rows, D]; the ignored tokens' grad_hidden rows,
// per-token losses and saved log Z set to 0.
struct KdCompactArgs {
  int dtype;
  int64_t D;
  const uint8_t* ignore;    // full [N]
  int64_t row0;
  int rows;
  const void* hidden;       // full [N, D]
  void* hcomp;
  int* rowmap;
  int* nrow;
  void* grad_hidden;        // full [N, D] or null
  int gh_f32;
  float* loss_per_token;    // full [N] or null
  float* logz_out;          // full [N] or null
};

extern "C" {
int kd_launch_prepare(const KdPrepareArgs* a, void* stream);
int kd_launch_chunk(const KdChunkArgs* a, void* stream);
int kd_launch_dh(const KdDhArgs* a, void* stream);
int kd_launch_dw(const KdDwArgs* a, void* stream);
int kd_launch_compact(const KdCompactArgs* a, void* stream);
int kd_launch_finalize(const float* partials, int n, const float* inv_nvalid, float* loss,
                       void* stream);
int kd_launch_scale(int out_bf16, const float* x, void* y, int64_t n, const float* g,
                    void* stream);
// the current device's scratch address (hipGetSymbolAddress on first use)
int kd_scratch_get(void** ptr);
// nonzero: the calling thread's launches record no profiling events
void kd_launch_suppress_profiling(int on);
int kd_launch_check_indices(const int32_t* idx, int64_t N, int K, int64_t V, int* flag,
                            int* host_flag, void* stream);
}
