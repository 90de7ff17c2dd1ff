/*
 * kdtopk.h - C ABI of the fused, chunked top-K KL distillation loss for
 * AMD MI355X (gfx950).
 *
 * The operation is the "full chunked KL computation" of §3.2.3 and
 * Algorithm 1 of "Efficient Knowledge Distillation for LLMs: Offline Top-K
 * Logits and a Fused Chunked KL Loss": the student output projection
 * z = h W^T is fused into a forward KL against a cached top-K teacher, the
 * rows are processed in chunks of C_s tokens, and the [N, V] logit tensor is
 * never stored. Per token t (Eq. 1 and its decomposition Eq. 2 in §3.2):
 *
 *     l_t = sum_{k} p_tk log p_tk  -  sum_{k} p_tk y_t[idx_tk]  +  M_t log Z_t
 *
 * with y_t = z_t / tau, log Z_t = logsumexp_v y_tv, p_t = softmax over the K
 * cached entries of teacher_logit_t / tau and M_t = sum_k p_tk. The loss is the
 * mean of l_t over non-ignored tokens (§3, after Eq. 1). Gradients use the
 * closed form of Eq. (3) (§3.2.3): dL/dz_tv = g_t / tau (M_t q_tv - p_tv) with
 * q_t = softmax(y_t) and g_t = 1/N_valid for non-ignored tokens, 0 otherwise;
 * grad_hidden = G W and grad_W (+)= G^T h, as in Algorithm 1's backward.
 *
 * Conventions for every entry point:
 *   - All tensor pointers are DEVICE pointers, row-major, densely packed.
 *   - The caller allocates and owns every buffer, including the workspace.
 *     The library never allocates, frees, or keeps a pointer after return.
 *   - Work is enqueued asynchronously on `hip_stream` (a hipStream_t passed as
 *     void*, NULL = the default stream). kd_topk_kl_fwd_bwd never
 *     synchronises: read `loss` after synchronising the stream.
 *   - Every argument is checked on the host before anything is enqueued. On
 *     any error nothing is launched, no output is touched, and the function
 *     returns the error code.
 *   - Results are deterministic: identical inputs and chunk size give
 *     bitwise identical outputs (no floating-point atomics).
 *   - Calls are reentrant; concurrent calls need distinct workspaces.
 */
#ifndef KDTOPK_H
#define KDTOPK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KDTOPK_ABI_VERSION 3

typedef enum kd_status {
  KD_OK = 0,
  KD_ERR_NULL_PTR = 1,           /* a required pointer is NULL */
  KD_ERR_BAD_SHAPE = 2,          /* N < 0, D/V/K <= 0, K > V, K > 4096, or a size limit */
  KD_ERR_BAD_ARG = 3,            /* chunk <= 0, tau not finite or <= 0, flags */
  KD_ERR_UNSUPPORTED = 4,        /* dtype, D % 64 != 0, misaligned pointer */
  KD_ERR_WORKSPACE_TOO_SMALL = 5,
  KD_ERR_BAD_INDEX = 6,          /* a teacher index outside [0, V) or repeated */
  KD_ERR_DEVICE = 7              /* a HIP launch or runtime error */
} kd_status;

typedef enum kd_dtype {
  KD_F32 = 0,                    /* fp32 inputs, fp32 arithmetic throughout */
  KD_BF16 = 1                    /* bf16 inputs, bf16 MFMA, fp32 accumulate */
} kd_dtype;

/* Problem description (Algorithm 1's inputs: h, W, the support and C_s). */
typedef struct kd_problem {
  int64_t N;           /* tokens = rows of hidden; 0 <= N < 2^31            */
  int64_t D;           /* hidden size d; 64 <= D <= 65536, D % 64 == 0       */
  int64_t V;           /* vocabulary size; 1 <= V <= 1048576                 */
  int64_t chunk;       /* rows per chunk C_s; >= 1 (min(chunk, N) is used)   */
  int32_t K;           /* cached teacher entries per token; 1 <= K <= V, K <= 4096 */
  int32_t dtype;       /* kd_dtype of hidden, W and grad_hidden              */
  float temperature;   /* tau; finite and > 0                                */
  int32_t flags;       /* 0 or KD_FLAG_TEACHER_LOGPROBS | KD_FLAG_GRAD_HIDDEN_F32 */
} kd_problem;

/*
 * Teacher representation (§3.2). Default (flags = 0): teacher_logit holds
 * logits of the K cached entries; the teacher distribution is their softmax
 * over the K entries at temperature tau (retained mass M = 1).
 * KD_FLAG_TEACHER_LOGPROBS: teacher_logit holds the teacher's log-probabilities
 * over the full vocabulary at the K cached entries (the partial-mass cache of
 * §3.2): p = exp(value) as given, M = sum_k p <= 1, no renormalisation and no
 * temperature (tau still divides the student's logits). Values must be <= 0
 * and sum_k exp(value) <= 1; this is not checked.
 */
#define KD_FLAG_TEACHER_LOGPROBS 1

/*
 * KD_FLAG_GRAD_HIDDEN_F32: grad_hidden is written as fp32 whatever the
 * problem's dtype (kd_topk_kl_fwd_bwd and kd_topk_kl_bwd), so that a caller
 * who scales it later (kd_scale_grads) rounds to the hidden dtype only once.
 * The pointer's buffer is then [N, D] fp32.
 */
#define KD_FLAG_GRAD_HIDDEN_F32 2

/*
 * Bytes of device workspace kd_topk_kl_fwd_bwd, kd_topk_kl_fwd,
 * kd_topk_kl_bwd and kd_topk_kl_check_indices need for problem *p. Pure host
 * function: touches no device. The size is O(N/4 + G C_s (V + K + 1) + D G C_s),
 * with G C_s <= 16384 the tokens whose dZ rows one grad_W contraction
 * gathers (at most 4 GiB of them), plus 64 MiB when grad_W's tiles leave the
 * last round of the compute units partly filled: it grows with N only
 * through an array of loss partials (one per 4 tokens), never as N*V.
 * Errors: KD_ERR_NULL_PTR if p or bytes is NULL; the shape/argument errors of
 * kd_topk_kl_fwd_bwd otherwise.
 */
kd_status kd_topk_kl_workspace_size(const kd_problem* p, size_t* bytes);

/*
 * Fused chunked top-K KL forward + backward (§3.2.3, Algorithm 1, Eqs. 1-3).
 *
 *   hidden        [N, D] dtype        student hidden states h (row t = token t)
 *   W             [V, D] dtype        output projection
 *   teacher_idx   [N, K] int32        support S_t: K indices in [0, V) per
 *                                     row (not range-checked here unless
 *                                     KD_DEBUG_CHECK=1; see
 *                                     kd_topk_kl_check_indices). An index
 *                                     outside [0, V) is skipped; an index
 *                                     repeated in a row counts once with the
 *                                     sum of the repeated entries'
 *                                     probabilities (the dense teacher row
 *                                     of §3.2.1)
 *   teacher_logit [N, K] fp32         teacher logits of the support; the
 *                                     teacher distribution is their softmax
 *                                     over the K entries at temperature tau
 *                                     (log-probabilities with
 *                                     KD_FLAG_TEACHER_LOGPROBS)
 *   ignore        [N] uint8 or NULL   nonzero = token excluded from the loss
 *                                     and from the mean's count; NULL = none
 *   loss          [1] fp32            out: mean of l_t over non-ignored
 *                                     tokens (0 if there are none)
 *   loss_per_token [N] fp32 or NULL   out: l_t (0 on ignored tokens)
 *   grad_hidden   [N, D] dtype or NULL  out: dL/dh (fp32 with
 *                                     KD_FLAG_GRAD_HIDDEN_F32); NULL skips
 *                                     its GEMMs
 *   grad_W        [V, D] fp32 or NULL   out: dL/dW; NULL skips its GEMMs
 *   accumulate_grad_W  0: grad_W = dL/dW;  1: grad_W += dL/dW (micro-batch
 *                                     accumulation)
 *   workspace, workspace_bytes        device scratch of at least
 *                                     kd_topk_kl_workspace_size bytes,
 *                                     16-byte aligned
 *   hip_stream                        hipStream_t or NULL
 *
 * Schedule: with grad_hidden or grad_W requested, each chunk is projected
 * once. A chunk's log Z is complete once its own projection has run, and the
 * upstream gradient of the mean is known up front, so the projection that
 * yields the normaliser also yields the gradient, stored up to a factor per
 * token that the dH and dW contractions apply once log Z is merged, in place
 * of Algorithm 1's logit recompute (which the split entry points below
 * keep). The transient [chunk, V] buffer is the same one; nothing of size
 * N x V exists. The stream's device must be the current device.
 *
 * With an ignore mask, the ignored tokens take no part in the contractions
 * (with or without gradients requested, and likewise in kd_topk_kl_fwd and
 * kd_topk_kl_bwd): their loss terms and gradient rows
 * are 0 (Eq. 3 weights every row of G by its mask), so each group of up to
 * 16384 tokens is first compacted to its tokens that are not ignored, the
 * projection, dH and dW run over those only (the count stays on the device:
 * no host synchronisation), and the ignored tokens' loss_per_token entries
 * and grad_hidden rows are written as 0. The results are those of the
 * uncompacted computation up to the order of fp32 sums.
 *
 * Pointers hidden, W, grad_hidden, grad_W and workspace must be 16-byte
 * aligned (KD_ERR_UNSUPPORTED otherwise). hidden, W, teacher_idx,
 * teacher_logit and loss are required (KD_ERR_NULL_PTR); with N == 0 only
 * loss (and grad_W when given) are written. Launch failures return
 * KD_ERR_DEVICE; work enqueued before the failure may have run.
 */
kd_status kd_topk_kl_fwd_bwd(const kd_problem* p,
                             const void* hidden,
                             const void* W,
                             const int32_t* teacher_idx,
                             const float* teacher_logit,
                             const uint8_t* ignore,
                             float* loss,
                             float* loss_per_token,
                             void* grad_hidden,
                             float* grad_W,
                             int accumulate_grad_W,
                             void* workspace,
                             size_t workspace_bytes,
                             void* hip_stream);

/*
 * Forward only: the loss of Algorithm 1's two forward passes (normaliser, then
 * the loss; §3.2.3), without any gradient work, plus the per-token
 * log-normaliser the backward needs.
 *
 *   hidden, W, teacher_idx, teacher_logit, ignore   as for kd_topk_kl_fwd_bwd
 *   loss          [1] fp32            out: mean of l_t over non-ignored tokens
 *   loss_per_token [N] fp32 or NULL   out: l_t (0 on ignored tokens)
 *   saved_logz    [N] fp32            out: log Z_t = logsumexp_v z_tv / tau
 *                                     (0 on ignored tokens, which are left
 *                                     out as in kd_topk_kl_fwd_bwd)
 *   workspace, workspace_bytes, hip_stream   as for kd_topk_kl_fwd_bwd
 *
 * One projection per chunk (the normaliser and the student logits at the
 * teacher entries come from the same tile). Values are bitwise identical to
 * the corresponding outputs of kd_topk_kl_fwd_bwd called without gradients.
 * Errors as for kd_topk_kl_fwd_bwd; saved_logz is required.
 */
kd_status kd_topk_kl_fwd(const kd_problem* p,
                         const void* hidden,
                         const void* W,
                         const int32_t* teacher_idx,
                         const float* teacher_logit,
                         const uint8_t* ignore,
                         float* loss,
                         float* loss_per_token,
                         float* saved_logz,
                         void* workspace,
                         size_t workspace_bytes,
                         void* hip_stream);

/*
 * Backward only (Algorithm 1's backward: per chunk the logits are recomputed,
 * q_t = exp(z_t / tau - log Z_t) with log Z_t from the forward, Eq. 3, then
 * grad_hidden = G W and grad_W (+)= G^T h).
 *
 *   hidden, W, teacher_idx, teacher_logit, ignore   as for the forward call
 *   saved_logz    [N] fp32            log Z_t written by kd_topk_kl_fwd (read
 *                                     for the tokens not ignored)
 *   grad_loss     [1] fp32 or NULL    upstream gradient of the mean loss
 *                                     (device scalar); NULL = 1
 *   grad_loss_per_token [N] fp32 or NULL   upstream gradients u_t of the
 *                                     per-token losses; when given, G uses
 *                                     g_t = u_t (ignored tokens 0) instead of
 *                                     grad_loss / N_valid
 *   grad_hidden   [N, D] dtype (fp32 with KD_FLAG_GRAD_HIDDEN_F32) or NULL,
 *   grad_W        [V, D] fp32 or NULL,
 *   accumulate_grad_W                 as for kd_topk_kl_fwd_bwd
 *
 * With grad_loss = NULL and no per-token gradients the results equal
 * kd_topk_kl_fwd_bwd's gradients up to the rounding of log Z through fp32.
 * Errors as for kd_topk_kl_fwd_bwd; saved_logz is required.
 */
kd_status kd_topk_kl_bwd(const kd_problem* p,
                         const void* hidden,
                         const void* W,
                         const int32_t* teacher_idx,
                         const float* teacher_logit,
                         const uint8_t* ignore,
                         const float* saved_logz,
                         const float* grad_loss,
                         const float* grad_loss_per_token,
                         void* grad_hidden,
                         float* grad_W,
                         int accumulate_grad_W,
                         void* workspace,
                         size_t workspace_bytes,
                         void* hip_stream);

/*
 * Checks that every teacher index lies in [0, V) and that no row repeats an
 * index (the support S_t of §3.2 is a set; the loss accepts repeats and sums
 * them, but a top-K cache never repeats an index, so a repeat points at a
 * broken cache). Synchronises `hip_stream`.
 * Returns KD_OK, KD_ERR_BAD_INDEX, or an argument/device error. Uses the
 * first bytes of `workspace` (same size rule as kd_topk_kl_fwd_bwd).
 *
 * Debug mode: with the environment variable KD_DEBUG_CHECK set to 1 when a
 * call is made, kd_topk_kl_fwd_bwd, kd_topk_kl_fwd and kd_topk_kl_bwd run
 * this check first (synchronising their stream, so the call is no longer
 * asynchronous) and return KD_ERR_BAD_INDEX with nothing else enqueued and no
 * output touched when it fails. Without it, indices are not checked.
 */
kd_status kd_topk_kl_check_indices(const kd_problem* p,
                                   const int32_t* teacher_idx,
                                   void* workspace,
                                   size_t workspace_bytes,
                                   void* hip_stream);

/*
 * kd_topk_kl_fwd_bwd for callers that cannot allocate device memory (code
 * being captured into a HIP graph, tight serving loops, harnesses that forbid
 * allocation): the same arguments without the workspace. The workspace is a
 * static per-device array of KD_SCRATCH_BYTES inside the library, which each
 * device the library runs on holds from the first use of the library on that
 * device until the process ends; the call itself allocates nothing (no
 * hipMalloc, no events, no allocating library routine) and only enqueues
 * kernels on hip_stream. The caller still provides every output.
 *
 * The plan is kd_topk_kl_fwd_bwd's when its workspace fits the array: results
 * are then bitwise identical to kd_topk_kl_fwd_bwd's. Otherwise fewer chunks'
 * dZ rows are gathered per grad_W contraction (grad_W differs only in the fp32
 * summation order); if one chunk's workspace does not fit (about
 * chunk * V * (element size) bytes plus small terms), the call returns
 * KD_ERR_WORKSPACE_TOO_SMALL before touching the device: use a smaller chunk.
 *
 * Every call on a device shares that device's array, and calls keep no state
 * in it (nothing in it has to start at zero; each call writes what it reads).
 * Calls that overlap in time on one device (two streams, two threads) race on
 * the array and give wrong results: order them on one stream. With
 * KD_DEBUG_CHECK=1 the index check synchronises the stream, as for the other
 * entry points. Errors as for kd_topk_kl_fwd_bwd, plus KD_ERR_WORKSPACE_TOO_SMALL
 * as above and KD_ERR_DEVICE if the array's address cannot be obtained.
 */
#define KD_SCRATCH_BYTES (256u << 20)

kd_status kd_topk_kl_fwd_bwd_noalloc(const kd_problem* p,
                                     const void* hidden,
                                     const void* W,
                                     const int32_t* teacher_idx,
                                     const float* teacher_logit,
                                     const uint8_t* ignore,
                                     float* loss,
                                     float* loss_per_token,
                                     void* grad_hidden,
                                     float* grad_W,
                                     int accumulate_grad_W,
                                     void* hip_stream);

/*
 * Scales the gradients of the mean loss by the upstream gradient g of that
 * mean, a device fp32 scalar: Algorithm 1's backward forms G = (M g) q - p g
 * (§3.2.3); the loss is linear in g, so the gradients kd_topk_kl_fwd_bwd
 * computed with g = 1 become those for any g by one multiplication. For a
 * caller (an autograd function) that runs the fused call in its forward,
 * before g is known: with KD_FLAG_GRAD_HIDDEN_F32 both gradients come out of
 * the fused call in fp32, and each is rounded once, here, to its dtype.
 *
 *   grad_loss        [1] fp32                g (device)
 *   grad_hidden_f32  [n_hidden] fp32 or NULL  input: dL/dh of the mean
 *   grad_hidden_out  [n_hidden] hidden_dtype or NULL   out: g * input
 *   grad_W_f32       [n_W] fp32 or NULL       input: dL/dW of the mean
 *   grad_W_out       [n_W] w_dtype or NULL    out: g * input
 *   hip_stream                                hipStream_t or NULL
 *
 * Each output is rounded once to its dtype (KD_F32 or KD_BF16). An fp32
 * output may be its input itself (in place); otherwise output and input must
 * not overlap. A NULL pair (or a zero count) skips that gradient.
 * Asynchronous on hip_stream. Errors, all detected before any launch:
 * KD_ERR_NULL_PTR (grad_loss NULL, or one of a pair NULL), KD_ERR_BAD_SHAPE
 * (a negative count), KD_ERR_UNSUPPORTED (an output dtype other than KD_F32
 * or KD_BF16, or a pointer not 16-byte aligned), KD_ERR_BAD_ARG (an output
 * overlapping its input other than in place); KD_ERR_DEVICE (launch).
 */
kd_status kd_scale_grads(const float* grad_loss,
                         const float* grad_hidden_f32,
                         int32_t hidden_dtype,
                         void* grad_hidden_out,
                         int64_t n_hidden,
                         const float* grad_W_f32,
                         int32_t w_dtype,
                         void* grad_W_out,
                         int64_t n_W,
                         void* hip_stream);

/*
 * Instrumentation, not part of the method: per-kernel timing with HIP events.
 * kd_profile_enable(mode), process-wide: 0 off; 1 the entry points record a
 * HIP event pair on their stream around each kernel launch; 2 only around the
 * contraction kernels (the projection, dH and dW launches, whose `flops` is
 * nonzero), which keeps the events' own cost out of the rest of the step.
 * Another mode gives KD_ERR_BAD_ARG. kd_profile_read waits for the recorded
 * events, writes up to `max` entries (one per kernel kind that ran), clears the
 * records and returns the number of entries written (negative on a HIP error).
 * `flops` is the algorithmic floating-point work of the recorded launches (the
 * 2*rows*D*V contractions of each chunk; 0 for the other kernels).
 * Creating events is an allocation: leave profiling off where that matters.
 */
typedef struct kd_kernel_time {
  char name[32];       /* kernel kind, e.g. "logits_lse", "dz", "dh", "dw" */
  int64_t launches;
  double total_ms;     /* sum of event-measured durations */
  double flops;        /* sum of algorithmic FLOP over the launches */
} kd_kernel_time;

kd_status kd_profile_enable(int mode);
int kd_profile_read(kd_kernel_time* out, int max);

/* Static, NUL-terminated description of a status code (never NULL). */
const char* kd_status_string(int status);

/* KDTOPK_ABI_VERSION of the loaded library. */
int kd_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KDTOPK_H */
