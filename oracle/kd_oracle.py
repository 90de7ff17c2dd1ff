"""fp64 CPU oracle for the fused chunked top-K KL distillation loss.

TEST INFRASTRUCTURE, NOT PRODUCT CODE. Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import or call anything in this package. The
HIP library and its Python binding never import, call or link it, and it shares
no code, constants or helpers with them.

Paper: "Efficient Knowledge Distillation for LLMs: Offline Top-K Logits and a
Fused Chunked KL Loss". What this module computes, and from which passage:

* The teacher distribution over the cached top-K support (§3.2). The inputs are
  teacher logits; the support probabilities are their softmax over the K entries
  at temperature tau (a reading: §3.2 caches probabilities with retained mass
  M <= 1; with logits renormalised over K, M = 1 up to rounding).
* The per-token forward KL of Eq. (1) in §3, evaluated densely: the top-K
  probabilities are scattered (summed) into a dense vocabulary row and compared
  against the student's dense log-softmax, as in the full dense evaluation of
  §3.2.1, which the paper names its correctness baseline. The GPU path instead
  evaluates the decomposition of Eq. (2); agreement therefore also checks the
  Eq. (1) = Eq. (2) identity.
* The mean over loss-masked (non-ignored) positions (§3, after Eq. 1); or, for
  the backward of Algorithm 1 driven by an upstream gradient, any per-token
  weights g_t of the token losses.
* The partial-mass teacher of §3.2: cached top-K probabilities with retained
  mass M = sum_k p_k <= 1, supplied as log-probabilities and used as they are
  (no renormalisation, no temperature).
* Gradients from the closed form of Eq. (3) in §3.2.3, dL/dz_v = M q_v - p_v,
  taken through the temperature (the 1/tau chain factor) and the mean weight
  g_t = 1/N_valid, then projected back as in Algorithm 1's backward:
  dh = G W and dW = G^T h.

Readings where the paper is silent (all only τ=1 is used in the paper):
  * temperature: q = softmax_V(z/tau), p = softmax_K(teacher_logit/tau), no tau^2
    factor, exact derivative including 1/tau;
  * 0 * log 0 = 0;
  * N_valid = 0 gives loss 0 and zero gradients;
  * duplicate indices in a row are summed (scatter-add, §3.2.2).

Everything is plain NumPy in float64; the dense [chunk, V] logits are
materialised one row chunk at a time, chunking exactly as Algorithm 1 does.
"""
from __future__ import annotations

import numpy as np


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def log_softmax_rows(y):
    """Row-wise log-softmax with the usual max shift (textbook definition)."""
    m = y.max(axis=1, keepdims=True)
    return y - (m + np.log(np.exp(y - m).sum(axis=1, keepdims=True)))


def teacher_distribution(teacher_logit, tau, mode="logits"):
    """Support probabilities p[N, K] of the offline top-K teacher (§3.2).

    mode "logits": softmax over the K cached entries of teacher_logit / tau
    (retained mass 1). mode "logprobs": the cached values are the teacher's
    log-probabilities over the full vocabulary, p = exp(value), retained mass
    M = sum_k p_k <= 1 (the partial-mass teacher)."""
    if mode == "logits":
        return np.exp(log_softmax_rows(_f64(teacher_logit) / float(tau)))
    if mode == "logprobs":
        return np.exp(_f64(teacher_logit))
    raise ValueError("mode must be 'logits' or 'logprobs'")


def kd_topk_kl(h, W, teacher_idx, teacher_logit, tau=1.0, ignore=None,
               chunk=None, mean_denominator=None, want_grads=True,
               token_weights=None, teacher_mode="logits"):
    """Loss, per-token loss, log-normaliser and gradients of the top-K forward KL.

    h [N, D], W [V, D] (any real dtype; computed in float64),
    teacher_idx [N, K] ints in [0, V), teacher_logit [N, K], ignore [N] (nonzero =
    excluded) or None, chunk = rows per chunk (None = all rows at once),
    mean_denominator = divisor of the mean (None = number of non-ignored rows;
    a caller checking a subset of a bigger batch passes the batch's count),
    token_weights [N] = weight g_t of each token's loss in the differentiated
    objective sum_t g_t l_t (None = the mean's 1/N_valid; ignored rows always 0),
    teacher_mode = "logits" or "logprobs" (see teacher_distribution).

    Returns a dict with: loss (float, the mean), loss_per_token [N] (0 on ignored
    rows), logZ [N] (log-normaliser of z/tau), M [N], and when want_grads the
    gradients of the objective: grad_hidden [N, D], grad_W [V, D].
    """
    h = _f64(h)
    W = _f64(W)
    idx = np.asarray(teacher_idx, dtype=np.int64)
    N, D = h.shape
    V = W.shape[0]
    if W.shape[1] != D:
        raise ValueError("W must be [V, D]")
    K = idx.shape[1]
    tau = float(tau)
    valid = np.ones(N, dtype=bool) if ignore is None else (np.asarray(ignore) == 0)
    n_valid = float(valid.sum()) if mean_denominator is None else float(mean_denominator)
    c = N if chunk is None else int(chunk)
    if c <= 0:
        raise ValueError("chunk must be positive")

    p = teacher_distribution(teacher_logit, tau, teacher_mode) if K > 0 else np.zeros((N, 0))
    M = p.sum(axis=1)
    # weight of each token in the objective: the mean's 1/N_valid over the
    # loss-masked positions (§3), or the caller's upstream per-token weights
    if token_weights is None:
        g = np.where(valid, 1.0 / n_valid, 0.0) if n_valid > 0 else np.zeros(N)
    else:
        g = np.where(valid, _f64(token_weights), 0.0)

    loss_tok = np.zeros(N)
    logZ = np.zeros(N)
    grad_h = np.zeros((N, D)) if want_grads else None
    grad_W = np.zeros((V, D)) if want_grads else None

    for s0 in range(0, N, c):                       # Algorithm 1: row chunks
        s1 = min(N, s0 + c)
        rows = np.arange(s1 - s0)
        z = h[s0:s1] @ W.T                          # transient logit chunk
        y = z / tau
        logq = log_softmax_rows(y)
        logZ[s0:s1] = y[:, 0] - logq[:, 0] if V > 0 else 0.0
        # dense teacher row: scatter-add of the K support probabilities
        P = np.zeros((s1 - s0, V))
        np.add.at(P, (np.repeat(rows, K), idx[s0:s1].reshape(-1)),
                  p[s0:s1].reshape(-1))
        # Eq. (1): sum_v P_v (log P_v - log q_v), with 0 log 0 = 0
        pos = P > 0
        term = np.zeros_like(P)
        term[pos] = P[pos] * (np.log(P[pos]) - logq[pos])
        ell = term.sum(axis=1)
        ell[~valid[s0:s1]] = 0.0
        loss_tok[s0:s1] = ell
        if want_grads:
            # Eq. (3): dL/dz = M q - P (support part scattered), times 1/tau
            # from z/tau and g_t from the mean.
            q = np.exp(logq)
            G = (g[s0:s1] / tau)[:, None] * (M[s0:s1, None] * q - P)
            grad_h[s0:s1] = G @ W                   # dh = G W
            grad_W += G.T @ h[s0:s1]                # dW += G^T h

    loss = float(loss_tok.sum() / n_valid) if n_valid > 0 else 0.0
    out = dict(loss=loss, loss_per_token=loss_tok, logZ=logZ, M=M)
    if want_grads:
        out["grad_hidden"] = grad_h
        out["grad_W"] = grad_W
    return out
