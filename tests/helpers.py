"""Shared test utilities: read device tensors back exactly and compare with the
oracle. bf16 -> fp32 -> fp64 is exact, so the oracle sees the same inputs."""
import numpy as np
import torch

# Tolerances (bf16 inputs with fp32 accumulation / fp32 throughout)
TOL = {
    "bf16": dict(loss=2e-3, grad=1e-2),
    "f32": dict(loss=1e-5, grad=1e-5),
}


def to64(t):
    if t is None:
        return None
    if t.dtype in (torch.bfloat16, torch.float16):
        t = t.float()
    return t.detach().cpu().numpy().astype(np.float64) if t.is_floating_point() else t.detach().cpu().numpy()


def rel_max(a, ref):
    """max|a - ref| / max|ref| (0 if both are all zero)."""
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.abs(ref).max() if ref.size else 0.0
    num = np.abs(a - ref).max() if ref.size else 0.0
    if den == 0.0:
        return num
    return num / den


def oracle_inputs(inp):
    return dict(h=to64(inp["hidden"]), W=to64(inp["W"]), teacher_idx=to64(inp["teacher_idx"]),
                teacher_logit=to64(inp["teacher_logit"]), ignore=to64(inp.get("ignore")))


def oracle_by_row_blocks(kd_topk_kl, h, W, teacher_idx, teacher_logit, tau, ignore=None,
                         block=2048, chunk=128, workers=None):
    """The oracle over all N rows, evaluated as independent row blocks on a
    thread pool (NumPy's ufuncs and BLAS release the GIL) with the batch's
    N_valid as every block's mean divisor: rows are independent given N_valid,
    so per-token losses and grad_hidden rows are the blocks' own, and grad_W is
    the sum of the blocks' grad_W (dW = sum_t G_t^T h_t). BLAS runs one thread
    per block to avoid oversubscription."""
    import os
    from concurrent.futures import ThreadPoolExecutor
    from threadpoolctl import threadpool_limits
    N = h.shape[0]
    valid = np.ones(N, dtype=bool) if ignore is None else (np.asarray(ignore) == 0)
    n_valid = int(valid.sum())
    if workers is None:
        workers = max(1, min(16, len(os.sched_getaffinity(0))))
    starts = list(range(0, N, block))

    def one(s0):
        s1 = min(N, s0 + block)
        return kd_topk_kl(h[s0:s1], W, teacher_idx[s0:s1], teacher_logit[s0:s1], tau=tau,
                          ignore=None if ignore is None else ignore[s0:s1],
                          mean_denominator=n_valid, chunk=chunk)

    with threadpool_limits(limits=1), ThreadPoolExecutor(max_workers=workers) as ex:
        parts = list(ex.map(one, starts))
    grad_W = parts[0]["grad_W"].copy()
    for p in parts[1:]:
        grad_W += p["grad_W"]
    lpt = np.concatenate([p["loss_per_token"] for p in parts])
    return dict(loss=float(lpt.sum() / n_valid) if n_valid else 0.0, loss_per_token=lpt,
                grad_hidden=np.concatenate([p["grad_hidden"] for p in parts]), grad_W=grad_W,
                logZ=np.concatenate([p["logZ"] for p in parts]))
