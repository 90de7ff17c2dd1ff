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
