"""Fused chunked top-K KL distillation loss on AMD MI355X (gfx950).

Python binding of libkdtopk.so (C ABI in include/kdtopk.h). The binding only
marshals arguments: PyTorch provides device memory and the current stream;
every step of the loss runs in the library's HIP kernels. There is no CPU or
PyTorch fallback: if the library is missing, the calls raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkdtopk.so")

KD_F32 = 0
KD_BF16 = 1
KD_FLAG_TEACHER_LOGPROBS = 1
KD_FLAG_GRAD_HIDDEN_F32 = 2

STATUS = {
    0: "KD_OK", 1: "KD_ERR_NULL_PTR", 2: "KD_ERR_BAD_SHAPE", 3: "KD_ERR_BAD_ARG",
    4: "KD_ERR_UNSUPPORTED", 5: "KD_ERR_WORKSPACE_TOO_SMALL", 6: "KD_ERR_BAD_INDEX",
    7: "KD_ERR_DEVICE",
}
EXPORTED = ("kd_topk_kl_workspace_size", "kd_topk_kl_fwd_bwd", "kd_topk_kl_fwd_bwd_noalloc",
            "kd_topk_kl_fwd",
            "kd_topk_kl_bwd", "kd_topk_kl_check_indices", "kd_scale_grads", "kd_status_string",
            "kd_abi_version", "kd_profile_enable", "kd_profile_read")


class KdError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {STATUS.get(code, code)}")


class KdProblem(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int64), ("D", ctypes.c_int64), ("V", ctypes.c_int64),
                ("chunk", ctypes.c_int64), ("K", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("temperature", ctypes.c_float), ("flags", ctypes.c_int32)]


class KdKernelTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double), ("flops", ctypes.c_double)]


_lib = None


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Loads libkdtopk.so (built by paper_2608_03796_amd.build). Raises if absent."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is not built; run `python -m paper_2608_03796_amd.build`")
    lib = ctypes.CDLL(p)
    vp, i64, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t
    lib.kd_topk_kl_workspace_size.argtypes = [ctypes.POINTER(KdProblem), ctypes.POINTER(sz)]
    lib.kd_topk_kl_workspace_size.restype = ctypes.c_int
    lib.kd_topk_kl_fwd_bwd.argtypes = [ctypes.POINTER(KdProblem), vp, vp, vp, vp, vp, vp, vp, vp,
                                       vp, ctypes.c_int, vp, sz, vp]
    lib.kd_topk_kl_fwd_bwd.restype = ctypes.c_int
    lib.kd_topk_kl_fwd_bwd_noalloc.argtypes = [ctypes.POINTER(KdProblem), vp, vp, vp, vp, vp,
                                               vp, vp, vp, vp, ctypes.c_int, vp]
    lib.kd_topk_kl_fwd_bwd_noalloc.restype = ctypes.c_int
    lib.kd_topk_kl_fwd.argtypes = [ctypes.POINTER(KdProblem), vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                   sz, vp]
    lib.kd_topk_kl_fwd.restype = ctypes.c_int
    lib.kd_topk_kl_bwd.argtypes = [ctypes.POINTER(KdProblem), vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                   vp, ctypes.c_int, vp, sz, vp]
    lib.kd_topk_kl_bwd.restype = ctypes.c_int
    lib.kd_topk_kl_check_indices.argtypes = [ctypes.POINTER(KdProblem), vp, vp, sz, vp]
    lib.kd_topk_kl_check_indices.restype = ctypes.c_int
    lib.kd_scale_grads.argtypes = [vp, vp, ctypes.c_int32, vp, i64, vp, ctypes.c_int32, vp, i64,
                                   vp]
    lib.kd_scale_grads.restype = ctypes.c_int
    lib.kd_status_string.argtypes = [ctypes.c_int]
    lib.kd_status_string.restype = ctypes.c_char_p
    lib.kd_abi_version.argtypes = []
    lib.kd_abi_version.restype = ctypes.c_int
    lib.kd_profile_enable.argtypes = [ctypes.c_int]
    lib.kd_profile_enable.restype = ctypes.c_int
    lib.kd_profile_read.argtypes = [ctypes.POINTER(KdKernelTime), ctypes.c_int]
    lib.kd_profile_read.restype = ctypes.c_int
    if path is None:
        _lib = lib
    return lib


def problem(N, D, V, K, chunk, tau, dtype, flags=0) -> KdProblem:
    return KdProblem(int(N), int(D), int(V), int(chunk), int(K), int(dtype), float(tau), int(flags))


def _flags(teacher_logprobs=False, grad_hidden_f32=False) -> int:
    return (KD_FLAG_TEACHER_LOGPROBS if teacher_logprobs else 0) | \
        (KD_FLAG_GRAD_HIDDEN_F32 if grad_hidden_f32 else 0)


def _dtype_code(t) -> int:
    import torch
    if t == torch.bfloat16:
        return KD_BF16
    if t == torch.float32:
        return KD_F32
    raise TypeError(f"unsupported dtype {t}")


def workspace_size(N, D, V, K, chunk, tau=1.0, dtype=KD_BF16) -> int:
    lib = load_library()
    pr = problem(N, D, V, K, chunk, tau, dtype)
    out = ctypes.c_size_t(0)
    rc = lib.kd_topk_kl_workspace_size(ctypes.byref(pr), ctypes.byref(out))
    if rc != 0:
        raise KdError(rc, "kd_topk_kl_workspace_size")
    return int(out.value)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream_handle(device):
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def alloc_workspace(N, D, V, K, chunk, tau, dtype, device):
    import torch
    n = workspace_size(N, D, V, K, chunk, tau, dtype)
    return torch.empty(n, dtype=torch.uint8, device=device)


def _check_inputs(hidden, W, teacher_idx, teacher_logit, ignore):
    """Dtypes, shapes, devices and layouts of the inputs. The library takes
    plain pointers, so every size it will index with is checked here."""
    import torch
    if hidden.device.type != "cuda":
        raise ValueError("tensors must be on a GPU")
    if hidden.dim() != 2 or W.dim() != 2:
        raise ValueError("hidden must be [N, D] and W [V, D]")
    if W.dtype != hidden.dtype:
        raise TypeError("hidden and W must share a dtype")
    for name, t, want in (("teacher_idx", teacher_idx, torch.int32),
                          ("teacher_logit", teacher_logit, torch.float32)):
        if t.dtype != want:
            raise TypeError(f"{name} must be {want}")
    if ignore is not None and ignore.dtype != torch.uint8:
        raise TypeError("ignore must be uint8")
    N, D = hidden.shape
    if W.shape[1] != D:
        raise ValueError(f"W is {tuple(W.shape)}, expected [V, {D}]")
    if teacher_idx.dim() != 2 or teacher_idx.shape[0] != N:
        raise ValueError(f"teacher_idx is {tuple(teacher_idx.shape)}, expected [{N}, K]")
    K = teacher_idx.shape[1]
    if tuple(teacher_logit.shape) != (N, K):
        raise ValueError(f"teacher_logit is {tuple(teacher_logit.shape)}, expected [{N}, {K}]")
    if ignore is not None and tuple(ignore.shape) != (N,):
        raise ValueError(f"ignore is {tuple(ignore.shape)}, expected [{N}]")
    tensors = [hidden, W, teacher_idx, teacher_logit] + ([ignore] if ignore is not None else [])
    for t in tensors:
        if not t.is_contiguous():
            raise ValueError("inputs must be contiguous")
        if t.device != hidden.device:
            raise ValueError("inputs must be on one device")
    return N, D, W.shape[0], K, _dtype_code(hidden.dtype)


def _check_tensor(name, t, shape, dtype, device):
    """A caller-provided output or extra input: exact shape, dtype, device, layout."""
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype or t.device != device \
            or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {dtype} tensor of shape {tuple(shape)} "
                         f"on {device} (got {t.dtype} {tuple(t.shape)} on {t.device})")


def _check_workspace(workspace, device):
    import torch
    if workspace.dtype != torch.uint8 or workspace.device != device \
            or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 tensor on the inputs' device")


def fwd_bwd(hidden, W, teacher_idx, teacher_logit, tau: float = 1.0, ignore=None,
            chunk: int = 4096, grad_hidden: bool = True, grad_W: bool = True,
            loss_per_token: bool = False, grad_W_out=None, accumulate_grad_W: bool = False,
            workspace=None, out=None, teacher_logprobs: bool = False,
            grad_hidden_f32: bool = False):
    """One call of kd_topk_kl_fwd_bwd on the current stream.

    hidden [N, D] and W [V, D] (bf16 or fp32, same dtype), teacher_idx [N, K]
    int32, teacher_logit [N, K] fp32 (log-probabilities of a partial-mass
    teacher when teacher_logprobs), ignore [N] uint8 or None. Returns a dict
    with 'loss' (0-d fp32 tensor), and 'loss_per_token', 'grad_hidden',
    'grad_W' when requested. grad_hidden is in hidden's dtype, or fp32 with
    grad_hidden_f32. `out` may carry preallocated output tensors (keys as
    returned) to make repeated calls allocation-free.
    """
    import torch
    lib = load_library()
    N, D, V, K, dt = _check_inputs(hidden, W, teacher_idx, teacher_logit, ignore)
    out = dict(out or {})
    dev = hidden.device
    if "loss" not in out:
        out["loss"] = torch.empty((), dtype=torch.float32, device=dev)
    if loss_per_token and "loss_per_token" not in out:
        out["loss_per_token"] = torch.empty(N, dtype=torch.float32, device=dev)
    gh_dtype = torch.float32 if grad_hidden_f32 else hidden.dtype
    if grad_hidden and "grad_hidden" not in out:
        out["grad_hidden"] = torch.empty(N, D, dtype=gh_dtype, device=dev)
    if grad_W:
        if grad_W_out is not None:
            out["grad_W"] = grad_W_out
        elif "grad_W" not in out:
            out["grad_W"] = torch.empty(V, D, dtype=torch.float32, device=dev)
    _check_tensor("loss", out["loss"], (), torch.float32, dev)
    if loss_per_token:
        _check_tensor("loss_per_token", out["loss_per_token"], (N,), torch.float32, dev)
    if grad_hidden:
        _check_tensor("grad_hidden", out["grad_hidden"], (N, D), gh_dtype, dev)
    if grad_W:
        _check_tensor("grad_W", out["grad_W"], (V, D), torch.float32, dev)
    pr = problem(N, D, V, K, chunk, tau, dt, _flags(teacher_logprobs, grad_hidden_f32))
    if workspace is None:
        workspace = alloc_workspace(N, D, V, K, chunk, tau, dt, dev)
    _check_workspace(workspace, dev)
    with torch.cuda.device(dev):
        rc = lib.kd_topk_kl_fwd_bwd(
            ctypes.byref(pr), _ptr(hidden), _ptr(W), _ptr(teacher_idx), _ptr(teacher_logit),
            _ptr(ignore), _ptr(out["loss"]), _ptr(out.get("loss_per_token") if loss_per_token else None),
            _ptr(out.get("grad_hidden") if grad_hidden else None),
            _ptr(out.get("grad_W") if grad_W else None), int(bool(accumulate_grad_W)),
            _ptr(workspace), ctypes.c_size_t(workspace.numel()), _stream_handle(dev))
    if rc != 0:
        raise KdError(rc, "kd_topk_kl_fwd_bwd")
    res = {"loss": out["loss"]}
    if loss_per_token:
        res["loss_per_token"] = out["loss_per_token"]
    if grad_hidden:
        res["grad_hidden"] = out["grad_hidden"]
    if grad_W:
        res["grad_W"] = out["grad_W"]
    return res


def fwd_bwd_noalloc(hidden, W, teacher_idx, teacher_logit, tau: float = 1.0, ignore=None,
                    chunk: int = 4096, out=None, grad_hidden: bool = True, grad_W: bool = True,
                    loss_per_token: bool = False, accumulate_grad_W: bool = False,
                    teacher_logprobs: bool = False):
    """kd_topk_kl_fwd_bwd_noalloc: kd_topk_kl_fwd_bwd with the library's own
    static per-device scratch as workspace. Pass every wanted output in `out`
    ('loss' 0-d fp32, 'loss_per_token' [N] fp32, 'grad_hidden' [N, D] in
    hidden's dtype, 'grad_W' [V, D] fp32) to make the call allocation-free;
    missing ones are allocated here. Returns the outputs as fwd_bwd does."""
    import torch
    lib = load_library()
    N, D, V, K, dt = _check_inputs(hidden, W, teacher_idx, teacher_logit, ignore)
    dev = hidden.device
    out = dict(out or {})
    want = {"loss": ((), torch.float32, True),
            "loss_per_token": ((N,), torch.float32, loss_per_token),
            "grad_hidden": ((N, D), hidden.dtype, grad_hidden),
            "grad_W": ((V, D), torch.float32, grad_W)}
    for k, (shape, dtype, on) in want.items():
        if not on:
            continue
        if k not in out:
            out[k] = torch.empty(shape, dtype=dtype, device=dev)
        _check_tensor(k, out[k], shape, dtype, dev)
    pr = problem(N, D, V, K, chunk, tau, dt, _flags(teacher_logprobs))
    with torch.cuda.device(dev):
        rc = lib.kd_topk_kl_fwd_bwd_noalloc(
            ctypes.byref(pr), _ptr(hidden), _ptr(W), _ptr(teacher_idx), _ptr(teacher_logit),
            _ptr(ignore), _ptr(out["loss"]),
            _ptr(out["loss_per_token"] if loss_per_token else None),
            _ptr(out["grad_hidden"] if grad_hidden else None),
            _ptr(out["grad_W"] if grad_W else None), int(bool(accumulate_grad_W)),
            _stream_handle(dev))
    if rc != 0:
        raise KdError(rc, "kd_topk_kl_fwd_bwd_noalloc")
    return {k: out[k] for k, (_, _, on) in want.items() if on}


def fwd(hidden, W, teacher_idx, teacher_logit, tau: float = 1.0, ignore=None,
        chunk: int = 4096, loss_per_token: bool = False, workspace=None,
        teacher_logprobs: bool = False):
    """kd_topk_kl_fwd: the loss without gradient work, plus the per-token
    log-normaliser log Z the backward needs. Returns a dict with 'loss' (0-d),
    'saved_logz' [N] and, when requested, 'loss_per_token' [N]."""
    import torch
    lib = load_library()
    N, D, V, K, dt = _check_inputs(hidden, W, teacher_idx, teacher_logit, ignore)
    dev = hidden.device
    res = {"loss": torch.empty((), dtype=torch.float32, device=dev),
           "saved_logz": torch.empty(N, dtype=torch.float32, device=dev)}
    if loss_per_token:
        res["loss_per_token"] = torch.empty(N, dtype=torch.float32, device=dev)
    pr = problem(N, D, V, K, chunk, tau, dt, _flags(teacher_logprobs))
    if workspace is None:
        workspace = alloc_workspace(N, D, V, K, chunk, tau, dt, dev)
    _check_workspace(workspace, dev)
    with torch.cuda.device(dev):
        rc = lib.kd_topk_kl_fwd(
            ctypes.byref(pr), _ptr(hidden), _ptr(W), _ptr(teacher_idx), _ptr(teacher_logit),
            _ptr(ignore), _ptr(res["loss"]), _ptr(res.get("loss_per_token")), _ptr(res["saved_logz"]),
            _ptr(workspace), ctypes.c_size_t(workspace.numel()), _stream_handle(dev))
    if rc != 0:
        raise KdError(rc, "kd_topk_kl_fwd")
    return res


def bwd(hidden, W, teacher_idx, teacher_logit, saved_logz, tau: float = 1.0, ignore=None,
        chunk: int = 4096, grad_loss=None, grad_loss_per_token=None, grad_hidden: bool = True,
        grad_W: bool = True, grad_W_out=None, accumulate_grad_W: bool = False, workspace=None,
        teacher_logprobs: bool = False, grad_hidden_f32: bool = False):
    """kd_topk_kl_bwd: gradients from the saved log-normaliser. grad_loss is the
    upstream gradient of the mean loss (0-d fp32 device tensor, None = 1);
    grad_loss_per_token [N] fp32 replaces it with per-token upstream gradients.
    Returns a dict with 'grad_hidden' (hidden's dtype, or fp32 with
    grad_hidden_f32) and 'grad_W' as requested."""
    import torch
    lib = load_library()
    N, D, V, K, dt = _check_inputs(hidden, W, teacher_idx, teacher_logit, ignore)
    dev = hidden.device
    _check_tensor("saved_logz", saved_logz, (N,), torch.float32, dev)
    if grad_loss is not None and grad_loss.numel() == 1:
        _check_tensor("grad_loss", grad_loss, tuple(grad_loss.shape), torch.float32, dev)
    elif grad_loss is not None:
        raise ValueError("grad_loss must hold one value (the upstream gradient of the mean)")
    if grad_loss_per_token is not None:
        _check_tensor("grad_loss_per_token", grad_loss_per_token, (N,), torch.float32, dev)
    res = {}
    if grad_hidden:
        res["grad_hidden"] = torch.empty(N, D, device=dev,
                                         dtype=torch.float32 if grad_hidden_f32 else hidden.dtype)
    if grad_W:
        res["grad_W"] = grad_W_out if grad_W_out is not None else torch.empty(
            V, D, dtype=torch.float32, device=dev)
        _check_tensor("grad_W", res["grad_W"], (V, D), torch.float32, dev)
    pr = problem(N, D, V, K, chunk, tau, dt, _flags(teacher_logprobs, grad_hidden_f32))
    if workspace is None:
        workspace = alloc_workspace(N, D, V, K, chunk, tau, dt, dev)
    _check_workspace(workspace, dev)
    with torch.cuda.device(dev):
        rc = lib.kd_topk_kl_bwd(
            ctypes.byref(pr), _ptr(hidden), _ptr(W), _ptr(teacher_idx), _ptr(teacher_logit),
            _ptr(ignore), _ptr(saved_logz), _ptr(grad_loss), _ptr(grad_loss_per_token),
            _ptr(res.get("grad_hidden")), _ptr(res.get("grad_W")), int(bool(accumulate_grad_W)),
            _ptr(workspace), ctypes.c_size_t(workspace.numel()), _stream_handle(dev))
    if rc != 0:
        raise KdError(rc, "kd_topk_kl_bwd")
    return res


def scale_grads(grad_loss, grad_hidden=None, grad_hidden_out=None, grad_W=None,
                grad_W_out=None):
    """kd_scale_grads on the current stream: out = grad_loss * in for the fp32
    gradients grad_hidden and grad_W of the mean loss, each written to its
    output (fp32 or bf16; an fp32 output may be its input). grad_loss is the
    upstream gradient of the mean, a one-element fp32 device tensor."""
    import torch
    lib = load_library()
    pairs = (("grad_hidden", grad_hidden, grad_hidden_out), ("grad_W", grad_W, grad_W_out))
    dev = None
    for name, x, y in pairs:
        if (x is None) != (y is None):
            raise ValueError(f"{name} and its output go together")
        if x is not None:
            dev = x.device if dev is None else dev
            _check_tensor(name, x, tuple(x.shape), torch.float32, dev)
            _check_tensor(name + "_out", y, tuple(x.shape), y.dtype, dev)
    if dev is None:
        return
    if grad_loss.numel() != 1:
        raise ValueError("grad_loss must hold one value")
    _check_tensor("grad_loss", grad_loss, tuple(grad_loss.shape), torch.float32, dev)

    def code(y):
        return _dtype_code(y.dtype) if y is not None else KD_F32

    with torch.cuda.device(dev):
        rc = lib.kd_scale_grads(
            _ptr(grad_loss), _ptr(grad_hidden), code(grad_hidden_out), _ptr(grad_hidden_out),
            grad_hidden.numel() if grad_hidden is not None else 0,
            _ptr(grad_W), code(grad_W_out), _ptr(grad_W_out),
            grad_W.numel() if grad_W is not None else 0, _stream_handle(dev))
    if rc != 0:
        raise KdError(rc, "kd_scale_grads")


def _autograd_functions():
    import torch

    class TopKKLLoss(torch.autograd.Function):
        """Mean top-K KL loss as an autograd function, Algorithm 1's schedule:
        forward runs kd_topk_kl_fwd and saves log Z; backward runs
        kd_topk_kl_bwd with the upstream gradient (logit recompute). grad_W is
        returned in W's dtype (fp32 accumulation inside one call; use
        bwd(..., accumulate_grad_W=True) to accumulate micro-batches in fp32)."""

        @staticmethod
        def forward(ctx, hidden, W, teacher_idx, teacher_logit, tau, ignore, chunk,
                    teacher_logprobs, workspace):
            res = fwd(hidden, W, teacher_idx, teacher_logit, tau=tau, ignore=ignore, chunk=chunk,
                      teacher_logprobs=teacher_logprobs, workspace=workspace)
            ctx.save_for_backward(hidden, W, teacher_idx, teacher_logit, res["saved_logz"],
                                  *([ignore] if ignore is not None else []))
            ctx.cfg = (tau, chunk, teacher_logprobs, ignore is not None)
            ctx.workspace = workspace
            return res["loss"]

        @staticmethod
        def backward(ctx, grad_out):
            tau, chunk, logprobs, has_ignore = ctx.cfg
            saved = ctx.saved_tensors
            hidden, W, idx, tl, logz = saved[:5]
            ignore = saved[5] if has_ignore else None
            g = grad_out.detach().to(torch.float32).contiguous()
            need_h, need_W = ctx.needs_input_grad[0], ctx.needs_input_grad[1]
            res = bwd(hidden, W, idx, tl, logz, tau=tau, ignore=ignore, chunk=chunk, grad_loss=g,
                      grad_hidden=need_h, grad_W=need_W, teacher_logprobs=logprobs,
                      workspace=ctx.workspace)
            gW = res.get("grad_W")
            if gW is not None and gW.dtype != W.dtype:
                gW = gW.to(W.dtype)
            return res.get("grad_hidden"), gW, None, None, None, None, None, None, None

    class TopKKLLossFused(torch.autograd.Function):
        """Mean top-K KL loss as an autograd function, one projection per chunk:
        when a gradient is wanted, forward runs kd_topk_kl_fwd_bwd and keeps the
        gradients of the mean (both in fp32); backward has kd_scale_grads
        multiply them by the upstream gradient (exact: the loss is linear in
        it) and round them once to the inputs' dtypes. The gradients are held
        from forward to backward; backward runs once per graph."""

        @staticmethod
        def forward(ctx, hidden, W, teacher_idx, teacher_logit, tau, ignore, chunk,
                    teacher_logprobs, workspace):
            need_h, need_W = ctx.needs_input_grad[0], ctx.needs_input_grad[1]
            ctx.grads = None
            if not (need_h or need_W):
                # the loss alone (no log Z to save): the fused call without
                # gradients, which leaves ignored tokens out
                return fwd_bwd(hidden, W, teacher_idx, teacher_logit, tau=tau, ignore=ignore,
                               chunk=chunk, grad_hidden=False, grad_W=False,
                               teacher_logprobs=teacher_logprobs, workspace=workspace)["loss"]
            out = fwd_bwd(hidden, W, teacher_idx, teacher_logit, tau=tau, ignore=ignore,
                          chunk=chunk, grad_hidden=need_h, grad_W=need_W,
                          teacher_logprobs=teacher_logprobs, workspace=workspace,
                          grad_hidden_f32=True)
            ctx.grads = [out.get("grad_hidden"), out.get("grad_W")]
            ctx.dtypes = (hidden.dtype, W.dtype)
            return out["loss"]

        @staticmethod
        def backward(ctx, grad_out):
            if ctx.grads is None:
                raise RuntimeError("topk_kl_loss(schedule='fused') supports one backward per "
                                   "graph; use schedule='recompute' to run backward again")
            gh, gW = ctx.grads
            ctx.grads = None
            h_dtype, w_dtype = ctx.dtypes
            g = grad_out.detach().to(torch.float32).contiguous()
            # both gradients are fp32 here: scaled by g in the library and
            # rounded once to the inputs' dtypes (in place when fp32)
            gh_out = None
            if gh is not None:
                gh_out = gh if h_dtype == torch.float32 else torch.empty_like(gh, dtype=h_dtype)
            gW_out = None
            if gW is not None:
                gW_out = gW if w_dtype == torch.float32 else torch.empty_like(gW, dtype=w_dtype)
            scale_grads(g, grad_hidden=gh, grad_hidden_out=gh_out, grad_W=gW, grad_W_out=gW_out)
            return gh_out, gW_out, None, None, None, None, None, None, None

    return {"recompute": TopKKLLoss, "fused": TopKKLLossFused}


_TOPK_KL = None


def topk_kl_loss(hidden, W, teacher_idx, teacher_logit, tau: float = 1.0, ignore=None,
                 chunk: int = 4096, teacher_logprobs: bool = False, schedule: str = "fused",
                 workspace=None):
    """Differentiable mean top-K KL loss.

    schedule="fused": when hidden or W needs a gradient, the forward computes
    the loss and the gradients of the mean in one kd_topk_kl_fwd_bwd call (one
    projection per chunk) and the backward scales them by the upstream
    gradient in the library (kd_scale_grads), rounding each once to its
    input's dtype; backward runs once per graph. Cost when no backward
    follows (a loss only logged with grad mode on): the forward still does
    all the gradient work (about 3x the forward-only time) and holds the fp32
    gradients ([N, D] and [V, D]: 2.5 GiB at N = 32768, D = 4096,
    V = 131072) until the graph is freed; they are kept on the autograd
    context, so saved-tensor hooks (offloading) do not see them. Compute such
    a loss under torch.no_grad() (the loss alone, through kd_topk_kl_fwd_bwd
    without gradients), or use schedule="recompute", whose forward is
    kd_topk_kl_fwd alone and which saves only log Z.
    schedule="recompute": Algorithm 1's schedule through the split entry
    points (forward saves log Z; backward recomputes the logits).
    workspace: a uint8 device tensor of at least workspace_size(...) bytes to
    reuse across calls (allocated per call when None)."""
    import torch
    global _TOPK_KL
    if schedule not in ("fused", "recompute"):
        raise ValueError("schedule must be 'fused' or 'recompute'")
    if not torch.is_grad_enabled():
        # no graph will be built: the loss alone (no gradient work; ignored
        # tokens left out)
        return fwd_bwd(hidden, W, teacher_idx, teacher_logit, tau=tau, ignore=ignore,
                       chunk=chunk, grad_hidden=False, grad_W=False,
                       teacher_logprobs=teacher_logprobs, workspace=workspace)["loss"]
    if _TOPK_KL is None:
        _TOPK_KL = _autograd_functions()
    return _TOPK_KL[schedule].apply(hidden, W, teacher_idx, teacher_logit, float(tau), ignore,
                                    int(chunk), bool(teacher_logprobs), workspace)


def check_indices(teacher_idx, V, chunk=4096, D=64, tau=1.0, dtype=KD_BF16, workspace=None):
    """True if every index is in [0, V) and no row repeats one (synchronises)."""
    import torch
    lib = load_library()
    if teacher_idx.device.type != "cuda" or teacher_idx.dtype != torch.int32 \
            or teacher_idx.dim() != 2 or not teacher_idx.is_contiguous():
        raise ValueError("teacher_idx must be a contiguous [N, K] int32 GPU tensor")
    N, K = teacher_idx.shape
    pr = problem(N, D, V, K, chunk, tau, dtype)
    if workspace is None:
        workspace = alloc_workspace(N, D, V, K, chunk, tau, dtype, teacher_idx.device)
    _check_workspace(workspace, teacher_idx.device)
    with torch.cuda.device(teacher_idx.device):
        rc = lib.kd_topk_kl_check_indices(ctypes.byref(pr), _ptr(teacher_idx), _ptr(workspace),
                                          ctypes.c_size_t(workspace.numel()),
                                          _stream_handle(teacher_idx.device))
    if rc == 6:
        return False
    if rc != 0:
        raise KdError(rc, "kd_topk_kl_check_indices")
    return True


def profile_enable(on: bool = True, contractions_only: bool = False):
    """Per-kernel HIP-event timing inside the library (instrumentation): off,
    around every kernel, or only around the contraction kernels."""
    rc = load_library().kd_profile_enable(0 if not on else (2 if contractions_only else 1))
    if rc != 0:
        raise KdError(rc, "kd_profile_enable")


def profile_read() -> dict:
    """{kernel kind: {launches, total_ms, flops}} recorded since the last read."""
    arr = (KdKernelTime * 32)()
    n = load_library().kd_profile_read(arr, 32)
    if n < 0:
        raise KdError(7, "kd_profile_read")
    return {arr[i].name.decode(): dict(launches=int(arr[i].launches),
                                       total_ms=float(arr[i].total_ms),
                                       flops=float(arr[i].flops)) for i in range(n)}
