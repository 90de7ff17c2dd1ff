"""The Python binding rejects inputs whose shapes, dtypes, devices or layouts
disagree before anything reaches the library (which takes plain pointers and
would index past a short buffer)."""
import pytest
import torch

import kd_inputs as ki

pytestmark = pytest.mark.gpu


def _inputs(N=64, D=64, V=300, K=5):
    dev = "cuda"
    hidden = ki.make_hidden(N, D, torch.float32, dev, seed=1)
    W = ki.make_weight(V, D, torch.float32, dev, seed=2)
    idx, logit = ki.make_teacher(N, K, V, dev, seed=3)
    return hidden, W, idx, logit


def test_mismatched_shapes_raise(gpu_lib):
    kd = gpu_lib
    h, W, idx, tl = _inputs()
    with pytest.raises(ValueError):
        kd.fwd_bwd(h, W, idx, tl[:-1].contiguous())          # fewer teacher rows
    with pytest.raises(ValueError):
        kd.fwd_bwd(h, W[:, :32].contiguous(), idx, tl)        # W's D differs
    with pytest.raises(ValueError):
        kd.fwd_bwd(h, W, idx[:, :4].contiguous(), tl)         # K differs
    with pytest.raises(ValueError):
        kd.fwd_bwd(h, W, idx, tl, ignore=torch.zeros(63, dtype=torch.uint8, device="cuda"))
    with pytest.raises(ValueError):
        kd.fwd_bwd(h[:, None, :], W, idx, tl)                 # not [N, D]


def test_bad_outputs_and_workspace_raise(gpu_lib):
    kd = gpu_lib
    h, W, idx, tl = _inputs()
    with pytest.raises(ValueError):
        kd.fwd_bwd(h, W, idx, tl, grad_W_out=torch.zeros(300, 32, device="cuda"))
    with pytest.raises(ValueError):
        kd.fwd_bwd(h, W, idx, tl, out={"grad_hidden": torch.empty(64, 64, dtype=torch.bfloat16,
                                                                   device="cuda")})
    ws = kd.alloc_workspace(64, 64, 300, 5, 4096, 1.0, kd.KD_F32, "cuda")
    with pytest.raises(ValueError):
        kd.fwd_bwd(h, W, idx, tl, workspace=ws.view(torch.int32))
    f = kd.fwd(h, W, idx, tl)
    with pytest.raises(ValueError):
        kd.bwd(h, W, idx, tl, f["saved_logz"][:-1].contiguous())
    with pytest.raises(ValueError):
        kd.bwd(h, W, idx, tl, f["saved_logz"], grad_loss=torch.ones(2, device="cuda"))
    with pytest.raises(ValueError):
        kd.bwd(h, W, idx, tl, f["saved_logz"], grad_loss_per_token=torch.ones(63, device="cuda"))
    # the well-formed calls still run
    out = kd.fwd_bwd(h, W, idx, tl, workspace=ws)
    torch.cuda.synchronize()
    assert torch.isfinite(out["loss"])
