"""The allocation-free entry point (kd_topk_kl_fwd_bwd_noalloc) against
kd_topk_kl_fwd_bwd, through the C ABI, on consecutive calls that share the
library's static scratch, each smaller than the one before:

  1. bf16, N=2048, D=64, V=131072, chunk 512: kd_topk_kl_fwd_bwd's plan
     (4 chunks per grad_W contraction, 512 MiB of dZ) does not fit the
     256 MiB scratch, so one chunk per contraction is used: loss and per-token
     losses are bitwise equal (the projections are the same), the gradients
     equal within the fp32 summation order (bf16 bound of the contract);
  2. bf16, N=1000, D=256, V=50000, chunk 256, tau 1.5, 10% ignored: the plan
     fits, so every output is bitwise equal;
  3. fp32, N=300, D=128, V=4133, K=7, chunk 100, tau 2, 20% ignored: bitwise.

The stale contents each call leaves in the scratch must not leak into the next.
Then the use it exists for: the call captured into a HIP graph and replayed.
"""
import pytest
import torch

import kd_inputs as ki
from tests.helpers import TOL, rel_max, to64

pytestmark = pytest.mark.gpu

CASES = [
    # N, D, V, K, chunk, tau, ignored, dtype, plan unchanged
    (2048, 64, 131072, 100, 512, 1.0, 0.0, torch.bfloat16, False),
    (1000, 256, 50000, 32, 256, 1.5, 0.1, torch.bfloat16, True),
    (300, 128, 4133, 7, 100, 2.0, 0.2, torch.float32, True),
]


def _inputs(N, D, V, K, dtype, ign, seed):
    dev = "cuda"
    hidden = ki.make_hidden(N, D, dtype, dev, seed=ki.SEED_HIDDEN + seed)
    W = ki.make_weight(V, D, dtype, dev, seed=ki.SEED_W + seed)
    idx, logit = ki.make_teacher(N, K, V, dev, seed=ki.SEED_TEACHER + seed)
    ignore = None
    if ign > 0:
        g = torch.Generator(device="cpu")
        g.manual_seed(ki.SEED_MASK + seed)
        ignore = (torch.rand(N, generator=g) < ign).to(torch.uint8).to(dev)
    return hidden, W, idx, logit, ignore


def test_noalloc_matches_fwd_bwd(gpu_lib):
    kd = gpu_lib
    for n, (N, D, V, K, chunk, tau, ign, dtype, same_plan) in enumerate(CASES):
        print(f"[noalloc] call {n + 1}: N={N} D={D} V={V} K={K} chunk={chunk} {dtype}",
              flush=True)
        hidden, W, idx, logit, ignore = _inputs(N, D, V, K, dtype, ign, seed=100 + n)
        ref = kd.fwd_bwd(hidden, W, idx, logit, tau=tau, ignore=ignore, chunk=chunk,
                         loss_per_token=True)
        out = {"loss": torch.empty((), dtype=torch.float32, device="cuda"),
               "loss_per_token": torch.full((N,), float("nan"), device="cuda"),
               "grad_hidden": torch.full((N, D), float("nan"), dtype=dtype, device="cuda"),
               "grad_W": torch.full((V, D), float("nan"), device="cuda")}
        got = kd.fwd_bwd_noalloc(hidden, W, idx, logit, tau=tau, ignore=ignore, chunk=chunk,
                                 out=out, loss_per_token=True)
        torch.cuda.synchronize()
        for k in ("loss", "loss_per_token", "grad_hidden", "grad_W"):
            assert got[k].data_ptr() == out[k].data_ptr()
        assert torch.equal(got["loss"], ref["loss"])
        assert torch.equal(got["loss_per_token"], ref["loss_per_token"])
        if same_plan:
            assert torch.equal(got["grad_hidden"], ref["grad_hidden"])
            assert torch.equal(got["grad_W"], ref["grad_W"])
        else:
            tol = TOL["bf16" if dtype == torch.bfloat16 else "f32"]["grad"]
            e_h = rel_max(to64(got["grad_hidden"]), to64(ref["grad_hidden"]))
            e_w = rel_max(to64(got["grad_W"]), to64(ref["grad_W"]))
            print(f"[noalloc] call {n + 1}: capped plan, grad_hidden {e_h:.2e}, "
                  f"grad_W {e_w:.2e}", flush=True)
            assert e_h <= tol and e_w <= tol


def test_noalloc_call_in_a_graph(gpu_lib):
    """The allocation-free call captured into a HIP graph (torch.cuda.graph) and
    replayed three times, with other eager work (a call through the workspace
    entry point on other inputs, and fills of the outputs) between the replays:
    every replay rewrites every output bitwise equal to the eager call's. A
    tenth of the tokens is ignored, so the captured call includes the gather
    of the tokens that are not ignored and the skip of the tiles past them."""
    kd = gpu_lib
    N, D, V, K, chunk, tau = 1000, 256, 50000, 32, 256, 1.5
    dev = "cuda"
    h = ki.make_hidden(N, D, torch.bfloat16, dev, seed=ki.SEED_HIDDEN + 61)
    W = ki.make_weight(V, D, torch.bfloat16, dev, seed=ki.SEED_W + 61)
    idx, logit = ki.make_teacher(N, K, V, dev, seed=ki.SEED_TEACHER + 61)
    h2 = ki.make_hidden(N, D, torch.bfloat16, dev, seed=ki.SEED_HIDDEN + 62)
    gm = torch.Generator(device="cpu")
    gm.manual_seed(ki.SEED_MASK + 61)
    ign = (torch.rand(N, generator=gm) < 0.1).to(torch.uint8).to(dev)

    def outs():
        return {"loss": torch.empty((), dtype=torch.float32, device=dev),
                "loss_per_token": torch.empty(N, dtype=torch.float32, device=dev),
                "grad_hidden": torch.empty(N, D, dtype=torch.bfloat16, device=dev),
                "grad_W": torch.empty(V, D, dtype=torch.float32, device=dev)}
    eager = kd.fwd_bwd_noalloc(h, W, idx, logit, tau=tau, ignore=ign, chunk=chunk, out=outs(),
                               loss_per_token=True)
    torch.cuda.synchronize()
    out = outs()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        kd.fwd_bwd_noalloc(h, W, idx, logit, tau=tau, ignore=ign, chunk=chunk, out=out,
                           loss_per_token=True)
    torch.cuda.synchronize()
    for rep in range(3):
        for t in out.values():
            t.fill_(float("nan"))
        other = kd.fwd_bwd(h2, W, idx, logit, tau=tau, ignore=ign, chunk=chunk)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        print(f"[graph] replay {rep}: loss {float(out['loss']):.6f}", flush=True)
        for k in out:
            assert torch.equal(out[k], eager[k]), (rep, k)
        assert not torch.equal(other["grad_W"], eager["grad_W"])


def test_noalloc_debug_index_check(gpu_lib, monkeypatch):
    """KD_DEBUG_CHECK=1 on the allocation-free call: the index check runs in the
    static scratch first; an index outside [0, V) gives KD_ERR_BAD_INDEX with no
    output touched, valid indices the same outputs as without the check."""
    kd = gpu_lib
    N, D, V, K, chunk = 300, 64, 1000, 20, 128
    dev = "cuda"
    h = ki.make_hidden(N, D, torch.float32, dev, seed=ki.SEED_HIDDEN + 71)
    W = ki.make_weight(V, D, torch.float32, dev, seed=ki.SEED_W + 71)
    idx, logit = ki.make_teacher(N, K, V, dev, seed=ki.SEED_TEACHER + 71)
    ref = kd.fwd_bwd_noalloc(h, W, idx, logit, chunk=chunk)
    torch.cuda.synchronize()
    monkeypatch.setenv("KD_DEBUG_CHECK", "1")
    out = kd.fwd_bwd_noalloc(h, W, idx, logit, chunk=chunk)
    torch.cuda.synchronize()
    for k in ref:
        assert torch.equal(out[k], ref[k]), k
    bad = idx.clone()
    bad[123, 4] = V
    sentinel = {"loss": torch.full((), 7.0, device=dev),
                "grad_hidden": torch.full((N, D), 7.0, device=dev),
                "grad_W": torch.full((V, D), 7.0, device=dev)}
    with pytest.raises(kd.KdError) as e:
        kd.fwd_bwd_noalloc(h, W, bad, logit, chunk=chunk, out=sentinel)
    assert e.value.code == 6
    torch.cuda.synchronize()
    for t in sentinel.values():
        assert bool((t == 7.0).all())
    monkeypatch.delenv("KD_DEBUG_CHECK")
