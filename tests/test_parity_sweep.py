"""Seeded random sweep of small problems, every output against the fp64 oracle,
through the fused call and through the split entry points (forward, then the
backward with its logit recompute).

The configurations are drawn once from a fixed seed: token counts from 1 to
700, hidden sizes 64 to 256, vocabularies from K to 70000 (the largest give
more than 256 grad_W tiles with a partly filled last round, which the dW
contraction splits along the tokens), chunks that are ragged, larger than N,
or multiples of 256 (which the schedule may merge per dW group), temperatures
0.5 to 2.5, fp32 and bf16, logits and log-probability teachers, 0 to 30% of
the tokens ignored, then sixteen more with half to all of the tokens ignored.
Each case prints its configuration before it runs.
"""
import numpy as np
import pytest
import torch

import kd_inputs as ki
from oracle import kd_topk_kl
from tests.helpers import TOL, oracle_inputs, rel_max, to64

pytestmark = pytest.mark.gpu


def _configs(n=24, seed=2024, n_masked=16, seed_masked=2025):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        N = int(rng.choice([1, 7, 63, 64, 255, 256, 257, 300, 511, 700]))
        D = int(rng.choice([64, 128, 192, 256]))
        K = int(rng.choice([1, 3, 16, 37, 64]))
        V = int(rng.choice([max(K, 40), 997, 4096, 5003, 70000 if D == 64 else 9000]))
        V = max(V, K)
        chunk = int(rng.choice([1, 7, 100, 256, 512, N + 5]))
        tau = float(np.round(rng.uniform(0.5, 2.5), 2))
        dtype = "bf16" if rng.random() < 0.5 else "f32"
        logprobs = bool(rng.random() < 0.25)
        ign = float(rng.choice([0.0, 0.1, 0.3]))
        out.append((i, N, D, V, K, chunk, tau, dtype, logprobs, ign))
    # heavier masks (every entry point leaves ignored tokens out), up to all
    # tokens ignored
    rng = np.random.default_rng(seed_masked)
    for i in range(n_masked):
        N = int(rng.choice([2, 65, 256, 300, 513, 700, 1200]))
        D = int(rng.choice([64, 128, 256]))
        K = int(rng.choice([1, 8, 16, 50]))
        V = max(K, int(rng.choice([300, 997, 4096, 9000])))
        chunk = int(rng.choice([1, 33, 100, 128, 256, N + 1]))
        tau = float(np.round(rng.uniform(0.5, 2.5), 2))
        dtype = "bf16" if rng.random() < 0.5 else "f32"
        logprobs = bool(rng.random() < 0.25)
        ign = float(rng.choice([0.5, 0.8, 0.97, 1.0]))
        out.append((100 + i, N, D, V, K, chunk, tau, dtype, logprobs, ign))
    # more than 256 grad_W tiles with a partly filled last round (split along
    # the tokens), in fp32 and in bf16 with a chunk the schedule merges
    out.append((n, 300, 64, 70000, 16, 100, 1.0, "f32", False, 0.1))
    out.append((n + 1, 700, 64, 70000, 32, 256, 1.5, "bf16", False, 0.2))
    return out


@pytest.mark.parametrize("cfg", _configs(), ids=lambda c: f"case{c[0]}")
def test_random_problem(gpu_lib, cfg):
    kd = gpu_lib
    i, N, D, V, K, chunk, tau, dtype, logprobs, ign = cfg
    print(f"[sweep] case {i}: N={N} D={D} V={V} K={K} chunk={chunk} tau={tau} {dtype} "
          f"logprobs={logprobs} ignored={ign}", flush=True)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    dev = "cuda"
    h = ki.make_hidden(N, D, tdt, dev, seed=ki.SEED_HIDDEN + 100 + i)
    W = ki.make_weight(V, D, tdt, dev, seed=ki.SEED_W + 100 + i, std=0.05)
    idx, logit = ki.make_teacher(N, K, V, dev, seed=ki.SEED_TEACHER + 100 + i)
    if logprobs:
        logit = (torch.log_softmax(logit, dim=1) - 0.2).contiguous()
    ignore = None
    if ign > 0:
        g = torch.Generator(device="cpu")
        g.manual_seed(ki.SEED_MASK + 100 + i)
        ignore = (torch.rand(N, generator=g) < ign).to(torch.uint8).to(dev)
    inp = dict(hidden=h, W=W, teacher_idx=idx, teacher_logit=logit, ignore=ignore)
    args = (h, W, idx, logit)
    fb = kd.fwd_bwd(*args, tau=tau, ignore=ignore, chunk=chunk, loss_per_token=True,
                    teacher_logprobs=logprobs)
    f = kd.fwd(*args, tau=tau, ignore=ignore, chunk=chunk, loss_per_token=True,
               teacher_logprobs=logprobs)
    b = kd.bwd(*args, f["saved_logz"], tau=tau, ignore=ignore, chunk=chunk,
               teacher_logprobs=logprobs)
    torch.cuda.synchronize()
    ref = kd_topk_kl(**oracle_inputs(inp), tau=tau, chunk=chunk,
                     teacher_mode="logprobs" if logprobs else "logits")
    tol = TOL[dtype]
    scale = max(abs(ref["loss"]), 1e-30)
    for res in (fb, f):
        assert abs(float(res["loss"]) - ref["loss"]) <= tol["loss"] * scale
        assert rel_max(to64(res["loss_per_token"]), ref["loss_per_token"]) <= tol["loss"]
    # saved log Z: ignored tokens are left out (0), the others against the oracle
    lz = to64(f["saved_logz"])
    keep = np.ones(N, bool) if ignore is None else to64(ignore) == 0
    assert np.all(lz[~keep] == 0.0)
    if keep.any():
        assert rel_max(lz[keep], ref["logZ"][keep]) <= tol["loss"]
    for res in (fb, b):
        assert rel_max(to64(res["grad_hidden"]), ref["grad_hidden"]) <= tol["grad"]
        assert rel_max(to64(res["grad_W"]), ref["grad_W"]) <= tol["grad"]
