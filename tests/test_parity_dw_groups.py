"""grad_W on the dW path the benchmark times, every element against the oracle.

At the benchmark's vocabulary (V = 131072) and chunk (4096 tokens), the fused
call gathers the dZ rows of 4 chunks (16384 tokens) before each grad_W
contraction: the K-major dZ operand then spans 4 GiB (its buffer resource is
re-based every K step), the transposed hidden rows have a pitch of 16384
tokens, and every group after the first accumulates into grad_W (beta = 1).
A small hidden size keeps the fp64 oracle to seconds while every one of those
conditions holds exactly as in the timed run; the oracle is evaluated over all
N rows (row blocks on a thread pool, summed for grad_W). Algorithm 1's
backward (dW += G^T h per chunk) and Eq. 3 define the reference.

  * N = 32768: two full groups (the loss32k token count and grouping);
  * N = 20000: a full group and a short last group of 3616 tokens (one
    partial chunk), with 5% of the tokens ignored.

grad_W is compared element by element, and so are grad_hidden (all rows), the
per-token losses and the loss.
"""
import numpy as np
import pytest
import torch

import kd_inputs as ki
from oracle import kd_topk_kl
from tests.helpers import TOL, oracle_by_row_blocks, rel_max, to64

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


@pytest.mark.parametrize("N,D,ign", [(32768, 64, 0.0), (20000, 128, 0.05)])
def test_grad_W_full_groups(gpu_lib, N, D, ign):
    V, K, chunk, tau = 131072, 100, 4096, 1.0
    print(f"[dw-groups] N={N} D={D} V={V} K={K} chunk={chunk} ignored={ign}", flush=True)
    dev = "cuda"
    hidden = ki.make_hidden(N, D, torch.bfloat16, dev)
    W = ki.make_weight(V, D, torch.bfloat16, dev)
    idx, logit = ki.make_teacher(N, K, V, dev)
    ignore = None
    if ign > 0:
        g = torch.Generator(device="cpu")
        g.manual_seed(ki.SEED_MASK)
        ignore = torch.zeros(N, dtype=torch.uint8)
        ignore[torch.randperm(N, generator=g)[:int(ign * N)]] = 1
        ignore = ignore.to(dev)
    # the grouping this test is about: 4 chunks per dW contraction, a 4 GiB
    # dZ buffer in the workspace
    ws = gpu_lib.workspace_size(N, D, V, K, chunk, tau, gpu_lib.KD_BF16)
    assert ws >= 16384 * V * 2
    out = gpu_lib.fwd_bwd(hidden, W, idx, logit, tau=tau, ignore=ignore, chunk=chunk,
                          loss_per_token=True)
    torch.cuda.synchronize()
    ref = oracle_by_row_blocks(kd_topk_kl, to64(hidden), to64(W), to64(idx), to64(logit), tau,
                               ignore=to64(ignore))
    e_l = abs(float(out["loss"]) - ref["loss"]) / abs(ref["loss"])
    e_t = rel_max(to64(out["loss_per_token"]), ref["loss_per_token"])
    e_h = rel_max(to64(out["grad_hidden"]), ref["grad_hidden"])
    e_w = rel_max(to64(out["grad_W"]), ref["grad_W"])
    print(f"[dw-groups] N={N}: loss rel {e_l:.2e}, l_t {e_t:.2e}, grad_hidden {e_h:.2e}, "
          f"grad_W {e_w:.2e}", flush=True)
    assert e_l <= TOL["bf16"]["loss"]
    assert e_t <= TOL["bf16"]["loss"]
    assert e_h <= TOL["bf16"]["grad"]
    assert e_w <= TOL["bf16"]["grad"]


@pytest.mark.parametrize("N,D,V,K,chunk,dtype,ign", [
    # 300 dW tiles (one full round of 256 and 44 tail tiles split 4 ways),
    # two groups: the second group's tail tiles add to grad_W (beta = 1)
    (20000, 64, 76800, 32, 4096, torch.bfloat16, 0.05),
    # fp32, 274 tiles (18 tail tiles), one group, a ragged vocabulary tile
    (300, 64, 70000, 8, 100, torch.float32, 0.0),
])
def test_grad_W_split_tail(gpu_lib, N, D, V, K, chunk, dtype, ign):
    """The dW contraction's last, partly filled round of tiles is split along
    the tokens and its parts are added to grad_W by a fixup pass: every grad_W
    element against the oracle, and accumulate_grad_W adds a second call's
    gradient on top (twice the first call's, to fp32 rounding)."""
    tol = TOL["bf16" if dtype == torch.bfloat16 else "f32"]
    print(f"[dw-split] N={N} D={D} V={V} K={K} chunk={chunk} {dtype}", flush=True)
    dev = "cuda"
    hidden = ki.make_hidden(N, D, dtype, dev, seed=ki.SEED_HIDDEN + 7)
    W = ki.make_weight(V, D, dtype, dev, seed=ki.SEED_W + 7)
    idx, logit = ki.make_teacher(N, K, V, dev, seed=ki.SEED_TEACHER + 7)
    ignore = None
    if ign > 0:
        g = torch.Generator(device="cpu")
        g.manual_seed(ki.SEED_MASK + 7)
        ignore = (torch.rand(N, generator=g) < ign).to(torch.uint8).to(dev)
    out = gpu_lib.fwd_bwd(hidden, W, idx, logit, tau=1.0, ignore=ignore, chunk=chunk)
    acc = out["grad_W"].clone()
    gpu_lib.fwd_bwd(hidden, W, idx, logit, tau=1.0, ignore=ignore, chunk=chunk, grad_hidden=False,
                    grad_W_out=acc, accumulate_grad_W=True)
    torch.cuda.synchronize()
    ref = oracle_by_row_blocks(kd_topk_kl, to64(hidden), to64(W), to64(idx), to64(logit), 1.0,
                               ignore=to64(ignore))
    e_w = rel_max(to64(out["grad_W"]), ref["grad_W"])
    e_h = rel_max(to64(out["grad_hidden"]), ref["grad_hidden"])
    e_a = rel_max(to64(acc), 2.0 * to64(out["grad_W"]))
    print(f"[dw-split] grad_W {e_w:.2e}, grad_hidden {e_h:.2e}, accumulated {e_a:.2e}",
          flush=True)
    assert e_w <= tol["grad"]
    assert e_h <= tol["grad"]
    assert e_a <= 1e-6


def test_merged_chunks_with_short_last_group(gpu_lib):
    """Chunks whose projection leaves the last round of tiles partly filled
    (2 x 196 = 392 tiles per 512-token chunk) while dH runs per group are
    processed as one chunk per dW group: 20000 tokens in chunks of 512 run as
    16384 + 3616 tokens. Every output against the oracle; the loss and the
    per-token losses equal those of a chunk size that is not merged (100)."""
    N, D, V, K, chunk, tau = 20000, 64, 50000, 16, 512, 2.0
    dev = "cuda"
    hidden = ki.make_hidden(N, D, torch.bfloat16, dev, seed=ki.SEED_HIDDEN + 9)
    W = ki.make_weight(V, D, torch.bfloat16, dev, seed=ki.SEED_W + 9)
    idx, logit = ki.make_teacher(N, K, V, dev, seed=ki.SEED_TEACHER + 9)
    g = torch.Generator(device="cpu")
    g.manual_seed(ki.SEED_MASK + 9)
    ignore = (torch.rand(N, generator=g) < 0.05).to(torch.uint8).to(dev)
    out = gpu_lib.fwd_bwd(hidden, W, idx, logit, tau=tau, ignore=ignore, chunk=chunk,
                          loss_per_token=True)
    other = gpu_lib.fwd_bwd(hidden, W, idx, logit, tau=tau, ignore=ignore, chunk=100,
                            loss_per_token=True, grad_hidden=False, grad_W=False)
    torch.cuda.synchronize()
    ref = oracle_by_row_blocks(kd_topk_kl, to64(hidden), to64(W), to64(idx), to64(logit), tau,
                               ignore=to64(ignore))
    e_l = abs(float(out["loss"]) - ref["loss"]) / abs(ref["loss"])
    e_t = rel_max(to64(out["loss_per_token"]), ref["loss_per_token"])
    e_h = rel_max(to64(out["grad_hidden"]), ref["grad_hidden"])
    e_w = rel_max(to64(out["grad_W"]), ref["grad_W"])
    print(f"[merged] loss rel {e_l:.2e}, l_t {e_t:.2e}, grad_hidden {e_h:.2e}, grad_W {e_w:.2e}",
          flush=True)
    assert e_l <= TOL["bf16"]["loss"] and e_t <= TOL["bf16"]["loss"]
    assert e_h <= TOL["bf16"]["grad"] and e_w <= TOL["bf16"]["grad"]
    # the per-token arithmetic does not depend on the chunking
    lt, lo = out["loss_per_token"], other["loss_per_token"]
    assert rel_max(to64(lt), to64(lo)) <= 1e-6
    assert torch.equal(lt[ignore.bool()], torch.zeros_like(lt[ignore.bool()]))
