"""Ignored tokens left out of the fused call's work, against the fp64 oracle.

With a mask, kd_topk_kl_fwd_bwd gathers each dW group's tokens that are not
ignored, runs the contractions on them only (tiles past their count are
skipped, the grad_W token range stops there), and writes 0 to the ignored
tokens' per-token losses and grad_hidden rows. These cases are built to reach
each consequence: heavy and structured masks (a whole dW group ignored, a
group with a few tokens at its end, every token ignored), a token count that
ends inside a chunk that is not a multiple of the 64-token K step (the dZ
rows past the tokens must not reach grad_W), the split grad_W tail, split dH,
fp32 grad_hidden, grad_W accumulation and the allocation-free entry point.
The workspace and the outputs start as NaN bytes, so any value the call
should have written and did not, or any stale row that leaks into a sum,
fails the comparison. Each case prints its configuration before it runs.
"""
import numpy as np
import pytest
import torch

import kd_inputs as ki
from oracle import kd_topk_kl
from tests.helpers import TOL, oracle_inputs, rel_max, to64

pytestmark = pytest.mark.gpu


def _mask(N, kind, seed):
    g = np.random.default_rng(seed)
    m = np.zeros(N, dtype=np.uint8)
    if kind == "half":
        m[:] = g.random(N) < 0.5
    elif kind == "all":
        m[:] = 1
    elif kind == "p90":
        m[:] = g.random(N) < 0.9
    elif kind == "groups":
        # first dW group half ignored, the second all ignored, the third only
        # its last 10 tokens kept (groups of 16384 tokens at chunk 4096)
        m[:16384] = g.random(16384) < 0.5
        m[16384:32768] = 1
        m[32768:] = 1
        m[-10:] = 0
    elif kind == "prefix199":
        # 199 tokens kept, at scattered places: the count ends inside the
        # second chunk of 100 rows, short of a 64-row boundary
        keep = g.choice(N, 199, replace=False)
        m[:] = 1
        m[keep] = 0
    elif kind == "p30":
        m[:] = g.random(N) < 0.3
    else:
        raise ValueError(kind)
    return torch.from_numpy(m)


# (name, N, D, V, K, chunk, dtype, mask, tau, extra)
CASES = [
    ("half_bf16", 1000, 128, 5003, 16, 256, "bf16", "half", 1.0, {}),
    ("half_f32_ragged", 700, 64, 997, 8, 100, "f32", "half", 1.5, {}),
    ("all_ignored", 300, 64, 1000, 8, 100, "bf16", "all", 1.0, {}),
    ("all_ignored_accumulate", 300, 64, 1000, 8, 100, "f32", "all", 1.0, {"accumulate": True}),
    ("p90_per_chunk_dh", 2048, 64, 3000, 8, 256, "bf16", "p90", 2.0, {}),
    ("groups_f32", 40000, 64, 1000, 8, 4096, "f32", "groups", 1.0, {}),
    ("groups_bf16_accumulate", 40000, 64, 1000, 8, 4096, "bf16", "groups", 0.7,
     {"accumulate": True}),
    ("count_in_ragged_chunk", 700, 64, 997, 8, 100, "bf16", "prefix199", 1.0, {}),
    ("count_in_ragged_chunk_f32", 700, 64, 997, 8, 100, "f32", "prefix199", 1.0, {}),
    ("split_dw_tail", 700, 64, 70000, 16, 256, "bf16", "p30", 1.0, {}),
    ("split_dh", 300, 256, 9000, 16, 300, "bf16", "half", 1.0, {}),
    ("groups_not_merged", 1000, 64, 65536, 16, 256, "bf16", "half", 1.0, {}),
    ("per_chunk_dh", 8192, 4096, 1000, 8, 4096, "bf16", "half", 1.0, {}),
    ("grad_hidden_f32", 1000, 128, 5003, 16, 256, "bf16", "half", 1.0, {"gh_f32": True}),
    ("logprobs", 600, 64, 4096, 37, 128, "bf16", "p30", 1.0, {"logprobs": True}),
    ("frozen_W", 600, 64, 4096, 16, 128, "bf16", "half", 1.0, {"grad_W": False}),
    ("no_grad_hidden", 600, 64, 4096, 16, 128, "bf16", "half", 1.0, {"grad_hidden": False}),
    ("mask_at_odd_address", 1000, 128, 5003, 16, 256, "bf16", "half", 1.0, {"mask_offset": 3}),
    ("loss_only", 1000, 128, 5003, 16, 256, "bf16", "half", 1.0,
     {"grad_hidden": False, "grad_W": False}),
    ("loss_only_f32_groups", 40000, 64, 1000, 8, 4096, "f32", "groups", 1.0,
     {"grad_hidden": False, "grad_W": False}),
    ("loss_only_all_ignored", 300, 64, 1000, 8, 100, "bf16", "all", 1.0,
     {"grad_hidden": False, "grad_W": False}),
]


def _nan_like(shape, dtype, dev):
    return torch.full(shape, float("nan"), dtype=dtype, device=dev)


@pytest.mark.parametrize("case", CASES, ids=lambda c: c[0])
def test_ignored_tokens(gpu_lib, case):
    kd = gpu_lib
    name, N, D, V, K, chunk, dtype, mkind, tau, ex = case
    print(f"[ignored] {name}: N={N} D={D} V={V} K={K} chunk={chunk} {dtype} mask={mkind} "
          f"tau={tau} {ex}", flush=True)
    dev = "cuda"
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    seed = 500 + CASES.index(case)
    h = ki.make_hidden(N, D, tdt, dev, seed=ki.SEED_HIDDEN + seed)
    W = ki.make_weight(V, D, tdt, dev, seed=ki.SEED_W + seed, std=0.05)
    idx, logit = ki.make_teacher(N, K, V, dev, seed=ki.SEED_TEACHER + seed)
    logprobs = ex.get("logprobs", False)
    if logprobs:
        logit = (torch.log_softmax(logit, dim=1) - 0.2).contiguous()
    ignore = _mask(N, mkind, ki.SEED_MASK + seed).to(dev)
    if ex.get("mask_offset"):
        # a mask that starts at an address that is not 4-byte aligned
        o = ex["mask_offset"]
        buf = torch.zeros(N + o, dtype=torch.uint8, device=dev)
        buf[o:] = ignore
        ignore = buf[o:]
        assert ignore.data_ptr() % 4 == o % 4
    want_h, want_W = ex.get("grad_hidden", True), ex.get("grad_W", True)
    gh_f32 = ex.get("gh_f32", False)
    acc = ex.get("accumulate", False)
    ws = torch.full((kd.workspace_size(N, D, V, K, chunk, tau, kd.KD_BF16 if dtype == "bf16"
                                       else kd.KD_F32),), 0xFF, dtype=torch.uint8, device=dev)
    out = {"loss_per_token": _nan_like((N,), torch.float32, dev)}
    if want_h:
        out["grad_hidden"] = _nan_like((N, D), torch.float32 if gh_f32 else tdt, dev)
    gW0 = None
    if want_W:
        if acc:
            gW0 = torch.randn(V, D, dtype=torch.float32, device=dev) * 1e-3
            out["grad_W"] = gW0.clone()
        else:
            out["grad_W"] = _nan_like((V, D), torch.float32, dev)
    res = kd.fwd_bwd(h, W, idx, logit, tau=tau, ignore=ignore, chunk=chunk,
                     loss_per_token=True, grad_hidden=want_h, grad_W=want_W,
                     accumulate_grad_W=acc, workspace=ws, out=out,
                     teacher_logprobs=logprobs, grad_hidden_f32=gh_f32)
    torch.cuda.synchronize()
    inp = dict(hidden=h, W=W, teacher_idx=idx, teacher_logit=logit, ignore=ignore)
    ref = kd_topk_kl(**oracle_inputs(inp), tau=tau, chunk=chunk,
                     teacher_mode="logprobs" if logprobs else "logits")
    tol = TOL[dtype]
    ign = ignore.cpu().numpy().astype(bool)
    lpt = to64(res["loss_per_token"])
    assert np.all(lpt[ign] == 0.0)
    if ign.all():
        assert float(res["loss"]) == 0.0
    else:
        scale = max(abs(ref["loss"]), 1e-30)
        assert abs(float(res["loss"]) - ref["loss"]) <= tol["loss"] * scale
        assert rel_max(lpt, ref["loss_per_token"]) <= tol["loss"]
    if want_h:
        gh = to64(res["grad_hidden"])
        assert np.all(gh[ign] == 0.0)
        if not ign.all():
            assert rel_max(gh, ref["grad_hidden"]) <= tol["grad"]
    if want_W:
        gW = to64(res["grad_W"])
        refW = ref["grad_W"] + (to64(gW0) if acc else 0.0)
        if ign.all():
            assert np.array_equal(gW, to64(gW0) if acc else np.zeros_like(gW))
        else:
            assert rel_max(gW - (to64(gW0) if acc else 0.0), ref["grad_W"]) <= tol["grad"]
            assert np.isfinite(gW).all() and rel_max(gW, refW) <= tol["grad"]


def test_ignored_tokens_deterministic_and_skipped(gpu_lib):
    """Two calls give the same bits; the gather runs only with a mask; a mask
    that ignores most tokens makes the projection cheaper."""
    kd = gpu_lib
    N, D, V, K, chunk = 4096, 1024, 32768, 16, 2048
    print(f"[ignored] deterministic: N={N} D={D} V={V} chunk={chunk}", flush=True)
    dev = "cuda"
    h = ki.make_hidden(N, D, torch.bfloat16, dev, seed=ki.SEED_HIDDEN + 600)
    W = ki.make_weight(V, D, torch.bfloat16, dev, seed=ki.SEED_W + 600, std=0.05)
    idx, logit = ki.make_teacher(N, K, V, dev, seed=ki.SEED_TEACHER + 600)
    ignore = _mask(N, "p90", ki.SEED_MASK + 600).to(dev)
    a = kd.fwd_bwd(h, W, idx, logit, ignore=ignore, chunk=chunk, loss_per_token=True)
    b = kd.fwd_bwd(h, W, idx, logit, ignore=ignore, chunk=chunk, loss_per_token=True)
    torch.cuda.synchronize()
    for k in ("loss", "loss_per_token", "grad_hidden", "grad_W"):
        assert torch.equal(a[k].view(torch.uint8) if a[k].dim() else a[k].reshape(1),
                           b[k].view(torch.uint8) if b[k].dim() else b[k].reshape(1)), k
    kd.profile_enable(True)
    kd.fwd_bwd(h, W, idx, logit, ignore=ignore, chunk=chunk)
    torch.cuda.synchronize()
    masked = kd.profile_read()
    kd.fwd_bwd(h, W, idx, logit, chunk=chunk)
    torch.cuda.synchronize()
    plain = kd.profile_read()
    kd.profile_enable(False)
    assert masked["compact"]["launches"] == 1 and "compact" not in plain
    # 90% of the tokens ignored: the projection covers 2 of 8 token tiles
    # per chunk (about 410 of 2048 rows)
    assert masked["logits_dz"]["total_ms"] < 0.6 * plain["logits_dz"]["total_ms"]


def test_ignored_tokens_noalloc(gpu_lib):
    """The allocation-free entry point takes the same path with a mask."""
    kd = gpu_lib
    N, D, V, K, chunk = 700, 64, 997, 8, 100
    print(f"[ignored] noalloc: N={N} D={D} V={V} chunk={chunk}", flush=True)
    dev = "cuda"
    h = ki.make_hidden(N, D, torch.bfloat16, dev, seed=ki.SEED_HIDDEN + 700)
    W = ki.make_weight(V, D, torch.bfloat16, dev, seed=ki.SEED_W + 700, std=0.05)
    idx, logit = ki.make_teacher(N, K, V, dev, seed=ki.SEED_TEACHER + 700)
    ignore = _mask(N, "prefix199", ki.SEED_MASK + 700).to(dev)
    a = kd.fwd_bwd(h, W, idx, logit, ignore=ignore, chunk=chunk, loss_per_token=True)
    b = kd.fwd_bwd_noalloc(h, W, idx, logit, ignore=ignore, chunk=chunk, loss_per_token=True)
    torch.cuda.synchronize()
    for k in ("loss", "loss_per_token", "grad_hidden", "grad_W"):
        assert torch.equal(a[k].float(), b[k].float()), k


def test_ignored_tokens_noalloc_smaller_groups(gpu_lib):
    """At V = 131072 the allocation-free call's 256 MiB scratch holds the dZ
    rows of one 512-token chunk, so its dW groups (and the gathers) are 512
    tokens where kd_topk_kl_fwd_bwd gathers 4096: both against the oracle."""
    kd = gpu_lib
    N, D, V, K, chunk = 4096, 64, 131072, 16, 512
    print(f"[ignored] noalloc, smaller groups: N={N} D={D} V={V} chunk={chunk}", flush=True)
    dev = "cuda"
    h = ki.make_hidden(N, D, torch.bfloat16, dev, seed=ki.SEED_HIDDEN + 800)
    W = ki.make_weight(V, D, torch.bfloat16, dev, seed=ki.SEED_W + 800, std=0.05)
    idx, logit = ki.make_teacher(N, K, V, dev, seed=ki.SEED_TEACHER + 800)
    ignore = _mask(N, "half", ki.SEED_MASK + 800).to(dev)
    a = kd.fwd_bwd(h, W, idx, logit, ignore=ignore, chunk=chunk, loss_per_token=True)
    b = kd.fwd_bwd_noalloc(h, W, idx, logit, ignore=ignore, chunk=chunk, loss_per_token=True)
    torch.cuda.synchronize()
    inp = dict(hidden=h, W=W, teacher_idx=idx, teacher_logit=logit, ignore=ignore)
    ref = kd_topk_kl(**oracle_inputs(inp), tau=1.0, chunk=chunk)
    tol = TOL["bf16"]
    ign = ignore.cpu().numpy().astype(bool)
    for res in (a, b):
        assert abs(float(res["loss"]) - ref["loss"]) <= tol["loss"] * abs(ref["loss"])
        lpt, gh = to64(res["loss_per_token"]), to64(res["grad_hidden"])
        assert np.all(lpt[ign] == 0.0) and np.all(gh[ign] == 0.0)
        assert rel_max(lpt, ref["loss_per_token"]) <= tol["loss"]
        assert rel_max(gh, ref["grad_hidden"]) <= tol["grad"]
        assert rel_max(to64(res["grad_W"]), ref["grad_W"]) <= tol["grad"]
    # each token's loss and grad_hidden row come from the same tiles either way
    assert torch.equal(a["loss_per_token"], b["loss_per_token"])
