"""GPU parity at sizes the oracle finishes in seconds: every element of the
loss, per-token loss and both gradients against the fp64 oracle on the same
seeded inputs. Shapes span several 256x256 tiles with ragged tails in N, V and
the chunk, plus the method's degenerate cases."""
import numpy as np
import pytest
import torch

import kd_inputs as ki
from oracle import kd_topk_kl
from tests.helpers import TOL, oracle_inputs, rel_max, to64

pytestmark = pytest.mark.gpu


def _inputs(N, D, V, K, dtype, seed=0, ignore_frac=0.0, wstd=0.02, hstd=1.0):
    dev = "cuda"
    hidden = ki.make_hidden(N, D, dtype, dev, seed=ki.SEED_HIDDEN + seed, std=hstd)
    W = ki.make_weight(V, D, dtype, dev, seed=ki.SEED_W + seed, std=wstd)
    idx, logit = ki.make_teacher(N, K, V, dev, seed=ki.SEED_TEACHER + seed)
    ignore = None
    if ignore_frac > 0:
        g = torch.Generator(device="cpu")
        g.manual_seed(ki.SEED_MASK + seed)
        ignore = (torch.rand(N, generator=g) < ignore_frac).to(torch.uint8).to(dev)
    return dict(hidden=hidden, W=W, teacher_idx=idx, teacher_logit=logit, ignore=ignore)


def _run_and_compare(kd, inp, tau, chunk, tol, grads=True):
    torch.cuda.synchronize()
    out = kd.fwd_bwd(inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"], tau=tau,
                     ignore=inp["ignore"], chunk=chunk, loss_per_token=True,
                     grad_hidden=grads, grad_W=grads)
    torch.cuda.synchronize()
    ref = kd_topk_kl(**oracle_inputs(inp), tau=tau, chunk=chunk, want_grads=grads)
    loss = float(out["loss"])
    assert np.isfinite(loss)
    assert abs(loss - ref["loss"]) <= tol["loss"] * max(abs(ref["loss"]), 1e-30), (loss, ref["loss"])
    lpt = to64(out["loss_per_token"])
    assert rel_max(lpt, ref["loss_per_token"]) <= tol["loss"]
    if grads:
        assert rel_max(to64(out["grad_hidden"]), ref["grad_hidden"]) <= tol["grad"]
        assert rel_max(to64(out["grad_W"]), ref["grad_W"]) <= tol["grad"]
    return out, ref


def test_tiny_fp32_workload(gpu_lib):
    """N=256, D=256, V=4096, K=16, chunk 64, tau 1, fp32."""
    w = ki.WORKLOADS["tiny_fp32"]
    inp = ki.make_workload_inputs(w, "cuda")
    _run_and_compare(gpu_lib, inp, w.tau, w.chunk, TOL["f32"])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("N,D,V,K,chunk,tau,ign", [
    (259, 128, 4133, 7, 100, 2.0, 0.2),      # ragged N, V, chunk; tau 2; mask
    (513, 192, 1000, 16, 513, 1.0, 0.0),     # one chunk, V < 4 tiles, D not /256
    (300, 64, 777, 1, 64, 0.5, 0.1),         # K = 1, tau < 1
    (64, 256, 2048, 40, 1000, 1.0, 0.0),     # chunk > N
])
def test_ragged_shapes(gpu_lib, dtype, N, D, V, K, chunk, tau, ign):
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    inp = _inputs(N, D, V, K, tdt, seed=N + V, ignore_frac=ign)
    _run_and_compare(gpu_lib, inp, tau, chunk, TOL[dtype])


def test_k_equals_v(gpu_lib):
    """The support is the whole vocabulary (P4 structure) on the GPU."""
    inp = _inputs(96, 64, 320, 320, torch.float32, seed=5)
    _run_and_compare(gpu_lib, inp, 1.0, 32, TOL["f32"])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_k_at_the_limit(gpu_lib, dtype):
    """K = 4096, the largest accepted: a 256-token tile carries 2^20 teacher
    entries through the bucket pass (ragged second tile, 5000-column V)."""
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    inp = _inputs(260, 64, 5000, 4096, tdt, seed=41)
    _run_and_compare(gpu_lib, inp, 1.3, 130, TOL[dtype])


def test_identity_head_kl_zero(gpu_lib):
    """W = I (D = V): hidden are the logits; teacher reproduced on its support
    and -1e4 elsewhere gives l = 0 and zero gradients (P2)."""
    V, K, N = 256, 12, 40
    idx, logit = ki.make_teacher(N, K, V, "cuda", seed=77)
    hidden = torch.full((N, V), -1e4, dtype=torch.float32, device="cuda")
    hidden.scatter_(1, idx.long(), logit)
    W = torch.eye(V, dtype=torch.float32, device="cuda")
    out = gpu_lib.fwd_bwd(hidden, W, idx, logit, tau=1.0, chunk=16, loss_per_token=True)
    torch.cuda.synchronize()
    assert abs(float(out["loss"])) < 1e-5
    assert float(out["grad_hidden"].abs().max()) < 1e-6


def test_identity_head_closed_form_gradient(gpu_lib):
    """W = I: grad_hidden is the logit gradient g/tau (M q - p) itself (P6)."""
    V, K, N, tau = 512, 9, 70, 2.0
    inp = _inputs(N, V, V, K, torch.float32, seed=8, hstd=3.0)
    inp["W"] = torch.eye(V, dtype=torch.float32, device="cuda")
    _run_and_compare(gpu_lib, inp, tau, 32, TOL["f32"])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("flag_every", [1, 3])
@pytest.mark.parametrize("top_z", [-40.0, -20.0])
@pytest.mark.parametrize("V", [512, 640])
def test_reference_logit_fallback(gpu_lib, dtype, flag_every, top_z, V):
    """The single projection stores 2^(y - R) with R the student logit at the
    teacher's top entry (+24, base 2); a tile row whose sum of 2^(y - R)
    exceeds 2^40 falls back to its own max and its row is rescaled to the
    largest reference of its runs. W = I puts z = top_z at the top teacher
    entry and z = +40 in another column of every flag_every-th row. With
    top_z = -40 every tile of those rows falls back (its ordinary columns
    alone sum past 2^40); with top_z = -20 only the tile holding the +40
    column does, so a row mixes runs stored against R and against a tile
    max. V = 640 leaves a partial last vocabulary tile. Loss and gradients
    against the oracle."""
    K, N, chunk = 6, 96, 64
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    inp = _inputs(N, V, V, K, torch.float32, seed=31, hstd=1.0)
    h = inp["hidden"]
    idx, logit = inp["teacher_idx"].long(), inp["teacher_logit"]
    top = idx.gather(1, logit.argmax(dim=1, keepdim=True)).squeeze(1)
    rows = torch.arange(0, N, flag_every, device="cuda")
    h[rows, top[rows]] = top_z
    # a column outside the row's teacher support gets the large logit
    far = (top[rows] + V // 2) % V
    mask = (idx[rows] == far[:, None]).any(dim=1)
    far = torch.where(mask, (far + 1) % V, far)
    h[rows, far] = 40.0
    inp["hidden"] = h.to(tdt).contiguous()
    inp["W"] = torch.eye(V, dtype=tdt, device="cuda")
    _run_and_compare(gpu_lib, inp, 1.0, chunk, TOL[dtype])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_small_temperature(gpu_lib, dtype):
    """tau = 0.02 stretches y = z log2(e) / tau to a spread of ~16 (base 2) per
    token on random inputs, so many tile rows sum past 2^40 against the
    reference logit and take the fallback to their own max (no constructed
    logits). Loss and gradients against the oracle."""
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    inp = _inputs(259, 128, 4133, 7, tdt, seed=23, ignore_frac=0.1)
    _run_and_compare(gpu_lib, inp, 0.02, 100, TOL[dtype])


def test_all_ignored(gpu_lib):
    inp = _inputs(200, 64, 600, 5, torch.float32, seed=9)
    inp["ignore"] = torch.ones(200, dtype=torch.uint8, device="cuda")
    out = gpu_lib.fwd_bwd(inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"],
                          ignore=inp["ignore"], chunk=64, loss_per_token=True)
    torch.cuda.synchronize()
    assert float(out["loss"]) == 0.0
    assert float(out["grad_hidden"].abs().max()) == 0.0
    assert float(out["grad_W"].abs().max()) == 0.0
    assert float(out["loss_per_token"].abs().max()) == 0.0


def test_empty_batch(gpu_lib):
    D, V, K = 64, 300, 4
    hidden = torch.empty(0, D, device="cuda")
    W = ki.make_weight(V, D, torch.float32, "cuda")
    idx = torch.empty(0, K, dtype=torch.int32, device="cuda")
    logit = torch.empty(0, K, dtype=torch.float32, device="cuda")
    gW = torch.full((V, D), 7.0, device="cuda")
    out = gpu_lib.fwd_bwd(hidden, W, idx, logit, chunk=16, grad_W_out=gW)
    torch.cuda.synchronize()
    assert float(out["loss"]) == 0.0
    assert float(gW.abs().max()) == 0.0


def test_accumulate_grad_W(gpu_lib):
    inp = _inputs(150, 64, 700, 6, torch.float32, seed=10)
    a = gpu_lib.fwd_bwd(inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"],
                        chunk=64)
    gW = a["grad_W"].clone()
    gpu_lib.fwd_bwd(inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"], chunk=64,
                    grad_W_out=gW, accumulate_grad_W=True, grad_hidden=False)
    torch.cuda.synchronize()
    assert rel_max(to64(gW), 2 * to64(a["grad_W"])) <= 1e-6


def test_forward_only_and_partial_grads(gpu_lib):
    inp = _inputs(260, 128, 900, 8, torch.bfloat16, seed=11, ignore_frac=0.1)
    args = (inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"])
    full = gpu_lib.fwd_bwd(*args, ignore=inp["ignore"], chunk=100)
    fwd = gpu_lib.fwd_bwd(*args, ignore=inp["ignore"], chunk=100, grad_hidden=False, grad_W=False)
    gh = gpu_lib.fwd_bwd(*args, ignore=inp["ignore"], chunk=100, grad_W=False)
    gw = gpu_lib.fwd_bwd(*args, ignore=inp["ignore"], chunk=100, grad_hidden=False)
    torch.cuda.synchronize()
    assert float(fwd["loss"]) == float(full["loss"])
    assert torch.equal(gh["grad_hidden"], full["grad_hidden"])
    assert torch.equal(gw["grad_W"], full["grad_W"])


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_deterministic(gpu_lib, dtype):
    inp = _inputs(600, 128, 3000, 10, dtype, seed=12, ignore_frac=0.05)
    args = (inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"])
    a = gpu_lib.fwd_bwd(*args, ignore=inp["ignore"], chunk=256, loss_per_token=True)
    b = gpu_lib.fwd_bwd(*args, ignore=inp["ignore"], chunk=256, loss_per_token=True)
    torch.cuda.synchronize()
    for k in a:
        assert torch.equal(a[k], b[k]), k


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_several_dw_groups(gpu_lib, dtype):
    """20000 tokens in chunks of 4096: dW gathers 4 chunks per contraction, so
    there are two groups, the second a single short chunk (3616 rows); dH runs
    per group with its vocabulary range split (a chunk alone has 16 tiles).
    Every element against the oracle."""
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    inp = _inputs(20000, 64, 1000, 8, tdt, seed=17, ignore_frac=0.05)
    _run_and_compare(gpu_lib, inp, 1.0, 4096, TOL[dtype])


@pytest.mark.parametrize("chunk", [1, 7, 64, 259, 300])
def test_chunk_invariance(gpu_lib, chunk):
    inp = _inputs(259, 64, 1500, 6, torch.float32, seed=13, ignore_frac=0.1)
    args = (inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"])
    ref = gpu_lib.fwd_bwd(*args, ignore=inp["ignore"], chunk=259)
    out = gpu_lib.fwd_bwd(*args, ignore=inp["ignore"], chunk=chunk)
    torch.cuda.synchronize()
    assert abs(float(out["loss"]) - float(ref["loss"])) <= 1e-6 * abs(float(ref["loss"]))
    assert rel_max(to64(out["grad_hidden"]), to64(ref["grad_hidden"])) <= 1e-6
    assert rel_max(to64(out["grad_W"]), to64(ref["grad_W"])) <= 1e-6


def test_debug_index_check(gpu_lib, monkeypatch):
    """KD_DEBUG_CHECK=1: the entry points check the indices first and return
    KD_ERR_BAD_INDEX (raised by the binding) with no output touched; valid
    indices give the same result as without the check."""
    inp = _inputs(300, 64, 1000, 20, torch.float32, seed=15)
    args = (inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"])
    ref = gpu_lib.fwd_bwd(*args, chunk=128)
    torch.cuda.synchronize()
    monkeypatch.setenv("KD_DEBUG_CHECK", "1")
    out = gpu_lib.fwd_bwd(*args, chunk=128)
    torch.cuda.synchronize()
    assert float(out["loss"]) == float(ref["loss"])
    assert torch.equal(out["grad_W"], ref["grad_W"])
    for bad in (1000, -1):
        idx = inp["teacher_idx"].clone()
        idx[123, 4] = bad
        for call in (lambda: gpu_lib.fwd_bwd(args[0], args[1], idx, args[3], chunk=128),
                     lambda: gpu_lib.fwd(args[0], args[1], idx, args[3], chunk=128)):
            with pytest.raises(gpu_lib.KdError) as e:
                call()
            assert e.value.code == 6
    idx = inp["teacher_idx"].clone()
    idx[7, 1] = idx[7, 0]  # a repeated index
    f = gpu_lib.fwd(*args, chunk=128)
    with pytest.raises(gpu_lib.KdError) as e:
        gpu_lib.bwd(args[0], args[1], idx, args[3], f["saved_logz"], chunk=128)
    assert e.value.code == 6
    monkeypatch.delenv("KD_DEBUG_CHECK")


def test_check_indices(gpu_lib):
    idx, _ = ki.make_teacher(300, 20, 1000, "cuda", seed=14)
    assert gpu_lib.check_indices(idx, V=1000)
    bad = idx.clone()
    bad[17, 3] = 1000
    assert not gpu_lib.check_indices(bad, V=1000)
    bad = idx.clone()
    bad[5, 0] = -1
    assert not gpu_lib.check_indices(bad, V=1000)
    dup = idx.clone()
    dup[123, 7] = dup[123, 2]
    assert not gpu_lib.check_indices(dup, V=1000)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("logprobs", [False, True])
def test_repeated_teacher_indices(gpu_lib, dtype, logprobs):
    """Rows that repeat a teacher index (twice, three times; the repeats far
    apart or adjacent) read as the dense teacher row that sums the repeated
    entries, as the oracle's scatter-add builds it: the fused call and the
    split entry points against the oracle, every output."""
    kd = gpu_lib
    N, D, V, K, chunk, tau = 300, 64, 2000, 12, 128, 1.5
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    inp = _inputs(N, D, V, K, tdt, seed=33, ignore_frac=0.1)
    idx = inp["teacher_idx"].cpu().clone()
    g = torch.Generator(device="cpu")
    g.manual_seed(ki.SEED_TEACHER + 33)
    rows = torch.randperm(N, generator=g)[:100]
    for n, r in enumerate(rows.tolist()):
        a, b = sorted(torch.randperm(K, generator=g)[:2].tolist())
        idx[r, b] = idx[r, a]                 # a pair
        if n % 3 == 0:
            c = int(torch.randint(0, K, (1,), generator=g))
            idx[r, c] = idx[r, a]             # possibly a triple
    inp["teacher_idx"] = idx.to("cuda").contiguous()
    assert not kd.check_indices(inp["teacher_idx"], V)
    if logprobs:
        u = inp["teacher_logit"]
        inp["teacher_logit"] = (torch.log_softmax(u, dim=1) - 0.3).contiguous()
    tol = TOL[dtype]
    ref = kd_topk_kl(**oracle_inputs(inp), tau=tau, chunk=chunk,
                     teacher_mode="logprobs" if logprobs else "logits")
    args = (inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"])
    fb = kd.fwd_bwd(*args, tau=tau, ignore=inp["ignore"], chunk=chunk, loss_per_token=True,
                    teacher_logprobs=logprobs)
    f = kd.fwd(*args, tau=tau, ignore=inp["ignore"], chunk=chunk, loss_per_token=True,
               teacher_logprobs=logprobs)
    b = kd.bwd(*args, f["saved_logz"], tau=tau, ignore=inp["ignore"], chunk=chunk,
               teacher_logprobs=logprobs)
    torch.cuda.synchronize()
    for res in (fb, f):
        assert abs(float(res["loss"]) - ref["loss"]) <= tol["loss"] * abs(ref["loss"])
        assert rel_max(to64(res["loss_per_token"]), ref["loss_per_token"]) <= tol["loss"]
    for res in (fb, b):
        assert rel_max(to64(res["grad_hidden"]), ref["grad_hidden"]) <= tol["grad"]
        assert rel_max(to64(res["grad_W"]), ref["grad_W"]) <= tol["grad"]
