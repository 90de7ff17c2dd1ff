"""GPU parity of the split forward/backward entry points (Algorithm 1's own
structure), the upstream gradients they take, the autograd wrapper built on
them, and the partial-mass teacher mode, all against the fp64 oracle on the
same seeded inputs."""
import numpy as np
import pytest
import torch

import kd_inputs as ki
from oracle import kd_topk_kl
from tests.helpers import TOL, oracle_inputs, rel_max, to64

pytestmark = pytest.mark.gpu

SHAPES = [  # N, D, V, K, chunk, tau, ignore fraction
    (259, 128, 4133, 7, 100, 2.0, 0.2),
    (513, 192, 1000, 16, 513, 1.0, 0.0),
]


def _inputs(N, D, V, K, dtype, seed=0, ignore_frac=0.0):
    dev = "cuda"
    hidden = ki.make_hidden(N, D, dtype, dev, seed=ki.SEED_HIDDEN + seed)
    W = ki.make_weight(V, D, dtype, dev, seed=ki.SEED_W + seed)
    idx, logit = ki.make_teacher(N, K, V, dev, seed=ki.SEED_TEACHER + seed)
    ignore = None
    if ignore_frac > 0:
        g = torch.Generator(device="cpu")
        g.manual_seed(ki.SEED_MASK + seed)
        ignore = (torch.rand(N, generator=g) < ignore_frac).to(torch.uint8).to(dev)
    return dict(hidden=hidden, W=W, teacher_idx=idx, teacher_logit=logit, ignore=ignore)


def _logprob_teacher(inp, seed):
    """Partial-mass cache: the K entries keep a per-row mass in [0.3, 0.95]."""
    tl = inp["teacher_logit"]
    g = torch.Generator(device="cpu")
    g.manual_seed(ki.SEED_TEACHER + 100 + seed)
    mass = (0.3 + 0.65 * torch.rand(tl.shape[0], generator=g)).to(tl.device)
    return (torch.log_softmax(tl, dim=1) + torch.log(mass)[:, None]).contiguous()


def _args(inp):
    return (inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("N,D,V,K,chunk,tau,ign", SHAPES)
def test_forward_matches_fused_and_oracle(gpu_lib, dtype, N, D, V, K, chunk, tau, ign):
    kd = gpu_lib
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    inp = _inputs(N, D, V, K, tdt, seed=N + 1, ignore_frac=ign)
    f = kd.fwd(*_args(inp), tau=tau, ignore=inp["ignore"], chunk=chunk, loss_per_token=True)
    fb = kd.fwd_bwd(*_args(inp), tau=tau, ignore=inp["ignore"], chunk=chunk, loss_per_token=True,
                    grad_hidden=False, grad_W=False)
    torch.cuda.synchronize()
    # the same kernels compute the loss in both entry points
    assert torch.equal(f["loss"], fb["loss"])
    assert torch.equal(f["loss_per_token"], fb["loss_per_token"])
    ref = kd_topk_kl(**oracle_inputs(inp), tau=tau, chunk=chunk, want_grads=False)
    tol = TOL[dtype]
    assert abs(float(f["loss"]) - ref["loss"]) <= tol["loss"] * abs(ref["loss"])
    # log Z from fp32 accumulation of the same inputs: absolute error ~1e-6 |log Z|;
    # ignored tokens are left out (0)
    lz = to64(f["saved_logz"])
    keep = np.ones(N, bool) if inp["ignore"] is None else to64(inp["ignore"]) == 0
    assert np.all(lz[~keep] == 0.0)
    assert np.abs(lz[keep] - ref["logZ"][keep]).max() <= 1e-5 * np.abs(ref["logZ"]).max()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("N,D,V,K,chunk,tau,ign", SHAPES)
def test_backward_matches_oracle(gpu_lib, dtype, N, D, V, K, chunk, tau, ign):
    kd = gpu_lib
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    inp = _inputs(N, D, V, K, tdt, seed=N + 2, ignore_frac=ign)
    f = kd.fwd(*_args(inp), tau=tau, ignore=inp["ignore"], chunk=chunk)
    b = kd.bwd(*_args(inp), f["saved_logz"], tau=tau, ignore=inp["ignore"], chunk=chunk)
    torch.cuda.synchronize()
    ref = kd_topk_kl(**oracle_inputs(inp), tau=tau, chunk=chunk)
    tol = TOL[dtype]
    assert rel_max(to64(b["grad_hidden"]), ref["grad_hidden"]) <= tol["grad"]
    assert rel_max(to64(b["grad_W"]), ref["grad_W"]) <= tol["grad"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("N,D,V,K,chunk,tau,ign", SHAPES + [(600, 128, 777, 5, 128, 0.5, 0.1)])
def test_fused_schedule_matches_split(gpu_lib, dtype, N, D, V, K, chunk, tau, ign):
    """The fused call projects each chunk once and stores dZ up to a factor per
    row (applied to the rows of dH and to the hidden rows for dW); the split
    entry points recompute the logits (Algorithm 1). Same loss up to the order
    of the normaliser's fp32 sums; gradients within one more bf16 rounding
    (2^-8 relative), or within the fp32 gradient tolerance."""
    kd = gpu_lib
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    inp = _inputs(N, D, V, K, tdt, seed=N + 5, ignore_frac=ign)
    fb = kd.fwd_bwd(*_args(inp), tau=tau, ignore=inp["ignore"], chunk=chunk, loss_per_token=True)
    f = kd.fwd(*_args(inp), tau=tau, ignore=inp["ignore"], chunk=chunk, loss_per_token=True)
    b = kd.bwd(*_args(inp), f["saved_logz"], tau=tau, ignore=inp["ignore"], chunk=chunk)
    torch.cuda.synchronize()
    assert abs(float(fb["loss"]) - float(f["loss"])) <= 1e-6 * abs(float(f["loss"]))
    assert rel_max(to64(fb["loss_per_token"]), to64(f["loss_per_token"])) <= 1e-6
    gt = TOL["f32"]["grad"] if dtype == "f32" else 2.0 ** -7
    assert rel_max(to64(fb["grad_hidden"]), to64(b["grad_hidden"])) <= gt
    assert rel_max(to64(fb["grad_W"]), to64(b["grad_W"])) <= gt


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_upstream_scalar_and_per_token(gpu_lib, dtype):
    kd = gpu_lib
    N, D, V, K, chunk, tau = 259, 128, 4133, 7, 100, 2.0
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    inp = _inputs(N, D, V, K, tdt, seed=3, ignore_frac=0.2)
    f = kd.fwd(*_args(inp), tau=tau, ignore=inp["ignore"], chunk=chunk)
    tol = TOL[dtype]
    o = oracle_inputs(inp)
    valid = (o["ignore"] == 0)
    # scalar upstream gradient of the mean
    gl = torch.tensor(-2.5, dtype=torch.float32, device="cuda")
    b = kd.bwd(*_args(inp), f["saved_logz"], tau=tau, ignore=inp["ignore"], chunk=chunk, grad_loss=gl)
    ref = kd_topk_kl(**o, tau=tau, chunk=chunk,
                     token_weights=np.full(N, -2.5 / valid.sum()))
    assert rel_max(to64(b["grad_hidden"]), ref["grad_hidden"]) <= tol["grad"]
    assert rel_max(to64(b["grad_W"]), ref["grad_W"]) <= tol["grad"]
    # per-token upstream gradients (ignored rows get none)
    g = torch.Generator(device="cpu")
    g.manual_seed(4242)
    u = (torch.rand(N, generator=g) * 3.0 - 1.0).to("cuda")
    b = kd.bwd(*_args(inp), f["saved_logz"], tau=tau, ignore=inp["ignore"], chunk=chunk,
               grad_loss_per_token=u)
    torch.cuda.synchronize()
    ref = kd_topk_kl(**o, tau=tau, chunk=chunk, token_weights=to64(u))
    assert rel_max(to64(b["grad_hidden"]), ref["grad_hidden"]) <= tol["grad"]
    assert rel_max(to64(b["grad_W"]), ref["grad_W"]) <= tol["grad"]
    assert torch.all(b["grad_hidden"][inp["ignore"].bool()] == 0)


def test_backward_accumulates_grad_W(gpu_lib):
    kd = gpu_lib
    inp = _inputs(300, 64, 777, 5, torch.float32, seed=9)
    f = kd.fwd(*_args(inp), tau=1.0, chunk=64)
    one = kd.bwd(*_args(inp), f["saved_logz"], tau=1.0, chunk=64, grad_hidden=False)["grad_W"]
    acc = one.clone()
    kd.bwd(*_args(inp), f["saved_logz"], tau=1.0, chunk=64, grad_hidden=False, grad_W_out=acc,
           accumulate_grad_W=True)
    torch.cuda.synchronize()
    assert torch.allclose(acc, 2 * one, rtol=1e-6, atol=1e-12)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("schedule", ["fused", "recompute"])
def test_autograd_wrapper(gpu_lib, dtype, schedule):
    kd = gpu_lib
    N, D, V, K, chunk, tau = 259, 128, 4133, 7, 100, 2.0
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    inp = _inputs(N, D, V, K, tdt, seed=11, ignore_frac=0.2)
    h = inp["hidden"].clone().requires_grad_(True)
    W = inp["W"].clone().requires_grad_(True)
    loss = kd.topk_kl_loss(h, W, inp["teacher_idx"], inp["teacher_logit"], tau=tau,
                           ignore=inp["ignore"], chunk=chunk, schedule=schedule)
    (3.0 * loss).backward()
    torch.cuda.synchronize()
    o = oracle_inputs(inp)
    valid = (o["ignore"] == 0)
    ref = kd_topk_kl(**o, tau=tau, chunk=chunk, token_weights=np.full(N, 3.0 / valid.sum()))
    tol = TOL[dtype]
    assert abs(float(loss.detach()) - ref["loss"]) <= tol["loss"] * abs(ref["loss"])
    assert h.grad.dtype == tdt and W.grad.dtype == tdt
    assert rel_max(to64(h.grad), ref["grad_hidden"]) <= tol["grad"]
    # grad_W comes back in W's dtype: bf16 rounding of an fp32 result
    assert rel_max(to64(W.grad), ref["grad_W"]) <= tol["grad"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("tau", [1.0, 2.0])
def test_partial_mass_teacher(gpu_lib, dtype, tau):
    """Cached log-probabilities (retained mass M < 1, §3.2): fused and split
    entry points against the oracle's partial-mass mode."""
    kd = gpu_lib
    N, D, V, K, chunk = 259, 128, 4133, 7, 100
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    inp = _inputs(N, D, V, K, tdt, seed=17, ignore_frac=0.1)
    inp["teacher_logit"] = _logprob_teacher(inp, 17)
    tol = TOL[dtype]
    ref = kd_topk_kl(**oracle_inputs(inp), tau=tau, chunk=chunk, teacher_mode="logprobs")
    fb = kd.fwd_bwd(*_args(inp), tau=tau, ignore=inp["ignore"], chunk=chunk, loss_per_token=True,
                    teacher_logprobs=True)
    f = kd.fwd(*_args(inp), tau=tau, ignore=inp["ignore"], chunk=chunk, teacher_logprobs=True)
    b = kd.bwd(*_args(inp), f["saved_logz"], tau=tau, ignore=inp["ignore"], chunk=chunk,
               teacher_logprobs=True)
    torch.cuda.synchronize()
    for loss in (fb["loss"], f["loss"]):
        assert abs(float(loss.detach()) - ref["loss"]) <= tol["loss"] * abs(ref["loss"])
    assert rel_max(to64(fb["loss_per_token"]), ref["loss_per_token"]) <= tol["loss"]
    for res in (fb, b):
        assert rel_max(to64(res["grad_hidden"]), ref["grad_hidden"]) <= tol["grad"]
        assert rel_max(to64(res["grad_W"]), ref["grad_W"]) <= tol["grad"]
    # Gibbs bound of the partial-mass loss, per token: l >= M log M
    M = ref["M"]
    lpt = to64(fb["loss_per_token"])
    valid = to64(inp["ignore"]) == 0
    assert np.all(lpt[valid] >= (M * np.log(M))[valid] - 1e-4)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_forward_teacher_crowding_one_vocab_tile(gpu_lib, dtype):
    """Every token's K = 128 entries lie in the same 256-column vocabulary tile,
    so the first 256-token tile has 32768 teacher cells in one output tile: more than
    the forward-only kernel numbers in LDS (28656), so some cells take the
    bucket-search path. The loss must match the fused entry point bit for bit
    and the oracle within tolerance."""
    kd = gpu_lib
    N, D, V, K, chunk, tau = 300, 64, 1100, 128, 300, 1.5
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    inp = _inputs(N, D, V, K, tdt, seed=21)
    g = torch.Generator(device="cpu")
    g.manual_seed(ki.SEED_TEACHER + 21)
    tile = torch.full((N,), 2)   # columns [512, 768), a full tile
    perm = torch.argsort(torch.rand(N, 256, generator=g), dim=1)[:, :K]
    inp["teacher_idx"] = (tile[:, None] * 256 + perm).to(torch.int32).to("cuda").contiguous()
    f = kd.fwd(*_args(inp), tau=tau, chunk=chunk, loss_per_token=True)
    fb = kd.fwd_bwd(*_args(inp), tau=tau, chunk=chunk, loss_per_token=True, grad_hidden=False,
                    grad_W=False)
    torch.cuda.synchronize()
    assert torch.equal(f["loss_per_token"], fb["loss_per_token"])
    ref = kd_topk_kl(**oracle_inputs(inp), tau=tau, chunk=chunk, want_grads=False)
    assert abs(float(f["loss"]) - ref["loss"]) <= TOL[dtype]["loss"] * abs(ref["loss"])


def test_autograd_fused_schedule_cases(gpu_lib):
    """The fused autograd schedule: a frozen W gets no gradient work and the
    same hidden gradient; under no_grad only the loss is computed; a second
    backward through the same graph is refused (the gradients are consumed);
    the recompute schedule agrees."""
    kd = gpu_lib
    N, D, V, K, chunk = 200, 64, 1500, 6, 64
    inp = _inputs(N, D, V, K, torch.float32, seed=12, ignore_frac=0.1)
    idx, tl, ign = inp["teacher_idx"], inp["teacher_logit"], inp["ignore"]
    h1 = inp["hidden"].clone().requires_grad_(True)
    kd.profile_read()
    kd.profile_enable(True)
    l1 = kd.topk_kl_loss(h1, inp["W"], idx, tl, ignore=ign, chunk=chunk)
    (0.5 * l1).backward()
    torch.cuda.synchronize()
    kd.profile_enable(False)
    ran = kd.profile_read()
    # W is frozen: the call ran the projection and dH, and no grad_W work
    assert "logits_dz" in ran and "dh" in ran
    assert "dw" not in ran and "transpose_rows" not in ran, ran
    h2 = inp["hidden"].clone().requires_grad_(True)
    l2 = kd.topk_kl_loss(h2, inp["W"], idx, tl, ignore=ign, chunk=chunk, schedule="recompute")
    (0.5 * l2).backward()
    torch.cuda.synchronize()
    assert abs(float(l1.detach()) - float(l2.detach())) <= 1e-6 * abs(float(l2.detach()))
    assert rel_max(to64(h1.grad), to64(h2.grad)) <= 1e-5
    kd.profile_enable(True)
    with torch.no_grad():
        l3 = kd.topk_kl_loss(inp["hidden"], inp["W"], idx, tl, ignore=ign, chunk=chunk)
    torch.cuda.synchronize()
    kd.profile_enable(False)
    ran = kd.profile_read()
    # no graph: the forward alone, no gradient contraction
    assert "logits_lse" in ran
    assert not ({"logits_dz", "dz", "dh", "dw", "transpose_rows"} & set(ran)), ran
    assert l3.grad_fn is None
    assert abs(float(l3) - float(l1.detach())) <= 1e-6 * abs(float(l1.detach()))
    h4 = inp["hidden"].clone().requires_grad_(True)
    ws = kd.alloc_workspace(N, D, V, K, chunk, 1.0, kd.KD_F32, h4.device)
    l4 = kd.topk_kl_loss(h4, inp["W"], idx, tl, ignore=ign, chunk=chunk, workspace=ws)
    l4.backward(retain_graph=True)
    torch.cuda.synchronize()
    assert rel_max(to64(h4.grad), to64(2.0 * h1.grad)) <= 1e-5
    with pytest.raises(RuntimeError):
        l4.backward()


@pytest.mark.parametrize("n", [1, 7, 8, 4097, 100003])
def test_scale_grads(gpu_lib, n):
    """kd_scale_grads: out = g * in from fp32 gradients, fp32 output exact (one
    fp32 multiply, in place too) and bf16 output rounded once to nearest even
    (compared with torch's own fp32 -> bf16 conversion of the fp32 product),
    on sizes with ragged tails of the 8-element vectors."""
    kd = gpu_lib
    g = torch.Generator(device="cpu")
    g.manual_seed(ki.SEED_TEACHER + n)
    x = (torch.randn(n, generator=g) * 1e-3).to("cuda")
    x2 = (torch.randn(n, generator=g) * 1e-6).to("cuda")
    gl = torch.tensor([-2.7182817], dtype=torch.float32, device="cuda")
    ref = (x.cpu() * gl.cpu()).contiguous()
    ref2 = (x2.cpu() * gl.cpu()).contiguous()
    out_bf = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    inplace = x2.clone()
    kd.scale_grads(gl, grad_hidden=x, grad_hidden_out=out_bf, grad_W=inplace,
                   grad_W_out=inplace)
    torch.cuda.synchronize()
    assert torch.equal(inplace.cpu(), ref2)
    assert torch.equal(out_bf.cpu(), ref.to(torch.bfloat16))
    # fp32 into a separate buffer, bf16 from the W slot
    out32 = torch.empty(n, dtype=torch.float32, device="cuda")
    out_bf2 = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    kd.scale_grads(gl, grad_hidden=x, grad_hidden_out=out32, grad_W=x2, grad_W_out=out_bf2)
    torch.cuda.synchronize()
    assert torch.equal(out32.cpu(), ref)
    assert torch.equal(out_bf2.cpu(), ref2.to(torch.bfloat16))


@pytest.mark.parametrize("chunk", [100, 300])
def test_grad_hidden_f32_flag(gpu_lib, chunk):
    """KD_FLAG_GRAD_HIDDEN_F32 (fused call and split backward): grad_hidden in
    fp32, whose single rounding to bf16 is bitwise the bf16 grad_hidden of the
    same call without the flag; the fp32 values match the oracle. chunk 100
    runs dH with a split vocabulary range (fp32 partials reduced), 300 without."""
    kd = gpu_lib
    N, D, V, K, tau = 600, 128, 4133, 7, 1.3
    inp = _inputs(N, D, V, K, torch.bfloat16, seed=44, ignore_frac=0.1)
    a = (inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"])
    fb16 = kd.fwd_bwd(*a, tau=tau, ignore=inp["ignore"], chunk=chunk, grad_W=False)
    fb32 = kd.fwd_bwd(*a, tau=tau, ignore=inp["ignore"], chunk=chunk, grad_W=False,
                      grad_hidden_f32=True)
    f = kd.fwd(*a, tau=tau, ignore=inp["ignore"], chunk=chunk)
    b16 = kd.bwd(*a, f["saved_logz"], tau=tau, ignore=inp["ignore"], chunk=chunk, grad_W=False)
    b32 = kd.bwd(*a, f["saved_logz"], tau=tau, ignore=inp["ignore"], chunk=chunk, grad_W=False,
                 grad_hidden_f32=True)
    torch.cuda.synchronize()
    assert fb32["grad_hidden"].dtype == torch.float32 and b32["grad_hidden"].dtype == torch.float32
    assert torch.equal(fb32["grad_hidden"].to(torch.bfloat16), fb16["grad_hidden"])
    assert torch.equal(b32["grad_hidden"].to(torch.bfloat16), b16["grad_hidden"])
    ref = kd_topk_kl(**oracle_inputs(inp), tau=tau, chunk=chunk)
    for res in (fb32, b32):
        assert rel_max(to64(res["grad_hidden"]), ref["grad_hidden"]) <= TOL["bf16"]["grad"]
