"""Pins for the oracle's two extensions, each against something other than the
oracle itself:

* per-token weights g_t of the token losses (the upstream gradient that
  Algorithm 1's backward receives): torch float64 autograd of sum_t g_t l_t;
* the partial-mass teacher of §3.2 (cached log-probabilities, retained mass
  M <= 1, no renormalisation): the Gibbs bound l >= M log M, the exact mass
  scaling identity l(c p) = c l(p) + c M log c, reduction to the renormalised
  mode when M = 1, and torch autograd of the dense Eq. (1) objective.
"""
import numpy as np
import pytest
import torch

from oracle import kd_topk_kl, teacher_distribution


def _case(N=7, D=5, V=17, K=4, seed=11, wscale=0.8):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((N, D))
    W = rng.standard_normal((V, D)) * wscale
    idx = np.stack([rng.choice(V, size=K, replace=False) for _ in range(N)])
    tl = np.sort(rng.standard_normal((N, K)) * 3.0, axis=1)[:, ::-1].copy()
    return h, W, idx, tl


def _partial_logprobs(tl, mass, seed=0):
    """Log-probabilities of a teacher whose K cached entries keep `mass` (per row)."""
    p = np.exp(tl - tl.max(axis=1, keepdims=True))
    p = p / p.sum(axis=1, keepdims=True) * np.asarray(mass)[:, None]
    return np.log(p)


@pytest.mark.parametrize("tau", [1.0, 1.7])
def test_token_weights_match_autograd(tau):
    h, W, idx, tl = _case()
    rng = np.random.default_rng(3)
    w = rng.uniform(-1.0, 2.0, size=h.shape[0])
    ign = np.zeros(h.shape[0], dtype=np.uint8)
    ign[2] = 1
    out = kd_topk_kl(h, W, idx, tl, tau=tau, ignore=ign, chunk=3, token_weights=w)
    th = torch.tensor(h, requires_grad=True)
    tW = torch.tensor(W, requires_grad=True)
    P = torch.zeros(h.shape[0], W.shape[0], dtype=torch.float64)
    P.scatter_(1, torch.tensor(idx), torch.softmax(torch.tensor(tl) / tau, dim=1))
    logq = torch.log_softmax(th @ tW.T / tau, dim=1)
    per = torch.nn.functional.kl_div(logq, P, reduction="none").sum(dim=1)
    obj = (per * torch.tensor(np.where(ign == 0, w, 0.0))).sum()
    obj.backward()
    np.testing.assert_allclose(out["grad_hidden"], th.grad.numpy(), rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(out["grad_W"], tW.grad.numpy(), rtol=1e-10, atol=1e-13)
    # the reported loss is still the mean over valid rows
    assert out["loss"] == pytest.approx(out["loss_per_token"][ign == 0].mean(), rel=1e-13)


def test_mean_weights_reproduce_default():
    h, W, idx, tl = _case(seed=5)
    a = kd_topk_kl(h, W, idx, tl, tau=1.3)
    b = kd_topk_kl(h, W, idx, tl, tau=1.3, token_weights=np.full(h.shape[0], 1.0 / h.shape[0]))
    np.testing.assert_allclose(a["grad_hidden"], b["grad_hidden"], rtol=1e-14, atol=1e-16)
    np.testing.assert_allclose(a["grad_W"], b["grad_W"], rtol=1e-14, atol=1e-16)


def test_partial_mass_gibbs_bound():
    h, W, idx, tl = _case(N=40, seed=8)
    mass = np.random.default_rng(2).uniform(0.05, 1.0, size=h.shape[0])
    lp = _partial_logprobs(tl, mass)
    out = kd_topk_kl(h, W, idx, lp, teacher_mode="logprobs")
    np.testing.assert_allclose(out["M"], mass, rtol=1e-13)
    assert np.all(out["loss_per_token"] >= mass * np.log(mass) - 1e-12)


@pytest.mark.parametrize("c", [0.25, 0.6])
def test_partial_mass_scaling_identity(c):
    """Scaling the cached probabilities by c scales Eq. (1) exactly:
    sum c p (log c p - log q) = c l(p) + c M log c."""
    h, W, idx, tl = _case(seed=9)
    mass = np.random.default_rng(4).uniform(0.3, 0.9, size=h.shape[0])
    lp = _partial_logprobs(tl, mass)
    a = kd_topk_kl(h, W, idx, lp, teacher_mode="logprobs")
    b = kd_topk_kl(h, W, idx, lp + np.log(c), teacher_mode="logprobs")
    np.testing.assert_allclose(b["loss_per_token"],
                               c * a["loss_per_token"] + c * a["M"] * np.log(c), rtol=1e-11, atol=1e-13)


def test_partial_mass_one_equals_renormalised_mode():
    h, W, idx, tl = _case(seed=10)
    lp = np.log(teacher_distribution(tl, 1.0))
    a = kd_topk_kl(h, W, idx, tl, tau=1.0)
    b = kd_topk_kl(h, W, idx, lp, teacher_mode="logprobs")
    assert a["loss"] == pytest.approx(b["loss"], rel=1e-13)
    np.testing.assert_allclose(a["grad_W"], b["grad_W"], rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("tau", [1.0, 2.0])
def test_partial_mass_autograd(tau):
    """The student temperature still applies; the cached log-probabilities are
    used as they are."""
    h, W, idx, tl = _case(seed=12)
    mass = np.random.default_rng(6).uniform(0.2, 1.0, size=h.shape[0])
    lp = _partial_logprobs(tl, mass)
    out = kd_topk_kl(h, W, idx, lp, tau=tau, chunk=2, teacher_mode="logprobs")
    th = torch.tensor(h, requires_grad=True)
    tW = torch.tensor(W, requires_grad=True)
    P = torch.zeros(h.shape[0], W.shape[0], dtype=torch.float64)
    P.scatter_(1, torch.tensor(idx), torch.exp(torch.tensor(lp)))
    logq = torch.log_softmax(th @ tW.T / tau, dim=1)
    per = (P * (torch.where(P > 0, torch.log(P), torch.zeros_like(P)) - logq)).sum(dim=1)
    loss = per.mean()
    loss.backward()
    assert out["loss"] == pytest.approx(float(loss.detach()), rel=1e-12)
    np.testing.assert_allclose(out["grad_hidden"], th.grad.numpy(), rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(out["grad_W"], tW.grad.numpy(), rtol=1e-10, atol=1e-13)


@pytest.mark.parametrize("tau", [1.0, 0.7])
def test_repeated_index_equals_merged_entry(tau):
    """A row that lists a vocabulary entry twice, with teacher logits t1 and t2,
    is the row that lists it once with the logit tau * logaddexp(t1/tau, t2/tau)
    (its softmax weight is the sum of the two): loss, per-token loss and both
    gradients agree. Pins the oracle's reading of repeats (the dense teacher row
    sums them) against a construction that has no repeat."""
    rng = np.random.default_rng(5)
    N, D, V, K = 6, 8, 40, 5
    h = rng.standard_normal((N, D))
    W = rng.standard_normal((V, D)) * 0.3
    idx = np.stack([rng.choice(V, K, replace=False) for _ in range(N)])
    tl = rng.standard_normal((N, K)) * 2
    rep = idx.copy()
    rep[:, 3] = rep[:, 1]                           # entry 3 repeats entry 1's index
    merged_idx = np.delete(idx, 3, axis=1)
    merged_tl = np.delete(tl, 3, axis=1)
    merged_tl[:, 1] = tau * np.logaddexp(tl[:, 1] / tau, tl[:, 3] / tau)
    a = kd_topk_kl(h, W, rep, tl, tau=tau)
    b = kd_topk_kl(h, W, merged_idx, merged_tl, tau=tau)
    assert abs(a["loss"] - b["loss"]) < 1e-12
    np.testing.assert_allclose(a["loss_per_token"], b["loss_per_token"], atol=1e-12)
    np.testing.assert_allclose(a["grad_hidden"], b["grad_hidden"], atol=1e-12)
    np.testing.assert_allclose(a["grad_W"], b["grad_W"], atol=1e-12)
