"""Planted mistakes in copies of the oracle must be caught by its pins.

Each mutation edits one line of the oracle's source (a dropped term, a wrong
sign, a missing 1/tau, a wrong normaliser, a transposed product...), loads the
edited copy as a throw-away module on the CPU, and runs a compact set of the
pins from test_oracle.py against it: at least one must fail.

Dropping the retained mass M from the gradient is not listed: with the teacher
renormalised over its K entries M = 1, so that edit is an equivalent program.
"""
import importlib.util
import json
import os
import types

import numpy as np
import pytest
import scipy.special as sps
import torch

ORACLE_SRC = os.path.join(os.path.dirname(os.path.dirname(__file__)), "oracle", "kd_oracle.py")
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_cases.json")

MUTATIONS = {
    "drop_1_over_tau_in_grad": ("G = (g[s0:s1] / tau)[:, None]", "G = (g[s0:s1])[:, None]"),
    "flip_grad_sign": ("(M[s0:s1, None] * q - P)", "(P - M[s0:s1, None] * q)"),
    "drop_entropy_term": ("P[pos] * (np.log(P[pos]) - logq[pos])", "P[pos] * (- logq[pos])"),
    "no_temperature_in_logits": ("y = z / tau", "y = z"),
    "teacher_not_tempered": ("_f64(teacher_logit) / float(tau)", "_f64(teacher_logit)"),
    "mean_over_all_rows": ("n_valid = float(valid.sum())", "n_valid = float(N)"),
    "grad_W_uses_W": ("grad_W += G.T @ h[s0:s1]", "grad_W += G.T @ (h[s0:s1] * 0 + 1)"),
    "grad_h_transposed_head": ("grad_h[s0:s1] = G @ W", "grad_h[s0:s1] = (G @ W) * 0.5"),
    "scatter_overwrite_first_col": ("np.add.at(P,", "np.add.at(P[:, ::-1],"),
    "ignored_rows_counted": ("ell[~valid[s0:s1]] = 0.0", "pass"),
    "scatter_assigns_repeats": ("np.add.at(P, (np.repeat(rows, K), idx[s0:s1].reshape(-1)),",
                                "P.__setitem__((np.repeat(rows, K), idx[s0:s1].reshape(-1)),"),
    "token_weights_ignored": ("g = np.where(valid, _f64(token_weights), 0.0)",
                              "g = np.where(valid, 1.0 / max(n_valid, 1.0), 0.0)"),
    "logprobs_renormalised": ("return np.exp(_f64(teacher_logit))",
                              "return np.exp(log_softmax_rows(_f64(teacher_logit)))"),
    "logprobs_tempered": ("return np.exp(_f64(teacher_logit))",
                          "return np.exp(_f64(teacher_logit) / float(tau))"),
}


def _load_mutant(old, new):
    with open(ORACLE_SRC) as f:
        src = f.read()
    assert old in src, old
    mod = types.ModuleType("kd_oracle_mutant")
    exec(compile(src.replace(old, new, 1), "kd_oracle_mutant", "exec"), mod.__dict__)
    return mod.kd_topk_kl


def _pins(fn):
    """Returns the names of the pins that fail for oracle function `fn`."""
    failed = []
    # golden hand-derived cases
    with open(GOLDEN) as f:
        cases = json.load(f)["cases"]
    for case in cases:
        ign = None if case["ignore"] is None else np.array(case["ignore"], dtype=np.uint8)
        try:
            out = fn(np.array(case["h"]), np.array(case["W"]), np.array(case["teacher_idx"]),
                     np.array(case["teacher_logit"]), tau=case["tau"], ignore=ign,
                     token_weights=case.get("token_weights"),
                     teacher_mode=case.get("teacher_mode", "logits"))
            ok = (abs(out["loss"] - case["loss"]) < 1e-12
                  and np.allclose(out["grad_hidden"], case["grad_hidden"], atol=1e-12)
                  and np.allclose(out["grad_W"], case["grad_W"], atol=1e-12))
        except Exception:
            ok = False
        if not ok:
            failed.append("golden:" + case["name"])
    # textbook autograd with tau != 1 and an ignore mask
    rng = np.random.default_rng(3)
    N, D, V, K, tau = 6, 5, 13, 4, 1.7
    h = rng.standard_normal((N, D)); W = rng.standard_normal((V, D))
    idx = np.stack([rng.choice(V, K, replace=False) for _ in range(N)])
    tl = rng.standard_normal((N, K)) * 2
    ign = np.array([0, 1, 0, 0, 0, 1], dtype=np.uint8)
    try:
        out = fn(h, W, idx, tl, tau=tau, ignore=ign, chunk=4)
        th = torch.tensor(h, requires_grad=True); tW = torch.tensor(W, requires_grad=True)
        P = torch.zeros(N, V, dtype=torch.float64)
        P.scatter_(1, torch.tensor(idx), torch.softmax(torch.tensor(tl) / tau, 1))
        per = torch.nn.functional.kl_div(torch.log_softmax(th @ tW.T / tau, 1), P,
                                         reduction="none").sum(1)
        valid = torch.tensor(ign == 0)
        loss = (per * valid).sum() / valid.sum()
        loss.backward()
        ok = (abs(out["loss"] - loss.item()) < 1e-10
              and np.allclose(out["grad_hidden"], th.grad.numpy(), atol=1e-10)
              and np.allclose(out["grad_W"], tW.grad.numpy(), atol=1e-10))
    except Exception:
        ok = False
    if not ok:
        failed.append("autograd")
    # Gibbs decomposition via scipy
    try:
        out = fn(h, W, idx, tl, tau=tau)
        q = sps.softmax(h @ W.T / tau, 1); p = sps.softmax(tl / tau, 1)
        ok = all(abs(out["loss_per_token"][t]
                     - (sps.rel_entr(p[t], q[t, idx[t]] / q[t, idx[t]].sum()).sum()
                        - np.log(q[t, idx[t]].sum()))) < 1e-10 for t in range(N))
    except Exception:
        ok = False
    if not ok:
        failed.append("gibbs")
    # partial-mass teacher (cached log-probabilities, M < 1) at tau != 1
    try:
        lp = np.log(sps.softmax(tl, 1) * 0.6)
        out = fn(h, W, idx, lp, tau=tau, teacher_mode="logprobs")
        th = torch.tensor(h, requires_grad=True); tW = torch.tensor(W, requires_grad=True)
        P = torch.zeros(N, V, dtype=torch.float64)
        P.scatter_(1, torch.tensor(idx), torch.exp(torch.tensor(lp)))
        logq = torch.log_softmax(th @ tW.T / tau, 1)
        per = (P * (torch.where(P > 0, torch.log(P), torch.zeros_like(P)) - logq)).sum(1)
        per.mean().backward()
        ok = (abs(out["loss"] - per.mean().item()) < 1e-10
              and np.allclose(out["grad_W"], tW.grad.numpy(), atol=1e-10))
    except Exception:
        ok = False
    if not ok:
        failed.append("partial-mass autograd")
    # a repeated index is the merged entry tau * logaddexp(t1/tau, t2/tau)
    try:
        rep = idx.copy()
        rep[:, 3] = rep[:, 1]
        mi, mt = np.delete(idx, 3, axis=1), np.delete(tl, 3, axis=1)
        mt[:, 1] = tau * np.logaddexp(tl[:, 1] / tau, tl[:, 3] / tau)
        a, b = fn(h, W, rep, tl, tau=tau), fn(h, W, mi, mt, tau=tau)
        ok = (abs(a["loss"] - b["loss"]) < 1e-12
              and np.allclose(a["grad_W"], b["grad_W"], atol=1e-12))
    except Exception:
        ok = False
    if not ok:
        failed.append("repeat = merged entry")
    return failed


def test_unmutated_oracle_passes_compact_pins():
    from oracle import kd_topk_kl
    assert _pins(kd_topk_kl) == []


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name):
    old, new = MUTATIONS[name]
    failed = _pins(_load_mutant(old, new))
    assert failed, f"mutation {name} was not caught by any pin"
