"""Seeded synthetic inputs for the fused top-K KL distillation loss.

This module only draws random tensors with fixed seeds and shapes; it holds
none of the loss arithmetic. Both the HIP path (through its binding) and the
fp64 oracle are fed from the same tensors drawn here: the oracle always reads
back the exact device tensors (bf16 -> fp64 is exact).

The paper's loss-only benchmark (§4.3 and Appendix B) uses deterministic
synthetic hidden states, output-projection weights and top-100 teacher targets
but names no distributions; the recipe below stands in for it:

  hidden ~ N(0, 1), W ~ N(0, 0.02) (second argument = standard deviation),
  per token K distinct uniform vocabulary indices, teacher logits = K draws
  of N(0, 3) sorted descending (the library renormalises them over K).

Seeds derive from the paper's training seed 1234 (Appendix A, Table 3).
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import torch

SEED_HIDDEN = 1234
SEED_W = 1235
SEED_TEACHER = 1236
SEED_MASK = 1237
SEED_ROWS = 1238
SEED_SUBBATCH = 1239


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    N: int
    D: int
    V: int
    K: int
    chunk: int
    tau: float
    dtype: str          # "f32" or "bf16"
    mask: str = "none"  # "none" or "packed5" (5% ignored, packed documents)

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


WORKLOADS = {
    "tiny_fp32": Workload("tiny_fp32", 256, 256, 4096, 16, 64, 1.0, "f32"),
    "loss4k": Workload("loss4k", 4096, 4096, 131072, 100, 4096, 1.0, "bf16"),
    "loss32k": Workload("loss32k", 32768, 4096, 131072, 100, 4096, 1.0, "bf16"),
    "packed": Workload("packed", 32768, 3072, 128256, 100, 2048, 2.0, "bf16",
                       mask="packed5"),
    "long256k": Workload("long256k", 262144, 4096, 131072, 100, 4096, 1.0, "bf16"),
}


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def make_hidden(N: int, D: int, dtype, device, seed: int = SEED_HIDDEN,
                std: float = 1.0) -> torch.Tensor:
    g = _gen(seed, device)
    x = torch.empty(N, D, dtype=torch.float32, device=device)
    for s in range(0, N, 16384):        # bounded fp32 temporaries
        e = min(N, s + 16384)
        x[s:e] = torch.randn(e - s, D, generator=g, device=device) * std
    return x.to(dtype)


def make_weight(V: int, D: int, dtype, device, seed: int = SEED_W,
                std: float = 0.02) -> torch.Tensor:
    return make_hidden(V, D, dtype, device, seed=seed, std=std)


def distinct_indices(N: int, K: int, V: int, g: torch.Generator, device) -> torch.Tensor:
    """[N, K] int32, each row K distinct uniform draws from [0, V) in random order."""
    if K > V:
        raise ValueError("K > V")
    if 2 * K > V:                      # dense regime: a random permutation prefix
        keys = torch.rand(N, V, generator=g, device=device)
        return keys.argsort(dim=1)[:, :K].to(torch.int32).contiguous()
    idx = torch.randint(0, V, (N, K), generator=g, device=device, dtype=torch.int64)
    while True:
        idx, _ = idx.sort(dim=1)
        dup = torch.zeros_like(idx, dtype=torch.bool)
        dup[:, 1:] = idx[:, 1:] == idx[:, :-1]
        n = int(dup.sum())
        if n == 0:
            break
        idx[dup] = torch.randint(0, V, (n,), generator=g, device=device, dtype=torch.int64)
    order = torch.rand(N, K, generator=g, device=device).argsort(dim=1)
    return idx.gather(1, order).to(torch.int32).contiguous()


def make_teacher(N: int, K: int, V: int, device, seed: int = SEED_TEACHER,
                 logit_std: float = 3.0):
    """(teacher_idx [N,K] int32, teacher_logit [N,K] fp32 sorted descending)."""
    g = _gen(seed, device)
    idx = distinct_indices(N, K, V, g, device)
    logit = torch.randn(N, K, generator=g, device=device) * logit_std
    logit, _ = logit.sort(dim=1, descending=True)
    return idx, logit.contiguous()


def make_packed_mask(N: int, device, seed: int = SEED_MASK, frac: float = 0.05):
    """Packed-documents structure: document lengths ~ U[512, 8192] concatenated
    and truncated to N (recorded only), and exactly floor(frac*N) positions,
    uniform without replacement, marked ignore (uint8, 1 = excluded)."""
    g = _gen(seed, "cpu")
    lengths = []
    total = 0
    while total < N:
        L = int(torch.randint(512, 8193, (1,), generator=g))
        L = min(L, N - total)
        lengths.append(L)
        total += L
    n_ign = int(frac * N)
    pos = torch.randperm(N, generator=g)[:n_ign]
    ignore = torch.zeros(N, dtype=torch.uint8)
    ignore[pos] = 1
    return ignore.to(device), lengths


def make_workload_inputs(w: Workload, device, N: Optional[int] = None):
    """All inputs of a workload on `device`. N overrides the token count (same
    generators, so rows are a prefix of the full workload's rows)."""
    n = w.N if N is None else N
    hidden = make_hidden(n, w.D, w.torch_dtype, device)
    W = make_weight(w.V, w.D, w.torch_dtype, device)
    idx, logit = make_teacher(n, w.K, w.V, device)
    ignore, lengths = (None, None)
    if w.mask == "packed5":
        ignore, lengths = make_packed_mask(n, device)
    return dict(hidden=hidden, W=W, teacher_idx=idx, teacher_logit=logit,
                ignore=ignore, doc_lengths=lengths, tau=w.tau, chunk=w.chunk)


def sample_rows(n_valid_rows: torch.Tensor, count: int = 64, seed: int = SEED_ROWS):
    """`count` row indices drawn uniformly without replacement from the given
    candidate rows (a 1-D CPU int tensor)."""
    g = _gen(seed, "cpu")
    perm = torch.randperm(n_valid_rows.numel(), generator=g)[:count]
    return n_valid_rows[perm].sort().values


def sub_batch(N: int, count: int = 512, seed: int = SEED_SUBBATCH):
    g = _gen(seed, "cpu")
    return torch.randperm(N, generator=g)[:count].sort().values
