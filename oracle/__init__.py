"""fp64 CPU oracle (test infrastructure only; see kd_oracle's header)."""
from .kd_oracle import kd_topk_kl, teacher_distribution, log_softmax_rows

__all__ = ["kd_topk_kl", "teacher_distribution", "log_softmax_rows"]
