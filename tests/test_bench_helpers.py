"""bench.py's bookkeeping of the committed counter summaries (CPU only): the
digest that ties a summary to the kernel sources ignores comments and layout
and sees code changes, and the stored traffic / MFMA counters are reported
only for the sources they were taken on."""
import os
import shutil

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_03796_amd", "csrc")


def _copy_csrc(tmp_path):
    d = tmp_path / "csrc"
    shutil.copytree(CSRC, d)
    return d


def test_digest_ignores_comments_and_layout(tmp_path):
    d = _copy_csrc(tmp_path)
    ref = bench.kernel_sources_sha256(str(d))
    assert ref == bench.kernel_sources_sha256(CSRC)
    f = d / "kd_kernels.hip"
    text = f.read_text()
    # a comment, a block comment and re-indented code: same digest
    f.write_text("// a note\n/* another\n note */\n" + text.replace("\n  ", "\n      ", 5))
    assert bench.kernel_sources_sha256(str(d)) == ref


def test_digest_sees_code_and_string_changes(tmp_path):
    d = _copy_csrc(tmp_path)
    ref = bench.kernel_sources_sha256(str(d))
    f = d / "kd_launch.h"
    text = f.read_text()
    f.write_text(text.replace("constexpr int kDwMaxSplit = 4;", "constexpr int kDwMaxSplit = 5;"))
    assert bench.kernel_sources_sha256(str(d)) != ref
    # inline assembly lives in strings: a change there is a code change too
    g = d / "kd_device.h"
    f.write_text(text)
    gt = g.read_text()
    assert "s_nop 0" in gt
    g.write_text(gt.replace("s_nop 0", "s_nop 1", 1))
    assert bench.kernel_sources_sha256(str(d)) != ref


def _summary_sha(path):
    with open(path) as f:
        for line in f:
            if line.startswith("source_sha256:"):
                return line.split(":", 1)[1].strip()
    return None


@pytest.mark.parametrize("kind,reader", [("hbm_traffic", bench.stored_traffic),
                                         ("mfma_counters", bench.stored_mfma_counters)])
def test_stored_counters_follow_the_sources(monkeypatch, kind, reader):
    path = os.path.join(ROOT, "profiles", f"dw_loss32k_{kind}.txt")
    sha = _summary_sha(path)
    assert sha is not None and len(sha) == 64
    monkeypatch.setattr(bench, "kernel_sources_sha256", lambda csrc_dir=None: sha)
    got = reader("dw", "loss32k")
    assert got is not None
    if kind == "hbm_traffic":
        assert got > 1e9  # bytes per launch of a 16384-token grad_W contraction
    else:
        assert got["counter_flop_per_launch"] == got["algorithmic_flop_per_launch"]
    monkeypatch.setattr(bench, "kernel_sources_sha256", lambda csrc_dir=None: "0" * 64)
    assert reader("dw", "loss32k") is None
    assert reader("dw", "no_such_workload") is None
