#!/usr/bin/env python3
"""Throughput of the fused chunked top-K KL loss (forward + backward) on one MI355X.

One step = one kd_topk_kl_fwd_bwd call over the whole workload: teacher
prologue, then for every chunk the projection with the online log-normaliser
and the provisional gradient, the normaliser merge with the per-token factors,
the teacher correction (Eq. 3), and the dH and dW contractions. The same step
through the split entry points (forward, then a backward that recomputes the
logits, as Algorithm 1 does) is timed beside it. Inputs are synthetic (seeded)
and resident in HBM before the timed region.

Prints one JSON line. `roofline` is for the kernel with the largest total time,
from HIP events the library records around each contraction launch during the
timed region (event pairs around every launch cost ~0.5% of a step, so the
per-kernel breakdown of all kernels comes from a second, untimed pass);
`cpu_baseline` times the fp64 CPU oracle on a bounded sample.
"""
import argparse
import json
import os
import sys
import time

METRIC = "fwd+bwd tokens/s of fused top-K KL loss (N=32K,D=4096,V=131K); MFMA %"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3       # MI355X fp32 (matrix and vector)
# The paper's fused chunked loss in its loss-only benchmark (D=4096, V=131072,
# K=100, chunk 4096, bf16): 5.04 it/s at 32K tokens and 0.630 it/s at 256K
# tokens, on 2x H200 with tensor parallelism 2 -> 165,151 tokens/s for both
# GPUs together. Another machine's number: context for the ratio, not a target.
PAPER_TOKENS_PER_S = {"loss32k": 32768 * 5.04, "long256k": 262144 * 0.630}
PAPER_REF = "paper's fused chunked loss, loss-only benchmark, 2x H200 with TP=2 (both GPUs)"


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="loss32k",
                    help="tiny_fp32 | loss4k | loss32k | packed | long256k")
    ap.add_argument("--cpu-rows", type=int, default=2048,
                    help="token rows of the oracle's CPU baseline sample (0 = skip)")
    ap.add_argument("--split-steps", type=int, default=3,
                    help="steps timed through the split fwd / bwd entry points (0 = skip)")
    ap.add_argument("--json-out", default=None, help="also append the JSON line to this file")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES bytes three times (the "
                         "reference kernel that scales the FETCH_SIZE / WRITE_SIZE counters)")
    ap.add_argument("--blas-reference", action="store_true",
                    help="only time the vendor GEMM (torch.matmul on hipBLASLt) on the "
                         "workload's three contraction shapes in bf16, as a reference for the "
                         "library's contraction kernels")
    ap.add_argument("--memory-sweep", action="store_true",
                    help="only measure peak allocated bytes of one fwd+bwd call at N = 4K..256K "
                         "(D=4096, V=131072, K=100, chunk 4096, bf16) and fit a + b N")
    return ap.parse_args()


def sclk_mhz():
    """Current shader clock from the driver's sysfs table (None if unreadable)."""
    import glob
    for f in sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk")):
        try:
            for line in open(f):
                if line.strip().endswith("*"):
                    return float(line.split(":")[1].strip().rstrip("*").strip().lower()
                                 .replace("mhz", ""))
        except (OSError, ValueError, IndexError):
            continue
    return None


def _hwmon_files(name):
    import glob
    return sorted(glob.glob(f"/sys/class/drm/card*/device/hwmon/hwmon*/{name}"))


def power_w():
    """Board power from the driver's hwmon (average, else instantaneous), in
    watts (None if unreadable)."""
    for name in ("power1_average", "power1_input"):
        for f in _hwmon_files(name):
            try:
                with open(f) as fh:
                    v = float(fh.read().strip()) / 1e6
                if v > 0:
                    return v
            except (OSError, ValueError):
                continue
    return None


def power_cap_w():
    """The board power cap the driver enforces, in watts (None if unreadable)."""
    for f in _hwmon_files("power1_cap"):
        try:
            with open(f) as fh:
                return float(fh.read().strip()) / 1e6
        except (OSError, ValueError):
            continue
    return None


class ClockSampler:
    """Samples the shader clock (and the board power) every `period` seconds
    on a background thread (the main thread sits in a blocking device
    synchronise meanwhile)."""

    def __init__(self, period=0.02):
        import threading
        self.period, self.samples, self.power = period, [], []
        self._stop = threading.Event()
        self._t = threading.Thread(target=self._run, daemon=True)

    def _run(self):
        while not self._stop.is_set():
            v = sclk_mhz()
            if v is not None:
                self.samples.append(v)
            w = power_w()
            if w is not None:
                self.power.append(w)
            self._stop.wait(self.period)

    def __enter__(self):
        self._t.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        self._t.join()

    def mean(self):
        return sum(self.samples) / len(self.samples) if self.samples else None

    def mean_power(self):
        return sum(self.power) / len(self.power) if self.power else None


def memory_sweep():
    """Peak allocated bytes (inputs + outputs + workspace) of one fwd+bwd call
    per N at the 4K-config shapes; least-squares fit peak = a + b N."""
    import numpy as np
    import torch
    import kd_inputs as ki
    import paper_2608_03796_amd as kd
    kd.load_library()
    dev = torch.device("cuda:0")
    base = ki.WORKLOADS["loss4k"]
    pts = []
    for N in (4096, 8192, 16384, 32768, 65536, 131072, 262144):
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats(dev)
        w = ki.Workload(name=f"sweep{N}", N=N, D=base.D, V=base.V, K=base.K, chunk=base.chunk,
                        tau=base.tau, dtype=base.dtype, mask=base.mask)
        inp = ki.make_workload_inputs(w, dev)
        out = kd.fwd_bwd(inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"],
                         tau=w.tau, ignore=inp["ignore"], chunk=w.chunk)
        torch.cuda.synchronize()
        assert np.isfinite(float(out["loss"]))
        pts.append((N, int(torch.cuda.max_memory_allocated(dev))))
        print(f"bench: memory N={N} peak {pts[-1][1] / 2**30:.3f} GiB", file=sys.stderr, flush=True)
        del inp, out
    # the dW gather buffer grows with the number of chunks up to 16384 tokens
    # (then stays fixed), so the linear law is fitted where the workspace is
    # constant
    n = np.array([p[0] for p in pts if p[0] >= 16384], dtype=np.float64)
    m = np.array([p[1] for p in pts if p[0] >= 16384], dtype=np.float64)
    b, a = np.polyfit(n, m, 1)
    resid = float(np.abs(m - (a + b * n)).max())
    dense = 262144 * base.V * 2
    print(json.dumps({"memory_sweep": [{"N": int(x), "peak_bytes": int(y)} for x, y in pts],
                      "fit": {"a_bytes": a, "b_bytes_per_token": b, "max_residual_bytes": resid,
                              "over": "N >= 16384 (constant workspace)"},
                      "shapes": {"D": base.D, "V": base.V, "K": base.K, "chunk": base.chunk,
                                 "dtype": base.dtype},
                      "bf16_logits_at_262144_bytes": dense}), flush=True)


def blas_reference(wname, reps=10):
    """torch.matmul (hipBLASLt) on the contraction shapes of one chunk / dW group
    of the workload, bf16 in and out, random operands of the workload's scales;
    HIP-event time per call and the sampled shader clock. A plain GEMM: no
    epilogue beyond the bf16 output write (the library's kernels add the
    normaliser and dZ epilogue, a row scale, or grad_W's fp32 read-modify-write)."""
    import torch
    import kd_inputs as ki
    w = ki.WORKLOADS[wname]
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(ki.SEED_HIDDEN)

    def rn(*shape, std=1.0):
        return (torch.randn(*shape, generator=g, device=dev) * std).to(torch.bfloat16)

    c = w.chunk
    T = max(1, 16384 // c) * c  # tokens of one dW group
    W = rn(w.V, w.D, std=0.02)
    H = rn(c, w.D)
    dZ = rn(c, w.V, std=1e-3)
    Ht = rn(w.D, T)
    dZg = rn(T, w.V, std=1e-3)
    cases = [("projection z^T = W H_c^T", lambda: torch.matmul(W, H.t()), 2.0 * c * w.D * w.V),
             ("dH = dZ W", lambda: torch.matmul(dZ, W), 2.0 * c * w.D * w.V),
             ("dW^T = H^T dZ (one group)", lambda: torch.matmul(Ht, dZg), 2.0 * T * w.D * w.V)]
    out = []
    for name, f, fl in cases:
        for _ in range(3):
            f()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        with ClockSampler(0.005) as ck:
            e0.record()
            for _ in range(reps):
                f()
            e1.record()
            torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        clk = ck.mean()
        out.append({"shape": name, "ms": round(ms, 4), "tflops": round(fl / ms / 1e9, 1),
                    "sclk_mhz": round(clk, 1) if clk else None})
        print(f"bench: blas {name}: {ms:.3f} ms, {fl / ms / 1e9:.0f} TFLOP/s", file=sys.stderr,
              flush=True)
    print(json.dumps({"blas_reference": out, "workload": wname,
                      "torch": torch.__version__}), flush=True)


def copy_calibration(nbytes):
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes, "launches": 3}))


def kernel_sources_sha256(csrc_dir=None):
    """Digest of the HIP sources' code, to tell whether stored counters still
    apply: comments and layout are left out, so that editing a comment keeps
    the counters taken on the same code."""
    import hashlib
    import re
    d = csrc_dir or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                 "paper_2608_03796_amd", "csrc")
    tok = re.compile(r'"(?:\\.|[^"\\])*"|\'(?:\\.|[^\'\\])*\'|//[^\n]*|/\*.*?\*/', re.S)
    h = hashlib.sha256()
    for name in sorted(os.listdir(d)):
        if name.endswith((".hip", ".h", ".cpp")):
            with open(os.path.join(d, name)) as f:
                text = f.read()
            code = tok.sub(lambda m: m.group(0) if m.group(0)[0] in "\"'" else " ", text)
            h.update(name.encode() + b"\0" + " ".join(code.split()).encode())
    return h.hexdigest()


def stored_traffic(kernel, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken for this kernel, this workload and the current sources."""
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles",
                        f"{kernel}_{workload}_hbm_traffic.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line:
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != kernel_sources_sha256():
        return None
    try:
        return float(kv["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def stored_mfma_counters(kernel, workload):
    """MFMA counters of one launch from the committed rocprofv3 summary
    (SQ_INSTS_VALU_MFMA_MOPS_BF16, SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE),
    if it was taken for this kernel, this workload and the current sources."""
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles",
                        f"{kernel}_{workload}_mfma_counters.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line:
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != kernel_sources_sha256():
        return None
    out = {"file": os.path.relpath(path, os.path.dirname(os.path.abspath(__file__)))}
    for k in ("counter_flop_per_launch", "algorithmic_flop_per_launch", "avg_launch_ms",
              "counter_tflops", "counter_frac_of_peak", "mfma_busy_pct", "gui_active_mhz"):
        try:
            out[k] = float(kv[k])
        except (KeyError, ValueError):
            out[k] = None
    return out


def cpu_baseline(inp, w, rows_count, single_rows=64):
    """fp64 oracle (fwd+bwd) on a random sub-batch of `rows_count` tokens at
    full D and V, timed on this host's cores; plus a one-thread run on
    `single_rows` sampled rows, and the linear extrapolation to the full step."""
    import numpy as np
    import torch
    import kd_inputs as ki
    from oracle import kd_topk_kl
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()
                     if i.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    sel = ki.sub_batch(w.N, rows_count).to(inp["hidden"].device)
    h = inp["hidden"].index_select(0, sel).float().cpu().numpy()
    W = inp["W"].float().cpu().numpy()
    idx = inp["teacher_idx"].index_select(0, sel).cpu().numpy()
    tl = inp["teacher_logit"].index_select(0, sel).cpu().numpy()
    ign = None
    if inp["ignore"] is not None:
        ign = inp["ignore"].index_select(0, sel).cpu().numpy()
    t0 = time.perf_counter()
    res = kd_topk_kl(h, W, idx, tl, tau=w.tau, ignore=ign, chunk=256, want_grads=True)
    dt = time.perf_counter() - t0
    assert np.isfinite(res["loss"])
    rec = {"value": rows_count / dt, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
           "sample": f"{rows_count}-token random sub-batch (seed {ki.SEED_SUBBATCH}) of the "
                     f"{w.name} workload at full D={w.D}, V={w.V}, K={w.K}; fp64 NumPy "
                     f"forward+backward, dense logits per 256-row chunk; {dt:.1f} s",
           "extrapolated_full_step_s": round(w.N * dt / rows_count, 1)}
    try:
        from threadpoolctl import threadpool_limits
        sel1 = ki.sample_rows(torch.arange(w.N), single_rows).to(inp["hidden"].device)
        h1 = inp["hidden"].index_select(0, sel1).float().cpu().numpy()
        i1 = inp["teacher_idx"].index_select(0, sel1).cpu().numpy()
        t1 = inp["teacher_logit"].index_select(0, sel1).cpu().numpy()
        g1 = None if inp["ignore"] is None else inp["ignore"].index_select(0, sel1).cpu().numpy()
        with threadpool_limits(limits=1):
            t0 = time.perf_counter()
            kd_topk_kl(h1, W, i1, t1, tau=w.tau, ignore=g1, chunk=64, want_grads=True)
            d1 = time.perf_counter() - t0
        rec["single_thread"] = {"value": single_rows / d1, "unit": "tokens/s", "cores": 1,
                                "sample": f"{single_rows} sampled rows (seed {ki.SEED_ROWS}); "
                                          f"{d1:.1f} s"}
    except ImportError:  # pragma: no cover
        pass
    return rec


def split_schedule(inp, w, steps, ws, step_flops, peak):
    """The same step through the split entry points (kd_topk_kl_fwd, then
    kd_topk_kl_bwd), i.e. Algorithm 1's schedule: the forward projects each
    chunk once for log Z and the teacher logits, the backward recomputes the
    logits from the saved log Z, then dH and dW (8 N D V FLOP per step)."""
    import torch
    import paper_2608_03796_amd as kd
    gw = torch.empty(w.V, w.D, dtype=torch.float32, device=inp["hidden"].device)

    def step():
        f = kd.fwd(inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"], tau=w.tau,
                   ignore=inp["ignore"], chunk=w.chunk, workspace=ws)
        kd.bwd(inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"], f["saved_logz"],
               tau=w.tau, ignore=inp["ignore"], chunk=w.chunk, grad_W_out=gw, workspace=ws)

    step()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    print(f"bench: split fwd + bwd {ms:.3f} ms/step", file=sys.stderr, flush=True)
    return {"entry_points": "kd_topk_kl_fwd + kd_topk_kl_bwd (logit recompute in the backward)",
            "steps": steps, "ms_per_step": round(ms, 4),
            "tokens_per_s": round(w.N / (ms / 1e3), 1),
            "flop_per_step": step_flops,
            "mfma_pct": round(100.0 * step_flops / (ms / 1e3) / (peak * 1e12), 2)}


def autograd_schedule(inp, w, steps, ws):
    """The step as a training loop takes it: topk_kl_loss(...).backward() with
    hidden and W requiring gradients, for both autograd schedules (fused: one
    kd_topk_kl_fwd_bwd call in the forward, the gradients scaled by the
    upstream gradient in the backward; recompute: the split entry points).
    Includes the autograd overhead and grad_W's conversion to W's dtype; the
    workspace is reused across calls, as a training loop would."""
    import torch
    import paper_2608_03796_amd as kd
    h = inp["hidden"].detach().clone().requires_grad_(True)
    Wp = inp["W"].detach().clone().requires_grad_(True)
    res = {}
    for sched in ("fused", "recompute"):
        def step():
            h.grad = None
            Wp.grad = None
            loss = kd.topk_kl_loss(h, Wp, inp["teacher_idx"], inp["teacher_logit"], tau=w.tau,
                                   ignore=inp["ignore"], chunk=w.chunk, schedule=sched,
                                   workspace=ws)
            loss.backward()

        step()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            step()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        print(f"bench: autograd {sched} {ms:.3f} ms/step", file=sys.stderr, flush=True)
        res[sched] = {"ms_per_step": round(ms, 4), "tokens_per_s": round(w.N / (ms / 1e3), 1)}
    del h, Wp
    torch.cuda.empty_cache()
    return {"call": "topk_kl_loss(...).backward(), hidden and W requiring gradients",
            "steps": steps, **res}


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.memory_sweep:
        memory_sweep()
        return
    if args.blas_reference:
        blas_reference(args.workload)
        return
    if args.gpus != 1:
        print(f"bench.py: --gpus {args.gpus} is not supported: the library runs the loss on one "
              f"GPU only (no collectives); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    import kd_inputs as ki
    import paper_2608_03796_amd as kd

    kd.load_library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = ki.WORKLOADS[args.workload]
    print(f"bench: workload {w.name} N={w.N} D={w.D} V={w.V} K={w.K} chunk={w.chunk} "
          f"tau={w.tau} {w.dtype}", file=sys.stderr, flush=True)
    torch.cuda.reset_peak_memory_stats(dev)
    inp = ki.make_workload_inputs(w, dev)
    dt_code = kd.KD_BF16 if w.dtype == "bf16" else kd.KD_F32
    ws = kd.alloc_workspace(w.N, w.D, w.V, w.K, w.chunk, w.tau, dt_code, dev)
    out = {"loss": torch.empty((), dtype=torch.float32, device=dev),
           "grad_hidden": torch.empty(w.N, w.D, dtype=w.torch_dtype, device=dev),
           "grad_W": torch.empty(w.V, w.D, dtype=torch.float32, device=dev)}

    def step():
        kd.fwd_bwd(inp["hidden"], inp["W"], inp["teacher_idx"], inp["teacher_logit"], tau=w.tau,
                   ignore=inp["ignore"], chunk=w.chunk, workspace=ws, out=out)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print("bench: warmup done", file=sys.stderr, flush=True)
    kd.profile_read()
    # event pairs only around the contraction kernels inside the timed region
    # (the dominant kernel is one of them); every kernel in a second pass below
    kd.profile_enable(True, contractions_only=True)
    stream = torch.cuda.current_stream(dev)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with ClockSampler() as clock:
        e0.record(stream)
        for _ in range(args.steps):
            step()
        e1.record(stream)
        torch.cuda.synchronize()
    kd.profile_enable(False)
    prof = kd.profile_read()
    ms = e0.elapsed_time(e1) / args.steps
    peak_alloc = torch.cuda.max_memory_allocated(dev)
    loss = float(out["loss"])
    print(f"bench: {ms:.3f} ms/step, loss {loss:.6f}", file=sys.stderr, flush=True)

    tokens_per_s = w.N / (ms / 1e3)
    n_valid = w.N if inp["ignore"] is None else int((inp["ignore"] == 0).sum())
    # 8 N D V: the metric's four contractions per chunk (Algorithm 1 with its
    # two forward passes in one); the fused call runs three (6 N D V), which
    # the library reports per launch and the MFMA fraction is taken on
    equiv_flops = 8.0 * w.N * w.D * w.V
    # With a mask the fused call leaves the ignored tokens out of its
    # contractions. The library counts each launch's FLOP over all the rows it
    # is given, so every contraction kind sums to 2 N D V per step; the tokens
    # that are not ignored make 2 N_valid D V of it, which is what the step
    # computes for the loss (the hardware also runs the rows that complete a
    # tile: under 256 per projection or dH launch and 64 per dW launch, which
    # the MFMA counters show and this leaves out).
    useful = n_valid / w.N if inp["ignore"] is not None else 1.0
    executed = sum(v["flops"] for v in prof.values()) / args.steps * useful
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    dom_name, dom = max(prof.items(), key=lambda kv: kv[1]["total_ms"])
    dom_flops = dom["flops"] * useful
    achieved = dom_flops / (dom["total_ms"] / 1e3) / 1e12 if dom["total_ms"] > 0 else 0.0
    roofline = {"bound": "mfma", "kernel": dom_name, "achieved": round(achieved, 2),
                "peak": peak, "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                "traffic": stored_traffic(dom_name, w.name),
                "avg_launch_ms": round(dom["total_ms"] / dom["launches"], 4),
                "flop_per_launch": dom_flops / dom["launches"]}
    # achieved HBM-side rate of the dominant kernel: the counters' bytes per
    # launch over this run's launch time
    roofline["traffic_gb_per_s"] = (
        round(roofline["traffic"] / (roofline["avg_launch_ms"] / 1e3) / 1e9, 1)
        if roofline["traffic"] else None)
    # every kernel's share of a step, from a second pass with an event pair
    # around every launch (the events' cost is why the timed pass above
    # records them around the contractions only)
    kd.profile_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    kd.profile_enable(False)
    prof_all = kd.profile_read()
    kernels = {k: {"launches": v["launches"], "ms_per_step": round(v["total_ms"] / args.steps, 4),
                   "tflops": (round(v["flops"] * useful / (v["total_ms"] / 1e3) / 1e12, 2)
                              if v["flops"] and v["total_ms"] > 0 else None)}
               for k, v in sorted(prof_all.items(), key=lambda kv: -kv[1]["total_ms"])}
    paper = PAPER_TOKENS_PER_S.get(w.name)
    clk = clock.mean()
    rec = {
        "metric": METRIC, "value": round(tokens_per_s, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak",
        "vs_baseline": round(tokens_per_s / paper, 4) if paper else None,
        "vs_baseline_ref": (f"{PAPER_REF}: {paper:.0f} tokens/s" if paper else None),
        "dtype": "bf16" if w.dtype == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": w.name, "N": w.N, "D": w.D, "V": w.V, "K": w.K, "chunk": w.chunk,
                   "tau": w.tau, "ignored_frac": 0.05 if w.mask == "packed5" else 0.0},
        "mfma_pct": round(100.0 * executed / (ms / 1e3) / (peak * 1e12), 2),
        "gemm_flop_per_step": executed,
        "mfma_pct_8ndv_equivalent": round(100.0 * equiv_flops / (ms / 1e3) / (peak * 1e12), 2),
        "flop_basis": ("mfma_pct = the FLOP the step's contraction kernels execute "
                       "(gemm_flop_per_step: one projection per chunk plus dH and dW, 6 N D V; "
                       "with a mask 6 N_valid D V, the ignored tokens being left out) "
                       "per second over the dense peak; mfma_pct_8ndv_equivalent counts the "
                       "metric's 8 N D V per step (all N positions) instead (an equivalent "
                       "rate, not utilisation: the fused call does not execute the fourth "
                       "contraction)"),
        "sclk_mhz": round(clk, 1) if clk else None,
        "sclk_samples": len(clock.samples),
        # board power during the timed region and the cap the driver enforces
        # (the clock under this load is set by power); the driver's reading
        # trails the load, so it means something over a second or more
        "power_w": round(clock.mean_power(), 1) if clock.mean_power() else None,
        "power_cap_w": power_cap_w(),
        "mfma_pct_at_measured_sclk": (round(100.0 * executed / (ms / 1e3)
                                            / (256 * 4096 * clk * 1e6), 2)
                                      if clk and w.dtype == "bf16" else None),
        "peak_alloc_bytes": int(peak_alloc),
        "valid_tokens_per_s": round(n_valid / (ms / 1e3), 1),
        "loss": loss,
        "roofline": roofline,
        "kernels": kernels,
    }
    # the dominant kernel's rocprofv3 MFMA counters (FLOP from
    # SQ_INSTS_VALU_MFMA_MOPS_BF16, busy cycles), when committed for the
    # current sources: the counter-derived rate beside the event-timed one
    rec["mfma_counters"] = stored_mfma_counters(dom_name, w.name)
    if args.split_steps > 0:
        rec["recompute_schedule"] = split_schedule(inp, w, args.split_steps, ws, equiv_flops, peak)
        rec["autograd"] = autograd_schedule(inp, w, args.split_steps, ws)
    if args.cpu_rows > 0:
        print("bench: timing the CPU oracle baseline", file=sys.stderr, flush=True)
        rec["cpu_baseline"] = cpu_baseline(inp, w, args.cpu_rows)
    line = json.dumps(rec)
    print(line, flush=True)
    if args.json_out:
        with open(args.json_out, "a") as f:
            f.write(line + "\n")


if __name__ == "__main__":
    main()
