#!/usr/bin/env python3
"""Throughput benchmark of oriented 1D depthwise convolution on one MI355X.

One step = the whole hot path on one batch: forward (o1d_fwd), then input and
weight gradients (o1d_bwd, one pass over x and dy for both), on the headline
workload 64 x 96 x 56 x 56, K = 31, float32, per-channel angles drawn from the
eight directions i * 22.5 degrees (ConvNeXt-T stage-1 shape, synthetic data).

Inputs are resident in HBM when the timed region starts.  Steps rotate over
several disjoint buffer sets whose total size far exceeds the 256 MB
Infinity Cache, so a step never finds its inputs cached by an earlier step.

Prints ONE JSON line: value = algorithmic bytes of the step divided by the
measured time, in GB/s.  The forward reads x and writes y; the backward reads
x and dy and writes dx (and the C*K weight gradient): 5 tensors of N*C*H*W
elements.  The "roofline" object reports the dominant kernel's algorithmic
bytes per launch over its mean duration (HIP events on the stream it runs on)
against the 8 TB/s HBM peak; "cpu_baseline" times the float64 CPU oracle on
the same workload.  "configs" holds the same per-op figures for the other
workloads (stage-2 and stage-3 shapes, NHWC, stride 2 on 224^2 planes,
bilinear sampling), "copy" a plain copy of one headline tensor (the
achievable-bandwidth reference) and "angle_cost" the time at arbitrary angles
over the time at theta = 0 for K in {7, 15, 31, 63}.
"""
from __future__ import annotations

import argparse
import gc
import hashlib
import json
import os
import statistics
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "oriented-1D DW conv fwd+bwd ms & GB/s (% HBM peak), K=31, 64×96×56×56"
HBM_PEAK_GBS = 8000.0
CSRC = os.path.join(ROOT, "paper_2309_15812_amd", "csrc")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_metric_workload.json")
THETA_TEXT = {
    "discrete8": "theta from the 8 directions i*22.5 deg",
    "uniform": "theta uniform in [0, 180) deg per channel",
    "zero": "theta = 0 for every channel",
    "ninety": "theta = 90 deg for every channel",
    "ramp": "theta_c = 22.5 c deg",
    "groups:4": "four equal channel groups at 0, 45, 90, 135 deg",
}


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h")):
            with open(os.path.join(CSRC, name), "rb") as f:
                h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def git_sha():
    try:
        r = subprocess.run(["git", "-C", ROOT, "rev-parse", "HEAD"], capture_output=True, text=True, timeout=10)
        return (r.stdout.strip() or None) if r.returncode == 0 else None
    except (OSError, subprocess.SubprocessError):
        return None


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="metric")
    ap.add_argument("--sets", type=int, default=6, help="rotating buffer sets (cache defeat)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-extra", action="store_true", help="only the headline step (no configs, sweep, copy)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU work for the oracle sample")
    ap.add_argument("--case", default="", help="profiling aid, with --only: run that op on one of the configs "
                    "of the bench line (nhwc_stage1, nhwc_stage3_bf16, stride2_224, bilinear_stage1, ...) "
                    "instead of the headline workload")
    ap.add_argument("--only", default="", help="profiling aid: run only this op (fwd|bwd|bwd_input|bwd_weight), or "
                    "'copy': a plain elementwise copy of one N*C*H*W tensor (reads T bytes, writes T bytes), "
                    "the calibration kernel for the HBM byte counters, or dsc_fwd|dsc_bwd: the depthwise "
                    "separable block at its Table 1 shape")
    return ap.parse_args()


def out_size(n, s):
    return (n - 1) // s + 1


class Case:
    """One timed configuration: a workload plus stride, layout and sampling."""

    def __init__(self, wl, stride=1, layout="nchw", sampling="floor", fused=True):
        self.wl, self.stride, self.layout, self.sampling, self.fused = wl, stride, layout, sampling, fused

    @property
    def plain(self):
        return self.stride == 1 and self.layout == "nchw" and self.sampling == "floor"

    def tensor_bytes(self):
        wl, s = self.wl, self.stride
        T_in = wl.elems * wl.elem_bytes
        T_out = wl.N * wl.C * out_size(wl.H, s) * out_size(wl.W, s) * wl.elem_bytes
        return T_in, T_out, wl.C * wl.K * wl.elem_bytes

    def algorithmic_bytes(self):
        """Bytes each op must move: read every input once, write every output once."""
        T_in, T_out, CK = self.tensor_bytes()
        return {"fwd": T_in + T_out, "bwd": 2 * T_in + T_out + CK, "bwd_input": T_out + T_in,
                "bwd_weight": T_in + T_out + CK, "copy": 2 * T_in}

    def describe(self):
        wl = self.wl
        return (f"{wl.N}x{wl.C}x{wl.H}x{wl.W} K={wl.K} {wl.dtype} {self.layout} stride {self.stride} "
                f"{self.sampling}, {THETA_TEXT.get(wl.theta, 'theta mode ' + wl.theta)}")


class BufferSet:
    def __init__(self, d, case, torch, dev, ops):
        wl = case.wl
        dt = torch.float32 if wl.dtype == "f32" else torch.bfloat16
        P, Q = out_size(wl.H, case.stride), out_size(wl.W, case.stride)
        x = torch.from_numpy(d["x"]).to(dev).to(dt)
        dy = torch.from_numpy(d["dy"][:, :, :P, :Q].copy()).to(dev).to(dt)
        if case.layout == "nhwc":
            x, dy = x.permute(0, 2, 3, 1).contiguous(), dy.permute(0, 2, 3, 1).contiguous()
        self.x, self.dy = x, dy
        self.w = torch.from_numpy(d["w"]).to(dev).to(dt)
        self.th = torch.from_numpy(d["theta"]).to(dev)
        self.y = torch.empty_like(self.dy)
        self.dx = torch.empty_like(self.x)
        self.dw = torch.empty_like(self.w)
        if case.plain:
            need = ops.workspace_bytes(wl.N, wl.C, wl.H, wl.W, wl.K, dt)
        else:
            need = ops.workspace_bytes_ex(wl.N, wl.C, wl.H, wl.W, wl.K, dt, case.stride, case.layout, case.sampling)
        self.ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)


def run_op(ops, case, b, name):
    wl = case.wl
    if name == "copy":
        # torch's vectorised elementwise kernel: reads x once, writes one tensor of x's size once
        import torch
        torch.neg(b.x, out=b.dx)
    elif case.plain:
        if name == "fwd":
            ops.fwd(b.x, b.w, b.th, out=b.y)
        elif name == "bwd":
            ops.bwd(b.x, b.dy, b.w, b.th, out=(b.dx, b.dw), workspace=b.ws)
        elif name == "bwd_input":
            ops.bwd_input(b.dy, b.w, b.th, out=b.dx)
        elif name == "bwd_weight":
            ops.bwd_weight(b.x, b.dy, b.th, wl.K, out=b.dw, workspace=b.ws)
    else:
        a = (case.stride, case.layout, case.sampling)
        if name == "fwd":
            ops.fwd_ex(b.x, b.w, b.th, *a, out=b.y)
        elif name == "bwd_input":
            ops.bwd_input_ex(b.dy, b.w, b.th, (wl.H, wl.W), *a, out=b.dx)
        elif name == "bwd_weight":
            ops.bwd_weight_ex(b.x, b.dy, b.th, wl.K, *a, out=b.dw, workspace=b.ws)
        else:
            raise ValueError(name)


def timed_steps(torch, dev, steps, names, launch):
    """Queues `steps` steps (launch(i, name) for every op name in turn) between two device
    synchronisations.  Returns (wall ms per step, {name: [event ms per launch]}).

    One event before every op; the event before a step's first op also ends the previous
    step's last op, and one more event ends the last step.  The events are created and
    recorded once before the timed region (the runtime creates an event at its first
    record, which can stall the host for a millisecond while the queue is still short),
    and the collector stays off while the steps are queued."""
    stream = torch.cuda.current_stream(dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps * len(names) + 1)]
    for e in ev:
        e.record(stream)
    torch.cuda.synchronize()
    gc_was_on = gc.isenabled()
    gc.disable()
    try:
        t0 = time.perf_counter()
        k = 0
        for i in range(steps):
            for nm in names:
                ev[k].record(stream)
                k += 1
                launch(i, nm)
        ev[k].record(stream)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
    finally:
        if gc_was_on:
            gc.enable()
    durs = {nm: [ev[i * len(names) + j].elapsed_time(ev[i * len(names) + j + 1]) for i in range(steps)]
            for j, nm in enumerate(names)}
    return (t1 - t0) * 1e3 / steps, durs


def config_cases(synth):
    """The other workloads of the bench line: {name: (Case, ops timed)}."""
    W = synth.WORKLOADS
    return {
        "c2_stage1_fwd": (Case(W["c2"]), ["fwd"]),
        "c3_stage2": (Case(W["c3"]), ["fwd", "bwd"]),
        "c4_stage3_bf16": (Case(W["c4"]), ["fwd", "bwd"]),
        "nhwc_stage1": (Case(W["metric"], layout="nhwc"), ["fwd", "bwd_input", "bwd_weight"]),
        "nhwc_stage3_bf16": (Case(W["c4"], layout="nhwc"), ["fwd", "bwd_input", "bwd_weight"]),
        "stride2_224": (Case(W["metric"].replace(name="s2", N=8, H=224, W=224), stride=2),
                        ["fwd", "bwd_input", "bwd_weight"]),
        "bilinear_stage1": (Case(W["metric"], sampling="bilinear"), ["fwd", "bwd_input", "bwd_weight"]),
    }


def time_case(case, names, steps, warmup, nsets, torch, ops, synth):
    """Returns (ms_per_step, {op: [durations ms]}) for the ops `names` run in turn per step."""
    dev = torch.device("cuda:0")
    d = synth.make_inputs(case.wl)
    sets = [BufferSet(d, case, torch, dev, ops) for _ in range(nsets)]
    del d
    for i in range(warmup):
        for nm in names:
            run_op(ops, case, sets[i % nsets], nm)
    ms, durs = timed_steps(torch, dev, steps, names, lambda i, nm: run_op(ops, case, sets[i % nsets], nm))
    del sets
    torch.cuda.empty_cache()
    return ms, durs


def op_stats(case, durs):
    ab = case.algorithmic_bytes()
    out = {}
    for nm, v in durs.items():
        mean = statistics.fmean(v)
        out[nm] = {"ms_mean": round(mean, 5), "ms_median": round(statistics.median(v), 5),
                   "ms_std": round(statistics.pstdev(v), 5),
                   "ms_max": round(max(v), 5), "max_at_step": v.index(max(v)), "bytes": ab[nm],
                   "GB/s": round(ab[nm] / (mean * 1e-3) / 1e9, 1),
                   "frac_hbm_peak": round(ab[nm] / (mean * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    return out


MFMA_F32_PEAK_TFLOPS = 157.3  # MI355X dense float32 matrix-core peak


class DscSet:
    """Device buffers of the depthwise separable block (Table 1 shape) for one rotating set."""

    def __init__(self, d, p, torch, dev, ops, cout, dtype):
        wl_dt = torch.float32 if dtype == "f32" else torch.bfloat16
        self.x = torch.from_numpy(d["x"]).to(dev).to(wl_dt)
        self.w = torch.from_numpy(d["w"]).to(dev).to(wl_dt)
        self.th = torch.from_numpy(d["theta"]).to(dev)
        self.w_pw = torch.from_numpy(p["w_pw"]).to(dev).to(wl_dt)
        self.dy = torch.from_numpy(p["dy_pw"]).to(dev).to(wl_dt)
        N, C, H, W = self.x.shape
        self.z = torch.empty_like(self.x)
        self.y = torch.empty((N, cout, H, W), dtype=wl_dt, device=dev)
        self.dx = torch.empty_like(self.x)
        self.dwd = torch.empty_like(self.w)
        self.dwp = torch.empty_like(self.w_pw)
        self.ws = torch.empty(max(1, ops.dsc_workspace_bytes(N, C, cout, H, W, self.w.shape[1], wl_dt)),
                              dtype=torch.uint8, device=dev)
        self.y_dw = torch.empty_like(self.x)


def run_dsc(ops, b, name):
    if name == "dsc_fwd":
        ops.dsc_fwd(b.x, b.w, b.th, b.w_pw, out=(b.z, b.y))
    elif name == "dsc_bwd":
        ops.dsc_bwd(b.x, b.z, b.dy, b.w, b.th, b.w_pw, out=(b.dx, b.dwd, b.dwp), workspace=b.ws)
    elif name == "dw_fwd":
        ops.fwd(b.x, b.w, b.th, out=b.y_dw)
    else:
        raise ValueError(name)


def time_dsc(wl, names, steps, warmup, nsets, torch, ops, synth):
    """(ms_per_step, {op: [ms]}) for the depthwise separable block at workload wl (C' = C)."""
    dev = torch.device("cuda:0")
    sets = []
    for i in range(nsets):
        d = synth.make_inputs(wl, seed=synth.BASE_SEED + 500 + i)
        p = synth.make_pointwise(wl, wl.C, seed=synth.BASE_SEED + 600 + i)
        sets.append(DscSet(d, p, torch, dev, ops, wl.C, wl.dtype))
        del d, p
    for i in range(warmup):
        for nm in names:
            run_dsc(ops, sets[i % nsets], nm)
    ms, durs = timed_steps(torch, dev, steps, names, lambda i, nm: run_dsc(ops, sets[i % nsets], nm))
    del sets
    torch.cuda.empty_cache()
    return ms, durs


def dsc_stats(wl, ms, durs):
    """The block's per-op times and the pointwise product's estimated matrix-core rate: its share of the
    forward pass is the forward minus the depthwise forward alone (the same shape, timed beside it)."""
    mean = {k: statistics.fmean(v) for k, v in durs.items()}
    flop = 2.0 * wl.N * wl.H * wl.W * wl.C * wl.C  # one pointwise product (C' = C)
    pw_ms = mean["dsc_fwd"] - mean["dw_fwd"]
    tflops = flop / (pw_ms * 1e-3) / 1e12 if pw_ms > 0 else None
    return {
        "workload": f"{wl.N}x{wl.C}->{wl.C}x{wl.H}x{wl.W} K={wl.K} {wl.dtype}, "
                    f"{THETA_TEXT.get(wl.theta, wl.theta)} (Table 1's block shape)",
        "ms_per_step": round(ms, 4),
        "ops_ms": {k: round(v, 4) for k, v in mean.items()},
        "pointwise_flop_per_product": flop,
        "pointwise_fwd_ms_est": round(pw_ms, 4),
        "pointwise_tflops_est": None if tflops is None else round(tflops, 1),
        "mfma_peak_tflops": MFMA_F32_PEAK_TFLOPS if wl.dtype == "f32" else 2500.0,
        "mfma_frac_est": None if tflops is None else round(
            tflops / (MFMA_F32_PEAK_TFLOPS if wl.dtype == "f32" else 2500.0), 4),
    }


def algorithmic_bytes(wl) -> dict:
    """Bytes each op of the plain (stride 1, NCHW) path must move (T = one N*C*H*W tensor): the forward
    reads x and writes y; the fused backward reads x and dy and writes dx and dw; the separate gradients
    read one or two tensors and write one (or dw)."""
    return Case(wl).algorithmic_bytes()


def traffic_for(op_name: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel sources."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_hash") != kernel_source_hash():
        return None
    ent = rec.get("ops", {}).get(op_name)
    return None if ent is None else ent.get("hbm_bytes_per_launch")


def cpu_baseline(wl, synth, seconds):
    import numpy as np

    import oracle

    threads = oracle.default_threads()
    d = synth.make_inputs(wl)
    x, dy, w = (np.asarray(d[k], np.float64) for k in ("x", "dy", "w"))
    th = np.asarray(d["theta"], np.float64)
    reps, t_total = 0, 0.0
    while t_total < seconds:
        t0 = time.perf_counter()
        oracle.fwd(x, w, th, threads)
        oracle.bwd_input(dy, w, th, threads)
        oracle.bwd_weight(x, dy, th, wl.K, threads)
        t_total += time.perf_counter() - t0
        reps += 1
    step_bytes = 5 * wl.elems * wl.elem_bytes + wl.C * wl.K * wl.elem_bytes  # as the GPU step
    out = {
        "value": round(step_bytes * reps / t_total / 1e9, 3),
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{reps} full step(s) of the same workload (fwd, then dx and dw, "
                  f"{wl.N}x{wl.C}x{wl.H}x{wl.W}, K={wl.K}) in float64 C loops, OpenMP over planes/channels; "
                  f"{t_total:.1f} s",
        "ms_per_step": round(t_total * 1e3 / reps, 1),
    }
    # single-threaded oracle on the small forward workload and on a bounded
    # sample (two images) of the stage-2 workload, scaled per image
    single = {}
    for name, planes in (("c1", None), ("c3", 2)):
        w2 = synth.WORKLOADS[name]
        d2 = synth.make_inputs(w2, planes=planes)
        t0 = time.perf_counter()
        oracle.fwd(d2["x"], d2["w"], d2["theta"], 1)
        if w2.ops == "fwd+bwd":
            oracle.bwd_input(d2["dy"], d2["w"], d2["theta"], 1)
            oracle.bwd_weight(d2["x"], d2["dy"], d2["theta"], w2.K, 1)
        dt_s = time.perf_counter() - t0
        n = d2["x"].shape[0]
        single[name] = {"images": n, "ops": w2.ops, "seconds": round(dt_s, 3),
                        "ms_per_image": round(dt_s * 1e3 / n, 2),
                        "ms_full_workload_est": round(dt_s * 1e3 * w2.N / n, 1)}
    out["single_thread"] = single
    return out


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU; the operation shards over channels "
                                   "or images with no exchange (see DESIGN.md), and multi-GPU runs are not "
                                   "part of this build", "n_gpus": args.gpus}), flush=True)
        sys.exit(2)

    import torch

    from paper_2309_15812_amd import ops, synth

    if args.only in ("dsc_fwd", "dsc_bwd"):
        # profiling aid: the depthwise separable block at its Table 1 shape
        dwl = synth.WORKLOADS["dsc"]
        m, dd = time_dsc(dwl, [args.only], args.steps, args.warmup, 2, torch, ops, synth)
        print(json.dumps({"only": args.only, "ms_per_step": round(m, 5),
                          "ms_mean": round(statistics.fmean(dd[args.only]), 5)}), flush=True)
        return
    wl = synth.WORKLOADS[args.workload]
    head = Case(wl)
    if args.case:
        if not args.only:
            sys.exit("--case needs --only")
        head = config_cases(synth)[args.case][0]
        wl = head.wl
    T = wl.elems * wl.elem_bytes
    print(f"[bench] workload {wl} T={T / 1e6:.2f} MB sets={args.sets}", file=sys.stderr, flush=True)
    names = [args.only] if args.only else ["fwd", "bwd"]
    ms, durs = time_case(head, names, args.steps, args.warmup, args.sets, torch, ops, synth)
    print(f"[bench] {ms:.4f} ms/step", file=sys.stderr, flush=True)

    per_op = op_stats(head, durs)
    dominant = max(per_op, key=lambda k: per_op[k]["ms_mean"])
    dom_ms = per_op[dominant]["ms_mean"]
    op_bytes = head.algorithmic_bytes()
    achieved = op_bytes[dominant] / (dom_ms * 1e-3) / 1e9
    step_bytes = sum(op_bytes[k] for k in durs)
    out = {
        "metric": METRIC,
        "value": round(step_bytes / (ms * 1e-3) / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: N={wl.N} C={wl.C} H={wl.H} W={wl.W} K={wl.K} {wl.dtype}, "
                        f"{THETA_TEXT.get(wl.theta, 'theta mode ' + wl.theta)}, "
                        f"one step = fwd + bwd (dx and dw in one pass)",
            "N": wl.N, "C": wl.C, "H": wl.H, "W": wl.W, "K": wl.K,
            "buffer_sets": args.sets,
            "step_bytes": step_bytes,
        },
        "frac_hbm_peak_step": round(step_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "roofline": {
            "bound": "hbm",
            "kernel": dominant,
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            # the committed counter summary covers the headline workload only
            "traffic": traffic_for(dominant) if args.workload == "metric" and not args.case else None,
            "algorithmic_bytes_per_launch": op_bytes[dominant],
            "ms_per_launch": dom_ms,
        },
        "ops": per_op,
        "kernel_source_hash": kernel_source_hash(),
        "git_sha": git_sha(),
    }

    if not args.only and not args.no_extra:
        # the achievable bandwidth: a plain copy of one headline tensor
        _, dc = time_case(head, ["copy"], 20, 5, args.sets, torch, ops, synth)
        out["copy"] = op_stats(head, dc)["copy"]
        print(f"[bench] copy: {out['copy']}", file=sys.stderr, flush=True)
        # the other workloads, per op
        W = synth.WORKLOADS
        cases = config_cases(synth)
        cfg = {}
        for key, (case, nm) in cases.items():
            m, dd = time_case(case, nm, 20, 5, 3, torch, ops, synth)
            cfg[key] = {"workload": case.describe(), "ms_per_step": round(m, 4), "ops": op_stats(case, dd)}
            print(f"[bench] {key}: {m:.4f} ms/step", file=sys.stderr, flush=True)
        out["configs"] = cfg
        # angle cost: the same shapes at theta = 0, 90 and uniform continuous angles
        sweep = {}
        for K in (7, 15, 31, 63):
            base = W["c5"].replace(K=K)
            res = {}
            for mode in ("zero", "ninety", "uniform"):
                m, dd = time_case(Case(base.replace(theta=mode)), ["fwd", "bwd"], 20, 5, 3, torch, ops, synth)
                res[mode] = {"step_ms": round(m, 4), "fwd_ms": round(statistics.fmean(dd["fwd"]), 4)}
            r_step = max(v["step_ms"] for v in res.values()) / res["zero"]["step_ms"]
            r_fwd = max(v["fwd_ms"] for v in res.values()) / res["zero"]["fwd_ms"]
            sweep[f"K{K}"] = {**res, "max_over_theta0_step": round(r_step, 3), "max_over_theta0_fwd": round(r_fwd, 3)}
            print(f"[bench] angle sweep K={K}: {sweep[f'K{K}']}", file=sys.stderr, flush=True)
        out["angle_cost"] = {"workload": "32x256x56x56 f32 fwd+bwd", **sweep}
        # the depthwise separable block (Sec. 3.2, Table 1): depthwise + pointwise on the matrix cores
        dwl = W["dsc"]
        m, dd = time_dsc(dwl, ["dsc_fwd", "dsc_bwd", "dw_fwd"], 10, 3, 2, torch, ops, synth)
        out["dsc_block"] = dsc_stats(dwl, m, dd)
        print(f"[bench] dsc block: {out['dsc_block']}", file=sys.stderr, flush=True)

    if not args.no_cpu and not args.only:
        print("[bench] timing the CPU oracle ...", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, synth, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
