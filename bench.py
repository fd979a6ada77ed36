#!/usr/bin/env python3
"""Benchmark: checksum-protected convolution layers on one MI355X.

Workload: the AlexNet-shaped stack of five convolution layers, fp32, batch 64
(synthetic U(0,1) inputs and He-normal weights at every layer's own input
shape; layers are independent).  One step runs the whole protected path of
every layer on one stream:

    conv_fwd_sums (+ encode of Cd1, Cd2) -> verify_correct_sums (+ Co5, Co6, Co7)

(two launches: the input checksums are encoded by extra workgroups of the
convolution launch and the CoC-D summations are taken in its epilogue; the
final launch computes the checksum-of-checksums Co5..Co7, tests every position
and runs the correction chain where one is flagged), following the paper's
error-injection protocol (Sec. 6.1): step i corrupts one output element of
layer (i mod 5) inside the convolution, before its output is summed, so every
step also detects, locates and repairs one fault.  Weight checksums are encoded
once at set-up (Sec. 4.2).

Reported: protected TFLOP/s (value), the error-free protected and the
unprotected (convolution only) rates, ABFT overhead percentages, per-layer
stage times, a roofline entry for the dominant convolution kernel, and the CPU
oracle timed on a sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_PEAK = {"f32": 157.3, "bf16": 2516.6}   # TFLOP/s, MI355X dense matrix peaks
# Additive corruption of one output element per step.  The outputs of these layers have an rms
# near 0.8, and the CoC location ratios (Sec. 3.6) resolve to the right block once a fault exceeds
# about 8 * max(N, M) times the detection threshold at its position: up to ~5e4 on the bf16
# layers with N * M = 65536 (ResNet-18 stage 4), where a smaller fault is still detected and
# corrected, but by the row or column schemes.  1e6 stays above that bound on every layer.
FAULT_VALUE = 1.0e6


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="lower bound on the CPU oracle's timed work (whole batch-64 passes)")
    ap.add_argument("--workload", default="alexnet",
                    choices=["alexnet", "vgg19", "vgg19_bf16", "resnet18", "darknet19"],
                    help="layer stack to time (the default is the benchmark's workload; the others report "
                         "the same figures for the remaining configurations)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="run a plain fp32 device copy of this size first (counter calibration)")
    ap.add_argument("--quiet", action="store_true")
    ap.add_argument("--schemes", action="store_true",
                    help="instead of the benchmark: the cost of every correction workflow (CoC, RC, ClC, FC, "
                         "recomputation) on each distinct layer, and the layerwise RC/ClC choice (one JSON "
                         "line per layer)")
    ap.add_argument("--scheme-reps", type=int, default=10)
    ap.add_argument("--groups", action="store_true",
                    help="AlexNet with Caffe's two groups on conv2, conv4 and conv5 (Sec. 5.2); flops counted "
                         "for the grouped layers")
    ap.add_argument("--chain", action="store_true",
                    help="the workload's layers chained into one network (ReLU, and max pooling where "
                         "the size drops, between layers): whole-network protected inference")
    ap.add_argument("--bias", action="store_true",
                    help="give every layer a seeded bias (Sec. 5.1): the output carries it and every check "
                         "applies its shares (the workloads themselves have none)")
    return ap.parse_args()


class LayerRun:
    def __init__(self, cfg, li, ft, torch, bias=False, groups=1):
        import workloads as wl
        self.spec = spec = cfg.layers[li]
        self.name = spec.name
        self.lay = ft.Layer(spec.n, spec.ch, spec.h, spec.w, spec.m, spec.r, spec.s, spec.stride,
                            spec.pad, spec.dtype, groups=groups)
        tdt = torch.bfloat16 if spec.dtype == "bf16" else torch.float32   # bf16 draws are exact in bf16
        self.D = torch.from_numpy(wl.gen_d(cfg, li)).to(tdt).cuda()
        # a grouped layer's filters see ch / groups channels (He-normal over that fan-in)
        self.W = torch.from_numpy(wl.gen_w(cfg, li, spec.with_(ch=spec.ch // groups))).to(tdt).cuda()
        self.O = self.lay.empty_output()
        self.lay.encode_weights(self.W)
        if bias:
            b = np.random.default_rng([12203, cfg.cid, li, 5]).uniform(-0.1, 0.1, size=spec.m)
            self.lay.set_bias(torch.from_numpy(b.astype(np.float32)).cuda())
        E, F = self.lay.E, self.lay.F
        self.flops = 2.0 * spec.n * spec.m * E * F * (spec.ch // groups) * spec.r * spec.s
        d = wl.fault_draws(cfg.cid, li, 1)[0]
        self.fault = {"n": int(d[0] * spec.n), "m": int(d[1] * spec.m), "x": int(d[2] * E),
                      "y": int(d[3] * F), "kind": "add", "value": FAULT_VALUE}


def scheme_table(args, cfg, runs, ft, torch):
    """Per distinct layer: the unprotected convolution, the error-free protected step (its excess
    is CoC-D), and each correction workflow of Sec. 4.3 on a fault pattern it must handle (the
    excess over the error-free step), all medians in microseconds; then the RC/ClC switch the
    paper's rule picks from those times."""
    import statistics

    from paper_2003_12203_amd import schemes

    seen = set()
    for li, r in enumerate(runs):
        s = cfg.layers[li]
        key = (s.n, s.ch, s.h, s.w, s.m, s.r, s.s, s.stride, s.pad, s.dtype)
        if key in seen:
            continue
        seen.add(key)
        L = r.lay
        ts = []
        L.conv_ws(r.D, r.W, r.O)
        for _ in range(args.scheme_reps):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            ev[0].record()
            L.conv_ws(r.D, r.W, r.O)
            ev[1].record()
            ev[1].synchronize()
            ts.append(ev[0].elapsed_time(ev[1]) * 1e3)
        t_conv = statistics.median(ts)
        res = schemes.measure(L, r.D, r.W, reps=args.scheme_reps)
        base = res["error-free"]["us"]
        flows = {}
        for name, v in res.items():
            if name == "error-free":
                continue
            flows[name] = {"extra_us": round(v["us"] - base, 2), "resolved": v["resolved"],
                           "as_expected": tuple(v["resolved"]) == schemes.WORKFLOWS[name][3]}
        line = {"workload": cfg.name, "layer": s.name, "dtype": s.dtype, "conv_us": round(t_conv, 2),
                "protected_us": round(base, 2), "coc_d_us": round(base - t_conv, 2), "workflows": flows}
        t = {k: v["us"] for k, v in res.items()}
        if all(k in t for k in schemes.WORKFLOWS):
            c = schemes.rc_clc_policy(t, s.n * s.ch * s.h * s.w, s.m * s.ch * s.r * s.s)
            line["policy"] = {"rc_on": c.rc_on, "clc_on": c.clc_on, "rc_gain_us": round(c.rc_gain, 2),
                              "rc_loss_us": round(c.rc_loss, 2), "clc_gain_us": round(c.clc_gain, 2),
                              "clc_loss_us": round(c.clc_loss, 2)}
        print(json.dumps(line), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the protected layer needs no communication; see DESIGN.md for how it would shard)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2003_12203_amd as ft
    import workloads as wl

    ft.lib()  # fails loudly if the HIP library is missing
    torch.cuda.set_device(0)
    cfg = {"alexnet": wl.config(1), "vgg19": wl.config(2), "vgg19_bf16": wl.vgg19_bf16(),
           "resnet18": wl.config(3), "darknet19": wl.config(4)}[args.workload]
    if args.groups and args.workload != "alexnet":
        print("bench.py: --groups applies to the AlexNet workload (Caffe's two groups)", file=sys.stderr)
        sys.exit(2)
    grouped = ("conv2", "conv4", "conv5") if args.groups else ()
    runs = [LayerRun(cfg, li, ft, torch, args.bias, 2 if cfg.layers[li].name in grouped else 1)
            for li in range(len(cfg.layers))]
    if args.schemes:
        scheme_table(args, cfg, runs, ft, torch)
        return
    if args.chain:
        return chain_bench(args, cfg, runs, ft, torch)
    dtype = cfg.layers[0].dtype
    peak = MFMA_PEAK[dtype]
    nl = len(runs)
    total_flops = sum(r.flops for r in runs)
    torch.cuda.synchronize()
    if args.copy_calibration_mib > 0:
        # a plain copy of known size: the scale of FETCH_SIZE / WRITE_SIZE per byte moved
        a = torch.ones(args.copy_calibration_mib << 18, device="cuda")
        b = torch.empty_like(a)
        for _ in range(2):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    # the dominant kernel for the roofline: the convolution of the largest layer (conv2, 42% of
    # the step's flops), timed inside the timed region with two events that the library records
    # immediately around that kernel's launch (ftcnn_set_kernel_events: the channels-last copy
    # launched before it by the same call falls outside the pair)
    dom = int(np.argmax([r.flops for r in runs]))

    def protected_step(i, inject=True, ev=None):
        for li, r in enumerate(runs):
            L = r.lay
            if ev is not None and li == dom:
                ft.set_kernel_events(ev[0], ev[1])
            L.conv_sums(r.D, r.W, r.O, [r.fault] if inject and li == i % nl else (), encode=True)
            L.verify_correct_sums(r.D, r.W, r.O, coc=True)

    def separate_step(i):
        # the same path from the separate kernels (detection re-reads O), error-free
        for r in runs:
            L = r.lay
            L.encode_input(r.D)
            L.conv(r.D, r.W, r.O)
            L.checksum_conv(ft.CO5 | ft.CO6 | ft.CO7)
            L.verify_correct(r.D, r.W, r.O)

    def conv_step(ev=None):
        for li, r in enumerate(runs):
            if ev is not None:
                ev[li][0].record()
            r.lay.conv_ws(r.D, r.W, r.O)
            if ev is not None:
                ev[li][1].record()

    def timed(fn, steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            fn(i)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / steps

    def mk_events():
        return [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in runs]

    # warm-up (also compiles nothing: kernels are prebuilt)
    for i in range(args.warmup):
        protected_step(i)
        conv_step()
    torch.cuda.synchronize()

    # ---- the timed region: K protected steps, one injected fault per step -------------
    step_events = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    for pair in step_events:   # create the HIP events outside the timed region
        for e in pair:
            e.record()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        protected_step(i, True, step_events[i])
    torch.cuda.synchronize()
    t_prot = (time.perf_counter() - t0) / args.steps

    # correctness of the last step: its faulted layer must report one CoC repair at the fault
    last = runs[(args.steps - 1) % nl]
    rep = last.lay.read_report()
    f = last.fault
    ok_fault = (rep.detected and rep.status == ft.STATUS_CORRECTED
                and rep.fixes == [(f["n"], f["m"], f["x"], f["y"], ft.SCHEME_COC)])
    clean_ok = all(not r.lay.read_report().detected for r in runs if r is not last)

    dom_conv_ms = np.array([step_events[i][0].elapsed_time(step_events[i][1]) for i in range(args.steps)])

    # ---- reference loops: the protected step again, error-free protected, unprotected and the
    # separate-kernel path, timed in four rounds of turns so that a drift of the clock over the
    # run falls on all of them alike (the overheads compare these)
    fns = [lambda i: protected_step(i, True), lambda i: protected_step(i, False), lambda i: conv_step(),
           separate_step]
    tot = [0.0] * len(fns)
    per = max(1, args.steps // 4)
    for _ in range(4):
        for k, fn in enumerate(fns):
            tot[k] += timed(fn, per)
    t_prot_r, t_clean, t_unprot, t_sep = (t / 4 for t in tot)

    # ---- per-layer stage breakdown (events between the calls) ------------------------
    stages = ["conv_sums_encode", "verify_correct_sums_coc"]
    reps = max(3, min(args.steps, 10))
    stage_ms = np.zeros((reps, nl, len(stages)))
    for k in range(reps):
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)] for _ in runs]
        for li, r in enumerate(runs):
            L = r.lay
            e = evs[li]
            e[0].record()
            L.conv_sums(r.D, r.W, r.O, encode=True)
            e[1].record()
            L.verify_correct_sums(r.D, r.W, r.O, coc=True)
            e[2].record()
        torch.cuda.synchronize()
        for li in range(nl):
            for s in range(len(stages)):
                stage_ms[k, li, s] = evs[li][s].elapsed_time(evs[li][s + 1])
    stage_med = np.median(stage_ms, axis=0)

    # the plain convolution alone, per layer (events), for the per-layer overheads
    plain_ms = np.zeros((reps, nl))
    for k in range(reps):
        evs = mk_events()
        conv_step(evs)
        torch.cuda.synchronize()
        for li in range(nl):
            plain_ms[k, li] = evs[li][0].elapsed_time(evs[li][1])
    plain_med = np.median(plain_ms, axis=0)

    per_layer = []
    for li, r in enumerate(runs):
        prot_t = float(stage_med[li].sum())
        per_layer.append({
            "layer": r.name, "gflop": round(r.flops / 1e9, 3),
            "conv_ms": round(float(plain_med[li]), 4),
            "conv_tflops": round(r.flops / float(plain_med[li]) / 1e9, 2),
            "protected_ms": round(prot_t, 4),
            "protected_tflops": round(r.flops / prot_t / 1e9, 2),
            "overhead_pct": round((prot_t / float(plain_med[li]) - 1) * 100, 2),
            "stage_ms": {s: round(float(stage_med[li][k]), 4) for k, s in enumerate(stages)},
        })

    # ---- roofline of the dominant kernel (its 128x128-tile kernel runs no other layer here)
    dom_flops = runs[dom].flops
    dom_ms = float(np.mean(dom_conv_ms))
    achieved = dom_flops / (dom_ms * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4),
                "traffic": measured_traffic() if args.workload == "alexnet" else None,
                "kernel": f"conv_kernel {dtype} with the CoC-D sums epilogue, the protected step "
                          f"({runs[dom].name})",
                "flop_per_launch": dom_flops, "avg_launch_ms": round(dom_ms, 4),
                "all_conv_tflops": round(total_flops / (float(plain_med.sum()) * 1e-3) / 1e12, 2)}

    # ---- CPU oracle on a bounded sample ----------------------------------------------
    cpu = None
    if not args.no_cpu_baseline and args.workload == "alexnet":
        cpu = cpu_baseline(cfg, args.cpu_seconds)

    value = total_flops / t_prot / 1e12
    out = {
        "metric": "protected conv TFLOP/s per layer + ABFT overhead % vs unprotected conv",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(t_prot * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": f"{cfg.name.split('_')[0]}-{nl}conv-{'fp32' if dtype == 'f32' else 'bf16'}"
                               f"-b{cfg.layers[0].n}",
                   "batch": cfg.layers[0].n, "layers": nl,
                   "faults_per_step": 1, "gflop_per_step": round(total_flops / 1e9, 3),
                   **({"bias": True} if args.bias else {}),
                   **({"groups": {"conv2": 2, "conv4": 2, "conv5": 2}} if args.groups else {})},
        "error_free_tflops": round(total_flops / t_clean / 1e12, 3),
        "unprotected_tflops": round(total_flops / t_unprot / 1e12, 3),
        "overhead_error_free_pct": round((t_clean / t_unprot - 1) * 100, 2),
        "overhead_erroneous_pct": round((t_prot_r / t_unprot - 1) * 100, 2),
        "overhead_timing": "protected (1 fault/step), error-free, unprotected and separate-kernel steps "
                           "timed in four rounds of turns after the timed region",
        "separate_kernels": {"error_free_tflops": round(total_flops / t_sep / 1e12, 3),
                             "overhead_error_free_pct": round((t_sep / t_unprot - 1) * 100, 2),
                             "note": "encode, conv_fwd, checksum_conv(Co5-Co7), verify_correct: "
                                     "five launches per layer, detection re-reads O"},
        "fault_corrected": bool(ok_fault),
        "clean_layers_clean": bool(clean_ok),
        "per_layer": per_layer,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))
    return 0 if ok_fault and clean_ok else 1


def chain_bench(args, cfg, runs, ft, torch):
    """Whole-network protected inference: every layer protected (conv_fwd_sums with the encode,
    verify_correct_sums with Co5..Co7) and ftcnn_relu_pool between layers, steps enqueued back to
    back as in the single-layer measurement; the host's recomputation check (every layer's report
    of a step) is timed on its own.  The unprotected network runs the same convolution kernels and
    the same operations between layers."""
    from paper_2003_12203_amd import network
    if any(r.lay.groups > 1 for r in runs) or args.bias:
        print("bench.py: --chain runs the dense, bias-free layers", file=sys.stderr)
        sys.exit(2)
    specs = [(l.n, l.ch, l.h, l.w, l.m, l.r, l.s, l.stride, l.pad) for l in cfg.layers]
    dtype = cfg.layers[0].dtype
    try:
        net = network.Chain(specs, dtype)
    except ft.FtcnnError as e:
        print(f"bench.py: the {cfg.name} layers do not form a chain ({e}); --chain runs AlexNet, VGG-19 "
              "and Darknet-19", file=sys.stderr)
        sys.exit(2)
    net.set_weights([r.W for r in runs])
    D0 = runs[0].D
    nl = len(runs)
    total_flops = sum(r.flops for r in runs)
    # the inputs of layers 1.. are the chain's own; free the per-layer bench tensors
    for r in runs[1:]:
        r.D = None
    faults = [[[r.fault] if li == i % nl else [] for li, r in enumerate(runs)] for i in range(nl)]

    def prot(i, inject=True):
        net.launch(D0, faults[i % nl] if inject else None)

    def plain(i):
        net.launch_plain(D0)

    def timed(fn, steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            fn(i)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / steps

    for i in range(args.warmup):
        prot(i)
        plain(i)
    # the fault-free output, for the check of the faulted steps
    prot(0, False)
    net.finish(D0)
    clean_out = net.outputs[-1].float().clone()
    def copy_clean(i):
        net.fuse_encode = False
        prot(i, False)
        net.fuse_encode = True

    # the four variants timed in turns (rounds of a quarter of the steps each), so that a drift
    # of the clock over the run falls on all of them alike
    fns = [prot, lambda i: prot(i, False), plain, copy_clean]
    tot = [0.0] * len(fns)
    per = max(1, args.steps // 4)
    for _ in range(4):
        for k, fn in enumerate(fns):
            tot[k] += timed(fn, per)
    t_prot, t_clean, t_plain, t_copy = (t / 4 for t in tot)
    # the fault of the last faulted step: run the faulted steps once more, in order
    for i in range(args.steps):
        prot(i)
    last = (args.steps - 1) % nl
    reps = net.finish(D0)
    f = runs[last].fault
    ok_fault = all((rep.fixes == [(f["n"], f["m"], f["x"], f["y"], ft.SCHEME_COC)] and
                    rep.status == ft.STATUS_CORRECTED) if li == last else not rep.detected
                   for li, rep in enumerate(reps))
    out = net.outputs[-1].float()
    rel = float(((out - clean_out).abs().max() / clean_out.abs().max().clamp_min(1e-30)).item())
    # the host's recomputation check of one step (one synchronization, the report headers of
    # every layer in one copy), after the GPU has finished
    chk = []
    for _ in range(5):
        prot(0, False)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        net.finish(D0)
        chk.append(time.perf_counter() - t0)

    # the operations between layers alone (events around them, in the unprotected pass)
    reps_n = max(3, min(args.steps, 10))
    link_ms = []
    for _ in range(reps_n):
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(nl - 1)]
        for l, lay in enumerate(net.layers):
            O = net.outputs[l]
            lay.conv_ws(D0 if l == 0 else net.inputs[l], net.W[l], O)
            if l + 1 < nl:
                evs[l][0].record()
                ft.relu_pool(O, *net.links[l], Y=net.inputs[l + 1])
                evs[l][1].record()
        torch.cuda.synchronize()
        link_ms.append(sum(a.elapsed_time(b) for a, b in evs))
    res = {
        "metric": "chained protected network, conv TFLOP/s + ABFT overhead % vs the unprotected network",
        "value": round(total_flops / t_prot / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(t_prot * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtype, "data": "synthetic",
        "config": {"workload": f"{cfg.name.split('_')[0]}-{nl}conv-chained-{'fp32' if dtype == 'f32' else 'bf16'}"
                               f"-b{cfg.layers[0].n}",
                   "batch": cfg.layers[0].n, "layers": nl, "links": [f"{k}x{k}/{s}" for k, s in net.links],
                   "faults_per_step": 1, "gflop_per_step": round(total_flops / 1e9, 3)},
        "error_free_tflops": round(total_flops / t_clean / 1e12, 3),
        "unprotected_tflops": round(total_flops / t_plain / 1e12, 3),
        "overhead_error_free_pct": round((t_clean / t_plain - 1) * 100, 2),
        "overhead_erroneous_pct": round((t_prot / t_plain - 1) * 100, 2),
        "links_ms": round(float(np.median(link_ms)), 4),
        "encode": "the link after each layer encodes the next layer's Cd1, Cd2 (ftcnn_relu_pool_encode, "
                  "ftcnn_conv_fwd_sums_given); the first layer encodes in its channels-last copy",
        "copy_encode": {"error_free_tflops": round(total_flops / t_copy / 1e12, 3),
                        "overhead_error_free_pct": round((t_copy / t_plain - 1) * 100, 2),
                        "note": "each layer encodes its input in its own channels-last copy"},
        "host_check_ms": round(float(np.median(chk)) * 1e3, 4),
        "timing": "steps enqueued back to back, the four variants (faulted, error-free, unprotected, copy-encode) "
                  "in four rounds of turns; every layer's report of a faulted run read after the timed region "
                  "(host_check_ms: that read for one step)",
        "fault_corrected": bool(ok_fault),
        "output_rel_diff_vs_fault_free": rel,
    }
    print(json.dumps(res))
    return 0 if ok_fault else 1


def measured_traffic():
    """HBM bytes per launch of the conv2 kernel from the committed FETCH_SIZE / WRITE_SIZE counter
    summary, scaled by the same counters read for a plain copy of known size.  None when the
    convolution source has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "conv2_fp32_alexnet_b64_traffic.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    h = hashlib.sha256()
    for f in ("conv_mfma.hip", "ftcnn_internal.h", "coc_tile.h", "encode_block.h"):
        with open(os.path.join(ROOT, "paper_2003_12203_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    if kv.get("source_sha256") != h.hexdigest():
        return None
    return float(kv["hbm_bytes_per_launch"])


def cpu_baseline(cfg, seconds):
    """The oracle's protected layer (encode, direct convolution, checksums, verify, correct) over the
    whole workload (five layers, batch 64, one fault in conv3), repeated until at least `seconds`
    of CPU time have been spent."""
    from oracle import core
    from oracle import workflow as wf
    import workloads as wl

    data = []
    for li, spec in enumerate(cfg.layers):
        E = core.out_extent(spec.h, spec.r, spec.stride, spec.pad)
        faults = [wf.Fault(0, 0, E // 2, E // 2, "add", value=FAULT_VALUE)] if li == 2 else []
        flops = 2.0 * spec.n * spec.m * E * E * spec.ch * spec.r * spec.s
        data.append((wl.gen_d(cfg, li), wl.gen_w(cfg, li), spec, faults, flops))
    passes, flops = 0, 0.0
    t0 = time.perf_counter()
    while True:
        for D, W, spec, faults, fl in data:
            wf.protect(D, W, spec.stride, spec.pad, spec.dtype, faults=faults)
            flops += fl
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= seconds:
            break
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": core.num_threads(),
            "kind": "oracle", "seconds": round(dt, 2),
            "sample": f"{passes} pass(es) of the whole workload (alexnet 5 conv layers, batch 64, "
                      "one fault in conv3)"}


if __name__ == "__main__":
    sys.exit(main())
