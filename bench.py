#!/usr/bin/env python3
"""Benchmark: checksum-protected convolution layers on one MI355X.

Workload (default): the VGG-19-shaped stack of sixteen 3x3 convolution layers, fp32, batch 32
(synthetic U(0,1) inputs and He-normal weights at every layer's own input shape; layers are
independent).  ``--workload`` selects AlexNet (fp32, batch 64), VGG-19 in bf16, ResNet-18 (bf16,
batch 128) or Darknet-19 (fp32, batch 16).  One step runs the whole protected path of every layer
on one stream:

    conv_fwd_sums (+ encode of Cd1, Cd2) -> verify_correct_sums (+ Co5, Co6, Co7)

(the input checksums are encoded by the channels-last copy or by extra workgroups of the
convolution launch, the CoC-D summations are taken in its epilogue; the final launch computes the
checksum-of-checksums Co5..Co7, tests every position and runs the correction chain where one is
flagged), following the paper's error-injection protocol (Sec. 6.1): step i corrupts one output
element of layer (i mod L) inside the convolution, before its output is summed, so every step also
detects, locates and repairs one fault.  Weight checksums are encoded once at set-up (Sec. 4.2).

Reported: protected TFLOP/s (value, wall clock over the timed steps), per-step medians and
percentiles, the error-free protected and the unprotected (same convolution kernels, no ABFT work)
rates and the ABFT overheads from steps timed in rounds of turns, per-layer times, rooflines and
overheads (warm, and cold after a cache flush), a roofline entry for the dominant convolution
kernel, and the CPU oracle timed on a sample of the same workload.

``--summarize DIR [DIR ...]`` turns rocprofv3 output of a bench run into the text summaries kept
under profiles/ (no GPU work).
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
HBM_PEAK_TBS = 8.0                            # TB/s, MI355X HBM3E
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
                    help="lower bound on the CPU oracle's timed work (whole passes over the sample)")
    ap.add_argument("--workload", default="vgg19",
                    choices=["alexnet", "vgg19", "vgg19_bf16", "resnet18", "darknet19"],
                    help="layer stack to time (the default is the benchmark's workload; the others report "
                         "the same figures for the remaining configurations)")
    ap.add_argument("--summarize", nargs="+", metavar="DIR",
                    help="no GPU work: summarize rocprofv3 output directories of a bench run of --workload "
                         "(a kernel trace, FETCH_SIZE / WRITE_SIZE passes, matrix-core counter passes)")
    ap.add_argument("--summary-out", default=None, help="with --summarize: also write the traffic file of "
                    "the dominant kernel to this path")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="run a plain fp32 device copy of this size first (counter calibration)")
    ap.add_argument("--quiet", action="store_true")
    ap.add_argument("--schemes", action="store_true",
                    help="instead of the benchmark: the cost of every correction workflow (CoC, RC, ClC, FC, "
                         "recomputation) on each distinct layer, and the layerwise RC/ClC choice (one JSON "
                         "line per layer)")
    ap.add_argument("--scheme-reps", type=int, default=10)
    ap.add_argument("--fault-protocol", action="store_true",
                    help="instead of the benchmark: the erroneous-run protocol of Sec. 6.1-6.2, one epoch per "
                         "layer with a row or column fault pattern in that layer, with RC/ClC disabled and with "
                         "the layerwise RC/ClC choice (one JSON line)")
    ap.add_argument("--protocol-rounds", type=int, default=5)
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


def workload_config(name):
    import workloads as wl
    return {"alexnet": wl.config(1), "vgg19": wl.config(2), "vgg19_bf16": wl.vgg19_bf16(),
            "resnet18": wl.config(3), "darknet19": wl.config(4)}[name]


class LayerRun:
    def __init__(self, cfg, li, ft, torch, bias=False, groups=1):
        import workloads as wl
        self.spec = spec = cfg.layers[li]
        self.name = spec.name
        self.groups = groups
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


def fault_protocol(args, cfg, runs, ft, torch):
    """The erroneous-case protocol of Sec. 6.1-6.2: L epochs for L layers, epoch i planting one
    fault pattern in layer i, every layer protected.  A pattern is a corrupted row (three filters of
    one image) or column (three images of one filter) of O at the centre position (schemes.pattern),
    row with probability |D| / (|D| + |W|) (a fault in D corrupts a row, one in W a column, Sec. 4.1),
    from a seeded draw per layer.  Two policies: RC and ClC disabled on every layer (CoC, then FC),
    and the layerwise choice of Sec. 4.3 from each layer's measured workflow times.  Each epoch's
    step is timed in rounds of turns with the error-free protected step and the unprotected one;
    the overhead is the mean over the epochs of the median step against the unprotected median."""
    import statistics

    import numpy as np

    from paper_2003_12203_amd import schemes

    nl = len(runs)
    kinds, patterns = [], []
    for li, r in enumerate(runs):
        sp = r.spec
        d_el = sp.n * sp.ch * sp.h * sp.w
        w_el = sp.m * (sp.ch // r.groups) * sp.r * sp.s
        g = np.random.default_rng([12203, cfg.cid, li, 61])
        kind = "row" if g.random() < d_el / (d_el + w_el) else "col"
        kinds.append(kind)
        patterns.append(schemes.pattern(kind, sp.n, sp.m, r.lay.E, r.lay.F))
    # the layerwise choice from each layer's own workflow times (the offline profiling of Sec. 4.3)
    need = ("CoC+FC/row", "CoC+RC", "CoC+RC+FC", "CoC+FC/col", "CoC+ClC", "CoC+ClC+FC")
    choice = []
    for r in runs:
        sp = r.spec
        t = schemes.measure(r.lay, r.D, r.W, reps=args.scheme_reps, workflows=need)
        c = schemes.rc_clc_policy({k: v["us"] for k, v in t.items()}, sp.n * sp.ch * sp.h * sp.w,
                                  sp.m * (sp.ch // r.groups) * sp.r * sp.s)
        choice.append((c.rc_on, c.clc_on))
    policies = {"rc_clc_off": [ft.make_policy(rc_on=False, clc_on=False)] * nl,
                "layerwise": [ft.make_policy(rc_on=a, clc_on=b) for a, b in choice]}

    def evp():
        return (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))

    def step(pols, fl):
        for li, r in enumerate(runs):
            r.lay.policy = pols[li]
            r.lay.conv_sums(r.D, r.W, r.O, patterns[li] if li == fl else (), encode=True)
            r.lay.verify_correct_sums(r.D, r.W, r.O, coc=True)

    def plain():
        for r in runs:
            r.lay.conv_ws(r.D, r.W, r.O)

    for _ in range(2):
        step(policies["layerwise"], -1)
        plain()
    torch.cuda.synchronize()
    # the outcome of every epoch, untimed: the faulted layer corrected, every other layer clean
    outcome = {k: [None] * nl for k in policies}
    ok = True
    for k, pols in policies.items():
        for i in range(nl):
            step(pols, i)
            rep = runs[i].lay.read_report()
            used = sorted({schemes.SCHEME_NAMES.get(fx[4], str(fx[4])) for fx in rep.fixes})
            outcome[k][i] = {"status": rep.status, "schemes": used}
            ok = ok and rep.status == ft.STATUS_CORRECTED and all(
                not runs[j].lay.read_report().detected for j in range(nl) if j != i)
    # timed: per round, every epoch of both policies, the error-free step and the unprotected one,
    # queued back to back with events between them (no host wait inside a round)
    times = {"unprotected": [], "error_free": []}
    epoch_ms = {k: [[] for _ in range(nl)] for k in policies}
    for _ in range(args.protocol_rounds):
        marks = []
        for k, pols in policies.items():
            for i in range(nl):
                a, b = evp()
                a.record()
                step(pols, i)
                b.record()
                marks.append((k, i, a, b))
            for v in ("error_free", "unprotected"):
                a, b = evp()
                a.record()
                if v == "error_free":
                    step(pols, -1)
                else:
                    plain()
                b.record()
                marks.append((v, -1, a, b))
        torch.cuda.synchronize()
        for k, i, a, b in marks:
            if i >= 0:
                epoch_ms[k][i].append(a.elapsed_time(b))
            else:
                times[k].append(a.elapsed_time(b))
    base = statistics.median(times["unprotected"])
    free = statistics.median(times["error_free"])
    out = {"mode": "fault_protocol", "workload": cfg.name, "layers": nl, "rounds": args.protocol_rounds,
           "unprotected_ms": round(base, 4), "error_free_ms": round(free, 4),
           "overhead_error_free_pct": round((free / base - 1) * 100, 2),
           "patterns": {"row": kinds.count("row"), "col": kinds.count("col")}}
    for k in policies:
        med = [statistics.median(x) for x in epoch_ms[k]]
        mean = sum(med) / nl
        used = {}
        for o in outcome[k]:
            for sname in o["schemes"]:
                used[sname] = used.get(sname, 0) + 1
        out[k] = {"mean_epoch_ms": round(mean, 4), "overhead_pct": round((mean / base - 1) * 100, 2),
                  "correction_pct": round((mean / free - 1) * 100, 2),
                  "resolved_by": used,
                  "per_layer": [{"layer": runs[i].name, "pattern": kinds[i], "ms": round(med[i], 4),
                                 "extra_us": round((med[i] - free) * 1e3, 1), **outcome[k][i]}
                                for i in range(nl)]}
    out["layerwise"]["rc_on_layers"] = sum(1 for a, _ in choice if a)
    out["layerwise"]["clc_on_layers"] = sum(1 for _, b in choice if b)
    out["all_corrected"] = bool(ok)
    print(json.dumps(out), flush=True)
    return 0 if ok else 1


def kernel_key(ft, lay, path=1):
    """The convolution kernel a layer launches (ftcnn_conv_tile): layers with the same key run the
    same kernel instantiation."""
    t = ft.conv_tile(lay.desc, path)
    return (t["tm"], t["tp"], t["tk"], t["loop"], t["nhwc"], t["group_skip"])


def kernel_label(key, dtype):
    tm, tp, tk, loop, nhwc, skip = key
    kinds = {0: "register-staged", 1: "gather woven between MFMAs", 2: "two chunks in flight", 3: "direct-to-LDS",
             4: "direct-to-LDS, three stages"}
    return (f"conv_kernel {dtype} {tm}x{tp} tile, {tk}-deep chunks, {kinds[loop]}"
            f"{', channels-last' if nhwc else ', NCHW gather'}{', grouped channel skip' if skip else ''}")


def layer_roof(spec, flops, groups, dtype, peak):
    """Compulsory bytes s (N Ch H W + M (Ch/G) R S + N M E F) and the roofline min(peak, AI x 8 TB/s)
    of one layer (flops / bytes = AI; TFLOP/s = AI x TB/s)."""
    s = 4 if dtype == "f32" else 2
    E = (spec.h + 2 * spec.pad - spec.r) // spec.stride + 1
    F = (spec.w + 2 * spec.pad - spec.s) // spec.stride + 1
    nbytes = s * (spec.n * spec.ch * spec.h * spec.w + spec.m * (spec.ch // groups) * spec.r * spec.s
                  + spec.n * spec.m * E * F)
    ai = flops / nbytes
    hbm_roof = ai * HBM_PEAK_TBS
    return nbytes, ("mfma" if hbm_roof >= peak else "hbm"), min(peak, hbm_roof)


def q(a, p):
    return float(np.percentile(np.asarray(a, dtype=np.float64), p))


def stats_ms(a):
    return {"median": round(q(a, 50), 4), "p10": round(q(a, 10), 4), "p90": round(q(a, 90), 4)}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the protected layer needs no communication; see DESIGN.md for how it would shard)",
              file=sys.stderr)
        sys.exit(2)
    if args.summarize:
        return summarize_profile(args)

    import torch

    import paper_2003_12203_amd as ft
    import workloads as wl

    ft.lib()  # fails loudly if the HIP library is missing
    torch.cuda.set_device(0)
    if args.copy_calibration_mib > 0:
        # a plain copy of known size: the scale of FETCH_SIZE / WRITE_SIZE per byte moved
        a = torch.ones(args.copy_calibration_mib << 18, device="cuda")
        b = torch.empty_like(a)
        for _ in range(2):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b
    cfg = workload_config(args.workload)
    if args.groups and args.workload != "alexnet":
        print("bench.py: --groups applies to the AlexNet workload (Caffe's two groups)", file=sys.stderr)
        sys.exit(2)
    grouped = ("conv2", "conv4", "conv5") if args.groups else ()
    runs = [LayerRun(cfg, li, ft, torch, args.bias, 2 if cfg.layers[li].name in grouped else 1)
            for li in range(len(cfg.layers))]
    if args.schemes:
        scheme_table(args, cfg, runs, ft, torch)
        return
    if args.fault_protocol:
        return fault_protocol(args, cfg, runs, ft, torch)
    if args.chain:
        return chain_bench(args, cfg, runs, ft, torch)
    dtype = cfg.layers[0].dtype
    peak = MFMA_PEAK[dtype]
    nl = len(runs)
    total_flops = sum(r.flops for r in runs)
    torch.cuda.synchronize()

    # the dominant kernel for the roofline: the convolution instantiation that carries the most
    # flops of the step (on VGG-19 fp32 the 128 x 128 channels-last tile of v3-v12); every one of
    # its launches in the timed steps is bracketed by two events that the library records
    # immediately around that kernel (ftcnn_set_kernel_events: the channels-last copy launched
    # before it by the same call falls outside the pair)
    keys = [kernel_key(ft, r.lay) for r in runs]
    key_flops = {}
    for k, r in zip(keys, runs):
        key_flops[k] = key_flops.get(k, 0.0) + r.flops
    dom_key = max(key_flops, key=key_flops.get)
    dom_set = {li for li, k in enumerate(keys) if k == dom_key}

    def evp():
        return (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))

    def protected_step(i, inject=True, dom_ev=None, lay_ev=None):
        fl = i % nl if inject else -1
        for li, r in enumerate(runs):
            L = r.lay
            if lay_ev is not None:
                lay_ev[li][0].record()
            if dom_ev is not None and li in dom_set and li != fl:
                ft.set_kernel_events(*dom_ev[li])
            L.conv_sums(r.D, r.W, r.O, [r.fault] if li == fl else (), encode=True)
            L.verify_correct_sums(r.D, r.W, r.O, coc=True)
            if lay_ev is not None:
                lay_ev[li][1].record()

    def separate_step(i, lay_ev=None):
        # the same path from the separate kernels (detection re-reads O), error-free
        for r in runs:
            L = r.lay
            L.encode_input(r.D)
            L.conv(r.D, r.W, r.O)
            L.checksum_conv(ft.CO5 | ft.CO6 | ft.CO7)
            L.verify_correct(r.D, r.W, r.O)

    def conv_step(i=0, lay_ev=None):
        for li, r in enumerate(runs):
            if lay_ev is not None:
                lay_ev[li][0].record()
            r.lay.conv_ws(r.D, r.W, r.O)
            if lay_ev is not None:
                lay_ev[li][1].record()

    # warm-up (also compiles nothing: kernels are prebuilt)
    for i in range(args.warmup):
        protected_step(i)
        conv_step()
    torch.cuda.synchronize()

    # ---- the timed region: K protected steps, one injected fault per step -------------
    step_ev = [evp() for _ in range(args.steps)]
    dom_ev = [{li: evp() for li in dom_set} for _ in range(args.steps)]
    for i in range(args.steps):   # create the HIP events outside the timed region
        for e in (*step_ev[i], *(x for p in dom_ev[i].values() for x in p)):
            e.record()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step_ev[i][0].record()
        protected_step(i, True, dom_ev[i])
        step_ev[i][1].record()
    torch.cuda.synchronize()
    t_prot = (time.perf_counter() - t0) / args.steps
    timed_step_ms = [a.elapsed_time(b) for a, b in step_ev]

    # correctness of the last step: its faulted layer must report one CoC repair at the fault
    last = runs[(args.steps - 1) % nl]
    rep = last.lay.read_report()
    f = last.fault
    ok_fault = (rep.detected and rep.status == ft.STATUS_CORRECTED
                and rep.fixes == [(f["n"], f["m"], f["x"], f["y"], ft.SCHEME_COC)])
    clean_ok = all(not r.lay.read_report().detected for r in runs if r is not last)

    dom_ms, dom_fl = 0.0, 0.0
    dom_launch_ms = []
    for i in range(args.steps):
        for li, (a, b) in dom_ev[i].items():
            if li == i % nl:
                continue   # the faulted layer's launch plants its fault (another instantiation)
            ms = a.elapsed_time(b)
            dom_ms += ms
            dom_fl += runs[li].flops
            dom_launch_ms.append(ms)

    # ---- reference loops in rounds of turns: the protected step with its fault, error-free,
    # unprotected (the same convolution kernels without any ABFT work) and the separate-kernel
    # path, so that a drift of the clock over the run falls on all of them alike; per-step events
    # give medians and percentiles, per-layer events (error-free and unprotected) the per-layer
    # overheads from the same steps
    # The per-layer events sit in steps of their own ("..._layers"): an event between layers costs
    # a few microseconds of the stream, which would otherwise weigh on the small-layer workloads'
    # aggregates.
    variants = ["erroneous", "error_free", "unprotected", "separate", "error_free_layers", "unprotected_layers"]
    per = max(2, args.steps // 4)
    rounds = 4
    steps_ms = {v: [] for v in variants}
    lay_ms = {v: [[] for _ in runs] for v in ("error_free", "unprotected")}
    for _ in range(rounds):
        for v in variants:
            evs = [evp() for _ in range(per)]
            lev = [[evp() for _ in runs] for _ in range(per)] if v.endswith("_layers") else None
            torch.cuda.synchronize()
            for i in range(per):
                evs[i][0].record()
                if v == "erroneous":
                    protected_step(i, True)
                elif v.startswith("error_free"):
                    protected_step(i, False, lay_ev=lev[i] if lev else None)
                elif v.startswith("unprotected"):
                    conv_step(i, lay_ev=lev[i] if lev else None)
                else:
                    separate_step(i)
                evs[i][1].record()
            torch.cuda.synchronize()
            steps_ms[v] += [a.elapsed_time(b) for a, b in evs]
            if lev is not None:
                base = v[:-len("_layers")]
                for i in range(per):
                    for li in range(nl):
                        lay_ms[base][li].append(lev[i][li][0].elapsed_time(lev[i][li][1]))
    med = {v: q(steps_ms[v], 50) for v in variants}

    # ---- cold caches: each layer alone after a 512 MiB write (twice the 256 MB last-level
    # cache), outside the events; protected (error-free) and unprotected in turns
    cold_reps = max(3, min(10, args.steps // 4))
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    cold = {v: [[] for _ in runs] for v in ("error_free", "unprotected")}
    for k in range(cold_reps):
        for li, r in enumerate(runs):
            for v in ("error_free", "unprotected"):
                flush.fill_(k & 0xFF)
                a, b = evp()
                a.record()
                if v == "error_free":
                    r.lay.conv_sums(r.D, r.W, r.O, (), encode=True)
                    r.lay.verify_correct_sums(r.D, r.W, r.O, coc=True)
                else:
                    r.lay.conv_ws(r.D, r.W, r.O)
                b.record()
                b.synchronize()
                cold[v][li].append(a.elapsed_time(b))
    del flush

    per_layer = []
    for li, r in enumerate(runs):
        prot = q(lay_ms["error_free"][li], 50)
        plain = q(lay_ms["unprotected"][li], 50)
        cprot = q(cold["error_free"][li], 50)
        cplain = q(cold["unprotected"][li], 50)
        _, bound, roof = layer_roof(r.spec, r.flops, r.groups, dtype, peak)
        per_layer.append({
            "layer": r.name, "gflop": round(r.flops / 1e9, 3), "kernel": "x".join(map(str, keys[li][:2])),
            "conv_ms": round(plain, 4), "conv_tflops": round(r.flops / plain / 1e9, 2),
            "protected_ms": round(prot, 4), "protected_tflops": round(r.flops / prot / 1e9, 2),
            "overhead_pct": round((prot / plain - 1) * 100, 2),
            "bound": bound, "roof_tflops": round(roof, 1),
            "protected_roof_frac": round(r.flops / prot / 1e9 / roof, 4),
            "cold": {"conv_ms": round(cplain, 4), "protected_ms": round(cprot, 4),
                     "overhead_pct": round((cprot / cplain - 1) * 100, 2)},
        })
    sum_prot = sum(p["protected_ms"] for p in per_layer)
    sum_plain = sum(p["conv_ms"] for p in per_layer)
    sum_cprot = sum(p["cold"]["protected_ms"] for p in per_layer)
    sum_cplain = sum(p["cold"]["conv_ms"] for p in per_layer)

    # ---- roofline of the dominant kernel ------------------------------------------------
    achieved = dom_fl / (dom_ms * 1e-3) / 1e12
    n_launch = len(dom_launch_ms)
    dom_layers = [runs[li].name for li in sorted(dom_set)]
    traffic = measured_traffic(args.workload, dom_key, dtype)
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4),
                "traffic": None if traffic is None else round(traffic, 0),
                "kernel": kernel_label(dom_key, dtype) + ", epilogue with the CoC-D sums (the protected step)",
                "layers": dom_layers,
                "flop_per_launch": round(dom_fl / n_launch, 0),
                "avg_launch_ms": round(dom_ms / n_launch, 4), "launches": n_launch,
                "timing": "HIP events recorded by the library immediately around every launch of this kernel "
                          "in the timed steps (the faulted layer's launch excluded)"}
    if traffic is not None:
        roofline["traffic_note"] = ("calibrated FETCH_SIZE + WRITE_SIZE bytes per launch, mean over the same "
                                    "layers' launches (profiles/)")

    # ---- CPU oracle on a bounded sample ----------------------------------------------
    cpu = None
    if not args.no_cpu_baseline and not args.bias and not args.groups:
        cpu = cpu_baseline(cfg, args.cpu_seconds)

    value = total_flops / t_prot / 1e12
    wname = f"{cfg.name.split('_')[0]}-{nl}conv-{'fp32' if dtype == 'f32' else 'bf16'}-b{cfg.layers[0].n}"
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
        "config": {"workload": wname,
                   "batch": cfg.layers[0].n, "layers": nl,
                   "faults_per_step": 1, "gflop_per_step": round(total_flops / 1e9, 3),
                   **({"bias": True} if args.bias else {}),
                   **({"groups": {"conv2": 2, "conv4": 2, "conv5": 2}} if args.groups else {})},
        "step_ms": stats_ms(timed_step_ms),
        "error_free_tflops": round(total_flops / med["error_free"] / 1e9, 3),
        "unprotected_tflops": round(total_flops / med["unprotected"] / 1e9, 3),
        "overhead_error_free_pct": round((med["error_free"] / med["unprotected"] - 1) * 100, 2),
        "overhead_erroneous_pct": round((med["erroneous"] / med["unprotected"] - 1) * 100, 2),
        "variants_step_ms": {v: stats_ms(steps_ms[v]) for v in variants},
        "overhead_timing": f"medians of per-step events; the variants in {rounds} rounds of turns of "
                           f"{per} steps after the timed region; per-layer times from events between the "
                           "layers of the error-free and unprotected steps of the same rounds "
                           "(variants ..._layers: those steps carry the per-layer events, the others none)",
        "per_layer_sum_ms": {"error_free": round(sum_prot, 4), "unprotected": round(sum_plain, 4),
                             "overhead_pct": round((sum_prot / sum_plain - 1) * 100, 2),
                             "steps_with_layer_events_ms": {
                                 "error_free": round(med["error_free_layers"], 4),
                                 "unprotected": round(med["unprotected_layers"], 4)}},
        "cold_cache": {"error_free_ms": round(sum_cprot, 4), "unprotected_ms": round(sum_cplain, 4),
                       "overhead_error_free_pct": round((sum_cprot / sum_cplain - 1) * 100, 2),
                       "note": f"each layer alone after a 512 MiB write, median of {cold_reps}; sums over the "
                               "layers"},
        "separate_kernels": {"error_free_tflops": round(total_flops / med["separate"] / 1e9, 3),
                             "overhead_error_free_pct": round((med["separate"] / med["unprotected"] - 1) * 100,
                                                              2),
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


CONV_SOURCES = ("conv_mfma.hip", "ftcnn_internal.h", "coc_tile.h", "encode_block.h")


def conv_source_hash():
    """sha256 over the convolution kernel's sources: counters taken on other sources are stale."""
    import hashlib
    h = hashlib.sha256()
    for f in CONV_SOURCES:
        with open(os.path.join(ROOT, "paper_2003_12203_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def traffic_path(workload):
    return os.path.join(ROOT, "profiles", f"conv_dominant_{workload}_traffic.txt")


def measured_traffic(workload, key, dtype):
    """HBM bytes per launch of the dominant convolution kernel from the committed FETCH_SIZE /
    WRITE_SIZE summary of this workload (mean over the launches of its layers), scaled by the same
    counters read for a plain copy of known size.  None when there is no summary, when it was taken
    on another kernel, or when the convolution source has changed since."""
    path = traffic_path(workload)
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != conv_source_hash() or kv.get("kernel_key") != ",".join(map(str, key)):
        return None
    return float(kv["hbm_bytes_per_launch"])


def cpu_baseline(cfg, seconds):
    """The oracle's protected layer (encode, direct convolution, checksums, verify, correct) over a
    bounded sample of the workload: every layer at an eighth of its batch (its first images), one
    fault in the middle layer, repeated until at least `seconds` have passed."""
    from oracle import core
    from oracle import workflow as wf
    import workloads as wl

    data = []
    nb = max(1, cfg.layers[0].n // 8)
    mid = len(cfg.layers) // 2
    for li, spec in enumerate(cfg.layers):
        E = core.out_extent(spec.h, spec.r, spec.stride, spec.pad)
        F = core.out_extent(spec.w, spec.s, spec.stride, spec.pad)
        faults = [wf.Fault(0, 0, E // 2, F // 2, "add", value=FAULT_VALUE)] if li == mid else []
        flops = 2.0 * nb * spec.m * E * F * spec.ch * spec.r * spec.s
        data.append((wl.gen_d(cfg, li)[:nb].copy(), wl.gen_w(cfg, li), spec, faults, flops))
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
            "sample": f"{passes} pass(es) over all {len(cfg.layers)} layers of {cfg.name} at batch {nb} of "
                      f"{cfg.layers[0].n} (each layer's first {nb} images), one fault in layer "
                      f"{cfg.layers[mid].name}; TFLOP/s of the sample"}


# ---- rocprofv3 summaries (no GPU work) --------------------------------------------------------

def _short(name):
    s = name.replace("ftcnn::(anonymous namespace)::", "").replace("ftcnn::", "")
    if s.startswith("void "):
        s = s[5:]
    depth = 0
    for i, ch in enumerate(s):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return s[:i]
    return s


def _conv_args(short):
    """(TM, TP, TK, loop, EPI, NHWC, GRP) of a conv_kernel instantiation name, else None."""
    import re
    # the last argument, when present, marks the stream-K form of the same tile
    m = re.match(r"conv_kernel<(F32T|BF16T)<(\d+)>, (\d+), (\d+), (\d+), (\d+), (\d+|true|false), "
                 r"(true|false), (\d), (true|false), (true|false)(?:, (?:true|false))?>", short)
    if not m:
        return None
    tk = int(m.group(2))
    wm, wp, fm, fp = (int(m.group(i)) for i in range(3, 7))
    loop = {"true": 1, "false": 0}.get(m.group(7), None)
    loop = int(m.group(7)) if loop is None else loop
    return (wm * fm * 32, wp * fp * 32, tk, loop, int(m.group(9)), m.group(10) == "true", m.group(11) == "true")


def _read_csv(path):
    import csv
    with open(path) as fh:
        return list(csv.DictReader(fh))


def summarize_profile(args):
    """Summaries of rocprofv3 output directories of one bench run of --workload: per-kernel
    durations (kernel trace), per-layer convolution, copy and final-launch durations, calibrated
    HBM bytes (FETCH_SIZE, WRITE_SIZE passes) and matrix-core busy fractions
    (SQ_VALU_MFMA_BUSY_CYCLES over GRBM_GUI_ACTIVE per XCD and 1024 SIMDs).  Conv dispatches of one
    epilogue kind cycle through the layers in order (every loop of the bench runs all layers once
    in order), which attributes them to layers; a mismatch with the layer's tile is reported."""
    import glob
    import paper_2003_12203_amd as ft

    cfg = workload_config(args.workload)
    specs = cfg.layers
    nl = len(specs)
    dtype = specs[0].dtype
    peak = MFMA_PEAK[dtype]
    flops, keys1, keys0 = [], [], []
    for sp in specs:
        d = ft.make_desc(sp.n, sp.ch, sp.h, sp.w, sp.m, sp.r, sp.s, sp.stride, sp.pad, sp.dtype)
        E, F = ft.out_shape(d)
        flops.append(2.0 * sp.n * sp.m * E * F * sp.ch * sp.r * sp.s)
        t1, t0 = ft.conv_tile(d, 1), ft.conv_tile(d, 0)
        keys1.append((t1["tm"], t1["tp"], t1["tk"], t1["loop"], t1["nhwc"], t1["group_skip"]))
        keys0.append((t0["tm"], t0["tp"], t0["tk"], t0["loop"], t0["nhwc"], t0["group_skip"]))
    key_flops = {}
    for k, fl in zip(keys1, flops):
        key_flops[k] = key_flops.get(k, 0.0) + fl
    dom_key = max(key_flops, key=key_flops.get)
    dom_layers = [li for li in range(nl) if keys1[li] == dom_key]

    trace, counters = None, {}
    for d in args.summarize:
        for p in glob.glob(os.path.join(d, "*kernel_trace.csv")):
            trace = _read_csv(p)
        for p in glob.glob(os.path.join(d, "*counter_collection.csv")):
            for r in _read_csv(p):
                e = counters.setdefault(int(r["Dispatch_Id"]), {"name": _short(r["Kernel_Name"]),
                                                                  "grid": int(r["Grid_Size"])})
                e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])

    def attribute(disp):
        """disp: list of (dispatch id, short name) in dispatch order -> {id: (layer, epi, key ok)}"""
        out, seq = {}, {0: 0, 1: 0}
        for did, nm in disp:
            ca = _conv_args(nm)
            if ca is None:
                continue
            epi = 0 if ca[4] == 0 else 1
            li = seq[epi] % nl
            seq[epi] += 1
            key = (ca[0], ca[1], ca[2], ca[3], ca[5], ca[6])
            # (layer, epilogue, the kernel of the workspace path (the protected step and its plain
            # twin), the kernel of ftcnn_conv_fwd)
            out[did] = (li, ca[4], key == keys1[li], epi == 0 and key == keys0[li])
        return out

    lines = []
    emit = lines.append
    if trace:
        rows = sorted(trace, key=lambda r: int(r["Dispatch_Id"]))
        disp = [(int(r["Dispatch_Id"]), _short(r["Kernel_Name"])) for r in rows]
        att = attribute(disp)
        bad = sum(1 for v in att.values() if not (v[2] or v[3]))
        total_ns = sum(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in rows)
        byname = {}
        for r in rows:
            nm = _short(r["Kernel_Name"])
            e = byname.setdefault(nm, {"n": 0, "ns": 0, "min": 1 << 62, "max": 0, "vgpr": r["VGPR_Count"],
                                       "agpr": r["Accum_VGPR_Count"], "lds": r["LDS_Block_Size"]})
            dur = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
            e["n"] += 1
            e["ns"] += dur
            e["min"] = min(e["min"], dur)
            e["max"] = max(e["max"], dur)
        emit("| kernel | calls | avg us | min us | max us | % time | VGPR | AGPR | LDS bytes |")
        emit("|---|---:|---:|---:|---:|---:|---:|---:|---:|")
        for nm, e in sorted(byname.items(), key=lambda kv: -kv[1]["ns"]):
            if e["ns"] < 0.001 * total_ns:
                continue
            emit(f"| `{nm}` | {e['n']} | {e['ns'] / e['n'] / 1e3:.2f} | {e['min'] / 1e3:.2f} | {e['max'] / 1e3:.2f} | "
                 f"{100.0 * e['ns'] / total_ns:.2f} | {e['vgpr']} | {e['agpr']} | {e['lds']} |")
        emit("")
        emit(f"Convolution launches per layer (dispatch order; {bad} launches did not match their layer's tile):")
        emit("")
        emit("| layer | GFLOP | tile | protected launch avg us (epilogue 1) | TFLOP/s | frac of peak | "
             "plain twin avg us (epilogue 0, same tile) | TFLOP/s |")
        emit("|---|---:|---|---:|---:|---:|---:|---:|")
        per = {li: {1: [], 0: []} for li in range(nl)}
        for r in rows:
            did = int(r["Dispatch_Id"])
            if did in att and att[did][2] and att[did][1] in (0, 1):
                per[att[did][0]][att[did][1]].append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
        dom_ns, dom_n, dom_fl = 0, 0, 0.0
        for li in range(nl):
            p1, p0 = per[li][1], per[li][0]
            a1 = sum(p1) / len(p1) / 1e3 if p1 else float("nan")
            a0 = sum(p0) / len(p0) / 1e3 if p0 else float("nan")
            if li in dom_layers and p1:
                dom_ns += sum(p1)
                dom_n += len(p1)
                dom_fl += flops[li] * len(p1)
            emit(f"| {specs[li].name} | {flops[li] / 1e9:.2f} | {keys1[li][0]}x{keys1[li][1]} | {a1:.1f} | "
                 f"{flops[li] / a1 / 1e6:.1f} | {flops[li] / a1 / 1e6 / peak:.3f} | {a0:.1f} | {flops[li] / a0 / 1e6:.1f} |")
        if dom_n:
            emit("")
            emit(f"Dominant kernel ({kernel_label(dom_key, dtype)}; layers "
                 f"{', '.join(specs[li].name for li in dom_layers)}), epilogue 1: {dom_n} launches, "
                 f"{dom_ns / dom_n / 1e3:.1f} us per launch on average, {dom_fl / dom_n / 1e9:.2f} GFLOP per launch "
                 f"on average, {dom_fl / dom_ns / 1e3:.1f} TFLOP/s = {dom_fl / dom_ns / 1e3 / peak:.3f} of {peak}.")
        emit("")
    if counters:
        cd = sorted(counters.items())
        att = attribute([(did, e["name"]) for did, e in cd])
        # calibration: the largest device copies
        mib = args.copy_calibration_mib or 1024
        copies = [e for _, e in cd if "copyBuffer" in e["name"]]
        scale_f = scale_w = None
        if copies:
            big = max(copies, key=lambda e: e.get("FETCH_SIZE", 0) + e.get("WRITE_SIZE", 0))
            if big.get("FETCH_SIZE"):
                scale_f = mib * 1024.0 / big["FETCH_SIZE"]
            if big.get("WRITE_SIZE"):
                scale_w = mib * 1024.0 / big["WRITE_SIZE"]
        emit(f"Counter calibration: a {mib} MiB device copy; FETCH_SIZE scale "
             f"{'n/a' if scale_f is None else f'{scale_f:.4f}'}, WRITE_SIZE scale "
             f"{'n/a' if scale_w is None else f'{scale_w:.4f}'} (bytes moved per counted byte).")
        emit("")
        agg = {}
        for did, e in cd:
            k = (e["name"], e["grid"])
            a = agg.setdefault(k, {"n": 0})
            a["n"] += 1
            for c, v in e.items():
                if c not in ("name", "grid"):
                    a[c] = a.get(c, 0.0) + v
        cols = sorted({c for a in agg.values() for c in a if c != "n"})
        emit("| kernel | grid (threads) | dispatches | " + " | ".join(f"{c} per dispatch" for c in cols) + " |")
        emit("|---|---:|---:|" + "---:|" * len(cols))
        for (nm, grid), a in sorted(agg.items(), key=lambda kv: -kv[1].get("FETCH_SIZE", kv[1].get(
                "SQ_VALU_MFMA_BUSY_CYCLES", 0))):
            vals = [a.get(c, 0.0) / a["n"] for c in cols]
            if max(vals + [0]) == 0:
                continue
            emit(f"| `{nm}` | {grid} | {a['n']} | " + " | ".join(f"{v:.6g}" for v in vals) + " |")
        emit("")
        # achieved HBM bandwidth of the memory-bound kernels: calibrated FETCH + WRITE bytes of a
        # dispatch over its duration in the kernel trace of the same command (matched by name and grid)
        if trace and scale_f and scale_w:
            tdur = {}
            for r in trace:
                k = (_short(r["Kernel_Name"]), int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"]))
                tdur.setdefault(k, []).append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
            emit("Memory-bound kernels (FETCH + WRITE per dispatch, calibrated; duration from the kernel trace):")
            emit("")
            emit("| kernel | grid (threads) | dispatches | MB read | MB written | avg us | GB/s | of 8 TB/s |")
            emit("|---|---:|---:|---:|---:|---:|---:|---:|")
            rows_bw = []
            for (nm, grid), a in agg.items():
                if nm.startswith("conv_kernel") or "copyBuffer" in nm or "FETCH_SIZE" not in a or "WRITE_SIZE" not in a:
                    continue
                if (nm, grid) not in tdur:
                    continue
                rb = a["FETCH_SIZE"] / a["n"] * 1024 * scale_f
                wb = a["WRITE_SIZE"] / a["n"] * 1024 * scale_w
                us = sum(tdur[(nm, grid)]) / len(tdur[(nm, grid)]) / 1e3
                if rb + wb < 1e6:
                    continue
                rows_bw.append((nm, grid, a["n"], rb, wb, us))
            for nm, grid, n, rb, wb, us in sorted(rows_bw, key=lambda x: -(x[3] + x[4])):
                gbs = (rb + wb) / us / 1e3
                emit(f"| `{nm}` | {grid} | {n} | {rb / 1e6:.1f} | {wb / 1e6:.1f} | {us:.1f} | {gbs:.0f} | "
                     f"{gbs / 1e3 / HBM_PEAK_TBS:.2f} |")
            emit("")
        # the dominant kernel's traffic and matrix-core busy fraction, per launch
        fsum = wsum = busy = gui = mops = 0.0
        nd = 0
        for did, e in cd:
            if did in att and att[did][2] and att[did][1] == 1 and att[did][0] in dom_layers:
                nd += 1
                fsum += e.get("FETCH_SIZE", 0.0)
                wsum += e.get("WRITE_SIZE", 0.0)
                busy += e.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
                gui += e.get("GRBM_GUI_ACTIVE", 0.0)
                mops += e.get("SQ_INSTS_VALU_MFMA_MOPS_F32", 0.0) + e.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0)
        if nd and gui > 0:
            emit(f"Dominant kernel, epilogue 1, {nd} dispatches: SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 "
                 f"XCDs x 1024 SIMDs) = {busy / (gui / 8 * 1024):.3f}; matrix-core flops counted "
                 f"(MOPS x 512) {mops * 512 / nd / 1e9:.2f} GFLOP per dispatch.")
        if nd and scale_f and scale_w and fsum > 0 and wsum > 0:
            fb = fsum / nd * 1024 * scale_f
            wb = wsum / nd * 1024 * scale_w
            emit(f"Dominant kernel, epilogue 1, {nd} dispatches: FETCH {fb / 1e6:.2f} MB, WRITE {wb / 1e6:.2f} MB "
                 f"per launch (calibrated).")
            if args.summary_out:
                with open(args.summary_out, "w") as fh:
                    fh.write(f"# FETCH_SIZE / WRITE_SIZE per launch of the dominant convolution kernel of "
                             f"{args.workload}, mean over {nd} launches of its layers, calibrated on a {mib} MiB copy\n")
                    fh.write(f"kernel={kernel_label(dom_key, dtype)}\n")
                    fh.write(f"kernel_key={','.join(map(str, dom_key))}\n")
                    fh.write(f"layers={','.join(specs[li].name for li in dom_layers)}\n")
                    fh.write(f"source_sha256={conv_source_hash()}\n")
                    fh.write(f"fetch_bytes_per_launch={fb:.0f}\n")
                    fh.write(f"write_bytes_per_launch={wb:.0f}\n")
                    fh.write(f"hbm_bytes_per_launch={fb + wb:.0f}\n")
    print("\n".join(lines))
    return 0


if __name__ == "__main__":
    sys.exit(main())
