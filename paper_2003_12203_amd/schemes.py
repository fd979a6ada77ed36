"""Per-layer cost of the correction schemes and the layerwise choice of RC and ClC.

The multischeme workflow (Sec. 4.3) always detects with CoC-D and corrects in the order CoC,
RC, ClC, FC, then recomputation.  RC and ClC are switched per layer: with t0 the runtime of
the workflow CoC+FC, t1 that of CoC+RC and t2 that of CoC+RC+FC (offline profiling), RC
saves p_r (t0 - t1) on the row errors it corrects and costs p_c (t2 - t0) on the column errors
it cannot, so it is worth enabling when the first exceeds the second; the ratio p_r / p_c of
row to column errors is estimated as the ratio of the element counts of D and W.  ClC is the
mirror image (it corrects column errors and fails on row errors).

A row error here is one corrupted input block D_n: every output block O[n][m] of that image
can be wrong at the same position.  A column error is one corrupted filter W_m: every O[n][m]
of that filter.  The workflows are timed by planting such patterns in the convolution's
output (inside its epilogue, before the output is summed) and timing the protected step
against the same step without faults.
"""
from __future__ import annotations

import dataclasses
import statistics
from typing import Dict, List, Sequence, Tuple

# workflow name -> (fault pattern, rc_on, clc_on, schemes expected to resolve it)
WORKFLOWS: Dict[str, Tuple[str, bool, bool, Tuple[str, ...]]] = {
    "CoC": ("single", True, True, ("coc",)),
    "CoC+FC/row": ("row", False, False, ("fc",)),
    "CoC+RC": ("row", True, False, ("rc",)),
    "CoC+RC+FC": ("col", True, False, ("fc",)),
    "CoC+FC/col": ("col", False, False, ("fc",)),
    "CoC+ClC": ("col", False, True, ("clc",)),
    "CoC+ClC+FC": ("row", False, True, ("fc",)),
    "recompute": ("square", True, True, ("unresolved",)),
}

def _frac_dist(r: float) -> float:
    return abs(r - round(r))


def _values(kind: str, pts: List[Tuple[int, int]], n: int, m: int) -> List[float]:
    """Fault magnitudes k * 2^14 (k in [64, 255]: exact in bf16, about 1e6 to 4e6, all positive so
    no two cancel in Co5 - So5), searched from a fixed seed so that every block-location ratio a
    scheme must fail on is at least a quarter away from an integer.  With hand-picked values
    such a ratio can land on an integer, and a wrong block then repairs into consistent
    checksums (Sec. 4.1: a multi-block error can defeat CoC)."""
    import numpy as np

    rng = np.random.default_rng([12203, len(pts), n, m])
    for _ in range(10000):
        k = rng.integers(64, 256, size=len(pts)).astype(np.float64)
        ratios = []
        if kind == "row":        # one image: CoC's filter ratio (and ClC's in that row)
            ratios.append(sum(b * w for (_, b), w in zip(pts, k)) / k.sum())
        elif kind == "col":      # one filter: CoC's image ratio (and RC's in that column)
            ratios.append(sum(a * w for (a, _), w in zip(pts, k)) / k.sum())
        elif kind == "square":   # CoC's two ratios, RC's two columns, ClC's two rows
            ratios.append(sum(a * w for (a, _), w in zip(pts, k)) / k.sum())
            ratios.append(sum(b * w for (_, b), w in zip(pts, k)) / k.sum())
            for key, other in ((1, 0), (0, 1)):
                for val in {q[key] for q in pts}:
                    sel = [(q, w) for q, w in zip(pts, k) if q[key] == val]
                    ratios.append(sum(q[other] * w for q, w in sel) / sum(w for _, w in sel))
        if all(_frac_dist(r) >= 0.25 for r in ratios):
            return [float(v) * 16384.0 for v in k]
    raise ValueError("no fault magnitudes keep the location ratios away from integers")


def pattern(kind: str, n: int, m: int, e: int, f: int) -> List[dict]:
    """Additive faults of one kind at the centre position of an [n][m][e][f] output.

    single: one block; row: three filters of one image; col: three images of one filter;
    square: a 2 x 2 set of blocks (two images x two filters), which neither RC nor ClC nor FC
    can resolve (Sec. 4.1).  Rows and columns need at least three blocks; square needs two."""
    x, y = e // 2, f // 2
    ms = sorted({0, m // 2, m - 1})
    ns = sorted({0, n // 2, n - 1})
    if kind == "single":
        pts = [(n // 2, m // 2)]
    elif kind == "row":
        if len(ms) < 3:
            raise ValueError("a row pattern needs at least three filters")
        pts = [(n // 2, mm) for mm in ms]
    elif kind == "col":
        if len(ns) < 3:
            raise ValueError("a column pattern needs at least three images")
        pts = [(nn, m // 2) for nn in ns]
    elif kind == "square":
        if n < 2 or m < 2:
            raise ValueError("a square pattern needs two images and two filters")
        pts = [(0, 0), (0, m - 1), (n - 1, 0), (n - 1, m - 1)]
    else:
        raise ValueError(kind)
    vals = _values(kind, pts, n, m)
    return [{"n": a, "m": b, "x": x, "y": y, "kind": "add", "value": v} for (a, b), v in zip(pts, vals)]


@dataclasses.dataclass
class Choice:
    rc_on: bool
    clc_on: bool
    rc_gain: float       # p_r (t0 - t1) / p_c, per unit of p_c
    rc_loss: float       # (t2 - t0)
    clc_gain: float      # (t0' - t1')
    clc_loss: float      # p_r (t2' - t0') / p_c


def rc_clc_policy(t: Dict[str, float], d_elems: int, w_elems: int) -> Choice:
    """The layerwise switch of Sec. 4.3 from the workflow times t (any unit, same for all):
    RC on iff p_r (t0 - t1) > p_c (t2 - t0), ClC on iff p_c (t0' - t1') > p_r (t2' - t0'),
    with p_r / p_c = |D| / |W| (element counts)."""
    ratio = float(d_elems) / float(w_elems)
    rc_gain = ratio * (t["CoC+FC/row"] - t["CoC+RC"])
    rc_loss = t["CoC+RC+FC"] - t["CoC+FC/col"]
    clc_gain = t["CoC+FC/col"] - t["CoC+ClC"]
    clc_loss = ratio * (t["CoC+ClC+FC"] - t["CoC+FC/row"])
    return Choice(rc_gain > rc_loss, clc_gain > clc_loss, rc_gain, rc_loss, clc_gain, clc_loss)


SCHEME_NAMES = {1: "coc", 2: "rc", 3: "clc", 4: "fc", 5: "cksum", 6: "unresolved"}


def measure(lay, D, W, reps: int = 10, workflows: Sequence[str] = tuple(WORKFLOWS)) -> Dict[str, dict]:
    """Time the protected step (conv_fwd_sums with the encode, verify_correct_sums with Co5..Co7)
    of one layer without faults and with each workflow's pattern; median of `reps` runs each,
    in microseconds, with the schemes the report says resolved the flagged positions."""
    import torch

    import paper_2003_12203_amd as ft

    n, m = lay.desc.n, lay.desc.m
    O = lay.empty_output()
    saved = lay.policy

    def run(faults, pol):
        lay.policy = pol
        lay.conv_sums(D, W, O, faults, encode=True)
        lay.verify_correct_sums(D, W, O, coc=True)

    def timeit(faults, pol):
        run(faults, pol)
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            ev[0].record()
            run(faults, pol)
            ev[1].record()
            ev[1].synchronize()
            ts.append(ev[0].elapsed_time(ev[1]) * 1e3)
        return statistics.median(ts)

    out = {}
    try:
        base_pol = ft.make_policy()
        out["error-free"] = {"us": timeit([], base_pol), "resolved": []}
        for name in workflows:
            kind, rc_on, clc_on, _ = WORKFLOWS[name]
            try:
                faults = pattern(kind, n, m, lay.E, lay.F)
            except ValueError:
                continue
            pol = ft.make_policy(rc_on=rc_on, clc_on=clc_on)
            us = timeit(faults, pol)
            rep = lay.read_report()
            resolved = sorted({SCHEME_NAMES.get(s, str(s)) for s in (fx[4] for fx in rep.fixes)})
            if rep.status == ft.STATUS_RECOMPUTED or rep.resolved_by[6]:
                resolved = sorted(set(resolved) | {"unresolved"})
            out[name] = {"us": us, "resolved": resolved, "status": rep.status}
    finally:
        lay.policy = saved
    return out
