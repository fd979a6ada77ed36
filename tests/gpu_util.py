"""Helpers shared by the GPU tests: device copies, the oracle side of a comparison."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2003_12203_amd as ft
import workloads as wl
from oracle import core
from oracle import workflow as wf

TOL = {"f32": 1e-4, "bf16": 2e-2}


def dev(x: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    if dtype == "bf16":
        t = t.to(torch.bfloat16)  # values are already bf16-representable: exact
    return t.cuda()


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def layer_for(spec: wl.LayerSpec, wbase: int = 0, **policy) -> ft.Layer:
    pol = ft.make_policy(**policy)
    return ft.Layer(spec.n, spec.ch, spec.h, spec.w, spec.m, spec.r, spec.s, spec.stride, spec.pad,
                    spec.dtype, wbase, policy=pol)


def assert_close_scaled(got: np.ndarray, ref: np.ndarray, rtol: float, what: str, slack=0.0) -> None:
    """|g - o| <= rtol * (|o| + rms(o)) + slack element by element."""
    rms = float(np.sqrt(np.mean(ref.astype(np.float64) ** 2))) if ref.size else 0.0
    err = np.abs(got - ref)
    lim = rtol * (np.abs(ref) + rms) + slack
    bad = err > lim
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError(f"{what}: {int(bad.sum())} of {ref.size} elements beyond rtol {rtol}; "
                             f"first {idx.tolist()} got {got[tuple(idx[0])]} ref {ref[tuple(idx[0])]}")


# The convolution epilogue of a bf16 layer sums each run of 16 filters in fp32 before adding the
# run in fp64: every term is exact in fp32, and the 15 additions of a run round by at most 2^-24
# of the run's sum of magnitudes.
EPI_RUN_EPS = 16 * 2.0 ** -24


def epi_slack(O: np.ndarray, dtype: str, wbase: int = 0) -> dict:
    """Per position ([E][F]), the rounding the bf16 epilogue sums may carry against float64 sums
    of the stored output O [N][M][E][F]: EPI_RUN_EPS times the weighted sum of magnitudes behind
    So5, So6, So7, and half of it relative to Q5.  Zero for fp32 layers (float64 throughout)."""
    shape = O.shape[2:]
    if dtype != "bf16":
        return {k: np.zeros(shape) for k in ("so5", "so6", "so7", "q5")}
    A = np.abs(O.astype(np.float64))
    wn = (np.arange(O.shape[0]) + wbase).astype(np.float64)[:, None, None, None]
    wm = (np.arange(O.shape[1]) + wbase).astype(np.float64)[None, :, None, None]
    q = np.sqrt((A ** 2).sum(axis=(0, 1)))
    return {"so5": EPI_RUN_EPS * A.sum(axis=(0, 1)), "so6": EPI_RUN_EPS * (wm * A).sum(axis=(0, 1)),
            "so7": EPI_RUN_EPS * (wn * A).sum(axis=(0, 1)), "q5": EPI_RUN_EPS * q}


def gpu_flags(layer: ft.Layer) -> np.ndarray:
    EF = layer.E * layer.F
    torch.cuda.synchronize()
    return layer.workspace[:4 * EF].view(torch.int32).cpu().numpy().copy()


def to_ft_faults(faults) -> list:
    out = []
    for f in faults:
        d = {"n": f.n, "m": f.m, "x": f.x, "y": f.y, "kind": f.kind}
        if f.kind == "flip":
            d["bit"] = f.bit
        else:
            d["value"] = f.value
        out.append(d)
    return out


def oracle_policy_from(pol: ft._lib.Policy, wbase: int = 0) -> wf.Policy:
    return wf.Policy(rc_on=bool(pol.rc_on), clc_on=bool(pol.clc_on),
                     repair="recompute" if pol.repair == ft.REPAIR_RECOMPUTE else "checksum",
                     kappa=pol.kappa, eta=pol.eta, wbase=wbase)


def workload_shapes():
    """Distinct layer shapes of all workloads, shrunk (batch, then spatial crop) to about a GFLOP."""
    seen, out = set(), []
    cfgs = wl.configs() + [wl.vgg19_bf16()]
    for cfg in cfgs:
        for li, L in enumerate(cfg.layers):
            key = (L.ch, L.h, L.m, L.r, L.stride, L.pad, L.dtype)
            if key in seen:
                continue
            seen.add(key)
            spec = L
            for n in (3, 2, 1):
                spec = spec.with_(n=min(n, L.n))
                E = core.out_extent(spec.h, spec.r, spec.stride, spec.pad)
                if 2 * spec.n * spec.m * E * E * spec.ch * spec.r * spec.s <= 1.5e9:
                    break
            h = spec.h
            while True:
                E = core.out_extent(h, spec.r, spec.stride, spec.pad)
                if 2 * spec.n * spec.m * E * E * spec.ch * spec.r * spec.s <= 1.5e9 or h <= 2 * spec.r:
                    break
                h = int(h * 0.8)
            spec = spec.with_(h=h, w=h)
            out.append(pytest.param(cfg, li, spec, id=f"{cfg.name}-{L.name}-n{spec.n}-h{spec.h}"))
    return out
