"""Every layer of every workload at its full size, through the path the benchmark times
(ftcnn_conv_fwd_sums with the encode, then ftcnn_verify_correct_sums with Co5..Co7):

* no position is flagged on the clean layer (no false positive at full size);
* 256 sampled output elements equal eq. (1) evaluated one by one by the oracle, within the
  output tolerance of the dtype;
* Cd1, Cd2 equal the oracle's block sums (Sec. 3.2) everywhere;
* Co5..Co7 at 64 sampled positions equal the oracle's convolutions of the checksum blocks, and
  So5..So7 there equal the float64 sums of the GPU's own output over all (n, m) blocks;
* the benchmark's planted fault (one additive 1e6 fault, Sec. 6.1) is detected and repaired by
  CoC at its element, back to the clean value within the repair tolerance.
"""
import numpy as np
import pytest
import torch

import paper_2003_12203_amd as ft
import workloads as wl
from gpu_util import EPI_RUN_EPS, TOL, dev, layer_for
from oracle import core
from oracle import workflow as wf

pytestmark = pytest.mark.gpu

FAULT_VALUE = 1.0e6


def _layers():
    out, seen = [], set()
    for cfg in wl.configs()[1:] + [wl.vgg19_bf16()]:
        for li, L in enumerate(cfg.layers):
            key = (cfg.name, L.dtype, L.n, L.ch, L.h, L.w, L.m, L.r, L.s, L.stride, L.pad)
            if key in seen:
                continue
            seen.add(key)
            out.append(pytest.param(cfg, li, id=f"{cfg.name}-{L.dtype}-{L.name}"))
    return out


@pytest.mark.parametrize("cfg,li", _layers())
def test_full_size_layer(cfg, li):
    spec = cfg.layers[li]
    dt = spec.dtype
    D, W = wl.gen_d(cfg, li), wl.gen_w(cfg, li)
    lay = layer_for(spec)
    Dd, Wd = dev(D, dt), dev(W, dt)
    lay.encode_weights(Wd)
    E, F = lay.E, lay.F
    print(f"[fullsize] {cfg.name} {dt} {spec.name} n{spec.n} c{spec.ch} h{spec.h} m{spec.m} r{spec.r} "
          f"u{spec.stride}", flush=True)

    # clean layer
    O = lay.empty_output()
    lay.conv_sums(Dd, Wd, O, encode=True)
    lay.verify_correct_sums(Dd, Wd, O, coc=True)
    rep = lay.read_report()
    assert not rep.detected and rep.n_flagged == 0 and rep.status == ft.STATUS_CLEAN

    rng = np.random.default_rng([12203, cfg.cid, li, 7])
    pts = np.stack([rng.integers(0, spec.n, 256), rng.integers(0, spec.m, 256),
                    rng.integers(0, E, 256), rng.integers(0, F, 256)], axis=1).astype(np.int32)
    Ot = O.float()
    got = Ot[pts[:, 0], pts[:, 1], pts[:, 2], pts[:, 3]].double().cpu().numpy()
    ref = core.conv_points(D, W, spec.stride, spec.pad, pts)
    rms = float(np.sqrt(np.mean(ref ** 2)))
    err = np.abs(got - ref) / (np.abs(ref) + rms)
    assert err.max() <= TOL[dt], (float(err.max()), pts[int(err.argmax())].tolist())

    b = {k: v.cpu().numpy() for k, v in lay.buf.items()}
    cd1, cd2 = core.block_sums(D, 0.0)
    for name, refc in (("cd1", cd1), ("cd2", cd2)):
        scale = np.abs(refc).max() + 1e-300
        assert np.abs(b[name] - refc.ravel()).max() <= 1e-12 * scale, name

    cw1, cw2 = core.block_sums(W, 0.0)
    pos = np.stack([rng.integers(0, E, 64), rng.integers(0, F, 64)], axis=1)
    zeros = np.zeros(64, dtype=np.int32)
    pq = np.stack([zeros, zeros, pos[:, 0], pos[:, 1]], axis=1).astype(np.int32)
    co5 = core.conv_points(cd1[None], cw1[None], spec.stride, spec.pad, pq)
    co6 = core.conv_points(cd1[None], cw2[None], spec.stride, spec.pad, pq)
    co7 = core.conv_points(cd2[None], cw1[None], spec.stride, spec.pad, pq)
    flat = pos[:, 0] * F + pos[:, 1]
    blocks = Ot[:, :, pos[:, 0], pos[:, 1]].double().cpu().numpy()   # [N][M][64]
    wn = np.arange(spec.n, dtype=np.float64)[:, None, None]
    wm = np.arange(spec.m, dtype=np.float64)[None, :, None]
    so5 = blocks.sum(axis=(0, 1))
    so6 = (wm * blocks).sum(axis=(0, 1))
    so7 = (wn * blocks).sum(axis=(0, 1))
    q = np.sqrt((blocks ** 2).sum(axis=(0, 1)))
    big = max(spec.n, spec.m)
    for name, refv in (("co5", co5), ("co6", co6), ("co7", co7)):
        lim = 1e-11 * (np.abs(refv) + big * q + 1e-300)
        assert np.all(np.abs(b[name][flat] - refv) <= lim), name
    # bf16: the epilogue's fp32 runs of 16 filters (every term exact, 15 roundings a run)
    mag = np.abs(blocks)
    eps = EPI_RUN_EPS if dt == "bf16" else 0.0
    slack = {"so5": eps * mag.sum(axis=(0, 1)), "so6": eps * (wm * mag).sum(axis=(0, 1)),
             "so7": eps * (wn * mag).sum(axis=(0, 1))}
    for name, refv in (("so5", so5), ("so6", so6), ("so7", so7)):
        lim = 1e-11 * (np.abs(refv) + big * q + 1e-300) + slack[name]
        assert np.all(np.abs(b[name][flat] - refv) <= lim), name

    # the benchmark's fault: planted in the convolution's output, detected and repaired by CoC
    d = wl.fault_draws(cfg.cid, li, 1)[0]
    f = {"n": int(d[0] * spec.n), "m": int(d[1] * spec.m), "x": int(d[2] * E), "y": int(d[3] * F),
         "kind": "add", "value": FAULT_VALUE}
    clean = float(Ot[f["n"], f["m"], f["x"], f["y"]])
    q_f = float(torch.sqrt((Ot[:, :, f["x"], f["y"]].double() ** 2).sum()))
    O2 = lay.empty_output()
    lay.conv_sums(Dd, Wd, O2, [f], encode=True)
    lay.verify_correct_sums(Dd, Wd, O2, coc=True)
    rep = lay.read_report()
    assert rep.detected and rep.n_flagged == 1 and rep.status == ft.STATUS_CORRECTED
    assert rep.fixes == [(f["n"], f["m"], f["x"], f["y"], ft.SCHEME_COC)]
    fixed = float(O2[f["n"], f["m"], f["x"], f["y"]].float())
    K = spec.ch * spec.r * spec.s
    tau = wf.tol_scale(K, dt, 16.0) * q_f
    assert abs(fixed - clean) <= tau + TOL[dt] * (abs(clean) + rms), (fixed, clean, tau)
