"""Bias (Sec. 5.1) through the C ABI against the oracle.

* the bias sums of ftcnn_encode(which = 2) equal sum_m b[m] and sum_m (m + wbase) b[m];
* the protected path with a bias (conv_fwd_sums + verify_correct_sums): O equals eq. (1) plus
  the bias (the oracle, within the dtype's tolerance) and bitwise ftcnn_conv_fwd_bias through
  the same kernels; Co5..Co7 stay the bias-free checksums; So5..So7 are the raw summations; a
  clean layer is not flagged (the Table 5 shares are applied);
* every correction workflow with a bias, on integer data: the schemes, repairs and final
  output are the oracle's (fp32 exactly);
* the separate-kernel path (conv_fwd_bias, checksum_conv, verify, correct) with a bias.
"""
import numpy as np
import pytest
import torch

import paper_2003_12203_amd as ft
import workloads as wl
from gpu_util import epi_slack, TOL, assert_close_scaled, dev, host, layer_for
from oracle import core
from oracle import workflow as wf
from paper_2003_12203_amd import schemes

pytestmark = pytest.mark.gpu

SHAPES = [
    # n, ch, h, m, r, stride, pad, dtype
    (4, 3, 17, 24, 3, 1, 1, "f32"),      # NCHW gather
    (5, 32, 12, 40, 3, 1, 1, "f32"),     # channels-last, CoC in the conv launch
    (6, 64, 9, 48, 3, 2, 1, "bf16"),     # channels-last, strided
    (40, 32, 7, 32, 1, 1, 0, "f32"),     # split images, 1x1
]


def _bias(m, seed, integer=False):
    g = np.random.default_rng([12203, 61, seed])
    return (g.integers(-5, 6, size=m) if integer else g.normal(0.0, 0.5, size=m)).astype(np.float32)


@pytest.mark.parametrize("wbase", [0, 1])
def test_bias_sums(wbase):
    spec = wl.LayerSpec("b", 3, 4, 6, 6, 37, 3, 3, 1, 1, "f32")
    lay = layer_for(spec, wbase=wbase)
    b = _bias(spec.m, 1)
    lay.set_bias(torch.from_numpy(b).cuda())
    torch.cuda.synchronize()
    cb = lay.buf["cb"].cpu().numpy()
    b64 = b.astype(np.float64)
    np.testing.assert_allclose(cb[0], b64.sum(), rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(cb[1], ((np.arange(spec.m) + wbase) * b64).sum(), rtol=1e-14, atol=1e-13)


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "-".join(map(str, s)))
def test_protected_path_with_bias(shape):
    n, ch, h, m, r, u, p, dt = shape
    spec = wl.LayerSpec("b", n, ch, h, h, m, r, r, u, p, dt)
    cfg = wl.Config(94, "bias", (spec,), "uniform", "he")
    D, W = wl.gen_d(cfg, 0, spec), wl.gen_w(cfg, 0, spec)
    b = _bias(m, sum(shape[:7]))
    lay = layer_for(spec)
    Dd, Wd = dev(D, dt), dev(W, dt)
    lay.encode_weights(Wd)
    lay.set_bias(torch.from_numpy(b).cuda())
    print(f"[bias] {shape}", flush=True)
    O = lay.empty_output()
    lay.conv_sums(Dd, Wd, O, encode=True)
    lay.verify_correct_sums(Dd, Wd, O, coc=True)
    rep = lay.read_report()
    assert not rep.detected and rep.n_flagged == 0
    ref = core.conv(D, W, u, p) + b.astype(np.float64)[None, :, None, None]
    assert_close_scaled(host(O), ref, TOL[dt], "O with bias")
    O2 = lay.empty_output()
    lay.conv_ws(Dd, Wd, O2)   # ftcnn_conv_fwd_bias through the protected path's kernels
    iv = torch.int16 if dt == "bf16" else torch.int32
    assert torch.equal(O.view(iv), O2.view(iv))
    bb = {k: v.cpu().numpy() for k, v in lay.buf.items()}
    cd1, cd2 = wf.encode(D, 0)
    ck = wf.Checksums(cd1, cd2, *wf.encode(W, 0))
    wf.coc_checksums(ck, u, p)
    for name, refc in (("co5", ck.co5), ("co6", ck.co6), ("co7", ck.co7)):
        assert_close_scaled(bb[name].reshape(refc.shape), refc, 1e-11, name)
    so5, so6, so7, q5, flags = wf.verify(host(O), ck.co5, ch * r * r, dt, wf.Policy(),
                                         wf.BiasTerms.make(b, n, m, 0))
    assert not flags.any()
    slack = epi_slack(host(O), dt)
    for name, refs in (("so5", so5), ("so6", so6), ("so7", so7)):
        assert_close_scaled(bb[name].reshape(refs.shape), refs, 1e-11, name, slack[name])


@pytest.mark.parametrize("name", list(schemes.WORKFLOWS))
@pytest.mark.parametrize("ch,dt", [(4, "f32"), (32, "f32"), (32, "bf16")])
def test_workflows_with_bias_match_oracle(name, ch, dt):
    kind, rc_on, clc_on, expect = schemes.WORKFLOWS[name]
    spec = wl.LayerSpec("b", 6, ch, 9, 9, 8, 3, 3, 1, 1, dt)
    D, W = wl.gen_int_d(spec, 23), wl.gen_int_w(spec, 23)
    b = _bias(spec.m, 23, integer=True)
    pattern = schemes.pattern(kind, spec.n, spec.m, 9, 9)
    pol = dict(rc_on=rc_on, clc_on=clc_on)
    lay = layer_for(spec, **pol)
    Dd, Wd = dev(D, dt), dev(W, dt)
    lay.encode_weights(Wd)
    lay.set_bias(torch.from_numpy(b).cuda())
    O = lay.empty_output()
    lay.conv_sums(Dd, Wd, O, pattern, encode=True)
    torch.cuda.synchronize()
    O_faulty = host(O)
    lay.verify_correct_sums(Dd, Wd, O, coc=True)
    rep = lay.read_report()
    res = wf.protect(D, W, 1, 1, dt, wf.Policy(**pol), O_in=O_faulty, bias=b.astype(np.float64))
    assert rep.detected and res.report.detected
    assert rep.n_flagged == res.report.n_flagged
    got = tuple(sorted({schemes.SCHEME_NAMES[f[4]] for f in rep.fixes}
                       | ({"unresolved"} if rep.resolved_by[6] else set())))
    assert got == expect
    if expect != ("unresolved",):
        assert rep.fixes == res.report.fixes
        if dt == "f32":
            np.testing.assert_array_equal(host(O), res.O)
        else:
            assert_close_scaled(host(O), res.O, TOL[dt], "repaired O")


def test_separate_path_with_bias():
    spec = wl.LayerSpec("b", 5, 8, 10, 10, 12, 3, 3, 1, 1, "f32")
    D, W = wl.gen_int_d(spec, 31), wl.gen_int_w(spec, 31)
    b = _bias(spec.m, 31, integer=True)
    lay = layer_for(spec)
    Dd, Wd = dev(D, "f32"), dev(W, "f32")
    lay.encode_weights(Wd)
    lay.set_bias(torch.from_numpy(b).cuda())
    lay.encode_input(Dd)
    O = lay.empty_output()
    lay.conv(Dd, Wd, O)
    clean = host(O).copy()
    np.testing.assert_array_equal(clean, core.conv(D, W, 1, 1) + b.astype(np.float64)[None, :, None, None])
    lay.checksum_conv(ft.CO5 | ft.CO6 | ft.CO7)
    lay.verify_correct(Dd, Wd, O)
    assert not lay.read_report().detected
    lay.inject(O, [{"n": 2, "m": 7, "x": 4, "y": 5, "kind": "add", "value": 321.0}])
    lay.verify(O)
    lay.correct(Dd, Wd, O)
    rep = lay.read_report()
    assert rep.detected and rep.status == ft.STATUS_CORRECTED
    assert rep.fixes == [(2, 7, 4, 5, ft.SCHEME_COC)]
    np.testing.assert_array_equal(host(O), clean)
    # the final launch reading Co5..Co7 from checksum_conv (no Co in the conv launch)
    O2 = lay.empty_output()
    lay.conv_sums(Dd, Wd, O2, [{"n": 1, "m": 3, "x": 2, "y": 2, "kind": "add", "value": 77.0}])
    lay.verify_correct_sums(Dd, Wd, O2, coc=False)
    rep = lay.read_report()
    assert rep.fixes == [(1, 3, 2, 2, ft.SCHEME_COC)]
    np.testing.assert_array_equal(host(O2), clean)
