"""GPU detection and correction decisions against the oracle (Sec. 4.1 scenarios and seeded faults).

Every case runs through each of the library's detection paths:

* ``separate``: ftcnn_verify then ftcnn_correct, faults injected into the stored O;
* ``fused``: ftcnn_verify_correct (one detection read of O, correction in the same launch);
* ``epilogue``: ftcnn_conv_fwd_sums (summations in the convolution's epilogue, faults planted
  in its outputs before they are summed) then ftcnn_verify_correct_sums;
* ``two_launch``: the same with the input checksums encoded inside the convolution launch and
  Co5..Co7 computed inside the final launch (ftcnn_protected_conv).  Cases that corrupt D or a
  checksum between the encode and the convolution do not apply to it.

Decisions are compared in decision-oracle mode: the oracle's workflow runs on
the GPU's own faulted output (before correction), so only the float64 order of
summation differs between the two sides.  Decisions, located indices and the
fix lists must then agree exactly; repaired values must agree to the output
tolerance (bit for bit on integer data).
"""
import numpy as np
import pytest
import torch

import paper_2003_12203_amd as ft
import workloads as wl
from gpu_util import TOL, assert_close_scaled, dev, gpu_flags, host, layer_for, to_ft_faults
from oracle import workflow as wf
from scenarios import all_scenarios

pytestmark = pytest.mark.gpu

SCN = all_scenarios()


def _flat(spec, target, index):
    if target == "cd1":
        c, h, w = index
        return (c * spec.h + h) * spec.w + w
    c, r, s = index
    return (c * spec.r + r) * spec.s + s


MODES = ["separate", "fused", "epilogue", "two_launch"]


def run_gpu(spec, D, W, faults, pol_kw, wbase=0, hook=None, mode="separate"):
    """Protected layer on the GPU; returns (first report, final status, faulted O, final O, flags)."""
    lay = layer_for(spec, wbase=wbase, **pol_kw)
    Dd, Wd = dev(D, spec.dtype), dev(W, spec.dtype)
    lay.encode_weights(Wd)
    if mode == "two_launch":
        assert hook is None, "no point between encode and convolution in the two-launch path"
    else:
        lay.encode_input(Dd)
    if hook is not None:
        t = hook["target"]
        if t == "D":
            Dd[hook["index"]] += hook["add"]
        elif t == "W":
            Wd[hook["index"]] += hook["add"]
        else:
            lay.buf[t][_flat(spec, t, hook["index"])] += hook["add"]
    O = lay.empty_output()
    if mode == "two_launch":
        lay.conv_sums(Dd, Wd, O, to_ft_faults(faults), encode=True)
        O_faulty = host(O)
        lay.verify_correct_sums(Dd, Wd, O, coc=True)
    elif mode == "epilogue":
        lay.conv_sums(Dd, Wd, O, to_ft_faults(faults))
        O_faulty = host(O)
        lay.checksum_conv(ft.CO5 | ft.CO6 | ft.CO7)
        lay.verify_correct_sums(Dd, Wd, O)
    else:
        lay.conv(Dd, Wd, O)
        lay.checksum_conv(ft.CO5 | ft.CO6 | ft.CO7)
        if faults:
            lay.inject(O, to_ft_faults(faults))
        O_faulty = host(O)
        if mode == "fused":
            lay.verify_correct(Dd, Wd, O)
        else:
            lay.verify(O)
            lay.correct(Dd, Wd, O)
    rep = lay.read_report()
    flags = gpu_flags(lay)
    status = rep.status
    if status == ft.STATUS_NEEDS_RECOMPUTE:
        if mode == "two_launch":
            lay.conv_sums(Dd, Wd, O, encode=True)
            lay.verify_correct_sums(Dd, Wd, O, coc=True)
        elif mode == "epilogue":
            lay.conv_sums(Dd, Wd, O)
            lay.verify_correct_sums(Dd, Wd, O)
        else:
            lay.conv(Dd, Wd, O)
            lay.verify(O)
        status = ft.STATUS_FAILED if lay.read_report().detected else ft.STATUS_RECOMPUTED
    return rep, status, O_faulty, host(O), flags


def compare(spec, D, W, rep, status, O_faulty, O_final, flags, policy, hook_fn=None, exact=False):
    res = wf.protect(D, W, spec.stride, spec.pad, spec.dtype, policy, O_in=O_faulty, after_encode=hook_fn)
    orep = res.report
    assert rep.detected == orep.detected
    assert sorted(np.flatnonzero(flags).tolist()) == orep.flagged
    assert rep.n_flagged == orep.n_flagged
    assert rep.resolved_by[1:] == orep.resolved_by()[1:], (rep.resolved_by, orep.resolved_by())
    assert rep.fixes == orep.fixes
    assert status == orep.status
    if exact:
        np.testing.assert_array_equal(O_final, res.O)
    else:
        assert_close_scaled(O_final, res.O, TOL[spec.dtype], "corrected O")
    return res


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("scn", SCN, ids=[s.name for s in SCN])
def test_scenario_matches_oracle(scn, mode):
    if mode == "two_launch" and scn.hook is not None:
        pytest.skip("corrupts D or a checksum between the encode and the convolution")
    D, W = scn.inputs()
    pol = scn.oracle_policy()
    kw = dict(rc_on=pol.rc_on, clc_on=pol.clc_on, repair=pol.repair, kappa=pol.kappa, eta=pol.eta)
    rep, status, O_faulty, O_final, flags = run_gpu(scn.spec, D, W, scn.faults, kw, pol.wbase, scn.hook, mode)
    res = compare(scn.spec, D, W, rep, status, O_faulty, O_final, flags, pol, scn.oracle_hook(),
                  exact=scn.data == "int")
    # and the outcome Sec. 4.1 predicts
    assert status == scn.expect_status
    if scn.expect_schemes:
        got = {s for s in range(1, 7) if rep.resolved_by[s]}
        assert got <= set(scn.expect_schemes), rep.resolved_by
    if scn.data == "int" and scn.expect_clean:
        np.testing.assert_array_equal(O_final, res.O_clean)


def _bitflip_faults(O, draws, dtype):
    """Sign/exponent bit flips on elements with |O| >= rms(O); the result must stay finite."""
    rms = np.sqrt(np.mean(O ** 2))
    big = np.argwhere(np.abs(O) >= rms)
    nbits, lo = (32, 23) if dtype == "f32" else (16, 7)
    out = []
    for d in draws:
        n, m, x, y = (int(v) for v in big[int(d[0] * len(big))])
        bit = lo + int(d[4] * (nbits - lo))
        f = wf.Fault(n, m, x, y, "flip", bit)
        tmp = O[n:n + 1, m:m + 1, x:x + 1, y:y + 1].copy()
        wf.apply_faults(tmp, dtype, [wf.Fault(0, 0, 0, 0, "flip", bit)])
        if np.isfinite(tmp).all() and tmp[0, 0, 0, 0] != O[n, m, x, y]:
            out.append(f)
    return out


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("trial", range(12))
def test_tiny_bitflip_detected_and_corrected(trial, mode):
    """The single-layer workload: one seeded bit flip in O, detected and corrected as the oracle does."""
    cfg = wl.config(0)
    spec = cfg.layers[0]
    D, W = wl.gen_d(cfg, 0), wl.gen_w(cfg, 0)
    clean = wf.protect(D, W, spec.stride, spec.pad, spec.dtype).O_clean
    faults = _bitflip_faults(clean, wl.fault_draws(0, 0, 1, variant=trial + 1), "f32")
    if not faults:
        pytest.skip("draw produced a non-finite or no-op flip")
    rep, status, O_faulty, O_final, flags = run_gpu(spec, D, W, faults, {}, mode=mode)
    compare(spec, D, W, rep, status, O_faulty, O_final, flags, wf.Policy())
    assert rep.detected and status == ft.STATUS_CORRECTED
    assert_close_scaled(O_final, clean, 1e-4, "recovered O")


def _pattern_faults(O, draws, count):
    """2-4 faults: a same-row group, a same-column group or scattered single blocks (one draw each)."""
    N, M, E, F = O.shape
    rms = float(np.sqrt(np.mean(O ** 2)))
    out = []
    for d in draws[:count]:
        kind = int(d[4] * 3)
        mag = (1.0 + 7.0 * d[5]) * rms * (1 if d[6] < 0.5 else -1) * 64
        n, m, x, y = int(d[0] * N), int(d[1] * M), int(d[2] * E), int(d[3] * F)
        if kind == 0:      # blocks of one row at one position
            for k in range(3):
                out.append(wf.Fault(n, (m + 5 * k) % M, x, y, "add", value=mag * (1 + 0.37 * k)))
        elif kind == 1:    # blocks of one column at one position
            for k in range(3):
                out.append(wf.Fault((n + 3 * k) % N, m, x, y, "add", value=mag * (1 + 0.41 * k)))
        else:              # one block, its own position
            out.append(wf.Fault(n, m, x, y, "add", value=mag))
    return out


@pytest.mark.parametrize("mode", ["fused", "epilogue", "two_launch"])
@pytest.mark.parametrize("li", [1, 5, 13, 14])
def test_darknet_multi_fault(li, mode):
    """Darknet-shaped layers (reduced batch and size) with seeded multi-fault injection."""
    cfg = wl.config(4)
    L = cfg.layers[li]
    spec = L.with_(n=4, h=min(L.h, 26), w=min(L.w, 26))
    D, W = wl.gen_d(cfg, li, spec), wl.gen_w(cfg, li, spec)
    clean = wf.protect(D, W, spec.stride, spec.pad, spec.dtype).O_clean
    draws = wl.fault_draws(4, li, 4)
    faults = _pattern_faults(clean, draws, 2 + int(draws[0, 6] * 3))
    rep, status, O_faulty, O_final, flags = run_gpu(spec, D, W, faults, {}, mode=mode)
    compare(spec, D, W, rep, status, O_faulty, O_final, flags, wf.Policy())
    assert rep.detected
    assert status in (ft.STATUS_CORRECTED, ft.STATUS_RECOMPUTED)
    assert_close_scaled(O_final, clean, 1e-3, "recovered O")


@pytest.mark.parametrize("mode", MODES)
def test_correct_is_noop_when_clean(mode):
    spec = wl.config(1).layers[3].with_(n=2)
    cfg = wl.config(1)
    D, W = wl.gen_d(cfg, 3, spec), wl.gen_w(cfg, 3, spec)
    rep, status, O_faulty, O_final, flags = run_gpu(spec, D, W, [], {}, mode=mode)
    assert not rep.detected and status == ft.STATUS_CLEAN and rep.fixes == []
    np.testing.assert_array_equal(O_faulty, O_final)


def test_report_capacity_overflow_counts_all():
    """More repairs than report slots: n_fixes still counts every repair."""
    scn = [s for s in SCN if s.name == "w_fault_col"][0]
    D, W = scn.inputs()
    lay = layer_for(scn.spec)
    lay.cap = 10
    lay.report = torch.zeros(ft.report_bytes(10), dtype=torch.uint8, device="cuda")
    Dd, Wd = dev(D, "f32"), dev(W, "f32")
    lay.encode_weights(Wd)
    lay.encode_input(Dd)
    Wd[scn.hook["index"]] += scn.hook["add"]
    O = lay.empty_output()
    lay.conv(Dd, Wd, O)
    lay.checksum_conv(ft.CO5 | ft.CO6 | ft.CO7)
    lay.verify(O)
    lay.correct(Dd, Wd, O)
    rep = lay.read_report()
    assert rep.n_fixes == 81 * 6 and len(rep.fixes) == 10 and rep.cap_fixes == 10
