"""Whole outputs at full size: for one full-size layer per convolution kernel that the workloads
launch (tests/fullsize_cases.py), every element of O against the oracle's float64 eq. (1), twice:

* workload data (U(0,1) inputs, He-normal weights): |g - o| <= rtol (|o| + rms(o)) at every
  element, rtol 1e-4 (fp32) or 2e-2 (bf16);
* integer data (D in {0..3}, W in {-2..2}, integer bias): every partial sum is an integer below
  2^24, so fp32 accumulation is exact and O must equal the oracle's rounded value bit for bit.

Path 1 (the protected path, ftcnn_conv_fwd_sums with the encode, then ftcnn_verify_correct_sums
with Co5..Co7) also checks, at every position: no false positive; Cd1, Cd2 against the oracle's
block sums (Sec. 3.2); Co5..Co7 against the oracle's convolutions of checksum blocks; So5..So7
and Q5 against the oracle's float64 summations of the stored output (Sec. 3.6); and that the
unprotected twin (ftcnn_conv_fwd_ws, the overhead baseline) stores the same bits.  Path 0 is
ftcnn_conv_fwd.
"""
import numpy as np
import pytest
import torch

import paper_2003_12203_amd as ft
import workloads as wl
from fullsize_cases import CASES, case_id, layer
from gpu_util import TOL, assert_close_scaled, dev, epi_slack, host
from oracle import workflow as wf

pytestmark = pytest.mark.gpu


def _bias(m: int, integer: bool, seed: int) -> np.ndarray:
    g = np.random.default_rng([12203, 17, seed])
    if integer:
        return g.integers(-3, 4, size=m).astype(np.float32)
    return g.uniform(-0.1, 0.1, size=m).astype(np.float32)


def _oracle_out(D, W, spec, groups, b):
    O = wf.grouped_conv(D, W, groups, spec.stride, spec.pad)
    if b is not None:
        O += b.astype(np.float64)[None, :, None, None]
    return wf.store(O, spec.dtype)


def _run_path1(spec, groups, D, W, b):
    dt = spec.dtype
    lay = ft.Layer(spec.n, spec.ch, spec.h, spec.w, spec.m, spec.r, spec.s, spec.stride, spec.pad, dt,
                   groups=groups)
    Dd, Wd = dev(D, dt), dev(W, dt)
    lay.encode_weights(Wd)
    if b is not None:
        lay.set_bias(torch.from_numpy(b).cuda())
    O = lay.empty_output()
    lay.conv_sums(Dd, Wd, O, encode=True)
    lay.verify_correct_sums(Dd, Wd, O, coc=True)
    rep = lay.read_report()
    assert not rep.detected and rep.n_flagged == 0 and rep.status == ft.STATUS_CLEAN, rep
    O_plain = lay.empty_output()
    lay.conv_ws(Dd, Wd, O_plain)
    iv = torch.int16 if dt == "bf16" else torch.int32
    assert torch.equal(O.view(iv), O_plain.view(iv)), "the unprotected twin stores other bits"
    bufs = {k: v.cpu().numpy() for k, v in lay.buf.items()}
    del O_plain, Dd, Wd
    return host(O), bufs, lay


def _check_checksums(spec, groups, D, W, b, Og, bufs, exact):
    """Cd1, Cd2, Co5..Co7 and So5..So7, Q5 at every position against the oracle."""
    dt = spec.dtype
    cd1, cd2 = wf.encode(D, 0)
    cw1, cw2 = wf.encode_weights(W, groups, 0)
    ck = wf.Checksums(cd1, cd2, cw1, cw2)
    wf.coc_checksums(ck, spec.stride, spec.pad)
    for name, ref in (("cd1", cd1), ("cd2", cd2)):
        got = bufs[name].reshape(ref.shape)
        if exact:
            np.testing.assert_array_equal(got, ref, err_msg=name)
        else:
            assert np.abs(got - ref).max() <= 1e-12 * (np.abs(ref).max() + 1e-300), name
    for name, ref in (("co5", ck.co5), ("co6", ck.co6), ("co7", ck.co7)):
        got = bufs[name].reshape(ref.shape)
        if exact:
            np.testing.assert_array_equal(got, ref, err_msg=name)
        else:
            assert_close_scaled(got, ref, 1e-11, name)
    bt = wf.BiasTerms.make(b, spec.n, spec.m, 0) if b is not None else None
    Kg = (spec.ch // groups) * spec.r * spec.s
    so5, so6, so7, q5, flags = wf.verify(Og, ck.co5, Kg, dt, wf.Policy(), bt)
    assert not flags.any(), "the oracle flags the GPU's clean output"
    slack = epi_slack(Og, dt)
    for name, ref in (("so5", so5), ("so6", so6), ("so7", so7), ("q5", q5)):
        got = bufs[name].reshape(ref.shape)
        if exact and dt == "f32" and name != "q5":
            np.testing.assert_array_equal(got, ref, err_msg=name)   # integer sums: exact in float64
        else:
            assert_close_scaled(got, ref, 1e-11, name, slack[name])


def _run_path0(spec, D, W):
    dt = spec.dtype
    desc = ft.make_desc(spec.n, spec.ch, spec.h, spec.w, spec.m, spec.r, spec.s, spec.stride, spec.pad, dt)
    Dd, Wd = dev(D, dt), dev(W, dt)
    E, F = ft.out_shape(desc)
    O = torch.empty((spec.n, spec.m, E, F), dtype=ft.DTYPES[dt][1], device="cuda")
    ft.conv_fwd(desc, Dd, Wd, O)
    torch.cuda.synchronize()
    return host(O)


@pytest.mark.parametrize("case", CASES, ids=case_id)
def test_full_size_whole_output(case):
    name, lname, groups, with_bias, path = case
    cfg, li = layer(name, lname)
    spec = cfg.layers[li]
    wspec = spec.with_(ch=spec.ch // groups)   # a grouped filter sees ch / groups channels
    kind = ft.conv_tile(ft.make_desc(spec.n, spec.ch, spec.h, spec.w, spec.m, spec.r, spec.s, spec.stride,
                                     spec.pad, spec.dtype, groups=groups), path)
    print(f"[fullsize-exact] {case_id(case)} n{spec.n} c{spec.ch} h{spec.h} m{spec.m} r{spec.r} "
          f"u{spec.stride} {spec.dtype} kernel {kind}", flush=True)
    for exact in (False, True):
        if exact:
            D, W = wl.gen_int_d(spec, 41), wl.gen_int_w(wspec, 41)
        else:
            D, W = wl.gen_d(cfg, li), wl.gen_w(cfg, li, wspec)
        b = _bias(spec.m, exact, li) if with_bias else None
        if path == 1:
            Og, bufs, _ = _run_path1(spec, groups, D, W, b)
        else:
            Og = _run_path0(spec, D, W)
        ref = _oracle_out(D, W, spec, groups, b)
        what = f"{case_id(case)} {'integer' if exact else 'workload'} data"
        if exact:
            bad = Og != ref
            assert not bad.any(), (f"{what}: {int(bad.sum())} of {ref.size} elements differ; first at "
                                   f"{np.argwhere(bad)[0].tolist()}")
        else:
            assert_close_scaled(Og, ref, TOL[spec.dtype], what)
        del ref
        if path == 1:
            _check_checksums(spec, groups, D, W, b, Og, bufs, exact)
