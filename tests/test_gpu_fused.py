"""The convolution with the CoC-D summations in its epilogue (ftcnn_conv_fwd_sums) against the
separate kernels and the oracle.

* O is bitwise the output of ftcnn_conv_fwd_ws (same kernels, same rounding);
* So5, So6, So7 and Q5 from the epilogue partials agree with the oracle's summations of the
  GPU's own output (Sec. 3.6) to float64 rounding, and exactly on integer data;
* faults planted in the epilogue give bitwise the output that ftcnn_inject gives afterwards;
* the two-launch path (input checksums encoded by extra workgroups of the convolution launch,
  Co5..Co7 computed in the final launch) gives the checksums of the separate kernels and the
  oracle;
* ftcnn_protected_conv (the whole path in one call) matches the step-by-step path.
"""
import numpy as np
import pytest
import torch

import paper_2003_12203_amd as ft
import workloads as wl
from gpu_util import epi_slack, assert_close_scaled, dev, gpu_flags, host, layer_for, to_ft_faults, workload_shapes
from oracle import workflow as wf

pytestmark = pytest.mark.gpu


def _sums(lay):
    torch.cuda.synchronize()
    return {k: lay.buf[k].cpu().numpy().copy() for k in ("so5", "so6", "so7", "q5")}


@pytest.mark.parametrize("cfg,li,spec", workload_shapes())
@pytest.mark.parametrize("wbase", [0, 1])
def test_epilogue_sums_match_oracle(cfg, li, spec, wbase):
    D, W = wl.gen_d(cfg, li, spec), wl.gen_w(cfg, li, spec)
    lay = layer_for(spec, wbase=wbase)
    Dd, Wd = dev(D, spec.dtype), dev(W, spec.dtype)
    lay.encode_weights(Wd)
    lay.encode_input(Dd)
    O_ref = lay.empty_output()
    lay.conv_ws(Dd, Wd, O_ref)
    O = lay.empty_output()
    lay.conv_sums(Dd, Wd, O)
    lay.checksum_conv(ft.CO5 | ft.CO6 | ft.CO7)
    lay.verify_correct_sums(Dd, Wd, O)
    torch.cuda.synchronize()
    assert torch.equal(O.view(torch.int16 if spec.dtype == "bf16" else torch.int32),
                       O_ref.view(torch.int16 if spec.dtype == "bf16" else torch.int32)), "O differs from conv_fwd_ws"
    got = _sums(lay)
    co5 = lay.buf["co5"].cpu().numpy().reshape(lay.E, lay.F)
    so5, so6, so7, q5, flags = wf.verify(host(O), co5, spec.ch * spec.r * spec.s, spec.dtype,
                                         wf.Policy(wbase=wbase))
    slack = epi_slack(host(O), spec.dtype, wbase)
    for name, ref in [("so5", so5), ("so6", so6), ("so7", so7), ("q5", q5)]:
        assert_close_scaled(got[name].reshape(ref.shape), ref, 1e-11, name, slack[name])
    assert not flags.any(), "clean layer flagged by the oracle"
    assert not gpu_flags(lay).any(), "clean layer flagged by the GPU"
    rep = lay.read_report()
    assert not rep.detected and rep.status == ft.STATUS_CLEAN and rep.n_flagged == 0


@pytest.mark.parametrize("cfg,li,spec", workload_shapes())
def test_two_launch_checksums_match_oracle(cfg, li, spec):
    D, W = wl.gen_d(cfg, li, spec), wl.gen_w(cfg, li, spec)
    lay = layer_for(spec)
    Dd, Wd = dev(D, spec.dtype), dev(W, spec.dtype)
    lay.encode_weights(Wd)
    O_ref = lay.empty_output()
    lay.conv_ws(Dd, Wd, O_ref)
    O = lay.empty_output()
    lay.conv_sums(Dd, Wd, O, encode=True)
    lay.verify_correct_sums(Dd, Wd, O, coc=True)
    torch.cuda.synchronize()
    iv = torch.int16 if spec.dtype == "bf16" else torch.int32
    assert torch.equal(O.view(iv), O_ref.view(iv)), "O differs from conv_fwd_ws"
    b = {k: v.cpu().numpy() for k, v in lay.buf.items()}
    cd1, cd2 = wf.encode(D, 0)
    np.testing.assert_allclose(b["cd1"], cd1.ravel(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(b["cd2"], cd2.ravel(), rtol=1e-12, atol=1e-10)
    ck = wf.Checksums(cd1, cd2, *wf.encode(W, 0))
    wf.coc_checksums(ck, spec.stride, spec.pad)
    for name, ref in [("co5", ck.co5), ("co6", ck.co6), ("co7", ck.co7)]:
        assert_close_scaled(b[name].reshape(ref.shape), ref, 1e-11, name)
    so5, so6, so7, q5, flags = wf.verify(host(O), ck.co5, spec.ch * spec.r * spec.s, spec.dtype, wf.Policy())
    slack = epi_slack(host(O), spec.dtype)
    for name, ref in [("so5", so5), ("so6", so6), ("so7", so7), ("q5", q5)]:
        assert_close_scaled(b[name].reshape(ref.shape), ref, 1e-11, name, slack[name])
    assert not flags.any() and not gpu_flags(lay).any()
    assert not lay.read_report().detected


@pytest.mark.parametrize("shape", [
    # n, ch, h, m, r, stride, pad: ragged pixel tails, partial filter tiles, several tiles per image
    (5, 6, 12, 9, 3, 1, 1),
    (3, 16, 10, 5, 3, 1, 1),
    (2, 7, 9, 33, 3, 2, 1),
    (4, 64, 7, 130, 1, 1, 0),
    (1, 3, 35, 96, 11, 4, 0),
    (2, 8, 13, 200, 5, 3, 2),
    (2, 5, 3, 7, 3, 1, 0),       # E = 1
])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_epilogue_sums_integer_exact(shape, dtype):
    """Integer data: the epilogue's summations equal the checksum convolutions exactly."""
    n, ch, h, m, r, u, p = shape
    spec = wl.LayerSpec("int", n, ch, h, h, m, r, r, u, p, dtype)
    D, W = wl.gen_int_d(spec, 7 + sum(shape)), wl.gen_int_w(spec, 7 + sum(shape))
    lay = layer_for(spec)
    Dd, Wd = dev(D, dtype), dev(W, dtype)
    lay.encode_weights(Wd)
    O = lay.empty_output()
    lay.conv_sums(Dd, Wd, O, encode=True)
    lay.verify_correct_sums(Dd, Wd, O, coc=True)
    torch.cuda.synchronize()
    b = {k: v.cpu().numpy() for k, v in lay.buf.items()}
    cd1, cd2 = wf.encode(D, 0)
    np.testing.assert_array_equal(b["cd1"], cd1.ravel())
    np.testing.assert_array_equal(b["cd2"], cd2.ravel())
    if dtype == "f32" or np.abs(host(O)).max() <= 256:
        np.testing.assert_array_equal(b["co5"], b["so5"])
        np.testing.assert_array_equal(b["co6"], b["so6"])
        np.testing.assert_array_equal(b["co7"], b["so7"])
    assert not lay.read_report().detected


def test_epilogue_sums_deterministic():
    cfg = wl.config(1)
    spec = cfg.layers[1].with_(n=6)
    lay = layer_for(spec)
    Dd, Wd = dev(wl.gen_d(cfg, 1, spec), "f32"), dev(wl.gen_w(cfg, 1, spec), "f32")
    lay.encode_weights(Wd)
    lay.encode_input(Dd)
    lay.checksum_conv(ft.CO5 | ft.CO6 | ft.CO7)
    O = lay.empty_output()
    lay.conv_sums(Dd, Wd, O)
    lay.verify_correct_sums(Dd, Wd, O)
    first = _sums(lay)
    lay.conv_sums(Dd, Wd, O)
    lay.verify_correct_sums(Dd, Wd, O)
    second = _sums(lay)
    for k in first:
        np.testing.assert_array_equal(first[k], second[k])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_planted_faults_equal_injected(dtype):
    """Faults planted in the epilogue (every kind, repeated hits on one element, NaN-producing
    flips) leave exactly the output that ftcnn_inject leaves on the plain convolution."""
    spec = wl.LayerSpec("f", 3, 8, 11, 11, 70, 3, 3, 1, 1, dtype)
    cfg = wl.Config(92, "f", (spec,), "uniform", "he")
    D, W = wl.gen_d(cfg, 0, spec), wl.gen_w(cfg, 0, spec)
    top = 30 if dtype == "f32" else 14
    faults = [
        wf.Fault(0, 0, 0, 0, "flip", top),
        wf.Fault(2, 69, 10, 10, "add", value=-3.5),
        wf.Fault(1, 33, 5, 7, "set", value=123.25),
        wf.Fault(1, 33, 5, 7, "add", value=0.5),          # second hit on one element
        wf.Fault(2, 64, 3, 9, "flip", top - 1),
        wf.Fault(0, 5, 4, 4, "set", value=float("inf")),
    ]
    lay = layer_for(spec)
    Dd, Wd = dev(D, dtype), dev(W, dtype)
    lay.encode_weights(Wd)
    lay.encode_input(Dd)
    O1 = lay.empty_output()
    lay.conv_ws(Dd, Wd, O1)
    lay.inject(O1, to_ft_faults(faults))
    O2 = lay.empty_output()
    lay.conv_sums(Dd, Wd, O2, to_ft_faults(faults))
    torch.cuda.synchronize()
    iv = torch.int16 if dtype == "bf16" else torch.int32
    assert torch.equal(O1.view(iv), O2.view(iv))
    O_faulty = host(O2)
    lay.checksum_conv(ft.CO5 | ft.CO6 | ft.CO7)
    lay.verify_correct_sums(Dd, Wd, O2)
    rep = lay.read_report()
    # the decisions on the planted faults are the oracle's on the same faulted output (a flip that
    # shrinks a bf16 value may stay inside the bf16 tolerance and go undetected on both sides)
    ores = wf.protect(D, W, spec.stride, spec.pad, dtype, O_in=O_faulty).report
    assert rep.detected and ores.detected
    assert rep.n_flagged == ores.n_flagged and rep.fixes == ores.fixes


def test_fault_list_is_validated():
    spec = wl.LayerSpec("v", 2, 3, 8, 8, 4, 3, 3, 1, 1, "f32")
    lay = layer_for(spec)
    D = torch.zeros(spec.n, spec.ch, spec.h, spec.w, device="cuda")
    W = torch.zeros(spec.m, spec.ch, spec.r, spec.s, device="cuda")
    O = lay.empty_output()
    with pytest.raises(ft.FtcnnError, match="out of range"):
        lay.conv_sums(D, W, O, [{"n": 2, "m": 0, "x": 0, "y": 0, "kind": "add", "value": 1.0}])
    with pytest.raises(ft.FtcnnError, match="bit"):
        lay.conv_sums(D, W, O, [{"n": 0, "m": 0, "x": 0, "y": 0, "kind": "flip", "bit": 32}])
    with pytest.raises(ft.FtcnnError, match="at most"):
        lay.conv_sums(D, W, O, [{"n": 0, "m": 0, "x": 0, "y": 0, "kind": "add", "value": 1.0}] * 65)


@pytest.mark.parametrize("li", [0, 1, 2])
def test_protected_conv_single_call(li):
    """ftcnn_protected_conv equals the step-by-step path (AlexNet layers, reduced batch)."""
    cfg = wl.config(1)
    spec = cfg.layers[li].with_(n=3)
    D, W = wl.gen_d(cfg, li, spec), wl.gen_w(cfg, li, spec)
    lay = layer_for(spec)
    Dd, Wd = dev(D, "f32"), dev(W, "f32")
    lay.encode_weights(Wd)
    O = lay.empty_output()
    lay.protected(Dd, Wd, O)
    one = _sums(lay)
    rep = lay.read_report()
    assert not rep.detected and rep.status == ft.STATUS_CLEAN
    O2 = lay.empty_output()
    lay.encode_input(Dd)
    lay.conv_ws(Dd, Wd, O2)
    lay.checksum_conv(ft.CO5 | ft.CO6 | ft.CO7)
    lay.verify(O2)
    torch.cuda.synchronize()
    assert torch.equal(O, O2)
    two = _sums(lay)
    Q = two["q5"]
    for k in ("so5", "so6", "so7"):
        np.testing.assert_allclose(one[k], two[k], rtol=0, atol=1e-12 * float(Q.max()) * max(spec.n, spec.m))


# Layers with many images and few 32 x 32 feature-map tiles: the channels-last copy encodes Cd1,
# Cd2 over several image ranges, the convolution launch combines them and computes the Co5..Co7
# partials from them (ranges of 16 images in fp32, 32 in bf16; uneven ranges with n = 50).
SPLIT_SHAPES = [
    # n, ch, h, m, r, stride, pad, dtype
    (64, 32, 9, 40, 3, 1, 1, "f32"),
    (50, 32, 10, 24, 3, 2, 1, "f32"),
    (40, 64, 5, 16, 1, 1, 0, "f32"),
    (64, 64, 7, 48, 3, 1, 1, "bf16"),
    (96, 64, 6, 70, 3, 2, 1, "bf16"),
]
# split images on layers with E*F*K of at least 1M: Co5..Co7 in the convolution launch, one pass
# per image range
SPLIT_COC_SHAPES = [
    (32, 32, 64, 32, 3, 1, 1, "f32"),
    (64, 64, 48, 64, 3, 1, 1, "bf16"),
]


def _split_spec(shape):
    n, ch, h, m, r, u, p, dtype = shape
    return wl.LayerSpec("split", n, ch, h, h, m, r, r, u, p, dtype)


@pytest.mark.parametrize("shape", SPLIT_SHAPES + SPLIT_COC_SHAPES,
                         ids=lambda s: "n{}-c{}-h{}-m{}-r{}-u{}-{}".format(*s[:6], s[7]))
def test_image_split_encode_integer_exact(shape):
    """Integer data: the combined image-range partials are exactly Cd1, Cd2, and the Co5..Co7
    partial products of the convolution launch add up exactly to the summations of O."""
    spec = _split_spec(shape)
    D, W = wl.gen_int_d(spec, 11), wl.gen_int_w(spec, 11)
    lay = layer_for(spec)
    Dd, Wd = dev(D, spec.dtype), dev(W, spec.dtype)
    lay.encode_weights(Wd)
    O_ref = lay.empty_output()
    lay.conv_ws(Dd, Wd, O_ref)
    O = lay.empty_output()
    lay.conv_sums(Dd, Wd, O, encode=True)
    lay.verify_correct_sums(Dd, Wd, O, coc=True)
    torch.cuda.synchronize()
    iv = torch.int16 if spec.dtype == "bf16" else torch.int32
    assert torch.equal(O.view(iv), O_ref.view(iv))
    b = {k: v.cpu().numpy() for k, v in lay.buf.items()}
    cd1, cd2 = wf.encode(D, 0)
    np.testing.assert_array_equal(b["cd1"], cd1.ravel())
    np.testing.assert_array_equal(b["cd2"], cd2.ravel())
    ck = wf.Checksums(cd1, cd2, *wf.encode(W, 0))
    wf.coc_checksums(ck, spec.stride, spec.pad)
    for name, ref in [("co5", ck.co5), ("co6", ck.co6), ("co7", ck.co7)]:
        np.testing.assert_array_equal(b[name].reshape(ref.shape), ref)
    if spec.dtype == "f32" or np.abs(host(O)).max() <= 256:
        for k in ("5", "6", "7"):
            np.testing.assert_array_equal(b["co" + k], b["so" + k])
    assert not lay.read_report().detected


@pytest.mark.parametrize("shape", SPLIT_SHAPES, ids=lambda s: "n{}-c{}-h{}-m{}-r{}-u{}-{}".format(*s[:6], s[7]))
def test_image_split_decisions_match_oracle(shape):
    """Random data with two planted faults (different positions): Cd, Co5..Co7 match the oracle,
    and the decisions and repairs are the oracle's on the same faulted output."""
    spec = _split_spec(shape)
    cfg = wl.Config(93, "split", (spec,), "uniform", "he")
    D, W = wl.gen_d(cfg, 0, spec), wl.gen_w(cfg, 0, spec)
    lay = layer_for(spec)
    Dd, Wd = dev(D, spec.dtype), dev(W, spec.dtype)
    lay.encode_weights(Wd)
    E, F = lay.E, lay.F
    faults = [wf.Fault(spec.n - 1, spec.m - 1, E - 1, F - 1, "add", value=1.0e5),
              wf.Fault(spec.n // 2, 1, 0, F // 2, "add", value=-2.0e5)]
    O = lay.empty_output()
    lay.conv_sums(Dd, Wd, O, to_ft_faults(faults), encode=True)
    torch.cuda.synchronize()
    O_faulty = host(O)
    lay.verify_correct_sums(Dd, Wd, O, coc=True)
    rep = lay.read_report()
    b = {k: v.cpu().numpy() for k, v in lay.buf.items()}
    cd1, cd2 = wf.encode(D, 0)
    np.testing.assert_allclose(b["cd1"], cd1.ravel(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(b["cd2"], cd2.ravel(), rtol=1e-12, atol=1e-10)
    ck = wf.Checksums(cd1, cd2, *wf.encode(W, 0))
    wf.coc_checksums(ck, spec.stride, spec.pad)
    for name, ref in [("co5", ck.co5), ("co6", ck.co6), ("co7", ck.co7)]:
        assert_close_scaled(b[name].reshape(ref.shape), ref, 1e-11, name)
    ores = wf.protect(D, W, spec.stride, spec.pad, spec.dtype, O_in=O_faulty).report
    assert rep.detected and ores.detected
    assert rep.n_flagged == ores.n_flagged == 2
    assert rep.fixes == ores.fixes
    assert sorted(f[:4] for f in rep.fixes) == sorted((f.n, f.m, f.x, f.y) for f in faults)
    assert rep.status == ft.STATUS_CORRECTED


def test_verify_taps_when_conv_launch_left_no_partials():
    """A channels-last layer whose convolution launch was given Cd but not Cw computes Co5..Co7
    from the taps in the final launch instead: same checksums and verdict."""
    spec = _split_spec((64, 32, 9, 40, 3, 1, 1, "f32"))
    D, W = wl.gen_int_d(spec, 5), wl.gen_int_w(spec, 5)
    lay = layer_for(spec)
    Dd, Wd = dev(D, "f32"), dev(W, "f32")
    lay.encode_weights(Wd)
    O = lay.empty_output()
    ck = ft._lib.Checksums()
    ck.cd1, ck.cd2 = lay.buf["cd1"].data_ptr(), lay.buf["cd2"].data_ptr()
    ft.conv_fwd_sums(lay.desc, Dd, Wd, O, ck, lay.report, lay.cap, lay.workspace)
    lay.verify_correct_sums(Dd, Wd, O, coc=True)
    torch.cuda.synchronize()
    b = {k: v.cpu().numpy() for k, v in lay.buf.items()}
    cd1, cd2 = wf.encode(D, 0)
    ckr = wf.Checksums(cd1, cd2, *wf.encode(W, 0))
    wf.coc_checksums(ckr, spec.stride, spec.pad)
    for name, ref in [("co5", ckr.co5), ("co6", ckr.co6), ("co7", ckr.co7)]:
        np.testing.assert_array_equal(b[name].reshape(ref.shape), ref)
        np.testing.assert_array_equal(b[name], b["so" + name[2]])
    assert not lay.read_report().detected
