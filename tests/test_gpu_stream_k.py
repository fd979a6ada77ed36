"""The stream-K schedule of the channels-last fp32 convolution (ftcnn_conv_stream_k): every
workgroup runs an equal run of the layer's (tile, chunk of K) pairs, and a tile split over several
workgroups is summed by the last of them, in chunk order, before its epilogue.  The cases are
layers on which the schedule is taken (asserted through the query), with tiles split over two to
four workgroups and, in one, a ragged last pixel tile:

* the whole output against the oracle's float64 eq. (1) (1e-4), and bit for bit on integer data;
* the unprotected twin storing the same bits as the protected convolution (both split K alike);
* So5..So7 and Q5 of the epilogue (run by each tile's last workgroup) against the oracle (Sec. 3.6);
* a planted multi-fault pattern detected and corrected as the oracle decides (Sec. 4.1, 4.3);
* a bias in the epilogue (Sec. 5.1), and a workspace full of garbage (the arrival counts are
  cleared by the channels-last copy before every such convolution).
"""
import numpy as np
import pytest
import torch

import paper_2003_12203_amd as ft
import workloads as wl
from gpu_util import TOL, assert_close_scaled, dev, host
from oracle import workflow as wf
from test_gpu_fullsize_exact import _bias, _check_checksums, _oracle_out, _run_path1
from test_gpu_workflow import _pattern_faults, compare, run_gpu

pytestmark = pytest.mark.gpu

# (workload config, layer index whose generators seed the data, shape): VGG-19 v13 at batch 16
# (64 x 64 tiles, 392 of them for 1024 resident workgroups) and Darknet-19 c9 at 25 x 25 (128 x 64
# tiles, the last pixel tile a quarter full)
CASES = {
    "v13-b16": (2, 12, wl.LayerSpec("v13-b16", 16, 512, 14, 14, 512, 3, 3, 1, 1, "f32")),
    "c9-25x25": (4, 8, wl.LayerSpec("c9-25x25", 16, 256, 25, 25, 512, 3, 3, 1, 1, "f32")),
}


def _desc(spec, groups=1):
    return ft.make_desc(spec.n, spec.ch, spec.h, spec.w, spec.m, spec.r, spec.s, spec.stride, spec.pad,
                        spec.dtype, groups=groups)


def _data(name, integer):
    cid, li, spec = CASES[name]
    if integer:
        return spec, wl.gen_int_d(spec, 43), wl.gen_int_w(spec, 43)
    cfg = wl.config(cid)
    return spec, wl.gen_d(cfg, li, spec), wl.gen_w(cfg, li, spec)


def test_schedule_is_taken_where_expected():
    for name in CASES:
        assert ft.conv_stream_k(_desc(CASES[name][2])) > 0, name
    vgg = {L.name: L for L in wl.config(2).layers}
    for lname in ("v10", "v13"):
        assert ft.conv_stream_k(_desc(vgg[lname])) > 0, lname
    # bf16 layers, grouped layers and the 3-channel stem (no channels-last copy) run whole tiles
    assert ft.conv_stream_k(_desc(vgg["v10"].with_(dtype="bf16"))) == 0
    assert ft.conv_stream_k(_desc(vgg["v1"])) == 0
    alex = {L.name: L for L in wl.config(1).layers}
    assert ft.conv_stream_k(_desc(alex["conv2"], groups=2)) == 0


@pytest.mark.parametrize("integer", [False, True], ids=["workload", "integer"])
@pytest.mark.parametrize("name", list(CASES))
def test_whole_output_and_sums(name, integer):
    spec, D, W = _data(name, integer)
    print(f"[stream-k] {name} {'integer' if integer else 'workload'} data, "
          f"{ft.conv_stream_k(_desc(spec))} workgroups", flush=True)
    Og, bufs, _ = _run_path1(spec, 1, D, W, None)   # also checks the twin's bits and no flag
    ref = _oracle_out(D, W, spec, 1, None)
    if integer:
        bad = Og != ref
        assert not bad.any(), f"{int(bad.sum())} of {ref.size} elements differ"
    else:
        assert_close_scaled(Og, ref, TOL["f32"], f"{name} O")
    _check_checksums(spec, 1, D, W, None, Og, bufs, integer)


def test_bias_and_dirty_workspace():
    spec, D, W = _data("c9-25x25", False)
    b = _bias(spec.m, False, 8)
    lay = ft.Layer(spec.n, spec.ch, spec.h, spec.w, spec.m, spec.r, spec.s, spec.stride, spec.pad, "f32")
    Dd, Wd = dev(D, "f32"), dev(W, "f32")
    lay.set_bias(torch.from_numpy(b).cuda())
    outs = []
    for fill in (0, 255):
        lay.workspace.fill_(fill)   # arrival counts of -1 unless the copy clears them
        O = lay.empty_output()
        lay.conv_ws(Dd, Wd, O)
        outs.append(host(O))
    np.testing.assert_array_equal(outs[0], outs[1])
    assert_close_scaled(outs[1], _oracle_out(D, W, spec, 1, b), TOL["f32"], "biased O")


def test_planted_faults_corrected():
    spec, D, W = _data("v13-b16", False)
    clean = wf.protect(D, W, spec.stride, spec.pad, spec.dtype).O_clean
    draws = wl.fault_draws(2, 12, 4)
    faults = _pattern_faults(clean, draws, 3)
    rep, status, O_faulty, O_final, flags = run_gpu(spec, D, W, faults, {}, mode="two_launch")
    compare(spec, D, W, rep, status, O_faulty, O_final, flags, wf.Policy())
    assert rep.detected and status in (ft.STATUS_CORRECTED, ft.STATUS_RECOMPUTED)
    assert_close_scaled(O_final, clean, 1e-3, "recovered O")
