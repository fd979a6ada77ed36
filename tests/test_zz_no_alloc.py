"""ftcnn_protected_conv_noalloc (the protected layer on the library's static device scratch, for
callers that cannot allocate) against ftcnn_protected_conv with a caller's workspace, through the
C ABI, on two calls in a row whose second input is smaller:

1. a layer whose channels-last workspace exceeds the 128 MiB static scratch, so the call takes the
   plan without channels-last copies: O within the output tolerance of the workspace call's O (the
   dot products are summed in another order), Cd1, Cd2, Co5..Co7 within float64 rounding of the
   workspace call's, So5..So7 and Q5 within float64 rounding of the oracle's summations of the
   call's own output (Sec. 3.6), both reports clean;
2. a smaller layer whose workspace fits, with one corrupted column of Cw1 so that detection and
   correction run in the scratch: the same kernels as the workspace call, so O, every checksum
   array and the report must be identical bit for bit, whatever the first call left in the
   scratch.
"""
import numpy as np
import pytest
import torch

import paper_2003_12203_amd as ft
import workloads as wl
from gpu_util import TOL, assert_close_scaled, dev, host
from oracle import workflow as wf

pytestmark = pytest.mark.gpu

CK_KEYS = ("cd1", "cd2", "co5", "co6", "co7", "so5", "so6", "so7", "q5")


def _two_layers(spec):
    mk = lambda: ft.Layer(spec.n, spec.ch, spec.h, spec.w, spec.m, spec.r, spec.s, spec.stride, spec.pad,
                          spec.dtype)
    return mk(), mk()


def _run_both(spec, D, W, corrupt_cw1=None):
    """(O, buffers, report) of ftcnn_protected_conv and of ftcnn_protected_conv_noalloc."""
    ref, na = _two_layers(spec)
    Dd, Wd = dev(D, spec.dtype), dev(W, spec.dtype)
    out = []
    for lay, noalloc in ((ref, False), (na, True)):
        lay.encode_weights(Wd)
        if corrupt_cw1 is not None:
            lay.buf["cw1"][corrupt_cw1] += 1.0
        O = lay.empty_output()
        if noalloc:
            ft.protected_conv_noalloc(lay.desc, Dd, Wd, O, lay.ck, lay.policy, lay.report, lay.cap)
        else:
            lay.protected(Dd, Wd, O)
        rep = lay.read_report()
        out.append((O, {k: lay.buf[k].cpu().numpy() for k in CK_KEYS}, rep))
    return out


def test_noalloc_matches_workspace_entry_point_on_two_calls():
    # call 1: 48 x 64 x 112 x 112 fp32, channels-last workspace ~170 MiB > 128 MiB
    big = wl.LayerSpec("big", 48, 64, 112, 112, 64, 3, 3, 1, 1, "f32")
    d = ft.make_desc(big.n, big.ch, big.h, big.w, big.m, big.r, big.s, big.stride, big.pad, big.dtype)
    assert ft.workspace_bytes(d) > (128 << 20), "the first layer must need the fallback plan"
    cfg = wl.config(2)
    D = wl.gen_d(cfg, 1, big)
    W = wl.gen_w(cfg, 1, big)
    print("[noalloc] call 1: 48x64x112x112 fp32, fallback plan", flush=True)
    (O_ref, b_ref, r_ref), (O_na, b_na, r_na) = _run_both(big, D, W)
    assert not r_ref.detected and not r_na.detected, (r_ref, r_na)
    assert r_na.status == ft.STATUS_CLEAN and r_na.n_flagged == 0
    Og = host(O_na)
    assert_close_scaled(Og, host(O_ref), TOL["f32"], "O (no-alloc vs workspace)")
    for k in ("cd1", "cd2", "co5", "co6", "co7"):
        assert_close_scaled(b_na[k], b_ref[k], 1e-11, k)
    E, F = O_na.shape[2:]
    so5, so6, so7, q5, flags = wf.verify(Og, b_na["co5"].reshape(E, F), big.ch * 9, "f32", wf.Policy())
    assert not flags.any()
    for k, ref in (("so5", so5), ("so6", so6), ("so7", so7), ("q5", q5)):
        assert_close_scaled(b_na[k].reshape(E, F), ref, 1e-11, k)
    del O_ref, O_na, Og

    # call 2: a smaller layer with a corrupted weight checksum: detection and correction run
    small = wl.LayerSpec("small", 6, 32, 14, 14, 24, 3, 3, 1, 1, "f32")
    D2, W2 = wl.gen_int_d(small, 5), wl.gen_int_w(small, 5)
    print("[noalloc] call 2: 6x32x14x14 fp32, corrupted Cw1, same plan as the workspace call", flush=True)
    (O_ref, b_ref, r_ref), (O_na, b_na, r_na) = _run_both(small, D2, W2, corrupt_cw1=4 * 9 + 4)
    assert r_ref.detected and r_ref.n_flagged > 0
    assert (r_na.detected, r_na.n_flagged, r_na.status, r_na.resolved_by, r_na.fixes, r_na.n_fixes) == \
           (r_ref.detected, r_ref.n_flagged, r_ref.status, r_ref.resolved_by, r_ref.fixes, r_ref.n_fixes)
    assert torch.equal(O_na.view(torch.int32), O_ref.view(torch.int32))
    for k in CK_KEYS:
        np.testing.assert_array_equal(b_na[k], b_ref[k], err_msg=k)


def test_noalloc_bf16_after_fp32():
    # a third, smaller call in another dtype on the same scratch: identical to the workspace call
    spec = wl.LayerSpec("tiny", 4, 64, 9, 9, 32, 3, 3, 1, 1, "bf16")
    cfg = wl.vgg19_bf16()
    D, W = wl.gen_d(cfg, 3, spec), wl.gen_w(cfg, 3, spec)
    print("[noalloc] call 3: 4x64x9x9 bf16", flush=True)
    (O_ref, b_ref, r_ref), (O_na, b_na, r_na) = _run_both(spec, D, W)
    assert not r_ref.detected and not r_na.detected
    assert torch.equal(O_na.view(torch.int16), O_ref.view(torch.int16))
    for k in CK_KEYS:
        np.testing.assert_array_equal(b_na[k], b_ref[k], err_msg=k)
