"""The oracle's grouped convolution (Sec. 5.2), pinned to what the definitions fix.

* the grouped convolution equals a brute-force loop over its definition (filter block m sees
  channel group m // (M/G) only) on tiny layers, for G = 2 and depthwise G = Ch, and equals the
  dense convolution of the block-diagonal expansion of W (an independent formulation);
* with the grouped Cw1/Cw2 (per-group filter sums side by side over the channels) all seven
  checksum identities Co_k = So_k hold exactly on integer data (the paper's proof), with block
  weights from 0 and from 1;
* every correction workflow on a grouped layer is resolved by its scheme and restores the clean
  output exactly; the weight check counts corrupted columns of a grouped W;
* G = 1 is the ungrouped layer.
"""
import numpy as np
import pytest

import workloads as wl
from oracle import core
from oracle import workflow as wf
from paper_2003_12203_amd import schemes


def _layer(n=3, ch=4, hw=6, m=6, groups=2, r=3, seed=5):
    g = np.random.default_rng([12203, 81, seed])
    D = g.integers(0, 4, size=(n, ch, hw, hw)).astype(np.float64)
    W = g.integers(-2, 3, size=(m, ch // groups, r, r)).astype(np.float64)
    return D, W


def _brute(D, W, groups, stride, pad):
    N, C, H, Wd = D.shape
    M, Cg, R, S = W.shape
    Mg = M // groups
    E, F = (H + 2 * pad - R) // stride + 1, (Wd + 2 * pad - S) // stride + 1
    O = np.zeros((N, M, E, F))
    for n in range(N):
        for m in range(M):
            g = m // Mg
            for x in range(E):
                for y in range(F):
                    acc = 0.0
                    for c in range(Cg):
                        for r in range(R):
                            for s in range(S):
                                ih, iw = x * stride + r - pad, y * stride + s - pad
                                if 0 <= ih < H and 0 <= iw < Wd:
                                    acc += D[n, g * Cg + c, ih, iw] * W[m, c, r, s]
                    O[n, m, x, y] = acc
    return O


def _expand(W, groups, C):
    M, Cg = W.shape[:2]
    Mg = M // groups
    Wf = np.zeros((M, C) + W.shape[2:])
    for m in range(M):
        g = m // Mg
        Wf[m, g * Cg:(g + 1) * Cg] = W[m]
    return Wf


@pytest.mark.parametrize("groups,ch,m", [(2, 4, 6), (4, 4, 8), (3, 6, 3)])
@pytest.mark.parametrize("stride,pad", [(1, 1), (2, 0)])
def test_grouped_conv_definition(groups, ch, m, stride, pad):
    D, W = _layer(ch=ch, m=m, groups=groups)
    got = wf.grouped_conv(D, W, groups, stride, pad)
    np.testing.assert_array_equal(got, _brute(D, W, groups, stride, pad))
    np.testing.assert_array_equal(got, core.conv(D, _expand(W, groups, ch), stride, pad))


@pytest.mark.parametrize("groups,ch,m", [(2, 4, 6), (4, 4, 8)])
@pytest.mark.parametrize("wbase", [0, 1])
def test_grouped_identities_exact(groups, ch, m, wbase):
    D, W = _layer(n=4, ch=ch, hw=7, m=m, groups=groups, seed=7)
    N, M = D.shape[0], W.shape[0]
    O = wf.grouped_conv(D, W, groups, 1, 1)
    cd1, cd2 = wf.encode(D, wbase)
    cw1, cw2 = wf.encode_weights(W, groups, wbase)
    assert cw1.shape == (ch,) + W.shape[2:]
    ck = wf.Checksums(cd1, cd2, cw1, cw2)
    wf.coc_checksums(ck, 1, 1)
    co1, co3 = wf.row_checksums(ck, W, 1, 1, groups)
    co2, co4 = wf.col_checksums(ck, D, 1, 1)
    wn = (np.arange(N) + wbase)[:, None, None, None].astype(np.float64)
    wm = (np.arange(M) + wbase)[None, :, None, None].astype(np.float64)
    np.testing.assert_array_equal(O.sum(axis=0), co1)
    np.testing.assert_array_equal((wn * O).sum(axis=0), co3)
    np.testing.assert_array_equal(O.sum(axis=1), co2)
    np.testing.assert_array_equal((wm * O).sum(axis=1), co4)
    np.testing.assert_array_equal(O.sum(axis=(0, 1)), ck.co5)
    np.testing.assert_array_equal((wm * O).sum(axis=(0, 1)), ck.co6)
    np.testing.assert_array_equal((wn * O).sum(axis=(0, 1)), ck.co7)
    # the grouped Cw1 is the ungrouped Cw1 of the block-diagonal expansion
    np.testing.assert_array_equal(cw1, wf.encode(_expand(W, groups, ch), wbase)[0])
    np.testing.assert_array_equal(cw2, wf.encode(_expand(W, groups, ch), wbase)[1])


@pytest.mark.parametrize("name", list(schemes.WORKFLOWS))
@pytest.mark.parametrize("groups,ch,m", [(2, 4, 8), (8, 8, 8)])
def test_workflows_on_grouped_layers(name, groups, ch, m):
    kind, rc_on, clc_on, expect = schemes.WORKFLOWS[name]
    D, W = _layer(n=6, ch=ch, hw=9, m=m, groups=groups, seed=11)
    faults = [wf.Fault(q["n"], q["m"], q["x"], q["y"], "add", value=q["value"])
              for q in schemes.pattern(kind, 6, m, 9, 9)]
    res = wf.protect(D, W, 1, 1, "f32", wf.Policy(rc_on=rc_on, clc_on=clc_on), faults, groups=groups)
    got = tuple(sorted({wf.SCHEME_NAMES[s] for s in res.report.scheme.values()}))
    assert got == expect
    np.testing.assert_array_equal(res.O, res.O_clean)
    np.testing.assert_array_equal(res.O_clean, wf.grouped_conv(D, W, groups, 1, 1))


def test_grouped_recompute_repair_and_weight_check():
    D, W = _layer(n=5, ch=6, hw=8, m=6, groups=3, seed=13)
    faults = [wf.Fault(2, 4, 3, 3, "add", value=1.0e6)]
    res = wf.protect(D, W, 1, 1, "f32", wf.Policy(repair="recompute"), faults, groups=3)
    assert res.report.fixes == [(2, 4, 3, 3, wf.SCHEME_COC)]
    np.testing.assert_array_equal(res.O, res.O_clean)
    cw1, _ = wf.encode_weights(W, 3)
    W2 = W.copy()
    W2[5, 1, 2, 0] += 1.0
    assert wf.check_weights(W2, cw1, groups=3) == 1 and wf.check_weights(W, cw1, groups=3) == 0


def test_one_group_is_ungrouped():
    spec = wl.LayerSpec("g", 4, 3, 8, 8, 5, 3, 3, 1, 1, "f32")
    D, W = wl.gen_int_d(spec, 3), wl.gen_int_w(spec, 3)
    faults = [wf.Fault(1, 2, 4, 4, "add", value=50.0)]
    a = wf.protect(D, W, 1, 1, "f32", faults=faults)
    b = wf.protect(D, W, 1, 1, "f32", faults=faults, groups=1)
    np.testing.assert_array_equal(a.O, b.O)
    assert a.report.fixes == b.report.fixes
