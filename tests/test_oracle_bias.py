"""The oracle's bias handling (Sec. 5.1, Table 5), pinned to what the definitions fix.

* Table 5's adjustments are identities: on integer data (every term exact in float64) the
  summations of the biased output, less the shares BiasTerms gives, equal the checksum
  convolutions of the bias-free checksum blocks, for all seven pairs (Co1..Co7 / So1..So7),
  with block weights starting at 0 and at 1.  A wrong share (N - 1 for N, sum n for
  sum (n + wbase), a dropped wbase) breaks one of them.
* The whole workflow with a bias: a clean layer is not flagged, and each fault pattern is
  resolved by the same scheme as without a bias, back to the biased clean output exactly.
* A zero bias changes nothing.
* The weight-memory check (Sec. 4.1.2) counts exactly the columns of W corrupted after Cw1
  was encoded.
"""
import numpy as np
import pytest

import workloads as wl
from oracle import core
from oracle import workflow as wf
from paper_2003_12203_amd import schemes


def _int_layer(n=5, ch=3, hw=8, m=6, seed=4):
    spec = wl.LayerSpec("bias", n, ch, hw, hw, m, 3, 3, 1, 1, "f32")
    D, W = wl.gen_int_d(spec, seed), wl.gen_int_w(spec, seed)
    bias = np.random.default_rng([12203, 51, seed]).integers(-7, 8, size=m).astype(np.float64)
    return spec, D.astype(np.float64), W.astype(np.float64), bias


@pytest.mark.parametrize("wbase", [0, 1])
def test_table5_identities_exact(wbase):
    spec, D, W, bias = _int_layer()
    N, M = spec.n, spec.m
    O = core.conv(D, W, 1, 1) + bias[None, :, None, None]
    cd1, cd2 = wf.encode(D, wbase)
    cw1, cw2 = wf.encode(W, wbase)
    ck = wf.Checksums(cd1, cd2, cw1, cw2)
    wf.coc_checksums(ck, 1, 1)
    co1, co3 = wf.row_checksums(ck, W, 1, 1)
    co2, co4 = wf.col_checksums(ck, D, 1, 1)
    bt = wf.BiasTerms.make(bias, N, M, wbase)
    wn = (np.arange(N) + wbase)[:, None, None, None].astype(np.float64)
    wm = (np.arange(M) + wbase)[None, :, None, None].astype(np.float64)
    so1, so3 = O.sum(axis=0), (wn * O).sum(axis=0)
    so2, so4 = O.sum(axis=1), (wm * O).sum(axis=1)
    so5, so6, so7 = O.sum(axis=(0, 1)), (wm * O).sum(axis=(0, 1)), (wn * O).sum(axis=(0, 1))
    np.testing.assert_array_equal(so1 - bt.s1[:, None, None], co1)
    np.testing.assert_array_equal(so3 - bt.s3[:, None, None], co3)
    np.testing.assert_array_equal(so2 - bt.b1, co2)
    np.testing.assert_array_equal(so4 - bt.b2, co4)
    np.testing.assert_array_equal(so5 - bt.s5, ck.co5)
    np.testing.assert_array_equal(so6 - bt.s6, ck.co6)
    np.testing.assert_array_equal(so7 - bt.s7, ck.co7)
    # the shares themselves, written out: sum over images of (n + wbase), and so on
    assert bt.wn == sum(n + wbase for n in range(N))
    assert bt.b2 == sum((m + wbase) * bias[m] for m in range(M))


def test_clean_biased_layer_not_flagged():
    spec, D, W, bias = _int_layer(seed=9)
    res = wf.protect(D, W, 1, 1, "f32", bias=bias)
    assert not res.report.detected and res.report.status == wf.STATUS_CLEAN
    np.testing.assert_array_equal(res.O, core.conv(D, W, 1, 1) + bias[None, :, None, None])
    # without the adjustment the same output is flagged everywhere the bias shares are nonzero
    *_, flags = wf.verify(res.O, res.ck.co5, spec.ch * 9, "f32", wf.Policy())
    assert flags.all()


@pytest.mark.parametrize("name", list(schemes.WORKFLOWS))
@pytest.mark.parametrize("repair", ["checksum", "recompute"])
def test_workflows_with_bias(name, repair):
    kind, rc_on, clc_on, expect = schemes.WORKFLOWS[name]
    spec, D, W, bias = _int_layer(n=6, ch=4, hw=9, m=8, seed=13)
    faults = [wf.Fault(q["n"], q["m"], q["x"], q["y"], "add", value=q["value"])
              for q in schemes.pattern(kind, spec.n, spec.m, 9, 9)]
    pol = wf.Policy(rc_on=rc_on, clc_on=clc_on, repair=repair)
    res = wf.protect(D, W, 1, 1, "f32", pol, faults, bias=bias)
    got = tuple(sorted({wf.SCHEME_NAMES[s] for s in res.report.scheme.values()}))
    assert got == expect
    np.testing.assert_array_equal(res.O, res.O_clean)
    np.testing.assert_array_equal(res.O_clean, core.conv(D, W, 1, 1) + bias[None, :, None, None])


def test_zero_bias_is_no_bias():
    spec, D, W, _ = _int_layer(seed=21)
    faults = [wf.Fault(2, 3, 4, 4, "add", value=99.0)]
    a = wf.protect(D, W, 1, 1, "f32", faults=faults)
    b = wf.protect(D, W, 1, 1, "f32", faults=faults, bias=np.zeros(spec.m))
    np.testing.assert_array_equal(a.O, b.O)
    assert a.report.fixes == b.report.fixes


@pytest.mark.parametrize("cols", [0, 1, 3])
def test_weight_check_counts_corrupted_columns(cols):
    """Sec. 4.1.2: corrupting elements of W after Cw1 is encoded shows in exactly the columns hit."""
    spec, _, W, _ = _int_layer(m=9, seed=37)
    cw1, _ = wf.encode(W, 0)
    W2 = W.copy()
    g = np.random.default_rng([12203, 71, cols])
    flat = g.choice(W.shape[1] * W.shape[2] * W.shape[3], size=cols, replace=False)
    for k in flat:
        c, rs = divmod(int(k), W.shape[2] * W.shape[3])
        r, s = divmod(rs, W.shape[3])
        W2[g.integers(0, W.shape[0]), c, r, s] += 0.5      # exact in float64
    assert wf.check_weights(W2, cw1) == cols
    assert wf.check_weights(W, cw1) == 0
