"""Pins for the oracle's checksums: closed forms, linearity and the location identities."""
import json
import os

import numpy as np
import pytest

from oracle import core, workflow as wf

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_encode_golden():
    with open(os.path.join(GOLD, "checksum_hand.json")) as f:
        g = json.load(f)["encode"]
    c1, c2 = wf.encode(np.array(g["X"], float))
    np.testing.assert_array_equal(c1, g["C1"])
    np.testing.assert_array_equal(c2, g["C2"])


def test_encode_per_image_constants():
    c = np.array([0.5, -2.0, 3.25, 7.0, 1.0])
    X = np.broadcast_to(c[:, None, None, None], (5, 3, 4, 4)).copy()
    c1, c2 = wf.encode(X)
    np.testing.assert_array_equal(c1, np.full((3, 4, 4), c.sum()))
    np.testing.assert_array_equal(c2, np.full((3, 4, 4), (np.arange(5) * c).sum()))
    c1b, c2b = wf.encode(X, wbase=1)
    np.testing.assert_array_equal(c2b, np.full((3, 4, 4), ((np.arange(5) + 1) * c).sum()))


def test_distributive_property():
    """Sec. 3.1: D1(x)W + D2(x)W = (D1+D2)(x)W and D(x)W1 + D(x)W2 = D(x)(W1+W2), exact on integers."""
    g = np.random.default_rng(11)
    D1, D2 = (g.integers(-3, 4, (2, 4, 9, 9)).astype(float) for _ in range(2))
    W1, W2 = (g.integers(-2, 3, (3, 4, 3, 3)).astype(float) for _ in range(2))
    for U, P in [(1, 1), (2, 0), (2, 1)]:
        np.testing.assert_array_equal(core.conv(D1, W1, U, P) + core.conv(D2, W1, U, P), core.conv(D1 + D2, W1, U, P))
        np.testing.assert_array_equal(core.conv(D1, W1, U, P) + core.conv(D1, W2, U, P), core.conv(D1, W1 + W2, U, P))


@pytest.mark.parametrize("wbase", [0, 1])
def test_checksum_identities_integer_exact(wbase):
    """Co_k equals the matching summation So_k exactly when nothing is corrupted (Sec. 3.3-3.6)."""
    g = np.random.default_rng(12 + wbase)
    N, M, U, P = 5, 6, 2, 1
    D = g.integers(0, 4, (N, 3, 11, 11)).astype(float)
    W = g.integers(-2, 3, (M, 3, 3, 3)).astype(float)
    O = core.conv(D, W, U, P)
    cd1, cd2 = wf.encode(D, wbase)
    cw1, cw2 = wf.encode(W, wbase)
    ck = wf.Checksums(cd1, cd2, cw1, cw2)
    wf.coc_checksums(ck, U, P)
    co1, co3 = wf.row_checksums(ck, W, U, P)
    co2, co4 = wf.col_checksums(ck, D, U, P)
    wn = (np.arange(N) + wbase)[:, None, None, None]
    wm = (np.arange(M) + wbase)[None, :, None, None]
    np.testing.assert_array_equal(co1, O.sum(0))
    np.testing.assert_array_equal(co3, (wn * O).sum(0))
    np.testing.assert_array_equal(co2, O.sum(1))
    np.testing.assert_array_equal(co4, (wm * O).sum(1))
    np.testing.assert_array_equal(ck.co5, O.sum((0, 1)))
    np.testing.assert_array_equal(ck.co6, (wm * O).sum((0, 1)))
    np.testing.assert_array_equal(ck.co7, (wn * O).sum((0, 1)))


def test_linearity_float_within_tolerance():
    """conv(sum_i D_i, W) = sum_i conv(D_i, W) up to float64 rounding on random data."""
    g = np.random.default_rng(13)
    D = g.random((8, 16, 13, 13))
    W = g.standard_normal((12, 16, 3, 3)) * np.sqrt(2 / 144)
    O = core.conv(D, W, 1, 1)
    cd1, cd2 = wf.encode(D)
    cw1, cw2 = wf.encode(W)
    ck = wf.Checksums(cd1, cd2, cw1, cw2)
    wf.coc_checksums(ck, 1, 1)
    so5, so6, so7, q5, flags = wf.verify(O, ck.co5, 144, "f32", wf.Policy())
    assert not flags.any()
    assert np.max(np.abs(ck.co5 - so5) / q5) < 1e-13
    np.testing.assert_allclose(ck.co6, so6, rtol=1e-12, atol=1e-12 * np.abs(so6).max())
    np.testing.assert_allclose(ck.co7, so7, rtol=1e-12, atol=1e-12 * np.abs(so7).max())


def test_location_identities_golden():
    with open(os.path.join(GOLD, "checksum_hand.json")) as f:
        g = json.load(f)["locate"]
    N, M = g["N"], g["M"]
    D = (np.arange(N, dtype=float) + 1)[:, None, None, None]
    W = (np.arange(M, dtype=float) + 1)[:, None, None, None]
    O = core.conv(D, W, 1, 0)
    ck = wf.Checksums(*wf.encode(D), *wf.encode(W))
    wf.coc_checksums(ck, 1, 0)
    O[g["i"], g["j"]] += g["add"]
    so5, so6, so7, _, _ = wf.verify(O, ck.co5, 1, "f32", wf.Policy())
    assert ck.co5[0, 0] - so5[0, 0] == g["d5"]
    assert ck.co6[0, 0] - so6[0, 0] == g["d6"]
    assert ck.co7[0, 0] - so7[0, 0] == g["d7"]


@pytest.mark.parametrize("i,j,delta", [(0, 0, 7.0), (3, 5, -11.0), (4, 0, 2.0), (0, 6, 1.0)])
def test_location_identities_closed_form(i, j, delta):
    """Sec. 3.6: one error of size delta in block (i, j) gives Co5-So5 = -delta, Co6-So6 = -j delta,
    Co7-So7 = -i delta, exactly on integer data."""
    g = np.random.default_rng(14)
    N, M = 5, 7
    D = g.integers(0, 4, (N, 2, 7, 7)).astype(float)
    W = g.integers(-2, 3, (M, 2, 3, 3)).astype(float)
    O = core.conv(D, W, 1, 1)
    ck = wf.Checksums(*wf.encode(D), *wf.encode(W))
    wf.coc_checksums(ck, 1, 1)
    O[i, j, 2, 3] += delta
    so5, so6, so7, _, _ = wf.verify(O, ck.co5, 18, "f32", wf.Policy())
    assert ck.co5[2, 3] - so5[2, 3] == -delta
    assert ck.co6[2, 3] - so6[2, 3] == -j * delta
    assert ck.co7[2, 3] - so7[2, 3] == -i * delta
    d = ck.co5 - so5
    d[2, 3] = 0
    assert not d.any()


def test_store_bf16_rounding():
    vals = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, 1.0 + 3 * 2 ** -9,
                     -2.5, 3.0e38, 1e-40, 0.0])
    got = wf.store(vals, "bf16")
    # ties go to even significands; 1 + 2^-8 is a tie between 1 and 1 + 2^-7
    assert got[0] == 1.0 and got[1] == 1.0 and got[2] == 1.0 + 2 ** -6
    assert got[3] == 1.0 and got[4] == 1.0 + 2 ** -7
    assert got[5] == -2.5 and got[8] == 0.0
    assert np.isfinite(got[6])
    # every result is a bf16 bit pattern
    f32 = got.astype(np.float32).view(np.uint32)
    assert not (f32 & 0xFFFF).any()


def test_fault_bit_flip():
    O = np.array([[[[1.5]]]])
    wf.apply_faults(O, "f32", [wf.Fault(0, 0, 0, 0, "flip", 31)])
    assert O[0, 0, 0, 0] == -1.5
    wf.apply_faults(O, "f32", [wf.Fault(0, 0, 0, 0, "flip", 23)])  # lowest exponent bit
    assert O[0, 0, 0, 0] == -0.75
    wf.apply_faults(O, "bf16", [wf.Fault(0, 0, 0, 0, "flip", 7)])
    assert O[0, 0, 0, 0] == -1.5
