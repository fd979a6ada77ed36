"""Pins for the oracle's convolution (eq. 1) against things other than itself."""
import json
import os

import numpy as np
import pytest
import torch

from oracle import core

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def brute_conv(D, W, U, P):
    """Seven nested Python loops over eq. (1) with an explicit zero border."""
    N, C, H, Wd = D.shape
    M, _, R, S = W.shape
    E = (H + 2 * P - R) // U + 1
    F = (Wd + 2 * P - S) // U + 1
    O = np.zeros((N, M, E, F))
    for n in range(N):
        for m in range(M):
            for x in range(E):
                for y in range(F):
                    acc = 0.0
                    for k in range(C):
                        for i in range(R):
                            for j in range(S):
                                h, w = U * x + i - P, U * y + j - P
                                if 0 <= h < H and 0 <= w < Wd:
                                    acc += D[n, k, h, w] * W[m, k, i, j]
                    O[n, m, x, y] = acc
    return O


def test_golden_hand_examples():
    with open(os.path.join(GOLD, "eq1_hand.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        O = core.conv(np.array(c["D"], float), np.array(c["W"], float), c["stride"], c["pad"])
        np.testing.assert_array_equal(O, np.array(c["O"], float))


@pytest.mark.parametrize("shape", [
    (2, 3, 5, 5, 4, 3, 3, 1, 1),
    (1, 2, 7, 6, 3, 3, 2, 2, 1),
    (3, 1, 6, 6, 2, 1, 1, 2, 0),
    (2, 2, 9, 9, 2, 5, 5, 4, 0),
    (1, 3, 5, 5, 2, 3, 3, 1, 2),   # padding larger than needed
])
def test_brute_force_tiny(shape):
    N, C, H, Wd, M, R, S, U, P = shape
    g = np.random.default_rng(sum(shape))
    D = g.standard_normal((N, C, H, Wd))
    W = g.standard_normal((M, C, R, S))
    np.testing.assert_allclose(core.conv(D, W, U, P), brute_conv(D, W, U, P), rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("shape", [
    (4, 3, 32, 32, 16, 3, 3, 1, 1),      # the tiny single-layer case
    (2, 3, 35, 35, 8, 11, 11, 4, 0),     # an 11x11 stride-4 stem
    (2, 5, 15, 15, 6, 7, 7, 2, 3),       # a 7x7 stride-2 stem
    (3, 8, 14, 14, 5, 1, 1, 2, 0),       # a 1x1 stride-2 projection
    (2, 6, 13, 11, 7, 3, 5, 1, 2),       # non-square input and kernel
])
def test_against_torch_float64(shape):
    N, C, H, Wd, M, R, S, U, P = shape
    g = np.random.default_rng(7 + sum(shape))
    D = g.standard_normal((N, C, H, Wd))
    W = g.standard_normal((M, C, R, S))
    ref = torch.nn.functional.conv2d(torch.from_numpy(D), torch.from_numpy(W), stride=U, padding=P).numpy()
    np.testing.assert_allclose(core.conv(D, W, U, P), ref, rtol=1e-12, atol=1e-12)


def test_one_hot_input_gives_shifted_kernel():
    N, C, H, M, R, U, P = 2, 3, 9, 4, 3, 2, 1
    g = np.random.default_rng(3)
    W = g.standard_normal((M, C, R, R))
    n0, c0, h0, w0 = 1, 2, 4, 5
    D = np.zeros((N, C, H, H))
    D[n0, c0, h0, w0] = 1.0
    O = core.conv(D, W, U, P)
    E = (H + 2 * P - R) // U + 1
    expect = np.zeros_like(O)
    for m in range(M):
        for x in range(E):
            for y in range(E):
                i, j = h0 - U * x + P, w0 - U * y + P
                if 0 <= i < R and 0 <= j < R:
                    expect[n0, m, x, y] = W[m, c0, i, j]
    np.testing.assert_array_equal(O, expect)


def test_constant_input_interior_sums():
    g = np.random.default_rng(4)
    W = g.standard_normal((3, 2, 3, 3))
    D = np.full((2, 2, 8, 8), 2.0)
    O = core.conv(D, W, 1, 1)
    # interior positions see the whole kernel; corner (0,0) misses the first row and column
    np.testing.assert_allclose(O[:, :, 1:-1, 1:-1], 2.0 * W.sum(axis=(1, 2, 3))[None, :, None, None]
                               * np.ones((2, 3, 6, 6)), rtol=1e-14)
    np.testing.assert_allclose(O[0, :, 0, 0], 2.0 * W[:, :, 1:, 1:].sum(axis=(1, 2, 3)), rtol=1e-14)


def test_integer_inputs_are_exact():
    g = np.random.default_rng(5)
    D = g.integers(0, 4, (3, 16, 10, 10)).astype(float)
    W = g.integers(-2, 3, (5, 16, 3, 3)).astype(float)
    O = core.conv(D, W, 1, 1)
    # integer arithmetic by einsum over an explicit zero-padded copy
    Dp = np.pad(D.astype(np.int64), ((0, 0), (0, 0), (1, 1), (1, 1)))
    Wi = W.astype(np.int64)
    exact = np.zeros(O.shape, dtype=np.int64)
    for i in range(3):
        for j in range(3):
            exact += np.einsum("nchw,mc->nmhw", Dp[:, :, i:i + 10, j:j + 10], Wi[:, :, i, j])
    np.testing.assert_array_equal(O, exact.astype(float))


def test_points_match_full_conv():
    g = np.random.default_rng(6)
    D = g.standard_normal((3, 4, 11, 11))
    W = g.standard_normal((5, 4, 3, 3))
    O = core.conv(D, W, 2, 1)
    pts = np.array([[n, m, x, y] for n in range(3) for m in range(5) for x in (0, 2, 5) for y in (0, 3, 5)])
    np.testing.assert_array_equal(core.conv_points(D, W, 2, 1, pts), O[pts[:, 0], pts[:, 1], pts[:, 2], pts[:, 3]])


@pytest.mark.parametrize("h,r,u,p,e", [(227, 11, 4, 0, 55), (224, 7, 2, 3, 112), (56, 1, 2, 0, 28),
                                       (56, 3, 2, 1, 28), (13, 3, 1, 1, 13), (416, 3, 1, 1, 416),
                                       (3, 5, 1, 0, 0)])
def test_out_extent(h, r, u, p, e):
    assert core.out_extent(h, r, u, p) == e
