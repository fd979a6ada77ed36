"""The oracle's chained protected inference, pinned to what the definitions fix.

* max pooling equals torch's max_pool2d (a library routine, float64 on the CPU) and a
  brute-force loop over its definition; ReLU satisfies relu(x) - relu(-x) = x and
  relu(x) + relu(-x) = |x|, and maps -0 and NaN to +0;
* the pooling chosen between layers is AlexNet's 3x3/2, VGG-19's and Darknet-19's 2x2/2 (the
  windows tile the map with nothing left over);
* a fault-free chain equals the plain composition conv -> ReLU -> pool written with torch's
  conv2d and max_pool2d (integer data: every value exact);
* with a fault planted in every layer, each layer corrects its own fault, receives the same
  input as in the fault-free chain, and the chain ends on the fault-free output bit for bit;
  a layer's Cd1, Cd2 are encoded from the corrected and pooled output of the layer before;
* a layer that falls back to recomputation still hands the clean output on.
"""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import chain
from oracle import workflow as wf
from paper_2003_12203_amd import schemes


def _brute_pool(x, k, s):
    N, C, H, W = x.shape
    Ho, Wo = (H - k) // s + 1, (W - k) // s + 1
    out = np.full((N, C, Ho, Wo), -np.inf)
    for n in range(N):
        for c in range(C):
            for i in range(Ho):
                for j in range(Wo):
                    for a in range(k):
                        for b in range(k):
                            out[n, c, i, j] = max(out[n, c, i, j], x[n, c, s * i + a, s * j + b])
    return out


@pytest.mark.parametrize("k,s,h", [(2, 2, 8), (2, 2, 9), (3, 2, 11), (3, 2, 7), (1, 1, 5)])
def test_max_pool(k, s, h):
    x = np.random.default_rng([12203, 91, k, h]).normal(size=(2, 3, h, h + 1))
    got = chain.max_pool(x, k, s)
    ref = torch.nn.functional.max_pool2d(torch.from_numpy(x), k, s).numpy()
    np.testing.assert_array_equal(got, ref)
    np.testing.assert_array_equal(got, _brute_pool(x, k, s))


def test_relu():
    x = np.random.default_rng([12203, 92]).normal(size=1000)
    np.testing.assert_array_equal(chain.relu(x) - chain.relu(-x), x)
    np.testing.assert_array_equal(chain.relu(x) + chain.relu(-x), np.abs(x))
    z = chain.relu(np.array([-0.0, 0.0, np.nan, -np.inf, np.inf]))
    assert list(z[:4]) == [0.0] * 4 and not np.signbit(z[:4]).any() and z[4] == np.inf


def test_links_of_the_networks():
    def links(cfg):
        return chain.links_for([(l.h, l.r, l.stride, l.pad, l.m) for l in cfg.layers])
    assert links(wl.config(1)) == [(3, 2), (3, 2), (1, 1), (1, 1)]                # AlexNet
    assert links(wl.config(2)) == [(1, 1), (2, 2), (1, 1), (2, 2)] + [(1, 1)] * 3 + [(2, 2)] \
        + [(1, 1)] * 3 + [(2, 2)] + [(1, 1)] * 3                                  # VGG-19
    assert links(wl.config(4))[:2] == [(2, 2), (2, 2)]                           # Darknet-19
    for e, h in ((10, 7), (8, 3)):      # no fit; 2x2/2 would drop a row of 8 -> 3 (and 3x3/2 too)
        with pytest.raises(ValueError):
            chain.pool_for(e, h)


def _int_chain(seed, n=5, chs=(3, 4, 6, 4), hs=(12, 12, 6), pads=(1, 1, 0), rs=(3, 3, 1)):
    g = np.random.default_rng([12203, 93, seed])
    D0 = g.integers(0, 3, size=(n, chs[0], hs[0], hs[0])).astype(np.float64)
    Ws = [g.integers(-1, 2, size=(chs[l + 1], chs[l], rs[l], rs[l])).astype(np.float64)
          for l in range(len(chs) - 1)]
    strides = [1] * len(Ws)
    shapes = [(hs[l], rs[l], 1, pads[l], chs[l + 1]) for l in range(len(Ws))]
    return D0, Ws, strides, list(pads[:len(Ws)]), chain.links_for(shapes)


def _torch_chain(D0, Ws, strides, pads, links):
    x = torch.from_numpy(D0)
    for l, W in enumerate(Ws):
        x = torch.nn.functional.conv2d(x, torch.from_numpy(W), stride=strides[l], padding=pads[l])
        if l + 1 < len(Ws):
            k, s = links[l]
            x = torch.relu(x)
            if (k, s) != (1, 1):
                x = torch.nn.functional.max_pool2d(x, k, s)
    return x.numpy()


def test_chain_fault_free_is_the_composition():
    D0, Ws, strides, pads, links = _int_chain(1)
    assert links == [(1, 1), (2, 2)]
    res = chain.protect_chain(D0, Ws, strides, pads, links, "f32")
    np.testing.assert_array_equal(res.output, _torch_chain(D0, Ws, strides, pads, links))
    assert all(not r.report.detected for r in res.layers)
    assert [x.shape[2] for x in res.inputs] == [12, 12, 6]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_chain_corrects_every_layer(dtype):
    D0, Ws, strides, pads, links = _int_chain(2)
    clean = chain.protect_chain(D0, Ws, strides, pads, links, dtype)
    faults = []
    for l, r in enumerate(clean.layers):
        N, M, E, F = r.O.shape
        faults.append([wf.Fault(l % N, (2 * l + 1) % M, E // 2, F - 1, "add", value=4096.0)])
    res = chain.protect_chain(D0, Ws, strides, pads, links, dtype, faults=faults)
    for l, r in enumerate(res.layers):
        f = faults[l][0]
        assert r.report.fixes == [(f.n, f.m, f.x, f.y, wf.SCHEME_COC)]
        assert r.report.status == wf.STATUS_CORRECTED
        np.testing.assert_array_equal(res.inputs[l], clean.inputs[l])
        # the layer's input checksums come from the corrected, pooled output of the layer before
        np.testing.assert_array_equal(r.ck.cd1, res.inputs[l].sum(axis=0))
        np.testing.assert_array_equal(r.ck.cd2, np.tensordot(np.arange(res.inputs[l].shape[0], dtype=np.float64),
                                                             res.inputs[l], axes=1))
    np.testing.assert_array_equal(res.output, clean.output)


def test_chain_recompute_hands_on_the_clean_output():
    D0, Ws, strides, pads, links = _int_chain(3, n=6, chs=(3, 8, 4), hs=(9, 9), pads=(1, 1), rs=(3, 3))
    clean = chain.protect_chain(D0, Ws, strides, pads, links, "f32")
    N, M, E, F = clean.layers[0].O.shape
    # four blocks in two images and two filters at one position: beyond every scheme
    pat = schemes.pattern("square", N, M, E, F)
    faults = [[wf.Fault(q["n"], q["m"], q["x"], q["y"], "add", value=q["value"]) for q in pat], []]
    res = chain.protect_chain(D0, Ws, strides, pads, links, "f32", wf.Policy(rc_on=False, clc_on=False),
                              faults)
    assert res.layers[0].report.status == wf.STATUS_RECOMPUTED
    np.testing.assert_array_equal(res.inputs[1], clean.inputs[1])
    np.testing.assert_array_equal(res.output, clean.output)
