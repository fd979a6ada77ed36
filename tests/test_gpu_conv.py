"""GPU parity of the main convolution (eq. 1) against the oracle, every layer shape of the workloads.

Both convolution paths are checked: ftcnn_conv_fwd (D and W as given) and ftcnn_conv_fwd_ws (the
path of the protected calls, which reads channels-last copies when Ch is a multiple of 32)."""
import numpy as np
import pytest
import torch

import workloads as wl
from gpu_util import TOL, assert_close_scaled, dev, host, layer_for, workload_shapes
from oracle import core
from oracle import workflow as wf

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("path", ["conv_fwd", "conv_fwd_ws"])
@pytest.mark.parametrize("cfg,li,spec", workload_shapes())
def test_conv_matches_oracle(cfg, li, spec, path):
    D = wl.gen_d(cfg, li, spec)
    W = wl.gen_w(cfg, li, spec)
    lay = layer_for(spec)
    Dd, Wd = dev(D, spec.dtype), dev(W, spec.dtype)
    O = lay.empty_output()
    if path == "conv_fwd":
        lay.conv(Dd, Wd, O)
    else:
        lay.conv_ws(Dd, Wd, O)
    torch.cuda.synchronize()
    ref = wf.store(core.conv(D, W, spec.stride, spec.pad), spec.dtype)
    assert_close_scaled(host(O), ref, TOL[spec.dtype], f"O {spec}")


@pytest.mark.parametrize("shape", [
    # n, ch, h, m, r, stride, pad: ragged pixel tails, partial M tiles, K tails, 1x1 outputs
    (3, 16, 10, 5, 3, 1, 1),
    (1, 3, 11, 96, 11, 4, 0),
    (2, 7, 9, 33, 3, 2, 1),
    (2, 5, 3, 7, 3, 1, 0),       # E = 1
    (1, 1, 1, 1, 1, 1, 0),       # a single multiply
    (4, 64, 7, 130, 1, 1, 0),    # M just past a 128 tile
    (2, 8, 13, 64, 5, 3, 2),
    # channels-last path (Ch a multiple of 32): ragged tiles, strides, 1x1, K tails of whole (r, s)
    (3, 32, 9, 40, 3, 1, 1),
    (2, 64, 7, 130, 1, 1, 0),
    (2, 96, 13, 70, 5, 2, 2),
    (1, 32, 5, 33, 3, 2, 0),
    (4, 128, 6, 256, 3, 1, 1),
])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("path", ["conv_fwd", "conv_fwd_ws"])
def test_conv_integer_inputs_bitwise(shape, dtype, path):
    """Integer inputs keep every partial sum exact, so the GPU result must equal the oracle bit for bit."""
    n, ch, h, m, r, u, p = shape
    spec = wl.LayerSpec("int", n, ch, h, h, m, r, r, u, p, dtype)
    D = wl.gen_int_d(spec, seed=sum(shape))
    W = wl.gen_int_w(spec, seed=sum(shape))
    lay = layer_for(spec)
    O = lay.empty_output()
    if path == "conv_fwd":
        lay.conv(dev(D, dtype), dev(W, dtype), O)
    else:
        lay.conv_ws(dev(D, dtype), dev(W, dtype), O)
    torch.cuda.synchronize()
    ref = wf.store(core.conv(D, W, u, p), dtype)  # exact sums, one rounding to the dtype on both sides
    np.testing.assert_array_equal(host(O), ref)


def test_conv_deterministic():
    cfg = wl.config(1)
    spec = cfg.layers[2].with_(n=4)
    lay = layer_for(spec)
    D, W = dev(wl.gen_d(cfg, 2, spec), "f32"), dev(wl.gen_w(cfg, 2, spec), "f32")
    O1, O2 = lay.empty_output(), lay.empty_output()
    lay.conv(D, W, O1)
    lay.conv(D, W, O2)
    torch.cuda.synchronize()
    assert torch.equal(O1, O2)
