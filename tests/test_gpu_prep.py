"""The channels-last copy that precedes the convolution on layers with 32-channel multiples
(and encodes Cd1, Cd2 of Sec. 3.2 on the way), on the layouts it distinguishes:

* H*W a multiple of the 16-byte vector (row segments start on a vector) or not (each channel
  row of a tile starts inside a vector, by a shift that depends on the channel);
* 32- or 64-channel tiles (bf16 layers with many tiles take 64);
* images split into ranges (partials combined by the convolution launch) or walked whole;
* D and W 16-byte aligned (vector loads) or not (element loads, same tile layout).

On integer data every sum is exact, so Cd1, Cd2 equal the oracle's encode bit for bit, the
output equals the oracle's eq. (1) within the dtype's rounding, the misaligned copies give
bitwise the aligned path's output, and no position is flagged.
"""
import numpy as np
import pytest
import torch

import workloads as wl
from gpu_util import TOL, assert_close_scaled, dev, host, layer_for
from oracle import core
from oracle import workflow as wf

pytestmark = pytest.mark.gpu

SHAPES = [
    # n, ch, h, m, r, u, p, dtype
    (4, 64, 14, 32, 3, 1, 1, "bf16"),     # H*W = 196: shifted rows
    (6, 64, 7, 64, 3, 1, 1, "bf16"),      # H*W = 49: odd
    (64, 32, 7, 32, 3, 1, 1, "bf16"),     # two image ranges
    (3, 32, 16, 32, 3, 2, 1, "bf16"),     # H*W = 256: aligned rows
    (2, 64, 170, 16, 3, 1, 1, "bf16"),    # 64-channel tiles with shifted rows
    (2, 64, 184, 16, 3, 1, 1, "bf16"),    # 64-channel tiles, aligned rows
    (3, 32, 13, 48, 3, 1, 1, "f32"),      # H*W = 169
    (2, 32, 27, 40, 5, 1, 2, "f32"),      # H*W = 729
    (40, 32, 9, 32, 1, 1, 0, "f32"),      # two image ranges, 1x1
    (3, 64, 12, 32, 3, 1, 1, "f32"),      # H*W = 144: aligned rows
]


def _misaligned(t: torch.Tensor) -> torch.Tensor:
    """A contiguous copy of t whose data starts one element past a 16-byte boundary."""
    buf = torch.empty(t.numel() + 1, dtype=t.dtype, device=t.device)
    out = buf[1:].view(t.shape)
    out.copy_(t)
    assert out.data_ptr() % 16 != 0
    return out


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "-".join(map(str, s)))
def test_channels_last_copy_layouts(shape):
    n, ch, h, m, r, u, p, dt = shape
    spec = wl.LayerSpec("prep", n, ch, h, h, m, r, r, u, p, dt)
    seed = 31 + sum(shape[:7])
    D, W = wl.gen_int_d(spec, seed), wl.gen_int_w(spec, seed)
    print(f"[prep] {shape}", flush=True)
    cd1, cd2 = wf.encode(D, 0)
    O_ref = core.conv(D, W, u, p)
    outs = []
    for misaligned in (False, True):
        lay = layer_for(spec)
        Dd, Wd = dev(D, dt), dev(W, dt)
        if misaligned:
            Dd, Wd = _misaligned(Dd), _misaligned(Wd)
        lay.encode_weights(Wd)
        O = lay.empty_output()
        lay.conv_sums(Dd, Wd, O, encode=True)
        lay.verify_correct_sums(Dd, Wd, O, coc=True)
        rep = lay.read_report()
        assert not rep.detected and rep.n_flagged == 0, ("flagged", misaligned)
        b = {k: v.cpu().numpy() for k, v in lay.buf.items()}
        np.testing.assert_array_equal(b["cd1"], cd1.ravel())
        np.testing.assert_array_equal(b["cd2"], cd2.ravel())
        if dt == "f32":
            np.testing.assert_array_equal(host(O), O_ref)
            np.testing.assert_array_equal(b["co5"], b["so5"])
        else:
            assert_close_scaled(host(O), O_ref, TOL[dt], "O")
        outs.append(O)
    view = torch.int16 if dt == "bf16" else torch.int32
    assert torch.equal(outs[0].view(view), outs[1].view(view)), "misaligned inputs changed the output"
