"""The weight-memory check (Sec. 4.1.2) through the C ABI: Cw1 re-encoded from the current W
against the Cw1 encoded at set-up; the count of mismatching columns equals the oracle's and
the number of columns corrupted, and an intact W gives 0."""
import numpy as np
import pytest
import torch

import workloads as wl
from gpu_util import dev, layer_for
from oracle import workflow as wf

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(4, 3, 9, 16, 3), (2, 64, 7, 96, 3), (2, 32, 5, 300, 1)])
def test_weight_check_matches_oracle(dt, shape):
    n, ch, h, m, r = shape
    spec = wl.LayerSpec("w", n, ch, h, h, m, r, r, 1, r // 2, dt)
    cfg = wl.Config(95, "w", (spec,), "uniform", "he")
    W = wl.gen_w(cfg, 0, spec)
    lay = layer_for(spec)
    Wd = dev(W, dt)
    lay.encode_weights(Wd)
    assert lay.check_weights(Wd) == 0
    cw1 = lay.buf["cw1"].cpu().numpy()
    g = np.random.default_rng([12203, 72, ch, m])
    K = ch * r * r
    cols = g.choice(K, size=min(5, K), replace=False)
    W2 = W.copy().reshape(m, K)
    for k in cols:
        W2[g.integers(0, m), k] *= -2.0           # a flipped sign and exponent step, exact in bf16
    W2 = W2.reshape(W.shape)
    W2d = dev(W2, dt)
    got = lay.check_weights(W2d)
    ref = wf.check_weights(W2d.double().cpu().numpy() if dt == "f32" else W2d.float().double().cpu().numpy(),
                           wf.encode(Wd.double().cpu().numpy(), 0)[0])
    assert got == ref == len(cols)
    # the oracle re-encoding of the intact weights reproduces the GPU's Cw1 (to rounding order)
    np.testing.assert_allclose(cw1, wf.encode(W.astype(np.float64), 0)[0].ravel(), rtol=1e-12, atol=1e-12)
    torch.cuda.synchronize()
