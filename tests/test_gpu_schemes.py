"""The correction-workflow measurement (bench.py --schemes) on small layers: every workflow's fault
pattern, with its RC/ClC switches, is resolved by the scheme the workflow table names, and a
repaired output equals the clean one (fp32 on integer data: exactly; bf16: within the output
rounding, since a repaired element is rebuilt from float64 checksums and rounded again)."""
import numpy as np
import pytest
import torch

import workloads as wl
from gpu_util import TOL, assert_close_scaled, dev, host, layer_for
from paper_2003_12203_amd import schemes

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("ch", [4, 32])   # NCHW gather and channels-last paths
def test_every_workflow_resolves_as_named(dtype, ch):
    spec = wl.LayerSpec("wf", 6, ch, 12, 12, 8, 3, 3, 1, 1, dtype)
    D, W = wl.gen_int_d(spec, 17), wl.gen_int_w(spec, 17)
    lay = layer_for(spec)
    Dd, Wd = dev(D, dtype), dev(W, dtype)
    lay.encode_weights(Wd)
    print(f"[schemes] {dtype} ch{ch}", flush=True)
    res = schemes.measure(lay, Dd, Wd, reps=2)
    assert set(res) == {"error-free"} | set(schemes.WORKFLOWS)
    for name, v in res.items():
        if name == "error-free":
            continue
        assert tuple(v["resolved"]) == schemes.WORKFLOWS[name][3], (name, v)
    clean = lay.empty_output()
    lay.conv_ws(Dd, Wd, clean)
    O = lay.empty_output()
    pol = lay.policy
    lay.conv_sums(Dd, Wd, O, schemes.pattern("row", 6, 8, lay.E, lay.F), encode=True)
    lay.verify_correct_sums(Dd, Wd, O, coc=True)
    torch.cuda.synchronize()
    if dtype == "f32":
        assert torch.equal(O.view(torch.int32), clean.view(torch.int32))
    else:
        assert_close_scaled(host(O), host(clean), TOL[dtype], "repaired O")
    assert lay.policy is pol
