"""Host-only: the full-size whole-output parity cases (tests/fullsize_cases.py) reach every
convolution kernel that the workloads' layers launch, on both paths (ftcnn_conv_tile), so that a
retuned tile choice cannot leave a kernel without a full-size comparison against the oracle."""
import pytest

import paper_2003_12203_amd as ft
import workloads as wl
from fullsize_cases import CASES, GROUPED_ALEXNET, layer


def _key(spec, groups, path):
    d = ft.make_desc(spec.n, spec.ch, spec.h, spec.w, spec.m, spec.r, spec.s, spec.stride, spec.pad,
                     spec.dtype, groups=groups)
    t = ft.conv_tile(d, path)
    # the kernel itself: a layer that reads D as given runs the same kernel on both paths
    return (spec.dtype, t["tm"], t["tp"], t["tk"], t["loop"], t["nhwc"], t["group_skip"])


def _workload_keys():
    keys = {}
    for cfg in wl.configs()[1:] + [wl.vgg19_bf16()]:
        for L in cfg.layers:
            for path in (0, 1):
                keys.setdefault(_key(L, 1, path), f"{cfg.name}.{L.name} path {path}")
    for L in wl.config(1).layers:
        if L.name in GROUPED_ALEXNET:
            keys.setdefault(_key(L, 2, 1), f"alexnet-g2.{L.name} path 1")
    return keys


def test_every_workload_kernel_has_a_full_size_case():
    covered = set()
    for name, lname, groups, _bias, path in CASES:
        cfg, li = layer(name, lname)
        covered.add(_key(cfg.layers[li], groups, path))
    missing = {k: v for k, v in _workload_keys().items() if k not in covered}
    assert not missing, f"kernels without a full-size whole-output case: {missing}"


def test_cases_name_real_layers():
    for c in CASES:
        cfg, li = layer(c[0], c[1])
        assert cfg.layers[li].name == c[1]
        if c[2] > 1:
            spec = cfg.layers[li]
            assert spec.ch % c[2] == 0 and spec.m % c[2] == 0


def test_conv_tile_query_rejects_bad_arguments():
    d = ft.make_desc(2, 3, 8, 8, 4, 3, 3)
    with pytest.raises(ft.FtcnnError):
        ft.conv_tile(d, 2)
    with pytest.raises(ft.FtcnnError):
        ft.conv_tile(ft.make_desc(0, 3, 8, 8, 4, 3, 3), 1)
