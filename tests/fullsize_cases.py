"""Full-size layers whose whole output the GPU tests compare with the oracle: one layer per
convolution kernel that the workloads launch (ftcnn_conv_tile), at its full batch and size.

Path 1 is every call that takes a workspace (the protected path and its unprotected baseline,
``ftcnn_conv_fwd_ws``); path 0 is ``ftcnn_conv_fwd`` (the separate-kernel path).  A case is
(workload name, layer name, groups, bias, path).  ``tests/test_tile_coverage.py`` checks on the
host that these cases reach every kernel that the workloads' layers reach.
"""
from __future__ import annotations

import workloads as wl

CASES = [
    # path 1: the protected convolution (epilogue with the CoC-D sums) and its plain twin
    ("darknet19", "c1", 1, False, 1),     # fp32 32 x 256, gathered from NCHW (3-channel stem)
    ("alexnet", "conv1", 1, False, 1),    # fp32 96 x 128, NCHW, 11x11 stride 4
    ("vgg19", "v1", 1, False, 1),         # fp32 64 x 128, NCHW
    ("darknet19", "c4", 1, False, 1),     # fp32 64 x 256, channels-last, 1x1
    ("alexnet", "conv5", 1, False, 1),    # fp32 128 x 64, channels-last, stream-K
    ("darknet19", "c10", 1, False, 1),    # fp32 64 x 64, channels-last, 1x1
    ("alexnet", "conv4", 1, False, 1),    # fp32 128 x 64, channels-last
    ("alexnet", "conv2", 1, False, 1),    # fp32 128 x 128, channels-last (the largest AlexNet layer), stream-K
    ("alexnet", "conv2", 1, True, 1),     # ... with a bias in the epilogue (Sec. 5.1)
    ("alexnet", "conv2", 2, False, 1),    # fp32 128 x 128, channels-last, grouped channel skip (Sec. 5.2)
    ("alexnet", "conv4", 2, False, 1),    # fp32 64 x 64, channels-last, grouped channel skip
    ("vgg19", "v10", 1, True, 1),         # fp32 128 x 128, 32-deep chunks, with a bias, stream-K
    ("vgg19_bf16", "v1", 1, False, 1),    # bf16 64 x 256, NCHW
    ("resnet18", "l1.0", 1, False, 1),    # bf16 64 x 128, direct-to-LDS
    ("resnet18", "l3.0", 1, False, 1),    # bf16 128 x 128, direct-to-LDS
    ("resnet18", "l4.0", 1, False, 1),    # bf16 128 x 64, direct-to-LDS (fewer 128 x 128 tiles than CUs)
    ("vgg19_bf16", "v10", 1, False, 1),   # bf16 256 x 256, direct-to-LDS
    ("vgg19_bf16", "v10", 1, True, 1),    # ... with a bias
    # path 0: ftcnn_conv_fwd on the layers whose kernel differs from path 1's
    ("alexnet", "conv5", 1, False, 0),    # fp32 64 x 64, NCHW
    ("alexnet", "conv4", 1, False, 0),    # fp32 128 x 64, NCHW
    ("alexnet", "conv2", 1, False, 0),    # fp32 128 x 128, NCHW
    ("darknet19", "c4", 1, False, 0),     # fp32 64 x 128, NCHW, 1x1
    ("resnet18", "l1.0", 1, False, 0),    # bf16 64 x 256, NCHW
    ("resnet18", "l3.0", 1, False, 0),    # bf16 128 x 128, 64-deep chunks
    ("vgg19_bf16", "v10", 1, False, 0),   # bf16 256 x 256, register-staged
]

# AlexNet with Caffe's two groups (the benchmark's --groups workload)
GROUPED_ALEXNET = ("conv2", "conv4", "conv5")


def workload(name: str) -> wl.Config:
    if name == "vgg19_bf16":
        return wl.vgg19_bf16()
    return {c.name: c for c in wl.configs()}[name]


def layer(name: str, lname: str):
    cfg = workload(name)
    for li, L in enumerate(cfg.layers):
        if L.name == lname:
            return cfg, li
    raise KeyError((name, lname))


def case_id(c) -> str:
    name, lname, groups, bias, path = c
    return f"{name}-{lname}" + (f"-g{groups}" if groups > 1 else "") + ("-bias" if bias else "") + f"-path{path}"
