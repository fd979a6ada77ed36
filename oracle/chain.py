"""Chained protected inference over a stack of convolution layers, in float64.

TEST INFRASTRUCTURE ONLY: the oracle that the HIP library's chained path is
checked against.  Only tests, the smoke check and the benchmark's CPU-baseline
leg use it.

The paper protects every convolution layer of a network on its own (Sec. 3,
Sec. 4.3; the networks of Sec. 6): a layer's input checksums Cd1, Cd2 are
encoded from the input that layer actually receives, which in a network is the
previous layer's output after that layer's correction and after the operations
between the two layers.  Here those operations are a ReLU and, where the
spatial size drops between the layers, a max pooling (window k, stride s,
no padding), as in AlexNet, VGG-19 and Darknet-19.  Both are applied to the
stored values, so they are exact in any dtype.

Readings (shared with the HIP library):

* ReLU maps every value that is not greater than zero (negative values, both
  zeros, NaN) to +0;
* the pooling between two layers is the one of (2, 2) and (3, 2) that maps the
  first layer's output size onto the second layer's input size with no row or
  column left over ((e - k) divisible by s: AlexNet's overlapping 3x3/2 on its
  odd maps, 2x2/2 on VGG-19's and Darknet-19's even ones); equal sizes mean no
  pooling.
"""
import dataclasses
from typing import List, Optional, Sequence, Tuple

import numpy as np

from . import workflow as wf


def relu(x: np.ndarray) -> np.ndarray:
    """max(x, 0) with every non-positive value (and NaN) mapped to +0."""
    x = np.asarray(x, dtype=np.float64)
    return np.where(x > 0.0, x, 0.0)


def max_pool(x: np.ndarray, k: int, s: int) -> np.ndarray:
    """Max over k x k windows at stride s, no padding: out[n][c][i][j] is the
    largest x[n][c][s*i + a][s*j + b] for 0 <= a, b < k."""
    x = np.asarray(x, dtype=np.float64)
    N, C, H, W = x.shape
    Ho, Wo = (H - k) // s + 1, (W - k) // s + 1
    out = np.empty((N, C, Ho, Wo))
    for i in range(Ho):
        for j in range(Wo):
            out[:, :, i, j] = x[:, :, s * i:s * i + k, s * j:s * j + k].max(axis=(2, 3))
    return out


def pool_for(e: int, h_next: int) -> Tuple[int, int]:
    """The (k, s) pooling that maps an output of size e onto the next layer's input size."""
    if e == h_next:
        return 1, 1
    for k, s in ((2, 2), (3, 2)):
        if e >= k and (e - k) % s == 0 and (e - k) // s + 1 == h_next:
            return k, s
    raise ValueError(f"no 2x2/2 or 3x3/2 max pooling maps {e} onto {h_next} exactly")


def link(O: np.ndarray, k: int, s: int) -> np.ndarray:
    """The operations between two layers: ReLU, then k x k / s max pooling (k = s = 1: none)."""
    a = relu(O)
    return a if k == 1 and s == 1 else max_pool(a, k, s)


@dataclasses.dataclass
class ChainResult:
    layers: List[wf.LayerResult]     # one protected layer each, in order
    inputs: List[np.ndarray]         # the input each layer received (float64)
    links: List[Tuple[int, int]]     # (k, s) after each layer but the last
    output: np.ndarray               # the last layer's corrected output


def links_for(shapes: Sequence[Tuple[int, int, int, int, int]]) -> List[Tuple[int, int]]:
    """shapes: per layer (h, r, stride, pad, m).  The pooling between consecutive layers."""
    out = []
    for a, b in zip(shapes[:-1], shapes[1:]):
        h, r, u, p, _ = a
        e = (h + 2 * p - r) // u + 1
        out.append(pool_for(e, b[0]))
    return out


def protect_chain(D0: np.ndarray, Ws: Sequence[np.ndarray], strides: Sequence[int], pads: Sequence[int],
                  links: Sequence[Tuple[int, int]], dtype: str, policy: Optional[wf.Policy] = None,
                  faults: Optional[Sequence[Sequence[wf.Fault]]] = None) -> ChainResult:
    """Protect each layer in turn; layer l + 1 receives link(corrected output of layer l, *links[l]).

    faults[l] are the faults planted in layer l's output (Sec. 6.1).
    """
    L = len(Ws)
    if len(links) != L - 1:
        raise ValueError("one (k, s) link between each pair of layers")
    faults = faults or [()] * L
    D = wf.store(np.asarray(D0, dtype=np.float64), dtype)
    results, inputs = [], []
    for l in range(L):
        inputs.append(D)
        res = wf.protect(D, Ws[l], strides[l], pads[l], dtype, policy, faults[l])
        results.append(res)
        if l + 1 < L:
            D = link(res.O, *links[l])
    return ChainResult(results, inputs, list(links), results[-1].O)
