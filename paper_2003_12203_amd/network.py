"""Chained protected inference over a stack of convolution layers.

Every convolution layer of the network is protected on its own (Sec. 3, Sec. 4.3; the
networks of Sec. 6): layer l + 1 receives ReLU and max pooling of layer l's output after
layer l's correction, and encodes its Cd1, Cd2 from exactly that input.  Everything runs
in the library's kernels on one stream:

    per layer: ftcnn_conv_fwd_sums_given (channels-last copy, convolution + sums)
               ftcnn_verify_correct_sums (Co5..Co7, CoC-D, the correction chain)
               ftcnn_relu_pool_encode into the next layer's input and its Cd1, Cd2

(the first layer encodes its own input in ftcnn_conv_fwd_sums' copy).  The next layer's
checksums are thus encoded in the pass that writes its input, from the corrected values.

and nothing waits on the host between layers.  Recomputation (Sec. 4.1.1) is the one
decision the host takes: after the pass, the reports are read once, and from the first
layer that asks for it the layer is recomputed and the layers after it run again.

The pooling between two layers is the one of 2x2/2 and 3x3/2 (no padding) that maps the
first layer's output size onto the second layer's input size with no row or column left
over (AlexNet's 3x3/2 on its odd maps, 2x2/2 on VGG-19's and Darknet-19's even ones);
equal sizes mean ReLU only.
"""
from __future__ import annotations

import ctypes as C
from typing import List, Optional, Sequence, Tuple

import torch

from . import _lib
from . import (STATUS_FAILED, STATUS_NEEDS_RECOMPUTE, STATUS_RECOMPUTED, FtcnnError, Layer, Report,
               make_policy, parse_report, relu_pool)


def pooling(e: int, h_next: int) -> Tuple[int, int]:
    """(k, s) between an output of size e and a next input of size h_next."""
    if e == h_next:
        return 1, 1
    for k, s in ((2, 2), (3, 2)):
        if e >= k and (e - k) % s == 0 and (e - k) // s + 1 == h_next:
            return k, s
    raise FtcnnError(f"no 2x2/2 or 3x3/2 max pooling maps an output of {e} onto an input of {h_next}")


class Chain:
    """Layers given as (n, ch, h, w, m, r, s, stride, pad), one dtype; consecutive layers must
    agree on the batch and on channels (m of layer l = ch of layer l + 1)."""

    def __init__(self, specs: Sequence[Tuple[int, ...]], dtype: str = "f32", policy=None,
                 device: str = "cuda", fuse_encode: bool = True):
        if not specs:
            raise FtcnnError("a chain needs at least one layer")
        # fuse_encode: the link between layers (ReLU, pooling) also encodes the next layer's
        # Cd1, Cd2 from the values it writes (ftcnn_relu_pool_encode), and that layer takes them
        # as given (ftcnn_conv_fwd_sums_given); otherwise each layer encodes in its own copy
        self.fuse_encode = fuse_encode
        self.policy = policy or make_policy()
        self.layers: List[Layer] = [Layer(*sp, dtype=dtype, policy=self.policy, device=device) for sp in specs]
        self.links: List[Tuple[int, int]] = []
        for a, b in zip(self.layers[:-1], self.layers[1:]):
            n, m, E, F = a.shape_o
            nb, cb, hb, wb = b.shape_d
            if (n, m) != (nb, cb):
                raise FtcnnError(f"layer output {a.shape_o} does not feed layer input {b.shape_d}")
            k, s = pooling(E, hb)
            if (F - k) // s + 1 != wb or (F - k) % s:
                raise FtcnnError(f"pooling {k}x{k}/{s} does not map width {F} onto {wb}")
            self.links.append((k, s))
        # every layer's report in one buffer, so that the host reads them all with one copy
        sizes = [lay.report.numel() for lay in self.layers]
        assert len(set(sizes)) == 1, "the layers of a chain share one fix capacity"
        self._reports = torch.zeros(sum(sizes), dtype=torch.uint8, device=self.layers[0].report.device)
        off = 0
        for lay, sz in zip(self.layers, sizes):
            lay.report = self._reports[off:off + sz]
            off += sz
        self._report_sizes = sizes
        self.outputs = [lay.empty_output() for lay in self.layers]
        self.inputs: List[Optional[torch.Tensor]] = [None] + [
            torch.empty(lay.shape_d, dtype=lay.tdtype, device=lay.buf["cd1"].device) for lay in self.layers[1:]]
        self.W: List[Optional[torch.Tensor]] = [None] * len(self.layers)

    def set_weights(self, Ws: Sequence[torch.Tensor], stream=None):
        """The filters of every layer; their Cw1, Cw2 are encoded once, before the application."""
        if len(Ws) != len(self.layers):
            raise FtcnnError("one weight tensor per layer")
        for l, (lay, W) in enumerate(zip(self.layers, Ws)):
            if tuple(W.shape) != lay.shape_w or W.dtype != lay.tdtype:
                raise FtcnnError(f"layer {l}: weights must be {lay.shape_w} {lay.tdtype}")
            self.W[l] = W.contiguous()
            lay.encode_weights(self.W[l], stream)

    def _input(self, l: int, D0: torch.Tensor) -> torch.Tensor:
        return D0 if l == 0 else self.inputs[l]

    def launch(self, D0: torch.Tensor, faults: Optional[Sequence[Sequence[dict]]] = None, start: int = 0,
               stream=None, linked: bool = False):
        """Enqueue the protected layers start.. on the stream (no host wait).  faults[l] (testing)
        are planted in layer l's outputs before they are summed.  linked: layer start's input (and,
        with fuse_encode, its Cd1, Cd2) was just written by the link from layer start - 1."""
        if tuple(D0.shape) != self.layers[0].shape_d or D0.dtype != self.layers[0].tdtype:
            raise FtcnnError(f"input must be {self.layers[0].shape_d} {self.layers[0].tdtype}")
        if any(W is None for W in self.W):
            raise FtcnnError("set_weights first")
        for l in range(start, len(self.layers)):
            lay, D, O = self.layers[l], self._input(l, D0), self.outputs[l]
            # with fuse_encode, a layer after the first gets its Cd1, Cd2 from the pass that wrote
            # its input (below); the first layer, and a restart, encode in the channels-last copy
            given = self.fuse_encode and (l > start or (linked and l > 0))
            lay.conv_sums(D, self.W[l], O, faults[l] if faults else (), stream, encode=not given, given=given)
            lay.verify_correct_sums(D, self.W[l], O, stream, coc=True)
            if l + 1 < len(self.layers):
                self._link(l, O, stream)

    def _link(self, l: int, O: torch.Tensor, stream=None):
        nxt = self.layers[l + 1]
        cd = (nxt.buf["cd1"], nxt.buf["cd2"]) if self.fuse_encode else None
        relu_pool(O, *self.links[l], Y=self.inputs[l + 1], stream=stream, cd=cd, wbase=nxt.desc.wbase)

    def launch_plain(self, D0: torch.Tensor, stream=None):
        """The same network unprotected: the same convolution kernels with no ABFT work, and the
        same operations between the layers."""
        for l, lay in enumerate(self.layers):
            O = self.outputs[l]
            lay.conv_ws(self._input(l, D0), self.W[l], O, stream)
            if l + 1 < len(self.layers):
                relu_pool(O, *self.links[l], Y=self.inputs[l + 1], stream=stream)

    def _read_reports(self) -> List[Report]:
        """Every layer's report: the headers of all layers in one small copy, then the fix list
        of each layer that detected something."""
        torch.cuda.synchronize()
        L, sz = len(self.layers), self._report_sizes[0]
        hb = C.sizeof(_lib.ReportHeader)
        heads = self._reports.view(L, sz)[:, :hb].cpu().numpy()
        reps = []
        for l in range(L):
            h = _lib.ReportHeader.from_buffer_copy(heads[l].tobytes())
            if h.detected:
                nf = min(h.n_fixes, h.cap_fixes)
                reps.append(parse_report(self._reports[l * sz:l * sz + hb + nf * C.sizeof(_lib.Fix)]))
            else:
                reps.append(Report(False, h.n_flagged, h.status, list(h.resolved_by), [], h.n_fixes, h.cap_fixes))
        return reps

    def finish(self, D0: torch.Tensor, stream=None) -> List[Report]:
        """Read every layer's report (one synchronization); recompute from the first layer that
        needs it and run the layers after it again (their reports replace the first pass's)."""
        reps = self._read_reports()
        for l, rep in enumerate(reps):
            if rep.status != STATUS_NEEDS_RECOMPUTE:
                continue
            lay, D, O = self.layers[l], self._input(l, D0), self.outputs[l]
            lay.conv_sums(D, self.W[l], O, (), stream, encode=True)
            lay.verify_correct_sums(D, self.W[l], O, stream, coc=True)
            again = lay.read_report()
            rep.status = STATUS_FAILED if again.detected else STATUS_RECOMPUTED
            if l + 1 < len(self.layers):
                self._link(l, O, stream)
                self.launch(D0, None, l + 1, stream, linked=True)
                for j in range(l + 1, len(self.layers)):
                    reps[j] = self.layers[j].read_report()
        return reps

    def run(self, D0: torch.Tensor, faults=None, stream=None) -> Tuple[torch.Tensor, List[Report]]:
        """The whole network: its output (the last layer's corrected output) and every report."""
        self.launch(D0, faults, 0, stream)
        return self.outputs[-1], self.finish(D0, stream)
