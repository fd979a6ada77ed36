"""Checksum-protected convolution (FT-CNN, arXiv 2003.12203) on MI355X.

A thin Python binding over the C ABI of ``include/ftcnn.h``: the functions
below have the names of the C entry points and only marshal arguments (torch
device tensors become raw device pointers, the current torch stream becomes
the HIP stream).  Every step of the protected layer runs in the library's HIP
kernels; if ``libftcnn.so`` is missing, every call raises.

``Layer`` bundles the per-layer device buffers (checksums, workspace, report)
for convenience.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
from typing import Dict, List, Optional, Sequence

import torch

from . import _lib
from ._lib import (BF16, CO1, CO2, CO3, CO4, CO5, CO6, CO7, F32, REPAIR_CHECKSUM,  # noqa: F401
                   REPAIR_RECOMPUTE, SCHEME_CKSUM, SCHEME_CLC, SCHEME_COC, SCHEME_FC, SCHEME_NONE,
                   SCHEME_RC, SCHEME_UNRESOLVED, STATUS_CLEAN, STATUS_CORRECTED, STATUS_FAILED,
                   STATUS_NEEDS_RECOMPUTE, STATUS_RECOMPUTED)

DTYPES = {"f32": (F32, torch.float32), "bf16": (BF16, torch.bfloat16)}


class FtcnnError(RuntimeError):
    pass


def lib():
    return _lib.load()


def _check(rc: int, what: str) -> None:
    if rc != 0:
        msg = lib().ftcnn_last_error().decode(errors="replace")
        raise FtcnnError(f"{what} failed ({rc}): {msg}")


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise FtcnnError("expected a device tensor")
    return C.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def make_desc(n, ch, h, w, m, r, s, stride=1, pad=0, dtype="f32", wbase=0, groups=1) -> _lib.ConvDesc:
    return _lib.ConvDesc(n, ch, h, w, m, r, s, stride, pad, groups, DTYPES[dtype][0], wbase)


def make_policy(rc_on=True, clc_on=True, repair="checksum", kappa=16.0, eta=0.1) -> _lib.Policy:
    rep = REPAIR_RECOMPUTE if repair == "recompute" else REPAIR_CHECKSUM
    return _lib.Policy(int(rc_on), int(clc_on), rep, 0, float(kappa), float(eta))


# ---- the C entry points --------------------------------------------------------

def out_shape(desc) -> tuple:
    E, F = C.c_int32(), C.c_int32()
    _check(lib().ftcnn_out_shape(C.byref(desc), C.byref(E), C.byref(F)), "ftcnn_out_shape")
    return E.value, F.value


def workspace_bytes(desc) -> int:
    return int(lib().ftcnn_workspace_bytes(C.byref(desc)))


def report_bytes(cap: int) -> int:
    return int(lib().ftcnn_report_bytes(cap))


def conv_tile(desc, path: int = 1) -> dict:
    """ftcnn_conv_tile: the convolution kernel a layer's calls launch (host-only query)."""
    out = (C.c_int32 * 6)()
    _check(lib().ftcnn_conv_tile(C.byref(desc), int(path), out), "ftcnn_conv_tile")
    return {"tm": out[0], "tp": out[1], "tk": out[2], "loop": out[3], "nhwc": bool(out[4]),
            "group_skip": bool(out[5])}


def conv_stream_k(desc) -> int:
    """ftcnn_conv_stream_k: stream-K workgroups of the layer's workspace-path convolution on the
    current device (0: one workgroup per tile)."""
    out = C.c_int32(0)
    _check(lib().ftcnn_conv_stream_k(C.byref(desc), C.byref(out)), "ftcnn_conv_stream_k")
    return int(out.value)


def last_error() -> str:
    return lib().ftcnn_last_error().decode(errors="replace")


def encode(desc, which: int, X: torch.Tensor, c1: torch.Tensor, c2: torch.Tensor,
           workspace: torch.Tensor, stream=None) -> None:
    _check(lib().ftcnn_encode(C.byref(desc), which, _ptr(X), _ptr(c1), _ptr(c2), _ptr(workspace),
                              _stream(stream)), "ftcnn_encode")


def conv_fwd(desc, D: torch.Tensor, W: torch.Tensor, O: torch.Tensor, stream=None) -> None:
    _check(lib().ftcnn_conv_fwd(C.byref(desc), _ptr(D), _ptr(W), _ptr(O), _stream(stream)), "ftcnn_conv_fwd")


def checksum_conv(desc, which: int, D, W, ck: _lib.Checksums, stream=None) -> None:
    _check(lib().ftcnn_checksum_conv(C.byref(desc), which, _ptr(D), _ptr(W), C.byref(ck), _stream(stream)),
           "ftcnn_checksum_conv")


def verify(desc, O, ck, policy, report: torch.Tensor, cap: int, workspace, stream=None) -> None:
    _check(lib().ftcnn_verify(C.byref(desc), _ptr(O), C.byref(ck), C.byref(policy), _ptr(report), cap,
                              _ptr(workspace), _stream(stream)), "ftcnn_verify")


def correct(desc, D, W, O, ck, policy, report, workspace, stream=None) -> None:
    _check(lib().ftcnn_correct(C.byref(desc), _ptr(D), _ptr(W), _ptr(O), C.byref(ck), C.byref(policy),
                               _ptr(report), _ptr(workspace), _stream(stream)), "ftcnn_correct")


def verify_correct(desc, D, W, O, ck, policy, report, cap, workspace, stream=None) -> None:
    _check(lib().ftcnn_verify_correct(C.byref(desc), _ptr(D), _ptr(W), _ptr(O), C.byref(ck), C.byref(policy),
                                      _ptr(report), cap, _ptr(workspace), _stream(stream)),
           "ftcnn_verify_correct")


def check_weights(desc, W, cw1, mismatches: torch.Tensor, workspace, stream=None) -> None:
    _check(lib().ftcnn_check_weights(C.byref(desc), _ptr(W), _ptr(cw1), _ptr(mismatches), _ptr(workspace),
                                     _stream(stream)), "ftcnn_check_weights")


def conv_fwd_bias(desc, D, W, bias, O, workspace=None, stream=None) -> None:
    _check(lib().ftcnn_conv_fwd_bias(C.byref(desc), _ptr(D), _ptr(W), _ptr(bias), _ptr(O), _ptr(workspace),
                                     _stream(stream)), "ftcnn_conv_fwd_bias")


def relu_pool(X: torch.Tensor, k: int = 1, s: int = 1, Y: Optional[torch.Tensor] = None,
              stream=None, cd=None, wbase: int = 0) -> torch.Tensor:
    """ftcnn_relu_pool: k x k / s max pooling of relu(X) (k = s = 1: ReLU only), the operations
    between two layers of a network.  X is [n][c][h][w] (float32, or bfloat16); Y is allocated
    when not given.  cd = (cd1, cd2): ftcnn_relu_pool_encode, which also writes the next layer's
    input checksums of Y there (float64 [c][h'][w'])."""
    if X.dim() != 4 or not X.is_contiguous():
        raise FtcnnError("relu_pool: X must be a contiguous [n][c][h][w] tensor")
    dt = {torch.float32: "f32", torch.bfloat16: "bf16"}.get(X.dtype)
    if dt is None:
        raise FtcnnError(f"relu_pool: dtype {X.dtype}")
    n, c, h, w = X.shape
    shape = (n, c, (h - k) // s + 1, (w - k) // s + 1)
    if Y is None:
        Y = torch.empty(shape, dtype=X.dtype, device=X.device)
    elif tuple(Y.shape) != shape or Y.dtype != X.dtype or not Y.is_contiguous():
        raise FtcnnError(f"relu_pool: Y must be a contiguous {shape} tensor of {X.dtype}")
    if cd is None:
        _check(lib().ftcnn_relu_pool(DTYPES[dt][0], n, c, h, w, k, s, _ptr(X), _ptr(Y), _stream(stream)),
               "ftcnn_relu_pool")
        return Y
    cd1, cd2 = cd
    plane = c * shape[2] * shape[3]
    for t in (cd1, cd2):
        if t.dtype != torch.float64 or t.numel() != plane or not t.is_contiguous():
            raise FtcnnError(f"relu_pool: checksums must be contiguous float64 of {plane} elements")
    _check(lib().ftcnn_relu_pool_encode(DTYPES[dt][0], n, c, h, w, k, s, wbase, _ptr(X), _ptr(Y), _ptr(cd1),
                                        _ptr(cd2), _stream(stream)), "ftcnn_relu_pool_encode")
    return Y


def conv_fwd_ws(desc, D, W, O, workspace, stream=None) -> None:
    _check(lib().ftcnn_conv_fwd_ws(C.byref(desc), _ptr(D), _ptr(W), _ptr(O), _ptr(workspace), _stream(stream)),
           "ftcnn_conv_fwd_ws")


def conv_fwd_sums(desc, D, W, O, ck, report, cap, workspace, faults: Sequence[dict] = (), stream=None,
                  given: bool = False) -> None:
    """ftcnn_conv_fwd_sums; given=True: ftcnn_conv_fwd_sums_given (Cd1, Cd2 in ck are inputs)."""
    arr = _fault_array(faults)
    fn = lib().ftcnn_conv_fwd_sums_given if given else lib().ftcnn_conv_fwd_sums
    _check(fn(C.byref(desc), _ptr(D), _ptr(W), _ptr(O), C.byref(ck) if ck else None,
              _ptr(report), cap, arr if faults else None, len(faults), _ptr(workspace), _stream(stream)),
           "ftcnn_conv_fwd_sums_given" if given else "ftcnn_conv_fwd_sums")


def verify_correct_sums(desc, D, W, O, ck, policy, report, workspace, which: int = 0, stream=None) -> None:
    _check(lib().ftcnn_verify_correct_sums(C.byref(desc), _ptr(D), _ptr(W), _ptr(O), C.byref(ck),
                                           C.byref(policy), _ptr(report), which, _ptr(workspace),
                                           _stream(stream)),
           "ftcnn_verify_correct_sums")


def protected_conv(desc, D, W, O, ck, policy, report, cap, workspace, stream=None) -> None:
    _check(lib().ftcnn_protected_conv(C.byref(desc), _ptr(D), _ptr(W), _ptr(O), C.byref(ck),
                                      C.byref(policy), _ptr(report), cap, _ptr(workspace),
                                      _stream(stream)), "ftcnn_protected_conv")


def protected_conv_noalloc(desc, D, W, O, ck, policy, report, cap, stream=None) -> None:
    """ftcnn_protected_conv_noalloc: the protected layer with the library's static device scratch in
    place of a workspace (for callers that cannot allocate)."""
    _check(lib().ftcnn_protected_conv_noalloc(C.byref(desc), _ptr(D), _ptr(W), _ptr(O), C.byref(ck),
                                              C.byref(policy), _ptr(report), cap, _stream(stream)),
           "ftcnn_protected_conv_noalloc")


def set_kernel_events(before, after) -> None:
    """ftcnn_set_kernel_events: record two torch.cuda.Event objects (timing enabled) around the next
    launch of the convolution kernel on this thread.  The events are recorded once here first so
    that their HIP handles exist."""
    handles = []
    for ev in (before, after):
        if ev is None:
            handles.append(None)
            continue
        if ev.cuda_event == 0:
            ev.record()
        handles.append(C.c_void_p(ev.cuda_event))
    _check(lib().ftcnn_set_kernel_events(*handles), "ftcnn_set_kernel_events")


def _fault_array(faults: Sequence[dict]):
    arr = (_lib.Fault * max(1, len(faults)))()
    kinds = {"flip": 0, "add": 1, "set": 2}
    for i, f in enumerate(faults):
        arr[i] = _lib.Fault(f["n"], f["m"], f["x"], f["y"], kinds[f["kind"]], f.get("bit", 0),
                            float(f.get("value", 0.0)))
    return arr


def inject(desc, O, faults: Sequence[dict], stream=None) -> None:
    _check(lib().ftcnn_inject(C.byref(desc), _ptr(O), _fault_array(faults), len(faults), _stream(stream)),
           "ftcnn_inject")


# ---- report ----------------------------------------------------------------------

@dataclasses.dataclass
class Report:
    detected: bool
    n_flagged: int
    status: int
    resolved_by: List[int]
    fixes: List[tuple]        # sorted (n, m, x, y, scheme)
    n_fixes: int
    cap_fixes: int


def parse_report(buf: torch.Tensor) -> Report:
    raw = bytes(buf.cpu().numpy().tobytes())
    h = _lib.ReportHeader.from_buffer_copy(raw[:C.sizeof(_lib.ReportHeader)])
    nf = min(h.n_fixes, h.cap_fixes)
    fixes = []
    base = C.sizeof(_lib.ReportHeader)
    for i in range(nf):
        fx = _lib.Fix.from_buffer_copy(raw[base + i * C.sizeof(_lib.Fix): base + (i + 1) * C.sizeof(_lib.Fix)])
        fixes.append((fx.n, fx.m, fx.x, fx.y, fx.scheme))
    fixes.sort()
    return Report(bool(h.detected), h.n_flagged, h.status, list(h.resolved_by), fixes, h.n_fixes, h.cap_fixes)


# ---- per-layer buffers --------------------------------------------------------------

class Layer:
    """Device buffers of one protected layer and the calls that use them."""

    def __init__(self, n, ch, h, w, m, r, s, stride=1, pad=0, dtype="f32", wbase=0,
                 policy: Optional[_lib.Policy] = None, cap_fixes: int = 4096, device="cuda", groups: int = 1):
        self.desc = make_desc(n, ch, h, w, m, r, s, stride, pad, dtype, wbase, groups)
        self.groups = groups
        self.dtype = dtype
        self.tdtype = DTYPES[dtype][1]
        self.E, self.F = out_shape(self.desc)
        self.shape_d = (n, ch, h, w)
        self.shape_w = (m, ch // groups, r, s)   # grouped (Sec. 5.2): each filter sees ch / groups channels
        self.shape_o = (n, m, self.E, self.F)
        self.policy = policy or make_policy()
        self.cap = cap_fixes
        dev = torch.device(device)
        f64 = dict(dtype=torch.float64, device=dev)
        EF = self.E * self.F
        self.buf: Dict[str, torch.Tensor] = {
            "cd1": torch.zeros(ch * h * w, **f64), "cd2": torch.zeros(ch * h * w, **f64),
            "cw1": torch.zeros(ch * r * s, **f64), "cw2": torch.zeros(ch * r * s, **f64),
        }
        for k in ("co5", "co6", "co7", "so5", "so6", "so7", "q5"):
            self.buf[k] = torch.zeros(EF, **f64)
        self.ck = _lib.Checksums()
        self.bias: Optional[torch.Tensor] = None
        self._sync_ck()
        nbytes = workspace_bytes(self.desc)
        self._ws_raw = torch.empty(nbytes + 256, dtype=torch.uint8, device=dev)
        off = (-self._ws_raw.data_ptr()) % 256
        self.workspace = self._ws_raw[off:off + nbytes]
        self.report = torch.zeros(report_bytes(cap_fixes), dtype=torch.uint8, device=dev)

    def _sync_ck(self):
        for k, t in self.buf.items():
            setattr(self.ck, k, t.data_ptr())

    def want_row_col(self, rows: bool = True, cols: bool = True):
        n, m = self.shape_d[0], self.shape_w[0]
        EF = self.E * self.F
        dev = self.buf["cd1"].device
        if rows and "co1" not in self.buf:
            self.buf["co1"] = torch.zeros(m * EF, dtype=torch.float64, device=dev)
            self.buf["co3"] = torch.zeros(m * EF, dtype=torch.float64, device=dev)
        if cols and "co2" not in self.buf:
            self.buf["co2"] = torch.zeros(n * EF, dtype=torch.float64, device=dev)
            self.buf["co4"] = torch.zeros(n * EF, dtype=torch.float64, device=dev)
        self._sync_ck()

    def set_bias(self, bias: Optional[torch.Tensor], stream=None):
        """A bias [M] added to every output block O[n][m] (Sec. 5.1), kept in fp32 on the device,
        with its sums encoded once (ftcnn_encode, which = 2); None removes it."""
        if bias is None:
            self.bias = None
            self.ck.bias = None
            self.ck.cb = None
            return
        b = bias.detach().to(device=self.buf["cd1"].device, dtype=torch.float32).contiguous().reshape(-1)
        if b.numel() != self.shape_w[0]:
            raise FtcnnError(f"bias has {b.numel()} elements, the layer {self.shape_w[0]} filters")
        self.bias = b
        if "cb" not in self.buf:
            self.buf["cb"] = torch.zeros(2, dtype=torch.float64, device=b.device)
        cb = self.buf["cb"]
        encode(self.desc, 2, b, cb[0:1], cb[1:2], self.workspace, stream)
        self._sync_ck()
        self.ck.bias = b.data_ptr()

    def empty_output(self) -> torch.Tensor:
        return torch.empty(self.shape_o, dtype=self.tdtype, device=self.buf["cd1"].device)

    # the entry points on this layer's buffers
    def encode_weights(self, W, stream=None):
        encode(self.desc, 1, W, self.buf["cw1"], self.buf["cw2"], self.workspace, stream)

    def check_weights(self, W, stream=None) -> int:
        """Columns of W whose sum no longer equals the Cw1 encoded at set-up (Sec. 4.1.2); 0 when
        W is intact, otherwise W should be reloaded.  Synchronizes."""
        out = torch.zeros(1, dtype=torch.int32, device=self.buf["cw1"].device)
        check_weights(self.desc, W, self.buf["cw1"], out, self.workspace, stream)
        return int(out.item())

    def encode_input(self, D, stream=None):
        encode(self.desc, 0, D, self.buf["cd1"], self.buf["cd2"], self.workspace, stream)

    def conv(self, D, W, O, stream=None):
        if self.groups > 1:   # grouped layers run on the expansion of W in the workspace
            self.conv_ws(D, W, O, stream)
        elif self.bias is not None:
            conv_fwd_bias(self.desc, D, W, self.bias, O, None, stream)
        else:
            conv_fwd(self.desc, D, W, O, stream)

    def checksum_conv(self, which, D=None, W=None, stream=None):
        checksum_conv(self.desc, which, D, W, self.ck, stream)

    def verify(self, O, stream=None):
        verify(self.desc, O, self.ck, self.policy, self.report, self.cap, self.workspace, stream)

    def correct(self, D, W, O, stream=None):
        correct(self.desc, D, W, O, self.ck, self.policy, self.report, self.workspace, stream)

    def verify_correct(self, D, W, O, stream=None):
        verify_correct(self.desc, D, W, O, self.ck, self.policy, self.report, self.cap, self.workspace, stream)

    def conv_ws(self, D, W, O, stream=None):
        """ftcnn_conv_fwd_ws (ftcnn_conv_fwd_bias with a bias): the convolution through the
        protected path's kernels."""
        if self.bias is not None:
            conv_fwd_bias(self.desc, D, W, self.bias, O, self.workspace, stream)
        else:
            conv_fwd_ws(self.desc, D, W, O, self.workspace, stream)

    def conv_sums(self, D, W, O, faults=(), stream=None, encode=False, given=False):
        """ftcnn_conv_fwd_sums; encode=True also encodes Cd1, Cd2 of D in the same pass and, on
        channels-last layers, computes the Co5..Co7 partials from them and Cw1, Cw2.  given=True:
        ftcnn_conv_fwd_sums_given, with this layer's Cd1, Cd2 already encoded (by
        relu_pool(..., cd=...) of the layer before)."""
        ck = None
        if encode or given or self.bias is not None:
            ck = _lib.Checksums()
            if encode or given:
                ck.cd1, ck.cd2 = self.buf["cd1"].data_ptr(), self.buf["cd2"].data_ptr()
                ck.cw1, ck.cw2 = self.buf["cw1"].data_ptr(), self.buf["cw2"].data_ptr()
            ck.bias, ck.cb = self.ck.bias, self.ck.cb   # the layer's bias goes into O
        conv_fwd_sums(self.desc, D, W, O, ck, self.report, self.cap, self.workspace, faults, stream, given)

    def verify_correct_sums(self, D, W, O, stream=None, coc=False):
        """ftcnn_verify_correct_sums; coc=True also computes Co5..Co7 in the same launch."""
        verify_correct_sums(self.desc, D, W, O, self.ck, self.policy, self.report, self.workspace,
                            (CO5 | CO6 | CO7) if coc else 0, stream)

    def protected(self, D, W, O, stream=None):
        protected_conv(self.desc, D, W, O, self.ck, self.policy, self.report, self.cap, self.workspace,
                       stream)

    def inject(self, O, faults, stream=None):
        inject(self.desc, O, faults, stream)

    def read_report(self) -> Report:
        torch.cuda.synchronize()
        return parse_report(self.report)

    def protected_fused(self, D, W, O, faults=(), stream=None):
        """The protected layer in two launches (what ftcnn_protected_conv does):
        conv_fwd_sums with the encode of D -> verify_correct_sums with Co5..Co7.
        ``faults`` (testing) are planted in the convolution's outputs before they are summed."""
        self.conv_sums(D, W, O, faults, stream, encode=True)
        self.verify_correct_sums(D, W, O, stream, coc=True)

    def run(self, D, W, O, faults=(), stream=None) -> Report:
        """The full workflow of Sec. 4.3 with recomputation of the layer when needed (Sec. 4.1.1)."""
        self.encode_input(D, stream)
        self.conv(D, W, O, stream)
        self.checksum_conv(CO5 | CO6 | CO7, stream=stream)
        if faults:
            self.inject(O, faults, stream)
        self.verify(O, stream)
        self.correct(D, W, O, stream)
        rep = self.read_report()
        if rep.status == STATUS_NEEDS_RECOMPUTE:
            first = rep
            self.conv(D, W, O, stream)
            self.verify(O, stream)
            again = self.read_report()
            first.status = STATUS_FAILED if again.detected else STATUS_RECOMPUTED
            rep = first
        return rep
