"""The FT-CNN protection workflow in float64 (Sec. 3 and Sec. 4.3).

TEST INFRASTRUCTURE ONLY: this is the oracle that the HIP library is checked
against.  Only tests, the smoke check and the benchmark's CPU-baseline leg
use it.

Everything here is a plain transcription of the paper's definitions:

* input checksums Cd1 = sum_n D_n, Cd2 = sum_n n D_n, Cw1 = sum_m W_m,
  Cw2 = sum_m m W_m (Sec. 3.2);
* output checksums Co1..Co7 as convolutions of checksum blocks (Sec. 3.2);
* output summations So1..So7 (Sec. 3.3-3.6);
* detection with CoC-D (Sec. 3.6, Sec. 4.3), then the correction chain
  CoC -> RC -> ClC -> FC -> recompute (Sec. 4.3, Fig. 7), each scheme located
  and repaired as in Sec. 3.3-3.6 and the FC fallbacks of Sec. 4.1.5.

Readings where the paper is silent (all shared with the HIP library):

* comparison tolerance: a difference d = Co - So at one element is "bad" when
  it is non-finite or |d| > kappa * (2^-24 sqrt(K) + u_out) * Q, where Q is the
  root sum of squares of the weighted terms that make up So, K = Ch*R*S, and
  u_out is 0 for fp32 outputs and 2^-8 for bf16 outputs;
* a located index is legal when the ratio is finite, within eta of an integer
  and inside [0, N) or [0, M);
* every scheme works per output element position p = (x, y) (Level 2 of
  Sec. 3.2); a scheme that repairs must leave Co5, Co6 and Co7 consistent with
  the re-summed output at p, otherwise its repairs are undone and the next
  scheme runs;
* a repair writes the exclusive sum (the correcting checksum minus the other
  blocks of its sum), which equals "add the difference" in exact arithmetic;
* when one of Co5/Co6/Co7 agrees with the output while the detection flagged
  p, the checksums are suspect (Sec. 4.1.4): they are re-encoded from D and W
  at p, and if the output agrees with the fresh ones p is closed as a checksum
  fault with no repair; otherwise the chain continues with the fresh ones;
* positions left unresolved trigger a recomputation of the whole layer
  (Sec. 4.1.1);
* with G groups (Sec. 5.2) filter block m convolves only with channel group
  m // (M/G) of every feature-map block; Cd stays, Cw1/Cw2 are the per-group filter
  sums laid side by side over the channels (m counted over all filters in Cw2), and
  the tolerance's K is the per-output dot length (Ch/G)*R*S;
* with a bias (Sec. 5.1) the output is eq. (1) plus Bias[m], the checksums stay
  those of the convolution, and every summation has the bias share of Table 5
  subtracted before it is compared or used in a repair (with the paper's index
  sums read as sums of the block weights n + wbase and m + wbase).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import core

U_ACC = 2.0 ** -24
U_OUT = {"f32": 0.0, "bf16": 2.0 ** -8}

SCHEME_NONE, SCHEME_COC, SCHEME_RC, SCHEME_CLC, SCHEME_FC, SCHEME_CKSUM, SCHEME_UNRESOLVED = range(7)
SCHEME_NAMES = ["none", "coc", "rc", "clc", "fc", "cksum", "unresolved"]

STATUS_CLEAN, STATUS_CORRECTED, STATUS_NEEDS_RECOMPUTE, STATUS_RECOMPUTED, STATUS_FAILED = range(5)


@dataclasses.dataclass
class Policy:
    rc_on: bool = True
    clc_on: bool = True
    repair: str = "checksum"  # or "recompute": re-evaluate eq. (1) for a located element
    kappa: float = 16.0
    eta: float = 0.1
    wbase: int = 0  # index weight of block 0 in Cd2/Cw2 (0 in the paper's definitions)


@dataclasses.dataclass
class Report:
    detected: bool = False
    flagged: List[int] = dataclasses.field(default_factory=list)  # flat positions x*F+y
    scheme: Dict[int, int] = dataclasses.field(default_factory=dict)  # position -> scheme
    fixes: List[Tuple[int, int, int, int, int]] = dataclasses.field(default_factory=list)
    status: int = STATUS_CLEAN

    @property
    def n_flagged(self) -> int:
        return len(self.flagged)

    def resolved_by(self) -> List[int]:
        counts = [0] * 7
        for s in self.scheme.values():
            counts[s] += 1
        return counts


# ----------------------------------------------------------------------------
# storage rounding and faults
# ----------------------------------------------------------------------------

def store(v: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 values to the output dtype (nearest, ties to even), returned as float64."""
    v = np.asarray(v, dtype=np.float64)
    if dtype == "f32":
        return v.astype(np.float32).astype(np.float64)
    if dtype != "bf16":
        raise ValueError(dtype)
    with np.errstate(over="ignore", invalid="ignore"):
        mant, ex = np.frexp(v)  # v = mant * 2^ex, 0.5 <= |mant| < 1
        ulp = np.ldexp(1.0, ex - 8)  # bf16 keeps 8 significant bits
        ulp = np.where(ex - 8 < -133, 2.0 ** -133, ulp)  # bf16 subnormal spacing
        q = np.rint(v / ulp) * ulp
        q = np.where(np.abs(q) > 3.3895313892515355e38, np.copysign(np.inf, v), q)
        q = np.where(np.isfinite(v), q, v)
    return q


def bits_of(v: float, dtype: str) -> int:
    if dtype == "f32":
        return int(np.array([v], dtype=np.float32).view(np.uint32)[0])
    return int(np.array([v], dtype=np.float32).view(np.uint32)[0]) >> 16


def value_of(bits: int, dtype: str) -> float:
    if dtype == "f32":
        return float(np.array([bits], dtype=np.uint32).view(np.float32)[0])
    return float(np.array([bits << 16], dtype=np.uint32).view(np.float32)[0])


@dataclasses.dataclass(frozen=True)
class Fault:
    """One corrupted output element: a bit flip of its stored pattern, or an additive error."""
    n: int
    m: int
    x: int
    y: int
    kind: str  # "flip", "add" or "set"
    bit: int = 0
    value: float = 0.0


def apply_faults(O: np.ndarray, dtype: str, faults: Sequence[Fault]) -> None:
    """Corrupt the stored output in place (the paper injects at source level, Sec. 6.1)."""
    for f in faults:
        old = O[f.n, f.m, f.x, f.y]
        if f.kind == "flip":
            O[f.n, f.m, f.x, f.y] = value_of(bits_of(old, dtype) ^ (1 << f.bit), dtype)
        elif f.kind == "add":
            O[f.n, f.m, f.x, f.y] = store(np.array([old + f.value]), dtype)[0]
        elif f.kind == "set":
            O[f.n, f.m, f.x, f.y] = store(np.array([f.value]), dtype)[0]
        else:
            raise ValueError(f.kind)


# ----------------------------------------------------------------------------
# checksums
# ----------------------------------------------------------------------------

def encode(X: np.ndarray, wbase: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """Sec. 3.2: (sum_r X_r, sum_r (r + wbase) X_r) over the leading block index."""
    return core.block_sums(X, float(wbase))


def encode_weights(W: np.ndarray, groups: int = 1, wbase: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """Cw1, Cw2 of Sec. 3.2; with G groups (Sec. 5.2) the sums over the filters of each group,
    laid side by side over the channels ([Ch][R][S] for W [M][Ch/G][R][S]), the weight of
    filter m being m + wbase with m counted over all filters."""
    if groups == 1:
        return encode(W, wbase)
    Mg = W.shape[0] // groups
    parts = [encode(W[g * Mg:(g + 1) * Mg], wbase + g * Mg) for g in range(groups)]
    return np.concatenate([a for a, _ in parts], axis=0), np.concatenate([b for _, b in parts], axis=0)


def grouped_conv(D: np.ndarray, W: np.ndarray, groups: int, stride: int, pad: int) -> np.ndarray:
    """Eq. (1) with G groups (Sec. 5.2): filter block m convolves with channel group m // (M/G)
    of every feature-map block only."""
    if groups == 1:
        return core.conv(D, W, stride, pad)
    Cg, Mg = D.shape[1] // groups, W.shape[0] // groups
    return np.concatenate([core.conv(D[:, g * Cg:(g + 1) * Cg], W[g * Mg:(g + 1) * Mg], stride, pad)
                           for g in range(groups)], axis=1)


@dataclasses.dataclass
class Checksums:
    cd1: np.ndarray
    cd2: np.ndarray
    cw1: np.ndarray
    cw2: np.ndarray
    co5: Optional[np.ndarray] = None
    co6: Optional[np.ndarray] = None
    co7: Optional[np.ndarray] = None


def checksum_conv(a: np.ndarray, b: np.ndarray, stride: int, pad: int) -> np.ndarray:
    """The block operator (x) applied to checksum blocks (Sec. 3.2)."""
    if a.ndim == 3:
        a = a[None]
    if b.ndim == 3:
        b = b[None]
    return core.conv(a, b, stride, pad)


def coc_checksums(ck: Checksums, stride: int, pad: int) -> None:
    """Co5 = Cd1 (x) Cw1, Co6 = Cd1 (x) Cw2, Co7 = Cd2 (x) Cw1 (Sec. 3.2), each [E][F]."""
    ck.co5 = checksum_conv(ck.cd1, ck.cw1, stride, pad)[0, 0]
    ck.co6 = checksum_conv(ck.cd1, ck.cw2, stride, pad)[0, 0]
    ck.co7 = checksum_conv(ck.cd2, ck.cw1, stride, pad)[0, 0]


def row_checksums(ck: Checksums, W: np.ndarray, stride: int, pad: int, groups: int = 1):
    """Co1 = Cd1 (x) W and Co3 = Cd2 (x) W (Sec. 3.2), each [M][E][F]; with G groups each
    filter block meets its own channel group of Cd1, Cd2 (Sec. 5.2)."""
    if groups == 1:
        return (checksum_conv(ck.cd1, W, stride, pad)[0], checksum_conv(ck.cd2, W, stride, pad)[0])
    Cg, Mg = ck.cd1.shape[0] // groups, W.shape[0] // groups
    rows = [(checksum_conv(ck.cd1[g * Cg:(g + 1) * Cg], W[g * Mg:(g + 1) * Mg], stride, pad)[0],
             checksum_conv(ck.cd2[g * Cg:(g + 1) * Cg], W[g * Mg:(g + 1) * Mg], stride, pad)[0])
            for g in range(groups)]
    return np.concatenate([a for a, _ in rows], axis=0), np.concatenate([b for _, b in rows], axis=0)


def col_checksums(ck: Checksums, D: np.ndarray, stride: int, pad: int):
    """Co2 = D (x) Cw1 and Co4 = D (x) Cw2 (Sec. 3.2), each [N][E][F]."""
    return (checksum_conv(D, ck.cw1, stride, pad)[:, 0], checksum_conv(D, ck.cw2, stride, pad)[:, 0])


def check_weights(W: np.ndarray, cw1: np.ndarray, wbase: int = 0, groups: int = 1) -> int:
    """Sec. 4.1.2: the columns (c, r, s) of W whose sum over the filters no longer equals the Cw1
    encoded before the application (a soft error in the weights in memory; the remedy is to
    reload W).  The same encode reproduces an intact column bit for bit."""
    fresh, _ = encode_weights(W, groups, wbase)
    return int(np.count_nonzero(fresh != cw1))


@dataclasses.dataclass
class BiasTerms:
    """The bias shares of the output summations (Sec. 5.1, Table 5), precomputed from Bias[m]:
    with wn = sum_n (n + wbase), b1 = sum_m Bias[m] and b2 = sum_m (m + wbase) Bias[m],
    So1[m] carries N Bias[m], So3[m] wn Bias[m], So2[n] b1, So4[n] b2, So5 N b1, So6 N b2 and
    So7 wn b1."""
    bias: np.ndarray
    wn: float
    b1: float
    b2: float
    N: int

    @staticmethod
    def make(bias: Optional[np.ndarray], N: int, M: int, wbase: int) -> "BiasTerms":
        b = np.zeros(M) if bias is None else np.asarray(bias, dtype=np.float64).reshape(M)
        wn = float(np.sum(np.arange(N, dtype=np.float64) + wbase))
        wm = np.arange(M, dtype=np.float64) + wbase
        return BiasTerms(b, wn, float(b.sum()), float((wm * b).sum()), N)

    @property
    def s5(self) -> float:
        return self.N * self.b1

    @property
    def s6(self) -> float:
        return self.N * self.b2

    @property
    def s7(self) -> float:
        return self.wn * self.b1

    @property
    def s1(self) -> np.ndarray:
        return self.N * self.bias

    @property
    def s3(self) -> np.ndarray:
        return self.wn * self.bias


# ----------------------------------------------------------------------------
# detection
# ----------------------------------------------------------------------------

def tol_scale(K: int, dtype: str, kappa: float) -> float:
    return kappa * (U_ACC * np.sqrt(float(K)) + U_OUT[dtype])


def bad(d, Q, scale):
    """A checksum difference that is non-finite or beyond the tolerance."""
    with np.errstate(invalid="ignore"):
        return np.logical_or(~np.isfinite(d), np.abs(d) > scale * Q)


def verify(O: np.ndarray, co5: np.ndarray, K: int, dtype: str, policy: Policy,
           bt: Optional[BiasTerms] = None):
    """CoC-D (Sec. 3.6): So5 = sum_{n,m} O_nm, less its bias share (Sec. 5.1), compared with
    Co5 at every position.

    Returns (So5, So6, So7, Q5, flags[E][F]), the summations as taken from O.  So6 and So7
    are the weighted summations of Sec. 3.6; they are reported for parity checks only.
    """
    N, M = O.shape[:2]
    wn = (np.arange(N, dtype=np.float64) + policy.wbase)[:, None, None, None]
    wm = (np.arange(M, dtype=np.float64) + policy.wbase)[None, :, None, None]
    with np.errstate(invalid="ignore", over="ignore"):
        so5 = O.sum(axis=(0, 1))
        so6 = (O * wm).sum(axis=(0, 1))
        so7 = (O * wn).sum(axis=(0, 1))
        q5 = np.sqrt((O * O).sum(axis=(0, 1)))
        share = bt.s5 if bt is not None else 0.0
        flags = bad(co5 - (so5 - share), q5, tol_scale(K, dtype, policy.kappa))
    return so5, so6, so7, q5, flags


# ----------------------------------------------------------------------------
# correction (per position p)
# ----------------------------------------------------------------------------

class _Layer:
    def __init__(self, O, D, W, ck, stride, pad, dtype, policy, bt=None, groups=1):
        self.O, self.D, self.W, self.ck = O, D, W, ck
        self.G = groups
        self.stride, self.pad, self.dtype, self.pol = stride, pad, dtype, policy
        self.N, self.M, self.E, self.F = O.shape
        self.K = W.shape[1] * W.shape[2] * W.shape[3]
        self.scale = tol_scale(self.K, dtype, policy.kappa)
        self.wn = np.arange(self.N, dtype=np.float64) + policy.wbase
        self.wm = np.arange(self.M, dtype=np.float64) + policy.wbase
        self._rows = self._cols = self._fresh = None
        self.bt = bt if bt is not None else BiasTerms.make(None, self.N, self.M, policy.wbase)

    # lazily computed per-layer checksum arrays (the paper computes them on demand, Sec. 4.3)
    def rows(self):
        if self._rows is None:
            self._rows = row_checksums(self.ck, self.W, self.stride, self.pad, self.G)
        return self._rows

    def cols(self):
        if self._cols is None:
            self._cols = col_checksums(self.ck, self.D, self.stride, self.pad)
        return self._cols

    def fresh_coc(self):
        """Co5..Co7 from input checksums re-encoded out of the current D and W."""
        if self._fresh is None:
            cd1, cd2 = encode(self.D, self.pol.wbase)
            cw1, cw2 = encode_weights(self.W, self.G, self.pol.wbase)
            f = Checksums(cd1, cd2, cw1, cw2)
            coc_checksums(f, self.stride, self.pad)
            self._fresh = (f.co5, f.co6, f.co7)
        return self._fresh

    # per-position helpers
    def block_sums_at(self, x, y):
        """So5, So6, So7 and their Q at p, from the current output."""
        Op = self.O[:, :, x, y]
        with np.errstate(invalid="ignore", over="ignore"):
            t6 = Op * self.wm[None, :]
            t7 = Op * self.wn[:, None]
            return (Op.sum(), t6.sum(), t7.sum(),
                    np.sqrt((Op * Op).sum()), np.sqrt((t6 * t6).sum()), np.sqrt((t7 * t7).sum()))

    def adjusted(self, s5, s6, s7):
        """So5, So6, So7 less their bias shares (Sec. 5.1, Table 5)."""
        return s5 - self.bt.s5, s6 - self.bt.s6, s7 - self.bt.s7

    def consistent(self, x, y, co):
        s5, s6, s7, q5, q6, q7 = self.block_sums_at(x, y)
        a5, a6, a7 = self.adjusted(s5, s6, s7)
        return not (bad(co[0] - a5, q5, self.scale) or bad(co[1] - a6, q6, self.scale)
                    or bad(co[2] - a7, q7, self.scale))

    def legal(self, r, hi):
        if not np.isfinite(r):
            return None
        i = np.rint(r)
        if abs(r - i) > self.pol.eta or i < 0 or i >= hi:
            return None
        return int(i)

    def element(self, n, m, x, y):
        """Eq. (1) for one element (over the filter's channel group), plus its bias (the RECOMPUTE
        repair option)."""
        Cg, g = self.D.shape[1] // self.G, m // (self.M // self.G)
        return core.conv_points(self.D[:, g * Cg:(g + 1) * Cg], self.W, self.stride, self.pad,
                                np.array([[n, m, x, y]], dtype=np.int32))[0] + self.bt.bias[m]

    def excl_row(self, co1m, m, i, x, y):
        """Co1[m] minus the other blocks of column m (exclusive sum over n != i), the sum less
        the bias share of So1[m]."""
        col = self.O[:, m, x, y]
        with np.errstate(invalid="ignore", over="ignore"):
            return co1m - (np.delete(col, i).sum() - self.bt.s1[m])

    def excl_col(self, co2n, n, j, x, y):
        row = self.O[n, :, x, y]
        with np.errstate(invalid="ignore", over="ignore"):
            return co2n - (np.delete(row, j).sum() - self.bt.b1)

    def excl_all(self, co5, i, j, x, y):
        others = np.delete(self.O[:, :, x, y].reshape(-1), i * self.M + j)
        with np.errstate(invalid="ignore", over="ignore"):
            return co5 - (others.sum() - self.bt.s5)

    def apply(self, fixes, x, y):
        """Write repaired values (rounded to the dtype); return the previous values."""
        old = []
        for (n, m, v) in fixes:
            old.append((n, m, self.O[n, m, x, y]))
            self.O[n, m, x, y] = store(np.array([v]), self.dtype)[0]
        return old

    def restore(self, old, x, y):
        for (n, m, v) in reversed(old):
            self.O[n, m, x, y] = v

    def try_fixes(self, fixes, x, y, co):
        old = self.apply(fixes, x, y)
        if self.consistent(x, y, co):
            return True
        self.restore(old, x, y)
        return False

    def value(self, n, m, x, y, checksum_value):
        if self.pol.repair == "recompute":
            return self.element(n, m, x, y)
        return checksum_value

    # schemes ------------------------------------------------------------------
    def row_sets(self, x, y):
        co1, co3 = self.rows()
        col = self.O[:, :, x, y]
        with np.errstate(invalid="ignore", over="ignore"):
            s1 = col.sum(axis=0)
            t3 = col * self.wn[:, None]
            s3 = t3.sum(axis=0)
            q1 = np.sqrt((col * col).sum(axis=0))
            d1 = co1[:, x, y] - (s1 - self.bt.s1)
            d3 = co3[:, x, y] - (s3 - self.bt.s3)
        mset = [m for m in range(self.M) if bad(d1[m], q1[m], self.scale)]
        return co1[:, x, y], d1, d3, mset

    def col_sets(self, x, y):
        co2, co4 = self.cols()
        row = self.O[:, :, x, y]
        with np.errstate(invalid="ignore", over="ignore"):
            s2 = row.sum(axis=1)
            t4 = row * self.wm[None, :]
            s4 = t4.sum(axis=1)
            q2 = np.sqrt((row * row).sum(axis=1))
            d2 = co2[:, x, y] - (s2 - self.bt.b1)
            d4 = co4[:, x, y] - (s4 - self.bt.b2)
        nset = [n for n in range(self.N) if bad(d2[n], q2[n], self.scale)]
        return co2[:, x, y], d2, d4, nset

    def coc(self, x, y, co, d):
        """Sec. 3.6: i = (Co7-So7)/delta, j = (Co6-So6)/delta, repair block (i, j)."""
        d5, d6, d7 = d
        with np.errstate(invalid="ignore", divide="ignore"):
            ri = d7 / d5 - self.pol.wbase
            rj = d6 / d5 - self.pol.wbase
        i, j = self.legal(ri, self.N), self.legal(rj, self.M)
        if i is None or j is None:
            return None
        v = self.value(i, j, x, y, self.excl_all(co[0], i, j, x, y))
        fixes = [(i, j, v)]
        return fixes if self.try_fixes(fixes, x, y, co) else None

    def rc(self, x, y, co):
        """Sec. 3.4: for each mismatching column m, i = (Co3-So3)/(Co1-So1); add Co1-So1."""
        co1, d1, d3, mset = self.row_sets(x, y)
        if not mset:
            return None
        fixes = []
        for m in mset:
            with np.errstate(invalid="ignore", divide="ignore"):
                r = d3[m] / d1[m] - self.pol.wbase
            i = self.legal(r, self.N)
            if i is None:
                return None
            fixes.append((i, m, self.value(i, m, x, y, self.excl_row(co1[m], m, i, x, y))))
        return fixes if self.try_fixes(fixes, x, y, co) else None

    def clc(self, x, y, co):
        """Sec. 3.5: for each mismatching row n, j = (Co4-So4)/(Co2-So2); add Co2-So2."""
        co2, d2, d4, nset = self.col_sets(x, y)
        if not nset:
            return None
        fixes = []
        for n in nset:
            with np.errstate(invalid="ignore", divide="ignore"):
                c = d4[n] / d2[n] - self.pol.wbase
            j = self.legal(c, self.M)
            if j is None:
                return None
            fixes.append((n, j, self.value(n, j, x, y, self.excl_col(co2[n], n, j, x, y))))
        return fixes if self.try_fixes(fixes, x, y, co) else None

    def fc(self, x, y, co, d):
        """Sec. 3.3 with the fallbacks of Sec. 4.1.5 (Fig. 5)."""
        co1, _, _, mset = self.row_sets(x, y)
        co2, _, _, nset = self.col_sets(x, y)
        d5, d6, d7 = d
        fixes = None
        if len(nset) == 1 and mset:  # one row of blocks, located by So2 (Fig. 5a)
            i = nset[0]
            fixes = [(i, m, self.value(i, m, x, y, self.excl_row(co1[m], m, i, x, y))) for m in mset]
        elif len(mset) == 1 and nset:  # one column of blocks, located by So1 (Fig. 5b)
            j = mset[0]
            fixes = [(n, j, self.value(n, j, x, y, self.excl_col(co2[n], n, j, x, y))) for n in nset]
        elif not mset and nset:  # Co1 blind to the error: column from Co6/Co5 (Fig. 5d)
            with np.errstate(invalid="ignore", divide="ignore"):
                j = self.legal(d6 / d5 - self.pol.wbase, self.M)
            if j is not None:
                fixes = [(n, j, self.value(n, j, x, y, self.excl_col(co2[n], n, j, x, y))) for n in nset]
        elif not nset and mset:  # Co2 blind to the error: row from Co7/Co5 (Fig. 5c)
            with np.errstate(invalid="ignore", divide="ignore"):
                i = self.legal(d7 / d5 - self.pol.wbase, self.N)
            if i is not None:
                fixes = [(i, m, self.value(i, m, x, y, self.excl_row(co1[m], m, i, x, y))) for m in mset]
        if fixes is None:
            return None
        return fixes if self.try_fixes(fixes, x, y, co) else None

    def resolve(self, x, y):
        """Run the correction chain at one flagged position; returns (scheme, fixes)."""
        ck = self.ck
        co = (ck.co5[x, y], ck.co6[x, y], ck.co7[x, y])
        s5, s6, s7, q5, q6, q7 = self.block_sums_at(x, y)
        s5, s6, s7 = self.adjusted(s5, s6, s7)
        d = (co[0] - s5, co[1] - s6, co[2] - s7)
        agree = [not bad(d[0], q5, self.scale), not bad(d[1], q6, self.scale),
                 not bad(d[2], q7, self.scale)]
        if any(agree):
            # an inconsistent pattern among Co5/Co6/Co7: suspect the checksums (Sec. 4.1.4)
            f5, f6, f7 = self.fresh_coc()
            co = (f5[x, y], f6[x, y], f7[x, y])
            if self.consistent(x, y, co):
                return SCHEME_CKSUM, []
            d = (co[0] - s5, co[1] - s6, co[2] - s7)
        fixes = self.coc(x, y, co, d)
        if fixes is not None:
            return SCHEME_COC, fixes
        if self.pol.rc_on:
            fixes = self.rc(x, y, co)
            if fixes is not None:
                return SCHEME_RC, fixes
        if self.pol.clc_on:
            fixes = self.clc(x, y, co)
            if fixes is not None:
                return SCHEME_CLC, fixes
        fixes = self.fc(x, y, co, d)
        if fixes is not None:
            return SCHEME_FC, fixes
        return SCHEME_UNRESOLVED, []


def correct(O: np.ndarray, D: np.ndarray, W: np.ndarray, ck: Checksums, flags: np.ndarray,
            stride: int, pad: int, dtype: str, policy: Policy, bt: Optional[BiasTerms] = None,
            groups: int = 1) -> Report:
    """Correction module of the multischeme workflow (Sec. 4.3), O repaired in place."""
    rep = Report()
    E, F = O.shape[2:]
    flat = np.flatnonzero(np.asarray(flags).reshape(-1))
    rep.flagged = [int(p) for p in flat]
    rep.detected = bool(len(flat))
    if not rep.detected:
        rep.status = STATUS_CLEAN
        return rep
    L = _Layer(O, D, W, ck, stride, pad, dtype, policy, bt, groups)
    for p in rep.flagged:
        x, y = divmod(p, F)
        scheme, fixes = L.resolve(x, y)
        rep.scheme[p] = scheme
        for (n, m, _) in fixes:
            rep.fixes.append((n, m, x, y, scheme))
    rep.fixes.sort()
    unresolved = sum(1 for s in rep.scheme.values() if s == SCHEME_UNRESOLVED)
    rep.status = STATUS_NEEDS_RECOMPUTE if unresolved else STATUS_CORRECTED
    return rep


# ----------------------------------------------------------------------------
# end to end
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class LayerResult:
    O: np.ndarray           # final output (stored values as float64)
    O_faulty: np.ndarray    # output after fault injection, before correction
    O_clean: np.ndarray     # fault-free stored output
    ck: Checksums
    so: tuple               # (So5, So6, So7, Q5) from the detection pass
    flags: np.ndarray
    report: Report


def protect(D: np.ndarray, W: np.ndarray, stride: int, pad: int, dtype: str,
            policy: Optional[Policy] = None, faults: Sequence[Fault] = (),
            O_in: Optional[np.ndarray] = None, after_encode=None,
            bias: Optional[np.ndarray] = None, groups: int = 1) -> LayerResult:
    """One protected layer: encode, convolve, checksum convs, verify, correct, recompute.

    ``after_encode(D, W, ck)`` may corrupt copies of D, W or the input
    checksums in place once they are encoded (memory faults of Sec. 4.1.2-4.1.4);
    the convolution and everything after it then see the corrupted data.
    ``O_in`` replaces the oracle's own convolution (decision-oracle mode: the
    caller supplies an output, e.g. a faulted one, and the workflow decides on
    it).  ``O_clean`` is always the output of the uncorrupted inputs.  ``bias`` [M] is added
    to every output block O[n][m] (Sec. 5.1).  ``groups`` G > 1: W is [M][Ch/G][R][S] and filter
    block m convolves with channel group m // (M/G) only (Sec. 5.2).
    """
    policy = policy or Policy()
    D = np.array(D, dtype=np.float64)
    W = np.array(W, dtype=np.float64)
    K = W.shape[1] * W.shape[2] * W.shape[3]
    bt = BiasTerms.make(bias, D.shape[0], W.shape[0], policy.wbase)

    def conv_b(D_, W_):
        return store(grouped_conv(D_, W_, groups, stride, pad) + bt.bias[None, :, None, None], dtype)

    O_clean = conv_b(D, W)
    cw1, cw2 = encode_weights(W, groups, policy.wbase)  # before the application (Sec. 4.2)
    cd1, cd2 = encode(D, policy.wbase)  # before the convolution (Sec. 3.3)
    ck = Checksums(cd1, cd2, cw1, cw2)
    touched = False
    if after_encode is not None:
        after_encode(D, W, ck)
        touched = True
    coc_checksums(ck, stride, pad)
    if O_in is not None:
        O = np.array(O_in, dtype=np.float64)
    elif touched:
        O = conv_b(D, W)
    else:
        O = O_clean.copy()
    apply_faults(O, dtype, faults)
    O_faulty = O.copy()
    so5, so6, so7, q5, flags = verify(O, ck.co5, K, dtype, policy, bt)
    rep = correct(O, D, W, ck, flags, stride, pad, dtype, policy, bt, groups)
    if rep.status == STATUS_NEEDS_RECOMPUTE:
        O[...] = conv_b(D, W)
        *_, flags2 = verify(O, ck.co5, K, dtype, policy, bt)
        rep.status = STATUS_FAILED if flags2.any() else STATUS_RECOMPUTED
    return LayerResult(O, O_faulty, O_clean, ck, (so5, so6, so7, q5), flags, rep)
