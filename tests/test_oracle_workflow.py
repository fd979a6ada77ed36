"""Pins for the oracle's workflow: the protection abilities of Sec. 4.1 on crafted faults."""
import numpy as np
import pytest

from oracle import workflow as wf
from scenarios import all_scenarios

SCN = all_scenarios()


@pytest.mark.parametrize("scn", SCN, ids=[s.name for s in SCN])
def test_protection_ability(scn):
    res = scn.run_oracle()
    rep = res.report
    assert rep.status == scn.expect_status, (rep.status, rep.scheme)
    if scn.expect_schemes:
        assert rep.detected
        assert set(rep.scheme.values()) <= set(scn.expect_schemes), rep.scheme
    else:
        assert not rep.detected
    if scn.data == "int" and scn.expect_clean:
        # integer data: every value is exact, so recovery must be bit for bit
        np.testing.assert_array_equal(res.O, res.O_clean)
    elif scn.expect_clean:
        scale = np.sqrt(np.mean(res.O_clean ** 2))
        N, M = res.O.shape[:2]
        tol = 8 * np.sqrt(N * M) * 2.0 ** -24 * scale
        assert np.max(np.abs(res.O - res.O_clean)) <= tol


def test_flagged_positions_are_the_corrupted_ones():
    from scenarios import by_name
    res = by_name("two_positions").run_oracle()
    assert res.report.flagged == [0 * 9 + 0, 6 * 9 + 1]
    assert res.report.fixes == [(0, 0, 0, 0, wf.SCHEME_COC), (5, 3, 6, 1, wf.SCHEME_COC)]


def test_w_fault_touches_whole_column():
    from scenarios import by_name
    res = by_name("w_fault_col").run_oracle()
    rep = res.report
    # the centre tap of filter 3 reaches every output position
    assert rep.n_flagged == 81
    assert {f[1] for f in rep.fixes} == {3}
    assert len(rep.fixes) == 81 * 6


def test_checksum_fault_leaves_output_untouched():
    from scenarios import by_name
    res = by_name("cd1_fault").run_oracle()
    assert res.report.fixes == []
    np.testing.assert_array_equal(res.O, res.O_clean)


def _swap_co6_co7(ck, stride, pad):
    _orig_coc(ck, stride, pad)
    ck.co6, ck.co7 = ck.co7, ck.co6


def _co1_from_cd2(ck, W, stride, pad, groups=1):
    co1, co3 = _orig_rows(ck, W, stride, pad, groups)
    return co3, co3


def _excl_keeps_element(self, co1m, m, i, x, y):
    return co1m - self.O[:, m, x, y].sum()


_orig_coc = wf.coc_checksums
_orig_rows = wf.row_checksums


@pytest.mark.parametrize("mistake,scenario", [
    ("swap_co6_co7", "single_block"),
    ("co1_from_cd2", "row_same_p"),
    ("excl_keeps_element", "row_same_p"),
])
def test_planted_mistake_is_caught(monkeypatch, mistake, scenario):
    """Plausible slips in the workflow must break the protection-ability pins."""
    from scenarios import by_name
    if mistake == "swap_co6_co7":
        monkeypatch.setattr(wf, "coc_checksums", _swap_co6_co7)
    elif mistake == "co1_from_cd2":
        monkeypatch.setattr(wf, "row_checksums", _co1_from_cd2)
    else:
        monkeypatch.setattr(wf._Layer, "excl_row", _excl_keeps_element)
    scn = by_name(scenario)
    res = scn.run_oracle()
    ok = (res.report.status == scn.expect_status
          and set(res.report.scheme.values()) <= set(scn.expect_schemes)
          and np.array_equal(res.O, res.O_clean))
    assert not ok


def test_large_random_bitflips_detected_and_fixed():
    """Sign and exponent bit flips on elements at least as large as rms(O) are always caught."""
    import workloads as wl
    cfg = wl.config(0)
    D, W = wl.gen_d(cfg, 0), wl.gen_w(cfg, 0)
    base = wf.protect(D, W, 1, 1, "f32")
    O = base.O_clean
    rms = np.sqrt(np.mean(O ** 2))
    draws = wl.fault_draws(0, 0, 40)
    big = np.argwhere(np.abs(O) >= rms)
    for d in draws:
        n, m, x, y = big[int(d[0] * len(big))]
        bit = 23 + int(d[4] * 9)
        f = wf.Fault(int(n), int(m), int(x), int(y), "flip", bit)
        tmp = O.copy()
        wf.apply_faults(tmp, "f32", [f])
        if not np.isfinite(tmp[n, m, x, y]):
            continue
        res = wf.protect(D, W, 1, 1, "f32", faults=[f])
        assert res.report.detected
        assert res.report.status in (wf.STATUS_CORRECTED, wf.STATUS_RECOMPUTED)
        assert np.max(np.abs(res.O - O)) <= 64 * 2.0 ** -24 * max(rms, abs(O[n, m, x, y]))
