"""The per-layer workflow measurement and the layerwise RC/ClC switch of Sec. 4.3 (host logic).

* the fault patterns have the structure each workflow needs (one block; three filters of one
  image; three images of one filter; a 2 x 2 set), inside the output;
* each workflow's pattern, replayed through the oracle with the workflow's switches, is resolved
  by the scheme the workflow table names (the expectation the GPU measurement checks against);
* the switch follows the paper's inequality on hand-worked times, including the case the paper
  gives (a layer where CoC+RC is barely faster than CoC+FC and CoC+RC+FC much slower: RC off).
"""
import numpy as np
import pytest

import workloads as wl
from oracle import workflow as wf
from paper_2003_12203_amd import schemes


@pytest.mark.parametrize("kind", ["single", "row", "col", "square"])
def test_pattern_structure(kind):
    n, m, e, f = 6, 8, 9, 7
    faults = schemes.pattern(kind, n, m, e, f)
    blocks = [(q["n"], q["m"]) for q in faults]
    assert len(set(blocks)) == len(blocks)
    assert {(q["x"], q["y"]) for q in faults} == {(e // 2, f // 2)}
    for q in faults:
        assert 0 <= q["n"] < n and 0 <= q["m"] < m and q["kind"] == "add" and q["value"] >= 1e6
        assert q["value"] % 16384 == 0 and 64 <= q["value"] // 16384 <= 255   # exact in bf16
    if kind == "single":
        assert len(blocks) == 1
    elif kind == "row":
        assert len(blocks) == 3 and len({b[0] for b in blocks}) == 1 and len({b[1] for b in blocks}) == 3
    elif kind == "col":
        assert len(blocks) == 3 and len({b[1] for b in blocks}) == 1 and len({b[0] for b in blocks}) == 3
    else:
        assert len(blocks) == 4 and len({b[0] for b in blocks}) == 2 and len({b[1] for b in blocks}) == 2


def test_pattern_too_small():
    with pytest.raises(ValueError):
        schemes.pattern("row", 4, 2, 3, 3)
    with pytest.raises(ValueError):
        schemes.pattern("square", 1, 4, 3, 3)
    with pytest.raises(ValueError):
        schemes.pattern("col", 2, 4, 3, 3)


@pytest.mark.parametrize("name", list(schemes.WORKFLOWS))
def test_workflow_expectations_match_oracle(name):
    kind, rc_on, clc_on, expect = schemes.WORKFLOWS[name]
    spec = wl.LayerSpec("wf", 6, 4, 9, 9, 8, 3, 3, 1, 1, "f32")
    D, W = wl.gen_int_d(spec, 3), wl.gen_int_w(spec, 3)
    faults = [wf.Fault(q["n"], q["m"], q["x"], q["y"], "add", value=q["value"])
              for q in schemes.pattern(kind, spec.n, spec.m, 9, 9)]
    res = wf.protect(D, W, 1, 1, "f32", wf.Policy(rc_on=rc_on, clc_on=clc_on), faults)
    got = tuple(sorted({wf.SCHEME_NAMES[s] for s in res.report.scheme.values()}))
    assert got == expect
    clean = wf.protect(D, W, 1, 1, "f32").O
    if expect != ("unresolved",):
        assert res.report.status == wf.STATUS_CORRECTED
    np.testing.assert_array_equal(res.O, clean)


def _times(**kw):
    t = {"CoC+FC/row": 100.0, "CoC+RC": 40.0, "CoC+RC+FC": 110.0,
         "CoC+FC/col": 100.0, "CoC+ClC": 60.0, "CoC+ClC+FC": 120.0}
    t.update(kw)
    return t


def test_switch_follows_the_inequality():
    # |D| / |W| = 10: RC gains 10 * 60 = 600 against a loss of 10; ClC gains 40 against 10 * 20
    c = schemes.rc_clc_policy(_times(), 1000, 100)
    assert (c.rc_on, c.clc_on) == (True, False)
    assert (c.rc_gain, c.rc_loss, c.clc_gain, c.clc_loss) == (600.0, 10.0, 40.0, 200.0)
    # |D| / |W| = 1/100: the roles swap
    c = schemes.rc_clc_policy(_times(), 10, 1000)
    assert (c.rc_on, c.clc_on) == (False, True)


def test_switch_paper_example():
    # CoC+RC close to CoC+FC, CoC+RC+FC much slower: RC stays off even with row errors likelier
    c = schemes.rc_clc_policy(_times(**{"CoC+RC": 98.0, "CoC+RC+FC": 190.0}), 200, 100)
    assert not c.rc_on
    # CoC+RC much faster and CoC+RC+FC slightly slower than CoC+FC: RC on at equal odds
    c = schemes.rc_clc_policy(_times(**{"CoC+RC": 30.0, "CoC+RC+FC": 104.0}), 100, 100)
    assert c.rc_on


def test_switch_ties_stay_off():
    t = {k: 50.0 for k in schemes.WORKFLOWS}
    c = schemes.rc_clc_policy(t, 1, 1)
    assert not c.rc_on and not c.clc_on
