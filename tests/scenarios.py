"""Fault scenarios of the paper's protection-ability analysis (Sec. 4.1, Figs. 2-5).

Each scenario is a small layer, its inputs, the corruption to apply and the
outcome Sec. 4.1 predicts.  The oracle tests check the predictions; the GPU
tests replay the same corruptions through the C ABI and compare with the
oracle.  Integer-valued inputs keep every fp32/bf16 result exact, so repaired
outputs must equal the clean ones bit for bit.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

import workloads as wl
from oracle import workflow as wf

S = wf  # scheme constants live in the oracle's workflow module


@dataclasses.dataclass
class Scenario:
    name: str
    spec: wl.LayerSpec
    data: str                       # "int" or "float"
    faults: List[wf.Fault]
    hook: Optional[Dict] = None     # {"target": "D"|"W"|"cd1"|"cw1", "index": (..), "add": v}
    policy: Dict = dataclasses.field(default_factory=dict)
    expect_schemes: Tuple[int, ...] = ()   # every flagged position resolved by one of these
    expect_status: int = wf.STATUS_CORRECTED
    expect_clean: bool = True       # final output equals the fault-free output

    def inputs(self):
        if self.data == "int":
            D = wl.gen_int_d(self.spec, seed=len(self.name))
            W = wl.gen_int_w(self.spec, seed=len(self.name))
        else:
            cfg = wl.Config(90, "scenario", (self.spec,), "uniform", "he")
            D = wl.gen_d(cfg, 0)
            W = wl.gen_w(cfg, 0)
        return D, W

    def oracle_hook(self):
        if self.hook is None:
            return None
        h = self.hook

        def fn(D, W, ck):
            arr = {"D": D, "W": W, "cd1": ck.cd1, "cw1": ck.cw1}[h["target"]]
            arr[h["index"]] += h["add"]
        return fn

    def oracle_policy(self) -> wf.Policy:
        return wf.Policy(**self.policy)

    def run_oracle(self):
        D, W = self.inputs()
        return wf.protect(D, W, self.spec.stride, self.spec.pad, self.spec.dtype,
                          self.oracle_policy(), self.faults, after_encode=self.oracle_hook())


def _layer(dtype="f32", n=6, m=8, ch=4, hw=9, r=3, u=1, p=1):
    return wl.LayerSpec("scn", n, ch, hw, hw, m, r, r, u, p, dtype)


def add(n, m, x, y, v):
    return wf.Fault(n, m, x, y, "add", value=float(v))


def all_scenarios() -> List[Scenario]:
    L = _layer()
    out = [
        Scenario("single_block", L, "int", [add(3, 5, 4, 2, 40)], expect_schemes=(S.SCHEME_COC,)),
        Scenario("single_block_corner", L, "int", [add(5, 7, 8, 8, -37)], expect_schemes=(S.SCHEME_COC,)),
        Scenario("row0_single", L, "int", [add(0, 6, 1, 7, 23)], expect_schemes=(S.SCHEME_COC,)),
        Scenario("two_positions", L, "int", [add(0, 0, 0, 0, 19), add(5, 3, 6, 1, -29)],
                 expect_schemes=(S.SCHEME_COC,)),
        Scenario("same_block_many_positions", L, "int",
                 [add(2, 2, x, y, 11 + x + 3 * y) for x, y in [(0, 1), (4, 4), (8, 3)]],
                 expect_schemes=(S.SCHEME_COC,)),
        Scenario("row_same_p", L, "int", [add(2, 1, 3, 3, 40), add(2, 4, 3, 3, 17), add(2, 6, 3, 3, 29)],
                 expect_schemes=(S.SCHEME_RC,)),
        Scenario("row_same_p_rc_off", L, "int",
                 [add(2, 1, 3, 3, 40), add(2, 4, 3, 3, 17), add(2, 6, 3, 3, 29)],
                 policy={"rc_on": False}, expect_schemes=(S.SCHEME_FC,)),
        Scenario("col_same_p", L, "int", [add(1, 5, 6, 2, 40), add(3, 5, 6, 2, 17), add(5, 5, 6, 2, 29)],
                 expect_schemes=(S.SCHEME_CLC,)),
        Scenario("col_same_p_clc_off", L, "int",
                 [add(1, 5, 6, 2, 40), add(3, 5, 6, 2, 17), add(5, 5, 6, 2, 29)],
                 policy={"clc_on": False}, expect_schemes=(S.SCHEME_FC,)),
        Scenario("col_same_p_all_off", L, "int",
                 [add(1, 5, 6, 2, 40), add(3, 5, 6, 2, 17), add(5, 5, 6, 2, 29)],
                 policy={"rc_on": False, "clc_on": False}, expect_schemes=(S.SCHEME_FC,)),
        Scenario("square_needs_recompute", L, "int",
                 [add(1, 2, 5, 5, 40), add(1, 6, 5, 5, 17), add(4, 2, 5, 5, 29), add(4, 6, 5, 5, 11)],
                 expect_schemes=(S.SCHEME_UNRESOLVED,), expect_status=wf.STATUS_RECOMPUTED),
        Scenario("nan_element", L, "int", [wf.Fault(4, 1, 2, 6, "set", value=float("nan"))],
                 expect_schemes=(S.SCHEME_FC,)),
        Scenario("inf_element", L, "int", [wf.Fault(1, 7, 7, 0, "set", value=float("inf"))],
                 expect_schemes=(S.SCHEME_FC,)),
        Scenario("single_block_recompute_repair", L, "int", [add(3, 5, 4, 2, 40)],
                 policy={"repair": "recompute"}, expect_schemes=(S.SCHEME_COC,)),
        Scenario("row_same_p_wbase1", L, "int",
                 [add(0, 1, 3, 3, 40), add(0, 4, 3, 3, 17), add(0, 6, 3, 3, 29)],
                 policy={"wbase": 1}, expect_schemes=(S.SCHEME_RC,)),
        Scenario("single_block_bf16", _layer("bf16"), "int", [add(3, 5, 4, 2, 40)],
                 expect_schemes=(S.SCHEME_COC,)),
        Scenario("row_same_p_bf16", _layer("bf16"), "int",
                 [add(2, 1, 3, 3, 40), add(2, 4, 3, 3, 17), add(2, 6, 3, 3, 29)],
                 expect_schemes=(S.SCHEME_RC,)),
        # memory faults after encoding (Sec. 4.1.2-4.1.5)
        Scenario("d_fault_row", L, "float", [], hook={"target": "D", "index": (2, 1, 4, 4), "add": 3.0},
                 expect_schemes=(S.SCHEME_RC,)),
        Scenario("d_fault_row_rc_off", L, "float", [], hook={"target": "D", "index": (2, 1, 4, 4), "add": 3.0},
                 policy={"rc_on": False}, expect_schemes=(S.SCHEME_FC,)),
        Scenario("w_fault_col", L, "float", [], hook={"target": "W", "index": (3, 2, 1, 1), "add": 3.0},
                 expect_schemes=(S.SCHEME_CLC,)),
        Scenario("w_fault_col_clc_off", L, "float", [], hook={"target": "W", "index": (3, 2, 1, 1), "add": 3.0},
                 policy={"clc_on": False}, expect_schemes=(S.SCHEME_FC,)),
        Scenario("cd1_fault", L, "float", [], hook={"target": "cd1", "index": (1, 4, 4), "add": 3.0},
                 expect_schemes=(S.SCHEME_CKSUM,)),
        Scenario("cw1_fault", L, "float", [], hook={"target": "cw1", "index": (2, 0, 2), "add": 3.0},
                 expect_schemes=(S.SCHEME_CKSUM,)),
        Scenario("strided_single", _layer(n=5, m=7, ch=3, hw=15, r=5, u=2, p=2), "int",
                 [add(4, 6, 7, 0, 31)], expect_schemes=(S.SCHEME_COC,)),
        Scenario("n1_single", _layer(n=1, m=5), "int", [add(0, 3, 2, 2, 21)], expect_schemes=(S.SCHEME_COC,)),
        Scenario("m1_single", _layer(n=4, m=1), "int", [add(2, 0, 5, 5, 21)], expect_schemes=(S.SCHEME_COC,)),
        Scenario("clean", L, "float", [], expect_schemes=(), expect_status=wf.STATUS_CLEAN),
    ]
    return out


def by_name(name: str) -> Scenario:
    for s in all_scenarios():
        if s.name == name:
            return s
    raise KeyError(name)
