"""Sec. 4.2 cost model and sparsity allocation: the oracle and libprox's host
calls against the paper's printed allocation table, closed forms, and each
other (no GPU)."""
import ctypes
import json
import os

import numpy as np
import pytest

from paper_2607_27591_amd import prox

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "cost_model_tables.json")))


@pytest.mark.parametrize("row", GOLDEN["allocation"], ids=lambda r: f"e{r['e']}")
def test_allocation_reproduces_printed_table(oracle_lib, row):
    s1, s2 = oracle_lib.allocate(row["e"])
    assert abs(s1 - row["s1"]) < 5e-4 and abs(s2 - row["s2"]) < 5e-4
    assert prox.allocate_sparsity(row["e"]) == pytest.approx((s1, s2), abs=1e-12)


def test_closed_forms(oracle_lib):
    a = 1.0 / 3.0
    assert oracle_lib.prox_cost(1.0, 1.0, a) == 0.0                  # nothing computed
    assert oracle_lib.prox_cost(1.0, 0.0, a) == 3.0                  # Stage 2 alone is dense
    assert oracle_lib.effective_sparsity(0.0, 0.0, a) == pytest.approx(-2 * a / 3)
    # the headline workload keeps 40% / 30%: e = 0.7 - (2/3)(0.4)/3
    assert oracle_lib.effective_sparsity(0.6, 0.7, a) == pytest.approx(0.7 - 0.8 / 9)
    assert prox.effective_sparsity(0.6, 0.7) == pytest.approx(0.7 - 0.8 / 9, abs=1e-15)


def test_allocation_round_trips_and_respects_bounds(oracle_lib):
    for e in np.linspace(-0.2, 0.95, 47):
        s1, s2 = oracle_lib.allocate(e)
        assert 0.0 <= s1 <= 0.7
        assert oracle_lib.effective_sparsity(s1, s2) == pytest.approx(e, abs=1e-12)
        if 0.0 < s1 < 0.7:
            assert s2 == 0.7                                         # the anchor holds
        assert prox.allocate_sparsity(e) == pytest.approx((s1, s2), abs=1e-12)


def test_alpha_table_summary_and_the_rounded_value():
    vals = np.array([v for g in GOLDEN["alpha_measured"].values() for row in g for v in row])
    s = GOLDEN["alpha_summary"]
    assert vals.size == 48
    assert vals.min() == s["min"] and vals.max() == s["max"]
    assert round(vals.mean(), 3) == s["mean"]
    assert s["min"] <= s["used"] <= s["max"]


def test_allocation_rejects_bad_arguments():
    L = prox.lib()
    a, b = ctypes.c_double(), ctypes.c_double()
    assert L.prox_allocate_sparsity(0.5, 0.0, 0.7, 0.0, 0.7, ctypes.byref(a), ctypes.byref(b)) == 1
    assert L.prox_allocate_sparsity(0.5, 1 / 3, 0.7, 0.8, 0.7, ctypes.byref(a), ctypes.byref(b)) == 1
    assert L.prox_allocate_sparsity(float("nan"), 1 / 3, 0.7, 0, 0.7, ctypes.byref(a),
                                    ctypes.byref(b)) == 1
    assert L.prox_allocate_sparsity(0.5, 1 / 3, 0.7, 0.0, 0.7, None, ctypes.byref(b)) == 1


@pytest.mark.parametrize("row", GOLDEN["cap_sensitivity"],
                         ids=lambda r: f"cap{r['s1_max']}_e{r['e']}")
def test_stage1_cap_rows_reproduce_printed_table(oracle_lib, row):
    """Every row of the cap-sensitivity table is an active cap: s1 sits at the
    cap and s2 is re-solved from the cost model to the printed value."""
    s1, s2 = oracle_lib.allocate(row["e"], s1_max=row["s1_max"])
    assert s1 == pytest.approx(row["s1_max"], abs=1e-15)
    assert abs(s2 - row["s2"]) < 5e-4
    assert oracle_lib.effective_sparsity(s1, s2) == pytest.approx(row["e"], abs=1e-12)
    assert prox.allocate_sparsity(row["e"], s1_max=row["s1_max"]) == pytest.approx(
        (s1, s2), abs=1e-12)


def test_stage1_cap_only_binds_at_high_sparsity(oracle_lib):
    """The table's text: at e = 40% and 50% every tested cap leaves the
    unconstrained allocation alone; at 60% only the 50% cap changes it."""
    unconstrained = {e: oracle_lib.allocate(e, s1_max=1.0) for e in (0.4, 0.5, 0.6)}
    for cap in GOLDEN["cap_tested"]:
        for e in (0.4, 0.5):
            assert oracle_lib.allocate(e, s1_max=cap) == unconstrained[e]
        changed = oracle_lib.allocate(0.6, s1_max=cap) != unconstrained[0.6]
        assert changed == (cap < 0.55)
        for e in (0.4, 0.5, 0.6):
            assert prox.allocate_sparsity(e, s1_max=cap) == pytest.approx(
                oracle_lib.allocate(e, s1_max=cap), abs=1e-12)
