"""libprox's host-side calibration calls (App. A.7 bounded sample and
empirical quantile) against the oracle's, on the CPU: they touch no GPU."""
import ctypes

import numpy as np
import pytest

from paper_2607_27591_amd import calibrate as C
from paper_2607_27591_amd import prox
from paper_2607_27591_amd import workloads as W

OK, INVALID = 0, 1


@pytest.mark.parametrize("s", [0.0, 0.25, 0.5, 0.7, 0.9, 0.999])
def test_quantile_matches_oracle(oracle_lib, s):
    rng = np.random.default_rng(int(s * 1000) + 1)
    for n in (1, 2, 7, 1000, 4097):
        v = np.abs(rng.standard_normal(n)).astype(np.float32)
        v[: n // 3] = v[0]   # ties
        assert C.quantile_threshold(v, s) == oracle_lib.quantile_threshold(v.astype(np.float64), s)


def test_reservoir_matches_oracle(oracle_lib):
    for cap in (1, 64, 300, 5000):
        a, b = C.Reservoir(cap), oracle_lib.Reservoir(cap)
        da, db = W.reservoir_draws(cap), W.reservoir_draws(cap)
        for k in range(6):
            vals = np.abs(np.random.default_rng(k).standard_normal(257)).astype(np.float32)
            a.add(vals, da(vals.size))
            b.add(vals.astype(np.float64), db(vals.size))
        assert np.array_equal(a.sample().astype(np.float64), b.sample())


def test_host_calls_reject_bad_arguments():
    L = prox.lib()
    buf = np.zeros(4, np.float32)
    tau = ctypes.c_float()
    assert L.prox_quantile_threshold(buf.ctypes.data, 0, 0.5, ctypes.byref(tau)) == INVALID
    assert L.prox_quantile_threshold(buf.ctypes.data, 4, 1.0, ctypes.byref(tau)) == INVALID
    assert L.prox_quantile_threshold(buf.ctypes.data, 4, -0.1, ctypes.byref(tau)) == INVALID
    assert L.prox_quantile_threshold(buf.ctypes.data, 4, float("nan"), ctypes.byref(tau)) == INVALID
    nan = np.array([1.0, np.nan], np.float32)
    assert L.prox_quantile_threshold(nan.ctypes.data, 2, 0.5, ctypes.byref(tau)) == INVALID
    assert L.prox_quantile_threshold(None, 4, 0.5, ctypes.byref(tau)) == INVALID
    assert L.prox_quantile_threshold(buf.ctypes.data, 4, 0.5, None) == INVALID
    seen = ctypes.c_uint64(0)
    draws = np.zeros(4, np.uint64)
    assert L.prox_reservoir_add(buf.ctypes.data, 0, ctypes.byref(seen), buf.ctypes.data, 4,
                                draws.ctypes.data) == INVALID
    assert L.prox_reservoir_add(buf.ctypes.data, 4, None, buf.ctypes.data, 4,
                                draws.ctypes.data) == INVALID
    assert L.prox_reservoir_add(buf.ctypes.data, 4, ctypes.byref(seen), None, 4,
                                draws.ctypes.data) == INVALID
    assert L.prox_reservoir_add(buf.ctypes.data, 4, ctypes.byref(seen), None, 0, None) == OK
    assert seen.value == 0
