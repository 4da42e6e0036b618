"""The library's APP capacity split (hill_app_balance, host-only C) against
the oracle's bisection of Eq. 2 (Sec. 4.3), and its argument checks.  No GPU
is needed: the function runs on the host."""
import ctypes
import math
import os

import pytest
from hypothesis import given, settings, strategies as st

from oracle import oracle as O


@pytest.fixture(scope="module")
def H():
    import paper_2602_18750_amd as H
    if not os.path.exists(H.hill.LIB_PATH):
        from paper_2602_18750_amd import _build
        _build.build()
    H.load_library()
    return H


rate = st.floats(1e7, 1e12)


@settings(max_examples=300, deadline=None)
@given(rate, rate, rate, rate, st.floats(0, 1), st.floats(0, 1), st.floats(1.0, 1e12), st.floats(-1.0, 1e12))
def test_app_balance_matches_oracle(H, f_c, f_s, b_c, b_s, a_c, a_s, m, m0):
    got = H.app_balance(f_c=f_c, f_s=f_s, b_c=b_c, b_s=b_s, alpha_c=a_c, alpha_s=a_s, m=m, m0=m0)
    beta, mc, ms, tc, ts, capped = O.app_split(f_c, f_s, b_c, b_s, a_c, a_s, m, m0)
    assert bool(got["capped"]) == capped
    assert math.isclose(got["m_c"], mc, rel_tol=1e-9, abs_tol=1e-9 * m)
    assert math.isclose(got["m_s"], ms, rel_tol=1e-9, abs_tol=1e-9 * m)
    assert math.isclose(got["t_c"], tc, rel_tol=1e-9, abs_tol=1e-12)
    assert math.isclose(got["t_s"], ts, rel_tol=1e-9, abs_tol=1e-12)
    if ms > 1e-6 * m:
        assert math.isclose(got["beta"], beta, rel_tol=1e-6)


def test_app_balance_worked_case(H):
    # Eq. 4 by hand: 25 * 10 * (6 + 0.2 * 2) / (6 * 2 * (25 + 0.2 * 10)) = 1600 / 324
    got = H.app_balance(f_c=10e9, f_s=2e9, b_c=25e9, b_s=6e9, alpha=0.2)
    assert math.isclose(got["beta"], 1600 / 324, rel_tol=1e-12) and not got["capped"]


@pytest.mark.parametrize("field,value", [("f_c", 0.0), ("f_s", -1.0), ("b_c", float("inf")), ("b_s", float("nan")),
                                         ("alpha_c", -0.1), ("alpha_s", 1.5), ("m", 0.0), ("m0", float("nan"))])
def test_app_balance_rejects_bad_arguments(H, field, value):
    lib = H.load_library()
    p = H.AppParams(10e9, 2e9, 25e9, 6e9, 0.2, 0.2, 1.0, 0.0)
    setattr(p, field, value)
    out = H.AppPlan()
    assert lib.hill_app_balance(ctypes.byref(p), ctypes.byref(out)) == 1
    assert lib.hill_app_balance(None, ctypes.byref(out)) == 1
    assert lib.hill_app_balance(ctypes.byref(H.AppParams(1, 1, 1, 1, 0, 0, 1, 0)), None) == 1
