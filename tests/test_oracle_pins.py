"""The oracle against facts that do not come from the oracle (CPU only)."""
import numpy as np
import pytest

import oracle
import pins


@pytest.mark.parametrize("pin", pins.FRONTIER_PINS, ids=lambda p: p.__name__)
def test_frontier_pin(pin):
    pin(oracle.frontier)


@pytest.mark.parametrize("pin", pins.SUMMARY_PINS, ids=lambda p: p.__name__)
def test_summary_pin(pin):
    pin(oracle.frontier, oracle.window_summary)


@pytest.mark.parametrize("pin", pins.LEAD_PINS, ids=lambda p: p.__name__)
def test_lead_exposed_pin(pin):
    pin(oracle.frontier, oracle.window_lead_exposed)


def test_lead_exposed_top2_cases():
    pins.pin_lead_top2_cases(oracle.frontier, oracle.window_lead_exposed, oracle.window_summary)


def test_twin_lead_exposed():
    pins.pin_lead_twin(oracle.frontier, oracle.window_lead_exposed, oracle.pyref)


@pytest.mark.parametrize("pin", pins.EVIDENCE_PINS, ids=lambda p: p.__name__)
def test_evidence_pin(pin):
    pin(oracle.frontier_evidence)


@pytest.mark.parametrize("pin", pins.SWITCH_PINS, ids=lambda p: p.__name__)
def test_switch_pin(pin):
    pin(oracle.frontier_evidence, oracle.window_leader_switches)


def test_twin_switches():
    pins.pin_switch_twin(oracle.frontier_evidence, oracle.window_leader_switches, oracle.pyref)


def test_twin_evidence():
    pins.pin_ev_twin(oracle.frontier_evidence, oracle.pyref)


def test_twin_frontier():
    pins.pin_twin(oracle.frontier, oracle.pyref)


def test_twin_summary():
    pins.pin_summary_twin(oracle.frontier, oracle.window_summary, oracle.pyref)


def test_pyref_against_pins():
    """The pure-Python twin passes the same printed examples."""
    def f(d):
        inc, lead = oracle.pyref.frontier(np.asarray(d).tolist())
        return np.array(inc, dtype=np.int64), np.array(lead, dtype=np.int32)
    pins.pin_golden(f)
    pins.pin_stall(f)


def test_empty_and_degenerate():
    inc, lead = oracle.frontier(np.zeros((0, 3, 4), dtype=np.int64))
    assert inc.shape == (0, 3) and lead.shape == (0, 3)
    ex, cnt, top2 = oracle.window_summary(inc, lead, 4, 10)
    assert ex.shape == (0, 3) and cnt.shape == (0, 3, 4) and top2.shape == (0, 2, 2)
    le, top2 = oracle.window_lead_exposed(inc, lead, 4, 10)
    assert le.shape == (0, 3, 4) and top2.shape == (0, 2, 2)
    # all-zero durations: zero advances, every boundary a full tie -> rank 0
    inc, lead = oracle.frontier(np.zeros((2, 3, 5), dtype=np.int64))
    assert (inc == 0).all() and (lead == 0).all()


def test_largest_prefix_is_exact():
    """int64 arithmetic stays exact up to the documented prefix bound."""
    big = (1 << 47) - 1
    d = np.zeros((1, 3, 3), dtype=np.int64)
    d[0, 0, 1] = big - 5
    d[0, 2, 1] = 5
    d[0, 1, 2] = big
    inc, lead = oracle.frontier(d)
    assert inc[0].tolist() == [big - 5, 5, 0]
    assert lead[0].tolist() == [1, 2, 1]


@pytest.mark.parametrize("pin", pins.INGEST_PINS, ids=lambda p: p.__name__)
def test_ingest_pin(pin):
    pin(oracle.ingest)


@pytest.mark.parametrize("pin", pins.ROUTE_PINS, ids=lambda p: p.__name__)
def test_route_pin(pin):
    pin(oracle.route)


def test_twin_ingest_route():
    pins.pin_ingest_twin(oracle.ingest, oracle.pyref)
    pins.pin_route_twin(oracle.route, oracle.pyref)


@pytest.mark.parametrize("pin", pins.GAIN_PINS, ids=lambda p: p.__name__)
def test_gain_pin(pin):
    pin(oracle.exposure_gain)


def test_twin_gain():
    pins.pin_gain_twin(oracle.exposure_gain, oracle.pyref)


@pytest.mark.parametrize("pin", pins.LAG_PINS, ids=lambda p: p.__name__)
def test_lag_pin(pin):
    pin(oracle.frontier_lag)


def test_twin_lag():
    pins.pin_lag_twin(oracle.frontier_lag, oracle.pyref)


@pytest.mark.parametrize("pin", pins.SPREAD_PINS, ids=lambda p: p.__name__)
def test_spread_pin(pin):
    pin(oracle.rank_spread)


def test_spread_first_boundary_is_lag():
    pins.pin_spread_first_boundary_is_lag(oracle.rank_spread, oracle.frontier_lag)


def test_twin_spread():
    pins.pin_spread_twin(oracle.rank_spread, oracle.pyref)


@pytest.mark.parametrize("pin", pins.MEDIAN_PINS, ids=lambda p: p.__name__)
def test_median_pin(pin):
    pin(oracle.window_median)


def test_twin_median():
    pins.pin_median_twin(oracle.window_median, oracle.pyref)


@pytest.mark.parametrize("pin", pins.RANGE_PINS, ids=lambda p: p.__name__)
def test_range_pin(pin):
    pin(oracle.range_status)


def test_twin_range():
    pins.pin_range_twin(oracle.range_status, oracle.pyref)
