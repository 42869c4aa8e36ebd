"""Pins for the oracle's Q-change and gate (CPU only)."""

import json
import math
import os

import numpy as np
import pytest

from oracle import COMPUTE, REACTIVATE, REUSE, gate, head_exposure, q_change
from oracle.stats import full_refresh_due

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")
NAMES = {"REUSE": REUSE, "REACTIVATE": REACTIVATE, "COMPUTE": COMPUTE}


def _golden(kind):
    with open(GOLDEN) as f:
        return json.load(f)[kind]


def test_q_change_hand_example():
    case = _golden("q_change")[0]
    eps = case["eps"]
    exp = np.array([[eval(v, {"eps": eps}) if isinstance(v, str) else v for v in row] for row in case["d"]])
    got = q_change(np.array(case["q_cur"], float), np.array(case["q_prev"], float), eps)
    np.testing.assert_allclose(got, exp, rtol=1e-15, atol=0)


@pytest.mark.parametrize("alpha", [0.0, 0.3, -0.3, -2.0, 1e-6])
def test_q_change_scaling_closed_form(alpha):
    """Q_t = (1 + alpha) Q_{t-1} gives |alpha| n / (n + eps) with n = ||Q_{t-1}||_F."""
    q = np.random.default_rng(1).standard_normal((2, 3, 17, 8))
    n = np.sqrt((q**2).sum(axis=(-2, -1)))
    eps = 1e-3
    np.testing.assert_allclose(q_change((1 + alpha) * q, q, eps), abs(alpha) * n / (n + eps), rtol=1e-12, atol=1e-15)


def test_q_change_zero_previous_is_norm_over_eps():
    cur = np.zeros((1, 1, 2, 2))
    cur[0, 0, 1] = (3.0, 4.0)
    np.testing.assert_allclose(q_change(cur, np.zeros_like(cur), 1e-8), 5.0 / 1e-8, rtol=1e-15)


def test_q_change_is_per_head():
    """Changing one head's rows changes only that head's statistic."""
    rng = np.random.default_rng(2)
    prev = rng.standard_normal((2, 4, 9, 8))
    cur = prev.copy()
    cur[1, 2] += 0.5
    got = q_change(cur, prev)
    assert got[1, 2] > 0
    mask = np.ones_like(got, bool)
    mask[1, 2] = False
    assert np.all(got[mask] == 0)


@pytest.mark.parametrize("sigma,t", [(0.3, 1), (0.3, 4), (0.01, 2), (0.2, 3)])
def test_q_change_random_walk_expectation(sigma, t):
    """X_{t-1} has per-element variance 1 + (t-1) sigma^2 and the increment
    sigma * N(0,1): for many elements D concentrates at sigma / sqrt(1 + (t-1) sigma^2)."""
    rng = np.random.default_rng(3)
    prev = rng.standard_normal((1, 4, 2048, 64)) * math.sqrt(1 + (t - 1) * sigma**2)
    cur = prev + sigma * rng.standard_normal(prev.shape)
    np.testing.assert_allclose(q_change(cur, prev), sigma / math.sqrt(1 + (t - 1) * sigma**2), rtol=5e-3)


def test_head_exposure_is_mean_over_target_queries():
    m = np.array([[[0.0, 1.0, 0.5, 0.5], [0.2, 0.2, 0.2, 0.2]]])
    np.testing.assert_allclose(head_exposure(m), [[0.5, 0.2]], rtol=0, atol=1e-16)


def test_gate_hand_examples():
    case = _golden("gate")[0]
    for c in case["cases"]:
        r = gate(np.array(case["d"]), np.array(case["mass_prev"]), c["theta"], c["reactivated"], mode=c["mode"], theta_m=c.get("theta_m"))
        assert r.decision == NAMES[c["decision"]], c
        assert r.reactivated == (r.decision != REUSE)
        assert math.isclose(r.g_mean, case["g_mean"], rel_tol=1e-14)
        assert math.isclose(r.d_mean, case["d_mean"], rel_tol=1e-14)
        assert math.isclose(r.m_mean, case["m_mean"], rel_tol=1e-14)


def test_gate_small_if_either_factor_is_zero():
    """The product score is zero when either cue is zero (the paper's remark that
    the score is small if either factor is weak), so any positive theta reuses."""
    rng = np.random.default_rng(4)
    mass = rng.random((1, 6, 32))
    d = rng.random((1, 6))
    d0 = d.copy()
    d0[:] = 0
    assert gate(d0, mass, 1e-12, False).decision == REUSE
    assert gate(d, np.zeros_like(mass), 1e-12, False).decision == REUSE
    assert gate(d, mass, 0.0, False).decision == REACTIVATE
    assert gate(d, mass, math.inf, False).decision == REUSE
    assert gate(d, mass, math.inf, True).decision == COMPUTE


def test_gate_pairs_product_per_head_before_mean():
    """High D on one head and high M on another head must not multiply across heads."""
    d = np.array([[1.0, 0.0]])
    mass = np.array([[[0.0, 0.0], [1.0, 1.0]]])
    r = gate(d, mass, 1e-9, False)
    assert r.g_mean == 0.0 and r.decision == REUSE
    assert r.d_mean * r.m_mean == 0.25  # the product of means would have crossed


def test_full_refresh_rule():
    assert full_refresh_due(0, 0, None)
    assert not full_refresh_due(5, 0, None)
    assert full_refresh_due(3, 1, 2) and not full_refresh_due(2, 1, 2)
    assert full_refresh_due(1, 0, 1)
