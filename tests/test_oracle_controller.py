"""Pins for the oracle's Alg. 1 controller (CPU only)."""

import json
import math
import os

import numpy as np
import pytest

from oracle import COMPUTE, REACTIVATE, REUSE, local_impact, run_controller

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")
NAMES = {"REUSE": REUSE, "REACTIVATE": REACTIVATE, "COMPUTE": COMPUTE}


def _scaled_inputs(case, heads=2, d=4):
    """Zero keys (uniform attention) and target Q = c[t][b] * Q0."""
    q0 = np.random.default_rng(0).standard_normal((1, heads, case["n_tgt"], d)) + 0.1
    nr, nt = case["n_ref"], case["n_tgt"]
    vr = np.random.default_rng(1).standard_normal((1, heads, nr, d))
    vt = np.random.default_rng(2).standard_normal((1, heads, nt, d))

    def inputs(t, b):
        return {
            "q_ref": np.ones((1, heads, nr, d)),
            "k_ref": np.zeros((1, heads, nr, d)),
            "v_ref": vr,
            "q_tgt": case["c"][t][b] * q0,
            "k_tgt": np.zeros((1, heads, nt, d)),
            "v_tgt": vt,
        }

    return inputs


def test_hand_scenario():
    case = json.load(open(GOLDEN))["controller"][0]
    T, nb = len(case["c"]), len(case["c"][0])
    tr = run_controller(_scaled_inputs(case), T, nb, case["theta"], eps=0.0)
    assert tr.decisions.tolist() == [[NAMES[x] for x in row] for row in case["decisions"]]
    assert tr.ages.tolist() == case["ages"]
    # The lagged mass is exactly n_ref / (n_ref + n_tgt) wherever the gate was read.
    m = tr.m_mean[~np.isnan(tr.m_mean)]
    np.testing.assert_allclose(m, 0.25, rtol=0, atol=1e-15)
    tr2 = run_controller(_scaled_inputs(case), T, nb, case["theta"], delta_max=2, eps=0.0)
    assert tr2.decisions.tolist() == [[NAMES[x] for x in row] for row in case["decisions_delta_max_2"]]
    assert tr2.ages.tolist() == case["ages_delta_max_2"]


def test_anchor_cue_closed_form():
    """Target Q_t = (1 + 0.1 t) Q0 under exactly uniform attention (mass 2/8 = 1/4).
    Consecutive change shrinks (0.1 / (1 + 0.1 (t-1))), so with theta = 0.04 every
    block reuses after step 0. Anchor change grows with the distance to the last
    COMPUTE step a (0.1 (t - a) / (1 + 0.1 a)): block 0 reaches 0.2 * 1/4 = 0.05 at
    step 2 and reactivates, block 1 then computes and moves its anchor to the step."""
    case = {"n_ref": 2, "n_tgt": 6, "c": [[1.0 + 0.1 * t] * 2 for t in range(4)]}
    C, R, U = COMPUTE, REACTIVATE, REUSE
    cons = run_controller(_scaled_inputs(case), 4, 2, 0.04, eps=0.0)
    assert cons.decisions.tolist() == [[C, C], [U, U], [U, U], [U, U]]
    np.testing.assert_allclose(cons.d_mean[1:, 0], [0.1, 0.1 / 1.1, 0.1 / 1.2], rtol=1e-12)
    anc = run_controller(_scaled_inputs(case), 4, 2, 0.04, eps=0.0, cue="anchor")
    assert anc.decisions.tolist() == [[C, C], [U, U], [R, C], [R, C]]
    assert anc.ages.tolist() == [[0, 0], [0, 0], [0, 2], [0, 3]]
    np.testing.assert_allclose(anc.d_mean[1:, 0], [0.1, 0.2, 0.3], rtol=1e-12)
    np.testing.assert_allclose(anc.g_mean[1:, 0], [0.025, 0.05, 0.075], rtol=1e-12)
    assert np.isnan(anc.d_mean[2, 1]) and np.isnan(anc.d_mean[3, 1])  # not read past the boundary


def _random_inputs(seed, n_ref=6, n_tgt=5, heads=3, d=4, drift=0.2):
    base = {r: np.random.default_rng([seed, i]).standard_normal((1, heads, n_ref if r.endswith("ref") else n_tgt, d)) for i, r in enumerate(("q_ref", "k_ref", "v_ref", "q_tgt", "k_tgt", "v_tgt"))}
    cache = {}

    def inputs(t, b):
        key = (t, b)
        if key not in cache:
            rng = np.random.default_rng([seed, t, b, 99])
            cache[key] = {r: v + drift * t * rng.standard_normal(v.shape) for r, v in base.items()}
        return cache[key]

    return inputs


def test_theta_zero_reactivates_at_block_zero_every_step():
    tr = run_controller(_random_inputs(1), 4, 5, 0.0)
    assert (tr.decisions[0] == COMPUTE).all()
    for t in range(1, 4):
        assert tr.decisions[t, 0] == REACTIVATE and (tr.decisions[t, 1:] == COMPUTE).all()


def test_theta_infinite_reuses_every_block_after_step_zero():
    tr = run_controller(_random_inputs(2), 4, 5, math.inf)
    assert (tr.decisions[1:] == REUSE).all()
    assert (tr.ages == 0).all()
    assert (tr.impact[1:] > 0).all()  # the cache is stale, so the output moves


def test_delta_max_one_is_always_full():
    tr = run_controller(_random_inputs(3), 4, 3, math.inf, delta_max=1)
    assert (tr.decisions == COMPUTE).all()
    assert (tr.impact == 0).all()
    assert tr.ages[-1].tolist() == [3, 3, 3]


@pytest.mark.parametrize("theta", [0.02, 0.05, 0.1, 0.2])
def test_one_monotone_switch_per_step(theta):
    """Each non-refresh step is REUSE* then at most one REACTIVATE followed by COMPUTE*."""
    tr = run_controller(_random_inputs(4, drift=0.3), 5, 8, theta)
    for t in range(1, 5):
        row = tr.decisions[t].tolist()
        k = next((i for i, x in enumerate(row) if x != REUSE), len(row))
        assert all(x == REUSE for x in row[:k])
        if k < len(row):
            assert row[k] == REACTIVATE and all(x == COMPUTE for x in row[k + 1 :])
            assert tr.g_mean[t, k] >= theta
        assert all(tr.g_mean[t, i] < theta for i in range(k))


def test_compute_blocks_match_full_fresh_and_refresh_cache_age():
    tr = run_controller(_random_inputs(5, drift=0.3), 3, 6, 0.0)
    assert (tr.impact[tr.decisions == COMPUTE] == 0).all()
    assert tr.ages[2].tolist() == [0, 2, 2, 2, 2, 2]


def test_boundary_reference_rows_attend_with_the_cached_state_queries():
    """Alg. 1 boundary branch: the restored reference state runs the reference-query
    computation. Scale 1, d = 2, one head, 2 reference + 2 target rows, theta = 0, so step 1
    reactivates block 0 and computes block 1. Reference keys (ln 5, 0) and (0, 0), target keys
    zero; reference queries are 0 at step 0 and (1, 0) at step 1. The boundary's reference rows
    therefore see all-zero logits (uniform attention): o = mean of [V_R(step 0); V_Y(step 1)] =
    ((4,0) + (0,4) + (0,0) + (8,8)) / 4 = (3, 3). The computing block uses the current queries:
    weights (5, 1, 1, 1) / 8, o = (5 (4,0) + (0,4) + (0,0) + (8,8)) / 8 = (3.5, 1.5)."""
    ln5 = math.log(5.0)

    def inputs(t, b):
        return {
            "q_ref": np.full((1, 1, 2, 2), 0.0) if t == 0 else np.tile([1.0, 0.0], (1, 1, 2, 1)),
            "k_ref": np.array([[[[ln5, 0.0], [0.0, 0.0]]]]),
            "v_ref": np.array([[[[4.0, 0.0], [0.0, 4.0]]]]) if t == 0 else np.array([[[[40.0, 0.0], [0.0, 40.0]]]]),
            "q_tgt": np.array([[[[1.0, 2.0], [3.0, -1.0]]]]) * (1.0 + t),
            "k_tgt": np.zeros((1, 1, 2, 2)),
            "v_tgt": np.array([[[[1.0, 1.0], [1.0, 1.0]]]]) if t == 0 else np.array([[[[0.0, 0.0], [8.0, 8.0]]]]),
        }

    tr = run_controller(inputs, 2, 2, 0.0, scale=1.0, keep_outputs=True)
    assert tr.decisions.tolist() == [[COMPUTE, COMPUTE], [REACTIVATE, COMPUTE]]
    boundary = tr.outputs[(1, 0)]["o_all"][0, 0, :2]
    np.testing.assert_allclose(boundary, [[3.0, 3.0], [3.0, 3.0]], rtol=0, atol=1e-14)
    # the computing block reads this step's reference Q and V: V_R = 10 x the step-0 rows
    computed = tr.outputs[(1, 1)]["o_all"][0, 0, :2]
    np.testing.assert_allclose(computed, [[(5 * 40 + 8) / 8, (40 + 8) / 8]] * 2, rtol=0, atol=1e-13)


def test_local_impact_closed_form():
    a = np.zeros((1, 1, 2, 2))
    b = np.zeros((1, 1, 2, 2))
    b[0, 0, 0] = (3, 4)
    a[0, 0, 0] = (3, 4)
    a[0, 0, 1] = (0, 5)
    np.testing.assert_allclose(local_impact(a, b, 0.0), [[1.0]], rtol=0, atol=0)
    np.testing.assert_allclose(local_impact(b, b), [[0.0]], rtol=0, atol=0)
