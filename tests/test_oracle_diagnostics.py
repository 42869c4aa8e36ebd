"""Pins for the oracle's diagnostic quantities (CPU only).

Each pin is fixed by the mathematics, not by re-typing the oracle's formula:
closed forms of scaled or rotated slices, a sigmoid closed form of the
reference mass for collinear keys, brute-force loops on tiny inputs and
hand-derived trajectories.
"""

import math

import numpy as np
import pytest

from oracle import diagnostics as dg


def _frob_loops(cur, base, eps):
    """Brute force over explicit element loops for one [n, d] slice."""
    num = den = 0.0
    for i in range(cur.shape[0]):
        for j in range(cur.shape[1]):
            num += (float(cur[i, j]) - float(base[i, j])) ** 2
            den += float(base[i, j]) ** 2
    return math.sqrt(num) / (math.sqrt(den) + eps)


def test_drifts_match_brute_force_per_head():
    rng = np.random.default_rng(3)
    cur, base = rng.standard_normal((2, 3, 5, 4)), rng.standard_normal((2, 3, 5, 4))
    eps = 1e-3
    for fn in (dg.consecutive_drift, dg.endpoint_drift):
        got = fn(cur, base, eps)
        for b in range(2):
            for h in range(3):
                assert got[b, h] == pytest.approx(_frob_loops(cur[b, h], base[b, h], eps), rel=1e-13)


@pytest.mark.parametrize("alpha", [0.0, 0.05, 0.7, -1.5])
def test_endpoint_drift_scaling_closed_form(alpha):
    """Z_t = (1 + alpha) Z_a gives exactly |alpha| at eps = 0 (denominator is the anchor norm)."""
    z = np.random.default_rng(5).standard_normal((1, 4, 9, 8))
    np.testing.assert_allclose(dg.endpoint_drift((1 + alpha) * z, z, 0.0), abs(alpha), rtol=1e-12, atol=1e-15)


def test_endpoint_drift_orthogonal_step():
    """Z_t = Z_a + c U with <U, Z_a>_F = 0 and ||U|| = ||Z_a|| gives c (Pythagoras plays no role)."""
    rng = np.random.default_rng(6)
    z = rng.standard_normal((6, 4))
    u = rng.standard_normal((6, 4))
    u -= (u * z).sum() / (z * z).sum() * z
    u *= np.linalg.norm(z) / np.linalg.norm(u)
    assert dg.endpoint_drift(z + 0.25 * u, z, 0.0) == pytest.approx(0.25, rel=1e-12)
    # Dividing by the current norm instead would give 0.25 / sqrt(1 + 0.25^2).
    assert dg.endpoint_drift(z + 0.25 * u, z, 0.0) != pytest.approx(0.25 / math.sqrt(1.0625), rel=1e-6)


def test_joint_endpoint_is_mean_of_kv_drifts():
    """Unequal K and V norms and drifts: E^KV is the mean of the two ratios, not the ratio of
    the concatenated slices (which would weight the larger tensor)."""
    rng = np.random.default_rng(7)
    k = rng.standard_normal((2, 2, 7, 8))
    v = 10.0 * rng.standard_normal((2, 2, 7, 8))
    dk, dv, e = dg.joint_endpoint(1.2 * k, k, 0.9 * v, v, 0.0)
    np.testing.assert_allclose(dk, 0.2, rtol=1e-12)
    np.testing.assert_allclose(dv, 0.1, rtol=1e-12)
    np.testing.assert_allclose(e, 0.15, rtol=1e-12)
    nk, nv = (k**2).sum(axis=(-2, -1)), (v**2).sum(axis=(-2, -1))
    concat = np.sqrt(0.04 * nk + 0.01 * nv) / np.sqrt(nk + nv)
    assert np.all(np.abs(e - concat) > 1e-3)


def test_drift_log_ratio_closed_form_and_sign():
    """Reference scaled by 1.02, target by 1.2 per step: rho = log10(0.02 / 0.2) = -1 at eps = 0."""
    rng = np.random.default_rng(8)
    zr, zt = rng.standard_normal((1, 3, 11, 8)), rng.standard_normal((1, 3, 5, 8))
    d_ref, d_tgt, rho = dg.drift_log_ratio(1.02 * zr, zr, 1.2 * zt, zt, 0.0)
    np.testing.assert_allclose(d_ref, 0.02, rtol=1e-11)
    np.testing.assert_allclose(d_tgt, 0.2, rtol=1e-11)
    np.testing.assert_allclose(rho, -1.0, rtol=1e-11)
    # Swapping the roles negates rho.
    _, _, rho2 = dg.drift_log_ratio(1.2 * zt, zt, 1.02 * zr, zr, 0.0)
    np.testing.assert_allclose(rho2, 1.0, rtol=1e-11)


def test_drift_log_ratio_eps_keeps_still_slices_finite():
    z = np.ones((1, 1, 2, 4))
    _, _, rho = dg.drift_log_ratio(z, z, z, z, 1e-8)
    np.testing.assert_allclose(rho, 0.0, atol=0)


def test_mass_mean_ramp_and_complement():
    m = np.linspace(0.1, 0.5, 9).reshape(1, 1, 9)
    np.testing.assert_allclose(dg.mass_mean(m), 0.3, rtol=1e-14)
    np.testing.assert_allclose(dg.mass_mean(m, complement=True), 0.7, rtol=1e-14)


def _collinear(n_q, n_ref, n_tgt, d, a, b, c):
    """Queries c e1, reference keys a e1, target keys b e1: every query sees reference logits
    s c a and target logits s c b, so its reference mass is the sigmoid closed form."""
    e1 = np.zeros(d)
    e1[0] = 1.0
    q = np.tile(c * e1, (1, 1, n_q, 1))
    kr = np.tile(a * e1, (1, 1, n_ref, 1))
    kt = np.tile(b * e1, (1, 1, n_tgt, 1))
    return q, kr, kt


def test_exposure_sigmoid_closed_form():
    n_ref, n_tgt, d = 6, 10, 16
    q, kr, kt = _collinear(4, n_ref, n_tgt, d, a=2.0, b=-1.0, c=1.5)
    s = 1.0 / math.sqrt(d)
    x, y = s * 1.5 * 2.0, s * 1.5 * -1.0
    want = n_ref * math.exp(x) / (n_ref * math.exp(x) + n_tgt * math.exp(y))
    np.testing.assert_allclose(dg.exposure(q, kr, kt), want, rtol=1e-13)


def test_uniform_attention_masses_are_segment_fractions():
    """Identical logits: target queries put n_ref / n on reference keys, reference queries
    put n_tgt / n on target keys."""
    rng = np.random.default_rng(9)
    n_ref, n_tgt = 5, 11
    q = rng.standard_normal((2, 3, 4, 8))
    kr = np.zeros((2, 3, n_ref, 8))
    kt = np.zeros((2, 3, n_tgt, 8))
    np.testing.assert_allclose(dg.exposure(q, kr, kt), n_ref / (n_ref + n_tgt), rtol=1e-14)
    np.testing.assert_allclose(dg.ref_query_target_mass(q, kr, kt), n_tgt / (n_ref + n_tgt), rtol=1e-14)


def test_cached_exposure_with_stale_reference_keys():
    """Same-step cached exposure: current queries and target keys, anchor reference keys. With
    collinear keys the anchor shift moves the mass along the sigmoid."""
    q, kr_now, kt = _collinear(3, 4, 8, 8, a=1.0, b=0.0, c=2.0)
    _, kr_anchor, _ = _collinear(3, 4, 8, 8, a=0.0, b=0.0, c=2.0)
    s = 1.0 / math.sqrt(8)
    fresh = 4 * math.exp(2 * s) / (4 * math.exp(2 * s) + 8)
    np.testing.assert_allclose(dg.exposure(q, kr_now, kt), fresh, rtol=1e-13)
    np.testing.assert_allclose(dg.exposure(q, kr_anchor, kt), 4 / 12, rtol=1e-13)


def test_adjacent_ref_change_hand_trajectory():
    """Head means 0.10, 0.12, 0.11, 0.11: |0.02| + |0.01| + 0 over T - 1 = 3 steps is 1.0 point."""
    heads = np.array([[0.05, 0.15], [0.10, 0.14], [0.11, 0.11], [0.02, 0.20]])  # [T, heads], means as above
    log = heads[:, None, None, :]  # [T, n_blocks=1, B=1, H=2]
    np.testing.assert_allclose(dg.adjacent_ref_change(log), [1.0], rtol=1e-12)


def test_adjacent_ref_change_per_block_and_edges():
    T, nb = 5, 3
    log = np.zeros((T, nb, 2))
    log[:, 1, :] = np.arange(T)[:, None] * 0.01  # rises 1 point per step
    log[::2, 2, :] = 0.3  # alternates 0.3, 0 -> 30 points per step
    np.testing.assert_allclose(dg.adjacent_ref_change(log), [0.0, 1.0, 30.0], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dg.adjacent_ref_change(log[:2]), [0.0, 1.0, 30.0], rtol=1e-12, atol=1e-12)
    with pytest.raises(ValueError):
        dg.adjacent_ref_change(log[:1])
