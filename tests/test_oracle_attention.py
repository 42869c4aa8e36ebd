"""Pins for the oracle's joint attention (CPU only).

Each test checks the oracle against something other than itself: hand-derived
worked examples (tests/golden), torch's scaled_dot_product_attention in fp64
(a library routine), scipy's logsumexp, closed forms and invariants of the
softmax-attention definition. Shapes are deliberately asymmetric
(n_ref != n_tgt != n_q != d) so that a transposed operand or a swapped segment
fails.
"""

import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

from oracle import joint_attention, joint_attention_loops

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")


def _val(x):
    if isinstance(x, str):
        if x == "-inf":
            return -math.inf
        if x.startswith("2ln"):
            return 2 * math.log(float(x[3:]))
        if x.startswith("ln"):
            return math.log(float(x[2:]))
        raise ValueError(x)
    return float(x)


def _arr(rows, d=None):
    a = np.array([[_val(v) for v in r] for r in rows], dtype=np.float64)
    if a.size == 0:
        a = np.zeros((0, d))
    return a


def _golden(kind):
    with open(GOLDEN) as f:
        return json.load(f)[kind]


@pytest.mark.parametrize("case", _golden("attention"), ids=lambda c: c["cite"][:40])
def test_hand_examples(case):
    q = _arr(case["q"])
    d = q.shape[1]
    kr, vr = _arr(case["k_ref"], d), _arr(case["v_ref"], d)
    kt, vt = _arr(case["k_tgt"], d), _arr(case["v_tgt"], d)
    out = joint_attention(q, kr, vr, kt, vt, scale=case["scale"])
    np.testing.assert_allclose(out["o"], _arr(case["o"]), rtol=0, atol=1e-12)
    np.testing.assert_allclose(out["ref_mass"], [_val(v) for v in case["ref_mass"]], rtol=0, atol=1e-14)
    np.testing.assert_allclose(out["lse_all"], [_val(v) for v in case["lse_all"]], rtol=0, atol=1e-12)
    np.testing.assert_allclose(out["lse_ref"], [_val(v) for v in case["lse_ref"]], rtol=0, atol=1e-12)
    # The loop form reaches the same values on the same worked example.
    lo = joint_attention_loops(q[None, None], kr[None, None], vr[None, None], kt[None, None], vt[None, None], case["scale"])
    np.testing.assert_allclose(lo["o"][0, 0], _arr(case["o"]), rtol=0, atol=1e-12)
    np.testing.assert_allclose(lo["ref_mass"][0, 0], [_val(v) for v in case["ref_mass"]], rtol=0, atol=1e-14)


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def _sdpa(q, k, v, scale):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(torch.float64)
    return torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), scale=scale).numpy()


@pytest.mark.parametrize("n_ref,n_tgt,n_q,d,scale", [(7, 5, 3, 4, None), (0, 9, 6, 8, None), (13, 1, 2, 16, 0.37), (40, 24, 31, 64, None)])
def test_output_matches_torch_sdpa_fp64(n_ref, n_tgt, n_q, d, scale):
    B, H = 2, 3
    q = _rand((B, H, n_q, d), 1)
    kr, vr = _rand((B, H, n_ref, d), 2), _rand((B, H, n_ref, d), 3)
    kt, vt = _rand((B, H, n_tgt, d), 4), _rand((B, H, n_tgt, d), 5)
    out = joint_attention(q, kr, vr, kt, vt, scale)
    s = 1 / math.sqrt(d) if scale is None else scale
    ref = _sdpa(q, np.concatenate([kr, kt], 2), np.concatenate([vr, vt], 2), s)
    np.testing.assert_allclose(out["o"], ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("n_ref,n_tgt", [(5, 11), (17, 3), (1, 1)])
def test_mass_is_attention_onto_reference_indicator(n_ref, n_tgt):
    """With V = indicator of the reference segment, softmax attention outputs
    exactly the per-query reference mass (computed here by torch SDPA)."""
    B, H, n_q, d = 1, 2, 6, 8
    q = _rand((B, H, n_q, d), 11, 2.0)
    kr, kt = _rand((B, H, n_ref, d), 12), _rand((B, H, n_tgt, d), 13)
    out = joint_attention(q, kr, np.zeros((B, H, n_ref, d)), kt, np.zeros((B, H, n_tgt, d)))
    ind = np.concatenate([np.ones((B, H, n_ref, 1)), np.zeros((B, H, n_tgt, 1))], 2)
    ref = _sdpa(q, np.concatenate([kr, kt], 2), ind, 1 / math.sqrt(d))[..., 0]
    np.testing.assert_allclose(out["ref_mass"], ref, rtol=0, atol=1e-13)
    assert np.all(out["ref_mass"] >= 0) and np.all(out["ref_mass"] <= 1)


def test_lse_matches_scipy_logsumexp_and_mass_identity():
    B, H, n_ref, n_tgt, n_q, d = 1, 2, 9, 4, 5, 16
    q = _rand((B, H, n_q, d), 21, 3.0)
    kr, kt = _rand((B, H, n_ref, d), 22), _rand((B, H, n_tgt, d), 23)
    vr, vt = _rand((B, H, n_ref, d), 24), _rand((B, H, n_tgt, d), 25)
    out = joint_attention(q, kr, vr, kt, vt)
    k = np.concatenate([kr, kt], 2)
    logits = (torch.from_numpy(q) @ torch.from_numpy(k).transpose(-1, -2)).numpy() / math.sqrt(d)
    np.testing.assert_allclose(out["lse_all"], scipy.special.logsumexp(logits, axis=-1), rtol=0, atol=1e-12)
    np.testing.assert_allclose(out["lse_ref"], scipy.special.logsumexp(logits[..., :n_ref], axis=-1), rtol=0, atol=1e-12)
    np.testing.assert_allclose(np.exp(out["lse_ref"] - out["lse_all"]), out["ref_mass"], rtol=1e-12, atol=0)


def test_uniform_attention_closed_form():
    """Identical keys make every softmax row uniform: O = mean of V and the
    reference mass is n_ref / (n_ref + n_tgt) exactly."""
    B, H, n_ref, n_tgt, n_q, d = 1, 2, 12, 21, 4, 8
    key = _rand((d,), 31)
    kr = np.broadcast_to(key, (B, H, n_ref, d))
    kt = np.broadcast_to(key, (B, H, n_tgt, d))
    vr, vt = _rand((B, H, n_ref, d), 32), _rand((B, H, n_tgt, d), 33)
    out = joint_attention(_rand((B, H, n_q, d), 34), kr, vr, kt, vt)
    mean_v = np.concatenate([vr, vt], 2).mean(axis=2, keepdims=True)
    np.testing.assert_allclose(out["o"], np.broadcast_to(mean_v, out["o"].shape), rtol=0, atol=1e-13)
    np.testing.assert_allclose(out["ref_mass"], n_ref / (n_ref + n_tgt), rtol=0, atol=1e-15)
    # A zero query sees uniform logits regardless of the keys.
    out0 = joint_attention(np.zeros((B, H, 1, d)), _rand((B, H, n_ref, d), 35), vr, _rand((B, H, n_tgt, d), 36), vt)
    np.testing.assert_allclose(out0["ref_mass"], n_ref / (n_ref + n_tgt), rtol=0, atol=1e-15)


def test_rows_sum_to_one_and_linearity_in_v():
    B, H, n_ref, n_tgt, n_q, d = 1, 1, 6, 10, 7, 4
    q = _rand((B, H, n_q, d), 41, 2.0)
    kr, kt = _rand((B, H, n_ref, d), 42), _rand((B, H, n_tgt, d), 43)
    ones = joint_attention(q, kr, np.ones((B, H, n_ref, d)), kt, np.ones((B, H, n_tgt, d)))
    np.testing.assert_allclose(ones["o"], 1.0, rtol=0, atol=1e-14)
    va, vb = _rand((B, H, n_ref + n_tgt, d), 44), _rand((B, H, n_ref + n_tgt, d), 45)
    f = lambda v: joint_attention(q, kr, v[:, :, :n_ref], kt, v[:, :, n_ref:])["o"]
    np.testing.assert_allclose(f(2.5 * va - 0.5 * vb), 2.5 * f(va) - 0.5 * f(vb), rtol=0, atol=1e-12)


def test_key_permutation_within_segment():
    B, H, n_ref, n_tgt, n_q, d = 1, 2, 9, 7, 3, 8
    q = _rand((B, H, n_q, d), 51)
    kr, vr = _rand((B, H, n_ref, d), 52), _rand((B, H, n_ref, d), 53)
    kt, vt = _rand((B, H, n_tgt, d), 54), _rand((B, H, n_tgt, d), 55)
    base = joint_attention(q, kr, vr, kt, vt)
    pr, pt = np.random.default_rng(5).permutation(n_ref), np.random.default_rng(6).permutation(n_tgt)
    perm = joint_attention(q, kr[:, :, pr], vr[:, :, pr], kt[:, :, pt], vt[:, :, pt])
    for key in ("o", "ref_mass", "lse_all", "lse_ref"):
        np.testing.assert_allclose(perm[key], base[key], rtol=0, atol=1e-13)
    # Moving one key from the target to the reference segment moves its weight into the mass.
    moved = joint_attention(q, np.concatenate([kr, kt[:, :, :1]], 2), np.concatenate([vr, vt[:, :, :1]], 2), kt[:, :, 1:], vt[:, :, 1:])
    np.testing.assert_allclose(moved["o"], base["o"], rtol=0, atol=1e-13)
    assert np.all(moved["ref_mass"] > base["ref_mass"])


def test_empty_reference_is_plain_self_attention():
    B, H, n, d = 1, 2, 11, 8
    q, k, v = _rand((B, H, n, d), 61), _rand((B, H, n, d), 62), _rand((B, H, n, d), 63)
    out = joint_attention(q, np.zeros((B, H, 0, d)), np.zeros((B, H, 0, d)), k, v)
    np.testing.assert_allclose(out["o"], _sdpa(q, k, v, 1 / math.sqrt(d)), rtol=0, atol=1e-13)
    assert np.all(out["ref_mass"] == 0.0)
    assert np.all(np.isneginf(out["lse_ref"]))


def test_loops_match_vectorised_on_random_tiny_shapes():
    B, H, n_ref, n_tgt, n_q, d = 1, 2, 5, 3, 4, 6
    args = [_rand((B, H, n, d), 70 + i) for i, n in enumerate((n_q, n_ref, n_ref, n_tgt, n_tgt))]
    a = joint_attention(*args, scale=0.3)
    b = joint_attention_loops(*args, scale=0.3)
    for key in ("o", "ref_mass", "lse_all", "lse_ref"):
        np.testing.assert_allclose(a[key], b[key], rtol=0, atol=1e-12)


def test_large_logits_do_not_overflow():
    """The definition is shift-invariant; huge logits must still give finite, exact rows."""
    q = np.array([[[[100.0, 0.0]]]])
    kr = np.array([[[[50.0, 0.0]]]])
    kt = np.array([[[[49.0, 0.0], [-10.0, 0.0]]]])
    out = joint_attention(q, kr, np.ones((1, 1, 1, 2)), kt, np.zeros((1, 1, 2, 2)), scale=1.0)
    # weights e^5000 : e^4900 : e^-1000 -> mass = 1 / (1 + e^-100 + ...)
    assert np.isfinite(out["o"]).all()
    np.testing.assert_allclose(out["ref_mass"], 1.0 / (1.0 + math.exp(-100.0)), rtol=1e-15)


def test_segment_masses_closed_forms():
    """Collinear keys: segment s (n_s keys at a_s e1), target (n_y keys at b e1), query c e1 ->
    mass_s = n_s e^{x_s} / (sum_s n_s e^{x_s} + n_y e^{y}) with x_s = scale c a_s, y = scale c b."""
    from oracle import segment_masses

    d, sizes, mags, n_y, b, c = 16, (3, 5, 2), (1.0, -2.0, 4.0), 7, 0.5, 1.5
    e1 = np.zeros(d)
    e1[0] = 1.0
    kr = np.concatenate([np.tile(m * e1, (n, 1)) for n, m in zip(sizes, mags)])[None, None]
    kt = np.tile(b * e1, (n_y, 1))[None, None]
    q = np.tile(c * e1, (4, 1))[None, None]
    s = 1.0 / np.sqrt(d)
    w = np.array([n * np.exp(s * c * m) for n, m in zip(sizes, mags)])
    want = w / (w.sum() + n_y * np.exp(s * c * b))
    got = segment_masses(q, kr, kt, np.cumsum(sizes).tolist())
    np.testing.assert_allclose(got[0, 0], np.tile(want, (4, 1)), rtol=1e-13)


def test_segment_masses_uniform_sum_and_permutation():
    from oracle import joint_attention, segment_masses

    rng = np.random.default_rng(12)
    q = rng.standard_normal((1, 2, 5, 8))
    np.testing.assert_allclose(segment_masses(q, np.zeros((1, 2, 10, 8)), np.zeros((1, 2, 6, 8)), [4, 10]),
                               np.broadcast_to([4 / 16, 6 / 16], (1, 2, 5, 2)), rtol=1e-14)
    kr, kt = rng.standard_normal((1, 2, 9, 8)), rng.standard_normal((1, 2, 4, 8))
    m = segment_masses(q, kr, kt, [3, 9])
    ref = joint_attention(q, kr, np.zeros_like(kr), kt, np.zeros_like(kt))["ref_mass"]
    np.testing.assert_allclose(m.sum(axis=-1), ref, rtol=1e-13)
    swapped = segment_masses(q, np.concatenate([kr[..., 3:, :], kr[..., :3, :]], axis=-2), kt, [6, 9])
    np.testing.assert_allclose(swapped[..., ::-1], m, rtol=1e-13)
    with pytest.raises(ValueError):
        segment_masses(q, kr, kt, [3, 8])
