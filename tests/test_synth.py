"""The seeded input generators are deterministic and round exactly to the run dtype."""

import hashlib

import numpy as np
import pytest
import torch

from paper_2609_32415_amd import synth


def _digest(t):
    h = hashlib.sha256()
    for k in sorted(t):
        h.update(k.encode())
        h.update(np.ascontiguousarray(t[k]).tobytes())
    return h.hexdigest()


def test_same_seed_same_bytes_and_different_blocks_differ():
    w = synth.workload("single_ref", heads=2, n_ref=96, n_tgt=64)
    a, b = synth.block_inputs(w, 0), synth.block_inputs(w, 0)
    assert _digest(a) == _digest(b)
    assert _digest(synth.block_inputs(w, 1)) != _digest(a)


def test_bf16_rounding_matches_torch_round_to_nearest_even():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 7
    ours = synth.round_to_dtype(x, "bf16")
    ref = torch.from_numpy(x).to(torch.bfloat16).float().numpy()
    assert np.array_equal(ours, ref)


def test_trajectory_drift_has_requested_scale():
    w = synth.workload("tiny")
    tr = synth.Trajectory(w, block=0)
    x0 = tr.step_tensors(0)
    x1 = tr.step_tensors(1)
    dq = np.std(x1["q_tgt"] - x0["q_tgt"])
    dk = np.std(x1["k_ref"] - x0["k_ref"])
    assert abs(dq - 0.3) < 0.01 and abs(dk - 0.01) < 0.001


def test_sweep_schedules():
    assert abs(synth.sweep_ref_drift(0) - 0.02) < 1e-12
    assert abs(synth.sweep_ref_drift(30) - 0.002) < 1e-12
    assert abs(synth.sweep_ref_drift(59) - 0.03) < 1e-12
    assert abs(synth.sweep_tgt_drift(1) - 0.3) < 1e-12 and abs(synth.sweep_tgt_drift(7) - 0.05) < 1e-12


def test_key_bias_sets_target_component():
    w = synth.workload("single_ref", heads=3, n_ref=32, n_tgt=200)
    t = synth.base_tensors(w)
    # Every target query's component along the bias direction is +1 or -lambda_h.
    rng_u = synth._rng(w.seed, 0, 0, synth.ROLE_IDS["bias"])
    u = rng_u.standard_normal((1, 3, 128), dtype=np.float32).astype(np.float64)
    u /= np.linalg.norm(u, axis=-1, keepdims=True)
    comp = np.einsum("bhnd,bhd->bhn", t["q_tgt"].astype(np.float64), u)
    for h, lam in enumerate([0.0, 3.0, 6.0]):
        vals = comp[0, h]
        ok = np.isclose(vals, 1.0, atol=1e-4) | np.isclose(vals, -lam, atol=1e-4)
        assert ok.all()
        frac = np.isclose(vals, 1.0, atol=1e-4).mean()
        assert 0.15 < frac < 0.45 or lam == 1.0


def test_per_segment_key_bias_weights():
    """Weights scale the reference-key bias per segment; no weights leaves the inputs unchanged."""
    base = synth.workload("tiny", dtype="bf16", heads=2, head_dim=64, n_ref=192, n_tgt=64, key_bias=True)
    w = synth.workload("tiny", dtype="bf16", heads=2, head_dim=64, n_ref=192, n_tgt=64, key_bias=True,
                       ref_segments=(128, 64), ref_bias_weights=(1.0, 0.0))
    a, b = synth.base_tensors(base), synth.base_tensors(w)
    np.testing.assert_array_equal(a["k_ref"][:, :, :128], b["k_ref"][:, :, :128])
    unbiased = synth.workload("tiny", dtype="bf16", heads=2, head_dim=64, n_ref=192, n_tgt=64, key_bias=False)
    np.testing.assert_array_equal(b["k_ref"][:, :, 128:], synth.base_tensors(unbiased)["k_ref"][:, :, 128:])
    np.testing.assert_array_equal(a["q_tgt"], b["q_tgt"])
    with pytest.raises(ValueError):
        synth.base_tensors(synth.workload("tiny", n_ref=192, key_bias=True, ref_segments=(100,),
                                          ref_bias_weights=(1.0,)))


def test_sweep_key_bias_depth_profile():
    """The sweep's lambda falls with depth (6 at block 0 to 0 at the deepest block) with a bounded
    per-head offset, so the head-mean reference exposure rises with depth."""
    w = synth.workload("sweep")
    lam = np.array([[synth._lambda(w, b, h) for h in range(w.heads)] for b in range(w.n_blocks)])
    assert lam.min() >= 0.0 and lam.max() <= 6.0
    mean = np.array([synth.sweep_lambda_mean(b, w.n_blocks) for b in range(w.n_blocks)])
    assert mean[0] == 6.0 and mean[-1] == 0.0 and np.all(np.diff(mean) < 0)
    inside = (mean[:, None] > synth.LAMBDA_JITTER) & (mean[:, None] < 6.0 - synth.LAMBDA_JITTER)
    assert np.all(np.abs(lam - mean[:, None])[inside.repeat(w.heads, 1)] <= synth.LAMBDA_JITTER)
    assert lam[:10].mean() > 4.0 and lam[-10:].mean() < 2.0
