"""Diagnostic quantities of the paper's analysis, in fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Definitions followed
--------------------
* Consecutive drift (Sec. 3.1, consecutive-drift equation):
  D_t(X) = ||X_t - X_{t-1}||_F / (||X_{t-1}||_F + eps) over the [n, d] slice of
  one (batch, head), for X a reference or a target slice of K or V.
* Matched log-ratio (Sec. 3.1, drift-log-ratio equation):
  rho = log10((D(Z_ref) + eps) / (D(Z_tgt) + eps)); negative when the reference
  slice moves more slowly than the target slice.
* Endpoint drift (Sec. 3.3, endpoint-drift equation):
  D_{t|a}(Z_ref) = ||Z_ref,t - Z_ref,a||_F / (||Z_ref,a||_F + eps) against an
  earlier anchor step a. The paper takes it separately on the head-resolved K
  and V slices and calls the result their joint endpoint scalar E^KV without
  printing the combination; this oracle reads it as the mean of the two
  drifts, E^KV = (D(K) + D(V)) / 2.
* Exposure (Sec. 3.2, directional-exposure equation): per head, the mean over
  target queries of the post-softmax mass on reference keys. The same-step
  cached exposure of App. A.2 is the same quantity with the reference keys
  taken at the anchor step and the target queries and keys at the current
  step.
* Reference-query mass on target keys (App., directional attention
  diagnostics): per head, the mean over reference queries of the mass on
  target keys, i.e. one minus their mass on reference keys.
* Adjacent reference-mass change (Sec. 3.2, adjacent-ref-change equation):
  per block, 100 / (T - 1) * sum_{t>=2} |Mbar_t - Mbar_{t-1}| in percentage
  points, Mbar_t the head mean of the exposure at step t.
"""

from __future__ import annotations

import numpy as np

from .joint_attention import joint_attention


def _frob_ratio(cur, base, eps):
    """||cur - base||_F / (||base||_F + eps) over the last two axes."""
    a = np.asarray(cur, dtype=np.float64)
    b = np.asarray(base, dtype=np.float64)
    if a.shape != b.shape:
        raise ValueError("the two slices must have the same shape")
    return np.sqrt(((a - b) ** 2).sum(axis=(-2, -1))) / (np.sqrt((b**2).sum(axis=(-2, -1))) + eps)


def consecutive_drift(z_cur, z_prev, eps=1e-8):
    """Sec. 3.1 consecutive drift per (batch, head): ``[..., n, d] -> [...]``."""
    return _frob_ratio(z_cur, z_prev, eps)


def endpoint_drift(z_cur, z_anchor, eps=1e-8):
    """Sec. 3.3 anchor-to-current drift per (batch, head): ``[..., n, d] -> [...]``."""
    return _frob_ratio(z_cur, z_anchor, eps)


def joint_endpoint(k_cur, k_anchor, v_cur, v_anchor, eps=1e-8):
    """(D(K), D(V), E^KV) of the reference K/V against the anchor; E^KV is the mean of the two."""
    dk = endpoint_drift(k_cur, k_anchor, eps)
    dv = endpoint_drift(v_cur, v_anchor, eps)
    return dk, dv, 0.5 * (dk + dv)


def drift_log_ratio(z_ref_cur, z_ref_prev, z_tgt_cur, z_tgt_prev, eps=1e-8):
    """(D_ref, D_tgt, rho) for one of K, V at adjacent steps (Sec. 3.1)."""
    d_ref = consecutive_drift(z_ref_cur, z_ref_prev, eps)
    d_tgt = consecutive_drift(z_tgt_cur, z_tgt_prev, eps)
    with np.errstate(divide="ignore", invalid="ignore"):
        rho = np.log10((d_ref + eps) / (d_tgt + eps))
    return d_ref, d_tgt, rho


def mass_mean(mass, complement=False):
    """Mean over the last axis of a per-query mass, or of one minus it."""
    m = np.asarray(mass, dtype=np.float64)
    return (1.0 - m).mean(axis=-1) if complement else m.mean(axis=-1)


def exposure(q_tgt, k_ref, k_tgt, scale=None):
    """Per-head exposure: mean over target queries of their mass on reference keys.

    The values do not enter the softmax, so zero values are passed to the
    attention oracle and only its ``ref_mass`` is used.
    """
    k_ref = np.asarray(k_ref, dtype=np.float64)
    k_tgt = np.asarray(k_tgt, dtype=np.float64)
    r = joint_attention(q_tgt, k_ref, np.zeros_like(k_ref), k_tgt, np.zeros_like(k_tgt), scale)
    return mass_mean(r["ref_mass"])


def ref_query_target_mass(q_ref, k_ref, k_tgt, scale=None):
    """Per-head mean over reference queries of their mass on target keys."""
    k_ref = np.asarray(k_ref, dtype=np.float64)
    k_tgt = np.asarray(k_tgt, dtype=np.float64)
    r = joint_attention(q_ref, k_ref, np.zeros_like(k_ref), k_tgt, np.zeros_like(k_tgt), scale)
    return mass_mean(r["ref_mass"], complement=True)


def adjacent_ref_change(mass_log):
    """Per block, in percentage points, from a ``[T, n_blocks, ...]`` log of per-head exposure.

    The head mean runs over every axis after the block axis.
    """
    m = np.asarray(mass_log, dtype=np.float64)
    if m.ndim < 2 or m.shape[0] < 2:
        raise ValueError("need a [T, n_blocks, ...] log with T >= 2")
    mbar = m.reshape(m.shape[0], m.shape[1], -1).mean(axis=-1)  # [T, n_blocks]
    return 100.0 / (m.shape[0] - 1) * np.abs(np.diff(mbar, axis=0)).sum(axis=0)
