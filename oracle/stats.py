"""Runtime cues and the reuse gate, in fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Definitions followed
--------------------
* Consecutive drift (paper Sec. 3.1, consecutive-drift equation):
  D_t(X) = ||X_t - X_{t-1}||_F / (||X_{t-1}||_F + eps), with token scope and
  head fixed. The controller applies it to each post-RoPE target-query head
  (Sec. 4, "Runtime cues observable under reuse"), so X is the [n_tgt, d]
  slice of one (batch, head).
* Directional exposure (Sec. 3.2, directional-exposure equation):
  M_h = (1/|Q_Y|) sum_{q in Q_Y} sum_{k in K_R} A_qk, i.e. the mean over target
  queries of the per-query reference mass; the controller reads the value
  recorded from the previous step's executed attention (Sec. 4).
* Interaction score (Sec. 4, factorized-risk equation): g_h = D_h * M_h,
  formed per head before aggregation.
* Head aggregate (App. A.2, candidate-head-aggregate equation): plain mean
  over heads. With more than one batch element the mean runs over
  batch x heads and yields one decision per block.
* Block decision (Sec. 4, depth-cutoff equation, and the block branch of
  Alg. 1): once the step has reactivated, every deeper block computes;
  otherwise a head-mean score below theta reuses, and a score reaching theta
  (>=) makes the block the reactivation boundary.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

# Block decisions of Alg. 1.
REUSE = 0  # skip reference rows; target attends to the cached reference K/V
REACTIVATE = 1  # boundary: target still on the cache, reference queries run
COMPUTE = 2  # fresh reference K/V, full joint attention, cache refreshed

GATE_MODES = ("product", "q_only", "mass_only", "and")


def q_change(q_cur, q_prev, eps=1e-8):
    """Relative Frobenius change per (batch, head) over the last two axes.

    ``q_cur``/``q_prev`` are ``[..., n_tgt, d]``; returns ``[...]`` fp64.
    """
    a = np.asarray(q_cur, dtype=np.float64)
    b = np.asarray(q_prev, dtype=np.float64)
    if a.shape != b.shape:
        raise ValueError("q_cur and q_prev must have the same shape")
    num = np.sqrt(((a - b) ** 2).sum(axis=(-2, -1)))
    den = np.sqrt((b**2).sum(axis=(-2, -1))) + eps
    return num / den


def head_exposure(ref_mass):
    """Mean over target queries of the per-query reference mass: ``[..., n_tgt] -> [...]``."""
    m = np.asarray(ref_mass, dtype=np.float64)
    return m.mean(axis=-1)


@dataclass
class GateResult:
    decision: int
    reactivated: bool
    d_mean: float  # mean over batch x heads of D
    m_mean: float  # mean over batch x heads of M
    g_mean: float  # mean over batch x heads of D * M (the paper's score)


def gate(d_cur, ref_mass_prev, theta, reactivated, mode="product", theta_m=None):
    """One block's decision.

    ``d_cur``: ``[B, H]`` target-Q change of this block at the current step.
    ``ref_mass_prev``: ``[B, H, n_tgt]`` per-query reference mass recorded
    from this block's executed attention at the previous step.
    ``theta``: this block's threshold. ``reactivated``: whether an earlier
    block of this step already reached its threshold.

    ``mode`` selects the score compared with ``theta``:
      ``product``   mean_h(D_h * M_h) (the paper's controller)
      ``q_only``    mean_h D_h          (target-Q cue alone)
      ``mass_only`` mean_h M_h          (exposure cue alone)
      ``and``       mean D >= theta and mean M >= theta_m
    """
    d = np.asarray(d_cur, dtype=np.float64)
    m = head_exposure(ref_mass_prev)
    if d.shape != m.shape:
        raise ValueError("d_cur must be [B, H] matching ref_mass_prev[..., :]")
    g = d * m
    d_mean, m_mean, g_mean = float(d.mean()), float(m.mean()), float(g.mean())
    if reactivated:
        return GateResult(COMPUTE, True, d_mean, m_mean, g_mean)
    if mode == "product":
        cross = g_mean >= theta
    elif mode == "q_only":
        cross = d_mean >= theta
    elif mode == "mass_only":
        cross = m_mean >= theta
    elif mode == "and":
        if theta_m is None:
            raise ValueError("mode 'and' needs theta_m")
        cross = d_mean >= theta and m_mean >= theta_m
    else:
        raise ValueError(f"unknown gate mode {mode!r}")
    if cross:
        return GateResult(REACTIVATE, True, d_mean, m_mean, g_mean)
    return GateResult(REUSE, False, d_mean, m_mean, g_mean)


def full_refresh_due(step, a_full, delta_max):
    """Bounded-age refresh test of Alg. 1: a step recomputes from block 0 when
    ``step - a_full >= delta_max``. Step 0 always materialises every block.
    ``delta_max`` of ``None`` disables the refresh."""
    if step == 0:
        return True
    if delta_max is None:
        return False
    return step - a_full >= delta_max
