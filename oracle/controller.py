"""Alg. 1 (monotone depth-adaptive reference reuse) over exogenous inputs, fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's executor runs a diffusion transformer; here the per-block,
per-step Q/K/V tensors are supplied by the caller (``inputs(t, b)``), so the
loop exercises exactly the parts of Alg. 1 that act on attention:

* step 0 materialises every block (full joint attention on fresh K/V), fills
  each block's cache with its reference Q/K/V and records target Q and the
  realised per-query reference mass;
* a step with ``t - a_full >= delta_max`` recomputes every block from block 0,
  refreshes all caches and sets ``a_full = t`` (bounded-age refresh);
* otherwise blocks are scanned shallow to deep: before the first crossing a
  block reuses (target queries attend to the cached reference K/V), the first
  block whose head-mean score reaches theta reactivates (the block's cached
  reference state is restored: its reference queries and the current target
  queries attend over the cached reference K/V and the current target K/V;
  cache unchanged), and every deeper block computes on fresh reference Q/K/V
  and refreshes its cache (age = t);
* every block records its target Q and the realised target->reference mass
  of the attention it executed, for the next step.

``cue="anchor"`` replaces the target-side cue by the change from the block's
most recent materialisation anchor (App. A.2, anchor-relative target-Q change):
D is measured against the target Q the block had at its last COMPUTE step
a_b, not at the previous step; the gate is otherwise the same (the paper's
Anchor-Q x Exposure ablation).

Reading taken where the paper relies on the DiT: at the boundary block the
paper restores the cached reference hidden state and runs the reference-query
computation from it (Alg. 1 boundary branch; Sec. 4 "Execution and cache
state": the block cache holds that state and its K/V). Without a DiT, the
cache keeps the state's reference Q, K and V from the block's last COMPUTE
step, so the boundary's reference rows attend with those cached queries over
[cached K_R; current K_Y], the target rows with their current queries over
the same keys, and the cache is left unchanged.

``local_impact`` is the Sec. 3.3 local-impact equation, used to report the
executed target output's relative change against the full-fresh output.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from .joint_attention import joint_attention
from .stats import COMPUTE, REACTIVATE, REUSE, full_refresh_due, gate, q_change


def local_impact(o_exec, o_fresh, eps=1e-8):
    """||O_exec - O_fresh||_F / (||O_fresh||_F + eps) over the last two axes."""
    a = np.asarray(o_exec, dtype=np.float64)
    b = np.asarray(o_fresh, dtype=np.float64)
    return np.sqrt(((a - b) ** 2).sum(axis=(-2, -1))) / (np.sqrt((b**2).sum(axis=(-2, -1))) + eps)


@dataclass
class ControllerTrace:
    decisions: np.ndarray  # [T, n_blocks] int (REUSE / REACTIVATE / COMPUTE)
    d_mean: np.ndarray  # [T, n_blocks] mean D where the gate was evaluated, else nan
    m_mean: np.ndarray  # [T, n_blocks] mean lagged M where evaluated, else nan
    g_mean: np.ndarray  # [T, n_blocks] mean D*M where evaluated, else nan
    impact: np.ndarray  # [T, n_blocks, B, H] I^KV of executed vs full-fresh target output
    ages: np.ndarray  # [T, n_blocks] a_b after the step
    outputs: dict = field(default_factory=dict)  # (t, b) -> executed target output / mass


def run_controller(
    inputs,
    n_steps,
    n_blocks,
    theta,
    delta_max=None,
    mode="product",
    theta_m=None,
    eps=1e-8,
    scale=None,
    keep_outputs=False,
    cue="consecutive",
):
    """Run Alg. 1 and return a ``ControllerTrace``.

    ``inputs(t, b)`` returns a dict with ``q_ref, k_ref, v_ref, q_tgt, k_tgt,
    v_tgt`` arrays of shape ``[B, H, n, d]`` (the fresh tensors of block ``b``
    at step ``t``). ``theta`` is a scalar or a per-block sequence.
    """
    if cue not in ("consecutive", "anchor"):
        raise ValueError(f"unknown cue {cue!r}")
    theta = np.broadcast_to(np.asarray(theta, dtype=np.float64), (n_blocks,))
    theta_m_arr = None
    if theta_m is not None:
        theta_m_arr = np.broadcast_to(np.asarray(theta_m, dtype=np.float64), (n_blocks,))

    decisions = np.full((n_steps, n_blocks), -1, dtype=np.int64)
    d_mean = np.full((n_steps, n_blocks), np.nan)
    m_mean = np.full((n_steps, n_blocks), np.nan)
    g_mean = np.full((n_steps, n_blocks), np.nan)
    ages = np.zeros((n_steps, n_blocks), dtype=np.int64)
    impact = None
    outputs = {}

    cache_k = [None] * n_blocks
    cache_v = [None] * n_blocks
    cache_q = [None] * n_blocks  # reference queries of the cached state
    q_rec = [None] * n_blocks
    q_anchor = [None] * n_blocks  # target Q at the block's last COMPUTE step
    mass_rec = [None] * n_blocks
    age = np.zeros(n_blocks, dtype=np.int64)
    a_full = 0

    for t in range(n_steps):
        full = full_refresh_due(t, a_full, delta_max)
        if full:
            a_full = t
        reactivated = False
        for b in range(n_blocks):
            x = inputs(t, b)
            n_ref = x["k_ref"].shape[-2]
            fresh = joint_attention(x["q_tgt"], x["k_ref"], x["v_ref"], x["k_tgt"], x["v_tgt"], scale)

            if full:
                dec = COMPUTE
            else:
                d = q_change(x["q_tgt"], q_anchor[b] if cue == "anchor" else q_rec[b], eps)
                res = gate(
                    d,
                    mass_rec[b],
                    theta[b],
                    reactivated,
                    mode=mode,
                    theta_m=None if theta_m_arr is None else theta_m_arr[b],
                )
                dec, reactivated = res.decision, res.reactivated
                if dec != COMPUTE:  # the gate is only read before the boundary
                    d_mean[t, b], m_mean[t, b], g_mean[t, b] = res.d_mean, res.m_mean, res.g_mean

            if dec == COMPUTE:
                q_all = np.concatenate([x["q_ref"], x["q_tgt"]], axis=-2)
                ex = joint_attention(q_all, x["k_ref"], x["v_ref"], x["k_tgt"], x["v_tgt"], scale)
                o_tgt = ex["o"][..., n_ref:, :]
                mass_tgt = ex["ref_mass"][..., n_ref:]
                cache_k[b] = np.array(x["k_ref"], dtype=np.float64)
                cache_v[b] = np.array(x["v_ref"], dtype=np.float64)
                cache_q[b] = np.array(x["q_ref"], dtype=np.float64)
                q_anchor[b] = np.array(x["q_tgt"], dtype=np.float64)
                age[b] = t
            elif dec == REACTIVATE:  # restored state: its reference queries, current target queries
                q_all = np.concatenate([cache_q[b], x["q_tgt"]], axis=-2)
                ex = joint_attention(q_all, cache_k[b], cache_v[b], x["k_tgt"], x["v_tgt"], scale)
                o_tgt = ex["o"][..., n_ref:, :]
                mass_tgt = ex["ref_mass"][..., n_ref:]
            else:  # REUSE
                ex = joint_attention(x["q_tgt"], cache_k[b], cache_v[b], x["k_tgt"], x["v_tgt"], scale)
                o_tgt = ex["o"]
                mass_tgt = ex["ref_mass"]

            imp = local_impact(o_tgt, fresh["o"], eps)
            if impact is None:
                impact = np.zeros((n_steps, n_blocks) + imp.shape)
            impact[t, b] = imp
            decisions[t, b] = dec
            q_rec[b] = np.array(x["q_tgt"], dtype=np.float64)
            mass_rec[b] = mass_tgt
            if keep_outputs:
                outputs[(t, b)] = {"o_tgt": o_tgt, "ref_mass": mass_tgt, "o_all": ex["o"] if dec != REUSE else None}
        ages[t] = age
    return ControllerTrace(decisions, d_mean, m_mean, g_mean, impact, ages, outputs)
