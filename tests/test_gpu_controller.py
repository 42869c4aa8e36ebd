"""End-to-end parity of the on-device Alg. 1 executor with the oracle controller.

Both run the same seeded trajectory (sweep recipe at reduced shapes, bf16
inputs; and the tiny fp32 workload): per-(step, block) decisions must be
identical, and the executed target outputs, recorded masses, the reference
outputs of every block that runs its reference rows (the boundary's restored
state and the computing blocks) and the cache ages must match the oracle's
within the bars of the run dtype. Every case's thresholds keep each evaluated
head-mean score at least 1e-3 from theta (a closer score may legitimately flip
under rounding); a case that loses that margin fails instead of passing
silently.
"""

import math

import numpy as np
import pytest
import torch

from gpu_helpers import MASS_TOL, O_TOL, TORCH_DTYPE, dev, host, max_abs
from oracle import REUSE, run_controller
from paper_2609_32415_amd import synth

pytestmark = pytest.mark.gpu

W = synth.workload("sweep", heads=4, n_ref=160, n_tgt=192, n_blocks=6, n_steps=4, seed=99)
# The tiny fp32 workload: 2 heads, head_dim 64, 256 + 256 tokens, 4 steps x 4 blocks,
# reference drift 0.01 and target drift 0.3 per step.
TINY = synth.workload("tiny")
MARGIN = 1e-3


def _inputs(w, sweep):
    if sweep:
        trajs = [synth.Trajectory(w, b, ref_sigma=lambda t, b=b: synth.sweep_ref_drift(b, w.n_blocks),
                                  tgt_sigma=lambda t: synth.sweep_tgt_drift(t, w.n_steps)) for b in range(w.n_blocks)]
    else:
        trajs = [synth.Trajectory(w, b) for b in range(w.n_blocks)]
    return {(t, b): trajs[b].step_tensors(t) for t in range(w.n_steps) for b in range(w.n_blocks)}


_X = {}


def _x(w=W):
    if w.name not in _X:
        _X[w.name] = _inputs(w, w.name == "sweep")
    return _X[w.name]


def _assert_margin(w, tr, theta, mode="product", theta_m=None):
    th = np.broadcast_to(np.asarray(theta, dtype=np.float64), (w.n_blocks,))
    score = {"product": tr.g_mean, "q_only": tr.d_mean, "mass_only": tr.m_mean, "and": tr.d_mean}[mode]
    mask = ~np.isnan(score)
    gap = np.abs(score - th[None, :])[mask]
    if mode == "and":
        gap = np.concatenate([gap, np.abs(tr.m_mean - theta_m)[~np.isnan(tr.m_mean)]])
    assert gap.size == 0 or gap.min() > MARGIN, f"a gate score lies {gap.min():.2e} from theta: pick another case"


def _run_gpu(w, theta, delta_max=None, fused=True, mode="product", theta_m=None, cue="consecutive"):
    from paper_2609_32415_amd.controller import Controller

    x = _x(w)
    ctl = Controller(w.n_blocks, w.n_steps, w.batch, w.heads, w.n_ref, w.n_tgt, w.head_dim, theta,
                     delta_max=delta_max, device="cuda:0", fused=fused, mode=mode, theta_m=theta_m, cue=cue,
                     dtype=TORCH_DTYPE[w.dtype])
    outs, masses, orefs, ages = {}, {}, {}, []
    for t in range(w.n_steps):
        xs = [{k: dev(v, w.dtype) for k, v in x[(t, b)].items()} for b in range(w.n_blocks)]
        ctl.step(t, xs)
        torch.cuda.synchronize()
        for b in range(w.n_blocks):
            outs[(t, b)] = host(ctl.o_tgt[b])
            masses[(t, b)] = host(ctl.recorded_mass(b))
            orefs[(t, b)] = host(ctl.o_ref[b])
        ages.append(ctl.age.cpu().tolist())
    return ctl.decisions.cpu().numpy(), outs, masses, orefs, np.array(ages)


def _compare(w, ref, dec, outs, masses, orefs, ages):
    assert dec.tolist() == ref.decisions.tolist()
    assert ages.tolist() == ref.ages.tolist()
    for (t, b), o in outs.items():
        assert max_abs(o, ref.outputs[(t, b)]["o_tgt"]) <= O_TOL[w.dtype], (t, b)
        assert max_abs(masses[(t, b)], ref.outputs[(t, b)]["ref_mass"]) <= MASS_TOL[w.dtype], (t, b)
        if dec[t, b] != REUSE:  # the boundary's restored reference rows and the computing blocks'
            o_all = ref.outputs[(t, b)]["o_all"]
            assert max_abs(orefs[(t, b)], o_all[..., : w.n_ref, :]) <= O_TOL[w.dtype], (t, b)


PER_BLOCK = (0.2, 0.2, 0.115, 0.115, 0.045, 0.045)
PER_BLOCK2 = (0.09, 0.09, 0.07, 0.05, 0.05, 0.05)
CASES = [(0.02, None), (0.05, None), (0.08, None), (0.05, 2), (0.0, None), (1e9, None), (PER_BLOCK, None),
         (PER_BLOCK2, None)]


@pytest.mark.parametrize("fused", [True, False], ids=["fused", "separate"])
@pytest.mark.parametrize("theta,delta_max", CASES, ids=lambda v: str(v))
def test_controller_matches_oracle(theta, delta_max, fused):
    print(f"controller theta={theta} delta_max={delta_max} fused={fused}", flush=True)
    x = _x()
    ref = run_controller(lambda t, b: x[(t, b)], W.n_steps, W.n_blocks, theta, delta_max=delta_max, keep_outputs=True)
    _assert_margin(W, ref, theta)
    _compare(W, ref, *_run_gpu(W, theta, delta_max, fused))


@pytest.mark.parametrize("theta", [0.02, 0.0, math.inf], ids=["theta0.02", "theta0", "theta_inf"])
def test_controller_fp32_tiny_matches_oracle(theta):
    """The tiny fp32 trajectory (theta_q 0.1 x theta_m 0.2 = 0.02; every step then reactivates at
    block 0) and the always-reactivate / always-reuse extremes, held to the fp32 bars (1e-5)."""
    print(f"controller fp32 tiny theta={theta}", flush=True)
    x = _x(TINY)
    ref = run_controller(lambda t, b: x[(t, b)], TINY.n_steps, TINY.n_blocks, theta, keep_outputs=True)
    _assert_margin(TINY, ref, theta)
    _compare(TINY, ref, *_run_gpu(TINY, theta))


# (theta, delta_max, gate mode, theta_m, target-side cue): the single-cue ablations, the
# two-threshold gate and the anchor-relative cue of the paper's ablation table.
VARIANTS = [
    (0.2, None, "q_only", None, "consecutive"),
    (0.3, None, "mass_only", None, "consecutive"),
    (0.2, None, "and", 0.35, "consecutive"),
    (0.05, None, "product", None, "anchor"),
    (0.08, 2, "product", None, "anchor"),
    (1e9, 3, "product", None, "consecutive"),  # fixed-interval refresh (every 3 steps)
]


@pytest.mark.parametrize("theta,delta_max,mode,theta_m,cue", VARIANTS, ids=lambda v: str(v))
def test_controller_variants_match_oracle(theta, delta_max, mode, theta_m, cue):
    print(f"controller variant theta={theta} delta_max={delta_max} mode={mode} theta_m={theta_m} cue={cue}",
          flush=True)
    x = _x()
    ref = run_controller(lambda t, b: x[(t, b)], W.n_steps, W.n_blocks, theta, delta_max=delta_max, mode=mode,
                         theta_m=theta_m, cue=cue, keep_outputs=True)
    _assert_margin(W, ref, theta, mode, theta_m)
    _compare(W, ref, *_run_gpu(W, theta, delta_max, True, mode, theta_m, cue))


def test_controller_cases_cover_every_decision_and_deep_boundaries():
    """The cases above contain REUSE, REACTIVATE and COMPUTE blocks after step 0 and
    reactivation boundaries below block 0, so the parity test covers every executed mode."""
    x = _x()
    seen, depths = set(), set()
    for theta, dm in CASES:
        ref = run_controller(lambda t, b: x[(t, b)], W.n_steps, W.n_blocks, theta, delta_max=dm)
        seen |= set(ref.decisions[1:].ravel().tolist())
        for row in ref.decisions[1:]:
            depths |= {i for i, d in enumerate(row) if d == 1}
    assert seen == {0, 1, 2}
    assert max(depths) >= 2
