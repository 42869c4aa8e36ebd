"""End-to-end parity of the on-device Alg. 1 executor with the oracle controller.

Both run the same seeded trajectory (sweep recipe at reduced shapes, bf16
inputs): per-(step, block) decisions must be identical, and the executed
target outputs, recorded masses and cache ages must match the oracle's within
the bf16 bars. Thresholds are chosen so that no evaluated head-mean score lies
within 1e-3 of theta (a closer score may legitimately flip under rounding).
"""

import numpy as np
import pytest
import torch

from gpu_helpers import MASS_TOL, O_TOL, dev, host, max_abs
from oracle import run_controller
from paper_2609_32415_amd import synth

pytestmark = pytest.mark.gpu

W = synth.workload("sweep", heads=4, n_ref=160, n_tgt=192, n_blocks=6, n_steps=4, seed=99)


def _inputs():
    trajs = [synth.Trajectory(W, b, ref_sigma=lambda t, b=b: synth.sweep_ref_drift(b, W.n_blocks),
                              tgt_sigma=lambda t: synth.sweep_tgt_drift(t, W.n_steps)) for b in range(W.n_blocks)]
    return {(t, b): trajs[b].step_tensors(t) for t in range(W.n_steps) for b in range(W.n_blocks)}


X = None


def _x():
    global X
    if X is None:
        X = _inputs()
    return X


def _margin_ok(tr, theta, mode="product", theta_m=None):
    th = np.broadcast_to(np.asarray(theta, dtype=np.float64), (W.n_blocks,))
    score = {"product": tr.g_mean, "q_only": tr.d_mean, "mass_only": tr.m_mean, "and": tr.d_mean}[mode]
    mask = ~np.isnan(score)
    ok = np.all(np.abs(score - th[None, :])[mask] > 1e-3)
    if mode == "and":
        ok = ok and np.all(np.abs(tr.m_mean - theta_m)[~np.isnan(tr.m_mean)] > 1e-3)
    return ok


def _run_gpu(theta, delta_max=None, fused=True, mode="product", theta_m=None, cue="consecutive"):
    from paper_2609_32415_amd.controller import Controller

    x = _x()
    ctl = Controller(W.n_blocks, W.n_steps, W.batch, W.heads, W.n_ref, W.n_tgt, W.head_dim, theta,
                     delta_max=delta_max, device="cuda:0", fused=fused, mode=mode, theta_m=theta_m, cue=cue)
    outs, masses, ages = {}, {}, []
    for t in range(W.n_steps):
        xs = [{k: dev(v, "bf16") for k, v in x[(t, b)].items()} for b in range(W.n_blocks)]
        ctl.step(t, xs)
        torch.cuda.synchronize()
        for b in range(W.n_blocks):
            outs[(t, b)] = host(ctl.o_tgt[b])
            masses[(t, b)] = host(ctl.recorded_mass(b))
        ages.append(ctl.age.cpu().tolist())
    return ctl.decisions.cpu().numpy(), outs, masses, np.array(ages)


PER_BLOCK = (0.2, 0.2, 0.115, 0.115, 0.045, 0.045)
CASES = [(0.02, None), (0.058, None), (0.105, None), (0.115, None), (0.05, 2), (0.0, None), (1e9, None),
         (PER_BLOCK, None)]


@pytest.mark.parametrize("fused", [True, False], ids=["fused", "separate"])
@pytest.mark.parametrize("theta,delta_max", CASES, ids=lambda v: str(v))
def test_controller_matches_oracle(theta, delta_max, fused):
    print(f"controller theta={theta} delta_max={delta_max} fused={fused}", flush=True)
    x = _x()
    ref = run_controller(lambda t, b: x[(t, b)], W.n_steps, W.n_blocks, theta, delta_max=delta_max, keep_outputs=True)
    if not _margin_ok(ref, theta):
        pytest.skip("a head-mean score lies within 1e-3 of theta for this seed")
    dec, outs, masses, ages = _run_gpu(theta, delta_max, fused)
    assert dec.tolist() == ref.decisions.tolist()
    assert ages.tolist() == ref.ages.tolist()
    for (t, b), o in outs.items():
        assert max_abs(o, ref.outputs[(t, b)]["o_tgt"]) <= O_TOL["bf16"], (t, b)
        assert max_abs(masses[(t, b)], ref.outputs[(t, b)]["ref_mass"]) <= MASS_TOL["bf16"], (t, b)


# (theta, delta_max, gate mode, theta_m, target-side cue): the single-cue ablations, the
# two-threshold gate and the anchor-relative cue of the paper's ablation table.
VARIANTS = [
    (0.1, None, "q_only", None, "consecutive"),
    (0.3, None, "mass_only", None, "consecutive"),
    (0.2, None, "and", 0.4, "consecutive"),
    (0.105, None, "product", None, "anchor"),
    (0.115, 2, "product", None, "anchor"),
    (1e9, 3, "product", None, "consecutive"),  # fixed-interval refresh (every 3 steps)
]


@pytest.mark.parametrize("theta,delta_max,mode,theta_m,cue", VARIANTS, ids=lambda v: str(v))
def test_controller_variants_match_oracle(theta, delta_max, mode, theta_m, cue):
    print(f"controller variant theta={theta} delta_max={delta_max} mode={mode} theta_m={theta_m} cue={cue}",
          flush=True)
    x = _x()
    ref = run_controller(lambda t, b: x[(t, b)], W.n_steps, W.n_blocks, theta, delta_max=delta_max, mode=mode,
                         theta_m=theta_m, cue=cue, keep_outputs=True)
    if not _margin_ok(ref, theta, mode, theta_m):
        pytest.skip("a head-mean score lies within 1e-3 of theta for this seed")
    dec, outs, masses, ages = _run_gpu(theta, delta_max, True, mode, theta_m, cue)
    assert dec.tolist() == ref.decisions.tolist()
    assert ages.tolist() == ref.ages.tolist()
    for (t, b), o in outs.items():
        assert max_abs(o, ref.outputs[(t, b)]["o_tgt"]) <= O_TOL["bf16"], (t, b)
        assert max_abs(masses[(t, b)], ref.outputs[(t, b)]["ref_mass"]) <= MASS_TOL["bf16"], (t, b)


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
