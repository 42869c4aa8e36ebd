"""The controller's steps captured as HIP graphs reproduce the eager trajectory.

Every step of a small trajectory is captured once; the trajectory is then
replayed twice, with eager copies of fresh inputs and synchronisations between
the replays, and every replay's decisions, executed outputs, recorded masses
and cache ages must equal the eager controller's bit for bit (same kernels on
the same inputs), and match the oracle controller's decisions.
"""

import numpy as np
import pytest
import torch

from gpu_helpers import dev
from oracle import run_controller
from paper_2609_32415_amd import synth

pytestmark = pytest.mark.gpu

W = synth.workload("sweep", heads=4, n_ref=160, n_tgt=192, n_blocks=6, n_steps=4, seed=99)
THETA = 0.058


def _inputs():
    trajs = [synth.Trajectory(W, b, ref_sigma=lambda t, b=b: synth.sweep_ref_drift(b, W.n_blocks),
                              tgt_sigma=lambda t: synth.sweep_tgt_drift(t, W.n_steps)) for b in range(W.n_blocks)]
    return {(t, b): trajs[b].step_tensors(t) for t in range(W.n_steps) for b in range(W.n_blocks)}


def _controller():
    from paper_2609_32415_amd.controller import Controller

    return Controller(W.n_blocks, W.n_steps, W.batch, W.heads, W.n_ref, W.n_tgt, W.head_dim, THETA,
                      delta_max=3, device="cuda:0")


def _snapshot(ctl, mass_of):
    return ([o.clone() for o in ctl.o_tgt], [mass_of(b).clone() for b in range(W.n_blocks)], ctl.age.clone())


def test_graph_replays_equal_eager_trajectory():
    from paper_2609_32415_amd.controller import StepGraphs

    x = _inputs()
    xs = {k: {n: dev(v, "bf16") for n, v in d.items()} for k, d in x.items()}

    eager = _controller()
    ref = []
    for t in range(W.n_steps):
        eager.step(t, [xs[(t, b)] for b in range(W.n_blocks)])
        torch.cuda.synchronize()
        ref.append(_snapshot(eager, eager.recorded_mass))
    ref_dec = eager.decisions.clone()

    oracle = run_controller(lambda t, b: x[(t, b)], W.n_steps, W.n_blocks, THETA, delta_max=3)
    assert ref_dec.cpu().numpy().tolist() == oracle.decisions.tolist()

    ctl = _controller()
    graphs = StepGraphs(ctl, lambda: [{n: torch.empty_like(v) for n, v in xs[(0, b)].items()}
                                      for b in range(W.n_blocks)])
    for rep in range(2):
        ctl.decisions.fill_(-1)
        for t in range(W.n_steps):
            for b, buf in enumerate(graphs.inputs(t)):
                for n, v in buf.items():
                    v.copy_(xs[(t, b)][n])
            torch.cuda.synchronize()
            graphs.replay(t)
            torch.cuda.synchronize()
            outs, masses, age = _snapshot(ctl, lambda b: graphs.recorded_mass(t, b))
            r_outs, r_masses, r_age = ref[t]
            for b in range(W.n_blocks):
                assert torch.equal(outs[b], r_outs[b]), (rep, t, b)
                assert torch.equal(masses[b], r_masses[b]), (rep, t, b)
            assert torch.equal(age, r_age), (rep, t)
        assert torch.equal(ctl.decisions, ref_dec), rep
        # eager work on the same stream between replays
        torch.cuda.synchronize()
        assert float(torch.stack([o.float().abs().sum() for o in ctl.o_tgt]).sum()) > 0
