"""fp64 CPU oracle for the RefAdapt-DiT hot path.

TEST INFRASTRUCTURE ONLY. This package is a plain, slow, obviously correct
implementation of what the GPU path computes, written from the definitions in
the paper (RefAdapt-DiT, arxiv 2609.32415). Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it. The product (the HIP library and its binding) never imports, calls
or links anything here, and this package imports nothing from the product.

Contents
--------
joint_attention      Sec. 3.3 fresh/stale-output equations + Sec. 3.2
                     directional-exposure equation: softmax attention of a
                     query set over [K_R; K_Y], per-query reference mass and
                     split log-sum-exp statistics (vectorised, fp64).
joint_attention_loops
                     The same definition as explicit Python loops, for tiny
                     shapes (brute force).
segment_masses       Per-query mass on each reference segment (the exposure of
                     one reference image).
q_change             Sec. 3.1 consecutive-drift equation applied to post-RoPE
                     target queries per head (Sec. 4, runtime cues).
head_exposure        Sec. 3.2 directional-exposure equation: mean over target
                     queries of the per-query reference mass.
gate                 Sec. 4 factorized-risk and depth-cutoff equations, with
                     the head aggregate of App. A.2 and the per-block branch
                     of Alg. 1.
run_controller       Alg. 1 (monotone depth-adaptive reference reuse) as a
                     step/block loop over exogenous synthetic inputs.
local_impact         Sec. 3.3 local-impact equation (relative Frobenius
                     change of the target attention output).
diagnostics          The analysis quantities of Secs. 3.1-3.3 and App. A.2:
                     consecutive and endpoint drift of K/V, the joint K/V
                     endpoint scalar, the matched drift log-ratio, per-head
                     exposure (fresh or with anchor reference keys), the
                     reference-query mass on target keys and the adjacent
                     reference-mass change.

Every function is pinned by ``-m "not gpu"`` tests in ``tests/`` against
closed forms, library routines (torch SDPA in fp64, scipy logsumexp),
hand-derived fixtures under ``tests/golden/`` and structural statements of
the paper.
"""

from .joint_attention import joint_attention, joint_attention_loops, segment_masses
from .stats import q_change, head_exposure, gate, GateResult, REUSE, REACTIVATE, COMPUTE
from .controller import run_controller, local_impact, ControllerTrace
from . import diagnostics

__all__ = [
    "joint_attention",
    "joint_attention_loops",
    "segment_masses",
    "q_change",
    "head_exposure",
    "gate",
    "GateResult",
    "REUSE",
    "REACTIVATE",
    "COMPUTE",
    "run_controller",
    "local_impact",
    "ControllerTrace",
    "diagnostics",
]
