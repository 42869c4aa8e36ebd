"""Alg. 1 (monotone depth-adaptive reference reuse) over the library's kernels.

Per denoising step and block the executor enqueues, on the current stream and
without any host synchronisation:

  refadapt_q_change_gate  D of this block's target Q against the recorded one and
                       the head-mean D*M against theta_b, decision written on the
                       device (block 0 also does the step bookkeeping: step 0 and
                       the bounded-age refresh make every block of the step compute);
                       two launches (fused=False: refadapt_q_change + refadapt_gate, three)
  refadapt_joint_attn  RA_KV_DEVICE: REUSE -> target queries over the cached
                       reference K/V; REACTIVATE -> current target queries and the
                       cached reference queries over the cache (the boundary
                       restores the block's cached reference state);
                       COMPUTE -> all queries over fresh K/V
  refadapt_cache_commit  fresh reference K/V and Q -> cache and a_b <- t on COMPUTE

and records the block's target Q (by reference) and the per-query reference
mass of the attention it executed (ping-pong buffers) for the next step. The
decisions stay on the device until the caller reads them. With
cue="anchor" the Q-change is taken against the target Q of the block's last
COMPUTE step (copied on the device by a K-only commit), the paper's
Anchor-Q x Exposure ablation.

The block inputs are exogenous here: the caller supplies each block's fresh
Q/K/V per step (the diffusion transformer whose hidden states would produce
them is outside this library).

``run_sweep`` runs the controller sweep: 60 blocks x 8 steps at the
single-reference shapes, 3 x 3 threshold cells, against a full-fresh
trajectory through the same harness.
"""

from __future__ import annotations

import math

import torch

from . import ops, synth
from .ops import COMPUTE, REACTIVATE, REUSE


class Controller:
    """Device-resident controller state and per-block buffers of one trajectory."""

    def __init__(self, n_blocks, n_steps, batch, heads, n_ref, n_tgt, head_dim, theta, delta_max=None,
                 mode="product", theta_m=None, dtype=torch.bfloat16, device="cuda:0", eps=1e-8, fused=True,
                 cue="consecutive", sidecar=None):
        self.nb, self.n_steps = n_blocks, n_steps
        self.shape_r = (batch, heads, n_ref, head_dim)
        self.shape_t = (batch, heads, n_tgt, head_dim)
        self.mode, self.eps, self.device = mode, eps, device
        tq = torch.as_tensor(theta, dtype=torch.float64).reshape(-1).expand(n_blocks)
        if mode == "and":  # (theta_q, theta_m) pairs per block
            tm = torch.as_tensor(theta_m, dtype=torch.float64).reshape(-1).expand(n_blocks)
            th = torch.stack([tq, tm], 1).reshape(-1)
        else:
            th = tq
        self.theta = th.to(torch.float32).contiguous().to(device)
        self.state = ops.new_gate_state(device, delta_max or 0)
        self.k_cache = [torch.empty(self.shape_r, dtype=dtype, device=device) for _ in range(n_blocks)]
        self.v_cache = [torch.empty(self.shape_r, dtype=dtype, device=device) for _ in range(n_blocks)]
        # reference queries of each block's cached state: the boundary restores that state, so
        # its reference rows attend with them (Alg. 1 boundary branch)
        self.q_cache = [torch.empty(self.shape_r, dtype=dtype, device=device) for _ in range(n_blocks)]
        self.mass = [[torch.zeros((batch, heads, n_tgt), dtype=torch.float32, device=device) for _ in range(2)]
                     for _ in range(n_blocks)]
        self.parity = [0] * n_blocks
        self.q_prev = [None] * n_blocks
        if cue not in ("consecutive", "anchor"):
            raise ValueError(f"unknown cue {cue!r}")
        self.cue = cue
        # anchor cue: the target Q of each block's last COMPUTE step
        self.q_anchor = ([torch.empty(self.shape_t, dtype=dtype, device=device) for _ in range(n_blocks)]
                         if cue == "anchor" else None)
        self.age = torch.zeros(n_blocks, dtype=torch.int32, device=device)
        self.d = torch.zeros((n_blocks, batch, heads), dtype=torch.float32, device=device)
        self.decisions = torch.full((n_steps, n_blocks), -1, dtype=torch.int32, device=device)
        self.scores = torch.zeros((n_steps, n_blocks, 3), dtype=torch.float32, device=device)
        self.o_tgt = [torch.empty(self.shape_t, dtype=dtype, device=device) for _ in range(n_blocks)]
        self.o_ref = [torch.empty(self.shape_r, dtype=dtype, device=device) for _ in range(n_blocks)]
        q_like = torch.empty(self.shape_t, dtype=dtype, device=device)
        self.fused = fused
        self.ws = ops.q_change_gate_workspace(q_like) if fused else ops.q_change_workspace(q_like)
        self.attn_ws = ops.attn_workspace(q_like, n_ref, kvsrc="device")
        self.sidecar = sidecar

    def block(self, t, b, x, mark=None, clock_probe=None):
        """Enqueue Alg. 1's work for block ``b`` at step ``t`` on fresh inputs ``x``.

        ``mark(name)`` (optional) is called after each enqueued phase ("gate", "attn",
        "commit"), e.g. to record timing events; ``clock_probe`` is passed to the attention
        launch (see ``ops.joint_attn``)."""
        if self.cue == "anchor":
            q_prev = self.q_anchor[b] if t > 0 else x["q_tgt"]
        else:
            q_prev = self.q_prev[b] if self.q_prev[b] is not None else x["q_tgt"]
        dec = self.decisions[t, b:b + 1]
        if self.fused:
            ops.q_change_gate(x["q_tgt"], q_prev, self.mass[b][self.parity[b]], self.theta, self.state, b, t,
                              self.mode, self.eps, d_out=self.d[b], decision_out=dec, score_out=self.scores[t, b],
                              workspace=self.ws)
        else:
            ops.q_change(x["q_tgt"], q_prev, self.eps, out=self.d[b], workspace=self.ws)
            ops.gate(self.d[b], self.mass[b][self.parity[b]], self.theta, self.state, b, t, self.mode,
                     decision_out=dec, score_out=self.scores[t, b])
        if mark:
            mark("gate")
        nxt = 1 - self.parity[b]
        ops.joint_attn(
            x["q_tgt"], x["k_tgt"], x["v_tgt"], q_ref=x["q_ref"], k_ref=x["k_ref"], v_ref=x["v_ref"],
            k_cache=self.k_cache[b], v_cache=self.v_cache[b], q_cache=self.q_cache[b], kvsrc="device", decision=dec,
            o_tgt=self.o_tgt[b], o_ref=self.o_ref[b], ref_mass=self.mass[b][nxt], workspace=self.attn_ws,
            clock_probe=clock_probe,
        )
        if mark:
            mark("attn")
        if self.sidecar is not None:  # read-only probes; the block's cache still holds its anchor K/V
            self.sidecar.block(t, b, x, self)
        ops.cache_commit(x["k_ref"], x["v_ref"], self.k_cache[b], self.v_cache[b], decision=dec,
                         age=self.age[b:b + 1], step=t, q_ref=x["q_ref"], q_cache=self.q_cache[b])
        if self.cue == "anchor":
            ops.cache_commit(x["q_tgt"], None, self.q_anchor[b], None, decision=dec)
        if mark:
            mark("commit")
        self.q_prev[b] = x["q_tgt"]
        self.parity[b] = nxt

    def step(self, t, inputs):
        """All blocks of step ``t``; ``inputs[b]`` is block b's dict of fresh tensors."""
        for b in range(self.nb):
            self.block(t, b, inputs[b])

    def recorded_mass(self, b):
        """Per-query reference mass of block b's most recently executed attention."""
        return self.mass[b][self.parity[b]]


class Sidecar:
    """Diagnostics sidecar of one controller trajectory: read-only probes per block and step.

    Called by ``Controller.block`` after the block's attention and before its cache
    commit, so the block's cache still holds the reference K/V of its last COMPUTE
    step (the anchor a_b). Everything is enqueued on the current stream into the
    sidecar's own buffers and device logs ``[n_steps, n_blocks, B, H]`` (NaN where
    a quantity is undefined, e.g. drifts at step 0); nothing the controller reads
    or writes is touched, so its outputs are bitwise the same with or without it.

    Logged per (t, b, batch, head):
      e_kv, d_k, d_v  endpoint drift of the fresh reference K and V against the
                      cached anchor values and their mean E^KV (t >= 1)
      rho_k, rho_v    matched log-ratio of reference vs target consecutive drift
                      of K and of V (t >= 1)
      impact          I^KV of the executed target output against the full-fresh
                      target output of the same step
      m_fresh         exposure of the current target queries over fresh keys
      m_cached        same-step exposure with the cached (anchor) reference keys
                      (t >= 1)
      m_refq_tgt      mean mass of the reference queries on target keys
    ``adjacent_change()`` gives the per-block adjacent reference-mass change (in
    percentage points) of the logged fresh exposure.
    """

    def __init__(self, n_blocks, n_steps, batch, heads, n_ref, n_tgt, head_dim, dtype=torch.bfloat16,
                 device="cuda:0", eps=1e-8):
        self.eps = eps
        shape = (n_steps, n_blocks, batch, heads)
        nan = lambda: torch.full(shape, float("nan"), dtype=torch.float32, device=device)
        self.e_kv, self.d_k, self.d_v = nan(), nan(), nan()
        self.rho_k, self.rho_v = nan(), nan()
        self.impact, self.m_fresh, self.m_cached, self.m_refq_tgt = nan(), nan(), nan(), nan()
        sr, st = (batch, heads, n_ref, head_dim), (batch, heads, n_tgt, head_dim)
        self.o_fresh = torch.empty(st, dtype=dtype, device=device)
        self.o_ref_fresh = torch.empty(sr, dtype=dtype, device=device)
        self.o_cached = torch.empty(st, dtype=dtype, device=device)
        self.mass_fresh = torch.empty((batch, heads, n_tgt), dtype=torch.float32, device=device)
        self.mass_refq = torch.empty((batch, heads, n_ref), dtype=torch.float32, device=device)
        self.mass_cached = torch.empty((batch, heads, n_tgt), dtype=torch.float32, device=device)
        q_like = torch.empty(st, dtype=dtype, device=device)
        r_like = torch.empty(sr, dtype=dtype, device=device)
        self.ws_full = ops.attn_workspace(q_like, n_ref, qset="all", kvsrc="fresh")
        self.ws_cached = ops.attn_workspace(q_like, n_ref, qset="target", kvsrc="cache")
        self.ws_kv = ops.kv_drift_workspace(r_like)
        self.ws_ratio = ops.drift_log_ratio_workspace(r_like, q_like)
        self.ws_impact = ops.output_impact_workspace(q_like)
        self.prev = [None] * n_blocks

    def block(self, t, b, x, ctl):
        eps = self.eps
        # Full-fresh joint attention of the step: target and reference queries over fresh K/V.
        ops.joint_attn(x["q_tgt"], x["k_tgt"], x["v_tgt"], q_ref=x["q_ref"], k_ref=x["k_ref"], v_ref=x["v_ref"],
                       qset="all", kvsrc="fresh", o_tgt=self.o_fresh, o_ref=self.o_ref_fresh,
                       ref_mass=self.mass_fresh, ref_mass_refq=self.mass_refq, workspace=self.ws_full)
        ops.mass_mean(self.mass_fresh, out=self.m_fresh[t, b])
        ops.mass_mean(self.mass_refq, complement=True, out=self.m_refq_tgt[t, b])
        ops.output_impact(ctl.o_tgt[b], self.o_fresh, eps, out=self.impact[t, b], workspace=self.ws_impact)
        if t > 0:
            ops.kv_drift(x["k_ref"], ctl.k_cache[b], x["v_ref"], ctl.v_cache[b], eps, d_k=self.d_k[t, b],
                         d_v=self.d_v[t, b], e_kv=self.e_kv[t, b], workspace=self.ws_kv)
            ops.joint_attn(x["q_tgt"], x["k_tgt"], x["v_tgt"], k_cache=ctl.k_cache[b], v_cache=ctl.v_cache[b],
                           qset="target", kvsrc="cache", o_tgt=self.o_cached, ref_mass=self.mass_cached,
                           workspace=self.ws_cached)
            ops.mass_mean(self.mass_cached, out=self.m_cached[t, b])
            p = self.prev[b]
            ops.drift_log_ratio(x["k_ref"], p["k_ref"], x["k_tgt"], p["k_tgt"], eps, rho=self.rho_k[t, b],
                                workspace=self.ws_ratio)
            ops.drift_log_ratio(x["v_ref"], p["v_ref"], x["v_tgt"], p["v_tgt"], eps, rho=self.rho_v[t, b],
                                workspace=self.ws_ratio)
        self.prev[b] = {k: x[k] for k in ("k_ref", "v_ref", "k_tgt", "v_tgt")}

    def adjacent_change(self):
        """Per-block adjacent reference-mass change (percentage points) of the fresh exposure."""
        return ops.adjacent_mass_change(self.m_fresh)


class StepGraphs:
    """HIP graphs of every step of one controller trajectory.

    Step t is captured once, from the controller's own per-block enqueues, as a
    graph that reads its fresh inputs from static per-block buffers
    ``inputs(t)`` (two sets, alternating with the step's parity, so step t's
    recorded target Q is still in place when step t+1 reads it). Replaying
    graphs 0..n_steps-1 in order runs the trajectory again: step 0's gate
    bookkeeping re-initialises the device state, so a new trajectory needs no
    reset. Capture must happen before any eager step of ``ctl`` (the captured
    pointers follow its ping-pong state from step 0). ``make_inputs()`` returns
    one list of per-block dicts of device tensors; it is called twice.
    """

    def __init__(self, ctl, make_inputs):
        self.ctl = ctl
        self.bufs = [make_inputs(), make_inputs()]
        self.graphs = []
        self._parity = []  # per step: the mass buffer each block's graph writes
        torch.cuda.synchronize()
        for t in range(ctl.n_steps):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                ctl.step(t, self.bufs[t % 2])
            self.graphs.append(g)
            self._parity.append(list(ctl.parity))
        torch.cuda.synchronize()

    def inputs(self, t):
        """Static input buffers read by step t's graph (fill them before replay(t))."""
        return self.bufs[t % 2]

    def replay(self, t):
        self.graphs[t].replay()

    def recorded_mass(self, t, b):
        """Per-query reference mass that block b's attention records at step t."""
        return self.ctl.mass[b][self._parity[t][b]]


def _sweep_inputs(w, device):
    trajs = [synth.DeviceTrajectory(w, b, device, ref_sigma=(lambda t, b=b: synth.sweep_ref_drift(b, w.n_blocks)),
                                    tgt_sigma=(lambda t: synth.sweep_tgt_drift(t, w.n_steps)))
             for b in range(w.n_blocks)]
    return trajs


def time_launches(fn, reps=10, warm_ms=50.0):
    """Mean time (ms) of ``fn`` over ``reps`` back-to-back launches, after at least ``warm_ms`` of
    warm-up launches: after host-side work the GPU clock needs tens of milliseconds of load to
    come back up, and a short warm-up then times the ramp, not the kernel."""
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    fn()
    b.record()
    torch.cuda.synchronize()
    for _ in range(max(5, int(warm_ms / max(a.elapsed_time(b), 1e-3)))):
        fn()
    a.record()
    for _ in range(reps):
        fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps

def _timed_run(w, device, theta, delta_max, mode="product", theta_m=None, keep=None, cue="consecutive",
               sidecar=None):
    """One trajectory; returns (controller, per-step attention-path milliseconds)."""
    ctl = Controller(w.n_blocks, w.n_steps, w.batch, w.heads, w.n_ref, w.n_tgt, w.head_dim, theta,
                     delta_max=delta_max, mode=mode, theta_m=theta_m, device=device, cue=cue, sidecar=sidecar)
    trajs = _sweep_inputs(w, device)
    step_ms = []
    for t in range(w.n_steps):
        xs = [tr.step_tensors(t) for tr in trajs]
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        ctl.step(t, xs)
        e1.record()
        if keep is not None:
            keep(t, ctl, xs)
        torch.cuda.synchronize()
        step_ms.append(e0.elapsed_time(e1))
    return ctl, step_ms


def _cell(w, device, full_ms, theta, delta_max=None, mode="product", theta_m=None, cue="consecutive"):
    """One controller configuration: timed trajectory, then an untimed replay that
    measures the executed target output's relative change against full-fresh attention."""
    ctl, ms = _timed_run(w, device, theta, delta_max, mode, theta_m, cue=cue)
    dec = ctl.decisions.cpu()
    after0 = dec[1:]
    errs = []

    def keep(t, c, xs):  # untimed: relative change of executed vs full-fresh target output
        for b in range(w.n_blocks):
            x = xs[b]
            fresh = ops.joint_attn(x["q_tgt"], x["k_tgt"], x["v_tgt"], k_ref=x["k_ref"], v_ref=x["v_ref"],
                                   ref_mass=False).o_tgt.float()
            diff = (c.o_tgt[b].float() - fresh).flatten(2).norm(dim=-1)
            errs.append((diff / (fresh.flatten(2).norm(dim=-1) + 1e-8)).flatten())

    _timed_run(w, device, theta, delta_max, mode, theta_m, keep=keep, cue=cue)
    e = torch.cat(errs).cpu()
    return {
        "mode": mode, "cue": cue, "theta": theta, "theta_m": theta_m, "delta_max": delta_max,
        "reuse_fraction": round(float((after0 == REUSE).float().mean()), 4),
        "reuse_or_reactivate_fraction": round(float((after0 != COMPUTE).float().mean()), 4),
        "attn_path_ms": round(sum(ms), 3),
        "speedup_vs_full_fresh": round(full_ms / sum(ms), 3),
        "boundary_block_per_step": [next((i for i, x in enumerate(row) if x == REACTIVATE), None)
                                    for row in dec.tolist()],
        "decisions": dec.tolist(),
        "impact_mean": round(float(e.mean()), 5),
        "impact_p99": round(float(e.quantile(0.99)), 5),
        "impact_max": round(float(e.max()), 5),
    }


def adaptive_cell(device="cuda:0", w=None, theta_q=0.2, theta_m=0.4, log=None):
    """One depth-adaptive controller trajectory against its full-fresh trajectory.

    The sweep workload (60 blocks x 8 steps at the single-reference shapes) runs once with a
    refresh every step (every block computes: the full-fresh trajectory) and once under the
    product gate at theta_q * theta_m, through the same harness. Reports the attention-path
    times, the attention-time speedup of adaptive reuse, the reuse fractions over steps >= 1,
    the reactivation boundary of every step and how many steps put it at each depth, the
    relative change of the executed target output against full-fresh attention, and the
    all-reuse bound of the speedup."""
    w = w or synth.workload("sweep")
    _, base_ms = _timed_run(w, device, 0.0, delta_max=1)
    full_ms = sum(base_ms)
    c = _cell(w, device, full_ms, theta_q * theta_m)
    bnd = c["boundary_block_per_step"][1:]
    hist = {}
    for b in bnd:
        key = "none" if b is None else str(b)
        hist[key] = hist.get(key, 0) + 1
    res = {
        "workload": f"{w.n_blocks} blocks x {w.n_steps} steps, batch {w.batch}, {w.heads} heads, head_dim "
                    f"{w.head_dim}, n_ref {w.n_ref}, n_tgt {w.n_tgt} (sweep recipe: exposure rising with depth, "
                    f"target change decaying over the steps)",
        "theta_q": theta_q, "theta_m": theta_m, "theta": theta_q * theta_m,
        "full_fresh_attn_path_ms": round(full_ms, 3),
        "adaptive_attn_path_ms": c["attn_path_ms"],
        "attn_time_speedup": c["speedup_vs_full_fresh"],
        "max_speedup_bound": round(w.n_steps / (1 + (w.n_steps - 1) * w.n_tgt / (w.n_ref + w.n_tgt)), 3),
        "reuse_fraction": c["reuse_fraction"],
        "reuse_or_reactivate_fraction": c["reuse_or_reactivate_fraction"],
        "boundary_block_per_step": c["boundary_block_per_step"],
        "boundary_depth_histogram": hist,
        "impact_mean": c["impact_mean"], "impact_p99": c["impact_p99"], "impact_max": c["impact_max"],
    }
    if log:
        log(f"adaptive reuse: {res['attn_time_speedup']}x over full-fresh ({res['full_fresh_attn_path_ms']} ms -> "
            f"{res['adaptive_attn_path_ms']} ms), boundaries {res['boundary_block_per_step']}")
    return res


def _graph_timed_run(w, device, theta, delta_max):
    """As _timed_run, with every step replayed from a captured HIP graph."""
    ctl = Controller(w.n_blocks, w.n_steps, w.batch, w.heads, w.n_ref, w.n_tgt, w.head_dim, theta,
                     delta_max=delta_max, device=device)
    trajs = _sweep_inputs(w, device)
    shapes = {"q_tgt": ctl.shape_t, "k_tgt": ctl.shape_t, "v_tgt": ctl.shape_t,
              "q_ref": ctl.shape_r, "k_ref": ctl.shape_r, "v_ref": ctl.shape_r}
    graphs = StepGraphs(ctl, lambda: [{n: torch.empty(sh, dtype=torch.bfloat16, device=device)
                                       for n, sh in shapes.items()} for _ in range(w.n_blocks)])
    step_ms = []
    for t in range(w.n_steps):
        for b, buf in enumerate(graphs.inputs(t)):
            x = trajs[b].step_tensors(t)
            for n, v in buf.items():
                v.copy_(x[n])
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        graphs.replay(t)
        e1.record()
        torch.cuda.synchronize()
        step_ms.append(e0.elapsed_time(e1))
    return ctl, step_ms


def run_sweep(device="cuda:0", w=None, log=None, delta_max_cells=((0.2, 0.4, 2), (0.2, 0.4, 4)),
              graph_cells=((0.2, 0.4),), ablation_cells=((0.05, 0.1), (0.1, 0.2), (0.2, 0.4))):
    """The controller sweep (60 blocks x 8 steps, single-reference shapes).

    For each (theta_q, theta_m) cell the product gate runs with
    theta = theta_q * theta_m (one threshold on the head-mean D*M score) and no
    bounded-age refresh; ``delta_max_cells`` adds (theta_q, theta_m, delta_max)
    cells with the refresh of Alg. 1 every delta_max steps. Reports the reuse
    fraction over steps >= 1, the attention-path time (Q-change, gate, attention
    and commit kernels of every block) against a full-fresh trajectory through
    the same harness (bounded-age refresh every step), and the relative change of
    the executed target output against full-fresh attention. ``ablation_cells``
    runs the cue ablation at those (theta_q, theta_m) pairs: Q-change alone
    (theta_q), mass alone (theta_m), both with separate thresholds, the product,
    the anchor-relative Q-change times mass, and a fixed refresh every 3 steps.
    ``graph_cells`` repeats cells (and the full-fresh baseline) as HIP-graph
    replays of captured steps.
    """
    w = w or synth.workload("sweep")
    base, base_ms = _timed_run(w, device, 0.0, delta_max=1)
    full_ms = sum(base_ms)
    if log:
        log(f"sweep: full-fresh trajectory {full_ms:.1f} ms")
    cells = []
    grid = [(tq, tm, None) for tq in w.theta_q for tm in w.theta_m] + list(delta_max_cells)
    for tq, tm, dmax in grid:
        c = _cell(w, device, full_ms, tq * tm, delta_max=dmax)
        c.update(theta_q=tq, theta_m=tm)
        cells.append(c)
        if log:
            log(f"sweep: cell theta_q={tq} theta_m={tm} delta_max={dmax}: {c['attn_path_ms']} ms, "
                f"speedup {c['speedup_vs_full_fresh']}, reuse {c['reuse_fraction']}")

    # Cue ablation (the paper's ablation table, on these synthetics): each target-side or
    # exposure cue alone, both with separate thresholds, the anchor-relative target-Q cue
    # times exposure, and a fixed refresh every 3 steps.
    ablation = []
    if ablation_cells:
        for tq, tm in ablation_cells:
            for mode, theta, theta_m, cue in (("q_only", tq, None, "consecutive"),
                                              ("mass_only", tm, None, "consecutive"),
                                              ("and", tq, tm, "consecutive"),
                                              ("product", tq * tm, None, "consecutive"),
                                              ("product", tq * tm, None, "anchor")):
                c = _cell(w, device, full_ms, theta, None, mode, theta_m, cue)
                c.update(theta_q=tq, theta_m=tm)
                c.pop("decisions")
                ablation.append(c)
                if log:
                    log(f"sweep: ablation {mode}/{cue} theta_q={tq} theta_m={tm}: speedup "
                        f"{c['speedup_vs_full_fresh']}, reuse {c['reuse_fraction']}, impact {c['impact_mean']}")
        c = _cell(w, device, full_ms, math.inf, delta_max=3)
        c.update(theta_q=None, theta_m=None, mode="fixed_interval_3")
        c.pop("decisions")
        ablation.append(c)
        if log:
            log(f"sweep: ablation fixed refresh every 3 steps: speedup {c['speedup_vs_full_fresh']}, "
                f"impact {c['impact_mean']}")

    # The same trajectories replayed from captured HIP graphs (one graph per step).
    g_base, g_base_ms = _graph_timed_run(w, device, 0.0, delta_max=1)
    graph = {"full_fresh_attn_path_ms": round(sum(g_base_ms), 3), "cells": []}
    for tq, tm in graph_cells:
        g_ctl, g_ms = _graph_timed_run(w, device, tq * tm, delta_max=None)
        eager = next(c for c in cells if c["theta_q"] == tq and c["theta_m"] == tm and c["delta_max"] is None)
        same = bool(torch.equal(g_ctl.decisions.cpu(), torch.tensor(eager["decisions"], dtype=torch.int32)))
        graph["cells"].append({"theta_q": tq, "theta_m": tm, "attn_path_ms": round(sum(g_ms), 3),
                               "speedup_vs_full_fresh": round(sum(g_base_ms) / sum(g_ms), 3),
                               "decisions_equal_eager": same})
    if log:
        log(f"sweep: graph replay full-fresh {graph['full_fresh_attn_path_ms']} ms, cells {graph['cells']}")
    for c in cells:
        c.pop("decisions")
    return {
        "ablation": ablation,
        "graph_replay": graph,
        "workload": f"{w.n_blocks} blocks x {w.n_steps} steps, batch {w.batch}, {w.heads} heads, head_dim "
                    f"{w.head_dim}, n_ref {w.n_ref}, n_tgt {w.n_tgt}",
        "full_fresh_attn_path_ms": round(full_ms, 3),
        "max_speedup_bound": round(w.n_steps / (1 + (w.n_steps - 1) * w.n_tgt / (w.n_ref + w.n_tgt)), 3),
        "cells": cells,
    }


def _ranks(a):
    """Ranks (average ranks for ties) of a 1-D array, for Spearman's correlation."""
    import numpy as np

    order = np.argsort(a, kind="stable")
    r = np.empty(len(a), dtype=np.float64)
    r[order] = np.arange(len(a), dtype=np.float64)
    vals, inv, counts = np.unique(a, return_inverse=True, return_counts=True)
    sums = np.bincount(inv, weights=r)
    return (sums / counts)[inv]


def run_diagnostics(device="cuda:0", w=None, theta=(0.1, 0.2), log=None):
    """The diagnostics sidecar over one controller trajectory (sweep shapes, 60 blocks x 8 steps).

    Runs the trajectory twice on the same inputs, without and with the sidecar,
    and checks that every controller output and state tensor is bitwise the same
    (the probe reads only). Summaries of the sidecar's device logs (steps >= 1
    where a quantity needs an anchor or a previous step):
      endpoint drift E^KV of the reference K/V against each block's anchor;
      median of the matched drift log-ratio rho for K and V and the ratio 10^rho;
      I^KV of the executed target output against full-fresh attention;
      per-block adjacent reference-mass change (percentage points);
      same-step cached vs fresh exposure: mean absolute difference, Pearson and
      Spearman correlation over (step, block, head) cells;
      mean mass of reference queries on target keys vs of target queries on
      reference keys, and the share of (step, block) cells where the first is larger;
      the sidecar's share of the attention-path time.
    Correlation statistics are computed on the host from the logged arrays.
    """
    import numpy as np

    w = w or synth.workload("sweep")
    th = theta[0] * theta[1]
    ctl_off, ms_off = _timed_run(w, device, th, None)
    final_off = [x.clone() for x in ctl_off.o_tgt + ctl_off.o_ref + [m for p in ctl_off.mass for m in p]
                 + ctl_off.k_cache + ctl_off.v_cache + [ctl_off.d, ctl_off.age, ctl_off.decisions, ctl_off.scores]]
    del ctl_off
    torch.cuda.empty_cache()
    sc = Sidecar(w.n_blocks, w.n_steps, w.batch, w.heads, w.n_ref, w.n_tgt, w.head_dim, device=device)
    ctl_on, ms_on = _timed_run(w, device, th, None, sidecar=sc)
    final_on = ctl_on.o_tgt + ctl_on.o_ref + [m for p in ctl_on.mass for m in p] + ctl_on.k_cache + \
        ctl_on.v_cache + [ctl_on.d, ctl_on.age, ctl_on.decisions, ctl_on.scores]
    identical = all(torch.equal(a, b) for a, b in zip(final_off, final_on))
    dbar = sc.adjacent_change()
    torch.cuda.synchronize()
    h = lambda x: x.cpu().numpy().astype(np.float64)
    e_kv, rho_k, rho_v, imp = h(sc.e_kv)[1:], h(sc.rho_k)[1:], h(sc.rho_v)[1:], h(sc.impact)
    m_f, m_c, m_q = h(sc.m_fresh), h(sc.m_cached)[1:], h(sc.m_refq_tgt)
    dec = ctl_on.decisions.cpu().numpy()
    reused = dec == REUSE
    mf1 = m_f[1:].reshape(-1)
    mc1 = m_c.reshape(-1)
    pearson = float(np.corrcoef(mf1, mc1)[0, 1])
    spearman = float(np.corrcoef(_ranks(mf1), _ranks(mc1))[0, 1])
    cell_refq = m_q.mean(axis=(2, 3))  # [T, n_blocks] head means
    cell_tgt = m_f.mean(axis=(2, 3))
    res = {
        "theta": list(theta),
        "bit_identical_with_sidecar": bool(identical),
        "attn_path_ms": round(sum(ms_off), 3),
        "attn_path_with_sidecar_ms": round(sum(ms_on), 3),
        "sidecar_share_of_path_time": round(sum(ms_on) / sum(ms_off) - 1.0, 3),
        "endpoint_e_kv": {"mean": round(float(e_kv.mean()), 5), "median": round(float(np.median(e_kv)), 5),
                          "max": round(float(e_kv.max()), 5)},
        "rho_k_median": round(float(np.median(rho_k)), 4),
        "rho_v_median": round(float(np.median(rho_v)), 4),
        "ref_over_tgt_drift_median_k": round(float(10 ** np.median(rho_k)), 4),
        "ref_over_tgt_drift_median_v": round(float(10 ** np.median(rho_v)), 4),
        "impact_mean": round(float(imp.mean()), 5),
        "impact_reused_blocks_mean": round(float(imp[reused].mean()), 5) if reused.any() else None,
        "impact_p99": round(float(np.quantile(imp, 0.99)), 5),
        "adjacent_ref_change_pp": {"max": round(float(h(dbar).max()), 4), "mean": round(float(h(dbar).mean()), 4)},
        "cached_vs_fresh_exposure": {"mad": round(float(np.abs(mf1 - mc1).mean()), 6),
                                     "pearson": round(pearson, 5), "spearman": round(spearman, 5)},
        "target_to_ref_mass_mean": round(float(m_f.mean()), 5),
        "ref_query_to_target_mass_mean": round(float(m_q.mean()), 5),
        "refq_gt_tgt_cell_share": round(float((cell_refq > cell_tgt).mean()), 4),
        "reuse_fraction": round(float(reused[1:].mean()), 4),
    }
    if log:
        log(f"diagnostics: bit-identical {identical}, sidecar +{100 * res['sidecar_share_of_path_time']:.0f}% of "
            f"path time, median 10^rho K {res['ref_over_tgt_drift_median_k']} V {res['ref_over_tgt_drift_median_v']}, "
            f"cached-vs-fresh MAD {res['cached_vs_fresh_exposure']['mad']}")
    return res


def run_ref_count_sweep(device="cuda:0", counts=(1, 2, 3, 4, 5, 6, 7, 8), n_blocks=8, theta_q=0.2, theta_m=0.4,
                        log=None):
    """Attention-time speedup against the number of reference images.

    For k reference images of 4096 tokens plus 256 text tokens (N_R = 4096 k + 256,
    N_Y = 4096, single-reference per-image shapes): the per-block attention times of a
    computed block (all queries, fresh K/V) and a reused block (target queries, cached
    K/V); the all-reuse bound of an n_steps trajectory, n t_full / (t_full + (n - 1)
    t_reuse); and a measured controller trajectory (n_blocks blocks x 8 steps, sweep
    recipe, product gate at theta_q * theta_m) against its full-fresh trajectory.
    """
    rows = []
    for k in counts:
        w = synth.workload("sweep", n_ref=4096 * k + 256, n_blocks=n_blocks)
        tr = synth.DeviceTrajectory(w, 0, device)
        tr.step_tensors(0)
        x = tr.step_tensors(1)
        del tr
        ws_r = ops.attn_workspace(x["q_tgt"], w.n_ref, "target", "cache")
        ws_f = ops.attn_workspace(x["q_tgt"], w.n_ref, "all", "fresh")

        t_reuse = time_launches(lambda: ops.joint_attn(x["q_tgt"], x["k_tgt"], x["v_tgt"], k_cache=x["k_ref"],
                                               v_cache=x["v_ref"], n_ref=w.n_ref, kvsrc="cache", workspace=ws_r))
        t_full = time_launches(lambda: ops.joint_attn(x["q_tgt"], x["k_tgt"], x["v_tgt"], q_ref=x["q_ref"], k_ref=x["k_ref"],
                                              v_ref=x["v_ref"], qset="all", workspace=ws_f))
        del x, ws_r, ws_f
        _, base_ms = _timed_run(w, device, 0.0, delta_max=1)
        ctl, ms = _timed_run(w, device, theta_q * theta_m, delta_max=None)
        after0 = ctl.decisions.cpu()[1:]
        n = w.n_steps
        rows.append({
            "ref_images": k, "n_ref": w.n_ref, "n_tgt": w.n_tgt,
            "full_block_ms": round(t_full, 4), "reuse_block_ms": round(t_reuse, 4),
            "block_speedup": round(t_full / t_reuse, 3),
            "all_reuse_bound": round(n * t_full / (t_full + (n - 1) * t_reuse), 3),
            "trajectory_full_fresh_ms": round(sum(base_ms), 3), "trajectory_adaptive_ms": round(sum(ms), 3),
            "trajectory_speedup": round(sum(base_ms) / sum(ms), 3),
            "reuse_fraction": round(float((after0 == REUSE).float().mean()), 4),
        })
        if log:
            log(f"ref-count sweep: {k} references: block {rows[-1]['block_speedup']}x, trajectory "
                f"{rows[-1]['trajectory_speedup']}x (reuse {rows[-1]['reuse_fraction']})")
        torch.cuda.empty_cache()
    return {"workload": f"{n_blocks} blocks x 8 steps, batch 1, 24 heads, head_dim 128, N_R = 4096 k + 256, "
                        f"N_Y 4096; product gate at theta_q {theta_q} x theta_m {theta_m}",
            "rows": rows}



def run_reference_segments(device="cuda:0", weights=(1.0, 0.5, 0.0, 1.0), sizes=(4096, 4096, 4096, 256),
                           cache_noise=0.02, log=None):
    """Per-reference exposure and individual stale impact at the multi-reference shapes.

    The reference rows are three 4096-token images and 256 text tokens. The synthetic key
    bias is weighted per segment (``weights``), so the references draw different attention,
    and the cache is the fresh reference K/V plus one drift step of ``cache_noise``. For
    each reference s: its exposure (per-head mean over target queries of the mass on its
    keys, from one fresh launch with per-segment masses) and its individual stale impact
    I^KV_s (target output with only segment s read from the cache against the fresh output,
    through ``RA_KV_SEGMENTS``); then the all-stale impact, the same table with the first
    two images swapped (the references are not interchangeable: values follow the image,
    not its position), and the time of a segment launch against a plain cached launch.
    """
    import numpy as np

    w = synth.workload("multi_ref", n_ref=sum(sizes), ref_segments=tuple(sizes), ref_bias_weights=tuple(weights),
                       cache_noise=cache_noise)
    x = synth.block_inputs(w)
    cache = synth.stale_cache(w, x)
    ends = np.cumsum(sizes).tolist()
    n_seg = len(sizes)

    def table(order):
        perm = np.concatenate([np.arange(e - n, e) for n, e in ((sizes[i], ends[i]) for i in order)])
        bf = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device).to(torch.bfloat16)
        t = {k: bf(v) for k, v in x.items() if k.endswith("_tgt")}
        kr, vr = bf(x["k_ref"][:, :, perm]), bf(x["v_ref"][:, :, perm])
        kc, vc = bf(cache["k_ref"][:, :, perm]), bf(cache["v_ref"][:, :, perm])
        ends_p = np.cumsum([sizes[i] for i in order]).tolist()
        fresh = ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], k_ref=kr, v_ref=vr, seg_end=ends_p, seg_mass=True,
                               workspace=False)
        expo = [ops.mass_mean(fresh.seg_mass[..., s].contiguous()) for s in range(n_seg)]
        imp = []
        for s in range(n_seg):
            o_s = ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], k_ref=kr, v_ref=vr, k_cache=kc, v_cache=vc,
                                 kvsrc="segments", seg_end=ends_p, seg_cache=[i == s for i in range(n_seg)]).o_tgt
            imp.append(ops.output_impact(o_s, fresh.o_tgt))
        o_all = ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], k_cache=kc, v_cache=vc, kvsrc="cache",
                               workspace=False).o_tgt
        imp_all = ops.output_impact(o_all, fresh.o_tgt)
        torch.cuda.synchronize()
        # rows in the original image order
        back = np.argsort(order)
        ex = np.array([float(e.mean()) for e in expo])[back]
        im = np.array([float(i.mean()) for i in imp])[back]
        return ex, im, float(imp_all.mean()), (t, kr, vr, kc, vc, ends_p)

    ex, im, im_all, (t, kr, vr, kc, vc, ends_p) = table(list(range(n_seg)))
    order2 = [1, 0] + list(range(2, n_seg))
    ex2, im2, im_all2, _ = table(order2)

    timed = lambda fn: time_launches(fn, reps=20)
    mixed = [i % 2 == 0 for i in range(n_seg)]
    ws = ops.attn_workspace(t["q_tgt"], sum(sizes), "target", "cache")
    ms_cache = timed(lambda: ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], k_cache=kc, v_cache=vc,
                                            kvsrc="cache", workspace=ws))
    ms_cache_whole = timed(lambda: ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], k_cache=kc, v_cache=vc,
                                                  kvsrc="cache", workspace=False))
    ms_seg = timed(lambda: ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], k_ref=kr, v_ref=vr, k_cache=kc,
                                          v_cache=vc, kvsrc="segments", seg_end=ends_p, seg_cache=mixed))
    ms_seg_cached = timed(lambda: ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], k_ref=kr, v_ref=vr, k_cache=kc,
                                                 v_cache=vc, kvsrc="segments", seg_end=ends_p,
                                                 seg_cache=[True] * n_seg))
    ws_sm = ops.attn_workspace(t["q_tgt"], sum(sizes), "target", "segments", n_seg_mass=n_seg)
    ms_seg_mass = timed(lambda: ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], k_ref=kr, v_ref=vr, k_cache=kc,
                                               v_cache=vc, kvsrc="segments", seg_end=ends_p, seg_cache=mixed,
                                               seg_mass=True, workspace=ws_sm))
    ms_seg_mass_whole = timed(lambda: ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], k_ref=kr, v_ref=vr,
                                                     k_cache=kc, v_cache=vc, kvsrc="segments", seg_end=ends_p,
                                                     seg_cache=mixed, seg_mass=True, workspace=False))
    names = [f"image{i}" for i in range(n_seg - 1)] + ["text"]
    res = {
        "segments": names, "sizes": list(sizes), "bias_weights": list(weights), "cache_noise": cache_noise,
        "exposure": [round(v, 5) for v in ex], "individual_stale_impact": [round(v, 6) for v in im],
        "all_stale_impact": round(im_all, 6), "exposure_sum": round(float(ex.sum()), 5),
        "swapped_first_two": {"exposure": [round(v, 5) for v in ex2],
                              "individual_stale_impact": [round(v, 6) for v in im2],
                              "all_stale_impact": round(im_all2, 6)},
        "reuse_attention_ms": {"cache_split": round(ms_cache, 4), "cache_whole": round(ms_cache_whole, 4),
                               "segments_all_cached": round(ms_seg_cached, 4),
                               "segments_mixed": round(ms_seg, 4), "segments_mixed_with_seg_mass": round(ms_seg_mass, 4),
                               "segments_mixed_with_seg_mass_whole": round(ms_seg_mass_whole, 4)},
    }
    if log:
        log(f"reference segments: exposure {res['exposure']}, individual stale impact "
            f"{res['individual_stale_impact']}, all-stale {res['all_stale_impact']}")
    return res
