"""Seeded synthetic workloads for the joint-attention hot path.

This module only draws inputs: random normal Q/K/V, the key-bias construction
that spreads each target query's reference mass, and random-walk drift across
denoising steps. It contains none of the method's arithmetic, so both the GPU
path and the fp64 oracle can consume its output.

Every tensor is drawn in fp32 with numpy's PCG64, then rounded once to the run
dtype (round-to-nearest-even to bf16 for bf16 workloads), so the values handed
to the GPU and to the oracle are identical. Sub-seeds are derived from
(workload seed, block, step, tensor role) through numpy's SeedSequence.

Workloads (the paper's models and benchmarks are not available, so these
shapes stand in for them: single- and multi-reference image editing, a
video-editing shape, and a controller sweep):

* ``tiny``        fp32, B1 H2 d64, 256 reference + 256 target tokens,
                  4 steps x 4 blocks, reference drift 0.01, target drift 0.3.
* ``single_ref``  bf16, B1 H24 d128, 4096 target, 4096 + 256 text reference.
* ``multi_ref``   bf16, B1 H24 d128, 4096 target, 3x4096 + 256 text reference.
* ``video``       bf16, B1 H24 d128, 16384 target + 16384 reference
                  (8 frames x 2048), reference drift 0.005, target drift 0.2.
* ``sweep``       bf16, ``single_ref`` shapes, 60 blocks x 8 steps, per-block
                  reference drift schedule and decaying target drift.

Key bias (bf16 workloads): per head h a random unit direction u_h is drawn;
every reference key gets +0.5*sqrt(d)*u_h, and each target query's component
along u_h is set to +1 in a seeded 30 % of target rows and to -lambda_h in
the rest (lambda_h = 6h/(H-1)). With the 1/sqrt(d) softmax scale this adds
+0.5 or -0.5*lambda_h to that query's reference logits, so per-query reference
mass spans about 0.05-0.65. In ``sweep`` lambda follows a depth profile: 6 at
block 0 falling linearly to 0 at the deepest block, plus a seeded per-(block,
head) offset uniform in [-1.5, 1.5], clipped to [0, 6]; the head-mean exposure
then rises from about 0.24 to 0.5 with depth, so the head-mean score crosses a
threshold at a depth that moves as the target change decays over the steps.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field, replace

import numpy as np

ROLE_IDS = {"q_ref": 0, "k_ref": 1, "v_ref": 2, "q_tgt": 3, "k_tgt": 4, "v_tgt": 5, "bias": 6, "cache": 7, "rows": 8}
ROLES = ("q_ref", "k_ref", "v_ref", "q_tgt", "k_tgt", "v_tgt")


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str  # "f32" or "bf16"
    batch: int
    heads: int
    head_dim: int
    n_ref: int  # reference segment length (reference image tokens + text tokens)
    n_tgt: int
    seed: int
    n_steps: int = 1
    n_blocks: int = 1
    ref_drift: float = 0.0  # std of the per-step reference K/V random-walk increment
    tgt_drift: float = 0.0  # std of the per-step target Q/K/V random-walk increment
    key_bias: bool = False
    cache_noise: float = 0.0  # std of the perturbation that makes a stale cache differ from fresh
    theta_q: tuple = ()
    theta_m: tuple = ()
    # Optional reference segments (row counts, e.g. reference images then text) and a weight
    # per segment on the key bias, so that the segments draw different attention.
    ref_segments: tuple = ()
    ref_bias_weights: tuple = ()
    meta: dict = field(default_factory=dict, compare=False, hash=False)

    @property
    def n_total(self):
        return self.n_ref + self.n_tgt


WORKLOADS = {
    "tiny": Workload(
        "tiny", "f32", 1, 2, 64, 256, 256, 1234, n_steps=4, n_blocks=4,
        ref_drift=0.01, tgt_drift=0.3, theta_q=(0.1,), theta_m=(0.2,),
    ),
    "single_ref": Workload(
        "single_ref", "bf16", 1, 24, 128, 4096 + 256, 4096, 1234,
        key_bias=True, cache_noise=0.01, meta={"n_ref_img": 4096, "n_text": 256},
    ),
    "multi_ref": Workload(
        "multi_ref", "bf16", 1, 24, 128, 3 * 4096 + 256, 4096, 1234,
        key_bias=True, cache_noise=0.01, meta={"n_ref_img": 3 * 4096, "n_text": 256},
    ),
    "video": Workload(
        "video", "bf16", 1, 24, 128, 16384, 16384, 42, n_steps=2,
        ref_drift=0.005, tgt_drift=0.2, key_bias=True, cache_noise=0.005,
        meta={"frames": 8, "tokens_per_frame": 2048},
    ),
    "sweep": Workload(
        "sweep", "bf16", 1, 24, 128, 4096 + 256, 4096, 1234, n_steps=8, n_blocks=60,
        key_bias=True, theta_q=(0.05, 0.1, 0.2), theta_m=(0.1, 0.2, 0.4),
    ),
}


def workload(name, **overrides):
    """A named workload, optionally with fields replaced (e.g. smaller shapes)."""
    w = WORKLOADS[name]
    return replace(w, **overrides) if overrides else w


def _rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(k) for k in key])))


def round_to_dtype(x, dtype):
    """Round fp32 values to the run dtype and return them as fp32 (exactly representable)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "f32":
        return x
    if dtype != "bf16":
        raise ValueError(dtype)
    u = x.view(np.uint32)
    # Round to nearest even on the top 16 bits (finite inputs cannot carry past bit 31).
    u = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return u.view(np.float32)


def _normal(rng, shape):
    return rng.standard_normal(shape, dtype=np.float32)


def sweep_ref_drift(block, n_blocks=60):
    """Per-block reference drift of the sweep: 0.02 at block 0, linear down to
    0.002 at the middle block, then linear up to 0.03 at the deepest block."""
    mid = n_blocks // 2
    if block <= mid:
        return 0.02 + (0.002 - 0.02) * block / mid
    return 0.002 + (0.03 - 0.002) * (block - mid) / (n_blocks - 1 - mid)


def sweep_tgt_drift(step, n_steps=8):
    """Per-step target drift of the sweep: 0.3 at step 1, linear down to 0.05 at the last step."""
    if step <= 0:
        return 0.0
    if n_steps <= 2:
        return 0.3
    return 0.3 + (0.05 - 0.3) * (step - 1) / (n_steps - 2)


LAMBDA_JITTER = 1.5  # per-head spread of the sweep's key-bias depth profile


def sweep_lambda_mean(block, n_blocks):
    """Depth profile of the sweep's key bias: 6 at block 0, linear down to 0 at the
    deepest block, so a target query's reference logits (and the head-mean exposure)
    rise with depth."""
    return 6.0 * (1.0 - block / (n_blocks - 1)) if n_blocks > 1 else 3.0


def _lambda(w, block, h):
    if w.name == "sweep":
        jit = _rng(w.seed, block, 0, ROLE_IDS["bias"], 1000 + h).uniform(-LAMBDA_JITTER, LAMBDA_JITTER)
        return float(min(6.0, max(0.0, sweep_lambda_mean(block, w.n_blocks) + jit)))
    return 6.0 * h / (w.heads - 1) if w.heads > 1 else 0.0


def _apply_key_bias(w, block, t):
    """Bias reference keys along a per-head unit direction and set each target
    query's component along it (see the module docstring)."""
    d = w.head_dim
    rng = _rng(w.seed, block, 0, ROLE_IDS["bias"])
    u = _normal(rng, (w.batch, w.heads, d)).astype(np.float64)
    u /= np.linalg.norm(u, axis=-1, keepdims=True)
    shared = _rng(w.seed, block, 0, ROLE_IDS["rows"]).random((w.batch, w.heads, w.n_tgt)) < 0.3
    lam = np.array([_lambda(w, block, h) for h in range(w.heads)])
    target_comp = np.where(shared, 1.0, -lam[None, :, None])  # [B, H, n_tgt]
    uq = u[:, :, None, :].astype(np.float32)
    k_bias = (0.5 * math.sqrt(d) * u[:, :, None, :]).astype(np.float32)
    if w.ref_bias_weights:  # per-segment weights on the bias (rows of R in segment order)
        if len(w.ref_bias_weights) != len(w.ref_segments) or sum(w.ref_segments) != w.n_ref:
            raise ValueError("ref_bias_weights needs one weight per segment of ref_segments summing to n_ref")
        wt = np.repeat(np.asarray(w.ref_bias_weights, dtype=np.float32), w.ref_segments)
        k_bias = k_bias * wt[None, None, :, None]
    t["k_ref"] += k_bias
    q = t["q_tgt"]
    cur = np.einsum("bhnd,bhd->bhn", q, u.astype(np.float32))
    q += (target_comp.astype(np.float32) - cur)[..., None] * uq


def base_tensors(w, block=0):
    """Fresh fp32 Q/K/V of one block at step 0 (before rounding to the run dtype)."""
    B, H, d = w.batch, w.heads, w.head_dim
    t = {}
    for role in ROLES:
        n = w.n_ref if role.endswith("_ref") else w.n_tgt
        t[role] = _normal(_rng(w.seed, block, 0, ROLE_IDS[role]), (B, H, n, d))
    if w.key_bias:
        _apply_key_bias(w, block, t)
    return t


def drift_increment(w, block, step, role, sigma):
    """Random-walk increment sigma * N(0, 1) for one tensor role at ``step``."""
    n = w.n_ref if role.endswith("_ref") else w.n_tgt
    rng = _rng(w.seed, block, step, ROLE_IDS[role])
    return sigma * _normal(rng, (w.batch, w.heads, n, w.head_dim))


class Trajectory:
    """Fresh tensors of one block across denoising steps (a seeded random walk).

    ``step_tensors(t)`` must be called with t = 0, 1, 2, ... in order; it
    returns the run-dtype-rounded tensors (as fp32 numpy arrays) of step t.
    Reference Q/K/V drift with the reference sigma and target Q/K/V with the
    target sigma (the target rows are the actively generated ones).
    """

    def __init__(self, w, block=0, ref_sigma=None, tgt_sigma=None):
        self.w, self.block = w, block
        self.ref_sigma = ref_sigma if ref_sigma is not None else (lambda t: w.ref_drift)
        self.tgt_sigma = tgt_sigma if tgt_sigma is not None else (lambda t: w.tgt_drift)
        self._state = None
        self._t = -1

    def step_tensors(self, t):
        if t != self._t + 1:
            raise ValueError("steps must be visited in order")
        if t == 0:
            self._state = base_tensors(self.w, self.block)
        else:
            for role in ROLES:
                sig = self.ref_sigma(t) if role.endswith("_ref") else self.tgt_sigma(t)
                if sig:
                    self._state[role] = self._state[role] + drift_increment(self.w, self.block, t, role, sig)
        self._t = t
        return {k: round_to_dtype(v, self.w.dtype) for k, v in self._state.items()}


def block_inputs(w, block=0):
    """Step-0 tensors of one block, rounded to the run dtype."""
    t = base_tensors(w, block)
    return {k: round_to_dtype(v, w.dtype) for k, v in t.items()}


def stale_cache(w, fresh, block=0):
    """A reference K/V cache that differs from ``fresh`` by one drift step of
    std ``w.cache_noise`` (so that a wrong source pointer fails parity)."""
    out = {}
    for i, role in enumerate(("k_ref", "v_ref")):
        rng = _rng(w.seed, block, 0, ROLE_IDS["cache"], i)
        noise = w.cache_noise * _normal(rng, fresh[role].shape)
        out[role] = round_to_dtype(fresh[role] + noise, w.dtype)
    return out


def sample_rows(n, count, seed, include_edges=True):
    """Sorted, distinct row indices for sampled-row parity checks; always
    includes the first and last rows when ``include_edges``."""
    count = min(count, n)
    rng = _rng(seed, 0, 0, ROLE_IDS["rows"], 7)
    idx = set(rng.choice(n, size=count, replace=False).tolist())
    if include_edges and n > 0:
        idx.update({0, n - 1})
    return np.array(sorted(idx), dtype=np.int64)


class DeviceTrajectory:
    """The same recipe as ``Trajectory`` drawn on a GPU with torch's generator.

    Used where host generation would be too slow (the 60-block sweep holds
    about 9 GB of base tensors): base Q/K/V ~ N(0, 1), the key-bias
    construction, then a random walk with per-step sigmas. Values are rounded
    to the run dtype. Seeded per (workload seed, block); not bit-identical to
    the numpy generator.
    """

    def __init__(self, w, block, device, ref_sigma=None, tgt_sigma=None):
        import torch

        self.torch = torch
        self.w, self.block, self.device = w, block, device
        self.ref_sigma = ref_sigma if ref_sigma is not None else (lambda t: w.ref_drift)
        self.tgt_sigma = tgt_sigma if tgt_sigma is not None else (lambda t: w.tgt_drift)
        self.gen = torch.Generator(device=device)
        self.gen.manual_seed(int(w.seed) * 1_000_003 + int(block))
        self._state = None
        self._t = -1

    def _randn(self, n):
        w = self.w
        return self.torch.randn((w.batch, w.heads, n, w.head_dim), generator=self.gen, device=self.device)

    def step_tensors(self, t):
        torch, w = self.torch, self.w
        if t != self._t + 1:
            raise ValueError("steps must be visited in order")
        if t == 0:
            st = {r: self._randn(w.n_ref if r.endswith("_ref") else w.n_tgt) for r in ROLES}
            if w.key_bias:
                u = torch.randn((w.batch, w.heads, w.head_dim), generator=self.gen, device=self.device)
                u = u / u.norm(dim=-1, keepdim=True)
                st["k_ref"] += 0.5 * math.sqrt(w.head_dim) * u[:, :, None, :]
                shared = torch.rand((w.batch, w.heads, w.n_tgt), generator=self.gen, device=self.device) < 0.3
                lam = torch.tensor([_lambda(w, self.block, h) for h in range(w.heads)], device=self.device)
                comp = torch.where(shared, torch.ones_like(shared, dtype=torch.float32), -lam[None, :, None])
                cur = torch.einsum("bhnd,bhd->bhn", st["q_tgt"], u)
                st["q_tgt"] += (comp - cur)[..., None] * u[:, :, None, :]
            self._state = st
        else:
            for role in ROLES:
                sig = self.ref_sigma(t) if role.endswith("_ref") else self.tgt_sigma(t)
                if sig:
                    n = w.n_ref if role.endswith("_ref") else w.n_tgt
                    self._state[role].add_(self._randn(n), alpha=sig)
        self._t = t
        dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        return {k: v.to(dt) for k, v in self._state.items()}
