"""Torch-tensor wrappers over the C ABI (device memory and streams only).

Each function checks devices, dtypes and layouts, allocates outputs with
torch (caching allocator) when the caller does not pass them, and calls the
C entry point of the same role on ``torch.cuda.current_stream()``. No torch
compute op runs on these paths; a tensor that is not on a GPU is an error.
"""

from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import Optional

import torch

from . import _lib as L

_DTYPES = {torch.bfloat16: L.RA_BF16, torch.float32: L.RA_F32}
_QSET = {"target": L.RA_Q_TARGET, "all": L.RA_Q_ALL}
_KVSRC = {"fresh": L.RA_KV_FRESH, "cache": L.RA_KV_CACHE, "device": L.RA_KV_DEVICE, "segments": L.RA_KV_SEGMENTS}
_GATE = {"product": L.RA_GATE_PRODUCT, "q_only": L.RA_GATE_Q_ONLY, "mass_only": L.RA_GATE_MASS_ONLY, "and": L.RA_GATE_AND}

REUSE, REACTIVATE, COMPUTE = L.RA_REUSE, L.RA_REACTIVATE, L.RA_COMPUTE


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _on_gpu(name, t):
    if t is not None and not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor (the HIP library is the only implementation)")


def _view(name, t, dtype=None, shape=None):
    if t is None:
        return L.ra_tensor()
    _on_gpu(name, t)
    if t.dim() != 4:
        raise ValueError(f"{name} must be [B, H, S, d], got {tuple(t.shape)}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)} != {tuple(shape)}")
    if t.numel() == 0:  # an empty segment is never read: pass a null view
        return L.ra_tensor()
    if t.stride(-1) != 1:
        raise ValueError(f"{name}: the head dimension must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype} differs from {dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)} != {tuple(shape)}")
    return L.ra_tensor(t.data_ptr(), t.stride(0), t.stride(1), t.stride(2))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _probe_ptr(t):
    _on_gpu("clock_probe", t)
    if t.dtype != torch.int64 or t.numel() != 2 or not t.is_contiguous():
        raise ValueError("clock_probe must be a contiguous int64 device tensor of 2 elements")
    return t.data_ptr()


@dataclass
class AttnOut:
    o_tgt: torch.Tensor
    o_ref: Optional[torch.Tensor]
    ref_mass: Optional[torch.Tensor]
    lse: Optional[torch.Tensor]
    ref_mass_refq: Optional[torch.Tensor]
    seg_mass: Optional[torch.Tensor] = None


def joint_attn(
    q_tgt,
    k_tgt,
    v_tgt,
    *,
    q_ref=None,
    k_ref=None,
    v_ref=None,
    k_cache=None,
    v_cache=None,
    q_cache=None,
    qset="target",
    kvsrc="fresh",
    decision=None,
    scale=None,
    n_ref=None,
    o_tgt=None,
    o_ref=None,
    ref_mass=True,
    lse=False,
    ref_mass_refq=False,
    workspace=None,
    seg_end=None,
    seg_cache=None,
    seg_mass=False,
    clock_probe=None,
):
    """Joint attention over [K_R; K_Y] through ``refadapt_joint_attn``.

    ``ref_mass``/``lse``/``ref_mass_refq`` may be booleans (allocate when True)
    or preallocated fp32 tensors. ``workspace``: None allocates the key-split
    workspace the library asks for (torch caching allocator), False runs
    without key splits, a uint8 device tensor is used as given (see
    ``attn_workspace``). Returns an ``AttnOut``.

    ``clock_probe``: an int64 device tensor of 2 elements that the bf16 kernel adds its
    workgroups' shader-clock cycles and 100 MHz reference ticks to (mean clock = 100 MHz x
    [0] / [1]); None disables it.

    ``q_cache``: reference queries of the cached state; reference queries that attend
    over the cached K/V (``kvsrc="cache"`` with ``qset="all"``, or REACTIVATE under
    ``kvsrc="device"``) read them instead of ``q_ref``.

    Reference segments (bf16): ``seg_end`` lists each segment's end row in R
    (multiples of 64 except the last, which is n_ref). With ``kvsrc="segments"``
    ``seg_cache`` (one bool per segment) picks the cached K/V for a segment, else
    the fresh K/V. ``seg_mass`` (bool or preallocated fp32 ``[B, H, n_tgt, n_seg]``)
    returns each target query's mass per segment in ``AttnOut.seg_mass``.
    """
    B, H, n_tgt, D = q_tgt.shape
    dt = q_tgt.dtype
    if dt not in _DTYPES:
        raise ValueError(f"unsupported dtype {dt}")
    if n_ref is None:
        src = next((t for t in (k_ref, k_cache, q_ref) if t is not None), None)
        n_ref = 0 if src is None else src.shape[2]
    dev = q_tgt.device
    device_mode = kvsrc == "device"
    ref_queries = (device_mode or qset == "all") and n_ref > 0
    if o_tgt is None:
        o_tgt = torch.empty((B, H, n_tgt, D), dtype=dt, device=dev)
    if ref_queries and o_ref is None:
        o_ref = torch.empty((B, H, n_ref, D), dtype=dt, device=dev)

    def _opt(flag, shape):
        if flag is True:
            return torch.empty(shape, dtype=torch.float32, device=dev)
        if flag is False or flag is None:
            return None
        if flag.dtype != torch.float32 or not flag.is_contiguous() or tuple(flag.shape) != shape:
            raise ValueError(f"output buffer must be contiguous fp32 of shape {shape}")
        return flag

    mass_t = _opt(ref_mass, (B, H, n_tgt))
    lse_t = _opt(lse, (B, H, n_tgt, 2))
    mrq_t = _opt(ref_mass_refq, (B, H, n_ref)) if n_ref > 0 else None
    n_seg = 0 if seg_end is None else len(seg_end)
    if (kvsrc == "segments" or seg_mass is not False) and not 1 <= n_seg <= L.RA_MAX_SEG:
        raise ValueError(f"seg_end must list 1..{L.RA_MAX_SEG} segment ends")
    smass_t = _opt(seg_mass, (B, H, n_tgt, n_seg)) if n_seg else None
    cache_bits = 0
    if kvsrc == "segments":
        if seg_cache is None or len(seg_cache) != n_seg:
            raise ValueError("seg_cache must give one flag per segment")
        cache_bits = sum(1 << i for i, c in enumerate(seg_cache) if c)
    if decision is not None:
        _on_gpu("decision", decision)
        if decision.dtype != torch.int32:
            raise ValueError("decision must be an int32 device tensor")

    shp_t = (B, H, n_tgt, D)
    shp_r = (B, H, n_ref, D)
    desc = L.ra_attn_desc(B, H, D, n_ref, n_tgt, _DTYPES[dt], float(scale or 0.0), _QSET[qset], _KVSRC[kvsrc])
    if workspace is None:
        if smass_t is not None:
            nbytes = L.refadapt_joint_attn_seg_workspace_size(desc, n_seg)
        else:
            nbytes = L.refadapt_joint_attn_workspace_size(desc)
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev) if nbytes else False
    if workspace is False:
        ws_ptr, ws_bytes = None, 0
    else:
        _on_gpu("workspace", workspace)
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    args = L.ra_attn_args(
        q_tgt=_view("q_tgt", q_tgt, dt, shp_t),
        k_tgt=_view("k_tgt", k_tgt, dt, shp_t),
        v_tgt=_view("v_tgt", v_tgt, dt, shp_t),
        q_ref=_view("q_ref", q_ref, dt, shp_r),
        k_ref=_view("k_ref", k_ref, dt, shp_r),
        v_ref=_view("v_ref", v_ref, dt, shp_r),
        k_cache=_view("k_cache", k_cache, dt, shp_r),
        v_cache=_view("v_cache", v_cache, dt, shp_r),
        decision=None if decision is None else decision.data_ptr(),
        o_tgt=_view("o_tgt", o_tgt, dt, shp_t),
        o_ref=_view("o_ref", o_ref, dt, shp_r),
        ref_mass=None if mass_t is None else mass_t.data_ptr(),
        lse_tgt=None if lse_t is None else lse_t.data_ptr(),
        ref_mass_refq=None if mrq_t is None else mrq_t.data_ptr(),
        workspace=ws_ptr,
        workspace_bytes=ws_bytes,
        n_seg=n_seg,
        seg_end=(ctypes.c_int32 * L.RA_MAX_SEG)(*(list(seg_end or []) + [0] * (L.RA_MAX_SEG - n_seg))),
        seg_cache=cache_bits,
        seg_mass=None if smass_t is None else smass_t.data_ptr(),
        q_cache=_view("q_cache", q_cache, dt, shp_r),
        clock_probe=None if clock_probe is None else _probe_ptr(clock_probe),
    )
    L.refadapt_joint_attn(desc, args, _stream())
    return AttnOut(o_tgt, o_ref if ref_queries else None, mass_t, lse_t, mrq_t, smass_t)


def attn_workspace(q_tgt, n_ref, qset="target", kvsrc="fresh", n_seg_mass=0):
    """Preallocated key-split workspace for ``joint_attn`` calls of this shape on
    ``q_tgt``'s device (False when the library would not split); ``n_seg_mass``
    segments with ``seg_mass`` need the larger segment workspace."""
    B, H, n_tgt, D = q_tgt.shape
    desc = L.ra_attn_desc(B, H, D, n_ref, n_tgt, _DTYPES[q_tgt.dtype], 0.0, _QSET[qset], _KVSRC[kvsrc])
    with torch.cuda.device(q_tgt.device):
        if n_seg_mass:
            nbytes = L.refadapt_joint_attn_seg_workspace_size(desc, n_seg_mass)
        else:
            nbytes = L.refadapt_joint_attn_workspace_size(desc)
    return torch.empty(nbytes, dtype=torch.uint8, device=q_tgt.device) if nbytes else False


def q_change_workspace(q_tgt):
    B, H, n, D = q_tgt.shape
    nbytes = L.refadapt_q_change_workspace_size(B, H, n, D)
    return torch.empty(max(nbytes, 8), dtype=torch.uint8, device=q_tgt.device)


def q_change(q_cur, q_prev, eps=1e-8, out=None, workspace=None):
    """D[b, h] = ||Q_cur - Q_prev||_F / (||Q_prev||_F + eps) through ``refadapt_q_change``."""
    B, H, n, D = q_cur.shape
    dt = q_cur.dtype
    if dt not in _DTYPES:
        raise ValueError(f"unsupported dtype {dt}")
    if out is None:
        out = torch.empty((B, H), dtype=torch.float32, device=q_cur.device)
    if workspace is None:
        workspace = q_change_workspace(q_cur)
    _on_gpu("out", out)
    _on_gpu("workspace", workspace)
    L.refadapt_q_change(
        B, H, n, D, _DTYPES[dt],
        _view("q_cur", q_cur, dt), _view("q_prev", q_prev, dt, q_cur.shape),
        float(eps), _ptr(out), _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(),
    )
    return out


def new_gate_state(device, delta_max=0):
    """Device-resident ra_gate_state {reactivated, a_full, delta_max, step} (int32[4])."""
    return torch.tensor([0, 0, int(delta_max or 0), 0], dtype=torch.int32, device=device)


def gate(d_cur, mass_prev, theta, state, block, step, mode="product", decision_out=None, score_out=None):
    """One block's decision through ``refadapt_gate``; returns (decision int32[1], scores fp32[3])."""
    B, H = d_cur.shape
    n_tgt = mass_prev.shape[-1]
    dev = d_cur.device
    for name, t in (("d_cur", d_cur), ("mass_prev", mass_prev), ("theta", theta), ("state", state)):
        _on_gpu(name, t)
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if tuple(mass_prev.shape) != (B, H, n_tgt) or mass_prev.dtype != torch.float32 or d_cur.dtype != torch.float32:
        raise ValueError("d_cur must be fp32 [B, H] and mass_prev fp32 [B, H, n_tgt]")
    if theta.dtype != torch.float32 or state.dtype != torch.int32 or state.numel() != 4:
        raise ValueError("theta must be fp32 and state int32[4]")
    need = 2 * (block + 1) if mode == "and" else block + 1
    if theta.numel() < need:
        raise ValueError(f"theta has {theta.numel()} entries; block {block} needs {need}")
    if decision_out is None:
        decision_out = torch.empty(1, dtype=torch.int32, device=dev)
    if score_out is None:
        score_out = torch.empty(3, dtype=torch.float32, device=dev)
    L.refadapt_gate(
        B, H, n_tgt, int(block), int(step), _GATE[mode],
        _ptr(d_cur), _ptr(mass_prev), _ptr(theta), _ptr(state), _ptr(decision_out), _ptr(score_out), _stream(),
    )
    return decision_out, score_out


def q_change_gate_workspace(q_tgt):
    """Workspace of ``q_change_gate`` for Q of this shape."""
    B, H, n, D = q_tgt.shape
    nbytes = L.refadapt_q_change_gate_workspace_size(B, H, n, D)
    return torch.empty(nbytes, dtype=torch.uint8, device=q_tgt.device)


def q_change_gate(q_cur, q_prev, mass_prev, theta, state, block, step, mode="product", eps=1e-8, d_out=None,
                  decision_out=None, score_out=None, workspace=None):
    """Q-change and gate fused through ``refadapt_q_change_gate``;
    returns (d [B, H], decision int32[1], scores fp32[3])."""
    B, H, n, D = q_cur.shape
    dt = q_cur.dtype
    if dt not in _DTYPES:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q_cur.device
    for name, t in (("mass_prev", mass_prev), ("theta", theta), ("state", state)):
        _on_gpu(name, t)
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if tuple(mass_prev.shape) != (B, H, n) or mass_prev.dtype != torch.float32:
        raise ValueError("mass_prev must be fp32 [B, H, n_tgt]")
    if theta.dtype != torch.float32 or state.dtype != torch.int32 or state.numel() != 4:
        raise ValueError("theta must be fp32 and state int32[4]")
    need = 2 * (block + 1) if mode == "and" else block + 1
    if theta.numel() < need:
        raise ValueError(f"theta has {theta.numel()} entries; block {block} needs {need}")
    if d_out is None:
        d_out = torch.empty((B, H), dtype=torch.float32, device=dev)
    if decision_out is None:
        decision_out = torch.empty(1, dtype=torch.int32, device=dev)
    if score_out is None:
        score_out = torch.empty(3, dtype=torch.float32, device=dev)
    if workspace is None:
        workspace = q_change_gate_workspace(q_cur)
    for name, t in (("d_out", d_out), ("decision_out", decision_out), ("score_out", score_out),
                    ("workspace", workspace)):
        _on_gpu(name, t)
    L.refadapt_q_change_gate(
        B, H, n, D, _DTYPES[dt], _view("q_cur", q_cur, dt), _view("q_prev", q_prev, dt, q_cur.shape), float(eps),
        int(block), int(step), _GATE[mode], _ptr(mass_prev), _ptr(theta), _ptr(state), _ptr(d_out),
        _ptr(decision_out), _ptr(score_out), _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(),
    )
    return d_out, decision_out, score_out


def q_change_gate_noalloc(q_cur, q_prev, mass_prev, theta, state, block, step, mode="product", eps=1e-8, d_out=None,
                          decision_out=None, score_out=None):
    """``q_change_gate`` through ``refadapt_q_change_gate_noalloc``: no workspace, the library's
    fixed device scratch holds the partial sums (for callers that cannot allocate; calls that
    overlap on one device race). Outputs must be passed in to allocate nothing here either."""
    B, H, n, D = q_cur.shape
    dt = q_cur.dtype
    if dt not in _DTYPES:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q_cur.device
    if d_out is None:
        d_out = torch.empty((B, H), dtype=torch.float32, device=dev)
    if decision_out is None:
        decision_out = torch.empty(1, dtype=torch.int32, device=dev)
    if score_out is None:
        score_out = torch.empty(3, dtype=torch.float32, device=dev)
    for name, t in (("mass_prev", mass_prev), ("theta", theta), ("state", state), ("d_out", d_out),
                    ("decision_out", decision_out), ("score_out", score_out)):
        _on_gpu(name, t)
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if tuple(mass_prev.shape) != (B, H, n) or mass_prev.dtype != torch.float32:
        raise ValueError("mass_prev must be fp32 [B, H, n_tgt]")
    if theta.dtype != torch.float32 or state.dtype != torch.int32 or state.numel() != 4:
        raise ValueError("theta must be fp32 and state int32[4]")
    need = 2 * (block + 1) if mode == "and" else block + 1
    if theta.numel() < need:
        raise ValueError(f"theta has {theta.numel()} entries; block {block} needs {need}")
    L.refadapt_q_change_gate_noalloc(
        B, H, n, D, _DTYPES[dt], _view("q_cur", q_cur, dt), _view("q_prev", q_prev, dt, q_cur.shape), float(eps),
        int(block), int(step), _GATE[mode], _ptr(mass_prev), _ptr(theta), _ptr(state), _ptr(d_out),
        _ptr(decision_out), _ptr(score_out), _stream(),
    )
    return d_out, decision_out, score_out


def cache_commit(k_ref, v_ref, k_cache, v_cache, decision=None, age=None, step=0, q_ref=None, q_cache=None):
    """Copy the fresh reference K, V (and Q when ``q_ref``/``q_cache`` are given) into the
    cache when ``decision`` is COMPUTE (or None); with ``v_ref`` and ``v_cache`` None only K
    is copied. One launch copies every pair."""
    B, H, n_ref, D = k_ref.shape
    dt = k_ref.dtype
    if (v_ref is None) != (v_cache is None):
        raise ValueError("v_ref and v_cache are both given or both None")
    if (q_ref is None) != (q_cache is None):
        raise ValueError("q_ref and q_cache are both given or both None")
    for name, t in (("decision", decision), ("age", age)):
        _on_gpu(name, t)
        if t is not None and t.dtype != torch.int32:
            raise ValueError(f"{name} must be int32")
    L.refadapt_cache_commit(
        B, H, n_ref, D, _DTYPES[dt],
        _view("k_ref", k_ref, dt), _view("v_ref", v_ref, dt, k_ref.shape), _view("q_ref", q_ref, dt, k_ref.shape),
        _view("k_cache", k_cache, dt, k_ref.shape), _view("v_cache", v_cache, dt, k_ref.shape),
        _view("q_cache", q_cache, dt, k_ref.shape),
        _ptr(decision), _ptr(age), int(step), _stream(),
    )


# ---- diagnostics sidecar (read-only probes of the controlled path)


def _f32_out(name, t, shape, device):
    if t is None:
        return torch.empty(shape, dtype=torch.float32, device=device)
    _on_gpu(name, t)
    if t.dtype != torch.float32 or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous float32 tensor of shape {tuple(shape)}")
    return t


def _nbytes(t):
    return t.numel() * t.element_size()


def kv_drift_workspace(k):
    B, H, n, D = k.shape
    return torch.empty(max(L.refadapt_kv_drift_workspace_size(B, H, n, D), 8), dtype=torch.uint8, device=k.device)


def kv_drift(k_cur, k_base, v_cur, v_base, eps=1e-8, d_k=None, d_v=None, e_kv=None, workspace=None):
    """Relative change of reference K and V against a base (the anchor for the endpoint
    drift) and their joint scalar E^KV = (D_K + D_V) / 2, per (b, h), through
    ``refadapt_kv_drift``. Returns (d_k, d_v, e_kv)."""
    B, H, n, D = k_cur.shape
    dt = k_cur.dtype
    if dt not in _DTYPES:
        raise ValueError(f"unsupported dtype {dt}")
    d_k = _f32_out("d_k", d_k, (B, H), k_cur.device)
    d_v = _f32_out("d_v", d_v, (B, H), k_cur.device)
    e_kv = _f32_out("e_kv", e_kv, (B, H), k_cur.device)
    workspace = kv_drift_workspace(k_cur) if workspace is None else workspace
    _on_gpu("workspace", workspace)
    L.refadapt_kv_drift(
        B, H, n, D, _DTYPES[dt], _view("k_cur", k_cur, dt), _view("k_base", k_base, dt, k_cur.shape),
        _view("v_cur", v_cur, dt, k_cur.shape), _view("v_base", v_base, dt, k_cur.shape), float(eps),
        _ptr(d_k), _ptr(d_v), _ptr(e_kv), _ptr(workspace), _nbytes(workspace), _stream(),
    )
    return d_k, d_v, e_kv


def drift_log_ratio_workspace(z_ref, z_tgt):
    B, H, n_ref, D = z_ref.shape
    nbytes = L.refadapt_drift_log_ratio_workspace_size(B, H, n_ref, z_tgt.shape[2], D)
    return torch.empty(max(nbytes, 8), dtype=torch.uint8, device=z_ref.device)


def drift_log_ratio(z_ref_cur, z_ref_prev, z_tgt_cur, z_tgt_prev, eps=1e-8, d_ref=None, d_tgt=None, rho=None,
                    workspace=None):
    """Consecutive drift of the reference and target slices of one of K, V and the matched
    log-ratio rho = log10((D_ref + eps) / (D_tgt + eps)) per (b, h), through
    ``refadapt_drift_log_ratio``. Returns (d_ref, d_tgt, rho)."""
    B, H, n_ref, D = z_ref_cur.shape
    n_tgt = z_tgt_cur.shape[2]
    dt = z_ref_cur.dtype
    if dt not in _DTYPES:
        raise ValueError(f"unsupported dtype {dt}")
    d_ref = _f32_out("d_ref", d_ref, (B, H), z_ref_cur.device)
    d_tgt = _f32_out("d_tgt", d_tgt, (B, H), z_ref_cur.device)
    rho = _f32_out("rho", rho, (B, H), z_ref_cur.device)
    workspace = drift_log_ratio_workspace(z_ref_cur, z_tgt_cur) if workspace is None else workspace
    _on_gpu("workspace", workspace)
    L.refadapt_drift_log_ratio(
        B, H, n_ref, n_tgt, D, _DTYPES[dt], _view("z_ref_cur", z_ref_cur, dt),
        _view("z_ref_prev", z_ref_prev, dt, z_ref_cur.shape), _view("z_tgt_cur", z_tgt_cur, dt, (B, H, n_tgt, D)),
        _view("z_tgt_prev", z_tgt_prev, dt, (B, H, n_tgt, D)), float(eps), _ptr(d_ref), _ptr(d_tgt), _ptr(rho),
        _ptr(workspace), _nbytes(workspace), _stream(),
    )
    return d_ref, d_tgt, rho


def output_impact_workspace(o):
    B, H, n, D = o.shape
    return torch.empty(max(L.refadapt_output_impact_workspace_size(B, H, n, D), 8), dtype=torch.uint8,
                       device=o.device)


def output_impact(o_stale, o_fresh, eps=1e-8, out=None, workspace=None):
    """I^KV[b, h] = ||O_stale - O_fresh||_F / (||O_fresh||_F + eps) through ``refadapt_output_impact``."""
    B, H, n, D = o_stale.shape
    dt = o_stale.dtype
    if dt not in _DTYPES:
        raise ValueError(f"unsupported dtype {dt}")
    out = _f32_out("out", out, (B, H), o_stale.device)
    workspace = output_impact_workspace(o_stale) if workspace is None else workspace
    _on_gpu("workspace", workspace)
    L.refadapt_output_impact(
        B, H, n, D, _DTYPES[dt], _view("o_stale", o_stale, dt), _view("o_fresh", o_fresh, dt, o_stale.shape),
        float(eps), _ptr(out), _ptr(workspace), _nbytes(workspace), _stream(),
    )
    return out


def mass_mean(mass, complement=False, out=None):
    """Per-(b, h) mean over rows of a [B, H, n] per-query mass (or of 1 - mass) through
    ``refadapt_mass_mean``."""
    _on_gpu("mass", mass)
    if mass.dim() != 3 or mass.dtype != torch.float32 or not mass.is_contiguous():
        raise ValueError("mass must be a contiguous float32 [B, H, n] tensor")
    B, H, n = mass.shape
    out = _f32_out("out", out, (B, H), mass.device)
    L.refadapt_mass_mean(B, H, n, _ptr(mass), int(bool(complement)), _ptr(out), _stream())
    return out


def adjacent_mass_change(mass_log, out=None):
    """Per block, 100 / (T - 1) * sum_t |Mbar_t - Mbar_{t-1}| (percentage points) from a
    [T, n_blocks, ...] log of per-head mass means, through ``refadapt_adjacent_mass_change``."""
    _on_gpu("mass_log", mass_log)
    if mass_log.dim() < 2 or mass_log.dtype != torch.float32 or not mass_log.is_contiguous():
        raise ValueError("mass_log must be a contiguous float32 [T, n_blocks, ...] tensor")
    T, nb = mass_log.shape[0], mass_log.shape[1]
    bh = mass_log[0, 0].numel()
    out = _f32_out("out", out, (nb,), mass_log.device)
    L.refadapt_adjacent_mass_change(T, nb, bh, _ptr(mass_log), _ptr(out), _stream())
    return out


def mfma_rate_probe(kind, operands, steps, workgroups=None, sink=None, clock_probe=None):
    """Runs ``refadapt_mfma_rate_probe`` (``kind`` "dense" or "mix") on the current stream and
    returns the sink. ``operands``: a device tensor of at least ``RA_PROBE_OPERAND_BYTES``
    bytes of bf16 values; ``workgroups`` defaults to the device's CU count (one per CU);
    FLOP = workgroups * 8 * steps * 32 * 32768."""
    _on_gpu("operands", operands)
    if operands.numel() * operands.element_size() < L.RA_PROBE_OPERAND_BYTES:
        raise ValueError(f"operands must hold at least {L.RA_PROBE_OPERAND_BYTES} bytes")
    if workgroups is None:
        workgroups = torch.cuda.get_device_properties(operands.device).multi_processor_count
    if sink is None:
        sink = torch.empty(workgroups * 512, dtype=torch.float32, device=operands.device)
    _on_gpu("sink", sink)
    if sink.dtype != torch.float32 or sink.numel() < workgroups * 512:
        raise ValueError("sink must be a float32 tensor of at least workgroups * 512 elements")
    probe = None if clock_probe is None else _ptr(clock_probe)
    L.refadapt_mfma_rate_probe({"dense": L.RA_PROBE_DENSE, "mix": L.RA_PROBE_MIX}[kind], int(workgroups), int(steps),
                               _ptr(operands), _ptr(sink), probe, _stream())
    return sink
