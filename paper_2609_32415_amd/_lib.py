"""ctypes binding of librefadapt.so (the C ABI declared in include/refadapt.h).

Argument marshalling only: every function here forwards to the exported C
symbol of the same name. The library is loaded from this package directory;
if it is missing the import fails loudly (there is no fallback path).
"""

from __future__ import annotations

import ctypes
import os

# torch must be imported before the library is loaded: torch ships its own HIP
# runtime (SONAME libamdhip64.so.7) and requests it as "libamdhip64.so"; loaded
# first, it also satisfies this library's libamdhip64.so.7 dependency, so the
# process holds ONE HIP runtime. Loading this library first would pull in a
# second runtime that torch then cannot share, and device calls would fail.
import torch  # noqa: F401

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librefadapt.so")

# ra_status
RA_OK, RA_EINVAL, RA_EUNSUPPORTED, RA_EWORKSPACE, RA_ELAUNCH = 0, -1, -2, -3, -4
# ra_dtype
RA_BF16, RA_F32 = 0, 1
# ra_qset
RA_Q_TARGET, RA_Q_ALL = 0, 1
# ra_kvsrc
RA_KV_FRESH, RA_KV_CACHE, RA_KV_DEVICE, RA_KV_SEGMENTS = 0, 1, 2, 3
RA_MAX_SEG = 16
# ra_decision
RA_REUSE, RA_REACTIVATE, RA_COMPUTE = 0, 1, 2
# ra_gate_mode
RA_GATE_PRODUCT, RA_GATE_Q_ONLY, RA_GATE_MASS_ONLY, RA_GATE_AND = 0, 1, 2, 3
# matrix-core rate probe
RA_PROBE_DENSE, RA_PROBE_MIX = 0, 1
RA_PROBE_OPERAND_BYTES = 65536

EXPORTED = (
    "refadapt_joint_attn",
    "refadapt_joint_attn_workspace_size",
    "refadapt_joint_attn_seg_workspace_size",
    "refadapt_q_change_workspace_size",
    "refadapt_q_change",
    "refadapt_gate",
    "refadapt_q_change_gate_workspace_size",
    "refadapt_q_change_gate",
    "refadapt_q_change_gate_noalloc",
    "refadapt_cache_commit",
    "refadapt_kv_drift_workspace_size",
    "refadapt_kv_drift",
    "refadapt_drift_log_ratio_workspace_size",
    "refadapt_drift_log_ratio",
    "refadapt_output_impact_workspace_size",
    "refadapt_output_impact",
    "refadapt_mass_mean",
    "refadapt_adjacent_mass_change",
    "refadapt_mfma_rate_probe",
    "refadapt_last_error",
    "refadapt_version",
)


class ra_tensor(ctypes.Structure):
    _fields_ = [
        ("data", ctypes.c_void_p),
        ("stride_b", ctypes.c_int64),
        ("stride_h", ctypes.c_int64),
        ("stride_s", ctypes.c_int64),
    ]


class ra_attn_desc(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("n_ref", ctypes.c_int32),
        ("n_tgt", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("scale", ctypes.c_float),
        ("qset", ctypes.c_int32),
        ("kvsrc", ctypes.c_int32),
    ]


class ra_attn_args(ctypes.Structure):
    _fields_ = [
        ("q_tgt", ra_tensor),
        ("k_tgt", ra_tensor),
        ("v_tgt", ra_tensor),
        ("q_ref", ra_tensor),
        ("k_ref", ra_tensor),
        ("v_ref", ra_tensor),
        ("k_cache", ra_tensor),
        ("v_cache", ra_tensor),
        ("decision", ctypes.c_void_p),
        ("o_tgt", ra_tensor),
        ("o_ref", ra_tensor),
        ("ref_mass", ctypes.c_void_p),
        ("lse_tgt", ctypes.c_void_p),
        ("ref_mass_refq", ctypes.c_void_p),
        ("workspace", ctypes.c_void_p),
        ("workspace_bytes", ctypes.c_size_t),
        ("n_seg", ctypes.c_int32),
        ("seg_end", ctypes.c_int32 * RA_MAX_SEG),
        ("seg_cache", ctypes.c_uint32),
        ("seg_mass", ctypes.c_void_p),
        ("q_cache", ra_tensor),
        ("clock_probe", ctypes.c_void_p),
    ]


class ra_gate_state(ctypes.Structure):
    _fields_ = [
        ("reactivated", ctypes.c_int32),
        ("a_full", ctypes.c_int32),
        ("delta_max", ctypes.c_int32),
        ("step", ctypes.c_int32),
    ]


class RefadaptError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"refadapt status {status}: {message}")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2609_32415_amd.csrc.build` "
            "(the HIP library is the only implementation; there is no fallback)"
        )
    lib = ctypes.CDLL(LIB_PATH)
    i32, vp, f32 = ctypes.c_int32, ctypes.c_void_p, ctypes.c_float
    lib.refadapt_joint_attn.argtypes = [ctypes.POINTER(ra_attn_desc), ctypes.POINTER(ra_attn_args), vp]
    lib.refadapt_joint_attn.restype = i32
    lib.refadapt_joint_attn_workspace_size.argtypes = [ctypes.POINTER(ra_attn_desc)]
    lib.refadapt_joint_attn_workspace_size.restype = ctypes.c_size_t
    lib.refadapt_joint_attn_seg_workspace_size.argtypes = [ctypes.POINTER(ra_attn_desc), ctypes.c_int32]
    lib.refadapt_joint_attn_seg_workspace_size.restype = ctypes.c_size_t
    lib.refadapt_q_change_workspace_size.argtypes = [i32, i32, i32, i32]
    lib.refadapt_q_change_workspace_size.restype = ctypes.c_size_t
    lib.refadapt_q_change.argtypes = [i32, i32, i32, i32, i32, ra_tensor, ra_tensor, f32, vp, vp, ctypes.c_size_t, vp]
    lib.refadapt_q_change.restype = i32
    lib.refadapt_gate.argtypes = [i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp]
    lib.refadapt_gate.restype = i32
    lib.refadapt_q_change_gate_workspace_size.argtypes = [i32, i32, i32, i32]
    lib.refadapt_q_change_gate_workspace_size.restype = ctypes.c_size_t
    lib.refadapt_q_change_gate.argtypes = [i32, i32, i32, i32, i32, ra_tensor, ra_tensor, f32, i32, i32, i32,
                                           vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.refadapt_q_change_gate.restype = i32
    lib.refadapt_q_change_gate_noalloc.argtypes = [i32, i32, i32, i32, i32, ra_tensor, ra_tensor, f32, i32, i32,
                                                   i32, vp, vp, vp, vp, vp, vp, vp]
    lib.refadapt_q_change_gate_noalloc.restype = i32
    lib.refadapt_cache_commit.argtypes = [i32, i32, i32, i32, i32, ra_tensor, ra_tensor, ra_tensor, ra_tensor,
                                          ra_tensor, ra_tensor, vp, vp, i32, vp]
    lib.refadapt_cache_commit.restype = i32
    lib.refadapt_kv_drift_workspace_size.argtypes = [i32, i32, i32, i32]
    lib.refadapt_kv_drift_workspace_size.restype = ctypes.c_size_t
    lib.refadapt_kv_drift.argtypes = [i32, i32, i32, i32, i32, ra_tensor, ra_tensor, ra_tensor, ra_tensor, f32,
                                      vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.refadapt_kv_drift.restype = i32
    lib.refadapt_drift_log_ratio_workspace_size.argtypes = [i32, i32, i32, i32, i32]
    lib.refadapt_drift_log_ratio_workspace_size.restype = ctypes.c_size_t
    lib.refadapt_drift_log_ratio.argtypes = [i32, i32, i32, i32, i32, i32, ra_tensor, ra_tensor, ra_tensor,
                                             ra_tensor, f32, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.refadapt_drift_log_ratio.restype = i32
    lib.refadapt_output_impact_workspace_size.argtypes = [i32, i32, i32, i32]
    lib.refadapt_output_impact_workspace_size.restype = ctypes.c_size_t
    lib.refadapt_output_impact.argtypes = [i32, i32, i32, i32, i32, ra_tensor, ra_tensor, f32, vp, vp,
                                           ctypes.c_size_t, vp]
    lib.refadapt_output_impact.restype = i32
    lib.refadapt_mass_mean.argtypes = [i32, i32, i32, vp, i32, vp, vp]
    lib.refadapt_mass_mean.restype = i32
    lib.refadapt_adjacent_mass_change.argtypes = [i32, i32, i32, vp, vp, vp]
    lib.refadapt_adjacent_mass_change.restype = i32
    lib.refadapt_mfma_rate_probe.argtypes = [i32, i32, i32, vp, vp, vp, vp]
    lib.refadapt_mfma_rate_probe.restype = i32
    lib.refadapt_last_error.argtypes = []
    lib.refadapt_last_error.restype = ctypes.c_char_p
    lib.refadapt_version.argtypes = []
    lib.refadapt_version.restype = ctypes.c_char_p
    return lib


LIB = _load()


def _check(status):
    if status != RA_OK:
        raise RefadaptError(status, LIB.refadapt_last_error().decode())
    return status


def refadapt_joint_attn(desc, args, stream):
    """Forward to ``refadapt_joint_attn``; raises RefadaptError on a non-OK status."""
    return _check(LIB.refadapt_joint_attn(ctypes.byref(desc), ctypes.byref(args), stream))


def refadapt_joint_attn_workspace_size(desc):
    return int(LIB.refadapt_joint_attn_workspace_size(ctypes.byref(desc)))


def refadapt_joint_attn_seg_workspace_size(desc, n_seg):
    return int(LIB.refadapt_joint_attn_seg_workspace_size(ctypes.byref(desc), n_seg))


def refadapt_q_change_workspace_size(batch, heads, n_tgt, head_dim):
    return int(LIB.refadapt_q_change_workspace_size(batch, heads, n_tgt, head_dim))


def refadapt_q_change(batch, heads, n_tgt, head_dim, dtype, q_cur, q_prev, eps, d_out, workspace, ws_bytes, stream):
    return _check(LIB.refadapt_q_change(batch, heads, n_tgt, head_dim, dtype, q_cur, q_prev, eps, d_out, workspace, ws_bytes, stream))


def refadapt_gate(batch, heads, n_tgt, block, step, mode, d_cur, mass_prev, theta, state, decision_out, score_out, stream):
    return _check(LIB.refadapt_gate(batch, heads, n_tgt, block, step, mode, d_cur, mass_prev, theta, state, decision_out, score_out, stream))


def refadapt_q_change_gate_workspace_size(batch, heads, n_tgt, head_dim):
    return int(LIB.refadapt_q_change_gate_workspace_size(batch, heads, n_tgt, head_dim))


def refadapt_q_change_gate(batch, heads, n_tgt, head_dim, dtype, q_cur, q_prev, eps, block, step, mode, mass_prev,
                           theta, state, d_out, decision_out, score_out, workspace, ws_bytes, stream):
    return _check(LIB.refadapt_q_change_gate(batch, heads, n_tgt, head_dim, dtype, q_cur, q_prev, eps, block, step,
                                             mode, mass_prev, theta, state, d_out, decision_out, score_out,
                                             workspace, ws_bytes, stream))


def refadapt_q_change_gate_noalloc(batch, heads, n_tgt, head_dim, dtype, q_cur, q_prev, eps, block, step, mode,
                                   mass_prev, theta, state, d_out, decision_out, score_out, stream):
    return _check(LIB.refadapt_q_change_gate_noalloc(batch, heads, n_tgt, head_dim, dtype, q_cur, q_prev, eps, block,
                                                     step, mode, mass_prev, theta, state, d_out, decision_out,
                                                     score_out, stream))


def refadapt_cache_commit(batch, heads, n_ref, head_dim, dtype, k_ref, v_ref, q_ref, k_cache, v_cache, q_cache,
                          decision, age, step, stream):
    return _check(LIB.refadapt_cache_commit(batch, heads, n_ref, head_dim, dtype, k_ref, v_ref, q_ref, k_cache,
                                            v_cache, q_cache, decision, age, step, stream))


def refadapt_kv_drift_workspace_size(batch, heads, n_rows, head_dim):
    return int(LIB.refadapt_kv_drift_workspace_size(batch, heads, n_rows, head_dim))


def refadapt_kv_drift(batch, heads, n_rows, head_dim, dtype, k_cur, k_base, v_cur, v_base, eps, d_k, d_v, e_kv,
                      workspace, ws_bytes, stream):
    return _check(LIB.refadapt_kv_drift(batch, heads, n_rows, head_dim, dtype, k_cur, k_base, v_cur, v_base, eps,
                                        d_k, d_v, e_kv, workspace, ws_bytes, stream))


def refadapt_drift_log_ratio_workspace_size(batch, heads, n_ref, n_tgt, head_dim):
    return int(LIB.refadapt_drift_log_ratio_workspace_size(batch, heads, n_ref, n_tgt, head_dim))


def refadapt_drift_log_ratio(batch, heads, n_ref, n_tgt, head_dim, dtype, z_ref_cur, z_ref_prev, z_tgt_cur,
                             z_tgt_prev, eps, d_ref, d_tgt, rho, workspace, ws_bytes, stream):
    return _check(LIB.refadapt_drift_log_ratio(batch, heads, n_ref, n_tgt, head_dim, dtype, z_ref_cur, z_ref_prev,
                                               z_tgt_cur, z_tgt_prev, eps, d_ref, d_tgt, rho, workspace, ws_bytes,
                                               stream))


def refadapt_output_impact_workspace_size(batch, heads, n_rows, head_dim):
    return int(LIB.refadapt_output_impact_workspace_size(batch, heads, n_rows, head_dim))


def refadapt_output_impact(batch, heads, n_rows, head_dim, dtype, o_stale, o_fresh, eps, impact, workspace,
                           ws_bytes, stream):
    return _check(LIB.refadapt_output_impact(batch, heads, n_rows, head_dim, dtype, o_stale, o_fresh, eps, impact,
                                             workspace, ws_bytes, stream))


def refadapt_mass_mean(batch, heads, n_rows, mass, complement, out, stream):
    return _check(LIB.refadapt_mass_mean(batch, heads, n_rows, mass, complement, out, stream))


def refadapt_adjacent_mass_change(n_steps, n_blocks, bh, mass_mean, out, stream):
    return _check(LIB.refadapt_adjacent_mass_change(n_steps, n_blocks, bh, mass_mean, out, stream))


def refadapt_mfma_rate_probe(kind, workgroups, steps, operands, sink, clock_probe, stream):
    return _check(LIB.refadapt_mfma_rate_probe(kind, workgroups, steps, operands, sink, clock_probe, stream))


def refadapt_last_error():
    return LIB.refadapt_last_error().decode()


def refadapt_version():
    return LIB.refadapt_version().decode()
