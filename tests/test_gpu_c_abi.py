"""The library called from plain C: paper_2609_32415_amd/examples/joint_attn_c (C99, the HIP
runtime API and include/refadapt.h only, built with the library) runs one joint attention
and writes its inputs and outputs; every output element matches the fp64 oracle."""

import os
import subprocess

import numpy as np
import pytest

from gpu_helpers import MASS_TOL, O_TOL, max_abs
from oracle import joint_attention

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "paper_2609_32415_amd", "examples", "joint_attn_c")


def _bf16(u16):
    return (u16.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def test_c_example_matches_oracle(tmp_path):
    assert os.path.exists(EXE), "the C example is built with the library (paper_2609_32415_amd.csrc.build)"
    out = tmp_path / "joint_attn_c.bin"
    print(f"C example {EXE}", flush=True)
    r = subprocess.run([EXE, str(out)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    raw = out.read_bytes()
    assert raw[:4] == b"RAC1"
    B, H, D, n_ref, n_tgt = (int(v) for v in np.frombuffer(raw, dtype=np.int32, count=5, offset=4))
    off = 24

    def take(dtype, shape):
        nonlocal off
        a = np.frombuffer(raw, dtype=dtype, count=int(np.prod(shape)), offset=off).reshape(shape)
        off += a.nbytes
        return a

    tgt, ref_shape = (B, H, n_tgt, D), (B, H, n_ref, D)
    q_tgt, k_tgt, v_tgt = (_bf16(take(np.uint16, tgt)) for _ in range(3))
    q_ref, k_ref, v_ref = (_bf16(take(np.uint16, ref_shape)) for _ in range(3))
    o_tgt, o_ref = _bf16(take(np.uint16, tgt)), _bf16(take(np.uint16, ref_shape))
    mass, lse = take(np.float32, (B, H, n_tgt)), take(np.float32, (B, H, n_tgt, 2))
    assert off == len(raw)
    want = joint_attention(q_tgt, k_ref, v_ref, k_tgt, v_tgt)
    want_ref = joint_attention(q_ref, k_ref, v_ref, k_tgt, v_tgt)
    assert max_abs(o_tgt, want["o"]) <= O_TOL["bf16"]
    assert max_abs(o_ref, want_ref["o"]) <= O_TOL["bf16"]
    assert max_abs(mass, want["ref_mass"]) <= MASS_TOL["bf16"]
    assert max_abs(lse[..., 0], want["lse_ref"]) <= 1e-3 and max_abs(lse[..., 1], want["lse_all"]) <= 1e-3
