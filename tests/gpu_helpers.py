"""Shared helpers of the GPU parity tests: move the seeded numpy inputs to the
device in the run dtype, and read results back for comparison with the oracle."""

import numpy as np
import torch

TORCH_DTYPE = {"bf16": torch.bfloat16, "f32": torch.float32}


def dev(x, dtype):
    """Copy an fp32 numpy array (already exactly representable in ``dtype``) to cuda:0."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda:0").to(TORCH_DTYPE[dtype])


def host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def max_abs(a, b):
    return float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64)))) if np.size(a) else 0.0


# Parity bars for floating point: attention output within 1e-2 (bf16) / 1e-5 (fp32)
# max-abs, reference mass within 1e-3.
O_TOL = {"bf16": 1e-2, "f32": 1e-5}
MASS_TOL = {"bf16": 1e-3, "f32": 1e-5}
