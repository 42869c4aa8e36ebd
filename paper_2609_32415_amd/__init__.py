"""MI355X-native hot path of RefAdapt-DiT (arxiv 2609.32415).

Joint attention over a [reference; target] token sequence whose reference K/V
come fresh or from a per-block cache, with each target query's reference
mass, plus the target-Q change and the reuse gate that drive the paper's
adaptive reuse controller. The compute lives in a C-ABI HIP library
(``librefadapt.so``); ``_lib`` binds it with ctypes, ``ops`` wraps it for torch
tensors (device memory and streams only), ``synth`` draws seeded inputs and
``controller`` runs Alg. 1 over the library's kernels.
"""

__all__ = ["ops", "synth", "controller"]
