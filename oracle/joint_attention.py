"""Joint attention over a [reference; target] key sequence, in fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Definitions followed
--------------------
* Attention operator: Attn(Q, K, V) = softmax(Q K^T / sqrt(d_h)) V, applied to
  the query set over the concatenated keys [K_R; K_Y] and values [V_R; V_Y]
  (paper Sec. 3.3, fresh/stale-output equations). Whether K_R/V_R are the
  current ("fresh") tensors or an earlier anchor ("stale", i.e. the cache) is
  decided by the caller, who passes whichever reference K/V the executed
  attention used.
* Directional exposure per query: m_q = sum over reference keys k of A_qk,
  where A is the post-softmax attention (paper Sec. 3.2, directional-exposure
  equation; that equation then averages m_q over target queries, which is
  ``head_exposure`` in ``stats.py``).
* Split statistics: lse_all = log sum_k exp(l_k) over all keys and lse_ref the
  same over reference keys only, so m_q = exp(lse_ref - lse_all).

The scale defaults to 1/sqrt(d). This is the definition written out, not a
tiled or online-softmax algorithm: the GPU kernel reaches the same values up
to rounding order, since tiling and online rescaling are re-associations.
"""

from __future__ import annotations

import math

import numpy as np


def _as64(x):
    return np.asarray(x, dtype=np.float64)


def joint_attention(q, k_ref, v_ref, k_tgt, v_tgt, scale=None):
    """Softmax attention of ``q`` over [k_ref; k_tgt] with values [v_ref; v_tgt].

    Shapes: ``q`` is ``[..., n_q, d]``; ``k_ref``/``v_ref`` are ``[..., n_ref, d]``
    (``n_ref`` may be 0); ``k_tgt``/``v_tgt`` are ``[..., n_tgt, d]`` with
    ``n_tgt >= 1``. Leading dimensions (batch, heads) must agree.

    Returns a dict of fp64 arrays:
      ``o``        ``[..., n_q, d]``  attention output
      ``ref_mass`` ``[..., n_q]``     sum of the softmax row over reference keys
      ``lse_ref``  ``[..., n_q]``     log-sum-exp of the scaled logits over
                                       reference keys (-inf when n_ref == 0)
      ``lse_all``  ``[..., n_q]``     log-sum-exp over all keys
    """
    q, k_ref, v_ref, k_tgt, v_tgt = map(_as64, (q, k_ref, v_ref, k_tgt, v_tgt))
    d = q.shape[-1]
    s = 1.0 / math.sqrt(d) if scale is None else float(scale)
    n_ref = k_ref.shape[-2]
    if k_tgt.shape[-2] < 1:
        raise ValueError("the target segment must hold at least one key")

    # The key sequence of the joint attention, reference rows first.
    k = np.concatenate([k_ref, k_tgt], axis=-2)
    v = np.concatenate([v_ref, v_tgt], axis=-2)

    logits = s * np.matmul(q, np.swapaxes(k, -1, -2))  # [..., n_q, n_k]
    mu = logits.max(axis=-1, keepdims=True)
    p = np.exp(logits - mu)
    z = p.sum(axis=-1, keepdims=True)
    a = p / z  # post-softmax attention rows
    o = np.matmul(a, v)

    ref_mass = a[..., :n_ref].sum(axis=-1)
    lse_all = mu[..., 0] + np.log(z[..., 0])
    if n_ref > 0:
        lr = logits[..., :n_ref]
        mu_r = lr.max(axis=-1, keepdims=True)
        lse_ref = mu_r[..., 0] + np.log(np.exp(lr - mu_r).sum(axis=-1))
    else:
        lse_ref = np.full(lse_all.shape, -np.inf)
    return {"o": o, "ref_mass": ref_mass, "lse_ref": lse_ref, "lse_all": lse_all}


def joint_attention_loops(q, k_ref, v_ref, k_tgt, v_tgt, scale=None):
    """The same definition as ``joint_attention`` as plain Python loops.

    Only for tiny shapes (a few dozen rows). Inputs are ``[B, H, n, d]``.
    Every softmax row is formed term by term with ``math.exp``: no max
    subtraction, no vector library call.
    """
    q, k_ref, v_ref, k_tgt, v_tgt = map(_as64, (q, k_ref, v_ref, k_tgt, v_tgt))
    B, H, n_q, d = q.shape
    n_ref = k_ref.shape[2]
    n_tgt = k_tgt.shape[2]
    s = 1.0 / math.sqrt(d) if scale is None else float(scale)
    o = np.zeros((B, H, n_q, d))
    ref_mass = np.zeros((B, H, n_q))
    lse_all = np.zeros((B, H, n_q))
    lse_ref = np.full((B, H, n_q), -np.inf)
    for b in range(B):
        for h in range(H):
            keys = [k_ref[b, h, j] for j in range(n_ref)] + [k_tgt[b, h, j] for j in range(n_tgt)]
            vals = [v_ref[b, h, j] for j in range(n_ref)] + [v_tgt[b, h, j] for j in range(n_tgt)]
            for i in range(n_q):
                weights = []
                for kk in keys:
                    dot = 0.0
                    for c in range(d):
                        dot += q[b, h, i, c] * kk[c]
                    weights.append(math.exp(s * dot))
                total = sum(weights)
                for j, w in enumerate(weights):
                    for c in range(d):
                        o[b, h, i, c] += (w / total) * vals[j][c]
                ref_total = sum(weights[:n_ref])
                ref_mass[b, h, i] = ref_total / total
                lse_all[b, h, i] = math.log(total)
                if n_ref > 0:
                    lse_ref[b, h, i] = math.log(ref_total)
    return {"o": o, "ref_mass": ref_mass, "lse_ref": lse_ref, "lse_all": lse_all}


def segment_masses(q, k_ref, k_tgt, seg_end, scale=None):
    """Per-query softmax mass on each reference segment (Sec. 3.2 directional exposure,
    restricted to the keys of one segment).

    ``seg_end`` lists the exclusive end row of each segment inside the reference rows
    (the last one is n_ref). Returns ``[..., n_q, n_seg]`` fp64: the sum of the softmax
    row over the keys of each segment, from the same logits as ``joint_attention``.
    """
    q, k_ref, k_tgt = map(_as64, (q, k_ref, k_tgt))
    d = q.shape[-1]
    s = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ends = list(seg_end)
    if not ends or ends[-1] != k_ref.shape[-2] or any(b <= a for a, b in zip([0] + ends[:-1], ends)):
        raise ValueError("segment ends must increase to n_ref")
    k = np.concatenate([k_ref, k_tgt], axis=-2)
    logits = s * np.matmul(q, np.swapaxes(k, -1, -2))
    p = np.exp(logits - logits.max(axis=-1, keepdims=True))
    a = p / p.sum(axis=-1, keepdims=True)
    starts = [0] + ends[:-1]
    return np.stack([a[..., lo:hi].sum(axis=-1) for lo, hi in zip(starts, ends)], axis=-1)
