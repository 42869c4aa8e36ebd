"""Benchmark of the RefAdapt-DiT joint-attention hot path on one MI355X.

One step = one pass of the whole path over one block of the multi-reference
image-editing workload (batch 1, 24 heads, head_dim 128, 4096 target tokens,
3 x 4096 reference-image + 256 text tokens = 12544 reference tokens, bf16):

  1+2. Q-change and gate, one launch:
                   D = ||Q_t - Q_{t-1}||_F / (||Q_{t-1}||_F + eps) per head, then the
                   head-mean D*M against theta, decision written on the device
  3. reuse attn    target queries over [cached K_R; K_Y]      (0.838 TFLOP)
  4. full attn     all queries over [fresh K_R; K_Y]          (3.402 TFLOP)
  5. cache commit  fresh reference K/V -> cache if the decision is COMPUTE

``value`` = attention FLOPs of (3)+(4) / measured step time (TFLOP/s). The
JSON line also carries each attention mode on its own, the attention-time
speedup of a reused block over a computed one, the roofline of the dominant
kernel (the full-fresh attention) measured live with HIP events on the launch
stream, and the fp64 CPU oracle timed on a bounded sample of the same work.

``--sweep`` additionally runs the 60-block x 8-step controller sweep
(single-reference shapes, 3 x 3 thresholds, cue ablation, graph replays) and
reports the reuse fraction, the attention-time speedup of adaptive reuse and
the output error against a full-fresh trajectory. ``--ref-sweep`` runs the
reference-count sweep (1..8 reference images). ``--shapes`` times the reuse and
full-fresh attention at the single-reference, multi-reference and video shapes.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
HBM_PEAK_GBS = 8000.0
WORKLOAD = "multi_ref"
PMC_SUMMARY = os.path.join(ROOT, "profiles", "attn_bf16_multi_ref_full_pmc.md")
KERNEL_SRC = os.path.join(ROOT, "paper_2609_32415_amd", "csrc", "attn_bf16.hip")


def attn_flops(heads, n_q, n_k, d, batch=1):
    """Dense joint-attention work: Q K^T and P V, 2 FLOP per multiply-add each."""
    return 4.0 * batch * heads * n_q * n_k * d


def parse_args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    # ~55 ms of steps: after the host-side input generation the GPU clock needs tens of
    # milliseconds of load to come back up
    ap.add_argument("--warmup", type=int, default=15)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="target duration of the oracle sample")
    ap.add_argument("--sweep", action="store_true", help="also run the 60-block x 8-step controller sweep")
    ap.add_argument("--diagnostics", action="store_true",
                    help="also run the diagnostics sidecar over a 60-block x 8-step controller trajectory")
    ap.add_argument("--segments", action="store_true",
                    help="also run the per-reference exposure / individual stale impact table")
    ap.add_argument("--ref-sweep", action="store_true",
                    help="also run the reference-count sweep (1..8 reference images at single-reference shapes)")
    ap.add_argument("--shapes", action="store_true",
                    help="also time the reuse and full-fresh attention at the single-reference, multi-reference and video shapes")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run the cache-commit copy over 2 x 512 MiB (a plain copy of known size, "
                    "for scaling the FETCH_SIZE / WRITE_SIZE counters) and exit")
    return ap.parse_args()


def copy_calibration():
    """A plain device copy of exactly 1 GiB read + 1 GiB written per launch
    (K and V of 24 heads x 87381 rows x 128 bf16 -> cache), run 5 times."""
    import torch

    from paper_2609_32415_amd import ops

    rows = (512 << 20) // (24 * 128 * 2)
    src = [torch.ones((1, 24, rows, 128), dtype=torch.bfloat16, device="cuda:0") for _ in range(2)]
    dst = [torch.empty_like(s) for s in src]
    for _ in range(5):
        ops.cache_commit(src[0], src[1], dst[0], dst[1])
    torch.cuda.synchronize()
    nbytes = 2 * src[0].numel() * 2
    print(json.dumps({"copy_calibration_bytes_read_per_launch": nbytes, "bytes_written_per_launch": nbytes}))


def _traffic_from_profile():
    """HBM bytes per launch of the dominant kernel from the committed rocprofv3
    --pmc summary, or None when absent or taken on a different kernel source."""
    if not os.path.exists(PMC_SUMMARY):
        return None
    text = open(PMC_SUMMARY).read()
    m_src = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", text)
    m_b = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_src or not m_b:
        return None
    cur = hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()
    return float(m_b.group(1)) if cur == m_src.group(1) else None


def time_shapes(dev, reps=10):
    """Reuse (target queries, cached K/V) and full-fresh (all queries, fresh K/V) attention at
    the single-reference, multi-reference and video workload shapes, seeded synthetic inputs
    (the fresh reference K/V stand in for the cache), event-timed over ``reps`` launches after
    warm-up."""
    import torch

    from paper_2609_32415_amd import ops, synth
    from paper_2609_32415_amd.controller import time_launches

    rows = []
    for name in ("single_ref", "multi_ref", "video"):
        w = synth.workload(name)
        x = synth.block_inputs(w)
        bf = lambda a: torch.from_numpy(a).to(dev).to(torch.bfloat16)
        t = {k: bf(x[k]) for k in ("q_tgt", "k_tgt", "v_tgt", "q_ref", "k_ref", "v_ref")}
        B, H, n_tgt, D = t["q_tgt"].shape
        n_ref = t["k_ref"].shape[2]
        ws_r = ops.attn_workspace(t["q_tgt"], n_ref, "target", "cache")
        ws_f = ops.attn_workspace(t["q_tgt"], n_ref, "all", "fresh")
        calls = {
            "reuse": (lambda: ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], k_cache=t["k_ref"], v_cache=t["v_ref"],
                                             n_ref=n_ref, qset="target", kvsrc="cache", workspace=ws_r),
                      attn_flops(H, n_tgt, n_ref + n_tgt, D, B)),
            "full_fresh": (lambda: ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], q_ref=t["q_ref"], k_ref=t["k_ref"],
                                                  v_ref=t["v_ref"], qset="all", kvsrc="fresh", workspace=ws_f),
                           attn_flops(H, n_ref + n_tgt, n_ref + n_tgt, D, B)),
        }
        row = {"workload": name, "heads": H, "head_dim": D, "n_ref": n_ref, "n_tgt": n_tgt}
        for mode, (fn, flop) in calls.items():
            ms = time_launches(fn, reps=reps)
            tf = flop / (ms * 1e-3) / 1e12
            row[mode] = {"ms": round(ms, 4), "tflops": round(tf, 2), "pct_peak": round(100 * tf / BF16_PEAK_TFLOPS, 2)}
        rows.append(row)
        print(f"shape {name}: reuse {row['reuse']}, full-fresh {row['full_fresh']}", file=sys.stderr, flush=True)
        del t, x
        torch.cuda.empty_cache()
    return rows


def cpu_baseline(x, seconds):
    """The fp64 oracle on a bounded sample of the full-fresh attention: all
    heads, all keys, a growing number of query rows until ~``seconds``."""
    import numpy as np

    from oracle import joint_attention

    try:
        from threadpoolctl import threadpool_info

        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count()
    H, n_ref, n_tgt, d = x["q_ref"].shape[1], x["k_ref"].shape[2], x["k_tgt"].shape[2], x["q_tgt"].shape[3]
    rows, spent, total_rows = 8, 0.0, 0
    q_all = np.concatenate([x["q_ref"], x["q_tgt"]], axis=2)
    rng = np.random.default_rng(0)
    while spent < seconds:
        idx = np.sort(rng.choice(q_all.shape[2], size=rows, replace=False))
        t0 = time.perf_counter()
        joint_attention(q_all[:, :, idx], x["k_ref"], x["v_ref"], x["k_tgt"], x["v_tgt"])
        spent += time.perf_counter() - t0
        total_rows += rows
        rows = min(rows * 2, 512)
    flops = attn_flops(H, total_rows, n_ref + n_tgt, d)
    return {
        "value": round(flops / spent / 1e12, 6),
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"full-fresh joint attention of {total_rows} sampled query rows x {H} heads over all "
        f"{n_ref + n_tgt} keys (fp64 numpy oracle, {spent:.1f} s)",
    }


def main():
    args = parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(
            "bench.py measures one MI355X: the hot path has no multi-GPU leg "
            "(heads would shard across GPUs with one head-mean all-reduce per gated block). "
            "Run with --gpus 1.",
            file=sys.stderr,
        )
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_32415_amd import ops, synth

    dev = torch.device("cuda:0")
    w = synth.workload(WORKLOAD, ref_drift=0.01, tgt_drift=0.3, n_steps=2)
    tr = synth.Trajectory(w)
    x0 = tr.step_tensors(0)  # previous step: cache contents and previous target Q
    x1 = tr.step_tensors(1)  # current step: fresh tensors
    bf = lambda a: torch.from_numpy(a).to(dev).to(torch.bfloat16)
    t = {k: bf(v) for k, v in x1.items()}
    cache_k, cache_v, q_prev = bf(x0["k_ref"]), bf(x0["v_ref"]), bf(x0["q_tgt"])
    B, H, n_tgt, D = t["q_tgt"].shape
    n_ref = t["k_ref"].shape[2]

    # Lagged per-query mass from the previous step's executed (full) attention.
    mass_prev = ops.joint_attn(bf(x0["q_tgt"]), bf(x0["k_tgt"]), bf(x0["v_tgt"]), k_ref=cache_k, v_ref=cache_v).ref_mass
    theta = torch.full((1,), 0.1 * 0.2, dtype=torch.float32, device=dev)
    state = ops.new_gate_state(dev)
    ws = ops.q_change_workspace(t["q_tgt"])
    ws_qg = ops.q_change_gate_workspace(t["q_tgt"])
    d_out = torch.empty((B, H), dtype=torch.float32, device=dev)
    dec = torch.empty(1, dtype=torch.int32, device=dev)
    score = torch.empty(3, dtype=torch.float32, device=dev)
    o_tgt_r = torch.empty_like(t["q_tgt"])
    o_tgt_f = torch.empty_like(t["q_tgt"])
    o_ref_f = torch.empty_like(t["q_ref"])
    mass_r = torch.empty((B, H, n_tgt), dtype=torch.float32, device=dev)
    mass_f = torch.empty((B, H, n_tgt), dtype=torch.float32, device=dev)
    commit_k, commit_v = cache_k.clone(), cache_v.clone()
    # Key-split workspaces (partial rows of the query tiles of a last, partly filled round).
    ws_r = ops.attn_workspace(t["q_tgt"], n_ref, "target", "cache")
    ws_f = ops.attn_workspace(t["q_tgt"], n_ref, "all", "fresh")

    ev = lambda: torch.cuda.Event(enable_timing=True)
    marks = {k: [] for k in ("qcg", "reuse", "full", "commit")}

    def step(record):
        e = [ev() for _ in range(5)] if record else None
        if record:
            e[0].record()
        ops.q_change_gate(t["q_tgt"], q_prev, mass_prev, theta, state, 0, 1, "product", d_out=d_out,
                          decision_out=dec, score_out=score, workspace=ws_qg)
        if record:
            e[1].record()
        ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], k_cache=cache_k, v_cache=cache_v, n_ref=n_ref,
                       qset="target", kvsrc="cache", o_tgt=o_tgt_r, ref_mass=mass_r, workspace=ws_r)
        if record:
            e[2].record()
        ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], q_ref=t["q_ref"], k_ref=t["k_ref"], v_ref=t["v_ref"],
                       qset="all", kvsrc="fresh", o_tgt=o_tgt_f, o_ref=o_ref_f, ref_mass=mass_f, workspace=ws_f)
        if record:
            e[3].record()
        ops.cache_commit(t["k_ref"], t["v_ref"], commit_k, commit_v, decision=dec)
        if record:
            e[4].record()
        return e

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    t0, t1 = ev(), ev()
    pending = []
    torch.cuda.synchronize()
    t0.record()
    for _ in range(args.steps):
        pending.append(step(True))
    t1.record()
    torch.cuda.synchronize()
    total_ms = t0.elapsed_time(t1)
    for e in pending:
        for k, (a, b) in zip(marks, zip(e[:-1], e[1:])):
            marks[k].append(a.elapsed_time(b))
    ms = {k: float(np.mean(v)) for k, v in marks.items()}
    ms_per_step = total_ms / args.steps

    # Outside the timed step: the separate Q-change and gate kernels the fused launch replaces,
    # and the diagnostics. Two figures each:
    #  * cold: one launch between events after a 512 MiB read (a reduction, so no dirty lines
    #    are left to write back) has evicted its inputs from the 256 MB last-level cache;
    #  * hot: n back-to-back launches replayed from a captured HIP graph (device time per
    #    launch with the inputs cache-resident; no host launch gaps).
    flush = torch.ones(128 << 20, dtype=torch.float32, device=dev)

    def timed(fn, n=20):
        for _ in range(3):
            fn()
        pairs = []
        for _ in range(n):
            flush.sum()
            a, b = ev(), ev()
            a.record()
            fn()
            b.record()
            pairs.append((a, b))
        torch.cuda.synchronize()
        return float(np.mean([a.elapsed_time(b) for a, b in pairs]))

    def timed_hot(fn, n=20):
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(n):
                fn()
        for _ in range(3):
            g.replay()
        a, b = ev(), ev()
        a.record()
        g.replay()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    def qcg():
        ops.q_change_gate(t["q_tgt"], q_prev, mass_prev, theta, state, 0, 1, "product", d_out=d_out,
                          decision_out=dec, score_out=score, workspace=ws_qg)

    def qc():
        ops.q_change(t["q_tgt"], q_prev, out=d_out, workspace=ws)

    def gate():
        ops.gate(d_out, mass_prev, theta, state, 0, 1, "product", decision_out=dec, score_out=score)

    ms["qcg_hot"] = timed_hot(qcg)
    ms["qc"], ms["qc_hot"] = timed(qc), timed_hot(qc)
    ms["gate"], ms["gate_hot"] = timed(gate), timed_hot(gate)
    # The cache commit of a computed block: copies the fresh reference K/V into the cache.
    ms["commit_copy"] = timed(lambda: ops.cache_commit(t["k_ref"], t["v_ref"], commit_k, commit_v))

    # Diagnostics sidecar kernels (read-only probes), at the same shapes.
    ws_kv = ops.kv_drift_workspace(t["k_ref"])
    ws_ratio = ops.drift_log_ratio_workspace(t["k_ref"], t["k_tgt"])
    ws_imp = ops.output_impact_workspace(o_tgt_r)
    diag_out = torch.empty((3, B, H), dtype=torch.float32, device=dev)
    ms["kv_drift"] = timed(lambda: ops.kv_drift(t["k_ref"], cache_k, t["v_ref"], cache_v, d_k=diag_out[0],
                                                d_v=diag_out[1], e_kv=diag_out[2], workspace=ws_kv))
    k_prev_tgt = bf(x0["k_tgt"])
    ms["ratio"] = timed(lambda: ops.drift_log_ratio(t["k_ref"], cache_k, t["k_tgt"], k_prev_tgt, d_ref=diag_out[0],
                                                    d_tgt=diag_out[1], rho=diag_out[2], workspace=ws_ratio))
    ms["impact"] = timed(lambda: ops.output_impact(o_tgt_r, o_tgt_f, out=diag_out[0], workspace=ws_imp))
    ms["mass_mean"] = timed(lambda: ops.mass_mean(mass_f, out=diag_out[0]))
    diag_bytes = {"kv_drift": 4 * B * H * n_ref * D * 2, "ratio": 2 * B * H * (n_ref + n_tgt) * D * 2,
                  "impact": 2 * B * H * n_tgt * D * 2, "mass_mean": B * H * n_tgt * 4}

    f_reuse = attn_flops(H, n_tgt, n_ref + n_tgt, D, B)
    f_full = attn_flops(H, n_ref + n_tgt, n_ref + n_tgt, D, B)
    value = (f_reuse + f_full) / (ms_per_step * 1e-3) / 1e12
    qc_bytes = 2 * B * H * n_tgt * D * 2
    full_tflops = f_full / (ms["full"] * 1e-3) / 1e12
    reuse_tflops = f_reuse / (ms["reuse"] * 1e-3) / 1e12

    out = {
        "metric": "joint-attn TFLOP/s (bf16, % MFMA peak) + attn-time speedup of adaptive reuse",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "multi-reference image edit: batch 1, 24 heads, head_dim 128, 4096 target + "
            "3x4096 reference-image + 256 text tokens (n_ref 12544); one block-step = Q-change, gate, "
            "reuse attention (target queries, cached reference K/V), full-fresh attention (all queries), "
            "cache commit",
            "batch": B, "heads": H, "head_dim": D, "n_ref": n_ref, "n_tgt": n_tgt,
        },
        "pct_bf16_peak": round(100 * value / BF16_PEAK_TFLOPS, 2),
        "modes": {
            "reuse": {"ms": round(ms["reuse"], 4), "tflops": round(reuse_tflops, 2),
                      "pct_peak": round(100 * reuse_tflops / BF16_PEAK_TFLOPS, 2), "flop": f_reuse},
            "full_fresh": {"ms": round(ms["full"], 4), "tflops": round(full_tflops, 2),
                           "pct_peak": round(100 * full_tflops / BF16_PEAK_TFLOPS, 2), "flop": f_full},
        },
        "reuse_block_attn_speedup": round(ms["full"] / ms["reuse"], 3),
        "small_kernels": {
            "q_change_gate_us": round(ms["qcg"] * 1e3, 2),
            "q_change_gate_gbs": round((qc_bytes + B * H * n_tgt * 4) / (ms["qcg"] * 1e-3) / 1e9, 1),
            "q_change_gate_hot_us": round(ms["qcg_hot"] * 1e3, 2),
            "q_change_us": round(ms["qc"] * 1e3, 2),
            "q_change_gbs": round(qc_bytes / (ms["qc"] * 1e-3) / 1e9, 1),
            "q_change_hot_us": round(ms["qc_hot"] * 1e3, 2),
            "gate_us": round(ms["gate"] * 1e3, 2),
            "gate_gbs": round((B * H * n_tgt * 4 + B * H * 4) / (ms["gate"] * 1e-3) / 1e9, 1),
            "gate_hot_us": round(ms["gate_hot"] * 1e3, 2),
            "commit_us": round(ms["commit"] * 1e3, 2),
            "commit_copy_us": round(ms["commit_copy"] * 1e3, 2),
            "commit_copy_gbs": round(4 * B * H * n_ref * D * 2 / (ms["commit_copy"] * 1e-3) / 1e9, 1),
            "diag_kv_drift_us": round(ms["kv_drift"] * 1e3, 2),
            "diag_kv_drift_gbs": round(diag_bytes["kv_drift"] / (ms["kv_drift"] * 1e-3) / 1e9, 1),
            "diag_drift_log_ratio_us": round(ms["ratio"] * 1e3, 2),
            "diag_drift_log_ratio_gbs": round(diag_bytes["ratio"] / (ms["ratio"] * 1e-3) / 1e9, 1),
            "diag_output_impact_us": round(ms["impact"] * 1e3, 2),
            "diag_output_impact_gbs": round(diag_bytes["impact"] / (ms["impact"] * 1e-3) / 1e9, 1),
            "diag_mass_mean_us": round(ms["mass_mean"] * 1e3, 2),
        },
        "roofline": {
            "kernel": "attn_bf16_kernel<128> (full-fresh mode, with the key-split merge of its last round)",
            "bound": "mfma",
            "achieved": round(full_tflops, 2),
            "peak": BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(full_tflops / BF16_PEAK_TFLOPS, 4),
            "traffic": _traffic_from_profile(),
        },
    }
    if not args.no_cpu_baseline:
        xs = {k: x1[k] for k in ("q_ref", "q_tgt", "k_ref", "v_ref", "k_tgt", "v_tgt")}
        out["cpu_baseline"] = cpu_baseline(xs, args.cpu_seconds)
    if args.sweep:
        from paper_2609_32415_amd.controller import run_sweep

        out["sweep"] = run_sweep(device=dev, log=lambda m: print(m, file=sys.stderr, flush=True))
    if args.diagnostics:
        from paper_2609_32415_amd.controller import run_diagnostics

        out["diagnostics"] = run_diagnostics(device=dev, log=lambda m: print(m, file=sys.stderr, flush=True))
    if args.segments:
        from paper_2609_32415_amd.controller import run_reference_segments

        out["reference_segments"] = run_reference_segments(device=dev, log=lambda m: print(m, file=sys.stderr, flush=True))
    if args.shapes:
        out["shapes"] = time_shapes(dev)
    if args.ref_sweep:
        from paper_2609_32415_amd.controller import run_ref_count_sweep

        out["ref_count_sweep"] = run_ref_count_sweep(device=dev, log=lambda m: print(m, file=sys.stderr, flush=True))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
