"""GPU parity of refadapt_q_change, refadapt_gate and refadapt_cache_commit
against the fp64 oracle (through the C ABI)."""

import math

import numpy as np
import pytest
import torch

from gpu_helpers import dev, host
from oracle import COMPUTE, REACTIVATE, REUSE, gate, q_change
from oracle.stats import full_refresh_due
from paper_2609_32415_amd import synth

pytestmark = pytest.mark.gpu

ops = None


@pytest.fixture(scope="module", autouse=True)
def _ops():
    global ops
    from paper_2609_32415_amd import ops as _o

    ops = _o
    yield


@pytest.mark.parametrize(
    "dtype,B,H,n,d,sigma",
    [("f32", 1, 2, 256, 64, 0.3), ("bf16", 1, 24, 4096, 128, 0.3), ("bf16", 2, 3, 333, 128, 0.05),
     ("bf16", 1, 2, 1, 64, 0.2), ("f32", 1, 1, 7, 128, 1e-3), ("bf16", 1, 24, 16384, 128, 0.2)],
)
def test_q_change_parity(dtype, B, H, n, d, sigma):
    print(f"q_change {dtype} {B}x{H}x{n}x{d}", flush=True)
    w = synth.workload("tiny", dtype=dtype, batch=B, heads=H, n_ref=1, n_tgt=n, head_dim=d, tgt_drift=sigma)
    tr = synth.Trajectory(w)
    prev = tr.step_tensors(0)["q_tgt"]
    cur = tr.step_tensors(1)["q_tgt"]
    got = ops.q_change(dev(cur, dtype), dev(prev, dtype), eps=1e-8)
    torch.cuda.synchronize()
    ref = q_change(cur, prev, 1e-8)
    np.testing.assert_allclose(host(got), ref, rtol=1e-5, atol=0)


def _layout(t, kind):
    """``t`` ([B, H, S, d]) as a head-interleaved view ([B, S, H, d] storage) or with its rows
    padded by 16 NaN elements; "plain" leaves it contiguous."""
    B, H, S, d = t.shape
    if kind == "bshd":
        return t.transpose(1, 2).contiguous().transpose(1, 2)
    if kind == "pad":
        buf = torch.full((B, H, S, d + 16), float("nan"), dtype=t.dtype, device=t.device)
        buf[..., :d] = t
        return buf[..., :d]
    return t


def _strided_cases(n=16, seed=99):
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        cases.append((i, str(rng.choice(["bf16", "f32"])), int(rng.integers(1, 3)), int(rng.integers(1, 33)),
                      int(rng.choice([1, 63, 65, int(rng.integers(2, 3000)), int(rng.integers(3000, 12000))])),
                      int(rng.choice([64, 128])), ["plain", "bshd", "pad"][i % 3]))
    return cases


@pytest.mark.parametrize("case", _strided_cases(), ids=lambda c: f"s{c[0]}-{c[1]}-{c[6]}")
def test_q_change_and_fused_gate_on_strided_views(case):
    """Q-change and the fused Q-change + gate on contiguous, head-interleaved and padded-row
    views (NaN in the padding): D matches the oracle and is identical between the two entry
    points; the fused gate's scores and decision follow the oracle gate."""
    i, dtype, B, H, n, d, kind = case
    print(f"q_change strided {case}", flush=True)
    rng = np.random.default_rng(500 + i)
    q0 = synth.round_to_dtype(rng.standard_normal((B, H, n, d)).astype(np.float32), dtype)
    sig = rng.uniform(1e-3, 0.8, (1, H, 1, 1)).astype(np.float32)
    q1 = synth.round_to_dtype(q0 + sig * rng.standard_normal(q0.shape).astype(np.float32), dtype)
    m = rng.uniform(0.0, 1.0, (B, H, n)).astype(np.float32)
    a, b = _layout(dev(q1, dtype), kind), _layout(dev(q0, dtype), kind)
    got = ops.q_change(a, b)
    theta = torch.tensor([0.15], dtype=torch.float32, device="cuda:0")
    d2, dec, score = ops.q_change_gate(a, b, dev(m, "f32"), theta, ops.new_gate_state("cuda:0"), 0, 1, "product")
    torch.cuda.synchronize()
    ref = q_change(q1, q0, 1e-8)
    np.testing.assert_allclose(host(got), ref, rtol=1e-5, atol=0)
    assert torch.equal(got, d2)
    exp = gate(ref, m, 0.15, False)
    np.testing.assert_allclose(host(score), [exp.d_mean, exp.m_mean, exp.g_mean], rtol=1e-5, atol=1e-7)
    assert abs(exp.g_mean - 0.15) > 1e-4, "the case must not sit on the threshold"
    assert int(dec.item()) == exp.decision


def test_q_change_closed_forms_on_device():
    q = np.random.default_rng(0).standard_normal((1, 3, 100, 64)).astype(np.float32)
    z = ops.q_change(dev(q, "f32"), dev(q, "f32"))
    neg = ops.q_change(dev(-q, "f32"), dev(q, "f32"), eps=0.0)
    zero_prev = ops.q_change(dev(q, "f32"), dev(np.zeros_like(q), "f32"), eps=1e-3)
    torch.cuda.synchronize()
    assert np.all(host(z) == 0)
    np.testing.assert_allclose(host(neg), 2.0, rtol=1e-6)
    np.testing.assert_allclose(host(zero_prev), np.sqrt((q.astype(np.float64) ** 2).sum((-2, -1))) / 1e-3, rtol=1e-5)


def test_q_change_is_deterministic():
    w = synth.workload("single_ref", heads=8, n_tgt=4096)
    x = synth.block_inputs(w)
    a, b = dev(x["q_tgt"], "bf16"), dev(x["q_ref"][:, :, :4096], "bf16")
    r1, r2 = ops.q_change(a, b), ops.q_change(a, b)
    torch.cuda.synchronize()
    assert torch.equal(r1, r2)


NAMES = {REUSE: "REUSE", REACTIVATE: "REACTIVATE", COMPUTE: "COMPUTE"}


def _gate_inputs(seed, B, H, n):
    rng = np.random.default_rng(seed)
    d = rng.uniform(0.0, 0.6, (B, H)).astype(np.float32)
    m = rng.uniform(0.0, 1.0, (B, H, n)).astype(np.float32)
    return d, m


@pytest.mark.parametrize("mode", ["product", "q_only", "mass_only", "and"])
def test_gate_sequence_matches_oracle(mode):
    """A sequence of steps x blocks of gate calls reproduces the oracle's decisions
    and scores on identical (D, M) inputs, including the step bookkeeping."""
    B, H, n, n_blocks, n_steps = 1, 24, 4096, 6, 4
    rng = np.random.default_rng(1)
    if mode == "and":
        th = np.stack([rng.uniform(0.1, 0.4, n_blocks), rng.uniform(0.3, 0.7, n_blocks)], 1).astype(np.float32)
    elif mode == "product":
        th = rng.uniform(0.05, 0.2, n_blocks).astype(np.float32)
    else:
        th = rng.uniform(0.2, 0.6, n_blocks).astype(np.float32)
    theta = torch.from_numpy(th.reshape(-1)).cuda()
    state = ops.new_gate_state("cuda:0", delta_max=3)
    a_full = 0
    for t in range(n_steps):
        full = full_refresh_due(t, a_full, 3)
        if full:
            a_full = t
        react = full
        for b in range(n_blocks):
            d, m = _gate_inputs(100 * t + b, B, H, n)
            dec, score = ops.gate(dev(d, "f32"), dev(m, "f32"), theta, state, b, t, mode)
            torch.cuda.synchronize()
            exp = gate(d, m, float(th[b][0] if mode == "and" else th[b]), react, mode=mode,
                       theta_m=float(th[b][1]) if mode == "and" else None)
            react = exp.reactivated
            got = int(dec.item())
            margin = {"product": exp.g_mean, "q_only": exp.d_mean, "mass_only": exp.m_mean, "and": exp.d_mean}[mode]
            thr = float(th[b][0] if mode == "and" else th[b])
            if abs(margin - thr) > 1e-4:
                assert got == exp.decision, (t, b, NAMES[got], NAMES[exp.decision])
            else:
                react = got != REUSE
            s = host(score)
            np.testing.assert_allclose(s, [exp.d_mean, exp.m_mean, exp.g_mean], rtol=1e-5, atol=1e-7)
        st = state.cpu().tolist()
        assert st[1] == a_full and st[3] == t


@pytest.mark.parametrize("B,H", [(1, 8192), (2, 4096)])
def test_gate_at_the_batch_heads_limit(B, H):
    """batch * heads = 8192, the largest the gate entry points take (their per-head
    D and mean-mass tables then fill 64 KiB of LDS): refadapt_gate and the fused
    refadapt_q_change_gate reproduce the oracle's D, scores and decision."""
    print(f"gate limit {B}x{H}", flush=True)
    n, d_head = 5, 64
    rng = np.random.default_rng(11)
    q0 = rng.standard_normal((B, H, n, d_head)).astype(np.float32)
    q1 = (q0 + 0.3 * rng.standard_normal(q0.shape)).astype(np.float32)
    m = rng.uniform(0.0, 1.0, (B, H, n)).astype(np.float32)
    d_ref = q_change(q1, q0, 1e-8)
    theta_v = 0.15
    theta = torch.full((1,), theta_v, dtype=torch.float32, device="cuda:0")
    exp = gate(d_ref.astype(np.float32), m, theta_v, False)
    # The separate gate on the oracle's D.
    state = ops.new_gate_state("cuda:0")
    ops.gate(dev(d_ref.astype(np.float32), "f32"), dev(m, "f32"), theta, state, 0, 0, "product")  # step 0
    dec, score = ops.gate(dev(d_ref.astype(np.float32), "f32"), dev(m, "f32"), theta, state, 0, 1, "product")
    torch.cuda.synchronize()
    np.testing.assert_allclose(host(score), [exp.d_mean, exp.m_mean, exp.g_mean], rtol=1e-5, atol=1e-7)
    if abs(exp.g_mean - theta_v) > 1e-4:
        assert int(dec.item()) == exp.decision
    # The fused path computes D itself.
    state = ops.new_gate_state("cuda:0")
    ops.gate(dev(d_ref.astype(np.float32), "f32"), dev(m, "f32"), theta, state, 0, 0, "product")  # step 0
    d_got, dec, score = ops.q_change_gate(dev(q1, "f32"), dev(q0, "f32"), dev(m, "f32"), theta, state, 0, 1,
                                          "product", eps=1e-8)
    torch.cuda.synchronize()
    np.testing.assert_allclose(host(d_got), d_ref, rtol=1e-5, atol=0)
    np.testing.assert_allclose(host(score), [exp.d_mean, exp.m_mean, exp.g_mean], rtol=1e-5, atol=1e-7)
    if abs(exp.g_mean - theta_v) > 1e-4:
        assert int(dec.item()) == exp.decision


@pytest.mark.parametrize("mode", ["product", "and"])
@pytest.mark.parametrize("dtype,B,H,n,d", [("bf16", 1, 24, 4096, 128), ("bf16", 2, 3, 333, 64), ("f32", 1, 2, 100, 64)])
def test_fused_q_change_gate_matches_oracle(mode, dtype, B, H, n, d):
    """refadapt_q_change_gate over steps x blocks with one reused workspace: D equals
    refadapt_q_change bit for bit, decisions and scores follow the oracle's Q-change
    and gate on the same inputs."""
    print(f"q_change_gate {mode} {dtype} {B}x{H}x{n}x{d}", flush=True)
    n_blocks, n_steps = 4, 3
    rng = np.random.default_rng(7)
    if mode == "and":
        th = np.stack([rng.uniform(0.2, 0.4, n_blocks), rng.uniform(0.3, 0.6, n_blocks)], 1).astype(np.float32)
    else:
        th = rng.uniform(0.1, 0.2, n_blocks).astype(np.float32)
    theta = torch.from_numpy(th.reshape(-1)).cuda()
    state = ops.new_gate_state("cuda:0", delta_max=2)
    q0 = synth.round_to_dtype(rng.standard_normal((B, H, n, d)).astype(np.float32), dtype)
    ws = ops.q_change_gate_workspace(dev(q0, dtype))
    a_full = 0
    for t in range(n_steps):
        full = full_refresh_due(t, a_full, 2)
        if full:
            a_full = t
        react = full
        for b in range(n_blocks):
            sig = rng.uniform(0.05, 0.6, (1, H, 1, 1)).astype(np.float32)
            q1 = synth.round_to_dtype(q0 + sig * rng.standard_normal(q0.shape).astype(np.float32), dtype)
            m = rng.uniform(0.0, 1.0, (B, H, n)).astype(np.float32)
            d_got, dec, score = ops.q_change_gate(dev(q1, dtype), dev(q0, dtype), dev(m, "f32"), theta, state, b, t,
                                                  mode, workspace=ws)
            d_ref = ops.q_change(dev(q1, dtype), dev(q0, dtype))
            torch.cuda.synchronize()
            assert torch.equal(d_got, d_ref)
            dq = q_change(q1, q0)
            np.testing.assert_allclose(host(d_got), dq, rtol=1e-5)
            thr = float(th[b][0] if mode == "and" else th[b])
            exp = gate(dq, m, thr, react, mode=mode, theta_m=float(th[b][1]) if mode == "and" else None)
            react = exp.reactivated
            got = int(dec.item())
            margin = exp.g_mean if mode == "product" else exp.d_mean
            if abs(margin - thr) > 1e-4 and (mode != "and" or abs(exp.m_mean - float(th[b][1])) > 1e-4):
                assert got == exp.decision, (t, b, NAMES[got], NAMES[exp.decision])
            else:
                react = got != REUSE
            np.testing.assert_allclose(host(score), [exp.d_mean, exp.m_mean, exp.g_mean], rtol=1e-5, atol=1e-7)
            q0 = q1
        st = state.cpu().tolist()
        assert st[1] == a_full and st[3] == t


def test_gate_thresholds_zero_and_infinite():
    B, H, n = 1, 4, 300
    d, m = _gate_inputs(5, B, H, n)
    for thv, expect in ((0.0, REACTIVATE), (math.inf, REUSE)):
        state = ops.new_gate_state("cuda:0")
        theta = torch.full((2,), thv, dtype=torch.float32, device="cuda:0")
        ops.gate(dev(d, "f32"), dev(m, "f32"), theta, state, 0, 1, "product")  # block 0 of step 1
        dec, _ = ops.gate(dev(d, "f32"), dev(m, "f32"), theta, state, 1, 1, "product")
        torch.cuda.synchronize()
        assert int(dec.item()) == (COMPUTE if expect == REACTIVATE else REUSE)
    # Step 0 computes every block whatever theta says.
    state = ops.new_gate_state("cuda:0")
    theta = torch.full((1,), math.inf, dtype=torch.float32, device="cuda:0")
    dec, _ = ops.gate(dev(d, "f32"), dev(m, "f32"), theta, state, 0, 0, "product")
    torch.cuda.synchronize()
    assert int(dec.item()) == COMPUTE


@pytest.mark.parametrize("decision,copied", [(2, True), (0, False)])
def test_cache_commit_k_only(decision, copied):
    """With both V views omitted only K is copied (the anchor-Q commit)."""
    src = torch.randn((1, 3, 77, 128), device="cuda:0").to(torch.bfloat16)
    dst = torch.zeros_like(src)
    dec = torch.tensor([decision], dtype=torch.int32, device="cuda:0")
    ops.cache_commit(src, None, dst, None, decision=dec)
    torch.cuda.synchronize()
    assert torch.equal(dst, src) if copied else bool((dst == 0).all())


@pytest.mark.parametrize("decision,copied", [(2, True), (0, False)])
def test_cache_commit_with_queries(decision, copied):
    """K, V and the reference queries of the state go to the cache in one launch."""
    rng = np.random.default_rng(4)
    shape = (2, 3, 130, 64)
    src = [dev(rng.standard_normal(shape).astype(np.float32), "bf16") for _ in range(3)]
    dst = [torch.zeros_like(x) for x in src]
    dec = torch.tensor([decision], dtype=torch.int32, device="cuda:0")
    ops.cache_commit(src[0], src[1], dst[0], dst[1], decision=dec, q_ref=src[2], q_cache=dst[2])
    torch.cuda.synchronize()
    for s_, d_ in zip(src, dst):
        assert torch.equal(d_, s_) if copied else bool((d_ == 0).all())


@pytest.mark.parametrize("decision,copied", [(2, True), (1, False), (0, False), (None, True)])
def test_cache_commit(decision, copied):
    rng = np.random.default_rng(3)
    shape = (1, 3, 200, 128)
    src_k, src_v = (dev(rng.standard_normal(shape).astype(np.float32), "bf16") for _ in range(2))
    ck, cv = torch.zeros_like(src_k), torch.zeros_like(src_v)
    age = torch.full((1,), -1, dtype=torch.int32, device="cuda:0")
    dec = None if decision is None else torch.tensor([decision], dtype=torch.int32, device="cuda:0")
    ops.cache_commit(src_k, src_v, ck, cv, decision=dec, age=age, step=5)
    torch.cuda.synchronize()
    if copied:
        assert torch.equal(ck, src_k) and torch.equal(cv, src_v) and int(age.item()) == 5
    else:
        assert torch.count_nonzero(ck) == 0 and torch.count_nonzero(cv) == 0 and int(age.item()) == -1


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("bf16", 64), ("f32", 64)])
def test_cache_commit_between_strided_views(dtype, d):
    """Head-interleaved sources into caches with padded rows (and the reverse for V): every row
    is copied, and the padding of the destination keeps its sentinel (nothing is written
    outside the view)."""
    rng = np.random.default_rng(11)
    B, H, n = 2, 3, 157
    src_k = _layout(dev(rng.standard_normal((B, H, n, d)).astype(np.float32), dtype), "bshd")
    src_v = _layout(dev(rng.standard_normal((B, H, n, d)).astype(np.float32), dtype), "pad")
    tdt = src_k.dtype
    buf_k = torch.full((B, H, n, d + 16), 7.0, dtype=tdt, device="cuda:0")
    dst_k = buf_k[..., :d]
    dst_k.zero_()
    dst_v = torch.zeros((B, n, H, d), dtype=tdt, device="cuda:0").transpose(1, 2)
    dec = torch.tensor([2], dtype=torch.int32, device="cuda:0")
    ops.cache_commit(src_k, src_v, dst_k, dst_v, decision=dec)
    torch.cuda.synchronize()
    assert torch.equal(dst_k, src_k) and torch.equal(dst_v, src_v)
    assert bool((buf_k[..., d:] == 7.0).all())


def test_mfma_rate_probe_runs_and_is_deterministic():
    """Both register-only MFMA probes finish, write finite, repeatable sinks and count a
    plausible shader clock."""
    ops_ = torch.randn(32768, generator=torch.Generator().manual_seed(0)).to(torch.bfloat16).cuda()
    for kind in ("dense", "mix"):
        print(f"mfma rate probe {kind}", flush=True)
        probe = torch.zeros(2, dtype=torch.int64, device="cuda:0")
        a = ops.mfma_rate_probe(kind, ops_, 64, workgroups=8, clock_probe=probe).clone()
        b = ops.mfma_rate_probe(kind, ops_, 64, workgroups=8)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(a).all()) and torch.equal(a, b)
        cyc, ticks = probe.cpu().tolist()
        assert ticks > 0 and 300.0 < 100.0 * cyc / ticks < 3000.0
