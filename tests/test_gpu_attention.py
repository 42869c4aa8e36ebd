"""GPU parity of refadapt_joint_attn against the fp64 oracle (through the C ABI).

Small cases compare every output element; shapes span several query and key
tiles and end in ragged tails. Full-size workloads compare sampled query rows
(each row of softmax attention is independent, so a sampled row is an exact
check of that row).
"""

import numpy as np
import pytest
import torch

from gpu_helpers import MASS_TOL, O_TOL, dev, host, max_abs
from oracle import joint_attention, segment_masses
from paper_2609_32415_amd import synth

pytestmark = pytest.mark.gpu

ops = None


@pytest.fixture(scope="module", autouse=True)
def _ops():
    global ops
    from paper_2609_32415_amd import ops as _o

    ops = _o
    yield


def _inputs(dtype, d, n_ref, n_tgt, B=1, H=2, seed=7, bias=True):
    base = "tiny" if dtype == "f32" else "single_ref"
    w = synth.workload(base, batch=B, heads=H, head_dim=d, n_ref=n_ref, n_tgt=n_tgt, seed=seed,
                       key_bias=bias and H > 1, cache_noise=0.01)
    x = synth.block_inputs(w)
    x.update({f"{k}_cache": v for k, v in synth.stale_cache(w, x).items()})
    return w, x


def _oracle(x, qset, use_cache, scale=None):
    kr = x["k_ref_cache"] if use_cache else x["k_ref"]
    vr = x["v_ref_cache"] if use_cache else x["v_ref"]
    n_ref = x["k_ref"].shape[2]
    res = {"tgt": joint_attention(x["q_tgt"], kr, vr, x["k_tgt"], x["v_tgt"], scale)}
    if qset == "all" and n_ref > 0:
        res["ref"] = joint_attention(x["q_ref"], kr, vr, x["k_tgt"], x["v_tgt"], scale)
    return res


def _gpu(x, dtype, qset, kvsrc, **kw):
    t = {k: dev(v, dtype) for k, v in x.items()}
    n_ref = x["k_ref"].shape[2]
    out = ops.joint_attn(
        t["q_tgt"], t["k_tgt"], t["v_tgt"], q_ref=t["q_ref"], k_ref=t["k_ref"], v_ref=t["v_ref"],
        k_cache=t["k_ref_cache"], v_cache=t["v_ref_cache"], qset=qset, kvsrc=kvsrc, n_ref=n_ref,
        lse=True, ref_mass_refq=True, **kw,
    )
    torch.cuda.synchronize()
    return out


SMALL = [
    # dtype, d, n_ref, n_tgt, B, H
    ("bf16", 128, 200, 333, 2, 3),
    ("bf16", 128, 64, 128, 1, 2),
    ("bf16", 128, 1, 1, 1, 2),
    ("bf16", 128, 129, 257, 1, 2),
    ("bf16", 128, 0, 130, 1, 2),
    ("bf16", 64, 200, 333, 1, 3),
    ("f32", 64, 256, 256, 1, 2),
    ("f32", 64, 100, 77, 2, 2),
    ("f32", 128, 70, 90, 1, 2),
    ("f32", 64, 0, 65, 1, 1),
]
MODES = [("target", "fresh"), ("target", "cache"), ("all", "fresh"), ("all", "cache")]


@pytest.mark.parametrize("case", SMALL, ids=lambda c: "-".join(map(str, c)))
@pytest.mark.parametrize("mode", MODES, ids=lambda m: "/".join(m))
def test_small_parity_all_elements(case, mode):
    dtype, d, n_ref, n_tgt, B, H = case
    qset, kvsrc = mode
    print(f"case {case} mode {mode}", flush=True)
    _, x = _inputs(dtype, d, n_ref, n_tgt, B, H)
    got = _gpu(x, dtype, qset, kvsrc)
    ref = _oracle(x, qset, kvsrc == "cache")
    assert max_abs(host(got.o_tgt), ref["tgt"]["o"]) <= O_TOL[dtype]
    assert max_abs(host(got.ref_mass), ref["tgt"]["ref_mass"]) <= MASS_TOL[dtype]
    lse = host(got.lse)
    assert max_abs(lse[..., 1], ref["tgt"]["lse_all"]) <= 1e-3
    if n_ref > 0:
        assert max_abs(lse[..., 0], ref["tgt"]["lse_ref"]) <= 1e-3
    else:
        assert np.all(np.isneginf(lse[..., 0]))
        assert np.all(host(got.ref_mass) == 0.0)
    m = host(got.ref_mass)
    assert np.all((m >= 0) & (m <= 1))
    if qset == "all" and n_ref > 0:
        assert max_abs(host(got.o_ref), ref["ref"]["o"]) <= O_TOL[dtype]
        assert max_abs(host(got.ref_mass_refq), ref["ref"]["ref_mass"]) <= MASS_TOL[dtype]


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("bf16", 64), ("f32", 64)])
@pytest.mark.parametrize("decision", [0, 1, 2], ids=["REUSE", "REACTIVATE", "COMPUTE"])
def test_device_mode_follows_decision_word(dtype, d, decision):
    print(f"device mode {dtype} d{d} decision {decision}", flush=True)
    _, x = _inputs(dtype, d, 150, 190, 1, 2)
    sentinel = 7.0
    o_ref = torch.full((1, 2, 150, d), sentinel, dtype=torch.bfloat16 if dtype == "bf16" else torch.float32, device="cuda:0")
    dec = torch.tensor([decision], dtype=torch.int32, device="cuda:0")
    got = _gpu(x, dtype, "target", "device", decision=dec, o_ref=o_ref)
    use_cache = decision != 2
    ref = _oracle(x, "all", use_cache)
    assert max_abs(host(got.o_tgt), ref["tgt"]["o"]) <= O_TOL[dtype]
    assert max_abs(host(got.ref_mass), ref["tgt"]["ref_mass"]) <= MASS_TOL[dtype]
    if decision == 0:
        assert np.all(host(o_ref) == sentinel)  # reference rows skipped on a reused block
    else:
        assert max_abs(host(o_ref), ref["ref"]["o"]) <= O_TOL[dtype]


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("f32", 64)])
def test_invariants_rows_sum_to_one_and_indicator_gives_mass(dtype, d):
    _, x = _inputs(dtype, d, 190, 230, 1, 3)
    ones = dict(x, v_ref=np.ones_like(x["v_ref"]), v_tgt=np.ones_like(x["v_tgt"]))
    got = _gpu(ones, dtype, "all", "fresh")
    assert max_abs(host(got.o_tgt), 1.0) <= (O_TOL["bf16"] if dtype == "bf16" else 1e-6)
    assert max_abs(host(got.o_ref), 1.0) <= (O_TOL["bf16"] if dtype == "bf16" else 1e-6)
    ind = dict(x, v_ref=np.ones_like(x["v_ref"]), v_tgt=np.zeros_like(x["v_tgt"]))
    got = _gpu(ind, dtype, "target", "fresh")
    o = host(got.o_tgt)
    m = host(got.ref_mass)
    assert max_abs(o, np.broadcast_to(m[..., None], o.shape)) <= (1e-2 if dtype == "bf16" else 1e-6)


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("f32", 64)])
def test_unchanged_cache_equals_full_fresh_target_rows(dtype, d):
    """Reuse with cache == fresh reproduces the full-fresh target rows bit for bit."""
    _, x = _inputs(dtype, d, 200, 260, 1, 2)
    same = dict(x, k_ref_cache=x["k_ref"], v_ref_cache=x["v_ref"])
    # Without key splits both launches reduce each target row in the same order.
    reuse = _gpu(same, dtype, "target", "cache", workspace=False)
    full = _gpu(same, dtype, "all", "fresh", workspace=False)
    assert torch.equal(reuse.o_tgt, full.o_tgt)
    assert torch.equal(reuse.ref_mass, full.ref_mass)


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("f32", 64)])
def test_mass_outputs_do_not_change_o_and_runs_are_deterministic(dtype, d):
    _, x = _inputs(dtype, d, 130, 300, 1, 2)
    t = {k: dev(v, dtype) for k, v in x.items()}
    kw = dict(k_ref=t["k_ref"], v_ref=t["v_ref"], qset="target", kvsrc="fresh")
    a = ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], ref_mass=False, lse=False, **kw)
    b = ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], ref_mass=True, lse=True, **kw)
    c = ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], ref_mass=True, lse=True, **kw)
    torch.cuda.synchronize()
    assert torch.equal(a.o_tgt, b.o_tgt)
    assert torch.equal(b.o_tgt, c.o_tgt) and torch.equal(b.ref_mass, c.ref_mass) and torch.equal(b.lse, c.lse)


# Shapes whose launches the host splits into key chunks of 4-5 key tiles (few
# query tiles, many key tiles): chunks wholly inside the reference segment, a
# chunk that spans the segment boundary through a ragged reference tile, a
# chunk that ends exactly at the boundary (576 = 9 key tiles), no reference.
SPLIT = [
    # d, n_ref, n_tgt, H
    (128, 1000, 100, 2),
    (128, 576, 576, 2),
    (128, 700, 300, 3),
    (128, 0, 1100, 2),
    (64, 1000, 100, 2),
]


def _workspace_bytes(n_ref, n_tgt, H, d, qset, kvsrc):
    from paper_2609_32415_amd import _lib as L

    desc = L.ra_attn_desc(1, H, d, n_ref, n_tgt, L.RA_BF16, 0.0, {"target": 0, "all": 1}[qset],
                          {"fresh": 0, "cache": 1, "device": 2, "segments": 3}[kvsrc])
    return L.refadapt_joint_attn_workspace_size(desc)


@pytest.mark.parametrize("case", SPLIT, ids=lambda c: "-".join(map(str, c)))
@pytest.mark.parametrize("mode", [("target", "cache"), ("all", "fresh")], ids=lambda m: "/".join(m))
def test_key_split_parity_all_elements(case, mode):
    d, n_ref, n_tgt, H = case
    qset, kvsrc = mode
    print(f"key split bf16 d{d} n_ref {n_ref} n_tgt {n_tgt} H {H} {qset}/{kvsrc}", flush=True)
    assert _workspace_bytes(n_ref, n_tgt, H, d, qset, kvsrc) > 0, "the launch should split key ranges"
    _, x = _inputs("bf16", d, n_ref, n_tgt, 1, H)
    ref = _oracle(x, qset, kvsrc == "cache")
    got = _gpu(x, "bf16", qset, kvsrc)
    whole = _gpu(x, "bf16", qset, kvsrc, workspace=False)
    assert max_abs(host(got.o_tgt), ref["tgt"]["o"]) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), ref["tgt"]["ref_mass"]) <= MASS_TOL["bf16"]
    lse = host(got.lse)
    if n_ref > 0:
        assert max_abs(lse[..., 0], ref["tgt"]["lse_ref"]) <= 1e-3
    else:
        assert np.all(np.isneginf(lse[..., 0]))
        assert np.all(host(got.ref_mass) == 0.0)
    assert max_abs(lse[..., 1], ref["tgt"]["lse_all"]) <= 1e-3
    assert max_abs(host(got.o_tgt), host(whole.o_tgt)) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), host(whole.ref_mass)) <= MASS_TOL["bf16"]
    if qset == "all" and n_ref > 0:
        assert max_abs(host(got.o_ref), ref["ref"]["o"]) <= O_TOL["bf16"]
        assert max_abs(host(got.ref_mass_refq), ref["ref"]["ref_mass"]) <= MASS_TOL["bf16"]


@pytest.mark.parametrize("mode", [("target", "cache"), ("all", "fresh")], ids=lambda m: "/".join(m))
def test_whole_and_split_tiles_spread_over_heads(mode):
    """A plan with whole rounds and split tiles whose count does not divide evenly over the
    heads (5 heads; 60 or 62 query tiles each, 256 run whole, 44 or 54 split): the split
    launch equals the unsplit one on every row, and sampled rows of every head's whole
    and split tiles match the oracle."""
    qset, kvsrc = mode
    d, n_ref, n_tgt, H = 128, 300, 15360, 5
    print(f"whole+split plan bf16 n_ref {n_ref} n_tgt {n_tgt} H {H} {qset}/{kvsrc}", flush=True)
    assert _workspace_bytes(n_ref, n_tgt, H, d, qset, kvsrc) > 0, "the launch should split key ranges"
    _, x = _inputs("bf16", d, n_ref, n_tgt, 1, H, seed=23)
    got = _gpu(x, "bf16", qset, kvsrc)
    whole = _gpu(x, "bf16", qset, kvsrc, workspace=False)
    assert max_abs(host(got.o_tgt), host(whole.o_tgt)) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), host(whole.ref_mass)) <= MASS_TOL["bf16"]
    if qset == "all":
        assert max_abs(host(got.o_ref), host(whole.o_ref)) <= O_TOL["bf16"]
    # the last 12 target tiles of a head hold its split tiles under either plan
    rng = np.random.default_rng(5)
    rows = np.sort(np.concatenate([rng.choice(n_tgt - 12 * 256, 24, replace=False),
                                   n_tgt - 12 * 256 + rng.choice(12 * 256, 40, replace=False)]))
    kr = x["k_ref_cache"] if kvsrc == "cache" else x["k_ref"]
    vr = x["v_ref_cache"] if kvsrc == "cache" else x["v_ref"]
    ref = joint_attention(x["q_tgt"][:, :, rows], kr, vr, x["k_tgt"], x["v_tgt"])
    assert max_abs(host(got.o_tgt)[:, :, rows], ref["o"]) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass)[:, :, rows], ref["ref_mass"]) <= MASS_TOL["bf16"]


@pytest.mark.parametrize("decision", [0, 1, 2], ids=["REUSE", "REACTIVATE", "COMPUTE"])
def test_key_split_device_mode_follows_decision_word(decision):
    """Under RA_KV_DEVICE each decision has its own split plan, chosen on the device."""
    print(f"key split device mode decision {decision}", flush=True)
    n_ref, n_tgt, H = 1000, 100, 2
    assert _workspace_bytes(n_ref, n_tgt, H, 128, "target", "device") > 0
    _, x = _inputs("bf16", 128, n_ref, n_tgt, 1, H)
    sentinel = 7.0
    o_ref = torch.full((1, H, n_ref, 128), sentinel, dtype=torch.bfloat16, device="cuda:0")
    dec = torch.tensor([decision], dtype=torch.int32, device="cuda:0")
    got = _gpu(x, "bf16", "target", "device", decision=dec, o_ref=o_ref)
    ref = _oracle(x, "all", decision != 2)
    assert max_abs(host(got.o_tgt), ref["tgt"]["o"]) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), ref["tgt"]["ref_mass"]) <= MASS_TOL["bf16"]
    if decision == 0:
        assert np.all(host(o_ref) == sentinel)
    else:
        assert max_abs(host(o_ref), ref["ref"]["o"]) <= O_TOL["bf16"]


def test_custom_scale_and_strided_views():
    """A non-default scale and non-contiguous [B, S, H, d] views (head-interleaved layout)."""
    _, x = _inputs("bf16", 128, 96, 200, 1, 2)
    ref = _oracle(x, "target", False, scale=0.05)
    t = {k: dev(v, "bf16").transpose(1, 2).contiguous().transpose(1, 2) for k, v in x.items()}
    assert t["q_tgt"].stride(1) == 128
    got = ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], k_ref=t["k_ref"], v_ref=t["v_ref"], scale=0.05)
    torch.cuda.synchronize()
    assert max_abs(host(got.o_tgt), ref["tgt"]["o"]) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), ref["tgt"]["ref_mass"]) <= MASS_TOL["bf16"]


def _layout(a, kind):
    """A device view of ``a`` ([B, H, S, d], bf16) in one of three memory layouts:
    contiguous, head-interleaved [B, S, H, d], or rows padded to 4 d elements."""
    t = dev(a, "bf16")
    if kind == "bshd":
        return t.transpose(1, 2).contiguous().transpose(1, 2)
    if kind == "pad":
        B, H, S, d = t.shape
        buf = torch.zeros((B, H, S, 4 * d), dtype=t.dtype, device=t.device)
        buf[..., d:2 * d] = t
        return buf[..., d:2 * d]
    return t


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("mode", [("target", "cache"), ("all", "fresh"), ("all", "cache")], ids=lambda m: "/".join(m))
def test_mixed_layouts_per_tensor(d, mode):
    """Every K/V tensor with its own row stride (contiguous, head-interleaved, padded rows),
    ragged reference and target tails: each view's tiles are addressed with its own stride."""
    qset, kvsrc = mode
    _, x = _inputs("bf16", d, 130, 333, B=2, H=3)
    ref = _oracle(x, qset, kvsrc == "cache")
    kinds = {"q_tgt": "pad", "k_tgt": "bshd", "v_tgt": "plain", "q_ref": "bshd", "k_ref": "pad", "v_ref": "bshd",
             "k_ref_cache": "bshd", "v_ref_cache": "pad"}
    t = {k: _layout(x[k], v) for k, v in kinds.items()}
    assert t["k_ref"].stride(2) == 4 * d and t["k_tgt"].stride(2) == 3 * d and t["v_tgt"].stride(2) == d
    got = ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], q_ref=t["q_ref"], k_ref=t["k_ref"], v_ref=t["v_ref"],
                         k_cache=t["k_ref_cache"], v_cache=t["v_ref_cache"], qset=qset, kvsrc=kvsrc, n_ref=130,
                         lse=True)
    torch.cuda.synchronize()
    assert max_abs(host(got.o_tgt), ref["tgt"]["o"]) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), ref["tgt"]["ref_mass"]) <= MASS_TOL["bf16"]
    if qset == "all":
        assert max_abs(host(got.o_ref), ref["ref"]["o"]) <= O_TOL["bf16"]


def _nan_padded(a, pad=64):
    """A device view of ``a`` ([B, H, S, d], bf16) whose buffer holds ``pad`` NaN rows after the
    S rows of every head: any load past a tensor's last row would poison the result."""
    t = dev(a, "bf16")
    B, H, S, d = t.shape
    buf = torch.full((B, H, S + pad, d), float("nan"), dtype=t.dtype, device=t.device)
    buf[:, :, :S] = t
    return buf[:, :, :S]


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("mode", [("target", "cache"), ("all", "fresh")], ids=lambda m: "/".join(m))
def test_ragged_tiles_never_read_past_the_last_row(d, mode):
    """Every K/V view sits in a buffer with NaN rows after its last row; ragged last tiles must
    load those rows as zeros (buffer range check), so O, mass and lse stay finite and exact."""
    qset, kvsrc = mode
    _, x = _inputs("bf16", d, 130, 77, B=1, H=2)
    ref = _oracle(x, qset, kvsrc == "cache")
    t = {k: (_nan_padded(v) if k[0] in "kv" else dev(v, "bf16")) for k, v in x.items()}
    got = ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], q_ref=t["q_ref"], k_ref=t["k_ref"], v_ref=t["v_ref"],
                         k_cache=t["k_ref_cache"], v_cache=t["v_ref_cache"], qset=qset, kvsrc=kvsrc, n_ref=130,
                         lse=True, workspace=False)
    torch.cuda.synchronize()
    assert np.isfinite(host(got.o_tgt)).all() and np.isfinite(host(got.lse)).all()
    assert max_abs(host(got.o_tgt), ref["tgt"]["o"]) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), ref["tgt"]["ref_mass"]) <= MASS_TOL["bf16"]
    if qset == "all":
        assert max_abs(host(got.o_ref), ref["ref"]["o"]) <= O_TOL["bf16"]


# Largest K/V row stride (elements) the bf16 attention accepts: the byte offsets of a 64-row
# key tile stay below 2^31 (the library rejects larger strides with RA_EUNSUPPORTED).
MAX_KV_ROW_STRIDE = (1 << 24) - 8


def _sparse_rows(a, stride):
    """A device view of ``a`` ([1, H, S, d], bf16) whose rows lie ``stride`` elements apart in a
    NaN-filled buffer: any element read outside a row poisons the result."""
    _, H, S, d = a.shape
    buf = torch.full((1, H, S, stride), float("nan"), dtype=torch.bfloat16, device="cuda:0")
    view = buf[..., :d]
    view.copy_(dev(a, "bf16"))
    return view


# d, n_ref, heads, key-split: two heads whose second starts more than 4 GiB into each buffer, run
# whole; one head with 10 + 2 key tiles, cut into key chunks by the workspace plan.
STRIDE_CASES = [(128, 130, 2, False), (64, 130, 2, False), (128, 578, 1, True)]


@pytest.mark.parametrize("case", STRIDE_CASES, ids=lambda c: f"d{c[0]}-nref{c[1]}-H{c[2]}-{'split' if c[3] else 'whole'}")
@pytest.mark.parametrize("mode", [("all", "fresh"), ("target", "cache")], ids=lambda m: "/".join(m))
def test_largest_kv_row_stride(case, mode):
    """Every K/V view at the largest accepted row stride (a 64-row key tile spans 2 GiB), with
    ragged reference and target tails: the 32-bit tile offsets and the 64-bit head, tile and
    key-chunk bases address the right rows; any other element read is NaN."""
    d, n_ref, H, split = case
    qset, kvsrc = mode
    n_tgt = 70
    print(f"largest K/V row stride {MAX_KV_ROW_STRIDE} bf16 d {d} n_ref {n_ref} H {H} {qset}/{kvsrc}", flush=True)
    if split:
        assert _workspace_bytes(n_ref, n_tgt, H, d, qset, kvsrc) > 0, "the launch should split key ranges"
    _, x = _inputs("bf16", d, n_ref, n_tgt, B=1, H=H)
    ref = _oracle(x, qset, kvsrc == "cache")
    kv = ["k_tgt", "v_tgt"] + (["k_ref_cache", "v_ref_cache"] if kvsrc == "cache" else ["k_ref", "v_ref"])
    t = {k: (_sparse_rows(v, MAX_KV_ROW_STRIDE) if k in kv else dev(v, "bf16")) for k, v in x.items()}
    assert t[kv[0]].stride(2) == MAX_KV_ROW_STRIDE
    if H > 1:
        assert t[kv[2]].stride(1) * 2 > 1 << 32
    got = ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], q_ref=t["q_ref"],
                         k_ref=t["k_ref"] if kvsrc == "fresh" else None,
                         v_ref=t["v_ref"] if kvsrc == "fresh" else None,
                         k_cache=t["k_ref_cache"] if kvsrc == "cache" else None,
                         v_cache=t["v_ref_cache"] if kvsrc == "cache" else None,
                         qset=qset, kvsrc=kvsrc, n_ref=n_ref, lse=True, workspace=None if split else False)
    torch.cuda.synchronize()
    del t
    torch.cuda.empty_cache()
    assert np.isfinite(host(got.o_tgt)).all() and np.isfinite(host(got.lse)).all()
    assert max_abs(host(got.o_tgt), ref["tgt"]["o"]) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), ref["tgt"]["ref_mass"]) <= MASS_TOL["bf16"]
    if qset == "all":
        assert max_abs(host(got.o_ref), ref["ref"]["o"]) <= O_TOL["bf16"]


def test_largest_kv_row_stride_segments():
    """Reference segments alternating between fresh and cached K/V, every K/V view at the
    largest accepted row stride and the second head more than 4 GiB into each buffer: a load
    cursor that moves between the two sources keeps its row (only the base pointer changes)."""
    d, sizes, n_tgt, H, cached = 128, (64, 64, 2), 70, 2, (True, False, True)
    print(f"largest K/V row stride {MAX_KV_ROW_STRIDE} segments {sizes} cached {cached}", flush=True)
    _, x = _inputs("bf16", d, sum(sizes), n_tgt, 1, H)
    kr, vr, ends = _seg_oracle_inputs(x, sizes, cached)
    big = ("k_tgt", "v_tgt", "k_ref", "v_ref", "k_ref_cache", "v_ref_cache")
    t = {k: (_sparse_rows(v, MAX_KV_ROW_STRIDE) if k in big else dev(v, "bf16")) for k, v in x.items()}
    got = ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], k_ref=t["k_ref"], v_ref=t["v_ref"],
                         k_cache=t["k_ref_cache"], v_cache=t["v_ref_cache"], qset="target", kvsrc="segments",
                         n_ref=sum(sizes), seg_end=ends, seg_cache=cached, seg_mass=True, workspace=False)
    torch.cuda.synchronize()
    del t
    torch.cuda.empty_cache()
    ref = joint_attention(x["q_tgt"], kr, vr, x["k_tgt"], x["v_tgt"])
    assert np.isfinite(host(got.o_tgt)).all()
    assert max_abs(host(got.o_tgt), ref["o"]) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), ref["ref_mass"]) <= MASS_TOL["bf16"]
    assert max_abs(host(got.seg_mass), segment_masses(x["q_tgt"], kr, x["k_tgt"], ends)) <= MASS_TOL["bf16"]


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("bf16", 64), ("f32", 64)])
@pytest.mark.parametrize("kvsrc,decision", [("cache", None), ("device", 1), ("device", 2), ("fresh", None)],
                         ids=["cache", "device-REACTIVATE", "device-COMPUTE", "fresh"])
def test_cached_reference_queries(dtype, d, kvsrc, decision):
    """q_cache (reference queries of the cached state) replaces q_ref exactly where reference
    queries attend over the cached K/V: ALL/CACHE and REACTIVATE; COMPUTE and FRESH ignore it."""
    print(f"q_cache {dtype} d{d} {kvsrc} {decision}", flush=True)
    _, x = _inputs(dtype, d, 150, 190, 1, 2)
    q_stale = synth.round_to_dtype(x["q_ref"] + 0.5 * np.random.default_rng(5).standard_normal(x["q_ref"].shape),
                                   dtype)
    t = {k: dev(v, dtype) for k, v in x.items()}
    dec = None if decision is None else torch.tensor([decision], dtype=torch.int32, device="cuda:0")
    got = ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], q_ref=t["q_ref"], k_ref=t["k_ref"], v_ref=t["v_ref"],
                         k_cache=t["k_ref_cache"], v_cache=t["v_ref_cache"], q_cache=dev(q_stale, dtype),
                         qset="all", kvsrc=kvsrc, decision=dec, ref_mass_refq=True)
    torch.cuda.synchronize()
    use_cache = kvsrc == "cache" or decision == 1
    kr = x["k_ref_cache"] if use_cache else x["k_ref"]
    vr = x["v_ref_cache"] if use_cache else x["v_ref"]
    refr = joint_attention(q_stale if use_cache else x["q_ref"], kr, vr, x["k_tgt"], x["v_tgt"])
    ref = joint_attention(x["q_tgt"], kr, vr, x["k_tgt"], x["v_tgt"])
    assert max_abs(host(got.o_ref), refr["o"]) <= O_TOL[dtype]
    assert max_abs(host(got.ref_mass_refq), refr["ref_mass"]) <= MASS_TOL[dtype]
    assert max_abs(host(got.o_tgt), ref["o"]) <= O_TOL[dtype]
    assert max_abs(host(got.ref_mass), ref["ref_mass"]) <= MASS_TOL[dtype]


FULL = [("single_ref", "target", "cache"), ("single_ref", "all", "fresh"), ("single_ref", "all", "cache"),
        ("multi_ref", "target", "cache"), ("multi_ref", "all", "fresh"), ("multi_ref", "all", "cache"),
        ("video", "target", "cache"), ("video", "all", "fresh"), ("video", "all", "cache"),
        ("ref8", "target", "cache"), ("ref8", "all", "fresh")]
_FULL_CACHE = {}
# eight 4096-token reference images plus 256 text tokens (the largest reference count swept)
_NAMED = {"ref8": ("single_ref", {"n_ref": 8 * 4096 + 256})}


def _full_inputs(name):
    if name not in _FULL_CACHE:
        _FULL_CACHE.clear()
        base, over = _NAMED.get(name, (name, {}))
        w = synth.workload(base, **over)
        x = synth.block_inputs(w)
        x.update({f"{k}_cache": v for k, v in synth.stale_cache(w, x).items()})
        _FULL_CACHE[name] = (w, x)
    return _FULL_CACHE[name]


@pytest.mark.parametrize("name,qset,kvsrc", FULL, ids=lambda v: str(v))
def test_full_size_sampled_rows(name, qset, kvsrc):
    print(f"full-size {name} {qset}/{kvsrc}", flush=True)
    w, x = _full_inputs(name)
    got = _gpu(x, "bf16", qset, kvsrc)
    use_cache = kvsrc == "cache"
    kr = x["k_ref_cache"] if use_cache else x["k_ref"]
    vr = x["v_ref_cache"] if use_cache else x["v_ref"]
    rows = synth.sample_rows(w.n_tgt, 48, 3)
    ref = joint_attention(x["q_tgt"][:, :, rows], kr, vr, x["k_tgt"], x["v_tgt"])
    assert max_abs(host(got.o_tgt[:, :, rows]), ref["o"]) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass[:, :, rows]), ref["ref_mass"]) <= MASS_TOL["bf16"]
    m = host(got.ref_mass)
    assert np.all((m >= 0) & (m <= 1))
    lse = host(got.lse[:, :, rows])
    assert max_abs(lse[..., 0], ref["lse_ref"]) <= 1e-3 and max_abs(lse[..., 1], ref["lse_all"]) <= 1e-3
    if qset == "all":
        rr = synth.sample_rows(w.n_ref, 48, 4)
        refr = joint_attention(x["q_ref"][:, :, rr], kr, vr, x["k_tgt"], x["v_tgt"])
        assert max_abs(host(got.o_ref[:, :, rr]), refr["o"]) <= O_TOL["bf16"]
        assert max_abs(host(got.ref_mass_refq[:, :, rr]), refr["ref_mass"]) <= MASS_TOL["bf16"]
        mr = host(got.ref_mass_refq)
        assert np.all((mr >= 0) & (mr <= 1))


def _jump_inputs(d, pattern, n_ref=600, n_tgt=300, H=2, seed=11):
    """Inputs whose row max rises sharply at chosen keys: every query gets a component c along
    a unit direction u and chosen keys get B u, so their logits stand far above the rest.
    ``spikes``: keys at offset 10 of reference tile 3 (first key block of a tile), offset 48 of
    reference tile 5 (second key block) and offset 56 of target tile 1 (after the reference
    statistics are frozen), each higher than the last; ``ramp``: every key gets a component
    growing with its index, so the max rises at every tile; ``huge``: one spike far beyond
    the fp32 range of 2^(logit - running max)."""
    _, x = _inputs("bf16", d, n_ref, n_tgt, 1, H, seed=seed, bias=False)
    rng = np.random.default_rng(seed)
    u = rng.standard_normal(d)
    u /= np.linalg.norm(u)
    x = {k: v.astype(np.float64) for k, v in x.items()}
    for k in ("q_tgt", "q_ref"):
        x[k] = x[k] + 2.0 * u
    n = n_ref + n_tgt
    k_all = np.concatenate([x["k_ref"], x["k_tgt"]], axis=2)
    if pattern == "spikes":
        for idx, b in ((3 * 64 + 10, 100.0), (5 * 64 + 48, 200.0), (n_ref + 64 + 56, 400.0)):
            k_all[:, :, idx, :] += b * u
    elif pattern == "ramp":
        k_all += (np.arange(n) / n * 400.0)[None, None, :, None] * u
    else:  # huge: about 2^700 above the running max in the exp2 domain
        k_all[:, :, 7 * 64 + 50, :] += 2000.0 * u
    x["k_ref"], x["k_tgt"] = k_all[:, :, :n_ref], k_all[:, :, n_ref:]
    x["k_ref_cache"] = x["k_ref"]
    x["v_ref_cache"] = x["v_ref"]
    return {k: synth.round_to_dtype(v, "bf16") for k, v in x.items()}


def _dominant_key_inputs(b, vscale, d=128, n_ref=300, n_tgt=400, H=2, seed=41):
    """One target key per head scores about 2b/sqrt(d) log2 units above the reference keys
    (every query gets a component 2u, the key b u): far enough to dominate its rows, not far
    enough to move the running max (its probability stays below the rescale bound), so the
    bf16 rounding of that one probability decides the output. Its value row is +-vscale."""
    _, x = _inputs("bf16", d, n_ref, n_tgt, 1, H, seed=seed, bias=False)
    rng = np.random.default_rng(seed)
    u = rng.standard_normal(d)
    u /= np.linalg.norm(u)
    x = {k: v.astype(np.float64) for k, v in x.items()}
    for k in ("q_tgt", "q_ref"):
        x[k] = x[k] + 2.0 * u
    idx = 2 * 64 + 17
    x["k_tgt"][:, :, idx, :] += b * u
    x["v_tgt"][:, :, idx, :] = vscale * np.sign(rng.standard_normal((1, H, d)))
    x["k_ref_cache"], x["v_ref_cache"] = x["k_ref"], x["v_ref"]
    return {k: synth.round_to_dtype(v, "bf16") for k, v in x.items()}


@pytest.mark.parametrize("b", [30.0, 40.0])
@pytest.mark.parametrize("mode", [("target", "fresh"), ("all", "fresh")], ids=lambda m: "/".join(m))
@pytest.mark.parametrize("split", [True, False], ids=["split", "whole"])
def test_dominant_key_below_the_rescale_bound(b, mode, split):
    """A dominant key whose probability is not rounded at 1 (the running max stays at the
    reference keys): outputs of magnitude up to 2.5 stay within the 1e-2 bar, which holds
    because O is divided by the sum of the rounded probabilities it accumulated."""
    qset, kvsrc = mode
    print(f"dominant key b={b} {qset}/{kvsrc} split={split}", flush=True)
    x = _dominant_key_inputs(b, 2.5)
    got = _gpu(x, "bf16", qset, kvsrc, **({} if split else {"workspace": False}))
    ref = _oracle(x, qset, False)
    err = max_abs(host(got.o_tgt), ref["tgt"]["o"])
    print(f"  max|o| {np.abs(ref['tgt']['o']).max():.3f} max|dO| {err:.5f}", flush=True)
    assert err <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), ref["tgt"]["ref_mass"]) <= MASS_TOL["bf16"]
    if qset == "all":
        assert max_abs(host(got.o_ref), ref["ref"]["o"]) <= O_TOL["bf16"]


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("pattern", ["spikes", "ramp", "huge"])
@pytest.mark.parametrize("mode", [("target", "fresh"), ("all", "fresh")], ids=lambda m: "/".join(m))
@pytest.mark.parametrize("split", [True, False], ids=["split", "whole"])
def test_running_max_moves(d, pattern, mode, split):
    """The probabilities are formed against the running max and the max moves only when a
    lane's partial row sum leaves its bound; these inputs force every such path (first and
    second half of a tile, after the reference freeze, at every tile, with overflow)."""
    qset, kvsrc = mode
    print(f"running max d{d} {pattern} {qset}/{kvsrc} split={split}", flush=True)
    x = _jump_inputs(d, pattern)
    got = _gpu(x, "bf16", qset, kvsrc, **({} if split else {"workspace": False}))
    ref = _oracle(x, qset, False)
    assert np.all(np.isfinite(host(got.o_tgt)))
    assert max_abs(host(got.o_tgt), ref["tgt"]["o"]) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), ref["tgt"]["ref_mass"]) <= MASS_TOL["bf16"]
    lse = host(got.lse)
    # The lse bar scales with the logit magnitude here: the fp32 accumulation of q.k in the
    # MFMA carries a relative error, and these logits reach hundreds.
    tol = 1e-3 * max(1.0, float(np.abs(ref["tgt"]["lse_all"]).max()) / 100)
    assert max_abs(lse[..., 0], ref["tgt"]["lse_ref"]) <= tol
    assert max_abs(lse[..., 1], ref["tgt"]["lse_all"]) <= tol
    if qset == "all":
        assert max_abs(host(got.o_ref), ref["ref"]["o"]) <= O_TOL["bf16"]
        assert max_abs(host(got.ref_mass_refq), ref["ref"]["ref_mass"]) <= MASS_TOL["bf16"]


# Reference segments: d, segment sizes (rows of R), n_tgt, H, cached segments.
SEG_CASES = [
    (128, (128, 192, 37), 200, 2, (True, False, True)),
    (64, (64, 64, 64, 100), 150, 3, (False, True, False, True)),
    (128, (300,), 100, 2, (True,)),
    (128, (64,) * 8 + (40,), 128, 2, (True, False) * 4 + (True,)),
    (128, (256, 256), 333, 2, (False, False)),
    (128, (64,) * 15 + (30,), 100, 2, (True, False, False) * 5 + (True,)),  # RA_MAX_SEG segments
]


def _seg_oracle_inputs(x, sizes, cached):
    """Reference K/V assembled per segment from the cached or the fresh rows."""
    ends = np.cumsum(sizes)
    kr, vr = x["k_ref"].copy(), x["v_ref"].copy()
    for lo, hi, c in zip(np.concatenate([[0], ends[:-1]]), ends, cached):
        if c:
            kr[..., lo:hi, :] = x["k_ref_cache"][..., lo:hi, :]
            vr[..., lo:hi, :] = x["v_ref_cache"][..., lo:hi, :]
    return kr, vr, ends.tolist()


@pytest.mark.parametrize("case", SEG_CASES, ids=lambda c: f"d{c[0]}-{len(c[1])}seg")
@pytest.mark.parametrize("qset", ["target", "all"])
def test_reference_segments_parity(case, qset):
    """RA_KV_SEGMENTS: each segment reads its own K/V source; per-segment masses match the
    oracle and add up to the reference mass."""
    d, sizes, n_tgt, H, cached = case
    print(f"segments d{d} sizes {sizes} cached {cached} {qset}", flush=True)
    _, x = _inputs("bf16", d, sum(sizes), n_tgt, 1, H)
    kr, vr, ends = _seg_oracle_inputs(x, sizes, cached)
    got = _gpu(x, "bf16", qset, "segments", seg_end=ends, seg_cache=cached, seg_mass=True)
    ref = joint_attention(x["q_tgt"], kr, vr, x["k_tgt"], x["v_tgt"])
    sm = segment_masses(x["q_tgt"], kr, x["k_tgt"], ends)
    assert max_abs(host(got.o_tgt), ref["o"]) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), ref["ref_mass"]) <= MASS_TOL["bf16"]
    lse = host(got.lse)
    assert max_abs(lse[..., 0], ref["lse_ref"]) <= 1e-3
    assert max_abs(lse[..., 1], ref["lse_all"]) <= 1e-3
    assert max_abs(host(got.seg_mass), sm) <= MASS_TOL["bf16"]
    assert max_abs(host(got.seg_mass).sum(-1), host(got.ref_mass)) <= 1e-5
    if qset == "all":
        rr = joint_attention(x["q_ref"], kr, vr, x["k_tgt"], x["v_tgt"])
        assert max_abs(host(got.o_ref), rr["o"]) <= O_TOL["bf16"]
        assert max_abs(host(got.ref_mass_refq), rr["ref_mass"]) <= MASS_TOL["bf16"]


@pytest.mark.parametrize("kvsrc", ["fresh", "cache"])
def test_segment_mass_with_one_source(kvsrc):
    """seg_mass under RA_KV_FRESH / RA_KV_CACHE: all segments read that source; the output,
    mass and lse equal those of the same launch without segments."""
    sizes = (64, 128, 90)
    _, x = _inputs("bf16", 128, sum(sizes), 300, 1, 2)
    ends = np.cumsum(sizes).tolist()
    got = _gpu(x, "bf16", "target", kvsrc, seg_end=ends, seg_mass=True)
    plain = _gpu(x, "bf16", "target", kvsrc, workspace=False)
    use = kvsrc == "cache"
    kr = x["k_ref_cache"] if use else x["k_ref"]
    np.testing.assert_allclose(host(got.seg_mass), segment_masses(x["q_tgt"], kr, x["k_tgt"], ends),
                               atol=MASS_TOL["bf16"], rtol=0)
    assert max_abs(host(got.o_tgt), host(plain.o_tgt)) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), host(plain.ref_mass)) <= 1e-5


@pytest.mark.parametrize("qset", ["target", "all"])
def test_reference_segments_key_split(qset):
    """Per-segment sources without seg_mass may split key ranges: chunks that start inside a
    segment pick up its source; results match the oracle and the unsplit launch."""
    sizes, cached = (256, 384, 360), (True, False, True)
    assert _workspace_bytes(sum(sizes), 100, 2, 128, qset, "segments") > 0, "the launch should split key ranges"
    _, x = _inputs("bf16", 128, sum(sizes), 100, 1, 2)
    kr, vr, ends = _seg_oracle_inputs(x, sizes, cached)
    got = _gpu(x, "bf16", qset, "segments", seg_end=ends, seg_cache=cached)
    whole = _gpu(x, "bf16", qset, "segments", seg_end=ends, seg_cache=cached, workspace=False)
    ref = joint_attention(x["q_tgt"], kr, vr, x["k_tgt"], x["v_tgt"])
    assert max_abs(host(got.o_tgt), ref["o"]) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), ref["ref_mass"]) <= MASS_TOL["bf16"]
    lse = host(got.lse)
    assert max_abs(lse[..., 0], ref["lse_ref"]) <= 1e-3 and max_abs(lse[..., 1], ref["lse_all"]) <= 1e-3
    assert max_abs(host(got.o_tgt), host(whole.o_tgt)) <= O_TOL["bf16"]
    if qset == "all":
        rr = joint_attention(x["q_ref"], kr, vr, x["k_tgt"], x["v_tgt"])
        assert max_abs(host(got.o_ref), rr["o"]) <= O_TOL["bf16"]


def _seg_workspace_bytes(n_ref, n_tgt, H, d, qset, kvsrc, n_seg):
    from paper_2609_32415_amd import _lib as L

    desc = L.ra_attn_desc(1, H, d, n_ref, n_tgt, L.RA_BF16, 0.0, {"target": 0, "all": 1}[qset],
                          {"fresh": 0, "cache": 1, "segments": 3}[kvsrc])
    return L.refadapt_joint_attn_seg_workspace_size(desc, n_seg)


SEG_SPLIT = [
    # segment sizes, cached segments, n_tgt
    ((256, 384, 360), (True, False, True), 100),
    ((128,) * 8 + (40,), (True, False) * 4 + (True,), 100),
    ((1000,), (False,), 1100),
    ((64,) * 15 + (30,), (False, True) * 8, 100),  # RA_MAX_SEG segments, mostly one key tile each
]


@pytest.mark.parametrize("case", SEG_SPLIT, ids=lambda c: f"{len(c[0])}seg-{c[2]}")
@pytest.mark.parametrize("qset", ["target", "all"])
@pytest.mark.parametrize("d", [128, 64])
def test_segment_mass_key_split(case, qset, d):
    """Per-segment masses with key splits: a chunk that starts or ends inside a segment
    records a partial log-sum-exp for it, the merge combines the chunks that overlap each
    segment; masses match the oracle and the whole-tile launch and add up to the reference
    mass."""
    sizes, cached, n_tgt = case
    n_ref, n_seg = sum(sizes), len(sizes)
    print(f"segment masses with key splits d{d} sizes {sizes} n_tgt {n_tgt} {qset}", flush=True)
    assert _seg_workspace_bytes(n_ref, n_tgt, 2, d, qset, "segments", n_seg) > 0, "the launch should split"
    _, x = _inputs("bf16", d, n_ref, n_tgt, 1, 2, seed=31)
    kr, vr, ends = _seg_oracle_inputs(x, sizes, cached)
    got = _gpu(x, "bf16", qset, "segments", seg_end=ends, seg_cache=cached, seg_mass=True)
    whole = _gpu(x, "bf16", qset, "segments", seg_end=ends, seg_cache=cached, seg_mass=True, workspace=False)
    ref = joint_attention(x["q_tgt"], kr, vr, x["k_tgt"], x["v_tgt"])
    sm = segment_masses(x["q_tgt"], kr, x["k_tgt"], ends)
    assert max_abs(host(got.o_tgt), ref["o"]) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), ref["ref_mass"]) <= MASS_TOL["bf16"]
    lse = host(got.lse)
    assert max_abs(lse[..., 0], ref["lse_ref"]) <= 1e-3 and max_abs(lse[..., 1], ref["lse_all"]) <= 1e-3
    assert max_abs(host(got.seg_mass), sm) <= MASS_TOL["bf16"]
    assert max_abs(host(got.seg_mass).sum(-1), host(got.ref_mass)) <= 1e-5
    assert max_abs(host(got.seg_mass), host(whole.seg_mass)) <= 1e-5
    if qset == "all":
        rr = joint_attention(x["q_ref"], kr, vr, x["k_tgt"], x["v_tgt"])
        assert max_abs(host(got.o_ref), rr["o"]) <= O_TOL["bf16"]
        assert max_abs(host(got.ref_mass_refq), rr["ref_mass"]) <= MASS_TOL["bf16"]


def test_segment_mass_with_plain_workspace_runs_whole():
    """seg_mass with a workspace sized for the plain split runs whole query tiles (the
    per-segment partials do not fit): results equal the whole-tile launch bitwise."""
    from paper_2609_32415_amd import _lib as L

    sizes, cached = (256, 384, 360), (True, False, True)
    _, x = _inputs("bf16", 128, sum(sizes), 100, 1, 2, seed=31)
    _, _, ends = _seg_oracle_inputs(x, sizes, cached)
    desc = L.ra_attn_desc(1, 2, 128, sum(sizes), 100, L.RA_BF16, 0.0, 0, 3)
    plain = L.refadapt_joint_attn_workspace_size(desc)
    assert 0 < plain < L.refadapt_joint_attn_seg_workspace_size(desc, 3)
    ws = torch.empty(plain, dtype=torch.uint8, device="cuda")
    got = _gpu(x, "bf16", "target", "segments", seg_end=ends, seg_cache=cached, seg_mass=True, workspace=ws)
    whole = _gpu(x, "bf16", "target", "segments", seg_end=ends, seg_cache=cached, seg_mass=True, workspace=False)
    assert torch.equal(got.o_tgt, whole.o_tgt) and torch.equal(got.seg_mass, whole.seg_mass)


def _random_cases(n=40, seed=2024, large=False, first=0):
    """Seeded random configurations: head dim, ragged reference/target sizes (including
    single rows and multiples of the 64-row tile), heads, batch, query set, K/V source,
    segments (with random tile-aligned boundaries and cache flags) and key splits. ``large``:
    up to 4000 reference and 2500 target rows, 8 heads and 16 segments."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(first, first + n):
        d = int(rng.choice([64, 128]))
        if large:
            n_ref = int(rng.choice([0, 64 * int(rng.integers(1, 60)), int(rng.integers(1, 4000))]))
            n_tgt = int(rng.choice([64 * int(rng.integers(1, 40)), int(rng.integers(1, 2500))]))
            B, H = int(rng.integers(1, 3)), int(rng.integers(1, 9))
        else:
            n_ref = int(rng.choice([0, 1, 63, 64, 65, int(rng.integers(2, 700))]))
            n_tgt = int(rng.choice([1, 64, int(rng.integers(2, 500))]))
            B, H = int(rng.integers(1, 3)), int(rng.integers(1, 4))
        qset = str(rng.choice(["target", "all"]))
        kv = str(rng.choice(["fresh", "cache", "segments"])) if n_ref > 0 else "fresh"
        segs, cached = None, None
        if kv == "segments" or (n_ref > 64 and rng.random() < 0.3):
            k = int(rng.integers(1, 16)) if large else 3
            cuts = sorted(set(int(x) * 64 for x in rng.integers(1, max(2, (n_ref + 63) // 64), size=k)
                              if int(x) * 64 < n_ref))
            segs = cuts + [n_ref]
            cached = [bool(x) for x in rng.integers(0, 2, size=len(segs))]
        split = bool(rng.random() < (0.6 if large else 0.5))
        cases.append((i, d, n_ref, n_tgt, B, H, qset, kv, segs, cached, split))
    return cases


@pytest.mark.parametrize("case", _random_cases() + [pytest.param(c, marks=pytest.mark.slow)
                                                     for c in _random_cases(30, 4242, large=True, first=1000)],
                         ids=lambda c: f"r{c[0]}")
def test_random_configurations_parity(case):
    i, d, n_ref, n_tgt, B, H, qset, kv, segs, cached, split = case
    print(f"random case {case}", flush=True)
    _, x = _inputs("bf16", d, n_ref, n_tgt, B, H, seed=100 + i)
    kw = {} if split else {"workspace": False}
    if kv == "segments":
        kr, vr, ends = _seg_oracle_inputs(x, np.diff([0] + segs).tolist(), cached)
        kw.update(seg_end=ends, seg_cache=cached)
    else:
        use = kv == "cache"
        kr = x["k_ref_cache"] if use else x["k_ref"]
        vr = x["v_ref_cache"] if use else x["v_ref"]
        if segs is not None:
            kw.update(seg_end=segs)
    want_seg = segs is not None
    got = _gpu(x, "bf16", qset, kv, seg_mass=want_seg, **kw)
    ref = joint_attention(x["q_tgt"], kr, vr, x["k_tgt"], x["v_tgt"])
    assert max_abs(host(got.o_tgt), ref["o"]) <= O_TOL["bf16"]
    assert max_abs(host(got.ref_mass), ref["ref_mass"]) <= MASS_TOL["bf16"]
    lse = host(got.lse)
    assert max_abs(lse[..., 1], ref["lse_all"]) <= 1e-3
    if n_ref > 0:
        assert max_abs(lse[..., 0], ref["lse_ref"]) <= 1e-3
    else:
        assert np.all(np.isneginf(lse[..., 0]))
    if want_seg:
        assert max_abs(host(got.seg_mass), segment_masses(x["q_tgt"], kr, x["k_tgt"], segs)) <= MASS_TOL["bf16"]
    if qset == "all" and n_ref > 0:
        rr = joint_attention(x["q_ref"], kr, vr, x["k_tgt"], x["v_tgt"])
        assert max_abs(host(got.o_ref), rr["o"]) <= O_TOL["bf16"]
        assert max_abs(host(got.ref_mass_refq), rr["ref_mass"]) <= MASS_TOL["bf16"]


def test_clock_probe_counts_and_leaves_outputs_unchanged():
    """The optional clock probe adds every workgroup's shader cycles and 100 MHz ticks; the
    outputs are bitwise those of the launch without it."""
    print("clock probe", flush=True)
    _, x = _inputs("bf16", 128, 700, 900, 1, 4)
    plain = _gpu(x, "bf16", "all", "fresh")
    probe = torch.zeros(2, dtype=torch.int64, device="cuda:0")
    got = _gpu(x, "bf16", "all", "fresh", clock_probe=probe)
    for a, b in ((plain.o_tgt, got.o_tgt), (plain.o_ref, got.o_ref), (plain.ref_mass, got.ref_mass),
                 (plain.lse, got.lse)):
        assert torch.equal(a, b)
    cyc, ticks = probe.cpu().tolist()
    assert ticks > 0 and cyc > 0
    mhz = 100.0 * cyc / ticks
    print(f"  mean shader clock {mhz:.0f} MHz", flush=True)
    assert 300.0 < mhz < 3000.0


def test_concurrent_launches_on_two_streams():
    """The library keeps no per-call state outside the caller's buffers: two key-split launches
    with their own workspaces, enqueued on two streams and running concurrently, give bitwise
    the outputs of the same launches run one after the other."""
    print("two streams", flush=True)
    _, xa = _inputs("bf16", 128, 700, 900, 1, 4, seed=61)
    _, xb = _inputs("bf16", 128, 300, 1300, 1, 4, seed=62)
    ta = {k: dev(v, "bf16") for k, v in xa.items()}
    tb = {k: dev(v, "bf16") for k, v in xb.items()}

    def run(t, kvsrc):
        return ops.joint_attn(t["q_tgt"], t["k_tgt"], t["v_tgt"], q_ref=t["q_ref"], k_ref=t["k_ref"],
                              v_ref=t["v_ref"], k_cache=t["k_ref_cache"], v_cache=t["v_ref_cache"], qset="all",
                              kvsrc=kvsrc, lse=True)

    seq_a, seq_b = run(ta, "fresh"), run(tb, "cache")
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    for _ in range(3):
        with torch.cuda.stream(s1):
            a = run(ta, "fresh")
        with torch.cuda.stream(s2):
            b = run(tb, "cache")
        outs.append((a, b))
    torch.cuda.synchronize()
    for a, b in outs:
        for x, y in ((a.o_tgt, seq_a.o_tgt), (a.o_ref, seq_a.o_ref), (a.ref_mass, seq_a.ref_mass), (a.lse, seq_a.lse),
                     (b.o_tgt, seq_b.o_tgt), (b.o_ref, seq_b.o_ref), (b.ref_mass, seq_b.ref_mass), (b.lse, seq_b.lse)):
            assert torch.equal(x, y)
