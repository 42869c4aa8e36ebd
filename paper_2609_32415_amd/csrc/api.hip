// C ABI of librefadapt: argument validation and kernel dispatch.
//
// Every entry point validates on the host, enqueues on the caller's stream and
// returns; nothing here allocates device memory or synchronises.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <algorithm>
#include <mutex>
#include <string>

#include "refadapt.h"
#include "internal.h"

using namespace refadapt;

namespace {

thread_local std::string g_last_error;

ra_status fail(ra_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

ra_status ok() {
  g_last_error.clear();
  return RA_OK;
}

View view(const ra_tensor& t) { return View{t.data, t.stride_b, t.stride_h, t.stride_s}; }

// Alignment rules for 16-byte vector access: base 16-byte aligned, strides in whole 16-byte units.
bool aligned(const ra_tensor& t, int dtype) {
  const int64_t unit = dtype == RA_BF16 ? 8 : 4;
  return (reinterpret_cast<uintptr_t>(t.data) & 15) == 0 && t.stride_b % unit == 0 && t.stride_h % unit == 0 &&
         t.stride_s % unit == 0;
}

ra_status check_tensor(const char* name, const ra_tensor& t, int dtype, int32_t rows, int32_t head_dim) {
  if (t.data == nullptr) return fail(RA_EINVAL, "%s: null data pointer", name);
  if (t.stride_b < 0 || t.stride_h < 0 || t.stride_s < 0)
    return fail(RA_EINVAL, "%s: negative stride", name);
  if (rows > 1 && t.stride_s < head_dim)
    return fail(RA_EINVAL, "%s: row stride %lld is smaller than head_dim %d", name, (long long)t.stride_s, head_dim);
  if (!aligned(t, dtype))
    return fail(RA_EUNSUPPORTED, "%s: base must be 16-byte aligned and strides multiples of %d elements", name,
                dtype == RA_BF16 ? 8 : 4);
  return RA_OK;
}

// ---- work decomposition of the bf16 attention launch
//
// All query tiles of a launch cost the same (each attends to every key tile),
// so the resident workgroups (slots = CUs x workgroups per CU) run them in
// rounds. Cost model in units of "one key tile processed by every resident
// workgroup": a round of items of L key tiles costs L, or kLoneRound * L when
// the round holds no more items than there are CUs (a workgroup alone on its
// CU runs faster); a chunk adds a fixed start-up and drain of kChunkOverhead
// key tiles; the merge costs its partial-result traffic. The plan keeps the
// largest number of whole rounds and splits only the remainder (plus, when it
// pays, one more round) into chunks of at least kMinChunk key tiles.
constexpr int kMinChunk = 4;
constexpr double kChunkOverhead = 2.0;
constexpr double kLoneRound = 0.67;
constexpr int kMaxChunks = 32;

SplitPlan whole_plan(int64_t tiles) {
  return SplitPlan{(int32_t)tiles, 0, 1, (int32_t)tiles};
}

// Cost of running `items` items of `len` key tiles each in rounds of `slots`.
double rounds_cost(int64_t items, double len, int64_t slots, int64_t cus) {
  const int64_t full = items / slots, last = items - full * slots;
  return full * len + (last == 0 ? 0.0 : last > cus ? len : kLoneRound * len);
}

SplitPlan plan_split(int64_t tiles, int nt, AttnSlots sl, int head_dim) {
  SplitPlan best = whole_plan(tiles);
  const int64_t slots = (int64_t)sl.cus * sl.per_cu;
  if (tiles <= 0 || slots <= 0 || nt < 2 * kMinChunk) return best;
  // A split must beat whole tiles by 3%; among splits the cheapest wins.
  double best_cost = 0.97 * rounds_cost(tiles, nt, slots, sl.cus);
  // Seconds for every resident workgroup to process one key tile (~1 PFLOP/s of
  // attention) and to move one split item's partial rows twice (~4 TB/s).
  const double tile_s = slots * 4.0 * kAttnBf16BM * kAttnBf16BN * head_dim / 1.0e15;
  const double item_s = 2.0 * kAttnBf16BM * (head_dim + 4) * 4.0 / 4.0e12;
  for (int extra = 0; extra < 2; ++extra) {
    const int64_t rem = tiles % slots + (int64_t)extra * slots;
    if (rem == 0 || rem > tiles) continue;
    const int64_t rounds = (tiles - rem) / slots;
    for (int c = 2; c <= kMaxChunks && c * kMinChunk <= nt; ++c) {
      const int64_t items = rem * c;
      if (items > 2 * slots) break;
      const int chunk = (nt + c - 1) / c;
      const double cost = (double)rounds * nt + rounds_cost(items, chunk + kChunkOverhead, slots, sl.cus) +
                          (items * item_s + 5e-6) / tile_s;
      if (cost < best_cost) {
        best_cost = cost;
        best = SplitPlan{(int32_t)(tiles - rem), (int32_t)rem, c, (int32_t)(tiles - rem + items)};
      }
    }
  }
  return best;
}

// Plans of one bf16 launch (plan[0]: the launch's query set, plan[1]: target
// query tiles only) and the workspace bytes their split items need.
struct LaunchPlan {
  SplitPlan plan[2];
  int64_t qt_ref, qt_tgt;
  int64_t items;  // split items of the larger plan
  size_t ws_bytes;
  size_t part_o_bytes;
};

// Workspace bytes of a split launch that also records per-segment masses: the partials plus
// one log-sum-exp per segment of each partial row, after them.
size_t seg_ws_bytes(const LaunchPlan& lp, int n_seg) {
  return lp.ws_bytes ? lp.ws_bytes + (size_t)lp.items * kAttnBf16BM * n_seg * sizeof(float) : 0;
}

LaunchPlan plan_launch(const ra_attn_desc& d, bool split) {
  LaunchPlan lp{};
  const bool device = d.kvsrc == RA_KV_DEVICE;
  const bool ref_queries = (device || d.qset == RA_Q_ALL) && d.n_ref > 0;
  const int bm = d.dtype == RA_BF16 ? kAttnBf16BM : kAttnF32BM;
  lp.qt_ref = ref_queries ? (d.n_ref + bm - 1) / bm : 0;
  lp.qt_tgt = (d.n_tgt + bm - 1) / bm;
  const int64_t bh = (int64_t)d.batch * d.heads;
  const int64_t all = bh * (lp.qt_ref + lp.qt_tgt), tgt = bh * lp.qt_tgt;
  lp.plan[0] = whole_plan(all);
  lp.plan[1] = device ? whole_plan(tgt) : lp.plan[0];
  if (!split || d.dtype != RA_BF16 || all > 0x7fffffff) return lp;
  const AttnSlots slots = attn_bf16_slots(d.head_dim);
  const int nt = (d.n_ref + kAttnBf16BN - 1) / kAttnBf16BN + (d.n_tgt + kAttnBf16BN - 1) / kAttnBf16BN;
  lp.plan[0] = plan_split(all, nt, slots, d.head_dim);
  lp.plan[1] = device ? plan_split(tgt, nt, slots, d.head_dim) : lp.plan[0];
  int64_t items = 0;
  for (const SplitPlan& pl : lp.plan) items = std::max<int64_t>(items, (int64_t)pl.split_tiles * pl.chunks);
  lp.items = items;
  lp.part_o_bytes = (size_t)items * kAttnBf16BM * d.head_dim * sizeof(float);
  lp.ws_bytes = items > 0 ? lp.part_o_bytes + (size_t)items * kAttnBf16BM * 5 * sizeof(float) : 0;
  return lp;
}

ra_status check_attn_desc(const ra_attn_desc* desc, const char* who) {
  if (!desc) return fail(RA_EINVAL, "%s: null desc", who);
  const ra_attn_desc& d = *desc;
  if (d.batch < 1 || d.heads < 1) return fail(RA_EINVAL, "%s: batch and heads must be >= 1", who);
  if (d.n_tgt < 1) return fail(RA_EINVAL, "%s: n_tgt must be >= 1 (got %d)", who, d.n_tgt);
  if (d.n_ref < 0) return fail(RA_EINVAL, "%s: n_ref must be >= 0 (got %d)", who, d.n_ref);
  if (d.dtype != RA_BF16 && d.dtype != RA_F32) return fail(RA_EINVAL, "%s: unknown dtype %d", who, d.dtype);
  if (d.qset != RA_Q_TARGET && d.qset != RA_Q_ALL) return fail(RA_EINVAL, "%s: unknown qset %d", who, d.qset);
  if (d.kvsrc < RA_KV_FRESH || d.kvsrc > RA_KV_SEGMENTS) return fail(RA_EINVAL, "%s: unknown kvsrc %d", who, d.kvsrc);
  if (d.head_dim != 64 && d.head_dim != 128)
    return fail(RA_EUNSUPPORTED, "%s: head_dim %d not supported (64 or 128)", who, d.head_dim);
  if (!std::isfinite(d.scale)) return fail(RA_EINVAL, "%s: scale must be finite", who);
  return RA_OK;
}

ra_status launch_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(RA_ELAUNCH, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

const char* refadapt_last_error(void) { return g_last_error.c_str(); }

const char* refadapt_version(void) { return "refadapt 0.1 gfx950"; }

size_t refadapt_joint_attn_workspace_size(const ra_attn_desc* desc) {
  if (check_attn_desc(desc, "joint_attn_workspace_size") != RA_OK) return 0;
  return plan_launch(*desc, true).ws_bytes;
}

size_t refadapt_joint_attn_seg_workspace_size(const ra_attn_desc* desc, int32_t n_seg) {
  if (check_attn_desc(desc, "joint_attn_seg_workspace_size") != RA_OK) return 0;
  const ra_attn_desc& d = *desc;
  if (n_seg < 1 || n_seg > RA_MAX_SEG || d.dtype != RA_BF16 || d.kvsrc == RA_KV_DEVICE || d.n_ref < 1) return 0;
  return seg_ws_bytes(plan_launch(d, true), n_seg);
}

ra_status refadapt_joint_attn(const ra_attn_desc* desc, const ra_attn_args* args, void* stream) {
  ra_status s;
  if ((s = check_attn_desc(desc, "joint_attn")) != RA_OK) return s;
  if (!args) return fail(RA_EINVAL, "joint_attn: null args");
  const ra_attn_desc& d = *desc;
  const ra_attn_args& a = *args;
  const bool device = d.kvsrc == RA_KV_DEVICE;
  const bool ref_queries = (device || d.qset == RA_Q_ALL) && d.n_ref > 0;
  // Reference segments: per-segment K/V sources or per-segment masses.
  const bool seg = d.kvsrc == RA_KV_SEGMENTS || a.seg_mass != nullptr;
  uint32_t seg_cache = 0;
  if (seg) {
    if (d.dtype != RA_BF16) return fail(RA_EUNSUPPORTED, "joint_attn: reference segments need RA_BF16");
    if (device) return fail(RA_EUNSUPPORTED, "joint_attn: reference segments are not available under RA_KV_DEVICE");
    if (d.n_ref < 1) return fail(RA_EINVAL, "joint_attn: reference segments need n_ref >= 1");
    if (a.n_seg < 1 || a.n_seg > RA_MAX_SEG)
      return fail(RA_EINVAL, "joint_attn: n_seg %d outside 1..%d", a.n_seg, RA_MAX_SEG);
    int32_t prev = 0;
    for (int i = 0; i < a.n_seg; ++i) {
      const int32_t e = a.seg_end[i];
      if (e <= prev) return fail(RA_EINVAL, "joint_attn: seg_end[%d] = %d does not increase", i, e);
      if (i + 1 < a.n_seg && e % kAttnBf16BN != 0)
        return fail(RA_EUNSUPPORTED, "joint_attn: seg_end[%d] = %d is not a multiple of %d", i, e, kAttnBf16BN);
      prev = e;
    }
    if (prev != d.n_ref) return fail(RA_EINVAL, "joint_attn: seg_end[n_seg-1] = %d != n_ref %d", prev, d.n_ref);
    const uint32_t all = (1u << a.n_seg) - 1u;
    seg_cache = d.kvsrc == RA_KV_SEGMENTS ? (a.seg_cache & all) : d.kvsrc == RA_KV_CACHE ? all : 0u;
  }
  const bool reads_fresh =
      d.n_ref > 0 && (d.kvsrc == RA_KV_FRESH || device || (d.kvsrc == RA_KV_SEGMENTS && seg_cache != ((1u << a.n_seg) - 1u)));
  const bool reads_cache = d.n_ref > 0 && (d.kvsrc == RA_KV_CACHE || device || (d.kvsrc == RA_KV_SEGMENTS && seg_cache != 0));
  if ((s = check_tensor("q_tgt", a.q_tgt, d.dtype, d.n_tgt, d.head_dim)) != RA_OK) return s;
  if ((s = check_tensor("k_tgt", a.k_tgt, d.dtype, d.n_tgt, d.head_dim)) != RA_OK) return s;
  if ((s = check_tensor("v_tgt", a.v_tgt, d.dtype, d.n_tgt, d.head_dim)) != RA_OK) return s;
  if ((s = check_tensor("o_tgt", a.o_tgt, d.dtype, d.n_tgt, d.head_dim)) != RA_OK) return s;
  if (reads_fresh) {
    if ((s = check_tensor("k_ref", a.k_ref, d.dtype, d.n_ref, d.head_dim)) != RA_OK) return s;
    if ((s = check_tensor("v_ref", a.v_ref, d.dtype, d.n_ref, d.head_dim)) != RA_OK) return s;
  }
  if (reads_cache) {
    if ((s = check_tensor("k_cache", a.k_cache, d.dtype, d.n_ref, d.head_dim)) != RA_OK) return s;
    if ((s = check_tensor("v_cache", a.v_cache, d.dtype, d.n_ref, d.head_dim)) != RA_OK) return s;
  }
  // Cached reference queries: read where reference queries attend over the cached K/V.
  const bool q_cache = ref_queries && a.q_cache.data != nullptr && (d.kvsrc == RA_KV_CACHE || device);
  if (ref_queries) {
    if (!(q_cache && d.kvsrc == RA_KV_CACHE))
      if ((s = check_tensor("q_ref", a.q_ref, d.dtype, d.n_ref, d.head_dim)) != RA_OK) return s;
    if (q_cache && (s = check_tensor("q_cache", a.q_cache, d.dtype, d.n_ref, d.head_dim)) != RA_OK) return s;
    if ((s = check_tensor("o_ref", a.o_ref, d.dtype, d.n_ref, d.head_dim)) != RA_OK) return s;
  }
  if (device && a.decision == nullptr) return fail(RA_EINVAL, "joint_attn: RA_KV_DEVICE needs a decision pointer");
  if (d.dtype == RA_BF16) {
    // K/V tiles are addressed with 32-bit buffer offsets: 64 rows of the row stride must fit.
    const ra_tensor* kv[] = {&a.k_tgt, &a.v_tgt, &a.k_ref, &a.v_ref, &a.k_cache, &a.v_cache};
    const char* kv_name[] = {"k_tgt", "v_tgt", "k_ref", "v_ref", "k_cache", "v_cache"};
    const bool used[] = {true, true, reads_fresh, reads_fresh, reads_cache, reads_cache};
    for (int i = 0; i < 6; ++i)
      if (used[i] && kv[i]->stride_s > kAttnMaxRowStride)
        return fail(RA_EUNSUPPORTED, "joint_attn: %s row stride %lld exceeds %lld elements", kv_name[i],
                    (long long)kv[i]->stride_s, (long long)kAttnMaxRowStride);
  }
  if (d.kvsrc == RA_KV_SEGMENTS && reads_fresh && reads_cache) {
    const auto same = [](const ra_tensor& x, const ra_tensor& y) {
      return x.stride_b == y.stride_b && x.stride_h == y.stride_h && x.stride_s == y.stride_s;
    };
    if (!same(a.k_ref, a.k_cache) || !same(a.v_ref, a.v_cache))
      return fail(RA_EUNSUPPORTED, "joint_attn: RA_KV_SEGMENTS needs the fresh and cached K/V to share strides");
  }

  AttnParams p{};
  p.q_tgt = view(a.q_tgt);
  p.k_tgt = view(a.k_tgt);
  p.v_tgt = view(a.v_tgt);
  p.q_ref = view(a.q_ref);
  p.q_cache = q_cache ? view(a.q_cache) : View{nullptr, 0, 0, 0};
  p.k_fresh = view(a.k_ref);
  p.v_fresh = view(a.v_ref);
  p.k_cache = view(a.k_cache);
  p.v_cache = view(a.v_cache);
  p.o_tgt = view(a.o_tgt);
  p.o_ref = view(a.o_ref);
  p.mass_tgt = a.ref_mass;
  p.lse_tgt = a.lse_tgt;
  p.mass_refq = a.ref_mass_refq;
  p.decision = a.decision;
  p.clock_probe = reinterpret_cast<unsigned long long*>(a.clock_probe);
  p.B = d.batch;
  p.H = d.heads;
  p.n_ref = d.n_ref;
  p.n_tgt = d.n_tgt;
  // With no reference rows there is nothing to choose between: read the (empty) fresh segment.
  p.kvsrc = d.n_ref == 0 ? RA_KV_FRESH : d.kvsrc;
  if (d.n_ref == 0 && device) p.kvsrc = RA_KV_FRESH;
  const float scale = d.scale > 0.f ? d.scale : 1.0f / std::sqrt((float)d.head_dim);
  p.sc_log2 = scale * 1.4426950408889634f;

  // Per-segment masses split key ranges only when the workspace also holds the per-segment
  // partials; with a smaller workspace the launch runs whole query tiles.
  LaunchPlan lp = plan_launch(d, a.workspace != nullptr);
  if (a.seg_mass != nullptr && a.workspace_bytes < seg_ws_bytes(lp, a.n_seg)) lp = plan_launch(d, false);
  const int64_t total = (int64_t)d.batch * d.heads * (lp.qt_ref + lp.qt_tgt);
  if (total > 0x7fffffff) return fail(RA_EUNSUPPORTED, "joint_attn: problem too large for one launch");
  if (a.workspace != nullptr) {
    if (a.workspace_bytes < lp.ws_bytes)
      return fail(RA_EWORKSPACE, "joint_attn: workspace needs %zu bytes (got %zu)", lp.ws_bytes, a.workspace_bytes);
    if ((reinterpret_cast<uintptr_t>(a.workspace) & 15) != 0)
      return fail(RA_EUNSUPPORTED, "joint_attn: workspace must be 16-byte aligned");
  }
  p.qt_ref = (int32_t)lp.qt_ref;
  p.qt_tgt = (int32_t)lp.qt_tgt;
  p.total_tiles = (int32_t)total;
  p.plan[0] = lp.plan[0];
  p.plan[1] = lp.plan[1];
  p.part_o = static_cast<float*>(a.workspace);
  p.part_st = lp.ws_bytes ? reinterpret_cast<float4*>(static_cast<char*>(a.workspace) + lp.part_o_bytes) : nullptr;
  p.part_lo = lp.ws_bytes ? reinterpret_cast<float*>(p.part_st + lp.items * kAttnBf16BM) : nullptr;
  p.part_seg = lp.ws_bytes && a.seg_mass ? reinterpret_cast<float*>(static_cast<char*>(a.workspace) + lp.ws_bytes)
                                         : nullptr;
  if (seg) {
    p.n_seg = a.n_seg;
    for (int i = 0; i < a.n_seg; ++i) {
      p.seg_tile_end[i] = (a.seg_end[i] + kAttnBf16BN - 1) / kAttnBf16BN;
      const bool c = (seg_cache >> i) & 1u;
      p.seg_kbase[i] = c ? a.k_cache.data : a.k_ref.data;
      p.seg_vbase[i] = c ? a.v_cache.data : a.v_ref.data;
    }
    p.seg_cache = seg_cache;
    p.seg_mass = a.seg_mass;
    // The kernel applies one set of strides to both sources: those of the fresh views when
    // any segment reads them, else those of the cached views.
    if (!reads_fresh) {
      p.k_fresh = p.k_cache;
      p.v_fresh = p.v_cache;
    }
  }

  const hipStream_t st = static_cast<hipStream_t>(stream);
  const hipError_t e = d.dtype == RA_BF16 ? launch_attn_bf16(p, d.head_dim, st) : launch_attn_f32(p, d.head_dim, st);
  return launch_status(e, "joint_attn");
}

size_t refadapt_q_change_workspace_size(int32_t batch, int32_t heads, int32_t n_tgt, int32_t head_dim) {
  if (batch < 1 || heads < 1 || n_tgt < 1 || head_dim < 1) return 0;
  return (size_t)batch * heads * q_change_chunks(n_tgt, head_dim) * 2 * sizeof(float);
}

ra_status refadapt_q_change(int32_t batch, int32_t heads, int32_t n_tgt, int32_t head_dim, int32_t dtype,
                            ra_tensor q_cur, ra_tensor q_prev, float eps, float* d_out, void* workspace,
                            size_t ws_bytes, void* stream) {
  if (batch < 1 || heads < 1 || n_tgt < 1) return fail(RA_EINVAL, "q_change: batch, heads, n_tgt must be >= 1");
  if (dtype != RA_BF16 && dtype != RA_F32) return fail(RA_EINVAL, "q_change: unknown dtype %d", dtype);
  if (head_dim < 1 || head_dim % (dtype == RA_BF16 ? 8 : 4) != 0)
    return fail(RA_EUNSUPPORTED, "q_change: head_dim %d must be a positive multiple of %d", head_dim,
                dtype == RA_BF16 ? 8 : 4);
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(RA_EINVAL, "q_change: eps must be finite and >= 0");
  ra_status s;
  if ((s = check_tensor("q_cur", q_cur, dtype, n_tgt, head_dim)) != RA_OK) return s;
  if ((s = check_tensor("q_prev", q_prev, dtype, n_tgt, head_dim)) != RA_OK) return s;
  if (d_out == nullptr) return fail(RA_EINVAL, "q_change: null d_out");
  const size_t need = refadapt_q_change_workspace_size(batch, heads, n_tgt, head_dim);
  if (workspace == nullptr || ws_bytes < need)
    return fail(RA_EWORKSPACE, "q_change: workspace needs %zu bytes (got %zu)", need, workspace ? ws_bytes : 0);
  if ((reinterpret_cast<uintptr_t>(workspace) & 7) != 0)
    return fail(RA_EUNSUPPORTED, "q_change: workspace must be 8-byte aligned");
  const hipError_t e = launch_q_change(dtype, batch, heads, n_tgt, head_dim, view(q_cur), view(q_prev), eps, d_out,
                                       workspace, static_cast<hipStream_t>(stream));
  return launch_status(e, "q_change");
}

ra_status refadapt_gate(int32_t batch, int32_t heads, int32_t n_tgt, int32_t block, int32_t step, int32_t mode,
                        const float* d_cur, const float* mass_prev, const float* theta, ra_gate_state* state,
                        int32_t* decision_out, float* score_out, void* stream) {
  if (batch < 1 || heads < 1 || n_tgt < 1) return fail(RA_EINVAL, "gate: batch, heads, n_tgt must be >= 1");
  if ((int64_t)batch * heads > 8192) return fail(RA_EUNSUPPORTED, "gate: batch*heads must be <= 8192");
  if (block < 0 || step < 0) return fail(RA_EINVAL, "gate: block and step must be >= 0");
  if (mode < RA_GATE_PRODUCT || mode > RA_GATE_AND) return fail(RA_EINVAL, "gate: unknown mode %d", mode);
  if (!d_cur || !mass_prev || !theta || !state || !decision_out || !score_out)
    return fail(RA_EINVAL, "gate: null pointer argument");
  const hipError_t e = launch_gate(batch, heads, n_tgt, block, step, mode, d_cur, mass_prev, theta,
                                   reinterpret_cast<GateState*>(state), decision_out, score_out,
                                   static_cast<hipStream_t>(stream));
  return launch_status(e, "gate");
}

size_t refadapt_q_change_gate_workspace_size(int32_t batch, int32_t heads, int32_t n_tgt, int32_t head_dim) {
  if (batch < 1 || heads < 1 || n_tgt < 1 || head_dim < 1) return 0;
  return q_change_gate_workspace_bytes(batch, heads, n_tgt, head_dim);
}

}  // extern "C"

namespace {

// Arguments of the fused Q-change + gate other than its workspace (`who` names the caller).
ra_status check_q_change_gate(const char* who, int32_t batch, int32_t heads, int32_t n_tgt, int32_t head_dim,
                              int32_t dtype, const ra_tensor& q_cur, const ra_tensor& q_prev, float eps,
                              int32_t block, int32_t step, int32_t mode, const float* mass_prev, const float* theta,
                              const ra_gate_state* state, const float* d_out, const int32_t* decision_out,
                              const float* score_out) {
  if (batch < 1 || heads < 1 || n_tgt < 1) return fail(RA_EINVAL, "%s: batch, heads, n_tgt must be >= 1", who);
  if ((int64_t)batch * heads > 8192) return fail(RA_EUNSUPPORTED, "%s: batch*heads must be <= 8192", who);
  if (dtype != RA_BF16 && dtype != RA_F32) return fail(RA_EINVAL, "%s: unknown dtype %d", who, dtype);
  if (head_dim < 1 || head_dim % (dtype == RA_BF16 ? 8 : 4) != 0)
    return fail(RA_EUNSUPPORTED, "%s: head_dim %d must be a positive multiple of %d", who, head_dim,
                dtype == RA_BF16 ? 8 : 4);
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(RA_EINVAL, "%s: eps must be finite and >= 0", who);
  if (block < 0 || step < 0) return fail(RA_EINVAL, "%s: block and step must be >= 0", who);
  if (mode < RA_GATE_PRODUCT || mode > RA_GATE_AND) return fail(RA_EINVAL, "%s: unknown mode %d", who, mode);
  ra_status s;
  if ((s = check_tensor("q_cur", q_cur, dtype, n_tgt, head_dim)) != RA_OK) return s;
  if ((s = check_tensor("q_prev", q_prev, dtype, n_tgt, head_dim)) != RA_OK) return s;
  if (!mass_prev || !theta || !state || !d_out || !decision_out || !score_out)
    return fail(RA_EINVAL, "%s: null pointer argument", who);
  return RA_OK;
}

}  // namespace

extern "C" {

ra_status refadapt_q_change_gate(int32_t batch, int32_t heads, int32_t n_tgt, int32_t head_dim, int32_t dtype,
                                 ra_tensor q_cur, ra_tensor q_prev, float eps, int32_t block, int32_t step,
                                 int32_t mode, const float* mass_prev, const float* theta, ra_gate_state* state,
                                 float* d_out, int32_t* decision_out, float* score_out, void* workspace,
                                 size_t ws_bytes, void* stream) {
  ra_status s;
  if ((s = check_q_change_gate("q_change_gate", batch, heads, n_tgt, head_dim, dtype, q_cur, q_prev, eps, block,
                               step, mode, mass_prev, theta, state, d_out, decision_out, score_out)) != RA_OK)
    return s;
  const size_t need = refadapt_q_change_gate_workspace_size(batch, heads, n_tgt, head_dim);
  if (workspace == nullptr || ws_bytes < need)
    return fail(RA_EWORKSPACE, "q_change_gate: workspace needs %zu bytes (got %zu)", need, workspace ? ws_bytes : 0);
  if ((reinterpret_cast<uintptr_t>(workspace) & 15) != 0)
    return fail(RA_EUNSUPPORTED, "q_change_gate: workspace must be 16-byte aligned");
  const hipError_t e = launch_q_change_gate(dtype, batch, heads, n_tgt, head_dim, view(q_cur), view(q_prev), eps,
                                            block, step, mode, mass_prev, theta, reinterpret_cast<GateState*>(state),
                                            d_out, decision_out, score_out, workspace,
                                            static_cast<hipStream_t>(stream));
  return launch_status(e, "q_change_gate");
}

}  // extern "C"

// ---- allocation-free Q-change + gate
//
// The fused Q-change + gate needs per-chunk partial sums between its two launches. This
// variant keeps them in one fixed device array instead of a caller workspace, for callers
// that cannot allocate. Each device holds its own copy of the array; host code takes its
// device address once per device (hipGetSymbolAddress) and passes that address to the
// kernels, never the array's name. Calls that overlap on one device share it and race.
namespace {

constexpr size_t kScratchBytes = size_t(1) << 20;  // 65536 partial records of 16 bytes
constexpr int kMaxScratchDevices = 64;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// Device address of the current device's `scratch`, looked up on the first call per device.
ra_status scratch_ptr(void** out) {
  int dev = -1;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(RA_ELAUNCH, "q_change_gate_noalloc: hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(RA_EUNSUPPORTED, "q_change_gate_noalloc: device %d outside 0..%d", dev, kMaxScratchDevices - 1);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    const hipError_t r = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (r != hipSuccess || p == nullptr)
      return fail(RA_ELAUNCH, "q_change_gate_noalloc: hipGetSymbolAddress(scratch): %s", hipGetErrorString(r));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return RA_OK;
}

}  // namespace

extern "C" {

ra_status refadapt_q_change_gate_noalloc(int32_t batch, int32_t heads, int32_t n_tgt, int32_t head_dim,
                                         int32_t dtype, ra_tensor q_cur, ra_tensor q_prev, float eps, int32_t block,
                                         int32_t step, int32_t mode, const float* mass_prev, const float* theta,
                                         ra_gate_state* state, float* d_out, int32_t* decision_out,
                                         float* score_out, void* stream) {
  ra_status s;
  if ((s = check_q_change_gate("q_change_gate_noalloc", batch, heads, n_tgt, head_dim, dtype, q_cur, q_prev, eps,
                               block, step, mode, mass_prev, theta, state, d_out, decision_out, score_out)) != RA_OK)
    return s;
  const size_t need = refadapt_q_change_gate_workspace_size(batch, heads, n_tgt, head_dim);
  if (need > kScratchBytes)
    return fail(RA_EUNSUPPORTED,
                "q_change_gate_noalloc: batch %d x heads %d x n_tgt %d x head_dim %d needs %zu bytes of partial sums; "
                "the fixed scratch holds %zu (use refadapt_q_change_gate with a workspace)",
                batch, heads, n_tgt, head_dim, need, kScratchBytes);
  void* ws = nullptr;
  if ((s = scratch_ptr(&ws)) != RA_OK) return s;
  return refadapt_q_change_gate(batch, heads, n_tgt, head_dim, dtype, q_cur, q_prev, eps, block, step, mode,
                                mass_prev, theta, state, d_out, decision_out, score_out, ws, kScratchBytes, stream);
}

ra_status refadapt_cache_commit(int32_t batch, int32_t heads, int32_t n_ref, int32_t head_dim, int32_t dtype,
                                ra_tensor k_ref, ra_tensor v_ref, ra_tensor q_ref, ra_tensor k_cache,
                                ra_tensor v_cache, ra_tensor q_cache, const int32_t* decision, int32_t* age,
                                int32_t step, void* stream) {
  if (batch < 1 || heads < 1 || n_ref < 0) return fail(RA_EINVAL, "cache_commit: bad sizes");
  if (dtype != RA_BF16 && dtype != RA_F32) return fail(RA_EINVAL, "cache_commit: unknown dtype %d", dtype);
  if (head_dim < 1 || (head_dim * (dtype == RA_BF16 ? 2 : 4)) % 16 != 0)
    return fail(RA_EUNSUPPORTED, "cache_commit: head_dim %d must fill whole 16-byte units", head_dim);
  if (n_ref == 0) return ok();
  ra_status s;
  CommitSet cs{};
  const ra_tensor* src[3] = {&k_ref, &v_ref, &q_ref};
  const ra_tensor* dst[3] = {&k_cache, &v_cache, &q_cache};
  const char* src_name[3] = {"k_ref", "v_ref", "q_ref"};
  const char* dst_name[3] = {"k_cache", "v_cache", "q_cache"};
  for (int i = 0; i < 3; ++i) {
    // K is required; V and Q are optional pairs (both sides given, or neither).
    if (i > 0 && src[i]->data == nullptr && dst[i]->data == nullptr) continue;
    if ((s = check_tensor(src_name[i], *src[i], dtype, n_ref, head_dim)) != RA_OK) return s;
    if ((s = check_tensor(dst_name[i], *dst[i], dtype, n_ref, head_dim)) != RA_OK) return s;
    cs.src[cs.n] = view(*src[i]);
    cs.dst[cs.n] = view(*dst[i]);
    ++cs.n;
  }
  const hipError_t e = launch_cache_commit(dtype, batch, heads, n_ref, head_dim, cs, decision, age, step,
                                           static_cast<hipStream_t>(stream));
  return launch_status(e, "cache_commit");
}

}  // extern "C"

// ---- diagnostics sidecar

namespace {

ra_status check_pair_common(const char* fn, int32_t batch, int32_t heads, int32_t head_dim, int32_t dtype,
                            float eps) {
  if (batch < 1 || heads < 1) return fail(RA_EINVAL, "%s: batch and heads must be >= 1", fn);
  if (dtype != RA_BF16 && dtype != RA_F32) return fail(RA_EINVAL, "%s: unknown dtype %d", fn, dtype);
  if (head_dim < 1 || head_dim % (dtype == RA_BF16 ? 8 : 4) != 0)
    return fail(RA_EUNSUPPORTED, "%s: head_dim %d must be a positive multiple of %d", fn, head_dim,
                dtype == RA_BF16 ? 8 : 4);
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(RA_EINVAL, "%s: eps must be finite and >= 0", fn);
  return RA_OK;
}

ra_status check_workspace(const char* fn, void* ws, size_t ws_bytes, size_t need) {
  if (ws == nullptr || ws_bytes < need)
    return fail(RA_EWORKSPACE, "%s: workspace needs %zu bytes (got %zu)", fn, need, ws ? ws_bytes : 0);
  if ((reinterpret_cast<uintptr_t>(ws) & 7) != 0) return fail(RA_EUNSUPPORTED, "%s: workspace must be 8-byte aligned", fn);
  return RA_OK;
}

}  // namespace

extern "C" {

size_t refadapt_kv_drift_workspace_size(int32_t batch, int32_t heads, int32_t n_rows, int32_t head_dim) {
  if (batch < 1 || heads < 1 || n_rows < 1 || head_dim < 1) return 0;
  const int32_t rows[2] = {n_rows, n_rows};
  return pair_workspace_bytes(batch, heads, head_dim, 2, rows);
}

ra_status refadapt_kv_drift(int32_t batch, int32_t heads, int32_t n_rows, int32_t head_dim, int32_t dtype,
                            ra_tensor k_cur, ra_tensor k_base, ra_tensor v_cur, ra_tensor v_base, float eps,
                            float* d_k, float* d_v, float* e_kv, void* workspace, size_t ws_bytes, void* stream) {
  ra_status s;
  if ((s = check_pair_common("kv_drift", batch, heads, head_dim, dtype, eps)) != RA_OK) return s;
  if (n_rows < 1) return fail(RA_EINVAL, "kv_drift: n_rows must be >= 1");
  if ((s = check_tensor("k_cur", k_cur, dtype, n_rows, head_dim)) != RA_OK) return s;
  if ((s = check_tensor("k_base", k_base, dtype, n_rows, head_dim)) != RA_OK) return s;
  if ((s = check_tensor("v_cur", v_cur, dtype, n_rows, head_dim)) != RA_OK) return s;
  if ((s = check_tensor("v_base", v_base, dtype, n_rows, head_dim)) != RA_OK) return s;
  if (e_kv == nullptr) return fail(RA_EINVAL, "kv_drift: null e_kv");
  if ((s = check_workspace("kv_drift", workspace, ws_bytes,
                           refadapt_kv_drift_workspace_size(batch, heads, n_rows, head_dim))) != RA_OK)
    return s;
  PairSet ps{};
  ps.cur[0] = view(k_cur);
  ps.base[0] = view(k_base);
  ps.cur[1] = view(v_cur);
  ps.base[1] = view(v_base);
  ps.n_rows[0] = ps.n_rows[1] = n_rows;
  const hipError_t e = launch_pair_change(dtype, batch, heads, head_dim, 2, ps, PAIR_KV, eps, d_k, d_v, e_kv,
                                          workspace, static_cast<hipStream_t>(stream));
  return launch_status(e, "kv_drift");
}

size_t refadapt_drift_log_ratio_workspace_size(int32_t batch, int32_t heads, int32_t n_ref, int32_t n_tgt,
                                               int32_t head_dim) {
  if (batch < 1 || heads < 1 || n_ref < 1 || n_tgt < 1 || head_dim < 1) return 0;
  const int32_t rows[2] = {n_ref, n_tgt};
  return pair_workspace_bytes(batch, heads, head_dim, 2, rows);
}

ra_status refadapt_drift_log_ratio(int32_t batch, int32_t heads, int32_t n_ref, int32_t n_tgt, int32_t head_dim,
                                   int32_t dtype, ra_tensor z_ref_cur, ra_tensor z_ref_prev, ra_tensor z_tgt_cur,
                                   ra_tensor z_tgt_prev, float eps, float* d_ref, float* d_tgt, float* rho,
                                   void* workspace, size_t ws_bytes, void* stream) {
  ra_status s;
  if ((s = check_pair_common("drift_log_ratio", batch, heads, head_dim, dtype, eps)) != RA_OK) return s;
  if (n_ref < 1 || n_tgt < 1) return fail(RA_EINVAL, "drift_log_ratio: n_ref and n_tgt must be >= 1");
  if ((s = check_tensor("z_ref_cur", z_ref_cur, dtype, n_ref, head_dim)) != RA_OK) return s;
  if ((s = check_tensor("z_ref_prev", z_ref_prev, dtype, n_ref, head_dim)) != RA_OK) return s;
  if ((s = check_tensor("z_tgt_cur", z_tgt_cur, dtype, n_tgt, head_dim)) != RA_OK) return s;
  if ((s = check_tensor("z_tgt_prev", z_tgt_prev, dtype, n_tgt, head_dim)) != RA_OK) return s;
  if (rho == nullptr) return fail(RA_EINVAL, "drift_log_ratio: null rho");
  if ((s = check_workspace("drift_log_ratio", workspace, ws_bytes,
                           refadapt_drift_log_ratio_workspace_size(batch, heads, n_ref, n_tgt, head_dim))) != RA_OK)
    return s;
  PairSet ps{};
  ps.cur[0] = view(z_ref_cur);
  ps.base[0] = view(z_ref_prev);
  ps.cur[1] = view(z_tgt_cur);
  ps.base[1] = view(z_tgt_prev);
  ps.n_rows[0] = n_ref;
  ps.n_rows[1] = n_tgt;
  const hipError_t e = launch_pair_change(dtype, batch, heads, head_dim, 2, ps, PAIR_RATIO, eps, d_ref, d_tgt, rho,
                                          workspace, static_cast<hipStream_t>(stream));
  return launch_status(e, "drift_log_ratio");
}

size_t refadapt_output_impact_workspace_size(int32_t batch, int32_t heads, int32_t n_rows, int32_t head_dim) {
  if (batch < 1 || heads < 1 || n_rows < 1 || head_dim < 1) return 0;
  return pair_workspace_bytes(batch, heads, head_dim, 1, &n_rows);
}

ra_status refadapt_output_impact(int32_t batch, int32_t heads, int32_t n_rows, int32_t head_dim, int32_t dtype,
                                 ra_tensor o_stale, ra_tensor o_fresh, float eps, float* impact, void* workspace,
                                 size_t ws_bytes, void* stream) {
  ra_status s;
  if ((s = check_pair_common("output_impact", batch, heads, head_dim, dtype, eps)) != RA_OK) return s;
  if (n_rows < 1) return fail(RA_EINVAL, "output_impact: n_rows must be >= 1");
  if ((s = check_tensor("o_stale", o_stale, dtype, n_rows, head_dim)) != RA_OK) return s;
  if ((s = check_tensor("o_fresh", o_fresh, dtype, n_rows, head_dim)) != RA_OK) return s;
  if (impact == nullptr) return fail(RA_EINVAL, "output_impact: null impact");
  if ((s = check_workspace("output_impact", workspace, ws_bytes,
                           refadapt_output_impact_workspace_size(batch, heads, n_rows, head_dim))) != RA_OK)
    return s;
  PairSet ps{};
  ps.cur[0] = view(o_stale);
  ps.base[0] = view(o_fresh);
  ps.cur[1] = ps.cur[0];
  ps.base[1] = ps.base[0];
  ps.n_rows[0] = ps.n_rows[1] = n_rows;
  const hipError_t e = launch_pair_change(dtype, batch, heads, head_dim, 1, ps, PAIR_SINGLE, eps, impact, nullptr,
                                          nullptr, workspace, static_cast<hipStream_t>(stream));
  return launch_status(e, "output_impact");
}

ra_status refadapt_mass_mean(int32_t batch, int32_t heads, int32_t n_rows, const float* mass, int32_t complement,
                             float* out, void* stream) {
  if (batch < 1 || heads < 1 || n_rows < 1) return fail(RA_EINVAL, "mass_mean: batch, heads, n_rows must be >= 1");
  if (mass == nullptr || out == nullptr) return fail(RA_EINVAL, "mass_mean: null pointer argument");
  if (complement != 0 && complement != 1) return fail(RA_EINVAL, "mass_mean: complement must be 0 or 1");
  const hipError_t e =
      launch_mass_mean(batch, heads, n_rows, mass, complement, out, static_cast<hipStream_t>(stream));
  return launch_status(e, "mass_mean");
}

ra_status refadapt_adjacent_mass_change(int32_t n_steps, int32_t n_blocks, int32_t bh, const float* mass_mean,
                                        float* out, void* stream) {
  if (n_steps < 2) return fail(RA_EINVAL, "adjacent_mass_change: n_steps must be >= 2");
  if (n_blocks < 1 || bh < 1) return fail(RA_EINVAL, "adjacent_mass_change: n_blocks and bh must be >= 1");
  if (mass_mean == nullptr || out == nullptr) return fail(RA_EINVAL, "adjacent_mass_change: null pointer argument");
  const hipError_t e =
      launch_adjacent_change(n_steps, n_blocks, bh, mass_mean, out, static_cast<hipStream_t>(stream));
  return launch_status(e, "adjacent_mass_change");
}

ra_status refadapt_mfma_rate_probe(int32_t kind, int32_t workgroups, int32_t steps, const void* operands,
                                   float* sink, uint64_t* clock_probe, void* stream) {
  static_assert(kProbeOperandBytes == RA_PROBE_OPERAND_BYTES, "probe operand size");
  if (kind != RA_PROBE_DENSE && kind != RA_PROBE_MIX) return fail(RA_EINVAL, "mfma_rate_probe: unknown kind %d", kind);
  if (workgroups < 1 || steps < 1) return fail(RA_EINVAL, "mfma_rate_probe: workgroups and steps must be >= 1");
  if (operands == nullptr || sink == nullptr) return fail(RA_EINVAL, "mfma_rate_probe: null pointer argument");
  if ((reinterpret_cast<uintptr_t>(operands) & 15) != 0)
    return fail(RA_EUNSUPPORTED, "mfma_rate_probe: operands must be 16-byte aligned");
  const hipError_t e = launch_mfma_rate(kind, workgroups, steps, operands, sink,
                                        reinterpret_cast<unsigned long long*>(clock_probe),
                                        static_cast<hipStream_t>(stream));
  return launch_status(e, "mfma_rate_probe");
}

}  // extern "C"
