// C ABI of librefadapt: argument validation and kernel dispatch.
//
// Every entry point validates on the host, enqueues on the caller's stream and
// returns; nothing here allocates device memory or synchronises.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>

#include "../../include/refadapt.h"
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

ra_status launch_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(RA_ELAUNCH, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

const char* refadapt_last_error(void) { return g_last_error.c_str(); }

const char* refadapt_version(void) { return "refadapt 0.1 gfx950"; }

ra_status refadapt_joint_attn(const ra_attn_desc* desc, const ra_attn_args* args, void* stream) {
  if (!desc || !args) return fail(RA_EINVAL, "joint_attn: null desc or args");
  const ra_attn_desc& d = *desc;
  if (d.batch < 1 || d.heads < 1) return fail(RA_EINVAL, "joint_attn: batch and heads must be >= 1");
  if (d.n_tgt < 1) return fail(RA_EINVAL, "joint_attn: n_tgt must be >= 1 (got %d)", d.n_tgt);
  if (d.n_ref < 0) return fail(RA_EINVAL, "joint_attn: n_ref must be >= 0 (got %d)", d.n_ref);
  if (d.dtype != RA_BF16 && d.dtype != RA_F32) return fail(RA_EINVAL, "joint_attn: unknown dtype %d", d.dtype);
  if (d.qset != RA_Q_TARGET && d.qset != RA_Q_ALL) return fail(RA_EINVAL, "joint_attn: unknown qset %d", d.qset);
  if (d.kvsrc < RA_KV_FRESH || d.kvsrc > RA_KV_DEVICE) return fail(RA_EINVAL, "joint_attn: unknown kvsrc %d", d.kvsrc);
  if (d.head_dim != 64 && d.head_dim != 128)
    return fail(RA_EUNSUPPORTED, "joint_attn: head_dim %d not supported (64 or 128)", d.head_dim);
  if (!std::isfinite(d.scale)) return fail(RA_EINVAL, "joint_attn: scale must be finite");

  const ra_attn_args& a = *args;
  const bool device = d.kvsrc == RA_KV_DEVICE;
  const bool ref_queries = (device || d.qset == RA_Q_ALL) && d.n_ref > 0;
  const bool reads_fresh = d.n_ref > 0 && (d.kvsrc == RA_KV_FRESH || device);
  const bool reads_cache = d.n_ref > 0 && (d.kvsrc == RA_KV_CACHE || device);
  ra_status s;
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
  if (ref_queries) {
    if ((s = check_tensor("q_ref", a.q_ref, d.dtype, d.n_ref, d.head_dim)) != RA_OK) return s;
    if ((s = check_tensor("o_ref", a.o_ref, d.dtype, d.n_ref, d.head_dim)) != RA_OK) return s;
  }
  if (device && a.decision == nullptr) return fail(RA_EINVAL, "joint_attn: RA_KV_DEVICE needs a decision pointer");

  AttnParams p{};
  p.q_tgt = view(a.q_tgt);
  p.k_tgt = view(a.k_tgt);
  p.v_tgt = view(a.v_tgt);
  p.q_ref = view(a.q_ref);
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
  p.B = d.batch;
  p.H = d.heads;
  p.n_ref = d.n_ref;
  p.n_tgt = d.n_tgt;
  // With no reference rows there is nothing to choose between: read the (empty) fresh segment.
  p.kvsrc = d.n_ref == 0 ? RA_KV_FRESH : d.kvsrc;
  if (d.n_ref == 0 && device) p.kvsrc = RA_KV_FRESH;
  const float scale = d.scale > 0.f ? d.scale : 1.0f / std::sqrt((float)d.head_dim);
  p.sc_log2 = scale * 1.4426950408889634f;

  const int bm = d.dtype == RA_BF16 ? kAttnBf16BM : kAttnF32BM;
  p.qt_ref = ref_queries ? (d.n_ref + bm - 1) / bm : 0;
  p.qt_tgt = (d.n_tgt + bm - 1) / bm;
  const int64_t total = (int64_t)d.batch * d.heads * (p.qt_ref + p.qt_tgt);
  if (total > 0x7fffffff) return fail(RA_EUNSUPPORTED, "joint_attn: problem too large for one launch");
  p.total_tiles = (int32_t)total;

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

ra_status refadapt_cache_commit(int32_t batch, int32_t heads, int32_t n_ref, int32_t head_dim, int32_t dtype,
                                ra_tensor k_ref, ra_tensor v_ref, ra_tensor k_cache, ra_tensor v_cache,
                                const int32_t* decision, int32_t* age, int32_t step, void* stream) {
  if (batch < 1 || heads < 1 || n_ref < 0) return fail(RA_EINVAL, "cache_commit: bad sizes");
  if (dtype != RA_BF16 && dtype != RA_F32) return fail(RA_EINVAL, "cache_commit: unknown dtype %d", dtype);
  if (head_dim < 1 || (head_dim * (dtype == RA_BF16 ? 2 : 4)) % 16 != 0)
    return fail(RA_EUNSUPPORTED, "cache_commit: head_dim %d must fill whole 16-byte units", head_dim);
  if (n_ref == 0) return ok();
  ra_status s;
  if ((s = check_tensor("k_ref", k_ref, dtype, n_ref, head_dim)) != RA_OK) return s;
  if ((s = check_tensor("v_ref", v_ref, dtype, n_ref, head_dim)) != RA_OK) return s;
  if ((s = check_tensor("k_cache", k_cache, dtype, n_ref, head_dim)) != RA_OK) return s;
  if ((s = check_tensor("v_cache", v_cache, dtype, n_ref, head_dim)) != RA_OK) return s;
  const hipError_t e = launch_cache_commit(dtype, batch, heads, n_ref, head_dim, view(k_ref), view(v_ref),
                                           view(k_cache), view(v_cache), decision, age, step,
                                           static_cast<hipStream_t>(stream));
  return launch_status(e, "cache_commit");
}

}  // extern "C"
