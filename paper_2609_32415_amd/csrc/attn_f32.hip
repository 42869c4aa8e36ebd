// Joint attention over [reference; target] keys in fp32 (vector ALU).
//
// The fp32 path serves small fp32 workloads where the output must match an
// fp64 evaluation to ~1e-5; it is not a throughput path. One workgroup = one
// wavefront = 64 query rows, one row per lane. Key/value tiles of 32 rows are
// staged in LDS (every lane reads the same key row: an LDS broadcast), the
// query tile sits in LDS with a padded row stride, and the online softmax
// keeps the same split (reference, target) statistics as the bf16 kernel.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace refadapt {
namespace {

constexpr int BQ = kAttnF32BM;
constexpr int BK = 32;

template <int D>
__global__ __launch_bounds__(BQ) void attn_f32_kernel(AttnParams p) {
  __shared__ float qs[BQ][D + 1];
  __shared__ float ks[BK][D];
  __shared__ float vs[BK][D];

  const int lane = threadIdx.x;
  const int tile = xcd_remap(blockIdx.x, p.total_tiles);
  const int qt_bh = p.qt_ref + p.qt_tgt;
  const int bh = tile / qt_bh;
  int qt = tile - bh * qt_bh;
  const int b = bh / p.H, h = bh - b * p.H;
  const bool ref_rows = qt < p.qt_ref;
  if (!ref_rows) qt -= p.qt_ref;

  bool use_cache = p.kvsrc == KV_CACHE;
  if (p.kvsrc == KV_DEVICE) {
    const int dec = *p.decision;
    if (ref_rows && dec == DEC_REUSE) return;
    use_cache = dec != DEC_COMPUTE;
  }
  const View& qv = ref_rows ? (use_cache && p.q_cache.p ? p.q_cache : p.q_ref) : p.q_tgt;
  const View& ov = ref_rows ? p.o_ref : p.o_tgt;
  const int n_rows = ref_rows ? p.n_ref : p.n_tgt;
  const View& krv = use_cache ? p.k_cache : p.k_fresh;
  const View& vrv = use_cache ? p.v_cache : p.v_fresh;

  const int row0 = qt * BQ;
  const float* qbase = static_cast<const float*>(qv.p) + b * qv.sb + h * qv.sh;
  for (int i = lane; i < BQ * D; i += BQ) {
    const int r = i / D, cidx = i % D;
    qs[r][cidx] = row0 + r < n_rows ? qbase[(int64_t)(row0 + r) * qv.ss + cidx] : 0.f;
  }

  float o[D];
#pragma unroll
  for (int i = 0; i < D; ++i) o[i] = 0.f;
  float m_run = -__builtin_inff(), l_run = 0.f, m_ref = -__builtin_inff(), l_ref = 0.f;
  const float c = p.sc_log2;

  const int n_rt = (p.n_ref + BK - 1) / BK;
  const int n_yt = (p.n_tgt + BK - 1) / BK;
  for (int j = 0; j < n_rt + n_yt; ++j) {
    const bool rseg = j < n_rt;
    const View& kv = rseg ? krv : p.k_tgt;
    const View& vv = rseg ? vrv : p.v_tgt;
    const int key0 = (rseg ? j : j - n_rt) * BK;
    const int valid = min(BK, (rseg ? p.n_ref : p.n_tgt) - key0);
    const float* kb = static_cast<const float*>(kv.p) + b * kv.sb + h * kv.sh + (int64_t)key0 * kv.ss;
    const float* vb = static_cast<const float*>(vv.p) + b * vv.sb + h * vv.sh + (int64_t)key0 * vv.ss;
    __syncthreads();
    for (int i = lane; i < BK * D; i += BQ) {
      const int r = i / D, cidx = i % D;
      ks[r][cidx] = r < valid ? kb[(int64_t)r * kv.ss + cidx] : 0.f;
      vs[r][cidx] = r < valid ? vb[(int64_t)r * vv.ss + cidx] : 0.f;
    }
    __syncthreads();

    float sc[BK];
    float mx = -__builtin_inff();
#pragma unroll
    for (int k = 0; k < BK; ++k) {
      float dot = 0.f;
#pragma unroll 16
      for (int i = 0; i < D; ++i) dot = fmaf(qs[lane][i], ks[k][i], dot);
      sc[k] = k < valid ? dot * c : -__builtin_inff();
      mx = fmaxf(mx, sc[k]);
    }
    const float m_new = fmaxf(m_run, mx);
    const float alpha = exp2f(m_run - m_new);
    float rs = 0.f;
#pragma unroll
    for (int k = 0; k < BK; ++k) {
      sc[k] = exp2f(sc[k] - m_new);
      rs += sc[k];
    }
    l_run = l_run * alpha + rs;
    m_run = m_new;
#pragma unroll 8
    for (int i = 0; i < D; ++i) {
      float acc = o[i] * alpha;
#pragma unroll
      for (int k = 0; k < BK; ++k) acc = fmaf(sc[k], vs[k][i], acc);
      o[i] = acc;
    }
    if (j == n_rt - 1) {
      m_ref = m_run;
      l_ref = l_run;
      l_run = 0.f;
    }
  }

  const int qrow = row0 + lane;
  if (qrow >= n_rows) return;
  const float L_R = l_ref > 0.f ? l_ref * exp2f(m_ref - m_run) : 0.f;
  const float total = L_R + l_run;
  float* op = static_cast<float*>(const_cast<void*>(ov.p)) + b * ov.sb + h * ov.sh + (int64_t)qrow * ov.ss;
#pragma unroll
  for (int i = 0; i < D; ++i) op[i] = o[i] / total;
  const int64_t row = (int64_t)bh * n_rows + qrow;
  const float mass = L_R / total;
  if (!ref_rows) {
    if (p.mass_tgt) p.mass_tgt[row] = mass;
    if (p.lse_tgt) {
      const float ln2 = 0.69314718055994531f;
      p.lse_tgt[2 * row] = (m_ref + log2f(l_ref)) * ln2;
      p.lse_tgt[2 * row + 1] = (m_run + log2f(total)) * ln2;
    }
  } else if (p.mass_refq) {
    p.mass_refq[row] = mass;
  }
}

}  // namespace

hipError_t launch_attn_f32(const AttnParams& p, int head_dim, hipStream_t stream) {
  if (p.total_tiles <= 0) return hipSuccess;
  const dim3 grid(p.total_tiles), block(BQ);
  return head_dim == 128 ? launch_kernel(attn_f32_kernel<128>, grid, block, 0, stream, p)
                         : launch_kernel(attn_f32_kernel<64>, grid, block, 0, stream, p);
}

}  // namespace refadapt
