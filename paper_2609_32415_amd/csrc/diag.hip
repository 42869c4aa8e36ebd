// Diagnostic sidecar kernels (gfx950). They only read the controller's tensors
// and write their own outputs, so the controlled path is bitwise unchanged with
// them on or off.
//   pair_partial / pair_final - relative Frobenius change ||cur - base||_F /
//       (||base||_F + eps) of one or two [B, H, n, d] slice pairs per (b, h), in
//       one launch pair, then combined per (b, h):
//         KV      endpoint drift of the reference K and of the reference V
//                 against their anchor values and the joint scalar E^KV, their
//                 mean (Sec. 3.3 endpoint-drift equation);
//         RATIO   consecutive drift of the reference and of the target slice of
//                 one of K, V and the matched log-ratio rho (Sec. 3.1
//                 consecutive-drift and drift-log-ratio equations);
//         SINGLE  the local perturbation I^KV of a stale-K/V output against the
//                 fresh output (Sec. 3.3 local-impact equation).
//   mass_mean - mean over query rows of the per-query reference mass, or of its
//       complement (the mass on target keys), per (b, h) (Sec. 3.2
//       directional-exposure equation, head-resolved).
//   adjacent_change - per block, the mean absolute change of the head-mean
//       reference mass between neighbouring steps, in percentage points
//       (Sec. 3.2 adjacent-ref-change equation).
// All are bandwidth- or latency-bound reductions with a fixed summation order:
// fp32 inside a workgroup, fp64 across workgroups and for the final ratios.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "internal.h"
#include "rowreduce.h"

namespace refadapt {
namespace {

constexpr int MM_THREADS = 256;
constexpr int MM_UNROLL = 8;
constexpr int AC_THREADS = 64;

// Pass 1: workgroup (chunk, bh, pair) sums (cur - base)^2 and base^2 over its rows.
template <bool BF16>
__global__ __launch_bounds__(QC_THREADS) void pair_partial(PairSet ps, int32_t H, int32_t head_dim,
                                                           int32_t chunks_max, float2* ws) {
  const int pair = blockIdx.z;
  const int chunks = ps.chunks[pair];
  if ((int)blockIdx.x >= chunks) return;  // whole workgroup: no barrier is skipped by part of it
  const int bh = blockIdx.y;
  const int b = bh / H, h = bh - b * H;
  const int2 rr = chunk_rows(ps.n_rows[pair], chunks);
  const float2 v = q_change_rows<BF16>(ps.cur[pair], ps.base[pair], b, h, rr.x, rr.y, head_dim);
  if (threadIdx.x == 0) ws[((int64_t)pair * gridDim.y + bh) * chunks_max + blockIdx.x] = v;
}

// Pass 2: a workgroup takes PF_HEADS (b, h) pairs, stages each pair's chunk partials in LDS
// (one coalesced memory round trip), and one thread per (b, h) adds them in chunk order in
// fp64 and combines the pairs.
constexpr int PF_THREADS = 256;
constexpr int PF_HEADS = 32;

__global__ __launch_bounds__(PF_THREADS) void pair_final(const float2* ws, PairSet ps, int32_t bh_total,
                                                         int32_t chunks_max, int32_t kind, float eps, float* out0,
                                                         float* out1, float* out2) {
  __shared__ float2 s_part[2][PF_HEADS * (QC_MAX_CHUNKS + 1)];
  const int h0 = blockIdx.x * PF_HEADS;
  const int nh = min(PF_HEADS, bh_total - h0);
  const int npairs = kind == PAIR_SINGLE ? 1 : 2;
  for (int pr = 0; pr < npairs; ++pr) {
    // pair pr's records of (b, h) lie at ws[(pr * bh_total + bh) * chunks_max + c], c < chunks
    const float2* src = ws + ((int64_t)pr * bh_total + h0) * chunks_max;
    const int n = nh * chunks_max;
    for (int i = threadIdx.x; i < n; i += PF_THREADS) {
      const int hh = i / chunks_max, c = i - hh * chunks_max;
      if (c < ps.chunks[pr]) s_part[pr][hh * (chunks_max + 1) + c] = src[i];
    }
  }
  __syncthreads();
  if ((int)threadIdx.x >= nh) return;
  const int bh = h0 + threadIdx.x;
  const double e = (double)eps;
  double d[2] = {0.0, 0.0};
  for (int pr = 0; pr < npairs; ++pr) {
    const float2* r = s_part[pr] + threadIdx.x * (chunks_max + 1);
    double a = 0.0, c = 0.0;
    for (int i = 0; i < ps.chunks[pr]; ++i) {
      a += r[i].x;
      c += r[i].y;
    }
    d[pr] = sqrt(a) / (sqrt(c) + e);
  }
  if (kind == PAIR_SINGLE) {
    out0[bh] = (float)d[0];
    return;
  }
  if (out0) out0[bh] = (float)d[0];
  if (out1) out1[bh] = (float)d[1];
  out2[bh] = (float)(kind == PAIR_KV ? 0.5 * (d[0] + d[1]) : log10((d[0] + e) / (d[1] + e)));
}

// One workgroup per (b, h): mean of mass (or 1 - mass) over n rows.
__global__ __launch_bounds__(MM_THREADS) void mass_mean_kernel(const float* mass, int32_t n, int32_t complement,
                                                               float* out) {
  const int bh = blockIdx.x;
  const float* m = mass + (int64_t)bh * n;
  float s = 0.f;
  // MM_UNROLL loads per thread in flight; the additions keep the plain strided order.
  for (int i0 = threadIdx.x; i0 < n; i0 += MM_UNROLL * MM_THREADS) {
    float v[MM_UNROLL];
#pragma unroll
    for (int u = 0; u < MM_UNROLL; ++u) v[u] = i0 + u * MM_THREADS < n ? m[i0 + u * MM_THREADS] : 0.f;
#pragma unroll
    for (int u = 0; u < MM_UNROLL; ++u) {
      if (i0 + u * MM_THREADS < n) s += complement ? 1.f - v[u] : v[u];
    }
  }
  s = wave_sum(s);
  __shared__ float red[MM_THREADS / 64];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    double a = 0.0;
#pragma unroll
    for (int w = 0; w < MM_THREADS / 64; ++w) a += red[w];
    out[bh] = (float)(a / n);
  }
}

// One thread per block: head means of the [T, n_blocks, bh] mass log, then
// 100 / (T - 1) * sum_t |mean_t - mean_{t-1}|.
__global__ __launch_bounds__(AC_THREADS) void adjacent_change_kernel(const float* m, int32_t T, int32_t nb,
                                                                     int32_t bh, float* out) {
  const int b = blockIdx.x * AC_THREADS + threadIdx.x;
  if (b >= nb) return;
  double prev = 0.0, acc = 0.0;
  for (int t = 0; t < T; ++t) {
    const float* row = m + ((int64_t)t * nb + b) * bh;
    double s = 0.0;
    for (int i = 0; i < bh; ++i) s += row[i];
    const double cur = s / bh;
    if (t > 0) acc += fabs(cur - prev);
    prev = cur;
  }
  out[b] = (float)(100.0 * acc / (T - 1));
}

}  // namespace

size_t pair_workspace_bytes(int32_t B, int32_t H, int32_t head_dim, int npairs, const int32_t* n_rows) {
  int cmax = 1;
  for (int i = 0; i < npairs; ++i) cmax = std::max(cmax, q_change_chunks(n_rows[i], head_dim));
  return (size_t)npairs * B * H * cmax * sizeof(float2);
}

hipError_t launch_pair_change(int dtype, int32_t B, int32_t H, int32_t head_dim, int npairs, PairSet ps, int kind,
                              float eps, float* out0, float* out1, float* out2, void* ws, hipStream_t stream) {
  int cmax = 1;
  for (int i = 0; i < npairs; ++i) {
    ps.chunks[i] = q_change_chunks(ps.n_rows[i], head_dim);
    cmax = std::max(cmax, ps.chunks[i]);
  }
  const dim3 grid(cmax, B * H, npairs);
  float2* w = static_cast<float2*>(ws);
  const hipError_t e =
      dtype == 0 ? launch_kernel(pair_partial<true>, grid, dim3(QC_THREADS), 0, stream, ps, H, head_dim, cmax, w)
                 : launch_kernel(pair_partial<false>, grid, dim3(QC_THREADS), 0, stream, ps, H, head_dim, cmax, w);
  if (e != hipSuccess) return e;
  const int bh = B * H;
  return launch_kernel(pair_final, dim3((bh + PF_HEADS - 1) / PF_HEADS), dim3(PF_THREADS), 0, stream, w, ps, bh,
                       cmax, kind, eps, out0, out1, out2);
}

hipError_t launch_mass_mean(int32_t B, int32_t H, int32_t n, const float* mass, int complement, float* out,
                            hipStream_t stream) {
  return launch_kernel(mass_mean_kernel, dim3(B * H), dim3(MM_THREADS), 0, stream, mass, n, complement, out);
}

hipError_t launch_adjacent_change(int32_t T, int32_t nb, int32_t bh, const float* m, float* out,
                                  hipStream_t stream) {
  return launch_kernel(adjacent_change_kernel, dim3((nb + AC_THREADS - 1) / AC_THREADS), dim3(AC_THREADS), 0,
                       stream, m, T, nb, bh, out);
}

}  // namespace refadapt
