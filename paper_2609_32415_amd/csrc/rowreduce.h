// Fixed-order row reductions shared by the statistics and diagnostics kernels.
// Every sum runs in the same order on every call, so results are bitwise
// reproducible. Device code only; the definitions have internal linkage in
// every source that includes this header.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace refadapt {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int QC_THREADS = 256;
constexpr int QC_TARGET_ELEMS = 16384;  // elements of one tensor per workgroup (32 KiB of bf16)
constexpr int QC_MAX_CHUNKS = 64;
constexpr int QC_UNROLL = 8;  // 16-byte vectors of each tensor per thread in flight

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Fixed-order wavefront reduction (butterfly over the 64 lanes).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// Stages the chunk partials of heads [h0, h0 + nh) (`chunks` records of T per head, head
// major) in LDS with coalesced loads by the whole workgroup, head i at s[i * (chunks + 1)]
// (the padding spreads the per-head rows over the banks). One memory round trip.
template <typename T>
__device__ __forceinline__ void stage_partials(T* s, const T* part, int h0, int nh, int chunks) {
  const int n = nh * chunks;
  const T* src = part + (int64_t)h0 * chunks;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const int hh = i / chunks, c = i - hh * chunks;
    s[hh * (chunks + 1) + c] = src[i];
  }
}

// Sums (cur - prev)^2 and prev^2 over rows [r0, r1) of one (b, h), returned to thread 0
// in a fixed order (per-thread fp32, wavefront butterfly, then wavefronts in order).
template <bool BF16>
__device__ __forceinline__ float2 q_change_rows(View cur, View prev, int b, int h, int r0, int r1, int32_t head_dim) {
  const int vec = BF16 ? 8 : 4;  // elements per 16-byte load
  const int vpr = head_dim / vec;
  const int nvec = max(0, r1 - r0) * vpr;
  const char* cb = static_cast<const char*>(cur.p);
  const char* pb = static_cast<const char*>(prev.p);
  const int esz = BF16 ? 2 : 4;
  const int64_t cbase = (b * cur.sb + h * cur.sh) * esz;
  const int64_t pbase = (b * prev.sb + h * prev.sh) * esz;

  float sd = 0.f, sp = 0.f;
  // QC_UNROLL vectors of each tensor are loaded before any is used, so each thread keeps
  // 2 * QC_UNROLL loads in flight. Vectors past the end load as zeros, which add exactly
  // +0 to both sums: the per-thread order is the plain strided order.
  for (int v0 = threadIdx.x; v0 < nvec; v0 += QC_UNROLL * QC_THREADS) {
    u32x4 xs[QC_UNROLL], ys[QC_UNROLL];
#pragma unroll
    for (int u = 0; u < QC_UNROLL; ++u) {
      const int v = v0 + u * QC_THREADS;
      xs[u] = ys[u] = u32x4{0u, 0u, 0u, 0u};
      if (v < nvec) {
        const int row = r0 + v / vpr, col = (v % vpr) * vec;
        xs[u] = *reinterpret_cast<const u32x4*>(cb + cbase + ((int64_t)row * cur.ss + col) * esz);
        ys[u] = *reinterpret_cast<const u32x4*>(pb + pbase + ((int64_t)row * prev.ss + col) * esz);
      }
    }
#pragma unroll
    for (int u = 0; u < QC_UNROLL; ++u) {
      const u32x4 x = xs[u], y = ys[u];
      if (BF16) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float a0 = bf16_lo(x[i]), a1 = bf16_hi(x[i]);
          const float p0 = bf16_lo(y[i]), p1 = bf16_hi(y[i]);
          const float d0 = a0 - p0, d1 = a1 - p1;
          sd = fmaf(d0, d0, sd);
          sd = fmaf(d1, d1, sd);
          sp = fmaf(p0, p0, sp);
          sp = fmaf(p1, p1, sp);
        }
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float a = __uint_as_float(x[i]), pp = __uint_as_float(y[i]);
          const float d = a - pp;
          sd = fmaf(d, d, sd);
          sp = fmaf(pp, pp, sp);
        }
      }
    }
  }
  sd = wave_sum(sd);
  sp = wave_sum(sp);
  __shared__ float red[2][QC_THREADS / 64];
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[0][wave] = sd;
    red[1][wave] = sp;
  }
  __syncthreads();
  float a = 0.f, c = 0.f;
#pragma unroll
  for (int w = 0; w < QC_THREADS / 64; ++w) {
    a += red[0][w];
    c += red[1][w];
  }
  return make_float2(a, c);
}

// Rows [r0, r1) of one (b, h) of chunk blockIdx.x out of `chunks` equal row ranges.
__device__ __forceinline__ int2 chunk_rows(int n_rows, int chunks) {
  const int rows_per = (n_rows + chunks - 1) / chunks;
  const int r0 = blockIdx.x * rows_per;
  return make_int2(r0, min(n_rows, r0 + rows_per));
}

}  // namespace
}  // namespace refadapt
