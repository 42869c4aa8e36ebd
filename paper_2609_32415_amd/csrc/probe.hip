// Matrix-core rate probes for the measurement harness (not part of the method): the bf16
// MFMA rate one MI355X sustains when every operand sits in registers, so no LDS read, no
// global load and no barrier takes part. The joint-attention kernel issues the same
// matrix instructions plus exactly those, so these rates bound it from above at the clock
// the device holds under such load.
//
//   RA_PROBE_DENSE: 32 v_mfma_f32_32x32x16_bf16 per step in two accumulation chains.
//   RA_PROBE_MIX:   the attention's per-key-tile register work: 16 MFMAs of a 64 x 32 score tile,
//                   then 16 MFMAs of a 128 x 32 output tile whose B operands are the bf16
//                   probabilities of the previous score tile; under the MFMAs, 16 pairs of
//                   scores each take two FMAs (scale, max), two exp2, two row-sum adds and
//                   one bf16 pack, spread over three consecutive MFMA slots as the attention
//                   does; after the last MFMA one dot2 per packed pair sums the rounded
//                   probabilities.
//
// One workgroup of eight wavefronts per CU (two per SIMD, as the attention runs). Operands
// are read once from a caller buffer of random bf16 values (their bit patterns, like the
// attention's inputs, set the matrix core's switching power).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace refadapt {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int PT = 512;  // threads per workgroup

template <typename T>
__device__ __forceinline__ void keep(T& v) {
  asm volatile("" : "+v"(v));
}

template <bool MIX>
__global__ __launch_bounds__(PT, 1) void mfma_rate_kernel(const bf16x8* operands, int32_t steps, float* sink,
                                                          unsigned long long* clock_probe) {
  // More than half of a CU's 160 KiB of LDS, so the device places one workgroup per CU, as
  // it does the attention's (whose register use allows no second one).
  __shared__ float hold[21 * 1024];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t clk0 = 0, rt0 = 0;
  if (clock_probe && threadIdx.x == 0) {
    clk0 = __builtin_amdgcn_s_memtime();
    rt0 = __builtin_amdgcn_s_memrealtime();
  }
  // 16 operand blocks of 8 bf16 per lane: four A (key), eight B (query), four A (value).
  bf16x8 a[4], b[8], v[4];
  const bf16x8* src = operands + (size_t)(wave & 3) * 64 * 16 + lane * 16;
#pragma unroll
  for (int i = 0; i < 4; ++i) a[i] = src[i];
#pragma unroll
  for (int i = 0; i < 8; ++i) b[i] = src[4 + i];
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = src[12 + i];
  float acc = 0.f;
  if constexpr (!MIX) {
    f32x16 c0 = {}, c1 = {};
    for (int s = 0; s < steps; ++s) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i & 3], b[i & 7], c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(i + 1) & 3], b[(i + 3) & 7], c1, 0, 0, 0);
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) acc += c0[r] + c1[r];
  } else {
    const float c = 0.12753102f;  // 1/sqrt(128) * log2(e), the head_dim-128 softmax scale
    const float m = 1.0f;
    f32x16 sa[2], sb[2], o[4] = {};
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      sa[mb] = f32x16{};
#pragma unroll
      for (int kk = 0; kk < 8; ++kk)
        sa[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(kk + mb) & 3], b[kk], sa[mb], 0, 0, 0);
    }
    float rs = 0.f, lo = 0.f;
    uint32_t pw[4][4];
    // One step: the score MFMAs of the next tile into s_next, the output MFMAs of this tile,
    // and the 16 probability pairs of s_cur (scores 2q, 2q + 1 -> P block q / 4, word q % 4).
    auto step = [&](f32x16(&s_cur)[2], f32x16(&s_next)[2]) {
      // Pair q (scores 2q, 2q + 1 -> P block q / 4, word q % 4) in three stages over three
      // consecutive MFMA slots, as the attention schedules them: exponent arguments, then
      // the exponentials, then the row-sum adds and the bf16 pack.
      float pa0 = 0.f, pa1 = 0.f, pe0 = 0.f, pe1 = 0.f;
      auto slot = [&](int k, int first, int end) {  // pairs first .. end - 1
        if (k - 2 >= first && k - 2 < end) {
          const int q = k - 2;
          rs = rs + (pe0 + pe1);
          keep(rs);
          bf16x2 pr;
          pr[0] = (__bf16)pe0;
          pr[1] = (__bf16)pe1;
          uint32_t w = __builtin_bit_cast(uint32_t, pr);
          keep(w);
          pw[q >> 2][q & 3] = w;
        }
        if (k - 1 >= first && k - 1 < end) {
          pe0 = __builtin_amdgcn_exp2f(pa0);
          pe1 = __builtin_amdgcn_exp2f(pa1);
          keep(pe0);
          keep(pe1);
        }
        if (k >= first && k < end) {
          const int mb = k >> 3, o2 = (2 * k) & 15;
          pa0 = fmaf(s_cur[mb][o2], c, -m);
          pa1 = fmaf(s_cur[mb][o2 + 1], c, -m);
          keep(pa0);
          keep(pa1);
        }
      };
      // The operands are opaque to the compiler at every step (as the attention's, read
      // from LDS, are), so no score MFMA is hoisted out of the loop.
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        keep(a[i]);
        keep(v[i]);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) keep(b[i]);
      s_next[0] = f32x16{};
      s_next[1] = f32x16{};
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        // key block i >> 3 pairs its A registers with the query blocks in another order
        s_next[i >> 3] =
            __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(i + (i >> 3)) & 3], b[i & 7], s_next[i >> 3], 0, 0, 0);
        if (i < 12) slot(i, 0, 10);  // pairs 0..9
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int blk = i >> 2;
        const u32x4 pv = {pw[blk][0], pw[blk][1], pw[blk][2], pw[blk][3]};
        o[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v[i & 3], __builtin_bit_cast(bf16x8, pv), o[i & 3], 0, 0, 0);
        if (i < 8) slot(10 + i, 10, 16);  // pairs 10..15, P blocks 2 and 3 complete before MFMA 8
        __builtin_amdgcn_sched_barrier(0);
      }
      // the sum of the rounded probabilities, one dot2 per packed pair after the last MFMA
      const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
      for (int w = 0; w < 16; ++w)
        lo = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw[w >> 2][w & 3]), one, lo, false);
      keep(lo);
    };
    int s = 0;
    for (; s + 1 < steps; s += 2) {  // two steps per iteration, so the score tiles swap roles
      step(sa, sb);
      step(sb, sa);
    }
    if (s < steps) step(sa, sb);
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc += o[d][r];
    acc += rs + lo;
  }
  if (steps < 0) {  // never taken (the host requires steps >= 1); keeps the LDS allocation
    hold[threadIdx.x] = acc;
    __syncthreads();
    acc += hold[threadIdx.x ^ 1];
  }
  sink[(size_t)blockIdx.x * PT + threadIdx.x] = acc;
  if (clock_probe && threadIdx.x == 0) {
    const uint64_t clk1 = __builtin_amdgcn_s_memtime(), rt1 = __builtin_amdgcn_s_memrealtime();
    atomicAdd(clock_probe, (unsigned long long)(clk1 - clk0));
    atomicAdd(clock_probe + 1, (unsigned long long)(rt1 - rt0));
  }
}

}  // namespace

hipError_t launch_mfma_rate(int kind, int32_t workgroups, int32_t steps, const void* operands, float* sink,
                            unsigned long long* clock_probe, hipStream_t stream) {
  const bf16x8* ops = static_cast<const bf16x8*>(operands);
  return kind == 0 ? launch_kernel(mfma_rate_kernel<false>, dim3(workgroups), dim3(PT), 0, stream, ops, steps, sink,
                                   clock_probe)
                   : launch_kernel(mfma_rate_kernel<true>, dim3(workgroups), dim3(PT), 0, stream, ops, steps, sink,
                                   clock_probe);
}

}  // namespace refadapt
