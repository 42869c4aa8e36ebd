// Controller statistics and cache maintenance (gfx950):
//   q_change  - relative Frobenius change of the target queries per (b, h)
//               (paper Sec. 3.1 consecutive-drift equation on post-RoPE target Q)
//   gate      - head-mean interaction score and the block decision
//               (Sec. 4 factorized-risk and depth-cutoff equations; Alg. 1)
//   q_change_gate - both in two launches: every Q-change workgroup also sums the
//               lagged mass over its rows; one workgroup then adds up and decides
//   commit    - device-conditional refresh of a block's cached reference state (K, V, Q)
//
// All are bandwidth- or latency-bound; they use 16-byte coalesced loads and
// fixed-order reductions, so every result is bitwise reproducible.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"
#include "rowreduce.h"

namespace refadapt {
namespace {

// Pass 1: one workgroup sums (cur - prev)^2 and prev^2 over a chunk of rows of one (b, h).
template <bool BF16>
__global__ __launch_bounds__(QC_THREADS) void q_change_partial(View cur, View prev, int32_t H, int32_t n_rows,
                                                               int32_t head_dim, int32_t chunks, float2* ws) {
  const int bh = blockIdx.y;
  const int b = bh / H, h = bh - b * H;
  const int2 rr = chunk_rows(n_rows, chunks);
  const float2 v = q_change_rows<BF16>(cur, prev, b, h, rr.x, rr.y, head_dim);
  if (threadIdx.x == 0) ws[(int64_t)bh * chunks + blockIdx.x] = v;
}

// Pass 2: a workgroup takes QF_HEADS (b, h) pairs, stages their chunk partials in LDS (one
// coalesced memory round trip), and one thread per pair adds them in chunk order in fp64.
constexpr int QF_THREADS = 256;
constexpr int QF_HEADS = 64;

__global__ __launch_bounds__(QF_THREADS) void q_change_final(const float2* ws, int32_t bh_total, int32_t chunks,
                                                             float eps, float* out) {
  __shared__ float2 s_part[QF_HEADS * (QC_MAX_CHUNKS + 1)];
  const int h0 = blockIdx.x * QF_HEADS;
  const int nh = min(QF_HEADS, bh_total - h0);
  stage_partials(s_part, ws, h0, nh, chunks);
  __syncthreads();
  if ((int)threadIdx.x >= nh) return;
  const float2* r = s_part + threadIdx.x * (chunks + 1);
  double a = 0.0, c = 0.0;
  for (int i = 0; i < chunks; ++i) {
    a += r[i].x;
    c += r[i].y;
  }
  out[h0 + threadIdx.x] = (float)(sqrt(a) / (sqrt(c) + (double)eps));
}

// Alg. 1 block branch on one thread: step bookkeeping at block 0 (step 0, or step -
// a_full >= delta_max with delta_max > 0, is a full refresh: every block of the step
// computes), then COMPUTE if an earlier block reactivated, else REACTIVATE when the
// head-mean score reaches theta, else REUSE. d[i], m[i] are the Q-change and the mean
// lagged mass of (b, h) pair i; the head means are taken in fp64 in index order.
// The state and this block's thresholds come in registers (the kernels load them before
// their reductions, so the loads' latency is hidden); the updated state is stored back.
struct GateInputs {
  GateState st;
  float th0, th1;  // theta[block], or theta[2 block], theta[2 block + 1] for the AND mode
};

__device__ __forceinline__ GateInputs gate_load(const GateState* st, const float* theta, int32_t block,
                                                int32_t mode) {
  GateInputs g;
  g.st = *st;
  g.th0 = theta[mode == 3 ? 2 * block : block];
  g.th1 = mode == 3 ? theta[2 * block + 1] : 0.f;
  return g;
}

__device__ void gate_decide(int32_t BH, int32_t block, int32_t step, int32_t mode, const float* d, const float* m,
                            GateInputs g, GateState* st, int32_t* decision_out, float* score_out) {
  GateState s = g.st;
  if (block == 0) {
    const bool full = step == 0 || (s.delta_max > 0 && step - s.a_full >= s.delta_max);
    if (full) s.a_full = step;
    s.reactivated = full ? 1 : 0;
    s.step = step;
  }
  double sd = 0.0, sm = 0.0, sg = 0.0;
  for (int i = 0; i < BH; ++i) {
    const double di = d[i], mi = m[i];
    sd += di;
    sm += mi;
    sg += di * mi;  // per-head product before the mean
  }
  const double dm = sd / BH, mm = sm / BH, gm = sg / BH;
  int dec;
  if (s.reactivated) {
    dec = DEC_COMPUTE;
  } else {
    bool cross;
    if (mode == 0) {
      cross = gm >= (double)g.th0;
    } else if (mode == 1) {
      cross = dm >= (double)g.th0;
    } else if (mode == 2) {
      cross = mm >= (double)g.th0;
    } else {
      cross = dm >= (double)g.th0 && mm >= (double)g.th1;
    }
    dec = cross ? DEC_REACTIVATE : DEC_REUSE;
    if (cross) s.reactivated = 1;
  }
  *st = s;
  *decision_out = dec;
  score_out[0] = (float)dm;
  score_out[1] = (float)mm;
  score_out[2] = (float)gm;
}

constexpr int GATE_THREADS = 1024;
constexpr int GATE_UNROLL = 16;  // 16-byte loads per lane in flight

__global__ __launch_bounds__(GATE_THREADS) void gate_kernel(int32_t BH, int32_t n_tgt, int32_t block, int32_t step,
                                                            int32_t mode, const float* d_cur, const float* mass_prev,
                                                            const float* theta, GateState* st, int32_t* decision_out,
                                                            float* score_out) {
  extern __shared__ float s_dm[];  // [2 * BH]: D (copied from d_cur), then the mean lagged mass
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  GateInputs gin{};
  if (tid == 0) gin = gate_load(st, theta, block, mode);
  for (int i = tid; i < BH; i += GATE_THREADS) s_dm[i] = d_cur[i];

  // Mean over target queries of the lagged per-query reference mass, one wavefront per
  // (b, h): 16-byte loads, GATE_UNROLL in flight per lane (a 4096-query row is one round
  // trip to memory), then a fixed-order butterfly. Loads past the row's end read as zeros,
  // which add exactly +0.
  for (int bh = wave; bh < BH; bh += GATE_THREADS / 64) {
    const float* row = mass_prev + (int64_t)bh * n_tgt;
    float s = 0.f;
    int i0 = 0;
    if ((reinterpret_cast<uintptr_t>(row) & 15) == 0) {
      const int n4 = n_tgt >> 2;
      const float4* r4 = reinterpret_cast<const float4*>(row);
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int k0 = lane; k0 < n4; k0 += 64 * GATE_UNROLL) {
        float4 v[GATE_UNROLL];
#pragma unroll
        for (int u = 0; u < GATE_UNROLL; ++u) {
          const int k = k0 + 64 * u;
          v[u] = k < n4 ? r4[k] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < GATE_UNROLL; ++u) {
          acc.x += v[u].x;
          acc.y += v[u].y;
          acc.z += v[u].z;
          acc.w += v[u].w;
        }
      }
      s = (acc.x + acc.y) + (acc.z + acc.w);
      i0 = n4 << 2;
    }
    for (int i = i0 + lane; i < n_tgt; i += 64) s += row[i];
    s = wave_sum(s);
    if (lane == 0) s_dm[BH + bh] = s / (float)n_tgt;
  }
  __syncthreads();
  if (tid == 0) gate_decide(BH, block, step, mode, s_dm, s_dm + BH, gin, st, decision_out, score_out);
}

// Q-change and gate in two launches (instead of three). Pass 1: workgroup (chunk, bh)
// sums the Q-change terms and the lagged mass over its rows. Pass 2 (one workgroup):
// per (b, h) the chunks are added in chunk order in fp64, D is written, and the mean
// mass and D feed the decision.
template <bool BF16>
__global__ __launch_bounds__(QC_THREADS) void q_change_mass_partial(View cur, View prev, int32_t H, int32_t n_rows,
                                                                    int32_t head_dim, int32_t chunks,
                                                                    const float* mass_prev, float4* part) {
  __shared__ float red[QC_THREADS / 64];
  const int bh = blockIdx.y;
  const int b = bh / H, h = bh - b * H;
  const int2 rr = chunk_rows(n_rows, chunks);
  // The first MP lagged-mass values of this thread's rows are loaded before the Q-change
  // loads, so both share one memory round trip; the per-thread order is the strided one.
  constexpr int MP = 4;
  const float* mrow = mass_prev + (int64_t)bh * n_rows;
  float mv[MP];
#pragma unroll
  for (int k = 0; k < MP; ++k) {
    const int i = rr.x + threadIdx.x + k * QC_THREADS;
    mv[k] = i < rr.y ? mrow[i] : 0.f;
  }
  const float2 v = q_change_rows<BF16>(cur, prev, b, h, rr.x, rr.y, head_dim);
  float sm = 0.f;
#pragma unroll
  for (int k = 0; k < MP; ++k) sm += mv[k];
  for (int i = rr.x + threadIdx.x + MP * QC_THREADS; i < rr.y; i += QC_THREADS) sm += mrow[i];
  sm = wave_sum(sm);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = sm;
  __syncthreads();
  if (threadIdx.x == 0) {
    float msum = 0.f;
#pragma unroll
    for (int w = 0; w < QC_THREADS / 64; ++w) msum += red[w];
    part[(int64_t)bh * chunks + blockIdx.x] = make_float4(v.x, v.y, msum, 0.f);
  }
}

constexpr int QG_THREADS = 256;
constexpr int QG_STAGE = 1024;  // float4 partial records staged in LDS per round (16 KiB)

// Pass 2 of the fused Q-change + gate (one workgroup): rounds of (b, h) pairs have their
// chunk partials staged in LDS (one coalesced memory round trip per round, a single round
// up to 1024 / chunks pairs); one thread per pair adds them in chunk order in fp64 and
// writes D and the mean lagged mass; then thread 0 decides.
__global__ __launch_bounds__(QG_THREADS) void q_change_gate_final(const float4* part, int32_t BH, int32_t chunks,
                                                                  int32_t n_rows, float eps, int32_t block,
                                                                  int32_t step, int32_t mode, const float* theta,
                                                                  GateState* st, float* d_out, int32_t* decision_out,
                                                                  float* score_out) {
  extern __shared__ float s_dm[];  // [2 * BH]: D, then the mean lagged mass of each (b, h)
  // a round holds nh <= QG_STAGE / chunks pairs (at most QG_THREADS) of chunks + 1 records
  __shared__ float4 s_part[QG_STAGE + QG_THREADS];
  GateInputs gin{};
  if (threadIdx.x == 0) gin = gate_load(st, theta, block, mode);
  const int per_round = max(1, min(QG_THREADS, QG_STAGE / chunks));
  for (int h0 = 0; h0 < BH; h0 += per_round) {
    const int nh = min(per_round, BH - h0);
    stage_partials(s_part, part, h0, nh, chunks);
    __syncthreads();
    if ((int)threadIdx.x < nh) {
      const float4* r = s_part + threadIdx.x * (chunks + 1);
      double a = 0.0, c = 0.0, ms = 0.0;
      for (int k = 0; k < chunks; ++k) {
        a += r[k].x;
        c += r[k].y;
        ms += r[k].z;
      }
      const int i = h0 + threadIdx.x;
      const float dv = (float)(sqrt(a) / (sqrt(c) + (double)eps));
      d_out[i] = dv;
      s_dm[i] = dv;
      s_dm[BH + i] = (float)(ms / n_rows);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) gate_decide(BH, block, step, mode, s_dm, s_dm + BH, gin, st, decision_out, score_out);
}

constexpr int CC_THREADS = 256;

// Copies pair blockIdx.z of `cs` (source -> destination, [B, H, n_rows, d]) with 16-byte
// vectors; exits at once unless the decision is COMPUTE (or absent).
__global__ __launch_bounds__(CC_THREADS) void cache_commit_kernel(CommitSet cs, int32_t H, int32_t n_rows,
                                                                  int32_t vpr, int32_t esz, const int32_t* decision,
                                                                  int32_t* age, int32_t step) {
  if (decision && *decision != DEC_COMPUTE) return;
  const int bh = blockIdx.y;
  const int b = bh / H, h = bh - b * H;
  const View src = cs.src[blockIdx.z], dst = cs.dst[blockIdx.z];
  const int64_t nvec = (int64_t)n_rows * vpr;
  const int vec = 16 / esz;
  const char* sb = static_cast<const char*>(src.p) + (b * src.sb + h * src.sh) * esz;
  char* db = static_cast<char*>(const_cast<void*>(dst.p)) + (b * dst.sb + h * dst.sh) * esz;
  for (int64_t v = (int64_t)blockIdx.x * CC_THREADS + threadIdx.x; v < nvec; v += (int64_t)gridDim.x * CC_THREADS) {
    const int64_t row = v / vpr;
    const int col = (int)(v % vpr) * vec;
    const u32x4 x = *reinterpret_cast<const u32x4*>(sb + (row * src.ss + col) * esz);
    *reinterpret_cast<u32x4*>(db + (row * dst.ss + col) * esz) = x;
  }
  if (age && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && threadIdx.x == 0) *age = step;
}

}  // namespace

int q_change_chunks(int32_t n_tgt, int32_t head_dim) {
  const int64_t elems = (int64_t)n_tgt * head_dim;
  int64_t c = (elems + QC_TARGET_ELEMS - 1) / QC_TARGET_ELEMS;
  if (c < 1) c = 1;
  if (c > QC_MAX_CHUNKS) c = QC_MAX_CHUNKS;
  if (c > n_tgt) c = n_tgt;
  return (int)c;
}

hipError_t launch_q_change(int dtype, int32_t B, int32_t H, int32_t n_tgt, int32_t head_dim, View cur, View prev,
                           float eps, float* d_out, void* ws, hipStream_t stream) {
  const int chunks = q_change_chunks(n_tgt, head_dim);
  const dim3 grid(chunks, B * H);
  float2* w = static_cast<float2*>(ws);
  const hipError_t e =
      dtype == 0
          ? launch_kernel(q_change_partial<true>, grid, dim3(QC_THREADS), 0, stream, cur, prev, H, n_tgt, head_dim,
                          chunks, w)
          : launch_kernel(q_change_partial<false>, grid, dim3(QC_THREADS), 0, stream, cur, prev, H, n_tgt, head_dim,
                          chunks, w);
  if (e != hipSuccess) return e;
  const int bh = B * H;
  return launch_kernel(q_change_final, dim3((bh + QF_HEADS - 1) / QF_HEADS), dim3(QF_THREADS), 0, stream, w, bh,
                       chunks, eps, d_out);
}

hipError_t launch_gate(int32_t B, int32_t H, int32_t n_tgt, int32_t block, int32_t step, int32_t mode,
                       const float* d_cur, const float* mass_prev, const float* theta, GateState* state,
                       int32_t* decision_out, float* score_out, hipStream_t stream) {
  const int bh = B * H;
  return launch_kernel(gate_kernel, dim3(1), dim3(GATE_THREADS), 2 * (size_t)bh * sizeof(float), stream, bh, n_tgt,
                       block, step, mode, d_cur, mass_prev, theta, state, decision_out, score_out);
}

size_t q_change_gate_workspace_bytes(int32_t B, int32_t H, int32_t n_tgt, int32_t head_dim) {
  return (size_t)B * H * q_change_chunks(n_tgt, head_dim) * sizeof(float4);
}

hipError_t launch_q_change_gate(int dtype, int32_t B, int32_t H, int32_t n_tgt, int32_t head_dim, View cur, View prev,
                                float eps, int32_t block, int32_t step, int32_t mode, const float* mass_prev,
                                const float* theta, GateState* state, float* d_out, int32_t* decision_out,
                                float* score_out, void* ws, hipStream_t stream) {
  const int chunks = q_change_chunks(n_tgt, head_dim);
  const dim3 grid(chunks, B * H);
  float4* part = static_cast<float4*>(ws);
  const hipError_t e =
      dtype == 0 ? launch_kernel(q_change_mass_partial<true>, grid, dim3(QC_THREADS), 0, stream, cur, prev, H, n_tgt,
                                 head_dim, chunks, mass_prev, part)
                 : launch_kernel(q_change_mass_partial<false>, grid, dim3(QC_THREADS), 0, stream, cur, prev, H, n_tgt,
                                 head_dim, chunks, mass_prev, part);
  if (e != hipSuccess) return e;
  const int bh = B * H;
  return launch_kernel(q_change_gate_final, dim3(1), dim3(QG_THREADS), 2 * (size_t)bh * sizeof(float), stream,
                       static_cast<const float4*>(part), bh, chunks, n_tgt, eps, block, step, mode, theta, state, d_out,
                       decision_out, score_out);
}

hipError_t launch_cache_commit(int dtype, int32_t B, int32_t H, int32_t n_ref, int32_t head_dim, CommitSet cs,
                               const int32_t* decision, int32_t* age, int32_t step, hipStream_t stream) {
  const int esz = dtype == 0 ? 2 : 4;
  const int vpr = head_dim * esz / 16;
  const int64_t nvec = (int64_t)n_ref * vpr;
  int gx = (int)((nvec + CC_THREADS * 4 - 1) / (CC_THREADS * 4));
  if (gx < 1) gx = 1;
  if (gx > 1024) gx = 1024;
  return launch_kernel(cache_commit_kernel, dim3(gx, B * H, cs.n), dim3(CC_THREADS), 0, stream, cs, H, n_ref, vpr,
                       esz, decision, age, step);
}

}  // namespace refadapt
