// Internal interface between the C-ABI layer (api.hip) and the kernels.
// Nothing here is exported from the shared library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <tuple>

namespace refadapt {

// A [B, H, S, d] view with element strides; d is contiguous.
struct View {
  const void* p;
  int64_t sb, sh, ss;
};

enum { KV_FRESH = 0, KV_CACHE = 1, KV_DEVICE = 2, KV_SEGMENTS = 3 };
constexpr int kMaxSeg = 16;
enum { DEC_REUSE = 0, DEC_REACTIVATE = 1, DEC_COMPUTE = 2 };

// Work decomposition of one bf16 attention launch over its query tiles (all
// tiles of a (batch, head) attend to every key tile, so they cost the same).
// Launch indices [0, whole) run whole query tiles; `split_tiles` query tiles
// (the last ones of each (batch, head), plan_split_tile; in the segment kernel
// the last ones in head-major order) are cut into `chunks` contiguous key-tile
// ranges each, launched at [whole, total_items), whose partial results a merge
// kernel combines.
struct SplitPlan {
  int32_t whole;        // query tiles run whole (a multiple of the resident workgroup slots)
  int32_t split_tiles;  // query tiles run in key chunks
  int32_t chunks;       // key chunks per split tile (1 when split_tiles == 0)
  int32_t total_items;  // whole + split_tiles * chunks (workgroups that do work)
};

struct AttnParams {
  View q_tgt, k_tgt, v_tgt;
  View q_ref, k_fresh, v_fresh, k_cache, v_cache;
  View q_cache;             // reference queries of the cached state; null p: q_ref serves
  View o_tgt, o_ref;        // written through const_cast
  float* mass_tgt;          // [B, H, n_tgt] or null
  float* lse_tgt;           // [B, H, n_tgt, 2] or null
  float* mass_refq;         // [B, H, n_ref] or null
  const int32_t* decision;  // KV_DEVICE only
  unsigned long long* clock_probe;  // [2] shader cycles, 100 MHz ticks (added to), or null
  int32_t B, H, n_ref, n_tgt;
  int32_t qt_ref;       // query tiles per (b, h) over reference rows (0 when they do not attend)
  int32_t qt_tgt;       // query tiles per (b, h) over target rows
  int32_t total_tiles;  // B * H * (qt_ref + qt_tgt) = grid size
  int32_t kvsrc;
  float sc_log2;  // softmax scale * log2(e)
  // bf16 path: plan[0] covers the launch's query set (under KV_DEVICE: every
  // query tile), plan[1] the target query tiles alone (KV_DEVICE on REUSE).
  SplitPlan plan[2];
  float* part_o;     // [items][BM][head_dim] unnormalised fp32 partial outputs of split items
  float4* part_st;   // [items][BM] (m, l_tgt, m_ref, l_ref) per partial row
  float* part_lo;    // [items][BM] sum of the bf16-rounded probabilities of a partial row
  float* part_seg;   // [items][BM][n_seg] per-segment log-sum-exp of partial rows (seg_mass), or null
  // Reference segments (bf16; seg_mass splits key ranges only with part_seg): n_seg > 0 selects the segment
  // kernel. Segment s covers reference key tiles [seg_tile_end[s-1], seg_tile_end[s]);
  // seg_cache bit s reads the cached K/V for it; seg_mass [B, H, n_tgt, n_seg] or null.
  int32_t n_seg;
  int32_t seg_tile_end[kMaxSeg];
  uint32_t seg_cache;
  float* seg_mass;
  // Per segment, the base of the K and V view it reads (fresh or cached; both views share
  // their strides, which are those of k_fresh / v_fresh).
  const void* seg_kbase[kMaxSeg];
  const void* seg_vbase[kMaxSeg];
};

// Query rows per workgroup of each attention kernel (the host sizes the grid with
// these) and keys per key tile of the bf16 kernel.
constexpr int kAttnBf16BM = 256;
constexpr int kAttnBf16BN = 64;
// Largest K/V row stride (elements) of the bf16 attention: a key tile spans 64 rows, addressed
// with 32-bit byte offsets.
constexpr int64_t kAttnMaxRowStride = (int64_t(1) << 24) - 8;
constexpr int kAttnF32BM = 64;

// Compute units of the current device and bf16 attention workgroups each holds
// at once; zeros if the device cannot be queried.
struct AttnSlots {
  int cus, per_cu;
};
AttnSlots attn_bf16_slots(int head_dim);
// Enqueues the bf16 attention kernel and, when a plan splits tiles, the merge.
hipError_t launch_attn_bf16(const AttnParams& p, int head_dim, hipStream_t stream);
hipError_t launch_attn_f32(const AttnParams& p, int head_dim, hipStream_t stream);

int q_change_chunks(int32_t n_tgt, int32_t head_dim);
hipError_t launch_q_change(int dtype, int32_t B, int32_t H, int32_t n_tgt, int32_t head_dim, View cur, View prev,
                           float eps, float* d_out, void* ws, hipStream_t stream);

struct GateState {
  int32_t reactivated, a_full, delta_max, step;
};
hipError_t launch_gate(int32_t B, int32_t H, int32_t n_tgt, int32_t block, int32_t step, int32_t mode,
                       const float* d_cur, const float* mass_prev, const float* theta, GateState* state,
                       int32_t* decision_out, float* score_out, hipStream_t stream);

size_t q_change_gate_workspace_bytes(int32_t B, int32_t H, int32_t n_tgt, int32_t head_dim);
hipError_t launch_q_change_gate(int dtype, int32_t B, int32_t H, int32_t n_tgt, int32_t head_dim, View cur, View prev,
                                float eps, int32_t block, int32_t step, int32_t mode, const float* mass_prev,
                                const float* theta, GateState* state, float* d_out, int32_t* decision_out,
                                float* score_out, void* ws, hipStream_t stream);

// Up to three (source, destination) pairs copied by one commit launch.
struct CommitSet {
  View src[3], dst[3];
  int32_t n;
};
hipError_t launch_cache_commit(int dtype, int32_t B, int32_t H, int32_t n_ref, int32_t head_dim, CommitSet cs,
                               const int32_t* decision, int32_t* age, int32_t step, hipStream_t stream);

// Up to two [B, H, n, d] slice pairs whose relative change the diagnostics
// reduce in one launch; chunks[] is filled by the launcher.
struct PairSet {
  View cur[2], base[2];
  int32_t n_rows[2];
  int32_t chunks[2];
};
enum { PAIR_SINGLE = 0, PAIR_KV = 1, PAIR_RATIO = 2 };
size_t pair_workspace_bytes(int32_t B, int32_t H, int32_t head_dim, int npairs, const int32_t* n_rows);
hipError_t launch_pair_change(int dtype, int32_t B, int32_t H, int32_t head_dim, int npairs, PairSet ps, int kind,
                              float eps, float* out0, float* out1, float* out2, void* ws, hipStream_t stream);
hipError_t launch_mass_mean(int32_t B, int32_t H, int32_t n, const float* mass, int complement, float* out,
                            hipStream_t stream);
hipError_t launch_adjacent_change(int32_t T, int32_t nb, int32_t bh, const float* m, float* out, hipStream_t stream);
// Matrix-core rate probe (measurement only): kind 0 back-to-back MFMAs, kind 1 the
// attention's per-tile register mix; operands >= kProbeOperandBytes of bf16 data.
constexpr size_t kProbeOperandBytes = 65536;
hipError_t launch_mfma_rate(int kind, int32_t workgroups, int32_t steps, const void* operands, float* sink,
                            unsigned long long* clock_probe, hipStream_t stream);

// Launches `kernel` and returns the status of THIS launch (hipLaunchKernel's
// return value), not a sticky error left by earlier runtime calls. Arguments
// are converted to the kernel's parameter types before their addresses are
// taken.
template <typename... KArgs, typename... Args>
hipError_t launch_kernel(void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t shmem, hipStream_t stream,
                         Args... args) {
  static_assert(sizeof...(KArgs) == sizeof...(Args), "kernel arity mismatch");
  std::tuple<KArgs...> held(static_cast<KArgs>(args)...);
  void* ptrs[sizeof...(KArgs) > 0 ? sizeof...(KArgs) : 1];
  std::apply(
      [&](auto&... e) {
        size_t i = 0;
        ((ptrs[i++] = static_cast<void*>(&e)), ...);
      },
      held);
  return hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, ptrs, shmem, stream);
}

// Maps a launch index to a tile index so that the workgroups the hardware
// sends to one XCD (round-robin over the 8 XCDs by launch index) get one
// contiguous range of tiles; consecutive tiles share (batch, head), so their
// K/V tiles are re-read from that XCD's L2. A bijection on [0, total).
__host__ __device__ __forceinline__ int xcd_remap(int w, int total) {
  const int per = total >> 3, rem = total & 7;
  const int xcd = w & 7, k = w >> 3;
  return xcd * per + (xcd < rem ? xcd : rem) + k;
}

// Query tiles in the order a split plan enumerates them. The plan's split tiles
// are spread evenly over the n_bh (batch, head) pairs, the last ones of each
// (pair h gets q + (h < r) of them, q = split / n_bh, r = split % n_bh); whole
// tiles are numbered pair by pair over the rest, and split tiles pair by pair too.
// Every pair keeps the same number of whole tiles (to within one), so with
// xcd_remap on top an XCD's rounds of whole tiles start at pair boundaries when
// that number is a multiple of the XCD's resident workgroups, and each round then
// streams the K/V of a single pair through the XCD's L2. Returns
// bh * tiles_bh + (tile within the pair); a bijection of [0, whole) and of
// [0, split) onto the whole and the split tiles.
__host__ __device__ __forceinline__ int plan_whole_tile(int i, int tiles_bh, int n_bh, int split) {
  const int q = split / n_bh, r = split - q * n_bh;
  const int few = tiles_bh - q - 1;  // whole tiles of heads h < r
  const int a = r * few;
  int h, t;
  if (i < a) {
    h = i / few;
    t = i - h * few;
  } else {
    const int j = i - a, many = tiles_bh - q;
    h = r + j / many;
    t = j - (h - r) * many;
  }
  return h * tiles_bh + t;
}

__host__ __device__ __forceinline__ int plan_split_tile(int st, int tiles_bh, int n_bh, int split) {
  const int q = split / n_bh, r = split - q * n_bh;
  const int b = r * (q + 1);
  int h, k;
  if (st < b) {
    h = st / (q + 1);
    k = st - h * (q + 1);
  } else {
    const int j = st - b;
    h = r + j / q;
    k = j - (h - r) * q;
  }
  const int s_h = q + (h < r ? 1 : 0);
  return h * tiles_bh + (tiles_bh - s_h) + k;
}

}  // namespace refadapt
