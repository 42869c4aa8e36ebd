// Joint attention over [reference; target] keys on bf16 MFMA (gfx950).
//
// One workgroup = 8 wavefronts = 256 query rows of one (batch, head); each
// wavefront owns 32 query rows. Key/value tiles of 64 rows stream through LDS,
// reference tiles first (from the fresh or the cached reference K/V, chosen
// once per workgroup) and then target tiles.
//
// Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16
// (keys on the M side, the wavefront's 32 queries on the N side), so every lane
// holds 32 scores of ONE query: row max and row sum are in-lane reductions plus
// one v_permlane32_swap. The probabilities P^T stay in registers and feed
// O^T += V^T P^T directly as the B operand; the V^T A operand is read from the
// row-major V tile with ds_read_b64_tr_b16 (LDS transpose read).
//
// Software pipeline (per wavefront): iteration j issues the 16 MFMAs of S_{j+1}
// with the probabilities of S_j pairs 0..9 formed under them (phase A), then
// the 16 MFMAs of O += V_j^T P_j^T, under the first eight of which the remaining
// pairs 10..15 are formed (phase B). A pair takes three MFMA slots (exponent
// arguments, exponentials, row-sum adds and bf16 pack), so the instructions of
// one slot never wait on each other. sched_barrier fences keep that order, so
// the vector ALU works while the matrix core runs. K tiles run one
// tile ahead of V tiles through two LDS buffers each. At the start of phase B of
// iteration j direct global-to-LDS loads (no staging registers, no LDS store
// instructions) fill the buffers that held K_j and V_{j-1} with K_{j+2} and
// V_{j+1}; the iteration's one barrier, after a wait for those loads, publishes
// them.
//
// One workgroup fills a CU with two wavefronts per SIMD (at most 256 vector
// registers per lane each): while one wavefront forms probabilities the other
// keeps the matrix core busy, and the eight wavefronts share every K/V tile
// in LDS (each wavefront loads two 1 KiB blocks of each tile). s_setprio
// alternates which wavefront of a SIMD wins issue ties between the phases, so
// the pair finishes a tile together instead of one idling at the barrier.
//
// Online softmax in the exp2 domain without a per-tile row max: probabilities
// are formed against the running max m, and a lane's partial row sum bounds
// each of its terms, so a sum within 2^12 proves that every probability is at
// most 2^12 and m may stay. The test runs (wave-wide, NaN and inf failing it)
// once for pairs 0..9 before any of them enters O and once for pairs 8..15
// (P blocks 2 and 3) before the first MFMA that reads them; when it fails (always at a
// workgroup's first tile, where m = -inf), a cold path takes the row max of
// the scores still to be formed, rescales O and l, and forms them again. The
// O rescale and the row max are thus almost never executed.
// Row sums add the fp32 probabilities, so the reference mass and the
// log-sum-exp carry no bf16 rounding. O is divided by a second sum, that of
// the bf16-rounded probabilities it accumulated (one v_dot2c_f32_bf16 per
// packed pair, after the tile's last MFMA), so the weights
// applied to V sum to one: with the fp32 sum, the rounding of a dominant
// probability (relative error up to 2^-8) moved the output by as much of V.
//
// Split statistics for the reference mass (paper Sec. 3.2, directional
// exposure): after the last reference tile the running (max, sum) pair is
// frozen as (m_R, l_R) and the sum restarts at zero, so at the end
// L_R = l_R * 2^(m_R - m) and L_Y = l are the reference and target parts of
// the softmax denominator in one scale; mass = L_R / (L_R + L_Y) lies in
// [0, 1] by construction and equals exp(lse_R - lse_all).
//
// Load balance: all query tiles cost the same, so the launch runs in rounds of
// as many workgroups as the device holds at once. When the last round would be
// only partly full, the host plan cuts its query tiles into key-tile chunks
// (more, shorter workgroups). A chunk keeps the same split statistics over its
// key range and writes its unnormalised output with (m, l_Y, m_R, l_R) to a
// workspace; attn_merge_kernel rescales the chunks to their common maximum and
// sums them, which is the same reduction the online softmax performs across
// key tiles. The split tiles are the last tiles of each (batch, head), spread
// evenly over the heads (plan_whole_tile, plan_split_tile), so an XCD's rounds
// of whole tiles stream few heads' K/V. With per-segment masses a chunk also
// records one log-sum-exp per reference segment it covers, which the merge
// combines per segment.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <type_traits>

#include "internal.h"

namespace refadapt {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr int BM = kAttnBf16BM;  // query rows per workgroup
constexpr int BN = kAttnBf16BN;  // keys per LDS tile
constexpr int NT = 512;          // threads per workgroup
constexpr float PBOUND = 4096.0f;  // bound on a probability against the running max (2^12)

// Row permutation of a 32-key MFMA block: swaps bits 2 and 3 of the row index.
// With key sigma(m) in A-row m of S^T = K Q^T, output register r of lane-half g
// holds key 16*(r/8) + 8*g + r%8: eight consecutive keys per lane-half, which is
// exactly the K-operand order of the B operand (P^T) of the PV product.
__device__ __forceinline__ int sigma(int m) { return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1); }

// max / sum of a value with its partner lane l ^ 32.
__device__ __forceinline__ float xor32_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor32_add(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Keeps a value in a register at this point of the program, so the optimizer
// cannot sink the instructions that produce it into a later block.
template <typename T>
__device__ __forceinline__ void pin(T& v) {
  asm volatile("" : "+v"(v));
}

// acc + lo + hi of a packed pair of bf16 values (one v_dot2c_f32_bf16 against (1, 1)).
__device__ __forceinline__ float add_bf16x2(uint32_t w, float acc) {
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), one, acc, false);
}

// LDS tiles are filled by direct global-to-LDS loads (buffer_load_dwordx4 ... lds):
// one wavefront instruction writes 64 lanes x 16 bytes = one contiguous 1 KiB block,
// lane L at byte 16 L. Each tile is D / 8 such blocks, and the lanes' global
// addresses decide what lands where (bf16 elements; b(x, k) = bit k of x):
//   K block kb = KS * mb + kk: 32 LDS rows n of 32 bytes, holding key 32 mb + sigma(n)
//     and head dims 16 kk .. 16 kk + 15; chunk g (dims 16 kk + 8 g .. + 7) sits at
//     byte 32 n + 16 (g ^ b(n, 3)). A-row n of an S^T block is LDS row n, and the 16
//     lanes of one read phase hit 16 distinct 16-byte bank groups.
//   V block vb = DB * s2 + db: 16 rows r of 64 bytes, holding key 16 s2 + r and head
//     dims 32 db .. 32 db + 31, with the dim offset XORed by 16 when b(r, 1) is set,
//     which makes the transpose reads of the V^T operand conflict-free.
// No padding, no staging registers and no LDS store instructions: a tile's loads are
// issued about a phase B ahead of the barrier that publishes it.
template <int D>
struct Layout {
  static constexpr int NB = D / 8;        // 1 KiB blocks per K or V tile
  static constexpr int TILE = NB * 512;   // elements per tile
  static constexpr int NLD = NB / 8;      // blocks each of the 8 wavefronts loads per tile
};

// Buffer resource of one K or V tile: base = its first row, range = its valid rows, so
// rows past a ragged tile's end load as zero (the range check covers the scalar offset
// too). The base and range are workgroup-uniform; readfirstlane states it, so the
// resource lives in scalar registers.
template <int D>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const uint16_t* base, int64_t ss, int valid) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  const uint32_t nbytes = __builtin_amdgcn_readfirstlane((uint32_t)((int64_t)(valid - 1) * ss * 2 + D * 2));
  void* ub = reinterpret_cast<void*>(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(ub, (short)0, (int)nbytes, 0x00020000);
}

// Per-lane byte offset of the direct loads (row part with row stride ss elements, plus
// the lane's 16-byte chunk); each block adds a uniform row and column offset.
template <bool IS_K>
__device__ __forceinline__ uint32_t dma_lane_offset(int lane, int64_t ss) {
  if (IS_K) return (uint32_t)(sigma(lane >> 1) * ss * 2 + 16 * ((lane & 1) ^ ((lane >> 4) & 1)));
  return (uint32_t)((lane >> 2) * ss * 2 + 16 * ((lane & 3) ^ (((lane >> 3) & 1) << 1)));
}

// This wavefront's blocks of one K or V tile, straight into the LDS tile.
template <int D, bool IS_K>
__device__ __forceinline__ void tile_dma(uint16_t* tile, __amdgpu_buffer_rsrc_t rs, uint32_t voff, int64_t ss,
                                         int wave) {
  constexpr int KS = D / 16, DB = D / 32;
#pragma unroll
  for (int i = 0; i < Layout<D>::NLD; ++i) {
    const int blk = wave + 8 * i;
    const int64_t soff = IS_K ? (int64_t)(blk / KS) * 32 * ss * 2 + (blk % KS) * 32
                              : (int64_t)(blk / DB) * 16 * ss * 2 + (blk % DB) * 64;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(tile + blk * 512), 16,
                                             voff, __builtin_amdgcn_readfirstlane((uint32_t)soff), 0, 0);
  }
}

// Direct-load cursor of one K or V stream: the next key tile to load, the first row of that
// tile, the rows of its view from there on, and the view's row stride, lane offset and the
// scalar offsets of this wavefront's blocks. Advancing to the next tile costs a 64-bit add;
// the view changes once, where the reference keys end and the target keys begin.
template <int D, bool IS_K>
struct DmaCursor {
  const uint16_t* ptr;
  int64_t ss;
  uint32_t voff;
  uint32_t soff[Layout<D>::NLD];
  int t, rows;

  __device__ __forceinline__ void set_view(const uint16_t* base, int64_t row_stride, uint32_t lane_off, int tile0,
                                           int first_row, int view_rows, int wave) {
    constexpr int KS = D / 16, DB = D / 32;
    ss = row_stride;
    voff = lane_off;
    ptr = base + (int64_t)first_row * ss;
    rows = view_rows - first_row;
    t = tile0;
#pragma unroll
    for (int i = 0; i < Layout<D>::NLD; ++i) {
      const int blk = wave + 8 * i;
      soff[i] = __builtin_amdgcn_readfirstlane(
          (uint32_t)(IS_K ? (int64_t)(blk / KS) * 32 * ss * 2 + (blk % KS) * 32
                          : (int64_t)(blk / DB) * 16 * ss * 2 + (blk % DB) * 64));
    }
  }
  // loads tile t into `tile` and advances to tile t + 1
  __device__ __forceinline__ void load(uint16_t* tile, int wave) {
    const int valid = min(BN, rows);
    const __amdgpu_buffer_rsrc_t rs = tile_rsrc<D>(ptr, ss, valid);
#pragma unroll
    for (int i = 0; i < Layout<D>::NLD; ++i) {
      const int blk = wave + 8 * i;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(tile + blk * 512), 16,
                                               voff, soff[i], 0, 0);
    }
    ptr += BN * ss;
    rows -= BN;
    t += 1;
  }
};

// SEG: reference segments: each reference key tile reads the fresh or the cached K/V of its
// segment. SEGM (with SEG, for a non-null seg_mass): each segment's log-sum-exp over the
// launch's key range is recorded; an instance of its own, so that launches without it carry
// none of its state (2% of the segment launch).
template <int D, bool SEG, bool SEGM>
__global__ __launch_bounds__(NT, 1) void attn_bf16_kernel(AttnParams p) {
  constexpr int KS = D / 16;   // MFMA k-steps over the head dim for S^T
  constexpr int DB = D / 32;   // 32-row blocks of the O^T accumulator
  constexpr int NQK = 2 * KS;  // MFMAs of one S^T tile
  constexpr int NPV = 4 * DB;  // MFMAs of one PV tile
  // Four separate arrays (not one indexed by a run-time buffer number), so the compiler
  // can tell the buffer a direct load fills from the ones being read and does not wait
  // for the load before those reads.
  __shared__ __attribute__((aligned(1024))) uint16_t kbuf0[Layout<D>::TILE];
  __shared__ __attribute__((aligned(1024))) uint16_t kbuf1[Layout<D>::TILE];
  __shared__ __attribute__((aligned(1024))) uint16_t vbuf0[Layout<D>::TILE];
  __shared__ __attribute__((aligned(1024))) uint16_t vbuf1[Layout<D>::TILE];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, n = lane & 31;

  // ---- which (batch, head, query tile) and which key tiles this workgroup owns
  bool use_cache = p.kvsrc == KV_CACHE;
  bool tgt_only = false;  // a reused block (KV_DEVICE): reference query rows are skipped
  if (p.kvsrc == KV_DEVICE) {
    const int dec = __builtin_amdgcn_readfirstlane(*p.decision);
    use_cache = dec != DEC_COMPUTE;
    tgt_only = dec == DEC_REUSE;
  }
  const SplitPlan pl = p.plan[tgt_only ? 1 : 0];
  const int qt_ref = tgt_only ? 0 : p.qt_ref;
  const int n_rt = (p.n_ref + BN - 1) / BN;
  const int n_yt = (p.n_tgt + BN - 1) / BN;
  const int nt = n_rt + n_yt;
  const int w = blockIdx.x;
  if (w >= pl.total_items) return;
  // Optional clock probe: shader-clock cycles and 100 MHz reference ticks over this
  // workgroup's life, added to the caller's counters by its first lane at exit.
  const bool probe = p.clock_probe != nullptr;
  uint64_t clk0 = 0, rt0 = 0;
  if (probe) {
    clk0 = __builtin_amdgcn_s_memtime();
    rt0 = __builtin_amdgcn_s_memrealtime();
  }
  auto probe_end = [&]() {
    if (probe && tid == 0) {
      const uint64_t clk1 = __builtin_amdgcn_s_memtime(), rt1 = __builtin_amdgcn_s_memrealtime();
      atomicAdd(p.clock_probe, (unsigned long long)(clk1 - clk0));
      atomicAdd(p.clock_probe + 1, (unsigned long long)(rt1 - rt0));
    }
  };
  const int qt_bh = qt_ref + p.qt_tgt;
  int tile, j0 = 0, j1 = nt, slot = -1;
  // The segment kernel keeps the plain head-major order (split tiles last): with per-segment
  // sources it ran 1% slower with the split tiles spread over the heads.
  if (w < pl.whole) {
    tile = xcd_remap(w, pl.whole);
    if constexpr (!SEG) tile = plan_whole_tile(tile, qt_bh, p.B * p.H, pl.split_tiles);
  } else {  // key chunk c of a split tile: key tiles [c * nt / chunks, (c + 1) * nt / chunks)
    // The chunks of neighbouring split tiles go to one XCD, as whole tiles do.
    slot = xcd_remap(w - pl.whole, pl.total_items - pl.whole);
    const int st = slot / pl.chunks, c = slot - st * pl.chunks;
    tile = SEG ? pl.whole + st : plan_split_tile(st, qt_bh, p.B * p.H, pl.split_tiles);
    j0 = c * nt / pl.chunks;
    j1 = (c + 1) * nt / pl.chunks;
  }
  const int bh = tile / qt_bh;
  int qt = tile - bh * qt_bh;
  const int b = bh / p.H, h = bh - b * p.H;
  const bool ref_rows = qt < qt_ref;
  if (!ref_rows) qt -= qt_ref;

  // Reference queries over the cached K/V read the cached queries when the caller gave them.
  const View qv = ref_rows ? (use_cache && p.q_cache.p ? p.q_cache : p.q_ref) : p.q_tgt;
  const View ov = ref_rows ? p.o_ref : p.o_tgt;
  const int n_rows = ref_rows ? p.n_ref : p.n_tgt;
  const View krv = use_cache ? p.k_cache : p.k_fresh;
  const View vrv = use_cache ? p.v_cache : p.v_fresh;
  const uint16_t* kr = static_cast<const uint16_t*>(krv.p) + b * krv.sb + h * krv.sh;
  const uint16_t* vr = static_cast<const uint16_t*>(vrv.p) + b * vrv.sb + h * vrv.sh;
  const uint16_t* ky = static_cast<const uint16_t*>(p.k_tgt.p) + b * p.k_tgt.sb + h * p.k_tgt.sh;
  const uint16_t* vy = static_cast<const uint16_t*>(p.v_tgt.p) + b * p.v_tgt.sb + h * p.v_tgt.sh;
  int64_t kr_ss = krv.ss, vr_ss = vrv.ss, ky_ss = p.k_tgt.ss, vy_ss = p.v_tgt.ss;

  auto tile_valid = [&](int j) { return j < n_rt ? min(BN, p.n_ref - j * BN) : min(BN, p.n_tgt - (j - n_rt) * BN); };
  const int rag_ref = p.n_ref % BN ? n_rt - 1 : -1;  // key tiles with fewer than BN keys
  const int rag_tgt = p.n_tgt % BN ? nt - 1 : -1;
  // Per-lane byte offsets of the direct loads, per source view (the segments of SEG share
  // the reference views' strides).
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t voff_r = dma_lane_offset<true>(lane, krv.ss);
  const uint32_t voff_rv = dma_lane_offset<false>(lane, vrv.ss);
  const uint32_t voff_yk = dma_lane_offset<true>(lane, p.k_tgt.ss);
  const uint32_t voff_yv = dma_lane_offset<false>(lane, p.v_tgt.ss);
  // SEG: each of the K and V streams visits reference tiles in increasing order, so it keeps
  // its current segment, that segment's base pointer (this (b, h) applied) and end tile, and
  // reads the next ones from the kernel arguments only when it crosses a segment end.
  int kseg = 0, kend = 0, vseg = 0, vend = 0;
  const uint16_t *kbase = nullptr, *vbase = nullptr;
  const int64_t kbh = b * krv.sb + h * krv.sh, vbh = b * vrv.sb + h * vrv.sh;
  if constexpr (SEG) {
    kend = vend = p.seg_tile_end[0];
    kbase = static_cast<const uint16_t*>(p.seg_kbase[0]) + kbh;
    vbase = static_cast<const uint16_t*>(p.seg_vbase[0]) + vbh;
  }
  // Loads reference tile j of one of K, V (strides ss, lane offset voff) from the base of
  // its segment into an LDS tile.
  auto load_ref_seg = [&](auto is_k, uint16_t* dst, int j, int& seg, int& end, const uint16_t*& base,
                          const void* const* seg_base, int64_t bh_off, int64_t ss, uint32_t voff) {
    while (j >= end && seg + 1 < p.n_seg) {
      end = p.seg_tile_end[++seg];
      base = static_cast<const uint16_t*>(seg_base[seg]) + bh_off;
    }
    tile_dma<D, decltype(is_k)::value>(dst, tile_rsrc<D>(base + (int64_t)j * BN * ss, ss, tile_valid(j)), voff, ss,
                                       wave_u);
  };
  auto load_k = [&](uint16_t* dst, int j) {
    const int valid = tile_valid(j);
    if constexpr (SEG) {
      if (j < n_rt) {
        load_ref_seg(std::true_type{}, dst, j, kseg, kend, kbase, p.seg_kbase, kbh, krv.ss, voff_r);
        return;
      }
    }
    if (j < n_rt)
      tile_dma<D, true>(dst, tile_rsrc<D>(kr + (int64_t)j * BN * kr_ss, kr_ss, valid), voff_r, kr_ss, wave_u);
    else
      tile_dma<D, true>(dst, tile_rsrc<D>(ky + (int64_t)(j - n_rt) * BN * ky_ss, ky_ss, valid), voff_yk, ky_ss,
                        wave_u);
  };
  auto load_v = [&](uint16_t* dst, int j) {
    const int valid = tile_valid(j);
    if constexpr (SEG) {
      if (j < n_rt) {
        load_ref_seg(std::false_type{}, dst, j, vseg, vend, vbase, p.seg_vbase, vbh, vrv.ss, voff_rv);
        return;
      }
    }
    if (j < n_rt)
      tile_dma<D, false>(dst, tile_rsrc<D>(vr + (int64_t)j * BN * vr_ss, vr_ss, valid), voff_rv, vr_ss, wave_u);
    else
      tile_dma<D, false>(dst, tile_rsrc<D>(vy + (int64_t)(j - n_rt) * BN * vy_ss, vy_ss, valid), voff_yv, vy_ss,
                         wave_u);
  };

  // ---- this lane's query row; Q^T as the B operand (query n, head-dim chunk 2*kk + g)
  const int qrow = qt * BM + wave * 32 + n;
  const bool qvalid = qrow < n_rows;
  bf16x8 qreg[KS];
  {
    const uint16_t* qp = static_cast<const uint16_t*>(qv.p) + b * qv.sb + h * qv.sh + (int64_t)qrow * qv.ss;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const u32x4 raw = qvalid ? *reinterpret_cast<const u32x4*>(qp + kk * 16 + g * 8) : u32x4{0, 0, 0, 0};
      qreg[kk] = __builtin_bit_cast(bf16x8, raw);
    }
  }

  // lane-dependent parts of the LDS operand addresses (everything else is an immediate)
  const int k_lane = 16 * n + 8 * (g ^ ((n >> 3) & 1));  // A-row n, head-dim chunk g
  const int tr_i = lane & 15, tr_G = lane >> 4;         // 16-lane group of the transpose read
  const int v_lane = 32 * (8 * (tr_G >> 1) + (tr_i >> 2)) + ((16 * (tr_G & 1) + 4 * (tr_i & 3)) ^ (16 * ((tr_i >> 3) & 1)));

  // ---- prologue: K_{j0}, K_{j0+1} and V_{j0} into LDS; S_{j0}. Tile j lives in
  // buffer (j - j0) & 1.
  load_k(kbuf0, j0);
  load_v(vbuf0, j0);
  if (j0 + 1 < j1) load_k(kbuf1, j0 + 1);
  __syncthreads();
  f32x16 sa[2], sb[2];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
    sa[mb] = f32x16{};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(kbuf0 + k_lane + 512 * (KS * mb + kk));
      sa[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[kk], sa[mb], 0, 0, 0);
    }
  }
  __syncthreads();  // every wavefront has read K_{j0} before the first iteration refills its buffer
  // cursors of the in-loop loads: K from tile j0 + 2, V from tile j0 + 1
  DmaCursor<D, true> kc;
  DmaCursor<D, false> vc;
  // SEG: the segment each cursor reads and the key tile that ends it. A cursor re-targets to
  // the next segment's base (this (b, h) applied) when it reaches that tile; segments share
  // the reference views' strides, so only the base pointer changes. The segment tables are
  // read through pointers into the kernel arguments (indexing the by-value copy at run time
  // would place it in scratch memory).
  int kc_seg = 0, kc_end = 0, vc_seg = 0, vc_end = 0;
  const int32_t* const seg_end_tab = p.seg_tile_end;
  const void* const* const seg_k_tab = p.seg_kbase;
  const void* const* const seg_v_tab = p.seg_vbase;
  auto cursor_view = [&](auto is_kc, auto& cur, int tile) __attribute__((always_inline)) {
    constexpr bool IS_K = decltype(is_kc)::value;
    if (tile < n_rt) {
      const uint16_t* base = IS_K ? kr : vr;
      if constexpr (SEG) {
        int sg = 0;
        while (tile >= seg_end_tab[sg] && sg + 1 < p.n_seg) ++sg;
        base = static_cast<const uint16_t*>((IS_K ? seg_k_tab : seg_v_tab)[sg]) + (IS_K ? kbh : vbh);
        (IS_K ? kc_seg : vc_seg) = sg;
        (IS_K ? kc_end : vc_end) = seg_end_tab[sg];
      }
      cur.set_view(base, IS_K ? kr_ss : vr_ss, IS_K ? voff_r : voff_rv, tile, tile * BN, p.n_ref, wave_u);
    } else {
      cur.set_view(IS_K ? ky : vy, IS_K ? ky_ss : vy_ss, IS_K ? voff_yk : voff_yv, tile, (tile - n_rt) * BN, p.n_tgt,
                   wave_u);
    }
  };
  // SEG: moves a cursor that reached its segment's last tile to the next segment (same rows,
  // same strides: the row pointer moves by the difference of the two segments' bases).
  auto cursor_next_seg = [&](auto is_kc, auto& cur) __attribute__((always_inline)) {
    constexpr bool IS_K = decltype(is_kc)::value;
    int& sg = IS_K ? kc_seg : vc_seg;
    const void* const* tab = IS_K ? seg_k_tab : seg_v_tab;
    const char* from = static_cast<const char*>(tab[sg]);
    ++sg;
    (IS_K ? kc_end : vc_end) = seg_end_tab[sg];
    cur.ptr = reinterpret_cast<const uint16_t*>(reinterpret_cast<const char*>(cur.ptr) +
                                                (static_cast<const char*>(tab[sg]) - from));
  };
  cursor_view(std::true_type{}, kc, j0 + 2);
  cursor_view(std::false_type{}, vc, j0 + 1);

  f32x16 o[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) o[i] = f32x16{};
  // l_run and l_ref hold this lane's half of the query's keys (its partner lane l ^ 32 the
  // other half; both see the same max): the halves are added where a whole sum is read.
  float m_run = -__builtin_inff(), l_run = 0.f;
  // Sum of the bf16-rounded probabilities that enter O (this lane's keys, against m_run): the
  // output is normalised by it, so the weights applied to V sum to one (l_run, the fp32 sum,
  // gives the mass and the log-sum-exp).
  float lo_run = 0.f;
  float m_ref = -__builtin_inff(), l_ref = 0.f;
  const float c = p.sc_log2;
  // SEG with seg_mass: the reference segment that holds this range's first key tile (a key
  // chunk may start inside one), the key tile that ends it, this row's seg_mass offset and,
  // for a key chunk, its row of per-segment partials.
  int seg_idx = 0;
  if constexpr (SEG)
    while (seg_idx < p.n_seg && j0 >= seg_end_tab[seg_idx]) ++seg_idx;
  const int seg_first = seg_idx;
  int seg_end_t = SEG && seg_idx < p.n_seg ? seg_end_tab[seg_idx] : -1;
  const int64_t seg_row = ((int64_t)bh * p.n_tgt + qrow) * p.n_seg;
  const int64_t seg_prow = ((int64_t)slot * BM + wave * 32 + n) * p.n_seg;
  // Closes the current segment: records its log-sum-exp (log2 domain) over this key range,
  // which the epilogue or the merge turns into a mass, then folds its sum into the reference
  // statistics, each kept against its own max, and restarts the running sum.
  auto close_segment = [&]() {
    const float l_seg = xor32_add(l_run);  // whole wavefront: the swap reads the partner lane
    if (!ref_rows && qvalid && g == 0) {
      const float lse_s = m_run + __log2f(l_seg);
      if (slot >= 0)
        p.part_seg[seg_prow + seg_idx] = lse_s;
      else
        p.seg_mass[seg_row + seg_idx] = lse_s;
    }
    l_ref = seg_idx == seg_first ? l_run : l_ref * __builtin_amdgcn_exp2f(m_ref - m_run) + l_run;
    m_ref = m_run;
    l_run = 0.f;
    ++seg_idx;
    seg_end_t = seg_idx < p.n_seg ? seg_end_tab[seg_idx] : -1;
  };

  // jbc: the LDS buffer of K_j and V_j, (j - j0) & 1, as a compile-time constant.
  auto iteration = [&](auto jbc, int j, f32x16(&s_cur)[2], f32x16(&s_next)[2]) {
    constexpr int jb = decltype(jbc)::value;
    // Global loads for the tiles this iteration stages: K_{j+2} and V_{j+1}, issued at the
    // start of phase B through the K and V cursors; past the workgroup's last key tile the
    // cursors skip the load.
    uint16_t* const kb_cur = jb ? kbuf1 : kbuf0;   // K_j (already read), refilled with K_{j+2}
    uint16_t* const kb_next = jb ? kbuf0 : kbuf1;  // K_{j+1}
    uint16_t* const vb_cur = jb ? vbuf1 : vbuf0;   // V_j
    uint16_t* const vb_next = jb ? vbuf0 : vbuf1;  // V_{j-1} (already read), refilled with V_{j+1}

    // The ragged last tile of each of the reference and target segments (if any) is known
    // up front: the test in the loop compares tile indices only.
    if (j == rag_ref || j == rag_tgt) {  // ragged last tile of a segment: drop keys past its end
      const int valid = tile_valid(j);
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = 32 * mb + 16 * (r >> 3) + 8 * g + (r & 7);
          if (key >= valid) s_cur[mb][r] = -__builtin_inff();
        }
    }

    // Issue priority: the first wavefront on a SIMD (waves 0-3) otherwise wins every tie,
    // finishes its tile early and waits at the barrier while its partner runs alone. The
    // partner gets the higher priority in phase A and the first one in phase B.
    const bool partner = __builtin_amdgcn_readfirstlane(wave) >= 4;
    if (partner) __builtin_amdgcn_s_setprio(1); else __builtin_amdgcn_s_setprio(0);
    // ---- phase A: the MFMAs of S_{j+1} (K_{j+1} is in LDS), with the probability pairs 0..9
    // of S_j (P blocks 0, 1 and half of block 2) formed under them, three slots per pair.
    // At the last iteration the K buffer holds no tile and S_{j+1} is discarded.
    const uint16_t* kb = kb_next;
    auto k_operand = [&](int i) {  // i = KS * mb + kk
      return *reinterpret_cast<const bf16x8*>(kb + k_lane + 512 * i);
    };
    uint32_t pw[4][4];  // packed bf16 probabilities: P block s2, keys 16*s2 + 8*g + 2w, +1
    // Row-sum chains: pairs 0..7 (P blocks 0, 1) and pairs 8..15 (P blocks 2, 3).
    float rs_a = 0.f, rs_b = 0.f, m_new = m_run;
    float a01 = 1.f;  // rescale of P blocks 0 and 1 by the second bound test
    // Adds a pair to its row-sum chain; the first pair of a chain starts it (0 + x is not
    // folded away: it would turn -0 into +0).
    auto row_add = [&](int q, float e0, float e1) {
      if (q < 8) {
        rs_a = q == 0 ? e0 + e1 : rs_a + (e0 + e1);
        pin(rs_a);
      } else {
        rs_b = q == 8 ? e0 + e1 : rs_b + (e0 + e1);
        pin(rs_b);
      }
    };
    auto prob_pair = [&](int q) {  // scores 2q, 2q+1 -> P block q/4, word q%4
      const int mb = q >> 3, o2 = (2 * q) & 15;
      const float e0 = __builtin_amdgcn_exp2f(fmaf(s_cur[mb][o2], c, -m_new));
      const float e1 = __builtin_amdgcn_exp2f(fmaf(s_cur[mb][o2 + 1], c, -m_new));
      row_add(q, e0, e1);
      bf16x2 pr;
      pr[0] = (__bf16)e0;
      pr[1] = (__bf16)e1;
      uint32_t w = __builtin_bit_cast(uint32_t, pr);
      pin(w);
      pw[q >> 2][q & 3] = w;
    };
    // Software pipeline of the pairs over the MFMA slots: a slot forms the exponent
    // arguments of pair k, the exponentials of pair k - 1 and the row-sum adds and bf16 pack
    // of pair k - 2, so no instruction of a slot waits on another of the same slot.
    float pa0 = 0.f, pa1 = 0.f;  // exponent arguments of the pair started one slot earlier
    float pe0 = 0.f, pe1 = 0.f;  // exponentials of the pair started two slots earlier
    auto pair_fin = [&](int q) {
      row_add(q, pe0, pe1);
      bf16x2 pr;
      pr[0] = (__bf16)pe0;
      pr[1] = (__bf16)pe1;
      uint32_t w = __builtin_bit_cast(uint32_t, pr);
      pin(w);
      pw[q >> 2][q & 3] = w;
    };
    auto pipe_slot = [&](int k, int lo, int hi) {  // pairs lo..hi-1
      if (k - 2 >= lo && k - 2 < hi) pair_fin(k - 2);
      if (k - 1 >= lo && k - 1 < hi) {
        pe0 = __builtin_amdgcn_exp2f(pa0);
        pe1 = __builtin_amdgcn_exp2f(pa1);
        pin(pe0);
        pin(pe1);
      }
      if (k >= lo && k < hi) {
        const int mb = k >> 3, o2 = (2 * k) & 15;
        pa0 = fmaf(s_cur[mb][o2], c, -m_new);
        pa1 = fmaf(s_cur[mb][o2 + 1], c, -m_new);
        pin(pa0);
        pin(pa1);
      }
    };
    // Row max of the lane's scores in key blocks mb0..1, shared by the lane pair of a query.
    auto tile_max = [&](int mb0) {
      float m = s_cur[1][0];
      pin(m);  // keeps the reduction in the cold path (it was otherwise begun in the hot block)
#pragma unroll
      for (int r = 1; r < 16; ++r) m = fmaxf(m, s_cur[1][r]);
      if (mb0 == 0) {
#pragma unroll
        for (int r = 0; r < 16; ++r) m = fmaxf(m, s_cur[0][r]);
      }
      return xor32_max(m) * c;
    };
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) s_next[mb] = f32x16{};
    bf16x8 ka[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) ka[i] = k_operand(i);
    __builtin_amdgcn_sched_barrier(0);
    // Probabilities against the running max: a lane's partial row sum bounds each of its
    // terms, so a sum within PBOUND (NaN and inf fail the test) proves that none exceeds
    // it and the running max may stay; otherwise a cold path moves the max.
#pragma unroll
    for (int i = 0; i < NQK; ++i) {
      s_next[i / KS] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[i & 3], qreg[i % KS], s_next[i / KS], 0, 0, 0);
      if (i + 4 < NQK) ka[i & 3] = k_operand(i + 4);
      if (i < 12) pipe_slot(i, 0, 10);  // pairs 0..9: P blocks 0, 1 and half of block 2
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int k = NQK; k < 12; ++k) pipe_slot(k, 0, 10);  // head_dim 64: fewer MFMAs than slots
    if (__any(!(rs_a + rs_b <= PBOUND))) {
      // Rare (always at a workgroup's first tile): move the max to the tile's row max
      // (nothing of this tile is in O^T yet) and form pairs 0..9 again.
      m_new = fmaxf(tile_max(0), m_run);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
      lo_run *= alpha;
#pragma unroll
      for (int i = 0; i < DB; ++i) o[i] *= alpha;
      m_run = m_new;
      rs_a = rs_b = 0.f;
#pragma unroll
      for (int q = 0; q < 10; ++q) prob_pair(q);
    }

    // ---- phase B: O^T += V_j^T P_j^T, P block-major; the probabilities of P blocks
    // 2 and 3 are formed under the MFMAs of blocks 0 and 1. V^T operands come from
    // LDS transpose reads issued two MFMAs ahead.
    if (partner) __builtin_amdgcn_s_setprio(0); else __builtin_amdgcn_s_setprio(1);
    // The next tiles' direct loads: issued here rather than at the top of the iteration, so
    // their LDS writes do not land under phase A's K operand reads (about -1.5%).
    if (kc.t < j1) {
      if (kc.t == n_rt) {
        cursor_view(std::true_type{}, kc, kc.t);
      } else if constexpr (SEG) {
        if (kc.t == kc_end) cursor_next_seg(std::true_type{}, kc);
      }
      kc.load(kb_cur, wave_u);
    }
    if (vc.t < j1) {
      if (vc.t == n_rt) {
        cursor_view(std::false_type{}, vc, vc.t);
      } else if constexpr (SEG) {
        if (vc.t == vc_end) cursor_next_seg(std::false_type{}, vc);
      }
      vc.load(vb_next, wave_u);
    }
    const uint16_t* vs = vb_cur;
    auto v_operand = [&](int i) {  // i = DB * s2 + db
      const uint16_t* a = vs + v_lane + 512 * i;
      const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(a));
      const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(a + 128));
      return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    };
    bf16x8 va[3];
    va[0] = v_operand(0);
    va[1] = v_operand(1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < NPV; ++i) {
      const int s2 = i / DB;
      const u32x4 pwv = {pw[s2][0], pw[s2][1], pw[s2][2], pw[s2][3]};
      o[i % DB] =
          __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[i % 3], __builtin_bit_cast(bf16x8, pwv), o[i % DB], 0, 0, 0);
      if (i + 2 < NPV) va[(i + 2) % 3] = v_operand(i + 2);
      // pairs 10..15 complete P blocks 2 and 3 before the first MFMA that reads them
      if (DB == 4 && i < 8) pipe_slot(10 + i, 10, 16);
      if (DB == 2 && i < 3) {
        prob_pair(10 + 2 * i);
        prob_pair(11 + 2 * i);
      }
      __builtin_amdgcn_sched_barrier(0);
      if (i == 2 * DB - 1 && __any(!(rs_b <= PBOUND))) {
        // Rare: pairs 8..15 exceed the bound. O^T holds this tile's P blocks 0 and 1
        // against the old max: rescale it with l and their sum, then form P blocks 2
        // and 3 against the new max before their MFMAs. Blocks 0 and 1 passed the first
        // test and only shrink, so the max of key block 1 suffices.
        m_new = fmaxf(tile_max(1), m_run);
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        l_run *= alpha;
        lo_run *= alpha;
        a01 = alpha;
        rs_a *= alpha;
#pragma unroll
        for (int k = 0; k < DB; ++k) o[k] *= alpha;
        m_run = m_new;
        rs_b = 0.f;
#pragma unroll
        for (int q = 8; q < 16; ++q) prob_pair(q);
      }
    }
    l_run += rs_a + rs_b;
    // The rounded sum of the tile's P after its last MFMA has issued: in the MFMA slots the
    // dot2 instructions slowed the matrix core's issue (+8% against +2.5% here).
    __builtin_amdgcn_sched_barrier(0);
    {
      float s01 = 0.f, s23 = 0.f;
#pragma unroll
      for (int wd = 0; wd < 8; ++wd) {
        s01 = add_bf16x2(pw[wd >> 2][wd & 3], s01);
        s23 = add_bf16x2(pw[2 + (wd >> 2)][wd & 3], s23);
      }
      lo_run += s01 * a01 + s23;
      pin(lo_run);
    }

    if (SEGM) {  // per-segment statistics
      if (j + 1 == seg_end_t) close_segment();  // end of reference segment seg_idx
    } else if (j == n_rt - 1) {  // end of the reference segment: freeze its statistics
      m_ref = m_run;
      l_ref = l_run;
      l_run = 0.f;
    }
    __syncthreads();
  };

  int j = j0;
  for (; j + 1 < j1; j += 2) {
    iteration(std::integral_constant<int, 0>{}, j, sa, sb);
    iteration(std::integral_constant<int, 1>{}, j + 1, sb, sa);
  }
  if (j < j1) iteration(std::integral_constant<int, 0>{}, j, sa, sb);
  if (j1 < n_rt) {  // a key chunk inside the reference segment: all of it is reference mass
    if (SEGM) {
      // The chunk ends inside a segment unless its end is a segment end: close its part.
      const int seg_start = seg_idx > 0 ? seg_end_tab[seg_idx - 1] : 0;
      if (max(seg_start, j0) < j1) close_segment();
    } else {
      m_ref = m_run;
      l_ref = l_run;
      l_run = 0.f;
    }
  }

  const float lo_sum = xor32_add(lo_run);  // both lanes of a query hold half its keys
  const float l_sum = xor32_add(l_run), l_ref_sum = xor32_add(l_ref);
  // ---- epilogue of a key chunk: unnormalised output and statistics to the workspace
  if (slot >= 0) {
    if (qvalid) {
      const int64_t prow = (int64_t)slot * BM + wave * 32 + n;
      float* po = p.part_o + prow * D;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr)
          *reinterpret_cast<float4*>(po + 32 * db + 8 * rr + 4 * g) =
              float4{o[db][4 * rr], o[db][4 * rr + 1], o[db][4 * rr + 2], o[db][4 * rr + 3]};
      if (g == 0) {
        p.part_st[prow] = float4{m_run, l_sum, m_ref, l_ref_sum};
        p.part_lo[prow] = lo_sum;
      }
    }
    probe_end();
    return;
  }

  // ---- epilogue
  const float L_R = l_ref_sum > 0.f ? l_ref_sum * __builtin_amdgcn_exp2f(m_ref - m_run) : 0.f;
  const float total = L_R + l_sum;
  const float inv = 1.f / total;
  const float inv_o = 1.f / lo_sum;
  if (qvalid) {
    uint16_t* op = static_cast<uint16_t*>(const_cast<void*>(ov.p)) + b * ov.sb + h * ov.sh + (int64_t)qrow * ov.ss;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        union {
          __bf16 h[4];
          u32x2 w;
        } pk;
#pragma unroll
        for (int i = 0; i < 4; ++i) pk.h[i] = (__bf16)(o[db][4 * rr + i] * inv_o);
        *reinterpret_cast<u32x2*>(op + 32 * db + 8 * rr + 4 * g) = pk.w;
      }
    if (g == 0) {
      const float mass = L_R * inv;
      const int64_t row = (int64_t)bh * n_rows + qrow;
      if (!ref_rows) {
        if (p.mass_tgt) p.mass_tgt[row] = mass;
        if (p.lse_tgt) {
          const float ln2 = 0.69314718055994531f;
          p.lse_tgt[2 * row] = (m_ref + __log2f(l_ref_sum)) * ln2;
          p.lse_tgt[2 * row + 1] = (m_run + __log2f(total)) * ln2;
        }
      } else if (p.mass_refq) {
        p.mass_refq[row] = mass;
      }
      if (SEGM && !ref_rows) {  // per-segment log-sum-exp -> mass, in place
        const float lt = m_run + __log2f(total);
        for (int s2 = 0; s2 < p.n_seg; ++s2)
          p.seg_mass[seg_row + s2] = __builtin_amdgcn_exp2f(p.seg_mass[seg_row + s2] - lt);
      }
    }
  }
  probe_end();
}

// Combines the key chunks of split query tiles: one row per D/4 threads, four
// output columns per thread. With M the largest running max over the chunks and
// M_R the largest reference max,
//   L'_R = sum_c l_R,c 2^(m_R,c - M_R),  L_R = L'_R 2^(M_R - M),
//   L_Y = sum_c l_Y,c 2^(m_c - M),  o = sum_c O_c 2^(m_c - M) / (L_R + L_Y),
//   mass = L_R / (L_R + L_Y),  lse_ref = M_R + log2 L'_R (times ln 2).
// A chunk's reference max never exceeds its running max, so M bounds both;
// summing the reference part against M_R keeps lse_ref finite when the target
// keys score so far above the reference keys that 2^(M_R - M) underflows.
template <int D, int MERGE_BATCH>
__device__ __forceinline__ void merge_rows(const AttnParams& p, const SplitPlan& pl, bool tgt_only) {
  constexpr int TPR = D / 4, RPB = 256 / TPR;
  const int qt_ref = tgt_only ? 0 : p.qt_ref;
  const int r = blockIdx.x * RPB + threadIdx.x / TPR, col = 4 * (threadIdx.x % TPR);
  const int st = r / BM, rr = r - st * BM;
  if (st >= pl.split_tiles) return;
  const int qt_bh = qt_ref + p.qt_tgt;
  const int tile = p.n_seg > 0 ? pl.whole + st : plan_split_tile(st, qt_bh, p.B * p.H, pl.split_tiles);
  const int bh = tile / qt_bh;
  int qt = tile - bh * qt_bh;
  const bool ref_rows = qt < qt_ref;
  if (!ref_rows) qt -= qt_ref;
  const int n_rows = ref_rows ? p.n_ref : p.n_tgt;
  const int qrow = qt * BM + rr;
  if (qrow >= n_rows) return;

  // Both passes load MERGE_BATCH chunks' partials before using any (one memory round trip
  // per batch instead of per chunk) and combine them in chunk order.
  const int nc = pl.chunks;
  const int64_t base = (int64_t)st * nc * BM + rr;  // partial row of chunk 0
  float M = -__builtin_inff(), M_R = -__builtin_inff();
  for (int c0 = 0; c0 < nc; c0 += MERGE_BATCH) {
    float4 sv[MERGE_BATCH];
#pragma unroll
    for (int u = 0; u < MERGE_BATCH; ++u)
      if (c0 + u < nc) sv[u] = p.part_st[base + (int64_t)(c0 + u) * BM];
#pragma unroll
    for (int u = 0; u < MERGE_BATCH; ++u) {
      if (c0 + u < nc) {
        M = fmaxf(M, sv[u].x);
        if (sv[u].w > 0.f) M_R = fmaxf(M_R, sv[u].z);
      }
    }
  }
  float L_Rr = 0.f, L_Y = 0.f;  // L_Rr: reference sum against M_R
  float L_o = 0.f;              // sum of the rounded probabilities that entered O
  float4 acc{0.f, 0.f, 0.f, 0.f};
  for (int c0 = 0; c0 < nc; c0 += MERGE_BATCH) {
    float4 sv[MERGE_BATCH], ov[MERGE_BATCH];
    float lv[MERGE_BATCH];
#pragma unroll
    for (int u = 0; u < MERGE_BATCH; ++u) {
      if (c0 + u < nc) {
        const int64_t prow = base + (int64_t)(c0 + u) * BM;
        sv[u] = p.part_st[prow];
        lv[u] = p.part_lo[prow];
        ov[u] = *reinterpret_cast<const float4*>(p.part_o + prow * D + col);
      }
    }
#pragma unroll
    for (int u = 0; u < MERGE_BATCH; ++u) {
      if (c0 + u < nc) {
        const float wgt = __builtin_amdgcn_exp2f(sv[u].x - M);
        L_Y += sv[u].y * wgt;
        L_o += lv[u] * wgt;
        if (sv[u].w > 0.f) L_Rr += sv[u].w * __builtin_amdgcn_exp2f(sv[u].z - M_R);
        acc.x += ov[u].x * wgt;
        acc.y += ov[u].y * wgt;
        acc.z += ov[u].z * wgt;
        acc.w += ov[u].w * wgt;
      }
    }
  }
  const float L_R = L_Rr > 0.f ? L_Rr * __builtin_amdgcn_exp2f(M_R - M) : 0.f;
  const float total = L_R + L_Y;
  const float inv = 1.f / total, inv_o = 1.f / L_o;
  const View ov = ref_rows ? p.o_ref : p.o_tgt;
  const int b = bh / p.H, h = bh - b * p.H;
  uint16_t* op = static_cast<uint16_t*>(const_cast<void*>(ov.p)) + b * ov.sb + h * ov.sh + (int64_t)qrow * ov.ss;
  union {
    __bf16 h[4];
    u32x2 w;
  } pk;
  pk.h[0] = (__bf16)(acc.x * inv_o);
  pk.h[1] = (__bf16)(acc.y * inv_o);
  pk.h[2] = (__bf16)(acc.z * inv_o);
  pk.h[3] = (__bf16)(acc.w * inv_o);
  *reinterpret_cast<u32x2*>(op + col) = pk.w;
  if (col == 0) {
    const float mass = L_R * inv;
    const int64_t row = (int64_t)bh * n_rows + qrow;
    if (!ref_rows) {
      if (p.mass_tgt) p.mass_tgt[row] = mass;
      if (p.lse_tgt) {
        const float ln2 = 0.69314718055994531f;
        p.lse_tgt[2 * row] = (M_R + __log2f(L_Rr)) * ln2;
        p.lse_tgt[2 * row + 1] = (M + __log2f(total)) * ln2;
      }
    } else if (p.mass_refq) {
      p.mass_refq[row] = mass;
    }
  }
  // Per-segment masses: thread col / 4 of the row combines segment s over the chunks whose
  // key range overlaps it, LSE_s = log2 sum_c 2^(lse_c,s), and stores 2^(LSE_s - LSE).
  const int s = col >> 2;
  if (p.seg_mass && !ref_rows && s < p.n_seg) {
    const int nt = (p.n_ref + BN - 1) / BN + (p.n_tgt + BN - 1) / BN;
    const int32_t* const ends = p.seg_tile_end;  // read through a pointer: no scratch copy
    const int s0 = s > 0 ? ends[s - 1] : 0, s1 = ends[s];
    const float* ps = p.part_seg + (int64_t)st * nc * BM * p.n_seg + (int64_t)rr * p.n_seg + s;
    float Ms = -__builtin_inff();
    for (int c = 0; c < nc; ++c)
      if (c * nt / nc < s1 && (c + 1) * nt / nc > s0) Ms = fmaxf(Ms, ps[(int64_t)c * BM * p.n_seg]);
    float Ls = 0.f;
    if (Ms > -__builtin_inff())
      for (int c = 0; c < nc; ++c)
        if (c * nt / nc < s1 && (c + 1) * nt / nc > s0) Ls += __builtin_amdgcn_exp2f(ps[(int64_t)c * BM * p.n_seg] - Ms);
    p.seg_mass[((int64_t)bh * p.n_tgt + qrow) * p.n_seg + s] =
        Ls > 0.f ? __builtin_amdgcn_exp2f(Ms + __log2f(Ls) - (M + __log2f(total))) : 0.f;
  }
}

template <int D, int MERGE_BATCH>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnParams p) {
  bool tgt_only = false;
  if (p.kvsrc == KV_DEVICE) tgt_only = __builtin_amdgcn_readfirstlane(*p.decision) == DEC_REUSE;
  const SplitPlan pl = p.plan[tgt_only ? 1 : 0];
  // Under a device-chosen plan the launch takes the wider instance for the plan with more
  // chunks; a two-chunk plan then runs the two-chunk body (one batch of loads, no guards).
  if constexpr (MERGE_BATCH > 2) {
    if (pl.chunks <= 2) {
      merge_rows<D, 2>(p, pl, tgt_only);
      return;
    }
  }
  merge_rows<D, MERGE_BATCH>(p, pl, tgt_only);
}

// Explicit instantiations: without them the host pass leaves the segment instances, which
// are only reached through the launcher's kernel-pointer argument, without launch stubs.
template __global__ void attn_bf16_kernel<128, false, false>(AttnParams);
template __global__ void attn_bf16_kernel<64, false, false>(AttnParams);
template __global__ void attn_bf16_kernel<128, true, false>(AttnParams);
template __global__ void attn_bf16_kernel<64, true, false>(AttnParams);
template __global__ void attn_bf16_kernel<128, true, true>(AttnParams);
template __global__ void attn_bf16_kernel<64, true, true>(AttnParams);

}  // namespace

AttnSlots attn_bf16_slots(int head_dim) {
  static std::atomic<int> cache[64][2][2];
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return AttnSlots{0, 0};
  const int di = head_dim == 128 ? 1 : 0;
  if (dev < 64) {
    const int c = cache[dev][di][0].load(std::memory_order_relaxed);
    if (c > 0) return AttnSlots{c, cache[dev][di][1].load(std::memory_order_relaxed)};
  }
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return AttnSlots{0, 0};
  const hipError_t e =
      head_dim == 128
          ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attn_bf16_kernel<128, false, false>, NT, 0)
          : hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attn_bf16_kernel<64, false, false>, NT, 0);
  if (e != hipSuccess || per_cu < 1 || cus < 1) return AttnSlots{0, 0};
  if (dev < 64) {
    cache[dev][di][1].store(per_cu, std::memory_order_relaxed);
    cache[dev][di][0].store(cus, std::memory_order_relaxed);
  }
  return AttnSlots{cus, per_cu};
}

hipError_t launch_attn_bf16(const AttnParams& p, int head_dim, hipStream_t stream) {
  const int items = max(p.plan[0].total_items, p.plan[1].total_items);
  if (items <= 0) return hipSuccess;
  const dim3 grid(items), block(NT);
  hipError_t e;
  if (p.n_seg > 0 && p.seg_mass) {
    e = head_dim == 128 ? launch_kernel(attn_bf16_kernel<128, true, true>, grid, block, 0, stream, p)
                        : launch_kernel(attn_bf16_kernel<64, true, true>, grid, block, 0, stream, p);
  } else if (p.n_seg > 0) {
    e = head_dim == 128 ? launch_kernel(attn_bf16_kernel<128, true, false>, grid, block, 0, stream, p)
                        : launch_kernel(attn_bf16_kernel<64, true, false>, grid, block, 0, stream, p);
  } else {
    e = head_dim == 128 ? launch_kernel(attn_bf16_kernel<128, false, false>, grid, block, 0, stream, p)
                        : launch_kernel(attn_bf16_kernel<64, false, false>, grid, block, 0, stream, p);
  }
  if (e != hipSuccess) return e;
  const int split = max(p.plan[0].split_tiles, p.plan[1].split_tiles);
  if (split == 0) return hipSuccess;
  const int rpb = 256 / (head_dim / 4);
  const dim3 mgrid((split * BM + rpb - 1) / rpb);
  // Loads in flight per merge thread: all chunks of a two-chunk split, else eight at a time.
  const bool two = max(p.plan[0].chunks, p.plan[1].chunks) <= 2;
  if (head_dim == 128)
    return two ? launch_kernel(attn_merge_kernel<128, 2>, mgrid, dim3(256), 0, stream, p)
               : launch_kernel(attn_merge_kernel<128, 8>, mgrid, dim3(256), 0, stream, p);
  return two ? launch_kernel(attn_merge_kernel<64, 2>, mgrid, dim3(256), 0, stream, p)
             : launch_kernel(attn_merge_kernel<64, 8>, mgrid, dim3(256), 0, stream, p);
}

}  // namespace refadapt
