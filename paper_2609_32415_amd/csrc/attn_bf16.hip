// Joint attention over [reference; target] keys on bf16 MFMA (gfx950).
//
// One workgroup = 4 wavefronts = 128 query rows of one (batch, head); each
// wavefront owns 32 query rows. Key/value tiles of 64 rows stream through a
// double-buffered LDS stage, reference tiles first (from the fresh or the
// cached reference K/V, chosen once per workgroup) and then target tiles.
//
// Per tile, a wavefront computes the transposed score block S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16 (keys on the M side, its 32 queries on the N side),
// so every lane holds 32 scores of ONE query: the row max and row sum of the
// online softmax are in-lane reductions plus one exchange with lane l^32. The
// probabilities P^T stay in registers and feed O^T += V^T P^T directly as the
// B operand; V^T comes from the LDS stage, where V is stored transposed.
//
// Split statistics for the reference mass: when the last reference tile is
// done the running (max, sum) pair is frozen as (m_R, l_R) and the sum restarts
// at zero for the target tiles, so at the end L_R = l_R * 2^(m_R - m) and
// L_Y = l are the reference and target parts of the softmax denominator in
// the same scale; mass = L_R / (L_R + L_Y) lies in [0, 1] by construction and
// equals exp(lse_R - lse_all) (paper Sec. 3.2 directional exposure).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace refadapt {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int BM = kAttnBf16BM;  // query rows per workgroup
constexpr int BN = 64;           // keys per LDS tile
constexpr int NT = 256;          // threads per workgroup

// Row permutation of a 32-key MFMA block: swaps bits 2 and 3 of the row index.
// Loading K row sigma(m) into A-row m makes output register r of lane-half g
// hold key 16*(r/8) + 8*g + r%8, i.e. eight consecutive keys per lane-half,
// which is exactly the K-operand order of the next MFMA's B operand (P^T).
__device__ __forceinline__ int sigma(int m) { return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1); }

__device__ __forceinline__ float wave_xor32_max(float v) { return fmaxf(v, __shfl_xor(v, 32)); }
__device__ __forceinline__ float wave_xor32_add(float v) { return v + __shfl_xor(v, 32); }

template <int D>
struct Prefetch {
  static constexpr int KCH = D / 8;               // 16-byte chunks per row
  static constexpr int NK = BN * KCH / NT;        // K chunks per thread
  static constexpr int NV = (BN / 2) * KCH / NT;  // V (key pair, chunk) units per thread
  u32x4 k[NK];
  u32x4 v[2 * NV];
};

template <int D>
__device__ __forceinline__ void load_tile(Prefetch<D>& pf, const uint16_t* kb, const uint16_t* vb, int64_t kss,
                                          int64_t vss, int valid, int tid) {
  constexpr int KCH = D / 8;
#pragma unroll
  for (int i = 0; i < Prefetch<D>::NK; ++i) {
    const int c = tid + NT * i;
    const int row = c / KCH, ch = c % KCH;
    pf.k[i] = row < valid ? *reinterpret_cast<const u32x4*>(kb + row * kss + ch * 8) : u32x4{0, 0, 0, 0};
  }
#pragma unroll
  for (int i = 0; i < Prefetch<D>::NV; ++i) {
    const int u = tid + NT * i;
    const int ch = u % KCH, pair = u / KCH;
    const int r0 = 2 * pair;
    pf.v[2 * i] = r0 < valid ? *reinterpret_cast<const u32x4*>(vb + r0 * vss + ch * 8) : u32x4{0, 0, 0, 0};
    pf.v[2 * i + 1] =
        r0 + 1 < valid ? *reinterpret_cast<const u32x4*>(vb + (r0 + 1) * vss + ch * 8) : u32x4{0, 0, 0, 0};
  }
}

// LDS layouts (bf16 elements):
//  K  tile: [BN][D], row r, 16-byte chunk c stored at chunk c ^ (sigma(r % 32) % 8)
//  V^T tile: [D][BN], row d, 16-byte chunk c (8 keys) stored at chunk c ^ ((d ^ (d / 8)) % 8)
// Both swizzles make the MFMA operand reads and the tile writes free of bank conflicts.
template <int D>
__device__ __forceinline__ void store_tile(const Prefetch<D>& pf, uint16_t* ks, uint16_t* vts, int tid) {
  constexpr int KCH = D / 8;
#pragma unroll
  for (int i = 0; i < Prefetch<D>::NK; ++i) {
    const int c = tid + NT * i;
    const int row = c / KCH, ch = c % KCH;
    const int phys = ch ^ (sigma(row & 31) & 7);
    *reinterpret_cast<u32x4*>(ks + row * D + phys * 8) = pf.k[i];
  }
#pragma unroll
  for (int i = 0; i < Prefetch<D>::NV; ++i) {
    const int u = tid + NT * i;
    const int ch = u % KCH, pair = u / KCH;
    const int key = 2 * pair;
    const u32x4 a = pf.v[2 * i], b = pf.v[2 * i + 1];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int d = ch * 8 + e;
      const uint32_t wa = a[e >> 1], wb = b[e >> 1];
      const uint32_t packed = (e & 1) ? ((wa >> 16) | (wb & 0xffff0000u)) : ((wa & 0xffffu) | (wb << 16));
      const int phys = (key >> 3) ^ ((d ^ (d >> 3)) & 7);
      *reinterpret_cast<uint32_t*>(vts + d * BN + phys * 8 + (key & 7)) = packed;
    }
  }
}

template <int D>
__global__ __launch_bounds__(NT, 2) void attn_bf16_kernel(AttnParams p) {
  constexpr int KS = D / 16;  // MFMA k-steps over the head dim for S^T
  constexpr int DB = D / 32;  // 32-row blocks of the O^T accumulator
  constexpr int TILE = BN * D;
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][2 * TILE];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, n = lane & 31;

  // ---- which (batch, head, query tile) this workgroup owns
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
    if (ref_rows && dec == DEC_REUSE) return;  // reference rows are skipped on a reused block
    use_cache = dec != DEC_COMPUTE;
  }

  const View& qv = ref_rows ? p.q_ref : p.q_tgt;
  const View& ov = ref_rows ? p.o_ref : p.o_tgt;
  const int n_rows = ref_rows ? p.n_ref : p.n_tgt;
  const View& krv = use_cache ? p.k_cache : p.k_fresh;
  const View& vrv = use_cache ? p.v_cache : p.v_fresh;

  const uint16_t* kr = static_cast<const uint16_t*>(krv.p) + b * krv.sb + h * krv.sh;
  const uint16_t* vr = static_cast<const uint16_t*>(vrv.p) + b * vrv.sb + h * vrv.sh;
  const uint16_t* ky = static_cast<const uint16_t*>(p.k_tgt.p) + b * p.k_tgt.sb + h * p.k_tgt.sh;
  const uint16_t* vy = static_cast<const uint16_t*>(p.v_tgt.p) + b * p.v_tgt.sb + h * p.v_tgt.sh;

  // ---- this lane's query row; Q^T as the B operand (query n, head-dim chunk 2*ks + g)
  const int qrow = qt * BM + wave * 32 + n;
  const bool qvalid = qrow < n_rows;
  bf16x8 qreg[KS];
  {
    const uint16_t* qp = static_cast<const uint16_t*>(qv.p) + b * qv.sb + h * qv.sh + (int64_t)qrow * qv.ss;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      u32x4 raw = qvalid ? *reinterpret_cast<const u32x4*>(qp + ks * 16 + g * 8) : u32x4{0, 0, 0, 0};
      qreg[ks] = __builtin_bit_cast(bf16x8, raw);
    }
  }

  const int n_rt = (p.n_ref + BN - 1) / BN;
  const int n_yt = (p.n_tgt + BN - 1) / BN;
  const int nt = n_rt + n_yt;

  auto tile_src = [&](int j, const uint16_t*& kb, const uint16_t*& vb, int64_t& kss, int64_t& vss, int& valid) {
    if (j < n_rt) {
      kb = kr + (int64_t)j * BN * krv.ss;
      vb = vr + (int64_t)j * BN * vrv.ss;
      kss = krv.ss;
      vss = vrv.ss;
      valid = min(BN, p.n_ref - j * BN);
    } else {
      const int jj = j - n_rt;
      kb = ky + (int64_t)jj * BN * p.k_tgt.ss;
      vb = vy + (int64_t)jj * BN * p.v_tgt.ss;
      kss = p.k_tgt.ss;
      vss = p.v_tgt.ss;
      valid = min(BN, p.n_tgt - jj * BN);
    }
  };

  f32x16 o[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) o[i] = f32x16{};
  float m_run = -__builtin_inff(), l_run = 0.f;
  float m_ref = -__builtin_inff(), l_ref = 0.f;
  const float c = p.sc_log2;

  Prefetch<D> pf;
  {
    const uint16_t *kb, *vb;
    int64_t kss, vss;
    int valid;
    tile_src(0, kb, vb, kss, vss, valid);
    load_tile<D>(pf, kb, vb, kss, vss, valid, tid);
    store_tile<D>(pf, lds[0], lds[0] + TILE, tid);
  }
  __syncthreads();

  for (int j = 0; j < nt; ++j) {
    int valid_next = 0;
    if (j + 1 < nt) {
      const uint16_t *kb, *vb;
      int64_t kss, vss;
      tile_src(j + 1, kb, vb, kss, vss, valid_next);
      load_tile<D>(pf, kb, vb, kss, vss, valid_next, tid);
    }
    const uint16_t* ks = lds[j & 1];
    const uint16_t* vts = ks + TILE;
    const int valid = j < n_rt ? min(BN, p.n_ref - j * BN) : min(BN, p.n_tgt - (j - n_rt) * BN);

    // ---- S^T = K Q^T for two 32-key blocks
    f32x16 s[2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      s[mb] = f32x16{};
      const uint16_t* krow = ks + (32 * mb + sigma(n)) * D;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const int phys = (2 * kk + g) ^ (n & 7);
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(krow + phys * 8);
        s[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[kk], s[mb], 0, 0, 0);
      }
    }
    if (valid < BN) {  // ragged last tile of a segment: drop keys past its end
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = 32 * mb + 16 * (r >> 3) + 8 * g + (r & 7);
          if (key >= valid) s[mb][r] = -__builtin_inff();
        }
    }

    // ---- online softmax in the exp2 domain (scores scaled by scale*log2(e))
    float mx = -__builtin_inff();
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[mb][r]);
    mx = wave_xor32_max(mx);
    const float m_new = fmaxf(m_run, mx * c);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    float rs = 0.f;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = __builtin_amdgcn_exp2f(fmaf(s[mb][r], c, -m_new));
        s[mb][r] = e;
        rs += e;
      }
    rs = wave_xor32_add(rs);
    l_run = l_run * alpha + rs;
    m_run = m_new;
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int i = 0; i < DB; ++i) o[i] *= alpha;
    }

    // ---- P^T to bf16 B operands: k-step s2 covers keys 16*s2 .. 16*s2+15
    bf16x8 pb[4];
#pragma unroll
    for (int s2 = 0; s2 < 4; ++s2)
#pragma unroll
      for (int i = 0; i < 8; ++i) pb[s2][i] = (__bf16)s[s2 >> 1][8 * (s2 & 1) + i];

    // ---- O^T += V^T P^T
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int d = 32 * db + n;
      const int swz = (d ^ (d >> 3)) & 7;
      const uint16_t* vrow = vts + d * BN;
#pragma unroll
      for (int s2 = 0; s2 < 4; ++s2) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(vrow + (((2 * s2 + g) ^ swz) * 8));
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[s2], o[db], 0, 0, 0);
      }
    }

    if (j == n_rt - 1) {  // end of the reference segment: freeze its statistics
      m_ref = m_run;
      l_ref = l_run;
      l_run = 0.f;
    }
    if (j + 1 < nt) store_tile<D>(pf, lds[(j + 1) & 1], lds[(j + 1) & 1] + TILE, tid);
    __syncthreads();
  }

  // ---- epilogue
  const float L_R = l_ref > 0.f ? l_ref * __builtin_amdgcn_exp2f(m_ref - m_run) : 0.f;
  const float total = L_R + l_run;
  const float inv = 1.f / total;
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
        for (int i = 0; i < 4; ++i) pk.h[i] = (__bf16)(o[db][4 * rr + i] * inv);
        *reinterpret_cast<u32x2*>(op + 32 * db + 8 * rr + 4 * g) = pk.w;
      }
    if (g == 0) {
      const float mass = L_R * inv;
      const int64_t row = (int64_t)bh * n_rows + qrow;
      if (!ref_rows) {
        if (p.mass_tgt) p.mass_tgt[row] = mass;
        if (p.lse_tgt) {
          const float ln2 = 0.69314718055994531f;
          p.lse_tgt[2 * row] = (m_ref + __log2f(l_ref)) * ln2;
          p.lse_tgt[2 * row + 1] = (m_run + __log2f(total)) * ln2;
        }
      } else if (p.mass_refq) {
        p.mass_refq[row] = mass;
      }
    }
  }
}

}  // namespace

hipError_t launch_attn_bf16(const AttnParams& p, int head_dim, hipStream_t stream) {
  if (p.total_tiles <= 0) return hipSuccess;
  const dim3 grid(p.total_tiles), block(NT);
  return head_dim == 128 ? launch_kernel(attn_bf16_kernel<128>, grid, block, 0, stream, p)
                         : launch_kernel(attn_bf16_kernel<64>, grid, block, 0, stream, p);
}

}  // namespace refadapt
