/*
 * refadapt.h - C ABI of the MI355X (gfx950) hot path of RefAdapt-DiT
 * (arxiv 2609.32415): joint attention over a [reference; target] token
 * sequence with fresh or cached reference K/V and per-query reference mass,
 * the consecutive target-Q change, the reuse gate and the cache commit.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Tensor pointers are DEVICE pointers (memory of the current HIP device);
 *   descriptors and argument structs are HOST memory read during the call.
 * - The caller owns every buffer. The library allocates no device memory and
 *   never synchronises: each call validates its arguments on the host, then
 *   enqueues kernels on `stream` (a hipStream_t; NULL is the null stream) and
 *   returns. All calls are stream-ordered and contain no host round-trip.
 * - Errors: arguments are validated synchronously and a non-zero ra_status is
 *   returned; nothing is enqueued in that case. refadapt_last_error() gives a
 *   message for the calling thread's last failing call. Device-side faults
 *   are asynchronous and surface at the caller's next synchronisation.
 * - Tensors are [B, H, S, d] with explicit element strides for B, H and S;
 *   the head dimension d is contiguous (stride 1). bf16 tensors need 16-byte
 *   aligned base pointers and strides that are multiples of 8 elements;
 *   fp32 tensors need 16-byte alignment and strides that are multiples of 4.
 */
#ifndef REFADAPT_H
#define REFADAPT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RA_OK = 0,
  RA_EINVAL = -1,        /* malformed argument (null pointer, bad size or enum) */
  RA_EUNSUPPORTED = -2,  /* well-formed but not implemented (head_dim, alignment) */
  RA_EWORKSPACE = -3,    /* workspace missing or too small */
  RA_ELAUNCH = -4        /* the HIP runtime refused a launch */
} ra_status;

typedef enum { RA_BF16 = 0, RA_F32 = 1 } ra_dtype;

/* Which query rows attend (paper App. A.4: a cached step drops the two
 * reference-query score regions). */
typedef enum {
  RA_Q_TARGET = 0, /* target queries only: o_tgt (and ref_mass) are written */
  RA_Q_ALL = 1     /* reference and target queries: o_ref and o_tgt written */
} ra_qset;

/* Source of the reference segment's K/V. */
typedef enum {
  RA_KV_FRESH = 0, /* k_ref / v_ref (this step's reference K/V) */
  RA_KV_CACHE = 1, /* k_cache / v_cache (the block cache of Sec. 4) */
  RA_KV_DEVICE = 2, /* chosen on the device from *decision (ra_decision):
                     *   REUSE      -> target queries only, cached K/V
                     *   REACTIVATE -> all queries, cached K/V
                     *   COMPUTE    -> all queries, fresh K/V */
  RA_KV_SEGMENTS = 3 /* per reference segment (ra_attn_args.seg_*): segment s
                      * reads the cached K/V when bit s of seg_cache is set,
                      * else the fresh K/V (bf16 only) */
} ra_kvsrc;

/* Most reference segments (e.g. reference images and text) one call can tell apart. */
#define RA_MAX_SEG 16

/* Block decisions of Alg. 1 (monotone depth-adaptive reference reuse). */
typedef enum { RA_REUSE = 0, RA_REACTIVATE = 1, RA_COMPUTE = 2 } ra_decision;

/* Score the gate compares with the block threshold. PRODUCT is the paper's
 * (Sec. 4 factorized-risk equation, head mean of App. A.2); Q_ONLY and
 * MASS_ONLY are the single-cue ablations; AND compares mean D and mean M with
 * a (theta_q, theta_m) pair. */
typedef enum {
  RA_GATE_PRODUCT = 0,
  RA_GATE_Q_ONLY = 1,
  RA_GATE_MASS_ONLY = 2,
  RA_GATE_AND = 3
} ra_gate_mode;

/* A [B, H, S, d] tensor: base pointer and element strides of B, H and S. */
typedef struct {
  void* data;
  int64_t stride_b, stride_h, stride_s;
} ra_tensor;

typedef struct {
  int32_t batch, heads, head_dim; /* head_dim in {64, 128} */
  int32_t n_ref;                  /* reference tokens (>= 0; 0 = plain self-attention) */
  int32_t n_tgt;                  /* target tokens (>= 1) */
  int32_t dtype;                  /* ra_dtype of Q/K/V and outputs */
  float scale;                    /* softmax scale; <= 0 selects 1/sqrt(head_dim) */
  int32_t qset;                   /* ra_qset (ignored for RA_KV_DEVICE) */
  int32_t kvsrc;                  /* ra_kvsrc */
} ra_attn_desc;

typedef struct {
  ra_tensor q_tgt, k_tgt, v_tgt; /* [B, H, n_tgt, d] target rows */
  ra_tensor q_ref;               /* [B, H, n_ref, d] reference queries (RA_Q_ALL / DEVICE) */
  ra_tensor k_ref, v_ref;        /* [B, H, n_ref, d] fresh reference K/V */
  ra_tensor k_cache, v_cache;    /* [B, H, n_ref, d] cached reference K/V */
  const int32_t* decision;       /* device word (ra_decision), RA_KV_DEVICE only */
  ra_tensor o_tgt;               /* out [B, H, n_tgt, d] */
  ra_tensor o_ref;               /* out [B, H, n_ref, d] (RA_Q_ALL / DEVICE) */
  float* ref_mass;               /* out [B, H, n_tgt] contiguous fp32, or NULL */
  float* lse_tgt;                /* out [B, H, n_tgt, 2] = (lse_ref, lse_all), or NULL */
  float* ref_mass_refq;          /* out [B, H, n_ref] reference-query mass on reference keys, or NULL */
  void* workspace;               /* device scratch for key-split partial results, or NULL (no split) */
  size_t workspace_bytes;        /* its size; >= refadapt_joint_attn_workspace_size(desc) when non-NULL */
  /* Reference segments (used with RA_KV_SEGMENTS or a non-NULL seg_mass; else ignored):
   * segment s holds reference rows [seg_end[s-1], seg_end[s]) (seg_end[-1] = 0). */
  int32_t n_seg;                 /* 1..RA_MAX_SEG */
  int32_t seg_end[RA_MAX_SEG];   /* increasing; multiples of 64 except seg_end[n_seg-1] == n_ref */
  uint32_t seg_cache;            /* RA_KV_SEGMENTS: bit s selects the cached K/V for segment s */
  float* seg_mass;               /* out [B, H, n_tgt, n_seg] target-query mass per segment, or NULL */
  /* Cached reference queries [B, H, n_ref, d] (the queries of the block's cached reference
   * state), or NULL data. When given, reference queries that attend over the cached
   * reference K/V read them instead of q_ref: under RA_KV_CACHE with RA_Q_ALL, and on
   * REACTIVATE under RA_KV_DEVICE (Alg. 1 boundary branch: the cached reference state is
   * restored and its queries attend to [cached K_R; current K_Y]). */
  ra_tensor q_cache;
  /* Optional clock probe (bf16 path; ignored by fp32), or NULL: the first lane of every
   * workgroup adds its shader-clock cycles to clock_probe[0] and the 100 MHz reference
   * ticks over the same interval to clock_probe[1] (device uint64, added to, so the caller
   * zeroes them). 100 MHz * [0] / [1] is the launch's mean shader clock. */
  uint64_t* clock_probe;
} ra_attn_args;

/*
 * refadapt_joint_attn - joint softmax attention over [K_R; K_Y].
 *
 * Computes, for every (b, h) and query row q of the selected query set,
 *   o_q = sum_k softmax_k(scale * q.k) v_k  over keys [K_R; K_Y], values [V_R; V_Y]
 * (paper Sec. 3.3, fresh/stale-output equations; App. A.4 score regions),
 * where K_R/V_R are the fresh or cached reference K/V per `kvsrc`, and for
 * every target query the reference mass
 *   ref_mass_q = sum_{k in R} A_qk = exp(lse_ref - lse_all)
 * (Sec. 3.2 directional-exposure equation, before its mean over queries),
 * obtained from split online-softmax statistics in the same pass; it lies in
 * [0, 1] by construction and is 0 when n_ref == 0. lse values are natural-log
 * log-sum-exp of the scaled logits over reference keys / all keys (lse_ref is
 * -inf when n_ref == 0). Outputs are written in `dtype` (accumulation is fp32,
 * bf16 MFMA for RA_BF16). Writing ref_mass / lse does not change o (the
 * attention output is bit-identical with them on or off). Requesting seg_mass
 * folds the reference sums segment by segment, so o then differs from the
 * launch without it by fp32 rounding only.
 *
 * Under RA_KV_DEVICE the launch is sized for every query and the workgroups
 * read *decision first: on RA_REUSE only target query rows are computed and
 * o_ref is left untouched.
 *
 * Reference segments (bf16): the reference rows may be split into n_seg
 * segments (the reference images and the text; App. "probe non-intrusiveness
 * and multi-reference controls": the references are not interchangeable).
 * Under RA_KV_SEGMENTS each segment reads fresh or cached K/V as seg_cache
 * says, so one launch evaluates a stale cache for any subset of the
 * references. seg_mass[b, h, q, s] = sum over the keys k of segment s of A_qk
 * (the directional exposure of Sec. 3.2 restricted to one segment); the
 * segments' masses add up to ref_mass. Segment boundaries must fall on 64-row
 * key tiles (the last one is n_ref), and under RA_KV_SEGMENTS the fresh and
 * cached K (and V) views must share their strides. With seg_mass the launch
 * splits key ranges only when workspace_bytes is at least
 * refadapt_joint_attn_seg_workspace_size(desc, n_seg) (each key chunk then
 * records a partial log-sum-exp per segment, which the merge combines);
 * with a smaller or no workspace it runs whole query tiles.
 *
 * Load balance (bf16): with a workspace, query tiles of a last, partly filled
 * round of workgroups are split into key-tile ranges whose partial softmax
 * statistics a second kernel merges (the same rescale-and-add the online
 * softmax applies across key tiles). Results then differ from the unsplit
 * launch only by fp32 rounding; a given desc on a given device always takes
 * the same split, so repeated calls are bitwise identical. With
 * workspace == NULL nothing is split. The workspace needs no initialisation,
 * must be 16-byte aligned and must not be used by another call that runs
 * concurrently. The fp32 path never splits.
 *
 * Errors: RA_EINVAL for a null desc/args, sizes out of range, unknown enums,
 * or a required pointer that is NULL (q/k/v/o_tgt always; k_ref/v_ref when
 * fresh K/V may be read and n_ref > 0; k_cache/v_cache when cached K/V may be
 * read and n_ref > 0; q_ref/o_ref when reference queries may attend and
 * n_ref > 0, except q_ref under RA_KV_CACHE when q_cache is given; decision
 * under RA_KV_DEVICE; n_seg outside 1..RA_MAX_SEG or
 * segment ends that do not increase to n_ref). RA_EUNSUPPORTED for head_dim not
 * in {64, 128} or misaligned tensors or workspace, and for segments with
 * RA_F32, RA_KV_DEVICE, an inner boundary off the 64-row key tiles, or (under
 * RA_KV_SEGMENTS) fresh and cached views with different strides, and (RA_BF16) for a
 * K/V row stride above 2^24 - 8 elements (key tiles use 32-bit offsets). RA_EWORKSPACE for a
 * non-NULL workspace smaller than refadapt_joint_attn_workspace_size(desc).
 */
ra_status refadapt_joint_attn(const ra_attn_desc* desc, const ra_attn_args* args, void* stream);

/*
 * refadapt_joint_attn_workspace_size - bytes of workspace that let
 * refadapt_joint_attn split key ranges for `desc` on the CURRENT device (the
 * split depends on the device's compute-unit count). 0 when no split pays or
 * for an invalid desc (refadapt_joint_attn then reports the error).
 */
size_t refadapt_joint_attn_workspace_size(const ra_attn_desc* desc);

/*
 * refadapt_joint_attn_seg_workspace_size - bytes of workspace that let a
 * refadapt_joint_attn call with seg_mass over n_seg reference segments split
 * key ranges for `desc` on the CURRENT device: the key-split partials plus one
 * fp32 log-sum-exp per segment of each partial row (per-segment masses of the
 * target queries, App. "probe non-intrusiveness and multi-reference
 * controls"). 0 when no split pays, for an invalid desc, for n_seg outside
 * 1..RA_MAX_SEG, and where segments are unavailable (RA_F32, RA_KV_DEVICE,
 * n_ref == 0).
 */
size_t refadapt_joint_attn_seg_workspace_size(const ra_attn_desc* desc, int32_t n_seg);

/*
 * refadapt_q_change - consecutive relative change of the target queries.
 *
 *   d_out[b, h] = ||Q_cur[b,h] - Q_prev[b,h]||_F / (||Q_prev[b,h]||_F + eps)
 * over the n_tgt x head_dim slice of each (b, h) (paper Sec. 3.1
 * consecutive-drift equation, applied to post-RoPE target-query heads as in
 * Sec. 4 "Runtime cues"). Sums are fp32 within a workgroup and fp64 across
 * workgroups in a fixed order, so the result is bitwise deterministic.
 *
 * `workspace` is device memory of at least
 * refadapt_q_change_workspace_size(...) bytes (scratch for per-chunk partial
 * sums; contents need no initialisation). d_out is [B, H] contiguous fp32.
 * Errors: RA_EINVAL (null pointers, sizes), RA_EUNSUPPORTED (alignment),
 * RA_EWORKSPACE (workspace NULL or smaller than required).
 */
size_t refadapt_q_change_workspace_size(int32_t batch, int32_t heads, int32_t n_tgt, int32_t head_dim);
ra_status refadapt_q_change(int32_t batch, int32_t heads, int32_t n_tgt, int32_t head_dim, int32_t dtype,
                            ra_tensor q_cur, ra_tensor q_prev, float eps, float* d_out, void* workspace,
                            size_t ws_bytes, void* stream);

/* Device-resident controller state of one denoising trajectory (Alg. 1). */
typedef struct {
  int32_t reactivated; /* an earlier block of the current step reached its threshold */
  int32_t a_full;      /* step of the last full refresh */
  int32_t delta_max;   /* bounded-age refresh period; <= 0 disables it */
  int32_t step;        /* step seen by the last block-0 call */
} ra_gate_state;

/*
 * refadapt_gate - one block's reuse decision, on the device.
 *
 * With M_h = mean over target queries of mass_prev[b, h, :] (the per-query
 * reference mass this block's executed attention produced at the previous
 * step; Sec. 3.2 directional-exposure equation, lagged as in Sec. 4) and
 * D_h = d_cur[b, h] (refadapt_q_change of this block), the score is
 * mean over (b, h) of D_h * M_h (Sec. 4 factorized-risk equation; head mean of
 * App. A.2). Decision (Sec. 4 depth-cutoff equation and the block branch of
 * Alg. 1): COMPUTE if state->reactivated; else REACTIVATE (and set
 * state->reactivated) if score >= theta; else REUSE.
 *
 * When block == 0 the call first performs the step bookkeeping of Alg. 1:
 * step 0, or step - a_full >= delta_max (delta_max > 0), is a full refresh
 * (a_full = step and reactivated = 1, so every block of the step computes);
 * otherwise reactivated = 0. `theta` is a device array indexed by block:
 * theta[block] for PRODUCT / Q_ONLY / MASS_ONLY, pairs theta[2*block],
 * theta[2*block+1] = (theta_q, theta_m) for AND.
 *
 * Outputs (device): *decision_out (ra_decision) and score_out[0..2] =
 * (mean D, mean M, mean D*M). Errors: RA_EINVAL for null pointers, sizes,
 * block < 0, step < 0 or an unknown mode.
 */
ra_status refadapt_gate(int32_t batch, int32_t heads, int32_t n_tgt, int32_t block, int32_t step, int32_t mode,
                        const float* d_cur, const float* mass_prev, const float* theta, ra_gate_state* state,
                        int32_t* decision_out, float* score_out, void* stream);

/*
 * refadapt_q_change_gate - refadapt_q_change and refadapt_gate fused.
 *
 * Computes d_out[b, h] exactly as refadapt_q_change (bitwise the same values)
 * and then the decision of refadapt_gate for `block` at `step` (same
 * bookkeeping, modes, theta layout and outputs). The mean lagged mass M_h is
 * summed by the Q-change workgroups over their rows (fp32 within a workgroup,
 * fp64 across workgroups in a fixed order), so the head reductions of both
 * steps run on every CU and the whole step is two kernels instead of three.
 *
 * `workspace`: device memory of at least refadapt_q_change_gate_workspace_size
 * bytes, 16-byte aligned; contents need no initialisation.
 * Errors: as refadapt_q_change and refadapt_gate together.
 */
size_t refadapt_q_change_gate_workspace_size(int32_t batch, int32_t heads, int32_t n_tgt, int32_t head_dim);
ra_status refadapt_q_change_gate(int32_t batch, int32_t heads, int32_t n_tgt, int32_t head_dim, int32_t dtype,
                                 ra_tensor q_cur, ra_tensor q_prev, float eps, int32_t block, int32_t step,
                                 int32_t mode, const float* mass_prev, const float* theta, ra_gate_state* state,
                                 float* d_out, int32_t* decision_out, float* score_out, void* workspace,
                                 size_t ws_bytes, void* stream);

/*
 * refadapt_q_change_gate_noalloc - refadapt_q_change_gate without a workspace.
 *
 * For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): the same computation
 * and outputs as refadapt_q_change_gate (bitwise), with the per-chunk partial
 * sums kept in a fixed 1 MiB device array of the library instead of a caller
 * workspace. Nothing is allocated: each device holds its copy of that array
 * from the library's load until the process ends; its address is looked up on
 * the first call on a device. Calls on one device share the array, so calls
 * that can overlap on a device (other streams, other threads) race and must be
 * serialised by the caller. Contents need no initialisation (every call writes
 * all the partials it reads).
 * Errors: as refadapt_q_change_gate; RA_EUNSUPPORTED when the shape needs more
 * than 1 MiB of partials (refadapt_q_change_gate_workspace_size > 1048576, e.g.
 * batch*heads > 1024 with 64 chunks per head) or the device index is 64 or
 * above; RA_ELAUNCH when the array's address cannot be obtained.
 */
ra_status refadapt_q_change_gate_noalloc(int32_t batch, int32_t heads, int32_t n_tgt, int32_t head_dim,
                                         int32_t dtype, ra_tensor q_cur, ra_tensor q_prev, float eps, int32_t block,
                                         int32_t step, int32_t mode, const float* mass_prev, const float* theta,
                                         ra_gate_state* state, float* d_out, int32_t* decision_out,
                                         float* score_out, void* stream);

/*
 * refadapt_cache_commit - refresh a block's cached reference state.
 *
 * Copies k_ref -> k_cache, v_ref -> v_cache and q_ref -> q_cache
 * ([B, H, n_ref, d]) when `decision` is NULL or *decision == RA_COMPUTE, and
 * then writes `step` to *age when age is non-NULL (Alg. 1: a computing block
 * updates its cached K/V and sets its materialisation step a_b; the cached
 * queries are those of the same state, read again at a later boundary). Otherwise
 * nothing is written. K is required; each of the V and Q pairs is copied when
 * both of its tensors have non-NULL data and skipped when both are NULL (e.g.
 * K alone for the target Q kept as the block's materialisation anchor). All
 * pairs are copied by one launch.
 * Errors: RA_EINVAL (null K tensors, a V or Q pair with one NULL side, sizes),
 * RA_EUNSUPPORTED (alignment).
 */
ra_status refadapt_cache_commit(int32_t batch, int32_t heads, int32_t n_ref, int32_t head_dim, int32_t dtype,
                                ra_tensor k_ref, ra_tensor v_ref, ra_tensor q_ref, ra_tensor k_cache,
                                ra_tensor v_cache, ra_tensor q_cache, const int32_t* decision, int32_t* age,
                                int32_t step, void* stream);

/* ---- Diagnostics sidecar --------------------------------------------------
 *
 * Read-only probes of the controlled path (paper App. "probe non-intrusiveness":
 * enabling them leaves every output of the path bitwise unchanged). Each call
 * reads its inputs, writes only its own outputs and workspace, and enqueues on
 * `stream` without synchronising. Sums are fp32 within a workgroup and fp64
 * across workgroups and for the final ratios, in a fixed order, so results are
 * bitwise reproducible. Tensors follow the ra_tensor rules of refadapt_q_change
 * (16-byte aligned base, strides in whole 16-byte units, d contiguous).
 * Workspaces need no initialisation and must be 8-byte aligned.
 */

/*
 * refadapt_kv_drift - relative change of a reference K/V pair against a base.
 *
 *   d_k[b, h]  = ||K_cur[b,h] - K_base[b,h]||_F / (||K_base[b,h]||_F + eps)
 *   d_v[b, h]  = the same for V
 *   e_kv[b, h] = (d_k[b, h] + d_v[b, h]) / 2
 * over the n_rows x head_dim slice of each (b, h). With K_base/V_base the
 * cached (anchor) reference K/V this is the endpoint drift D_{t|a} of Sec. 3.3
 * (endpoint-drift equation) and e_kv its joint K/V scalar E^KV (the mean of the
 * two head-resolved drifts); with the previous step's K/V it is the consecutive
 * drift of Sec. 3.1. d_k and d_v may be NULL; e_kv is required. Outputs are
 * [B, H] contiguous fp32. One launch pair covers both tensors.
 * Errors: RA_EINVAL (sizes, dtype, eps, null tensors or e_kv), RA_EUNSUPPORTED
 * (head_dim, alignment), RA_EWORKSPACE (workspace NULL or smaller than
 * refadapt_kv_drift_workspace_size).
 */
size_t refadapt_kv_drift_workspace_size(int32_t batch, int32_t heads, int32_t n_rows, int32_t head_dim);
ra_status refadapt_kv_drift(int32_t batch, int32_t heads, int32_t n_rows, int32_t head_dim, int32_t dtype,
                            ra_tensor k_cur, ra_tensor k_base, ra_tensor v_cur, ra_tensor v_base, float eps,
                            float* d_k, float* d_v, float* e_kv, void* workspace, size_t ws_bytes, void* stream);

/*
 * refadapt_drift_log_ratio - matched reference/target drift log-ratio.
 *
 *   d_ref[b, h] = ||Z_ref_cur - Z_ref_prev||_F / (||Z_ref_prev||_F + eps)   (n_ref rows)
 *   d_tgt[b, h] = ||Z_tgt_cur - Z_tgt_prev||_F / (||Z_tgt_prev||_F + eps)   (n_tgt rows)
 *   rho[b, h]   = log10((d_ref + eps) / (d_tgt + eps))
 * for one tensor Z of K or V at adjacent steps (Sec. 3.1 consecutive-drift and
 * drift-log-ratio equations): rho < 0 means the reference slice moves more
 * slowly than the target slice. d_ref and d_tgt may be NULL; rho is required.
 * With eps == 0 a zero drift gives an infinite or NaN rho (IEEE division).
 * Errors: as refadapt_kv_drift, with refadapt_drift_log_ratio_workspace_size.
 */
size_t refadapt_drift_log_ratio_workspace_size(int32_t batch, int32_t heads, int32_t n_ref, int32_t n_tgt,
                                               int32_t head_dim);
ra_status refadapt_drift_log_ratio(int32_t batch, int32_t heads, int32_t n_ref, int32_t n_tgt, int32_t head_dim,
                                   int32_t dtype, ra_tensor z_ref_cur, ra_tensor z_ref_prev, ra_tensor z_tgt_cur,
                                   ra_tensor z_tgt_prev, float eps, float* d_ref, float* d_tgt, float* rho,
                                   void* workspace, size_t ws_bytes, void* stream);

/*
 * refadapt_output_impact - local perturbation of a stale-K/V attention output.
 *
 *   impact[b, h] = ||O_stale[b,h] - O_fresh[b,h]||_F / (||O_fresh[b,h]||_F + eps)
 * over the n_rows x head_dim slice (Sec. 3.3 local-impact equation, I^KV):
 * O_stale is the target output over cached reference K/V (refadapt_joint_attn
 * with RA_KV_CACHE, or the executed output of a reused block), O_fresh the
 * target output over fresh K/V. Both outputs are read once, in one pass.
 * impact is [B, H] contiguous fp32.
 * Errors: as refadapt_kv_drift, with refadapt_output_impact_workspace_size.
 */
size_t refadapt_output_impact_workspace_size(int32_t batch, int32_t heads, int32_t n_rows, int32_t head_dim);
ra_status refadapt_output_impact(int32_t batch, int32_t heads, int32_t n_rows, int32_t head_dim, int32_t dtype,
                                 ra_tensor o_stale, ra_tensor o_fresh, float eps, float* impact, void* workspace,
                                 size_t ws_bytes, void* stream);

/*
 * refadapt_mass_mean - head-resolved mean of per-query reference mass.
 *
 *   out[b, h] = mean over r < n_rows of mass[b, h, r]          (complement == 0)
 *   out[b, h] = mean over r < n_rows of (1 - mass[b, h, r])    (complement == 1)
 * with mass [B, H, n_rows] contiguous fp32 as written by refadapt_joint_attn.
 * From ref_mass (target queries) this is the head exposure M_{t,b,h} of
 * Sec. 3.2 (directional-exposure equation); from a REUSE launch's ref_mass it is
 * the same-step cached exposure M^cached of App. A.2; complement = 1 over
 * ref_mass_refq (reference queries) gives the reference-query mass on target
 * keys (App. directional attention diagnostics). out is [B, H] fp32.
 * Errors: RA_EINVAL (sizes, null pointers, complement not 0 or 1).
 */
ra_status refadapt_mass_mean(int32_t batch, int32_t heads, int32_t n_rows, const float* mass, int32_t complement,
                             float* out, void* stream);

/*
 * refadapt_adjacent_mass_change - mean adjacent-step change of head-mean mass.
 *
 * With mass_mean [n_steps, n_blocks, bh] contiguous fp32 (per step and block,
 * the bh values M_{t,b,(b',h)} of refadapt_mass_mean) and Mbar_{t,b} their mean
 * over bh, writes per block
 *   out[b] = 100 / (n_steps - 1) * sum_{t >= 1} |Mbar_{t,b} - Mbar_{t-1,b}|
 * in percentage points (Sec. 3.2 adjacent-ref-change equation).
 * Errors: RA_EINVAL (n_steps < 2, n_blocks or bh < 1, null pointers).
 */
ra_status refadapt_adjacent_mass_change(int32_t n_steps, int32_t n_blocks, int32_t bh, const float* mass_mean,
                                        float* out, void* stream);

/* ---- measurement probe (not part of the method) ----
 *
 * refadapt_mfma_rate_probe: the bf16 matrix-core rate this device sustains with every
 * operand in registers (no LDS, no global loads, no barrier), an upper bound on the joint
 * attention's rate at the clock the device holds under that load. kind 0
 * (RA_PROBE_DENSE): 32 back-to-back 32x32x16 bf16 MFMAs per step; kind 1 (RA_PROBE_MIX):
 * per step the attention's register work of one 64-key tile, 16 score MFMAs and 16
 * output MFMAs with 16 pairs of probabilities (scale, exp2, row-sum add, bf16 pack) formed
 * under them. `workgroups` workgroups of 512 threads (one per CU fills the device) each
 * run `steps` steps: workgroups x 8 x steps x 32 MFMAs of 32768 FLOP.
 *   operands     device, >= RA_PROBE_OPERAND_BYTES bytes of bf16 values, read once (their
 *                bit patterns set the matrix core's switching power: pass data like the
 *                attention's, e.g. standard normal)
 *   sink         device fp32 [workgroups * 512], written (keeps the work observable)
 *   clock_probe  device uint64[2] or NULL: thread 0 of each workgroup adds its shader
 *                cycles and 100 MHz reference ticks (as ra_attn_args.clock_probe)
 * Errors: RA_EINVAL (kind not 0 or 1, workgroups or steps < 1, null operands or sink),
 *         RA_EUNSUPPORTED (operands not 16-byte aligned).
 */
#define RA_PROBE_OPERAND_BYTES 65536
enum { RA_PROBE_DENSE = 0, RA_PROBE_MIX = 1 };
ra_status refadapt_mfma_rate_probe(int32_t kind, int32_t workgroups, int32_t steps, const void* operands,
                                   float* sink, uint64_t* clock_probe, void* stream);

/* Message describing the calling thread's last non-OK status ("" if none). */
const char* refadapt_last_error(void);

/* Library version string. */
const char* refadapt_version(void);

#ifdef __cplusplus
}
#endif

#endif /* REFADAPT_H */
