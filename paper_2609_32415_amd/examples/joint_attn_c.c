/*
 * joint_attn_c.c - calling the refadapt C ABI from plain C (no Python, no torch).
 *
 * Builds seeded bf16 Q/K/V for a small [reference; target] problem on the host, runs
 * refadapt_joint_attn on the current HIP device with all queries over the fresh
 * reference K/V (per-query reference mass, log-sum-exp pair, key-split workspace), and
 * writes the inputs and outputs to a binary file:
 *
 *   "RAC1", int32 batch, heads, head_dim, n_ref, n_tgt,
 *   bf16 q_tgt, k_tgt, v_tgt [B, H, n_tgt, d], q_ref, k_ref, v_ref [B, H, n_ref, d],
 *   bf16 o_tgt [B, H, n_tgt, d], o_ref [B, H, n_ref, d],
 *   fp32 ref_mass [B, H, n_tgt], lse [B, H, n_tgt, 2]
 *
 * (all contiguous, little-endian). Usage: joint_attn_c OUTPUT_FILE. Exit status 0 on
 * success; a failing call prints refadapt_last_error() and exits non-zero.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "refadapt.h"

enum { B = 1, H = 3, D = 128, N_REF = 300, N_TGT = 333 };

#define HIP_OK(call)                                                                    \
  do {                                                                                  \
    hipError_t e_ = (call);                                                             \
    if (e_ != hipSuccess) {                                                             \
      fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));                 \
      exit(2);                                                                          \
    }                                                                                   \
  } while (0)

/* xorshift64* stream and Box-Muller normals: the inputs only need to be seeded. */
static uint64_t rng = 0x9E3779B97F4A7C15ull;
static double uniform01(void) {
  rng ^= rng >> 12;
  rng ^= rng << 25;
  rng ^= rng >> 27;
  return ((rng * 0x2545F4914F6CDD1Dull) >> 11) * (1.0 / 9007199254740992.0);
}
static float normal(void) {
  const double u1 = uniform01() + 1e-300, u2 = uniform01();
  return (float)(sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2));
}
static uint16_t to_bf16(float f) { /* round to nearest even */
  uint32_t u;
  memcpy(&u, &f, 4);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

/* A contiguous [B, H, rows, D] bf16 tensor: host copy, device copy and its ra_tensor view. */
typedef struct {
  size_t n;
  uint16_t* host;
  void* dev;
  ra_tensor view;
} tensor;

static tensor make(int rows, int fill, float scale) {
  tensor t;
  t.n = (size_t)B * H * rows * D;
  t.host = (uint16_t*)calloc(t.n ? t.n : 1, 2);
  if (!t.host) exit(3);
  if (fill)
    for (size_t i = 0; i < t.n; ++i) t.host[i] = to_bf16(scale * normal());
  HIP_OK(hipMalloc(&t.dev, t.n * 2));
  HIP_OK(hipMemcpy(t.dev, t.host, t.n * 2, hipMemcpyHostToDevice));
  t.view.data = t.dev;
  t.view.stride_b = (int64_t)H * rows * D;
  t.view.stride_h = (int64_t)rows * D;
  t.view.stride_s = D;
  return t;
}

int main(int argc, char** argv) {
  if (argc != 2) {
    fprintf(stderr, "usage: %s OUTPUT_FILE\n", argv[0]);
    return 1;
  }
  printf("%s: joint attention B %d H %d d %d n_ref %d n_tgt %d\n", refadapt_version(), B, H, D, N_REF, N_TGT);
  tensor q_tgt = make(N_TGT, 1, 1.0f), k_tgt = make(N_TGT, 1, 1.0f), v_tgt = make(N_TGT, 1, 1.0f);
  tensor q_ref = make(N_REF, 1, 1.0f), k_ref = make(N_REF, 1, 1.0f), v_ref = make(N_REF, 1, 1.0f);
  tensor o_tgt = make(N_TGT, 0, 0.f), o_ref = make(N_REF, 0, 0.f);
  float *mass, *lse;
  HIP_OK(hipMalloc((void**)&mass, sizeof(float) * B * H * N_TGT));
  HIP_OK(hipMalloc((void**)&lse, sizeof(float) * B * H * N_TGT * 2));

  ra_attn_desc desc = {B, H, D, N_REF, N_TGT, RA_BF16, 0.0f, RA_Q_ALL, RA_KV_FRESH};
  ra_attn_args args;
  memset(&args, 0, sizeof args);
  args.q_tgt = q_tgt.view;
  args.k_tgt = k_tgt.view;
  args.v_tgt = v_tgt.view;
  args.q_ref = q_ref.view;
  args.k_ref = k_ref.view;
  args.v_ref = v_ref.view;
  args.o_tgt = o_tgt.view;
  args.o_ref = o_ref.view;
  args.ref_mass = mass;
  args.lse_tgt = lse;
  args.workspace_bytes = refadapt_joint_attn_workspace_size(&desc);
  if (args.workspace_bytes > 0) HIP_OK(hipMalloc(&args.workspace, args.workspace_bytes));
  printf("key-split workspace: %zu bytes\n", args.workspace_bytes);

  hipStream_t stream;
  HIP_OK(hipStreamCreate(&stream));
  const ra_status s = refadapt_joint_attn(&desc, &args, stream);
  if (s != RA_OK) {
    fprintf(stderr, "refadapt_joint_attn: status %d: %s\n", (int)s, refadapt_last_error());
    return 4;
  }
  HIP_OK(hipStreamSynchronize(stream));

  float* h_mass = (float*)malloc(sizeof(float) * B * H * N_TGT);
  float* h_lse = (float*)malloc(sizeof(float) * B * H * N_TGT * 2);
  if (!h_mass || !h_lse) return 3;
  HIP_OK(hipMemcpy(o_tgt.host, o_tgt.dev, o_tgt.n * 2, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(o_ref.host, o_ref.dev, o_ref.n * 2, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(h_mass, mass, sizeof(float) * B * H * N_TGT, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(h_lse, lse, sizeof(float) * B * H * N_TGT * 2, hipMemcpyDeviceToHost));

  FILE* f = fopen(argv[1], "wb");
  if (!f) {
    perror(argv[1]);
    return 5;
  }
  const int32_t dims[5] = {B, H, D, N_REF, N_TGT};
  fwrite("RAC1", 1, 4, f);
  fwrite(dims, sizeof dims, 1, f);
  const tensor* order[8] = {&q_tgt, &k_tgt, &v_tgt, &q_ref, &k_ref, &v_ref, &o_tgt, &o_ref};
  for (int i = 0; i < 8; ++i) fwrite(order[i]->host, 2, order[i]->n, f);
  fwrite(h_mass, sizeof(float), (size_t)B * H * N_TGT, f);
  fwrite(h_lse, sizeof(float), (size_t)B * H * N_TGT * 2, f);
  if (fclose(f) != 0) return 5;

  const tensor* all[8] = {&q_tgt, &k_tgt, &v_tgt, &q_ref, &k_ref, &v_ref, &o_tgt, &o_ref};
  for (int i = 0; i < 8; ++i) {
    HIP_OK(hipFree(all[i]->dev));
    free(all[i]->host);
  }
  HIP_OK(hipFree(mass));
  HIP_OK(hipFree(lse));
  if (args.workspace) HIP_OK(hipFree(args.workspace));
  HIP_OK(hipStreamDestroy(stream));
  free(h_mass);
  free(h_lse);
  printf("wrote %s\n", argv[1]);
  return 0;
}
