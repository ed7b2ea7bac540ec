/*
 * A plain C client of libxattn (no Python, no torch): the library used the way
 * a C or C++ inference engine would use it, through include/xattn.h and the
 * HIP runtime only. On one GPU it
 *   1. runs the chained forward (score -> select -> sparse attention,
 *      Fig. 1) at tau = 1, which selects every causal block, and checks the
 *      output bitwise against the dense mode;
 *   2. runs it at tau = 0.9 and checks the selection it leaves in the
 *      workspace: every row's list non-empty, ascending, inside the causal
 *      candidates, and holding the diagonal block whenever its score is the
 *      row's largest;
 *   3. checks that an invalid shape is rejected before anything is enqueued,
 *      with a message.
 * Prints "c client ok" and exits 0 on success; any failure prints a reason
 * and exits 1. Built by the package's build step (tests/c_client.c ->
 * paper_2503_16428_amd/lib/xattn_c_client) and run by a GPU test.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "xattn.h"

#define CHECK_HIP(x)                                                              \
  do {                                                                            \
    hipError_t e_ = (x);                                                          \
    if (e_ != hipSuccess) {                                                       \
      fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));              \
      exit(1);                                                                    \
    }                                                                             \
  } while (0)

#define CHECK_X(x)                                                                \
  do {                                                                            \
    int s_ = (x);                                                                 \
    if (s_ != XATTN_OK) {                                                         \
      fprintf(stderr, "%s failed: %s (%s)\n", #x, xattn_strerror(s_),             \
              xattn_last_error());                                                \
      exit(1);                                                                    \
    }                                                                             \
  } while (0)

/* bf16 bit pattern of a float (round to nearest even; inputs are finite) */
static uint16_t to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* deterministic N(0, 1)-like values: sum of four uniforms from a 64-bit LCG */
static uint64_t lcg_state = 0x9E3779B97F4A7C15ull;
static float next_gauss(void) {
  float s = 0.f;
  for (int i = 0; i < 4; ++i) {
    lcg_state = lcg_state * 6364136223846793005ull + 1442695040888963407ull;
    s += (float)((lcg_state >> 40) & 0xFFFFFF) / 16777216.0f;
  }
  return (s - 2.0f) * 1.7320508f;
}

static void *upload(const uint16_t *h, size_t n) {
  void *d = NULL;
  CHECK_HIP(hipMalloc(&d, n * sizeof(uint16_t)));
  CHECK_HIP(hipMemcpy(d, h, n * sizeof(uint16_t), hipMemcpyHostToDevice));
  return d;
}

int main(void) {
  const int L = 2048, HQ = 4, HKV = 2, D = 128, B = 128, S = 8, NB = L / B;
  xattn_dims dims = {1, HQ, HKV, L, D, 1};
  const size_t nq = (size_t)HQ * L * D, nkv = (size_t)HKV * L * D;

  /* inputs: keys drawn around a few shared directions so that attention is
   * concentrated (a meaningful selection at tau = 0.9), values N(0, 1) */
  uint16_t *hq = malloc(nq * 2), *hk = malloc(nkv * 2), *hv = malloc(nkv * 2);
  float centre[8][128];
  for (int c = 0; c < 8; ++c)
    for (int e = 0; e < D; ++e) centre[c][e] = 2.0f * next_gauss();
  for (size_t r = 0; r < nkv / D; ++r) {
    const int c = (int)(r * 2654435761u % 8u);
    for (int e = 0; e < D; ++e) {
      hk[r * D + e] = to_bf16(centre[c][e] + next_gauss());
      hv[r * D + e] = to_bf16(next_gauss());
    }
  }
  for (size_t r = 0; r < nq / D; ++r) {
    const int c = (int)(r * 40503u % 8u);
    for (int e = 0; e < D; ++e) hq[r * D + e] = to_bf16(centre[c][e] + next_gauss());
  }
  void *q = upload(hq, nq), *k = upload(hk, nkv), *v = upload(hv, nkv);

  hipStream_t st;
  CHECK_HIP(hipStreamCreate(&st));
  size_t ws_bytes = 0, sc_off = 0, idx_off = 0, cnt_off = 0, scr_off = 0;
  CHECK_X(xattn_forward_workspace_size(&dims, B, S, &ws_bytes));
  CHECK_X(xattn_forward_layout(&dims, B, S, &sc_off, &idx_off, &cnt_off, &scr_off));
  void *ws = NULL, *o_fwd = NULL, *o_dense = NULL;
  CHECK_HIP(hipMalloc(&ws, ws_bytes));
  CHECK_HIP(hipMalloc(&o_fwd, nq * 2));
  CHECK_HIP(hipMalloc(&o_dense, nq * 2));

  /* 1. tau = 1: every causal block, bitwise the dense mode */
  CHECK_X(xattn_forward(q, k, v, &dims, B, S, 1.0f, o_fwd, NULL, ws, ws_bytes, st));
  CHECK_X(xattn_dense_attn(q, k, v, &dims, o_dense, NULL, st));
  CHECK_HIP(hipStreamSynchronize(st));
  uint16_t *a = malloc(nq * 2), *b = malloc(nq * 2);
  CHECK_HIP(hipMemcpy(a, o_fwd, nq * 2, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(b, o_dense, nq * 2, hipMemcpyDeviceToHost));
  if (memcmp(a, b, nq * 2) != 0) {
    fprintf(stderr, "forward at tau = 1 differs from the dense mode\n");
    return 1;
  }
  int32_t *hcnt = malloc((size_t)HQ * NB * 4);
  CHECK_HIP(hipMemcpy(hcnt, (char *)ws + cnt_off, (size_t)HQ * NB * 4, hipMemcpyDeviceToHost));
  for (int r = 0; r < HQ * NB; ++r)
    if (hcnt[r] != r % NB + 1) {
      fprintf(stderr, "tau = 1: row %d selected %d of %d blocks\n", r, hcnt[r], r % NB + 1);
      return 1;
    }

  /* 2. tau = 0.9: the lists left in the workspace */
  CHECK_X(xattn_forward(q, k, v, &dims, B, S, 0.9f, o_fwd, NULL, ws, ws_bytes, st));
  CHECK_HIP(hipStreamSynchronize(st));
  float *hsc = malloc((size_t)HQ * NB * NB * 4);
  int32_t *hidx = malloc((size_t)HQ * NB * NB * 4);
  CHECK_HIP(hipMemcpy(hsc, (char *)ws + sc_off, (size_t)HQ * NB * NB * 4, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(hidx, (char *)ws + idx_off, (size_t)HQ * NB * NB * 4, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(hcnt, (char *)ws + cnt_off, (size_t)HQ * NB * 4, hipMemcpyDeviceToHost));
  long selected = 0;
  for (int r = 0; r < HQ * NB; ++r) {
    const int bq = r % NB, c = hcnt[r];
    const int32_t *row = hidx + (size_t)r * NB;
    const float *srow = hsc + (size_t)r * NB;
    if (c < 1 || c > bq + 1) {
      fprintf(stderr, "row %d: count %d outside [1, %d]\n", r, c, bq + 1);
      return 1;
    }
    int argmax = 0;
    for (int j = 1; j <= bq; ++j)
      if (srow[j] > srow[argmax]) argmax = j;
    int has_argmax = 0;
    for (int i = 0; i < c; ++i) {
      if (row[i] < 0 || row[i] > bq || (i > 0 && row[i] <= row[i - 1])) {
        fprintf(stderr, "row %d: list not ascending inside the causal candidates\n", r);
        return 1;
      }
      has_argmax |= row[i] == argmax;
    }
    if (!has_argmax) {
      fprintf(stderr, "row %d: the highest-scoring block %d was not selected\n", r, argmax);
      return 1;
    }
    selected += c;
  }

  /* 3. a shape the library rejects before enqueueing anything */
  xattn_dims bad = dims;
  bad.seq = L + 64;
  const int rc = xattn_forward(q, k, v, &bad, B, S, 0.9f, o_fwd, NULL, ws, ws_bytes, st);
  if (rc == XATTN_OK || strlen(xattn_last_error()) == 0) {
    fprintf(stderr, "a sequence length of %d was accepted\n", bad.seq);
    return 1;
  }

  printf("c client ok: library version %d, workspace %zu bytes, density %.3f at tau 0.9, "
         "rejected seq %d with \"%s\"\n",
         xattn_version(), ws_bytes, (double)selected / (HQ * NB * (NB + 1) / 2), bad.seq,
         xattn_last_error());
  free(hq); free(hk); free(hv); free(a); free(b); free(hcnt); free(hsc); free(hidx);
  CHECK_HIP(hipFree(q)); CHECK_HIP(hipFree(k)); CHECK_HIP(hipFree(v));
  CHECK_HIP(hipFree(ws)); CHECK_HIP(hipFree(o_fwd)); CHECK_HIP(hipFree(o_dense));
  CHECK_HIP(hipStreamDestroy(st));
  return 0;
}
