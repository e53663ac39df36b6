/* A plain C99 client of libestp.
 *
 * Without arguments it checks what needs no GPU: estp.h compiles as C, the
 * exports link, and host-side validation rejects bad arguments with a status
 * and a message before any device work.  With --gpu it allocates device
 * memory through the HIP runtime and runs two closed forms through the
 * library, for both input types:
 *   - W = 0 makes every logit 0, so each token's next-token distribution is
 *     uniform and its entropy is ln V (Eq. 2); all V logits tie, so the mode
 *     (vocab_argmax) is index 0, the lowest;
 *   - K = 0 makes every score 0, so the causal attention of query i is 1/(i+1)
 *     on keys 0..i and the importance of key j in a prompt of N tokens is
 *     S_j = (H_N - H_j) / N with harmonic numbers H_n = sum_{k=1..n} 1/k (Eq. 1).
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "estp.h"

static int fail(const char* what) {
  fprintf(stderr, "FAIL: %s (last error: %s)\n", what, estp_last_error());
  return 1;
}

static int host_checks(void) {
  size_t ws;
  if (estp_version() <= 0) return fail("estp_version");
  if (strlen(estp_status_string(ESTP_ERR_INVALID_ARG)) == 0) return fail("estp_status_string");
  ws = estp_token_entropy_workspace_size(100, 64, 1000, ESTP_BF16);
  if (ws == 0) return fail("estp_token_entropy_workspace_size");
  if (estp_token_entropy(NULL, NULL, 100, 64, 1000, ESTP_BF16, NULL, NULL, NULL, ws, NULL) != ESTP_ERR_INVALID_ARG)
    return fail("null inputs not rejected");
  if (estp_last_error()[0] == '\0') return fail("no error message");
  if (estp_attn_importance(NULL, NULL, NULL, 1, 1, 1, 1, 1, 1, 64, 0.125f, ESTP_BF16, NULL, NULL, 0, NULL) !=
      ESTP_ERR_INVALID_ARG)
    return fail("importance: null inputs not rejected");
  printf("host checks passed (libestp version %d)\n", estp_version());
  return 0;
}

#define HIP_OK(call)                                                    \
  do {                                                                  \
    if ((call) != hipSuccess) {                                         \
      fprintf(stderr, "FAIL: %s at line %d\n", #call, __LINE__);        \
      return 1;                                                         \
    }                                                                   \
  } while (0)

/* bf16 bit pattern of a float (round to nearest even; the values here are exact) */
static uint16_t to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

/* copy n floats to the device as `dtype` (fp32 or bf16) */
static int upload(void** dst, const float* src, size_t n, int dtype) {
  size_t i;
  if (dtype == ESTP_F32) {
    HIP_OK(hipMalloc(dst, n * sizeof(float)));
    HIP_OK(hipMemcpy(*dst, src, n * sizeof(float), hipMemcpyHostToDevice));
  } else {
    uint16_t* h = (uint16_t*)malloc(n * sizeof(uint16_t));
    if (!h) return 1;
    for (i = 0; i < n; ++i) h[i] = to_bf16(src[i]);
    HIP_OK(hipMalloc(dst, n * sizeof(uint16_t)));
    HIP_OK(hipMemcpy(*dst, h, n * sizeof(uint16_t), hipMemcpyHostToDevice));
    free(h);
  }
  return 0;
}

static int entropy_uniform(int dtype) {
  const int n = 300, d = 64, V = 1000;
  float* x = (float*)malloc((size_t)n * d * sizeof(float));
  float* w = (float*)calloc((size_t)V * d, sizeof(float));
  float* h = (float*)malloc((size_t)n * sizeof(float));
  void *X = NULL, *W = NULL, *ws = NULL;
  float* H = NULL;
  int32_t* A = NULL;
  int32_t* am = (int32_t*)malloc((size_t)n * sizeof(int32_t));
  size_t wsb, i;
  double err = 0.0;
  int n_bad = 0;
  if (!x || !w || !h || !am) return fail("host allocation");
  for (i = 0; i < (size_t)n * d; ++i) x[i] = (float)sin(0.37 * (double)i);
  if (upload(&X, x, (size_t)n * d, dtype) || upload(&W, w, (size_t)V * d, dtype)) return 1;
  HIP_OK(hipMalloc((void**)&H, (size_t)n * sizeof(float)));
  wsb = estp_token_entropy_workspace_size(n, d, V, dtype);
  HIP_OK(hipMalloc(&ws, wsb));
  if (estp_token_entropy(X, W, n, d, V, dtype, H, NULL, ws, wsb, NULL) != ESTP_OK) return fail("estp_token_entropy");
  HIP_OK(hipDeviceSynchronize());
  HIP_OK(hipMemcpy(h, H, (size_t)n * sizeof(float), hipMemcpyDeviceToHost));
  for (i = 0; i < (size_t)n; ++i) err = fmax(err, fabs((double)h[i] - log((double)V)));
  printf("entropy, uniform logits (%s): max |H - ln V| = %.3g\n", dtype == ESTP_F32 ? "f32" : "bf16", err);
  /* the same call with the mode: every logit ties, the lowest index wins */
  HIP_OK(hipMalloc((void**)&A, (size_t)n * sizeof(int32_t)));
  HIP_OK(hipMemset(A, 0xff, (size_t)n * sizeof(int32_t)));
  if (estp_token_entropy(X, W, n, d, V, dtype, H, A, ws, wsb, NULL) != ESTP_OK) return fail("estp_token_entropy (mode)");
  HIP_OK(hipDeviceSynchronize());
  HIP_OK(hipMemcpy(am, A, (size_t)n * sizeof(int32_t), hipMemcpyDeviceToHost));
  for (i = 0; i < (size_t)n; ++i) n_bad += am[i] != 0;
  printf("next-token mode, all logits tied (%s): %d of %d rows not index 0\n", dtype == ESTP_F32 ? "f32" : "bf16",
         n_bad, n);
  HIP_OK(hipFree(A));
  free(am);
  if (n_bad) return fail("tied-logit mode");
  HIP_OK(hipFree(X));
  HIP_OK(hipFree(W));
  HIP_OK(hipFree(H));
  HIP_OK(hipFree(ws));
  free(x);
  free(w);
  free(h);
  return err <= 1e-4 ? 0 : fail("uniform-logit entropy");
}

static int importance_uniform(int dtype) {
  enum { B = 3, L = 1, HQ = 4, HKV = 2, DH = 64 };
  const int lens[B] = {1, 37, 300};
  int cu[B + 1], b, j, max_len = 0;
  size_t n, i, wsb;
  float *q, *k, *s;
  void *Q = NULL, *K = NULL, *ws = NULL;
  int32_t* CU = NULL;
  float* S = NULL;
  double err = 0.0;
  cu[0] = 0;
  for (b = 0; b < B; ++b) {
    cu[b + 1] = cu[b] + lens[b];
    if (lens[b] > max_len) max_len = lens[b];
  }
  n = (size_t)cu[B];
  q = (float*)malloc(n * HQ * DH * sizeof(float));
  k = (float*)calloc(n * HKV * DH, sizeof(float));
  s = (float*)malloc(n * sizeof(float));
  if (!q || !k || !s) return fail("host allocation");
  for (i = 0; i < n * HQ * DH; ++i) q[i] = (float)cos(0.11 * (double)i);
  if (upload(&Q, q, n * HQ * DH, dtype) || upload(&K, k, n * HKV * DH, dtype)) return 1;
  HIP_OK(hipMalloc((void**)&CU, sizeof cu));
  HIP_OK(hipMemcpy(CU, cu, sizeof cu, hipMemcpyHostToDevice));
  HIP_OK(hipMalloc((void**)&S, n * sizeof(float)));
  wsb = estp_attn_importance_workspace_size((int64_t)n, B, max_len, L, HQ, HKV, DH, dtype);
  HIP_OK(hipMalloc(&ws, wsb));
  if (estp_attn_importance(Q, K, CU, B, max_len, (int64_t)n, L, HQ, HKV, DH, 0.125f, dtype, S, ws, wsb, NULL) !=
      ESTP_OK)
    return fail("estp_attn_importance");
  HIP_OK(hipDeviceSynchronize());
  HIP_OK(hipMemcpy(s, S, n * sizeof(float), hipMemcpyDeviceToHost));
  for (b = 0; b < B; ++b) {
    const int N = lens[b];
    double tail = 0.0; /* H_N - H_j, built from j = N - 1 down */
    for (j = N - 1; j >= 0; --j) {
      double ref;
      tail += 1.0 / (double)(j + 1);
      ref = tail / (double)N;
      err = fmax(err, fabs((double)s[cu[b] + j] - ref) / ref);
    }
  }
  printf("importance, zero keys (%s): max relative |S - (H_N - H_j)/N| = %.3g\n", dtype == ESTP_F32 ? "f32" : "bf16",
         err);
  HIP_OK(hipFree(Q));
  HIP_OK(hipFree(K));
  HIP_OK(hipFree(CU));
  HIP_OK(hipFree(S));
  HIP_OK(hipFree(ws));
  free(q);
  free(k);
  free(s);
  return err <= 1e-4 ? 0 : fail("uniform-attention importance");
}

int main(int argc, char** argv) {
  if (host_checks()) return 1;
  if (argc > 1 && strcmp(argv[1], "--gpu") == 0) {
    if (entropy_uniform(ESTP_F32) || entropy_uniform(ESTP_BF16)) return 1;
    if (importance_uniform(ESTP_F32) || importance_uniform(ESTP_BF16)) return 1;
    printf("gpu checks passed\n");
  }
  return 0;
}
