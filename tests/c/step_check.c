/* Two training steps of one class shard driven from C through libpfc's C
 * ABI, with device memory from hipMalloc and no other runtime: sampling
 * (Sec. 3.3.1-3.3.2), forward loss (Sec. 3.1) and backward + momentum
 * update (Sec. 3.2.1) in bf16.  Checks properties that hold whatever the
 * exact values are: status codes, the size and order of the active set, the
 * label remap, finite loss and feature gradient, rows outside both active
 * sets untouched bit for bit and rows inside them changed.  (Element-wise
 * agreement with the CPU oracle is checked by the Python parity tests.)
 * Exit status 0 on success, else the number of the failing check; 77 when
 * no GPU is present. */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "pfc.h"

#define CHECK(n, cond)                                       \
  do {                                                       \
    if (!(cond)) {                                           \
      fprintf(stderr, "check %d failed: %s\n", n, #cond);    \
      return n;                                              \
    }                                                        \
  } while (0)
#define HIPOK(n, call) CHECK(n, (call) == hipSuccess)

enum { B = 64, D = 128, C = 5000, OFFSET = 100, STEPS = 2 };
static const double R = 0.1;

/* xorshift64* uniform in [-1, 1) */
static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static double uniform(void) {
  rng_state ^= rng_state >> 12;
  rng_state ^= rng_state << 25;
  rng_state ^= rng_state >> 27;
  return (double)((rng_state * 2685821657736338717ull) >> 11) * (2.0 / 9007199254740992.0) - 1.0;
}

/* float -> bf16, round to nearest even (finite inputs) */
static uint16_t to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static int cmp_i32(const void* a, const void* b) {
  const int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
  return (x > y) - (x < y);
}

int main(void) {
  int n_dev = 0;
  if (hipGetDeviceCount(&n_dev) != hipSuccess || n_dev < 1) {
    fprintf(stderr, "no GPU\n");
    return 77;
  }
  size_t ws_bytes = 0;
  int64_t cap = 0;
  CHECK(1, pfc_workspace_bytes(B, D, C, R, PFC_BF16, &ws_bytes, &cap) == PFC_OK);

  uint16_t* hX = malloc(sizeof(uint16_t) * B * D);
  uint16_t* hW0 = malloc(sizeof(uint16_t) * C * D);
  uint16_t* hW1 = malloc(sizeof(uint16_t) * C * D);
  float* hM1 = malloc(sizeof(float) * C * D);
  float* hdX = malloc(sizeof(float) * B * D);
  int64_t* hL = malloc(sizeof(int64_t) * B);
  int32_t* hA = malloc(sizeof(int32_t) * cap);
  int32_t* hY = malloc(sizeof(int32_t) * B);
  unsigned char* touched = calloc(C, 1);
  CHECK(2, hX && hW0 && hW1 && hM1 && hdX && hL && hA && hY && touched);
  for (int i = 0; i < B * D; ++i) hX[i] = to_bf16((float)uniform());
  for (int i = 0; i < C * D; ++i) hW0[i] = to_bf16((float)(0.01 * uniform()));

  void *X, *W, *ws;
  float *M, *loss, *lse, *dX;
  int64_t* labels;
  int32_t *active, *n_active, *mapped;
  hipStream_t stream;
  HIPOK(3, hipStreamCreate(&stream));
  HIPOK(4, hipMalloc(&X, sizeof(uint16_t) * B * D));
  HIPOK(5, hipMalloc(&W, sizeof(uint16_t) * C * D));
  HIPOK(6, hipMalloc((void**)&M, sizeof(float) * C * D));
  HIPOK(7, hipMalloc(&ws, ws_bytes));
  HIPOK(8, hipMalloc((void**)&loss, sizeof(float)));
  HIPOK(9, hipMalloc((void**)&lse, sizeof(float) * B));
  HIPOK(10, hipMalloc((void**)&dX, sizeof(float) * B * D));
  HIPOK(11, hipMalloc((void**)&labels, sizeof(int64_t) * B));
  HIPOK(12, hipMalloc((void**)&active, sizeof(int32_t) * cap));
  HIPOK(13, hipMalloc((void**)&n_active, sizeof(int32_t)));
  HIPOK(14, hipMalloc((void**)&mapped, sizeof(int32_t) * B));
  HIPOK(15, hipMemcpy(X, hX, sizeof(uint16_t) * B * D, hipMemcpyHostToDevice));
  HIPOK(16, hipMemcpy(W, hW0, sizeof(uint16_t) * C * D, hipMemcpyHostToDevice));
  HIPOK(17, hipMemset(M, 0, sizeof(float) * C * D));

  for (int t = 0; t < STEPS; ++t) {
    /* Labels: mostly in the shard, a few outside it. */
    for (int n = 0; n < B; ++n) {
      const double u = 0.5 * (uniform() + 1.0);
      hL[n] = (n % 16 == 15) ? (int64_t)(OFFSET + C + 7 * n) : (int64_t)(OFFSET + u * C);
      if (hL[n] >= OFFSET + C && n % 16 != 15) hL[n] = OFFSET + C - 1;
    }
    HIPOK(20, hipMemcpy(labels, hL, sizeof(int64_t) * B, hipMemcpyHostToDevice));
    CHECK(21, pfc_sample(labels, B, C, OFFSET, R, (uint64_t)t, active, cap, n_active, mapped,
                         ws, ws_bytes, stream) == PFC_OK);
    CHECK(22, pfc_forward_loss(X, PFC_BF16, B, D, W, PFC_BF16, C, active, n_active, cap, mapped,
                               PFC_BF16, 64.0f, 0.5f, PFC_ARCFACE, 2.0f, loss, lse, ws, ws_bytes,
                               stream) == PFC_OK);
    CHECK(23, pfc_backward_update(X, PFC_BF16, B, D, W, PFC_BF16, NULL, M, C, active, n_active,
                                  cap, mapped, PFC_BF16, 64.0f, 0.5f, PFC_ARCFACE, lse, 0.1f,
                                  0.9f, dX, ws, ws_bytes, stream) == PFC_OK);
    HIPOK(24, hipStreamSynchronize(stream));

    int32_t k = 0;
    float hloss = 0.0f;
    HIPOK(25, hipMemcpy(&k, n_active, sizeof(int32_t), hipMemcpyDeviceToHost));
    HIPOK(26, hipMemcpy(&hloss, loss, sizeof(float), hipMemcpyDeviceToHost));
    HIPOK(27, hipMemcpy(hA, active, sizeof(int32_t) * cap, hipMemcpyDeviceToHost));
    HIPOK(28, hipMemcpy(hY, mapped, sizeof(int32_t) * B, hipMemcpyDeviceToHost));
    HIPOK(29, hipMemcpy(hdX, dX, sizeof(float) * B * D, hipMemcpyDeviceToHost));

    /* |S| = max(b, |P|) with b = r C = 500; distinct owned labels here are < 500. */
    int32_t pos[B];
    int np = 0;
    for (int n = 0; n < B; ++n)
      if (hL[n] >= OFFSET && hL[n] < OFFSET + C) pos[np++] = (int32_t)(hL[n] - OFFSET);
    qsort(pos, (size_t)np, sizeof(int32_t), cmp_i32);
    int n_distinct = 0;
    for (int i = 0; i < np; ++i)
      if (i == 0 || pos[i] != pos[i - 1]) ++n_distinct;
    CHECK(30, k == (n_distinct > 500 ? n_distinct : 500) && k <= cap);
    for (int j = 0; j < k; ++j) {
      CHECK(31, hA[j] >= 0 && hA[j] < C);
      CHECK(32, j == 0 || hA[j] > hA[j - 1]);
      touched[hA[j]] = 1;
    }
    for (int n = 0; n < B; ++n) {
      if (hL[n] >= OFFSET && hL[n] < OFFSET + C) {
        CHECK(33, hY[n] >= 0 && hY[n] < k && hA[hY[n]] == (int32_t)(hL[n] - OFFSET));
      } else {
        CHECK(34, hY[n] == -1);
      }
    }
    CHECK(35, isfinite(hloss) && hloss > 0.0f);
    for (int i = 0; i < B * D; ++i) CHECK(36, isfinite(hdX[i]));
    printf("step %d: |S| = %d, loss = %.6f\n", t, k, hloss);
  }

  HIPOK(40, hipMemcpy(hW1, W, sizeof(uint16_t) * C * D, hipMemcpyDeviceToHost));
  HIPOK(41, hipMemcpy(hM1, M, sizeof(float) * C * D, hipMemcpyDeviceToHost));
  int n_changed = 0, n_touched = 0;
  for (int c = 0; c < C; ++c) {
    const int same_w = memcmp(hW1 + (size_t)c * D, hW0 + (size_t)c * D, sizeof(uint16_t) * D) == 0;
    int zero_m = 1;
    for (int i = 0; i < D; ++i) zero_m &= hM1[(size_t)c * D + i] == 0.0f;
    if (!touched[c]) {
      CHECK(42, same_w && zero_m);   /* rows outside both active sets are untouched */
    } else {
      ++n_touched;
      n_changed += !zero_m;
    }
  }
  CHECK(43, n_touched > 0 && n_changed == n_touched);   /* every active row got momentum */
  printf("step_check ok: %d rows updated, %d untouched\n", n_touched, C - n_touched);
  hipFree(X);
  hipFree(W);
  hipFree(M);
  hipFree(ws);
  hipFree(loss);
  hipFree(lse);
  hipFree(dX);
  hipFree(labels);
  hipFree(active);
  hipFree(n_active);
  hipFree(mapped);
  hipStreamDestroy(stream);
  return 0;
}
