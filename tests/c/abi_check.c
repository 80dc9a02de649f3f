/* Compiles include/pfc.h as C99 and calls the host-side entry points of
 * libpfc (sizes, capacity, status strings and argument checks), none of which
 * touches a GPU.  Exit status 0 when every check holds; otherwise the number
 * of the first failing check. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "pfc.h"

#define CHECK(n, cond)                                  \
  do {                                                  \
    if (!(cond)) {                                      \
      fprintf(stderr, "check %d failed: %s\n", n, #cond); \
      return n;                                         \
    }                                                   \
  } while (0)

int main(void) {
  size_t bytes = 0;
  int64_t cap = 0;
  int64_t labels_dummy = 0;

  /* Capacity of the 8M-class shard at r = 0.1: the budget (800,000). */
  CHECK(1, pfc_workspace_bytes(1024, 512, 8000000, 0.1, PFC_F16, &bytes, &cap) == PFC_OK);
  CHECK(2, cap == 800000 && bytes > (size_t)1024 * 800000 * 2);
  /* Positives above the budget: |S| may reach min(B, C). */
  CHECK(3, pfc_workspace_bytes(64, 128, 100, 0.01, PFC_F32, &bytes, &cap) == PFC_OK);
  CHECK(4, cap == 64);
  /* Argument checks. */
  CHECK(5, pfc_workspace_bytes(0, 128, 100, 0.1, PFC_F32, &bytes, &cap) == PFC_ERR_INVALID_ARG);
  CHECK(6, pfc_workspace_bytes(16, 12, 100, 0.1, PFC_F32, &bytes, &cap) == PFC_ERR_INVALID_ARG);
  CHECK(7, pfc_workspace_bytes(16, 128, 100, 1.5, PFC_F32, &bytes, &cap) == PFC_ERR_INVALID_ARG);
  CHECK(8, pfc_workspace_bytes(PFC_MAX_BATCH + 1, 128, 100000, 0.1, PFC_F32, &bytes, &cap) ==
               PFC_ERR_INVALID_ARG);
  CHECK(9, pfc_sample(NULL, 16, 1000, 0, 0.1, 0, NULL, 100, NULL, NULL, NULL, 0, NULL) ==
               PFC_ERR_INVALID_ARG);
  /* A workspace that is not 256-byte aligned is refused before any launch. */
  CHECK(10, pfc_sample(&labels_dummy, 16, 1000, 0, 0.1, 0, (int32_t*)0x1000, 100,
                       (int32_t*)0x1000, (int32_t*)0x1000, (void*)0x1010, (size_t)1 << 40,
                       NULL) == PFC_ERR_WORKSPACE);
  /* Status strings. */
  CHECK(11, strlen(pfc_status_string(PFC_OK)) > 0);
  CHECK(12, strcmp(pfc_status_string(99), "unknown status") == 0);
  printf("abi_check ok\n");
  return 0;
}
