/*
 * The C ABI from plain C (C99, no C++ and no Python): every entry point that
 * needs no GPU.  Built and run by tests/test_c_abi.py:
 *   c_abi_host q0 q1 q2 p      (three NTT primes for N = 256 and one more)
 * Prints "ok" and returns 0, or names the first failed check and returns 1.
 */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "fiona.h"

#define CHECK(c)                                                  \
  do {                                                            \
    if (!(c)) {                                                   \
      printf("FAIL line %d: %s\n", __LINE__, #c);                 \
      return 1;                                                   \
    }                                                             \
  } while (0)

/* Two inputs, two outputs.  Output 0: one raw term (input 0, plaintext 0)
 * and the group {+A0, -A1} with scale 0.  Output 1: the group {-A0, +A1}
 * (the same sum reversed) with scale 1, and a sign-0 member of input 1. */
static const uint32_t pm_off[3] = {0, 1, 1}, pm_input[1] = {0}, pm_pt[1] = {0};
static const uint32_t grp_off[3] = {0, 1, 2}, grp_mem_off[3] = {0, 2, 5};
static const uint32_t mem_input[5] = {0, 1, 0, 1, 1}, grp_scale[2] = {0, 1};
static const int8_t mem_sign[5] = {1, -1, -1, 1, 0};

static fiona_layer_desc layer(uint32_t flags) {
  fiona_layer_desc d;
  memset(&d, 0, sizeof d);
  d.n_in = 2;
  d.n_out = 2;
  d.n_pt = 1;
  d.n_scale = 2;
  d.pm_off = pm_off;
  d.pm_input = pm_input;
  d.pm_pt = pm_pt;
  d.grp_off = grp_off;
  d.grp_mem_off = grp_mem_off;
  d.mem_input = mem_input;
  d.mem_sign = mem_sign;
  d.grp_scale = grp_scale;
  d.flags = flags;
  return d;
}

int main(int argc, char **argv) {
  if (argc != 5) {
    printf("usage: %s q0 q1 q2 p\n", argv[0]);
    return 2;
  }
  uint64_t q[4];
  for (int i = 0; i < 4; ++i) q[i] = strtoull(argv[i + 1], NULL, 10);

  /* context */
  fiona_ctx *ctx = NULL, *none = NULL;
  CHECK(fiona_ctx_create(256, 3, q, &ctx) == FIONA_OK && ctx != NULL);
  CHECK(fiona_ctx_create(256, 3, NULL, &none) == FIONA_ERR_ARG);
  CHECK(fiona_ctx_create(0, 3, q, &none) != FIONA_OK);
  const uint64_t small[1] = {1u << 20};   /* not above 2^20 */
  CHECK(fiona_ctx_create(256, 1, small, &none) == FIONA_ERR_UNSUPPORTED);
  CHECK(fiona_pt_pitch_hint(ctx) >= 3u * 256u && fiona_pt_pitch_hint(NULL) == 0);

  /* a host-only checking plan: the reversed sum is shared */
  fiona_layer_desc d = layer(FIONA_PLAN_HOST_ONLY | FIONA_PLAN_CHECK_INPUTS);
  fiona_plan *plan = NULL;
  CHECK(fiona_plan_create(ctx, &d, &plan) == FIONA_OK && plan != NULL);
  fiona_plan_stats_t st;
  CHECK(fiona_plan_stats(plan, &st) == FIONA_OK);
  CHECK(st.ct_terms == 6 && st.n_pmult == 1 && st.n_member == 5 && st.n_member_nonzero == 4);
  CHECK(st.n_use == 2 && st.n_sum_distinct == 1 && st.pmult_per_contribution == 5 && st.pmult_grouped == 3);
  CHECK(st.input_passes == 1 && st.tile == 64 && st.grid == 3 * 4);
  CHECK(fiona_plan_stats(NULL, &st) == FIONA_ERR_ARG);

  /* without sharing the two sums are formed separately */
  fiona_layer_desc d2 = layer(FIONA_PLAN_HOST_ONLY | FIONA_PLAN_NO_SHARING);
  fiona_plan *plan2 = NULL;
  CHECK(fiona_plan_create(ctx, &d2, &plan2) == FIONA_OK);
  CHECK(fiona_plan_stats(plan2, &st) == FIONA_OK && st.n_sum_distinct == 2 && st.n_use == 2);

  /* the checking plan's preconditions on host arrays */
  const uint64_t scales[2] = {5, (1u << 20) - 1};
  const uint64_t big_scale[2] = {5, 1u << 20};
  int8_t flipped[5];
  memcpy(flipped, mem_sign, sizeof flipped);
  flipped[4] = 1;
  CHECK(fiona_plan_check_inputs(plan, mem_sign, scales, NULL, NULL) == FIONA_OK);
  CHECK(fiona_plan_check_inputs(plan, flipped, scales, NULL, NULL) == FIONA_ERR_PRECONDITION);
  CHECK(fiona_plan_check_inputs(plan, mem_sign, big_scale, NULL, NULL) == FIONA_ERR_PRECONDITION);
  CHECK(fiona_plan_check_inputs(plan2, mem_sign, scales, NULL, NULL) == FIONA_ERR_ARG);

  /* a host-only plan launches nothing */
  CHECK(fiona_hybrid_linear(plan, NULL, NULL, NULL, NULL, NULL, NULL) == FIONA_ERR_NODEVICE);
  CHECK(fiona_hybrid_linear_static(plan, NULL, NULL, NULL, NULL, NULL, NULL) == FIONA_ERR_NODEVICE);
  CHECK(fiona_hybrid_linear(NULL, NULL, NULL, NULL, NULL, NULL, NULL) == FIONA_ERR_ARG);

  /* inconsistent descriptions */
  fiona_layer_desc bad = layer(FIONA_PLAN_HOST_ONLY);
  bad.n_in = 1;   /* member input 1 out of range */
  fiona_plan *none_plan = NULL;
  CHECK(fiona_plan_create(ctx, &bad, &none_plan) == FIONA_ERR_PLAN && none_plan == NULL);
  bad = layer(FIONA_PLAN_HOST_ONLY);
  bad.pt_pitch = 3u * 256u - 1u;   /* below L*N */
  CHECK(fiona_plan_create(ctx, &bad, &none_plan) == FIONA_ERR_ARG);

  fiona_plan_destroy(plan2);
  fiona_plan_destroy(plan);
  fiona_plan_destroy(NULL);

  /* host replay of the NTT passes' accesses: in bounds, and an output one
   * word short is found */
  char msg[256];
  CHECK(fiona_check_ntt_offsets(0, 256, 3, q, 4, 4, 0, msg, sizeof msg) == FIONA_OK && msg[0] == 0);
  CHECK(fiona_check_ntt_offsets(0, 256, 3, q, 4, 4, 8, msg, sizeof msg) == FIONA_ERR_BOUNDS && msg[0] != 0);
  CHECK(fiona_check_ntt_offsets(1, 256, 3, q, 5, 5, 0, msg, sizeof msg) == FIONA_OK);

  /* status strings */
  for (int s = FIONA_ERR_BOUNDS; s <= FIONA_OK; ++s) CHECK(fiona_status_string(s) != NULL);
  CHECK(strcmp(fiona_status_string(FIONA_OK), fiona_status_string(FIONA_ERR_ARG)) != 0);
  CHECK(fiona_status_string(-1000) != NULL);

  fiona_ctx_destroy(ctx);
  fiona_ctx_destroy(NULL);
  printf("ok\n");
  return 0;
}
