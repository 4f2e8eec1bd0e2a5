/*
 * The hot path from plain C (C99, the HIP runtime's C API, no Python): a
 * seeded layer with raw terms, shared and reversed signed sums and sign-0
 * members is compiled, its inputs are copied to the device, and
 * fiona_hybrid_linear and fiona_hybrid_linear_static run on a stream of the
 * program's own.  Both results must equal the oracle's (oracle_weighted_sum,
 * the plain per-contribution evaluation in liboracle.so) word for word.
 * Built and run by tests/test_c_abi.py:
 *   c_abi_gpu q0 q1 q2 seed
 * Prints "ok" and returns 0, or names the first failed check and returns 1.
 */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "fiona.h"

/* the oracle (test infrastructure): see oracle/fiona_oracle.c */
int oracle_weighted_sum(uint32_t n_pos, const uint64_t *q, uint32_t n_in, const uint64_t *x, const uint64_t *pt,
                        uint32_t n_out, const uint32_t *pm_off, const uint32_t *pm_input, const uint32_t *pm_pt,
                        const uint32_t *grp_off, const uint32_t *grp_mem_off, const uint32_t *mem_input,
                        const int8_t *mem_sign, const uint32_t *grp_scale, const uint64_t *scales, uint64_t *out,
                        int n_threads);

#define CHECK(c)                                                  \
  do {                                                            \
    if (!(c)) {                                                   \
      printf("FAIL line %d: %s\n", __LINE__, #c);                 \
      return 1;                                                   \
    }                                                             \
  } while (0)
#define HIP(c) CHECK((c) == hipSuccess)

enum { N = 300, L = 3, N_IN = 20, N_OUT = 9, N_SCALE = 4, MAX_PM = 64, MAX_GRP = 8, MAX_MEM = 24 };

static uint64_t state;
static uint64_t next(void) {   /* xorshift64*: test inputs only */
  state ^= state >> 12;
  state ^= state << 25;
  state ^= state >> 27;
  return state * 2685821657736338717ull;
}

int main(int argc, char **argv) {
  if (argc != 5) {
    printf("usage: %s q0 q1 q2 seed\n", argv[0]);
    return 2;
  }
  uint64_t q[L];
  for (int l = 0; l < L; ++l) q[l] = strtoull(argv[l + 1], NULL, 10);
  state = strtoull(argv[4], NULL, 10) * 0x9E3779B97F4A7C15ull + 1;

  /* the layer: per output some raw terms and groups; every third group
   * repeats an earlier one, reversed every other time */
  static uint32_t pm_off[N_OUT + 1], pm_input[N_OUT * MAX_PM], pm_pt[N_OUT * MAX_PM];
  static uint32_t grp_off[N_OUT + 1], grp_mem_off[N_OUT * MAX_GRP + 1], mem_input[N_OUT * MAX_GRP * MAX_MEM];
  static uint32_t grp_scale[N_OUT * MAX_GRP];
  static int8_t mem_sign[N_OUT * MAX_GRP * MAX_MEM];
  uint32_t n_pm = 0, n_grp = 0, n_mem = 0;
  for (uint32_t j = 0; j < N_OUT; ++j) {
    const uint32_t raw = (uint32_t)(next() % MAX_PM), grp = (uint32_t)(next() % MAX_GRP);
    for (uint32_t t = 0; t < raw; ++t) {
      pm_input[n_pm] = (uint32_t)(next() % N_IN);
      pm_pt[n_pm] = n_pm;
      ++n_pm;
    }
    for (uint32_t g = 0; g < grp; ++g) {
      if (n_grp >= 2 && n_grp % 3 == 0) {   /* repeat group n_grp - 2 */
        const uint32_t src = n_grp - 2, m0 = grp_mem_off[src], m1 = grp_mem_off[src + 1];
        const int8_t s = (n_grp % 2) ? -1 : 1;
        for (uint32_t m = m0; m < m1; ++m) {
          mem_input[n_mem] = mem_input[m];
          mem_sign[n_mem] = (int8_t)(s * mem_sign[m]);
          ++n_mem;
        }
      } else {
        const uint32_t size = (uint32_t)(next() % MAX_MEM);
        for (uint32_t m = 0; m < size; ++m) {
          mem_input[n_mem] = (uint32_t)(next() % N_IN);
          mem_sign[n_mem] = (int8_t)((int)(next() % 3) - 1);
          ++n_mem;
        }
      }
      grp_scale[n_grp] = (uint32_t)(next() % N_SCALE);
      grp_mem_off[++n_grp] = n_mem;
    }
    pm_off[j + 1] = n_pm;
    grp_off[j + 1] = n_grp;
  }
  const uint32_t n_pt = n_pm ? n_pm : 1;
  uint64_t scales[N_SCALE];
  for (int c = 0; c < N_SCALE; ++c) scales[c] = 1 + next() % ((1u << 20) - 1);

  /* inputs and plaintexts: residues below each limb's modulus */
  const size_t LN = (size_t)L * N, n_x = (size_t)N_IN * 2 * LN, n_p = (size_t)n_pt * LN, n_y = (size_t)N_OUT * 2 * LN;
  uint64_t *x = malloc(n_x * 8), *pt = malloc(n_p * 8), *expect = malloc(n_y * 8), *got = malloc(n_y * 8);
  uint64_t *qpos = malloc(LN * 8);
  CHECK(x && pt && expect && got && qpos);
  for (size_t s = 0; s < LN; ++s) qpos[s] = q[s / N];
  for (size_t w = 0; w < n_x; ++w) x[w] = next() % qpos[w % LN];
  for (size_t w = 0; w < n_p; ++w) pt[w] = next() % qpos[w % LN];
  CHECK(oracle_weighted_sum((uint32_t)LN, qpos, N_IN, x, pt, N_OUT, pm_off, pm_input, pm_pt, grp_off, grp_mem_off,
                            mem_input, mem_sign, grp_scale, scales, expect, 4) == 0);

  /* the library */
  fiona_ctx *ctx = NULL;
  CHECK(fiona_ctx_create(N, L, q, &ctx) == FIONA_OK);
  fiona_layer_desc d;
  memset(&d, 0, sizeof d);
  d.n_in = N_IN;
  d.n_out = N_OUT;
  d.n_pt = n_pt;
  d.n_scale = N_SCALE;
  d.pm_off = pm_off;
  d.pm_input = pm_input;
  d.pm_pt = pm_pt;
  d.grp_off = grp_off;
  d.grp_mem_off = grp_mem_off;
  d.mem_input = mem_input;
  d.mem_sign = mem_sign;
  d.grp_scale = grp_scale;
  fiona_plan *plan = NULL;
  CHECK(fiona_plan_create(ctx, &d, &plan) == FIONA_OK);
  fiona_plan_stats_t st;
  CHECK(fiona_plan_stats(plan, &st) == FIONA_OK && st.ct_terms == (uint64_t)n_pm + n_mem);

  uint64_t *dx, *dp, *ds, *dy;
  int8_t *dsg;
  HIP(hipMalloc((void **)&dx, n_x * 8));
  HIP(hipMalloc((void **)&dp, n_p * 8));
  HIP(hipMalloc((void **)&ds, sizeof scales));
  HIP(hipMalloc((void **)&dy, n_y * 8));
  HIP(hipMalloc((void **)&dsg, n_mem ? n_mem : 1));
  HIP(hipMemcpy(dx, x, n_x * 8, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dp, pt, n_p * 8, hipMemcpyHostToDevice));
  HIP(hipMemcpy(ds, scales, sizeof scales, hipMemcpyHostToDevice));
  if (n_mem) HIP(hipMemcpy(dsg, mem_sign, n_mem, hipMemcpyHostToDevice));
  hipStream_t stream;
  HIP(hipStreamCreate(&stream));

  for (int entry = 0; entry < 2; ++entry) {
    HIP(hipMemset(dy, 0xFF, n_y * 8));
    const int rc = entry == 0 ? fiona_hybrid_linear(plan, dx, dp, dsg, ds, dy, stream)
                              : fiona_hybrid_linear_static(plan, dx, dp, dsg, ds, dy, stream);
    if (rc != FIONA_OK) printf("entry %d: %s\n", entry, fiona_status_string(rc));
    CHECK(rc == FIONA_OK);
    HIP(hipStreamSynchronize(stream));
    HIP(hipMemcpy(got, dy, n_y * 8, hipMemcpyDeviceToHost));
    for (size_t w = 0; w < n_y; ++w)
      if (got[w] != expect[w]) {
        printf("entry %d: word %zu (output %zu, poly %zu, limb %zu, coeff %zu): gpu %llu, oracle %llu\n", entry, w,
               w / (2 * LN), (w / LN) % 2, (w % LN) / N, w % N, (unsigned long long)got[w],
               (unsigned long long)expect[w]);
        return 1;
      }
  }
  /* an unaligned pointer and an output that overlaps an input are refused */
  CHECK(fiona_hybrid_linear(plan, (const uint64_t *)((const char *)dx + 4), dp, dsg, ds, dy, stream) ==
        FIONA_ERR_ALIGN);
  CHECK(fiona_hybrid_linear(plan, dx, dp, dsg, ds, dx, stream) == FIONA_ERR_ALIAS);

  HIP(hipStreamDestroy(stream));
  HIP(hipFree(dx));
  HIP(hipFree(dp));
  HIP(hipFree(ds));
  HIP(hipFree(dy));
  HIP(hipFree(dsg));
  fiona_plan_destroy(plan);
  fiona_ctx_destroy(ctx);
  free(x);
  free(pt);
  free(expect);
  free(got);
  free(qpos);
  printf("ok: %u raw terms, %u groups, %u members, %llu distinct sums\n", n_pm, n_grp, n_mem,
         (unsigned long long)st.n_sum_distinct);
  return 0;
}
