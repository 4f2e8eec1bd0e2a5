/*
 * Oracle for the hybrid weighted sum -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow CPU statement of what the GPU path must compute.  Only the
 * tests, the smoke check and the benchmark's CPU-baseline leg may load it; the
 * library under paper_2609_35352_amd/ never does, and the two share no code.
 *
 * What is computed (paper Sec. 4.2, "Exact Compilation of Routed Linear
 * Operators", Eq. (routed-example)): every packed output y_j is a sum of raw
 * terms, each a slot-wise product of a plaintext weight vector with an input
 * ciphertext (one PMult), and of signed terms, each an input ciphertext that a
 * pure group adds (h=+1), subtracts (h=-1) or skips (h=0) after applying the
 * output's reconstruction factor.  The paper's grouped and shared forms are
 * algebraic rewrites of this per-contribution form (Sec. 4.2), so the
 * per-contribution form is the plain definition, and it is what this file
 * evaluates: every signed term is applied on its own with weight h*c mod q.
 *
 * Representation (CKKS in RNS and NTT form; the paper's executor keeps this
 * inside its FHE library): a ciphertext is two polynomials; each polynomial is
 * stored per RNS prime q_l as N residues in the negacyclic NTT domain, where a
 * PMult is the element-wise product mod q_l and Add/Sub are element-wise.  A
 * constant reconstruction factor c encodes to the constant polynomial c, whose
 * NTT is c in every slot, so it is a scalar product mod q_l.
 *
 * Every position (limb l, coefficient k) is independent, so the data are
 * addressed by a flat position index s with modulus q[s]:
 *   x  [(i*2 + p) * n_pos + s]   input ciphertext i, polynomial p
 *   pt [pi * n_pos + s]          plaintext pi
 *   out[(j*2 + p) * n_pos + s]   output ciphertext j, polynomial p
 * With n_pos = L*N and s = l*N + k this is the limb-major ciphertext layout.
 *
 * Arithmetic: unsigned __int128 products and the C remainder operator, one
 * reduction per term.  Results are canonical residues in [0, q).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <pthread.h>

typedef unsigned __int128 u128;

static uint64_t mulmod(uint64_t a, uint64_t b, uint64_t q) {
  return (uint64_t)(((u128)a * (u128)b) % q);
}

static uint64_t addmod(uint64_t a, uint64_t b, uint64_t q) {
  return (uint64_t)(((u128)a + (u128)b) % q);
}

static uint64_t submod(uint64_t a, uint64_t b, uint64_t q) {
  return (uint64_t)(((u128)(a % q) + (u128)(q - b % q)) % q);
}

static uint64_t powmod(uint64_t b, uint64_t e, uint64_t q) {
  uint64_t r = 1 % q;
  b %= q;
  while (e) {
    if (e & 1) r = mulmod(r, b, q);
    b = mulmod(b, b, q);
    e >>= 1;
  }
  return r;
}

/* Weight of one signed term: its group's sign h in {-1,0,+1} times the group's
 * integer reconstruction factor c, as a residue mod q (Sec. 2.3 ternary
 * weights; Sec. 3 Obs. 2: Add for +1, Sub for -1, skip for 0). */
static uint64_t signed_weight(int h, uint64_t c, uint64_t q) {
  if (h > 0) return c % q;
  if (h < 0) return (q - c % q) % q;
  return 0;
}

typedef struct {
  uint32_t n_pos;
  const uint64_t *q;
  uint32_t n_in;
  const uint64_t *x;
  const uint64_t *pt;
  uint32_t n_out;
  const uint32_t *pm_off, *pm_input, *pm_pt;
  const uint32_t *grp_off, *grp_mem_off, *mem_input;
  const int8_t *mem_sign;
  const uint32_t *grp_scale;
  const uint64_t *scales;
  uint64_t *out;
  uint32_t s_begin, s_end;
} ws_job;

static void *ws_worker(void *arg) {
  const ws_job *a = (const ws_job *)arg;
  const size_t n_pos = a->n_pos;
  for (uint32_t s = a->s_begin; s < a->s_end; ++s) {
    const uint64_t q = a->q[s];
    for (uint32_t j = 0; j < a->n_out; ++j) {
      for (uint32_t p = 0; p < 2; ++p) {
        uint64_t acc = 0;
        /* raw route: one PMult per term */
        for (uint32_t t = a->pm_off[j]; t < a->pm_off[j + 1]; ++t) {
          const uint64_t w = a->pt[(size_t)a->pm_pt[t] * n_pos + s];
          const uint64_t xv = a->x[((size_t)a->pm_input[t] * 2 + p) * n_pos + s];
          acc = addmod(acc, mulmod(w, xv, q), q);
        }
        /* signed route, per contribution: weight h*c of the member's group */
        for (uint32_t g = a->grp_off[j]; g < a->grp_off[j + 1]; ++g) {
          const uint64_t c = a->scales[a->grp_scale[g]];
          for (uint32_t m = a->grp_mem_off[g]; m < a->grp_mem_off[g + 1]; ++m) {
            const uint64_t w = signed_weight(a->mem_sign[m], c, q);
            const uint64_t xv = a->x[((size_t)a->mem_input[m] * 2 + p) * n_pos + s];
            acc = addmod(acc, mulmod(w, xv, q), q);
          }
        }
        a->out[((size_t)j * 2 + p) * n_pos + s] = acc;
      }
    }
  }
  return NULL;
}

/* Per-contribution hybrid weighted sum over n_pos positions; see the file
 * comment for the layouts.  Returns 0, or -1 on a bad argument. */
int oracle_weighted_sum(uint32_t n_pos, const uint64_t *q, uint32_t n_in, const uint64_t *x,
                        const uint64_t *pt, uint32_t n_out, const uint32_t *pm_off,
                        const uint32_t *pm_input, const uint32_t *pm_pt, const uint32_t *grp_off,
                        const uint32_t *grp_mem_off, const uint32_t *mem_input,
                        const int8_t *mem_sign, const uint32_t *grp_scale, const uint64_t *scales,
                        uint64_t *out, int n_threads) {
  if (!q || !x || !pm_off || !grp_off || !out || n_threads < 1) return -1;
  if (n_threads > 256) n_threads = 256;
  if ((uint32_t)n_threads > n_pos) n_threads = n_pos ? (int)n_pos : 1;
  pthread_t th[256];
  ws_job jobs[256];
  for (int t = 0; t < n_threads; ++t) {
    ws_job *jb = &jobs[t];
    jb->n_pos = n_pos; jb->q = q; jb->n_in = n_in; jb->x = x; jb->pt = pt; jb->n_out = n_out;
    jb->pm_off = pm_off; jb->pm_input = pm_input; jb->pm_pt = pm_pt;
    jb->grp_off = grp_off; jb->grp_mem_off = grp_mem_off; jb->mem_input = mem_input;
    jb->mem_sign = mem_sign; jb->grp_scale = grp_scale; jb->scales = scales; jb->out = out;
    jb->s_begin = (uint32_t)((uint64_t)n_pos * t / n_threads);
    jb->s_end = (uint32_t)((uint64_t)n_pos * (t + 1) / n_threads);
  }
  if (n_threads == 1) {
    ws_worker(&jobs[0]);
    return 0;
  }
  for (int t = 0; t < n_threads; ++t) pthread_create(&th[t], NULL, ws_worker, &jobs[t]);
  for (int t = 0; t < n_threads; ++t) pthread_join(th[t], NULL);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Negacyclic NTT, used only by the tests that pin the meaning of the        */
/* element-wise product (PMult) and by the toy CKKS round trip.              */
/* ------------------------------------------------------------------------ */

/* psi: a primitive 2N-th root of unity mod q, x^((q-1)/2N) for the smallest
 * x >= 2 with psi^N = -1 (mod q).  Returns 0 if q != 1 (mod 2N) or none found. */
uint64_t oracle_find_psi(uint32_t N, uint64_t q) {
  if (N == 0 || (q - 1) % (2ull * N) != 0) return 0;
  for (uint64_t x = 2; x < 1000000; ++x) {
    uint64_t psi = powmod(x, (q - 1) / (2ull * N), q);
    if (powmod(psi, N, q) == q - 1) return psi;
  }
  return 0;
}

/* Definition: out_k = sum_n a_n psi^((2k+1) n) mod q, k = 0..N-1 (O(N^2)). */
void oracle_ntt_naive(const uint64_t *a, uint64_t *out, uint32_t N, uint64_t q, uint64_t psi) {
  for (uint32_t k = 0; k < N; ++k) {
    const uint64_t w = powmod(psi, 2ull * k + 1, q);
    uint64_t wn = 1, acc = 0;
    for (uint32_t n = 0; n < N; ++n) {
      acc = addmod(acc, mulmod(a[n] % q, wn, q), q);
      wn = mulmod(wn, w, q);
    }
    out[k] = acc;
  }
}

/* Definition of the inverse: a_n = N^-1 sum_k out_k psi^(-(2k+1) n) mod q. */
void oracle_intt_naive(const uint64_t *in, uint64_t *a, uint32_t N, uint64_t q, uint64_t psi) {
  const uint64_t psi_inv = powmod(psi, q - 2, q);
  const uint64_t n_inv = powmod(N % q, q - 2, q);
  for (uint32_t n = 0; n < N; ++n) {
    const uint64_t w = powmod(psi_inv, n, q);   /* psi^-n */
    const uint64_t w2 = mulmod(w, w, q);        /* psi^-2n */
    uint64_t wk = w, acc = 0;                   /* psi^-(2k+1)n, k = 0 */
    for (uint32_t k = 0; k < N; ++k) {
      acc = addmod(acc, mulmod(in[k] % q, wk, q), q);
      wk = mulmod(wk, w2, q);
    }
    a[n] = mulmod(acc, n_inv, q);
  }
}

/* Cyclic DFT of length n (a power of two) with root omega, by the textbook
 * radix-2 recursion: X_k = E_k + omega^k O_k, X_{k+n/2} = E_k - omega^k O_k. */
static void dft_rec(uint64_t *v, uint32_t n, uint64_t omega, uint64_t q, uint64_t *tmp) {
  if (n == 1) return;
  const uint32_t h = n / 2;
  for (uint32_t i = 0; i < h; ++i) {
    tmp[i] = v[2 * i];
    tmp[h + i] = v[2 * i + 1];
  }
  memcpy(v, tmp, n * sizeof(uint64_t));
  const uint64_t omega2 = mulmod(omega, omega, q);
  dft_rec(v, h, omega2, q, tmp);
  dft_rec(v + h, h, omega2, q, tmp);
  uint64_t wk = 1;
  for (uint32_t k = 0; k < h; ++k) {
    const uint64_t e = v[k], o = mulmod(wk, v[h + k], q);
    tmp[k] = addmod(e, o, q);
    tmp[h + k] = submod(e, o, q);
    wk = mulmod(wk, omega, q);
  }
  memcpy(v, tmp, n * sizeof(uint64_t));
}

/* Same transform as oracle_ntt_naive in O(N log N): twist a_n by psi^n, then a
 * cyclic DFT with omega = psi^2, since psi^((2k+1)n) = psi^n (psi^2)^(kn).
 * N must be a power of two.  Returns -1 if it is not. */
int oracle_ntt_fast(const uint64_t *a, uint64_t *out, uint32_t N, uint64_t q, uint64_t psi) {
  if (N == 0 || (N & (N - 1))) return -1;
  uint64_t *tmp = (uint64_t *)malloc(sizeof(uint64_t) * N);
  if (!tmp) return -1;
  uint64_t pn = 1;
  for (uint32_t n = 0; n < N; ++n) {
    out[n] = mulmod(a[n] % q, pn, q);
    pn = mulmod(pn, psi, q);
  }
  dft_rec(out, N, mulmod(psi, psi, q), q, tmp);
  free(tmp);
  return 0;
}

/* Inverse of oracle_ntt_fast: cyclic DFT with omega^-1, scale by N^-1, untwist
 * by psi^-n. */
int oracle_intt_fast(const uint64_t *in, uint64_t *a, uint32_t N, uint64_t q, uint64_t psi) {
  if (N == 0 || (N & (N - 1))) return -1;
  uint64_t *tmp = (uint64_t *)malloc(sizeof(uint64_t) * N);
  if (!tmp) return -1;
  const uint64_t psi_inv = powmod(psi, q - 2, q);
  const uint64_t n_inv = powmod(N % q, q - 2, q);
  for (uint32_t k = 0; k < N; ++k) a[k] = in[k] % q;
  dft_rec(a, N, mulmod(psi_inv, psi_inv, q), q, tmp);
  uint64_t pn = n_inv;
  for (uint32_t n = 0; n < N; ++n) {
    a[n] = mulmod(a[n], pn, q);
    pn = mulmod(pn, psi_inv, q);
  }
  free(tmp);
  return 0;
}

/* Schoolbook product in Z_q[X]/(X^N + 1): X^N = -1 folds the high half back
 * with a minus sign. */
void oracle_negacyclic_mul(const uint64_t *a, const uint64_t *b, uint64_t *c, uint32_t N, uint64_t q) {
  for (uint32_t k = 0; k < N; ++k) c[k] = 0;
  for (uint32_t i = 0; i < N; ++i) {
    for (uint32_t j = 0; j < N; ++j) {
      const uint64_t prod = mulmod(a[i] % q, b[j] % q, q);
      const uint32_t d = i + j;
      if (d < N) c[d] = addmod(c[d], prod, q);
      else c[d - N] = submod(c[d - N], prod, q);
    }
  }
}

/* acc_k = (acc_k + a_k b_k) mod q for k < N: one term of an element-wise
 * (NTT-domain) inner product, used by the rotation oracle's key switching. */
void oracle_mul_acc(uint64_t *acc, const uint64_t *a, const uint64_t *b, uint32_t N, uint64_t q) {
  for (uint32_t k = 0; k < N; ++k) acc[k] = addmod(acc[k], mulmod(a[k] % q, b[k] % q, q), q);
}
