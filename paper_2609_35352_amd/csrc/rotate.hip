// Hoisted baby-step rotations: the step that produces the hot path's input
// ciphertexts.  A linear layer's inputs A_i are the packed input rotated by
// the packing layout's baby steps (paper Sec. 2, "Homomorphic Operations":
// Rot cyclically shifts the slots; Sec. 4.2: the A_i are prepared according
// to the packing layout).  Rot by r slots is the automorphism
// sigma_g: a(X) -> a(X^g), g = 5^r mod 2N, on both polynomials, then a key
// switch of the second one from sigma_g(s) back to s, by RNS digits (digit j
// = the coefficients of c1 mod q_j, in [0, q_j)), over the data moduli and
// one special prime P, with a rounded division by P at the end.
//
// In the NTT domain a_hat_k = a(psi^(2k+1)), the automorphism is the slot
// gather (sigma a)_hat[k] = a_hat[pi(k)], pi(k) = k g + (g - 1) / 2 mod N.
// Per call (one input ciphertext, several rotations):
//   1. digits, once (hoisting): D_j = INTT_{q_j}(c1_j) and
//      Dhat[j][m] = NTT_m(D_j mod m) for every modulus m of q_0 .. q_{L-1}, P;
//   2. per rotation, the key-switch inner product in the pi^-1 frame:
//      u'_p[m][i] = sum_j Dhat[j][m][i] * K'[j][p][m][i]  mod m, where the
//      library's key layout holds K'[j][p][m][i] = ksk_hat[j][p][m][pi^-1(i)],
//      so that no digit is gathered;
//   3. the division by P with rounding (the rescale of the chain
//      q_0 .. q_{L-1}, P): v' = round(u' / P), with c0 added to v'_0;
//   4. the gather back: out_0[k] = (c0 + v'_0)[pi(k)], out_1[k] = v'_1[pi(k)],
//      exact because the automorphism permutes the coefficients up to sign
//      and the rounding division is odd-symmetric (P is odd: no ties).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <algorithm>
#include <cstring>
#include <new>
#include <vector>

#include "fiona.h"
#include "fiona_ctx.hpp"
#include "modarith.hpp"
#include "ntt_host.hpp"

using namespace fiona_host;

namespace fiona {

constexpr uint32_t kKsTile = 128;   // coefficients per workgroup of the inner product (two per lane)
constexpr uint32_t kKsWaves = 8;    // wavefronts per workgroup; rotations are dealt out to them
constexpr uint32_t kKsRoundMax = 64;   // rotations whose outputs are buffered in LDS per round, at most
constexpr size_t kKsLdsMax = 160 * 1024;

typedef uint32_t ks_u4 __attribute__((ext_vector_type(4)));
typedef uint64_t ks_q2 __attribute__((ext_vector_type(2)));

// LDS of the inner product: the digits, the zero row and `round` rotations'
// outputs (2 KiB per row of a tile).
__host__ __device__ constexpr size_t ks_lds_bytes(uint32_t L, uint32_t round) {
  return (size_t)(L + 1) * kKsTile * sizeof(uint2) + (size_t)round * 2 * kKsTile * sizeof(uint64_t);
}
// The most rotations per round that fit the LDS next to the digits.
inline uint32_t ks_round(uint32_t L) {
  const size_t free = kKsLdsMax - ks_lds_bytes(L, 0);
  const size_t r = free / (2 * kKsTile * sizeof(uint64_t));
  return r < kKsRoundMax ? (uint32_t)r : kKsRoundMax;
}

// Step 2.  Workgroup = (modulus m, tile of 128 coefficients); lane l takes
// coefficients 2l and 2l + 1 of the tile, so that every key and digit load is
// 16 bytes per lane and 1 KiB per wavefront.  The L digits of the tile are
// staged in LDS as radix-2^25 digit pairs; each wavefront then takes
// rotations r = wave, wave + kKsWaves, ..., loads the 2 L key word pairs of
// each lane in batches of JB digits (both polynomials), and accumulates the
// exact products (modarith.hpp), reduced once per output.  Padding terms of a
// batch read the zero row and repeat a real key address.  The outputs of up
// to `round` rotations wait in LDS and leave together after a barrier
// (writes mixed one by one into the key stream cost more: 2-3% measured).
// Measured against one coefficient per lane (512-byte loads, 2 workgroups
// per CU): VGG11's 63 rotations 1.75 -> 1.58 ms, BERT's 31 1.67 -> 1.50 ms,
// Large's 127 10.0 -> 9.5 ms; with one workgroup per CU here (the LDS of a
// 64-rotation round).
template <uint32_t JB>
__global__ void __launch_bounds__(kKsWaves * 64) ks_inner_kernel(const uint64_t *__restrict__ dhat,
                                                                  const uint64_t *__restrict__ keys,
                                                                  uint64_t *__restrict__ u,
                                                                  const LimbConst *__restrict__ limbs, uint32_t N,
                                                                  uint32_t L, uint32_t n_rot, uint32_t round) {
  extern __shared__ uint4 ks_lds[];   // [L + 1][64] two digit pairs per lane (the last row zero),
                                      // then [round][2][64] two outputs per lane
  uint4 *xs = ks_lds;
  const uint32_t tiles = N / kKsTile;
  const uint32_t m = blockIdx.x / tiles, t = blockIdx.x - m * tiles;
  const uint32_t lane = threadIdx.x & 63u, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t k = t * kKsTile + 2 * lane;
  const uint32_t M = L + 1;
  for (uint32_t j = wave; j < L; j += kKsWaves) {
    const ks_q2 x = __builtin_nontemporal_load((const ks_q2 *)(dhat + ((size_t)j * M + m) * N + k));
    xs[j * 64 + lane] = make_uint4(lo_digit(x.x), hi_digit(x.x), lo_digit(x.y), hi_digit(x.y));
  }
  if (wave == 0) xs[L * 64 + lane] = make_uint4(0, 0, 0, 0);
  __syncthreads();
  const LimbConst lc = limbs[m];
  const size_t poly = (size_t)M * N;           // words between the two polynomials of a digit
  const size_t rot_words = (size_t)L * 2 * poly;
  ks_q2 *obuf = (ks_q2 *)(xs + M * 64);
  for (uint32_t r0 = 0; r0 < n_rot; r0 += round) {   // uniform over the workgroup
    const uint32_t nr = n_rot - r0 < round ? n_rot - r0 : round;
    for (uint32_t rr = wave; rr < nr; rr += kKsWaves) {
      const uint64_t *kr = keys + (size_t)(r0 + rr) * rot_words + (size_t)m * N + k;
      Acc a00, a01, a10, a11;   // [coefficient 2l, 2l + 1][polynomial]
      acc_zero(a00);
      acc_zero(a01);
      acc_zero(a10);
      acc_zero(a11);
      for (uint32_t j0 = 0; j0 < L; j0 += JB) {
        ks_u4 w0[JB], w1[JB];
#pragma unroll
        for (uint32_t b = 0; b < JB; ++b) {
          const uint32_t j = j0 + b < L ? j0 + b : L - 1;
          w0[b] = __builtin_nontemporal_load((const ks_u4 *)(kr + (size_t)j * 2 * poly));
          w1[b] = __builtin_nontemporal_load((const ks_u4 *)(kr + (size_t)j * 2 * poly + poly));
        }
#pragma unroll
        for (uint32_t b = 0; b < JB; ++b) {
          const uint32_t row = j0 + b < L ? j0 + b : L;
          const uint4 x = xs[row * 64 + lane];
          mac(a00, x.x, x.y, w0[b].x, w0[b].y);
          mac(a01, x.x, x.y, w1[b].x, w1[b].y);
          mac(a10, x.z, x.w, w0[b].z, w0[b].w);
          mac(a11, x.z, x.w, w1[b].z, w1[b].w);
        }
      }
      obuf[(2 * rr) * 64 + lane] = (ks_q2){finish(a00, 0, lc), finish(a10, 0, lc)};
      obuf[(2 * rr + 1) * 64 + lane] = (ks_q2){finish(a01, 0, lc), finish(a11, 0, lc)};
    }
    __syncthreads();
    for (uint32_t e = wave; e < 2 * nr; e += kKsWaves) {   // u: [2][n_rot][L + 1][N]
      const uint32_t p = e & 1u, r = r0 + (e >> 1);
      __builtin_nontemporal_store(obuf[e * 64 + lane], (ks_q2 *)(u + (((size_t)p * n_rot + r) * M + m) * N + k));
    }
    __syncthreads();   // the next round refills the buffer
  }
}

// Steps 3-4 fused: the forward pass B of the division by P that also applies
// the automorphism.  With d = d_lo + N2 d_hi and A = (g d_lo + c) mod N
// (c = (g - 1) / 2), pi(d) = k2 + N2 k1 where k2 = A mod N2 depends on d_lo
// only and k1 = (A / N2 + g d_hi) mod N1.  A workgroup takes 16 consecutive
// destination columns d_lo, transforms the 16 intermediate rows k2 they read
// (contiguous rows of N1 words), finishes the division there (u' and c0 are
// in the transposed layout, so row k2 is contiguous too), and then stores
// each destination row d_hi as a run of 16 words, picking k1 in LDS.
// Vectors: set = data limb l, vector lv = p n_rot + r in the set.
template <uint32_t LOGM>
__global__ void __launch_bounds__(kNttThreads) ntt_pass_b_rot(const NttPass P, const RotArgs R) {
  using D = DftShape<LOGM>;
  using G = GeomRot<LOGM>;
  constexpr uint32_t M = D::M, PM = D::PM, PER = G::PER;
  extern __shared__ double xs[];   // [kNttCols][PM], then the M/2 DFT twiddles
  Tw *tw = (Tw *)(xs + kNttCols * PM);
  const uint32_t set = blockIdx.y / P.vps, lv = blockIdx.y - set * P.vps;
  const uint32_t p = lv / R.n_rot, r = lv - p * R.n_rot;
  const NttSet S = P.sets[set];
  stage_twiddles(tw, S.dft_b, LOGM);
  Tw t1[8];
  first_twiddles<LOGM>(t1, S.dft_b);
  const uint32_t log_n2 = P.log_n2, N2 = 1u << log_n2, N = M << log_n2;   // M = N1
  const uint32_t g = R.g[r], cg = (g - 1) / 2, o0 = blockIdx.x * kNttCols;
  const double q = S.q, qinv = S.qinv;
  const Buf tmp(P.tmp + (uint64_t)blockIdx.y * N, P.tmp_end);
#pragma unroll 1
  for (uint32_t it = threadIdx.x; it < D::IT1; it += kNttThreads) {
    const uint32_t row = G::row(it), ip = G::grp(it);
    const uint32_t k2 = G::src_row(g, o0 + row, N2);
    double x[16];
#pragma unroll
    for (uint32_t u = 0; u < 16; ++u) {
      const Off ot = G::tmp(k2, ip, u);
      x[u] = tmp.f64_once(ot.v, ot.s);
    }
    first_stages<LOGM>(x, t1, q, qinv);
    put_first<LOGM>(xs, row, ip, x);
  }
  middle_stages<LOGM>(xs, tw, q, qinv);
  const Buf base(P.base + set * P.base_set_stride + lv * P.base_stride, P.base_end),
      add(P.add + set * P.add_set_stride, P.add_end);
  // row cc of the workgroup (k2 of destination column o0 + cc), outputs k1:
  // (u' - transform) * P^-1, plus c0 for the first polynomial, into LDS
#pragma unroll 1
  for (uint32_t it = threadIdx.x; it < D::IT2; it += kNttThreads) {
    const uint32_t cc = G::row2(it), o = G::off2(it);
    const uint32_t k2c = G::src_row(g, o0 + cc, N2);
    double y[D::E2];
    last_stages<LOGM>(xs, cc, o, tw, y, q, qinv);
    uint64_t bv[D::E2];
#pragma unroll
    for (uint32_t u = 0; u < D::E2; ++u) {
      const Off ow = G::word(k2c, o, u);
      bv[u] = base.u64_once(ow.v, ow.s);
    }
#pragma unroll
    for (uint32_t u = 0; u < D::E2; ++u) y[u] = canonical(mul_tw(to_f64(bv[u]) - y[u], S.inv, q), q, qinv);
    if (p == 0) {
      uint64_t av[D::E2];
#pragma unroll
      for (uint32_t u = 0; u < D::E2; ++u) {
        const Off ow = G::word(k2c, o, u);
        av[u] = add.u64(ow.v, ow.s);
      }
#pragma unroll
      for (uint32_t u = 0; u < D::E2; ++u) {
        const double z = y[u] + to_f64(av[u]);
        y[u] = z >= q ? z - q : z;
      }
    }
#pragma unroll
    for (uint32_t u = 0; u < D::E2; ++u) xs[cc * PM + pidx(o + (u << D::S0L))] = y[u];
  }
  __syncthreads();
  // destination column o0 + c, rows d_hi = rr + 16 j: runs of 16 words
  const uint32_t c = threadIdx.x % kNttCols, rr = threadIdx.x / kNttCols;
  const uint32_t hi = ((g * (o0 + c) + cg) & (N - 1)) >> log_n2;
  const Buf out((uint64_t *)P.out + ((size_t)(r * 2 + p) * R.L + set) * N, P.out_end);
#pragma unroll
  for (uint32_t j = 0; j < PER; ++j) {
    const uint32_t d_hi = rr + j * kNttCols;
    const uint32_t k1 = (hi + g * d_hi) & (M - 1);
    const Off oo = G::out(o0, threadIdx.x, j, N2);
    out.put(to_u64(xs[c * PM + pidx(k1)]), oo.v, oo.s);
  }
}

// c0 of the input ciphertext in the transposed layout (L limbs), for the
// fused division: out[l][k2 N1 + k1] = c0[l][k2 + N2 k1].
__global__ void __launch_bounds__(256) transpose_kernel(const uint64_t *__restrict__ in, uint64_t *__restrict__ out,
                                                        uint32_t log_n1, uint32_t log_n2) {
  const uint32_t N = 1u << (log_n1 + log_n2);
  const uint32_t a = blockIdx.x * 256 + threadIdx.x;   // destination index
  const size_t limb = (size_t)blockIdx.y * N;
  if (a >= N) return;
  const uint32_t k2 = a >> log_n1, k1 = a & ((1u << log_n1) - 1);
  out[limb + a] = in[limb + k2 + ((size_t)k1 << log_n2)];
}

// The library's key layout: every row of N words permuted by pi^-1 and stored
// transposed, K'[row][k2 N1 + k1] = K[row][pi^-1(k2 + N2 k1)], with
// pi^-1(i) = (i - (g - 1) / 2) g^-1 mod N.
__global__ void __launch_bounds__(256) key_layout_kernel(const uint64_t *__restrict__ key,
                                                         uint64_t *__restrict__ out, uint32_t log_n1,
                                                         uint32_t log_n2, uint32_t rows, uint32_t g, uint32_t ginv) {
  const uint32_t N = 1u << (log_n1 + log_n2);
  const uint32_t row = blockIdx.y;
  const uint32_t a = blockIdx.x * 256 + threadIdx.x;
  if (row >= rows || a >= N) return;
  const uint32_t i = (a >> log_n1) + ((a & ((1u << log_n1) - 1)) << log_n2);
  const uint32_t src = ((i - (g - 1) / 2) * ginv) & (N - 1);
  out[(size_t)row * N + a] = key[(size_t)row * N + src];
}

}  // namespace fiona

struct fiona_rotator {
  const fiona_ctx *ctx = nullptr;
  fiona_ctx *ext = nullptr;            // q_0 .. q_{L-1}, P (their multiply-add constants)
  uint32_t N = 0, L = 0, log_n1 = 0, log_n2 = 0, max_rot = 0;
  uint64_t P = 0;
  int device = -1;
  void *dev = nullptr;
  const NttSet *inv_sets = nullptr;    // [L] inverse transforms of q_0 .. q_{L-1}
  const NttSet *fwd_sets = nullptr;    // [L + 1] forward transforms of q_0 .. q_{L-1}, P
  const NttSet *down_sets = nullptr;   // [L] forward transforms of q_0 .. q_{L-1}, inv = P^-1 mod q_l
  const NttSet *p_inv_set = nullptr;   // [1] inverse transform of P
  const fiona::LimbConst *limbs = nullptr;   // [L + 1] on the device
  uint64_t *D = nullptr;               // [L][N] digits
  uint64_t *Dhat = nullptr;            // [L][L + 1][N], transposed layout
  uint64_t *c0t = nullptr;             // [L][N] c0 of the call, transposed layout
  double *T = nullptr;                 // NTT intermediates: max(L (L + 1), 2 L max_rot) vectors
  double *W = nullptr;                 // [2 max_rot][N] centred coefficients of u'_P
  uint64_t *U = nullptr;               // [2][n_rot][L + 1][N], transposed layout
  const void *D_end = nullptr, *Dhat_end = nullptr, *c0t_end = nullptr, *T_end = nullptr, *W_end = nullptr,
             *U_end = nullptr;
  size_t limb_bytes = 0;
};

namespace {

size_t round256(size_t x) { return (x + 255) / 256 * 256; }

template <uint32_t LOG>
void launch_rot_b(dim3 grid, size_t smem, hipStream_t stream, const NttPass &P, const fiona::RotArgs &G) {
  hipLaunchKernelGGL(fiona::ntt_pass_b_rot<LOG>, grid, dim3(fiona::kNttThreads), smem, stream, P, G);
}

// The fused pass B over V vectors: grid (N2 / 16 destination blocks, V).
void launch_rot_pass_b(uint32_t log_n1, uint32_t log_n2, uint32_t V, hipStream_t stream, const NttPass &P,
                       const fiona::RotArgs &G) {
  if (LaunchRecord *rec = launch_recorder()) {
    rec->passes.push_back(PassLaunch{PassLaunch::kPassBRot, log_n1, log_n2, V, P, G});
    return;
  }
  const dim3 grid((1u << log_n2) / fiona::kNttCols, V);
  const size_t smem = fiona::kNttCols * fiona::padded_len(1u << log_n1) * sizeof(double) +
                      (1u << log_n1) / 2 * sizeof(Tw);
  switch (log_n1) {
    case 4: launch_rot_b<4>(grid, smem, stream, P, G); break;
    case 5: launch_rot_b<5>(grid, smem, stream, P, G); break;
    case 6: launch_rot_b<6>(grid, smem, stream, P, G); break;
    case 7: launch_rot_b<7>(grid, smem, stream, P, G); break;
    case 8: launch_rot_b<8>(grid, smem, stream, P, G); break;
    default: launch_rot_b<9>(grid, smem, stream, P, G); break;
  }
}

template <uint32_t LOG>
bool allow_rot_one(int bytes) {
  return hipFuncSetAttribute((const void *)fiona::ntt_pass_b_rot<LOG>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             bytes) == hipSuccess;
}

bool allow_rot_smem(int bytes) {
  return allow_rot_one<4>(bytes) && allow_rot_one<5>(bytes) && allow_rot_one<6>(bytes) &&
         allow_rot_one<7>(bytes) && allow_rot_one<8>(bytes) && allow_rot_one<9>(bytes);
}

bool overlap(const void *a, size_t na, const void *b, size_t nb) {
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + nb && b0 < a0 + na;
}

// Checks the parameters and sizes a rotator: its tables (img) and the bytes
// of its device buffer.  R->ext (host only) is created here.
int rotator_layout(const fiona_ctx *ctx, uint64_t special_prime, const uint64_t *psi, uint32_t max_rot,
                   fiona_rotator *R, TableImage &img, size_t &total) {
  if (max_rot == 0) return FIONA_ERR_ARG;
  const uint32_t N = ctx->N, L = ctx->L;
  uint32_t logN = 0;
  while ((1u << logN) < N) ++logN;
  if ((1u << logN) != N || logN < 8 || logN > 17 || L < 1 || L + 1 > FIONA_MAX_L) return FIONA_ERR_UNSUPPORTED;
  if ((size_t)L * (L + 1) > 65535 || max_rot > fiona::kRotMax) return FIONA_ERR_UNSUPPORTED;
  const uint64_t P = special_prime;
  if (P <= (1ull << FIONA_SCALE_BITS) || P >= (1ull << FIONA_MODULUS_BITS) || (P - 1) % (2ull * N) != 0)
    return FIONA_ERR_UNSUPPORTED;
  std::vector<uint64_t> mods(ctx->q.begin(), ctx->q.end());
  for (uint64_t q : mods)
    if (q == P) return FIONA_ERR_UNSUPPORTED;
  mods.push_back(P);
  std::vector<uint64_t> roots(L + 1);
  for (uint32_t i = 0; i <= L; ++i) {
    const uint64_t q = mods[i];
    if ((q - 1) % (2ull * N) != 0) return FIONA_ERR_UNSUPPORTED;
    roots[i] = psi ? psi[i] % q : default_psi(N, q);
    if (roots[i] == 0 || powmod_h(roots[i], N, q) != q - 1) return FIONA_ERR_UNSUPPORTED;
  }
  R->ctx = ctx;
  R->N = N;
  R->L = L;
  R->P = P;
  R->log_n1 = (logN + 1) / 2;
  R->log_n2 = logN / 2;
  R->max_rot = max_rot;
  const int rc = fiona_ctx_create(N, L + 1, mods.data(), &R->ext);
  if (rc != FIONA_OK) return rc;
  for (uint32_t j = 0; j < L; ++j) img.add(make_tables(R->log_n1, R->log_n2, mods[j], roots[j], true), mods[j]);
  for (uint32_t i = 0; i <= L; ++i) img.add(make_tables(R->log_n1, R->log_n2, mods[i], roots[i], false), mods[i]);
  for (uint32_t l = 0; l < L; ++l)
    img.add(make_tables(R->log_n1, R->log_n2, mods[l], roots[l], false), mods[l],
            make_tw(powmod_h(P % mods[l], mods[l] - 2, mods[l]), mods[l]));
  img.add(make_tables(R->log_n1, R->log_n2, P, roots[L], true), P);
  const size_t vec = (size_t)N * 8;
  R->limb_bytes = round256((L + 1) * sizeof(fiona::LimbConst));
  const size_t t_vectors = std::max((size_t)L * (L + 1), (size_t)2 * L * max_rot);
  total = img.bytes() + R->limb_bytes + round256(L * vec) + round256((size_t)L * (L + 1) * vec) +
          round256(L * vec) + round256(t_vectors * vec) + round256((size_t)2 * max_rot * vec) +
          round256((size_t)max_rot * 2 * (L + 1) * vec);
  return FIONA_OK;
}

// Points the rotator's parts into its device buffer at dev.
void rotator_place(fiona_rotator *R, const TableImage &img, void *dev) {
  const uint32_t L = R->L;
  const size_t vec = (size_t)R->N * 8;
  const size_t t_vectors = std::max((size_t)L * (L + 1), (size_t)2 * L * R->max_rot);
  R->dev = dev;
  const NttSet *sets = img.sets_addr(dev);
  R->inv_sets = sets;
  R->fwd_sets = sets + L;
  R->down_sets = sets + 2 * L + 1;
  R->p_inv_set = sets + 3 * L + 1;
  char *p = (char *)dev + img.bytes();
  auto take = [&](size_t bytes, const void *&end) {
    char *at = p;
    end = at + bytes;
    p += round256(bytes);
    return at;
  };
  const void *limbs_end = nullptr;
  R->limbs = (const fiona::LimbConst *)take((L + 1) * sizeof(fiona::LimbConst), limbs_end);
  R->D = (uint64_t *)take(L * vec, R->D_end);
  R->Dhat = (uint64_t *)take((size_t)L * (L + 1) * vec, R->Dhat_end);
  R->c0t = (uint64_t *)take(L * vec, R->c0t_end);
  R->T = (double *)take(t_vectors * vec, R->T_end);
  R->W = (double *)take((size_t)2 * R->max_rot * vec, R->W_end);
  R->U = (uint64_t *)take((size_t)R->max_rot * 2 * (L + 1) * vec, R->U_end);
}

// The launches of one call (arguments already checked).
void rotate_enqueue(const fiona_rotator *R, const uint64_t *ct, uint32_t n_rot, const uint32_t *galois,
                    const uint64_t *keys, uint64_t *out_cts, hipStream_t stream) {
  const uint32_t N = R->N, L = R->L;
  const uint32_t M = L + 1;
  const void *ct_end = ct + (size_t)2 * L * N, *out_end = out_cts + (size_t)n_rot * 2 * L * N;

  // 1. digits of c1, once: D_j = INTT_{q_j}(c1_j), then Dhat[j][m] = NTT_m(D_j)
  //    (transposed layout); c0 transposed for step 3
  NttPass A{};
  A.sets = R->inv_sets;
  A.vps = 1;
  A.log_n1 = R->log_n1;
  A.log_n2 = R->log_n2;
  A.in = ct + (size_t)L * N;
  A.in_end = ct_end;
  A.in_set_stride = N;
  A.tmp = R->T;
  A.tmp_end = R->T_end;
  A.out = R->D;
  A.out_end = R->D_end;
  A.out_set_stride = N;
  A.load = fiona::kLoadU64;
  A.store = fiona::kStoreU64;
  launch_transform(R->log_n1, R->log_n2, L, stream, A);
  NttPass B{};
  B.sets = R->fwd_sets;
  B.vps = L;
  B.log_n1 = R->log_n1;
  B.log_n2 = R->log_n2;
  B.in = R->D;
  B.in_end = R->D_end;
  B.in_stride = N;
  B.tmp = R->T;
  B.tmp_end = R->T_end;
  B.out = R->Dhat;
  B.out_end = R->Dhat_end;
  B.out_stride = (size_t)M * N;
  B.out_set_stride = N;
  B.load = fiona::kLoadU64;
  B.store = fiona::kStoreU64;
  B.out_transposed = 1;
  B.nsets_shared = ((1u << R->log_n1) / fiona::kNttCols * L) % 8 == 0 ? M : 0;   // every modulus reads D_j
  launch_transform(R->log_n1, R->log_n2, L * M, stream, B);
  // transpose_kernel: reads limbs 0 .. L-1 of c0, writes L vectors of c0t
  if (launch_recorder()) {
    record_span("transpose: c0", ct, 0, (uint64_t)L * N * 8);
    record_span("transpose: c0t", R->c0t, 0, (uint64_t)L * N * 8);
  } else {
    hipLaunchKernelGGL(fiona::transpose_kernel, dim3((N + 255) / 256, L), dim3(256), 0, stream, ct, R->c0t,
                       R->log_n1, R->log_n2);
  }

  // 2. the inner products of every rotation (transposed layout, pi^-1 frame)
  //    (batches of 8 digits, or of 4 where that pads fewer: L = 8, 16 take 8, L = 10, 12 take 4)
  const dim3 ks_grid(M * (N / fiona::kKsTile));
  const uint32_t round = fiona::ks_round(L);
  const size_t ks_smem = fiona::ks_lds_bytes(L, round);
  const uint32_t pad8 = (L + 7) / 8 * 8 - L, pad4 = (L + 3) / 4 * 4 - L;
  // ks_inner_kernel: digits (j < L, m < M, 16 bytes per lane pair), keys of
  // rotations r < n_rot (digit j, polynomial p, modulus m), u' of every
  // rotation, the limb constants of every modulus
  const uint64_t key_words = (uint64_t)L * 2 * M * N;
  if (launch_recorder()) {
    record_span("ks_inner: Dhat", R->Dhat, 0, (uint64_t)L * M * N * 8);
    record_span("ks_inner: keys", keys, 0, (uint64_t)n_rot * key_words * 8);
    record_span("ks_inner: U", R->U, 0, (uint64_t)2 * n_rot * M * N * 8);
    record_span("ks_inner: limbs", R->limbs, 0, (uint64_t)M * sizeof(fiona::LimbConst));
  } else if (pad8 <= pad4) {
    hipLaunchKernelGGL(fiona::ks_inner_kernel<8>, ks_grid, dim3(fiona::kKsWaves * 64), ks_smem, stream, R->Dhat, keys,
                       R->U, R->limbs, N, L, n_rot, round);
  } else {
    hipLaunchKernelGGL(fiona::ks_inner_kernel<4>, ks_grid, dim3(fiona::kKsWaves * 64), ks_smem, stream, R->Dhat,
                       keys, R->U, R->limbs, N, L, n_rot, round);
  }

  // 3. the division by P: u'_P back to centred coefficients (W), then per
  //    data limb its transform, the subtraction from u', the product with
  //    P^-1, c0 for the first polynomials and the automorphism, written to out
  const uint32_t V = 2 * n_rot;
  NttPass C{};
  C.sets = R->p_inv_set;
  C.vps = V;
  C.log_n1 = R->log_n1;
  C.log_n2 = R->log_n2;
  C.in = R->U + (size_t)L * N;
  C.in_end = R->U_end;
  C.in_stride = (size_t)M * N;
  C.tmp = R->T;
  C.tmp_end = R->T_end;
  C.out = R->W;
  C.out_end = R->W_end;
  C.out_stride = N;
  C.load = fiona::kLoadU64T;
  C.store = fiona::kStoreF64;
  launch_transform(R->log_n1, R->log_n2, V, stream, C);
  NttPass Q{};
  Q.sets = R->down_sets;
  Q.vps = V;
  Q.log_n1 = R->log_n1;
  Q.log_n2 = R->log_n2;
  Q.in = R->W;
  Q.in_end = R->W_end;
  Q.in_stride = N;
  Q.tmp = R->T;
  Q.tmp_end = R->T_end;
  Q.out = out_cts;
  Q.out_end = out_end;
  Q.base = R->U;
  Q.base_end = R->U_end;
  Q.base_stride = (size_t)M * N;
  Q.base_set_stride = N;
  Q.add = R->c0t;
  Q.add_end = R->c0t_end;
  Q.add_set_stride = N;
  Q.load = fiona::kLoadF64;
  const uint32_t col_blocks = (1u << R->log_n1) / fiona::kNttCols;
  Q.nsets_shared = L > 1 && (col_blocks * V) % 8 == 0 ? L : 0;
  launch_pass(true, R->log_n2, R->log_n1, L * V, stream, Q);
  fiona::RotArgs G{};
  for (uint32_t r = 0; r < n_rot; ++r) G.g[r] = galois[r];
  G.n_rot = n_rot;
  G.L = L;
  launch_rot_pass_b(R->log_n1, R->log_n2, L * V, stream, Q, G);
}

}  // namespace

namespace fiona_host {

// A rotator laid out at fake device addresses, one call with n_rot
// rotations recorded (Galois elements 5^r mod 2N for r = 1 .. n_rot - 2,
// then the conjugation 2N - 1 and the identity 1) and every access of its
// launches checked; the output region is out_shrink bytes short.
int rotate_replay(const uint64_t *moduli, uint32_t N, uint32_t L, uint32_t max_rot, uint32_t n_rot,
                  uint64_t out_shrink, std::string &err) {
  fiona_ctx *ctx = nullptr;
  int rc = fiona_ctx_create(N, L, moduli, &ctx);
  if (rc != FIONA_OK) return rc;
  fiona_rotator R;
  TableImage img;
  size_t total = 0;
  rc = rotator_layout(ctx, moduli[L], nullptr, max_rot, &R, img, total);
  if (rc == FIONA_OK && (n_rot == 0 || n_rot > max_rot)) rc = FIONA_ERR_ARG;
  if (rc != FIONA_OK) {
    fiona_ctx_destroy(R.ext);
    fiona_ctx_destroy(ctx);
    return rc;
  }
  std::vector<uint32_t> galois(n_rot);
  uint64_t g = 1;
  for (uint32_t r = 0; r < n_rot; ++r) {
    g = g * 5 % (2ull * N);
    galois[r] = (uint32_t)g;
  }
  if (n_rot >= 2) galois[n_rot - 2] = 2 * N - 1;
  galois[n_rot - 1] = 1;
  // (each starts with bit 31 of its low address half set: the replay
  // rebuilds every descriptor base from its halves as the kernels do)
  const uint64_t kGap = 1ull << 44, kLow = 0x80000000ull;
  char *dev = (char *)(uintptr_t)(1 * kGap + kLow);
  const uint64_t *ct = (const uint64_t *)(uintptr_t)(2 * kGap + kLow);
  const uint64_t *keys = (const uint64_t *)(uintptr_t)(3 * kGap + kLow);
  uint64_t *out = (uint64_t *)(uintptr_t)(4 * kGap + kLow);
  rotator_place(&R, img, dev);
  std::vector<Region> regions = table_regions(img, dev);
  regions.push_back(Region{(uint64_t)R.limbs, (uint64_t)R.limbs + (L + 1) * sizeof(fiona::LimbConst), "limbs"});
  regions.push_back(Region{(uint64_t)R.D, (uint64_t)R.D_end, "D"});
  regions.push_back(Region{(uint64_t)R.Dhat, (uint64_t)R.Dhat_end, "Dhat"});
  regions.push_back(Region{(uint64_t)R.c0t, (uint64_t)R.c0t_end, "c0t"});
  regions.push_back(Region{(uint64_t)R.T, (uint64_t)R.T_end, "T"});
  regions.push_back(Region{(uint64_t)R.W, (uint64_t)R.W_end, "W"});
  regions.push_back(Region{(uint64_t)R.U, (uint64_t)R.U_end, "U"});
  regions.push_back(Region{(uint64_t)ct, (uint64_t)(ct + (size_t)2 * L * N), "ct"});
  regions.push_back(Region{(uint64_t)keys, (uint64_t)(keys + (size_t)n_rot * fiona_rotation_key_words(&R)), "keys"});
  regions.push_back(Region{(uint64_t)out, (uint64_t)(out + (size_t)n_rot * 2 * L * N) - out_shrink, "out_cts"});
  LaunchRecord rec;
  launch_recorder() = &rec;
  rotate_enqueue(&R, ct, n_rot, galois.data(), keys, out, nullptr);
  launch_recorder() = nullptr;
  err = check_launches(rec, regions, (uint64_t)img.sets_addr(dev), img.sets_at(dev));
  fiona_ctx_destroy(R.ext);
  fiona_ctx_destroy(ctx);
  return err.empty() ? FIONA_OK : FIONA_ERR_BOUNDS;
}

}  // namespace fiona_host

extern "C" {

int fiona_rotator_create(const fiona_ctx *ctx, uint64_t special_prime, const uint64_t *psi, uint32_t max_rot,
                         fiona_rotator **out) {
  if (!out) return FIONA_ERR_ARG;
  *out = nullptr;
  if (!ctx) return FIONA_ERR_ARG;
  fiona_rotator *R = new (std::nothrow) fiona_rotator;
  if (!R) return FIONA_ERR_NOMEM;
  try {
    TableImage img;
    size_t total = 0;
    const int rc = rotator_layout(ctx, special_prime, psi, max_rot, R, img, total);
    if (rc != FIONA_OK) {
      fiona_rotator_destroy(R);
      return rc;
    }
    if (hipGetDevice(&R->device) != hipSuccess) {
      fiona_rotator_destroy(R);
      return FIONA_ERR_HIP;
    }
    void *dev = nullptr;
    if (hipMalloc(&dev, total) != hipSuccess) {
      fiona_rotator_destroy(R);
      return FIONA_ERR_NOMEM;
    }
    rotator_place(R, img, dev);
    if (!img.upload(R->dev) || hipMemcpy((void *)R->limbs, R->ext->limbs.data(),
                                         (R->L + 1) * sizeof(fiona::LimbConst), hipMemcpyHostToDevice) != hipSuccess) {
      fiona_rotator_destroy(R);
      return FIONA_ERR_HIP;
    }
    const int ks_smem = (int)fiona::ks_lds_bytes(R->L, fiona::ks_round(R->L));
    const int nt_smem = (int)(fiona::kNttCols * fiona::padded_len(fiona::kNttMaxSide) * sizeof(double) +
                              fiona::kNttMaxSide / 2 * sizeof(Tw));
    if (!allow_smem() || !allow_rot_smem(nt_smem) ||
        hipFuncSetAttribute((const void *)fiona::ks_inner_kernel<8>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            ks_smem) != hipSuccess ||
        hipFuncSetAttribute((const void *)fiona::ks_inner_kernel<4>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            ks_smem) != hipSuccess) {
      fiona_rotator_destroy(R);
      return FIONA_ERR_HIP;
    }
  } catch (...) {
    fiona_rotator_destroy(R);
    return FIONA_ERR_NOMEM;
  }
  *out = R;
  return FIONA_OK;
}

void fiona_rotator_destroy(fiona_rotator *R) {
  if (!R) return;
  if (R->dev) (void)hipFree(R->dev);
  fiona_ctx_destroy(R->ext);
  delete R;
}

uint64_t fiona_rotation_key_words(const fiona_rotator *R) {
  return R ? (uint64_t)R->L * 2 * (R->L + 1) * R->N : 0;
}

int fiona_rotation_key_layout(const fiona_rotator *R, uint32_t galois, const uint64_t *key, uint64_t *key_out,
                              hipStream_t stream) {
  if (!R || !key || !key_out) return FIONA_ERR_ARG;
  const uint32_t N = R->N;
  if ((galois & 1u) == 0 || galois >= 2 * N) return FIONA_ERR_ARG;
  if (((uintptr_t)key | (uintptr_t)key_out) & 7u) return FIONA_ERR_ALIGN;
  const size_t words = fiona_rotation_key_words(R);
  if (overlap(key, words * 8, key_out, words * 8)) return FIONA_ERR_ALIAS;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != R->device) return FIONA_ERR_ARG;
  uint32_t ginv = 1;   // g^-1 mod N by Newton's iteration (g odd, N a power of two)
  for (int i = 0; i < 5; ++i) ginv *= 2u - galois * ginv;
  const uint32_t rows = R->L * 2 * (R->L + 1);
  hipLaunchKernelGGL(fiona::key_layout_kernel, dim3(N / 256, rows), dim3(256), 0, stream, key, key_out, R->log_n1,
                     R->log_n2, rows, galois, ginv & (N - 1));
  return hipGetLastError() == hipSuccess ? FIONA_OK : FIONA_ERR_HIP;
}

int fiona_hoisted_rotate(const fiona_rotator *R, const uint64_t *ct, uint32_t n_rot, const uint32_t *galois,
                         const uint64_t *keys, uint64_t *out_cts, hipStream_t stream) {
  if (!R) return FIONA_ERR_ARG;
  if (n_rot == 0) return FIONA_OK;
  if (!ct || !galois || !keys || !out_cts || n_rot > R->max_rot) return FIONA_ERR_ARG;
  const uint32_t N = R->N, L = R->L;
  for (uint32_t r = 0; r < n_rot; ++r)
    if ((galois[r] & 1u) == 0 || galois[r] >= 2 * N) return FIONA_ERR_ARG;
  if ((((uintptr_t)ct | (uintptr_t)out_cts) & 7u) || ((uintptr_t)keys & 15u)) return FIONA_ERR_ALIGN;
  const size_t ct_bytes = (size_t)2 * L * N * 8, out_bytes = (size_t)n_rot * ct_bytes;
  const size_t key_bytes = (size_t)n_rot * fiona_rotation_key_words(R) * 8;
  if (overlap(out_cts, out_bytes, ct, ct_bytes) || overlap(out_cts, out_bytes, keys, key_bytes))
    return FIONA_ERR_ALIAS;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != R->device) return FIONA_ERR_ARG;
  rotate_enqueue(R, ct, n_rot, galois, keys, out_cts, stream);
  return hipGetLastError() == hipSuccess ? FIONA_OK : FIONA_ERR_HIP;
}

}  // extern "C"
