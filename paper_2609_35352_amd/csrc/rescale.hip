// Host side of the rescale epilogue (include/fiona.h): twiddle tables, the
// workspace and the launches of the NTT passes in ntt_kernel.hpp.
//
// Rescaling (paper Sec. 2, "Levels and Bootstrapping"; applied once per output
// after its routes are summed, Sec. 4.2 "Combining the Signed and Raw Routes")
// divides each coefficient's integer by the last modulus q_t = q_{L-1} with
// rounding.  In RNS form, for every other limb l:
//     out_l = (in_l - NTT_l([INTT_t(in_t)]_centred mod q_l)) * q_t^-1  mod q_l,
// where the centred remainder r in (-q_t/2, q_t/2] makes (C - r) / q_t the
// rounded quotient.  Only the last limb leaves the NTT domain.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

#include "fiona.h"
#include "fiona_ctx.hpp"
#include "ntt_kernel.hpp"

using fiona::NttPass;
using fiona::Tw;

namespace {

uint64_t mulmod_h(uint64_t a, uint64_t b, uint64_t q) { return (uint64_t)((unsigned __int128)a * b % q); }

uint64_t powmod_h(uint64_t b, uint64_t e, uint64_t q) {
  uint64_t r = 1 % q;
  b %= q;
  while (e) {
    if (e & 1) r = mulmod_h(r, b, q);
    b = mulmod_h(b, b, q);
    e >>= 1;
  }
  return r;
}

Tw make_tw(uint64_t w, uint64_t q) { return Tw{(double)w, (double)w / (double)q}; }

// The default root: psi = x^((q-1)/2N) for the smallest x >= 2 with psi^N = -1.
uint64_t default_psi(uint32_t N, uint64_t q) {
  for (uint64_t x = 2; x < 1000000; ++x) {
    const uint64_t psi = powmod_h(x, (q - 1) / (2ull * N), q);
    if (powmod_h(psi, N, q) == q - 1) return psi;
  }
  return 0;
}

// Tables of one direction of one limb.  Forward: pre = psi^n, mid = omega^(n1 k2) at k2 N1 + n1,
// DFT roots omega^N1 (size N2) and omega^N2 (size N1).  Inverse: omega -> omega^-1,
// no pre, post = N^-1 psi^-k.
struct TableSet {
  std::vector<Tw> pre, mid, dft_a, dft_b, post;
};

TableSet make_tables(uint32_t log_n1, uint32_t log_n2, uint64_t q, uint64_t psi, bool inverse) {
  const uint32_t N1 = 1u << log_n1, N2 = 1u << log_n2, N = N1 * N2;
  const uint64_t psi_inv = powmod_h(psi, q - 2, q);
  const uint64_t omega = inverse ? mulmod_h(psi_inv, psi_inv, q) : mulmod_h(psi, psi, q);
  TableSet t;
  if (!inverse) {
    t.pre.resize(N);
    uint64_t p = 1;
    for (uint32_t n = 0; n < N; ++n, p = mulmod_h(p, psi, q)) t.pre[n] = make_tw(p, q);
  } else {
    t.post.resize(N);
    uint64_t p = powmod_h(N, q - 2, q);
    for (uint32_t n = 0; n < N; ++n, p = mulmod_h(p, psi_inv, q)) t.post[n] = make_tw(p, q);
  }
  t.mid.resize(N);
  for (uint32_t n1 = 0; n1 < N1; ++n1) {
    const uint64_t step = powmod_h(omega, n1, q);
    uint64_t p = 1;
    for (uint32_t k2 = 0; k2 < N2; ++k2, p = mulmod_h(p, step, q)) t.mid[(size_t)k2 * N1 + n1] = make_tw(p, q);
  }
  const uint64_t w2 = powmod_h(omega, N1, q), w1 = powmod_h(omega, N2, q);
  t.dft_a.resize(N2 / 2);
  uint64_t p = 1;
  for (uint32_t i = 0; i < N2 / 2; ++i, p = mulmod_h(p, w2, q)) t.dft_a[i] = make_tw(p, q);
  t.dft_b.resize(N1 / 2);
  p = 1;
  for (uint32_t i = 0; i < N1 / 2; ++i, p = mulmod_h(p, w1, q)) t.dft_b[i] = make_tw(p, q);
  return t;
}

// The passes are instantiated per DFT side 2^4 .. 2^9.
template <uint32_t LOG>
void launch_pair(bool a, dim3 grid, size_t smem, hipStream_t stream, const NttPass &P) {
  if (a) hipLaunchKernelGGL(fiona::ntt_pass_a<LOG>, grid, dim3(fiona::kNttThreads), smem, stream, P);
  else hipLaunchKernelGGL(fiona::ntt_pass_b<LOG>, grid, dim3(fiona::kNttThreads), smem, stream, P);
}

void launch_pass(bool a, uint32_t log_side, dim3 grid, hipStream_t stream, const NttPass &P) {
  const size_t smem = fiona::kNttCols * fiona::padded_len(1u << log_side) * sizeof(double) +
                      (1u << log_side) / 2 * sizeof(Tw);
  switch (log_side) {
    case 4: launch_pair<4>(a, grid, smem, stream, P); break;
    case 5: launch_pair<5>(a, grid, smem, stream, P); break;
    case 6: launch_pair<6>(a, grid, smem, stream, P); break;
    case 7: launch_pair<7>(a, grid, smem, stream, P); break;
    case 8: launch_pair<8>(a, grid, smem, stream, P); break;
    default: launch_pair<9>(a, grid, smem, stream, P); break;
  }
}

template <uint32_t LOG>
bool allow_smem(int bytes) {
  return hipFuncSetAttribute((const void *)fiona::ntt_pass_a<LOG>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             bytes) == hipSuccess &&
         hipFuncSetAttribute((const void *)fiona::ntt_pass_b<LOG>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             bytes) == hipSuccess;
}

struct LimbTables {
  const Tw *pre = nullptr, *mid = nullptr, *dft_a = nullptr, *dft_b = nullptr, *post = nullptr;
};

}  // namespace

struct fiona_rescaler {
  const fiona_ctx *ctx = nullptr;
  uint32_t N = 0, L = 0, log_n1 = 0, log_n2 = 0, max_ct = 0;
  int device = -1;
  void *dev = nullptr;
  std::vector<LimbTables> fwd;   // limbs 0 .. L-2
  LimbTables inv;                // limb L-1
  std::vector<Tw> inv_qt;        // q_t^-1 mod q_l
  double *W = nullptr;           // the centred remainders [INTT_t(in_t)], one vector per polynomial
  double *T = nullptr;           // the transposed intermediate of the passes
};

extern "C" {

int fiona_rescaler_create(const fiona_ctx *ctx, const uint64_t *psi, uint32_t max_ct, fiona_rescaler **out) {
  if (!out) return FIONA_ERR_ARG;
  *out = nullptr;
  if (!ctx || max_ct == 0) return FIONA_ERR_ARG;
  const uint32_t N = ctx->N, L = ctx->L;
  uint32_t logN = 0;
  while ((1u << logN) < N) ++logN;
  if ((1u << logN) != N || logN < 8 || logN > 17 || L < 2) return FIONA_ERR_UNSUPPORTED;
  std::vector<uint64_t> roots(L);
  for (uint32_t l = 0; l < L; ++l) {
    const uint64_t q = ctx->q[l];
    if ((q - 1) % (2ull * N) != 0) return FIONA_ERR_UNSUPPORTED;
    roots[l] = psi ? psi[l] % q : default_psi(N, q);
    if (roots[l] == 0 || powmod_h(roots[l], N, q) != q - 1) return FIONA_ERR_UNSUPPORTED;
  }
  fiona_rescaler *R = new (std::nothrow) fiona_rescaler;
  if (!R) return FIONA_ERR_NOMEM;
  R->ctx = ctx;
  R->N = N;
  R->L = L;
  R->log_n1 = (logN + 1) / 2;
  R->log_n2 = logN / 2;
  R->max_ct = max_ct;
  try {
    // every table of every limb, then the workspace, in one device buffer
    std::vector<TableSet> sets;
    for (uint32_t l = 0; l + 1 < L; ++l) sets.push_back(make_tables(R->log_n1, R->log_n2, ctx->q[l], roots[l], false));
    sets.push_back(make_tables(R->log_n1, R->log_n2, ctx->q[L - 1], roots[L - 1], true));
    std::vector<Tw> all;
    struct Off { size_t pre, mid, dft_a, dft_b, post; };
    std::vector<Off> offs;
    auto put = [&](const std::vector<Tw> &v) {
      const size_t o = all.size();
      all.insert(all.end(), v.begin(), v.end());
      return v.empty() ? (size_t)-1 : o;
    };
    for (auto &t : sets) offs.push_back(Off{put(t.pre), put(t.mid), put(t.dft_a), put(t.dft_b), put(t.post)});
    const size_t table_bytes = (all.size() * sizeof(Tw) + 255) / 256 * 256;
    const size_t vec_bytes = (size_t)2 * max_ct * N * sizeof(double);
    if (hipGetDevice(&R->device) != hipSuccess) {
      delete R;
      return FIONA_ERR_HIP;
    }
    if (hipMalloc(&R->dev, table_bytes + 2 * vec_bytes) != hipSuccess) {
      R->dev = nullptr;
      delete R;
      return FIONA_ERR_NOMEM;
    }
    if (hipMemcpy(R->dev, all.data(), all.size() * sizeof(Tw), hipMemcpyHostToDevice) != hipSuccess) {
      fiona_rescaler_destroy(R);
      return FIONA_ERR_HIP;
    }
    const Tw *tb = (const Tw *)R->dev;
    auto at = [&](size_t o) { return o == (size_t)-1 ? nullptr : tb + o; };
    for (uint32_t l = 0; l < L; ++l) {
      LimbTables lt{at(offs[l].pre), at(offs[l].mid), at(offs[l].dft_a), at(offs[l].dft_b), at(offs[l].post)};
      if (l + 1 < L) R->fwd.push_back(lt);
      else R->inv = lt;
    }
    R->W = (double *)((char *)R->dev + table_bytes);
    R->T = (double *)((char *)R->dev + table_bytes + vec_bytes);
    const uint64_t qt = ctx->q[L - 1];
    for (uint32_t l = 0; l + 1 < L; ++l) {
      const uint64_t q = ctx->q[l];
      R->inv_qt.push_back(make_tw(powmod_h(qt % q, q - 2, q), q));
    }
    const int smem = (int)(fiona::kNttCols * fiona::padded_len(fiona::kNttMaxSide) * sizeof(double) +
                           fiona::kNttMaxSide / 2 * sizeof(Tw));
    if (!allow_smem<4>(smem) || !allow_smem<5>(smem) || !allow_smem<6>(smem) || !allow_smem<7>(smem) ||
        !allow_smem<8>(smem) || !allow_smem<9>(smem)) {
      fiona_rescaler_destroy(R);
      return FIONA_ERR_HIP;
    }
  } catch (...) {
    fiona_rescaler_destroy(R);
    return FIONA_ERR_NOMEM;
  }
  *out = R;
  return FIONA_OK;
}

void fiona_rescaler_destroy(fiona_rescaler *R) {
  if (!R) return;
  if (R->dev) (void)hipFree(R->dev);
  delete R;
}

int fiona_rescale(const fiona_rescaler *R, const uint64_t *in_cts, uint32_t n_ct, uint64_t *out_cts,
                  hipStream_t stream) {
  if (!R) return FIONA_ERR_ARG;
  if (n_ct == 0) return FIONA_OK;
  if (!in_cts || !out_cts || n_ct > R->max_ct) return FIONA_ERR_ARG;
  if (((uintptr_t)in_cts | (uintptr_t)out_cts) & 7u) return FIONA_ERR_ALIGN;
  const size_t N = R->N, L = R->L;
  const size_t in_bytes = (size_t)n_ct * 2 * L * N * 8, out_bytes = (size_t)n_ct * 2 * (L - 1) * N * 8;
  const uintptr_t a0 = (uintptr_t)in_cts, b0 = (uintptr_t)out_cts;
  if (a0 < b0 + out_bytes && b0 < a0 + in_bytes) return FIONA_ERR_ALIAS;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != R->device) return FIONA_ERR_ARG;
  const uint32_t V = 2 * n_ct, N1 = 1u << R->log_n1, N2 = 1u << R->log_n2;
  const dim3 grid_a(N1 / fiona::kNttCols, V), grid_b(N2 / fiona::kNttCols, V);

  // 1. the last limb back to its coefficients, kept as centred residues mod q_t
  const uint64_t qt = R->ctx->q[L - 1];
  NttPass P{};
  P.q = (double)qt;
  P.qinv = 1.0 / (double)qt;
  P.log_n1 = R->log_n1;
  P.log_n2 = R->log_n2;
  P.in = in_cts + (L - 1) * N;
  P.in_stride = L * N;
  P.tmp = R->T;
  P.out = R->W;
  P.out_stride = N;
  P.mid = R->inv.mid;
  P.dft_a = R->inv.dft_a;
  P.dft_b = R->inv.dft_b;
  P.post = R->inv.post;
  P.load = fiona::kLoadU64;
  P.store = fiona::kStoreF64;
  launch_pass(true, R->log_n2, grid_a, stream, P);
  launch_pass(false, R->log_n1, grid_b, stream, P);

  // 2. every other limb: the centred remainder (a signed integer, so its
  //    residue mod q_l comes with the first product) into its NTT domain,
  //    subtracted, multiplied by q_t^-1
  for (uint32_t l = 0; l + 1 < L; ++l) {
    NttPass Q{};
    Q.q = (double)R->ctx->q[l];
    Q.qinv = 1.0 / (double)R->ctx->q[l];
    Q.log_n1 = R->log_n1;
    Q.log_n2 = R->log_n2;
    Q.in = R->W;
    Q.in_stride = N;
    Q.tmp = R->T;
    Q.out = out_cts + l * N;
    Q.out_stride = (L - 1) * N;
    Q.base = in_cts + l * N;
    Q.base_stride = L * N;
    Q.pre = R->fwd[l].pre;
    Q.mid = R->fwd[l].mid;
    Q.dft_a = R->fwd[l].dft_a;
    Q.dft_b = R->fwd[l].dft_b;
    Q.inv = R->inv_qt[l];
    Q.load = fiona::kLoadF64;
    Q.store = fiona::kStoreRescale;
    launch_pass(true, R->log_n2, grid_a, stream, Q);
    launch_pass(false, R->log_n1, grid_b, stream, Q);
  }
  if (hipGetLastError() != hipSuccess) return FIONA_ERR_HIP;
  return FIONA_OK;
}

}  // extern "C"
