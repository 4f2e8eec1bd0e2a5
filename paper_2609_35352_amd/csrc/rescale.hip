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
#include "ntt_host.hpp"

using namespace fiona_host;

constexpr size_t kMaxTmpBytes = (size_t)8 << 30;   // cap on the intermediates of one launch pair


struct fiona_rescaler {
  const fiona_ctx *ctx = nullptr;
  uint32_t N = 0, L = 0, log_n1 = 0, log_n2 = 0, max_ct = 0;
  uint32_t limbs_per_launch = 1;   // forward limbs transformed together (room for them in T)
  int device = -1;
  void *dev = nullptr;
  const NttSet *sets = nullptr;  // limbs 0 .. L-2 forward (inv = q_t^-1 mod q_l), then limb L-1 inverse
  double *W = nullptr;           // the centred remainders [INTT_t(in_t)], one vector per polynomial
  double *T = nullptr;           // the transposed intermediate of the passes
  const void *W_end = nullptr, *T_end = nullptr;
};

namespace {

// Checks the parameters and sizes a rescaler: its tables (img) and the
// bytes of its device buffer (the table image, then W and T).
int rescaler_layout(const fiona_ctx *ctx, const uint64_t *psi, uint32_t max_ct, fiona_rescaler *R,
                    TableImage &img, size_t &total) {
  if (max_ct == 0) return FIONA_ERR_ARG;
  if (2ull * max_ct > 65535) return FIONA_ERR_UNSUPPORTED;   // a launch holds at most 65535 vectors
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
  R->ctx = ctx;
  R->N = N;
  R->L = L;
  R->log_n1 = (logN + 1) / 2;
  R->log_n2 = logN / 2;
  R->max_ct = max_ct;
  // every table of every limb and the set records, then the workspace
  const uint64_t qt = ctx->q[L - 1];
  for (uint32_t l = 0; l + 1 < L; ++l) {
    const uint64_t q = ctx->q[l];
    img.add(make_tables(R->log_n1, R->log_n2, q, roots[l], false), q, make_tw(powmod_h(qt % q, q - 2, q), q));
  }
  img.add(make_tables(R->log_n1, R->log_n2, qt, roots[L - 1], true), qt);
  const size_t vec_bytes = (size_t)2 * max_ct * N * sizeof(double);
  // All forward limbs go in one launch pair, so T holds L - 1 intermediates.
  // Measured against one limb per launch (in-process A/B, same buffers):
  // 256 vectors (VGG11's outputs) 1.25 -> 1.18 ms, 192 (BERT's) 1.32 -> 1.30.
  // Very large max_ct takes fewer limbs per launch, so that T stays within
  // kMaxTmpBytes (and every launch within the grid's 65535 vectors).
  const size_t fit = kMaxTmpBytes / vec_bytes;
  const size_t fit_grid = 65535 / (2 * (size_t)max_ct);
  size_t lpl = L - 1;
  if (lpl > fit) lpl = fit;
  if (lpl > fit_grid) lpl = fit_grid;
  R->limbs_per_launch = lpl < 1 ? 1 : (uint32_t)lpl;
  total = img.bytes() + (1 + R->limbs_per_launch) * vec_bytes;
  return FIONA_OK;
}

// Points the rescaler's parts into its device buffer at dev.
void rescaler_place(fiona_rescaler *R, const TableImage &img, void *dev) {
  const size_t vec_bytes = (size_t)2 * R->max_ct * R->N * sizeof(double);
  R->dev = dev;
  R->sets = img.sets_addr(dev);
  R->W = (double *)((char *)dev + img.bytes());
  R->T = (double *)((char *)dev + img.bytes() + vec_bytes);
  R->W_end = (const char *)R->W + vec_bytes;
  R->T_end = (const char *)R->T + R->limbs_per_launch * vec_bytes;
}

// The launches of one rescale (arguments already checked).
void rescale_enqueue(const fiona_rescaler *R, const uint64_t *in_cts, uint32_t n_ct, uint64_t *out_cts,
                     hipStream_t stream) {
  const size_t N = R->N, L = R->L;
  const uint32_t V = 2 * n_ct;
  const void *in_end = in_cts + (size_t)n_ct * 2 * L * N, *out_end = out_cts + (size_t)n_ct * 2 * (L - 1) * N;

  // 1. the last limb back to its coefficients, kept as centred residues mod q_t
  NttPass P{};
  P.sets = R->sets + (L - 1);
  P.vps = V;
  P.log_n1 = R->log_n1;
  P.log_n2 = R->log_n2;
  P.in = in_cts + (L - 1) * N;
  P.in_end = in_end;
  P.in_stride = L * N;
  P.tmp = R->T;
  P.tmp_end = R->T_end;
  P.out = R->W;
  P.out_end = R->W_end;
  P.out_stride = N;
  P.load = fiona::kLoadU64;
  P.store = fiona::kStoreF64;
  launch_transform(R->log_n1, R->log_n2, V, stream, P);

  // 2. every other limb: the centred remainder (a signed integer, so its
  //    residue mod q_l comes with the first product) into its NTT domain,
  //    subtracted, multiplied by q_t^-1; all limbs in one launch pair (one
  //    set per limb, the vectors of a set share its modulus), pass A in the
  //    order that fetches each input block once per XCD
  const uint32_t lpl = R->limbs_per_launch;
  for (uint32_t l0 = 0; l0 + 1 < L; l0 += lpl) {
    const uint32_t nl = (uint32_t)(L - 1 - l0) < lpl ? (uint32_t)(L - 1 - l0) : lpl;
    NttPass Q{};
    Q.sets = R->sets + l0;
    Q.vps = V;
    Q.log_n1 = R->log_n1;
    Q.log_n2 = R->log_n2;
    Q.in = R->W;
    Q.in_end = R->W_end;
    Q.in_stride = N;
    Q.tmp = R->T;
    Q.tmp_end = R->T_end;
    Q.out = out_cts + l0 * N;
    Q.out_end = out_end;
    Q.out_stride = (L - 1) * N;
    Q.out_set_stride = N;
    Q.base = in_cts + l0 * N;
    Q.base_end = in_end;
    Q.base_stride = L * N;
    Q.base_set_stride = N;
    Q.load = fiona::kLoadF64;
    Q.store = fiona::kStoreRescale;
    const uint32_t col_blocks = (1u << R->log_n1) / fiona::kNttCols;
    Q.nsets_shared = nl > 1 && (col_blocks * V) % 8 == 0 ? nl : 0;
    launch_transform(R->log_n1, R->log_n2, nl * V, stream, Q);
  }
}

}  // namespace

namespace fiona_host {

// A rescaler laid out at fake device addresses, one rescale of n_ct
// ciphertexts recorded and every access of its launches checked.  The
// caller's output region is out_shrink bytes short of its size (a check of
// the checker).
int rescale_replay(const uint64_t *moduli, uint32_t N, uint32_t L, uint32_t max_ct, uint32_t n_ct,
                   uint64_t out_shrink, std::string &err) {
  fiona_ctx *ctx = nullptr;
  int rc = fiona_ctx_create(N, L, moduli, &ctx);
  if (rc != FIONA_OK) return rc;
  fiona_rescaler R;
  TableImage img;
  size_t total = 0;
  rc = rescaler_layout(ctx, nullptr, max_ct, &R, img, total);
  if (rc == FIONA_OK && (n_ct == 0 || n_ct > max_ct)) rc = FIONA_ERR_ARG;
  if (rc != FIONA_OK) {
    fiona_ctx_destroy(ctx);
    return rc;
  }
  // separate fake allocations, 2^44 bytes apart
  // (each starts with bit 31 of its low address half set: the replay
  // rebuilds every descriptor base from its halves as the kernels do)
  const uint64_t kGap = 1ull << 44, kLow = 0x80000000ull;
  char *dev = (char *)(uintptr_t)(1 * kGap + kLow);
  const uint64_t *in = (const uint64_t *)(uintptr_t)(2 * kGap + kLow);
  uint64_t *out = (uint64_t *)(uintptr_t)(3 * kGap + kLow);
  rescaler_place(&R, img, dev);
  std::vector<Region> regions = table_regions(img, dev);
  regions.push_back(Region{(uint64_t)R.W, (uint64_t)R.W_end, "rescaler W"});
  regions.push_back(Region{(uint64_t)R.T, (uint64_t)R.T_end, "rescaler T"});
  regions.push_back(Region{(uint64_t)in, (uint64_t)(in + (size_t)n_ct * 2 * L * N), "in_cts"});
  regions.push_back(Region{(uint64_t)out, (uint64_t)(out + (size_t)n_ct * 2 * (L - 1) * N) - out_shrink, "out_cts"});
  LaunchRecord rec;
  launch_recorder() = &rec;
  rescale_enqueue(&R, in, n_ct, out, nullptr);
  launch_recorder() = nullptr;
  err = check_launches(rec, regions, (uint64_t)R.sets, img.sets_at(dev));
  fiona_ctx_destroy(ctx);
  return err.empty() ? FIONA_OK : FIONA_ERR_BOUNDS;
}

}  // namespace fiona_host

extern "C" {

int fiona_rescaler_create(const fiona_ctx *ctx, const uint64_t *psi, uint32_t max_ct, fiona_rescaler **out) {
  if (!out) return FIONA_ERR_ARG;
  *out = nullptr;
  if (!ctx) return FIONA_ERR_ARG;
  fiona_rescaler *R = new (std::nothrow) fiona_rescaler;
  if (!R) return FIONA_ERR_NOMEM;
  try {
    TableImage img;
    size_t total = 0;
    const int rc = rescaler_layout(ctx, psi, max_ct, R, img, total);
    if (rc != FIONA_OK) {
      delete R;
      return rc;
    }
    if (hipGetDevice(&R->device) != hipSuccess) {
      delete R;
      return FIONA_ERR_HIP;
    }
    void *dev = nullptr;
    if (hipMalloc(&dev, total) != hipSuccess) {
      delete R;
      return FIONA_ERR_NOMEM;
    }
    rescaler_place(R, img, dev);
    if (!img.upload(R->dev) || !allow_smem()) {
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
  rescale_enqueue(R, in_cts, n_ct, out_cts, stream);
  if (hipGetLastError() != hipSuccess) return FIONA_ERR_HIP;
  return FIONA_OK;
}

}  // extern "C"
