// Negacyclic NTT passes for gfx950 and the rescale epilogue built on them.
//
// Convention (the NTT domain the library's ciphertexts live in):
//     a_hat_k = sum_n a_n psi^((2k+1) n)  mod q,   k = 0 .. N-1 in natural order,
// psi a primitive 2N-th root of unity mod q.  With omega = psi^2 this is the
// cyclic DFT of the twisted sequence a_n psi^n; its inverse is
//     a_n = N^-1 psi^-n sum_k a_hat_k omega^(-nk).
//
// Both run as a four-step transform, N = N1 * N2 (256 x 256 for N = 2^16):
// index n = n1 + N1 n2 on the input side and k = k2 + N2 k1 on the output
// side, so that omega^(nk) = omega^(n1 k2) (omega^N2)^(n1 k1) (omega^N1)^(n2 k2).
//   pass A: for each n1, a DFT of size N2 over n2 (optionally after a
//           multiplication of each input by pre[n]), then a multiplication by
//           mid[n1 N2 + k2] = omega^(n1 k2); stored transposed as T[k2 N1 + n1];
//   pass B: for each k2, a DFT of size N1 over n1, giving output k2 + N2 k1.
// A workgroup takes kCols columns (pass A) or rows (pass B) at once, so every
// global access is a run of kCols consecutive words; the DFTs run in LDS
// (radix 2, input in bit-reversed order, output natural), up to four stages
// at a time in registers.
//
// Arithmetic is in fp64, on exact integers (q < 2^50): a double holds any
// integer below 2^53, and gfx950 issues fp64 FMA at full rate where 32-bit
// integer multiplies run at quarter rate.  A modular product b * w follows the
// FMA method of van der Hoeven, Lecerf and Quintin ("Modular SIMD arithmetic in
// Mathemagix", 2016): h = fl(b w) and its exact error l = b w - h (one FMA);
// the quotient k = rint(b * w/q) from one FMA against a rounding constant;
// then b w - k q = (h - k q) + l exactly.  For |b| < 2^51 and 0 <= w < q the
// result r satisfies r = b w (mod q) and |r| <= q (1/2 + |b| 2^-54).  Values
// between stages are signed and lazily reduced; reduce() brings any |x| < 2^52
// to the exact centred residue, |x| <= (q-1)/2 (the FMA's error |x/q| 2^-53 is
// below 1/(2q), the distance from x/q to the nearest half-integer).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fiona {

constexpr uint32_t kNttCols = 16;      // columns (pass A) or rows (pass B) per workgroup
constexpr uint32_t kNttThreads = 256;
constexpr uint32_t kNttMaxSide = 512;  // N1, N2 <= 512: N <= 2^17

struct Tw {   // a twiddle w, an integer in [0, q), and fl(w / q)
  double w, wq;
};

// 1.5 * 2^52: adding it to |v| < 2^51 rounds v to the nearest integer.
constexpr double kRound = 6755399441055744.0;

__device__ __forceinline__ double mul_tw(double b, const Tw &t, double q) {
#pragma clang fp contract(off)
  const double h = b * t.w;
  const double l = __builtin_fma(b, t.w, -h);
  const double k = __builtin_fma(b, t.wq, kRound) - kRound;
  return __builtin_fma(-k, q, h) + l;
}

__device__ __forceinline__ double reduce(double x, double q, double qinv) {
#pragma clang fp contract(off)
  const double k = __builtin_fma(x, qinv, kRound) - kRound;
  return __builtin_fma(-k, q, x);
}

// x an integer, |x| < 2^52 -> its residue in [0, q)
__device__ __forceinline__ double canonical(double x, double q, double qinv) {
  const double z = reduce(x, q, qinv);
  return z < 0.0 ? z + q : z;
}

__device__ __forceinline__ double to_f64(uint64_t x) {   // x < 2^53
  return __builtin_fma((double)(uint32_t)(x >> 32), 4294967296.0, (double)(uint32_t)x);
}
__device__ __forceinline__ uint64_t to_u64(double y) {   // y an integer in [0, 2^53)
  const uint32_t hi = (uint32_t)(y * 0x1p-32);
  const uint32_t lo = (uint32_t)__builtin_fma(-(double)hi, 4294967296.0, y);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint32_t bit_reverse(uint32_t x, uint32_t bits) { return __brev(x) >> (32 - bits); }

// LDS layout of the kNttCols columns.  The 16 lanes of a quarter wave work on
// the same word of 16 different columns (the DFT's twiddle reads are then
// broadcasts), so the column stride is odd: those lanes fall into 16
// different banks.  Within a column one padding word follows every 16, so
// that 16 consecutive bit-reversed positions (the row loads of pass B) fall
// into different banks too.
__device__ __forceinline__ uint32_t pidx(uint32_t i) { return i + (i >> 4); }
__host__ __device__ constexpr uint32_t padded_len(uint32_t m) { return m + m / 16 + 1; }

// Stages s0 .. s0+R-1 of the radix-2 DFT for the groups of one 16-word item:
// a group is the 2^R words base + (u << s0) that these stages combine; the
// item holds 16 >> R groups, kept in registers across the R stages.
// Entries are |x| <= 0.57 q; every second stage and the last one end with a
// reduction.  A product's output is below 0.5 q (1 + 2^-3); the unit-twiddle
// butterflies of the first pass add their input unmultiplied, so a product's
// input stays below 1.2 q, every value below 2.3 q (< 2^52, within reduce's
// range), and the item leaves |x| <= q/2 behind.
template <int R>
__device__ __forceinline__ void dft_item(double *col, uint32_t logM, uint32_t s0, uint32_t item, const Tw *tw,
                                         double q, double qinv) {
  constexpr uint32_t S = 1u << R, G = 16u >> R;
#pragma unroll
  for (uint32_t g = 0; g < G; ++g) {
    const uint32_t gi = item * G + g;
    const uint32_t o = gi & ((1u << s0) - 1);
    const uint32_t base = ((gi >> s0) << (s0 + R)) + o;
    double r[S];
#pragma unroll
    for (uint32_t u = 0; u < S; ++u) r[u] = col[pidx(base + (u << s0))];
#pragma unroll
    for (uint32_t st = 0; st < (uint32_t)R; ++st) {
      const uint32_t hh = 1u << st, shift = logM - 1 - (s0 + st);
#pragma unroll
      for (uint32_t u0 = 0; u0 < S; ++u0) {
        if ((u0 & (2 * hh - 1)) >= hh) continue;
        const uint32_t pos = o + ((u0 & (hh - 1)) << s0);
        // in the first pass (s0 = 0, so o = 0) the butterflies with pos = 0
        // have the twiddle 1: no product (their t is at most the input bound)
        const bool unit = s0 == 0 && (u0 & (hh - 1)) == 0;
        const double a = r[u0], t = unit ? r[u0 + hh] : mul_tw(r[u0 + hh], tw[pos << shift], q);
        r[u0] = a + t;
        r[u0 + hh] = a - t;
      }
      if ((st & 1) || st + 1 == (uint32_t)R) {
#pragma unroll
        for (uint32_t u = 0; u < S; ++u) r[u] = reduce(r[u], q, qinv);
      }
    }
#pragma unroll
    for (uint32_t u = 0; u < S; ++u) col[pidx(base + (u << s0))] = r[u];
  }
}

// Radix-2 DFT of size M = 2^LOGM (16 <= M <= kNttMaxSide) on kNttCols
// columns held in LDS (column c at x + c * padded_len(M), loaded in
// bit-reversed order, entries |x| <= 0.57 q); natural order on return, each
// entry the centred residue.  tw[t] = w_M^t for t < M/2 (in LDS).  Up to four
// stages per pass over LDS, in registers; item it works on column
// it % kNttCols.
template <uint32_t LOGM>
__device__ __forceinline__ void lds_dft(double *x, const Tw *tw, double q, double qinv) {
  constexpr uint32_t M = 1u << LOGM, PM = padded_len(M), items = kNttCols * (M >> 4);
#pragma unroll
  for (uint32_t s0 = 0; s0 < LOGM; s0 += 4) {
    __syncthreads();
    for (uint32_t it = threadIdx.x; it < items; it += kNttThreads) {
      double *col = x + (it % kNttCols) * PM;
      const uint32_t item = it / kNttCols;
      if (LOGM - s0 >= 4) dft_item<4>(col, LOGM, s0, item, tw, q, qinv);
      else if (LOGM - s0 == 3) dft_item<3>(col, LOGM, s0, item, tw, q, qinv);
      else if (LOGM - s0 == 2) dft_item<2>(col, LOGM, s0, item, tw, q, qinv);
      else dft_item<1>(col, LOGM, s0, item, tw, q, qinv);
    }
  }
  __syncthreads();
}

// Copy the M/2 twiddles of the size-M DFT into LDS.
__device__ __forceinline__ void stage_twiddles(Tw *dst, const Tw *__restrict__ src, uint32_t logM) {
  for (uint32_t i = threadIdx.x; i < (1u << logM) / 2; i += kNttThreads) dst[i] = src[i];
}

// What a pass reads (pass A) and writes (pass B).
// The transposed layout of an N-word vector: element i = k2 + N2 k1
// (k2 < N2, k1 < N1, the split of the four-step transform's output) at
// k2 N1 + k1, so that one pass-B row k2 is N1 contiguous words.
enum NttLoad : uint32_t {
  kLoadU64 = 0,    // residues in [0, q) as uint64
  kLoadF64 = 1,    // signed integers as doubles, |x| < 2^49 (a centred residue of another modulus)
  kLoadU64T = 2,   // residues in [0, q) as uint64, each vector in the transposed layout (no pre)
};
enum NttStore : uint32_t {
  kStoreU64 = 0,      // the transform, residues in [0, q) as uint64
  kStoreF64 = 1,      // the transform, centred residues as doubles
  kStoreRescale = 2,  // (base - transform) * inv mod q, in [0, q) as uint64
};

// One modulus of a pass and its tables.
struct NttSet {
  const Tw *pre;     // pass A: multiply input n by pre[n] (null: by 1)
  const Tw *mid;     // pass A: mid[k2 N1 + n1] = omega^(n1 k2)
  const Tw *dft_a;   // size-N2 DFT twiddles (N2 / 2)
  const Tw *dft_b;   // size-N1 DFT twiddles (N1 / 2)
  const Tw *post;    // pass B: multiply output k by post[k] (null: by 1)
  Tw inv;            // kStoreRescale: the factor applied after the subtraction
  double q, qinv;    // the modulus and fl(1 / q)
};

// A launch covers vectors v = 0 .. gridDim.y - 1, grouped into sets of vps
// consecutive vectors that share one modulus: vector v is number v % vps of
// set v / vps, whose modulus and tables are sets[v / vps].  Its words sit at
//   in   + (v / vps) * in_set_stride   + (v % vps) * in_stride   + n,
// and likewise for out and base; the intermediate of vector v at tmp + v * N.
struct NttPass {
  const void *in;        // pass A input
  double *tmp;           // the transposed intermediates
  void *out;             // pass B output
  const uint64_t *base;  // kStoreRescale: residues in [0, q)
  const NttSet *sets;    // device array, one entry per set
  const uint64_t *add;   // ntt_pass_b_rot: residues in [0, q) added to the first polynomials
  uint64_t in_stride, out_stride, base_stride;
  uint64_t in_set_stride, out_set_stride, base_set_stride, add_set_stride;
  uint32_t vps, log_n1, log_n2, load, store;
  uint32_t out_transposed;  // pass B, kStoreU64 and kStoreRescale: write the transposed layout
  uint32_t nsets_shared;   // pass A: 0, or the number of sets when they all read the same input
                           // vectors (in_set_stride 0) and gridDim.x * vps is a multiple of 8
};

// Global loads and stores go in batches of up to kNttBatch per thread, all
// issued before the first is used (8: measured faster than 16, which took
// the passes past 128 VGPRs).
constexpr uint32_t kNttBatch = 8;

// Pass A, N2 = 2^LOGM: grid (N1 / kNttCols, vectors).  Thread t handles
// column c0 + t % kNttCols, rows n2 = t / kNttCols + j * (kNttThreads / kNttCols).
template <uint32_t LOGM>
__global__ void __launch_bounds__(kNttThreads) ntt_pass_a(const NttPass P) {
  constexpr uint32_t M = 1u << LOGM, PM = padded_len(M), PER = kNttCols * M / kNttThreads;
  constexpr uint32_t B = PER < kNttBatch ? PER : kNttBatch, RSTEP = kNttThreads / kNttCols;
  extern __shared__ double xs[];   // [kNttCols][PM], then the M/2 DFT twiddles
  Tw *tw = (Tw *)(xs + kNttCols * PM);
  uint32_t set = blockIdx.y / P.vps, lv = blockIdx.y - set * P.vps, cb = blockIdx.x;
  if (P.nsets_shared) {
    // The sets read the same input vectors: give the nsets_shared workgroups
    // of one (vector, column block) consecutive turns on one XCD (workgroup
    // ids i, i + 8, ... run there), so that the input is fetched once into
    // its L2.  The launch covers gridDim.x * vps units, a multiple of 8.
    const uint32_t id = blockIdx.y * gridDim.x + blockIdx.x;
    const uint32_t u = id >> 3, unit = (id & 7u) + 8u * (u / P.nsets_shared);
    set = u % P.nsets_shared;
    lv = unit / gridDim.x;
    cb = unit - lv * gridDim.x;
  }
  const NttSet S = P.sets[set];
  stage_twiddles(tw, S.dft_a, LOGM);
  const uint32_t N1 = 1u << P.log_n1, c = threadIdx.x % kNttCols, r = threadIdx.x / kNttCols;
  const uint32_t n1 = cb * kNttCols + c;
  const uint64_t v = (uint64_t)set * P.vps + lv;
  const uint64_t in_off = set * P.in_set_stride + lv * P.in_stride;
  const double q = S.q, qinv = S.qinv;
  if (P.load == kLoadU64T) {   // uniform: thread t reads column cb*16 + t/16, so that each
                               // quarter wave reads 16 consecutive words of the transposed layout
    const uint32_t cc = threadIdx.x / kNttCols, kk = threadIdx.x % kNttCols, col = cb * kNttCols + cc;
    const uint64_t *in = (const uint64_t *)P.in + in_off;
    const uint32_t N2 = 1u << P.log_n2;
#pragma unroll 1
    for (uint32_t b0 = 0; b0 < PER; b0 += B) {
      double x[B];
#pragma unroll
      for (uint32_t j = 0; j < B; ++j) {
        const uint32_t n = col + N1 * (kk + (b0 + j) * kNttCols);   // element n = n1 + N1 n2
        x[j] = reduce(to_f64(in[(size_t)(n & (N2 - 1)) * N1 + (n >> P.log_n2)]), q, qinv);
      }
#pragma unroll
      for (uint32_t j = 0; j < B; ++j) xs[cc * PM + pidx(bit_reverse(kk + (b0 + j) * kNttCols, LOGM))] = x[j];
    }
  } else {
  // batches one after the other (not unrolled): fewer registers, more waves
#pragma unroll 1
  for (uint32_t b0 = 0; b0 < PER; b0 += B) {
    double x[B];
    if (P.load == kLoadF64) {
      const double *in = (const double *)P.in + in_off + n1;
#pragma unroll
      for (uint32_t j = 0; j < B; ++j) x[j] = in[(size_t)N1 * (r + (b0 + j) * RSTEP)];
    } else {
      const uint64_t *in = (const uint64_t *)P.in + in_off + n1;
#pragma unroll
      for (uint32_t j = 0; j < B; ++j) x[j] = to_f64(in[(size_t)N1 * (r + (b0 + j) * RSTEP)]);
    }
    if (S.pre) {
      Tw t[B];
#pragma unroll
      for (uint32_t j = 0; j < B; ++j) t[j] = S.pre[n1 + N1 * (r + (b0 + j) * RSTEP)];
#pragma unroll
      for (uint32_t j = 0; j < B; ++j) x[j] = mul_tw(x[j], t[j], q);
    } else {
#pragma unroll
      for (uint32_t j = 0; j < B; ++j) x[j] = reduce(x[j], q, qinv);
    }
#pragma unroll
    for (uint32_t j = 0; j < B; ++j) xs[c * PM + pidx(bit_reverse(r + (b0 + j) * RSTEP, LOGM))] = x[j];
  }
  }
  lds_dft<LOGM>(xs, tw, q, qinv);
  double *tmp = P.tmp + v * ((uint64_t)N1 * M) + n1;
#pragma unroll 1
  for (uint32_t b0 = 0; b0 < PER; b0 += B) {
    Tw t[B];
#pragma unroll
    for (uint32_t j = 0; j < B; ++j) t[j] = S.mid[(size_t)(r + (b0 + j) * RSTEP) * N1 + n1];
#pragma unroll
    for (uint32_t j = 0; j < B; ++j) {
      const uint32_t k2 = r + (b0 + j) * RSTEP;
      tmp[(size_t)k2 * N1] = mul_tw(xs[c * PM + pidx(k2)], t[j], q);
    }
  }
}

// Pass B, N1 = 2^LOGM: grid (N2 / kNttCols, vectors).  Rows of the
// intermediate are loaded whole; thread t stores column k2 = r0 + t % kNttCols.
template <uint32_t LOGM>
__global__ void __launch_bounds__(kNttThreads) ntt_pass_b(const NttPass P) {
  constexpr uint32_t M = 1u << LOGM, PM = padded_len(M), PER = kNttCols * M / kNttThreads;
  constexpr uint32_t B = PER < kNttBatch ? PER : kNttBatch, RSTEP = kNttThreads / kNttCols;
  extern __shared__ double xs[];   // [kNttCols][PM], then the M/2 DFT twiddles
  Tw *tw = (Tw *)(xs + kNttCols * PM);
  const uint32_t set = blockIdx.y / P.vps, lv = blockIdx.y - set * P.vps;
  const NttSet S = P.sets[set];
  stage_twiddles(tw, S.dft_b, LOGM);
  const uint32_t N2 = 1u << P.log_n2, r0 = blockIdx.x * kNttCols;
  const uint64_t v = blockIdx.y;
  const double q = S.q, qinv = S.qinv;
  const double *tmp = P.tmp + v * ((uint64_t)N2 * M) + (size_t)r0 * M;
#pragma unroll
  for (uint32_t b0 = 0; b0 < PER; b0 += B) {
    double x[B];
#pragma unroll
    for (uint32_t j = 0; j < B; ++j) x[j] = tmp[threadIdx.x + (b0 + j) * kNttThreads];
#pragma unroll
    for (uint32_t j = 0; j < B; ++j) {
      const uint32_t idx = threadIdx.x + (b0 + j) * kNttThreads;
      xs[(idx >> LOGM) * PM + pidx(bit_reverse(idx & (M - 1), LOGM))] = x[j];
    }
  }
  lds_dft<LOGM>(xs, tw, q, qinv);
  const uint32_t c = threadIdx.x % kNttCols, r = threadIdx.x / kNttCols, k2 = r0 + c;
  const bool transposed = P.out_transposed != 0 && P.store != kStoreF64;
  const bool rescale = P.store == kStoreRescale;
  const uint64_t *base = rescale ? P.base + set * P.base_set_stride + lv * P.base_stride + k2 : nullptr;
#pragma unroll
  for (uint32_t b0 = 0; b0 < PER; b0 += B) {
    double y[B];
#pragma unroll
    for (uint32_t j = 0; j < B; ++j) y[j] = xs[c * PM + pidx(r + (b0 + j) * RSTEP)];
    if (S.post) {
      Tw t[B];
#pragma unroll
      for (uint32_t j = 0; j < B; ++j) t[j] = S.post[k2 + (size_t)N2 * (r + (b0 + j) * RSTEP)];
#pragma unroll
      for (uint32_t j = 0; j < B; ++j) y[j] = mul_tw(y[j], t[j], q);
    }
    if (P.store == kStoreF64) {
      double *out = (double *)P.out + set * P.out_set_stride + lv * P.out_stride + k2;
#pragma unroll
      for (uint32_t j = 0; j < B; ++j) out[(size_t)N2 * (r + (b0 + j) * RSTEP)] = reduce(y[j], q, qinv);
      continue;
    }
    if (rescale) {
      uint64_t bv[B];
#pragma unroll
      for (uint32_t j = 0; j < B; ++j) bv[j] = base[(size_t)N2 * (r + (b0 + j) * RSTEP)];
#pragma unroll
      for (uint32_t j = 0; j < B; ++j) y[j] = mul_tw(to_f64(bv[j]) - y[j], S.inv, q);
    }
#pragma unroll
    for (uint32_t j = 0; j < B; ++j) y[j] = canonical(y[j], q, qinv);
    if (transposed) {
#pragma unroll
      for (uint32_t j = 0; j < B; ++j) xs[c * PM + pidx(r + (b0 + j) * RSTEP)] = y[j];
    } else {
      uint64_t *out = (uint64_t *)P.out + set * P.out_set_stride + lv * P.out_stride + k2;
#pragma unroll
      for (uint32_t j = 0; j < B; ++j) out[(size_t)N2 * (r + (b0 + j) * RSTEP)] = to_u64(y[j]);
    }
  }
  if (transposed) {   // uniform over the workgroup
    // each quarter wave stores kNttCols consecutive k1 of one row k2
    __syncthreads();
    const uint32_t cc = threadIdx.x / kNttCols, kk = threadIdx.x % kNttCols;
    uint64_t *out = (uint64_t *)P.out + set * P.out_set_stride + lv * P.out_stride + (size_t)(r0 + cc) * M;
#pragma unroll
    for (uint32_t j = 0; j < PER; ++j) {
      const uint32_t k1 = kk + j * kNttCols;
      out[k1] = to_u64(xs[cc * PM + pidx(k1)]);
    }
  }
}

}  // namespace fiona
