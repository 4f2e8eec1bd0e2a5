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
// Modular products use Shoup's method with precomputed companions
// ws = floor(w 2^64 / q) (q < 2^50), giving x w mod q in [0, 2q) before one
// correction.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "modarith.hpp"

namespace fiona {

constexpr uint32_t kNttCols = 16;      // columns (pass A) or rows (pass B) per workgroup
constexpr uint32_t kNttThreads = 256;
constexpr uint32_t kNttMaxSide = 512;  // N1, N2 <= 512: N <= 2^17

struct Tw {   // a twiddle and its Shoup companion
  uint64_t w, ws;
};

__device__ __forceinline__ uint64_t mul_tw(uint64_t x, const Tw &t, uint64_t q) {
  const uint64_t r = x * t.w - __umul64hi(x, t.ws) * q;   // in [0, 2q) for x < 2^64
  return r >= q ? r - q : r;
}
__device__ __forceinline__ uint64_t add_q(uint64_t a, uint64_t b, uint64_t q) {
  const uint64_t s = a + b;
  return s >= q ? s - q : s;
}
__device__ __forceinline__ uint64_t sub_q(uint64_t a, uint64_t b, uint64_t q) { return a >= b ? a - b : a + q - b; }

__device__ __forceinline__ uint32_t bit_reverse(uint32_t x, uint32_t bits) { return __brev(x) >> (32 - bits); }

// LDS column layout: one padding word after every 16, so that the 16-word
// groups a thread reads (consecutive words, or words 16 apart) fall into
// different banks.
__device__ __forceinline__ uint32_t pidx(uint32_t i) { return i + (i >> 4); }
__host__ __device__ constexpr uint32_t padded_len(uint32_t m) { return m + m / 16; }

// Stages s0 .. s0+R-1 of the radix-2 DFT for the groups of one 16-word item:
// a group is the 2^R words base + (u << s0) that these stages combine; the
// item holds 16 >> R groups, kept in registers across the R stages.
template <int R>
__device__ __forceinline__ void dft_item(uint64_t *col, uint32_t logM, uint32_t s0, uint32_t item,
                                         const Tw *tw, uint64_t q) {
  constexpr uint32_t S = 1u << R, G = 16u >> R;
#pragma unroll
  for (uint32_t g = 0; g < G; ++g) {
    const uint32_t gi = item * G + g;
    const uint32_t o = gi & ((1u << s0) - 1);
    const uint32_t base = ((gi >> s0) << (s0 + R)) + o;
    uint64_t r[S];
#pragma unroll
    for (uint32_t u = 0; u < S; ++u) r[u] = col[pidx(base + (u << s0))];
#pragma unroll
    for (uint32_t st = 0; st < (uint32_t)R; ++st) {
      const uint32_t hh = 1u << st, shift = logM - 1 - (s0 + st);
#pragma unroll
      for (uint32_t u0 = 0; u0 < S; ++u0) {
        if ((u0 & (2 * hh - 1)) >= hh) continue;
        const uint32_t pos = o + ((u0 & (hh - 1)) << s0);
        const uint64_t a = r[u0], t = mul_tw(r[u0 + hh], tw[pos << shift], q);
        r[u0] = add_q(a, t, q);
        r[u0 + hh] = sub_q(a, t, q);
      }
    }
#pragma unroll
    for (uint32_t u = 0; u < S; ++u) col[pidx(base + (u << s0))] = r[u];
  }
}

// Radix-2 DFT of size M = 2^logM (16 <= M <= kNttMaxSide) on kNttCols
// columns held in LDS (column c at x + c * padded_len(M), loaded in
// bit-reversed order); natural order on return.  tw[t] = w_M^t for t < M/2
// (in LDS).  Up to four stages per pass over LDS, in registers.
__device__ __forceinline__ void lds_dft(uint64_t *x, uint32_t logM, const Tw *tw, uint64_t q) {
  const uint32_t M = 1u << logM, PM = padded_len(M), per_col = M >> 4;
  const uint32_t items = kNttCols * per_col;
  for (uint32_t s0 = 0; s0 < logM; s0 += 4) {
    const uint32_t R = min(4u, logM - s0);
    __syncthreads();
    for (uint32_t it = threadIdx.x; it < items; it += kNttThreads) {
      uint64_t *col = x + (it / per_col) * PM;
      const uint32_t item = it % per_col;
      if (R == 4) dft_item<4>(col, logM, s0, item, tw, q);
      else if (R == 3) dft_item<3>(col, logM, s0, item, tw, q);
      else if (R == 2) dft_item<2>(col, logM, s0, item, tw, q);
      else dft_item<1>(col, logM, s0, item, tw, q);
    }
  }
  __syncthreads();
}

// Copy the M/2 twiddles of the size-M DFT into LDS.
__device__ __forceinline__ void stage_twiddles(Tw *dst, const Tw *__restrict__ src, uint32_t logM) {
  for (uint32_t i = threadIdx.x; i < (1u << logM) / 2; i += kNttThreads) dst[i] = src[i];
}

// What a pass does with the values it loads (pass A) or stores (pass B).
enum NttLoad : uint32_t {
  kLoadPlain = 0,    // the input is already a residue mod q
  kLoadCentred = 1,  // the input is a residue mod q_src: take its centred value mod q
};
enum NttStore : uint32_t {
  kStorePlain = 0,    // store the transform
  kStoreRescale = 1,  // store (base - transform) * inv mod q
};

struct NttPass {
  const uint64_t *in;    // pass A: vector v, element n at in + v * in_stride + n
  uint64_t *tmp;         // the transposed intermediate, vector v at tmp + v * N
  uint64_t *out;         // pass B: vector v, element k at out + v * out_stride + k
  const uint64_t *base;  // kStoreRescale: base + v * base_stride + k
  const Tw *pre;         // pass A: multiply input n by pre[n] (null: by 1)
  const Tw *mid;         // pass A: mid[n1 N2 + k2]
  const Tw *dft_a;       // size-N2 DFT twiddles (N2 / 2)
  const Tw *dft_b;       // size-N1 DFT twiddles (N1 / 2)
  const Tw *post;        // pass B: multiply output k by post[k] (null: by 1)
  Tw inv;                // kStoreRescale: q_src^-1 mod q
  uint64_t q, q_src, q_src_mod_q;
  double qinv;           // 1 / q, for reducing a residue mod q_src
  uint64_t in_stride, out_stride, base_stride;
  uint32_t log_n1, log_n2, load, store;
};

// Pass A: grid (N1 / kNttCols, vectors).
__global__ void __launch_bounds__(kNttThreads) ntt_pass_a(const NttPass P) {
  extern __shared__ uint64_t xs[];   // [kNttCols][padded N2], then the N2/2 DFT twiddles
  const uint32_t N1 = 1u << P.log_n1, N2 = 1u << P.log_n2, PM = padded_len(N2);
  Tw *tw = (Tw *)(xs + kNttCols * PM);
  stage_twiddles(tw, P.dft_a, P.log_n2);
  const uint32_t c0 = blockIdx.x * kNttCols;
  const uint64_t v = blockIdx.y;
  const uint64_t *in = P.in + v * P.in_stride;
  const uint64_t half_src = P.q_src >> 1;
  for (uint32_t idx = threadIdx.x; idx < kNttCols * N2; idx += kNttThreads) {
    const uint32_t c = idx & (kNttCols - 1), n2 = idx / kNttCols;
    const uint32_t n = c0 + c + N1 * n2;
    uint64_t x = in[n];
    if (P.load == kLoadCentred) {   // x in [0, q_src): its centred value mod q
      const bool neg = x > half_src;
      x = reduce_small(x, P.q, P.qinv);
      if (neg) x = sub_q(x, P.q_src_mod_q, P.q);
    }
    if (P.pre) x = mul_tw(x, P.pre[n], P.q);
    xs[c * PM + pidx(bit_reverse(n2, P.log_n2))] = x;
  }
  lds_dft(xs, P.log_n2, tw, P.q);
  uint64_t *tmp = P.tmp + v * ((uint64_t)N1 * N2);
  for (uint32_t idx = threadIdx.x; idx < kNttCols * N2; idx += kNttThreads) {
    const uint32_t c = idx & (kNttCols - 1), k2 = idx / kNttCols;
    const uint32_t n1 = c0 + c;
    tmp[k2 * N1 + n1] = mul_tw(xs[c * PM + pidx(k2)], P.mid[n1 * N2 + k2], P.q);
  }
}

// Pass B: grid (N2 / kNttCols, vectors).
__global__ void __launch_bounds__(kNttThreads) ntt_pass_b(const NttPass P) {
  extern __shared__ uint64_t xs[];   // [kNttCols][padded N1], then the N1/2 DFT twiddles
  const uint32_t N1 = 1u << P.log_n1, N2 = 1u << P.log_n2, PM = padded_len(N1);
  Tw *tw = (Tw *)(xs + kNttCols * PM);
  stage_twiddles(tw, P.dft_b, P.log_n1);
  const uint32_t r0 = blockIdx.x * kNttCols;
  const uint64_t v = blockIdx.y;
  const uint64_t *tmp = P.tmp + v * ((uint64_t)N1 * N2);
  for (uint32_t idx = threadIdx.x; idx < kNttCols * N1; idx += kNttThreads) {
    const uint32_t c = idx / N1, n1 = idx & (N1 - 1);
    xs[c * PM + pidx(bit_reverse(n1, P.log_n1))] = tmp[(r0 + c) * N1 + n1];
  }
  lds_dft(xs, P.log_n1, tw, P.q);
  uint64_t *out = P.out + v * P.out_stride;
  const uint64_t *base = P.base ? P.base + v * P.base_stride : nullptr;
  for (uint32_t idx = threadIdx.x; idx < kNttCols * N1; idx += kNttThreads) {
    const uint32_t c = idx & (kNttCols - 1), k1 = idx / kNttCols;
    const uint32_t k = r0 + c + N2 * k1;
    uint64_t y = xs[c * PM + pidx(k1)];
    if (P.post) y = mul_tw(y, P.post[k], P.q);
    if (P.store == kStoreRescale) y = mul_tw(sub_q(base[k], y, P.q), P.inv, P.q);
    out[k] = y;
  }
}

}  // namespace fiona
