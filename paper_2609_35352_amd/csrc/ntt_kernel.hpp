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
// (radix 2, input in bit-reversed order, output natural).
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

// Radix-2 DFT of size M = 2^logM on kNttCols columns held in LDS (column c at
// x + c*M, loaded in bit-reversed order); natural order on return.
// tw[t] = w_M^t for t < M/2.
__device__ __forceinline__ void lds_dft(uint64_t *x, uint32_t logM, const Tw *__restrict__ tw, uint64_t q) {
  const uint32_t M = 1u << logM, halfM = M >> 1;
  const uint32_t nb = kNttCols * halfM;
  for (uint32_t s = 0; s < logM; ++s) {
    const uint32_t half = 1u << s;
    __syncthreads();
    for (uint32_t b = threadIdx.x; b < nb; b += kNttThreads) {
      const uint32_t c = b >> (logM - 1), j = b & (halfM - 1);
      const uint32_t pos = j & (half - 1);
      const uint32_t i0 = ((j >> s) << (s + 1)) | pos, i1 = i0 + half;
      uint64_t *col = x + c * M;
      const uint64_t u = col[i0], t = mul_tw(col[i1], tw[pos << (logM - 1 - s)], q);
      col[i0] = add_q(u, t, q);
      col[i1] = sub_q(u, t, q);
    }
  }
  __syncthreads();
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
  extern __shared__ uint64_t xs[];   // [kNttCols][N2]
  const uint32_t N1 = 1u << P.log_n1, N2 = 1u << P.log_n2;
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
    xs[c * N2 + bit_reverse(n2, P.log_n2)] = x;
  }
  lds_dft(xs, P.log_n2, P.dft_a, P.q);
  uint64_t *tmp = P.tmp + v * ((uint64_t)N1 * N2);
  for (uint32_t idx = threadIdx.x; idx < kNttCols * N2; idx += kNttThreads) {
    const uint32_t c = idx & (kNttCols - 1), k2 = idx / kNttCols;
    const uint32_t n1 = c0 + c;
    tmp[k2 * N1 + n1] = mul_tw(xs[c * N2 + k2], P.mid[n1 * N2 + k2], P.q);
  }
}

// Pass B: grid (N2 / kNttCols, vectors).
__global__ void __launch_bounds__(kNttThreads) ntt_pass_b(const NttPass P) {
  extern __shared__ uint64_t xs[];   // [kNttCols][N1]
  const uint32_t N1 = 1u << P.log_n1, N2 = 1u << P.log_n2;
  const uint32_t r0 = blockIdx.x * kNttCols;
  const uint64_t v = blockIdx.y;
  const uint64_t *tmp = P.tmp + v * ((uint64_t)N1 * N2);
  for (uint32_t idx = threadIdx.x; idx < kNttCols * N1; idx += kNttThreads) {
    const uint32_t c = idx / N1, n1 = idx & (N1 - 1);
    xs[c * N1 + bit_reverse(n1, P.log_n1)] = tmp[(r0 + c) * N1 + n1];
  }
  lds_dft(xs, P.log_n1, P.dft_b, P.q);
  uint64_t *out = P.out + v * P.out_stride;
  const uint64_t *base = P.base ? P.base + v * P.base_stride : nullptr;
  for (uint32_t idx = threadIdx.x; idx < kNttCols * N1; idx += kNttThreads) {
    const uint32_t c = idx & (kNttCols - 1), k1 = idx / kNttCols;
    const uint32_t k = r0 + c + N2 * k1;
    uint64_t y = xs[c * N1 + k1];
    if (P.post) y = mul_tw(y, P.post[k], P.q);
    if (P.store == kStoreRescale) y = mul_tw(sub_q(base[k], y, P.q), P.inv, P.q);
    out[k] = y;
  }
}

}  // namespace fiona
