// Modular arithmetic for residues below 2^50 on gfx950, built from 32-bit
// integer multiplies with 64-bit results (v_mad_u64_u32 / v_mad_i64_i32).
//
// A residue x < 2^50 is split into two radix-2^25 digits, x = x0 + 2^25 x1.
// A product x * w is accumulated digit by digit,
//     x * w = x0 w0 + 2^25 (x0 w1 + x1 w0) + 2^50 x1 w1,
// four 32x32->64 multiply-adds per polynomial with the accumulation folded
// into the multiply-add.  Nothing is reduced per term: the accumulators hold
// the exact integer sum, and one reduction per output brings it to the
// canonical residue in [0, q).  The bounds below keep every accumulator exact
// for up to kFoldTerms terms; longer sums are folded into a running residue.
//
// A signed sum U = sum h_m x_m (h in {-1, 0, +1}, at most kMaxMembers members)
// is kept digit-wise as two signed 32-bit values (U0, U1), U = U0 + 2^25 U1,
// and a scalar c < 2^20 multiplies it with two 32x32->64 signed multiply-adds.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fiona {

constexpr uint32_t kDigitMask = 0x1FFFFFFu;  // 2^25 - 1
constexpr uint32_t kFoldTerms = 1024;        // terms (or uses) per exact accumulation
constexpr uint32_t kMaxMembers = 48;         // members per signed sum: |U0|, |U1| < 48 * 2^25 < 2^31

// Per-limb constants, computed on the host (2^20 < q < 2^50).
struct LimbConst {
  uint64_t q;
  uint64_t r50;        // 2^50 mod q
  uint64_t r50_shoup;  // floor(r50 * 2^64 / q)
  double qinv;         // 1.0 / q rounded to double
};

// Exact sum of one output polynomial at one position.
//   value = a0 + s0 + 2^25 (a1 + s1) + 2^50 a2
// Bounds for at most kFoldTerms raw terms and kFoldTerms uses:
//   a0, a2 < 2^10 * 2^50 = 2^60;  a1 < 2^10 * 2^51 = 2^61;
//   |s0|, |s1| < 2^10 * 2^20 * 2^31 = 2^61.
struct Acc {
  uint64_t a0, a1, a2;
  int64_t s0, s1;
};

__device__ __forceinline__ void acc_zero(Acc &a) {
  a.a0 = 0; a.a1 = 0; a.a2 = 0; a.s0 = 0; a.s1 = 0;
}

// Digits of a residue below 2^50.
__device__ __forceinline__ uint32_t lo_digit(uint64_t x) { return (uint32_t)x & kDigitMask; }
__device__ __forceinline__ uint32_t hi_digit(uint64_t x) {
  return __builtin_amdgcn_alignbit((uint32_t)(x >> 32), (uint32_t)x, 25);
}

// acc += x * w for x = x0 + 2^25 x1 and w = w0 + 2^25 w1.
__device__ __forceinline__ void mac(Acc &a, uint32_t x0, uint32_t x1, uint32_t w0, uint32_t w1) {
  a.a0 += (uint64_t)x0 * w0;
  a.a1 += (uint64_t)x0 * w1;
  a.a1 += (uint64_t)x1 * w0;
  a.a2 += (uint64_t)x1 * w1;
}

// acc += c * U for a signed scale c (|c| < 2^20) and U = u0 + 2^25 u1.
__device__ __forceinline__ void smac(Acc &a, int32_t c, int32_t u0, int32_t u1) {
  a.s0 += (int64_t)c * u0;
  a.s1 += (int64_t)c * u1;
}

// v mod q in [0, q) for |v| < 2^62 and 2 <= q < 2^50.  Two rounds of a
// floating-point quotient estimate.  The estimate of v / q has relative error
// below 3 * 2^-53, so the first round leaves |r| <= |v| * 3 * 2^-53 + q
// < 2^11 + q; the second is then off by at most one multiple of q, which the
// final corrections remove.
__device__ __forceinline__ uint64_t reduce_i64(int64_t v, uint64_t q, double qinv) {
  const int64_t qs = (int64_t)q;
  double t = floor((double)v * qinv);
  int64_t r = v - (int64_t)t * qs;
  t = floor((double)r * qinv);
  r -= (int64_t)t * qs;
  if (r < 0) r += qs;
  if (r < 0) r += qs;
  if (r >= qs) r -= qs;
  if (r >= qs) r -= qs;
  return (uint64_t)r;
}

// v mod q in [0, q) for 0 <= v < 2^52 and 2^20 < q < 2^50: v converts to
// double exactly, the quotient is below 2^32 and its estimate is off by at
// most one.
__device__ __forceinline__ uint64_t reduce_small(uint64_t v, uint64_t q, double qinv) {
  const uint32_t t = (uint32_t)((double)v * qinv);   // truncation = floor for v >= 0
  int64_t r = (int64_t)(v - (uint64_t)t * q);
  if (r < 0) r += (int64_t)q;
  if (r >= (int64_t)q) r -= (int64_t)q;
  return (uint64_t)r;
}

// h * w mod q, in [0, 2q), for h < 2^64, w < q < 2^63, ws = floor(w 2^64 / q)
// (Shoup's multiplication by a precomputed constant).
__device__ __forceinline__ uint64_t mul_shoup_lazy(uint64_t h, uint64_t w, uint64_t ws, uint64_t q) {
  const uint64_t qhat = __umul64hi(h, ws);
  return h * w - qhat * q;
}

// Canonical residue of (racc + value of a) mod q, racc < q.
__device__ __forceinline__ uint64_t finish(const Acc &a, uint64_t racc, const LimbConst &lc) {
  int64_t lo = (int64_t)a.a0 + a.s0;              // |lo| < 2^62
  int64_t md = (int64_t)a.a1 + a.s1;              // |md| < 2^62
  int64_t hi = (int64_t)a.a2;
  // carry-normalise to value = lo + 2^25 md + 2^50 hi with lo, md in [0, 2^25)
  int64_t c = lo >> 25;                           // arithmetic shift: floor division
  lo &= (int64_t)kDigitMask;
  md += c;
  c = md >> 25;
  md &= (int64_t)kDigitMask;
  hi += c;                                        // |hi| < 2^61
  const uint64_t base = (uint64_t)lo + ((uint64_t)md << 25);   // < 2^50
  // 2^50 hi mod q: |hi| * (2^50 mod q) in [0, 2q), negated for hi < 0
  const uint64_t mag = (uint64_t)(hi < 0 ? -hi : hi);
  uint64_t t = mul_shoup_lazy(mag, lc.r50, lc.r50_shoup, lc.q);
  if (hi < 0) t = 2 * lc.q - t;                   // in (0, 2q]
  return reduce_small(base + t + racc, lc.q, lc.qinv);   // < 2^50 + 2q + q < 2^52
}

}  // namespace fiona
