// Modular arithmetic for residues below 2^50 on gfx950, built from 32-bit
// integer multiplies with 64-bit results (v_mad_u64_u32 / v_mad_i64_i32).
//
// A ciphertext residue x < 2^50 is split into two radix-2^25 digits,
// x = x0 + 2^25 x1 (done once, when the input is staged), and a plaintext
// word w < 2^50 is used as its two 32-bit halves, w = wl + 2^32 wh (wh < 2^18),
// which needs no instruction at all.  A product x * w is accumulated as
//     x * w = x0 wl + 2^25 x1 wl + 2^32 x0 wh + 2^57 x1 wh,
// four 32x32->64 multiply-adds per polynomial, with the accumulation folded
// into the multiply-add.  Nothing is reduced per term: the accumulators hold
// the exact integer sum and one reduction per output brings it to the
// canonical residue in [0, q).  A cheap carry step once per chunk of at most
// kChunkTerms terms keeps the two low partial sums below 2^64; much longer
// sums are folded into a running residue.
//
// A signed sum U = sum h_m x_m (h in {-1, 0, +1}, at most kMaxMembers members)
// is kept digit-wise as two signed 32-bit values (U0, U1), U = U0 + 2^25 U1,
// and a scalar c < 2^20 multiplies it with two 32x32->64 signed multiply-adds.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fiona {

constexpr uint32_t kDigitMask = 0x1FFFFFFu;  // 2^25 - 1
constexpr uint32_t kChunkTerms = 56;         // raw terms between two carry steps
constexpr uint32_t kFoldChunks = 4096;       // chunks of raw terms per exact accumulation
constexpr uint32_t kFoldUses = 1024;         // signed-sum uses per exact accumulation
constexpr uint32_t kMaxMembers = 48;         // members per signed sum: |U0|, |U1| < 48 * 2^25 < 2^31

// Per-limb constants, computed on the host (2^20 < q < 2^50).
struct LimbConst {
  uint64_t q;
  uint64_t r32, r32_shoup;   // 2^32 mod q and floor(r32 * 2^64 / q)
  uint64_t r57, r57_shoup;   // 2^57 mod q and floor(r57 * 2^64 / q)
  double qinv;               // 1.0 / q rounded to double
};

// Exact sum of one output polynomial at one position:
//   value = A0 + 2^25 A1 + 2^32 A2 + 2^57 A3 + s0 + 2^25 s1.
// Bounds (x0, x1 < 2^25, wl < 2^32, wh < 2^18, |c| < 2^20, |U0|, |U1| < 2^31):
//   a raw term adds < 2^57 to A0 and A1 and < 2^43 to A2 and A3;
//   after a carry step A0, A1 < 2^32, so one chunk leaves them < 2^32 + 56 * 2^57 < 2^63;
//   a chunk plus its carry adds < 2^49 to A2 and A3: < 2^61 over kFoldChunks chunks;
//   a use adds |c U| < 2^51 to s0 and s1: |s0|, |s1| < 2^61 over kFoldUses uses.
struct Acc {
  uint64_t A0, A1, A2, A3;
  int64_t s0, s1;
};

__device__ __forceinline__ void acc_zero(Acc &a) {
  a.A0 = 0; a.A1 = 0; a.A2 = 0; a.A3 = 0; a.s0 = 0; a.s1 = 0;
}

// Digits of a residue below 2^50.
__device__ __forceinline__ uint32_t lo_digit(uint64_t x) { return (uint32_t)x & kDigitMask; }
__device__ __forceinline__ uint32_t hi_digit(uint64_t x) {
  return __builtin_amdgcn_alignbit((uint32_t)(x >> 32), (uint32_t)x, 25);
}

// acc += x * w for x = x0 + 2^25 x1 and w = wl + 2^32 wh.
__device__ __forceinline__ void mac(Acc &a, uint32_t x0, uint32_t x1, uint32_t wl, uint32_t wh) {
  a.A0 += (uint64_t)x0 * wl;
  a.A1 += (uint64_t)x1 * wl;
  a.A2 += (uint64_t)x0 * wh;
  a.A3 += (uint64_t)x1 * wh;
}

// Moves the upper halves of A0 and A1 up to the partial sums of the same
// weight: 2^32 (A0 >> 32) has A2's weight and 2^25 2^32 (A1 >> 32) has A3's.
__device__ __forceinline__ void carry(Acc &a) {
  a.A2 += a.A0 >> 32;
  a.A0 &= 0xFFFFFFFFull;
  a.A3 += a.A1 >> 32;
  a.A1 &= 0xFFFFFFFFull;
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

// v mod q in [0, q) for 0 <= v < 2^53 and v < 2^32 q: v converts to double
// exactly, the quotient fits 32 bits and its estimate (relative error below
// 2^-51) is off by at most one.
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
__device__ __forceinline__ uint64_t finish(Acc a, uint64_t racc, const LimbConst &lc) {
  carry(a);                                       // A0, A1 < 2^32
  int64_t p0 = (int64_t)a.A0 + a.s0;              // |p0| < 2^61 + 2^32
  int64_t p1 = (int64_t)a.A1 + a.s1;
  // value = p0 + 2^25 p1 + 2^32 A2 + 2^57 A3; carry p0 into p1 and p1 into A2
  int64_t c = p0 >> 25;                           // arithmetic shift: floor division
  p0 &= (int64_t)kDigitMask;
  p1 += c;
  c = p1 >> 7;
  p1 &= 0x7F;
  const int64_t h = (int64_t)a.A2 + c;            // |h| < 2^62
  const uint64_t base = (uint64_t)p0 + ((uint64_t)p1 << 25);   // < 2^32
  // 2^32 h mod q and 2^57 A3 mod q, each in [0, 2q]
  uint64_t th = mul_shoup_lazy((uint64_t)(h < 0 ? -h : h), lc.r32, lc.r32_shoup, lc.q);
  if (h < 0) th = 2 * lc.q - th;
  const uint64_t t3 = mul_shoup_lazy(a.A3, lc.r57, lc.r57_shoup, lc.q);
  return reduce_small(base + th + t3 + racc, lc.q, lc.qinv);   // < 2^32 + 5q < 2^53
}

}  // namespace fiona
