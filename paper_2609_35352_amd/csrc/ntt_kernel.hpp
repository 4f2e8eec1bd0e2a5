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
//           multiplication of each input by pre[n2]), then a multiplication by
//           mid[k2 N1 + n1]; stored transposed as T[k2 N1 + n1];
//   pass B: for each k2, a DFT of size N1 over n1, giving output k2 + N2 k1
//           (optionally multiplied by post[k1]).
// The twist psi^n of the forward transform and the factor N^-1 psi^-k of the
// inverse split into a part that pre or post applies and a part that is
// constant along one pass's DFT and rides in mid (the tables are built on the
// host).  A workgroup takes kNttCols columns (pass A) or rows (pass B) at
// once, so every global access is a run of at least kNttCols consecutive
// words.  The DFTs are radix 2 with the input in bit-reversed order and the
// output natural; a thread takes groups of up to 16 words through four
// stages at a time in registers, and LDS carries the data between groups.
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

#include "buffer.hpp"

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

// Integers below 2^52 to and from doubles: 2^52 + x has the bits of x in its
// mantissa, so the conversion is one bitwise operation and one exact add.
__device__ __forceinline__ double to_f64(uint64_t x) {   // x < 2^52
  return __builtin_bit_cast(double, x | 0x4330000000000000ull) - 4503599627370496.0;
}
__device__ __forceinline__ uint64_t to_u64(double y) {   // y an integer in [0, 2^52)
  return __builtin_bit_cast(uint64_t, y + 4503599627370496.0) & 0x000FFFFFFFFFFFFFull;
}

// A buffer view of global memory for the passes' per-group accesses.  The
// descriptor holds the base and the bytes left in the buffer; the byte
// offset splits into the lane's part (a VGPR) and a part the workgroup
// shares (an SGPR or a constant), so that the 16 accesses of a group need no
// vector address arithmetic.  Offsets stay below 2^32 bytes (one vector or
// one table per view).
typedef uint32_t nv2 __attribute__((ext_vector_type(2)));
typedef uint32_t nv4 __attribute__((ext_vector_type(4)));
struct Buf {
  __amdgpu_buffer_rsrc_t rs;
  // p is the same in every lane; readfirstlane keeps the descriptor in SGPRs
  // where the compiler has computed p in vector registers.  end: the end of
  // the buffer p points into.
  __device__ __forceinline__ Buf(const void *p, const void *end) : rs(make(p, end)) {}
  static __device__ __forceinline__ __amdgpu_buffer_rsrc_t make(const void *p, const void *end) {
    const uint64_t a = (uint64_t)p;
    // readfirstlane returns an int; join_halves takes it as unsigned
    const uint64_t u = join_halves((uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)),
                                   (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a));
    return __builtin_amdgcn_make_buffer_rsrc((void *)u, (short)0, (int)buffer_extent(u, (uint64_t)end), 0x00020000);
  }
  __device__ __forceinline__ uint64_t u64(uint32_t voff, uint32_t soff) const {
    const nv2 w = __builtin_amdgcn_raw_buffer_load_b64(rs, voff, soff, 0);
    return (uint64_t)w.x | ((uint64_t)w.y << 32);
  }
  __device__ __forceinline__ double f64(uint32_t voff, uint32_t soff) const {
    return __builtin_bit_cast(double, u64(voff, soff));
  }
  // Nontemporal loads (cache policy 2) for words read once: pass B's
  // intermediate and the words it subtracts from (rescale VGG11 / BERT /
  // Large a further 0.5 / 2 / 1% faster).
  __device__ __forceinline__ uint64_t u64_once(uint32_t voff, uint32_t soff) const {
    const nv2 w = __builtin_amdgcn_raw_buffer_load_b64(rs, voff, soff, 2);
    return (uint64_t)w.x | ((uint64_t)w.y << 32);
  }
  __device__ __forceinline__ double f64_once(uint32_t voff, uint32_t soff) const {
    return __builtin_bit_cast(double, u64_once(voff, soff));
  }
  __device__ __forceinline__ Tw tw(uint32_t voff, uint32_t soff) const {
    const nv4 w = __builtin_amdgcn_raw_buffer_load_b128(rs, voff, soff, 0);
    return Tw{__builtin_bit_cast(double, (uint64_t)w.x | ((uint64_t)w.y << 32)),
              __builtin_bit_cast(double, (uint64_t)w.z | ((uint64_t)w.w << 32))};
  }
  // Stores are nontemporal (cache policy 2): measured against the default
  // policy, the rescale of VGG11's outputs 1.11 -> 1.08 ms, BERT's 1.25 ->
  // 1.19, Large's 2.29 -> 2.16; the rotations 0-2% faster.
  __device__ __forceinline__ void put(uint64_t x, uint32_t voff, uint32_t soff) const {
    __builtin_amdgcn_raw_buffer_store_b64((nv2){(uint32_t)x, (uint32_t)(x >> 32)}, rs, voff, soff, 2);
  }
  __device__ __forceinline__ void put(double y, uint32_t voff, uint32_t soff) const {
    put(__builtin_bit_cast(uint64_t, y), voff, soff);
  }
};

__device__ __forceinline__ uint32_t bit_reverse(uint32_t x, uint32_t bits) { return __brev(x) >> (32 - bits); }
// The four-bit reversal of u < 16 (a group's position in the bit-reversed order).
__host__ __device__ constexpr uint32_t rev4(uint32_t u) {
  return ((u & 1u) << 3) | ((u & 2u) << 1) | ((u & 4u) >> 1) | ((u & 8u) >> 3);
}

// LDS layout of the kNttCols columns.  The 16 lanes of a quarter wave work on
// the same word of 16 different columns (the DFT's twiddle reads are then
// broadcasts), so the column stride is odd: those lanes fall into 16
// different banks.  Within a column one padding word follows every 16, so
// that 16 consecutive bit-reversed positions (the row loads of pass B) fall
// into different banks too.
__device__ __forceinline__ uint32_t pidx(uint32_t i) { return i + (i >> 4); }
__host__ __device__ constexpr uint32_t padded_len(uint32_t m) { return m + m / 16 + 1; }

// Stages S0 .. S0+R-1 of the radix-2 DFT on one group of 2^R words held in
// registers: r[u] is the word at position o + (u << S0) of a group whose
// offset below 2^S0 is o (positions in the DFT's bit-reversed input order).
// tw_at(t) returns w_M^t.  Entries are |x| <= 0.57 q; every second stage and
// the last one end with a reduction.  A product's output is below 0.5 q
// (1 + 2^-3); the unit-twiddle butterflies of the first stages (S0 = 0) add
// their input unmultiplied, so a product's input stays below 1.2 q, every
// value below 2.3 q (< 2^52, within reduce's range), and the group leaves
// |x| <= q/2 behind.
template <uint32_t LOGM, uint32_t S0, uint32_t R, typename TwAt>
__device__ __forceinline__ void butterflies(double (&r)[1u << R], uint32_t o, TwAt tw_at, double q, double qinv) {
  constexpr uint32_t S = 1u << R;
#pragma unroll
  for (uint32_t st = 0; st < R; ++st) {
    const uint32_t hh = 1u << st, shift = LOGM - 1 - (S0 + st);
#pragma unroll
    for (uint32_t u0 = 0; u0 < S; ++u0) {
      if ((u0 & (2 * hh - 1)) >= hh) continue;
      // with S0 = 0 (so o = 0) the butterflies with offset 0 have the twiddle 1
      const bool unit = S0 == 0 && (u0 & (hh - 1)) == 0;
      const double a = r[u0];
      const double t = unit ? r[u0 + hh] : mul_tw(r[u0 + hh], tw_at((o + ((u0 & (hh - 1)) << S0)) << shift), q);
      r[u0] = a + t;
      r[u0 + hh] = a - t;
    }
    if ((st & 1) || st + 1 == R) {
#pragma unroll
      for (uint32_t u = 0; u < S; ++u) r[u] = reduce(r[u], q, qinv);
    }
  }
}

// How a size-M DFT (16 <= M <= kNttMaxSide) splits over a workgroup's
// kNttCols columns.  The first four stages run on groups of 16 words that a
// thread loads straight from global memory (natural index i' + I1 v,
// v < 16: position 16 i + bitrev4(v) of the bit-reversed input order,
// i = bitrev(i') over log2(I1) bits); the last R2 stages run on groups of
// 2^R2 words (positions o + (u << S0L), o < I2) whose results, the outputs
// k = o + (u << S0L) in natural order, the thread stores straight to global
// memory; what lies between (M = 512: one stage) runs in LDS.
template <uint32_t LOGM>
struct DftShape {
  static constexpr uint32_t M = 1u << LOGM, PM = padded_len(M);
  static constexpr uint32_t I1 = M / 16;                       // first groups per column
  static constexpr uint32_t R2 = LOGM <= 8 ? LOGM - 4 : 4;      // stages of the last groups
  static constexpr uint32_t S0L = LOGM - R2;                   // the last groups' first stage
  static constexpr uint32_t E2 = 1u << R2, I2 = 1u << S0L;     // last group size and count per column
  static constexpr uint32_t IT1 = kNttCols * I1, IT2 = kNttCols * I2;
};

// The twiddles of the first four stages, w_M^(j M/16) for j < 8: uniform
// over the workgroup, read once into scalar registers.
template <uint32_t LOGM>
__device__ __forceinline__ void first_twiddles(Tw (&t1)[8], const Tw *__restrict__ dft) {
#pragma unroll
  for (uint32_t j = 0; j < 8; ++j) t1[j] = dft[j << (LOGM - 4)];
}

template <uint32_t LOGM>
__device__ __forceinline__ void first_stages(double (&r)[16], const Tw (&t1)[8], double q, double qinv) {
  butterflies<LOGM, 0, 4>(r, 0, [&](uint32_t t) { return t1[t >> (LOGM - 4)]; }, q, qinv);
}

// The first groups' results go to LDS: column col, group i' (natural order).
template <uint32_t LOGM>
__device__ __forceinline__ void put_first(double *xs, uint32_t col, uint32_t ip, const double (&r)[16]) {
  using D = DftShape<LOGM>;
  const uint32_t i = LOGM > 4 ? bit_reverse(ip, LOGM - 4) : 0u;   // (M = 16: one group, i' = 0)
#pragma unroll
  for (uint32_t u = 0; u < 16; ++u) xs[col * D::PM + pidx(16 * i + u)] = r[u];
}

// Between the first and the last groups: the middle stages in LDS (M = 512),
// each thread taking groups of two in turn; barriers on both sides.
template <uint32_t LOGM>
__device__ __forceinline__ void middle_stages(double *xs, const Tw *tw, double q, double qinv) {
  using D = DftShape<LOGM>;
  __syncthreads();
  if constexpr (D::S0L > 4) {
    static_assert(D::S0L == 5, "one middle stage at most");
    for (uint32_t it = threadIdx.x; it < kNttCols * D::M / 2; it += kNttThreads) {
      const uint32_t col = it % kNttCols, gi = it / kNttCols, o = gi & 15u, base = ((gi >> 4) << 5) + o;
      double r[2] = {xs[col * D::PM + pidx(base)], xs[col * D::PM + pidx(base + 16)]};
      butterflies<LOGM, 4, 1>(r, o, [&](uint32_t t) { return tw[t]; }, q, qinv);
      xs[col * D::PM + pidx(base)] = r[0];
      xs[col * D::PM + pidx(base + 16)] = r[1];
    }
    __syncthreads();
  }
}

// The last groups: column col, offset o; on return r[u] is output o + (u << S0L).
template <uint32_t LOGM>
__device__ __forceinline__ void last_stages(const double *xs, uint32_t col, uint32_t o, const Tw *tw,
                                            double (&r)[DftShape<LOGM>::E2], double q, double qinv) {
  using D = DftShape<LOGM>;
#pragma unroll
  for (uint32_t u = 0; u < D::E2; ++u) r[u] = xs[col * D::PM + pidx(o + (u << D::S0L))];
  butterflies<LOGM, D::S0L, D::R2>(r, o, [&](uint32_t t) { return tw[t]; }, q, qinv);
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
  const Tw *pre;     // pass A: multiply input n1 + N1 n2 by pre[n2] (null: by 1)
  const Tw *mid;     // pass A: multiply output (n1, k2) by mid[k2 N1 + n1]
  const Tw *dft_a;   // size-N2 DFT twiddles (N2 / 2)
  const Tw *dft_b;   // size-N1 DFT twiddles (N1 / 2)
  const Tw *post;    // pass B: multiply output k2 + N2 k1 by post[k1] (null: by 1)
  Tw inv;            // kStoreRescale: the factor applied after the subtraction
  double q, qinv;    // the modulus and fl(1 / q)
};

// A launch covers vectors v = 0 .. gridDim.y - 1, grouped into sets of vps
// consecutive vectors that share one modulus: vector v is number v % vps of
// set v / vps, whose modulus and tables are sets[v / vps].  Its words sit at
//   in   + (v / vps) * in_set_stride   + (v % vps) * in_stride   + n,
// and likewise for out and base; the intermediate of vector v at tmp + v * N.
// Each buffer's end bounds the descriptors of its accesses (buffer_extent).
struct NttPass {
  const void *in;        // pass A input
  double *tmp;           // the transposed intermediates
  void *out;             // pass B output
  const uint64_t *base;  // kStoreRescale: residues in [0, q)
  const NttSet *sets;    // device array, one entry per set
  const uint64_t *add;   // ntt_pass_b_rot: residues in [0, q) added to the first polynomials
  const void *in_end, *tmp_end, *out_end, *base_end, *add_end;   // ends of the buffers above
  uint64_t in_stride, out_stride, base_stride;
  uint64_t in_set_stride, out_set_stride, base_set_stride, add_set_stride;
  uint32_t vps, log_n1, log_n2, load, store;
  uint32_t out_transposed;  // pass B, kStoreU64 and kStoreRescale: write the transposed layout
  uint32_t nsets_shared;   // pass A: 0, or the number of sets when they all read the same input
                           // vectors (in_set_stride 0) and gridDim.x * vps is a multiple of 8
};

// The passes' global accesses.  These helpers give the work split and the
// byte offsets of every buffer access (VGPR part v, SGPR part s); the
// kernels address memory only through them, and the host replay of a
// launch (ntt_check.hip) runs the same helpers over every workgroup and
// thread to check each access against the buffer it falls in.
struct Off {
  uint32_t v, s;
};

// Pass A over DFT side N2 = 2^LOGM (other side N1): the unit of workgroup
// (bx, by) of a grid gx workgroups wide.
struct UnitA {
  uint32_t set, lv, cb;
};
__host__ __device__ inline UnitA pass_a_unit(uint32_t vps, uint32_t nsets_shared, uint32_t bx, uint32_t by,
                                             uint32_t gx) {
  UnitA a;
  a.set = by / vps;
  a.lv = by - a.set * vps;
  a.cb = bx;
  if (nsets_shared) {
    // The sets read the same input vectors: give the nsets_shared workgroups
    // of one (vector, column block) consecutive turns on one XCD (workgroup
    // ids i, i + 8, ... run there), so that the input is fetched once into
    // its L2.  The launch covers gx * vps units, a multiple of 8.
    const uint32_t id = by * gx + bx;
    const uint32_t u = id >> 3, unit = (id & 7u) + 8u * (u / nsets_shared);
    a.set = u % nsets_shared;
    a.lv = unit / gx;
    a.cb = unit - a.lv * gx;
  }
  return a;
}

template <uint32_t LOGM>
struct GeomA {
  using D = DftShape<LOGM>;
  // first groups, loop index it < IT1: column and group (kLoadU64T walks a column's groups first)
  static __host__ __device__ uint32_t col(uint32_t it, bool trans) { return trans ? it / D::I1 : it % kNttCols; }
  static __host__ __device__ uint32_t grp(uint32_t it, bool trans) { return trans ? it % D::I1 : it / kNttCols; }
  // word u of the first group ip of column n1 (row n2 = ip + I1 rev4(u))
  static __host__ __device__ Off in(uint32_t n1, uint32_t ip, uint32_t u, uint32_t N1) {
    return Off{(n1 + N1 * ip) * 8, N1 * D::I1 * 8 * rev4(u)};
  }
  // the same element in the transposed layout: n = n1 + N1 n2 at (n mod N2) N1 + n / N2
  static __host__ __device__ Off in_t(uint32_t n1, uint32_t ip, uint32_t u, uint32_t N1) {
    const uint32_t n = n1 + N1 * (ip + D::I1 * rev4(u));
    return Off{((n & (D::M - 1)) * N1 + (n >> LOGM)) * 8, 0};
  }
  static __host__ __device__ Off pre(uint32_t ip, uint32_t u) { return Off{ip * 16, D::I1 * 16 * rev4(u)}; }
  // last groups, loop index it < IT2: column, offset; word u is row k2 = o + (u << S0L)
  static __host__ __device__ uint32_t col2(uint32_t it) { return it % kNttCols; }
  static __host__ __device__ uint32_t off2(uint32_t it) { return it / kNttCols; }
  static __host__ __device__ Off tmp(uint32_t o, uint32_t n1, uint32_t u, uint32_t N1) {
    return Off{(o * N1 + n1) * 8, ((u << D::S0L) * N1) * 8};
  }
  static __host__ __device__ Off mid(uint32_t o, uint32_t n1, uint32_t u, uint32_t N1) {
    return Off{(o * N1 + n1) * 16, ((u << D::S0L) * N1) * 16};
  }
};

// Pass B over DFT side N1 = 2^LOGM (other side N2), workgroup rows r0 .. r0 + 15.
template <uint32_t LOGM>
struct GeomB {
  using D = DftShape<LOGM>;
  // first groups, it < IT1: row of the workgroup and group; word u from the row's start
  static __host__ __device__ uint32_t row(uint32_t it) { return it / D::I1; }
  static __host__ __device__ uint32_t grp(uint32_t it) { return it % D::I1; }
  static __host__ __device__ Off tmp(uint32_t row, uint32_t ip, uint32_t u) {
    return Off{(row * D::M + ip) * 8, D::I1 * 8 * rev4(u)};
  }
  // last groups, it < IT2: row and offset (out_transposed walks a row's offsets first)
  static __host__ __device__ uint32_t row2(uint32_t it, bool trans) { return trans ? it / D::I2 : it % kNttCols; }
  static __host__ __device__ uint32_t off2(uint32_t it, bool trans) { return trans ? it % D::I2 : it / kNttCols; }
  static __host__ __device__ Off post(uint32_t o, uint32_t u) { return Off{o * 16, (u << D::S0L) * 16}; }
  // output k2 + N2 k1, k1 = o + (u << S0L), in natural order and transposed
  static __host__ __device__ Off col(uint32_t k2, uint32_t o, uint32_t u, uint32_t N2) {
    return Off{(k2 + N2 * o) * 8, (N2 * 8 << D::S0L) * u};
  }
  static __host__ __device__ Off row_t(uint32_t k2, uint32_t o, uint32_t u) {
    return Off{(k2 * D::M + o) * 8, (u << D::S0L) * 8};
  }
};

// The fused pass B of the rotations (ntt_pass_b_rot, rotate.hip) over DFT
// side N1 = 2^LOGM: destination columns d_lo = o0 .. o0 + 15 of the rotation
// by Galois element g.
constexpr uint32_t kRotMax = 256;   // rotations per call (their Galois elements ride in the arguments)

struct RotArgs {
  uint32_t g[kRotMax];
  uint32_t n_rot, L;
};

template <uint32_t LOGM>
struct GeomRot {
  using D = DftShape<LOGM>;
  static constexpr uint32_t PER = kNttCols * D::M / kNttThreads;   // stores per thread
  // first groups, it < IT1: the workgroup's column and group
  static __host__ __device__ uint32_t row(uint32_t it) { return it / D::I1; }
  static __host__ __device__ uint32_t grp(uint32_t it) { return it % D::I1; }
  // the intermediate row k2 that destination column d_lo reads
  static __host__ __device__ uint32_t src_row(uint32_t g, uint32_t d_lo, uint32_t N2) {
    return (g * d_lo + (g - 1) / 2) & (N2 - 1);
  }
  static __host__ __device__ Off tmp(uint32_t k2, uint32_t ip, uint32_t u) {
    return Off{(k2 * D::M + ip) * 8, D::I1 * 8 * rev4(u)};
  }
  // last groups, it < IT2: the workgroup's column and offset; word k1 = o + (u << S0L) of row k2
  static __host__ __device__ uint32_t row2(uint32_t it) { return it / D::I2; }
  static __host__ __device__ uint32_t off2(uint32_t it) { return it % D::I2; }
  static __host__ __device__ Off word(uint32_t k2, uint32_t o, uint32_t u) {
    return Off{(k2 * D::M + o) * 8, (u << D::S0L) * 8};
  }
  // store j of thread t: column o0 + t mod 16, destination row d_hi = t / 16 + 16 j
  static __host__ __device__ Off out(uint32_t o0, uint32_t t, uint32_t j, uint32_t N2) {
    return Off{(o0 + t % kNttCols + (t / kNttCols) * N2) * 8, j * kNttCols * N2 * 8};
  }
};

// Pass A, N2 = 2^LOGM: grid (N1 / kNttCols, vectors).  The first groups of
// column n1 hold rows n2 = i' + I1 v; the quarter waves read runs of
// kNttCols columns of one row (kLoadU64T: runs of consecutive rows of one
// column, which are contiguous there).  The last groups store rows
// k2 = o + (u << S0L) of the intermediate, again in runs of kNttCols columns.
template <uint32_t LOGM>
__global__ void __launch_bounds__(kNttThreads) ntt_pass_a(const NttPass P) {
  using D = DftShape<LOGM>;
  using G = GeomA<LOGM>;
  extern __shared__ double xs[];   // [kNttCols][PM], then the M/2 DFT twiddles
  Tw *tw = (Tw *)(xs + kNttCols * D::PM);
  const UnitA un = pass_a_unit(P.vps, P.nsets_shared, blockIdx.x, blockIdx.y, gridDim.x);
  const uint32_t set = un.set, lv = un.lv, cb = un.cb;
  const NttSet S = P.sets[set];
  stage_twiddles(tw, S.dft_a, LOGM);
  Tw t1[8];
  first_twiddles<LOGM>(t1, S.dft_a);
  const uint32_t log_n1 = P.log_n1, N1 = 1u << log_n1, N2 = D::M;
  const uint64_t v = (uint64_t)set * P.vps + lv;
  const uint64_t in_off = set * P.in_set_stride + lv * P.in_stride;
  const double q = S.q, qinv = S.qinv;
  const bool trans = P.load == kLoadU64T;   // uniform
  const Buf in((const char *)P.in + in_off * 8, P.in_end);
#pragma unroll 1
  for (uint32_t it = threadIdx.x; it < D::IT1; it += kNttThreads) {
    const uint32_t cl = G::col(it, trans), ip = G::grp(it, trans);
    const uint32_t n1 = cb * kNttCols + cl;
    double r[16];
    if (trans) {   // no pre
      uint64_t w[16];
#pragma unroll
      for (uint32_t u = 0; u < 16; ++u) {
        const Off o = G::in_t(n1, ip, u, N1);
        w[u] = in.u64(o.v, o.s);
      }
#pragma unroll
      for (uint32_t u = 0; u < 16; ++u) r[u] = reduce(to_f64(w[u]), q, qinv);
    } else {
      if (P.load == kLoadF64) {
#pragma unroll
        for (uint32_t u = 0; u < 16; ++u) {
          const Off o = G::in(n1, ip, u, N1);
          r[u] = in.f64(o.v, o.s);
        }
      } else {
        uint64_t w[16];
#pragma unroll
        for (uint32_t u = 0; u < 16; ++u) {
          const Off o = G::in(n1, ip, u, N1);
          w[u] = in.u64(o.v, o.s);
        }
#pragma unroll
        for (uint32_t u = 0; u < 16; ++u) r[u] = to_f64(w[u]);
      }
      if (S.pre) {
        const Buf pre(S.pre, S.pre + N2);
#pragma unroll
        for (uint32_t u = 0; u < 16; ++u) {
          const Off o = G::pre(ip, u);
          r[u] = mul_tw(r[u], pre.tw(o.v, o.s), q);
        }
      } else {
#pragma unroll
        for (uint32_t u = 0; u < 16; ++u) r[u] = reduce(r[u], q, qinv);
      }
    }
    first_stages<LOGM>(r, t1, q, qinv);
    put_first<LOGM>(xs, cl, ip, r);
  }
  middle_stages<LOGM>(xs, tw, q, qinv);
  const Buf tmp(P.tmp + v * ((uint64_t)N1 * N2), P.tmp_end), mid(S.mid, S.mid + (size_t)N1 * N2);
#pragma unroll 1
  for (uint32_t it = threadIdx.x; it < D::IT2; it += kNttThreads) {
    const uint32_t cl = G::col2(it), o = G::off2(it), n1 = cb * kNttCols + cl;
    double r[D::E2];
    last_stages<LOGM>(xs, cl, o, tw, r, q, qinv);
#pragma unroll
    for (uint32_t u = 0; u < D::E2; ++u) {
      const Off om = G::mid(o, n1, u, N1), ot = G::tmp(o, n1, u, N1);
      tmp.put(mul_tw(r[u], mid.tw(om.v, om.s), q), ot.v, ot.s);
    }
  }
}

// Pass B, N1 = 2^LOGM: grid (N2 / kNttCols, vectors).  The first groups read
// runs of I1 consecutive words of one intermediate row k2; the last groups
// store column k2 = r0 + (lane mod kNttCols), rows k1, as runs of kNttCols
// words (out_transposed: runs of consecutive k1 of one row k2).
template <uint32_t LOGM>
__global__ void __launch_bounds__(kNttThreads) ntt_pass_b(const NttPass P) {
  using D = DftShape<LOGM>;
  using G = GeomB<LOGM>;
  extern __shared__ double xs[];   // [kNttCols][PM], then the M/2 DFT twiddles
  Tw *tw = (Tw *)(xs + kNttCols * D::PM);
  const uint32_t set = blockIdx.y / P.vps, lv = blockIdx.y - set * P.vps;
  const NttSet S = P.sets[set];
  stage_twiddles(tw, S.dft_b, LOGM);
  Tw t1[8];
  first_twiddles<LOGM>(t1, S.dft_b);
  const uint32_t N2 = 1u << P.log_n2, r0 = blockIdx.x * kNttCols, M = D::M;
  const uint64_t v = blockIdx.y;
  const double q = S.q, qinv = S.qinv;
  const Buf tmp(P.tmp + v * ((uint64_t)N2 * M) + (size_t)r0 * M, P.tmp_end);
#pragma unroll 1
  for (uint32_t it = threadIdx.x; it < D::IT1; it += kNttThreads) {
    const uint32_t row = G::row(it), ip = G::grp(it);
    double r[16];
#pragma unroll
    for (uint32_t u = 0; u < 16; ++u) {
      const Off o = G::tmp(row, ip, u);
      r[u] = tmp.f64_once(o.v, o.s);
    }
    first_stages<LOGM>(r, t1, q, qinv);
    put_first<LOGM>(xs, row, ip, r);
  }
  middle_stages<LOGM>(xs, tw, q, qinv);
  const bool transposed = P.out_transposed != 0 && P.store != kStoreF64;   // uniform
  const bool rescale = P.store == kStoreRescale;
  const Buf out((const char *)P.out + (set * P.out_set_stride + lv * P.out_stride) * 8, P.out_end);
  const Buf base(rescale ? P.base + set * P.base_set_stride + lv * P.base_stride : nullptr,
                 rescale ? P.base_end : nullptr);
#pragma unroll 1
  for (uint32_t it = threadIdx.x; it < D::IT2; it += kNttThreads) {
    const uint32_t row = G::row2(it, transposed), o = G::off2(it, transposed);
    const uint32_t k2 = r0 + row;   // output k2 + N2 k1, k1 = o + (u << S0L)
    double y[D::E2];
    last_stages<LOGM>(xs, row, o, tw, y, q, qinv);
    if (S.post) {
      const Buf post(S.post, S.post + M);
#pragma unroll
      for (uint32_t u = 0; u < D::E2; ++u) {
        const Off op = G::post(o, u);
        y[u] = mul_tw(y[u], post.tw(op.v, op.s), q);
      }
    }
    if (P.store == kStoreF64) {
#pragma unroll
      for (uint32_t u = 0; u < D::E2; ++u) {
        const Off oc = G::col(k2, o, u, N2);
        out.put(reduce(y[u], q, qinv), oc.v, oc.s);
      }
      continue;
    }
    if (rescale) {
      uint64_t bv[D::E2];
#pragma unroll
      for (uint32_t u = 0; u < D::E2; ++u) {
        const Off oc = G::col(k2, o, u, N2);
        bv[u] = base.u64_once(oc.v, oc.s);
      }
#pragma unroll
      for (uint32_t u = 0; u < D::E2; ++u) y[u] = mul_tw(to_f64(bv[u]) - y[u], S.inv, q);
    }
    if (transposed) {
#pragma unroll
      for (uint32_t u = 0; u < D::E2; ++u) {
        const Off ot = G::row_t(k2, o, u);
        out.put(to_u64(canonical(y[u], q, qinv)), ot.v, ot.s);
      }
    } else {
#pragma unroll
      for (uint32_t u = 0; u < D::E2; ++u) {
        const Off oc = G::col(k2, o, u, N2);
        out.put(to_u64(canonical(y[u], q, qinv)), oc.v, oc.s);
      }
    }
  }
}

}  // namespace fiona
