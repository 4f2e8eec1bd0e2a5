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
// descriptor holds the base; the byte offset splits into the lane's part (a
// VGPR) and a part the workgroup shares (an SGPR or a constant), so that the
// 16 accesses of a group need no vector address arithmetic.  Offsets stay
// below 2^32 bytes (one vector or one table per view).
typedef uint32_t nv2 __attribute__((ext_vector_type(2)));
typedef uint32_t nv4 __attribute__((ext_vector_type(4)));
struct Buf {
  __amdgpu_buffer_rsrc_t rs;
  // p is the same in every lane; readfirstlane keeps the descriptor in SGPRs
  // where the compiler has computed p in vector registers.
  __device__ __forceinline__ explicit Buf(const void *p) : rs(make(p)) {}
  static __device__ __forceinline__ __amdgpu_buffer_rsrc_t make(const void *p) {
    const uint64_t a = (uint64_t)p;
    // (readfirstlane returns an int: through uint32_t, so that the low half
    // is not sign-extended into the high half)
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a);
    const uint64_t u = ((uint64_t)hi << 32) | lo;
    return __builtin_amdgcn_make_buffer_rsrc((void *)u, (short)0, (int)0xFFFFFFFF, 0x00020000);
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

// Pass A, N2 = 2^LOGM: grid (N1 / kNttCols, vectors).  The first groups of
// column n1 hold rows n2 = i' + I1 v; the quarter waves read runs of
// kNttCols columns of one row (kLoadU64T: runs of consecutive rows of one
// column, which are contiguous there).  The last groups store rows
// k2 = o + (u << S0L) of the intermediate, again in runs of kNttCols columns.
template <uint32_t LOGM>
__global__ void __launch_bounds__(kNttThreads) ntt_pass_a(const NttPass P) {
  using D = DftShape<LOGM>;
  extern __shared__ double xs[];   // [kNttCols][PM], then the M/2 DFT twiddles
  Tw *tw = (Tw *)(xs + kNttCols * D::PM);
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
  Tw t1[8];
  first_twiddles<LOGM>(t1, S.dft_a);
  const uint32_t log_n1 = P.log_n1, N1 = 1u << log_n1, N2 = D::M;
  const uint64_t v = (uint64_t)set * P.vps + lv;
  const uint64_t in_off = set * P.in_set_stride + lv * P.in_stride;
  const double q = S.q, qinv = S.qinv;
  const bool trans = P.load == kLoadU64T;   // uniform
  const Buf in((const char *)P.in + in_off * 8);
  const uint32_t row_step = N1 * D::I1 * 8;   // bytes between the group's rows n2 and n2 + I1
#pragma unroll 1
  for (uint32_t it = threadIdx.x; it < D::IT1; it += kNttThreads) {
    const uint32_t cl = trans ? it / D::I1 : it % kNttCols, ip = trans ? it % D::I1 : it / kNttCols;
    const uint32_t n1 = cb * kNttCols + cl;
    double r[16];
    if (trans) {   // element n = n1 + N1 n2 sits at (n mod N2) N1 + n / N2; no pre
      uint64_t w[16];
#pragma unroll
      for (uint32_t u = 0; u < 16; ++u) {
        const uint32_t n = n1 + N1 * (ip + D::I1 * bit_reverse(u, 4));
        w[u] = in.u64(((n & (N2 - 1)) * N1 + (n >> LOGM)) * 8, 0);
      }
#pragma unroll
      for (uint32_t u = 0; u < 16; ++u) r[u] = reduce(to_f64(w[u]), q, qinv);
    } else {
      const uint32_t lane = (n1 + N1 * ip) * 8;
      if (P.load == kLoadF64) {
#pragma unroll
        for (uint32_t u = 0; u < 16; ++u) r[u] = in.f64(lane, row_step * bit_reverse(u, 4));
      } else {
        uint64_t w[16];
#pragma unroll
        for (uint32_t u = 0; u < 16; ++u) w[u] = in.u64(lane, row_step * bit_reverse(u, 4));
#pragma unroll
        for (uint32_t u = 0; u < 16; ++u) r[u] = to_f64(w[u]);
      }
      if (S.pre) {
        const Buf pre(S.pre);
#pragma unroll
        for (uint32_t u = 0; u < 16; ++u) r[u] = mul_tw(r[u], pre.tw(ip * 16, D::I1 * 16 * bit_reverse(u, 4)), q);
      } else {
#pragma unroll
        for (uint32_t u = 0; u < 16; ++u) r[u] = reduce(r[u], q, qinv);
      }
    }
    first_stages<LOGM>(r, t1, q, qinv);
    put_first<LOGM>(xs, cl, ip, r);
  }
  middle_stages<LOGM>(xs, tw, q, qinv);
  const Buf tmp(P.tmp + v * ((uint64_t)N1 * N2)), mid(S.mid);
#pragma unroll 1
  for (uint32_t it = threadIdx.x; it < D::IT2; it += kNttThreads) {
    const uint32_t cl = it % kNttCols, o = it / kNttCols, n1 = cb * kNttCols + cl;
    double r[D::E2];
    last_stages<LOGM>(xs, cl, o, tw, r, q, qinv);
    const uint32_t k = o * N1 + n1;   // the word k2 N1 + n1 of row k2 = o + (u << S0L)
#pragma unroll
    for (uint32_t u = 0; u < D::E2; ++u) {
      const uint32_t ku = (u << D::S0L) * N1;
      tmp.put(mul_tw(r[u], mid.tw(k * 16, ku * 16), q), k * 8, ku * 8);
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
  const Buf tmp(P.tmp + v * ((uint64_t)N2 * M) + (size_t)r0 * M);
#pragma unroll 1
  for (uint32_t it = threadIdx.x; it < D::IT1; it += kNttThreads) {
    const uint32_t row = it / D::I1, ip = it % D::I1;
    double r[16];
#pragma unroll
    for (uint32_t u = 0; u < 16; ++u) r[u] = tmp.f64_once((row * M + ip) * 8, D::I1 * 8 * bit_reverse(u, 4));
    first_stages<LOGM>(r, t1, q, qinv);
    put_first<LOGM>(xs, row, ip, r);
  }
  middle_stages<LOGM>(xs, tw, q, qinv);
  const bool transposed = P.out_transposed != 0 && P.store != kStoreF64;   // uniform
  const bool rescale = P.store == kStoreRescale;
  const Buf out((const char *)P.out + (set * P.out_set_stride + lv * P.out_stride) * 8);
  const Buf base(rescale ? P.base + set * P.base_set_stride + lv * P.base_stride : nullptr);
  const uint32_t col_step = N2 * 8 << D::S0L;   // bytes between outputs k1 and k1 + 2^S0L of one column
#pragma unroll 1
  for (uint32_t it = threadIdx.x; it < D::IT2; it += kNttThreads) {
    const uint32_t row = transposed ? it / D::I2 : it % kNttCols, o = transposed ? it % D::I2 : it / kNttCols;
    const uint32_t k2 = r0 + row, lane = (k2 + N2 * o) * 8;   // output k2 + N2 k1, k1 = o + (u << S0L)
    double y[D::E2];
    last_stages<LOGM>(xs, row, o, tw, y, q, qinv);
    if (S.post) {
      const Buf post(S.post);
#pragma unroll
      for (uint32_t u = 0; u < D::E2; ++u) y[u] = mul_tw(y[u], post.tw(o * 16, (u << D::S0L) * 16), q);
    }
    if (P.store == kStoreF64) {
#pragma unroll
      for (uint32_t u = 0; u < D::E2; ++u) out.put(reduce(y[u], q, qinv), lane, col_step * u);
      continue;
    }
    if (rescale) {
      uint64_t bv[D::E2];
#pragma unroll
      for (uint32_t u = 0; u < D::E2; ++u) bv[u] = base.u64_once(lane, col_step * u);
#pragma unroll
      for (uint32_t u = 0; u < D::E2; ++u) y[u] = mul_tw(to_f64(bv[u]) - y[u], S.inv, q);
    }
    if (transposed) {
#pragma unroll
      for (uint32_t u = 0; u < D::E2; ++u) out.put(to_u64(canonical(y[u], q, qinv)), (k2 * M + o) * 8, (u << D::S0L) * 8);
    } else {
#pragma unroll
      for (uint32_t u = 0; u < D::E2; ++u) out.put(to_u64(canonical(y[u], q, qinv)), lane, col_step * u);
    }
  }
}

}  // namespace fiona
