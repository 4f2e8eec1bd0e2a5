// Fused hybrid weighted-sum kernel for gfx950 (CDNA4).
//
// One workgroup owns one position tile: one RNS limb l and 64 consecutive
// coefficients k (lane = coefficient).  Every position is independent in the
// NTT domain, so a tile needs no data from any other tile.  Per tile:
//   1. each input ciphertext's two polynomials are read once from HBM and kept
//      in LDS as radix-2^25 digits (16 B per input and lane);
//   2. the signed sums that several outputs share are formed once, by Add/Sub
//      of LDS-resident inputs, and kept in LDS (Sec. 4.2 "Sharing Signed Sums");
//   3. each wavefront works through its list of work items.  An item is one
//      output, or one segment of a long output: its raw terms stream their
//      plaintext slices from HBM (each plaintext word feeds the products with
//      both ciphertext polynomials, two batches of loads in flight) and its
//      signed sums are read from LDS or formed in place and multiplied once by
//      the group's scale (Sec. 4.2 "Grouping Reconstruction Operations").  Raw
//      and signed results share one exact accumulator ("Combining the Signed
//      and Raw Routes"), reduced once to a canonical residue.  A whole output
//      is written at once; the segments of a split output leave their
//      residues in LDS and are added after a barrier.
// Plan records are wave-uniform: a wavefront loads 64 records with one vector
// load (one per lane) and broadcasts them with v_readlane into scalar registers,
// so all control flow is uniform.  No MFMA: this is modular integer arithmetic.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "modarith.hpp"

namespace fiona {

constexpr uint32_t kTile = 64;            // coefficients per workgroup (one per lane)
constexpr uint32_t kInlineSum = 0xFFFFFFFFu;
constexpr uint32_t kRawBatch = 8;         // plaintext loads per batch; two batches in flight
constexpr uint32_t kSumBatch = 8;         // member reads issued before their additions
constexpr uint32_t kSegmentFlag = 0x80000000u;

struct KParams {
  const uint64_t *in;       // [n_in][2][L][N]
  const uint64_t *pt;       // [n_pt][L][N]
  const int8_t *signs;      // [n_member of the layer description]
  const uint64_t *scales;   // [n_scale]
  uint64_t *out;            // [n_out][2][L][N]
  const LimbConst *limbs;   // [L]
  const uint4 *items;       // per work item: raw begin, raw count, use begin, use count
  const uint32_t *dest;     // per work item: output index, or kSegmentFlag | LDS segment slot
  const uint2 *waves;       // per wavefront: first item, item count
  const uint4 *splits;      // per split output: output index, first segment slot, segments, 0
  const uint2 *pm;          // per raw term: plaintext index, input index
  const uint4 *uses;        // per use: member begin, member count, LDS slot or kInlineSum, scale index | negate << 31
  const uint2 *mats;        // per LDS-resident sum: member begin, member count
  const uint2 *members;     // per member: input index, index into signs
  const uint2 *sums;        // per distinct sum: member begin, member count
  uint32_t *words;          // per member, rewritten on every call: LDS row | class << 30,
                            // each sum's members ordered added, subtracted, skipped
  uint32_t N, L, n_in, n_mat, n_split, n_sums, zero_row, tiles;
};

__device__ __forceinline__ uint64_t pair64(uint32_t lo, uint32_t hi) { return ((uint64_t)hi << 32) | lo; }

// Member words of every distinct signed sum for this call: each sum's members
// are reordered by their run-time sign (added, then subtracted, then skipped:
// Sec. 3 Obs. 2), one wavefront per sum, so that the hot loop needs no
// per-member branch.  A word is the member's LDS row (its input) | class << 30.
__global__ void __launch_bounds__(256) pack_members_kernel(const KParams P) {
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t s = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (s >= P.n_sums) return;
  const uint2 sm = P.sums[s];
  const bool valid = lane < sm.y;
  uint32_t cls = 3, row = 0;
  if (valid) {
    const uint2 m = P.members[sm.x + lane];
    const int32_t h = P.signs[m.y];
    cls = h > 0 ? 0u : (h < 0 ? 1u : 2u);
    row = m.x;
  }
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  const uint64_t b0 = __ballot(cls == 0), b1 = __ballot(cls == 1), b2 = __ballot(cls == 2);
  const uint32_t n0 = __popcll(b0), n1 = __popcll(b1);
  uint32_t pos;
  if (cls == 0) pos = __popcll(b0 & below);
  else if (cls == 1) pos = n0 + __popcll(b1 & below);
  else pos = n0 + n1 + __popcll(b2 & below);
  if (valid) P.words[sm.x + pos] = row | (cls << 30);
}

// Signed sum U = sum h x of one distinct sum, digit-wise: (U0, U1) for each
// polynomial.  wv holds the sum's member words, one per lane (lanes past the
// sum hold class 3).  The two 25-bit digits of an input are added as one 64-bit
// word (the halves never carry into each other for at most 64 members), in
// batches of 8 LDS reads; a batch past the end of its class reads the zero row.
__device__ __forceinline__ uint4 signed_sum(const KParams &P, const uint4 *lds, uint32_t wv, uint32_t lane) {
  const uint32_t cls = wv >> 30;
  const uint32_t n_pos = __popcll(__ballot(cls == 0));
  const uint32_t n_neg = __popcll(__ballot(cls == 1));
  uint64_t pa = 0, pb = 0, na = 0, nb = 0;
  for (uint32_t r = 0; r < n_pos; r += kSumBatch) {
    uint4 x[kSumBatch];
#pragma unroll
    for (uint32_t u = 0; u < kSumBatch; ++u) {
      const uint32_t w = __builtin_amdgcn_readlane(wv, r + u);
      const uint32_t row = r + u < n_pos ? (w & 0x3FFFFFFFu) : P.zero_row;
      x[u] = lds[row * kTile + lane];
    }
#pragma unroll
    for (uint32_t u = 0; u < kSumBatch; ++u) {
      pa += pair64(x[u].x, x[u].y);
      pb += pair64(x[u].z, x[u].w);
    }
  }
  const uint32_t end = n_pos + n_neg;
  for (uint32_t r = n_pos; r < end; r += kSumBatch) {
    uint4 x[kSumBatch];
#pragma unroll
    for (uint32_t u = 0; u < kSumBatch; ++u) {
      const uint32_t w = __builtin_amdgcn_readlane(wv, (r + u) & 63u);
      const uint32_t row = r + u < end ? (w & 0x3FFFFFFFu) : P.zero_row;
      x[u] = lds[row * kTile + lane];
    }
#pragma unroll
    for (uint32_t u = 0; u < kSumBatch; ++u) {
      na += pair64(x[u].x, x[u].y);
      nb += pair64(x[u].z, x[u].w);
    }
  }
  return make_uint4((uint32_t)pa - (uint32_t)na, (uint32_t)(pa >> 32) - (uint32_t)(na >> 32),
                    (uint32_t)pb - (uint32_t)nb, (uint32_t)(pb >> 32) - (uint32_t)(nb >> 32));
}

// Member words of a sum (one per lane; class 3 past its members).
__device__ __forceinline__ uint32_t load_words(const KParams &P, uint32_t mbeg, uint32_t mcnt, uint32_t lane) {
  return lane < mcnt ? P.words[mbeg + lane] : (3u << 30);
}

// Issue the plaintext loads of 8 raw terms (records r0 .. r0+7 of this chunk).
__device__ __forceinline__ void raw_issue(uint64_t (&w)[kRawBatch], const uint2 rec, uint32_t r0,
                                          const uint64_t *pt_tile, size_t LN, uint32_t lane_off) {
#pragma unroll
  for (uint32_t u = 0; u < kRawBatch; ++u) {
    const uint32_t pti = __builtin_amdgcn_readlane(rec.x, r0 + u);
    w[u] = __builtin_nontemporal_load(pt_tile + (size_t)pti * LN + lane_off);
  }
}

// Multiply-accumulate 8 raw terms whose plaintext words are in w.
__device__ __forceinline__ void raw_consume(Acc &a0, Acc &a1, const uint64_t (&w)[kRawBatch], const uint2 rec,
                                            uint32_t r0, const uint4 *lds_in, uint32_t lane) {
  uint4 x[kRawBatch];
#pragma unroll
  for (uint32_t u = 0; u < kRawBatch; ++u) {
    const uint32_t ini = __builtin_amdgcn_readlane(rec.y, r0 + u);
    x[u] = lds_in[ini * kTile + lane];
  }
#pragma unroll
  for (uint32_t u = 0; u < kRawBatch; ++u) {
    const uint32_t w0 = lo_digit(w[u]), w1 = hi_digit(w[u]), ws = w0 + w1;
    mac(a0, x[u].x, x[u].y, w0, w1, ws);
    mac(a1, x[u].z, x[u].w, w0, w1, ws);
  }
}

template <int NW>
__global__ void __launch_bounds__(NW * 64) hybrid_linear_kernel(const KParams P) {
  extern __shared__ uint4 lds[];   // [n_in + n_mat + segment slots][kTile]
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t limb = blockIdx.x / P.tiles;
  const uint32_t tile = blockIdx.x - limb * P.tiles;
  const uint32_t k0 = tile * kTile;
  const uint32_t k = k0 + lane;
  // lanes past N (partial last tile) read a valid coefficient and store nothing
  const uint32_t lane_off = (k < P.N ? k : P.N - 1) - k0;
  const size_t LN = (size_t)P.L * P.N;
  const LimbConst lc = P.limbs[limb];

  // 1. stage this tile of every input ciphertext (read once)
  for (uint32_t i = wave; i < P.n_in; i += NW) {
    const uint64_t *src = P.in + ((size_t)i * 2 * P.L + limb) * P.N + k0;
    const uint64_t a = __builtin_nontemporal_load(src + lane_off);
    const uint64_t b = __builtin_nontemporal_load(src + LN + lane_off);
    lds[i * kTile + lane] = make_uint4(lo_digit(a), hi_digit(a), lo_digit(b), hi_digit(b));
  }
  if (wave == NW - 1) lds[P.zero_row * kTile + lane] = make_uint4(0, 0, 0, 0);   // padding row of sums
  __syncthreads();

  // 2. shared signed sums, formed once per tile
  uint4 *sums = lds + (size_t)P.n_in * kTile;
  for (uint32_t s = wave; s < P.n_mat; s += NW) {
    const uint2 m = P.mats[s];
    sums[s * kTile + lane] = signed_sum(P, lds, load_words(P, m.x, m.y, lane), lane);
  }
  __syncthreads();

  // 3. this wavefront's work items
  uint4 *segs = sums + (size_t)P.n_mat * kTile;
  const uint64_t *pt_tile = P.pt + (size_t)limb * P.N + k0;
  const uint2 wr = P.waves[wave];
  for (uint32_t it = wr.x; it < wr.x + wr.y; ++it) {
    const uint4 item = P.items[it];
    const uint32_t dest = P.dest[it];
    Acc a0, a1;
    acc_zero(a0);
    acc_zero(a1);
    uint64_t r0 = 0, r1 = 0;

    // raw route: one PMult per term
    uint32_t since_fold = 0;
    for (uint32_t base = 0; base < item.y; base += 64) {
      const uint32_t n = min(64u, item.y - base);
      uint2 rec = make_uint2(0, 0);
      if (lane < n) rec = P.pm[item.x + base + lane];
      if (since_fold + n > kFoldTerms) {   // keep the accumulators exact
        r0 = finish(a0, r0, lc);
        r1 = finish(a1, r1, lc);
        acc_zero(a0);
        acc_zero(a1);
        since_fold = 0;
      }
      since_fold += n;
      const uint32_t nb = n / kRawBatch;
      uint64_t wa[kRawBatch], wb[kRawBatch];
      if (nb > 0) raw_issue(wa, rec, 0, pt_tile, LN, lane_off);
      for (uint32_t b = 0; b < nb; b += 2) {
        if (b + 1 < nb) raw_issue(wb, rec, (b + 1) * kRawBatch, pt_tile, LN, lane_off);
        raw_consume(a0, a1, wa, rec, b * kRawBatch, lds, lane);
        if (b + 1 < nb) {
          if (b + 2 < nb) raw_issue(wa, rec, (b + 2) * kRawBatch, pt_tile, LN, lane_off);
          raw_consume(a0, a1, wb, rec, (b + 1) * kRawBatch, lds, lane);
        }
      }
      for (uint32_t r = nb * kRawBatch; r < n; ++r) {
        const uint32_t pti = __builtin_amdgcn_readlane(rec.x, r);
        const uint32_t ini = __builtin_amdgcn_readlane(rec.y, r);
        const uint64_t w = __builtin_nontemporal_load(pt_tile + (size_t)pti * LN + lane_off);
        const uint4 x = lds[ini * kTile + lane];
        const uint32_t w0 = lo_digit(w), w1 = hi_digit(w), ws = w0 + w1;
        mac(a0, x.x, x.y, w0, w1, ws);
        mac(a1, x.z, x.w, w0, w1, ws);
      }
    }

    // signed route: each use applies its group's scale once to a signed sum
    since_fold = 0;
    for (uint32_t base = 0; base < item.w; base += 64) {
      const uint32_t n = min(64u, item.w - base);
      uint4 rec = make_uint4(0, 0, kInlineSum, 0);
      uint32_t scl = 0;
      if (lane < n) {
        rec = P.uses[item.z + base + lane];
        scl = (uint32_t)P.scales[rec.w & 0x7FFFFFFFu];   // scales are < 2^20
      }
      if (since_fold + n > kFoldTerms) {
        r0 = finish(a0, r0, lc);
        r1 = finish(a1, r1, lc);
        acc_zero(a0);
        acc_zero(a1);
        since_fold = 0;
      }
      since_fold += n;
      // member words of the next in-place sum are loaded while the current one is added
      uint32_t wnext = __builtin_amdgcn_readlane(rec.z, 0) == kInlineSum
                           ? load_words(P, __builtin_amdgcn_readlane(rec.x, 0), __builtin_amdgcn_readlane(rec.y, 0), lane)
                           : (3u << 30);
      for (uint32_t r = 0; r < n; ++r) {
        const uint32_t slot = __builtin_amdgcn_readlane(rec.z, r);
        const uint32_t sc = __builtin_amdgcn_readlane(rec.w, r);
        const uint32_t wcur = wnext;
        if (r + 1 < n && __builtin_amdgcn_readlane(rec.z, r + 1) == kInlineSum)
          wnext = load_words(P, __builtin_amdgcn_readlane(rec.x, r + 1), __builtin_amdgcn_readlane(rec.y, r + 1), lane);
        const uint4 U = slot != kInlineSum ? sums[slot * kTile + lane] : signed_sum(P, lds, wcur, lane);
        const int32_t cabs = (int32_t)__builtin_amdgcn_readlane(scl, r);
        const int32_t c = (sc >> 31) ? -cabs : cabs;
        smac(a0, c, (int32_t)U.x, (int32_t)U.y);
        smac(a1, c, (int32_t)U.z, (int32_t)U.w);
      }
    }

    const uint64_t y0 = finish(a0, r0, lc);
    const uint64_t y1 = finish(a1, r1, lc);
    if (dest & kSegmentFlag) {
      segs[(dest & ~kSegmentFlag) * kTile + lane] =
          make_uint4((uint32_t)y0, (uint32_t)(y0 >> 32), (uint32_t)y1, (uint32_t)(y1 >> 32));
    } else if (k < P.N) {
      uint64_t *dst = P.out + ((size_t)dest * 2 * P.L + limb) * P.N + k;
      __builtin_nontemporal_store(y0, dst);
      __builtin_nontemporal_store(y1, dst + LN);
    }
  }

  // 4. outputs that were split across wavefronts: add their segments' residues
  if (P.n_split) {
    __syncthreads();
    for (uint32_t s = wave; s < P.n_split; s += NW) {
      const uint4 sp = P.splits[s];
      uint64_t y0 = 0, y1 = 0;   // at most kMaxSegments residues < 2^50: no overflow
      for (uint32_t g = 0; g < sp.z; ++g) {
        const uint4 v = segs[(sp.y + g) * kTile + lane];
        y0 += pair64(v.x, v.y);
        y1 += pair64(v.z, v.w);
      }
      y0 = reduce_i64((int64_t)y0, lc.q, lc.qinv);
      y1 = reduce_i64((int64_t)y1, lc.q, lc.qinv);
      if (k < P.N) {
        uint64_t *dst = P.out + ((size_t)sp.x * 2 * P.L + limb) * P.N + k;
        __builtin_nontemporal_store(y0, dst);
        __builtin_nontemporal_store(y1, dst + LN);
      }
    }
  }
}

}  // namespace fiona
