// Fused hybrid weighted-sum kernel for gfx950 (CDNA4).
//
// One workgroup owns one position tile: one RNS limb l and 64 consecutive
// coefficients k (lane = coefficient).  Every position is independent in the
// NTT domain, so a tile needs no data from any other tile.  Per tile:
//   1. each input ciphertext's two polynomials are read once from HBM and kept
//      in LDS as radix-2^25 digits (16 B per input and lane);
//   2. the signed sums that several outputs share are formed once, by Add/Sub
//      of LDS-resident inputs, and kept in LDS (Sec. 4.2 "Sharing Signed Sums");
//   3. the wavefronts take outputs in turn; for each output the raw terms
//      stream their plaintext slices from HBM (each plaintext word feeds the
//      products with both ciphertext polynomials) and the output's signed sums
//      are either read from LDS or formed in place and multiplied once by the
//      group's scale (Sec. 4.2 "Grouping Reconstruction Operations"); raw and
//      signed results share one exact accumulator ("Combining the Signed and
//      Raw Routes"), reduced once to a canonical residue and written once.
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
constexpr uint32_t kRawBatch = 8;         // plaintext loads issued before their products

struct KParams {
  const uint64_t *in;      // [n_in][2][L][N]
  const uint64_t *pt;      // [n_pt][L][N]
  const int8_t *signs;     // [n_member of the layer description]
  const uint64_t *scales;  // [n_scale]
  uint64_t *out;           // [n_out][2][L][N]
  const LimbConst *limbs;  // [L]
  const uint4 *outs;       // per output: raw begin, raw count, use begin, use count
  const uint2 *pm;         // per raw term: plaintext index, input index
  const uint4 *uses;       // per use: member begin, member count, LDS slot or kInlineSum, scale index | negate << 31
  const uint2 *mats;       // per LDS-resident sum: member begin, member count
  const uint2 *members;    // per member: input index, index into signs
  uint32_t N, L, n_in, n_out, n_mat, tiles;
};

// Signed sum of up to 64 members, digit-wise: (U0, U1) for each polynomial.
// Member signs are read from the run-time sign array; +1 adds, -1 subtracts,
// 0 skips (Sec. 3 Obs. 2).
__device__ __forceinline__ uint4 signed_sum(const KParams &P, const uint4 *lds_in, uint32_t mbeg,
                                            uint32_t mcnt, uint32_t lane) {
  uint32_t packed = 0;
  if (lane < mcnt) {
    const uint2 m = P.members[mbeg + lane];
    const int32_t h = P.signs[m.y];
    packed = m.x | ((uint32_t)(h & 3) << 30);   // +1 -> 1, -1 -> 3, 0 -> 0
  }
  int32_t u0a = 0, u1a = 0, u0b = 0, u1b = 0;
  for (uint32_t r = 0; r < mcnt; ++r) {
    const uint32_t pk = __builtin_amdgcn_readlane(packed, r);
    const uint32_t code = pk >> 30;
    if (code == 1) {
      const uint4 x = lds_in[(pk & 0x3FFFFFFFu) * kTile + lane];
      u0a += (int32_t)x.x; u1a += (int32_t)x.y; u0b += (int32_t)x.z; u1b += (int32_t)x.w;
    } else if (code == 3) {
      const uint4 x = lds_in[(pk & 0x3FFFFFFFu) * kTile + lane];
      u0a -= (int32_t)x.x; u1a -= (int32_t)x.y; u0b -= (int32_t)x.z; u1b -= (int32_t)x.w;
    }
  }
  return make_uint4((uint32_t)u0a, (uint32_t)u1a, (uint32_t)u0b, (uint32_t)u1b);
}

template <int NW>
__global__ void __launch_bounds__(NW * 64) hybrid_linear_kernel(const KParams P) {
  extern __shared__ uint4 lds[];   // [n_in + n_mat][kTile]
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t limb = blockIdx.x / P.tiles;
  const uint32_t tile = blockIdx.x - limb * P.tiles;
  const uint32_t k0 = tile * kTile;
  const uint32_t k = k0 + lane;
  // lanes past N (partial last tile) read a valid coefficient and store nothing
  const uint32_t lc_off = (k < P.N ? k : P.N - 1) - k0;
  const size_t LN = (size_t)P.L * P.N;
  const LimbConst lc = P.limbs[limb];

  // 1. stage this tile of every input ciphertext (read once)
  for (uint32_t i = wave; i < P.n_in; i += NW) {
    const uint64_t *src = P.in + ((size_t)i * 2 * P.L + limb) * P.N + k0;
    const uint64_t a = __builtin_nontemporal_load(src + lc_off);
    const uint64_t b = __builtin_nontemporal_load(src + LN + lc_off);
    lds[i * kTile + lane] = make_uint4(lo_digit(a), hi_digit(a), lo_digit(b), hi_digit(b));
  }
  __syncthreads();

  // 2. shared signed sums, formed once per tile
  uint4 *sums = lds + (size_t)P.n_in * kTile;
  for (uint32_t s = wave; s < P.n_mat; s += NW) {
    const uint2 m = P.mats[s];
    sums[s * kTile + lane] = signed_sum(P, lds, m.x, m.y, lane);
  }
  __syncthreads();

  // 3. outputs, one wavefront each in turn
  const uint64_t *pt_tile = P.pt + (size_t)limb * P.N + k0;
  for (uint32_t j = wave; j < P.n_out; j += NW) {
    const uint4 od = P.outs[j];
    Acc a0, a1;
    acc_zero(a0);
    acc_zero(a1);
    uint64_t r0 = 0, r1 = 0;

    // raw route: one PMult per term, plaintexts streamed from HBM
    for (uint32_t f = 0; f < od.y; f += kFoldTerms) {
      const uint32_t fend = min(od.y, f + kFoldTerms);
      for (uint32_t base = f; base < fend; base += 64) {
        const uint32_t n = min(64u, fend - base);
        uint2 rec = make_uint2(0, 0);
        if (lane < n) rec = P.pm[od.x + base + lane];
        uint32_t r = 0;
        for (; r + kRawBatch <= n; r += kRawBatch) {
          uint64_t w[kRawBatch];
          uint4 x[kRawBatch];
#pragma unroll
          for (uint32_t u = 0; u < kRawBatch; ++u) {
            const uint32_t pti = __builtin_amdgcn_readlane(rec.x, r + u);
            const uint32_t ini = __builtin_amdgcn_readlane(rec.y, r + u);
            w[u] = __builtin_nontemporal_load(pt_tile + (size_t)pti * LN + lc_off);
            x[u] = lds[ini * kTile + lane];
          }
#pragma unroll
          for (uint32_t u = 0; u < kRawBatch; ++u) {
            const uint32_t w0 = lo_digit(w[u]), w1 = hi_digit(w[u]), ws = w0 + w1;
            mac(a0, x[u].x, x[u].y, w0, w1, ws);
            mac(a1, x[u].z, x[u].w, w0, w1, ws);
          }
        }
        for (; r < n; ++r) {
          const uint32_t pti = __builtin_amdgcn_readlane(rec.x, r);
          const uint32_t ini = __builtin_amdgcn_readlane(rec.y, r);
          const uint64_t w = __builtin_nontemporal_load(pt_tile + (size_t)pti * LN + lc_off);
          const uint4 x = lds[ini * kTile + lane];
          const uint32_t w0 = lo_digit(w), w1 = hi_digit(w), ws = w0 + w1;
          mac(a0, x.x, x.y, w0, w1, ws);
          mac(a1, x.z, x.w, w0, w1, ws);
        }
      }
      if (fend < od.y) {   // keep the accumulators exact: fold into the running residue
        r0 = finish(a0, r0, lc);
        r1 = finish(a1, r1, lc);
        acc_zero(a0);
        acc_zero(a1);
      }
    }

    // signed route: each use applies its group's scale once to a signed sum
    for (uint32_t f = 0; f < od.w; f += kFoldTerms) {
      const uint32_t fend = min(od.w, f + kFoldTerms);
      for (uint32_t base = f; base < fend; base += 64) {
        const uint32_t n = min(64u, fend - base);
        uint4 rec = make_uint4(0, 0, 0, 0);
        if (lane < n) rec = P.uses[od.z + base + lane];
        for (uint32_t r = 0; r < n; ++r) {
          const uint32_t mbeg = __builtin_amdgcn_readlane(rec.x, r);
          const uint32_t mcnt = __builtin_amdgcn_readlane(rec.y, r);
          const uint32_t slot = __builtin_amdgcn_readlane(rec.z, r);
          const uint32_t sc = __builtin_amdgcn_readlane(rec.w, r);
          const uint4 U = slot != kInlineSum ? sums[slot * kTile + lane]
                                             : signed_sum(P, lds, mbeg, mcnt, lane);
          const int32_t cabs = (int32_t)(uint32_t)P.scales[sc & 0x7FFFFFFFu];
          const int32_t c = (sc >> 31) ? -cabs : cabs;
          smac(a0, c, (int32_t)U.x, (int32_t)U.y);
          smac(a1, c, (int32_t)U.z, (int32_t)U.w);
        }
      }
      if (fend < od.w) {
        r0 = finish(a0, r0, lc);
        r1 = finish(a1, r1, lc);
        acc_zero(a0);
        acc_zero(a1);
      }
    }

    const uint64_t y0 = finish(a0, r0, lc);
    const uint64_t y1 = finish(a1, r1, lc);
    if (k < P.N) {
      uint64_t *dst = P.out + ((size_t)j * 2 * P.L + limb) * P.N + k;
      __builtin_nontemporal_store(y0, dst);
      __builtin_nontemporal_store(y1, dst + LN);
    }
  }
}

}  // namespace fiona
