// Fused hybrid weighted-sum kernel for gfx950 (CDNA4).
//
// One workgroup owns one position tile: one RNS limb l and 64 consecutive
// coefficients k (lane = coefficient).  Every position is independent in the
// NTT domain, so a tile needs no data from any other tile.  Per tile:
//   1. each input ciphertext's two polynomials are read once from HBM and kept
//      in LDS as radix-2^25 digits (16 B per input and lane);
//   2. signed terms common to several sums (partial overlaps) are formed once,
//      reduced to residues and kept in LDS as extra rows (Sec. 4.2, the
//      sharing candidates); the signed sums that several outputs share are
//      formed once, by Add/Sub of LDS rows, and kept in LDS (Sec. 4.2
//      "Sharing Signed Sums");
//   3. each wavefront works through its list of work items.  An item is one
//      output, or one segment of a long output: its raw terms stream their
//      plaintext slices from HBM (each plaintext word feeds the products with
//      both ciphertext polynomials, two batches of loads in flight) and its
//      signed sums, formed between the raw batches while their loads are in
//      flight, are read from LDS or formed in place and multiplied once by
//      the group's scale (Sec. 4.2 "Grouping Reconstruction Operations").  Raw
//      and signed results share one exact accumulator ("Combining the Signed
//      and Raw Routes"), reduced once to a canonical residue.  A whole output
//      is written at once; the segments of a split output leave their
//      residues in LDS and are added after a barrier.
// Plan records are wave-uniform.  Work items, raw-term records, use headers
// and the member words of signed sums are all read with scalar loads straight
// into SGPRs (every tile reads the same records, so they stay in the scalar
// cache).  All control flow is uniform.  No MFMA: this is modular integer
// arithmetic.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "buffer.hpp"
#include "modarith.hpp"

namespace fiona {

constexpr uint32_t kTile = 64;            // coefficients per workgroup (one per lane)
constexpr uint32_t kRowBytes = kTile * 16;   // one LDS row: 16 B per lane
constexpr uint32_t kInlineSum = 0xFFFFFFFFu;
constexpr uint32_t kRawBatch = 8;         // plaintext loads per batch; two batches in flight
constexpr uint32_t kRawBatches = kChunkTerms / kRawBatch;   // batches per chunk of raw records
constexpr uint32_t kChunkSlots = 64;      // records per chunk block; the last one is the header
constexpr uint32_t kSumBatch = 4;         // member reads issued before their additions
constexpr uint32_t kSumBatches = kMaxMembers / kSumBatch;
constexpr uint32_t kSumWords = 64;        // words per block: 4 header words + member rows
constexpr uint32_t kAddWord = 4;          // first word of the rows to add
constexpr uint32_t kUseBlock = 0x40000000u;   // block flag: a use (its header carries a slot and a signed scale)
constexpr uint32_t kSegmentFlag = 0x80000000u;   // item destination: a segment slot in LDS
constexpr uint32_t kBufferFlag = 0x40000000u;    // item destination: a row of the output buffer in LDS
constexpr uint32_t kNormaliseSigns = 0x80000000u;   // block flag: signs relative to the first member's
constexpr uint32_t kMaxLevels = 4;        // levels of common partial sums
constexpr int kLoadNT = 2;                // cache policy of the plaintext stream: nontemporal
constexpr int kStoreNT = 2;               // cache policy of the output stores: nontemporal
static_assert(kChunkTerms % kRawBatch == 0 && kChunkTerms < kChunkSlots, "chunk layout");
// header, rows to add from word 4 up, rows to subtract from word 63 down; a batch read of either list
// (four words) stays inside the block
static_assert(kAddWord + kMaxMembers <= kSumWords && kAddWord + kSumBatch * kSumBatches <= kSumWords,
              "sum block layout");
static_assert(kAddWord % kSumBatch == 0 && kSumWords % kSumBatch == 0, "member batches are 16-byte aligned");

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Per-call description for the sign-packing kernel.  Word blocks: the common
// partial sums, the resident signed sums, then one block per use.
struct PackParams {
  const int8_t *signs;      // [n_member of the layer description]
  const uint2 *members;     // per member: LDS row, index into signs
  const uint4 *blocks;      // per block: member begin, member count (<= kMaxMembers) | kNormaliseSigns |
                            // kUseBlock, resident slot or kInlineSum, scale index | negate << 31
  uint32_t *words;          // per block: kSumWords words
  const uint64_t *scales;   // [n_scale of the layer description]
  uint32_t n_blocks;
};

// Scalars of the main kernel.  LDS rows: inputs, common partial sums (level by
// level; level l ends at level_end[l]), resident signed sums, segment slots,
// the zero row, then the output buffer (from row obuf_row).  The outputs are
// produced in n_rounds rounds; each round ends with a barrier after which the
// round's buffered outputs and split outputs are written out together.
struct KShape {
  uint32_t N, L, n_in, n_part, n_levels, n_mat, zero_row, tiles, n_rounds, obuf_row, use_block0;
  uint32_t level_end[kMaxLevels];
};

__device__ __forceinline__ uint64_t pair64(uint32_t lo, uint32_t hi) { return ((uint64_t)hi << 32) | lo; }

// The word blocks of this call.  Word 0 holds the numbers of rows to add and
// to subtract; word 1 the LDS slot of a resident sum (a use of it) or
// kInlineSum; word 2 a use's signed scale (-1)^negate * c (c < 2^20); word 3
// is 0.  The rows to add follow from word 4 upwards and the rows to subtract
// from word 63 downwards; a row is given as its LDS byte offset.  Members
// whose run-time sign is 0 are left out (Sec. 3 Obs. 2, the skip).  A common
// partial sum takes its signs relative to its first member's, so it is the
// same term in every sum that contains it.  One wavefront per block.
__global__ void __launch_bounds__(256) pack_members_kernel(const PackParams P) {
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= P.n_blocks) return;
  const uint4 bk = P.blocks[b];
  const uint32_t cnt = bk.y & 0xFFFFu;
  const int32_t h0 = (bk.y & kNormaliseSigns) ? (int32_t)P.signs[P.members[bk.x].y] : 1;
  uint32_t cls = 3, row = 0;
  if (lane < cnt) {
    const uint2 m = P.members[bk.x + lane];
    const int32_t h = P.signs[m.y] * h0;
    cls = h > 0 ? 0u : (h < 0 ? 1u : 2u);
    row = m.x;
  }
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  const uint64_t b0 = __ballot(cls == 0), b1 = __ballot(cls == 1);
  const uint32_t n0 = __popcll(b0), n1 = __popcll(b1);
  uint32_t *w = P.words + (size_t)b * kSumWords;
  if (cls == 0) w[kAddWord + __popcll(b0 & below)] = row * kRowBytes;
  if (cls == 1) w[kSumWords - 1 - __popcll(b1 & below)] = row * kRowBytes;
  if (lane == 0) w[0] = n0 | (n1 << 16);
  if (lane == 1) w[1] = bk.z;
  if (lane == 2) {
    int32_t sc = 0;
    if (bk.y & kUseBlock) {
      const int32_t c = (int32_t)P.scales[bk.w & 0x7FFFFFFFu];
      sc = (bk.w >> 31) ? -c : c;
    }
    w[2] = (uint32_t)sc;
  }
  if (lane == 3) w[3] = 0;
}

__device__ __forceinline__ const uint4 &lds_row(const uint4 *lds, uint32_t row_bytes, uint32_t lane_bytes) {
  return *(const uint4 *)((const char *)lds + row_bytes + lane_bytes);
}

// Scalar (SMEM) loads of plan records.  Every wavefront of every tile reads
// the same records, so they come from the scalar cache straight into SGPRs:
// no vector load and no v_readlane per record.  The address must be uniform.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x8 __attribute__((ext_vector_type(8)));
typedef const __attribute__((address_space(4))) uint32_t *cu32p;
typedef const __attribute__((address_space(4))) u32x2 *cu32x2p;
typedef const __attribute__((address_space(4))) u32x4 *cu32x4p;
typedef const __attribute__((address_space(4))) u32x8 *cu32x8p;
__device__ __forceinline__ uint32_t sload1(const void *p) { return *(cu32p)p; }
__device__ __forceinline__ u32x2 sload2(const void *p) { return *(cu32x2p)p; }
__device__ __forceinline__ u32x4 sload4(const void *p) { return *(cu32x4p)p; }
__device__ __forceinline__ u32x8 sload8(const void *p) { return *(cu32x8p)p; }
__device__ __forceinline__ uint4 as_uint4(u32x4 v) { return make_uint4(v.x, v.y, v.z, v.w); }
__device__ __forceinline__ uint2 as_uint2(u32x2 v) { return make_uint2(v.x, v.y); }

// Adds the kSumBatch rows whose LDS byte offsets are in r into the packed digit sums.
__device__ __forceinline__ void sum_batch(uint64_t &a, uint64_t &b, u32x4 r, const uint4 *lds, uint32_t lane16) {
  uint4 x[kSumBatch];
#pragma unroll
  for (int u = 0; u < (int)kSumBatch; ++u) x[u] = lds_row(lds, r[u], lane16);
#pragma unroll
  for (int u = 0; u < (int)kSumBatch; ++u) {
    a += pair64(x[u].x, x[u].y);
    b += pair64(x[u].z, x[u].w);
  }
}

// Signed sum U = sum h x of the word block blk (uniform address; hdr = its
// word 0), digit-wise: (U0, U1) for each polynomial.  The two 25-bit digits
// of an input are added as one 64-bit word (the halves never carry into each
// other for at most 48 members), in batches of kSumBatch LDS reads whose row
// offsets come from scalar loads.
// The first n (1 .. 3) rows of a batch whose offsets are in r (first, the
// rows to add) or its last n (the rows to subtract, stored downwards).
__device__ __forceinline__ void sum_tail(uint64_t &a, uint64_t &b, u32x4 r, uint32_t n, bool first, const uint4 *lds,
                                         uint32_t lane16) {
  const uint32_t o = first ? 0u : kSumBatch - n;
  uint4 x = lds_row(lds, r[o], lane16);
  a += pair64(x.x, x.y);
  b += pair64(x.z, x.w);
  if (n > 1) {
    x = lds_row(lds, r[o + 1], lane16);
    a += pair64(x.x, x.y);
    b += pair64(x.z, x.w);
  }
  if (n > 2) {
    x = lds_row(lds, r[o + 2], lane16);
    a += pair64(x.x, x.y);
    b += pair64(x.z, x.w);
  }
}

// Full batches of four rows, then the rest one row at a time: padding the
// lists to whole batches with the zero row cost about three extra row reads
// per sum (BERT: a fifth of all LDS reads); exact counts measured 0.8-1.4%
// faster on BERT and the kernel's code 40% smaller (rolled batch loops).
__device__ __forceinline__ uint4 signed_sum(const uint32_t *blk, uint32_t hdr, const uint4 *lds, uint32_t lane16) {
  const uint32_t np = hdr & 0xFFFFu, nn = hdr >> 16;
  uint64_t pa = 0, pb = 0, na = 0, nb = 0;
  uint32_t k = 0;
  for (; (k + 1) * kSumBatch <= np; ++k) sum_batch(pa, pb, sload4(blk + kAddWord + k * kSumBatch), lds, lane16);
  if (k * kSumBatch < np) sum_tail(pa, pb, sload4(blk + kAddWord + k * kSumBatch), np - k * kSumBatch, true, lds, lane16);
  k = 0;
  for (; (k + 1) * kSumBatch <= nn; ++k)
    sum_batch(na, nb, sload4(blk + kSumWords - (k + 1) * kSumBatch), lds, lane16);
  if (k * kSumBatch < nn)
    sum_tail(na, nb, sload4(blk + kSumWords - (k + 1) * kSumBatch), nn - k * kSumBatch, false, lds, lane16);
  return make_uint4((uint32_t)pa - (uint32_t)na, (uint32_t)(pa >> 32) - (uint32_t)(na >> 32),
                    (uint32_t)pb - (uint32_t)nb, (uint32_t)(pb >> 32) - (uint32_t)(nb >> 32));
}

// Raw-term chunks.  A chunk block holds kChunkSlots plaintext offsets, then
// kChunkSlots input rows; record r < 8 nb is (offset r, row r): the byte
// offset of the term's plaintext from the chunk base and the LDS byte offset
// of its input row.  Padding records point at offset 0 and the all-zero row,
// so they add nothing.  Slot kChunkSlots-1 of the two halves is the header:
// chunk base bits 0..31, and bits 32..47 | nb << 16; the chunk base is a byte
// offset into the plaintext table.  A plaintext is read with a buffer load:
// descriptor base = this tile's plaintext column at the chunk base, and lane
// offset plus record offset in the VGPR offset (an SGPR offset that changes
// from load to load streamed measurably slower).  A batch's offsets and rows
// are loaded separately, so only the offsets of the batch about to be issued
// and the rows of the batch being multiplied occupy SGPRs.
__device__ __forceinline__ u32x8 batch_offsets(const uint32_t *blk, uint32_t b) { return sload8(blk + b * kRawBatch); }
__device__ __forceinline__ u32x8 batch_rows(const uint32_t *blk, uint32_t b) {
  return sload8(blk + kChunkSlots + b * kRawBatch);
}

// Issue the plaintext loads of one batch, offsets in SGPRs.
__device__ __forceinline__ void raw_issue_s(u32x2 (&w)[kRawBatch], __amdgpu_buffer_rsrc_t rs, u32x8 off,
                                            uint32_t voff) {
#pragma unroll
  for (uint32_t u = 0; u < kRawBatch; ++u) w[u] = __builtin_amdgcn_raw_buffer_load_b64(rs, voff + off[u], 0, kLoadNT);
}

// Multiply-accumulate one batch whose plaintext words are in w, input rows in SGPRs.
__device__ __forceinline__ void raw_consume_s(Acc &a0, Acc &a1, const u32x2 (&w)[kRawBatch], u32x8 row,
                                              const uint4 *lds, uint32_t lane16) {
#pragma unroll
  for (uint32_t h = 0; h < kRawBatch; h += 4) {
    uint4 x[4];
#pragma unroll
    for (uint32_t u = 0; u < 4; ++u) x[u] = lds_row(lds, row[h + u], lane16);
#pragma unroll
    for (uint32_t u = 0; u < 4; ++u) {
      mac(a0, x[u].x, x[u].y, w[h + u].x, w[h + u].y);
      mac(a1, x[u].z, x[u].w, w[h + u].x, w[h + u].y);
    }
  }
}

__device__ __forceinline__ const uint32_t *sload_block(const uint2 *pm, uint32_t chunk) {
  return (const uint32_t *)(pm + (size_t)chunk * kChunkSlots);
}

// All batches of the chunk block blk (uniform address), records in SGPRs:
// batch b+1 is in flight while batch b is multiplied, and fill() (signed-
// route work, which reads no HBM) runs before each batch is multiplied, so
// that the batch's plaintext loads have longer to arrive.  pt_end: the end
// of the plaintext table.
template <typename Fill>
__device__ __forceinline__ void raw_chunk(const uint32_t *blk, const char *pt_tile, const void *pt_end, uint32_t voff,
                                          Acc &a0, Acc &a1, const uint4 *lds, uint32_t lane16, Fill &&fill) {
  const uint32_t hlo = sload1(blk + kChunkSlots - 1), hhi = sload1(blk + 2 * kChunkSlots - 1);
  const uint32_t nb = hhi >> 16;
  const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(pt_tile + pair64(hlo, hhi & 0xFFFFu), pt_end);
  u32x2 wa[kRawBatch], wb[kRawBatch];
  raw_issue_s(wa, rs, batch_offsets(blk, 0), voff);
  uint32_t b = 0;
  for (; b + 2 < nb; b += 2) {   // batch b is in flight in wa
    raw_issue_s(wb, rs, batch_offsets(blk, b + 1), voff);
    fill();
    raw_consume_s(a0, a1, wa, batch_rows(blk, b), lds, lane16);
    raw_issue_s(wa, rs, batch_offsets(blk, b + 2), voff);
    fill();
    raw_consume_s(a0, a1, wb, batch_rows(blk, b + 1), lds, lane16);
  }
  if (b + 1 < nb) {   // two batches left, the first in flight in wa
    raw_issue_s(wb, rs, batch_offsets(blk, b + 1), voff);
    fill();
    raw_consume_s(a0, a1, wa, batch_rows(blk, b), lds, lane16);
    fill();
    raw_consume_s(a0, a1, wb, batch_rows(blk, b + 1), lds, lane16);
  } else {
    fill();
    raw_consume_s(a0, a1, wa, batch_rows(blk, b), lds, lane16);
  }
}

// Stores one output position of both polynomials: row = the output's limb
// row at this tile (polynomial 0), poly_bytes = the distance to polynomial 1,
// out_end = the end of the output array.  Nontemporal buffer stores
// (measured faster than default-policy stores by 13% on a VGG11-sized layer,
// and than device-scope ones by 2%).
// ADD (a later input pass): y += the stored output, mod q.
template <bool ADD>
__device__ __forceinline__ void store_out(uint64_t *row, const void *out_end, uint32_t lane_bytes, uint32_t poly_bytes,
                                          uint64_t y0, uint64_t y1, uint64_t q) {
  const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(row, out_end);
  if constexpr (ADD) {
    const u32x2 o0 = __builtin_amdgcn_raw_buffer_load_b64(rs, lane_bytes, 0, 0);
    const u32x2 o1 = __builtin_amdgcn_raw_buffer_load_b64(rs, lane_bytes + poly_bytes, 0, 0);
    y0 += pair64(o0.x, o0.y);
    y1 += pair64(o1.x, o1.y);
    if (y0 >= q) y0 -= q;
    if (y1 >= q) y1 -= q;
  }
  __builtin_amdgcn_raw_buffer_store_b64((u32x2){(uint32_t)y0, (uint32_t)(y0 >> 32)}, rs, lane_bytes, 0, kStoreNT);
  __builtin_amdgcn_raw_buffer_store_b64((u32x2){(uint32_t)y1, (uint32_t)(y1 >> 32)}, rs, lane_bytes + poly_bytes, 0,
                                        kStoreNT);
}

__device__ __forceinline__ void fold(Acc &a0, Acc &a1, uint64_t &r0, uint64_t &r1, const LimbConst &lc) {
  r0 = finish(a0, r0, lc);
  r1 = finish(a1, r1, lc);
  acc_zero(a0);
  acc_zero(a1);
}


// Plan records of the main kernel (device pointers into the plan's image).
struct KPlan {
  const LimbConst *limbs;   // [L]
  const uint4 *items;       // per work item: first chunk, chunks, first use, uses
  const uint32_t *dest;     // per work item: output, kSegmentFlag | slot or kBufferFlag | row
  const uint2 *waves;       // per (round, wavefront): first item, item count
  const uint4 *rounds;      // per round: first flush entry, buffered outputs, first split, split outputs
  const uint32_t *flush;    // per buffered output: its output index (buffer row = entry - first)
  const uint4 *splits;      // per split output: output, first segment slot, segments
  const uint2 *pm;          // raw-term chunk blocks
  const uint32_t *words;    // word blocks: common partial sums, resident signed sums, uses
};

// pt_end, out_end: the ends of the plaintext table and of the output array.
// ADD: a later pass over an input range, which adds its sums to the outputs.
template <int NW, bool ADD>
__global__ void __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(4, 4))) hybrid_linear_kernel(
    const uint64_t *__restrict__ in, const uint64_t *__restrict__ pt, uint64_t *__restrict__ out, const KPlan K,
    const KShape S, const void *pt_end, const void *out_end) {
  extern __shared__ uint4 lds[];   // [n_in + n_part + n_mat + segment slots + zero row + output buffer][kTile]
  const LimbConst *__restrict__ limbs = K.limbs;
  const uint4 *__restrict__ items = K.items;
  const uint32_t *__restrict__ dest = K.dest;
  const uint2 *__restrict__ pm = K.pm;
  const uint32_t *__restrict__ words = K.words;
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t lane16 = lane * 16u;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t limb = blockIdx.x / S.tiles;
  const uint32_t tile = blockIdx.x - limb * S.tiles;
  const uint32_t k0 = tile * kTile;
  const uint32_t k = k0 + lane;
  // lanes past N (partial last tile) read a valid coefficient and store nothing
  const uint32_t lane_off = (k < S.N ? k : S.N - 1) - k0;
  const size_t LN = (size_t)S.L * S.N;
  const LimbConst lc = limbs[limb];

  // 1. stage this tile of every input ciphertext (read once)
  for (uint32_t i = wave; i < S.n_in; i += NW) {
    const uint64_t *src = in + ((size_t)i * 2 * S.L + limb) * S.N + k0;
    const uint64_t a = __builtin_nontemporal_load(src + lane_off);
    const uint64_t b = __builtin_nontemporal_load(src + LN + lane_off);
    lds[i * kTile + lane] = make_uint4(lo_digit(a), hi_digit(a), lo_digit(b), hi_digit(b));
  }
  if (wave == NW - 1) lds[S.zero_row * kTile + lane] = make_uint4(0, 0, 0, 0);   // padding row
  __syncthreads();

  // 2. common partial sums, level by level, each kept as a canonical residue
  // in the inputs' digit form so that it enters other sums as one member
  uint4 *parts = lds + (size_t)S.n_in * kTile;
  for (uint32_t lv = 0, p0 = 0; lv < S.n_levels; ++lv) {
    const uint32_t p1 = S.level_end[lv];
    for (uint32_t p = p0 + wave; p < p1; p += NW) {
      const uint32_t *blk = words + (size_t)p * kSumWords;
      const uint4 U = signed_sum(blk, sload1(blk), lds, lane16);
      const uint64_t v0 = reduce_i64((int64_t)(int32_t)U.x + ((int64_t)(int32_t)U.y << 25), lc.q, lc.qinv);
      const uint64_t v1 = reduce_i64((int64_t)(int32_t)U.z + ((int64_t)(int32_t)U.w << 25), lc.q, lc.qinv);
      parts[p * kTile + lane] = make_uint4(lo_digit(v0), hi_digit(v0), lo_digit(v1), hi_digit(v1));
    }
    p0 = p1;
    __syncthreads();
  }

  // 3. shared signed sums, formed once per tile
  uint4 *sums = parts + (size_t)S.n_part * kTile;
  if (S.n_mat) {   // uniform over the workgroup
    for (uint32_t s = wave; s < S.n_mat; s += NW) {
      const uint32_t *blk = words + (size_t)(S.n_part + s) * kSumWords;
      sums[s * kTile + lane] = signed_sum(blk, sload1(blk), lds, lane16);
    }
    __syncthreads();
  }

  // 4. this wavefront's work items of each round; the first records of each
  // item are loaded while the previous item runs
  uint4 *segs = sums + (size_t)S.n_mat * kTile;
  uint4 *obuf = lds + (size_t)S.obuf_row * kTile;
  const char *pt_tile = (const char *)(pt + (size_t)limb * S.N + k0);
  const uint32_t voff = lane_off * 8u;
  const uint32_t out_row = limb * S.N + k0;   // offset of this tile in one output polynomial
  for (uint32_t rd = 0; rd < S.n_rounds; ++rd) {
  const uint2 wr = as_uint2(sload2(K.waves + rd * NW + wave));
  for (uint32_t it = wr.x; it < wr.x + wr.y; ++it) {
    const uint4 item = as_uint4(sload4(items + it));   // first chunk, chunks, first use, uses
    Acc a0, a1;
    acc_zero(a0);
    acc_zero(a1);
    uint64_t r0 = 0, r1 = 0;

    // signed route: each use applies its group's scale once to a signed sum,
    // read from LDS (a resident sum) or formed in place from the use's block
    const uint32_t *ub = words + (size_t)(S.use_block0 + item.z) * kSumWords;
    uint32_t u = 0;
    auto use_one = [&]() {
      if (u && u % kFoldUses == 0) fold(a0, a1, r0, r1, lc);
      const uint32_t *blk = ub + (size_t)u * kSumWords;
      const u32x4 hd = sload4(blk);   // row counts, resident slot or kInlineSum, signed scale
      const uint4 U = hd.y != kInlineSum ? sums[hd.y * kTile + lane] : signed_sum(blk, hd.x, lds, lane16);
      const int32_t c = (int32_t)hd.z;
      smac(a0, c, (int32_t)U.x, (int32_t)U.y);
      smac(a1, c, (int32_t)U.z, (int32_t)U.w);
      ++u;
    };
    // raw route: one PMult per term, chunk by chunk; within a chunk batch b+1
    // is in flight while batch b is multiplied.  The uses are spread over the
    // batches (per of them before each batch is multiplied; the rest after
    // the last chunk): a wavefront then keeps plaintext loads in flight while
    // it forms signed sums.  Measured against all uses after the raw route
    // (in-process A/B, both load orders): VGG11 +4%, BERT +1%, Large +2-3%,
    // ViT within the order spread.  The exact sum allows any order; chunks
    // and uses keep their own fold counts (A0..A3 and s0, s1 bounds).
    const uint32_t per = item.y ? (item.w + item.y * kRawBatches - 1) / (item.y * kRawBatches) : 0;
    auto fill = [&]() {
      for (uint32_t k = 0; k < per && u < item.w; ++k) use_one();
    };
    for (uint32_t c = 0; c < item.y; ++c) {
      if (c) {
        if (c % kFoldChunks == 0) fold(a0, a1, r0, r1, lc);   // keep the accumulators exact
        else { carry(a0); carry(a1); }
      }
      raw_chunk(sload_block(pm, item.x + c), pt_tile, pt_end, voff, a0, a1, lds, lane16, fill);
    }
    while (u < item.w) use_one();

    const uint64_t y0 = finish(a0, r0, lc);
    const uint64_t y1 = finish(a1, r1, lc);
    const uint32_t d = sload1(dest + it);
    if (d & kSegmentFlag) {
      segs[(d & ~kSegmentFlag) * kTile + lane] =
          make_uint4((uint32_t)y0, (uint32_t)(y0 >> 32), (uint32_t)y1, (uint32_t)(y1 >> 32));
    } else if (d & kBufferFlag) {
      obuf[(d & ~kBufferFlag) * kTile + lane] =
          make_uint4((uint32_t)y0, (uint32_t)(y0 >> 32), (uint32_t)y1, (uint32_t)(y1 >> 32));
    } else if (k < S.N) {
      store_out<ADD>(out + (size_t)d * 2 * LN + out_row, out_end, lane * 8u, (uint32_t)(LN * 8), y0, y1, lc.q);
    }
  }

  // 5. end of the round: outputs that were split across wavefronts add their
  // segments' residues, and the buffered outputs leave LDS in one burst
  const uint4 rr = K.rounds[rd];   // first flush entry, buffered outputs, first split, split outputs
  if (rr.y | rr.w) {               // uniform over the workgroup
    __syncthreads();
    for (uint32_t s = wave; s < rr.w; s += NW) {
      const uint4 sp = K.splits[rr.z + s];
      uint64_t y0 = 0, y1 = 0;   // at most 64 residues < 2^50: below 2^56
      for (uint32_t g = 0; g < sp.z; ++g) {
        const uint4 v = segs[(sp.y + g) * kTile + lane];
        y0 += pair64(v.x, v.y);
        y1 += pair64(v.z, v.w);
      }
      y0 = reduce_i64((int64_t)y0, lc.q, lc.qinv);
      y1 = reduce_i64((int64_t)y1, lc.q, lc.qinv);
      if (k < S.N) store_out<ADD>(out + (size_t)sp.x * 2 * LN + out_row, out_end, lane * 8u, (uint32_t)(LN * 8), y0, y1, lc.q);
    }
    for (uint32_t e = wave; e < rr.y; e += NW) {
      const uint4 v = obuf[e * kTile + lane];
      const uint32_t j = K.flush[rr.x + e];
      if (k < S.N)
        store_out<ADD>(out + (size_t)j * 2 * LN + out_row, out_end, lane * 8u, (uint32_t)(LN * 8), pair64(v.x, v.y),
                       pair64(v.z, v.w), lc.q);
    }
    if (rd + 1 < S.n_rounds) __syncthreads();   // the next round refills the buffer
  }
  }   // rounds
}

}  // namespace fiona
