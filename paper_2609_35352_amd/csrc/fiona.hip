// Host side of the C ABI in include/fiona.h: parameter checks, the plan
// compiler (grouping, sharing, LDS residency) and the kernel launch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <unordered_map>
#include <vector>

#include "fiona.h"
#include "fiona_ctx.hpp"
#include "hybrid_kernel.hpp"

using fiona::KShape;
using fiona::PackParams;
using fiona::LimbConst;

namespace {

constexpr uint32_t kLdsBytes = 160u * 1024u;    // gfx950 LDS per workgroup (and per CU)
constexpr uint32_t kSlotBytes = fiona::kTile * 16u;   // one input or sum tile in LDS
constexpr uint32_t kMaxInputs = kLdsBytes / kSlotBytes;   // LDS rows of one workgroup
static_assert(FIONA_MAX_INPUTS + 1 == kMaxInputs, "inputs plus the zero row fill the LDS");
constexpr uint32_t kMaxSegments = 64;           // segments of one split output
constexpr uint32_t kMinBurstRows = 8;           // free LDS rows needed for output bursts
constexpr double kMinBurstShare = 0.025;        // output share of a launch's HBM bytes for bursts
// Relative costs used to balance work items over wavefronts (units: one raw term).
constexpr double kCostUseResident = 0.6;
constexpr double kCostUseInline = 0.5;
constexpr double kCostMember = 0.25;
constexpr double kCostFinish = 6.0;
constexpr double kCostChunk = 3.0;
constexpr double kMinSegmentCost = 128.0;
// LDS residency and common partial sums must save at least this share of a
// tile's estimated work, else the plan keeps neither (each costs LDS rows, a
// barrier and a pass over its sums per tile).
constexpr double kMinShareGain = 0.02;

LimbConst make_limb_const(uint64_t q) {
  LimbConst c;
  c.q = q;
  c.r32 = (uint64_t)((((unsigned __int128)1) << 32) % q);
  c.r32_shoup = (uint64_t)((((unsigned __int128)c.r32) << 64) / q);
  c.r57 = (uint64_t)((((unsigned __int128)1) << 57) % q);
  c.r57_shoup = (uint64_t)((((unsigned __int128)c.r57) << 64) / q);
  c.qinv = 1.0 / (double)q;
  return c;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool ranges_overlap(const void *a, size_t na, const void *b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + nb && b0 < a0 + na;
}

}  // namespace

struct fiona_plan {
  const fiona_ctx *ctx = nullptr;
  uint32_t n_in = 0, n_out = 0, n_pt = 0, n_scale = 0, n_member_desc = 0;
  uint64_t pt_pitch = 0;   // words from one plaintext to the next
  uint32_t n_mat = 0;
  uint32_t n_part = 0, n_levels = 0;   // common partial sums and their levels
  std::vector<uint32_t> part_levels;
  uint32_t flags = 0;
  fiona_plan_stats_t st{};
  std::vector<uint4> items;
  std::vector<uint32_t> dest;
  std::vector<uint2> waves;    // [n_rounds][nw]
  std::vector<uint4> splits;
  std::vector<uint4> rounds;   // per round: first flush entry, buffered outputs, first split, split outputs
  std::vector<uint32_t> flush; // output index of each buffered output, round by round
  uint32_t n_rounds = 1, obuf_rows = 0;
  uint32_t nw = 8, n_seg_slots = 0;
  std::vector<uint2> pm;
  uint32_t n_uses = 0;
  std::vector<uint2> members;
  std::vector<uint4> blocks;   // word blocks: common partial sums, resident sums, uses (see PackParams)
  std::vector<int8_t> signs;   // a checking plan: the layer description's mem_sign
  bool any_raw = false;
  // A layer with more inputs than the LDS of one tile holds runs in passes
  // over ranges of its inputs: the plan then keeps one plan per pass (the
  // first stores the outputs, the later ones add to them) and no image of
  // its own.  A pass reads inputs in_base .. in_base + n_in - 1.
  std::vector<fiona_plan *> passes;
  uint32_t in_base = 0;
  bool accumulate = false;   // a pass after the first: adds to the outputs
  void *dev = nullptr;
  int device = -1;
  // device pointers into dev
  const LimbConst *d_limbs = nullptr;
  const uint4 *d_items = nullptr, *d_splits = nullptr, *d_rounds = nullptr, *d_blocks = nullptr;
  const uint32_t *d_dest = nullptr, *d_flush = nullptr;
  const uint2 *d_waves = nullptr, *d_pm = nullptr, *d_members = nullptr;
  uint32_t *d_words = nullptr;
  KShape shape{};
  uint32_t lds_bytes = 0, grid = 0, tiles = 0;
  bool any_signed = false;
};

extern "C" {

const char *fiona_status_string(int status) {
  switch (status) {
    case FIONA_OK: return "ok";
    case FIONA_ERR_ARG: return "invalid argument";
    case FIONA_ERR_PLAN: return "inconsistent layer description";
    case FIONA_ERR_UNSUPPORTED: return "unsupported size or modulus";
    case FIONA_ERR_ALIGN: return "device pointer not aligned";
    case FIONA_ERR_ALIAS: return "output overlaps an input";
    case FIONA_ERR_HIP: return "HIP runtime error";
    case FIONA_ERR_NOMEM: return "out of host memory";
    case FIONA_ERR_NODEVICE: return "plan has no device image";
    case FIONA_ERR_PRECONDITION: return "an input breaks a precondition";
    case FIONA_ERR_BOUNDS: return "a replayed access falls outside its buffer";
    default: return "unknown status";
  }
}

int fiona_ctx_create(uint32_t N, uint32_t L, const uint64_t *moduli, fiona_ctx **out) {
  if (!out) return FIONA_ERR_ARG;
  *out = nullptr;
  if (!moduli) return FIONA_ERR_ARG;
  if (N == 0 || N > FIONA_MAX_N || L == 0 || L > FIONA_MAX_L) return FIONA_ERR_UNSUPPORTED;
  for (uint32_t l = 0; l < L; ++l)
    if (moduli[l] <= (1ull << FIONA_SCALE_BITS) || moduli[l] >= (1ull << FIONA_MODULUS_BITS))
      return FIONA_ERR_UNSUPPORTED;
  fiona_ctx *c = new (std::nothrow) fiona_ctx;
  if (!c) return FIONA_ERR_NOMEM;
  try {
    c->N = N;
    c->L = L;
    c->q.assign(moduli, moduli + L);
    for (uint32_t l = 0; l < L; ++l) c->limbs.push_back(make_limb_const(moduli[l]));
  } catch (...) {
    delete c;
    return FIONA_ERR_NOMEM;
  }
  *out = c;
  return FIONA_OK;
}

void fiona_ctx_destroy(fiona_ctx *ctx) { delete ctx; }

uint64_t fiona_pt_pitch_hint(const fiona_ctx *ctx) {
  if (!ctx) return 0;
  const uint64_t ln = (uint64_t)ctx->L * ctx->N;
  return (ln + 63) / 64 * 64 + 128;
}

}  // extern "C"

namespace {

// Checks every index of the description (no partial trust).
int validate_desc(const fiona_layer_desc *d) {
  if (!d->pm_off || !d->grp_off) return FIONA_ERR_ARG;
  if (d->n_in == 0) return FIONA_ERR_ARG;
  if (d->n_out >= (1u << 30) || d->n_pt >= (1u << 31) || d->n_scale >= (1u << 31)) return FIONA_ERR_PLAN;
  if (d->pm_off[0] != 0 || d->grp_off[0] != 0) return FIONA_ERR_PLAN;
  for (uint32_t j = 0; j < d->n_out; ++j)
    if (d->pm_off[j + 1] < d->pm_off[j] || d->grp_off[j + 1] < d->grp_off[j]) return FIONA_ERR_PLAN;
  const uint32_t n_pm = d->pm_off[d->n_out];
  const uint32_t n_group = d->grp_off[d->n_out];
  if (n_pm && (!d->pm_input || !d->pm_pt)) return FIONA_ERR_ARG;
  for (uint32_t t = 0; t < n_pm; ++t)
    if (d->pm_input[t] >= d->n_in || d->pm_pt[t] >= d->n_pt) return FIONA_ERR_PLAN;
  if (n_group) {
    if (!d->grp_mem_off || !d->grp_scale) return FIONA_ERR_ARG;
    if (d->grp_mem_off[0] != 0) return FIONA_ERR_PLAN;
    for (uint32_t g = 0; g < n_group; ++g) {
      if (d->grp_mem_off[g + 1] < d->grp_mem_off[g]) return FIONA_ERR_PLAN;
      if (d->grp_scale[g] >= d->n_scale) return FIONA_ERR_PLAN;
    }
    const uint32_t n_member = d->grp_mem_off[n_group];
    if (n_member >= (1u << 31)) return FIONA_ERR_PLAN;
    if (n_member && (!d->mem_input || !d->mem_sign)) return FIONA_ERR_ARG;
    for (uint32_t m = 0; m < n_member; ++m) {
      if (d->mem_input[m] >= d->n_in) return FIONA_ERR_PLAN;
      if (d->mem_sign[m] < -1 || d->mem_sign[m] > 1) return FIONA_ERR_PLAN;
    }
  }
  return FIONA_OK;
}

// A member of a signed sum or of a common partial sum: an LDS row (an input,
// or a common partial sum at row n_in + p), the index of the sign that this
// member's run-time sign is read from, and its sign when the plan was made.
struct MemberRef {
  uint32_t row, slot;
  int32_t sign;
};

struct SumBuild {
  std::vector<MemberRef> members;   // of the representative group, sorted by row
  bool flip = false;                // representative's canonicalisation flipped its signs
  uint32_t n_use = 0;
  uint32_t slot = fiona::kInlineSum;
  uint32_t member_begin = 0;        // its members in the device member list
};

// A common partial sum: first + rel * second (rows as in MemberRef).  Its two
// members' slots are those of the first sum it was found in; at run time its
// value is normalised by the first member's sign.
struct PartialBuild {
  MemberRef first, second;
  uint32_t level = 1;
};

constexpr uint32_t kMaxPartialLevels = fiona::kMaxLevels;   // barriers between levels of common terms per tile
// A common term costs its reduction to a residue and an LDS row once per tile
// (about as much work as a dozen member additions) before it saves anything.
constexpr uint64_t kMinPartialReuse = 16;

// Sec. 4.2 candidate search, greedy: repeatedly take the signed pair that
// the most sum evaluations contain, if the paper's estimate k*m - m - k of the
// Add/Sub it saves (m = 2 members, k = evaluations containing it) is positive,
// k reaches kMinPartialReuse and an LDS row is left.  A pair may combine
// earlier common terms (the level counts how deep); each sum then holds the
// common term once in place of the two members (so overlapping candidates
// never both apply to one sum).
void find_partial_sums(std::vector<SumBuild> &sums, const std::vector<uint64_t> &weight, uint32_t n_in,
                       uint32_t max_rows, std::vector<PartialBuild> &parts) {
  std::vector<uint32_t> level_of;   // per partial
  auto level = [&](uint32_t row) { return row < n_in ? 0u : level_of[row - n_in]; };
  std::unordered_map<uint64_t, uint64_t> count;
  std::vector<uint64_t> keys;
  while (parts.size() < max_rows) {
    count.clear();
    for (size_t s = 0; s < sums.size(); ++s) {
      // members are sorted by row; a group may name one input twice, and a
      // pair of one input with itself is no common term.  Each candidate
      // counts once per sum, as at most one copy of it is replaced there.
      const auto &m = sums[s].members;
      keys.clear();
      for (size_t i = 0; i < m.size(); ++i)
        for (size_t j = i + 1; j < m.size(); ++j) {
          if (m[i].row == m[j].row) continue;
          if (std::max(level(m[i].row), level(m[j].row)) + 1 > kMaxPartialLevels) continue;
          keys.push_back(((uint64_t)m[i].row << 33) | ((uint64_t)m[j].row << 1) | (m[i].sign != m[j].sign));
        }
      std::sort(keys.begin(), keys.end());
      keys.erase(std::unique(keys.begin(), keys.end()), keys.end());
      for (uint64_t key : keys) count[key] += weight[s];
    }
    uint64_t best = 0, best_k = 0;
    for (const auto &kv : count)
      if (kv.second > best_k || (kv.second == best_k && kv.first < best)) {
        best = kv.first;
        best_k = kv.second;
      }
    const uint64_t m = 2, k = best_k;
    if (k * m <= m + k || k < kMinPartialReuse) break;
    const uint32_t ra = (uint32_t)(best >> 33), rb = (uint32_t)((best >> 1) & 0xFFFFFFFFu);
    const int32_t rel = (best & 1) ? -1 : 1;
    const uint32_t row = n_in + (uint32_t)parts.size();
    bool first_use = true;
    PartialBuild pb;
    for (auto &sb : sums) {
      auto &mm = sb.members;
      // two distinct members (ra != rb) with this relative sign; with a
      // repeated input, any copy that fits
      size_t ia = mm.size(), ib = mm.size();
      for (size_t t = 0; t < mm.size() && ib == mm.size(); ++t) {
        if (mm[t].row != ra) continue;
        for (size_t v = 0; v < mm.size(); ++v)
          if (mm[v].row == rb && mm[t].sign * mm[v].sign == rel) {
            ia = t;
            ib = v;
            break;
          }
      }
      if (ib == mm.size()) continue;
      if (first_use) {
        pb.first = MemberRef{ra, mm[ia].slot, 1};
        pb.second = MemberRef{rb, mm[ib].slot, rel};
        first_use = false;
      }
      const MemberRef joined{row, mm[ia].slot, mm[ia].sign};
      mm.erase(mm.begin() + std::max(ia, ib));
      mm.erase(mm.begin() + std::min(ia, ib));
      mm.push_back(joined);   // rows of common terms are above every input row
    }
    pb.level = std::max(level(ra), level(rb)) + 1;
    level_of.push_back(pb.level);
    parts.push_back(pb);
  }
}

int compile_plan(fiona_plan *P, const fiona_layer_desc *d) {
  // Per-contribution compilation applies every signed term's factor on its
  // own: each nonzero member is a sum of one member, nothing is shared.
  const bool per_contribution = (d->flags & FIONA_PLAN_PER_CONTRIBUTION) != 0;
  const bool share = !(d->flags & FIONA_PLAN_NO_SHARING) && !per_contribution;
  const bool partial = share && !(d->flags & FIONA_PLAN_NO_PARTIAL_SHARING);
  const size_t part_members = per_contribution ? 1 : fiona::kMaxMembers;
  const uint32_t n_pm = d->pm_off[d->n_out];
  const uint32_t n_group = d->grp_off[d->n_out];
  P->n_member_desc = n_group ? d->grp_mem_off[n_group] : 0;

  std::vector<SumBuild> sums;
  std::map<std::vector<uint64_t>, uint32_t> index;   // canonical signed sum -> sum id
  struct Use { uint32_t sum, scale; bool neg; };
  std::vector<std::vector<Use>> out_uses(d->n_out);

  uint64_t nz_members = 0, addsub_unshared = 0;
  for (uint32_t j = 0; j < d->n_out; ++j) {
    for (uint32_t g = d->grp_off[j]; g < d->grp_off[j + 1]; ++g) {
      // nonzero members of the group, split into sub-sums of at most kMaxMembers
      std::vector<std::pair<uint64_t, uint32_t>> nz;   // (input*2 + negative, member index)
      for (uint32_t m = d->grp_mem_off[g]; m < d->grp_mem_off[g + 1]; ++m) {
        if (d->mem_sign[m] == 0) continue;
        nz.push_back({(uint64_t)d->mem_input[m] * 2 + (d->mem_sign[m] < 0 ? 1 : 0), m});
      }
      nz_members += nz.size();
      for (size_t c0 = 0; c0 < nz.size(); c0 += part_members) {
        const size_t c1 = std::min(nz.size(), c0 + part_members);
        std::vector<std::pair<uint64_t, uint32_t>> part(nz.begin() + c0, nz.begin() + c1);
        std::sort(part.begin(), part.end());
        const bool flip = (part[0].first & 1) != 0;   // canonical form: first member positive
        std::vector<uint64_t> key(part.size());
        for (size_t t = 0; t < part.size(); ++t) key[t] = part[t].first ^ (flip ? 1 : 0);
        addsub_unshared += part.size() - 1;
        uint32_t sid;
        auto it = share ? index.find(key) : index.end();
        if (it == index.end()) {
          sid = (uint32_t)sums.size();
          SumBuild sb;
          sb.flip = flip;
          for (auto &pr : part)
            sb.members.push_back(MemberRef{(uint32_t)(pr.first >> 1), pr.second, (pr.first & 1) ? -1 : 1});
          sums.push_back(std::move(sb));
          if (share) index.emplace(std::move(key), sid);
        } else {
          sid = it->second;
        }
        sums[sid].n_use++;
        out_uses[j].push_back(Use{sid, d->grp_scale[g], flip != sums[sid].flip});
      }
    }
  }
  uint64_t addsub_shared = 0;
  for (const auto &sb : sums) addsub_shared += sb.members.size() - 1;

  // Candidates for LDS residency: sums used more than once, most used first.
  const bool lds_sums = !(d->flags & FIONA_PLAN_NO_LDS_SUMS);
  std::vector<uint32_t> cand;
  for (uint32_t s = 0; s < sums.size(); ++s)
    if (lds_sums && sums[s].n_use >= 2) cand.push_back(s);
  std::stable_sort(cand.begin(), cand.end(),
                   [&](uint32_t a, uint32_t b) { return sums[a].n_use > sums[b].n_use; });
  const uint32_t lds_free = kMaxInputs - d->n_in - 1;   // slots left after the inputs and the zero row
  if (cand.size() > lds_free) cand.resize(lds_free);
  // estimated work of a tile without residency or common terms (cost units of
  // the work-item balance below), and what residency would save
  double tile_work = (double)n_pm;
  for (const auto &sb : sums)
    tile_work += sb.n_use * (kCostUseInline + kCostMember * (double)sb.members.size());
  double res_gain = 0;
  for (uint32_t s : cand) res_gain += (sums[s].n_use - 1) * kCostMember * (double)sums[s].members.size();
  std::vector<char> resident(sums.size(), 0);
  for (uint32_t s : cand) resident[s] = 1;

  // Common partial sums in the LDS rows that residency leaves free.  A sum is
  // evaluated once per tile if resident, else once per use.
  // An image of at most half the LDS lets two workgroups share a CU; common
  // terms do not push an image that fits past that line.
  std::vector<PartialBuild> parts;
  std::vector<std::vector<MemberRef>> members_before;   // restored if the sharing is not kept
  for (const auto &sb : sums) members_before.push_back(sb.members);
  double part_gain = 0;
  if (partial && lds_free > cand.size()) {
    std::vector<uint64_t> weight(sums.size());
    for (uint32_t s = 0; s < sums.size(); ++s) weight[s] = resident[s] ? 1 : sums[s].n_use;
    const uint32_t base_rows = d->n_in + 1 + (uint32_t)cand.size();
    const uint32_t cap = base_rows * 2 <= kMaxInputs ? kMaxInputs / 2 : kMaxInputs;
    if (cap > base_rows) find_partial_sums(sums, weight, d->n_in, cap - base_rows, parts);
    double saved = -2.0 * (double)parts.size();   // each common pair is formed once per tile
    for (uint32_t s = 0; s < sums.size(); ++s)
      saved += (double)weight[s] * ((double)members_before[s].size() - (double)sums[s].members.size());
    part_gain = kCostMember * saved;
  }
  if (res_gain + part_gain < kMinShareGain * tile_work) {
    // not worth its LDS rows and barriers: every signed sum is formed in place
    for (uint32_t s = 0; s < sums.size(); ++s) sums[s].members = members_before[s];
    parts.clear();
    for (uint32_t s : cand) resident[s] = 0;
    cand.clear();
  }
  const uint32_t n_part = (uint32_t)parts.size();
  uint64_t addsub_partial = n_part;   // one Add/Sub forms each common pair
  for (const auto &sb : sums) addsub_partial += sb.members.size() - 1;
  const uint32_t rows_free = lds_free - n_part;   // for resident sums and segments

  // One workgroup per CU when the LDS image exceeds half the CU: then 16 wavefronts.
  const uint32_t est_slots = d->n_in + n_part + std::min<uint32_t>((uint32_t)cand.size(), rows_free);
  P->nw = est_slots * 2 > kMaxInputs ? 16 : 8;
  // Output bursts: one workgroup per CU (16 wavefronts) that keeps finished
  // outputs in the LDS rows its image leaves free and writes them together at
  // the end of a round.  Output stores spread among the plaintext reads cost
  // far more HBM time than the same bytes written in bursts.
  // They pay when outputs are a fair share of the launch's bytes; else one
  // workgroup per CU and the barriers that end the rounds cost more.
  const double out_share = 2.0 * d->n_out / (2.0 * d->n_in + (double)n_pm + 2.0 * d->n_out);
  bool bursts = !(d->flags & FIONA_PLAN_NO_OUTPUT_BURSTS) && d->n_out > 0 && out_share >= kMinBurstShare &&
                est_slots + 1 + kMinBurstRows <= kMaxInputs;
  if (bursts) P->nw = 16;

  // Work items: whole outputs, or segments of outputs that are long compared
  // with the share of one wavefront.
  auto use_cost = [&](const Use &u) {
    return resident[u.sum] ? kCostUseResident
                           : kCostUseInline + kCostMember * (double)sums[u.sum].members.size();
  };
  std::vector<double> out_cost(d->n_out);
  double total = 0;
  for (uint32_t j = 0; j < d->n_out; ++j) {
    double c = kCostFinish + (double)(d->pm_off[j + 1] - d->pm_off[j]);
    for (const Use &u : out_uses[j]) c += use_cost(u);
    out_cost[j] = c;
    total += c;
  }
  const double target = total / P->nw;
  std::vector<uint32_t> nseg(d->n_out, 1);
  uint32_t seg_slots = 0;
  for (uint32_t j = 0; j < d->n_out; ++j) {
    if (out_cost[j] <= 1.25 * target) continue;
    uint32_t S = (uint32_t)(out_cost[j] / target + 0.5);
    S = std::min<uint32_t>(S, (uint32_t)(out_cost[j] / kMinSegmentCost));
    S = std::min<uint32_t>(S, kMaxSegments);
    if (S >= 2 && seg_slots + S <= rows_free) {
      nseg[j] = S;
      seg_slots += S;
    }
  }
  P->n_seg_slots = seg_slots;
  if (cand.size() > rows_free - seg_slots) {   // segments take precedence over the least used residents
    for (size_t c = rows_free - seg_slots; c < cand.size(); ++c) resident[cand[c]] = 0;
    cand.resize(rows_free - seg_slots);
  }
  // Rounds of outputs: consecutive outputs, as many whole (unsplit) outputs per
  // round as the free LDS rows hold.
  std::vector<uint32_t> round_of(d->n_out, 0);
  {
    const uint32_t image = d->n_in + n_part + (uint32_t)cand.size() + seg_slots + 1;
    const uint32_t avail = kMaxInputs > image ? kMaxInputs - image : 0;
    uint32_t n_whole = 0;
    for (uint32_t j = 0; j < d->n_out; ++j) n_whole += nseg[j] == 1;
    if (avail < kMinBurstRows || n_whole == 0) bursts = false;
    P->n_rounds = 1;
    if (bursts) {
      uint32_t n_rounds = (n_whole + avail - 1) / avail;
      for (;; ++n_rounds) {   // outputs in order, evenly over the rounds
        std::vector<uint32_t> cnt(n_rounds, 0);
        uint32_t most = 0;
        for (uint32_t j = 0; j < d->n_out; ++j) {
          round_of[j] = (uint32_t)((uint64_t)j * n_rounds / d->n_out);
          if (nseg[j] == 1) most = std::max(most, ++cnt[round_of[j]]);
        }
        if (most <= avail) {
          P->obuf_rows = most;
          break;
        }
      }
      P->n_rounds = n_rounds;
    }
  }

  // Device records.  Word blocks: one per common partial sum, one per resident
  // signed sum, then one per use; the sign-packing kernel fills them on every
  // call.  Block = {member begin, count | flags, resident slot, scale | negate}.
  for (uint32_t p = 0; p < n_part; ++p) {
    const uint32_t mb = (uint32_t)P->members.size();
    P->members.push_back(make_uint2(parts[p].first.row, parts[p].first.slot));
    P->members.push_back(make_uint2(parts[p].second.row, parts[p].second.slot));
    P->blocks.push_back(make_uint4(mb, 2u | fiona::kNormaliseSigns, fiona::kInlineSum, 0));
  }
  for (auto &sb : sums) {
    sb.member_begin = (uint32_t)P->members.size();
    for (auto &m : sb.members) P->members.push_back(make_uint2(m.row, m.slot));
  }
  // Rows of common terms are numbered level by level (a term only reads rows
  // of lower levels), so each level is formed after a barrier; part_levels[l]
  // is the end of the rows of level l+1.
  P->n_part = n_part;
  uint32_t n_levels = 0;
  {
    std::vector<uint32_t> order(n_part);
    for (uint32_t p = 0; p < n_part; ++p) order[p] = p;
    std::stable_sort(order.begin(), order.end(),
                     [&](uint32_t a, uint32_t b) { return parts[a].level < parts[b].level; });
    std::vector<uint32_t> new_row(n_part);
    for (uint32_t t = 0; t < n_part; ++t) new_row[order[t]] = t;
    for (auto &m : P->members)
      if (m.x >= d->n_in) m.x = d->n_in + new_row[m.x - d->n_in];
    const std::vector<uint4> blocks(P->blocks.begin(), P->blocks.begin() + n_part);
    for (uint32_t p = 0; p < n_part; ++p) P->blocks[new_row[p]] = blocks[p];
    P->part_levels.assign(kMaxPartialLevels, 0);
    for (uint32_t t = 0; t < n_part; ++t) {
      const uint32_t lv = parts[order[t]].level;
      n_levels = std::max(n_levels, lv);
      for (uint32_t l = lv - 1; l < kMaxPartialLevels; ++l) P->part_levels[l] = t + 1;
    }
  }
  P->n_levels = n_levels;
  for (uint32_t s : cand) {
    sums[s].slot = P->n_mat++;
    P->blocks.push_back(make_uint4(sums[s].member_begin, (uint32_t)sums[s].members.size(), fiona::kInlineSum, 0));
  }
  std::vector<uint32_t> use_begin(d->n_out);
  for (uint32_t j = 0; j < d->n_out; ++j) {
    use_begin[j] = P->n_uses;
    for (const Use &u : out_uses[j]) {
      const SumBuild &sb = sums[u.sum];
      const uint32_t sc = u.scale | (u.neg ? 0x80000000u : 0u);
      if (sb.slot != fiona::kInlineSum)   // a resident sum: no members, its LDS slot
        P->blocks.push_back(make_uint4(0, fiona::kUseBlock, sb.slot, sc));
      else
        P->blocks.push_back(make_uint4(sb.member_begin, (uint32_t)sb.members.size() | fiona::kUseBlock,
                                       fiona::kInlineSum, sc));
      P->n_uses++;
    }
  }
  P->st.addsub_partial = addsub_partial;
  P->st.n_partial = n_part;
  P->st.partial_levels = n_levels;

  // Raw-term records, per work item, in chunks of at most kChunkTerms terms
  // (one block of kChunkSlots records each, see hybrid_kernel.hpp).  The
  // terms of an output may be taken in any order (the sum is exact), so they
  // are sorted by plaintext offset: a chunk then covers a short stretch of the
  // plaintext table, and its terms' offsets from the chunk base fit 31 bits.
  const uint32_t zero_row = d->n_in + n_part + P->n_mat + seg_slots;
  const uint64_t ln8 = P->pt_pitch * 8;
  auto emit_chunks = [&](const std::vector<std::pair<uint64_t, uint32_t>> &terms, size_t t0, size_t t1) {
    const uint32_t first = (uint32_t)(P->pm.size() / fiona::kChunkSlots);
    size_t t = t0;
    while (t < t1) {
      const uint64_t cbase = terms[t].first;
      size_t e = t;
      while (e < t1 && e - t < fiona::kChunkTerms && terms[e].first - cbase < (1ull << 31)) ++e;
      const uint32_t n = (uint32_t)(e - t), nb = (n + fiona::kRawBatch - 1) / fiona::kRawBatch;
      // block: kChunkSlots plaintext offsets, then kChunkSlots input rows (as
      // kChunkSlots uint2 words); slot kChunkSlots-1 of each half is the header
      const size_t blk = P->pm.size();
      P->pm.resize(blk + fiona::kChunkSlots, make_uint2(0, 0));
      uint32_t *w = (uint32_t *)&P->pm[blk];
      for (uint32_t r = 0; r < nb * fiona::kRawBatch; ++r) {
        w[r] = r < n ? (uint32_t)(terms[t + r].first - cbase) : 0u;
        w[fiona::kChunkSlots + r] = (r < n ? terms[t + r].second : zero_row) * kSlotBytes;
      }
      w[fiona::kChunkSlots - 1] = (uint32_t)cbase;
      w[2 * fiona::kChunkSlots - 1] = (uint32_t)(cbase >> 32) | (nb << 16);
      t = e;
    }
    return make_uint2(first, (uint32_t)(P->pm.size() / fiona::kChunkSlots) - first);
  };

  // items, each with its cost; segments of a split output get consecutive LDS
  // slots; buffered outputs get the next row of their round's output buffer
  struct Item { uint4 rec; uint32_t dest; double cost; uint32_t round; };
  std::vector<Item> items;
  uint32_t slot = 0;
  P->rounds.assign(P->n_rounds, make_uint4(0, 0, 0, 0));
  for (uint32_t j = 0, r = 0; j < d->n_out; ++j) {   // first entries of each round
    for (; r < round_of[j]; ++r) {
      P->rounds[r + 1].x = P->rounds[r].x + P->rounds[r].y;
      P->rounds[r + 1].z = P->rounds[r].z + P->rounds[r].w;
    }
    if (nseg[j] > 1) P->rounds[r].w++;
    else if (bursts) P->rounds[r].y++;
  }
  for (uint32_t r = 1; r < P->n_rounds; ++r) {   // rounds after the last output's
    if (P->rounds[r].x < P->rounds[r - 1].x + P->rounds[r - 1].y) {
      P->rounds[r].x = P->rounds[r - 1].x + P->rounds[r - 1].y;
      P->rounds[r].z = P->rounds[r - 1].z + P->rounds[r - 1].w;
    }
  }
  P->flush.assign(P->rounds.empty() ? 0 : P->rounds.back().x + P->rounds.back().y, 0);
  std::vector<uint32_t> buf_row(P->n_rounds, 0);
  std::vector<std::pair<uint64_t, uint32_t>> terms;   // (plaintext byte offset, input)
  for (uint32_t j = 0; j < d->n_out; ++j) {
    const uint32_t pb = d->pm_off[j], pc = d->pm_off[j + 1] - pb;
    terms.clear();
    for (uint32_t t = pb; t < pb + pc; ++t) terms.push_back({(uint64_t)d->pm_pt[t] * ln8, d->pm_input[t]});
    std::stable_sort(terms.begin(), terms.end(),
                     [](const std::pair<uint64_t, uint32_t> &a, const std::pair<uint64_t, uint32_t> &b) {
                       return a.first < b.first;
                     });
    const uint32_t ub = use_begin[j], uc = (uint32_t)out_uses[j].size();
    const uint32_t S = nseg[j];
    if (S > 1) P->splits.push_back(make_uint4(j, slot, S, 0));
    for (uint32_t g = 0; g < S; ++g) {
      const uint32_t r0 = (uint32_t)((uint64_t)pc * g / S), r1 = (uint32_t)((uint64_t)pc * (g + 1) / S);
      const uint32_t u0 = (uint32_t)((uint64_t)uc * g / S), u1 = (uint32_t)((uint64_t)uc * (g + 1) / S);
      const uint2 ch = emit_chunks(terms, r0, r1);
      double c = kCostFinish + (double)(r1 - r0) + kCostChunk * ch.y;
      for (uint32_t u = u0; u < u1; ++u) c += use_cost(out_uses[j][u]);
      uint32_t dst = j;
      if (S > 1) {
        dst = fiona::kSegmentFlag | (slot + g);
      } else if (bursts) {
        const uint32_t r = round_of[j], row = buf_row[r]++;
        P->flush[P->rounds[r].x + row] = j;
        dst = fiona::kBufferFlag | row;
      }
      items.push_back(Item{make_uint4(ch.x, ch.y, ub + u0, u1 - u0), dst, c, round_of[j]});
    }
    if (S > 1) slot += S;
  }
  // per round: longest item first onto the least loaded wavefront
  for (uint32_t r = 0; r < P->n_rounds; ++r) {
    std::vector<uint32_t> order;
    for (uint32_t t = 0; t < items.size(); ++t)
      if (items[t].round == r) order.push_back(t);
    std::stable_sort(order.begin(), order.end(),
                     [&](uint32_t a, uint32_t b) { return items[a].cost > items[b].cost; });
    std::vector<double> load(P->nw, 0.0);
    std::vector<std::vector<uint32_t>> per_wave(P->nw);
    for (uint32_t t : order) {
      const uint32_t w = (uint32_t)(std::min_element(load.begin(), load.end()) - load.begin());
      load[w] += items[t].cost;
      per_wave[w].push_back(t);
    }
    for (uint32_t w = 0; w < P->nw; ++w) {
      std::sort(per_wave[w].begin(), per_wave[w].end());
      P->waves.push_back(make_uint2((uint32_t)P->items.size(), (uint32_t)per_wave[w].size()));
      for (uint32_t t : per_wave[w]) {
        P->items.push_back(items[t].rec);
        P->dest.push_back(items[t].dest);
      }
    }
  }

  fiona_plan_stats_t &st = P->st;
  st.n_pmult = n_pm;
  st.n_member = P->n_member_desc;
  st.ct_terms = (uint64_t)n_pm + P->n_member_desc;
  st.n_member_nonzero = nz_members;
  st.n_use = P->n_uses;
  st.n_sum_distinct = sums.size();
  st.n_sum_resident = P->n_mat;
  st.pmult_per_contribution = (uint64_t)n_pm + nz_members;
  st.pmult_grouped = (uint64_t)n_pm + P->n_uses;
  st.addsub_unshared = addsub_unshared;
  st.addsub_shared = addsub_shared;
  P->any_signed = P->n_uses > 0;
  P->any_raw = n_pm > 0;
  return FIONA_OK;
}

int upload_plan(fiona_plan *P) {
  const fiona_ctx *C = P->ctx;
  const size_t a = 256;
  const size_t o_limbs = 0;
  const size_t o_items = align_up(o_limbs + sizeof(LimbConst) * C->L, a);
  const size_t o_dest = align_up(o_items + sizeof(uint4) * P->items.size(), a);
  const size_t o_waves = align_up(o_dest + sizeof(uint32_t) * P->dest.size(), a);
  const size_t o_splits = align_up(o_waves + sizeof(uint2) * P->waves.size(), a);
  const size_t o_rounds = align_up(o_splits + sizeof(uint4) * P->splits.size(), a);
  const size_t o_flush = align_up(o_rounds + sizeof(uint4) * P->rounds.size(), a);
  const size_t o_pm = align_up(o_flush + sizeof(uint32_t) * P->flush.size(), a);
  const size_t o_mem = align_up(o_pm + sizeof(uint2) * P->pm.size(), a);
  const size_t o_blocks = align_up(o_mem + sizeof(uint2) * P->members.size(), a);
  const size_t o_words = align_up(o_blocks + sizeof(uint4) * P->blocks.size(), a);
  const size_t n_words = P->blocks.size() * fiona::kSumWords;
  const size_t total = align_up(o_words + sizeof(uint32_t) * n_words, a);
  std::vector<unsigned char> host(total, 0);
  auto put = [&](size_t off, const void *src, size_t n) { if (n) std::memcpy(host.data() + off, src, n); };
  put(o_limbs, C->limbs.data(), sizeof(LimbConst) * C->L);
  put(o_items, P->items.data(), sizeof(uint4) * P->items.size());
  put(o_dest, P->dest.data(), sizeof(uint32_t) * P->dest.size());
  put(o_waves, P->waves.data(), sizeof(uint2) * P->waves.size());
  put(o_splits, P->splits.data(), sizeof(uint4) * P->splits.size());
  put(o_rounds, P->rounds.data(), sizeof(uint4) * P->rounds.size());
  put(o_flush, P->flush.data(), sizeof(uint32_t) * P->flush.size());
  put(o_pm, P->pm.data(), sizeof(uint2) * P->pm.size());
  put(o_mem, P->members.data(), sizeof(uint2) * P->members.size());
  put(o_blocks, P->blocks.data(), sizeof(uint4) * P->blocks.size());
  if (hipGetDevice(&P->device) != hipSuccess) return FIONA_ERR_HIP;
  if (hipMalloc(&P->dev, total) != hipSuccess) {
    P->dev = nullptr;
    return FIONA_ERR_HIP;
  }
  if (hipMemcpy(P->dev, host.data(), total, hipMemcpyHostToDevice) != hipSuccess) return FIONA_ERR_HIP;
  // the kernels' LDS limit, set on the current device with every plan (cheap,
  // and correct whatever device the plan lives on)
  const void *kernels[4] = {(const void *)fiona::hybrid_linear_kernel<8, false>,
                            (const void *)fiona::hybrid_linear_kernel<16, false>,
                            (const void *)fiona::hybrid_linear_kernel<8, true>,
                            (const void *)fiona::hybrid_linear_kernel<16, true>};
  for (const void *k : kernels)
    if (hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsBytes) != hipSuccess)
      return FIONA_ERR_HIP;
  unsigned char *base = (unsigned char *)P->dev;
  P->d_limbs = (const LimbConst *)(base + o_limbs);
  P->d_items = (const uint4 *)(base + o_items);
  P->d_dest = (const uint32_t *)(base + o_dest);
  P->d_waves = (const uint2 *)(base + o_waves);
  P->d_splits = (const uint4 *)(base + o_splits);
  P->d_rounds = (const uint4 *)(base + o_rounds);
  P->d_flush = (const uint32_t *)(base + o_flush);
  P->d_pm = (const uint2 *)(base + o_pm);
  P->d_members = (const uint2 *)(base + o_mem);
  P->d_blocks = (const uint4 *)(base + o_blocks);
  P->d_words = (uint32_t *)(base + o_words);
  return FIONA_OK;
}

// The word blocks of fiona_hybrid_linear_static live in a file-scope device
// array, one copy per device, looked up once per device (hipGetSymbolAddress
// with that device current) and kept for the life of the process.
constexpr size_t kScratchBytes = (size_t)4 << 20;   // 16384 word blocks
constexpr int kScratchDevices = 64;
std::mutex scratch_mutex;
uint32_t *scratch_addr[kScratchDevices] = {};

}  // namespace

static __device__ __align__(256) uint32_t scratch[kScratchBytes / sizeof(uint32_t)];

namespace {

// This device's copy of scratch (dev is current).
int scratch_on(int dev, uint32_t **out) {
  if (dev < 0 || dev >= kScratchDevices) return FIONA_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(scratch_mutex);
  if (!scratch_addr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return FIONA_ERR_HIP;
    scratch_addr[dev] = (uint32_t *)p;
  }
  *out = scratch_addr[dev];
  return FIONA_OK;
}

// Byte sizes of one call's arrays.
struct CallBytes {
  size_t in, pt, out, sign, scale;
};

// The argument checks of a call (nothing is launched on an error).
int check_call(const fiona_plan *plan, const uint64_t *in_cts, const uint64_t *pt_diags, const int8_t *ternary_groups,
               const uint64_t *scales, const uint64_t *out_cts, CallBytes &b) {
  if (!plan) return FIONA_ERR_ARG;
  if (!(plan->passes.empty() ? plan->dev : plan->passes[0]->dev)) return FIONA_ERR_NODEVICE;
  const fiona_ctx *C = plan->ctx;
  const size_t LN = (size_t)C->L * C->N;
  b.in = (size_t)plan->n_in * 2 * LN * 8;
  b.pt = plan->n_pt ? ((size_t)(plan->n_pt - 1) * plan->pt_pitch + LN) * 8 : 0;
  b.out = (size_t)plan->n_out * 2 * LN * 8;
  b.sign = plan->n_member_desc;
  b.scale = (size_t)plan->n_scale * 8;
  if (!in_cts) return FIONA_ERR_ARG;
  if (plan->n_out && !out_cts) return FIONA_ERR_ARG;
  if (plan->any_raw && !pt_diags) return FIONA_ERR_ARG;
  if (plan->any_signed && (!ternary_groups || !scales)) return FIONA_ERR_ARG;
  if (((uintptr_t)in_cts | (uintptr_t)pt_diags | (uintptr_t)scales | (uintptr_t)out_cts) & 7u)
    return FIONA_ERR_ALIGN;
  if (ranges_overlap(out_cts, b.out, in_cts, b.in) || ranges_overlap(out_cts, b.out, pt_diags, b.pt) ||
      ranges_overlap(out_cts, b.out, ternary_groups, b.sign) || ranges_overlap(out_cts, b.out, scales, b.scale))
    return FIONA_ERR_ALIAS;
  if (plan->n_out == 0) return FIONA_OK;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != plan->device) return FIONA_ERR_ARG;
  return FIONA_OK;
}

// The launches of one call: the sign-packing kernel writes this call's word
// blocks at words (plan->blocks.size() blocks of kSumWords words), then the
// main kernel reads them.
int enqueue_one(const fiona_plan *plan, const uint64_t *in_cts, const uint64_t *pt_diags,
                  const int8_t *ternary_groups, const uint64_t *scales, uint64_t *out_cts, uint32_t *words,
                  const CallBytes &b, hipStream_t stream) {
  const uint32_t n_blocks = (uint32_t)plan->blocks.size();
  if (n_blocks) {   // this call's signs and scales: the word blocks
    PackParams pp;
    pp.signs = ternary_groups;
    pp.members = plan->d_members;
    pp.blocks = plan->d_blocks;
    pp.words = words;
    pp.scales = scales;
    pp.n_blocks = n_blocks;
    hipLaunchKernelGGL(fiona::pack_members_kernel, dim3((n_blocks + 3) / 4), dim3(256), 0, stream, pp);
    if (hipGetLastError() != hipSuccess) return FIONA_ERR_HIP;
  }
  auto kernel = plan->nw == 16 ? (plan->accumulate ? fiona::hybrid_linear_kernel<16, true>
                                                  : fiona::hybrid_linear_kernel<16, false>)
                                : (plan->accumulate ? fiona::hybrid_linear_kernel<8, true>
                                                    : fiona::hybrid_linear_kernel<8, false>);
  fiona::KPlan kp;
  kp.limbs = plan->d_limbs;
  kp.items = plan->d_items;
  kp.dest = plan->d_dest;
  kp.waves = plan->d_waves;
  kp.rounds = plan->d_rounds;
  kp.flush = plan->d_flush;
  kp.splits = plan->d_splits;
  kp.pm = plan->d_pm;
  kp.words = words;
  hipLaunchKernelGGL(kernel, dim3(plan->grid), dim3(plan->nw * 64), plan->lds_bytes, stream, in_cts, pt_diags,
                     out_cts, kp, plan->shape, (const void *)((const char *)pt_diags + b.pt),
                     (const void *)((const char *)out_cts + b.out));
  if (hipGetLastError() != hipSuccess) return FIONA_ERR_HIP;
  return FIONA_OK;
}

// A call of a plan with or without passes; words: the word blocks of each
// pass (null: each pass's own workspace).  The passes run in turn on the
// stream, so that a later pass adds to the outputs of the earlier ones and
// may reuse the same word blocks.
int enqueue_layer(const fiona_plan *plan, const uint64_t *in_cts, const uint64_t *pt_diags,
                  const int8_t *ternary_groups, const uint64_t *scales, uint64_t *out_cts, uint32_t *words,
                  const CallBytes &b, hipStream_t stream) {
  if (plan->passes.empty())
    return enqueue_one(plan, in_cts, pt_diags, ternary_groups, scales, out_cts, words ? words : plan->d_words, b,
                       stream);
  const size_t LN = (size_t)plan->ctx->L * plan->ctx->N;
  for (const fiona_plan *S : plan->passes) {
    CallBytes bs = b;
    bs.in = (size_t)S->n_in * 2 * LN * 8;
    const int rc = enqueue_one(S, in_cts + (size_t)S->in_base * 2 * LN, pt_diags, ternary_groups, scales, out_cts,
                               words ? words : S->d_words, bs, stream);
    if (rc != FIONA_OK) return rc;
  }
  return FIONA_OK;
}

// Inputs per pass of a layer with more than FIONA_MAX_INPUTS inputs: room
// for common partial sums, resident sums and output rows beside them.
constexpr uint32_t kPassInputs = 128;

// Compiles one plan over all of d's inputs and, unless host-only, uploads it.
// slot_map (or null): for each member of d, its index in the caller's
// ternary_groups; n_member: the caller's member count.
int build_plan(const fiona_ctx *ctx, const fiona_layer_desc *d, uint64_t pitch, const std::vector<uint32_t> *slot_map,
               uint32_t n_member, fiona_plan **out) {
  fiona_plan *P = new (std::nothrow) fiona_plan;
  if (!P) return FIONA_ERR_NOMEM;
  P->ctx = ctx;
  P->n_in = d->n_in;
  P->n_out = d->n_out;
  P->n_pt = d->n_pt;
  P->pt_pitch = pitch;
  P->n_scale = d->n_scale;
  P->flags = d->flags;
  int rc;
  try {
    rc = compile_plan(P, d);
    if (rc == FIONA_OK && slot_map)
      for (auto &m : P->members) m.y = (*slot_map)[m.y];
  } catch (...) {
    rc = FIONA_ERR_NOMEM;
  }
  if (rc != FIONA_OK) {
    delete P;
    return rc;
  }
  P->n_member_desc = n_member;
  P->tiles = (ctx->N + fiona::kTile - 1) / fiona::kTile;
  P->grid = P->tiles * ctx->L;
  P->lds_bytes = (P->n_in + P->n_part + P->n_mat + P->n_seg_slots + 1 + P->obuf_rows) * kSlotBytes;
  P->st.tile = fiona::kTile;
  P->st.waves = P->nw;
  P->st.split_outputs = (uint32_t)P->splits.size();
  P->st.segment_slots = P->n_seg_slots;
  P->st.output_rounds = P->n_rounds;
  P->st.output_buffer_rows = P->obuf_rows;
  P->st.lds_bytes = P->lds_bytes;
  P->st.grid = P->grid;
  P->st.input_passes = 1;
  KShape &k = P->shape;
  k.N = ctx->N;
  k.L = ctx->L;
  k.n_in = P->n_in;
  k.n_mat = P->n_mat;
  k.zero_row = P->n_in + P->n_part + P->n_mat + P->n_seg_slots;
  k.n_rounds = P->n_rounds;
  k.obuf_row = k.zero_row + 1;
  k.use_block0 = P->n_part + P->n_mat;
  k.n_part = P->n_part;
  k.n_levels = P->n_levels;
  for (uint32_t l = 0; l < fiona::kMaxLevels; ++l) k.level_end[l] = P->part_levels[l];
  k.tiles = P->tiles;
  if (!(d->flags & FIONA_PLAN_HOST_ONLY)) {
    rc = upload_plan(P);
    if (rc != FIONA_OK) {
      fiona_plan_destroy(P);
      return rc;
    }
  }
  *out = P;
  return FIONA_OK;
}

// The passes of a layer with more inputs than one tile's LDS holds: the
// inputs are cut into consecutive ranges of at most kPassInputs, and pass g
// takes the raw terms and the group members whose input falls in its range.
// A group whose members span several ranges becomes one sub-sum per range,
// each with the group's scale (exact: c (U1 + U2) = c U1 + c U2).
int build_passes(const fiona_ctx *ctx, const fiona_layer_desc *d, uint64_t pitch, fiona_plan *P) {
  const uint32_t n_pass = (d->n_in + kPassInputs - 1) / kPassInputs;
  const uint32_t per = (d->n_in + n_pass - 1) / n_pass;
  const uint32_t n_group = d->grp_off[d->n_out];
  const uint32_t n_member = n_group ? d->grp_mem_off[n_group] : 0;
  fiona_plan_stats_t &st = P->st;
  for (uint32_t g = 0; g < n_pass; ++g) {
    const uint32_t i0 = g * per, i1 = std::min(d->n_in, i0 + per);
    std::vector<uint32_t> pm_off(d->n_out + 1, 0), pm_input, pm_pt, grp_off(d->n_out + 1, 0), grp_mem_off(1, 0),
        mem_input, grp_scale, slot_map;
    std::vector<int8_t> mem_sign;
    for (uint32_t j = 0; j < d->n_out; ++j) {
      for (uint32_t t = d->pm_off[j]; t < d->pm_off[j + 1]; ++t)
        if (d->pm_input[t] >= i0 && d->pm_input[t] < i1) {
          pm_input.push_back(d->pm_input[t] - i0);
          pm_pt.push_back(d->pm_pt[t]);
        }
      pm_off[j + 1] = (uint32_t)pm_input.size();
      for (uint32_t q = d->grp_off[j]; q < d->grp_off[j + 1]; ++q) {
        const size_t before = mem_input.size();
        for (uint32_t m = d->grp_mem_off[q]; m < d->grp_mem_off[q + 1]; ++m)
          if (d->mem_input[m] >= i0 && d->mem_input[m] < i1) {
            mem_input.push_back(d->mem_input[m] - i0);
            mem_sign.push_back(d->mem_sign[m]);
            slot_map.push_back(m);
          }
        if (mem_input.size() > before) {
          grp_mem_off.push_back((uint32_t)mem_input.size());
          grp_scale.push_back(d->grp_scale[q]);
        }
      }
      grp_off[j + 1] = (uint32_t)grp_scale.size();
    }
    // a range that no term reads adds nothing: no pass (unless every range
    // is empty, when the first pass still writes the zero outputs)
    if (pm_input.empty() && grp_scale.empty() && (g + 1 < n_pass || !P->passes.empty())) continue;
    fiona_layer_desc sd = *d;
    sd.n_in = i1 - i0;
    sd.pm_off = pm_off.data();
    sd.pm_input = pm_input.data();
    sd.pm_pt = pm_pt.data();
    sd.grp_off = grp_off.data();
    sd.grp_mem_off = grp_mem_off.data();
    sd.mem_input = mem_input.data();
    sd.mem_sign = mem_sign.data();
    sd.grp_scale = grp_scale.data();
    sd.flags = d->flags & ~FIONA_PLAN_CHECK_INPUTS;
    sd.pt_pitch = pitch;
    fiona_plan *S = nullptr;
    const int rc = build_plan(ctx, &sd, pitch, &slot_map, n_member, &S);
    if (rc != FIONA_OK) return rc;
    S->in_base = i0;
    S->accumulate = !P->passes.empty();
    P->passes.push_back(S);
    // counts add up over the passes; the launch shape is the widest pass's
    const fiona_plan_stats_t &a = S->st;
    st.ct_terms += a.ct_terms;
    st.n_pmult += a.n_pmult;
    st.n_member += a.n_member;
    st.n_member_nonzero += a.n_member_nonzero;
    st.n_use += a.n_use;
    st.n_sum_distinct += a.n_sum_distinct;
    st.n_sum_resident += a.n_sum_resident;
    st.pmult_per_contribution += a.pmult_per_contribution;
    st.pmult_grouped += a.pmult_grouped;
    st.addsub_unshared += a.addsub_unshared;
    st.addsub_shared += a.addsub_shared;
    st.addsub_partial += a.addsub_partial;
    st.tile = a.tile;
    st.waves = std::max(st.waves, a.waves);
    st.lds_bytes = std::max(st.lds_bytes, a.lds_bytes);
    st.grid = a.grid;
    st.split_outputs += a.split_outputs;
    st.segment_slots = std::max(st.segment_slots, a.segment_slots);
    st.n_partial += a.n_partial;
    st.partial_levels = std::max(st.partial_levels, a.partial_levels);
    st.output_rounds = std::max(st.output_rounds, a.output_rounds);
    st.output_buffer_rows = std::max(st.output_buffer_rows, a.output_buffer_rows);
    P->any_signed = P->any_signed || S->any_signed;
    P->any_raw = P->any_raw || S->any_raw;
    P->device = S->device;
  }
  st.input_passes = (uint32_t)P->passes.size();
  return FIONA_OK;
}

}  // namespace

extern "C" {

int fiona_plan_create(const fiona_ctx *ctx, const fiona_layer_desc *desc, fiona_plan **out) {
  if (!out) return FIONA_ERR_ARG;
  *out = nullptr;
  if (!ctx || !desc) return FIONA_ERR_ARG;
  int rc = validate_desc(desc);
  if (rc != FIONA_OK) return rc;
  if (desc->n_in > FIONA_MAX_LAYER_INPUTS) return FIONA_ERR_UNSUPPORTED;
  const uint64_t ln = (uint64_t)ctx->L * ctx->N;
  const uint64_t pitch = desc->pt_pitch ? desc->pt_pitch : ln;
  if (pitch < ln || pitch > (1ull << 45)) return FIONA_ERR_ARG;
  // raw-term records hold 48-bit byte offsets into the plaintext table
  if (((uint64_t)desc->n_pt * pitch) * 8 > (1ull << 48)) return FIONA_ERR_UNSUPPORTED;
  const uint32_t n_group = desc->grp_off[desc->n_out];
  const uint32_t n_member = n_group ? desc->grp_mem_off[n_group] : 0;
  fiona_plan *P = nullptr;
  if (desc->n_in <= FIONA_MAX_INPUTS) {
    rc = build_plan(ctx, desc, pitch, nullptr, n_member, &P);
    if (rc != FIONA_OK) return rc;
  } else {
    P = new (std::nothrow) fiona_plan;
    if (!P) return FIONA_ERR_NOMEM;
    P->ctx = ctx;
    P->n_in = desc->n_in;
    P->n_out = desc->n_out;
    P->n_pt = desc->n_pt;
    P->pt_pitch = pitch;
    P->n_scale = desc->n_scale;
    P->flags = desc->flags;
    P->n_member_desc = n_member;
    try {
      rc = build_passes(ctx, desc, pitch, P);
    } catch (...) {
      rc = FIONA_ERR_NOMEM;
    }
    if (rc != FIONA_OK) {
      fiona_plan_destroy(P);
      return rc;
    }
  }
  if ((desc->flags & FIONA_PLAN_CHECK_INPUTS) && n_member) {
    try {
      P->signs.assign(desc->mem_sign, desc->mem_sign + n_member);
    } catch (...) {
      fiona_plan_destroy(P);
      return FIONA_ERR_NOMEM;
    }
  }
  *out = P;
  return FIONA_OK;
}

void fiona_plan_destroy(fiona_plan *plan) {
  if (!plan) return;
  for (fiona_plan *S : plan->passes) fiona_plan_destroy(S);
  if (plan->dev) (void)hipFree(plan->dev);
  delete plan;
}

int fiona_plan_stats(const fiona_plan *plan, fiona_plan_stats_t *out) {
  if (!plan || !out) return FIONA_ERR_ARG;
  *out = plan->st;
  return FIONA_OK;
}

int fiona_plan_check_inputs(const fiona_plan *plan, const int8_t *signs, const uint64_t *scales, const uint64_t *in,
                            const uint64_t *pt) {
  if (!plan || !(plan->flags & FIONA_PLAN_CHECK_INPUTS)) return FIONA_ERR_ARG;
  if ((plan->n_member_desc && !signs) || (plan->n_scale && !scales)) return FIONA_ERR_ARG;
  if (plan->n_member_desc && std::memcmp(signs, plan->signs.data(), plan->n_member_desc) != 0)
    return FIONA_ERR_PRECONDITION;
  for (uint32_t c = 0; c < plan->n_scale; ++c)
    if (scales[c] >> FIONA_SCALE_BITS) return FIONA_ERR_PRECONDITION;
  const size_t LN = (size_t)plan->ctx->L * plan->ctx->N;
  if (in)
    for (size_t w = 0; w < (size_t)plan->n_in * 2 * LN; ++w)
      if (in[w] >> FIONA_MODULUS_BITS) return FIONA_ERR_PRECONDITION;
  if (pt)
    for (size_t r = 0; r < plan->n_pt; ++r)
      for (size_t w = 0; w < LN; ++w)
        if (pt[r * plan->pt_pitch + w] >> FIONA_MODULUS_BITS) return FIONA_ERR_PRECONDITION;
  return FIONA_OK;
}

int fiona_hybrid_linear(const fiona_plan *plan, const uint64_t *in_cts, const uint64_t *pt_diags,
                        const int8_t *ternary_groups, const uint64_t *scales, uint64_t *out_cts,
                        hipStream_t stream) {
  CallBytes b;
  int rc = check_call(plan, in_cts, pt_diags, ternary_groups, scales, out_cts, b);
  if (rc != FIONA_OK || plan->n_out == 0) return rc;
  if (plan->flags & FIONA_PLAN_CHECK_INPUTS) {   // a checking plan: the preconditions, on host copies
    try {
      std::vector<int8_t> hs(b.sign);
      std::vector<uint64_t> hc(plan->n_scale), hi(b.in / 8), hp(b.pt / 8);
      auto back = [&](void *dst, const void *src, size_t n) {
        return n == 0 || hipMemcpyAsync(dst, src, n, hipMemcpyDeviceToHost, stream) == hipSuccess;
      };
      if (!back(hs.data(), ternary_groups, b.sign) || !back(hc.data(), scales, b.scale) ||
          !back(hi.data(), in_cts, b.in) || !back(hp.data(), pt_diags, b.pt) ||
          hipStreamSynchronize(stream) != hipSuccess)
        return FIONA_ERR_HIP;
      rc = fiona_plan_check_inputs(plan, hs.data(), hc.data(), hi.data(), b.pt ? hp.data() : nullptr);
    } catch (...) {
      return FIONA_ERR_NOMEM;
    }
    if (rc != FIONA_OK) return rc;
  }
  return enqueue_layer(plan, in_cts, pt_diags, ternary_groups, scales, out_cts, nullptr, b, stream);
}

int fiona_hybrid_linear_static(const fiona_plan *plan, const uint64_t *in_cts, const uint64_t *pt_diags,
                               const int8_t *ternary_groups, const uint64_t *scales, uint64_t *out_cts,
                               hipStream_t stream) {
  CallBytes b;
  int rc = check_call(plan, in_cts, pt_diags, ternary_groups, scales, out_cts, b);
  if (rc != FIONA_OK || plan->n_out == 0) return rc;
  if (plan->flags & FIONA_PLAN_CHECK_INPUTS) return FIONA_ERR_ARG;   // its check copies into host memory
  size_t blocks = plan->blocks.size();
  for (const fiona_plan *S : plan->passes) blocks = std::max(blocks, S->blocks.size());
  if (blocks * fiona::kSumWords * sizeof(uint32_t) > kScratchBytes) return FIONA_ERR_UNSUPPORTED;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return FIONA_ERR_HIP;
  uint32_t *words = nullptr;
  rc = scratch_on(dev, &words);
  if (rc != FIONA_OK) return rc;
  return enqueue_layer(plan, in_cts, pt_diags, ternary_groups, scales, out_cts, words, b, stream);
}

}  // extern "C"
