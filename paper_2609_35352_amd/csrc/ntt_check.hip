// Host replay of the NTT passes' memory accesses.
//
// A rescaler or rotator is laid out at fake device addresses, one call is
// recorded instead of launched (ntt_host.hpp), and every global access of
// every workgroup and thread of every recorded pass is recomputed on the host
// through the same offset helpers the kernels use (GeomA, GeomB, GeomRot in
// ntt_kernel.hpp).  Each access must lie inside the buffer that holds its
// descriptor's base, every offset must stay below 2^32 bytes, and every
// descriptor's end pointer must be that buffer's end.  No device is needed.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <string>
#include <vector>

#include "fiona.h"
#include "ntt_host.hpp"

namespace fiona_host {

namespace {

using fiona::DftShape;
using fiona::GeomA;
using fiona::GeomB;
using fiona::GeomRot;
using fiona::Off;
using fiona::kNttCols;

struct Checker {
  const std::vector<Region> &regions;
  uint64_t sets_dev;
  const std::vector<NttSet> &sets_host;
  std::string err, end_err;   // end_err: a descriptor end that differs (reported after the accesses)
  size_t launch = 0;

  const Region *find(uint64_t a) const {
    for (const Region &r : regions)
      if (a >= r.lo && a < r.hi) return &r;
    return nullptr;
  }
  bool fail(const std::string &m) {
    if (err.empty()) err = "launch " + std::to_string(launch) + ": " + m;
    return false;
  }
  // bytes [base + lo, base + hi) must lie in the region that holds base;
  // end (if not null) must be that region's end
  bool span(const char *what, uint64_t base, uint64_t lo, uint64_t hi, const void *end) {
    if (hi <= lo) return true;
    if (fiona::join_halves((uint32_t)(base >> 32), (uint32_t)base) != base)
      return fail(std::string(what) + ": base not rebuilt from its halves");
    const Region *r = find(base);
    if (!r) return fail(std::string(what) + ": base outside every buffer");
    if (base + hi > r->hi)
      return fail(std::string(what) + ": bytes up to " + std::to_string(base + hi - r->lo) + " of " + r->name +
                  " (" + std::to_string(r->hi - r->lo) + " bytes)");
    if (end && (uint64_t)end != r->hi && end_err.empty())
      end_err = "launch " + std::to_string(launch) + ": " + what + ": descriptor end differs from the end of " +
                r->name;
    return true;
  }
  // the largest end (offset + bytes) of accesses with offsets o, and the 2^32 limit
  bool grow(uint64_t &hi, Off o, uint32_t bytes, const char *what) {
    const uint64_t off = (uint64_t)o.v + o.s;
    if (off + bytes > 0xFFFFFFFFull) return fail(std::string(what) + ": offset beyond 2^32 bytes");
    hi = std::max(hi, off + bytes);
    return true;
  }
  const NttSet *set(const NttSet *p, uint32_t s) {
    const uint64_t a = (uint64_t)(p + s);
    if (a < sets_dev || (a - sets_dev) % sizeof(NttSet) != 0 || (a - sets_dev) / sizeof(NttSet) >= sets_host.size()) {
      fail("set record " + std::to_string(s) + " outside the NttSet array");
      return nullptr;
    }
    return &sets_host[(a - sets_dev) / sizeof(NttSet)];
  }
  bool tables(const NttSet &S, const Tw *dft, uint32_t logm) {
    return span("DFT twiddles", (uint64_t)dft, 0, (uint64_t)(1u << logm) / 2 * sizeof(Tw), nullptr);
  }
};

template <uint32_t LOGM>
bool pass_a(Checker &C, const PassLaunch &L) {
  using D = DftShape<LOGM>;
  using G = GeomA<LOGM>;
  const NttPass &P = L.P;
  const uint32_t N1 = 1u << P.log_n1, N2 = D::M, gx = N1 / kNttCols;
  if (P.log_n1 != L.log_other || N1 < kNttCols) return C.fail("pass A: bad sides");
  const bool trans = P.load == fiona::kLoadU64T;
  // per column block: the largest ends of the accesses relative to each descriptor's base
  std::vector<uint64_t> in_hi(gx, 0), pre_hi(gx, 0), tmp_hi(gx, 0), mid_hi(gx, 0);
  for (uint32_t cb = 0; cb < gx; ++cb) {
    for (uint32_t it = 0; it < D::IT1; ++it) {
      const uint32_t cl = G::col(it, trans), ip = G::grp(it, trans), n1 = cb * kNttCols + cl;
      for (uint32_t u = 0; u < 16; ++u) {
        if (!C.grow(in_hi[cb], trans ? G::in_t(n1, ip, u, N1) : G::in(n1, ip, u, N1), 8, "pass A input"))
          return false;
        if (!trans && !C.grow(pre_hi[cb], G::pre(ip, u), 16, "pass A pre")) return false;
      }
    }
    for (uint32_t it = 0; it < D::IT2; ++it) {
      const uint32_t cl = G::col2(it), o = G::off2(it), n1 = cb * kNttCols + cl;
      for (uint32_t u = 0; u < D::E2; ++u)
        if (!C.grow(tmp_hi[cb], G::tmp(o, n1, u, N1), 8, "pass A tmp") ||
            !C.grow(mid_hi[cb], G::mid(o, n1, u, N1), 16, "pass A mid"))
          return false;
    }
  }
  for (uint32_t by = 0; by < L.V; ++by)
    for (uint32_t bx = 0; bx < gx; ++bx) {
      const fiona::UnitA un = fiona::pass_a_unit(P.vps, P.nsets_shared, bx, by, gx);
      const NttSet *S = C.set(P.sets, un.set);
      if (!S) return false;
      const uint64_t v = (uint64_t)un.set * P.vps + un.lv;
      const uint64_t in_base = (uint64_t)P.in + (un.set * P.in_set_stride + un.lv * P.in_stride) * 8;
      const uint64_t tmp_base = (uint64_t)P.tmp + v * N1 * N2 * 8;
      if (!C.span("pass A input", in_base, 0, in_hi[un.cb], P.in_end) ||
          !C.span("pass A tmp", tmp_base, 0, tmp_hi[un.cb], P.tmp_end) ||
          !C.span("pass A mid", (uint64_t)S->mid, 0, mid_hi[un.cb], nullptr) ||
          !C.span("pass A mid table", (uint64_t)S->mid, 0, (uint64_t)N1 * N2 * sizeof(Tw), nullptr) ||
          !C.tables(*S, S->dft_a, LOGM))
        return false;
      if (!trans && S->pre &&
          (!C.span("pass A pre", (uint64_t)S->pre, 0, pre_hi[un.cb], nullptr) ||
           !C.span("pass A pre table", (uint64_t)S->pre, 0, (uint64_t)N2 * sizeof(Tw), nullptr)))
        return false;
    }
  return true;
}

template <uint32_t LOGM>
bool pass_b(Checker &C, const PassLaunch &L) {
  using D = DftShape<LOGM>;
  using G = GeomB<LOGM>;
  const NttPass &P = L.P;
  const uint32_t M = D::M, N2 = 1u << P.log_n2, gx = N2 / kNttCols;
  if (P.log_n2 != L.log_other || N2 < kNttCols) return C.fail("pass B: bad sides");
  const bool transposed = P.out_transposed != 0 && P.store != fiona::kStoreF64;
  const bool rescale = P.store == fiona::kStoreRescale;
  uint64_t tmp_hi = 0;
  for (uint32_t it = 0; it < D::IT1; ++it)
    for (uint32_t u = 0; u < 16; ++u)
      if (!C.grow(tmp_hi, G::tmp(G::row(it), G::grp(it), u), 8, "pass B tmp")) return false;
  std::vector<uint64_t> out_hi(gx, 0), base_hi(gx, 0);
  uint64_t post_hi = 0;
  for (uint32_t x = 0; x < gx; ++x) {
    const uint32_t r0 = x * kNttCols;
    for (uint32_t it = 0; it < D::IT2; ++it) {
      const uint32_t row = G::row2(it, transposed), o = G::off2(it, transposed), k2 = r0 + row;
      for (uint32_t u = 0; u < D::E2; ++u) {
        if (!C.grow(post_hi, G::post(o, u), 16, "pass B post")) return false;
        const Off oc = G::col(k2, o, u, N2);
        if (rescale && !C.grow(base_hi[x], oc, 8, "pass B base")) return false;
        if (!C.grow(out_hi[x], transposed ? G::row_t(k2, o, u) : oc, 8, "pass B output")) return false;
      }
    }
  }
  for (uint32_t by = 0; by < L.V; ++by) {
    const uint32_t set = by / P.vps, lv = by - set * P.vps;
    const NttSet *S = C.set(P.sets, set);
    if (!S || !C.tables(*S, S->dft_b, LOGM)) return false;
    if (S->post && (!C.span("pass B post", (uint64_t)S->post, 0, post_hi, nullptr) ||
                    !C.span("pass B post table", (uint64_t)S->post, 0, (uint64_t)M * sizeof(Tw), nullptr)))
      return false;
    for (uint32_t x = 0; x < gx; ++x) {
      const uint64_t tmp_base = (uint64_t)P.tmp + ((uint64_t)by * N2 * M + (uint64_t)x * kNttCols * M) * 8;
      const uint64_t out_base = (uint64_t)P.out + (set * P.out_set_stride + lv * P.out_stride) * 8;
      if (!C.span("pass B tmp", tmp_base, 0, tmp_hi, P.tmp_end) ||
          !C.span("pass B output", out_base, 0, out_hi[x], P.out_end))
        return false;
      if (rescale &&
          !C.span("pass B base", (uint64_t)P.base + (set * P.base_set_stride + lv * P.base_stride) * 8, 0, base_hi[x],
                  P.base_end))
        return false;
    }
  }
  return true;
}

template <uint32_t LOGM>
bool pass_b_rot(Checker &C, const PassLaunch &L) {
  using D = DftShape<LOGM>;
  using G = GeomRot<LOGM>;
  const NttPass &P = L.P;
  const RotArgs &R = L.G;
  const uint32_t N2 = 1u << P.log_n2, N = D::M << P.log_n2, gx = N2 / kNttCols;
  if (P.log_n2 != L.log_other || N2 < kNttCols || R.n_rot == 0 || R.n_rot > fiona::kRotMax)
    return C.fail("rotation pass B: bad shape");
  // per (column block, rotation): the rows read depend on the Galois element
  std::vector<uint64_t> tmp_hi((size_t)gx * R.n_rot, 0), word_hi((size_t)gx * R.n_rot, 0), out_hi(gx, 0);
  for (uint32_t x = 0; x < gx; ++x) {
    const uint32_t o0 = x * kNttCols;
    for (uint32_t r = 0; r < R.n_rot; ++r) {
      const uint32_t g = R.g[r];
      uint64_t &th = tmp_hi[(size_t)x * R.n_rot + r], &wh = word_hi[(size_t)x * R.n_rot + r];
      for (uint32_t it = 0; it < D::IT1; ++it) {
        const uint32_t k2 = G::src_row(g, o0 + G::row(it), N2);
        for (uint32_t u = 0; u < 16; ++u)
          if (!C.grow(th, G::tmp(k2, G::grp(it), u), 8, "rotation pass B tmp")) return false;
      }
      for (uint32_t it = 0; it < D::IT2; ++it) {
        const uint32_t k2c = G::src_row(g, o0 + G::row2(it), N2);
        for (uint32_t u = 0; u < D::E2; ++u)
          if (!C.grow(wh, G::word(k2c, G::off2(it), u), 8, "rotation pass B u'/c0")) return false;
      }
    }
    for (uint32_t t = 0; t < fiona::kNttThreads; ++t)
      for (uint32_t j = 0; j < G::PER; ++j)
        if (!C.grow(out_hi[x], G::out(o0, t, j, N2), 8, "rotation pass B output")) return false;
  }
  for (uint32_t by = 0; by < L.V; ++by) {
    const uint32_t set = by / P.vps, lv = by - set * P.vps, p = lv / R.n_rot, r = lv - p * R.n_rot;
    if (p > 1) return C.fail("rotation pass B: more than two polynomials per rotation");
    const NttSet *S = C.set(P.sets, set);
    if (!S || !C.tables(*S, S->dft_b, LOGM)) return false;
    for (uint32_t x = 0; x < gx; ++x) {
      const size_t xr = (size_t)x * R.n_rot + r;
      if (!C.span("rotation pass B tmp", (uint64_t)P.tmp + (uint64_t)by * N * 8, 0, tmp_hi[xr], P.tmp_end) ||
          !C.span("rotation pass B u'", (uint64_t)P.base + (set * P.base_set_stride + lv * P.base_stride) * 8, 0,
                  word_hi[xr], P.base_end) ||
          (p == 0 && !C.span("rotation pass B c0", (uint64_t)P.add + set * P.add_set_stride * 8, 0, word_hi[xr],
                             P.add_end)) ||
          !C.span("rotation pass B output", (uint64_t)P.out + (((uint64_t)r * 2 + p) * R.L + set) * N * 8, 0,
                  out_hi[x], P.out_end))
        return false;
    }
  }
  return true;
}

template <uint32_t LOGM>
bool replay_one(Checker &C, const PassLaunch &L) {
  switch (L.kind) {
    case PassLaunch::kPassA: return pass_a<LOGM>(C, L);
    case PassLaunch::kPassB: return pass_b<LOGM>(C, L);
    default: return pass_b_rot<LOGM>(C, L);
  }
}

}  // namespace

std::string check_launches(const LaunchRecord &rec, const std::vector<Region> &regions, uint64_t sets_dev,
                           const std::vector<NttSet> &sets_host) {
  Checker C{regions, sets_dev, sets_host, std::string()};
  for (const SpanAccess &s : rec.spans)
    if (!C.span(s.what, s.base, s.lo, s.hi, nullptr)) return C.err;
  for (const PassLaunch &L : rec.passes) {
    if (L.V == 0 || L.V > 65535 || L.P.vps == 0) {
      C.fail("bad vector count");
      return C.err;
    }
    bool ok = false;
    switch (L.log_side) {
      case 4: ok = replay_one<4>(C, L); break;
      case 5: ok = replay_one<5>(C, L); break;
      case 6: ok = replay_one<6>(C, L); break;
      case 7: ok = replay_one<7>(C, L); break;
      case 8: ok = replay_one<8>(C, L); break;
      case 9: ok = replay_one<9>(C, L); break;
      default: C.fail("DFT side outside 2^4 .. 2^9"); break;
    }
    if (!ok) return C.err;
    ++C.launch;
  }
  return C.end_err;
}

}  // namespace fiona_host

extern "C" int fiona_check_ntt_offsets(uint32_t op, uint32_t N, uint32_t L, const uint64_t *moduli,
                                       uint32_t capacity, uint32_t n_call, uint64_t out_shrink, char *msg,
                                       size_t msg_len) {
  if (!moduli || op > 1) return FIONA_ERR_ARG;
  std::string err;
  int rc;
  try {
    rc = op == 0 ? fiona_host::rescale_replay(moduli, N, L, capacity, n_call, out_shrink, err)
                 : fiona_host::rotate_replay(moduli, N, L, capacity, n_call, out_shrink, err);
  } catch (...) {
    return FIONA_ERR_NOMEM;
  }
  if (msg && msg_len) {
    std::strncpy(msg, err.c_str(), msg_len - 1);
    msg[msg_len - 1] = '\0';
  }
  return rc;
}
