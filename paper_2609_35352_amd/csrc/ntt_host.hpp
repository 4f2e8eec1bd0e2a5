// Host side of the NTT passes (ntt_kernel.hpp): twiddle tables, the table
// image in device memory, and the launch of one pass.  Shared by the rescale
// epilogue (rescale.hip) and the rotation producer (rotate.hip).
#pragma once
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "ntt_kernel.hpp"

namespace fiona_host {

using fiona::NttPass;
using fiona::NttSet;
using fiona::RotArgs;
using fiona::Tw;

// A launch as the host replay sees it (ntt_check.hip).  With a recorder
// installed, the launch helpers below record their launches instead of
// issuing them; the other kernels of a call record the byte ranges they
// touch.
struct PassLaunch {
  enum Kind : uint32_t { kPassA, kPassB, kPassBRot } kind;
  uint32_t log_side, log_other, V;   // DFT side, the other side, vectors (gridDim.y)
  NttPass P;
  RotArgs G;                         // kPassBRot only
};
struct SpanAccess {   // a kernel that is not an NTT pass: bytes [lo, hi) of the buffer at base
  const char *what;
  uint64_t base, lo, hi;
};
struct LaunchRecord {
  std::vector<PassLaunch> passes;
  std::vector<SpanAccess> spans;
};
inline LaunchRecord *&launch_recorder() {
  static thread_local LaunchRecord *rec = nullptr;
  return rec;
}
inline bool record_span(const char *what, const void *base, uint64_t lo, uint64_t hi) {
  LaunchRecord *rec = launch_recorder();
  if (!rec) return false;
  rec->spans.push_back(SpanAccess{what, (uint64_t)base, lo, hi});
  return true;
}

// A buffer of the replayed layout: bytes [lo, hi) of a fake address space.
struct Region {
  uint64_t lo, hi;
  std::string name;
};
// Checks every access of the recorded launches: each must fall inside the
// region that holds its descriptor's base, and each descriptor's end pointer
// must be that region's end.  sets_dev / sets_host: the device address of
// the table image's NttSet array and its host copy.  Returns "" or the
// first violation.
std::string check_launches(const LaunchRecord &rec, const std::vector<Region> &regions, uint64_t sets_dev,
                           const std::vector<NttSet> &sets_host);
// The replays of a rescale and of a rotation call (rescale.hip, rotate.hip).
int rescale_replay(const uint64_t *moduli, uint32_t N, uint32_t L, uint32_t max_ct, uint32_t n_ct,
                   uint64_t out_shrink, std::string &err);
int rotate_replay(const uint64_t *moduli, uint32_t N, uint32_t L, uint32_t max_rot, uint32_t n_rot,
                  uint64_t out_shrink, std::string &err);

inline uint64_t mulmod_h(uint64_t a, uint64_t b, uint64_t q) { return (uint64_t)((unsigned __int128)a * b % q); }

inline uint64_t powmod_h(uint64_t b, uint64_t e, uint64_t q) {
  uint64_t r = 1 % q;
  b %= q;
  while (e) {
    if (e & 1) r = mulmod_h(r, b, q);
    b = mulmod_h(b, b, q);
    e >>= 1;
  }
  return r;
}

inline Tw make_tw(uint64_t w, uint64_t q) { return Tw{(double)w, (double)w / (double)q}; }

// The default root: psi = x^((q-1)/2N) for the smallest x >= 2 with psi^N = -1.
inline uint64_t default_psi(uint32_t N, uint64_t q) {
  for (uint64_t x = 2; x < 1000000; ++x) {
    const uint64_t psi = powmod_h(x, (q - 1) / (2ull * N), q);
    if (powmod_h(psi, N, q) == q - 1) return psi;
  }
  return 0;
}

// Tables of one direction of one modulus, for n = n1 + N1 n2 on the input
// side and k = k2 + N2 k1 on the output side.  Forward: the twist psi^n
// splits as psi^(N1 n2) psi^n1; pre = psi^(N1 n2) (N2 entries) and the
// factor psi^n1, constant along pass A's DFT, joins mid = omega^(n1 k2)
// psi^n1 at k2 N1 + n1.  Inverse (omega -> omega^-1): the factor
// N^-1 psi^-k = N^-1 psi^-k2 psi^(-N2 k1); the part in k2, constant along
// pass B's DFT, joins mid = omega^(-n1 k2) N^-1 psi^-k2, and post =
// psi^(-N2 k1) (N1 entries).  DFT roots omega^N1 (size N2) and omega^N2
// (size N1).
struct TableSet {
  std::vector<Tw> pre, mid, dft_a, dft_b, post;
};

inline TableSet make_tables(uint32_t log_n1, uint32_t log_n2, uint64_t q, uint64_t psi, bool inverse) {
  const uint32_t N1 = 1u << log_n1, N2 = 1u << log_n2, N = N1 * N2;
  const uint64_t psi_inv = powmod_h(psi, q - 2, q);
  const uint64_t omega = inverse ? mulmod_h(psi_inv, psi_inv, q) : mulmod_h(psi, psi, q);
  TableSet t;
  if (!inverse) {
    t.pre.resize(N2);
    const uint64_t step = powmod_h(psi, N1, q);
    uint64_t p = 1;
    for (uint32_t n2 = 0; n2 < N2; ++n2, p = mulmod_h(p, step, q)) t.pre[n2] = make_tw(p, q);
  } else {
    t.post.resize(N1);
    const uint64_t step = powmod_h(psi_inv, N2, q);
    uint64_t p = 1;
    for (uint32_t k1 = 0; k1 < N1; ++k1, p = mulmod_h(p, step, q)) t.post[k1] = make_tw(p, q);
  }
  t.mid.resize(N);
  const uint64_t n_inv = powmod_h(N, q - 2, q);
  for (uint32_t n1 = 0; n1 < N1; ++n1) {
    const uint64_t step = powmod_h(omega, n1, q);
    uint64_t p = inverse ? n_inv : powmod_h(psi, n1, q);   // the k2 = 0 entry
    for (uint32_t k2 = 0; k2 < N2; ++k2) {
      t.mid[(size_t)k2 * N1 + n1] = make_tw(p, q);
      p = mulmod_h(p, inverse ? mulmod_h(step, psi_inv, q) : step, q);
    }
  }
  const uint64_t w2 = powmod_h(omega, N1, q), w1 = powmod_h(omega, N2, q);
  t.dft_a.resize(N2 / 2);
  uint64_t p = 1;
  for (uint32_t i = 0; i < N2 / 2; ++i, p = mulmod_h(p, w2, q)) t.dft_a[i] = make_tw(p, q);
  t.dft_b.resize(N1 / 2);
  p = 1;
  for (uint32_t i = 0; i < N1 / 2; ++i, p = mulmod_h(p, w1, q)) t.dft_b[i] = make_tw(p, q);
  return t;
}

// Host image of table sets: all tables back to back (Tw), then the NttSet
// records, which point into the device copy of the same image.
struct TableImage {
  std::vector<Tw> tw;
  struct Entry {
    size_t pre, mid, dft_a, dft_b, post;
    uint64_t q;
    Tw inv;
  };
  std::vector<Entry> entries;

  // Appends the tables of one modulus; returns its set index.
  uint32_t add(const TableSet &t, uint64_t q, Tw inv = Tw{0.0, 0.0}) {
    auto put = [&](const std::vector<Tw> &v) {
      const size_t o = tw.size();
      tw.insert(tw.end(), v.begin(), v.end());
      return v.empty() ? (size_t)-1 : o;
    };
    Entry e{put(t.pre), put(t.mid), put(t.dft_a), put(t.dft_b), put(t.post), q, inv};
    entries.push_back(e);
    return (uint32_t)entries.size() - 1;
  }

  size_t table_bytes() const { return (tw.size() * sizeof(Tw) + 255) / 256 * 256; }
  size_t bytes() const { return table_bytes() + (entries.size() * sizeof(NttSet) + 255) / 256 * 256; }

  // The NttSet records of an image placed at device address dev.
  std::vector<NttSet> sets_at(const void *dev) const {
    const Tw *tb = (const Tw *)dev;
    auto at = [&](size_t o) { return o == (size_t)-1 ? nullptr : tb + o; };
    std::vector<NttSet> sets;
    for (const Entry &e : entries)
      sets.push_back(NttSet{at(e.pre), at(e.mid), at(e.dft_a), at(e.dft_b), at(e.post), e.inv, (double)e.q,
                            1.0 / (double)e.q});
    return sets;
  }
  NttSet *sets_addr(void *dev) const { return (NttSet *)((char *)dev + table_bytes()); }

  // Copies the image to dev (bytes() long); returns the device NttSet array.
  NttSet *upload(void *dev) const {
    const std::vector<NttSet> sets = sets_at(dev);
    NttSet *dsets = sets_addr(dev);
    if (hipMemcpy(dev, tw.data(), tw.size() * sizeof(Tw), hipMemcpyHostToDevice) != hipSuccess) return nullptr;
    if (hipMemcpy(dsets, sets.data(), sets.size() * sizeof(NttSet), hipMemcpyHostToDevice) != hipSuccess)
      return nullptr;
    return dsets;
  }
};

// The regions of an image placed at dev: each table of each set on its own,
// then the NttSet array.
inline std::vector<Region> table_regions(const TableImage &img, const void *dev) {
  std::vector<Region> r;
  const uint64_t base = (uint64_t)dev;
  const size_t n = img.tw.size();
  for (size_t s = 0; s < img.entries.size(); ++s) {
    const TableImage::Entry &e = img.entries[s];
    const size_t offs[5] = {e.pre, e.mid, e.dft_a, e.dft_b, e.post};
    const char *names[5] = {"pre", "mid", "dft_a", "dft_b", "post"};
    for (int t = 0; t < 5; ++t) {
      if (offs[t] == (size_t)-1) continue;
      size_t end = n;   // the next table's start, else the end of the tables
      for (const TableImage::Entry &f : img.entries) {
        const size_t o2[5] = {f.pre, f.mid, f.dft_a, f.dft_b, f.post};
        for (size_t o : o2)
          if (o != (size_t)-1 && o > offs[t] && o < end) end = o;
      }
      r.push_back(Region{base + offs[t] * sizeof(Tw), base + end * sizeof(Tw),
                         "set " + std::to_string(s) + " " + names[t]});
    }
  }
  r.push_back(Region{base + img.table_bytes(), base + img.table_bytes() + img.entries.size() * sizeof(NttSet),
                     "NttSet records"});
  return r;
}

// The passes are instantiated per DFT side 2^4 .. 2^9.
template <uint32_t LOG>
void launch_pair(bool a, dim3 grid, size_t smem, hipStream_t stream, const NttPass &P) {
  if (a) hipLaunchKernelGGL(fiona::ntt_pass_a<LOG>, grid, dim3(fiona::kNttThreads), smem, stream, P);
  else hipLaunchKernelGGL(fiona::ntt_pass_b<LOG>, grid, dim3(fiona::kNttThreads), smem, stream, P);
}

// One pass over gridDim.y = V vectors (V <= 65535).
inline void launch_pass(bool a, uint32_t log_side, uint32_t log_other, uint32_t V, hipStream_t stream,
                        const NttPass &P) {
  if (LaunchRecord *rec = launch_recorder()) {
    rec->passes.push_back(PassLaunch{a ? PassLaunch::kPassA : PassLaunch::kPassB, log_side, log_other, V, P, {}});
    return;
  }
  const dim3 grid((1u << log_other) / fiona::kNttCols, V);
  const size_t smem = fiona::kNttCols * fiona::padded_len(1u << log_side) * sizeof(double) +
                      (1u << log_side) / 2 * sizeof(Tw);
  switch (log_side) {
    case 4: launch_pair<4>(a, grid, smem, stream, P); break;
    case 5: launch_pair<5>(a, grid, smem, stream, P); break;
    case 6: launch_pair<6>(a, grid, smem, stream, P); break;
    case 7: launch_pair<7>(a, grid, smem, stream, P); break;
    case 8: launch_pair<8>(a, grid, smem, stream, P); break;
    default: launch_pair<9>(a, grid, smem, stream, P); break;
  }
}

// Both passes of one transform.
inline void launch_transform(uint32_t log_n1, uint32_t log_n2, uint32_t V, hipStream_t stream, const NttPass &P) {
  launch_pass(true, log_n2, log_n1, V, stream, P);
  launch_pass(false, log_n1, log_n2, V, stream, P);
}

template <uint32_t LOG>
bool allow_smem_one(int bytes) {
  return hipFuncSetAttribute((const void *)fiona::ntt_pass_a<LOG>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             bytes) == hipSuccess &&
         hipFuncSetAttribute((const void *)fiona::ntt_pass_b<LOG>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             bytes) == hipSuccess;
}

// Lets every pass use the LDS of its largest side.
inline bool allow_smem() {
  const int smem = (int)(fiona::kNttCols * fiona::padded_len(fiona::kNttMaxSide) * sizeof(double) +
                         fiona::kNttMaxSide / 2 * sizeof(Tw));
  return allow_smem_one<4>(smem) && allow_smem_one<5>(smem) && allow_smem_one<6>(smem) &&
         allow_smem_one<7>(smem) && allow_smem_one<8>(smem) && allow_smem_one<9>(smem);
}

}  // namespace fiona_host
