// Device-side generator of the synthetic inputs (the same counter-based
// definition as the NumPy generator in synth/__init__.py):
//   mix64  = SplitMix64 output function (Steele, Lea, Flood, OOPSLA 2014)
//   key    = mix64(mix64(seed) + tag * GOLDEN)
//   u(idx) = mix64(key + (idx + 1) * GOLDEN)
//   residue uniform in [0, q) = floor(u * q / 2^64)
// It fills ciphertext and plaintext tables in HBM so that large layers need
// no host-to-device copies.  It contains none of the weighted-sum arithmetic.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;
constexpr uint32_t kMaxL = 64;

struct Moduli {
  uint64_t q[kMaxL];
};

__host__ __device__ inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

uint64_t stream_key(uint64_t seed, uint64_t tag) { return mix64(mix64(seed) + tag * kGolden); }

// One workgroup per row of N coefficients; row r covers limb r % L.
__global__ void __launch_bounds__(256) fill_rows_kernel(uint64_t *dst, uint32_t rows, uint32_t L, uint32_t N,
                                                        uint64_t key, Moduli m) {
  const uint32_t r = blockIdx.x;
  if (r >= rows) return;
  const uint64_t q = m.q[r % L];
  const uint64_t base = (uint64_t)r * N;
  for (uint32_t k = threadIdx.x; k < N; k += blockDim.x) {
    const uint64_t idx = base + k;
    dst[idx] = __umul64hi(mix64(key + (idx + 1) * kGolden), q);
  }
}

// Plaintext rows: row r = local plaintext p * L + limb.  A uniform plaintext
// takes stream positions of its global id; a constant plaintext (pt_const >= 0,
// sign code in bits 32..33, scale in bits 0..31) holds h*c mod q everywhere.
__global__ void __launch_bounds__(256) fill_pts_kernel(uint64_t *dst, uint32_t n_pt, uint32_t L, uint32_t N,
                                                       uint64_t pitch, const uint64_t *pt_global,
                                                       const int64_t *pt_const, uint64_t key, Moduli m) {
  const uint32_t r = blockIdx.x;
  const uint32_t p = r / L, l = r - p * L;
  if (p >= n_pt) return;
  const uint64_t q = m.q[l];
  uint64_t *row = dst + (uint64_t)p * pitch + (uint64_t)l * N;
  const int64_t c = pt_const ? pt_const[p] : -1;
  if (c >= 0) {
    const uint64_t code = (uint64_t)c >> 32, s = (uint64_t)c & 0xFFFFFFFFull;
    const uint64_t sm = s % q;
    const uint64_t v = code == 1 ? sm : (code == 2 ? (sm ? q - sm : 0) : 0);
    for (uint32_t k = threadIdx.x; k < N; k += blockDim.x) row[k] = v;
    return;
  }
  const uint64_t base = (pt_global[p] * L + l) * (uint64_t)N;
  for (uint32_t k = threadIdx.x; k < N; k += blockDim.x) {
    const uint64_t idx = base + k;
    row[k] = __umul64hi(mix64(key + (idx + 1) * kGolden), q);
  }
}

int make_moduli(const uint64_t *moduli, uint32_t L, Moduli *m) {
  if (!moduli || L == 0 || L > kMaxL) return -1;
  for (uint32_t l = 0; l < kMaxL; ++l) m->q[l] = l < L ? moduli[l] : 1;
  return 0;
}

}  // namespace

extern "C" {

// dst: device [n_rows][N] with row r in limb r % L (a ciphertext array has
// n_rows = n_ct * 2 * L); element (r, k) takes stream index r * N + k.
int synth_fill_uniform(uint64_t *dst, uint32_t n_rows, uint32_t L, uint32_t N, uint64_t seed, uint64_t tag,
                       const uint64_t *moduli_host, hipStream_t stream) {
  Moduli m;
  if (!dst || N == 0 || make_moduli(moduli_host, L, &m) != 0) return -1;
  if (n_rows == 0) return 0;
  hipLaunchKernelGGL(fill_rows_kernel, dim3(n_rows), dim3(256), 0, stream, dst, n_rows, L, N,
                     stream_key(seed, tag), m);
  return hipGetLastError() == hipSuccess ? 0 : -2;
}

// dst: device, n_pt plaintexts of [L][N], plaintext p at word p * pitch
// (pitch >= L * N; the words between rows are left as they are);
// pt_global: device [n_pt]; pt_const: device [n_pt] or null.
int synth_fill_pts(uint64_t *dst, uint32_t n_pt, uint32_t L, uint32_t N, uint64_t pitch, const uint64_t *pt_global,
                   const int64_t *pt_const, uint64_t seed, uint64_t tag, const uint64_t *moduli_host,
                   hipStream_t stream) {
  Moduli m;
  if (!dst || !pt_global || N == 0 || make_moduli(moduli_host, L, &m) != 0) return -1;
  if (pitch < (uint64_t)L * N) return -1;
  if (n_pt == 0) return 0;
  const uint64_t rows = (uint64_t)n_pt * L;
  if (rows >= (1ull << 31)) return -1;
  hipLaunchKernelGGL(fill_pts_kernel, dim3((uint32_t)rows), dim3(256), 0, stream, dst, n_pt, L, N, pitch,
                     pt_global, pt_const, stream_key(seed, tag), m);
  return hipGetLastError() == hipSuccess ? 0 : -2;
}

}  // extern "C"
