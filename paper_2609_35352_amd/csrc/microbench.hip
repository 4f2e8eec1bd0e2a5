// Register-only rate of the raw route's arithmetic, for comparing the hybrid
// kernel's multiply-add rate with what the VALU sustains when nothing else
// runs (a measurement helper; the weighted sum does not call it).
//
// Per plaintext word the kernel does what hybrid_linear_kernel does for one
// raw term at one position: the exact multiply-add of the word into both
// polynomials' accumulators (modarith.hpp mac: four 32x32->64 multiply-adds
// each) and a carry step every kChunkTerms words.  The words and digits live
// in registers; an empty asm statement after every block of eight words makes
// the compiler treat the words as new values, so that no product is folded
// or hoisted.  No memory is read; one word per thread is written at the end.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "fiona.h"
#include "modarith.hpp"

namespace fiona {

constexpr uint32_t kMicroThreads = 256;

__global__ void __launch_bounds__(kMicroThreads) mac_microbench_kernel(uint32_t chunks, uint64_t *sink) {
  const uint32_t t = blockIdx.x * kMicroThreads + threadIdx.x;
  const uint32_t x0 = (t * 2654435761u) & kDigitMask, x1 = (t * 40503u + 7u) & kDigitMask;
  const uint32_t y0 = (t * 97u + 3u) & kDigitMask, y1 = (t * 2246822519u) & kDigitMask;
  uint32_t wl[8], wh[8];
#pragma unroll
  for (uint32_t k = 0; k < 8; ++k) {
    wl[k] = t * 0x9E3779B9u + k * 0x85EBCA6Bu;
    wh[k] = (t + 977u * k) & 0x3FFFFu;
  }
  Acc a0, a1;
  acc_zero(a0);
  acc_zero(a1);
  for (uint32_t c = 0; c < chunks; ++c) {
#pragma unroll
    for (uint32_t k = 0; k < kChunkTerms; ++k) {
      mac(a0, x0, x1, wl[k & 7], wh[k & 7]);
      mac(a1, y0, y1, wl[k & 7], wh[k & 7]);
      if ((k & 7) == 7) {
        asm volatile("" : "+v"(wl[0]), "+v"(wl[1]), "+v"(wl[2]), "+v"(wl[3]), "+v"(wl[4]), "+v"(wl[5]),
                     "+v"(wl[6]), "+v"(wl[7]));
        asm volatile("" : "+v"(wh[0]), "+v"(wh[1]), "+v"(wh[2]), "+v"(wh[3]), "+v"(wh[4]), "+v"(wh[5]),
                     "+v"(wh[6]), "+v"(wh[7]));
      }
    }
    carry(a0);
    carry(a1);
  }
  sink[t] = a0.A0 ^ a0.A1 ^ a0.A2 ^ a0.A3 ^ a1.A0 ^ a1.A1 ^ a1.A2 ^ a1.A3;
}

typedef uint32_t sv4 __attribute__((ext_vector_type(4)));

// Stream probes: the HBM bandwidth a plain contiguous read and a plain copy
// reach, as ceilings to set the kernels' rates against.  Grid-stride over
// 16-byte words, four loads in flight per thread, nontemporal loads and
// stores (each word is touched once).  The read probe folds what it reads
// into one word per workgroup, so that no load can be dropped.
__global__ void __launch_bounds__(kMicroThreads) stream_read_kernel(const sv4 *__restrict__ src, uint64_t n16,
                                                                    uint64_t *__restrict__ sink) {
  const uint64_t step = (uint64_t)gridDim.x * kMicroThreads * 4;
  uint32_t acc = 0;
  for (uint64_t i = (uint64_t)blockIdx.x * kMicroThreads * 4 + threadIdx.x; i < n16; i += step) {
    sv4 v[4];
#pragma unroll
    for (uint32_t u = 0; u < 4; ++u) {
      const uint64_t j = i + u * kMicroThreads;
      v[u] = j < n16 ? __builtin_nontemporal_load(src + j) : (sv4){0, 0, 0, 0};
    }
#pragma unroll
    for (uint32_t u = 0; u < 4; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  __shared__ uint32_t red[kMicroThreads];
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t a = 0;
    for (uint32_t t = 0; t < kMicroThreads; ++t) a ^= red[t];
    sink[blockIdx.x] = a;
  }
}

__global__ void __launch_bounds__(kMicroThreads) stream_copy_kernel(const sv4 *__restrict__ src,
                                                                    sv4 *__restrict__ dst, uint64_t n16) {
  const uint64_t step = (uint64_t)gridDim.x * kMicroThreads * 4;
  for (uint64_t i = (uint64_t)blockIdx.x * kMicroThreads * 4 + threadIdx.x; i < n16; i += step) {
    sv4 v[4];
#pragma unroll
    for (uint32_t u = 0; u < 4; ++u) {
      const uint64_t j = i + u * kMicroThreads;
      v[u] = j < n16 ? __builtin_nontemporal_load(src + j) : (sv4){0, 0, 0, 0};
    }
#pragma unroll
    for (uint32_t u = 0; u < 4; ++u) {
      const uint64_t j = i + u * kMicroThreads;
      if (j < n16) __builtin_nontemporal_store(v[u], dst + j);
    }
  }
}

// Every 16-byte slot of dst gets (seed, seed + slot, ...): a write-only stream.
__global__ void __launch_bounds__(kMicroThreads) stream_write_kernel(sv4 *__restrict__ dst, uint64_t n16,
                                                                     uint32_t seed) {
  const uint64_t step = (uint64_t)gridDim.x * kMicroThreads * 4;
  for (uint64_t i = (uint64_t)blockIdx.x * kMicroThreads * 4 + threadIdx.x; i < n16; i += step) {
#pragma unroll
    for (uint32_t u = 0; u < 4; ++u) {
      const uint64_t j = i + u * kMicroThreads;
      if (j < n16) __builtin_nontemporal_store((sv4){seed, (uint32_t)j, (uint32_t)(j >> 32), seed ^ u}, dst + j);
    }
  }
}

}  // namespace fiona

extern "C" {

int fiona_stream_read(const uint64_t *src, uint64_t words, uint32_t blocks, uint64_t *sink, hipStream_t stream) {
  if (!src || !sink || blocks == 0 || words == 0 || (words & 1u)) return FIONA_ERR_ARG;
  if ((uintptr_t)src & 15u) return FIONA_ERR_ALIGN;
  hipLaunchKernelGGL(fiona::stream_read_kernel, dim3(blocks), dim3(fiona::kMicroThreads), 0, stream,
                     (const fiona::sv4 *)src, words / 2, sink);
  return hipGetLastError() == hipSuccess ? FIONA_OK : FIONA_ERR_HIP;
}

int fiona_stream_copy(const uint64_t *src, uint64_t *dst, uint64_t words, uint32_t blocks, hipStream_t stream) {
  if (!src || !dst || blocks == 0 || words == 0 || (words & 1u)) return FIONA_ERR_ARG;
  if (((uintptr_t)src | (uintptr_t)dst) & 15u) return FIONA_ERR_ALIGN;
  const uintptr_t a = (uintptr_t)src, b = (uintptr_t)dst;
  if (a < b + words * 8 && b < a + words * 8) return FIONA_ERR_ALIAS;
  hipLaunchKernelGGL(fiona::stream_copy_kernel, dim3(blocks), dim3(fiona::kMicroThreads), 0, stream,
                     (const fiona::sv4 *)src, (fiona::sv4 *)dst, words / 2);
  return hipGetLastError() == hipSuccess ? FIONA_OK : FIONA_ERR_HIP;
}

int fiona_stream_write(uint64_t *dst, uint64_t words, uint32_t blocks, hipStream_t stream) {
  if (!dst || blocks == 0 || words == 0 || (words & 1u)) return FIONA_ERR_ARG;
  if ((uintptr_t)dst & 15u) return FIONA_ERR_ALIGN;
  hipLaunchKernelGGL(fiona::stream_write_kernel, dim3(blocks), dim3(fiona::kMicroThreads), 0, stream,
                     (fiona::sv4 *)dst, words / 2, 0x9E3779B9u);
  return hipGetLastError() == hipSuccess ? FIONA_OK : FIONA_ERR_HIP;
}

uint64_t fiona_mac_microbench_words(uint32_t blocks, uint32_t chunks) {
  return (uint64_t)blocks * fiona::kMicroThreads * chunks * fiona::kChunkTerms;
}

int fiona_mac_microbench(uint32_t blocks, uint32_t chunks, uint64_t *sink, hipStream_t stream) {
  if (blocks == 0 || chunks == 0 || sink == nullptr) return FIONA_ERR_ARG;
  hipLaunchKernelGGL(fiona::mac_microbench_kernel, dim3(blocks), dim3(fiona::kMicroThreads), 0, stream, chunks,
                     sink);
  return hipGetLastError() == hipSuccess ? FIONA_OK : FIONA_ERR_HIP;
}

}  // extern "C"
