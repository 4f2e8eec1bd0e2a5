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

}  // namespace fiona

extern "C" {

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
