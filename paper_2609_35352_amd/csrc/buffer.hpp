// Buffer descriptors of the kernels' global accesses.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fiona {

// The 64-bit address whose halves are hi and lo.  Both are taken as
// unsigned 32-bit values: widening a signed low half would copy its bit 31
// into the whole high half (an address far outside the GPU's address space).
__host__ __device__ constexpr uint64_t join_halves(uint32_t hi, uint32_t lo) { return ((uint64_t)hi << 32) | lo; }

// num_records of a buffer descriptor at byte address base for a buffer that
// ends at byte address end (end >= base): the bytes left, at most 2^32 - 1.
// An access at or past it reads zero and a store there is dropped, instead
// of reaching memory outside the buffer.
__host__ __device__ constexpr uint32_t buffer_extent(uint64_t base, uint64_t end) {
  return end - base > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)(end - base);
}

// A raw buffer descriptor (stride 0) over [base, end).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *base, const void *end) {
  return __builtin_amdgcn_make_buffer_rsrc((void *)base, (short)0, (int)buffer_extent((uint64_t)base, (uint64_t)end),
                                           0x00020000);
}

}  // namespace fiona
