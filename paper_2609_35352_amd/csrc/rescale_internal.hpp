// The rescale's vector-level entry, shared by the rescale epilogue and the
// rotation producer's division by the special prime (host only).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fiona.h"

// V polynomials of L limbs (in: vector v at in + v L N) divided by q_{L-1}
// with rounding, L - 1 limbs out (vector v at out + v (L - 1) N); with add,
// the first add_count vectors get add (L - 1 limbs, the same for all of
// them) added after the division; transposed stores every limb as k2 N1 + k1
// instead of k2 + N2 k1 (the four-step index k = k2 + N2 k1).  Arguments are
// the caller's to check (V <= 2 max_ct).  Returns FIONA_OK or FIONA_ERR_HIP.
int fiona_rescale_vectors(const fiona_rescaler *R, const uint64_t *in, uint32_t V, uint64_t *out,
                          const uint64_t *add, uint32_t add_count, bool transposed, hipStream_t stream);
