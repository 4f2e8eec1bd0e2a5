// The RNS context shared by the library's translation units (host only).
#pragma once
#include <stdint.h>

#include <vector>

#include "modarith.hpp"

struct fiona_ctx {
  uint32_t N = 0, L = 0;
  std::vector<uint64_t> q;
  std::vector<fiona::LimbConst> limbs;
};
