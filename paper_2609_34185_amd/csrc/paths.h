// Decode kernel families and the host rule that picks one per tensor.
#pragma once
#include <cstdint>

#include "../../include/entropack.h"

namespace ep {

enum DecodePath : uint32_t {
  kPathNone = 0,    // no kernel family in this build can hold the tables
  kPathLut = 1,     // packed slot table in LDS: one 32-bit lookup per symbol
  kPathSearch = 2,  // cumulative table in LDS, branch-free binary search per symbol
};

// LDS bytes of the packed slot table (16 tables x 2^b slots x 4 B) and of the
// cumulative scratch it is built from.
constexpr uint32_t kLutMaxBits = 11;
constexpr int32_t kLutValueMin = -256;   // packed doubled coordinate: signed 9 bits
constexpr int32_t kLutValueMax = 255;
constexpr uint32_t kSearchLdsBytes = 128 * 1024;   // the payload rings take the other 32 KiB

inline uint32_t choose_path(const ep_tensor_info& I) {
  if (I.prob_bits <= kLutMaxBits && I.coord2_min >= kLutValueMin && I.coord2_max <= kLutValueMax)
    return kPathLut;
  if (4ull * (I.sum_alphabet + 48) + 16 <= kSearchLdsBytes) return kPathSearch;
  return kPathNone;
}

}  // namespace ep
