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

// Search path: 2^8 buckets per table (257 bounds), u16 cumulative tables.
constexpr uint32_t kBucketBits = 8;
constexpr uint32_t kBuckets1 = (1u << kBucketBits) + 1;

struct SearchLayout {
  uint32_t bucket, meta, total;   // byte offsets of the buckets and metadata; bytes in all
};

constexpr SearchLayout search_layout(uint32_t sum_A) {
  // u16 cumulative values: sum_A + one end value per table, padded to 4 bytes
  const uint32_t cum = (2 * (sum_A + 16) + 3) & ~3u;
  const uint32_t bucket = cum;
  const uint32_t meta = (bucket + 2 * 16 * kBuckets1 + 3) & ~3u;
  const uint32_t total = (meta + 4 * 32 + 15) & ~15u;
  return SearchLayout{bucket, meta, total};
}

constexpr uint32_t search_table_bytes(uint32_t sum_A) {
  return search_layout(sum_A).total;
}

inline uint32_t choose_path(const ep_tensor_info& I) {
  if (I.prob_bits <= kLutMaxBits && I.coord2_min >= kLutValueMin && I.coord2_max <= kLutValueMax)
    return kPathLut;
  if (I.sum_alphabet <= 0xFFFF0u && search_table_bytes(I.sum_alphabet) <= kSearchLdsBytes)
    return kPathSearch;
  return kPathNone;
}

}  // namespace ep
