// Decode kernel families and the host rule that picks one per tensor.
#pragma once
#include <cstdint>

#include "../../include/entropack.h"

namespace ep {

enum DecodePath : uint32_t {
  kPathNone = 0,    // no kernel family in this build can hold the tables
  kPathLut = 1,     // packed slot table in LDS: one 32-bit lookup per symbol
  kPathSearch = 2,  // cumulative table in LDS, branch-free binary search per symbol
  kPathWide = 3,    // packed slot table with a 10-bit coordinate field (wider ranges)
};

// LDS bytes of the packed slot table (16 tables x 2^b slots x 4 B) and of the
// cumulative scratch it is built from.
constexpr uint32_t kLutMaxBits = 11;
constexpr int32_t kLutValueMin = -256;   // doubled coordinates whose integer part fits a signed byte
constexpr int32_t kLutValueMax = 255;
constexpr int32_t kWideValueMin = -1024; // ... a signed 10-bit field (wide entries)
constexpr int32_t kWideValueMax = 1023;
constexpr uint32_t kSearchLdsBytes = 128 * 1024;   // the payload rings take the other 32 KiB

// Search path: u16 cumulative tables plus, per table, 2^k + 1 u16 bucket
// bounds (bucket j starts at slot j * 2^(b-k)); k is the largest of
// min(b, 11) .. 8 whose tables fit, so that for b <= 11 and moderate table
// sizes every bucket is a single slot and no search remains.
constexpr uint32_t kBucketBitsMin = 8;
constexpr uint32_t kBucketBitsMax = 11;

struct SearchLayout {
  uint32_t bucket_bits;           // k (0 when no k fits)
  uint32_t bucket, meta, total;   // byte offsets of the buckets and metadata; bytes in all
};

constexpr SearchLayout search_layout_k(uint32_t sum_A, uint32_t k) {
  // u16 cumulative values: sum_A + one end value per table, padded to 4 bytes
  const uint32_t cum = (2 * (sum_A + 16) + 3) & ~3u;
  const uint32_t bucket = cum;
  const uint32_t meta = (bucket + 2 * 16 * ((1u << k) + 1) + 3) & ~3u;
  // the payload rings that follow are addressed as base | offset: 512-byte aligned
  const uint32_t total = (meta + 4 * 32 + 511) & ~511u;
  return SearchLayout{k, bucket, meta, total};
}

constexpr SearchLayout search_layout(uint32_t b, uint32_t sum_A) {
  for (uint32_t k = (b < kBucketBitsMax ? b : kBucketBitsMax); k >= kBucketBitsMin; k--) {
    const SearchLayout S = search_layout_k(sum_A, k);
    if (S.total <= kSearchLdsBytes) return S;
  }
  return SearchLayout{0, 0, 0, 0};
}

inline uint32_t choose_path(const ep_tensor_info& I) {
  if (I.prob_bits <= kLutMaxBits && I.coord2_min >= kLutValueMin && I.coord2_max <= kLutValueMax)
    return kPathLut;
  if (I.prob_bits <= kLutMaxBits && I.coord2_min >= kWideValueMin && I.coord2_max <= kWideValueMax)
    return kPathWide;
  if (I.sum_alphabet <= 0xFFFF0u && search_layout(I.prob_bits, I.sum_alphabet).bucket_bits)
    return kPathSearch;
  return kPathNone;
}

}  // namespace ep
