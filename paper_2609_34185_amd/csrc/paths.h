// Decode kernel families and the host rule that picks one per tensor.
#pragma once
#include <cstdint>
#include <initializer_list>

#include "../../include/entropack.h"

namespace ep {

enum DecodePath : uint32_t {
  kPathNone = 0,    // not a decodable tensor (never chosen for a blob that passes validation)
  kPathLut = 1,     // packed slot table in LDS: one 32-bit lookup per symbol
  kPathSearch = 2,  // cumulative table in LDS, branch-free binary search per symbol
  kPathWide = 3,    // packed slot table with a 10-bit coordinate field (wider ranges)
  kPathGlobal = 4,  // frequencies read from the blob in global memory, coarse cumulative index in LDS
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

// Global-table path (tables too large for the LDS paths; App. C.3 places the decode
// tables in shared or packed global memory by alphabet size).  The blob's own u16
// frequency arrays are read from global memory; LDS holds every G-th cumulative
// value of each table (G = 2^g), u16, n_t = ceil(A_t / G) entries per table, then
// u32 metadata for t < 16: the first coarse entry of the table, its min, n_t and
// the byte offset of its frequencies in the blob.  A symbol is found by a binary
// search over the coarse entries and a scan of at most G frequencies.
constexpr uint32_t kGlobalBitsMin = 3;
constexpr uint32_t kGlobalBitsMax = 6;

struct GlobalLayout {
  uint32_t g_bits;        // log2 G (0 when nothing fits)
  uint32_t meta, total;   // byte offset of the metadata; bytes in all (512-byte aligned)
};

inline GlobalLayout global_layout(const uint32_t* A) {
  for (uint32_t g = kGlobalBitsMin; g <= kGlobalBitsMax; g++) {
    uint64_t n = 0;
    for (int t = 0; t < 16; t++) n += (A[t] + (1u << g) - 1) >> g;
    const uint64_t meta = (2 * n + 3) & ~3ull;
    const uint64_t total = (meta + 4 * 64 + 511) & ~511ull;
    if (total <= kSearchLdsBytes) return GlobalLayout{g, (uint32_t)meta, (uint32_t)total};
  }
  return GlobalLayout{0, 0, 0};
}

// Whether path P can hold the tables of tensor I.
inline bool path_fits(uint32_t P, const ep_tensor_info& I) {
  switch (P) {
    case kPathLut:
      return I.prob_bits <= kLutMaxBits && I.coord2_min >= kLutValueMin && I.coord2_max <= kLutValueMax;
    case kPathWide:
      return I.prob_bits <= kLutMaxBits && I.coord2_min >= kWideValueMin && I.coord2_max <= kWideValueMax;
    case kPathSearch:
      return I.sum_alphabet <= 0xFFFF0u && search_layout(I.prob_bits, I.sum_alphabet).bucket_bits != 0;
    case kPathGlobal:
      return I.prob_bits >= 9 && I.prob_bits <= 15 && global_layout(I.table_A).g_bits != 0;
    default:
      return false;
  }
}

// The fastest path that holds the tables.  Every blob that passes validation (A <= 2^b
// <= 2^15 per table) fits the global-table path: 16 tables of at most 2^15 symbols
// need 2^16 coarse entries at G = 8 (128 KiB) or half that at G = 16.
inline uint32_t choose_path(const ep_tensor_info& I) {
  for (uint32_t P : {kPathLut, kPathWide, kPathSearch, kPathGlobal})
    if (path_fits(P, I)) return P;
  return kPathNone;
}

}  // namespace ep
