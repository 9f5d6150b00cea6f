// Internal declarations shared by the host sources of libentropack.so.
#pragma once
#include <cstdint>

namespace ep {

constexpr uint32_t kMagic = 0x314B5045u;   // "EPK1"
constexpr uint32_t kVersion = 1;
constexpr uint32_t kHeaderBytes = 48;

// Section offsets of a blob (byte layout in include/entropack.h).
struct Layout {
  uint64_t off_tables, off_sigma, off_delta, off_states, off_offsets, off_payload, total;
};

inline Layout layout_of(uint32_t rows, uint32_t table_bytes, uint32_t n_tiles, uint32_t container,
                        uint32_t payload_words) {
  Layout L;
  L.off_tables = kHeaderBytes;
  L.off_sigma = L.off_tables + table_bytes;
  L.off_delta = L.off_sigma + 4ull * rows;
  L.off_states = L.off_delta + (container ? 4ull * rows : 0ull);
  L.off_offsets = L.off_states + 128ull * n_tiles;
  L.off_payload = L.off_offsets + 4ull * (n_tiles + 1ull);
  L.total = L.off_payload + ((2ull * payload_words + 3) / 4) * 4;
  return L;
}

// Records a thread-local message for ep_last_error and returns code.
int fail(int code, const char* msg);

}  // namespace ep
