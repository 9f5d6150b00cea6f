// Host-side blob validation (ep_blob_info) and error reporting of libentropack.so.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <string>

#include "../../include/entropack.h"
#include "common.h"
#include "paths.h"

namespace ep {

namespace {
thread_local std::string g_err;
}

int fail(int code, const char* msg) {
  g_err = msg ? msg : "";
  return code;
}

namespace {

uint32_t rd32(const uint8_t* p) {
  uint32_t v;
  std::memcpy(&v, p, 4);
  return v;
}

}  // namespace

int blob_info(const void* host_blob, uint64_t n, ep_tensor_info* info) {
  if (!host_blob || !info) return fail(EP_ERR_ARG, "ep_blob_info: null argument");
  std::memset(info, 0, sizeof(*info));
  const uint8_t* b = static_cast<const uint8_t*>(host_blob);
  if (n < kHeaderBytes) return fail(EP_ERR_FORMAT, "ep_blob_info: shorter than the header");
  if (rd32(b) != kMagic) return fail(EP_ERR_FORMAT, "ep_blob_info: bad magic");
  if (rd32(b + 4) != kVersion) return fail(EP_ERR_FORMAT, "ep_blob_info: unsupported version");
  ep_tensor_info I;
  std::memset(&I, 0, sizeof I);
  I.rows = rd32(b + 8);
  I.cols = rd32(b + 12);
  I.prob_bits = rd32(b + 16);
  I.tile_vectors = rd32(b + 20);
  I.n_tiles = rd32(b + 24);
  I.container = rd32(b + 28);
  I.table_bytes = rd32(b + 32);
  I.payload_words = rd32(b + 36);
  std::memcpy(&I.total_bytes, b + 40, 8);
  if (I.total_bytes != n) return fail(EP_ERR_FORMAT, "ep_blob_info: size field differs from blob size");
  if (!I.rows || !I.cols || I.cols % 8) return fail(EP_ERR_FORMAT, "ep_blob_info: bad shape");
  if (I.prob_bits < 9 || I.prob_bits > 15) return fail(EP_ERR_FORMAT, "ep_blob_info: b outside 9..15");
  if (!I.tile_vectors || I.container > 4) return fail(EP_ERR_FORMAT, "ep_blob_info: bad tile size or container");
  const uint64_t nvec = (uint64_t)I.rows * I.cols / 8;
  if (nvec > 0xFFFFFFFFull) return fail(EP_ERR_FORMAT, "ep_blob_info: tensor too large");
  if ((uint64_t)I.n_tiles != (nvec + I.tile_vectors - 1) / I.tile_vectors)
    return fail(EP_ERR_FORMAT, "ep_blob_info: tile count does not match the shape");
  Layout L = layout_of(I.rows, I.table_bytes, I.n_tiles, I.container, I.payload_words);
  if (L.total != n) return fail(EP_ERR_FORMAT, "ep_blob_info: section sizes do not add up");
  I.off_tables = L.off_tables;
  I.off_sigma = L.off_sigma;
  I.off_delta = I.container ? L.off_delta : 0;
  I.off_states = L.off_states;
  I.off_offsets = L.off_offsets;
  I.off_payload = L.off_payload;

  // tables
  const uint32_t M = 1u << I.prob_bits;
  const uint8_t* p = b + L.off_tables;
  const uint8_t* end = b + L.off_sigma;
  if (p + 4 > end) return fail(EP_ERR_FORMAT, "ep_blob_info: truncated coset table");
  uint16_t cf[2];
  std::memcpy(cf, p, 4);
  if ((uint32_t)cf[0] + cf[1] != M) return fail(EP_ERR_FORMAT, "ep_blob_info: coset frequencies do not sum to 2^b");
  p += 4;
  int64_t lo2 = INT64_MAX, hi2 = INT64_MIN;
  uint32_t amax = 0, asum = 0;
  I.coset_f0 = cf[0];
  I.coset_f1 = cf[1];
  for (int c = 0; c < 2; c++) {
    for (int i = 1; i <= 8; i++) {
      if (p + 8 > end) return fail(EP_ERR_FORMAT, "ep_blob_info: truncated field table");
      int32_t mn = (int32_t)rd32(p);
      uint32_t A = rd32(p + 4);
      const int ti = 8 * c + (i - 1);
      I.table_off[ti] = (uint32_t)(p + 8 - b);
      I.table_min[ti] = mn;
      I.table_A[ti] = A;
      asum += A;
      uint64_t sz = 8 + ((2ull * A + 3) / 4) * 4;
      if (A > M || p + sz > end) return fail(EP_ERR_FORMAT, "ep_blob_info: field table larger than 2^b or truncated");
      if (!A && cf[c]) return fail(EP_ERR_FORMAT, "ep_blob_info: empty table of a used coset");
      uint64_t sum = 0;
      for (uint32_t z = 0; z < A; z++) {
        uint16_t f;
        std::memcpy(&f, p + 8 + 2 * z, 2);
        sum += f;
      }
      if (A && sum != M) return fail(EP_ERR_FORMAT, "ep_blob_info: field frequencies do not sum to 2^b");
      if (A && cf[c]) {
        int64_t vmin = mn, vmax = (int64_t)mn + A - 1;
        if (vmin < -(1 << 27) || vmax > (1 << 27))
          return fail(EP_ERR_FORMAT, "ep_blob_info: coordinate value out of range");
        int64_t a2, b2;
        if (i <= 7) {
          a2 = 2 * vmin + c;
          b2 = 2 * vmax + c;
        } else {
          a2 = 4 * vmin + c;
          b2 = 4 * vmax + 2 + c;
        }
        lo2 = std::min(lo2, a2);
        hi2 = std::max(hi2, b2);
        amax = std::max(amax, A);
      }
      p += sz;
    }
  }
  if (p != end) return fail(EP_ERR_FORMAT, "ep_blob_info: table section size mismatch");
  I.max_alphabet = amax;
  I.sum_alphabet = asum;
  I.coord2_min = (int32_t)lo2;
  I.coord2_max = (int32_t)hi2;

  // scales
  const float* sg = reinterpret_cast<const float*>(b + L.off_sigma);
  double smax = 0;
  for (uint32_t r = 0; r < I.rows; r++) {
    float v;
    std::memcpy(&v, sg + r, 4);
    if (!std::isfinite(v)) return fail(EP_ERR_FORMAT, "ep_blob_info: non-finite row scale");
    smax = std::max(smax, (double)std::fabs(v));
  }
  if (I.container) {
    const float* dl = reinterpret_cast<const float*>(b + L.off_delta);
    for (uint32_t r = 0; r < I.rows; r++) {
      float v;
      std::memcpy(&v, dl + r, 4);
      if (!std::isfinite(v)) return fail(EP_ERR_FORMAT, "ep_blob_info: non-finite dequant scale");
    }
  }
  double pmax = std::max(std::fabs((double)lo2), std::fabs((double)hi2)) / 2.0;
  double bound = smax * pmax * (1.0 + 1.0 / 8388608.0);
  I.max_abs_weight = bound > 3.0e38 ? 3.0e38f : (float)bound;

  // offsets
  const uint32_t* off = reinterpret_cast<const uint32_t*>(b + L.off_offsets);
  uint32_t prev = 0;
  for (uint32_t t = 0; t <= I.n_tiles; t++) {
    uint32_t o;
    std::memcpy(&o, off + t, 4);
    if ((t == 0 && o != 0) || o < prev) return fail(EP_ERR_FORMAT, "ep_blob_info: payload offsets not monotone from 0");
    prev = o;
  }
  if (prev != I.payload_words) return fail(EP_ERR_FORMAT, "ep_blob_info: last offset differs from the payload size");
  I.path = choose_path(I);
  *info = I;
  return EP_OK;
}

}  // namespace ep

extern "C" {

int ep_blob_info(const void* host_blob, uint64_t n, ep_tensor_info* info) {
  return ep::blob_info(host_blob, n, info);
}

const char* ep_last_error(void) { return ep::g_err.c_str(); }

}  // extern "C"
