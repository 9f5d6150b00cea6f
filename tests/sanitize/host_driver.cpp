// Host-code driver for the AddressSanitizer / UndefinedBehaviorSanitizer run of
// the CPU test suite: the oracle (oracle/oracle.c) and the library's host
// sources (encoder, blob validation) are built with the sanitizers and
// exercised on small tensors, then on a loop of malformed blobs.  Both sides
// must agree byte for byte on every encode, and neither may fault, read out
// of bounds or hit undefined behaviour on any input.  Test code only.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <cmath>
#include <vector>

#include "../../include/entropack.h"

extern "C" {
struct ora_params {
  double target_bpp;
  int32_t tile_vectors, prob_bits, search_steps, container;
  double scale_lo, scale_hi;
  int64_t sample_vectors;
  double state_credit_bits;
  int32_t rdo_candidates, rdo_sweeps;
};
int ora_encode(const void* w, int dtype, int64_t R, int64_t C, const ora_params* prm,
               uint8_t** out_blob, uint64_t* out_size, double* stats);
void ora_blob_free(uint8_t* blob);
int ora_decode(const uint8_t* blob, uint64_t n, int out_dtype, void* out, float* dequant,
               uint32_t t0, uint32_t t1);
}

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint64_t next_u64() {   // SplitMix64
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
double uniform() { return ((next_u64() >> 11) + 0.5) * (1.0 / 9007199254740992.0); }
double gauss() { return std::sqrt(-2.0 * std::log(uniform())) * std::cos(6.283185307179586 * uniform()); }

uint16_t to_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

std::vector<uint16_t> tensor(int64_t R, int64_t C, double scale, double outlier_rate) {
  std::vector<uint16_t> w((size_t)(R * C));
  for (int64_t r = 0; r < R; r++) {
    const double s = scale * std::exp(0.4 * gauss());
    for (int64_t c = 0; c < C; c++) {
      double v = s * gauss();
      if (uniform() < outlier_rate) v *= 8.0;
      w[(size_t)(r * C + c)] = to_bf16((float)v);
    }
  }
  return w;
}

int failures = 0;
void check(bool ok, const char* what) {
  if (!ok) {
    std::fprintf(stderr, "FAIL: %s\n", what);
    failures++;
  }
}

struct Case {
  int64_t R, C;
  double target;
  int V, b, container, rdo_k, rdo_t;
  double credit;
};

}  // namespace

int main(int argc, char** argv) {
  const int mutations = argc > 1 ? std::atoi(argv[1]) : 3000;
  const Case cases[] = {
      {64, 512, 4.0, 512, 12, 0, 0, 0, 8.0},   {37, 136, 3.3, 45, 0, 0, 0, 0, 8.0},
      {300, 8, 4.0, 33, 0, 0, 0, 0, 8.0},      {128, 512, 4.0, 512, 0, 1, 0, 0, 8.0},
      {128, 512, 6.0, 512, 0, 2, 0, 0, 8.0},   {96, 512, 4.0, 64, 0, 3, 0, 0, 8.0},
      {80, 520, 4.0, 512, 0, 4, 0, 0, 8.0},    {64, 1024, 9.0, 512, 0, 0, 0, 0, 8.0},
      {64, 256, 2.0, 512, 9, 0, 0, 0, 8.0},    {96, 512, 3.0, 512, 0, 0, 0, 0, 16.0},
      {96, 512, 3.0, 128, 0, 0, 5, 1, 8.0},    {77, 136, 6.0, 45, 0, 2, 4, 3, 8.0},
      {1, 8, 4.0, 1, 0, 0, 0, 0, 8.0},         {32, 64, 14.0, 7, 0, 0, 0, 0, 8.0},
  };
  std::vector<uint8_t> keep;   // one valid blob for the mutation loop
  for (const Case& k : cases) {
    std::vector<uint16_t> w = tensor(k.R, k.C, 0.02, k.container ? 5e-4 : 1e-3);
    ora_params op{k.target, k.V, k.b, 12, k.container, 1e-3, 8.0, 1 << 18, k.credit, k.rdo_k, k.rdo_t};
    uint8_t* ob = nullptr;
    uint64_t on = 0;
    check(ora_encode(w.data(), EP_BF16, k.R, k.C, &op, &ob, &on, nullptr) == 0, "oracle encode");
    ep_encode_params pp;
    ep_encode_params_default(&pp);
    pp.target_bpp = k.target;
    pp.tile_vectors = k.V;
    pp.prob_bits = k.b;
    pp.container = k.container;
    pp.state_credit_bits = k.credit;
    pp.rdo_candidates = k.rdo_k;
    pp.rdo_sweeps = k.rdo_t;
    pp.nthreads = 2;
    ep_blob pb{nullptr, 0};
    ep_encode_stats st;
    check(ep_encode_cpu(w.data(), EP_BF16, k.R, k.C, &pp, &pb, &st) == EP_OK, "library encode");
    check(ob && pb.data && on == pb.size && std::memcmp(ob, pb.data, on) == 0, "encoders agree");
    ep_tensor_info info;
    check(ep_blob_info(pb.data, pb.size, &info) == EP_OK, "blob info");
    for (int dt : {EP_BF16, EP_FP16, EP_FP32, EP_FP8_E4M3, EP_INT8, EP_FP8_E5M2, EP_UINT8, EP_COORD2_I32}) {
      std::vector<uint8_t> out((size_t)(k.R * k.C) * 4);
      std::vector<float> dq((size_t)k.R);
      check(ora_decode(ob, on, dt, out.data(), dq.data(), 0, info.n_tiles) == 0, "oracle decode");
    }
    if (k.R == 64 && k.C == 512) keep.assign(ob, ob + on);
    ora_blob_free(ob);
    ep_blob_free(&pb);
  }
  std::printf("encode cases: %zu\n", sizeof cases / sizeof cases[0]);

  // malformed blobs: truncations, bit flips in every section, random words
  const size_t n0 = keep.size();
  int accepted = 0;
  for (int it = 0; it < mutations; it++) {
    std::vector<uint8_t> m = keep;
    const int kind = it % 4;
    size_t n = n0;
    if (kind == 0) {
      n = (size_t)(next_u64() % n0);
    } else if (kind == 1) {
      const int flips = 1 + (int)(next_u64() % 4);
      for (int f = 0; f < flips; f++) m[next_u64() % n0] ^= (uint8_t)(1u << (next_u64() % 8));
    } else if (kind == 2) {
      const size_t at = next_u64() % (n0 < 256 ? n0 : 256);   // header and tables
      m[at] = (uint8_t)next_u64();
    } else {
      const size_t at = next_u64() % (n0 - 4);
      const uint32_t v = (uint32_t)next_u64();
      std::memcpy(&m[at & ~size_t(3)], &v, 4);
    }
    std::vector<uint8_t> exact(m.begin(), m.begin() + n);   // no slack after the blob
    ep_tensor_info info;
    const int rc = ep_blob_info(exact.data(), n, &info);
    check(rc == EP_OK || rc == EP_ERR_FORMAT, "blob info status");
    if (rc != EP_OK) continue;
    accepted++;
    if ((uint64_t)info.rows * info.cols > 64ull * 1024 * 1024) continue;
    std::vector<uint8_t> out((size_t)info.rows * info.cols * 4);
    std::vector<float> dq(info.rows);
    const int orc = ora_decode(exact.data(), n, EP_COORD2_I32, out.data(), dq.data(), 0, info.n_tiles);
    check(orc == 0 || orc == -2 || orc == -6, "oracle decode status on a malformed blob");
  }
  std::printf("mutations: %d, accepted by validation: %d\n", mutations, accepted);
  if (failures) {
    std::fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  std::printf("sanitized host run: ok\n");
  return 0;
}
