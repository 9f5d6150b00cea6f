// Fused tile-parallel EntroPack decode for gfx950 (Section 3.7).
//
// One wavefront (64 lanes) decodes two tiles at once: lanes 0-31 hold the 32
// interleaved rANS states of the first tile, lanes 32-63 those of the second.
// Each lane decodes whole 8-vectors: the coset symbol with the two-entry coset
// table, then the eight fields with the tables selected by that coset
// (eq. rans_decode), refilling its state with 16-bit payload words consumed in
// lane order inside each half-wave (ballot + prefix count).  As soon as a
// vector's ninth symbol is known the lane inverts the field map
// (eq. point_inverse), multiplies by the FP32 row scale and snaps to the
// output dtype (eq. recon), and stores the eight weights; no symbol tensor is
// ever written.
//
// Workgroups are persistent: each takes a contiguous range of two-tile tasks,
// builds the decode tables of the layer it is working on in LDS, and its 16
// waves walk the range.  Two table families exist:
//   kPathLut    packed slot table, one LDS read per symbol: for table
//               (field i, coset c) and slot u in [0, 2^b) the 32-bit entry
//               holds f (bits 0-11), u - F (bits 12-22) and the doubled
//               coordinate value (bits 23-31, signed) -- b <= 11 only;
//   kPathSearch per-symbol cumulative table (F | f << 16) searched with a
//               fixed-trip binary search -- any b, alphabets up to the LDS size.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/entropack.h"
#include "common.h"
#include "paths.h"

namespace ep {
namespace {

constexpr int kWaveSize = 64;
constexpr int kWavesPerGroup = 16;
constexpr int kThreads = kWaveSize * kWavesPerGroup;
constexpr uint32_t kStateLow = 1u << 15;

struct LayerDev {
  const uint8_t* blob;
  void* out;
  float* dequant;
  uint32_t rows, cols, cvec, b, V, n_tiles, container;
  uint32_t tile_begin, tile_end;  // tiles decoded
  uint32_t task_begin, n_tasks;   // this layer's slice of the global task list
  uint32_t out_dtype, saturate;
  uint32_t coset_f0, coset_f1;
  uint32_t sum_A, search_iters;
  uint32_t pay_bytes;             // payload section bytes (bounds of the buffer resource)
  uint32_t div_magic, div_shift, div_pow2;  // floor(v / (C/8))
  uint64_t off_sigma, off_delta, off_states, off_offsets, off_payload;
  uint32_t tab_off[16];
  int32_t tab_min[16];
  uint32_t tab_A[16];
  uint32_t tab_base[16];          // prefix of tab_A (search path)
};

// ---- output snapping (eq. recon) --------------------------------------------
__device__ __forceinline__ float sat(float y, float m) { return __builtin_amdgcn_fmed3f(y, -m, m); }

__device__ __forceinline__ uint32_t bf16_pair(float a, float b) {
  typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
  typedef float f2 __attribute__((ext_vector_type(2)));
  f2 v = {a, b};
  bf2 h = __builtin_convertvector(v, bf2);
  uint32_t r;
  __builtin_memcpy(&r, &h, 4);
  return r;
}

__device__ __forceinline__ uint32_t fp16_pair(float a, float b) {
  _Float16 ha = (_Float16)a, hb = (_Float16)b;
  uint16_t ua, ub;
  __builtin_memcpy(&ua, &ha, 2);
  __builtin_memcpy(&ub, &hb, 2);
  return (uint32_t)ua | ((uint32_t)ub << 16);
}

__device__ __forceinline__ uint32_t fp8_quad(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
  return (uint32_t)w;
}

__device__ __forceinline__ uint32_t int8_quad(float a, float b, float c, float d) {
  int ia = (int)__builtin_rintf(sat(a, 128.0f)), ib = (int)__builtin_rintf(sat(b, 128.0f));
  int ic = (int)__builtin_rintf(sat(c, 128.0f)), id = (int)__builtin_rintf(sat(d, 128.0f));
  ia = min(ia, 127), ib = min(ib, 127), ic = min(ic, 127), id = min(id, 127);
  return (uint32_t)(ia & 0xFF) | ((uint32_t)(ib & 0xFF) << 8) | ((uint32_t)(ic & 0xFF) << 16) |
         ((uint32_t)(id & 0xFF) << 24);
}

// Store the eight weights of vector v (elements 8v..8v+7).
__device__ __forceinline__ void store_vector(const LayerDev& L, uint32_t v, const int32_t* p2,
                                             float half_sigma) {
  float y[8];
#pragma unroll
  for (int j = 0; j < 8; j++) y[j] = half_sigma * (float)p2[j];
  switch (L.out_dtype) {
    case EP_BF16: {
      if (L.saturate)
#pragma unroll
        for (int j = 0; j < 8; j++) y[j] = sat(y[j], 3.38953139e38f);
      uint4 o = {bf16_pair(y[0], y[1]), bf16_pair(y[2], y[3]), bf16_pair(y[4], y[5]),
                 bf16_pair(y[6], y[7])};
      reinterpret_cast<uint4*>(L.out)[v] = o;
      break;
    }
    case EP_FP16: {
      if (L.saturate)
#pragma unroll
        for (int j = 0; j < 8; j++) y[j] = sat(y[j], 65504.0f);
      uint4 o = {fp16_pair(y[0], y[1]), fp16_pair(y[2], y[3]), fp16_pair(y[4], y[5]),
                 fp16_pair(y[6], y[7])};
      reinterpret_cast<uint4*>(L.out)[v] = o;
      break;
    }
    case EP_FP32: {
      float4* o = reinterpret_cast<float4*>(L.out) + 2ull * v;
      o[0] = make_float4(y[0], y[1], y[2], y[3]);
      o[1] = make_float4(y[4], y[5], y[6], y[7]);
      break;
    }
    case EP_FP8_E4M3: {
      if (L.saturate)
#pragma unroll
        for (int j = 0; j < 8; j++) y[j] = sat(y[j], 448.0f);
      uint2 o = {fp8_quad(y[0], y[1], y[2], y[3]), fp8_quad(y[4], y[5], y[6], y[7])};
      reinterpret_cast<uint2*>(L.out)[v] = o;
      break;
    }
    case EP_INT8: {
      uint2 o = {int8_quad(y[0], y[1], y[2], y[3]), int8_quad(y[4], y[5], y[6], y[7])};
      reinterpret_cast<uint2*>(L.out)[v] = o;
      break;
    }
    default: {  // EP_COORD2_I32
      int4* o = reinterpret_cast<int4*>(L.out) + 2ull * v;
      o[0] = make_int4(p2[0], p2[1], p2[2], p2[3]);
      o[1] = make_int4(p2[4], p2[5], p2[6], p2[7]);
      break;
    }
  }
}

// ---- table construction in LDS ------------------------------------------------
// Cumulative entries F_s | f_s << 16 of the 16 field tables at lds[base_t + s];
// wave w scans table w (and w + 16 ... when fewer waves exist).
__device__ void build_cumulative(const LayerDev& L, uint32_t* cum) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int t = wave; t < 16; t += kWavesPerGroup) {
    const uint16_t* f = reinterpret_cast<const uint16_t*>(L.blob + L.tab_off[t]);
    const uint32_t A = L.tab_A[t], base = L.tab_base[t];
    uint32_t running = 0;
    for (uint32_t s0 = 0; s0 < A; s0 += kWaveSize) {
      uint32_t s = s0 + lane;
      uint32_t fs = s < A ? f[s] : 0u;
      uint32_t incl = fs;
#pragma unroll
      for (int d = 1; d < kWaveSize; d <<= 1) {
        uint32_t o = __shfl_up(incl, d, kWaveSize);
        if (lane >= d) incl += o;
      }
      if (s < A) cum[base + s] = (running + incl - fs) | (fs << 16);
      running += __shfl(incl, kWaveSize - 1, kWaveSize);
    }
  }
}

__device__ __forceinline__ int32_t doubled_value(int32_t z, int field, uint32_t c) {
  return field < 8 ? 2 * z + (int32_t)c : 4 * z + (int32_t)c;
}

// Packed slot table: lut[t * M + u] for the 16 field tables (b <= 11).
__device__ void build_lut(const LayerDev& L, uint32_t* lut, const uint32_t* cum) {
  const uint32_t M = 1u << L.b;
  const uint32_t per = M / 64;                     // slots per thread: 16 tables x 64 threads
  const int t = threadIdx.x >> 6, j = threadIdx.x & 63;
  const uint32_t A = L.tab_A[t], base = L.tab_base[t];
  const uint32_t u0 = j * per;
  uint32_t* row = lut + t * M;
  if (A == 0) {
    for (uint32_t u = u0; u < u0 + per; u++) row[u] = 0;
    return;
  }
  // largest s with F_s <= u0
  uint32_t s = 0, n = A;
  while (n > 1) {
    uint32_t h = n >> 1;
    if ((cum[base + s + h] & 0xFFFF) <= u0) s += h;
    n -= h;
  }
  const int field = (t & 7) + 1;
  const uint32_t c = (uint32_t)t >> 3;
  uint32_t e = cum[base + s];
  for (uint32_t u = u0; u < u0 + per; u++) {
    while (s + 1 < A && (e & 0xFFFF) + (e >> 16) <= u) e = cum[base + ++s];
    uint32_t F = e & 0xFFFF, f = e >> 16;
    int32_t val = doubled_value((int32_t)s + L.tab_min[t], field, c);
    row[u] = f | ((u - F) << 12) | (((uint32_t)val & 0x1FFu) << 23);
  }
}

// ---- the decode of one two-tile task -------------------------------------------
// Payload staging: each half-wave owns a 512-word ring in LDS.  Word w of the
// payload section lives in slot w & 511.  Chunks of 256 words (aligned to 256
// in w) are fetched with four coalesced buffer_load_dword per lane (a raw
// buffer resource bounds every read to the payload section) into registers,
// and written to the ring ("committed") only when the consumer gets within 64
// words of the committed end, by which time the loads have long returned; the
// following chunk is requested right after each commit.  A commit overwrites
// the slots of words [Qc - 512, Qc - 256), all consumed by then.
constexpr uint32_t kRingWords = 512;
constexpr uint32_t kChunkWords = 256;
constexpr uint32_t kRingBytesPerWave = 2 * 2 * kRingWords;   // two halves, u16 words
constexpr uint32_t kRingBytes = kWavesPerGroup * kRingBytesPerWave;

struct Stage {
  __amdgpu_buffer_rsrc_t rsrc;   // payload section
  uint32_t ring;                 // LDS byte address of this half's ring
  uint32_t Qc;                   // committed end (words)
  uint32_t T;                    // commit trigger: P >= T
  uint32_t Pend;
  uint32_t pend[4];              // fetched, not yet committed chunk
};

__device__ __forceinline__ void fetch_chunk(Stage& S, uint32_t l, uint32_t start) {
#pragma unroll
  for (int k = 0; k < 4; k++)
    S.pend[k] = __builtin_amdgcn_raw_buffer_load_b32(S.rsrc, 2 * start + 4 * (l + 32 * k), 0, 0);
}

__device__ __forceinline__ void store_chunk(uint8_t* lds_base, const Stage& S, uint32_t l,
                                            uint32_t start) {
#pragma unroll
  for (int k = 0; k < 4; k++) {
    const uint32_t slot = (start + 2 * (l + 32 * k)) & (kRingWords - 1);
    *reinterpret_cast<uint32_t*>(lds_base + S.ring + 2 * slot) = S.pend[k];
  }
}

// Commit the pending chunk if this half is within 64 words of the committed end.
__device__ __forceinline__ void stage_check(uint8_t* lds_base, Stage& S, uint32_t P, uint32_t l) {
  const bool due = P >= S.T;
  if (__ballot(due)) {
    if (due) {
      store_chunk(lds_base, S, l, S.Qc);
      S.Qc += kChunkWords;
      S.T = S.Qc - 64;
      if (S.Qc < S.Pend) fetch_chunk(S, l, S.Qc);
    }
  }
}

// Refill states below 2^15 from the half-wave's ring (lane order inside each half).
__device__ __forceinline__ void renorm(uint32_t& x, bool act, uint32_t& P, const uint8_t* lds_base,
                                       const Stage& S, uint32_t half) {
  const uint64_t m = __ballot(act && x < kStateLow);
  const uint32_t lo = (uint32_t)m, hi = (uint32_t)(m >> 32);
  uint32_t idx;
  if (half) {
    idx = __builtin_amdgcn_mbcnt_hi(hi, P);
    P += (uint32_t)__builtin_popcount(hi);
  } else {
    idx = __builtin_amdgcn_mbcnt_lo(lo, P);
    P += (uint32_t)__builtin_popcount(lo);
  }
  if (act && x < kStateLow) {
    const uint32_t word =
        *reinterpret_cast<const uint16_t*>(lds_base + S.ring + 2 * (idx & (kRingWords - 1)));
    x = (x << 16) | word;
  }
}

// One field symbol.  Slot-table path: entry = lut[(8c + i - 1) * 2^B + u]; the
// coset part cb = 8c * 2^B is per lane, the field part a constant offset.
template <int PATH, int B>
__device__ __forceinline__ void decode_field(const LayerDev& L, const uint32_t* lds, int field,
                                             uint32_t cb, uint32_t c, uint32_t& x, int32_t& dval) {
  if (PATH == kPathLut) {
    constexpr uint32_t M = 1u << B;
    const uint32_t u = x & (M - 1);
    const uint32_t e = lds[cb + u + (uint32_t)(field - 1) * M];
    x = __umul24(e & 0xFFFu, x >> B) + ((e >> 12) & 0x7FFu);
    dval = (int32_t)e >> 23;
  } else {
    const uint32_t u = x & ((1u << L.b) - 1);
    const uint32_t base = c ? L.tab_base[8 + field - 1] : L.tab_base[field - 1];
    const uint32_t A = c ? L.tab_A[8 + field - 1] : L.tab_A[field - 1];
    uint32_t s = 0, n = A;
    for (uint32_t it = 0; it < L.search_iters; it++) {
      const uint32_t h = n >> 1;
      if ((lds[base + s + h] & 0xFFFFu) <= u) s += h;
      n -= h;
    }
    const uint32_t e = lds[base + s];
    x = __umul24(e >> 16, x >> L.b) + u - (e & 0xFFFFu);
    const int32_t mn = c ? L.tab_min[8 + field - 1] : L.tab_min[field - 1];
    dval = doubled_value((int32_t)s + mn, field, c);
  }
}

// floor(v / C8) with the host-computed magic (Granlund-Montgomery).
__device__ __forceinline__ uint32_t row_of(const LayerDev& L, uint32_t v) {
  if (L.div_pow2) return v >> L.div_shift;
  const uint32_t q = __umulhi(v, L.div_magic);
  return (q + ((v - q) >> 1)) >> L.div_shift;
}

template <int PATH, int B>
__device__ void decode_task(const LayerDev& L, const uint32_t* lds, uint8_t* lds_base,
                            uint32_t ring_area, uint32_t task, int32_t* status) {
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t half = lane >> 5, l = lane & 31;
  const uint32_t tile = L.tile_begin + 2 * task + half;
  const bool tile_ok = tile < L.tile_end;
  const uint32_t nvec = L.rows * L.cvec;
  const uint32_t v0 = tile_ok ? tile * L.V : 0;
  const uint32_t nv = tile_ok ? min(L.V, nvec - v0) : 0;
  const uint32_t n_l = l < nv ? (nv - 1 - l) / 32 + 1 : 0;
  const uint32_t r_here = (nv + 31) / 32;
  const uint32_t rounds = max(__builtin_amdgcn_readlane(r_here, 0), __builtin_amdgcn_readlane(r_here, 32));

  const uint32_t* states = reinterpret_cast<const uint32_t*>(L.blob + L.off_states);
  const uint32_t* offs = reinterpret_cast<const uint32_t*>(L.blob + L.off_offsets);
  const float* sigma = reinterpret_cast<const float*>(L.blob + L.off_sigma);
  uint32_t x = tile_ok ? states[(uint64_t)tile * 32 + l] : kStateLow;
  const uint32_t P0 = tile_ok ? offs[tile] : 0;
  Stage S;
  S.rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(L.blob + L.off_payload), (short)0,
                                             (int)L.pay_bytes, 0x00020000);
  S.ring = ring_area + wave * kRingBytesPerWave + half * (2 * kRingWords);
  S.Pend = tile_ok ? offs[tile + 1] : 0;
  const uint32_t C0 = P0 & ~(kChunkWords - 1);
  S.Qc = C0;
  S.T = 0xFFFFFFFFu;
  if (tile_ok) {
    fetch_chunk(S, l, C0);
    store_chunk(lds_base, S, l, C0);
    S.Qc = C0 + kChunkWords;
    if (S.Qc < S.Pend) {
      fetch_chunk(S, l, S.Qc);
      store_chunk(lds_base, S, l, S.Qc);
    }
    S.Qc += kChunkWords;
    S.T = S.Qc - 64;
    if (S.Qc < S.Pend) fetch_chunk(S, l, S.Qc);
  }
  uint32_t P = P0;
  const uint32_t mask = (1u << L.b) - 1;

  for (uint32_t k = 0; k < rounds; k++) {
    const bool act = k < n_l;
    const uint32_t v = v0 + l + 32 * k;
    const float sg = act ? sigma[row_of(L, v)] : 0.0f;
    // coset symbol
    uint32_t c = 0, cb = 0;
    if (act) {
      const uint32_t u = x & mask;
      c = u >= L.coset_f0 ? 1u : 0u;
      const uint32_t f = c ? L.coset_f1 : L.coset_f0;
      const uint32_t F = c ? L.coset_f0 : 0u;
      x = __umul24(f, x >> L.b) + u - F;
      cb = c << (L.b + 3);
    }
    stage_check(lds_base, S, P, l);
    renorm(x, act, P, lds_base, S, half);
    int32_t d[9];
#pragma unroll
    for (int i = 1; i <= 8; i++) {
      if (act) decode_field<PATH, B>(L, lds, i, cb, c, x, d[i]);
      stage_check(lds_base, S, P, l);
      renorm(x, act, P, lds_base, S, half);
    }
    if (act) {
      // field inverse: 2p_i = 2 z_i + c; 2p_8 = 4m + c + 2 pi, pi = sum z_1..7 mod 2
      int32_t p2[8];
      int32_t acc = (int32_t)c;
#pragma unroll
      for (int i = 1; i <= 7; i++) {
        p2[i - 1] = d[i];
        acc += d[i];
      }
      p2[7] = d[8] + (acc & 2);
      store_vector(L, v, p2, 0.5f * sg);
    }
  }
  uint32_t err = 0;
  if (tile_ok) {
    if (x != kStateLow) err |= EP_STATUS_BAD_FINAL_STATE;
    if (l == 0 && P != S.Pend) err |= P > S.Pend ? EP_STATUS_PAYLOAD_OVERRUN : EP_STATUS_BAD_END_OFFSET;
    if (L.container && L.dequant) {
      const float* delta = reinterpret_cast<const float*>(L.blob + L.off_delta);
      const uint32_t r_first = (v0 + L.cvec - 1) / L.cvec;
      const uint32_t r_last = (v0 + nv - 1) / L.cvec;
      for (uint32_t r = r_first + l; r <= r_last; r += 32) L.dequant[r] = delta[r];
    }
  }
  if (err && status) atomicOr(status, (int32_t)err);
}

// LDS byte offset of the payload rings: after the slot table (LUT path) or
// after the cumulative table (search path).
template <int PATH>
__device__ __forceinline__ uint32_t ring_offset(const LayerDev& L) {
  return PATH == kPathLut ? (64u << L.b) : ((4u * L.sum_A + 15u) & ~15u);
}

template <int PATH>
__device__ void build_tables(const LayerDev& L, uint32_t* lds) {
  if (PATH == kPathLut) {
    uint32_t* cum = lds + (16u << L.b);   // scratch inside the ring area
    build_cumulative(L, cum);
    __syncthreads();
    build_lut(L, lds, cum);
  } else {
    build_cumulative(L, lds);
  }
}

// Decode global tasks [t_begin, t_end) of a layer list: per layer segment the
// workgroup builds that layer's tables, then its waves take tasks in turn.
template <int PATH>
__device__ void run_layers(const LayerDev* layers, int n_layers, uint32_t total,
                           uint32_t per_group, int32_t* status) {
  extern __shared__ uint32_t lds[];
  const uint32_t t_begin = blockIdx.x * per_group;
  const uint32_t t_end = min(total, t_begin + per_group);
  if (t_begin >= t_end) return;
  const uint32_t wave = threadIdx.x >> 6;
  int li = 0;
  while (li + 1 < n_layers && layers[li + 1].task_begin <= t_begin) li++;
  for (uint32_t seg = t_begin; seg < t_end && li < n_layers; li++) {
    const LayerDev& L = layers[li];
    const uint32_t seg_end = min(t_end, L.task_begin + L.n_tasks);
    if (seg_end <= seg) continue;
    __syncthreads();
    build_tables<PATH>(L, lds);
    __syncthreads();
    const uint32_t ring_area = ring_offset<PATH>(L);
    uint8_t* lb = reinterpret_cast<uint8_t*>(lds);
    for (uint32_t task = seg + wave; task < seg_end; task += kWavesPerGroup) {
      if (PATH == kPathSearch) decode_task<PATH, 0>(L, lds, lb, ring_area, task - L.task_begin, status);
      else if (L.b == 11) decode_task<PATH, 11>(L, lds, lb, ring_area, task - L.task_begin, status);
      else if (L.b == 10) decode_task<PATH, 10>(L, lds, lb, ring_area, task - L.task_begin, status);
      else decode_task<PATH, 9>(L, lds, lb, ring_area, task - L.task_begin, status);
    }
    seg = seg_end;
  }
}

// Up to kArgLayers descriptors travel as a kernel argument (no copy before
// the launch); longer lists are read from the caller's device workspace.
constexpr int kArgLayers = 8;
struct LayerList {
  LayerDev L[kArgLayers];
};
static_assert(sizeof(LayerList) + 64 <= 4096, "kernel arguments are limited to 4 KiB");

template <int PATH>
__global__ __launch_bounds__(kThreads) void decode_args_kernel(const LayerList list, int n_layers,
                                                               uint32_t total, uint32_t per_group,
                                                               int32_t* status) {
  run_layers<PATH>(list.L, n_layers, total, per_group, status);
}

template <int PATH>
__global__ __launch_bounds__(kThreads) void decode_ws_kernel(const LayerDev* layers, int n_layers,
                                                             uint32_t total, uint32_t per_group,
                                                             int32_t* status) {
  run_layers<PATH>(layers, n_layers, total, per_group, status);
}

// ---- host side ---------------------------------------------------------------------
struct DeviceProps {
  int cus = 0;
  size_t max_lds = 0;
};

DeviceProps device_props() {
  static std::mutex mu;
  static std::vector<DeviceProps> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return DeviceProps{};
  std::lock_guard<std::mutex> g(mu);
  if ((int)cache.size() <= dev) cache.resize(dev + 1);
  if (!cache[dev].cus) {
    int cus = 0, lds = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) cus = 0;
    if (hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) lds = 0;
    cache[dev].cus = cus;
    cache[dev].max_lds = (size_t)lds;
  }
  return cache[dev];
}

uint32_t lds_bytes(uint32_t path, const ep_tensor_info& I) {
  if (path == kPathLut) return (64u << I.prob_bits) + kRingBytes;
  return ((4u * I.sum_alphabet + 15u) & ~15u) + kRingBytes;
}

float dtype_max(int dt) {
  switch (dt) {
    case EP_BF16: return 3.38953139e38f;
    case EP_FP16: return 65504.0f;
    case EP_FP8_E4M3: return 448.0f;
    default: return 3.4e38f;
  }
}

bool valid_out_dtype(int dt) {
  return dt == EP_BF16 || dt == EP_FP16 || dt == EP_FP32 || dt == EP_FP8_E4M3 || dt == EP_INT8 ||
         dt == EP_COORD2_I32;
}

int fill_layer(const ep_tensor_info& I, const void* d_blob, int out_dtype, void* d_out,
               float* d_dequant, uint32_t t0, uint32_t t1, LayerDev& D) {
  if (!d_blob || !d_out) return fail(EP_ERR_ARG, "decode: null device pointer");
  if (!valid_out_dtype(out_dtype)) return fail(EP_ERR_ARG, "decode: unknown output dtype");
  if (t0 > t1 || t1 > I.n_tiles) return fail(EP_ERR_ARG, "decode: tile range outside the tensor");
  if (!I.rows || !I.cols || I.cols % 8 || I.prob_bits < 9 || I.prob_bits > 15 || !I.tile_vectors)
    return fail(EP_ERR_ARG, "decode: tensor info not filled by ep_blob_info");
  if (I.path == kPathNone)
    return fail(EP_ERR_UNSUPPORTED, "decode: the frequency tables do not fit a decode path of this build");
  std::memset(&D, 0, sizeof D);
  D.blob = static_cast<const uint8_t*>(d_blob);
  D.out = d_out;
  D.dequant = d_dequant;
  D.rows = I.rows;
  D.cols = I.cols;
  D.cvec = I.cols / 8;
  D.b = I.prob_bits;
  D.V = I.tile_vectors;
  D.n_tiles = I.n_tiles;
  D.container = I.container;
  D.tile_begin = t0;
  D.tile_end = t1;
  D.n_tasks = (t1 - t0 + 1) / 2;
  D.out_dtype = (uint32_t)out_dtype;
  D.saturate = I.max_abs_weight >= dtype_max(out_dtype) ? 1u : 0u;
  D.coset_f0 = I.coset_f0;
  D.coset_f1 = I.coset_f1;
  D.sum_A = I.sum_alphabet;
  uint32_t amax = 1, it = 0;
  for (int t = 0; t < 16; t++) amax = std::max(amax, I.table_A[t]);
  while ((1u << it) < amax) it++;
  D.search_iters = it;
  const uint64_t pay = (2ull * I.payload_words + 3) / 4 * 4;
  if (pay > 0xFFFFFFF0ull) return fail(EP_ERR_UNSUPPORTED, "decode: payload section above 4 GiB");
  D.pay_bytes = (uint32_t)pay;
  const uint32_t d = D.cvec;
  if ((d & (d - 1)) == 0) {
    D.div_pow2 = 1;
    D.div_shift = 0;
    while ((1u << D.div_shift) < d) D.div_shift++;
  } else {
    uint32_t lg = 0;
    while ((1ull << lg) < d) lg++;
    D.div_pow2 = 0;
    D.div_magic = (uint32_t)(((1ull << 32) * ((1ull << lg) - d)) / d + 1);
    D.div_shift = lg - 1;
  }
  D.off_sigma = I.off_sigma;
  D.off_delta = I.off_delta;
  D.off_states = I.off_states;
  D.off_offsets = I.off_offsets;
  D.off_payload = I.off_payload;
  uint32_t base = 0;
  for (int t = 0; t < 16; t++) {
    D.tab_off[t] = I.table_off[t];
    D.tab_min[t] = I.table_min[t];
    D.tab_A[t] = I.table_A[t];
    D.tab_base[t] = base;
    base += I.table_A[t];
  }
  return EP_OK;
}

uint32_t groups_for(uint32_t path, uint32_t lds, uint32_t tasks, const DeviceProps& P) {
  uint32_t per_cu = path == kPathLut ? 1u : (uint32_t)std::max<size_t>(1, std::min<size_t>(2, 160 * 1024 / std::max<uint32_t>(lds, 1)));
  uint32_t g = (uint32_t)P.cus * per_cu;
  uint32_t need = (tasks + kWavesPerGroup - 1) / kWavesPerGroup;
  return std::max(1u, std::min(g, need));
}

}  // namespace

template <int PATH>
int set_lds_limit(size_t bytes) {
  hipError_t e1 = hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_args_kernel<PATH>),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  hipError_t e2 = hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_ws_kernel<PATH>),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  return (e1 == hipSuccess && e2 == hipSuccess) ? EP_OK : EP_ERR_HIP;
}

// Launch the layers of one decode path: by-value descriptors when they fit,
// else from d_ws (copied there first on the same stream).
int launch_layers(uint32_t path, const std::vector<LayerDev>& D, uint32_t total, uint32_t lds,
                  void* d_ws, uint64_t ws_bytes, int32_t* d_status, hipStream_t s,
                  const char* who) {
  DeviceProps P = device_props();
  if (!P.cus) return fail(EP_ERR_HIP, "decode: no HIP device");
  if (lds > P.max_lds) return fail(EP_ERR_UNSUPPORTED, "decode: tables exceed the device LDS");
  uint32_t G = groups_for(path, lds, total, P);
  uint32_t per = (total + G - 1) / G;
  G = (total + per - 1) / per;
  const int n = (int)D.size();
  int rc = path == kPathLut ? set_lds_limit<kPathLut>(lds) : set_lds_limit<kPathSearch>(lds);
  if (rc) return fail(EP_ERR_HIP, "decode: cannot raise the kernel's LDS limit");
  if (n <= kArgLayers) {
    LayerList list;
    std::memset(&list, 0, sizeof list);
    for (int i = 0; i < n; i++) list.L[i] = D[i];
    if (path == kPathLut)
      hipLaunchKernelGGL(decode_args_kernel<kPathLut>, dim3(G), dim3(kThreads), lds, s, list, n, total, per, d_status);
    else
      hipLaunchKernelGGL(decode_args_kernel<kPathSearch>, dim3(G), dim3(kThreads), lds, s, list, n, total, per, d_status);
  } else {
    if (!d_ws || ws_bytes < sizeof(LayerDev) * (uint64_t)n)
      return fail(EP_ERR_ARG, "ep_decode_layers: workspace too small");
    if (hipMemcpyAsync(d_ws, D.data(), sizeof(LayerDev) * D.size(), hipMemcpyHostToDevice, s) != hipSuccess)
      return fail(EP_ERR_HIP, "ep_decode_layers: descriptor copy failed");
    const LayerDev* dl = static_cast<const LayerDev*>(d_ws);
    if (path == kPathLut)
      hipLaunchKernelGGL(decode_ws_kernel<kPathLut>, dim3(G), dim3(kThreads), lds, s, dl, n, total, per, d_status);
    else
      hipLaunchKernelGGL(decode_ws_kernel<kPathSearch>, dim3(G), dim3(kThreads), lds, s, dl, n, total, per, d_status);
  }
  if (hipGetLastError() != hipSuccess) return fail(EP_ERR_HIP, (std::string(who) + ": launch failed").c_str());
  return EP_OK;
}

int decode_tiles(const ep_tensor_info* info, const void* d_blob, int out_dtype, void* d_out,
                 float* d_dequant, uint32_t t0, uint32_t t1, int32_t* d_status, void* stream) {
  if (!info) return fail(EP_ERR_ARG, "ep_decode_tiles: null info");
  std::vector<LayerDev> D(1);
  int rc = fill_layer(*info, d_blob, out_dtype, d_out, d_dequant, t0, t1, D[0]);
  if (rc) return rc;
  if (D[0].n_tasks == 0) return EP_OK;
  return launch_layers(info->path, D, D[0].n_tasks, lds_bytes(info->path, *info), nullptr, 0,
                       d_status, static_cast<hipStream_t>(stream), "ep_decode_tiles");
}

uint64_t decode_layers_workspace(int n) {
  return n > kArgLayers ? (uint64_t)n * sizeof(LayerDev) : 0;
}

int decode_layers(const ep_layer* layers, int n, void* d_ws, uint64_t ws_bytes, int32_t* d_status,
                  void* stream) {
  if (n < 0 || (n > 0 && !layers)) return fail(EP_ERR_ARG, "ep_decode_layers: bad layer list");
  if (n == 0) return EP_OK;
  const uint32_t path = layers[0].info.path;
  std::vector<LayerDev> D((size_t)n);
  uint32_t total = 0, lds = 0;
  for (int i = 0; i < n; i++) {
    const ep_layer& Lr = layers[i];
    if (Lr.info.path != path)
      return fail(EP_ERR_UNSUPPORTED, "ep_decode_layers: layers need different decode paths");
    int rc = fill_layer(Lr.info, Lr.d_blob, Lr.out_dtype, Lr.d_out, Lr.d_dequant, 0,
                        Lr.info.n_tiles, D[i]);
    if (rc) return rc;
    D[i].task_begin = total;
    total += D[i].n_tasks;
    lds = std::max(lds, lds_bytes(path, Lr.info));
  }
  if (total == 0) return EP_OK;
  return launch_layers(path, D, total, lds, d_ws, ws_bytes, d_status,
                       static_cast<hipStream_t>(stream), "ep_decode_layers");
}

}  // namespace ep

extern "C" {

int ep_decode_tiles(const ep_tensor_info* info, const void* d_blob, int out_dtype, void* d_out,
                    float* d_dequant, uint32_t tile_begin, uint32_t tile_end, int32_t* d_status,
                    void* hip_stream) {
  return ep::decode_tiles(info, d_blob, out_dtype, d_out, d_dequant, tile_begin, tile_end,
                          d_status, hip_stream);
}

uint64_t ep_decode_layers_workspace(int n) { return ep::decode_layers_workspace(n); }

int ep_decode_layers(const ep_layer* layers, int n, void* d_workspace, uint64_t ws_bytes,
                     int32_t* d_status, void* hip_stream) {
  return ep::decode_layers(layers, n, d_workspace, ws_bytes, d_status, hip_stream);
}

}  // extern "C"
