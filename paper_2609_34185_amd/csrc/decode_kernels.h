// Device side of the fused decode (Section 3.7): tables, steady states,
// generic loop and the kernel templates.  Included by decode.hip (host code
// and most kernels), decode_args.hip, decode_mixed.hip and decode_gemm.hip,
// which instantiate the remaining kernels, so that the four compile
// concurrently.
//
// A chain is one wavefront (64 lanes) over two tiles: lanes 0-31 hold the 32
// interleaved rANS states of the first tile, lanes 32-63 those of the second.
// Each lane decodes whole 8-vectors: the coset symbol with the two-entry coset
// table, then the eight fields with the tables selected by that coset
// (eq. rans_decode), refilling its state with 16-bit payload words consumed in
// lane order inside each half-wave (ballot + prefix count).  As soon as a
// vector's ninth symbol is known the lane inverts the field map
// (eq. point_inverse), multiplies by the FP32 row scale and snaps to the
// output dtype (eq. recon), and stores the eight weights; no symbol tensor is
// ever written.  A wave interleaves two chains (a four-tile task), or runs one
// (a two-tile task) in launches with too few four-tile tasks to fill the SIMDs.
//
// Workgroups are persistent: each takes a contiguous range of tasks, builds
// (or copies in) the decode tables of the layer it is working on in LDS, and
// its 16 waves walk the range.  Four table layouts exist:
//   kPathLut    packed slot table, one LDS read per symbol: for table
//               (field i, coset c) and slot u in [0, 2^b) the 32-bit entry
//               holds f (bits 0-11), u - F (bits 12-22) and, as a signed
//               byte in bits 24-31, the integer part z of the coordinate
//               (2p_i = 2z + c; for field 8, z = 2m, so 2p_8 = 2(z + pi) + c)
//               -- b <= 11 only;
//   kPathWide   the same table with wide entries for larger coordinates:
//               f - 1 (bits 0-10), u - F (bits 11-21) and z as a signed
//               10-bit field (bits 22-31); one more add per symbol;
//   kPathSearch per-symbol cumulative table (F | f << 16) searched with a
//               fixed-trip binary search -- any b, alphabets up to the LDS size;
//   kPathGlobal every G-th cumulative value in LDS, the frequencies themselves
//               read from the blob in global memory -- any valid table.
#pragma once
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <string>
#include <type_traits>
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
// Internal output mode of the fused product (never a public dtype code): the
// decoded INT8 container values are multiplied into a small int8 batch X and
// summed into Y (int32) instead of being stored.
constexpr int kOutDotI8 = 0x200;
constexpr uint32_t kDotMaxTokens = 8;

// Index of the calling wave in its workgroup, as a wave-uniform (scalar) value.
__device__ __forceinline__ uint32_t wave_id() {
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
}

// Global-memory views of the caller's pointers.  Accesses through them are
// global (not flat) instructions, so they count only against vmcnt and never
// delay the waits for LDS reads.
#define EP_GLOBAL __attribute__((address_space(1)))
template <class T>
__device__ __forceinline__ EP_GLOBAL T* gptr(const void* p) {
  return (EP_GLOBAL T*)const_cast<void*>(p);
}
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct LayerDev {
  const uint8_t* blob;
  void* out;
  float* dequant;
  uint32_t rows, cols, cvec, b, V, n_tiles, container;
  uint32_t tile_begin, tile_end;  // tiles decoded
  uint32_t task_begin, n_tasks;   // this layer's slice of the global task list
  uint32_t out_dtype, saturate;
  uint32_t coset_f0, coset_f1;
  uint32_t sum_A;
  uint32_t pay_bytes;             // payload section bytes (bounds of the buffer resource)
  uint32_t div_magic, div_shift, div_pow2;  // floor(v / (C/8))
  uint64_t off_sigma, off_delta, off_states, off_offsets, off_payload;
  uint32_t tab_off[16];
  int32_t tab_min[16];
  uint32_t tab_A[16];
  uint32_t tab_base[16];          // prefix of tab_A (search path)
  const int8_t* x;                // fused product: X (m x cols, row-major), Y in `out`
  uint32_t m;
  uint32_t path;                  // decode path of the layer (DecodePath)
  uint32_t tpt;                   // tiles per task: 4 (two chains per wave) or 2 (one chain)
  uint32_t g_bits, g_meta;        // global-table path: log2 G, byte offset of its metadata
  const uint8_t* tables;          // prepared stacks: the layer's decode tables as built in LDS
                                  // (ring_offset bytes), copied in instead of rebuilt; or null
};

// The scalars the decode loop needs, read once per layer segment and forced
// into scalar registers (whatever memory the descriptor list lives in).
struct Hot {
  const uint8_t* blob;
  void* out;
  float* dequant;
  uint32_t rows, cvec, V, tile_begin, tile_end, b, container;
  uint32_t out_dtype, saturate, coset_f0, coset_f1;
  uint32_t pay_bytes, div_magic, div_shift, div_pow2;
  uint32_t meta, bucket;          // search path: u32 index of the metadata, u16 index of the buckets
  uint32_t bucket_shift, bucket_n1; // search path: b - k and 2^k + 1
  uint32_t off_sigma, off_delta, off_states, off_offsets, off_payload;
  const int8_t* x;
  uint32_t m, cols;
  uint32_t g_bits, g_meta;        // global-table path: log2 G, u32 index of the metadata
  uint32_t tab_bytes;             // end of the tables section (bounds of their loads)
  uint32_t tpt;                   // tiles per task (LayerDev::tpt)
};

__device__ __forceinline__ uint32_t uni(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
}
template <class T>
__device__ __forceinline__ T* uni_ptr(T* p) {
  const uint64_t a = (uint64_t)p;
  return (T*)((uint64_t)uni((uint32_t)a) | ((uint64_t)uni((uint32_t)(a >> 32)) << 32));
}

__device__ __forceinline__ Hot make_hot(const LayerDev& L) {
  Hot H;
  H.blob = uni_ptr(L.blob);
  H.out = uni_ptr(L.out);
  H.dequant = uni_ptr(L.dequant);
  H.rows = uni(L.rows);
  H.cvec = uni(L.cvec);
  H.V = uni(L.V);
  H.tile_begin = uni(L.tile_begin);
  H.tile_end = uni(L.tile_end);
  H.b = uni(L.b);
  H.container = uni(L.container);
  H.out_dtype = uni(L.out_dtype);
  H.saturate = uni(L.saturate);
  H.coset_f0 = uni(L.coset_f0);
  H.coset_f1 = uni(L.coset_f1);
  H.pay_bytes = uni(L.pay_bytes);
  H.div_magic = uni(L.div_magic);
  H.div_shift = uni(L.div_shift);
  H.div_pow2 = uni(L.div_pow2);
  {
    const SearchLayout S = search_layout(L.b, L.sum_A);
    H.meta = uni(S.meta / 4);
    H.bucket = uni(S.bucket / 2);
    H.bucket_shift = uni(L.b - S.bucket_bits);
    H.bucket_n1 = uni((1u << S.bucket_bits) + 1);
  }
  H.off_sigma = uni((uint32_t)L.off_sigma);
  H.off_delta = uni((uint32_t)L.off_delta);
  H.off_states = uni((uint32_t)L.off_states);
  H.off_offsets = uni((uint32_t)L.off_offsets);
  H.off_payload = uni((uint32_t)L.off_payload);
  H.x = uni_ptr(L.x);
  H.m = uni(L.m);
  H.cols = uni(L.cols);
  H.g_bits = uni(L.g_bits);
  H.g_meta = uni(L.g_meta / 4);
  H.tab_bytes = uni((uint32_t)L.off_sigma);
  H.tpt = uni(L.tpt);
  return H;
}

// ---- output snapping (eq. recon) --------------------------------------------
__device__ __forceinline__ float sat(float y, float m) { return __builtin_amdgcn_fmed3f(y, -m, m); }

// Two FP32 values to a BF16 pair (round to nearest even), converted where it
// stands: left to itself the compiler keeps the eight FP32 values of a vector
// alive until its store, which costs a scratch spill in the steady state.
__device__ __forceinline__ uint32_t bf16_pair(float a, float b) {
  uint32_t r;
  asm("v_cvt_pk_bf16_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

__device__ __forceinline__ uint32_t fp16_pair(float a, float b) {
  // The product is rounded to FP32 first: keep the compiler from fusing the
  // multiply into a mixed-precision FMA that rounds once, to FP16.
  asm("" : "+v"(a), "+v"(b));
  _Float16 ha = (_Float16)a, hb = (_Float16)b;
  uint16_t ua, ub;
  __builtin_memcpy(&ua, &ha, 2);
  __builtin_memcpy(&ub, &hb, 2);
  return (uint32_t)ua | ((uint32_t)ub << 16);
}

__device__ __forceinline__ uint32_t fp8_quad(float a, float b, float c, float d) {
  // the first conversion fills the low half; its high half is overwritten next
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)__float_as_uint(a), false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
  return (uint32_t)w;
}

// The same for OCP e5m2 (v_cvt_pk_bf8_f32: round to nearest even).
__device__ __forceinline__ uint32_t e5m2_quad(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_bf8_f32(a, b, (int)__float_as_uint(a), false);
  w = __builtin_amdgcn_cvt_pk_bf8_f32(c, d, w, true);
  return (uint32_t)w;
}

__device__ __forceinline__ uint32_t uint8_quad(float a, float b, float c, float d) {
  const int ia = (int)__builtin_rintf(__builtin_amdgcn_fmed3f(a, 0.0f, 255.0f));
  const int ib = (int)__builtin_rintf(__builtin_amdgcn_fmed3f(b, 0.0f, 255.0f));
  const int ic = (int)__builtin_rintf(__builtin_amdgcn_fmed3f(c, 0.0f, 255.0f));
  const int id = (int)__builtin_rintf(__builtin_amdgcn_fmed3f(d, 0.0f, 255.0f));
  return (uint32_t)ia | ((uint32_t)ib << 8) | ((uint32_t)ic << 16) | ((uint32_t)id << 24);
}

__device__ __forceinline__ uint32_t int8_quad(float a, float b, float c, float d) {
  int ia = (int)__builtin_rintf(sat(a, 128.0f)), ib = (int)__builtin_rintf(sat(b, 128.0f));
  int ic = (int)__builtin_rintf(sat(c, 128.0f)), id = (int)__builtin_rintf(sat(d, 128.0f));
  ia = min(ia, 127), ib = min(ib, 127), ic = min(ic, 127), id = min(id, 127);
  return (uint32_t)(ia & 0xFF) | ((uint32_t)(ib & 0xFF) << 8) | ((uint32_t)(ic & 0xFF) << 16) |
         ((uint32_t)(id & 0xFF) << 24);
}

// Store the eight weights of vector v (elements 8v..8v+7), output type DT,
// saturating to the type's finite range when SAT.
template <int DT, bool SAT>
__device__ __forceinline__ void store_vec(void* out, uint32_t v, const int32_t* p2,
                                          float half_sigma) {
  float y[8];
#pragma unroll
  for (int j = 0; j < 8; j++) y[j] = half_sigma * (float)p2[j];
  if constexpr (DT == EP_BF16) {
    if constexpr (SAT)
#pragma unroll
      for (int j = 0; j < 8; j++) y[j] = sat(y[j], 3.38953139e38f);
    const u32x4 o = {bf16_pair(y[0], y[1]), bf16_pair(y[2], y[3]), bf16_pair(y[4], y[5]),
                     bf16_pair(y[6], y[7])};
    gptr<u32x4>(out)[v] = o;
  } else if constexpr (DT == EP_FP16) {
    if constexpr (SAT)
#pragma unroll
      for (int j = 0; j < 8; j++) y[j] = sat(y[j], 65504.0f);
    const u32x4 o = {fp16_pair(y[0], y[1]), fp16_pair(y[2], y[3]), fp16_pair(y[4], y[5]),
                     fp16_pair(y[6], y[7])};
    gptr<u32x4>(out)[v] = o;
  } else if constexpr (DT == EP_FP32) {
    EP_GLOBAL u32x4* o = gptr<u32x4>(out) + 2ull * v;
    o[0] = u32x4{__float_as_uint(y[0]), __float_as_uint(y[1]), __float_as_uint(y[2]),
                 __float_as_uint(y[3])};
    o[1] = u32x4{__float_as_uint(y[4]), __float_as_uint(y[5]), __float_as_uint(y[6]),
                 __float_as_uint(y[7])};
  } else if constexpr (DT == EP_FP8_E4M3) {
    if constexpr (SAT)
#pragma unroll
      for (int j = 0; j < 8; j++) y[j] = sat(y[j], 448.0f);
    const u32x2 o = {fp8_quad(y[0], y[1], y[2], y[3]), fp8_quad(y[4], y[5], y[6], y[7])};
    gptr<u32x2>(out)[v] = o;
  } else if constexpr (DT == EP_FP8_E5M2) {
    if constexpr (SAT)
#pragma unroll
      for (int j = 0; j < 8; j++) y[j] = sat(y[j], 57344.0f);
    const u32x2 o = {e5m2_quad(y[0], y[1], y[2], y[3]), e5m2_quad(y[4], y[5], y[6], y[7])};
    gptr<u32x2>(out)[v] = o;
  } else if constexpr (DT == EP_INT8) {
    const u32x2 o = {int8_quad(y[0], y[1], y[2], y[3]), int8_quad(y[4], y[5], y[6], y[7])};
    gptr<u32x2>(out)[v] = o;
  } else if constexpr (DT == EP_UINT8) {
    const u32x2 o = {uint8_quad(y[0], y[1], y[2], y[3]), uint8_quad(y[4], y[5], y[6], y[7])};
    gptr<u32x2>(out)[v] = o;
  } else {  // EP_COORD2_I32
    EP_GLOBAL u32x4* o = gptr<u32x4>(out) + 2ull * v;
    o[0] = u32x4{(uint32_t)p2[0], (uint32_t)p2[1], (uint32_t)p2[2], (uint32_t)p2[3]};
    o[1] = u32x4{(uint32_t)p2[4], (uint32_t)p2[5], (uint32_t)p2[6], (uint32_t)p2[7]};
  }
}

__device__ __forceinline__ uint32_t row_of(const Hot& L, uint32_t v);

// *p += v as a global-memory atomic (never a flat one: flat instructions also
// count against lgkmcnt, which the decode steps' LDS waits rely on).
__device__ __forceinline__ void add_i32(EP_GLOBAL int32_t* p, int32_t v) {
#if defined(__HIP_DEVICE_COMPILE__)
  __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#else
  (void)p;
  (void)v;
#endif
}

// Fused product, one vector at a time: the eight INT8 weights (w0: elements
// 0-3, w1: 4-7, one byte each) of vector v times the same eight columns of
// every row t of X, added to Y[t][row] (int32, exact).
__device__ __forceinline__ void dot_add(const Hot& L, uint32_t w0, uint32_t w1, uint32_t v,
                                        uint32_t r) {
  const uint32_t col8 = 8 * (v - r * L.cvec);
  const EP_GLOBAL int8_t* xp = gptr<const int8_t>(L.x) + col8;
  EP_GLOBAL int32_t* y = gptr<int32_t>(L.out) + r;
  for (uint32_t t = 0; t < L.m; t++) {
    const u32x2 xv = *reinterpret_cast<const EP_GLOBAL u32x2*>(xp + (uint64_t)t * L.cols);
    const int d = __builtin_amdgcn_sdot4((int)w1, (int)xv.y, __builtin_amdgcn_sdot4((int)w0, (int)xv.x, 0, false), false);
    add_i32(y + (uint64_t)t * L.rows, d);
  }
}

__device__ __forceinline__ void dot_vec(const Hot& L, uint32_t v, const int32_t* p2, float half_sigma) {
  float y[8];
#pragma unroll
  for (int j = 0; j < 8; j++) y[j] = half_sigma * (float)p2[j];
  dot_add(L, int8_quad(y[0], y[1], y[2], y[3]), int8_quad(y[4], y[5], y[6], y[7]), v, row_of(L, v));
}

template <bool DOT = false>
__device__ __forceinline__ void store_vector(const Hot& L, uint32_t v, const int32_t* p2,
                                             float half_sigma) {
  if constexpr (DOT) {
    dot_vec(L, v, p2, half_sigma);
    return;
  }
  switch (L.out_dtype) {
    case EP_BF16:
      if (L.saturate) store_vec<EP_BF16, true>(L.out, v, p2, half_sigma);
      else store_vec<EP_BF16, false>(L.out, v, p2, half_sigma);
      break;
    case EP_FP16:
      if (L.saturate) store_vec<EP_FP16, true>(L.out, v, p2, half_sigma);
      else store_vec<EP_FP16, false>(L.out, v, p2, half_sigma);
      break;
    case EP_FP32: store_vec<EP_FP32, false>(L.out, v, p2, half_sigma); break;
    case EP_FP8_E4M3:
      if (L.saturate) store_vec<EP_FP8_E4M3, true>(L.out, v, p2, half_sigma);
      else store_vec<EP_FP8_E4M3, false>(L.out, v, p2, half_sigma);
      break;
    case EP_FP8_E5M2:
      if (L.saturate) store_vec<EP_FP8_E5M2, true>(L.out, v, p2, half_sigma);
      else store_vec<EP_FP8_E5M2, false>(L.out, v, p2, half_sigma);
      break;
    case EP_INT8: store_vec<EP_INT8, false>(L.out, v, p2, half_sigma); break;
    case EP_UINT8: store_vec<EP_UINT8, false>(L.out, v, p2, half_sigma); break;
    default: store_vec<EP_COORD2_I32, false>(L.out, v, p2, half_sigma); break;
  }
}

// ---- table construction in LDS ------------------------------------------------
// Prefix sums of the 16 field tables' frequencies: put(t, s, F_s, f_s) for every
// symbol s of table t, and end(t, M) once per table with the total (= 2^b).
// Wave w scans table w (and w + kWavesPerGroup ... when fewer waves exist).
// The frequencies of up to kScanAhead chunks of 64 symbols are requested
// together before any of them is scanned, so a table of a few hundred symbols
// waits for memory once rather than once per chunk (every workgroup builds its
// tables at the same moment, when loads are slowest).  Lanes past the end read
// the table's last entry (in bounds) and use 0.
constexpr int kScanAhead = 4;
template <class Put, class End>
__device__ __forceinline__ void scan_tables(const LayerDev& L, Put put, End end) {
  const int lane = threadIdx.x & 63, wave = (int)wave_id();
  for (int t = wave; t < 16; t += kWavesPerGroup) {
    const EP_GLOBAL uint16_t* f = gptr<const uint16_t>(L.blob + L.tab_off[t]);
    const uint32_t A = L.tab_A[t];
    uint32_t running = 0;
    for (uint32_t g0 = 0; g0 < A; g0 += kScanAhead * kWaveSize) {
      uint32_t fa[kScanAhead];
#pragma unroll
      for (int k = 0; k < kScanAhead; k++) {
        const uint32_t s = g0 + k * kWaveSize + lane;
        const uint32_t v = f[s < A ? s : A - 1];
        fa[k] = s < A ? v : 0u;
      }
#pragma unroll
      for (int k = 0; k < kScanAhead; k++) {
        const uint32_t s0 = g0 + k * kWaveSize;
        if (s0 >= A) break;
        const uint32_t s = s0 + lane, fs = fa[k];
        uint32_t incl = fs;
#pragma unroll
        for (int d = 1; d < kWaveSize; d <<= 1) {
          uint32_t o = __shfl_up(incl, d, kWaveSize);
          if (lane >= d) incl += o;
        }
        if (s < A) put(t, s, running + incl - fs, fs);
        running += __shfl(incl, kWaveSize - 1, kWaveSize);
      }
    }
    if (lane == 0) end(t, running);
  }
}

// Cumulative entries F_s | f_s << 16 at cum[base_t + s] (slot-table build).
__device__ __forceinline__ void build_cumulative(const LayerDev& L, uint32_t* cum) {
  scan_tables(L, [&](int t, uint32_t s, uint32_t F, uint32_t f) { cum[L.tab_base[t] + s] = F | (f << 16); },
              [](int, uint32_t) {});
}

__device__ __forceinline__ int32_t doubled_value(int32_t z, int field, uint32_t c) {
  return field < 8 ? 2 * z + (int32_t)c : 4 * z + (int32_t)c;
}

// Packed slot table: lut[t * M + u] for the 16 field tables (b <= 11).  Wave
// w fills tables w, w + kWavesPerGroup, ...; each lane a run of M/64 slots.
// The byte z of an entry is the field value for fields 1-7 and twice the
// value m for field 8, so that every coordinate is 2z + c before field 8's
// parity bit (2 pi) is added; the host admits a tensor to this path only when
// every doubled coordinate lies in [-256, 255], i.e. z fits a signed byte.
// Wide entries (WIDE) hold f - 1 in 11 bits (f = 2^b only for a one-symbol
// table), u - F in 11 bits and z in a signed 10-bit field: doubled coordinates
// in [-1024, 1023].
template <bool WIDE>
__device__ __forceinline__ void build_lut_table(const LayerDev& L, uint32_t* lut,
                                                const uint32_t* cum, int t, int j) {
  const uint32_t M = 1u << L.b;
  const uint32_t per = M / 64;
  const uint32_t A = L.tab_A[t], base = L.tab_base[t];
  const uint32_t u0 = j * per;
  uint32_t* row = lut + t * M;
  // Lane j owns slots u0 .. u0 + per - 1 but writes them starting at offset
  // j mod per and wrapping, so that at each store the wave's lanes hit
  // different banks (in order, every lane would hit the same bank: runs of
  // per = 32 slots are 128 bytes apart).  Both starting symbols are found
  // before the loop, so the wrap is a select, not a divergent search.
  const uint32_t i0 = (uint32_t)j & (per - 1);
  if (A == 0) {
    for (uint32_t k = 0; k < per; k++) row[u0 + ((i0 + k) & (per - 1))] = 0;
    return;
  }
  // largest s with F_s <= u, for u = u0 + i0 and u = u0 (the two searches
  // advance together, their reads in flight at once)
  uint32_t s_mid = 0, s_start = 0;
  for (uint32_t n = A; n > 1;) {
    const uint32_t h = n >> 1;
    const uint32_t c_mid = cum[base + s_mid + h], c_start = cum[base + s_start + h];
    if ((c_mid & 0xFFFF) <= u0 + i0) s_mid += h;
    if ((c_start & 0xFFFF) <= u0) s_start += h;
    n -= h;
  }
  const int field = (t & 7) + 1;
  const uint32_t e_mid = cum[base + s_mid], e_start = cum[base + s_start];
  uint32_t s = s_mid, e = e_mid;
  for (uint32_t k = 0; k < per; k++) {
    const uint32_t i = (i0 + k) & (per - 1);
    const uint32_t u = u0 + i;
    if (i == 0) {   // wrapped to the start of the run
      s = s_start;
      e = e_start;
    }
    while (s + 1 < A && (e & 0xFFFF) + (e >> 16) <= u) e = cum[base + ++s];
    uint32_t F = e & 0xFFFF, f = e >> 16;
    const int32_t v = (int32_t)s + L.tab_min[t];
    const int32_t z = field < 8 ? v : 2 * v;
    row[u] = WIDE ? (f - 1) | ((u - F) << 11) | ((uint32_t)(z & 0x3FF) << 22)
                  : f | ((u - F) << 12) | ((uint32_t)(z & 0xFF) << 24);
  }
}

template <bool WIDE>
__device__ __forceinline__ void build_lut(const LayerDev& L, uint32_t* lut, const uint32_t* cum) {
  for (int t = (int)wave_id(); t < 16; t += kWavesPerGroup)
    build_lut_table<WIDE>(L, lut, cum, t, threadIdx.x & 63);
}

// LDS bytes of the payload rings of a workgroup (all waves, all halves).
constexpr uint32_t kRingBytes = 32 * 1024;

// ---- the decode of one wave task ---------------------------------------------------
// A wave task is NC chains; chain j decodes two tiles, the first on lanes 0-31
// (half A), the second on lanes 32-63 (half B).  Every half owns a payload ring
// in LDS: a logical ring of RW words stored twice (physical slots s and s + RW
// hold the same word), so the up-to-32 words a step reads never wrap.  Chunks
// of CW = RW/2 words are fetched with bounded raw-buffer loads into registers
// and written to the ring ("committed") when the consumer pointer reaches the
// last CW committed words; the next chunk is requested right after.  A commit
// overwrites words [Qc - RW, Qc - CW), all consumed by then.  The read pointer
// of each half is kept as a wave-uniform LDS byte address; the per-lane word
// address is base + 2 * (prefix of the 64-lane refill ballot, corrected for
// the upper half).
template <int NC>
struct RingGeom {
  static constexpr uint32_t RW = NC == 1 ? 256 : 128;   // logical ring words
  static constexpr uint32_t CW = RW / 2;                 // chunk words
  static constexpr uint32_t DW = CW / 64;                // chunk dwords per lane
  static constexpr uint32_t HALF_BYTES = 4 * RW;         // two copies of RW u16 words
};
static_assert(kWavesPerGroup * 2 * 1 * RingGeom<1>::HALF_BYTES <= kRingBytes, "ring area");
static_assert(kWavesPerGroup * 2 * 2 * RingGeom<2>::HALF_BYTES <= kRingBytes, "ring area");

template <int NC>
struct HalfRing {          // wave-uniform state of one half's ring
  uint32_t rbase;          // LDS byte address of the ring
  uint32_t S2;             // LDS byte address of the next word to read
  uint32_t T2;             // commit when S2 >= T2
  uint32_t Qc;             // committed end (payload words)
  uint32_t base;           // payload word held at physical slot 0 (mod RW)
  uint32_t C0;             // first chunk start of the tile
  uint32_t Pend;           // end of the tile's payload window
};

template <int NC>
__device__ __forceinline__ void fetch(uint32_t* pend, __amdgpu_buffer_rsrc_t rsrc, uint32_t l,
                                      uint32_t start) {
#pragma unroll
  for (uint32_t k = 0; k < RingGeom<NC>::DW; k++)
    pend[k] = __builtin_amdgcn_raw_buffer_load_b32(rsrc, 2 * start + 4 * (l + 32 * k), 0, 0);
}

template <int NC>
__device__ __forceinline__ void commit_lanes(uint8_t* lds, const uint32_t* pend, uint32_t rbase,
                                             uint32_t slot0, uint32_t l) {
  constexpr uint32_t RW = RingGeom<NC>::RW;
#pragma unroll
  for (uint32_t k = 0; k < RingGeom<NC>::DW; k++) {
    const uint32_t a = rbase + 2 * (slot0 + 2 * (l + 32 * k));
    *reinterpret_cast<uint32_t*>(lds + a) = pend[k];
    *reinterpret_cast<uint32_t*>(lds + a + 2 * RW) = pend[k];
  }
}

// Commit the pending chunk of one half (lanes of that half write), advance the
// window, rebase the read address, and request the following chunk.
template <int NC>
__device__ __forceinline__ void commit_half(uint8_t* lds, HalfRing<NC>& R, uint32_t* pend,
                                            __amdgpu_buffer_rsrc_t rsrc, bool mine, uint32_t l) {
  constexpr uint32_t RW = RingGeom<NC>::RW, CW = RingGeom<NC>::CW;
  if (mine) commit_lanes<NC>(lds, pend, R.rbase, (R.Qc - R.C0) & (RW - 1), l);
  R.Qc += CW;
  R.T2 += 2 * CW;
  if (R.S2 - R.rbase >= 2 * RW) {
    R.S2 -= 2 * RW;
    R.T2 -= 2 * RW;
    R.base += RW;
  }
  if (mine && R.Qc < R.Pend) fetch<NC>(pend, rsrc, l, R.Qc);
}

template <int NC>
__device__ __forceinline__ void ring_start(uint8_t* lds, HalfRing<NC>& R, uint32_t* pend,
                                           __amdgpu_buffer_rsrc_t rsrc, bool mine, uint32_t l,
                                           uint32_t P0, uint32_t Pend, uint32_t rbase) {
  constexpr uint32_t RW = RingGeom<NC>::RW, CW = RingGeom<NC>::CW;
  R.rbase = rbase;
  R.C0 = P0 & ~(CW - 1);
  R.base = R.C0;
  R.Pend = Pend;
  R.S2 = rbase + 2 * (P0 - R.C0);
  if (mine) {
    fetch<NC>(pend, rsrc, l, R.C0);
    commit_lanes<NC>(lds, pend, rbase, 0, l);
    if (R.C0 + CW < Pend) {
      fetch<NC>(pend, rsrc, l, R.C0 + CW);
      commit_lanes<NC>(lds, pend, rbase, CW, l);
    }
  }
  R.Qc = R.C0 + RW;
  R.T2 = rbase + 2 * CW;
  if (mine && R.Qc < Pend) fetch<NC>(pend, rsrc, l, R.Qc);
}

// One refill step of one chain: 64-lane ballot of states below 2^15, words read
// from each half's ring in lane order, uniform pointers advanced, commits done.
template <int NC, bool FULL>
__device__ __forceinline__ void refill(uint32_t& x, bool act, uint64_t act_mask, HalfRing<NC>& A,
                                       HalfRing<NC>& Bh, uint8_t* lds, uint32_t* pend,
                                       __amdgpu_buffer_rsrc_t rsrc, uint32_t half, uint32_t l) {
  uint64_t m = __ballot(x < kStateLow);
  if (!FULL) m &= act_mask;
  const uint32_t lo = (uint32_t)m, hi = (uint32_t)(m >> 32);
  const uint32_t clo = (uint32_t)__builtin_popcount(lo), chi = (uint32_t)__builtin_popcount(hi);
  const uint32_t pre = __builtin_amdgcn_mbcnt_hi(hi, __builtin_amdgcn_mbcnt_lo(lo, 0u));
  const int32_t dd = (int32_t)((Bh.S2 - A.S2) >> 1) - (int32_t)clo;
  const uint32_t widx = (uint32_t)(__mul24((int32_t)half, dd) + (int32_t)pre);
  const uint32_t w = *reinterpret_cast<const uint16_t*>(lds + A.S2 + 2 * widx);
  const bool need = (FULL || act) && x < kStateLow;
  x = need ? ((x << 16) | w) : x;
  A.S2 += 2 * clo;
  Bh.S2 += 2 * chi;
  if (A.S2 >= A.T2) commit_half<NC>(lds, A, pend, rsrc, half == 0, l);
  if (Bh.S2 >= Bh.T2) commit_half<NC>(lds, Bh, pend, rsrc, half == 1, l);
}

// One field symbol.  Slot-table path: entry = lut[(8c + i - 1) * 2^B + u]; the
// coset part cb = 8c * 2^B is per lane, the field part a constant offset.
template <int PATH, int B>
__device__ __forceinline__ void decode_field(const Hot& L, const uint32_t* lds, int field,
                                             uint32_t cb, uint32_t c, uint32_t& x, int32_t& dval) {
  if (PATH == kPathLut) {
    constexpr uint32_t M = 1u << B;
    const uint32_t u = x & (M - 1);
    const uint32_t e = lds[cb + u + (uint32_t)(field - 1) * M];
    x = __umul24(e & 0xFFFu, x >> B) + ((e >> 12) & 0x7FFu);
    dval = 2 * ((int32_t)e >> 24) + (int32_t)c;
  } else if (PATH == kPathWide) {
    constexpr uint32_t M = 1u << B;
    const uint32_t u = x & (M - 1);
    const uint32_t e = lds[cb + u + (uint32_t)(field - 1) * M];
    const uint32_t g = x >> B;
    x = __umul24(e & 0x7FFu, g) + g + ((e >> 11) & 0x7FFu);   // (f - 1) g + g + (u - F)
    dval = 2 * ((int32_t)e >> 22) + (int32_t)c;
  } else if (PATH == kPathGlobal) {
    // Coarse search: C_j = F_{jG} of table t in LDS (C_0 = 0 <= u), the largest j
    // with C_j <= u, then a scan of the block's frequencies f_{jG} .. f_{jG+G-1},
    // two per dword, from the blob's table in global memory.  The block holds the
    // symbol (its successor's C exceeds u, or it is the last block, whose
    // frequencies run up to 2^b), so the scan ends inside it.
    const uint16_t* cum = reinterpret_cast<const uint16_t*>(lds);
    const uint32_t u = x & ((1u << L.b) - 1);
    const uint32_t t = 8 * c + (uint32_t)(field - 1);
    const uint32_t base = lds[L.g_meta + t], n = lds[L.g_meta + 32 + t];
    uint32_t lo = 0, hi = n ? n - 1 : 0;
    while (lo < hi) {
      const uint32_t mid = (lo + hi + 1) >> 1;
      if (cum[base + mid] <= u) lo = mid;
      else hi = mid - 1;
    }
    uint32_t F = cum[base + lo], s = lo << L.g_bits, f = 0;
    const __amdgpu_buffer_rsrc_t trsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(L.blob), (short)0, (int)L.tab_bytes, 0x00020000);
    const uint32_t off = lds[L.g_meta + 48 + t] + 2 * s;
    for (uint32_t k = 0; k < (1u << L.g_bits); k += 2) {
      const uint32_t w = __builtin_amdgcn_raw_buffer_load_b32(trsrc, off + 2 * k, 0, 0);
      const uint32_t f0 = w & 0xFFFFu, f1 = w >> 16;
      if (u < F + f0) {
        f = f0;
        s += k;
        break;
      }
      F += f0;
      if (u < F + f1) {
        f = f1;
        s += k + 1;
        break;
      }
      F += f1;
    }
    x = __umul24(f, x >> L.b) + u - F;
    dval = doubled_value((int32_t)s + (int32_t)lds[L.g_meta + 16 + t], field, c);
  } else {
    // Bucketed search: the bucket j of u (its top k bits) bounds the symbol to
    // [bk[j], bk[j + 1]]; a binary search on the u16 cumulative table narrows
    // it (nothing to search when buckets are single slots).
    const uint16_t* cum = reinterpret_cast<const uint16_t*>(lds);
    const uint32_t u = x & ((1u << L.b) - 1);
    const uint32_t t = 8 * c + (uint32_t)(field - 1);
    const uint32_t base = lds[L.meta + t];
    const uint16_t* bk = cum + L.bucket + t * L.bucket_n1;
    const uint32_t j = u >> L.bucket_shift;
    uint32_t lo = bk[j], hi = L.bucket_shift ? bk[j + 1] : lo;
    while (lo < hi) {
      const uint32_t mid = (lo + hi + 1) >> 1;
      if (cum[base + mid] <= u) lo = mid;
      else hi = mid - 1;
    }
    const uint32_t F = cum[base + lo], Fn = cum[base + lo + 1];
    x = __umul24(Fn - F, x >> L.b) + u - F;
    dval = doubled_value((int32_t)lo + (int32_t)lds[L.meta + 16 + t], field, c);
  }
}

// floor(v / (C/8)) with the host-computed magic (Granlund-Montgomery).
__device__ __forceinline__ uint32_t row_of(const Hot& L, uint32_t v) {
  if (L.div_pow2) return v >> L.div_shift;
  const uint32_t q = __umulhi(v, L.div_magic);
  return (q + ((v - q) >> 1)) >> L.div_shift;
}

template <int PATH, int B, int NC, bool FULL, bool DOT = false>
__device__ __forceinline__ void decode_task(const Hot& L, const uint32_t* tab, uint8_t* lds,
                            uint32_t ring_area, uint32_t task, int32_t* status) {
  const uint32_t lane = threadIdx.x & 63, wave = wave_id();
  const uint32_t half = lane >> 5, l = lane & 31;
  const uint32_t nvec = L.rows * L.cvec;
  const EP_GLOBAL uint32_t* states = gptr<const uint32_t>(L.blob + L.off_states);
  const EP_GLOBAL uint32_t* offs = gptr<const uint32_t>(L.blob + L.off_offsets);
  const EP_GLOBAL float* sigma = gptr<const float>(L.blob + L.off_sigma);
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(L.blob + L.off_payload), (short)0, (int)L.pay_bytes, 0x00020000);
  const uint32_t mask = (1u << L.b) - 1;

  uint32_t x[NC], v0[NC], n_l[NC], pend[NC][RingGeom<NC>::DW];
  uint64_t am[NC];
  HalfRing<NC> RA[NC], RB[NC];
  uint32_t rounds = 0;
#pragma unroll
  for (int j = 0; j < NC; j++) {
    const uint32_t tA = L.tile_begin + 2 * (NC * task + j);      // uniform
    const uint32_t tB = tA + 1;
    const bool okA = tA < L.tile_end, okB = tB < L.tile_end;   // uniform
    const uint32_t tile = half ? tB : tA;
    const bool ok = half ? okB : okA;
    v0[j] = ok ? tile * L.V : 0;
    const uint32_t nv = ok ? min(L.V, nvec - v0[j]) : 0;
    n_l[j] = l < nv ? (nv - 1 - l) / 32 + 1 : 0;
    const uint32_t nvA = okA ? min(L.V, nvec - tA * L.V) : 0;
    const uint32_t nvB = okB ? min(L.V, nvec - tB * L.V) : 0;
    rounds = max(rounds, (max(nvA, nvB) + 31) / 32);
    x[j] = ok ? states[(uint64_t)tile * 32 + l] : kStateLow;
    const uint32_t rb = ring_area + (wave * NC + j) * 2 * RingGeom<NC>::HALF_BYTES;
    const uint32_t pa0 = okA ? offs[tA] : 0, pa1 = okA ? offs[tA + 1] : 0;
    const uint32_t pb0 = okB ? offs[tB] : 0, pb1 = okB ? offs[tB + 1] : 0;
    ring_start<NC>(lds, RA[j], pend[j], rsrc, half == 0 && okA, l, pa0, pa1, rb);
    ring_start<NC>(lds, RB[j], pend[j], rsrc, half == 1 && okB, l, pb0, pb1,
                   rb + RingGeom<NC>::HALF_BYTES);
  }

  for (uint32_t k = 0; k < rounds; k++) {
    uint32_t c[NC], cb[NC], v[NC];
    float sg[NC];
    bool act[NC];
    int32_t d[NC][9];
#pragma unroll
    for (int j = 0; j < NC; j++) {
      act[j] = FULL || k < n_l[j];
      am[j] = FULL ? ~0ull : __ballot(act[j]);
      v[j] = v0[j] + l + 32 * k;
      sg[j] = act[j] ? sigma[row_of(L, v[j])] : 0.0f;
      c[j] = 0;
      cb[j] = 0;
      if (act[j]) {   // coset symbol
        const uint32_t u = x[j] & mask;
        c[j] = u >= L.coset_f0 ? 1u : 0u;
        const uint32_t f = c[j] ? L.coset_f1 : L.coset_f0;
        const uint32_t F = c[j] ? L.coset_f0 : 0u;
        x[j] = __umul24(f, x[j] >> L.b) + u - F;
        cb[j] = c[j] << (L.b + 3);
      }
    }
#pragma unroll
    for (int j = 0; j < NC; j++)
      refill<NC, FULL>(x[j], act[j], am[j], RA[j], RB[j], lds, pend[j], rsrc, half, l);
#pragma unroll
    for (int i = 1; i <= 8; i++) {
#pragma unroll
      for (int j = 0; j < NC; j++)
        if (act[j]) decode_field<PATH, B>(L, tab, i, cb[j], c[j], x[j], d[j][i]);
#pragma unroll
      for (int j = 0; j < NC; j++)
        refill<NC, FULL>(x[j], act[j], am[j], RA[j], RB[j], lds, pend[j], rsrc, half, l);
    }
#pragma unroll
    for (int j = 0; j < NC; j++) {
      if (act[j]) {
        // field inverse: 2p_i = 2 z_i + c; 2p_8 = 4m + c + 2 pi, pi = sum z_1..7 mod 2
        int32_t p2[8];
        int32_t acc = (int32_t)c[j];
#pragma unroll
        for (int i = 1; i <= 7; i++) {
          p2[i - 1] = d[j][i];
          acc += d[j][i];
        }
        p2[7] = d[j][8] | (acc & 2);
        store_vector<DOT>(L, v[j], p2, 0.5f * sg[j]);
      }
    }
  }

  uint32_t err = 0;
#pragma unroll
  for (int j = 0; j < NC; j++) {
    const uint32_t tile = L.tile_begin + 2 * (NC * task + j) + half;
    if (tile < L.tile_end) {
      if (x[j] != kStateLow) err |= EP_STATUS_BAD_FINAL_STATE;
      const HalfRing<NC>& R = half ? RB[j] : RA[j];
      const uint32_t P = R.base + (R.S2 - R.rbase) / 2;
      if (l == 0 && P != R.Pend) err |= P > R.Pend ? EP_STATUS_PAYLOAD_OVERRUN : EP_STATUS_BAD_END_OFFSET;
      if (L.container && L.dequant) {
        const EP_GLOBAL float* delta = gptr<const float>(L.blob + L.off_delta);
        const uint32_t nv = min(L.V, nvec - v0[j]);
        const uint32_t r_first = (v0[j] + L.cvec - 1) / L.cvec;
        const uint32_t r_last = (v0[j] + nv - 1) / L.cvec;
        for (uint32_t r = r_first + l; r <= r_last; r += 32) gptr<float>(L.dequant)[r] = delta[r];
      }
    }
  }
  if (err && status) atomicOr(status, (int32_t)err);
}

// ---- steady state of the bucketed-search path: full four-tile tasks, two chains ---
// Payload staging.  Each half (one tile's stream) owns a 512-byte ring in LDS
// (256 words) that is addressed modulo its size, so a step's reads need no
// second copy of the ring.  Words arrive in 128-word blocks, one dwordx2 per
// lane of the half: a block is requested into registers (pend) and committed
// to the ring at a later symbol round, once the ring has room for it.  The
// output of a round waits for the global loads in flight, so a block requested
// at the start of a round has landed by the start of the next one; there is no
// other wait on global memory in the loop.  Between commits the reads of a
// step stay inside committed words: a step reads at most 32 words per half,
// and the committed margin is restored to >= 128 words at the start of a
// round and to >= 96 words after steps 3 and 6.
constexpr uint32_t kFastRingBytes = 512;
constexpr uint32_t kFastRingWords = kFastRingBytes / 2;
constexpr uint32_t kFastBlockWords = 128;
constexpr uint32_t kFastChainBytes = 2 * kFastRingBytes;
constexpr uint32_t kFastOob = 0x80000000u;   // buffer offset past any payload section
constexpr uint32_t kPinnedState = 0x7FFFFFFFu; // a state that takes no refill for one symbol
static_assert(kWavesPerGroup * 2 * kFastChainBytes <= kRingBytes, "fast ring area");
static_assert(search_layout(11, 0).total % kFastRingBytes == 0 &&
                  search_layout(12, 12345).total % kFastRingBytes == 0 &&
                  (64u << 9) % kFastRingBytes == 0,
              "ring areas start on a ring-size boundary (rings are addressed as base | offset)");

struct FastChain {     // wave-uniform, in payload words
  uint32_t OA, D;      // read position of half A, from the first block of its stream, and
                       // the read position of half B (same origin for B) minus OA
  uint32_t QA, QB;     // committed end, same origin
  uint32_t CA, CB;     // payload word index of that first block
  uint32_t EA, EB;     // end of each tile's stream, same origin as CA / CB
};

// Commit the staged block of half A (lanes 0-31, registers pendA) if its
// margin is below `limit`, and request its next block; likewise half B (lanes
// 32-63, pendB).  The positions stay wave-uniform (scalar registers); only the
// commit and the request are per lane.  Separate staging registers per half
// keep a commit of one half from waiting for the other half's request.
__device__ __forceinline__ void fast_stage(FastChain& F, u32x2& pendA, u32x2& pendB, uint8_t* lds,
                                           uint32_t vrb8,
                                           uint32_t vl8, __amdgpu_buffer_rsrc_t rsrc,
                                           uint32_t half, uint32_t limit) {
  const bool cA = uni(F.QA - F.OA) < limit, cB = uni(F.QB - F.OA - F.D) < limit;
  if (cA || cB) {
    if (cA && half == 0) {
      *reinterpret_cast<u32x2*>(lds + vrb8 + 2 * (F.QA & (kFastRingWords - 1))) = pendA;
      const uint32_t a = F.QA + kFastBlockWords;
      pendA = __builtin_amdgcn_raw_buffer_load_b64(
          rsrc, uni(a < F.EA ? 2 * (F.CA + a) : kFastOob) + vl8, 0, 0);
    }
    if (cB && half == 1) {
      *reinterpret_cast<u32x2*>(lds + vrb8 + 2 * (F.QB & (kFastRingWords - 1))) = pendB;
      const uint32_t a = F.QB + kFastBlockWords;
      pendB = __builtin_amdgcn_raw_buffer_load_b64(
          rsrc, uni(a < F.EB ? 2 * (F.CB + a) : kFastOob) + vl8, 0, 0);
    }
    F.QA = uni(F.QA + (cA ? kFastBlockWords : 0u));
    F.QB = uni(F.QB + (cB ? kFastBlockWords : 0u));
  }
}

// The same refill in plain code, for the search path's steady state.
__device__ __forceinline__ void refill_staged(uint32_t& x, uint32_t& SA, uint32_t& D,
                                              const uint8_t* lds, uint32_t vrb, uint32_t vH) {
  const uint64_t m = __ballot(x < kStateLow);
  const uint32_t lo = (uint32_t)m, hi = (uint32_t)(m >> 32);
  const uint32_t clo = uni((uint32_t)__builtin_popcount(lo));
  const uint32_t chi = uni((uint32_t)__builtin_popcount(hi));
  const uint32_t pre = __builtin_amdgcn_mbcnt_hi(hi, __builtin_amdgcn_mbcnt_lo(lo, 0u));
  const int32_t dd = (int32_t)D - (int32_t)clo;
  const uint32_t idx = (uint32_t)(__mul24((int32_t)vH, dd) + (int32_t)pre);
  const uint32_t a = vrb | (((idx + SA) << 1) & (kFastRingBytes - 1));
  const uint32_t w = *reinterpret_cast<const uint16_t*>(lds + a);
  if (x < kStateLow) x = (x << 16) | w;
  SA = uni(SA + clo);
  D = uni((uint32_t)dd + chi);
}

// Coset and field steps of the search path for both chains (plain code).
__device__ __forceinline__ void coset_step_search(const Hot& L, uint32_t* x, uint32_t* c,
                                                  FastChain& F0, FastChain& F1, const uint8_t* lds,
                                                  uint32_t vrb0, uint32_t vrb1, uint32_t vH) {
  const uint32_t mask = (1u << L.b) - 1;
#pragma unroll
  for (int j = 0; j < 2; j++) {
    const uint32_t u = x[j] & mask;
    c[j] = u >= L.coset_f0 ? 1u : 0u;
    const uint32_t f = c[j] ? L.coset_f1 : L.coset_f0;
    const uint32_t F = c[j] ? L.coset_f0 : 0u;
    x[j] = __umul24(f, x[j] >> L.b) + u - F;
  }
  refill_staged(x[0], F0.OA, F0.D, lds, vrb0, vH);
  refill_staged(x[1], F1.OA, F1.D, lds, vrb1, vH);
}

template <int FIELD>
__device__ __forceinline__ void field_step_search(const Hot& L, const uint32_t* tab, uint32_t* x,
                                                  const uint32_t* c, int32_t (*d)[9], FastChain& F0,
                                                  FastChain& F1, const uint8_t* lds, uint32_t vrb0,
                                                  uint32_t vrb1, uint32_t vH) {
#pragma unroll
  for (int j = 0; j < 2; j++) decode_field<kPathSearch, 0>(L, tab, FIELD, 0, c[j], x[j], d[j][FIELD]);
  refill_staged(x[0], F0.OA, F0.D, lds, vrb0, vH);
  refill_staged(x[1], F1.OA, F1.D, lds, vrb1, vH);
}

// Set up one chain (tiles tA on lanes 0-31, tA + 1 on lanes 32-63) from the
// word offsets pA0..pA1 and pB0..pB1 of the two streams: request the first two
// blocks of each stream (returned, for the ring) and the third (into pend).
// Minimum of two wave-uniform values on the scalar unit (left to itself the
// compiler computes it on the vector unit and reads the result back).
__device__ __forceinline__ uint32_t smin(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("s_min_u32 %0, %1, %2" : "=s"(r) : "s"(a), "s"(b));
  return r;
}

// Both chains' staging at one point of the round: a single scalar test of the
// smallest of the four margins skips the per-half work when no half needs it
// (the common case: at typical rates a half consumes well under a block per
// round).
__device__ __forceinline__ void fast_stage_both(FastChain& F0, FastChain& F1, u32x2& pendA0,
                                                u32x2& pendB0, u32x2& pendA1, u32x2& pendB1,
                                                uint8_t* lds, uint32_t vrb08, uint32_t vrb18,
                                                uint32_t vl8, __amdgpu_buffer_rsrc_t rsrc,
                                                uint32_t half, uint32_t limit) {
  const uint32_t m = smin(smin(F0.QA - F0.OA, F0.QB - F0.OA - F0.D),
                          smin(F1.QA - F1.OA, F1.QB - F1.OA - F1.D));
  if (__builtin_expect(m < limit, 0)) {
    fast_stage(F0, pendA0, pendB0, lds, vrb08, vl8, rsrc, half, limit);
    fast_stage(F1, pendA1, pendB1, lds, vrb18, vl8, rsrc, half, limit);
  }
}

__device__ __forceinline__ u32x4 fast_start(FastChain& F, u32x2& pend, __amdgpu_buffer_rsrc_t rsrc,
                                            uint32_t half, uint32_t l, uint32_t pA0, uint32_t pA1,
                                            uint32_t pB0, uint32_t pB1) {
  F.CA = pA0 & ~(kFastBlockWords - 1);
  F.CB = pB0 & ~(kFastBlockWords - 1);
  F.OA = pA0 - F.CA;
  F.D = (pB0 - F.CB) - F.OA;
  F.QA = F.QB = kFastRingWords;
  F.EA = pA1 - F.CA;
  F.EB = pB1 - F.CB;
  const uint32_t c = half ? F.CB : F.CA, e = half ? F.EB : F.EA;
  const u32x4 first = __builtin_amdgcn_raw_buffer_load_b128(rsrc, 2 * c + 16 * l, 0, 0);
  pend = __builtin_amdgcn_raw_buffer_load_b64(
      rsrc, (kFastRingWords < e ? 2 * (c + kFastRingWords) : kFastOob) + 8 * l, 0, 0);
  return first;
}

// The steady-state task of the search path: four full tiles (two chains),
// output type DT.
template <int PATH, int B, int DT, bool SAT>
__device__ __forceinline__ void decode_task_fast(const Hot& L, uint8_t* lds, uint32_t ring_area,
                                                 uint32_t task, int32_t* status) {
  const uint32_t* tab = reinterpret_cast<const uint32_t*>(lds);
  const uint32_t lane = threadIdx.x & 63, wave = wave_id();
  const uint32_t half = lane >> 5, l = lane & 31;
  const EP_GLOBAL uint32_t* states = gptr<const uint32_t>(L.blob + L.off_states);
  const EP_GLOBAL uint32_t* offs = gptr<const uint32_t>(L.blob + L.off_offsets);
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(L.blob + L.off_payload), (short)0, (int)L.pay_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t srsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(L.blob + L.off_sigma), (short)0, (int)(4 * L.rows), 0x00020000);

  const uint32_t t0 = L.tile_begin + 4 * task;      // tiles t0 .. t0 + 3, all full
  const uint32_t vrb0 = ring_area + wave * 2 * kFastChainBytes + half * kFastRingBytes;
  const uint32_t vrb1 = vrb0 + kFastChainBytes;
  const uint32_t vl8 = 8 * l;
  // Tile offsets, states and the first blocks are all requested before the
  // one wait below.
  uint32_t o[5];
#pragma unroll
  for (int i = 0; i < 5; i++) o[i] = offs[t0 + i];
  uint32_t x[2], v0[2], row[2], col[2];
#pragma unroll
  for (int j = 0; j < 2; j++) {
    const uint32_t tile = t0 + 2 * j + half;
    v0[j] = tile * L.V;
    x[j] = states[(uint64_t)tile * 32 + l];
    const uint32_t vv = v0[j] + l;
    row[j] = row_of(L, vv);
    col[j] = vv - row[j] * L.cvec;
  }
  FastChain F0, F1;
  u32x2 pend0, pend1, pendB0, pendB1;
#pragma unroll
  for (int i = 0; i < 5; i++) o[i] = uni(o[i]);
  const u32x4 fill0 = fast_start(F0, pend0, rsrc, half, l, o[0], o[1], o[1], o[2]);
  const u32x4 fill1 = fast_start(F1, pend1, rsrc, half, l, o[2], o[3], o[3], o[4]);
  // One wait for everything requested so far, so that no load is in flight
  // when the loop starts (the loop's own waits then stay one round behind).
  __builtin_amdgcn_s_waitcnt(0);
  *reinterpret_cast<u32x4*>(lds + vrb0 + 16 * l) = fill0;
  *reinterpret_cast<u32x4*>(lds + vrb1 + 16 * l) = fill1;
  pendB0 = pend0;   // pend* serve lanes 0-31, pendB* lanes 32-63
  pendB1 = pend1;

  const uint32_t vH = half;
  const uint32_t rounds = L.V / 32;
  const bool wide = L.cvec >= 32;
  const uint32_t vrb08 = vrb0 + vl8, vrb18 = vrb1 + vl8;

  for (uint32_t k = 0; k < rounds; k++) {
    // room for a block: margin <= ring - block
    fast_stage_both(F0, F1, pend0, pendB0, pend1, pendB1, lds, vrb08, vrb18, vl8, rsrc, half,
                    kFastRingWords - kFastBlockWords + 1);
    float sg[2];
#pragma unroll
    for (int j = 0; j < 2; j++)
      sg[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(srsrc, 4 * row[j], 0, 0));
    uint32_t c[2];
    int32_t d[2][9];
    coset_step_search(L, x, c, F0, F1, lds, vrb0, vrb1, vH);
#define EP_FIELD(I) field_step_search<I>(L, tab, x, c, d, F0, F1, lds, vrb0, vrb1, vH);
    EP_FIELD(1) EP_FIELD(2)
    fast_stage_both(F0, F1, pend0, pendB0, pend1, pendB1, lds, vrb08, vrb18, vl8, rsrc, half, 3 * 32);
    EP_FIELD(3) EP_FIELD(4) EP_FIELD(5)
    fast_stage_both(F0, F1, pend0, pendB0, pend1, pendB1, lds, vrb08, vrb18, vl8, rsrc, half, 3 * 32);
    EP_FIELD(6) EP_FIELD(7) EP_FIELD(8)
#undef EP_FIELD
#pragma unroll
    for (int j = 0; j < 2; j++) {
      int32_t p2[8];
      int32_t acc = (int32_t)c[j];
#pragma unroll
      for (int i = 1; i <= 7; i++) {
        p2[i - 1] = d[j][i];
        acc += d[j][i];
      }
      p2[7] = d[j][8] | (acc & 2);
      if constexpr (DT == kOutDotI8) dot_vec(L, v0[j] + l + 32 * k, p2, 0.5f * sg[j]);
      else store_vec<DT, SAT>(L.out, v0[j] + l + 32 * k, p2, 0.5f * sg[j]);
      // next vector of this lane: 32 vectors further
      if (wide) {
        col[j] += 32;
        if (col[j] >= L.cvec) {
          col[j] -= L.cvec;
          row[j] += 1;
        }
      } else {
        row[j] = row_of(L, v0[j] + l + 32 * (k + 1));
      }
    }
  }

  uint32_t err = 0;
#pragma unroll
  for (int j = 0; j < 2; j++) {
    if (x[j] != kStateLow) err |= EP_STATUS_BAD_FINAL_STATE;
    const FastChain& F = j ? F1 : F0;
    const uint32_t P = half ? F.OA + F.D : F.OA, E = half ? F.EB : F.EA;
    if (l == 0 && P != E) err |= P > E ? EP_STATUS_PAYLOAD_OVERRUN : EP_STATUS_BAD_END_OFFSET;
    if (L.container && L.dequant) {
      const EP_GLOBAL float* delta = gptr<const float>(L.blob + L.off_delta);
      const uint32_t r_first = (v0[j] + L.cvec - 1) / L.cvec;
      const uint32_t r_last = (v0[j] + L.V - 1) / L.cvec;
      for (uint32_t r = r_first + l; r <= r_last; r += 32) gptr<float>(L.dequant)[r] = delta[r];
    }
  }
  if (err && status) atomicOr(status, (int32_t)err);
}

// ---- hand-scheduled steady state of the slot-table path: full tasks, two chains -------
// Same staging as the search path's steady state (512-byte rings, 128-word
// blocks, commits at a round's start and after steps 3 and 6).  One symbol
// step of both chains: chain 0's refill ballot lives in VCC, chain 1's in
// s[94:95] (clobbered), so the two refills interleave instruction by
// instruction.  Per chain: 64-lane ballot of states below 2^15, per-half word
// index from v_mbcnt (upper-half lanes corrected by the distance between the
// two read positions less the lower half's count, dd = D - popcount(lower
// half), where the chain keeps D = SB - SA in place of SB), the ring read at
// byte vrb | (2 (SA + index) mod 512), the scalar advance SA += popcount(lower),
// D = dd + popcount(upper), and the merge x = x << 16 | w on the refilling
// lanes only (EXEC narrowed to each chain's ballot, then restored).  The wave's
// issue priority drops back to 0 once both ring reads are in flight (a field
// step raises it while its table entries are in hand).  WORK is independent
// vector work placed in the wait for the ring words.
#define EP_REFILL_BOTH_W(WORK)                                              \
  "v_cmp_gt_u32_e32 vcc, 0x8000, %[x0]\n\t"                                 \
  "v_cmp_gt_u32_e64 s[94:95], %[k15], %[x1]\n\t"                            \
  "s_bcnt1_i32_b32 %[c0lo], vcc_lo\n\t"                                    \
  "v_mbcnt_lo_u32_b32 %[t0], vcc_lo, 0\n\t"                                 \
  "s_bcnt1_i32_b32 %[c0hi], vcc_hi\n\t"                                    \
  "v_mbcnt_lo_u32_b32 %[t1], s94, 0\n\t"                                    \
  "v_mbcnt_hi_u32_b32 %[t0], vcc_hi, %[t0]\n\t"                             \
  "s_sub_u32 %[d0], %[D0], %[c0lo]\n\t"                                    \
  "v_mbcnt_hi_u32_b32 %[t1], s95, %[t1]\n\t"                                \
  "s_bcnt1_i32_b32 %[c1lo], s94\n\t"                                       \
  "v_mad_i32_i24 %[t0], %[vH], %[d0], %[t0]\n\t"                            \
  "s_bcnt1_i32_b32 %[c1hi], s95\n\t"                                       \
  "v_add_lshl_u32 %[t0], %[t0], %[SA0], 1\n\t"                              \
  "v_and_or_b32 %[t0], %[t0], %[rmask], %[vrb0]\n\t"                        \
  "s_sub_u32 %[d1], %[D1], %[c1lo]\n\t"                                    \
  "ds_read_u16 %[w0], %[t0]\n\t"                                            \
  "v_mad_i32_i24 %[t1], %[vH], %[d1], %[t1]\n\t"                            \
  "s_add_u32 %[SA0], %[SA0], %[c0lo]\n\t"                                  \
  "v_add_lshl_u32 %[t1], %[t1], %[SA1], 1\n\t"                              \
  "s_add_u32 %[D0], %[d0], %[c0hi]\n\t"                                  \
  "v_and_or_b32 %[t1], %[t1], %[rmask], %[vrb1]\n\t"                        \
  "s_add_u32 %[SA1], %[SA1], %[c1lo]\n\t"                                  \
  "ds_read_u16 %[w1], %[t1]\n\t"                                            \
  "s_setprio 0\n\t"                                                        \
  "s_add_u32 %[D1], %[d1], %[c1hi]\n\t"                                  \
  WORK                                                                     \
  "s_and_saveexec_b64 %[ex], vcc\n\t"                                       \
  "s_waitcnt lgkmcnt(1)\n\t"                                                \
  "v_lshl_or_b32 %[x0], %[x0], 16, %[w0]\n\t"                               \
  "s_and_b64 exec, %[ex], s[94:95]\n\t"                                     \
  "s_waitcnt lgkmcnt(0)\n\t"                                                \
  "v_lshl_or_b32 %[x1], %[x1], 16, %[w1]\n\t"                               \
  "s_mov_b64 exec, %[ex]\n\t"

#define EP_REFILL_BOTH EP_REFILL_BOTH_W("")

#define EP_STEP_OUTS                                                                      \
  [x0] "+v"(x0), [x1] "+v"(x1), [SA0] "+s"(F0.OA), [D0] "+s"(F0.D), [SA1] "+s"(F1.OA),  \
      [D1] "+s"(F1.D), [u0] "=&v"(u0), [u1] "=&v"(u1), [g0] "=&v"(g0), [g1] "=&v"(g1),  \
      [t0] "=&v"(t0), [t1] "=&v"(t1), [w0] "=&v"(w0), [w1] "=&v"(w1),                     \
      [c0lo] "=&s"(c0lo), [c0hi] "=&s"(c0hi), [c1lo] "=&s"(c1lo), [c1hi] "=&s"(c1hi),     \
      [d0] "=&s"(dd0), [d1] "=&s"(dd1), [ex] "=&s"(ex)

#define EP_STEP_TEMPS                                                                     \
  uint32_t u0, u1, g0, g1, t0, t1, w0, w1, c0lo, c0hi, c1lo, c1hi, dd0, dd1;             \
  uint64_t ex

#define EP_STEP_INS                                                                          \
  [vH] "v"(vH), [vrb0] "v"(vrb0), [vrb1] "v"(vrb1), [rmask] "s"(kFastRingBytes - 1),         \
      [k15] "s"(kStateLow), [mk] "i"((1 << B) - 1), [b] "i"(B)

#define EP_STEP_CLOBBERS "vcc", "scc", "exec", "s94", "s95", "memory"

// Field symbol (table 8c + FIELD - 1, entry at byte cb + 4u + (FIELD - 1) 4 * 2^B)
// for both chains, then the refill; e0, e1 receive the slot entries, kept for the
// reconstruction.  Chain 0's decode starts as soon as its own table read
// returns.  From then until the ring reads are issued the wave runs at raised
// issue priority: the dependent ALU chain of a wave whose table reads have
// landed goes ahead of waves that are still waiting, which shortens every
// wave's step latency.
//
// While the ring words are in flight the step turns its own entries into
// weights (YM = 1: y = fma(sg, z, hc); YM = 2: also clamped to [-m, m]; YM = 0:
// nothing), z being the entry's top byte (top 10 bits for wide entries).  For
// field 8 the parity bit of z_1 + ... + z_7 (the low bit of z in X) is first
// merged into the entry.
#define EP_Y_CVT                                                                      \
  "v_cvt_f32_i32_sdwa %[y0], sext(%[e0]) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n\t" \
  "v_cvt_f32_i32_sdwa %[y1], sext(%[e1]) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n\t" \
  "v_fma_f32 %[y0], %[sg0], %[y0], %[hc0]\n\t"                                        \
  "v_fma_f32 %[y1], %[sg1], %[y1], %[hc1]\n\t"
#define EP_Y_CVT_WIDE                                                                 \
  "v_ashrrev_i32 %[y0], 22, %[e0]\n\t"                                                \
  "v_ashrrev_i32 %[y1], 22, %[e1]\n\t"                                                \
  "v_cvt_f32_i32_e32 %[y0], %[y0]\n\t"                                                \
  "v_cvt_f32_i32_e32 %[y1], %[y1]\n\t"                                                \
  "v_fma_f32 %[y0], %[sg0], %[y0], %[hc0]\n\t"                                        \
  "v_fma_f32 %[y1], %[sg1], %[y1], %[hc1]\n\t"
#define EP_Y_SAT                                                                      \
  "v_med3_f32 %[y0], %[y0], %[nm], %[m]\n\t"                                          \
  "v_med3_f32 %[y1], %[y1], %[nm], %[m]\n\t"
#define EP_Y_PAR                                                                      \
  "v_and_or_b32 %[e0], %[X0], %[bit], %[e0]\n\t"                                      \
  "v_and_or_b32 %[e1], %[X1], %[bit], %[e1]\n\t"
// x = f (x >> b) + (u - F) from a narrow entry, chain j
#define EP_DEC(j)                                                                     \
  "v_and_b32 %[u" #j "], 0xfff, %[e" #j "]\n\t"                                        \
  "v_bfe_u32 %[t" #j "], %[e" #j "], 12, 11\n\t"                                       \
  "v_mad_u32_u24 %[x" #j "], %[u" #j "], %[g" #j "], %[t" #j "]\n\t"
// the same from a wide entry: (f - 1) (x >> b) + (x >> b) + (u - F)
#define EP_DEC_WIDE(j)                                                                \
  "v_and_b32 %[u" #j "], 0x7ff, %[e" #j "]\n\t"                                        \
  "v_bfe_u32 %[t" #j "], %[e" #j "], 11, 11\n\t"                                       \
  "v_add_u32_e32 %[t" #j "], %[g" #j "], %[t" #j "]\n\t"                                \
  "v_mad_u32_u24 %[x" #j "], %[u" #j "], %[g" #j "], %[t" #j "]\n\t"

#define EP_FIELD_ASM(DEC0, DEC1, WORK)                                                   \
  asm volatile(                                                                          \
      "v_and_b32 %[u0], %[mk], %[x0]\n\t"                                                \
      "v_and_b32 %[u1], %[mk], %[x1]\n\t"                                                \
      "v_lshl_add_u32 %[u0], %[u0], 2, %[cb0]\n\t"                                       \
      "v_lshl_add_u32 %[u1], %[u1], 2, %[cb1]\n\t"                                       \
      "ds_read_b32 %[e0], %[u0] offset:%[off]\n\t"                                       \
      "ds_read_b32 %[e1], %[u1] offset:%[off]\n\t"                                       \
      "v_lshrrev_b32 %[g0], %[b], %[x0]\n\t"                                             \
      "v_lshrrev_b32 %[g1], %[b], %[x1]\n\t"                                             \
      "s_waitcnt lgkmcnt(1)\n\t"                                                         \
      "s_setprio 2\n\t"                                                                  \
      DEC0                                                                               \
      "s_waitcnt lgkmcnt(0)\n\t"                                                         \
      DEC1                                                                               \
      EP_REFILL_BOTH_W(WORK)                                                             \
      : EP_STEP_OUTS, [e0] "=&v"(e0), [e1] "=&v"(e1), [y0] "=&v"(y0), [y1] "=&v"(y1)     \
      : [cb0] "v"(cb0), [cb1] "v"(cb1), [off] "i"((FIELD - 1) * (4 << B)), [sg0] "v"(sg0), \
        [sg1] "v"(sg1), [hc0] "v"(hc0), [hc1] "v"(hc1), [m] "s"(m), [nm] "v"(-m),        \
        [X0] "v"(X0), [X1] "v"(X1), [bit] "s"(zbit), EP_STEP_INS                         \
      : EP_STEP_CLOBBERS)

template <int B, int FIELD, int YM, bool WIDE>
__device__ __forceinline__ void field_step2(uint32_t& x0, uint32_t& x1, uint32_t cb0, uint32_t cb1,
                                            uint32_t& e0, uint32_t& e1, float& y0, float& y1,
                                            float sg0, float sg1, float hc0, float hc1,
                                            uint32_t X0, uint32_t X1, float m, FastChain& F0,
                                            FastChain& F1, uint32_t vH, uint32_t vrb0, uint32_t vrb1) {
  EP_STEP_TEMPS;
  const uint32_t zbit = 1u << (WIDE ? 22 : 24);   // low bit of the entry's z
  if constexpr (WIDE) {
    if constexpr (YM == 0) EP_FIELD_ASM(EP_DEC_WIDE(0), EP_DEC_WIDE(1), "");
    else if constexpr (FIELD == 8 && YM == 1) EP_FIELD_ASM(EP_DEC_WIDE(0), EP_DEC_WIDE(1), EP_Y_PAR EP_Y_CVT_WIDE);
    else if constexpr (FIELD == 8) EP_FIELD_ASM(EP_DEC_WIDE(0), EP_DEC_WIDE(1), EP_Y_PAR EP_Y_CVT_WIDE EP_Y_SAT);
    else if constexpr (YM == 1) EP_FIELD_ASM(EP_DEC_WIDE(0), EP_DEC_WIDE(1), EP_Y_CVT_WIDE);
    else EP_FIELD_ASM(EP_DEC_WIDE(0), EP_DEC_WIDE(1), EP_Y_CVT_WIDE EP_Y_SAT);
  } else {
    if constexpr (YM == 0) EP_FIELD_ASM(EP_DEC(0), EP_DEC(1), "");
    else if constexpr (FIELD == 8 && YM == 1) EP_FIELD_ASM(EP_DEC(0), EP_DEC(1), EP_Y_PAR EP_Y_CVT);
    else if constexpr (FIELD == 8) EP_FIELD_ASM(EP_DEC(0), EP_DEC(1), EP_Y_PAR EP_Y_CVT EP_Y_SAT);
    else if constexpr (YM == 1) EP_FIELD_ASM(EP_DEC(0), EP_DEC(1), EP_Y_CVT);
    else EP_FIELD_ASM(EP_DEC(0), EP_DEC(1), EP_Y_CVT EP_Y_SAT);
  }
}

// Coset symbol (two-entry table f0, f1) for both chains, then the refill.
// Returns cb = 4 * 8c * 2^B (the byte offset of the lane's coset tables) and
// hc = c * sg / 2 (half the row scale when the point lies in the half-integer
// coset, else 0).
template <int B>
__device__ __forceinline__ void coset_step2(uint32_t& x0, uint32_t& x1, uint32_t& cb0, uint32_t& cb1,
                                            float& hc0, float& hc1, float sg0, float sg1,
                                            uint32_t vf0, uint32_t vf1, uint32_t vcb, FastChain& F0,
                                            FastChain& F1, uint32_t vH, uint32_t vrb0, uint32_t vrb1) {
  EP_STEP_TEMPS;
  asm volatile(
      "v_and_b32 %[u0], %[mk], %[x0]\n\t"
      "v_and_b32 %[u1], %[mk], %[x1]\n\t"
      "v_lshrrev_b32 %[g0], %[b], %[x0]\n\t"
      "v_lshrrev_b32 %[g1], %[b], %[x1]\n\t"
      "v_cmp_le_u32_e32 vcc, %[vf0], %[u0]\n\t"
      "v_cndmask_b32_e32 %[w0], %[vf0], %[vf1], vcc\n\t"
      "v_cndmask_b32_e32 %[t0], 0, %[vf0], vcc\n\t"
      "v_cndmask_b32_e32 %[cb0], 0, %[vcb], vcc\n\t"
      "v_mad_u32_u24 %[x0], %[w0], %[g0], %[u0]\n\t"
      "v_mul_f32_e32 %[w0], 0.5, %[sg0]\n\t"
      "v_cndmask_b32_e32 %[hc0], 0, %[w0], vcc\n\t"
      "v_sub_u32_e32 %[x0], %[x0], %[t0]\n\t"
      "v_cmp_le_u32_e32 vcc, %[vf0], %[u1]\n\t"
      "v_cndmask_b32_e32 %[w1], %[vf0], %[vf1], vcc\n\t"
      "v_cndmask_b32_e32 %[t1], 0, %[vf0], vcc\n\t"
      "v_cndmask_b32_e32 %[cb1], 0, %[vcb], vcc\n\t"
      "v_mad_u32_u24 %[x1], %[w1], %[g1], %[u1]\n\t"
      "v_mul_f32_e32 %[w1], 0.5, %[sg1]\n\t"
      "v_cndmask_b32_e32 %[hc1], 0, %[w1], vcc\n\t"
      "v_sub_u32_e32 %[x1], %[x1], %[t1]\n\t"
      EP_REFILL_BOTH
      : EP_STEP_OUTS, [cb0] "=&v"(cb0), [cb1] "=&v"(cb1), [hc0] "=&v"(hc0), [hc1] "=&v"(hc1)
      : [vf0] "v"(vf0), [vf1] "v"(vf1), [vcb] "v"(vcb), [sg0] "v"(sg0), [sg1] "v"(sg1), EP_STEP_INS
      : EP_STEP_CLOBBERS);
}

// ---- one chain per wave (small launches) ----------------------------------------
// The same steps for a wave that advances a single chain (two tiles, one per
// half): each step's instructions are chain 0's of the two-chain steps.  A
// wave alone on its SIMD issues about one instruction per four cycles, so a
// launch with too few tasks to put several waves on every SIMD finishes
// sooner when each wave issues half the instructions per symbol and there are
// twice as many waves.
#define EP_REFILL_ONE_W(WORK)                                               \
  "v_cmp_gt_u32_e32 vcc, 0x8000, %[x0]\n\t"                                 \
  "s_bcnt1_i32_b32 %[c0lo], vcc_lo\n\t"                                    \
  "v_mbcnt_lo_u32_b32 %[t0], vcc_lo, 0\n\t"                                 \
  "s_bcnt1_i32_b32 %[c0hi], vcc_hi\n\t"                                    \
  "v_mbcnt_hi_u32_b32 %[t0], vcc_hi, %[t0]\n\t"                             \
  "s_sub_u32 %[d0], %[D0], %[c0lo]\n\t"                                    \
  "v_mad_i32_i24 %[t0], %[vH], %[d0], %[t0]\n\t"                            \
  "v_add_lshl_u32 %[t0], %[t0], %[SA0], 1\n\t"                              \
  "v_and_or_b32 %[t0], %[t0], %[rmask], %[vrb0]\n\t"                        \
  "ds_read_u16 %[w0], %[t0]\n\t"                                            \
  "s_add_u32 %[SA0], %[SA0], %[c0lo]\n\t"                                  \
  "s_setprio 0\n\t"                                                        \
  "s_add_u32 %[D0], %[d0], %[c0hi]\n\t"                                  \
  WORK                                                                     \
  "s_and_saveexec_b64 %[ex], vcc\n\t"                                       \
  "s_waitcnt lgkmcnt(0)\n\t"                                                \
  "v_lshl_or_b32 %[x0], %[x0], 16, %[w0]\n\t"                               \
  "s_mov_b64 exec, %[ex]\n\t"

#define EP_STEP1_OUTS                                                                    \
  [x0] "+v"(x0), [SA0] "+s"(F0.OA), [D0] "+s"(F0.D), [u0] "=&v"(u0), [g0] "=&v"(g0),   \
      [t0] "=&v"(t0), [w0] "=&v"(w0), [c0lo] "=&s"(c0lo), [c0hi] "=&s"(c0hi),           \
      [d0] "=&s"(dd0), [ex] "=&s"(ex)

#define EP_STEP1_TEMPS                                                                   \
  uint32_t u0, g0, t0, w0, c0lo, c0hi, dd0;                                              \
  uint64_t ex

#define EP_STEP1_INS                                                                     \
  [vH] "v"(vH), [vrb0] "v"(vrb0), [rmask] "s"(kFastRingBytes - 1), [mk] "i"((1 << B) - 1), \
      [b] "i"(B)

#define EP_STEP1_CLOBBERS "vcc", "scc", "exec", "memory"

#define EP_Y_CVT1                                                                     \
  "v_cvt_f32_i32_sdwa %[y0], sext(%[e0]) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n\t" \
  "v_fma_f32 %[y0], %[sg0], %[y0], %[hc0]\n\t"
#define EP_Y_CVT1_WIDE                                                                \
  "v_ashrrev_i32 %[y0], 22, %[e0]\n\t"                                                \
  "v_cvt_f32_i32_e32 %[y0], %[y0]\n\t"                                                \
  "v_fma_f32 %[y0], %[sg0], %[y0], %[hc0]\n\t"
#define EP_Y_SAT1 "v_med3_f32 %[y0], %[y0], %[nm], %[m]\n\t"
#define EP_Y_PAR1 "v_and_or_b32 %[e0], %[X0], %[bit], %[e0]\n\t"

#define EP_FIELD1_ASM(DEC0, WORK)                                                        \
  asm volatile(                                                                          \
      "v_and_b32 %[u0], %[mk], %[x0]\n\t"                                                \
      "v_lshl_add_u32 %[u0], %[u0], 2, %[cb0]\n\t"                                       \
      "ds_read_b32 %[e0], %[u0] offset:%[off]\n\t"                                       \
      "v_lshrrev_b32 %[g0], %[b], %[x0]\n\t"                                             \
      "s_waitcnt lgkmcnt(0)\n\t"                                                         \
      "s_setprio 2\n\t"                                                                  \
      DEC0                                                                               \
      EP_REFILL_ONE_W(WORK)                                                              \
      : EP_STEP1_OUTS, [e0] "=&v"(e0), [y0] "=&v"(y0)                                    \
      : [cb0] "v"(cb0), [off] "i"((FIELD - 1) * (4 << B)), [sg0] "v"(sg0), [hc0] "v"(hc0), \
        [m] "s"(m), [nm] "v"(-m), [X0] "v"(X0), [bit] "s"(zbit), EP_STEP1_INS            \
      : EP_STEP1_CLOBBERS)

// Field symbol of the single chain (see field_step2).
template <int B, int FIELD, int YM, bool WIDE>
__device__ __forceinline__ void field_step1(uint32_t& x0, uint32_t cb0, uint32_t& e0, float& y0,
                                            float sg0, float hc0, uint32_t X0, float m, FastChain& F0,
                                            uint32_t vH, uint32_t vrb0) {
  EP_STEP1_TEMPS;
  const uint32_t zbit = 1u << (WIDE ? 22 : 24);   // low bit of the entry's z
  if constexpr (WIDE) {
    if constexpr (YM == 0) EP_FIELD1_ASM(EP_DEC_WIDE(0), "");
    else if constexpr (FIELD == 8 && YM == 1) EP_FIELD1_ASM(EP_DEC_WIDE(0), EP_Y_PAR1 EP_Y_CVT1_WIDE);
    else if constexpr (FIELD == 8) EP_FIELD1_ASM(EP_DEC_WIDE(0), EP_Y_PAR1 EP_Y_CVT1_WIDE EP_Y_SAT1);
    else if constexpr (YM == 1) EP_FIELD1_ASM(EP_DEC_WIDE(0), EP_Y_CVT1_WIDE);
    else EP_FIELD1_ASM(EP_DEC_WIDE(0), EP_Y_CVT1_WIDE EP_Y_SAT1);
  } else {
    if constexpr (YM == 0) EP_FIELD1_ASM(EP_DEC(0), "");
    else if constexpr (FIELD == 8 && YM == 1) EP_FIELD1_ASM(EP_DEC(0), EP_Y_PAR1 EP_Y_CVT1);
    else if constexpr (FIELD == 8) EP_FIELD1_ASM(EP_DEC(0), EP_Y_PAR1 EP_Y_CVT1 EP_Y_SAT1);
    else if constexpr (YM == 1) EP_FIELD1_ASM(EP_DEC(0), EP_Y_CVT1);
    else EP_FIELD1_ASM(EP_DEC(0), EP_Y_CVT1 EP_Y_SAT1);
  }
}

// Coset symbol of the single chain (see coset_step2).
template <int B>
__device__ __forceinline__ void coset_step1(uint32_t& x0, uint32_t& cb0, float& hc0, float sg0,
                                            uint32_t vf0, uint32_t vf1, uint32_t vcb, FastChain& F0,
                                            uint32_t vH, uint32_t vrb0) {
  EP_STEP1_TEMPS;
  asm volatile(
      "v_and_b32 %[u0], %[mk], %[x0]\n\t"
      "v_lshrrev_b32 %[g0], %[b], %[x0]\n\t"
      "v_cmp_le_u32_e32 vcc, %[vf0], %[u0]\n\t"
      "v_cndmask_b32_e32 %[w0], %[vf0], %[vf1], vcc\n\t"
      "v_cndmask_b32_e32 %[t0], 0, %[vf0], vcc\n\t"
      "v_cndmask_b32_e32 %[cb0], 0, %[vcb], vcc\n\t"
      "v_mad_u32_u24 %[x0], %[w0], %[g0], %[u0]\n\t"
      "v_mul_f32_e32 %[w0], 0.5, %[sg0]\n\t"
      "v_cndmask_b32_e32 %[hc0], 0, %[w0], vcc\n\t"
      "v_sub_u32_e32 %[x0], %[x0], %[t0]\n\t"
      EP_REFILL_ONE_W("")
      : EP_STEP1_OUTS, [cb0] "=&v"(cb0), [hc0] "=&v"(hc0)
      : [vf0] "v"(vf0), [vf1] "v"(vf1), [vcb] "v"(vcb), [sg0] "v"(sg0), EP_STEP1_INS
      : EP_STEP1_CLOBBERS);
}

__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t r;
  asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Reconstruction of one vector as its slot entries arrive (eq. point_inverse,
// eq. recon).  Bit 24 of an entry is the low bit of its z, so bit 24 of
// e1 ^ ... ^ e7 is pi = (z_1 + ... + z_7) mod 2, and field 8's z becomes z + pi
// (z is even there).  Each weight is fp32(sigma * (z + c/2)), formed as the
// single rounding fma(sigma, z, c * sigma / 2) -- equal to the product of the
// FP32 row scale with the coordinate -- and snapped to the output type.  The
// entry of an odd field waits in `ep` for its even partner; the pair is then
// converted and packed into the output words w.  The weights themselves are
// formed inside the symbol steps (field_step2).
struct QAcc {
  uint32_t X;     // xor of the entries of fields 1..7 so far
  uint32_t ep;    // entry of the pending odd field
  float yp;       // its weight
  uint32_t w[8];  // packed output words (the output type uses 2, 4 or 8 of them)
};

// clamp(RNE(a), -128, 127) and the same of b as two bytes (low half-word):
// round to nearest even, convert (the conversion saturates to the int32
// range), then an arithmetic shift by 0 with saturation to int8, packed into
// the low half of the destination (whose high half the instruction leaves as
// it was, hence the mask).
__device__ __forceinline__ uint32_t int8_pair(float a, float b) {
  const int ia = (int)__builtin_rintf(a), ib = (int)__builtin_rintf(b);
  uint32_t r;
  asm("v_ashr_pk_i8_i32 %0, %1, %2, 0" : "=v"(r) : "v"(ia), "v"(ib));
  return r & 0xFFFFu;
}

// The same with saturation to [0, 255] (unsigned bytes).
__device__ __forceinline__ uint32_t uint8_pair(float a, float b) {
  const int ia = (int)__builtin_rintf(a), ib = (int)__builtin_rintf(b);
  uint32_t r;
  asm("v_ashr_pk_u8_i32 %0, %1, %2, 0" : "=v"(r) : "v"(ia), "v"(ib));
  return r & 0xFFFFu;
}

// Fold field FIELD's entry e and weight y (computed in the step, see
// field_step2) into the chain's accumulator; c is the coset bit.
template <int DT, int FIELD, bool WIDE>
__device__ __forceinline__ void q_take(QAcc& a, uint32_t e, float y, uint32_t c) {
  constexpr int ZS = WIDE ? 22 : 24;   // position of z in the entry
  if constexpr (FIELD % 2 == 1) {
    if constexpr (FIELD == 7) a.X ^= e;
    a.ep = e;
    a.yp = y;
    return;
  } else {
    if constexpr (FIELD == 2) a.X = a.ep ^ e;
    else if constexpr (FIELD < 8) a.X = xor3(a.X, a.ep, e);
    constexpr int p = FIELD / 2 - 1;   // pair index 0..3
    if constexpr (DT == EP_COORD2_I32) {
      if constexpr (FIELD == 8) e |= a.X & (1u << ZS);
      a.w[2 * p] = (uint32_t)(2 * ((int32_t)a.ep >> ZS) + (int32_t)c);
      a.w[2 * p + 1] = (uint32_t)(2 * ((int32_t)e >> ZS) + (int32_t)c);
      return;
    }
    const float y0 = a.yp, y1 = y;
    if constexpr (DT == EP_BF16) {
      a.w[p] = bf16_pair(y0, y1);
    } else if constexpr (DT == EP_FP16) {
      a.w[p] = fp16_pair(y0, y1);
    } else if constexpr (DT == EP_FP32) {
      a.w[2 * p] = __float_as_uint(y0);
      a.w[2 * p + 1] = __float_as_uint(y1);
    } else if constexpr (DT == EP_FP8_E4M3) {
      // the low half is written first; its high half is overwritten by the next pair
      a.w[p / 2] = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(
          y0, y1, (int)(p & 1 ? a.w[p / 2] : __float_as_uint(y0)), (p & 1) != 0);
    } else if constexpr (DT == EP_FP8_E5M2) {
      a.w[p / 2] = (uint32_t)__builtin_amdgcn_cvt_pk_bf8_f32(
          y0, y1, (int)(p & 1 ? a.w[p / 2] : __float_as_uint(y0)), (p & 1) != 0);
    } else if constexpr (DT == EP_UINT8) {
      const uint32_t h = uint8_pair(y0, y1);
      a.w[p / 2] = p & 1 ? (a.w[p / 2] | (h << 16)) : h;
    } else {  // EP_INT8
      const uint32_t h = int8_pair(y0, y1);
      a.w[p / 2] = p & 1 ? (a.w[p / 2] | (h << 16)) : h;
    }
  }
}

// Store the packed vector at base + off.
template <int DT>
__device__ __forceinline__ void q_put(EP_GLOBAL uint8_t* base, uint32_t off, const QAcc& a) {
  if constexpr (DT == EP_BF16 || DT == EP_FP16) {
    *reinterpret_cast<EP_GLOBAL u32x4*>(base + off) = u32x4{a.w[0], a.w[1], a.w[2], a.w[3]};
  } else if constexpr (DT == EP_FP8_E4M3 || DT == EP_FP8_E5M2 || DT == EP_INT8 || DT == EP_UINT8) {
    *reinterpret_cast<EP_GLOBAL u32x2*>(base + off) = u32x2{a.w[0], a.w[1]};
  } else {
    EP_GLOBAL u32x4* o = reinterpret_cast<EP_GLOBAL u32x4*>(base + off);
    o[0] = u32x4{a.w[0], a.w[1], a.w[2], a.w[3]};
    o[1] = u32x4{a.w[4], a.w[5], a.w[6], a.w[7]};
  }
}

// Bytes of one 8-weight vector in output type DT.
template <int DT>
constexpr uint32_t vec_bytes() {
  return DT == EP_FP8_E4M3 || DT == EP_FP8_E5M2 || DT == EP_INT8 || DT == EP_UINT8 ? 8u
         : (DT == EP_BF16 || DT == EP_FP16) ? 16u : 32u;
}

// Sum of v over the 32 lanes of each half-wave, valid in lanes 0 and 32 (the
// lanes that add it to Y).  DPP moves and lane reads only, no LDS instruction:
// the LDS waits inside the decode steps count on their own reads alone.
// Every lane of the wave must be active.
__device__ __forceinline__ int32_t half_sum(int32_t v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);    // lane i ^ 1
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);    // lane i ^ 2
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);   // the other quad of 8
  v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);   // the other 8 of 16
  const int32_t a = __builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16);
  const int32_t b = __builtin_amdgcn_readlane(v, 32) + __builtin_amdgcn_readlane(v, 48);
  return (threadIdx.x & 32) ? b : a;
}

// The steady-state task of the slot-table path: four full tiles t0 .. t0 + 3
// (two chains).  TWO: every lane's vectors v, v + 32, ... of a tile lie in at
// most two rows (C/8 >= 32 (ceil(V / 32) - 1)), so each lane holds both row
// scales and switches at round kc; otherwise the row scale is loaded every round.
//
// Fused product (DT = kOutDotI8): each round's eight INT8 weights go straight
// into two dot4 instructions per row of X.  With TWO (the caller guarantees
// C/8 >= V here, so a tile spans at most rows r0 and r0 + 1) each lane keeps
// MT int32 sums per chain: at the start of the round where a lane's vectors
// pass into row r0 + 1 its sums so far are summed over its half-wave and
// added to Y[t][r0], and at the end of the task the remaining sums go to r0
// or r0 + 1.  Columns 0-3 of X for a round are requested at its start and
// used once the vector's first four weights are known (after field 4), when
// columns 4-7 are requested, used at the end of the round.
// Without TWO every vector is added to Y on its own.
template <int B, int DT, bool SAT, bool TWO, bool WIDE, int MT = 1>
__device__ __forceinline__ void lut_task(const Hot& L, uint8_t* lds, uint32_t ring_area, uint32_t t0,
                                         int32_t* status) {
  const uint32_t lane = threadIdx.x & 63, wave = wave_id();
  const uint32_t half = lane >> 5, l = lane & 31;
  const EP_GLOBAL uint32_t* states = gptr<const uint32_t>(L.blob + L.off_states);
  const EP_GLOBAL uint32_t* offs = gptr<const uint32_t>(L.blob + L.off_offsets);
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(L.blob + L.off_payload), (short)0, (int)L.pay_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t srsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(L.blob + L.off_sigma), (short)0, (int)(4 * L.rows), 0x00020000);
  constexpr uint32_t VB = vec_bytes<DT>();
  // weights formed in the steps: none for the doubled-coordinate output,
  // clamped to the type's finite range when SAT
  constexpr int YM = DT == EP_COORD2_I32 ? 0 : SAT ? 2 : 1;
  const float ymax = DT == EP_FP8_E4M3 ? 448.0f : DT == EP_FP8_E5M2 ? 57344.0f
                     : DT == EP_FP16 ? 65504.0f : 3.38953139e38f;

  const uint32_t vrb0 = ring_area + wave * 2 * kFastChainBytes + half * kFastRingBytes;
  const uint32_t vrb1 = vrb0 + kFastChainBytes;
  const uint32_t vl8 = 8 * l;
  uint32_t o[5];
#pragma unroll
  for (int i = 0; i < 5; i++) o[i] = offs[t0 + i];
  uint32_t x[2], vb[2], voff[2], kc[2];
  float sa[2], sb[2];
#pragma unroll
  for (int j = 0; j < 2; j++) {
    const uint32_t tile = t0 + 2 * j + half;
    x[j] = states[(uint64_t)tile * 32 + l];
    vb[j] = tile * L.V + l;
    voff[j] = ((2 * j + half) * L.V + l) * VB;
    if constexpr (TWO) {
      const uint32_t r = row_of(L, vb[j]);
      kc[j] = ((r + 1) * L.cvec - vb[j] + 31) >> 5;
      sa[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(srsrc, 4 * r, 0, 0));
      sb[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(srsrc, 4 * r + 4, 0, 0));
    }
  }
  constexpr bool DOT = DT == kOutDotI8;
  constexpr bool ACC = DOT && TWO;
  int32_t dacc[2][MT];
  uint32_t r0[2], kd[2], colb[2];
  __amdgpu_buffer_rsrc_t xrsrc;
  if constexpr (ACC) {
    xrsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(L.x), (short)0,
                                              (int)(L.m * L.cols), 0x00020000);
#pragma unroll
    for (int j = 0; j < 2; j++) {
      r0[j] = row_of(L, (t0 + 2 * j + half) * L.V);   // first row of the lane's tile
      kd[j] = row_of(L, vb[j]) == r0[j] ? kc[j] : 0u;   // first round in row r0 + 1
      colb[j] = vb[j] - r0[j] * L.cvec;
#pragma unroll
      for (int t = 0; t < MT; t++) dacc[j][t] = 0;
    }
  }
  FastChain F0, F1;
  u32x2 pend0, pend1, pendB0, pendB1;
#pragma unroll
  for (int i = 0; i < 5; i++) o[i] = uni(o[i]);
  const u32x4 fill0 = fast_start(F0, pend0, rsrc, half, l, o[0], o[1], o[1], o[2]);
  const u32x4 fill1 = fast_start(F1, pend1, rsrc, half, l, o[2], o[3], o[3], o[4]);
  // One wait for everything requested so far, so that no load is in flight
  // when the loop starts (the loop's own waits then stay one round behind).
  __builtin_amdgcn_s_waitcnt(0);
  *reinterpret_cast<u32x4*>(lds + vrb0 + 16 * l) = fill0;
  *reinterpret_cast<u32x4*>(lds + vrb1 + 16 * l) = fill1;
  pendB0 = pend0;   // pend* serve lanes 0-31, pendB* lanes 32-63
  pendB1 = pend1;

  EP_GLOBAL uint8_t* obase = gptr<uint8_t>(L.out) + (uint64_t)t0 * L.V * VB;
  const uint32_t vH = half;
  const uint32_t vf0 = L.coset_f0, vf1 = L.coset_f1, vcb = 32u << B;
  // V = 32 * full + tail vectors: `full` rounds in which every lane decodes a
  // vector, then (tail > 0, store outputs only) one round in which lanes
  // l >= tail have none.  That round runs the same steps with those lanes'
  // states pinned at 2^31 - 1 before every symbol: x >> b then exceeds 2^15 / f
  // for any f >= 1, so they never take a refill word, and the staging commits
  // stay outside any divergent region.  Their decoded values are not stored,
  // and their real final states (saved first) are checked at the end.
  const uint32_t full = L.V / 32, tail = L.V % 32;
  const uint32_t rounds = full + (tail ? 1 : 0);
  const uint32_t vrb08 = vrb0 + vl8, vrb18 = vrb1 + vl8;
  uint32_t xsave[2] = {0, 0};
  const bool pin = l >= tail;

  auto round = [&](uint32_t k, auto part) {
    constexpr bool PART = decltype(part)::value;
    if constexpr (PART) {
      xsave[0] = x[0];
      xsave[1] = x[1];
    }
    // room for a block: margin <= ring - block
    fast_stage_both(F0, F1, pend0, pendB0, pend1, pendB1, lds, vrb08, vrb18, vl8, rsrc, half,
                    kFastRingWords - kFastBlockWords + 1);
    float sg[2], hc[2];
#pragma unroll
    for (int j = 0; j < 2; j++) {
      if constexpr (TWO) sg[j] = k < kc[j] ? sa[j] : sb[j];
      else sg[j] = __uint_as_float(
          __builtin_amdgcn_raw_buffer_load_b32(srsrc, 4 * row_of(L, vb[j] + 32 * k), 0, 0));
    }
    uint32_t xo[2], xq[2][MT];
    if constexpr (ACC) {
      EP_GLOBAL int32_t* y = gptr<int32_t>(L.out);
#pragma unroll
      for (int j = 0; j < 2; j++) {
        // lanes whose vectors pass into row r0 + 1 this round: their sums so far belong to r0
        const bool dep = k == kd[j];
        if (__builtin_expect(__ballot(dep) != 0, 0)) {
#pragma unroll
          for (int t = 0; t < MT; t++) {
            const int32_t sum = half_sum(dep ? dacc[j][t] : 0);
            if (l == 0 && (uint32_t)t < L.m && sum != 0) add_i32(y + (uint64_t)t * L.rows + r0[j], sum);
            if (dep) dacc[j][t] = 0;
          }
        }
        xo[j] = 8 * (colb[j] + 32 * k - (k >= kd[j] ? L.cvec : 0u));
        // columns 0-3 of the vector now, 4-7 once the first four weights are known
#pragma unroll
        for (int t = 0; t < MT; t++) xq[j][t] = __builtin_amdgcn_raw_buffer_load_b32(xrsrc, xo[j], t * L.cols, 0);
      }
    }
    uint32_t cb[2], e0, e1;
    float y0, y1;
    QAcc acc[2];
    acc[0].X = acc[1].X = 0;
#define EP_PIN                            \
  if constexpr (PART) {                   \
    x[0] = pin ? kPinnedState : x[0];     \
    x[1] = pin ? kPinnedState : x[1];     \
  }
    EP_PIN
    coset_step2<B>(x[0], x[1], cb[0], cb[1], hc[0], hc[1], sg[0], sg[1], vf0, vf1, vcb, F0, F1, vH,
                   vrb0, vrb1);
#define EP_FIELD(I)                                                                           \
  EP_PIN                                                                                      \
  field_step2<B, I, YM, WIDE>(x[0], x[1], cb[0], cb[1], e0, e1, y0, y1, sg[0], sg[1], hc[0],  \
                              hc[1], acc[0].X, acc[1].X, ymax, F0, F1, vH, vrb0, vrb1);       \
  q_take<DT, I, WIDE>(acc[0], e0, y0, cb[0] >> (B + 5));                                      \
  q_take<DT, I, WIDE>(acc[1], e1, y1, cb[1] >> (B + 5));
    EP_FIELD(1) EP_FIELD(2)
    fast_stage_both(F0, F1, pend0, pendB0, pend1, pendB1, lds, vrb08, vrb18, vl8, rsrc, half, 3 * 32);
    EP_FIELD(3) EP_FIELD(4)
    if constexpr (ACC) {
#pragma unroll
      for (int j = 0; j < 2; j++) {
#pragma unroll
        for (int t = 0; t < MT; t++) {
          dacc[j][t] = __builtin_amdgcn_sdot4((int)acc[j].w[0], (int)xq[j][t], dacc[j][t], false);
          xq[j][t] = __builtin_amdgcn_raw_buffer_load_b32(xrsrc, xo[j] + 4, t * L.cols, 0);
        }
      }
    }
    EP_FIELD(5)
    fast_stage_both(F0, F1, pend0, pendB0, pend1, pendB1, lds, vrb08, vrb18, vl8, rsrc, half, 3 * 32);
    EP_FIELD(6) EP_FIELD(7) EP_FIELD(8)
#undef EP_FIELD
#undef EP_PIN
    if constexpr (ACC) {
#pragma unroll
      for (int j = 0; j < 2; j++)
#pragma unroll
        for (int t = 0; t < MT; t++)
          dacc[j][t] = __builtin_amdgcn_sdot4((int)acc[j].w[1], (int)xq[j][t], dacc[j][t], false);
    } else if constexpr (DOT) {
#pragma unroll
      for (int j = 0; j < 2; j++) {
        const uint32_t v = vb[j] + 32 * k;
        dot_add(L, acc[j].w[0], acc[j].w[1], v, row_of(L, v));
      }
    } else {
      if (!PART || !pin) {
        q_put<DT>(obase, voff[0], acc[0]);
        q_put<DT>(obase, voff[1], acc[1]);
      }
      obase += 32 * VB;
    }
  };
  for (uint32_t k = 0; k < full; k++) round(k, std::false_type{});
  if constexpr (!DOT) {
    if (tail) {
      round(full, std::true_type{});
      x[0] = pin ? xsave[0] : x[0];
      x[1] = pin ? xsave[1] : x[1];
    }
  }
  if constexpr (ACC) {
    EP_GLOBAL int32_t* y = gptr<int32_t>(L.out);
#pragma unroll
    for (int j = 0; j < 2; j++) {
      const bool moved = rounds > kd[j];   // the lane's last vector lies in row r0 + 1
#pragma unroll
      for (int t = 0; t < MT; t++) {
        const int32_t s0 = half_sum(moved ? 0 : dacc[j][t]);
        const int32_t s1 = half_sum(moved ? dacc[j][t] : 0);
        if (l == 0 && (uint32_t)t < L.m) {
          if (s0 != 0) add_i32(y + (uint64_t)t * L.rows + r0[j], s0);
          if (s1 != 0) add_i32(y + (uint64_t)t * L.rows + r0[j] + 1, s1);
        }
      }
    }
  }

  uint32_t err = 0;
#pragma unroll
  for (int j = 0; j < 2; j++) {
    if (x[j] != kStateLow) err |= EP_STATUS_BAD_FINAL_STATE;
    const FastChain& F = j ? F1 : F0;
    const uint32_t P = half ? F.OA + F.D : F.OA, E = half ? F.EB : F.EA;
    if (l == 0 && P != E) err |= P > E ? EP_STATUS_PAYLOAD_OVERRUN : EP_STATUS_BAD_END_OFFSET;
    if (L.container && L.dequant) {
      const EP_GLOBAL float* delta = gptr<const float>(L.blob + L.off_delta);
      const uint32_t v0 = (t0 + 2 * j + half) * L.V;
      const uint32_t r_first = (v0 + L.cvec - 1) / L.cvec;
      const uint32_t r_last = (v0 + L.V - 1) / L.cvec;
      for (uint32_t r = r_first + l; r <= r_last; r += 32) gptr<float>(L.dequant)[r] = delta[r];
    }
  }
  if (err && status) atomicOr(status, (int32_t)err);
}

// The slot-table steady state with one chain: a task of two tiles, t0 in
// lanes 0-31 and t0 + 1 in lanes 32-63, for launches with too few four-tile
// tasks to fill the SIMDs (see field_step1), and for the fused product with
// more than four rows of X, whose sums then fit the registers.  The structure
// is lut_task's with the second chain removed.
template <int B, int DT, bool SAT, bool TWO, bool WIDE, int MT = 1>
__device__ __forceinline__ void lut_task1(const Hot& L, uint8_t* lds, uint32_t ring_area, uint32_t t0,
                                          int32_t* status) {
  constexpr bool DOT = DT == kOutDotI8;
  static_assert(!DOT || TWO, "the fused product runs the steady state on rows of at least a tile");
  const uint32_t lane = threadIdx.x & 63, wave = wave_id();
  const uint32_t half = lane >> 5, l = lane & 31;
  const EP_GLOBAL uint32_t* states = gptr<const uint32_t>(L.blob + L.off_states);
  const EP_GLOBAL uint32_t* offs = gptr<const uint32_t>(L.blob + L.off_offsets);
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(L.blob + L.off_payload), (short)0, (int)L.pay_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t srsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(L.blob + L.off_sigma), (short)0, (int)(4 * L.rows), 0x00020000);
  constexpr uint32_t VB = vec_bytes<DT>();
  constexpr int YM = DT == EP_COORD2_I32 ? 0 : SAT ? 2 : 1;
  const float ymax = DT == EP_FP8_E4M3 ? 448.0f : DT == EP_FP8_E5M2 ? 57344.0f
                     : DT == EP_FP16 ? 65504.0f : 3.38953139e38f;

  // the wave's first ring (the two-chain layout's chain 0)
  const uint32_t vrb0 = ring_area + wave * 2 * kFastChainBytes + half * kFastRingBytes;
  const uint32_t vl8 = 8 * l;
  uint32_t o[3];
#pragma unroll
  for (int i = 0; i < 3; i++) o[i] = offs[t0 + i];
  const uint32_t tile = t0 + half;
  uint32_t x = states[(uint64_t)tile * 32 + l];
  const uint32_t vb = tile * L.V + l;
  const uint32_t voff = (half * L.V + l) * VB;
  uint32_t kc = 0;
  float sa = 0.0f, sb = 0.0f;
  if constexpr (TWO) {
    const uint32_t r = row_of(L, vb);
    kc = ((r + 1) * L.cvec - vb + 31) >> 5;
    sa = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(srsrc, 4 * r, 0, 0));
    sb = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(srsrc, 4 * r + 4, 0, 0));
  }
  int32_t dacc[MT];
  uint32_t r0 = 0, kd = 0, colb = 0;
  __amdgpu_buffer_rsrc_t xrsrc;
  if constexpr (DOT) {
    xrsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(L.x), (short)0,
                                              (int)(L.m * L.cols), 0x00020000);
    r0 = row_of(L, tile * L.V);                 // first row of the lane's tile
    kd = row_of(L, vb) == r0 ? kc : 0u;         // first round in row r0 + 1
    colb = vb - r0 * L.cvec;
#pragma unroll
    for (int t = 0; t < MT; t++) dacc[t] = 0;
  }
  FastChain F0;
  u32x2 pend0, pendB0;
#pragma unroll
  for (int i = 0; i < 3; i++) o[i] = uni(o[i]);
  const u32x4 fill0 = fast_start(F0, pend0, rsrc, half, l, o[0], o[1], o[1], o[2]);
  __builtin_amdgcn_s_waitcnt(0);
  *reinterpret_cast<u32x4*>(lds + vrb0 + 16 * l) = fill0;
  pendB0 = pend0;   // pend0 serves lanes 0-31, pendB0 lanes 32-63

  EP_GLOBAL uint8_t* obase = gptr<uint8_t>(L.out) + (uint64_t)t0 * L.V * VB;
  const uint32_t vH = half;
  const uint32_t vf0 = L.coset_f0, vf1 = L.coset_f1, vcb = 32u << B;
  // full rounds, then a partial one with the states of lanes past the tile
  // pinned (see lut_task)
  const uint32_t full = L.V / 32, tail = L.V % 32;
  const uint32_t vrb08 = vrb0 + vl8;
  uint32_t xsave = 0;
  const bool pin = l >= tail;

  auto round = [&](uint32_t k, auto part) {
    constexpr bool PART = decltype(part)::value;
    if constexpr (PART) xsave = x;
    fast_stage(F0, pend0, pendB0, lds, vrb08, vl8, rsrc, half, kFastRingWords - kFastBlockWords + 1);
    float sg;
    if constexpr (TWO) sg = k < kc ? sa : sb;
    else sg = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(srsrc, 4 * row_of(L, vb + 32 * k), 0, 0));
    uint32_t xo = 0, xq[MT];
    if constexpr (DOT) {
      EP_GLOBAL int32_t* y = gptr<int32_t>(L.out);
      // lanes whose vectors pass into row r0 + 1 this round: their sums so far belong to r0
      const bool dep = k == kd;
      if (__builtin_expect(__ballot(dep) != 0, 0)) {
#pragma unroll
        for (int t = 0; t < MT; t++) {
          const int32_t sum = half_sum(dep ? dacc[t] : 0);
          if (l == 0 && (uint32_t)t < L.m && sum != 0) add_i32(y + (uint64_t)t * L.rows + r0, sum);
          if (dep) dacc[t] = 0;
        }
      }
      xo = 8 * (colb + 32 * k - (k >= kd ? L.cvec : 0u));
      // columns 0-3 of the vector now, 4-7 once the first four weights are known
#pragma unroll
      for (int t = 0; t < MT; t++) xq[t] = __builtin_amdgcn_raw_buffer_load_b32(xrsrc, xo, t * L.cols, 0);
    }
    uint32_t cb, e0;
    float y0, hc;
    QAcc acc;
    acc.X = 0;
#define EP_PIN1                       \
  if constexpr (PART) x = pin ? kPinnedState : x;
    EP_PIN1
    coset_step1<B>(x, cb, hc, sg, vf0, vf1, vcb, F0, vH, vrb0);
#define EP_FIELD(I)                                                                        \
  EP_PIN1                                                                                  \
  field_step1<B, I, YM, WIDE>(x, cb, e0, y0, sg, hc, acc.X, ymax, F0, vH, vrb0);           \
  q_take<DT, I, WIDE>(acc, e0, y0, cb >> (B + 5));
    EP_FIELD(1) EP_FIELD(2)
    fast_stage(F0, pend0, pendB0, lds, vrb08, vl8, rsrc, half, 3 * 32);
    EP_FIELD(3) EP_FIELD(4)
    if constexpr (DOT) {
#pragma unroll
      for (int t = 0; t < MT; t++) {
        dacc[t] = __builtin_amdgcn_sdot4((int)acc.w[0], (int)xq[t], dacc[t], false);
        xq[t] = __builtin_amdgcn_raw_buffer_load_b32(xrsrc, xo + 4, t * L.cols, 0);
      }
    }
    EP_FIELD(5)
    fast_stage(F0, pend0, pendB0, lds, vrb08, vl8, rsrc, half, 3 * 32);
    EP_FIELD(6) EP_FIELD(7) EP_FIELD(8)
#undef EP_FIELD
#undef EP_PIN1
    if constexpr (DOT) {
#pragma unroll
      for (int t = 0; t < MT; t++)
        dacc[t] = __builtin_amdgcn_sdot4((int)acc.w[1], (int)xq[t], dacc[t], false);
    } else {
      if (!PART || !pin) q_put<DT>(obase, voff, acc);
      obase += 32 * VB;
    }
  };
  for (uint32_t k = 0; k < full; k++) round(k, std::false_type{});
  if constexpr (!DOT) {
    if (tail) {
      round(full, std::true_type{});
      x = pin ? xsave : x;
    }
  } else {
    EP_GLOBAL int32_t* y = gptr<int32_t>(L.out);
    const bool moved = full > kd;   // the lane's last vector lies in row r0 + 1
#pragma unroll
    for (int t = 0; t < MT; t++) {
      const int32_t s0 = half_sum(moved ? 0 : dacc[t]);
      const int32_t s1 = half_sum(moved ? dacc[t] : 0);
      if (l == 0 && (uint32_t)t < L.m) {
        if (s0 != 0) add_i32(y + (uint64_t)t * L.rows + r0, s0);
        if (s1 != 0) add_i32(y + (uint64_t)t * L.rows + r0 + 1, s1);
      }
    }
  }

  uint32_t err = 0;
  if (x != kStateLow) err |= EP_STATUS_BAD_FINAL_STATE;
  const uint32_t P = half ? F0.OA + F0.D : F0.OA, E = half ? F0.EB : F0.EA;
  if (l == 0 && P != E) err |= P > E ? EP_STATUS_PAYLOAD_OVERRUN : EP_STATUS_BAD_END_OFFSET;
  if (L.container && L.dequant) {
    const EP_GLOBAL float* delta = gptr<const float>(L.blob + L.off_delta);
    const uint32_t v0 = tile * L.V;
    const uint32_t r_first = (v0 + L.cvec - 1) / L.cvec;
    const uint32_t r_last = (v0 + L.V - 1) / L.cvec;
    for (uint32_t r = r_first + l; r <= r_last; r += 32) gptr<float>(L.dequant)[r] = delta[r];
  }
  if (err && status) atomicOr(status, (int32_t)err);
}

// NCH: chains per wave (2: a four-tile task, 1: a two-tile task).
template <int B, int DT, bool SAT, bool WIDE, int NCH = 2>
__device__ __forceinline__ void lut_task_rows(const Hot& L, uint8_t* lds, uint32_t ring_area,
                                              uint32_t t0, int32_t* status) {
  static_assert(NCH == 2 || DT == EP_BF16 || DT == EP_FP16 || DT == EP_FP8_E4M3 || DT == EP_INT8 ||
                    DT == kOutDotI8,
                "one-chain tasks cover the common output types");
  if constexpr (NCH == 1 && DT == kOutDotI8) {
    // more than four rows of X (the only product that runs one chain); rows
    // of at least a tile (lut_task_any checks)
    lut_task1<B, DT, false, true, WIDE, kDotMaxTokens>(L, lds, ring_area, t0, status);
  } else if constexpr (NCH == 1) {
    if (L.cvec >= 32 * ((L.V - 1) / 32)) lut_task1<B, DT, SAT, true, WIDE>(L, lds, ring_area, t0, status);
    else lut_task1<B, DT, SAT, false, WIDE>(L, lds, ring_area, t0, status);
  } else if constexpr (DT == kOutDotI8) {
    // up to four rows of X (more take one chain per wave, lut_task_any)
    if (L.cvec >= L.V) {
      if (L.m <= 1) lut_task<B, DT, false, true, WIDE, 1>(L, lds, ring_area, t0, status);
      else if (L.m <= 2) lut_task<B, DT, false, true, WIDE, 2>(L, lds, ring_area, t0, status);
      else lut_task<B, DT, false, true, WIDE, 4>(L, lds, ring_area, t0, status);
    } else {
      lut_task<B, DT, false, false, WIDE>(L, lds, ring_area, t0, status);
    }
  } else {
    // a lane's vectors v, v + 32, ..., v + 32 (ceil(V / 32) - 1) lie in at most two rows when
    // C/8 is at least their span
    if (L.cvec >= 32 * ((L.V - 1) / 32)) lut_task<B, DT, SAT, true, WIDE>(L, lds, ring_area, t0, status);
    else lut_task<B, DT, SAT, false, WIDE>(L, lds, ring_area, t0, status);
  }
}

// Output-type dispatch of a full slot-table task (narrow or wide entries;
// four tiles, or two with NCH = 1).  Returns false for the combinations the
// steady state does not cover (they take the generic loop).
template <int B, bool WIDE, bool DOT = false, int NCH = 2>
__device__ __forceinline__ bool lut_task_any(const Hot& L, uint8_t* lds, uint32_t ring_area,
                                             uint32_t t0, int32_t* status) {
  if constexpr (DOT) {
    if (NCH == 1 && L.cvec < L.V) return false;   // the generic loop adds vector by vector
    // two chains hold the sums of at most four rows of X in registers
    if (NCH == 2 && L.m > 4) return false;
    lut_task_rows<B, kOutDotI8, false, WIDE, NCH>(L, lds, ring_area, t0, status);
    return true;
  }
  if constexpr (NCH == 1) {
    // the output types small layers are decoded to; the rest take the generic loop
    switch (L.out_dtype) {
      case EP_BF16:
        if (L.saturate) lut_task_rows<B, EP_BF16, true, WIDE, 1>(L, lds, ring_area, t0, status);
        else lut_task_rows<B, EP_BF16, false, WIDE, 1>(L, lds, ring_area, t0, status);
        return true;
      case EP_FP16:
        if (L.saturate) lut_task_rows<B, EP_FP16, true, WIDE, 1>(L, lds, ring_area, t0, status);
        else lut_task_rows<B, EP_FP16, false, WIDE, 1>(L, lds, ring_area, t0, status);
        return true;
      case EP_FP8_E4M3:
        if (L.saturate) lut_task_rows<B, EP_FP8_E4M3, true, WIDE, 1>(L, lds, ring_area, t0, status);
        else lut_task_rows<B, EP_FP8_E4M3, false, WIDE, 1>(L, lds, ring_area, t0, status);
        return true;
      case EP_INT8: lut_task_rows<B, EP_INT8, false, WIDE, 1>(L, lds, ring_area, t0, status); return true;
      default: return false;
    }
  } else {
    switch (L.out_dtype) {
      case EP_BF16:
        if (L.saturate) lut_task_rows<B, EP_BF16, true, WIDE, NCH>(L, lds, ring_area, t0, status);
        else lut_task_rows<B, EP_BF16, false, WIDE, NCH>(L, lds, ring_area, t0, status);
        return true;
      case EP_FP16:
        if (L.saturate) lut_task_rows<B, EP_FP16, true, WIDE, NCH>(L, lds, ring_area, t0, status);
        else lut_task_rows<B, EP_FP16, false, WIDE, NCH>(L, lds, ring_area, t0, status);
        return true;
      case EP_FP8_E4M3:
        if (L.saturate) lut_task_rows<B, EP_FP8_E4M3, true, WIDE, NCH>(L, lds, ring_area, t0, status);
        else lut_task_rows<B, EP_FP8_E4M3, false, WIDE, NCH>(L, lds, ring_area, t0, status);
        return true;
      case EP_FP8_E5M2:
        if (L.saturate) lut_task_rows<B, EP_FP8_E5M2, true, WIDE, NCH>(L, lds, ring_area, t0, status);
        else lut_task_rows<B, EP_FP8_E5M2, false, WIDE, NCH>(L, lds, ring_area, t0, status);
        return true;
      case EP_INT8: lut_task_rows<B, EP_INT8, false, WIDE, NCH>(L, lds, ring_area, t0, status); return true;
      case EP_UINT8: lut_task_rows<B, EP_UINT8, false, WIDE, NCH>(L, lds, ring_area, t0, status); return true;
      case EP_FP32: lut_task_rows<B, EP_FP32, false, WIDE, NCH>(L, lds, ring_area, t0, status); return true;
      case EP_COORD2_I32:
        lut_task_rows<B, EP_COORD2_I32, false, WIDE, NCH>(L, lds, ring_area, t0, status);
        return true;
      default: return false;
    }
  }
}

// Output-type dispatch of a full search-path task (four tiles, two chains).  Returns
// false for the combinations the steady state does not cover (they take the generic loop).
template <int PATH, int B, bool DOT = false>
__device__ __forceinline__ bool decode_task_fast_any(const Hot& L, uint8_t* lds, uint32_t ring_area,
                                                     uint32_t task, int32_t* status) {
  if constexpr (DOT) {
    decode_task_fast<PATH, B, kOutDotI8, false>(L, lds, ring_area, task, status);
    return true;
  }
  switch (L.out_dtype) {
    case EP_BF16:
      if (L.saturate) return false;
      decode_task_fast<PATH, B, EP_BF16, false>(L, lds, ring_area, task, status);
      return true;
    case EP_FP16:
      if (L.saturate) decode_task_fast<PATH, B, EP_FP16, true>(L, lds, ring_area, task, status);
      else decode_task_fast<PATH, B, EP_FP16, false>(L, lds, ring_area, task, status);
      return true;
    case EP_FP8_E4M3:
      if (L.saturate) decode_task_fast<PATH, B, EP_FP8_E4M3, true>(L, lds, ring_area, task, status);
      else decode_task_fast<PATH, B, EP_FP8_E4M3, false>(L, lds, ring_area, task, status);
      return true;
    case EP_FP8_E5M2:
      if (L.saturate) decode_task_fast<PATH, B, EP_FP8_E5M2, true>(L, lds, ring_area, task, status);
      else decode_task_fast<PATH, B, EP_FP8_E5M2, false>(L, lds, ring_area, task, status);
      return true;
    case EP_INT8:
      decode_task_fast<PATH, B, EP_INT8, false>(L, lds, ring_area, task, status);
      return true;
    case EP_UINT8:
      decode_task_fast<PATH, B, EP_UINT8, false>(L, lds, ring_area, task, status);
      return true;
    case EP_FP32:
      decode_task_fast<PATH, B, EP_FP32, false>(L, lds, ring_area, task, status);
      return true;
    case EP_COORD2_I32:
      decode_task_fast<PATH, B, EP_COORD2_I32, false>(L, lds, ring_area, task, status);
      return true;
    default:
      return false;
  }
}

// LDS byte offset of the payload rings: after the slot table (LUT path) or
// after the search tables (search path).
template <int PATH>
__device__ __forceinline__ uint32_t ring_offset(const LayerDev& L) {
  if (PATH == kPathGlobal) return (L.g_meta + 4 * 64 + 511) & ~511u;   // GlobalLayout::total
  return PATH != kPathSearch ? (64u << L.b) : search_layout(L.b, L.sum_A).total;
}

// Search-path tables (byte layout from search_layout): u16 cumulative values
// of table t at [base_t + t, base_t + t + A_t] (the last one = 2^b), the u16
// bucket bounds bk[t][0 .. 2^k] (bk[t][j] = the symbol whose slot range holds
// slot j * 2^(b-k); bk[t][2^k] = A_t - 1), and u32 metadata base'[16], min[16].
// Each symbol writes the bucket starts inside its own slot range.
__device__ __forceinline__ void build_search(const LayerDev& L, uint32_t* lds) {
  uint16_t* cum = reinterpret_cast<uint16_t*>(lds);
  const SearchLayout S = search_layout(L.b, L.sum_A);
  uint16_t* bk = cum + S.bucket / 2;
  const uint32_t shift = L.b - S.bucket_bits, n1 = (1u << S.bucket_bits) + 1;
  scan_tables(
      L,
      [&](int t, uint32_t s, uint32_t F, uint32_t f) {
        cum[L.tab_base[t] + t + s] = (uint16_t)F;
        const uint32_t j0 = (F + (1u << shift) - 1) >> shift, j1 = (F + f + (1u << shift) - 1) >> shift;
        for (uint32_t j = j0; j < j1; j++) bk[t * n1 + j] = (uint16_t)s;
      },
      [&](int t, uint32_t M) {
        cum[L.tab_base[t] + t + L.tab_A[t]] = (uint16_t)M;
        bk[t * n1 + n1 - 1] = (uint16_t)(L.tab_A[t] ? L.tab_A[t] - 1 : 0);
      });
  if (threadIdx.x < 32) {
    const uint32_t t = threadIdx.x & 15;
    lds[S.meta / 4 + threadIdx.x] = threadIdx.x < 16 ? L.tab_base[t] + t : (uint32_t)L.tab_min[t];
  }
}

// Global-table path: C_j = F_{jG} of every table (u16, table t's entries from the
// sum of ceil(A_t' / G) over t' < t) and the metadata (GlobalLayout).
__device__ __forceinline__ uint32_t global_base(const LayerDev& L, uint32_t t) {
  uint32_t acc = 0;
  for (uint32_t i = 0; i < t; i++) acc += (L.tab_A[i] + (1u << L.g_bits) - 1) >> L.g_bits;
  return acc;
}

__device__ __forceinline__ void build_global(const LayerDev& L, uint32_t* lds) {
  uint16_t* cum = reinterpret_cast<uint16_t*>(lds);
  const uint32_t g = L.g_bits, G = 1u << g;
  scan_tables(
      L,
      [&](int t, uint32_t s, uint32_t F, uint32_t) {
        if ((s & (G - 1)) == 0) cum[global_base(L, (uint32_t)t) + (s >> g)] = (uint16_t)F;
      },
      [](int, uint32_t) {});
  if (threadIdx.x < 64) {
    const uint32_t t = threadIdx.x & 15, q = threadIdx.x >> 4;
    lds[L.g_meta / 4 + threadIdx.x] = q == 0 ? global_base(L, t)
                                      : q == 1 ? (uint32_t)L.tab_min[t]
                                      : q == 2 ? (L.tab_A[t] + G - 1) >> g
                                               : L.tab_off[t];
  }
}

template <int PATH>
__device__ __forceinline__ void build_tables(const LayerDev& L, uint32_t* lds) {
  if (PATH == kPathGlobal) {
    build_global(L, lds);
  } else if (PATH != kPathSearch && L.sum_A <= kRingBytes / 4) {
    uint32_t* cum = lds + (16u << L.b);   // scratch inside the ring area
    build_cumulative(L, cum);
    __syncthreads();
    build_lut<PATH == kPathWide>(L, lds, cum);
  } else if (PATH != kPathSearch) {
    // more symbols than the scratch holds (wide tables): every lane fills the
    // slot range of its own symbol straight from the table's prefix scan
    scan_tables(L, [&](int t, uint32_t s, uint32_t F, uint32_t f) {
      uint32_t* row = lds + ((uint32_t)t << L.b);
      const int field = (t & 7) + 1;
      const int32_t v = (int32_t)s + L.tab_min[t];
      const uint32_t z = (uint32_t)(field < 8 ? v : 2 * v);
      for (uint32_t i = 0; i < f; i++)
        row[F + i] = PATH == kPathWide ? (f - 1) | (i << 11) | ((z & 0x3FF) << 22)
                                       : f | (i << 12) | ((z & 0xFF) << 24);
    }, [](int, uint32_t) {});
  } else {
    build_search(L, lds);
  }
}

// A wave task is four tiles (two chains of two).  When all four are full (V
// vectors each, V a multiple of 32) the slot-table paths at b = 11 (the
// precision the encoder starts from for targets up to 7 bpp) and the search
// path decode them in a steady-state pass; otherwise the generic loop does.
constexpr int kChains = 2;                 // chains of the generic loop
// A task is one pass of a wave: two chains of two tiles, or in a launch with
// few tasks (LayerDev::tpt = 2) one chain of two tiles.
constexpr uint32_t kTilesPerTask = 4;
static_assert(kChains == 2, "the generic loop and the search steady state advance two chains");
static_assert(kTilesPerTask == 2 * kChains, "task granularity: one four-tile pass");

// SMALL: the kernel may run two-tile tasks (see use_small_tasks).
template <int PATH, int B, bool DOT, bool SMALL>
__device__ __forceinline__ void task_b(const Hot& L, const uint32_t* tab, uint8_t* lb,
                                       uint32_t ring_area, uint32_t task, int32_t* status) {
  const uint32_t nvec = L.rows * L.cvec;
  if constexpr (SMALL && (PATH == kPathLut || PATH == kPathWide) && B == 11) {
    if (L.tpt == 2) {
      // two-tile tasks, one chain per wave (the fused product needs whole rounds)
      const uint32_t t0 = L.tile_begin + 2 * task;
      const bool whole = t0 + 2 <= L.tile_end && (uint64_t)(t0 + 2) * L.V <= nvec;
      if (whole && L.V >= 32 && (!DOT || L.V % 32 == 0) && L.pay_bytes < kFastOob &&
          lut_task_any<B, PATH == kPathWide, DOT, 1>(L, lb, ring_area, t0, status))
        return;
      if (whole && L.V % 32 == 0) decode_task<PATH, B, 1, true, DOT>(L, tab, lb, ring_area, task, status);
      else decode_task<PATH, B, 1, false, DOT>(L, tab, lb, ring_area, task, status);
      return;
    }
  }
  const uint32_t t0 = L.tile_begin + kTilesPerTask * task;
  const bool whole = t0 + kTilesPerTask <= L.tile_end && (uint64_t)(t0 + kTilesPerTask) * L.V <= nvec;
  const bool full = whole && L.V % 32 == 0;   // every lane has a vector in every round
  // The slot-table steady state also takes tiles of any length V >= 32 (a
  // partial last round, see lut_task); the fused product and the search path's
  // steady state need whole rounds.
  const bool lut_ok = whole && (full || (!DOT && L.V >= 32));
  if (L.pay_bytes < kFastOob && ((PATH == kPathSearch && full) || (B == 11 && lut_ok))) {
    if constexpr (PATH != kPathSearch && B == 11) {
      if (lut_task_any<B, PATH == kPathWide, DOT>(L, lb, ring_area, t0, status)) return;
    } else if constexpr (PATH == kPathSearch) {
      if (decode_task_fast_any<PATH, B, DOT>(L, lb, ring_area, task, status)) return;
    }
  }
  // generic loop
  if (full) decode_task<PATH, B, kChains, true, DOT>(L, tab, lb, ring_area, task, status);
  else decode_task<PATH, B, kChains, false, DOT>(L, tab, lb, ring_area, task, status);
}

template <int PATH, bool DOT, bool SMALL = false>
__device__ __forceinline__ void dispatch_task(const Hot& L, const uint32_t* tab, uint8_t* lb,
                                              uint32_t ring_area, uint32_t task, int32_t* status) {
  if (PATH == kPathSearch || PATH == kPathGlobal) task_b<PATH, 0, DOT, SMALL>(L, tab, lb, ring_area, task, status);
  else if (L.b == 11) task_b<PATH, 11, DOT, SMALL>(L, tab, lb, ring_area, task, status);
  else if (L.b == 10) task_b<PATH, 10, DOT, SMALL>(L, tab, lb, ring_area, task, status);
  else task_b<PATH, 9, DOT, SMALL>(L, tab, lb, ring_area, task, status);
}

// Decode global tasks [t_begin, t_end) of a layer list: per layer segment the
// workgroup builds that layer's tables, then its waves take tasks in turn.
// DOT: the fused product (every layer's output mode is kOutDotI8).
// Prepared stacks: copy the layer's decode tables, built once by the stack's
// preparation, from global memory into LDS with direct loads (memory to LDS,
// no registers): one wave instruction moves 1 KiB, lane l writing 16 bytes at
// l * 16.  Bytes past the image read as 0 (buffer bounds) and land in the ring
// area, which every task initialises after the barrier that follows.
typedef __attribute__((address_space(3))) uint8_t lds_u8;
template <int PATH>
__device__ __forceinline__ void load_tables(const LayerDev& L, uint32_t* lds) {
  const uint32_t bytes = ring_offset<PATH>(L);
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(L.tables), (short)0, (int)bytes, 0x00020000);
  const uint32_t lane = threadIdx.x & 63;
  for (uint32_t c = wave_id() * 1024u; c < bytes; c += kWavesPerGroup * 1024u)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_u8*)lds + c, 16, c + 16 * lane, 0, 0, 0);
  __builtin_amdgcn_s_waitcnt(0);
}

// One layer segment of a workgroup: build (or copy) the layer's tables, then
// the waves take tasks [seg, seg_end) in turn.
template <int PATH, bool DOT, bool SMALL = false>
__device__ __forceinline__ void run_segment(const LayerDev& L, uint32_t* lds, uint32_t seg,
                                            uint32_t seg_end, int32_t* status) {
  if (L.tables) load_tables<PATH>(L, lds);
  else build_tables<PATH>(L, lds);
  __syncthreads();
  const uint32_t ring_area = uni(ring_offset<PATH>(L));
  const uint32_t first = uni(L.task_begin);
  const Hot H = make_hot(L);
  uint8_t* lb = reinterpret_cast<uint8_t*>(lds);
  for (uint32_t task = seg + wave_id(); task < seg_end; task += kWavesPerGroup)
    dispatch_task<PATH, DOT, SMALL>(H, lds, lb, ring_area, task - first, status);
}

// A layer list whose layers take different decode paths: each segment runs
// the kernel family of its own layer (the path is uniform over the workgroup).
constexpr int kPathMixed = 15;

// Decode global tasks [t_begin, t_end) of a layer list: per layer segment the
// workgroup builds that layer's tables, then its waves take tasks in turn.
// DOT: the fused product (every layer's output mode is kOutDotI8).
template <int PATH, bool DOT = false>
__device__ __forceinline__ void run_layers(const LayerDev* layers, int n_layers, uint32_t total,
                           uint32_t per_group, int32_t* status) {
  extern __shared__ uint32_t lds[];
  const uint32_t t_begin = blockIdx.x * per_group;
  const uint32_t t_end = min(total, t_begin + per_group);
  if (t_begin >= t_end) return;
  int li = 0;
  while (li + 1 < n_layers && layers[li + 1].task_begin <= t_begin) li++;
  for (uint32_t seg = t_begin; seg < t_end && li < n_layers; li++) {
    const LayerDev& L = layers[li];
    const uint32_t seg_end = min(t_end, L.task_begin + L.n_tasks);
    if (seg_end <= seg) continue;
    __syncthreads();
    if constexpr (PATH == kPathMixed) {
      switch (uni(L.path)) {
        case kPathLut: run_segment<kPathLut, DOT>(L, lds, seg, seg_end, status); break;
        case kPathWide: run_segment<kPathWide, DOT>(L, lds, seg, seg_end, status); break;
        case kPathSearch: run_segment<kPathSearch, DOT>(L, lds, seg, seg_end, status); break;
        default: run_segment<kPathGlobal, DOT>(L, lds, seg, seg_end, status); break;
      }
    } else {
      // a single-path kernel may run two-tile tasks; the mixed-path kernel
      // (above) never does (use_small_tasks)
      run_segment<PATH, DOT, true>(L, lds, seg, seg_end, status);
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
  // The list is the first kernel argument: index it in the kernel-argument
  // segment itself (scalar loads) instead of copying the by-value struct.
#if defined(__HIP_DEVICE_COMPILE__)
  (void)list;
  const LayerDev* layers = (const LayerDev*)__builtin_amdgcn_kernarg_segment_ptr();
#else
  const LayerDev* layers = list.L;
#endif
  run_layers<PATH>(layers, n_layers, total, per_group, status);
}

// The fused decode and product, in kernels of its own: its steady state needs
// more registers than the decode's, and sharing a kernel would give every
// decode launch its scratch allocation.
template <int PATH>
__global__ __launch_bounds__(kThreads) void decode_dot_kernel(const LayerList list, int n_layers,
                                                              uint32_t total, uint32_t per_group,
                                                              int32_t* status) {
#if defined(__HIP_DEVICE_COMPILE__)
  (void)list;
  const LayerDev* layers = (const LayerDev*)__builtin_amdgcn_kernarg_segment_ptr();
#else
  const LayerDev* layers = list.L;
#endif
  run_layers<PATH, true>(layers, n_layers, total, per_group, status);
}

template <int PATH>
__global__ __launch_bounds__(kThreads) void decode_ws_kernel(const LayerDev* __restrict__ layers,
                                                             int n_layers,
                                                             uint32_t total, uint32_t per_group,
                                                             int32_t* status) {
  run_layers<PATH>(layers, n_layers, total, per_group, status);
}

// ---- fused decode and MFMA product (any number of rows of X) ----------------------
// Y[t][r] = sum_j X[t][j] W'[r][j] for an INT8-container tensor, with W' never
// written as a whole.  A matrix core needs 16 rows of W' at the same columns,
// and the tiles of the format are row segments, so each workgroup owns a block
// of RB consecutive rows (RB = ceil(R / CUs), so that every block runs at once):
// it decodes every tile that touches its block (the row-major INT8 values) into
// a slab of the caller's workspace, which stays in L2 and the last-level cache,
// then its waves multiply X by the slab's rows with v_mfma_i32_16x16x64_i8.  A
// tile can span a block boundary: both blocks decode it, each keeping the rows
// it owns (the slab has `margin` rows on either side for the rest).
struct GemmArgs {
  const void* x;         // m x C, row-major: int8, or bf16 for the BF16 product
  void* y;               // m x R, row-major: int32, or fp32 (cleared first when K is split over waves)
  uint8_t* slabs;        // one slab per workgroup
  uint64_t slab_bytes;   // (RB + 2 margin) x C, rounded up to 256
  uint32_t m, margin, n_blocks, rows_per_block;
};

struct GemmLaunch {
  LayerDev L;
  GemmArgs g;
};

constexpr uint32_t kGemmMaxTiles = 4;   // NT <= 4: blocks of at most 64 rows

// Whether a product of T tiles of X (16 rows each) takes the kernels whose work
// items hold several X tiles: more than 32 rows of X.
__host__ __device__ inline bool gemm_wide(uint32_t t) { return t > 2; }

// X tiles per work item of a block's product, for NT slab tiles and T tiles of
// X: one in the kernels for up to 32 rows of X; above, four when the block has
// a single slab tile, two when it has two or three.  2 kGroup (XT + NT)
// fragments and XT NT accumulators of 4 VGPRs each (at most 64 registers)
// then fit in what the decode leaves.  Every item reads the block's slab once,
// so fewer items read it fewer times.
__host__ __device__ constexpr uint32_t gemm_x_tiles(uint32_t nt, bool wide) {
  return !wide || nt > 3 ? 1u : nt == 1 ? 4u : 2u;
}

// Whether the product splits K over waves, adding partial sums to Y with
// atomics (Y must then start at zero): fewer work items than waves.
__host__ __device__ inline bool gemm_splits_k(uint32_t nt, uint32_t t) {
  const uint32_t xt = gemm_x_tiles(nt, gemm_wide(t));
  return (t + xt - 1) / xt < (uint32_t)kWavesPerGroup;
}

// The product kernels (decode_gemm_kernel) are in decode_gemm.hip.

// Prepared stacks: workgroup i builds layer i's decode tables in LDS, exactly as
// a decode launch would, and writes them to the layer's table image.
template <int PATH>
__device__ __forceinline__ void build_and_store(const LayerDev& L, uint32_t* lds) {
  build_tables<PATH>(L, lds);
  __syncthreads();
  const uint32_t n16 = ring_offset<PATH>(L) / 16;
  EP_GLOBAL u32x4* dst = gptr<u32x4>(L.tables);
  const u32x4* src = reinterpret_cast<const u32x4*>(lds);
  for (uint32_t i = threadIdx.x; i < n16; i += kThreads) dst[i] = src[i];
}

__global__ __launch_bounds__(kThreads) void stack_tables_kernel(const LayerDev* __restrict__ layers) {
  extern __shared__ uint32_t lds[];
  const LayerDev& L = layers[blockIdx.x];
  switch (uni(L.path)) {
    case kPathLut: build_and_store<kPathLut>(L, lds); break;
    case kPathWide: build_and_store<kPathWide>(L, lds); break;
    case kPathSearch: build_and_store<kPathSearch>(L, lds); break;
    default: build_and_store<kPathGlobal>(L, lds); break;
  }
}

}  // namespace
}  // namespace ep
