// INT8 x INT8 -> INT32 matrix product on gfx950 MFMA, for decode-then-GEMM:
// Y[M x N] = A[M x K] * B[N x K]^T, both operands K-contiguous (row-major A,
// row-major B = the decoded weight matrix as stored), exact int32 accumulation.
//
// Tiling: a workgroup of 256 threads (4 waves, 2 x 2) owns a 256 x 256 tile of
// Y; each wave owns 128 x 128 = 4 x 4 blocks of v_mfma_i32_32x32x32_i8 (256
// accumulator registers), which reads 8 KiB of LDS operands (eight 16-byte
// fragments per lane) per 32-byte K chunk for 16 MFMAs.  One workgroup per
// CU, one wave per SIMD.  K is walked in steps of 128 bytes (four chunks).
//
// Operands reach LDS by direct loads (buffer_load ... lds: memory to LDS
// without passing through registers), one wave instruction per 8 rows x 128
// bytes, so that eight lanes cover one whole 128-byte line of a row.  (With
// 64-byte row pieces each line is requested twice, in consecutive steps, and
// a CU's stream of direct loads runs at about 60 % of the rate it reaches
// with whole lines.)  Two stage buffers of 64 KiB alternate.  Per step s
// (buffer s mod 2 holds step s, and step s + 1 is in flight):
//   chunks 1..3: the MFMAs of chunk c - 1 while the fragments of chunk c are
//           read;
//   barrier (this wave's loads of step s + 1 landed, its LDS reads returned);
//   then step s + 2 is requested into buffer s mod 2, which every wave has
//   finished reading, and the MFMAs of chunk 3 run while the chunk-0
//   fragments of step s + 1 are read.
// A step's loads thus have a whole step of MFMAs to land.  The single barrier
// sits between two MFMA groups whose operands are already in registers.
// Direct loads are bounded buffer loads: out-of-range chunks land as zeros.
//
// Tile order: workgroups are dealt to the 8 XCDs round-robin, so the
// workgroup id is remapped so that each XCD runs a contiguous range of tiles,
// walked in groups of four tile rows (the 32 tiles an XCD holds at once share
// 4 A panels and 8 B panels in its L2).  When the last round of whole tiles
// would occupy at most half of the CUs, its tiles are issued as twice as many
// 256 x 128 halves instead, so that round takes about half as long.
//
// LDS rows are 128 bytes (eight 16-byte chunks) without padding; the chunk j
// of row r is stored at position j ^ swz(r), swz(r) = (r mod 8) ^ ((r / 8)
// mod 2).  Any 8 consecutive rows then hold one chunk in 8 different 16-byte
// bank groups (32 banks), and any 16 consecutive rows in 16 different groups
// of a 256-byte bank row (64 banks), so the fragment reads (32 consecutive
// rows at one chunk) are free of bank conflicts; the direct loads write 1 KiB
// contiguously.
//
// MFMA operand layout (32x32x32, int8): lane l supplies row (l mod 32) of the
// A block and column (l mod 32) of the B block, 16 consecutive k bytes each,
// lanes 0-31 the k bytes [0, 16) and lanes 32-63 [16, 32) of the 32-byte k
// chunk.  Accumulator register r of lane l holds element
// (8 (r / 4) + 4 (l / 32) + r mod 4, l mod 32) of the 32 x 32 block.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <type_traits>

#include "../../include/entropack.h"
#include "common.h"

namespace ep {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kTileM = 256, kTileK = 128;
constexpr int kWaveM = 128;                         // per wave: 4 x (TN / 64) blocks of 32 x 32
constexpr int kBlocksM = kWaveM / 32;
constexpr int kGemmThreads = 256;
constexpr int kRowBytes = kTileK;                   // no padding: chunks are swizzled

#define EP_GLOBAL __attribute__((address_space(1)))

constexpr uint32_t kOutside = 0x80000000u;   // operands are limited to 2^31 bytes

__device__ __forceinline__ uint32_t swz(uint32_t r) { return (r & 7) ^ ((r >> 3) & 1); }

typedef __attribute__((address_space(3))) uint8_t lds_u8;

// Per-thread part of the direct (global -> LDS) loads of one K step: an
// operand's 128-byte pieces of 256 (A) or TN (B) rows go to one 32 KiB slot,
// cut into 1 KiB segments of 8 rows; one wave instruction fills one segment,
// lane l writing the 16 bytes at l * 16, i.e. slot (l mod 8) of row l / 8 of
// the segment, so the lane loads chunk (l mod 8) ^ swz(row) of that row.
// Wave w fills segments w + 4 q.
template <int TN>
struct PanelLoader {
  static constexpr int kSegsA = kTileM / 32, kSegsB = TN / 32;   // per wave
  uint32_t a_off[kSegsA], b_off[kSegsB];   // byte offset of the row start, or kOutside
  uint32_t chunk;            // byte offset of the lane's chunk within a 128-byte K step
  uint32_t seg0;             // LDS offset of the wave's first segment

  __device__ __forceinline__ void init(int64_t m, int64_t n, int64_t k, int64_t m0, int64_t n0,
                                       int wave, int lane) {
    const uint32_t r = (uint32_t)lane >> 3;   // row within the segment
    // slot row 8 (wave + 4 q) + r: its value mod 16 is 8 (wave mod 2) + r for every q
    chunk = 16 * (((uint32_t)lane & 7) ^ swz(8 * ((uint32_t)wave & 1) + r));
    seg0 = 1024 * wave;
#pragma unroll
    for (int q = 0; q < kSegsA; q++) {
      const int64_t g = m0 + 8 * (wave + 4 * q) + r;
      a_off[q] = g < m ? (uint32_t)(g * k) : kOutside;
    }
#pragma unroll
    for (int q = 0; q < kSegsB; q++) {
      const int64_t g = n0 + 8 * (wave + 4 * q) + r;
      b_off[q] = g < n ? (uint32_t)(g * k) : kOutside;
    }
  }
  // segments [Q0, Q1) of the step at K offset k0 into `slot`; bytes at or past
  // k_end land as zeros
  template <int Q0, int Q1, int NQ>
  __device__ __forceinline__ static void fetch(const uint32_t (&off)[NQ], uint32_t chunk, uint32_t seg0,
                                               __amdgpu_buffer_rsrc_t rsrc, int64_t k_end, int64_t k0,
                                               lds_u8* slot) {
    const int64_t kk = k0 + chunk;
#pragma unroll
    for (int q = Q0; q < Q1; q++) {
      const uint32_t o = (kk < k_end && off[q] != kOutside) ? off[q] + (uint32_t)kk : kOutside;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, slot + seg0 + 4096 * q, 16, o, 0, 0, 0);
    }
  }
  template <int Q0, int Q1>
  __device__ __forceinline__ void fetch_a(__amdgpu_buffer_rsrc_t ra, int64_t k_end, int64_t k0, lds_u8* slot) const {
    fetch<Q0, Q1>(a_off, chunk, seg0, ra, k_end, k0, slot);
  }
  template <int Q0, int Q1>
  __device__ __forceinline__ void fetch_b(__amdgpu_buffer_rsrc_t rb, int64_t k_end, int64_t k0, lds_u8* slot) const {
    fetch<Q0, Q1>(b_off, chunk, seg0, rb, k_end, k0, slot);
  }
};

// Workgroup barrier for the direct-load pipeline: this wave's LDS reads have
// returned and at most N of its direct loads are still in flight, then
// s_barrier.  (A fenced barrier would also wait for the N newest direct
// loads, which are meant to stay in flight across it.)  The scheduling
// barriers keep the compiler from moving LDS accesses across it.
template <int N>
__device__ __forceinline__ void stage_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));   // vmcnt(N) lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

constexpr int kXcds = 8, kGroupRows = 4;

// Workgroups are dealt to the XCDs round-robin: spread the ids [0, count) so
// that each XCD takes a contiguous range of `per` indices.
__device__ __forceinline__ uint32_t xcd_spread(uint32_t id, uint32_t count) {
  const uint32_t per = count / kXcds;
  return id < per * kXcds ? (id % kXcds) * per + id / kXcds : id;
}

// Tile (row, column) of tile index `idx` among tm x tn tiles, taken in groups
// of kGroupRows tile rows, column by column within a group.
__device__ __forceinline__ void tile_of(uint32_t idx, uint32_t tm, uint32_t tn, uint32_t& ti,
                                        uint32_t& tj) {
  const uint32_t group = idx / (kGroupRows * tn), first = group * kGroupRows;
  const uint32_t rows = tm - first < kGroupRows ? tm - first : kGroupRows;
  const uint32_t q = idx - first * tn;
  ti = first + q % rows;
  tj = q / rows;
}

constexpr int kTileN = 256;
constexpr int kSlots = 5;                          // LDS ring of operand panels
constexpr int kSlotBytes = kTileM * kRowBytes;     // 32 KiB: one operand's rows for one K step
constexpr int kChunks = kTileK / 32;               // 32-byte MFMA K chunks per step

// Y[m0 .. m0 + 256, n0 .. n0 + TN), summed over K in [k_lo, k_hi) (k_lo a
// multiple of the 128-byte step); a wave owns 128 x TN / 2.  With ADD the
// sums are added to Y by atomics (a K range of a split tile), else stored.
//
// The ring: slot j mod 5 holds the j-th panel of the sequence A(0), B(0),
// A(1), B(1), ... (A(t), B(t): the operands' rows for K step t).  Iteration t
// reads A(t), B(t) and loads B(t + 1), A(t + 2) into the slots of A(t - 1),
// B(t - 1), which the barrier ending iteration t - 1 released.  Its barrier
// waits for B(t + 1) (A(t + 1) is older) and lets A(t + 2) stay in flight.
// Each of the four sections of an iteration runs the MFMAs of one chunk,
// with the fragment reads of the next chunk and a quarter of the loads
// between them, so the loads are spread thinly over the whole step: issued
// in bursts they stall the wave (its SIMD has no other wave to feed the
// matrix pipe) while the CU's load path drains.
template <int TN, bool ADD>
__device__ __forceinline__ void tile_product(const int8_t* a, const int8_t* b, int32_t* y, int64_t m,
                                             int64_t n, int64_t k, int64_t m0, int64_t n0,
                                             int64_t k_lo, int64_t k_hi, lds_u8* lds) {
  constexpr int kWaveN = TN / 2, kBlocksN = kWaveN / 32;
  constexpr int kFrags = kBlocksM + kBlocksN, kMfmas = kBlocksM * kBlocksN;
  using Loader = PanelLoader<TN>;
  constexpr int kSegsA = Loader::kSegsA, kSegsB = Loader::kSegsB;
  static_assert(kWaveN % 32 == 0 && TN % 64 == 0 && TN <= kTileM, "tile width");
  static_assert(kFrags < kMfmas && kSegsB % 2 == 0 && kSegsA % 2 == 0, "schedule");
  static_assert(kChunks == 4, "an iteration walks four chunks");
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wm = wave >> 1, wn = wave & 1;   // wave's 128 x TN / 2 block of the tile
  const int64_t steps = (k_hi - k_lo + kTileK - 1) / kTileK;

  v16i acc[kBlocksM][kBlocksN];
#pragma unroll
  for (int i = 0; i < kBlocksM; i++)
#pragma unroll
    for (int j = 0; j < kBlocksN; j++) acc[i][j] = v16i{};

  const __amdgpu_buffer_rsrc_t ra =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(a), (short)0, (int)(m * k), 0x00020000);
  const __amdgpu_buffer_rsrc_t rb =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(b), (short)0, (int)(n * k), 0x00020000);
  Loader ld;
  ld.init(m, n, k, m0, n0, wave, lane);

  // fragment addresses: row (l mod 32) of each block, 16-byte chunk 2 c + l / 32
  // for the 32-byte K chunk c, swizzled (row mod 16 = l mod 16 for every block)
  const uint32_t fr = lane & 31, fh = lane >> 5, fs = swz(lane & 15);
  const uint32_t fa = (kWaveM * wm + fr) * kRowBytes, fb = (kWaveN * wn + fr) * kRowBytes;

  v4i xa0[kBlocksM], xb0[kBlocksN], xa1[kBlocksM], xb1[kBlocksN];   // fragments of two chunks

  auto read_frags = [&](const lds_u8* pa, const lds_u8* pb, int c, v4i* xa, v4i* xb) {
    const uint32_t o = 16 * ((2 * c + fh) ^ fs);
#pragma unroll
    for (int i = 0; i < kBlocksM; i++)
      xa[i] = *reinterpret_cast<const __attribute__((address_space(3))) v4i*>(pa + fa + o + 32 * kRowBytes * i);
#pragma unroll
    for (int j = 0; j < kBlocksN; j++)
      xb[j] = *reinterpret_cast<const __attribute__((address_space(3))) v4i*>(pb + fb + o + 32 * kRowBytes * j);
  };
  auto mfmas = [&](const v4i* xa, const v4i* xb) {
#pragma unroll
    for (int i = 0; i < kBlocksM; i++)
#pragma unroll
      for (int j = 0; j < kBlocksN; j++)
        acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(xa[i], xb[j], acc[i][j], 0, 0, 0);
  };
  // one section's order: an MFMA, then a fragment read, until the reads are
  // out; then an MFMA and its share of the section's L loads.  The reads come
  // first in program order too: the compiler keeps LDS reads and direct loads
  // in the order written.
  auto section = [&](auto loads) {
    constexpr int L = decltype(loads)::value;
    constexpr int kPer = (L + kMfmas - kFrags - 1) / (kMfmas - kFrags);
#pragma unroll
    for (int r = 0; r < kMfmas; r++) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (r < kFrags) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      else if ((r - kFrags) * kPer < L) __builtin_amdgcn_sched_group_barrier(0x020, kPer, 0);
    }
  };
  using HalfB = std::integral_constant<int, kSegsB / 2>;
  using HalfA = std::integral_constant<int, kSegsA / 2>;

  auto slot = [&](uint32_t j) { return lds + kSlotBytes * (j < kSlots ? j : j - kSlots); };
  ld.template fetch_a<0, kSegsA>(ra, k_hi, k_lo, slot(0));
  ld.template fetch_b<0, kSegsB>(rb, k_hi, k_lo, slot(1));
  ld.template fetch_a<0, kSegsA>(ra, k_hi, k_lo + kTileK, slot(2));
  stage_barrier<kSegsA>();
#pragma unroll
  for (int i = 0; i < kBlocksM; i++) xa1[i] = v4i{};
#pragma unroll
  for (int j = 0; j < kBlocksN; j++) xb1[j] = v4i{};

  uint32_t j0 = 0;   // slot of A(t)
  for (int64_t s = 0; s < steps; s++) {
    const lds_u8* const pa = slot(j0);
    const lds_u8* const pb = slot(j0 + 1);
    lds_u8* const qb = slot(j0 + 3);   // B(s + 1)
    lds_u8* const qa = slot(j0 + 4);   // A(s + 2)
    const int64_t kb = k_lo + (s + 1) * kTileK, ka = k_lo + (s + 2) * kTileK;
    // chunk 3 of step s - 1 (zeros before the first step) while chunk 0 is read
    read_frags(pa, pb, 0, xa0, xb0);
    ld.template fetch_b<0, kSegsB / 2>(rb, k_hi, kb, qb);
    mfmas(xa1, xb1);
    section(HalfB{});
    read_frags(pa, pb, 1, xa1, xb1);
    ld.template fetch_b<kSegsB / 2, kSegsB>(rb, k_hi, kb, qb);
    mfmas(xa0, xb0);
    section(HalfB{});
    read_frags(pa, pb, 2, xa0, xb0);
    ld.template fetch_a<0, kSegsA / 2>(ra, k_hi, ka, qa);
    mfmas(xa1, xb1);
    section(HalfA{});
    read_frags(pa, pb, 3, xa1, xb1);
    ld.template fetch_a<kSegsA / 2, kSegsA>(ra, k_hi, ka, qa);
    mfmas(xa0, xb0);
    section(HalfA{});
    // B(s + 1) has landed for this wave and every read of A(s), B(s) is done;
    // then for every wave
    stage_barrier<kSegsA>();
    j0 = j0 + 2 < kSlots ? j0 + 2 : j0 + 2 - kSlots;
  }
  mfmas(xa1, xb1);                 // chunk 3 of the last step
  __builtin_amdgcn_s_waitcnt(0);   // direct loads still in flight land before the wave ends

  const int half = lane >> 5;
#pragma unroll
  for (int i = 0; i < kBlocksM; i++)
#pragma unroll
    for (int j = 0; j < kBlocksN; j++) {
      const int64_t col = n0 + kWaveN * wn + 32 * j + fr;
#pragma unroll
      for (int r = 0; r < 16; r++) {
        const int64_t row = m0 + kWaveM * wm + 32 * i + 8 * (r >> 2) + 4 * half + (r & 3);
        if (row < m && col < n) {
          EP_GLOBAL int32_t* const p = (EP_GLOBAL int32_t*)y + row * n + col;
          if (ADD) __hip_atomic_fetch_add(p, acc[i][j][r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          else *p = acc[i][j][r];
        }
      }
    }
}

// Workgroups [0, full) take whole 256 x 256 tiles; when the last round of
// whole tiles would fill at most half the CUs, its `split` tiles are instead
// taken as 2 * split half-width (256 x 128) tiles by workgroups [full, ..),
// so that round lasts about half as long.  With parts > 1 (a launch of few
// tiles) each of those units is taken by `parts` workgroups, each summing a
// range of `part_steps` K steps into Y with atomics (Y cleared before).
template <bool ADD>
__device__ __forceinline__ void gemm_unit(const int8_t* a, const int8_t* b, int32_t* y, int64_t m,
                                          int64_t n, int64_t k, uint32_t tm, uint32_t tn,
                                          uint32_t full, uint32_t split, uint32_t id, int64_t k_lo,
                                          int64_t k_hi, lds_u8* lds) {
  uint32_t ti, tj;
  if (id < full) {
    tile_of(xcd_spread(id, full), tm, tn, ti, tj);
    tile_product<kTileN, ADD>(a, b, y, m, n, k, (int64_t)ti * kTileM, (int64_t)tj * kTileN, k_lo,
                              k_hi, lds);
  } else {
    const uint32_t u = xcd_spread(id - full, 2 * split);
    tile_of(full + u / 2, tm, tn, ti, tj);
    tile_product<kTileN / 2, ADD>(a, b, y, m, n, k, (int64_t)ti * kTileM,
                                  (int64_t)tj * kTileN + (kTileN / 2) * (u & 1), k_lo, k_hi, lds);
  }
}

__global__ __launch_bounds__(kGemmThreads) void gemm_i8_nt_kernel(const int8_t* __restrict__ a,
                                                                  const int8_t* __restrict__ b,
                                                                  int32_t* __restrict__ y,
                                                                  int64_t m, int64_t n, int64_t k,
                                                                  uint32_t tm, uint32_t tn,
                                                                  uint32_t full, uint32_t split,
                                                                  uint32_t parts, uint32_t part_steps) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds_mem[kSlots * kSlotBytes];
  lds_u8* const lds = (lds_u8*)lds_mem;
  if (parts == 1) {
    gemm_unit<false>(a, b, y, m, n, k, tm, tn, full, split, blockIdx.x, 0, k, lds);
  } else {
    const uint32_t unit = blockIdx.x / parts, part = blockIdx.x % parts;
    const int64_t k_lo = (int64_t)part * part_steps * kTileK;
    const int64_t k_hi = k_lo + (int64_t)part_steps * kTileK < k ? k_lo + (int64_t)part_steps * kTileK : k;
    if (k_lo < k_hi) gemm_unit<true>(a, b, y, m, n, k, tm, tn, full, split, unit, k_lo, k_hi, lds);
  }
}

__global__ void zero_i32_kernel(int32_t* __restrict__ y, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * blockDim.x)
    ((EP_GLOBAL int32_t*)y)[i] = 0;
}

}  // namespace
}  // namespace ep

extern "C" int ep_gemm_i8_nt(const int8_t* d_a, const int8_t* d_b, int32_t* d_y, int64_t m,
                             int64_t n, int64_t k, void* hip_stream) {
  if (!d_a || !d_b || !d_y) return ep::fail(EP_ERR_ARG, "ep_gemm_i8_nt: null pointer");
  if (m <= 0 || n <= 0 || k <= 0 || k % 16)
    return ep::fail(EP_ERR_ARG, "ep_gemm_i8_nt: need m, n, k > 0 and k % 16 == 0");
  if ((reinterpret_cast<uintptr_t>(d_a) | reinterpret_cast<uintptr_t>(d_b)) & 15)
    return ep::fail(EP_ERR_ARG, "ep_gemm_i8_nt: operands must be 16-byte aligned");
  // |a * b| <= 128 * 128 = 2^14, so a K-term sum stays below 2^31 for K <= 131071
  if (k > 131071)
    return ep::fail(EP_ERR_ARG, "ep_gemm_i8_nt: k above 131071 may overflow the int32 sums");
  if (m * k >= (int64_t)ep::kOutside || n * k >= (int64_t)ep::kOutside)
    return ep::fail(EP_ERR_ARG, "ep_gemm_i8_nt: an operand above 2^31 bytes");
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return ep::fail(EP_ERR_HIP, "ep_gemm_i8_nt: no device");
  const int64_t tm = (m + ep::kTileM - 1) / ep::kTileM, tn = (n + ep::kTileN - 1) / ep::kTileN;
  const int64_t tiles = tm * tn, last = tiles % cus;
  if (tiles + last > 0x7FFFFFFF) return ep::fail(EP_ERR_ARG, "ep_gemm_i8_nt: matrix too large");
  const int64_t split = (last > 0 && 2 * last <= cus) ? last : 0;   // one workgroup per CU
  // A launch of at most half as many units (whole or half tiles) as CUs splits
  // K over `parts` workgroups per unit, at least four 128-byte steps each.
  const int64_t units = tiles + split, steps = (k + ep::kTileK - 1) / ep::kTileK;
  int64_t parts = 1;
  if (2 * units <= cus) parts = std::max<int64_t>(1, std::min<int64_t>(cus / units, steps / 4));
  const int64_t part_steps = (steps + parts - 1) / parts;
  const hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  if (parts > 1) {
    const int64_t count = m * n;
    const unsigned blocks = (unsigned)std::min<int64_t>((count + 255) / 256, 4096);
    hipLaunchKernelGGL(ep::zero_i32_kernel, dim3(blocks), dim3(256), 0, stream, d_y, count);
  }
  hipLaunchKernelGGL(ep::gemm_i8_nt_kernel, dim3((unsigned)(units * parts)), dim3(ep::kGemmThreads), 0,
                     stream, d_a, d_b, d_y, m, n, k, (uint32_t)tm, (uint32_t)tn,
                     (uint32_t)(tiles - split), (uint32_t)split, (uint32_t)parts, (uint32_t)part_steps);
  if (hipGetLastError() != hipSuccess) return ep::fail(EP_ERR_HIP, "ep_gemm_i8_nt: launch failed");
  return EP_OK;
}
