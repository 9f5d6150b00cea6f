// INT8 x INT8 -> INT32 matrix product on gfx950 MFMA, for decode-then-GEMM:
// Y[M x N] = A[M x K] * B[N x K]^T, both operands K-contiguous (row-major A,
// row-major B = the decoded weight matrix as stored), exact int32 accumulation.
//
// Tiling: a workgroup of 256 threads (4 waves, 2 x 2) owns a 256 x 256 tile of
// Y; each wave owns 128 x 128 = 4 x 4 blocks of v_mfma_i32_32x32x32_i8 (256
// accumulator registers), which reads 8 KiB of LDS operands (eight 16-byte
// fragments per lane) per 32-byte K chunk for 16 MFMAs.  One workgroup per
// CU, one wave per SIMD.  K is walked in steps of 64 bytes (two chunks).
//
// Operands reach LDS by direct loads (buffer_load ... lds: memory to LDS
// without passing through registers) into four rotating stage buffers, three
// steps ahead.  Per step s (buffer s mod 4 holds step s):
//   half A: MFMAs of chunk 0 (fragments already in registers); meanwhile
//           step s + 3 is requested into the buffer step s - 1 used and the
//           chunk-1 fragments of step s are read;
//   barrier (this wave's loads of step s + 1 landed, its LDS reads returned);
//   half B: MFMAs of chunk 1; meanwhile the chunk-0 fragments of step s + 1
//           are read.
// The single barrier sits between two MFMA halves whose operands are already
// in registers, so the matrix pipe does not wait on LDS latency, and it
// orders every wave's last read of a buffer before the next load into it.
// Direct loads are bounded buffer loads: out-of-range chunks land as zeros.
//
// Tile order: workgroups are dealt to the 8 XCDs round-robin, so the
// workgroup id is remapped so that each XCD runs a contiguous range of tiles,
// walked in groups of four tile rows (the 32 tiles an XCD holds at once share
// 4 A panels and 8 B panels in its L2).  When the last round of whole tiles
// would occupy at most half of the CUs, its tiles are issued as twice as many
// 256 x 128 halves instead, so that round takes about half as long.
//
// LDS rows are 64 bytes (four 16-byte chunks) without padding; the chunk j of
// row r is stored at position j ^ swz(r), with swz a fixed 16-entry table over
// r mod 16 chosen so that neither the direct loads (16 rows x 64 bytes per
// wave instruction) nor the fragment reads (32 consecutive rows at one chunk)
// put two lanes of an LDS cycle on the same bank, for 32 or 64 banks.
//
// MFMA operand layout (32x32x32, int8): lane l supplies row (l mod 32) of the
// A block and column (l mod 32) of the B block, 16 consecutive k bytes each,
// lanes 0-31 the k bytes [0, 16) and lanes 32-63 [16, 32) of the 32-byte k
// chunk.  Accumulator register r of lane l holds element
// (8 (r / 4) + 4 (l / 32) + r mod 4, l mod 32) of the 32 x 32 block.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/entropack.h"
#include "common.h"

namespace ep {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kTileM = 256, kTileK = 64;
constexpr int kWaveM = 128;                         // per wave: 4 x (TN / 64) blocks of 32 x 32
constexpr int kBlocksM = kWaveM / 32;
constexpr int kGemmThreads = 256;
constexpr int kRowBytes = kTileK;                   // no padding: chunks are swizzled
constexpr int kABytes = kTileM * kRowBytes;
constexpr uint32_t kSwizzle = 0x63c99e34u;          // swz(r) = bits [2 (r mod 16), +2)

#define EP_GLOBAL __attribute__((address_space(1)))

constexpr uint32_t kOutside = 0x80000000u;   // operands are limited to 2^31 bytes

__device__ __forceinline__ uint32_t swz(uint32_t r) { return (kSwizzle >> (2 * (r & 15))) & 3; }

typedef __attribute__((address_space(3))) uint8_t lds_u8;

// Per-thread part of the direct (global -> LDS) load of one K step of the
// stage: the stage is 16 KiB of A rows then TN / 16 KiB of B rows, cut into
// 1 KiB segments of 16 rows; one wave instruction fills one segment, lane l
// writing the 16 bytes at l * 16, i.e. slot (l mod 4) of row l / 4 of the
// segment, so the lane loads chunk (l mod 4) ^ swz(row) of that row.  Wave w
// fills segments w + 4 q.
template <int TN>
struct StageLoader {
  static constexpr int kSegs = (kTileM + TN) / 16 / 4;   // per wave
  uint32_t row_off[kSegs];   // byte offset of the row start in its operand, or kOutside
  uint32_t chunk;            // byte offset of the lane's chunk within a 64-byte K step
  uint32_t seg0;             // LDS offset of the wave's first segment

  __device__ __forceinline__ void init(int64_t m, int64_t n, int64_t k, int64_t m0, int64_t n0,
                                       int wave, int lane) {
    const uint32_t r = (uint32_t)lane >> 2;   // row within the segment = row mod 16
    chunk = 16 * (((uint32_t)lane & 3) ^ swz(r));
    seg0 = 1024 * wave;
#pragma unroll
    for (int q = 0; q < kSegs; q++) {
      const int64_t row = 16 * (wave + 4 * q) + r;   // stage row
      const bool is_a = q < kTileM / 64;
      const int64_t g = is_a ? m0 + row : n0 + row - kTileM;
      row_off[q] = g < (is_a ? m : n) ? (uint32_t)(g * k) : kOutside;
    }
  }
  __device__ __forceinline__ void fetch(__amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rb,
                                        int64_t k, int64_t k0, lds_u8* stage) const {
    const int64_t kk = k0 + chunk;
#pragma unroll
    for (int q = 0; q < kSegs; q++) {
      const uint32_t off = (kk < k && row_off[q] != kOutside) ? row_off[q] + (uint32_t)kk : kOutside;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(q < kTileM / 64 ? ra : rb, stage + seg0 + 4096 * q, 16,
                                               off, 0, 0, 0);
    }
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
constexpr int kStages = 4;   // LDS stage buffers: loads run kStages - 1 steps ahead
constexpr int stage_bytes(int tn) { return kABytes + tn * kRowBytes; }   // A tile then B tile

// Y[m0 .. m0 + 256, n0 .. n0 + TN) over all of K; a wave owns 128 x TN / 2.
template <int TN>
__device__ __forceinline__ void tile_product(const int8_t* a, const int8_t* b, int32_t* y, int64_t m,
                                             int64_t n, int64_t k, int64_t m0, int64_t n0,
                                             lds_u8* lds) {
  constexpr int kWaveN = TN / 2, kBlocksN = kWaveN / 32;
  constexpr int kStageBytes = stage_bytes(TN);
  constexpr int kFrags = kBlocksM + kBlocksN, kMfmas = kBlocksM * kBlocksN;
  constexpr int kSegs = StageLoader<TN>::kSegs;
  static_assert(kWaveN % 32 == 0 && TN % 64 == 0, "tile width");
  // half A puts the direct loads behind the first MFMAs and the fragment
  // reads, kPer at a time, behind the rest
  static_assert(kSegs < kMfmas && kFrags <= kMfmas, "schedule");
  constexpr int kPer = (kFrags + kMfmas - kSegs - 1) / (kMfmas - kSegs);
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wm = wave >> 1, wn = wave & 1;   // wave's 128 x TN / 2 block of the tile
  const int64_t steps = (k + kTileK - 1) / kTileK;

  v16i acc[kBlocksM][kBlocksN];
#pragma unroll
  for (int i = 0; i < kBlocksM; i++)
#pragma unroll
    for (int j = 0; j < kBlocksN; j++) acc[i][j] = v16i{};

  const __amdgpu_buffer_rsrc_t ra =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(a), (short)0, (int)(m * k), 0x00020000);
  const __amdgpu_buffer_rsrc_t rb =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(b), (short)0, (int)(n * k), 0x00020000);
  StageLoader<TN> ld;
  ld.init(m, n, k, m0, n0, wave, lane);

  // fragment addresses: row (l mod 32) of each block, chunk (l / 32) of the
  // 32-byte K chunk, swizzled (row mod 16 = l mod 16 for every block)
  const uint32_t fr = lane & 31, fh = lane >> 5, fs = swz(lane & 15);
  const uint32_t fa[2] = {(kWaveM * wm + fr) * kRowBytes + 16 * (fh ^ fs),
                          (kWaveM * wm + fr) * kRowBytes + 16 * ((2 + fh) ^ fs)};
  const uint32_t fb[2] = {kABytes + (kWaveN * wn + fr) * kRowBytes + 16 * (fh ^ fs),
                          kABytes + (kWaveN * wn + fr) * kRowBytes + 16 * ((2 + fh) ^ fs)};

  v4i xa0[kBlocksM], xb0[kBlocksN], xa1[kBlocksM], xb1[kBlocksN];   // chunk-0 / chunk-1 fragments

  auto read_frags = [&](const lds_u8* buf, int kc, v4i* xa, v4i* xb) {
#pragma unroll
    for (int i = 0; i < kBlocksM; i++)
      xa[i] = *reinterpret_cast<const __attribute__((address_space(3))) v4i*>(buf + fa[kc] + 32 * kRowBytes * i);
#pragma unroll
    for (int j = 0; j < kBlocksN; j++)
      xb[j] = *reinterpret_cast<const __attribute__((address_space(3))) v4i*>(buf + fb[kc] + 32 * kRowBytes * j);
  };
  auto mfmas = [&](const v4i* xa, const v4i* xb) {
#pragma unroll
    for (int i = 0; i < kBlocksM; i++)
#pragma unroll
      for (int j = 0; j < kBlocksN; j++)
        acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(xa[i], xb[j], acc[i][j], 0, 0, 0);
  };
  // One step: `cur` holds step s, `nxt` step s + 1 (in flight), `fut` (read
  // during step s - 1, released by its barrier) receives step s + kStages - 1.
  auto step = [&](const lds_u8* cur, const lds_u8* nxt, lds_u8* fut, int64_t s) {
    ld.fetch(ra, rb, k, (s + kStages - 1) * kTileK, fut);
    read_frags(cur, 1, xa1, xb1);
    mfmas(xa0, xb0);
#pragma unroll
    for (int r = 0; r < kSegs; r++) {
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
#pragma unroll
    for (int r = 0; r < kMfmas - kSegs; r++) {
      __builtin_amdgcn_sched_group_barrier(0x100, kPer, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
    // every wave's part of step s + 1 has landed, every read of step s is done
    stage_barrier<(kStages - 2) * kSegs>();
    read_frags(nxt, 0, xa0, xb0);
    mfmas(xa1, xb1);
#pragma unroll
    for (int r = 0; r < kFrags; r++) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
  };

  lds_u8* const b0 = lds;
  lds_u8* const b1 = lds + kStageBytes;
  lds_u8* const b2 = lds + 2 * kStageBytes;
  lds_u8* const b3 = lds + 3 * kStageBytes;
  ld.fetch(ra, rb, k, 0, b0);
  ld.fetch(ra, rb, k, kTileK, b1);
  ld.fetch(ra, rb, k, 2 * kTileK, b2);
  stage_barrier<(kStages - 2) * kSegs>();
  read_frags(b0, 0, xa0, xb0);

  // Four steps per trip, the buffers rotating; steps past the end (up to
  // three in the last trip) are zero tiles and add nothing.
  static_assert(kStages == 4, "the trip below rotates four buffers");
  for (int64_t s = 0; s < steps; s += 4) {
    step(b0, b1, b3, s);
    step(b1, b2, b0, s + 1);
    step(b2, b3, b1, s + 2);
    step(b3, b0, b2, s + 3);
  }
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
        if (row < m && col < n) ((EP_GLOBAL int32_t*)y)[row * n + col] = acc[i][j][r];
      }
    }
}

// Workgroups [0, full) take whole 256 x 256 tiles; when the last round of
// whole tiles would fill at most half the CUs, its `split` tiles are instead
// taken as 2 * split half-width (256 x 128) tiles by workgroups [full, ..),
// so that round lasts about half as long.
__global__ __launch_bounds__(kGemmThreads) void gemm_i8_nt_kernel(const int8_t* __restrict__ a,
                                                                  const int8_t* __restrict__ b,
                                                                  int32_t* __restrict__ y,
                                                                  int64_t m, int64_t n, int64_t k,
                                                                  uint32_t tm, uint32_t tn,
                                                                  uint32_t full, uint32_t split) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds_mem[kStages * stage_bytes(kTileN)];
  lds_u8* const lds = (lds_u8*)lds_mem;
  const uint32_t id = blockIdx.x;
  uint32_t ti, tj;
  if (id < full) {
    tile_of(xcd_spread(id, full), tm, tn, ti, tj);
    tile_product<kTileN>(a, b, y, m, n, k, (int64_t)ti * kTileM, (int64_t)tj * kTileN, lds);
  } else {
    const uint32_t u = xcd_spread(id - full, 2 * split);
    tile_of(full + u / 2, tm, tn, ti, tj);
    tile_product<kTileN / 2>(a, b, y, m, n, k, (int64_t)ti * kTileM,
                             (int64_t)tj * kTileN + (kTileN / 2) * (u & 1), lds);
  }
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
  hipLaunchKernelGGL(ep::gemm_i8_nt_kernel, dim3((unsigned)(tiles + split)), dim3(ep::kGemmThreads), 0,
                     static_cast<hipStream_t>(hip_stream), d_a, d_b, d_y, m, n, k, (uint32_t)tm,
                     (uint32_t)tn, (uint32_t)(tiles - split), (uint32_t)split);
  if (hipGetLastError() != hipSuccess) return ep::fail(EP_ERR_HIP, "ep_gemm_i8_nt: launch failed");
  return EP_OK;
}
