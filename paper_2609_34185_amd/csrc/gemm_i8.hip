// INT8 x INT8 -> INT32 matrix product on gfx950 MFMA, for decode-then-GEMM:
// Y[M x N] = A[M x K] * B[N x K]^T, both operands K-contiguous (row-major A,
// row-major B = the decoded weight matrix as stored), exact int32 accumulation.
//
// Tiling: a workgroup of 256 threads (4 waves, 2 x 2) owns a 256 x 128 tile of
// Y; each wave owns 128 x 64 = 4 x 2 blocks of v_mfma_i32_32x32x32_i8 (128
// accumulator registers), which reads 12 KiB of LDS operands per 64-byte K
// step for 16 MFMAs.  K is walked in steps of 64 bytes through double-buffered
// LDS tiles (one barrier per step).  Operands are fetched two steps ahead into
// two alternating register stages with bounded buffer loads (out-of-range
// chunks read as zero without touching memory), so a step's loads have two
// steps of MFMA work to land in.
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

constexpr int kTileM = 256, kTileN = 128, kTileK = 64;
constexpr int kWaveM = 128, kWaveN = 64;            // per wave: 4 x 2 blocks of 32 x 32
constexpr int kBlocksM = kWaveM / 32, kBlocksN = kWaveN / 32;
constexpr int kGemmThreads = 256;
constexpr int kRowBytes = kTileK + 16;              // padded LDS row: shifts banks by 4 per row
constexpr int kABytes = kTileM * kRowBytes, kBBytes = kTileN * kRowBytes;
constexpr int kStageBytes = kABytes + kBBytes;      // A tile then B tile

#define EP_GLOBAL __attribute__((address_space(1)))

constexpr uint32_t kOutside = 0x80000000u;   // operands are limited to 2^31 bytes

// Load the 16-byte chunks of one ROWS x 64 operand tile owned by this thread
// (ROWS / 64 per thread); chunks outside [0, rows) x [0, k) get an offset past
// the buffer's end and read as zero.
template <int ROWS>
__device__ __forceinline__ void fetch_tile(__amdgpu_buffer_rsrc_t rsrc, int64_t rows, int64_t k,
                                           int64_t r0, int64_t k0, int t, v4i* out) {
#pragma unroll
  for (int i = 0; i < ROWS / 64; i++) {
    const int c = t + kGemmThreads * i;   // chunk: row c / 4, 16-byte column c % 4
    const int64_t r = r0 + (c >> 2), kk = k0 + 16 * (c & 3);
    const uint32_t off = (r < rows && kk < k) ? (uint32_t)(r * k + kk) : kOutside;
    out[i] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, 0));
  }
}

template <int ROWS>
__device__ __forceinline__ void stash_tile(uint8_t* lds, int t, const v4i* in) {
#pragma unroll
  for (int i = 0; i < ROWS / 64; i++) {
    const int c = t + kGemmThreads * i;
    *reinterpret_cast<v4i*>(lds + (c >> 2) * kRowBytes + 16 * (c & 3)) = in[i];
  }
}

__global__ __launch_bounds__(kGemmThreads) void gemm_i8_nt_kernel(const int8_t* __restrict__ a,
                                                                  const int8_t* __restrict__ b,
                                                                  int32_t* __restrict__ y,
                                                                  int64_t m, int64_t n, int64_t k) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * kStageBytes];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wm = wave >> 1, wn = wave & 1;   // wave's 128 x 64 block of the tile
  const int64_t m0 = (int64_t)blockIdx.y * kTileM, n0 = (int64_t)blockIdx.x * kTileN;
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
  v4i ga0[kTileM / 64], gb0[kTileN / 64], ga1[kTileM / 64], gb1[kTileN / 64];
  fetch_tile<kTileM>(ra, m, k, m0, 0, t, ga0);
  fetch_tile<kTileN>(rb, n, k, n0, 0, t, gb0);
  fetch_tile<kTileM>(ra, m, k, m0, kTileK, t, ga1);
  fetch_tile<kTileN>(rb, n, k, n0, kTileK, t, gb1);
  stash_tile<kTileM>(lds, t, ga0);
  stash_tile<kTileN>(lds + kABytes, t, gb0);
  __syncthreads();

  const int fr = lane & 31, fk = 16 * (lane >> 5);   // fragment row and k byte offset
  auto compute = [&](const uint8_t* cur) {
#pragma unroll
    for (int kc = 0; kc < kTileK; kc += 32) {
      v4i fa[kBlocksM], fb[kBlocksN];
#pragma unroll
      for (int i = 0; i < kBlocksM; i++)
        fa[i] = *reinterpret_cast<const v4i*>(cur + (kWaveM * wm + 32 * i + fr) * kRowBytes + kc + fk);
#pragma unroll
      for (int j = 0; j < kBlocksN; j++)
        fb[j] = *reinterpret_cast<const v4i*>(cur + kABytes + (kWaveN * wn + 32 * j + fr) * kRowBytes +
                                              kc + fk);
#pragma unroll
      for (int i = 0; i < kBlocksM; i++)
#pragma unroll
        for (int j = 0; j < kBlocksN; j++)
          acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
  };
  // Steps s and s + 1 per trip: buffer 0 holds step s (stage-0 registers
  // refill with s + 2), buffer 1 step s + 1 (stage-1 registers with s + 3).
  // Steps past the end (the second half of the last trip when the step count
  // is odd) are zero tiles and add nothing.
  for (int64_t s = 0; s < steps; s += 2) {
    fetch_tile<kTileM>(ra, m, k, m0, (s + 2) * kTileK, t, ga0);
    fetch_tile<kTileN>(rb, n, k, n0, (s + 2) * kTileK, t, gb0);
    __builtin_amdgcn_sched_barrier(0);   // issue the loads before this step's MFMAs
    compute(lds);
    stash_tile<kTileM>(lds + kStageBytes, t, ga1);
    stash_tile<kTileN>(lds + kStageBytes + kABytes, t, gb1);
    __syncthreads();
    fetch_tile<kTileM>(ra, m, k, m0, (s + 3) * kTileK, t, ga1);
    fetch_tile<kTileN>(rb, n, k, n0, (s + 3) * kTileK, t, gb1);
    __builtin_amdgcn_sched_barrier(0);
    compute(lds + kStageBytes);
    stash_tile<kTileM>(lds, t, ga0);
    stash_tile<kTileN>(lds + kABytes, t, gb0);
    __syncthreads();
  }

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

}  // namespace
}  // namespace ep

extern "C" int ep_gemm_i8_nt(const int8_t* d_a, const int8_t* d_b, int32_t* d_y, int64_t m,
                             int64_t n, int64_t k, void* hip_stream) {
  if (!d_a || !d_b || !d_y) return ep::fail(EP_ERR_ARG, "ep_gemm_i8_nt: null pointer");
  if (m <= 0 || n <= 0 || k <= 0 || k % 16)
    return ep::fail(EP_ERR_ARG, "ep_gemm_i8_nt: need m, n, k > 0 and k % 16 == 0");
  if ((reinterpret_cast<uintptr_t>(d_a) | reinterpret_cast<uintptr_t>(d_b)) & 15)
    return ep::fail(EP_ERR_ARG, "ep_gemm_i8_nt: operands must be 16-byte aligned");
  if (k > (int64_t(1) << 24))
    return ep::fail(EP_ERR_ARG, "ep_gemm_i8_nt: k above 2^24 may overflow int32 sums");
  if (m * k >= (int64_t)ep::kOutside || n * k >= (int64_t)ep::kOutside)
    return ep::fail(EP_ERR_ARG, "ep_gemm_i8_nt: an operand above 2^31 bytes");
  const int64_t gx = (n + ep::kTileN - 1) / ep::kTileN, gy = (m + ep::kTileM - 1) / ep::kTileM;
  if (gx > 0x7FFFFFFF || gy > 65535) return ep::fail(EP_ERR_ARG, "ep_gemm_i8_nt: matrix too large");
  hipLaunchKernelGGL(ep::gemm_i8_nt_kernel, dim3((unsigned)gx, (unsigned)gy), dim3(ep::kGemmThreads), 0,
                     static_cast<hipStream_t>(hip_stream), d_a, d_b, d_y, m, n, k);
  if (hipGetLastError() != hipSuccess) return ep::fail(EP_ERR_HIP, "ep_gemm_i8_nt: launch failed");
  return EP_OK;
}
