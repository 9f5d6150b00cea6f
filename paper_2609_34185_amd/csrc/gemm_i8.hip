// INT8 x INT8 -> INT32 matrix product on gfx950 MFMA, for decode-then-GEMM:
// Y[M x N] = A[M x K] * B[N x K]^T, both operands K-contiguous (row-major A,
// row-major B = the decoded weight matrix as stored), exact int32 accumulation.
//
// Tiling: a workgroup of 256 threads (4 waves, 2 x 2) owns a 128 x 128 tile of
// Y; each wave owns 64 x 64 = 2 x 2 blocks of v_mfma_i32_32x32x32_i8.  K is
// walked in steps of 64 bytes through double-buffered LDS tiles (one barrier
// per step); the next step's operands are fetched into registers while the
// current step's MFMAs run.
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

constexpr int kTileM = 128, kTileN = 128, kTileK = 64;
constexpr int kGemmThreads = 256;
constexpr int kRowBytes = kTileK + 16;             // padded LDS row: shifts banks by 4 per row
constexpr int kOperandBytes = kTileM * kRowBytes;  // one operand tile in LDS
constexpr int kStageBytes = 2 * kOperandBytes;     // A tile then B tile

#define EP_GLOBAL __attribute__((address_space(1)))

// Load the 16-byte chunks of one 128 x 64 operand tile owned by this thread
// (two per thread), zero outside [0, rows) x [0, k).
__device__ __forceinline__ void fetch_tile(const int8_t* base, int64_t rows, int64_t k, int64_t r0,
                                           int64_t k0, int t, v4i* out) {
#pragma unroll
  for (int i = 0; i < 2; i++) {
    const int c = t + kGemmThreads * i;   // chunk: row c / 4, 16-byte column c % 4
    const int64_t r = r0 + (c >> 2), kk = k0 + 16 * (c & 3);
    if (r < rows && kk < k)
      out[i] = *reinterpret_cast<const EP_GLOBAL v4i*>((const EP_GLOBAL int8_t*)base + r * k + kk);
    else
      out[i] = v4i{0, 0, 0, 0};
  }
}

__device__ __forceinline__ void stash_tile(uint8_t* lds, int t, const v4i* in) {
#pragma unroll
  for (int i = 0; i < 2; i++) {
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
  const int wm = wave >> 1, wn = wave & 1;   // wave's 64 x 64 quadrant
  const int64_t m0 = (int64_t)blockIdx.y * kTileM, n0 = (int64_t)blockIdx.x * kTileN;
  const int64_t steps = (k + kTileK - 1) / kTileK;

  v16i acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; i++)
#pragma unroll
    for (int j = 0; j < 2; j++) acc[i][j] = v16i{};

  v4i ga[2], gb[2];
  fetch_tile(a, m, k, m0, 0, t, ga);
  fetch_tile(b, n, k, n0, 0, t, gb);
  stash_tile(lds, t, ga);
  stash_tile(lds + kOperandBytes, t, gb);
  __syncthreads();

  const int fr = lane & 31, fk = 16 * (lane >> 5);   // fragment row and k byte offset
  for (int64_t s = 0; s < steps; s++) {
    uint8_t* cur = lds + (s & 1) * kStageBytes;
    const bool more = s + 1 < steps;
    if (more) {
      fetch_tile(a, m, k, m0, (s + 1) * kTileK, t, ga);
      fetch_tile(b, n, k, n0, (s + 1) * kTileK, t, gb);
    }
#pragma unroll
    for (int kc = 0; kc < kTileK; kc += 32) {
      v4i fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; i++)
        fa[i] = *reinterpret_cast<const v4i*>(cur + (64 * wm + 32 * i + fr) * kRowBytes + kc + fk);
#pragma unroll
      for (int j = 0; j < 2; j++)
        fb[j] = *reinterpret_cast<const v4i*>(cur + kOperandBytes +
                                              (64 * wn + 32 * j + fr) * kRowBytes + kc + fk);
#pragma unroll
      for (int i = 0; i < 2; i++)
#pragma unroll
        for (int j = 0; j < 2; j++)
          acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      uint8_t* nxt = lds + ((s + 1) & 1) * kStageBytes;
      stash_tile(nxt, t, ga);
      stash_tile(nxt + kOperandBytes, t, gb);
    }
    __syncthreads();
  }

  const int half = lane >> 5;
#pragma unroll
  for (int i = 0; i < 2; i++)
#pragma unroll
    for (int j = 0; j < 2; j++) {
      const int64_t col = n0 + 64 * wn + 32 * j + fr;
#pragma unroll
      for (int r = 0; r < 16; r++) {
        const int64_t row = m0 + 64 * wm + 32 * i + 8 * (r >> 2) + 4 * half + (r & 3);
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
  const int64_t gx = (n + ep::kTileN - 1) / ep::kTileN, gy = (m + ep::kTileM - 1) / ep::kTileM;
  if (gx > 0x7FFFFFFF || gy > 65535) return ep::fail(EP_ERR_ARG, "ep_gemm_i8_nt: matrix too large");
  hipLaunchKernelGGL(ep::gemm_i8_nt_kernel, dim3((unsigned)gx, (unsigned)gy), dim3(ep::kGemmThreads), 0,
                     static_cast<hipStream_t>(hip_stream), d_a, d_b, d_y, m, n, k);
  if (hipGetLastError() != hipSuccess) return ep::fail(EP_ERR_HIP, "ep_gemm_i8_nt: launch failed");
  return EP_OK;
}
