// The kernels of the fused decode and MFMA product (ep_decode_gemm_i8,
// ep_decode_gemm_bf16 and their prepared forms; App. D): each workgroup
// decodes a block of rows into its slab with the decode machinery of
// decode_kernels.h, then multiplies X by the slab on the matrix cores.
#include "decode_kernels.h"
#include "decode_launch.h"

namespace ep {
namespace {

typedef int v4i_t __attribute__((ext_vector_type(4)));
typedef float v4f_t __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf_t __attribute__((ext_vector_type(8)));

// The product of one block: a work item is XT tiles of 16 rows of X against
// all NT = ceil(RB / 16) tiles of 16 block rows, so each X fragment is loaded
// once per block and each slab fragment once per item; items are dealt to the
// waves, and when there are fewer items than waves K is split over the idle
// waves and the partial sums are added with atomics (exact, order-free integer
// additions).  NT and XT are template arguments so that no load is issued for
// a tile the block does not have.  MFMA operands: lane l supplies row l mod 16
// of an X tile and of a slab tile, 16 consecutive bytes of K each
// (k = 16 (l / 16) + 0..15 of a 64-byte step); accumulator r of lane l is
// element (4 (l / 16) + r, l mod 16) of a 16 x 16 result.
//
// BF: the BF16 product (bf16 X and slab, v_mfma_f32_16x16x32_bf16, fp32 Y).
// A lane's 16 bytes of a 64-byte K step are then 8 bf16 elements, the same
// bytes as 16 int8 ones, so the addressing below is in bytes for both; the
// sums are fp32 and K slices add them with float atomics.
template <uint32_t NT, uint32_t XT, bool BF>
__device__ __forceinline__ void block_product_nt(const LayerDev& L, const GemmArgs& g,
                                                 const uint8_t* slab, uint32_t b) {
  const uint32_t wave = wave_id(), lane = threadIdx.x & 63;
  const uint32_t C = L.cols * (BF ? 2 : 1), m = g.m, RB = g.rows_per_block;   // C: row bytes
  const uint32_t T = (m + 15) / 16, I = (T + XT - 1) / XT;   // X tiles, items
  const uint32_t S = I >= kWavesPerGroup ? 1u : kWavesPerGroup / I;   // K slices
  if (I < kWavesPerGroup && wave >= I * S) return;
  const uint32_t slice = I >= kWavesPerGroup ? 0u : wave / I;
  const uint32_t it0 = I >= kWavesPerGroup ? wave : wave % I;
  const uint32_t istep = I >= kWavesPerGroup ? kWavesPerGroup : I;
  // 64-byte K steps per group: two groups' fragments stay within the
  // registers the decode leaves (2 (XT + NT) kGroup fragments of 4 VGPRs)
  constexpr uint32_t kGroup = XT + NT <= 3 ? 2 : 1;
  // slices are cut at 128-byte boundaries whatever the group
  const uint32_t groups = (C + 127) / 128, gper = (groups + S - 1) / S;
  const uint32_t k_begin = slice * gper * 128, k_end = min(C, (slice + 1) * gper * 128);
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(g.x), (short)0, (int)((uint64_t)m * C), 0x00020000);
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(slab), (short)0, (int)g.slab_bytes, 0x00020000);
  const uint32_t li = lane & 15, q = lane >> 4;
  const uint32_t row0 = b * RB;
  using Acc = typename std::conditional<BF, v4f_t, v4i_t>::type;
  using Out = typename std::conditional<BF, float, int32_t>::type;
  EP_GLOBAL Out* y = gptr<Out>(g.y);
  // one group's fragments: XT X tiles and the NT slab tiles for kGroup 64-byte K steps
  struct Frags {
    v4i_t a[kGroup][XT], w[kGroup][NT];
  };
  for (uint32_t it = it0; it < I; it += istep) {
    Acc acc[XT][NT];
#pragma unroll
    for (uint32_t x = 0; x < XT; x++)
#pragma unroll
      for (uint32_t c = 0; c < NT; c++) acc[x][c] = Acc{0, 0, 0, 0};
    // bytes at or past k_end read as zeros (bounded buffer loads), so the
    // prefetch past the slice's end and a partial last group add nothing; so
    // do the rows of X past m (a last item with fewer than XT tiles)
    auto load = [&](uint32_t k0, Frags& f) {
#pragma unroll
      for (uint32_t u = 0; u < kGroup; u++) {
        const uint32_t kq = k0 + 64 * u + 16 * q;
#pragma unroll
        for (uint32_t x = 0; x < XT; x++) {
          const uint32_t tok = 16 * (XT * it + x) + li;
          // K beyond the row (C % 64 != 0) reads as zeros of X: C is a multiple of 8
          // bytes, so a lane's 16 bytes are whole, half (the upper 8 beyond C) or none
          const bool in = kq < k_end && tok < m;
          v4i_t av = (v4i_t)__builtin_amdgcn_raw_buffer_load_b128(xr, in ? tok * C + kq : 0x80000000u, 0, 0);
          if (in && kq + 8 >= C) av[2] = av[3] = 0;
          f.a[u][x] = av;
        }
#pragma unroll
        for (uint32_t c = 0; c < NT; c++) {
          const uint32_t wrow = (g.margin + 16 * c + li) * C;   // slab offset of the lane's W' row
          f.w[u][c] = (v4i_t)__builtin_amdgcn_raw_buffer_load_b128(
              wr, kq < k_end ? wrow + kq : 0x80000000u, 0, 0);
        }
      }
    };
    auto mma = [&](const Frags& f) {
#pragma unroll
      for (uint32_t u = 0; u < kGroup; u++)
#pragma unroll
        for (uint32_t x = 0; x < XT; x++)
#pragma unroll
          for (uint32_t c = 0; c < NT; c++) {
            if constexpr (BF)
              acc[x][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  __builtin_bit_cast(v8bf_t, f.a[u][x]), __builtin_bit_cast(v8bf_t, f.w[u][c]), acc[x][c],
                  0, 0, 0);
            else
              acc[x][c] = __builtin_amdgcn_mfma_i32_16x16x64_i8(f.a[u][x], f.w[u][c], acc[x][c], 0, 0, 0);
          }
    };
    // two groups in flight: the next group's loads are issued before this
    // group's MFMAs wait for their operands
    Frags f0, f1;
    load(k_begin, f0);
    for (uint32_t k0 = k_begin; k0 < k_end; k0 += 2 * 64 * kGroup) {
      load(k0 + 64 * kGroup, f1);
      mma(f0);
      if (k0 + 64 * kGroup >= k_end) break;
      load(k0 + 2 * 64 * kGroup, f0);
      mma(f1);
    }
#pragma unroll
    for (uint32_t x = 0; x < XT; x++)
#pragma unroll
      for (uint32_t c = 0; c < NT; c++) {
        const uint32_t rl = 16 * c + li, row = row0 + rl;
#pragma unroll
        for (uint32_t r = 0; r < 4; r++) {
          const uint32_t t = 16 * (XT * it + x) + 4 * q + r;
          if (t < m && rl < RB && row < L.rows) {
            if (S > 1) {
              if constexpr (BF)
                __hip_atomic_fetch_add(y + (uint64_t)t * L.rows + row, acc[x][c][r], __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
              else
                add_i32(y + (uint64_t)t * L.rows + row, acc[x][c][r]);
            } else {
              y[(uint64_t)t * L.rows + row] = acc[x][c][r];
            }
          }
        }
      }
  }
}

// Block b's rows times X, from the slab (row i of the block at slab row
// margin + i), for NT = ceil(RB / 16) tiles of 16 block rows.  WIDE: more
// than 32 rows of X.
template <bool BF, bool WIDE>
__device__ __forceinline__ void block_product(const LayerDev& L, const GemmArgs& g,
                                              const uint8_t* slab, uint32_t b) {
  switch (uni((g.rows_per_block + 15) / 16)) {
    case 1: block_product_nt<1, gemm_x_tiles(1, WIDE), BF>(L, g, slab, b); break;
    case 2: block_product_nt<2, gemm_x_tiles(2, WIDE), BF>(L, g, slab, b); break;
    case 3: block_product_nt<3, gemm_x_tiles(3, WIDE), BF>(L, g, slab, b); break;
    default: block_product_nt<4, gemm_x_tiles(4, WIDE), BF>(L, g, slab, b); break;
  }
}

// BF: the BF16 product (the slab holds the bf16 decode of the tiles).  WIDE:
// more than 32 rows of X.
template <int PATH, bool BF, bool WIDE>
__global__ __launch_bounds__(kThreads) void decode_gemm_kernel(const GemmLaunch launch, int32_t* status) {
#if defined(__HIP_DEVICE_COMPILE__)
  (void)launch;
  const GemmLaunch& A = *(const GemmLaunch*)__builtin_amdgcn_kernarg_segment_ptr();
#else
  const GemmLaunch& A = launch;
#endif
  extern __shared__ uint32_t lds[];
  const LayerDev& L = A.L;
  const GemmArgs& g = A.g;
  if (L.tables) load_tables<PATH>(L, lds);   // prepared by ep_decode_gemm_prepare
  else build_tables<PATH>(L, lds);
  __syncthreads();
  const uint32_t ring_area = uni(ring_offset<PATH>(L));
  uint8_t* lb = reinterpret_cast<uint8_t*>(lds);
  uint8_t* slab = g.slabs + (uint64_t)blockIdx.x * g.slab_bytes;
  const uint64_t nvec = (uint64_t)L.rows * L.cvec;
  const uint32_t RB = g.rows_per_block;
  for (uint32_t b = blockIdx.x; b < g.n_blocks; b += gridDim.x) {
    // tiles touching rows [RB b, RB (b + 1)), widened to whole tasks (task
    // boundaries at multiples of kTilesPerTask tiles, so that every task but
    // the tensor's last runs the steady state): decoded into the slab, row r
    // at slab row r - RB b + margin
    const uint64_t v_first = (uint64_t)b * RB * L.cvec;
    const uint64_t v_end_b = (uint64_t)(b + 1) * RB * L.cvec;
    const uint64_t v_end = v_end_b < nvec ? v_end_b : nvec;
    Hot H = make_hot(L);
    const uint32_t t_end = (uint32_t)((v_end + L.V - 1) / L.V);
    H.tile_begin = uni((uint32_t)(v_first / L.V) / kTilesPerTask * kTilesPerTask);
    H.tile_end = uni(min(L.tile_end, (t_end + kTilesPerTask - 1) / kTilesPerTask * kTilesPerTask));
    const int64_t shift = ((int64_t)b * RB - (int64_t)g.margin) * (int64_t)L.cols * (BF ? 2 : 1);
    H.out = uni_ptr(reinterpret_cast<void*>(reinterpret_cast<intptr_t>(slab) - (intptr_t)shift));
    const uint32_t tasks = (H.tile_end - H.tile_begin + kTilesPerTask - 1) / kTilesPerTask;
    for (uint32_t task = wave_id(); task < tasks; task += kWavesPerGroup)
      dispatch_task<PATH, false>(H, lds, lb, ring_area, task, status);
    __syncthreads();   // the block's rows are in the slab
    block_product<BF, WIDE>(L, g, slab, b);
    __syncthreads();   // every wave is done with the slab
  }
}

template <bool BF, bool WIDE>
const void* gemm_fn(uint32_t path) {
  return path == kPathLut ? reinterpret_cast<const void*>(&decode_gemm_kernel<kPathLut, BF, WIDE>)
         : path == kPathWide ? reinterpret_cast<const void*>(&decode_gemm_kernel<kPathWide, BF, WIDE>)
         : path == kPathSearch ? reinterpret_cast<const void*>(&decode_gemm_kernel<kPathSearch, BF, WIDE>)
                               : reinterpret_cast<const void*>(&decode_gemm_kernel<kPathGlobal, BF, WIDE>);
}

template <bool BF, bool WIDE>
void launch_one(uint32_t path, const GemmLaunch& A, uint32_t groups, uint32_t lds, int32_t* st,
                hipStream_t s) {
  if (path == kPathLut)
    hipLaunchKernelGGL((decode_gemm_kernel<kPathLut, BF, WIDE>), dim3(groups), dim3(kThreads), lds, s, A, st);
  else if (path == kPathWide)
    hipLaunchKernelGGL((decode_gemm_kernel<kPathWide, BF, WIDE>), dim3(groups), dim3(kThreads), lds, s, A, st);
  else if (path == kPathSearch)
    hipLaunchKernelGGL((decode_gemm_kernel<kPathSearch, BF, WIDE>), dim3(groups), dim3(kThreads), lds, s, A, st);
  else
    hipLaunchKernelGGL((decode_gemm_kernel<kPathGlobal, BF, WIDE>), dim3(groups), dim3(kThreads), lds, s, A, st);
}

}  // namespace

hipError_t set_gemm_lds_limit(uint32_t path, bool bf, bool wide, size_t bytes) {
  const void* fn = bf ? (wide ? gemm_fn<true, true>(path) : gemm_fn<true, false>(path))
                      : (wide ? gemm_fn<false, true>(path) : gemm_fn<false, false>(path));
  return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

void launch_gemm(uint32_t path, bool bf, bool wide, const void* launch, uint32_t groups,
                 uint32_t lds, int32_t* status, hipStream_t s) {
  const GemmLaunch& A = *static_cast<const GemmLaunch*>(launch);
  if (bf) {
    if (wide) launch_one<true, true>(path, A, groups, lds, status, s);
    else launch_one<true, false>(path, A, groups, lds, status, s);
  } else {
    if (wide) launch_one<false, true>(path, A, groups, lds, status, s);
    else launch_one<false, false>(path, A, groups, lds, status, s);
  }
}

}  // namespace ep
