// The kernels of the fused decode and MFMA product (ep_decode_gemm_i8,
// ep_decode_gemm_bf16 and their prepared forms; App. D): each workgroup
// decodes a block of rows into its slab and multiplies X by it.  The device
// code is in decode_kernels.h.
#include "decode_kernels.h"
#include "decode_launch.h"

namespace ep {
namespace {

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
