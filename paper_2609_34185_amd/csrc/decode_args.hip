// The decode kernels of a by-value descriptor list (up to eight layers of one
// decode path), for ep_decode_tiles and short ep_decode_layers lists
// (Section 3.7).  The device code is in decode_kernels.h.
#include "decode_kernels.h"
#include "decode_launch.h"

namespace ep {

hipError_t set_args_lds_limit(uint32_t path, size_t bytes) {
  const void* fn = path == kPathLut ? reinterpret_cast<const void*>(&decode_args_kernel<kPathLut>)
                   : path == kPathWide ? reinterpret_cast<const void*>(&decode_args_kernel<kPathWide>)
                   : path == kPathSearch ? reinterpret_cast<const void*>(&decode_args_kernel<kPathSearch>)
                                         : reinterpret_cast<const void*>(&decode_args_kernel<kPathGlobal>);
  return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

void launch_args(uint32_t path, const void* list, int n, uint32_t total, uint32_t per,
                 uint32_t groups, uint32_t lds, int32_t* status, hipStream_t s) {
  const LayerList& L = *static_cast<const LayerList*>(list);
  if (path == kPathLut)
    hipLaunchKernelGGL(decode_args_kernel<kPathLut>, dim3(groups), dim3(kThreads), lds, s, L, n, total, per, status);
  else if (path == kPathWide)
    hipLaunchKernelGGL(decode_args_kernel<kPathWide>, dim3(groups), dim3(kThreads), lds, s, L, n, total, per, status);
  else if (path == kPathSearch)
    hipLaunchKernelGGL(decode_args_kernel<kPathSearch>, dim3(groups), dim3(kThreads), lds, s, L, n, total, per, status);
  else
    hipLaunchKernelGGL(decode_args_kernel<kPathGlobal>, dim3(groups), dim3(kThreads), lds, s, L, n, total, per, status);
}

}  // namespace ep
