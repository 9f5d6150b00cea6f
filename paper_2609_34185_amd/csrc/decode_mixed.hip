// The decode kernels of a layer list over several decode paths: each segment
// of the list runs the code of its own layer's path (Section 3.7).  The device
// code is in decode_kernels.h.
#include "decode_kernels.h"
#include "decode_launch.h"

namespace ep {

hipError_t set_mixed_lds_limit(size_t bytes) {
  hipError_t e1 = hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_args_kernel<kPathMixed>),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  hipError_t e2 = hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_ws_kernel<kPathMixed>),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  return e1 != hipSuccess ? e1 : e2;
}

void launch_mixed_args(const void* list, int n, uint32_t total, uint32_t per, uint32_t groups,
                       uint32_t lds, int32_t* status, hipStream_t s) {
  const LayerList& L = *static_cast<const LayerList*>(list);
  hipLaunchKernelGGL(decode_args_kernel<kPathMixed>, dim3(groups), dim3(kThreads), lds, s, L, n, total, per,
                     status);
}

void launch_mixed_ws(const void* layers, int n, uint32_t total, uint32_t per, uint32_t groups,
                     uint32_t lds, int32_t* status, hipStream_t s) {
  hipLaunchKernelGGL(decode_ws_kernel<kPathMixed>, dim3(groups), dim3(kThreads), lds, s,
                     static_cast<const LayerDev*>(layers), n, total, per, status);
}

}  // namespace ep
