// INT8 matrix product on MFMA for decode-then-GEMM (placeholder until the tiled kernel lands).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/entropack.h"
#include "common.h"

extern "C" int ep_gemm_i8_nt(const int8_t* d_a, const int8_t* d_b, int32_t* d_y, int64_t m,
                             int64_t n, int64_t k, void* hip_stream) {
  (void)d_a, (void)d_b, (void)d_y, (void)m, (void)n, (void)k, (void)hip_stream;
  return ep::fail(EP_ERR_UNSUPPORTED, "ep_gemm_i8_nt: not built yet");
}
