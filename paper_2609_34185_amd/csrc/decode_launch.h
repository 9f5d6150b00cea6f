// Launches of the decode kernels that are compiled in their own source files
// (decode_args.hip, decode_mixed.hip, decode_gemm.hip), so that the four
// decode sources build concurrently.  Plain types only: each source holds its own copy of the
// device code and descriptor types (decode_kernels.h).
#pragma once
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace ep {

// decode_args.hip: a descriptor list passed by value (`list` points to a
// LayerList on the host), one decode path (`path`: the slot-table, wide,
// search or global-table path).
hipError_t set_args_lds_limit(uint32_t path, size_t bytes);
void launch_args(uint32_t path, const void* list, int n, uint32_t total, uint32_t per,
                 uint32_t groups, uint32_t lds, int32_t* status, hipStream_t s);

// decode_mixed.hip: a list whose layers take several decode paths, by value
// (`list`, a LayerList on the host) or in device memory (`layers`, LayerDev[n]).
hipError_t set_mixed_lds_limit(size_t bytes);
void launch_mixed_args(const void* list, int n, uint32_t total, uint32_t per, uint32_t groups,
                       uint32_t lds, int32_t* status, hipStream_t s);
void launch_mixed_ws(const void* layers, int n, uint32_t total, uint32_t per, uint32_t groups,
                     uint32_t lds, int32_t* status, hipStream_t s);

// decode_gemm.hip: the fused decode and MFMA product of one tensor (`launch`
// points to a GemmLaunch on the host), one decode path; `bf`: bf16 operands
// and fp32 Y, else int8 and int32; `wide`: more than 32 rows of X.
hipError_t set_gemm_lds_limit(uint32_t path, bool bf, bool wide, size_t bytes);
void launch_gemm(uint32_t path, bool bf, bool wide, const void* launch, uint32_t groups,
                 uint32_t lds, int32_t* status, hipStream_t s);

}  // namespace ep
