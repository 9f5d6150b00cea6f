// Stand-ins for the device half of the GPU encoder, so that the library's host
// sources link without HIP in the sanitized CPU build.  Every call reports
// that the GPU encoder is unavailable; the driver never reaches them.
#include <cstdint>

#include "../../include/entropack.h"

namespace ep {
namespace genc {
struct Ctx {};
int open(Ctx**, const void*, int, int64_t, int64_t, int, void*) { return EP_ERR_UNSUPPORTED; }
void close(Ctx*) {}
int prep(Ctx*, float*, double*) { return EP_ERR_UNSUPPORTED; }
int quantize(Ctx*, const int64_t*, int64_t, double, int32_t*) { return EP_ERR_UNSUPPORTED; }
int count(Ctx*, bool, const int32_t*, const int32_t*, uint64_t*) { return EP_ERR_UNSUPPORTED; }
int refit(Ctx*, double*, double*) { return EP_ERR_UNSUPPORTED; }
int rans(Ctx*, int, uint32_t, uint64_t, const int32_t*, const int32_t*, const uint32_t*, uint32_t*,
         uint64_t*) { return EP_ERR_UNSUPPORTED; }
int payload(Ctx*, const uint32_t*, uint64_t, uint64_t, uint8_t*) { return EP_ERR_UNSUPPORTED; }
int errors(Ctx*, const float*, int, double*) { return EP_ERR_UNSUPPORTED; }
int cand_alloc(Ctx*, int) { return EP_ERR_UNSUPPORTED; }
int cand_quantize(Ctx*, int, double, int32_t*) { return EP_ERR_UNSUPPORTED; }
int cand_refit(Ctx*, int, double*, double*) { return EP_ERR_UNSUPPORTED; }
int cand_distortion(Ctx*, int, const float*, double*) { return EP_ERR_UNSUPPORTED; }
int cand_rate(Ctx*, int, const double*, const int32_t*, const int32_t*, double*) { return EP_ERR_UNSUPPORTED; }
int cand_select(Ctx*, const int32_t*, int32_t*) { return EP_ERR_UNSUPPORTED; }
int cand_count(Ctx*, int, const int32_t*, const int32_t*, uint64_t*) { return EP_ERR_UNSUPPORTED; }
}  // namespace genc
}  // namespace ep
