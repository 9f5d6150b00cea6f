// Device half of the GPU encoder (encode_gpu.hip): the bulk passes of the
// encoding pipeline on gfx950.  The search, table normalisation, refit
// division and serialisation stay on the host (encode.cpp), shared with the
// CPU encoder; every function here returns EP_OK or a negative ep_status and
// leaves a message for ep_last_error.  Host arrays are plain host memory; all
// work runs on the stream given to open() and each call returns after its
// results are on the host.
#pragma once
#include <cstdint>

namespace ep {
namespace genc {

struct Ctx;

// d_w: device input (R x C row-major, dtype EP_BF16 / EP_FP16 bits or EP_FP32).
int open(Ctx** ctx, const void* d_w, int dt, int64_t R, int64_t C, int container, void* stream);
void close(Ctx* ctx);

// Coded values, delta_r (0 for direct coding) and mu_r; EP_ERR_ARG on a
// non-finite input value.  delta and mu: R entries.
int prep(Ctx* ctx, float* delta, double* mu);

// Fields of the vectors of `rows` (ascending row indices; null = every row,
// written to the full field set, else to the sample set) at scale s, and the
// observed [min, max] of each field table: lohi[2 i], lohi[2 i + 1] for
// tables i = 1..16 (table 0 is the coset, always [0, 1]); an unobserved table
// reports min > max.
int quantize(Ctx* ctx, const int64_t* rows, int64_t nrows, double s, int32_t* lohi);

// Counts of the sample (sample = true) or full field set into n: table i
// occupies n[base_i .. base_i + A[i]) with base_0 = 0 and base_{i+1} = base_i
// + A[i]; lo[i] is table i's minimum (lo[0] = 0, A[0] = 2).
int count(Ctx* ctx, bool sample, const int32_t* lo, const int32_t* A, uint64_t* n);

// Refit sums of every row over the full field set (eq. scale_fit):
// num_r = sum x p, den_r = sum p^2, each accumulated in element order.
int refit(Ctx* ctx, double* num, double* den);

// Interleaved rANS encode of every tile of the full field set with b-bit
// frequencies f (same table layout as count): terminal states (32 per tile)
// and the number of 16-bit words of each tile.
int rans(Ctx* ctx, int b, uint32_t V, uint64_t tiles, const int32_t* lo, const int32_t* A,
         const uint32_t* f, uint32_t* states, uint64_t* words);

// The tiles' words (forward order) copied to dst (host) at offs[t] words.
int payload(Ctx* ctx, const uint32_t* offs, uint64_t tiles, uint64_t total_words, uint8_t* dst);

// Per row r: acc[4r..4r+3] = squared error and squared norm against the coded
// values, then against the input (decoded weights snapped to rdt).
int errors(Ctx* ctx, const float* sigma, int rdt, double* acc);

// Per-row refinement (Section 3.5, App. C.2): K candidate field sets of the
// whole tensor held on the device.
int cand_alloc(Ctx* ctx, int K);
// Candidate k <- every row's fields at scale s; extents as quantize().
int cand_quantize(Ctx* ctx, int k, double s, int32_t* lohi);
// Refit sums of candidate k (as refit()).
int cand_refit(Ctx* ctx, int k, double* num, double* den);
// D_r = sum_j (x_rj - sigma_r p_rj)^2 of candidate k in element order (sigma: R FP32).
int cand_distortion(Ctx* ctx, int k, const float* sigma, double* D);
// R_r of candidate k: the sum, in symbol order (per vector: coset, fields 1..8),
// of lq at each symbol's cell (table layout lo, A as count()).
int cand_rate(Ctx* ctx, int k, const double* lq, const int32_t* lo, const int32_t* A, double* Rt);
// The full field set <- row r of candidate sel[r]; extents of the result.
int cand_select(Ctx* ctx, const int32_t* sel, int32_t* lohi);
// Counts of candidate k, or of the full field set for k < 0 (as count()).
int cand_count(Ctx* ctx, int k, const int32_t* lo, const int32_t* A, uint64_t* n);

}  // namespace genc
}  // namespace ep
