// GPU encoder passes on gfx950 (declared in encode_gpu.h).
//
// The bulk of encoding runs here: input conversion and the container route
// (App. A.6, B.1), the row RMS (Section 3.2), nearest-E8 quantisation and the
// field map of every vector at a trial or final scale (Section 3.2, eqs. d8,
// parity), per-table extents and counts (Section 3.3), the refit sums
// (eq. scale_fit), the 32-state interleaved rANS encode of every tile (eq.
// rans_encode, App. C.3) and the per-row error sums of the statistics.  The
// per-value arithmetic is the CPU encoder's own (encode_math.h) compiled for
// the device, and every sum that reaches the blob is accumulated in the CPU
// encoder's element order, so the blob is byte-identical to the CPU encoder's.
//
// Mapping: element-wise passes take one thread per vector (or a workgroup
// per row for the conversion and the error sums); passes whose double sums
// decide the blob (row RMS, refit) take one thread per row, summing in
// element order out of coalesced LDS-staged chunks; counts go through a
// workgroup histogram in LDS when all tables fit (else straight to memory);
// the rANS encode runs two tiles per wave, one per half, each lane one state,
// words placed by a 32-lane ballot in the order the decoder consumes them.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <thread>
#include <vector>

#include <sys/mman.h>

#include "../../include/entropack.h"
#include "common.h"
#include "encode_gpu.h"
#include "encode_math.h"

namespace ep {
namespace genc {
namespace {

constexpr int kTablesN = 17;
constexpr uint32_t kLanesN = 32;
constexpr uint32_t kLdsBins = 36864;   // histogram in LDS when all tables fit (144 KiB)
constexpr uint32_t kMaxCells = 2 + 16 * 32768;   // counted tables have A <= 2^15

__device__ __forceinline__ float load_input(const void* w, int dt, int64_t i) {
  if (dt == EP_FP32) return static_cast<const float*>(w)[i];
  const uint16_t h = static_cast<const uint16_t*>(w)[i];
  if (dt == EP_FP16) return (float)__builtin_bit_cast(_Float16, h);
  return __builtin_bit_cast(float, (uint32_t)h << 16);
}

// One workgroup per row: input -> coded values (container route), delta_r.
// The unsigned container scales the whole tensor at once: its first pass
// (tmax < 0) only writes each row's amax into delta, the second quantises
// with tmax, the largest of them.
__global__ __launch_bounds__(256) void k_prep_rows(const void* w, int dt, int64_t C, int cont,
                                                   double tmax, float* x, float* delta, int* bad) {
  __shared__ double s_amax[256];
  __shared__ int s_bad;
  const int64_t r = blockIdx.x, base = r * C;
  const int t = threadIdx.x;
  if (t == 0) s_bad = 0;
  __syncthreads();
  double amax = 0;
  int nb = 0;
  for (int64_t j = t; j < C; j += 256) {
    const float v = load_input(w, dt, base + j);
    if (!__builtin_isfinite(v)) nb = 1;
    const double a = __builtin_fabs((double)v);
    if (a > amax) amax = a;
    if (!cont) x[base + j] = v;
  }
  if (nb) s_bad = 1;
  s_amax[t] = amax;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (t < h && s_amax[t + h] > s_amax[t]) s_amax[t] = s_amax[t + h];
    __syncthreads();
  }
  if (t == 0 && s_bad) atomicOr(bad, 1);
  if (!cont) return;
  amax = s_amax[0];
  if (cont == EP_CONT_UINT8_TENSOR) {
    if (tmax < 0) {
      if (t == 0) delta[r] = (float)amax;   // exact: amax is an FP32 value
      return;
    }
    amax = tmax;
  }
  const float d = amax > 0 ? (float)(amax / em::container_max(cont)) : 1.0f;
  if (t == 0) delta[r] = d;
  for (int64_t j = t; j < C; j += 256) {
    const double q = (double)load_input(w, dt, base + j) / (double)d;
    x[base + j] = (float)em::container_snap(cont, q);
  }
}

constexpr int kRowsPerBlock = 64;   // row-ordered sums: one thread per row, 64 rows per workgroup
constexpr int kFetchThreads = 256;  // threads of a workgroup of k_prep_mu and k_refit (rows' threads first)

// mu_r = max(sqrt(sum x^2 / C), eta), summed in element order by the row's
// thread (the first wave); the four waves of the workgroup stage 64 x 64
// chunks of its rows through LDS with 16-byte loads, the next chunk's loads in
// flight while the rows' threads sum the current one.
__global__ __launch_bounds__(kFetchThreads) void k_prep_mu(const float* x, int64_t R, int64_t C, double* mu) {
  __shared__ float tile[kRowsPerBlock][65];
  const int t = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.x * kRowsPerBlock;
  const int nr = (int)(R - r0 < kRowsPerBlock ? R - r0 : kRowsPerBlock);
  // a chunk is 64 rows x 16 groups of 4 values; this thread moves groups t + 256 k
  float4 v[4];
  auto fetch = [&](int64_t j0) {
#pragma unroll
    for (int k = 0; k < 4; k++) {
      const int i = t + kFetchThreads * k, row = i >> 4, g = i & 15;
      const bool in = row < nr && j0 + 4 * g < C;   // C % 8 == 0: groups are whole
      v[k] = in ? *reinterpret_cast<const float4*>(x + (r0 + row) * C + j0 + 4 * g)
                : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  double ss = 0;
  fetch(0);
  for (int64_t j0 = 0; j0 < C; j0 += 64) {
    const int ne = (int)(C - j0 < 64 ? C - j0 : 64);
#pragma unroll
    for (int k = 0; k < 4; k++) {
      const int i = t + kFetchThreads * k, row = i >> 4, g = i & 15;
      tile[row][4 * g] = v[k].x;
      tile[row][4 * g + 1] = v[k].y;
      tile[row][4 * g + 2] = v[k].z;
      tile[row][4 * g + 3] = v[k].w;
    }
    __syncthreads();
    if (j0 + 64 < C) fetch(j0 + 64);
    if (t < nr)
      for (int e = 0; e < ne; e++) ss += (double)tile[t][e] * (double)tile[t][e];
    __syncthreads();
  }
  if (t < nr) {
    const double m = __builtin_sqrt(ss / (double)C);
    mu[r0 + t] = m > em::kEta ? m : em::kEta;
  }
}

// One thread per vector: fields at scale s, table extents.
__global__ __launch_bounds__(256) void k_quantize(const float* x, const double* mu,
                                                  const int64_t* rows, int64_t nrows, int64_t cvec,
                                                  int64_t C, double s, int32_t* fl, int32_t* lohi) {
  __shared__ int32_t s_lo[16], s_hi[16];
  const int t = threadIdx.x;
  if (t < 16) {
    s_lo[t] = INT_MAX;
    s_hi[t] = INT_MIN;
  }
  __syncthreads();
  const int64_t id = (int64_t)blockIdx.x * 256 + t;
  if (id < nrows * cvec) {
    const int64_t k = id / cvec, jv = id - k * cvec;
    const int64_t r = rows ? rows[k] : k;
    const float4* xv = reinterpret_cast<const float4*>(x + r * C + 8 * jv);
    const float4 a = xv[0], b = xv[1];
    const float xs[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    const double m = mu[r];
    double y[8];
    for (int j = 0; j < 8; j++) y[j] = ((double)xs[j] / m) / s;
    int32_t p2[8], f[9];
    em::e8_point(y, p2);
    em::split_fields(p2, f);
    int32_t* o = fl + 9 * id;
    for (int i = 0; i < 9; i++) o[i] = f[i];
    for (int i = 1; i <= 8; i++) {
      const int ti = em::table_index(i, f[0]) - 1;
      atomicMin(&s_lo[ti], f[i]);
      atomicMax(&s_hi[ti], f[i]);
    }
  }
  __syncthreads();
  if (t < 16 && s_lo[t] <= s_hi[t]) {
    atomicMin(&lohi[2 * (t + 1)], s_lo[t]);
    atomicMax(&lohi[2 * (t + 1) + 1], s_hi[t]);
  }
}

struct TableDesc {
  int32_t lo[kTablesN];
  uint32_t base[kTablesN];
};

__device__ __forceinline__ uint32_t bin_of(const TableDesc& td, const int32_t* q, int i) {
  if (i == 0) return (uint32_t)q[0];
  const int ti = em::table_index(i, q[0]);
  return td.base[ti] + (uint32_t)(q[i] - td.lo[ti]);
}

// Counts with a workgroup histogram in LDS (cells <= kLdsBins).
__global__ __launch_bounds__(256) void k_count_lds(const int32_t* fl, int64_t nv, TableDesc td,
                                                   uint32_t cells, uint32_t* counts) {
  extern __shared__ uint32_t h[];
  for (uint32_t i = threadIdx.x; i < cells; i += 256) h[i] = 0;
  __syncthreads();
  for (int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x; id < nv; id += (int64_t)gridDim.x * 256) {
    const int32_t* q = fl + 9 * id;
    for (int i = 0; i < 9; i++) atomicAdd(&h[bin_of(td, q, i)], 1u);
  }
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < cells; i += 256)
    if (h[i]) atomicAdd(&counts[i], h[i]);
}

// Counts straight into memory (tables too wide for LDS).
__global__ __launch_bounds__(256) void k_count_mem(const int32_t* fl, int64_t nv, TableDesc td,
                                                   uint32_t* counts) {
  for (int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x; id < nv; id += (int64_t)gridDim.x * 256) {
    const int32_t* q = fl + 9 * id;
    for (int i = 0; i < 9; i++) atomicAdd(&counts[bin_of(td, q, i)], 1u);
  }
}

// Refit sums in element order by the row's thread (the first wave), 8 vectors
// (64 values and 72 fields) of each of the workgroup's 64 rows staged through
// LDS at a time by its four waves: values in 16-byte groups, fields one by
// one; the next chunk's loads are in flight while the rows' threads sum the
// current one.
__global__ __launch_bounds__(kFetchThreads) void k_refit(const float* x, const int32_t* fl, int64_t R,
                                                         int64_t cvec, double* num, double* den) {
  __shared__ float tx[kRowsPerBlock][65];
  __shared__ int32_t tf[kRowsPerBlock][73];   // 72 fields used
  const int t = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.x * kRowsPerBlock, C = cvec * 8;
  const int nr = (int)(R - r0 < kRowsPerBlock ? R - r0 : kRowsPerBlock);
  // values: 64 rows x 16 groups of 4, groups t + 256 k; fields: 64 rows x 72,
  // fields t + 256 k
  constexpr int kF = kRowsPerBlock * 72 / kFetchThreads;   // 18
  float4 xv[4];
  int32_t fv[kF];
  auto fetch = [&](int64_t v0) {
    const int nvv = (int)(cvec - v0 < 8 ? cvec - v0 : 8);
#pragma unroll
    for (int k = 0; k < 4; k++) {
      const int i = t + kFetchThreads * k, row = i >> 4, g = i & 15;
      const bool in = row < nr && 4 * g < 8 * nvv;
      xv[k] = in ? *reinterpret_cast<const float4*>(x + (r0 + row) * C + 8 * v0 + 4 * g)
                 : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int k = 0; k < kF; k++) {
      const int i = t + kFetchThreads * k, row = i / 72, c = i % 72;
      fv[k] = (row < nr && c < 9 * nvv) ? fl[9 * ((r0 + row) * cvec + v0) + c] : 0;
    }
  };
  double sn = 0, sd = 0;
  fetch(0);
  for (int64_t v0 = 0; v0 < cvec; v0 += 8) {
    const int nvv = (int)(cvec - v0 < 8 ? cvec - v0 : 8);
#pragma unroll
    for (int k = 0; k < 4; k++) {
      const int i = t + kFetchThreads * k, row = i >> 4, g = i & 15;
      tx[row][4 * g] = xv[k].x;
      tx[row][4 * g + 1] = xv[k].y;
      tx[row][4 * g + 2] = xv[k].z;
      tx[row][4 * g + 3] = xv[k].w;
    }
#pragma unroll
    for (int k = 0; k < kF; k++) {
      const int i = t + kFetchThreads * k;
      tf[i / 72][i % 72] = fv[k];
    }
    __syncthreads();
    if (v0 + 8 < cvec) fetch(v0 + 8);
    if (t < nr)
      for (int v = 0; v < nvv; v++) {
        int32_t p2[8];
        em::join_fields(&tf[t][9 * v], p2);
        for (int j = 0; j < 8; j++) {
          const double pj = p2[j] / 2.0;
          sn += (double)tx[t][8 * v + j] * pj;
          sd += pj * pj;
        }
      }
    __syncthreads();
  }
  if (t < nr) {
    num[r0 + t] = sn;
    den[r0 + t] = sd;
  }
}

// Two tiles per wave (one per half), lane = state.  Steps run backwards
// (last vector's last field first); within a step the words pushed by the
// renormalising lanes go, in descending lane order, to the end of the tile's
// scratch row moving towards its start, so the row ends with the tile's
// stream in the decoder's (step ascending, lane ascending) order.
__global__ __launch_bounds__(64) void k_rans(const int32_t* fl, uint64_t nvec, uint32_t V,
                                             uint32_t rounds_max, uint64_t tiles, TableDesc td,
                                             const uint2* tab, int b, uint32_t* states,
                                             uint32_t* cnt, uint16_t* scratch, uint32_t cap) {
  const uint32_t lane = threadIdx.x, half = lane >> 5, l = lane & 31;
  const uint64_t t = 2ull * blockIdx.x + half;
  const bool tile_ok = t < tiles;
  const uint64_t v0 = t * V;
  const uint64_t nv = tile_ok ? (nvec - v0 < V ? nvec - v0 : V) : 0;
  const uint32_t M = 1u << b;
  uint16_t* out = scratch + t * cap + cap - 1;
  uint32_t st = 1u << 15, pos = 0;
  for (uint32_t step = 9 * rounds_max; step-- > 0;) {
    const uint32_t k = step / 9, fi = step - 9 * k;
    const uint64_t li = l + kLanesN * (uint64_t)k;
    const bool active = li < nv;
    uint32_t f = 1, F = 0;
    if (active) {
      const int32_t* q = fl + 9 * (v0 + li);
      const uint2 e = tab[bin_of(td, q, (int)fi)];
      f = e.x;
      F = e.y;
    }
    uint32_t xs = st;
    const bool push = active && (uint64_t)xs >= ((uint64_t)f << (31 - b));
    const uint64_t mask = __ballot(push);
    const uint32_t m = (uint32_t)(mask >> (32 * half));
    if (push) {
      const uint32_t idx = pos + (uint32_t)__popcll((uint64_t)m >> (l + 1));
      out[-(int64_t)idx] = (uint16_t)(xs & 0xFFFF);
      xs >>= 16;
    }
    pos += (uint32_t)__popc(m);
    if (active) st = (xs / f) * M + xs % f + F;
  }
  if (tile_ok) {
    states[t * kLanesN + l] = st;
    if (l == 0) cnt[t] = pos;
  }
}

// One workgroup per tile: the tile's words from the end of its scratch row to
// the payload at its offset.
__global__ __launch_bounds__(256) void k_gather(const uint16_t* scratch, uint32_t cap,
                                                const uint32_t* cnt, const uint32_t* offs,
                                                uint16_t* payload) {
  const uint64_t t = blockIdx.x;
  const uint32_t n = cnt[t];
  const uint16_t* src = scratch + t * cap + cap - n;
  uint16_t* dst = payload + offs[t];
  for (uint32_t i = threadIdx.x; i < n; i += 256) dst[i] = src[i];
}

// One workgroup per row: error sums, each thread over a strided subset of the
// row's vectors, combined by a fixed tree (deterministic, but not the CPU
// encoder's element order: these statistics agree with its to rounding).
__global__ __launch_bounds__(256) void k_errors(const void* w, int dt, const float* x,
                                                const int32_t* fl, const float* sigma,
                                                const float* delta, int rdt, int cont, int64_t cvec,
                                                double* acc) {
  __shared__ double red[4][256];
  const int64_t r = blockIdx.x, C = cvec * 8;
  const int t = threadIdx.x;
  double ec = 0, rc = 0, eo = 0, ro = 0;
  for (int64_t jv = t; jv < cvec; jv += 256) {
    int32_t two[8];
    em::join_fields(fl + 9 * (r * cvec + jv), two);
    for (int j = 0; j < 8; j++) {
      const double y = (double)(float)((double)sigma[r] * (two[j] / 2.0));
      const double v = em::snap_out(rdt, y);
      const double xc = x[r * C + 8 * jv + j];
      const double off = em::container_offset(cont);
      ec += (v - xc) * (v - xc);
      rc += (xc - off) * (xc - off);
      const double wo = (double)load_input(w, dt, r * C + 8 * jv + j);
      const double vo = cont ? (v - off) * (double)delta[r] : v;
      eo += (vo - wo) * (vo - wo);
      ro += wo * wo;
    }
  }
  red[0][t] = ec;
  red[1][t] = rc;
  red[2][t] = eo;
  red[3][t] = ro;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (t < h)
      for (int q = 0; q < 4; q++) red[q][t] += red[q][t + h];
    __syncthreads();
  }
  if (t < 4) acc[4 * r + t] = red[t][0];
}

// Per-row refinement, candidate k: D_r = sum_j (x_rj - sigma_r p_rj)^2 in
// element order (one thread per row, which also loads the 64 x 8-vector chunks
// that the workgroup stages through LDS).
__global__ __launch_bounds__(64) void k_dist(const float* x, const int32_t* fl, const float* sigma,
                                             int64_t R, int64_t cvec, double* D) {
  __shared__ float tx[kRowsPerBlock][65];
  __shared__ int32_t tf[kRowsPerBlock][73];
  const int t = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.x * kRowsPerBlock, C = cvec * 8;
  const int nr = (int)(R - r0 < kRowsPerBlock ? R - r0 : kRowsPerBlock);
  const double sg = t < nr ? (double)sigma[r0 + t] : 0.0;
  double d = 0;
  for (int64_t v0 = 0; v0 < cvec; v0 += 8) {
    const int nvv = (int)(cvec - v0 < 8 ? cvec - v0 : 8);
    float xv[kRowsPerBlock];
    int32_t f0[kRowsPerBlock], f1[kRowsPerBlock];
#pragma unroll
    for (int i = 0; i < kRowsPerBlock; i++) {
      const bool row = i < nr;
      const int64_t fb = 9 * ((r0 + i) * cvec + v0);
      xv[i] = (row && t < 8 * nvv) ? x[(r0 + i) * C + 8 * v0 + t] : 0.0f;
      f0[i] = (row && t < 9 * nvv) ? fl[fb + t] : 0;
      f1[i] = (row && t + 64 < 9 * nvv) ? fl[fb + t + 64] : 0;
    }
#pragma unroll
    for (int i = 0; i < kRowsPerBlock; i++) {
      tx[i][t] = xv[i];
      tf[i][t] = f0[i];
      if (t < 9) tf[i][t + 64] = f1[i];
    }
    __syncthreads();
    if (t < nr)
      for (int v = 0; v < nvv; v++) {
        int32_t p2[8];
        em::join_fields(&tf[t][9 * v], p2);
        for (int j = 0; j < 8; j++) {
          const double e = (double)tx[t][8 * v + j] - sg * (p2[j] / 2.0);
          d += e * e;
        }
      }
    __syncthreads();
  }
  if (t < nr) D[r0 + t] = d;
}

// Per-row refinement, candidate k: R_r = sum over the row's symbols (coset,
// then fields 1..8 of each vector, vectors in order) of lq[base_t + v - lo_t].
__global__ __launch_bounds__(64) void k_rate(const int32_t* fl, const double* lq, TableDesc td,
                                             int64_t R, int64_t cvec, double* Rt) {
  __shared__ int32_t tf[kRowsPerBlock][73];
  const int t = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.x * kRowsPerBlock;
  const int nr = (int)(R - r0 < kRowsPerBlock ? R - r0 : kRowsPerBlock);
  double acc = 0;
  for (int64_t v0 = 0; v0 < cvec; v0 += 8) {
    const int nvv = (int)(cvec - v0 < 8 ? cvec - v0 : 8);
    int32_t f0[kRowsPerBlock], f1[kRowsPerBlock];
#pragma unroll
    for (int i = 0; i < kRowsPerBlock; i++) {
      const bool row = i < nr;
      const int64_t fb = 9 * ((r0 + i) * cvec + v0);
      f0[i] = (row && t < 9 * nvv) ? fl[fb + t] : 0;
      f1[i] = (row && t + 64 < 9 * nvv) ? fl[fb + t + 64] : 0;
    }
#pragma unroll
    for (int i = 0; i < kRowsPerBlock; i++) {
      tf[i][t] = f0[i];
      if (t < 9) tf[i][t + 64] = f1[i];
    }
    __syncthreads();
    if (t < nr)
      for (int v = 0; v < nvv; v++) {
        const int32_t* q = &tf[t][9 * v];
        acc += lq[bin_of(td, q, 0)];
        for (int i = 1; i <= 8; i++) acc += lq[bin_of(td, q, i)];
      }
    __syncthreads();
  }
  if (t < nr) Rt[r0 + t] = acc;
}

// The full field set <- row r of candidate sel[r], with the result's table extents.
__global__ __launch_bounds__(256) void k_select(const int32_t* cand, uint64_t cand_stride,
                                                const int32_t* sel, int64_t nvec, int64_t cvec,
                                                int32_t* fl, int32_t* lohi) {
  __shared__ int32_t s_lo[16], s_hi[16];
  const int t = threadIdx.x;
  if (t < 16) {
    s_lo[t] = INT_MAX;
    s_hi[t] = INT_MIN;
  }
  __syncthreads();
  const int64_t id = (int64_t)blockIdx.x * 256 + t;
  if (id < nvec) {
    const int32_t* q = cand + (uint64_t)sel[id / cvec] * cand_stride + 9 * id;
    int32_t f[9];
    for (int i = 0; i < 9; i++) f[i] = q[i];
    for (int i = 0; i < 9; i++) fl[9 * id + i] = f[i];
    for (int i = 1; i <= 8; i++) {
      const int ti = em::table_index(i, f[0]) - 1;
      atomicMin(&s_lo[ti], f[i]);
      atomicMax(&s_hi[ti], f[i]);
    }
  }
  __syncthreads();
  if (t < 16 && s_lo[t] <= s_hi[t]) {
    atomicMin(&lohi[2 * (t + 1)], s_lo[t]);
    atomicMax(&lohi[2 * (t + 1) + 1], s_hi[t]);
  }
}

unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

// Two pinned host buffers through which large device-to-host copies are
// staged: a copy into pageable memory runs at a few GB/s, while a pinned one
// runs at the link's rate and, chunk by chunk, overlaps the host copy of the
// previous chunk into place.  Allocated on first use and kept until the
// process ends; one copy uses them at a time.
constexpr uint64_t kStageBytes = 8ull << 20;
struct Stage {
  std::mutex mu;
  void* buf[2] = {nullptr, nullptr};
  bool tried = false;
};
Stage& stage() {
  static Stage* s = new Stage;   // never destroyed: no HIP call at exit
  return *s;
}

// Touch every page of a large, freshly allocated host range from several
// threads before it is copied into: the page faults of first use, taken one
// at a time by a single copying thread, cost more than the copy itself.  The
// range's whole 2 MiB pages are offered to the kernel as huge pages first
// (where transparent huge pages are enabled, one fault then maps 2 MiB).
void prefault(uint8_t* d, uint64_t n) {
  const unsigned T = std::min(8u, std::max(1u, std::thread::hardware_concurrency()));
  if (n < (8ull << 20) || T < 2) return;
  constexpr uintptr_t kHuge = 2ull << 20;
  const uintptr_t lo = ((uintptr_t)d + kHuge - 1) & ~(kHuge - 1), hi = ((uintptr_t)d + n) & ~(kHuge - 1);
  if (hi > lo) (void)madvise(reinterpret_cast<void*>(lo), hi - lo, MADV_HUGEPAGE);
  const uint64_t part = (n / T + 4095) & ~4095ull;
  std::vector<std::thread> th;
  for (unsigned t = 0; t < T; t++) {
    const uint64_t lo = t * part, hi = std::min(n, lo + part);
    if (lo >= hi) break;
    th.emplace_back([d, lo, hi] {
      volatile uint8_t* v = d;
      for (uint64_t i = lo; i < hi; i += 4096) v[i] = 0;
      v[hi - 1] = 0;
    });
  }
  for (auto& x : th) x.join();
}

}  // namespace

struct Ctx {
  const void* w = nullptr;
  int dt = 0, cont = 0;
  int64_t R = 0, C = 0, cvec = 0;
  hipStream_t st = nullptr;
  std::vector<void*> owned;
  float* x = nullptr;
  float* delta = nullptr;
  double* mu = nullptr;
  int* bad = nullptr;
  int64_t* rows = nullptr;
  int32_t* sfl = nullptr;
  int64_t sfl_vectors = 0, sample_vectors = 0;
  int32_t* fl = nullptr;
  int32_t* lohi = nullptr;
  uint16_t* words = nullptr;   // rANS output rows (cap words per tile), rans() -> payload()
  uint32_t* words_n = nullptr;
  uint32_t cap = 0;
  uint32_t* counts = nullptr;  // kMaxCells histogram cells
  double *num = nullptr, *den = nullptr, *acc = nullptr;
  float* sigma = nullptr;
  std::vector<int64_t> rows_up;   // the row list last uploaded to `rows`
  int32_t* cand = nullptr;        // K candidate field sets of the per-row refinement
  int cand_k = 0;
  int32_t* sel = nullptr;
  float* csig = nullptr;
  double* lq = nullptr;
  uint32_t lq_cells = 0;

  template <class T>
  int alloc(T** p, uint64_t count, const char* what) {
    void* q = nullptr;
    if (hipMalloc(&q, count * sizeof(T) > 0 ? count * sizeof(T) : 1) != hipSuccess) {
      (void)hipGetLastError();
      return fail(EP_ERR_HIP, what);
    }
    owned.push_back(q);
    *p = static_cast<T*>(q);
    return EP_OK;
  }
  void release(void* p) {
    for (auto& q : owned)
      if (q == p) {
        (void)hipFree(q);
        q = nullptr;
      }
  }
  int sync(const char* what) {
    if (hipStreamSynchronize(st) != hipSuccess || hipGetLastError() != hipSuccess)
      return fail(EP_ERR_HIP, what);
    return EP_OK;
  }
  int to_host(void* dst, const void* src, uint64_t bytes, const char* what) {
    if (bytes && hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, st) != hipSuccess)
      return fail(EP_ERR_HIP, what);
    return sync(what);
  }
  // The same copy staged through the pinned buffers (chunks of kStageBytes):
  // the transfer of chunk i runs while chunk i - 1 is copied into place, and
  // the destination's pages are mapped first.  Without the pinned buffers
  // (their allocation failed), a plain copy.
  int to_host_staged(void* dst, const void* src, uint64_t bytes, const char* what) {
    Stage& S = stage();
    std::lock_guard<std::mutex> lock(S.mu);
    if (!S.tried) {
      S.tried = true;
      for (void*& b : S.buf)
        if (hipHostMalloc(&b, kStageBytes, hipHostMallocDefault) != hipSuccess) {
          (void)hipGetLastError();
          b = nullptr;
        }
    }
    if (!S.buf[0] || !S.buf[1]) return to_host(dst, src, bytes, what);
    uint8_t* d = static_cast<uint8_t*>(dst);
    const uint8_t* g = static_cast<const uint8_t*>(src);
    prefault(d, bytes);
    uint64_t prev_off = 0, prev_n = 0;
    int prev_b = 0;
    for (uint64_t off = 0, i = 0; off < bytes || prev_n; i++) {
      const uint64_t n = off < bytes ? std::min(kStageBytes, bytes - off) : 0;
      const int b = (int)(i & 1);
      if (n && hipMemcpyAsync(S.buf[b], g + off, n, hipMemcpyDeviceToHost, st) != hipSuccess)
        return fail(EP_ERR_HIP, what);
      if (prev_n) std::memcpy(d + prev_off, S.buf[prev_b], prev_n);
      if (n && sync(what) != EP_OK) return EP_ERR_HIP;
      prev_off = off;
      prev_n = n;
      prev_b = b;
      off += n;
    }
    return EP_OK;
  }
  int to_dev(void* dst, const void* src, uint64_t bytes, const char* what) {
    if (bytes && hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, st) != hipSuccess)
      return fail(EP_ERR_HIP, what);
    return EP_OK;
  }
};

#define EP_GTRY(call)             \
  do {                            \
    int rc_ = (call);             \
    if (rc_ != EP_OK) return rc_; \
  } while (0)
#define EP_LAUNCHED(what) \
  if (hipGetLastError() != hipSuccess) return fail(EP_ERR_HIP, what)

int open(Ctx** out, const void* d_w, int dt, int64_t R, int64_t C, int container, void* stream) {
  *out = nullptr;
  if (R >= (int64_t(1) << 31)) return fail(EP_ERR_UNSUPPORTED, "ep_encode_gpu: more than 2^31 rows");
  Ctx* c = new Ctx;
  c->w = d_w;
  c->dt = dt;
  c->cont = container;
  c->R = R;
  c->C = C;
  c->cvec = C / 8;
  c->st = static_cast<hipStream_t>(stream);
  const uint64_t N = (uint64_t)R * (uint64_t)C;
  int rc = EP_OK;
  if ((rc = c->alloc(&c->x, N, "ep_encode_gpu: device allocation (values)")) != EP_OK ||
      (rc = c->alloc(&c->delta, R, "ep_encode_gpu: device allocation")) != EP_OK ||
      (rc = c->alloc(&c->mu, R, "ep_encode_gpu: device allocation")) != EP_OK ||
      (rc = c->alloc(&c->bad, 1, "ep_encode_gpu: device allocation")) != EP_OK ||
      (rc = c->alloc(&c->rows, R, "ep_encode_gpu: device allocation")) != EP_OK ||
      (rc = c->alloc(&c->fl, N / 8 * 9, "ep_encode_gpu: device allocation (fields)")) != EP_OK ||
      (rc = c->alloc(&c->lohi, 2 * kTablesN, "ep_encode_gpu: device allocation")) != EP_OK ||
      (rc = c->alloc(&c->counts, kMaxCells, "ep_encode_gpu: device allocation")) != EP_OK ||
      (rc = c->alloc(&c->num, R, "ep_encode_gpu: device allocation")) != EP_OK ||
      (rc = c->alloc(&c->den, R, "ep_encode_gpu: device allocation")) != EP_OK ||
      (rc = c->alloc(&c->acc, 4 * (uint64_t)R, "ep_encode_gpu: device allocation")) != EP_OK ||
      (rc = c->alloc(&c->sigma, R, "ep_encode_gpu: device allocation")) != EP_OK) {
    close(c);
    return rc;
  }
  *out = c;
  return EP_OK;
}

void close(Ctx* c) {
  if (!c) return;
  if (c->st) (void)hipStreamSynchronize(c->st);
  for (void* q : c->owned)
    if (q) (void)hipFree(q);
  delete c;
}

int prep(Ctx* c, float* delta, double* mu) {
  const int zero = 0;
  EP_GTRY(c->to_dev(c->bad, &zero, sizeof(int), "ep_encode_gpu: copy"));
  if (hipMemsetAsync(c->delta, 0, 4 * (size_t)c->R, c->st) != hipSuccess)
    return fail(EP_ERR_HIP, "ep_encode_gpu: clear");
  double tmax = -1.0;
  if (c->cont == EP_CONT_UINT8_TENSOR) {
    hipLaunchKernelGGL(k_prep_rows, dim3((unsigned)c->R), dim3(256), 0, c->st, c->w, c->dt, c->C,
                       c->cont, -1.0, c->x, c->delta, c->bad);
    EP_LAUNCHED("ep_encode_gpu: launch (row amax)");
    std::vector<float> am((size_t)c->R);
    EP_GTRY(c->to_host(am.data(), c->delta, 4 * (uint64_t)c->R, "ep_encode_gpu: prep"));
    tmax = 0.0;
    for (float a : am) tmax = a > tmax ? (double)a : tmax;
  }
  hipLaunchKernelGGL(k_prep_rows, dim3((unsigned)c->R), dim3(256), 0, c->st, c->w, c->dt, c->C,
                     c->cont, tmax, c->x, c->delta, c->bad);
  EP_LAUNCHED("ep_encode_gpu: launch (prep)");
  hipLaunchKernelGGL(k_prep_mu, dim3(blocks_for(c->R, kRowsPerBlock)), dim3(kFetchThreads), 0, c->st,
                     c->x, c->R, c->C, c->mu);
  EP_LAUNCHED("ep_encode_gpu: launch (row rms)");
  int bad = 0;
  EP_GTRY(c->to_host(&bad, c->bad, sizeof(int), "ep_encode_gpu: prep"));
  if (bad) return fail(EP_ERR_ARG, "ep_encode: non-finite input value");
  EP_GTRY(c->to_host(delta, c->delta, 4 * (uint64_t)c->R, "ep_encode_gpu: prep"));
  return c->to_host(mu, c->mu, 8 * (uint64_t)c->R, "ep_encode_gpu: prep");
}

int quantize(Ctx* c, const int64_t* rows, int64_t nrows, double s, int32_t* lohi) {
  int32_t* dst = c->fl;
  const int64_t nv = nrows * c->cvec;
  if (rows) {
    if (nv > c->sfl_vectors) {
      if (c->sfl) c->release(c->sfl);
      c->sfl = nullptr;
      EP_GTRY(c->alloc(&c->sfl, (uint64_t)nv * 9, "ep_encode_gpu: device allocation (sample)"));
      c->sfl_vectors = nv;
    }
    dst = c->sfl;
    c->sample_vectors = nv;
    if ((int64_t)c->rows_up.size() != nrows ||
        std::memcmp(c->rows_up.data(), rows, 8 * (size_t)nrows) != 0) {
      c->rows_up.assign(rows, rows + nrows);
      EP_GTRY(c->to_dev(c->rows, c->rows_up.data(), 8 * (uint64_t)nrows, "ep_encode_gpu: copy (rows)"));
    }
  }
  int32_t init[2 * kTablesN];
  for (int i = 0; i < kTablesN; i++) {
    init[2 * i] = INT_MAX;
    init[2 * i + 1] = INT_MIN;
  }
  EP_GTRY(c->to_dev(c->lohi, init, sizeof(init), "ep_encode_gpu: copy"));
  hipLaunchKernelGGL(k_quantize, dim3(blocks_for(nv, 256)), dim3(256), 0, c->st, c->x, c->mu,
                     rows ? c->rows : nullptr, nrows, c->cvec, c->C, s, dst, c->lohi);
  EP_LAUNCHED("ep_encode_gpu: launch (quantize)");
  return c->to_host(lohi, c->lohi, sizeof(init), "ep_encode_gpu: quantize");
}

namespace {
TableDesc desc_of(const int32_t* lo, const int32_t* A, uint32_t* cells) {
  TableDesc td;
  uint32_t base = 0;
  for (int i = 0; i < kTablesN; i++) {
    td.lo[i] = lo[i];
    td.base[i] = base;
    base += (uint32_t)A[i];
  }
  *cells = base;
  return td;
}
}  // namespace

namespace {
int count_on(Ctx* c, const int32_t* src, int64_t nv, const int32_t* lo, const int32_t* A, uint64_t* n) {
  uint32_t cells = 0;
  const TableDesc td = desc_of(lo, A, &cells);
  if (cells > kMaxCells) return fail(EP_ERR_ARG, "ep_encode_gpu: count of a table wider than 2^15");
  uint32_t* d = c->counts;
  if (hipMemsetAsync(d, 0, 4ull * cells, c->st) != hipSuccess) return fail(EP_ERR_HIP, "ep_encode_gpu: clear");
  const unsigned grid = (unsigned)std::min<int64_t>(256, (nv + 255) / 256);
  if (grid) {
    if (cells <= kLdsBins) {
      if (hipFuncSetAttribute((const void*)k_count_lds, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)(4 * kLdsBins)) != hipSuccess)
        return fail(EP_ERR_HIP, "ep_encode_gpu: LDS limit");
      hipLaunchKernelGGL(k_count_lds, dim3(grid), dim3(256), 4 * cells, c->st, src, nv, td, cells, d);
    } else {
      hipLaunchKernelGGL(k_count_mem, dim3(grid), dim3(256), 0, c->st, src, nv, td, d);
    }
    EP_LAUNCHED("ep_encode_gpu: launch (count)");
  }
  std::vector<uint32_t> h(cells);
  EP_GTRY(c->to_host(h.data(), d, 4ull * cells, "ep_encode_gpu: count"));
  for (uint32_t i = 0; i < cells; i++) n[i] = h[i];
  return EP_OK;
}
}  // namespace

int count(Ctx* c, bool sample, const int32_t* lo, const int32_t* A, uint64_t* n) {
  return count_on(c, sample ? c->sfl : c->fl, sample ? c->sample_vectors : c->R * c->cvec, lo, A, n);
}

int refit(Ctx* c, double* num, double* den) {
  hipLaunchKernelGGL(k_refit, dim3(blocks_for(c->R, kRowsPerBlock)), dim3(kFetchThreads), 0, c->st,
                     c->x, c->fl, c->R, c->cvec, c->num, c->den);
  EP_LAUNCHED("ep_encode_gpu: launch (refit)");
  EP_GTRY(c->to_host(num, c->num, 8 * (uint64_t)c->R, "ep_encode_gpu: refit"));
  return c->to_host(den, c->den, 8 * (uint64_t)c->R, "ep_encode_gpu: refit");
}

int rans(Ctx* c, int b, uint32_t V, uint64_t tiles, const int32_t* lo, const int32_t* A,
         const uint32_t* f, uint32_t* states, uint64_t* words) {
  uint32_t cells = 0;
  const TableDesc td = desc_of(lo, A, &cells);
  std::vector<uint2> tab(cells);
  for (int i = 0; i < kTablesN; i++) {
    uint32_t F = 0;
    for (int32_t z = 0; z < A[i]; z++) {
      tab[td.base[i] + z] = make_uint2(f[td.base[i] + z], F);
      F += f[td.base[i] + z];
    }
  }
  const uint32_t rounds_max = (V + kLanesN - 1) / kLanesN;
  const uint64_t cap = 9ull * rounds_max * kLanesN;
  if (cap > 0xFFFFFFFFull) return fail(EP_ERR_UNSUPPORTED, "ep_encode_gpu: tile too large");
  uint2* dtab = nullptr;
  uint32_t *dst = nullptr, *dcnt = nullptr;
  uint16_t* scr = nullptr;
  EP_GTRY(c->alloc(&dtab, cells, "ep_encode_gpu: device allocation"));
  EP_GTRY(c->alloc(&dst, tiles * kLanesN, "ep_encode_gpu: device allocation"));
  EP_GTRY(c->alloc(&dcnt, tiles, "ep_encode_gpu: device allocation"));
  EP_GTRY(c->alloc(&scr, tiles * cap, "ep_encode_gpu: device allocation (rANS words)"));
  EP_GTRY(c->to_dev(dtab, tab.data(), 8ull * cells, "ep_encode_gpu: copy (tables)"));
  hipLaunchKernelGGL(k_rans, dim3((unsigned)((tiles + 1) / 2)), dim3(64), 0, c->st, c->fl,
                     (uint64_t)(c->R * c->cvec), V, rounds_max, tiles, td, dtab, b, dst, dcnt, scr,
                     (uint32_t)cap);
  EP_LAUNCHED("ep_encode_gpu: launch (rANS)");
  std::vector<uint32_t> cnt(tiles);
  EP_GTRY(c->to_host(states, dst, 4 * tiles * kLanesN, "ep_encode_gpu: rANS"));
  EP_GTRY(c->to_host(cnt.data(), dcnt, 4 * tiles, "ep_encode_gpu: rANS"));
  for (uint64_t t = 0; t < tiles; t++) words[t] = cnt[t];
  c->release(dtab);
  c->release(dst);
  c->words = scr;
  c->words_n = dcnt;
  c->cap = (uint32_t)cap;
  return EP_OK;
}

int payload(Ctx* c, const uint32_t* offs, uint64_t tiles, uint64_t total_words, uint8_t* dst) {
  if (!c->words) return fail(EP_ERR_ARG, "ep_encode_gpu: payload before rans");
  uint32_t* doffs = nullptr;
  uint16_t* dpay = nullptr;
  EP_GTRY(c->alloc(&doffs, tiles + 1, "ep_encode_gpu: device allocation"));
  EP_GTRY(c->alloc(&dpay, total_words, "ep_encode_gpu: device allocation (payload)"));
  EP_GTRY(c->to_dev(doffs, offs, 4 * (tiles + 1), "ep_encode_gpu: copy (offsets)"));
  if (tiles) {
    hipLaunchKernelGGL(k_gather, dim3((unsigned)tiles), dim3(256), 0, c->st, c->words, c->cap,
                       c->words_n, doffs, dpay);
    EP_LAUNCHED("ep_encode_gpu: launch (payload)");
  }
  EP_GTRY(c->to_host_staged(dst, dpay, 2 * total_words, "ep_encode_gpu: payload"));
  c->release(doffs);
  c->release(dpay);
  c->release(c->words);
  c->release(c->words_n);
  c->words = nullptr;
  c->words_n = nullptr;
  return EP_OK;
}

int errors(Ctx* c, const float* sigma, int rdt, double* acc) {
  EP_GTRY(c->to_dev(c->sigma, sigma, 4 * (uint64_t)c->R, "ep_encode_gpu: copy (scales)"));
  hipLaunchKernelGGL(k_errors, dim3((unsigned)c->R), dim3(256), 0, c->st, c->w, c->dt, c->x, c->fl,
                     c->sigma, c->delta, rdt, c->cont, c->cvec, c->acc);
  EP_LAUNCHED("ep_encode_gpu: launch (errors)");
  return c->to_host(acc, c->acc, 32 * (uint64_t)c->R, "ep_encode_gpu: errors");
}

// ---- per-row refinement ----------------------------------------------------
namespace {
int32_t* cand_ptr(Ctx* c, int k) { return c->cand + (uint64_t)k * (uint64_t)(c->R * c->cvec) * 9; }
void init_lohi(int32_t* init) {
  for (int i = 0; i < kTablesN; i++) {
    init[2 * i] = INT_MAX;
    init[2 * i + 1] = INT_MIN;
  }
}
}  // namespace

int cand_alloc(Ctx* c, int K) {
  if (c->cand) return fail(EP_ERR_ARG, "ep_encode_gpu: candidates already allocated");
  const uint64_t nvec = (uint64_t)(c->R * c->cvec);
  EP_GTRY(c->alloc(&c->cand, nvec * 9 * (uint64_t)K, "ep_encode_gpu: device allocation (candidates)"));
  EP_GTRY(c->alloc(&c->sel, (uint64_t)c->R, "ep_encode_gpu: device allocation"));
  c->cand_k = K;
  return EP_OK;
}

int cand_quantize(Ctx* c, int k, double s, int32_t* lohi) {
  if (k < 0 || k >= c->cand_k) return fail(EP_ERR_ARG, "ep_encode_gpu: candidate index");
  int32_t init[2 * kTablesN];
  init_lohi(init);
  EP_GTRY(c->to_dev(c->lohi, init, sizeof(init), "ep_encode_gpu: copy"));
  const int64_t nv = c->R * c->cvec;
  hipLaunchKernelGGL(k_quantize, dim3(blocks_for(nv, 256)), dim3(256), 0, c->st, c->x, c->mu,
                     nullptr, c->R, c->cvec, c->C, s, cand_ptr(c, k), c->lohi);
  EP_LAUNCHED("ep_encode_gpu: launch (candidate quantize)");
  return c->to_host(lohi, c->lohi, sizeof(init), "ep_encode_gpu: candidate quantize");
}

int cand_refit(Ctx* c, int k, double* num, double* den) {
  hipLaunchKernelGGL(k_refit, dim3(blocks_for(c->R, kRowsPerBlock)), dim3(kFetchThreads), 0, c->st,
                     c->x, cand_ptr(c, k), c->R, c->cvec, c->num, c->den);
  EP_LAUNCHED("ep_encode_gpu: launch (candidate refit)");
  EP_GTRY(c->to_host(num, c->num, 8 * (uint64_t)c->R, "ep_encode_gpu: candidate refit"));
  return c->to_host(den, c->den, 8 * (uint64_t)c->R, "ep_encode_gpu: candidate refit");
}

int cand_distortion(Ctx* c, int k, const float* sigma, double* D) {
  EP_GTRY(c->to_dev(c->sigma, sigma, 4 * (uint64_t)c->R, "ep_encode_gpu: copy (scales)"));
  hipLaunchKernelGGL(k_dist, dim3(blocks_for(c->R, kRowsPerBlock)), dim3(kRowsPerBlock), 0, c->st,
                     c->x, cand_ptr(c, k), c->sigma, c->R, c->cvec, c->num);
  EP_LAUNCHED("ep_encode_gpu: launch (distortion)");
  return c->to_host(D, c->num, 8 * (uint64_t)c->R, "ep_encode_gpu: distortion");
}

int cand_rate(Ctx* c, int k, const double* lq, const int32_t* lo, const int32_t* A, double* Rt) {
  uint32_t cells = 0;
  const TableDesc td = desc_of(lo, A, &cells);
  if (cells > c->lq_cells) {
    if (c->lq) c->release(c->lq);
    c->lq = nullptr;
    EP_GTRY(c->alloc(&c->lq, cells, "ep_encode_gpu: device allocation"));
    c->lq_cells = cells;
  }
  EP_GTRY(c->to_dev(c->lq, lq, 8ull * cells, "ep_encode_gpu: copy (model)"));
  hipLaunchKernelGGL(k_rate, dim3(blocks_for(c->R, kRowsPerBlock)), dim3(kRowsPerBlock), 0, c->st,
                     cand_ptr(c, k), c->lq, td, c->R, c->cvec, c->num);
  EP_LAUNCHED("ep_encode_gpu: launch (rate)");
  return c->to_host(Rt, c->num, 8 * (uint64_t)c->R, "ep_encode_gpu: rate");
}

int cand_select(Ctx* c, const int32_t* sel, int32_t* lohi) {
  int32_t init[2 * kTablesN];
  init_lohi(init);
  EP_GTRY(c->to_dev(c->lohi, init, sizeof(init), "ep_encode_gpu: copy"));
  EP_GTRY(c->to_dev(c->sel, sel, 4 * (uint64_t)c->R, "ep_encode_gpu: copy (selection)"));
  const int64_t nv = c->R * c->cvec;
  hipLaunchKernelGGL(k_select, dim3(blocks_for(nv, 256)), dim3(256), 0, c->st, c->cand,
                     (uint64_t)nv * 9, c->sel, nv, c->cvec, c->fl, c->lohi);
  EP_LAUNCHED("ep_encode_gpu: launch (select)");
  return c->to_host(lohi, c->lohi, sizeof(init), "ep_encode_gpu: select");
}

int cand_count(Ctx* c, int k, const int32_t* lo, const int32_t* A, uint64_t* n) {
  return count_on(c, k < 0 ? c->fl : cand_ptr(c, k), c->R * c->cvec, lo, A, n);
}

}  // namespace genc
}  // namespace ep
