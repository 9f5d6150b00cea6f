// CPU encoder of the MI355X EntroPack library (ep_encode_cpu).
//
// Implements the paper's encoding pipeline (Figure "pipeline", upper path):
// row normalisation and nearest-E8 quantisation (Section 3.2), the integer
// field map (eq. parity), the 17-table coset-conditioned model with b-bit
// frequencies (Section 3.3), sampled-row rate estimation with geometric scale
// search and precision escalation (Section 3.4, Alg. rate selection,
// Appendix C.1), the least-squares row-scale refit (Section 3.5, eq.
// scale_fit), and tiled 32-state interleaved rANS (Section 3.6,
// Appendix C.3).  The byte layout is documented in include/entropack.h.
//
// Work is split over rows (quantisation, refit), per-thread histograms
// (counts) and tiles (rANS); every reduction that involves rounding runs in a
// fixed order, so the blob does not depend on the thread count.
#include <algorithm>
#include <array>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <limits>
#include <new>
#include <thread>
#include <vector>

#include "../../include/entropack.h"
#include "common.h"
#include "encode_gpu.h"
#include "encode_math.h"

namespace ep {
namespace {

constexpr uint32_t kLanes = 32;        // interleaved states per tile
constexpr uint32_t kStateLow = 1u << 15;
constexpr int kTables = 17;            // coset + (8 fields x 2 cosets)

// ---- small parallel-for over [0, n) with static contiguous chunks ---------
void parallel_for(int64_t n, int nthreads, const std::function<void(int64_t, int64_t, int)>& fn) {
  if (n <= 0) return;
  int T = (int)std::min<int64_t>(nthreads, n);
  if (T <= 1) {
    fn(0, n, 0);
    return;
  }
  std::vector<std::thread> th;
  th.reserve(T);
  for (int t = 0; t < T; t++) {
    int64_t b = n * t / T, e = n * (t + 1) / T;
    th.emplace_back([&fn, b, e, t] { fn(b, e, t); });
  }
  for (auto& x : th) x.join();
}

using em::int8_snap;
using em::kEta;
using em::table_index;
using em::to_bf16;
using em::to_e4m3;
using em::to_fp16;

double half_bits_to_double(uint16_t h) {
  int e = (h >> 10) & 0x1F, m = h & 0x3FF;
  double v = e == 0 ? std::ldexp((double)m, -24)
                    : (e == 31 ? (m ? NAN : INFINITY) : std::ldexp(1024.0 + m, e - 25));
  return (h & 0x8000) ? -v : v;
}

double input_at(const void* w, int dt, int64_t i) {
  if (dt == EP_FP32) return (double)static_cast<const float*>(w)[i];
  uint16_t h = static_cast<const uint16_t*>(w)[i];
  if (dt == EP_FP16) return half_bits_to_double(h);
  uint32_t u = (uint32_t)h << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

// ---- lattice: em::d8_point, em::e8_point, em::split_fields (encode_math.h)

// ---- model ---------------------------------------------------------------
struct Table {
  int32_t lo = 0;
  int32_t A = 0;
  std::vector<uint64_t> n;
  std::vector<uint32_t> f;
};

struct Model {
  Table t[kTables];
  int32_t max_field_alphabet() const {
    int32_t m = 0;
    for (int i = 1; i < kTables; i++) m = std::max(m, t[i].A);
    return m;
  }
  uint64_t serialized_bytes() const {
    uint64_t s = 4;
    for (int i = 1; i < kTables; i++) s += 8 + ((2ull * (uint64_t)t[i].A + 3) / 4) * 4;
    return s;
  }
};

// Counts of the field values of nv vectors (9 int32 each), built with
// per-thread histograms.
void count_fields(const int32_t* fl, int64_t nv, int nthreads, Model& md) {
  int T = (int)std::max<int64_t>(1, std::min<int64_t>(nthreads, nv / 4096 + 1));
  std::vector<std::array<int32_t, 2 * kTables>> ext(T);
  for (auto& e : ext)
    for (int i = 0; i < kTables; i++) {
      e[2 * i] = std::numeric_limits<int32_t>::max();
      e[2 * i + 1] = std::numeric_limits<int32_t>::min();
    }
  parallel_for(nv, T, [&](int64_t b, int64_t e, int tid) {
    auto& x = ext[tid];
    for (int64_t v = b; v < e; v++) {
      const int32_t* q = fl + 9 * v;
      for (int i = 1; i <= 8; i++) {
        int ti = table_index(i, q[0]);
        x[2 * ti] = std::min(x[2 * ti], q[i]);
        x[2 * ti + 1] = std::max(x[2 * ti + 1], q[i]);
      }
    }
  });
  for (int i = 0; i < kTables; i++) {
    int32_t lo = std::numeric_limits<int32_t>::max(), hi = std::numeric_limits<int32_t>::min();
    if (i == 0) {
      lo = 0;
      hi = 1;
    }
    for (auto& x : ext) {
      lo = std::min(lo, x[2 * i]);
      hi = std::max(hi, x[2 * i + 1]);
    }
    Table& tb = md.t[i];
    tb.lo = hi >= lo ? lo : 0;
    tb.A = hi >= lo ? (int32_t)((int64_t)hi - lo + 1) : 0;
    tb.n.assign((size_t)tb.A, 0);
    tb.f.assign((size_t)tb.A, 0);
  }
  // counting: per-thread arrays when small, else a single pass
  uint64_t cells = 0;
  for (int i = 0; i < kTables; i++) cells += md.t[i].A;
  std::vector<std::vector<uint64_t>> part(T, std::vector<uint64_t>(cells, 0));
  std::vector<uint64_t> base(kTables, 0);
  for (int i = 1; i < kTables; i++) base[i] = base[i - 1] + md.t[i - 1].A;
  parallel_for(nv, T, [&](int64_t b, int64_t e, int tid) {
    uint64_t* h = part[tid].data();
    for (int64_t v = b; v < e; v++) {
      const int32_t* q = fl + 9 * v;
      h[q[0]]++;
      for (int i = 1; i <= 8; i++) {
        int ti = table_index(i, q[0]);
        h[base[ti] + (q[i] - md.t[ti].lo)]++;
      }
    }
  });
  for (int i = 0; i < kTables; i++)
    for (int32_t z = 0; z < md.t[i].A; z++) {
      uint64_t s = 0;
      for (int t = 0; t < T; t++) s += part[t][base[i] + z];
      md.t[i].n[z] = s;
    }
}

// b-bit frequencies: floor share (at least 1 for observed symbols); missing
// units to the largest shortfall M n - f N (smaller symbol first); surplus
// taken one unit at a time from the largest frequency above 1 (smaller symbol
// first).  Section 3.3 requires only sum = 2^b and f > 0 on observed symbols.
bool quantize_freqs(Table& tb, int b) {
  const uint64_t M = 1ull << b;
  uint64_t N = 0, K = 0;
  for (auto c : tb.n) {
    N += c;
    K += c != 0;
  }
  std::fill(tb.f.begin(), tb.f.end(), 0u);
  if (!N) return true;
  if (K > M) return false;
  int64_t assigned = 0;
  for (int32_t z = 0; z < tb.A; z++) {
    if (!tb.n[z]) continue;
    uint64_t share = (M * tb.n[z]) / N;
    tb.f[z] = (uint32_t)std::max<uint64_t>(1, share);
    assigned += tb.f[z];
  }
  int64_t missing = (int64_t)M - assigned;
  if (missing > 0) {
    std::vector<std::pair<int64_t, int32_t>> cand;
    cand.reserve(K);
    for (int32_t z = 0; z < tb.A; z++)
      if (tb.n[z]) cand.emplace_back((int64_t)(M * tb.n[z]) - (int64_t)tb.f[z] * (int64_t)N, z);
    std::sort(cand.begin(), cand.end(), [](const auto& a, const auto& b) {
      return a.first != b.first ? a.first > b.first : a.second < b.second;
    });
    for (int64_t i = 0; i < missing; i++) tb.f[cand[i].second]++;
  }
  for (; missing < 0; missing++) {
    int32_t arg = -1;
    for (int32_t z = 0; z < tb.A; z++)
      if (tb.f[z] > 1 && (arg < 0 || tb.f[z] > tb.f[arg])) arg = z;
    tb.f[arg]--;
  }
  return true;
}

// Model code length C_CE in bits (eq. length), summed per table then over
// tables in index order.
double model_bits(const Model& md, int b) {
  double total = 0;
  for (int i = 0; i < kTables; i++) {
    double part = 0;
    const Table& tb = md.t[i];
    for (int32_t z = 0; z < tb.A; z++)
      if (tb.n[z]) part += (double)tb.n[z] * ((double)b - std::log2((double)tb.f[z]));
    total += part;
  }
  return total;
}

// Stored-size estimate in bits (eq. estimate, eq. outer_estimate); all terms
// except the payload are the exact serialized sizes.
double estimated_bits(double cce, uint64_t tiles, double credit, const Model& md, uint64_t rows,
                      int container) {
  double rest = cce - credit * (double)kLanes * (double)tiles;
  if (rest < 0) rest = 0;
  double words = std::ceil(rest / 16.0);
  double payload = 16.0 * words;
  double pad = std::fmod(words, 2.0) == 1.0 ? 16.0 : 0.0;
  double meta = 8.0 * (double)(132ull * tiles + 4ull);
  double tables = 8.0 * (double)md.serialized_bytes();
  double scales = 32.0 * (double)rows * (container ? 2.0 : 1.0);
  double header = 8.0 * kHeaderBytes;
  return payload + pad + meta + tables + scales + header;
}

// ---- sampling --------------------------------------------------------------
uint64_t splitmix_next(uint64_t& s) {
  s += 0x9E3779B97F4A7C15ull;
  uint64_t z = s;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

std::vector<int64_t> pick_rows(int64_t R, int64_t C, int64_t nominal_vectors) {
  int64_t per_row = C / 8;
  int64_t want = (nominal_vectors + per_row - 1) / per_row;
  std::vector<int64_t> idx((size_t)R);
  for (int64_t r = 0; r < R; r++) idx[r] = r;
  if (want >= R) return idx;
  uint64_t s = ((uint64_t)R << 32) ^ (uint64_t)C;
  for (int64_t i = 0; i < want; i++) {
    int64_t j = i + (int64_t)(splitmix_next(s) % (uint64_t)(R - i));
    std::swap(idx[i], idx[j]);
  }
  idx.resize((size_t)want);
  std::sort(idx.begin(), idx.end());
  return idx;
}

#define EP_TRY_G(call)          \
  do {                          \
    int rcg_ = (call);          \
    if (rcg_ != EP_OK) return rcg_; \
  } while (0)

// ---- backends -----------------------------------------------------------
// The search, refit, table and serialisation logic below is shared; a
// backend supplies the bulk work on its own device:
//   prep      coded values, container scales delta_r and row RMS mu_r;
//   quantize  fields of a row set at scale s, model extents, counts (when
//             every field table fits `cap`), refit sums;
//   rans      terminal states and words per tile;
//   payload   the tiles' words at their offsets;
//   errors    per-row squared errors and norms for the statistics.
struct CpuBackend {
  const void* w;
  int dt;
  int64_t R, C, cvec;
  int T;
  std::vector<float> x;       // coded values (fp32-exact)
  std::vector<float> delta;   // container scales
  std::vector<double> mu;     // row RMS
  std::vector<int32_t> sfl, fl;                  // sample / full fields, 9 per vector
  std::vector<std::vector<uint16_t>> tile_words;

  int prep(int cont) {
    const int64_t N = R * C;
    x.resize((size_t)N);
    delta.assign((size_t)R, 0.0f);
    mu.resize((size_t)R);
    std::vector<char> bad((size_t)R, 0);
    std::vector<double> am((size_t)R, 0.0);
    parallel_for(R, T, [&](int64_t b, int64_t e, int) {
      for (int64_t r = b; r < e; r++) {
        double amax = 0;
        float* xr = x.data() + r * C;
        for (int64_t j = 0; j < C; j++) {
          float v = (float)input_at(w, dt, r * C + j);
          if (!std::isfinite(v)) bad[r] = 1;
          xr[j] = v;
          amax = std::max(amax, std::fabs((double)v));
        }
        am[r] = amax;
      }
    });
    double tmax = 0;   // one scale for the whole tensor (unsigned container)
    for (double a : am) tmax = std::max(tmax, a);
    parallel_for(R, T, [&](int64_t b, int64_t e, int) {
      for (int64_t r = b; r < e; r++) {
        const double amax = cont == EP_CONT_UINT8_TENSOR ? tmax : am[r];
        float* xr = x.data() + r * C;
        if (cont) {
          float d = amax > 0 ? (float)(amax / em::container_max(cont)) : 1.0f;
          delta[r] = d;
          for (int64_t j = 0; j < C; j++) {
            double q = (double)xr[j] / (double)d;
            xr[j] = (float)em::container_snap(cont, q);
          }
        }
        double ss = 0;
        for (int64_t j = 0; j < C; j++) ss += (double)xr[j] * (double)xr[j];
        double m = std::sqrt(ss / (double)C);
        mu[r] = m > kEta ? m : kEta;
      }
    });
    for (char c : bad)
      if (c) return fail(EP_ERR_ARG, "ep_encode: non-finite input value");
    return EP_OK;
  }

  // quantise rows (all rows when `rows` is null) into fields; optional refit sums
  int quantize(const std::vector<int64_t>* rows, double s, Model& md, int64_t /*cap*/,
               double* num, double* den) {
    const int64_t nr = rows ? (int64_t)rows->size() : R;
    std::vector<int32_t>& out = rows ? sfl : fl;
    out.resize((size_t)(nr * cvec * 9));
    int32_t* f9 = out.data();
    parallel_for(nr, T, [&](int64_t b, int64_t e, int) {
      for (int64_t k = b; k < e; k++) {
        int64_t r = rows ? (*rows)[k] : k;
        const float* xr = x.data() + r * C;
        double sn = 0, sd = 0;
        for (int64_t jv = 0; jv < cvec; jv++) {
          double y[8];
          int32_t p2[8];
          for (int j = 0; j < 8; j++) y[j] = ((double)xr[8 * jv + j] / mu[r]) / s;
          em::e8_point(y, p2);
          em::split_fields(p2, f9 + 9 * (k * cvec + jv));
          if (num)
            for (int j = 0; j < 8; j++) {
              double pj = p2[j] / 2.0;
              sn += (double)xr[8 * jv + j] * pj;
              sd += pj * pj;
            }
        }
        if (num) {
          num[r] = sn;
          den[r] = sd;
        }
      }
    });
    md = Model();
    count_fields(f9, nr * cvec, T, md);
    return EP_OK;
  }

  int rans(const Model& full, int b, uint32_t V, uint64_t tiles, std::vector<uint32_t>& states,
           std::vector<uint64_t>& words) {
    const uint64_t nvec = (uint64_t)(R * cvec);
    const uint32_t M = 1u << b;
    std::vector<std::vector<uint32_t>> cum(kTables);
    for (int i = 0; i < kTables; i++) {
      cum[i].assign((size_t)full.t[i].A + 1, 0);
      for (int32_t z = 0; z < full.t[i].A; z++) cum[i][z + 1] = cum[i][z] + full.t[i].f[z];
    }
    states.assign(tiles * kLanes, 0);
    words.assign(tiles, 0);
    tile_words.assign(tiles, {});
    parallel_for((int64_t)tiles, T, [&](int64_t tb, int64_t te, int) {
      for (int64_t t = tb; t < te; t++) {
        uint64_t v0 = (uint64_t)t * V;
        uint64_t nv = std::min<uint64_t>(V, nvec - v0);
        uint64_t rounds = (nv + kLanes - 1) / kLanes;
        uint32_t st[kLanes];
        for (auto& q : st) q = kStateLow;
        std::vector<uint16_t>& out_w = tile_words[t];
        for (uint64_t step = 9 * rounds; step-- > 0;) {
          uint64_t k = step / 9;
          int fi = (int)(step % 9);
          for (int l = (int)kLanes - 1; l >= 0; l--) {
            uint64_t li = (uint64_t)l + kLanes * k;
            if (li >= nv) continue;
            const int32_t* q = fl.data() + 9 * (v0 + li);
            int ti = table_index(fi, q[0]);
            int32_t z = fi == 0 ? q[0] : q[fi] - full.t[ti].lo;
            uint64_t f = full.t[ti].f[z], F = cum[ti][z];
            uint64_t xs = st[l];
            if (xs >= (f << (31 - b))) {
              out_w.push_back((uint16_t)(xs & 0xFFFF));
              xs >>= 16;
            }
            st[l] = (uint32_t)((xs / f) * M + xs % f + F);
          }
        }
        std::reverse(out_w.begin(), out_w.end());
        for (uint32_t l = 0; l < kLanes; l++) states[t * kLanes + l] = st[l];
        words[t] = out_w.size();
      }
    });
    return EP_OK;
  }

  // ---- per-row refinement primitives (the algorithm is rdo_run below) ----
  std::vector<std::vector<int32_t>> cf;   // candidate field sets

  int rdo_alloc(int K) {
    cf.assign((size_t)K, {});
    return EP_OK;
  }
  // candidate k <- every row's fields at scale sk; extents; refit sums in element order
  int rdo_quantize(int k, double sk, int32_t* lo, int32_t* hi, double* num, double* den) {
    cf[k].resize((size_t)(R * cvec) * 9);
    int32_t* f9 = cf[k].data();
    parallel_for(R, T, [&](int64_t rb, int64_t re, int) {
      for (int64_t r = rb; r < re; r++) {
        const float* xr = x.data() + r * C;
        double sn = 0, sd = 0;
        for (int64_t jv = 0; jv < cvec; jv++) {
          double y[8];
          int32_t p2[8];
          for (int j = 0; j < 8; j++) y[j] = ((double)xr[8 * jv + j] / mu[r]) / sk;
          em::e8_point(y, p2);
          em::split_fields(p2, f9 + 9 * (r * cvec + jv));
          for (int j = 0; j < 8; j++) {
            double pj = p2[j] / 2.0;
            sn += (double)xr[8 * jv + j] * pj;
            sd += pj * pj;
          }
        }
        num[r] = sn;
        den[r] = sd;
      }
    });
    extents(f9, lo, hi);
    return EP_OK;
  }
  void extents(const int32_t* f9, int32_t* lo, int32_t* hi) const {
    for (int t = 0; t < kTables; t++) {
      lo[t] = std::numeric_limits<int32_t>::max();
      hi[t] = std::numeric_limits<int32_t>::min();
    }
    for (int64_t v = 0; v < R * cvec; v++) {
      const int32_t* q = f9 + 9 * v;
      for (int i = 1; i <= 8; i++) {
        int t = table_index(i, q[0]);
        lo[t] = std::min(lo[t], q[i]);
        hi[t] = std::max(hi[t], q[i]);
      }
    }
  }
  // D_r = sum_j (x_rj - sigma_r p_rj)^2 of candidate k, in element order
  int rdo_distortion(int k, const float* sig, double* D) {
    const int32_t* f9 = cf[k].data();
    parallel_for(R, T, [&](int64_t rb, int64_t re, int) {
      for (int64_t r = rb; r < re; r++) {
        const float* xr = x.data() + r * C;
        double d = 0;
        for (int64_t jv = 0; jv < cvec; jv++) {
          int32_t p2[8];
          em::join_fields(f9 + 9 * (r * cvec + jv), p2);
          for (int j = 0; j < 8; j++) {
            double e = (double)xr[8 * jv + j] - (double)sig[r] * (p2[j] / 2.0);
            d += e * e;
          }
        }
        D[r] = d;
      }
    });
    return EP_OK;
  }
  // R_r of candidate k: sum of lq over the row's symbols in symbol order
  int rdo_rate(int k, const double* lq, const int32_t* lo, const int32_t* A, double* Rt) {
    uint64_t base[kTables];
    uint64_t at = 0;
    for (int t = 0; t < kTables; t++) {
      base[t] = at;
      at += (uint64_t)A[t];
    }
    const int32_t* f9 = cf[k].data();
    parallel_for(R, T, [&](int64_t rb, int64_t re, int) {
      for (int64_t r = rb; r < re; r++) {
        double acc = 0;
        for (int64_t jv = 0; jv < cvec; jv++) {
          const int32_t* q = f9 + 9 * (r * cvec + jv);
          acc += lq[q[0]];
          for (int i = 1; i <= 8; i++) {
            int t = table_index(i, q[0]);
            acc += lq[base[t] + (uint64_t)(q[i] - lo[t])];
          }
        }
        Rt[r] = acc;
      }
    });
    return EP_OK;
  }
  // the full field set <- row r of candidate sel[r]; its extents
  int rdo_select(const int32_t* sel, int32_t* lo, int32_t* hi) {
    fl.resize((size_t)(R * cvec) * 9);
    for (int64_t r = 0; r < R; r++)
      std::copy(cf[sel[r]].begin() + 9 * r * cvec, cf[sel[r]].begin() + 9 * (r + 1) * cvec,
                fl.begin() + 9 * r * cvec);
    extents(fl.data(), lo, hi);
    return EP_OK;
  }
  // counts of candidate k, or of the full set for k < 0 (layout as the GPU backend's)
  int rdo_counts(int k, const int32_t* lo, const int32_t* A, uint64_t* n) {
    const int32_t* f9 = k < 0 ? fl.data() : cf[k].data();
    uint64_t base[kTables];
    uint64_t at = 0;
    for (int t = 0; t < kTables; t++) {
      base[t] = at;
      at += (uint64_t)A[t];
    }
    std::fill(n, n + at, 0);
    for (int64_t v = 0; v < R * cvec; v++) {
      const int32_t* q = f9 + 9 * v;
      n[q[0]]++;
      for (int i = 1; i <= 8; i++) {
        int t = table_index(i, q[0]);
        n[base[t] + (uint64_t)(q[i] - lo[t])]++;
      }
    }
    return EP_OK;
  }



  int payload(uint8_t* dst, const std::vector<uint32_t>& offs) {
    parallel_for((int64_t)tile_words.size(), T, [&](int64_t tb, int64_t te, int) {
      for (int64_t t = tb; t < te; t++)
        if (!tile_words[t].empty())
          std::memcpy(dst + 2ull * offs[t], tile_words[t].data(), 2 * tile_words[t].size());
    });
    return EP_OK;
  }

  // per row: squared error and norm in coded units, then against the input
  int errors(const std::vector<float>& sigma, int rdt, int cont, std::vector<double>& acc) {
    acc.assign((size_t)R * 4, 0.0);
    parallel_for(R, T, [&](int64_t rb, int64_t re, int) {
      for (int64_t r = rb; r < re; r++) {
        double ec = 0, rc = 0, eo = 0, ro = 0;
        for (int64_t jv = 0; jv < cvec; jv++) {
          int32_t two[8];
          em::join_fields(fl.data() + 9 * (r * cvec + jv), two);
          for (int j = 0; j < 8; j++) {
            double y = (double)(float)((double)sigma[r] * (two[j] / 2.0));
            double v = em::snap_out(rdt, y);
            double xc = x[r * C + 8 * jv + j];
            const double off = em::container_offset(cont);
            ec += (v - xc) * (v - xc);
            rc += (xc - off) * (xc - off);
            double wo = (double)(float)input_at(w, dt, r * C + 8 * jv + j);
            double vo = cont ? (v - off) * (double)delta[r] : v;
            eo += (vo - wo) * (vo - wo);
            ro += wo * wo;
          }
        }
        acc[4 * r] = ec;
        acc[4 * r + 1] = rc;
        acc[4 * r + 2] = eo;
        acc[4 * r + 3] = ro;
      }
    });
    return EP_OK;
  }
};

// Bulk passes on the GPU (encode_gpu.hip); extents come back from the
// quantisation pass, counts only when every field table fits `cap` (the
// search discards the counts otherwise).
struct GpuBackend {
  genc::Ctx* c = nullptr;
  int64_t R = 0;
  std::vector<float> delta;
  std::vector<double> mu;
  ~GpuBackend() { genc::close(c); }

  int prep(int) {
    delta.resize((size_t)R);
    mu.resize((size_t)R);
    return genc::prep(c, delta.data(), mu.data());
  }

  int quantize(const std::vector<int64_t>* rows, double s, Model& md, int64_t cap, double* num,
               double* den) {
    int32_t lohi[2 * kTables];
    EP_TRY_G(genc::quantize(c, rows ? rows->data() : nullptr, rows ? (int64_t)rows->size() : R, s, lohi));
    md = Model();
    int32_t lo[kTables], A[kTables];
    for (int i = 0; i < kTables; i++) {
      int32_t l = i ? lohi[2 * i] : 0, h = i ? lohi[2 * i + 1] : 1;
      Table& tb = md.t[i];
      tb.lo = h >= l ? l : 0;
      tb.A = h >= l ? (int32_t)((int64_t)h - l + 1) : 0;
      lo[i] = tb.lo;
      A[i] = tb.A;
    }
    if (md.max_field_alphabet() <= cap) {
      uint64_t cells = 0;
      for (int i = 0; i < kTables; i++) cells += (uint64_t)A[i];
      std::vector<uint64_t> n(cells);
      EP_TRY_G(genc::count(c, rows != nullptr, lo, A, n.data()));
      uint64_t at = 0;
      for (int i = 0; i < kTables; i++) {
        Table& tb = md.t[i];
        tb.n.assign(n.begin() + at, n.begin() + at + tb.A);
        tb.f.assign((size_t)tb.A, 0);
        at += tb.A;
      }
    }
    if (num) EP_TRY_G(genc::refit(c, num, den));
    return EP_OK;
  }

  int rans(const Model& full, int b, uint32_t V, uint64_t tiles, std::vector<uint32_t>& states,
           std::vector<uint64_t>& words) {
    int32_t lo[kTables], A[kTables];
    std::vector<uint32_t> f;
    for (int i = 0; i < kTables; i++) {
      lo[i] = full.t[i].lo;
      A[i] = full.t[i].A;
      f.insert(f.end(), full.t[i].f.begin(), full.t[i].f.end());
    }
    states.assign(tiles * kLanes, 0);
    words.assign(tiles, 0);
    return genc::rans(c, b, V, tiles, lo, A, f.data(), states.data(), words.data());
  }

  // ---- per-row refinement primitives (device passes; see CpuBackend) ----
  int rdo_alloc(int K) { return genc::cand_alloc(c, K); }
  int rdo_quantize(int k, double sk, int32_t* lo, int32_t* hi, double* num, double* den) {
    int32_t lohi[2 * kTables];
    EP_TRY_G(genc::cand_quantize(c, k, sk, lohi));
    for (int t = 0; t < kTables; t++) {
      lo[t] = t ? lohi[2 * t] : std::numeric_limits<int32_t>::max();
      hi[t] = t ? lohi[2 * t + 1] : std::numeric_limits<int32_t>::min();
    }
    return genc::cand_refit(c, k, num, den);
  }
  int rdo_distortion(int k, const float* sig, double* D) { return genc::cand_distortion(c, k, sig, D); }
  int rdo_rate(int k, const double* lq, const int32_t* lo, const int32_t* A, double* Rt) {
    return genc::cand_rate(c, k, lq, lo, A, Rt);
  }
  int rdo_select(const int32_t* sel, int32_t* lo, int32_t* hi) {
    int32_t lohi[2 * kTables];
    EP_TRY_G(genc::cand_select(c, sel, lohi));
    for (int t = 0; t < kTables; t++) {
      lo[t] = t ? lohi[2 * t] : std::numeric_limits<int32_t>::max();
      hi[t] = t ? lohi[2 * t + 1] : std::numeric_limits<int32_t>::min();
    }
    return EP_OK;
  }
  int rdo_counts(int k, const int32_t* lo, const int32_t* A, uint64_t* n) {
    return genc::cand_count(c, k, lo, A, n);
  }

  int payload(uint8_t* dst, const std::vector<uint32_t>& offs) {
    const uint64_t tiles = offs.size() - 1;
    return genc::payload(c, offs.data(), tiles, offs[tiles], dst);
  }

  int errors(const std::vector<float>& sigma, int rdt, int, std::vector<double>& acc) {
    acc.assign((size_t)R * 4, 0.0);
    return genc::errors(c, sigma.data(), rdt, acc.data());
  }
};

// Per-row rate-distortion refinement (Section 3.5, eqs. rdo_rate, rdo_budget,
// rdo_choice; App. C.2, Alg. rdo) of the full field set at baseline (s, b),
// over a backend's bulk passes: candidates at rho_k s (rho_0 = 1, then
// log-midpoints of the widest gap of {0.70, ratios so far, 1.45}), each row
// refit; D_{r,k} the squared error with the stored FP32 scale; a candidate
// joins only if every table's index range, joined with those already
// admitted, stays within 2^b; the shared model adds 1/2 to each count over
// those joined ranges; B and B_mix are eq. estimate with the b-bit tables of
// the baseline and of the mixture; the lambda bracket starts at
// 2^-20 sum D / sum R and doubles.  Every sum runs in the order of the oracle's
// definition.  On return the backend's full field set, `full` (b-bit) and
// sigma are those of the selected candidates.
template <class BK>
int rdo_run(BK& E, int64_t R, int64_t cvec, const std::vector<double>& mu, double s, int b,
            uint32_t V, double kappa, int cont, int K, int sweeps, std::vector<float>& sigma,
            Model& full, uint32_t& moved) {
  if (K > 64) return fail(EP_ERR_ARG, "ep_encode: at most 64 refinement candidates");
  const int64_t nvec = R * cvec;
  std::vector<double> rho((size_t)K);
  {
    std::vector<double> pts = {std::log(0.70), 0.0, std::log(1.45)};
    rho[0] = 1.0;
    for (int k = 1; k < K; k++) {
      size_t g = 0;
      for (size_t i = 1; i + 1 < pts.size(); i++)
        if (pts[i + 1] - pts[i] > pts[g + 1] - pts[g]) g = i;
      double mid = 0.5 * (pts[g] + pts[g + 1]);
      pts.insert(pts.begin() + (long)g + 1, mid);
      rho[k] = std::exp(mid);
    }
  }
  EP_TRY_G(E.rdo_alloc(K));
  std::vector<float> csig((size_t)(R * K)), sk_sig((size_t)R);
  std::vector<double> D((size_t)(R * K)), Rt((size_t)(R * K), 0.0), col((size_t)R);
  std::vector<double> num((size_t)R), den((size_t)R);
  std::vector<std::array<int32_t, kTables>> clo((size_t)K), chi((size_t)K);
  for (int k = 0; k < K; k++) {
    const double sk = rho[k] * s;
    EP_TRY_G(E.rdo_quantize(k, sk, clo[k].data(), chi[k].data(), num.data(), den.data()));
    for (int64_t r = 0; r < R; r++) {
      double sg = den[r] > 0 ? (num[r] / den[r] < kEta ? kEta : num[r] / den[r]) : sk * mu[r];
      sk_sig[r] = (float)sg;
      csig[r * K + k] = sk_sig[r];
    }
    EP_TRY_G(E.rdo_distortion(k, sk_sig.data(), col.data()));
    for (int64_t r = 0; r < R; r++) D[r * K + k] = col[r];
  }

  // admission and the joined ranges
  std::vector<char> adm((size_t)K, 0);
  int32_t ulo[kTables], uhi[kTables];
  for (int t = 0; t < kTables; t++) {
    ulo[t] = std::numeric_limits<int32_t>::max();
    uhi[t] = std::numeric_limits<int32_t>::min();
  }
  ulo[0] = 0;
  uhi[0] = 1;
  for (int k = 0; k < K; k++) {
    int32_t lo[kTables], hi[kTables];
    bool fits = true;
    for (int t = 0; t < kTables; t++) {
      lo[t] = std::min(ulo[t], clo[k][t]);
      hi[t] = std::max(uhi[t], chi[k][t]);
      if (t && hi[t] >= lo[t] && (int64_t)hi[t] - lo[t] + 1 > (1 << b)) fits = false;
    }
    if (k == 0 || fits) {
      adm[k] = 1;
      std::copy(lo, lo + kTables, ulo);
      std::copy(hi, hi + kTables, uhi);
    }
  }

  const uint64_t tiles = ((uint64_t)nvec + V - 1) / V;
  // b-bit model of a field set with extents lo/hi (table 0: [0, 1])
  auto model_of = [&](int k, const int32_t* lo, const int32_t* hi, Model& md) {
    int32_t mlo[kTables], mA[kTables];
    uint64_t cells = 0;
    for (int t = 0; t < kTables; t++) {
      const int32_t l = t ? lo[t] : 0, h = t ? hi[t] : 1;
      mlo[t] = h >= l ? l : 0;
      mA[t] = h >= l ? (int32_t)((int64_t)h - l + 1) : 0;
      cells += (uint64_t)mA[t];
    }
    std::vector<uint64_t> n(cells);
    const int rc = E.rdo_counts(k, mlo, mA, n.data());
    if (rc != EP_OK) return rc;
    md = Model();
    uint64_t at = 0;
    for (int t = 0; t < kTables; t++) {
      Table& tb = md.t[t];
      tb.lo = mlo[t];
      tb.A = mA[t];
      tb.n.assign(n.begin() + (long)at, n.begin() + (long)(at + mA[t]));
      tb.f.assign((size_t)mA[t], 0);
      at += (uint64_t)mA[t];
    }
    return (int)EP_OK;
  };
  auto est_bytes = [&](Model& md) {
    for (auto& tb : md.t) quantize_freqs(tb, b);
    return estimated_bits(model_bits(md, b), tiles, kappa, md, (uint64_t)R, cont) / 8.0;
  };
  auto choose = [&](double lambda, std::vector<int32_t>& out) {
    for (int64_t r = 0; r < R; r++) {
      int best = 0;
      double bv = D[r * K] + lambda * Rt[r * K];
      for (int k = 1; k < K; k++) {
        if (!adm[k]) continue;
        double v = D[r * K + k] + lambda * Rt[r * K + k];
        if (v < bv) {
          bv = v;
          best = k;
        }
      }
      out[r] = best;
    }
  };
  auto length = [&](const std::vector<int32_t>& sel) {
    double L = 0;
    for (int64_t r = 0; r < R; r++) L += Rt[r * K + sel[r]];
    return L;
  };

  Model md;
  EP_TRY_G(model_of(0, clo[0].data(), chi[0].data(), md));
  const double B = est_bytes(md);
  std::vector<int32_t> sel((size_t)R, 0), cand((size_t)R), tmp((size_t)R);
  int32_t ulo_t[kTables], uA[kTables];
  uint64_t ucells = 0;
  for (int t = 0; t < kTables; t++) {
    ulo_t[t] = uhi[t] >= ulo[t] ? ulo[t] : 0;
    uA[t] = uhi[t] >= ulo[t] ? (int32_t)((int64_t)uhi[t] - ulo[t] + 1) : 0;
    ucells += (uint64_t)uA[t];
  }
  std::vector<double> lq(ucells);
  for (int sw = 0; sw < sweeps; sw++) {
    int32_t mlo[kTables], mhi[kTables];
    EP_TRY_G(E.rdo_select(sel.data(), mlo, mhi));
    EP_TRY_G(model_of(-1, mlo, mhi, md));
    // shared model: counts of the selection plus 1/2 over the joined ranges
    uint64_t at = 0;
    for (int t = 0; t < kTables; t++) {
      double tot = 0;
      for (int32_t z = 0; z < md.t[t].A; z++) tot += (double)md.t[t].n[z];
      const double A = (double)uA[t];
      for (int32_t z = 0; z < uA[t]; z++) {
        const int32_t v = ulo_t[t] + z;
        const int32_t mz = v - md.t[t].lo;
        const double n = (mz >= 0 && mz < md.t[t].A) ? (double)md.t[t].n[mz] : 0.0;
        lq[at + z] = -std::log2((n + 0.5) / (tot + 0.5 * A));
      }
      at += (uint64_t)uA[t];
    }
    // R_{r,k} (eq. rdo_rate)
    for (int k = 0; k < K; k++) {
      if (!adm[k]) continue;
      EP_TRY_G(E.rdo_rate(k, lq.data(), ulo_t, uA, col.data()));
      for (int64_t r = 0; r < R; r++) Rt[r * K + k] = col[r];
    }
    const double Bmix = est_bytes(md);
    const double budget = length(sel) + 8.0 * (B - Bmix);   // eq. rdo_budget
    choose(0.0, cand);                                       // eq. rdo_choice
    if (length(cand) > budget) {
      double sd = 0, sr = 0;
      for (int64_t r = 0; r < R; r++) {
        sd += D[r * K];
        sr += Rt[r * K];
      }
      double lo = 0, hi = (sd > 0 && sr > 0) ? std::ldexp(sd / sr, -20) : std::ldexp(1.0, -20);
      for (int it = 0; it < 2000; it++) {
        choose(hi, tmp);
        if (length(tmp) <= budget) break;
        hi *= 2.0;
      }
      for (int j = 0; j < 20; j++) {
        double lam = lo == 0 ? hi / 2.0 : std::sqrt(lo * hi);
        choose(lam, tmp);
        if (length(tmp) > budget) {
          lo = lam;
        } else {
          hi = lam;
          cand = tmp;
        }
      }
    }
    sel = cand;
  }

  moved = 0;
  for (int64_t r = 0; r < R; r++) {
    moved += sel[r] != 0;
    sigma[r] = csig[r * K + sel[r]];
  }
  int32_t flo[kTables], fhi[kTables];
  EP_TRY_G(E.rdo_select(sel.data(), flo, fhi));
  EP_TRY_G(model_of(-1, flo, fhi, full));
  for (auto& tb : full.t) quantize_freqs(tb, b);
  return EP_OK;
}

int check_args(const void* w, int w_dtype, int64_t R, int64_t C, const ep_encode_params* prm,
               ep_blob* out) {
  if (!w || !prm || !out) return fail(EP_ERR_ARG, "ep_encode: null argument");
  out->data = nullptr;
  out->size = 0;
  if (R <= 0 || C <= 0 || C % 8) return fail(EP_ERR_ARG, "ep_encode: need R, C > 0 and C % 8 == 0");
  if (w_dtype != EP_BF16 && w_dtype != EP_FP16 && w_dtype != EP_FP32)
    return fail(EP_ERR_ARG, "ep_encode: input dtype must be BF16, FP16 or FP32");
  if (!(prm->target_bpp > 0) || prm->tile_vectors < 1 || prm->search_steps < 0 ||
      prm->container < 0 || prm->container > 4 || !(prm->scale_lo > 0) ||
      !(prm->scale_hi > prm->scale_lo) || prm->sample_vectors < 1 ||
      (prm->prob_bits && (prm->prob_bits < 9 || prm->prob_bits > 15)) ||
      prm->rdo_candidates > 64 || prm->rdo_sweeps < 0)
    return fail(EP_ERR_ARG, "ep_encode: invalid parameters");
  if (R > 0xFFFFFFFFll || C > 0xFFFFFFFFll || (R * C) / 8 > 0xFFFFFFFFll)
    return fail(EP_ERR_ARG, "ep_encode: tensor too large");
  return EP_OK;
}


template <class BK>
int encode_impl(BK& E, int w_dtype, int64_t R, int64_t C, const ep_encode_params* prm,
                ep_blob* out, ep_encode_stats* stats) {
  const int64_t N = R * C, nvec = N / 8;
  const int cont = prm->container;
  const uint32_t V = (uint32_t)prm->tile_vectors;

  // input values, container route, row RMS (Section 3.2; App. A.6, B.1)
  EP_TRY_G(E.prep(cont));

  // scale search on a fixed row sample (Alg. rate selection; App. C.1)
  std::vector<int64_t> srows = pick_rows(R, C, prm->sample_vectors);
  const bool sample_all = (int64_t)srows.size() == R;
  const int64_t snv = (int64_t)srows.size() * (C / 8);
  const uint64_t stiles = ((uint64_t)snv + V - 1) / V;
  const double nsub = (double)((int64_t)srows.size() * C);
  std::vector<double> num((size_t)R), den((size_t)R);

  const int b_first = prm->prob_bits ? prm->prob_bits : (prm->target_bpp <= 7.0 ? 11 : 12);
  int b = b_first;
  double s = 1.0, rhat = 0;
  uint32_t escal = 0, coarse = 0;
  bool fits = false;
  Model full;
  for (; b <= 15 && !fits; b++) {
    double lo = prm->scale_lo, hi = prm->scale_hi;
    for (int it = 0; it < prm->search_steps; it++) {
      s = std::sqrt(lo * hi);
      Model sm;
      EP_TRY_G(E.quantize(sample_all ? nullptr : &srows, s, sm, 1 << b, nullptr, nullptr));
      if (sm.max_field_alphabet() > (1 << b)) {
        rhat = std::numeric_limits<double>::infinity();
      } else {
        for (auto& tb : sm.t) quantize_freqs(tb, b);
        rhat = estimated_bits(model_bits(sm, b), stiles, prm->state_credit_bits, sm,
                              srows.size(), cont) / nsub;
      }
      if (rhat > prm->target_bpp) lo = s;
      else hi = s;
    }
    s = std::sqrt(lo * hi);
    EP_TRY_G(E.quantize(nullptr, s, full, 1 << b, num.data(), den.data()));
    fits = full.max_field_alphabet() <= (1 << b);
    if (!fits) escal++;
  }
  if (fits) b--;  // the loop advanced past the accepted precision
  else {
    b = 15;
    while (full.max_field_alphabet() > (1 << b)) {
      s = 1.05 * s * (double)full.max_field_alphabet() / (double)(1 << b);
      EP_TRY_G(E.quantize(nullptr, s, full, 1 << b, num.data(), den.data()));
      coarse++;
    }
  }
  for (auto& tb : full.t) quantize_freqs(tb, b);

  // row reconstruction scales (eq. scale_fit)
  std::vector<float> sigma((size_t)R);
  for (int64_t r = 0; r < R; r++) {
    double sg;
    if (den[r] > 0) {
      sg = num[r] / den[r];
      if (sg < kEta) sg = kEta;
    } else {
      sg = s * E.mu[r];
    }
    sigma[r] = (float)sg;
  }

  // optional per-row refinement (Section 3.5; App. C.2); the tables follow the new fields
  uint32_t moved = 0;
  if (prm->rdo_candidates > 1 && prm->rdo_sweeps > 0) {
    EP_TRY_G(rdo_run(E, R, C / 8, E.mu, s, b, V, prm->state_credit_bits, cont, prm->rdo_candidates,
                   prm->rdo_sweeps, sigma, full, moved));
  }

  // interleaved rANS per tile (eq. rans_encode; App. C.3)
  const uint64_t tiles = ((uint64_t)nvec + V - 1) / V;
  std::vector<uint32_t> states;
  std::vector<uint64_t> tw;
  EP_TRY_G(E.rans(full, b, V, tiles, states, tw));
  uint64_t words = 0;
  std::vector<uint32_t> offs(tiles + 1);
  for (uint64_t t = 0; t < tiles; t++) {
    offs[t] = (uint32_t)words;
    words += tw[t];
    if (words > 0xFFFFFFFFull) return fail(EP_ERR_UNSUPPORTED, "ep_encode: payload too large");
  }
  offs[tiles] = (uint32_t)words;

  // serialise
  Layout L = layout_of((uint32_t)R, (uint32_t)full.serialized_bytes(), (uint32_t)tiles,
                       (uint32_t)cont, (uint32_t)words);
  uint8_t* blob = static_cast<uint8_t*>(std::calloc((size_t)L.total, 1));
  if (!blob) return fail(EP_ERR_NOMEM, "ep_encode: out of host memory");
  auto w32 = [&](uint64_t off, uint32_t v) { std::memcpy(blob + off, &v, 4); };
  w32(0, kMagic);
  w32(4, kVersion);
  w32(8, (uint32_t)R);
  w32(12, (uint32_t)C);
  w32(16, (uint32_t)b);
  w32(20, V);
  w32(24, (uint32_t)tiles);
  w32(28, (uint32_t)cont);
  w32(32, (uint32_t)full.serialized_bytes());
  w32(36, (uint32_t)words);
  std::memcpy(blob + 40, &L.total, 8);
  uint8_t* q = blob + L.off_tables;
  uint16_t cf[2] = {(uint16_t)full.t[0].f[0], (uint16_t)full.t[0].f[1]};
  std::memcpy(q, cf, 4);
  q += 4;
  for (int i = 1; i < kTables; i++) {
    const Table& tb = full.t[i];
    std::memcpy(q, &tb.lo, 4);
    uint32_t A = (uint32_t)tb.A;
    std::memcpy(q + 4, &A, 4);
    for (int32_t z = 0; z < tb.A; z++) {
      uint16_t v = (uint16_t)tb.f[z];
      std::memcpy(q + 8 + 2 * z, &v, 2);
    }
    q += 8 + ((2ull * A + 3) / 4) * 4;
  }
  std::memcpy(blob + L.off_sigma, sigma.data(), 4 * (size_t)R);
  if (cont) std::memcpy(blob + L.off_delta, E.delta.data(), 4 * (size_t)R);
  std::memcpy(blob + L.off_states, states.data(), 4 * states.size());
  std::memcpy(blob + L.off_offsets, offs.data(), 4 * offs.size());
  int rc = E.payload(blob + L.off_payload, offs);
  if (rc != EP_OK) {
    std::free(blob);
    return rc;
  }

  if (stats) {
    // reconstruction error in the dtype of the coded values
    int rdt = em::container_dtype(cont, w_dtype);
    std::vector<double> acc;
    rc = E.errors(sigma, rdt, cont, acc);
    if (rc != EP_OK) {
      std::free(blob);
      return rc;
    }
    double ec = 0, rc2 = 0, eo = 0, ro = 0, sb = 0;
    for (int64_t r = 0; r < R; r++) {
      ec += acc[4 * r];
      rc2 += acc[4 * r + 1];
      eo += acc[4 * r + 2];
      ro += acc[4 * r + 3];
    }
    // sum over a tile's lanes of log2(x / 2^15), as the log of the product: each
    // factor lies in [1, 2^16), so 32 of them stay below 2^512
    for (uint64_t t = 0; t < tiles; t++) {
      double prod = 1.0;
      for (uint32_t l = 0; l < kLanes; l++) prod *= (double)states[t * kLanes + l] / (double)kStateLow;
      sb += std::log2(prod);
    }
    stats->scale = s;
    stats->rate_estimate_sample = rhat;
    stats->rate_stored = 8.0 * (double)L.total / (double)N;
    stats->code_length_bits = model_bits(full, b);
    stats->erel_coded = rc2 > 0 ? std::sqrt(ec / rc2) : 0;
    stats->erel_original = ro > 0 ? std::sqrt(eo / ro) : 0;
    stats->mean_state_bits = sb / (double)(tiles * kLanes);
    stats->bytes = L.total;
    stats->payload_bits = 16ull * words;
    stats->prob_bits = (uint32_t)b;
    stats->n_tiles = (uint32_t)tiles;
    stats->max_alphabet = (uint32_t)full.max_field_alphabet();
    stats->sample_rows = (uint32_t)srows.size();
    stats->escalations = escal;
    stats->coarsenings = coarse;
    stats->rdo_rows_moved = moved;
  }
  out->data = blob;
  out->size = L.total;
  return EP_OK;
}

}  // namespace

int encode_cpu(const void* w, int w_dtype, int64_t R, int64_t C, const ep_encode_params* prm,
               ep_blob* out, ep_encode_stats* stats) {
  EP_TRY_G(check_args(w, w_dtype, R, C, prm, out));
  try {
    CpuBackend E;
    E.w = w;
    E.dt = w_dtype;
    E.R = R;
    E.C = C;
    E.cvec = C / 8;
    int hw = (int)std::thread::hardware_concurrency();
    E.T = prm->nthreads > 0 ? prm->nthreads : std::max(1, hw);
    return encode_impl(E, w_dtype, R, C, prm, out, stats);
  } catch (const std::bad_alloc&) {
    return fail(EP_ERR_NOMEM, "ep_encode_cpu: out of host memory");
  }
}

int encode_gpu(const void* d_w, int w_dtype, int64_t R, int64_t C, const ep_encode_params* prm,
               ep_blob* out, ep_encode_stats* stats, void* stream) {
  EP_TRY_G(check_args(d_w, w_dtype, R, C, prm, out));
  try {
    GpuBackend E;
    E.R = R;
    EP_TRY_G(genc::open(&E.c, d_w, w_dtype, R, C, prm->container, stream));
    return encode_impl(E, w_dtype, R, C, prm, out, stats);
  } catch (const std::bad_alloc&) {
    return fail(EP_ERR_NOMEM, "ep_encode_gpu: out of host memory");
  }
}

}  // namespace ep

extern "C" {

void ep_encode_params_default(ep_encode_params* p) {
  if (!p) return;
  std::memset(p, 0, sizeof(*p));
  p->target_bpp = 4.0;
  p->tile_vectors = 512;
  p->prob_bits = 0;
  p->search_steps = 12;
  p->container = EP_CONT_DIRECT;
  p->scale_lo = 1e-3;
  p->scale_hi = 8.0;
  p->sample_vectors = 1 << 18;
  p->state_credit_bits = 8.0;
  p->nthreads = 0;
}

int ep_encode_cpu(const void* w, int w_dtype, int64_t rows, int64_t cols,
                  const ep_encode_params* params, ep_blob* out, ep_encode_stats* stats) {
  return ep::encode_cpu(w, w_dtype, rows, cols, params, out, stats);
}

int ep_encode_gpu(const void* d_w, int w_dtype, int64_t rows, int64_t cols,
                  const ep_encode_params* params, ep_blob* out, ep_encode_stats* stats,
                  void* hip_stream) {
  return ep::encode_gpu(d_w, w_dtype, rows, cols, params, out, stats, hip_stream);
}

void ep_blob_free(ep_blob* blob) {
  if (!blob) return;
  std::free(blob->data);
  blob->data = nullptr;
  blob->size = 0;
}

}  // extern "C"
