// Per-value and per-vector arithmetic of the encoder, shared by the CPU
// encoder (g++) and the GPU encoder's kernels (hipcc), so that both run the
// same IEEE double sequence and produce the same blob.  Both are compiled
// with floating-point contraction off.
#pragma once
#include <cmath>
#include <cstdint>

#include "../../include/entropack.h"

#if defined(__HIPCC__)
#define EP_HD __host__ __device__
#else
#define EP_HD
#endif

namespace ep {
namespace em {

constexpr double kEta = 1e-12;   // floor of the row RMS and of refitted scales

// Round-half-even of v onto a binary float format with `frac` fraction bits,
// minimum normal exponent emin and largest finite value vmax (saturating).
EP_HD inline double round_to_format(double v, int frac, int emin, double vmax) {
  if (v == 0.0) return v;
  double mag = std::fabs(v);
  int ex = std::ilogb(mag);   // mag in [2^ex, 2^(ex+1))
  if (ex < emin) ex = emin;
  double ulp = std::ldexp(1.0, ex - frac);
  double q = std::nearbyint(mag / ulp) * ulp;
  if (q > vmax) q = vmax;
  return std::signbit(v) ? -q : q;
}

EP_HD inline double to_e4m3(double v) { return round_to_format(v, 3, -6, 448.0); }
EP_HD inline double to_e5m2(double v) { return round_to_format(v, 2, -14, 57344.0); }

// Largest magnitude of a row container (delta_r = amax_r / qmax) and the
// rounding of a quotient W / delta_r into it.
EP_HD inline double container_max(int cont) {
  return cont == EP_CONT_FP8_ROW ? 448.0 : cont == EP_CONT_FP8E5M2_ROW ? 57344.0 : 127.0;
}
EP_HD inline double container_snap(int cont, double q) {
  if (cont == EP_CONT_FP8_ROW) return to_e4m3(q);
  if (cont == EP_CONT_FP8E5M2_ROW) return to_e5m2(q);
  const double r = std::nearbyint(q);
  return (r > 127.0 ? 127.0 : (r < -127.0 ? -127.0 : r)) + (cont == EP_CONT_UINT8_TENSOR ? 128.0 : 0.0);
}
// Offset of a container's values (the unsigned container's 128; 0 otherwise).
EP_HD inline double container_offset(int cont) { return cont == EP_CONT_UINT8_TENSOR ? 128.0 : 0.0; }
// Output type in which a container's values are reconstructed.
EP_HD inline int container_dtype(int cont, int direct) {
  return cont == EP_CONT_FP8_ROW ? EP_FP8_E4M3 : cont == EP_CONT_FP8E5M2_ROW ? EP_FP8_E5M2
         : cont == EP_CONT_INT8_ROW ? EP_INT8 : cont == EP_CONT_UINT8_TENSOR ? EP_UINT8 : direct;
}
EP_HD inline double to_bf16(double v) { return round_to_format(v, 7, -126, 3.3895313892515355e38); }
EP_HD inline double to_fp16(double v) { return round_to_format(v, 10, -14, 65504.0); }

EP_HD inline double int8_snap(double v) {
  double r = std::nearbyint(v);
  return r > 127 ? 127 : (r < -128 ? -128 : r);
}

// y snapped to output type dt (FP32 and others: y itself).
EP_HD inline double snap_out(int dt, double y) {
  if (dt == EP_UINT8) {
    const double r = std::nearbyint(y);
    return r > 255 ? 255 : (r < 0 ? 0 : r);
  }
  return dt == EP_BF16 ? to_bf16(y) : dt == EP_FP16 ? to_fp16(y) : dt == EP_FP8_E4M3 ? to_e4m3(y)
         : dt == EP_FP8_E5M2 ? to_e5m2(y) : dt == EP_INT8 ? int8_snap(y) : y;
}

// Nearest point of D8: coordinate rounding (ties to even), then, if the sum is
// odd, the coordinate with the largest residual (first on ties) moves by one
// towards its input (a zero residual moves up).  Section 3.2, eq. d8.
EP_HD inline void d8_point(const double* y, double* z) {
  double r[8], tot = 0;
  for (int j = 0; j < 8; j++) {
    z[j] = std::nearbyint(y[j]);
    r[j] = y[j] - z[j];
    tot += z[j];
  }
  if (std::fmod(std::fabs(tot), 2.0) == 1.0) {
    int k = 0;
    double best = std::fabs(r[0]);
    for (int j = 1; j < 8; j++) {
      double a = std::fabs(r[j]);
      if (a > best) {
        best = a;
        k = j;
      }
    }
    z[k] += r[k] < 0 ? -1.0 : 1.0;
  }
}

EP_HD inline double sqdist(const double* y, const double* p) {
  double s = 0;
  for (int j = 0; j < 8; j++) s += (y[j] - p[j]) * (y[j] - p[j]);
  return s;
}

// Nearest E8 point as doubled coordinates; the shifted coset replaces the D8
// candidate only when strictly closer.
EP_HD inline void e8_point(const double* y, int32_t* p2) {
  double a[8], h[8], yh[8];
  d8_point(y, a);
  for (int j = 0; j < 8; j++) yh[j] = y[j] - 0.5;
  d8_point(yh, h);
  for (int j = 0; j < 8; j++) h[j] += 0.5;
  const double* win = sqdist(y, h) < sqdist(y, a) ? h : a;
  for (int j = 0; j < 8; j++) p2[j] = (int32_t)(2.0 * win[j]);
}

// Field tuple (c, z1..z7, m) of a doubled point (eq. parity).
EP_HD inline void split_fields(const int32_t* p2, int32_t* f) {
  int32_t c = p2[0] & 1, par = 0;
  for (int j = 0; j < 7; j++) {
    f[1 + j] = (p2[j] - c) >> 1;
    par += f[1 + j];
  }
  f[0] = c;
  int32_t z8 = (p2[7] - c) >> 1;
  f[8] = (z8 - (par & 1)) >> 1;
}

// Doubled point of a field tuple (inverse of split_fields, eq. point_inverse).
EP_HD inline void join_fields(const int32_t* f, int32_t* p2) {
  int32_t par = 0;
  for (int j = 0; j < 7; j++) {
    par += f[1 + j];
    p2[j] = 2 * f[1 + j] + f[0];
  }
  p2[7] = 2 * (2 * f[8] + (par & 1)) + f[0];
}

// Model table of field `field` (0 = coset) under coset c: 0, or 1 + 8c + field - 1.
EP_HD inline int table_index(int field, int c) { return field == 0 ? 0 : 1 + 8 * c + field - 1; }

}  // namespace em
}  // namespace ep
