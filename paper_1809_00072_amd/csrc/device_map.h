// W -> G of one device (RxNN Sec. V-A, model generator steps 1 and 2): tiling
// with zero padding, the differential / bit-sliced mapping of the weight, the
// device characteristic and the device's variation factor.  Shared by the
// G' builds (nested dissection and row sweep).
#pragma once

#include "common.h"

namespace rxnn {

// Philox-4x64 with 10 rounds (Salmon, Moraes, Dror and Shaw, "Parallel random
// numbers: as easy as 1, 2, 3", SC 2011): counter (c0..c3), key (k0, k1).
__device__ __forceinline__ void philox4x64_10(uint64_t& c0, uint64_t& c1, uint64_t& c2,
                                              uint64_t& c3, uint64_t k0, uint64_t k1) {
  constexpr uint64_t kM0 = 0xD2E7470EE14C6C93ull, kM1 = 0xCA5A826395121157ull;
  constexpr uint64_t kW0 = 0x9E3779B97F4A7C15ull, kW1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int rnd = 0; rnd < 10; ++rnd) {
    if (rnd) {
      k0 += kW0;
      k1 += kW1;
    }
    const uint64_t hi0 = __umul64hi(kM0, c0), lo0 = kM0 * c0;
    const uint64_t hi1 = __umul64hi(kM1, c2), lo1 = kM1 * c2;
    const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
}

// Generated variation factor of device d: max(0, 1 + sigma z), z from
// Box-Muller on the first two Philox words of counter (d, 0, 0, 0) under key
// (seed, 0): u1 = ((x0 >> 11) + 1) 2^-53 in (0, 1], u2 = (x1 >> 11) 2^-53.
__device__ __forceinline__ double generated_factor(uint64_t d, uint64_t seed, double sigma) {
  uint64_t c0 = d, c1 = 0, c2 = 0, c3 = 0;
  philox4x64_10(c0, c1, c2, c3, seed, 0);
  const double u1 = ((double)(c0 >> 11) + 1.0) * 0x1.0p-53;
  const double u2 = (double)(c1 >> 11) * 0x1.0p-53;
  const double z = sqrt(-2.0 * log(u1)) * cos(2.0 * M_PI * u2);
  return fmax(0.0, 1.0 + sigma * z);
}

// Device characteristic: linear interpolation of the table (n samples at
// levels k / (n - 1)) at level u, clamped to [0, 1].
__device__ __forceinline__ double characteristic(const double* lut, int n, double u) {
  const double pos = fmin(fmax(u, 0.0), 1.0) * (double)(n - 1);
  const int k = min((int)floor(pos), n - 2);
  const double t = pos - (double)k;
  return lut[k] + t * (lut[k + 1] - lut[k]);
}

// Conductance of device (i, j) of array `arr` = (c R + r) A + a of the layer
// (tile row r, tile column c, array a = 2 slice + side).
__device__ __forceinline__ double device_g(const MapScalars& ms, const float* W, double wmax,
                                           int64_t arr, int i, int j) {
  const int a = (int)(arr % ms.A);
  const int64_t rc = arr / ms.A;
  const int r = (int)(rc % ms.R), c = (int)(rc / ms.R);
  const int64_t p = (int64_t)r * ms.M + i, q = (int64_t)c * ms.N + j;
  const float wf = (p < ms.P && q < ms.Q) ? W[p * ms.Q + q] : 0.0f;
  const double w = (double)wf;
  const int side = a & 1, s = a >> 1;
  const double range = ms.g_max - ms.g_min;
  double G;
  if (ms.slice_bits == 0) {
    const double mag = side ? fmax(-w, 0.0) : fmax(w, 0.0);
    if (!(wmax > 0.0)) G = ms.g_min;
    else if (!ms.lut) G = ms.g_min + (range / wmax) * mag;
    else G = ms.g_min + range * characteristic(ms.lut, ms.lut_n, fmin(mag / wmax, 1.0));
  } else {
    const int levels = (1 << ms.slice_bits) - 1;
    const double lw = (double)((1 << ms.weight_bits) - 1);
    double qv = 0.0;
    if (wmax > 0.0) qv = fmin(lw, rint(fabs(w) * (lw / wmax)));
    const int64_t qi = (int64_t)qv;
    const int64_t d = (qi >> (ms.slice_bits * s)) & levels;
    const bool on = side ? (wf < 0.0f) : (wf > 0.0f);
    if (!on) G = ms.g_min;
    else if (!ms.lut) G = ms.g_min + (double)d * (range / (double)levels);
    else G = ms.g_min + range * characteristic(ms.lut, ms.lut_n, (double)d / (double)levels);
  }
  const int64_t dev = arr * ((int64_t)ms.M * ms.N) + (int64_t)i * ms.N + j;
  if (ms.vf) G *= (double)ms.vf[dev];
  else if (ms.vf_sigma > 0.0) G *= generated_factor((uint64_t)dev, ms.vf_seed, ms.vf_sigma);
  return G;
}

}  // namespace rxnn
