// Element-wise mathematics of the learnable modulation and the softened
// ternarisation (Sec. 2.2-2.3, Eq. 2-6), shared by the LM+ST kernels and by
// the weight-gradient GEMM's fused factor-gradient epilogue.
#pragma once

#include <cmath>

#include "kernels.h"

namespace catq {

// Constants of f at sharpness s (StConst), formed on the host in double.
static inline StConst make_st(double s) {
  StConst c;
  const double l2e = 1.4426950408889634;
  c.c2s = (float)(2.0 * s * l2e);
  c.s4 = (float)(4.0 * s);
  c.s4l = (float)(4.0 * s * l2e);
  c.k2 = (float)(1.0 / std::tanh(s));
  c.sk4 = (float)(2.0 * s / std::tanh(s));
  return c;
}

// 1 - exp(-t) for t >= 0 without cancellation: a degree-7 Taylor polynomial
// below t = 1/4 (truncation < 2e-9 relative), the exponential above it.
__device__ __forceinline__ float one_minus_exp_neg(float t, float t_log2e) {
  if (t < 0.25f) {
    float p = 1.0f / 5040.0f;
    p = fmaf(p, t, -1.0f / 720.0f);
    p = fmaf(p, t, 1.0f / 120.0f);
    p = fmaf(p, t, -1.0f / 24.0f);
    p = fmaf(p, t, 1.0f / 6.0f);
    p = fmaf(p, t, -0.5f);
    p = fmaf(p, t, 1.0f);
    return t * p;
  }
  return 1.0f - __builtin_amdgcn_exp2f(-t_log2e);
}

// Per-group scalars of Eq. 3-4 from fp32 stats and factors.  mu and alpha are
// formed in double (the products of two fp32 values are exact there) and
// rounded once to fp32; Delta likewise.
struct GroupScalars {
  float mu, alpha, alpha_div, delta;
};

__device__ __forceinline__ GroupScalars group_scalars(float mu0, float alpha0, float dmu, float dal,
                                                      float dde, float delta0) {
  GroupScalars g;
  g.mu = (float)((double)mu0 + (double)dmu * (double)alpha0);
  g.alpha = (float)((double)dal * (double)alpha0);
  g.delta = (float)((double)dde * (double)delta0);
  g.alpha_div = fmaxf(g.alpha, 1.17549435e-38f);  // smallest normal: constant groups stay finite
  if (g.alpha != g.alpha) g.alpha_div = g.alpha;  // keep NaN
  return g;
}

// Exact hard decision of Eq. 2 on W_hat = (w - mu)/alpha against Delta,
// without dividing: compare r = w - mu with theta = Delta*alpha in double.
__device__ __forceinline__ float hard_code(float w, float mu, double theta) {
  double r = (double)w - (double)mu;
  return (float)((r > theta) - (r < -theta));
}

// The same decision with a float32 screen.  With r = w - mu and
// theta = Delta*alpha exact, r32 = fl(r) and b = fl(Delta*alpha) each carry a
// relative error of at most 2^-24 (a difference of floats that falls below
// the normal range is exact), so |r32| > b (1 + 2^-21) proves |r| > theta
// and |r32| < b (1 - 2^-21) proves |r| < theta; only the band between them,
// and thresholds outside [2^-120, 2^120] (zero, negative, NaN, huge), go to
// the exact float64 comparison.
struct HardThresh {
  double theta;
  float hi, lo;
};
__device__ __forceinline__ HardThresh hard_thresh(float delta, float alpha_div) {
  HardThresh t;
  t.theta = (double)delta * (double)alpha_div;
  const float b = delta * alpha_div;
  const bool ok = b >= 0x1p-120f && b <= 0x1p+120f;  // false for NaN
  t.hi = ok ? b * (1.0f + 0x1p-21f) : __builtin_inff();
  t.lo = ok ? b * (1.0f - 0x1p-21f) : -1.0f;
  return t;
}
// Codes of N weights of one group: the screen for all N, and the exact
// comparison for all N when any of them falls in the band (rare; one branch).
template <int N>
__device__ __forceinline__ void hard_codes_n(const float (&w)[N], float mu, const HardThresh& t,
                                             float (&c)[N]) {
  bool band = false;
#pragma unroll
  for (int j = 0; j < N; ++j) {
    const float r = w[j] - mu;
    const float a = fabsf(r);
    c[j] = a > t.hi ? copysignf(1.0f, r) : 0.0f;
    band |= !(a > t.hi) && !(a < t.lo);
  }
  if (band) {
#pragma unroll
    for (int j = 0; j < N; ++j) c[j] = hard_code(w[j], mu, t.theta);
  }
}
__device__ __forceinline__ void hard_codes8(const float (&w)[8], float mu, const HardThresh& t,
                                            float (&c)[8]) {
  hard_codes_n<8>(w, mu, t, c);
}

// Transition function f of Eq. 5 at x_hat (cancellation-free form).
__device__ __forceinline__ float transition_f(float xs, float delta, float ED, const StConst& c) {
  float x = fabsf(xs);
  float d = x - delta;
  float qa = __builtin_amdgcn_exp2f(-fabsf(d) * c.c2s);
  float E = one_minus_exp_neg(x * c.s4, x * c.s4l);
  bool ge = d >= 0.0f;
  float eb = ge ? ED : E;
  float qb = fmaf(-qa, eb, qa);
  float den = (1.0f + qa) * (1.0f + qb);
  float num = ge ? E : qa * E;
  float F = num * __builtin_amdgcn_rcpf(den) * c.k2;
  return copysignf(F, xs);
}

// f, f_W and f_Delta together (backward).
__device__ __forceinline__ void transition_parts(float xs, float delta, float ED, const StConst& c,
                                                 float& f, float& fW, float& fD) {
  float x = fabsf(xs);
  float d = x - delta;
  float qa = __builtin_amdgcn_exp2f(-fabsf(d) * c.c2s);
  float E = one_minus_exp_neg(x * c.s4, x * c.s4l);
  bool ge = d >= 0.0f;
  float eb = ge ? ED : E;
  float qb = fmaf(-qa, eb, qa);
  float ra = __builtin_amdgcn_rcpf(1.0f + qa);
  float rb = __builtin_amdgcn_rcpf(1.0f + qb);
  float num = ge ? E : qa * E;
  f = copysignf(num * ra * rb * c.k2, xs);
  float ra2 = ra * ra, rb2 = rb * rb;
  fW = c.sk4 * fmaf(qa, ra2, qb * rb2);
  float om = ge ? E : ED;  // 1 - qa*qb
  fD = copysignf(c.sk4 * (qa * eb) * om * (ra2 * rb2), -xs);
  if (xs == 0.0f) fD = 0.0f;
}

}  // namespace catq
