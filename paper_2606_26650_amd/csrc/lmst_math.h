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

// The softened ternarisation of one group in the base-2 exponent domain.
// With z = (w - mu) * sc = 2 s W_hat log2(e), y = |z| and x = |W_hat|:
//   q_a = e^{-2 s |x - Delta|} = 2^{-|y - dz|},   e^{-4 s x} = 2^{-2 y},
//   E = 1 - e^{-4 s x},  q_b = q_a (1 - E) (x < Delta) or q_a (1 - E_Delta),
//   alpha f = copysign(num / ((1 + q_a)(1 + q_b)), z) * alpha / tanh(s),
//   num = E (x >= Delta) or q_a E (x < Delta)
// (the cancellation-free form of Eq. 5; the scalings of the exponents and of
// the output are folded into per-group constants).
struct SoftGroup {
  float mu;     // mu of Eq. 3
  float sc;     // 2 s log2(e) / alpha:  z = (w - mu) * sc
  float inv_a;  // 1 / alpha  (when sc does not fit a float)
  float c2s;    // 2 s log2(e)
  float dz;     // 2 s Delta log2(e)
  float ed;     // E_Delta = 1 - e^{-4 s Delta}
  float ak;     // alpha / tanh(s)
  bool fast;    // sc finite: z in one product
};

__device__ __forceinline__ SoftGroup soft_group(const GroupScalars& gs, const StConst& c) {
  SoftGroup q;
  q.mu = gs.mu;
  q.inv_a = __builtin_amdgcn_rcpf(gs.alpha_div);  // 1 ulp; W_hat needs no more
  q.c2s = c.c2s;
  q.sc = q.inv_a * c.c2s;
  q.fast = fabsf(q.sc) <= 3.0e38f;  // false for inf and NaN
  q.dz = gs.delta * c.c2s;
  q.ed = one_minus_exp_neg(gs.delta * c.s4, gs.delta * c.s4l);
  q.ak = gs.alpha * c.k2;
  return q;
}

// 1 - 2^{-2y} (= 1 - e^{-t}, t = 2 y ln 2) for y >= 0 given T = 2^{-2y}:
// below t = 1/8 the series of 1 - e^{-t} to t^5 in powers of y (truncation
// below 5e-8 relative), above it 1 - T (no cancellation: T < 0.89).
__device__ __forceinline__ float one_minus_exp2_neg2(float y, float T) {
  if (y < 0.09016844f) {
    float p = 0.04266738519f;
    p = fmaf(p, y, -0.1538900584f);
    p = fmaf(p, y, 0.4440328777f);
    p = fmaf(p, y, -0.9609060287f);
    p = fmaf(p, y, 1.386294365f);
    return y * p;
  }
  return 1.0f - T;
}

// alpha * f(W_hat; s, Delta) of one weight (Eq. 5 times the group scale).
template <bool FAST>
__device__ __forceinline__ float soft_value(float w, const SoftGroup& q) {
  const float z = FAST ? (w - q.mu) * q.sc : ((w - q.mu) * q.inv_a) * q.c2s;
  const float y = fabsf(z);
  const float d = y - q.dz;
  const float qa = __builtin_amdgcn_exp2f(-fabsf(d));
  const float T = __builtin_amdgcn_exp2f(-(y + y));
  const float E = one_minus_exp2_neg2(y, T);
  const bool ge = d >= 0.0f;
  const float eb = ge ? q.ed : E;
  const float qb = fmaf(-qa, eb, qa);
  const float opa = 1.0f + qa;
  const float den = fmaf(opa, qb, opa);
  const float num = ge ? E : qa * E;
  return copysignf(num * __builtin_amdgcn_rcpf(den), z) * q.ak;
}

template <int N>
__device__ __forceinline__ void soft_values(const float (&w)[N], const SoftGroup& q,
                                            float (&out)[N]) {
  if (q.fast) {
#pragma unroll
    for (int j = 0; j < N; ++j) out[j] = soft_value<true>(w[j], q);
  } else {
#pragma unroll
    for (int j = 0; j < N; ++j) out[j] = soft_value<false>(w[j], q);
  }
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

// f, f_W and f_Delta without their constant factors, in the base-2 exponent
// domain of soft_value: with z = xs * c2s (c2s = 2 s log2 e), y = |z|,
// dz = Delta * c2s and ed = E_Delta,
//   f = k2 * fp,   f_W = sk4 * fwp,   f_Delta = sk4 * fdp,
// 1/(1 + q_a) and 1/(1 + q_b) from one reciprocal of their product.  The
// factor-gradient sums apply k2 and sk4 once per group.
__device__ __forceinline__ void transition_parts_z(float xs, float c2s, float dz, float ed,
                                                   float& fp, float& fwp, float& fdp) {
  const float z = xs * c2s;
  const float y = fabsf(z);
  const float d = y - dz;
  const float qa = __builtin_amdgcn_exp2f(-fabsf(d));
  const float T = __builtin_amdgcn_exp2f(-(y + y));
  const float E = one_minus_exp2_neg2(y, T);
  const bool ge = d >= 0.0f;
  const float eb = ge ? ed : E;
  const float qb = fmaf(-qa, eb, qa);
  const float opa = 1.0f + qa, opb = 1.0f + qb;
  const float rden = __builtin_amdgcn_rcpf(opa * opb);
  const float num = ge ? E : qa * E;
  fp = copysignf(num * rden, xs);
  const float ra = opb * rden, rb = opa * rden;  // 1/(1 + q_a), 1/(1 + q_b)
  fwp = fmaf(qa * ra, ra, (qb * rb) * rb);
  const float om = ge ? E : ed;  // 1 - q_a q_b / ... (see transition_parts)
  fdp = copysignf((qa * eb) * om * (rden * rden), -xs);
}

// The same parts from z itself with E = 1 - 2^(-2|z|) given (the GEMM
// epilogue forms E for a whole pass of weights, taking the series only where
// some lane of the wave needs it), 1/(1 + q_a)^2 and 1/(1 + q_b)^2 as
// (1 + q_b)^2 r^2 and (1 + q_a)^2 r^2 from the one reciprocal r.
__device__ __forceinline__ void transition_parts_zE(float z, float dz, float ed, float E,
                                                    float& fp, float& fwp, float& fdp) {
  const float y = fabsf(z);
  const float d = y - dz;
  const float qa = __builtin_amdgcn_exp2f(-fabsf(d));
  const bool ge = d >= 0.0f;
  const float eb = ge ? ed : E;
  const float qb = fmaf(-qa, eb, qa);
  const float opa = 1.0f + qa, opb = 1.0f + qb;
  const float rden = __builtin_amdgcn_rcpf(opa * opb);
  const float r2 = rden * rden;
  const float num = ge ? E : qa * E;
  fp = copysignf(num * rden, z);
  fwp = fmaf(qa, opb * opb, qb * (opa * opa)) * r2;
  const float om = ge ? E : ed;
  fdp = copysignf((qa * eb) * om * r2, -z);
}

// Scales of the per-group sums of transition_parts_z: f is the hard code
// (HARD, no scale) or k2 fp; f_W is 1 under the straight-through estimator;
// wz turns a sum of g f_W z (z = xs c2s) into that of g f_W xs.
struct FacScale {
  float f, w, d, wz;
};
__device__ __forceinline__ FacScale fac_scale(int mode, int ste, const StConst& c) {
  FacScale k;
  k.f = (mode == CATQ_SOFT) ? c.k2 : 1.0f;
  k.w = ste ? 1.0f : c.sk4;
  k.d = c.sk4;
  k.wz = k.w / c.c2s;
  return k;
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
