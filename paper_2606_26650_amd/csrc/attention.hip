// Causal grouped-query attention of the decoder block (forward and backward),
// built from the matrix-core GEMM plus row kernels (gfx950).
//
//   prep      per (token, head): optional RMSNorm of q and k, rotary embedding,
//             q/k re-laid out head-major [B][H][S][d]
//   scores    S = (1/sqrt d) Q K^T per (batch, q head), tiles above the
//             diagonal skipped                                   (MFMA GEMM)
//   softmax   P = softmax over the causal prefix of each row; zeros written
//             from the diagonal to the next multiple of 256 so that the
//             tiles of the following GEMMs read defined values
//   output    O = P V, contraction cut at the tile diagonal      (MFMA GEMM)
// The backward recomputes nothing: P is kept.  dP = dO V^T, dS = P*(dP - D)/sqrt d
// with D = rowsum(P*dP), dQ = dS K, dK = dS^T Q and dV = P^T dO per q head
// (fp32), and the prep-backward sums the q heads of each kv group, undoes the
// rotation and the q/k RMSNorm and writes d(qkv).
#include <cmath>
#include <cstring>

#include "kernels.h"

namespace catq {

struct AttnLayout {
  int64_t B, S, Hq, Hkv, d, G, ld;  // ld = (Hq + 2 Hkv) d
  bool flash;                        // fused kernels (head_dim 64 or 128)
  int hs;                            // flash dK/dV: q heads of a group split over hs blocks
  // saved buffer (byte offsets)
  size_t o_qh, o_kh, o_vh, o_lse, o_p, o_rstd, o_cos, o_sin, o_sc, saved_total;
  // backward workspace
  size_t o_dp, o_ds, o_dq, o_dk, o_dv, o_dsum, bwd_total;
};

static AttnLayout attn_layout(const catq_attn_desc* a) {
  AttnLayout L;
  L.B = a->batch;
  L.S = a->seq;
  L.Hq = a->n_q;
  L.Hkv = a->n_kv;
  L.d = a->head_dim;
  L.G = L.Hq / (L.Hkv > 0 ? L.Hkv : 1);
  L.ld = (L.Hq + 2 * L.Hkv) * L.d;
  L.flash = (L.d == 64 || L.d == 128);
  // The dK/dV kernel runs one block per (batch, kv head, 128 keys) and loops
  // over the group's q heads; with few kv heads (a high q:kv ratio) that is
  // too few blocks for the chip, so the group's heads are split over hs
  // blocks (the smallest divisor of G giving >= 512 blocks), each writing
  // its own partial dK/dV, summed in chunk order by the q/k backward.
  L.hs = 1;
  if (L.flash) {
    const int64_t nb = L.B * L.Hkv * ((L.S + 127) / 128);
    for (int h = 1; h <= L.G; ++h)
      if (L.G % h == 0) {
        L.hs = h;
        if (nb * h >= 512) break;
      }
  }
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = round_up(off + bytes, 256);
    return o;
  };
  const size_t BHq = (size_t)(L.B * L.Hq), BHk = (size_t)(L.B * L.Hkv),
               SS = (size_t)(L.S * L.S);
  L.o_qh = take(BHq * L.S * L.d * 2);
  L.o_kh = take(BHk * L.S * L.d * 2);
  L.o_rstd = take((size_t)(L.B * L.S) * (L.Hq + L.Hkv) * 4);
  L.o_cos = take((size_t)L.S * (L.d / 2) * 4);
  L.o_sin = take((size_t)L.S * (L.d / 2) * 4);
  if (L.flash) {
    L.o_vh = take(BHk * L.S * L.d * 2);
    L.o_lse = take(BHq * L.S * 4);
    L.o_p = L.o_sc = 0;
  } else {
    L.o_p = take(BHq * SS * 2);
    L.o_sc = take(BHq * SS * 4);
    L.o_vh = L.o_lse = 0;
  }
  L.saved_total = off;
  off = 0;
  if (L.flash) {
    L.o_dsum = take(BHq * L.S * 4);
    L.o_dq = take(BHq * L.S * L.d * 4);
    L.o_dk = take((size_t)L.hs * BHk * L.S * L.d * 4);
    L.o_dv = take((size_t)L.hs * BHk * L.S * L.d * 4);
    L.o_dp = L.o_ds = 0;
  } else {
    L.o_dp = take(BHq * SS * 4);
    L.o_ds = take(BHq * SS * 2);
    L.o_dq = take(BHq * L.S * L.d * 4);
    L.o_dk = take(BHq * L.S * L.d * 4);
    L.o_dv = take(BHq * L.S * L.d * 4);
    L.o_dsum = 0;
  }
  L.bwd_total = off;
  return L;
}

static catq_status check_desc(const catq_attn_desc* a) {
  CATQ_REQUIRE(a != nullptr, CATQ_ERR_NULL, "attention descriptor is NULL");
  CATQ_REQUIRE(a->batch > 0 && a->seq > 0 && a->n_q > 0 && a->n_kv > 0, CATQ_ERR_SHAPE,
               "batch, seq and head counts must be > 0");
  CATQ_REQUIRE(a->n_q % a->n_kv == 0, CATQ_ERR_SHAPE, "n_q must be a multiple of n_kv");
  CATQ_REQUIRE(count_ok((int64_t)a->batch * a->seq, (int64_t)a->n_q + 2 * (int64_t)a->n_kv,
                        a->head_dim > 0 ? a->head_dim : 1) &&
                   count_ok((int64_t)a->batch * a->n_q, a->seq, a->seq),
               CATQ_ERR_SHAPE, "batch, seq and heads too large (more than 2^38 elements)");
  CATQ_REQUIRE(a->head_dim == 64 || a->head_dim == 128 || a->head_dim == 256, CATQ_ERR_SHAPE,
               "head_dim must be 64, 128 or 256");
  CATQ_REQUIRE(a->seq % 8 == 0 && a->seq <= 8192, CATQ_ERR_SHAPE,
               "seq must be a multiple of 8 and <= 8192");
  CATQ_REQUIRE(a->rope_theta > 1.0f && a->eps >= 0.0f, CATQ_ERR_VALUE, "bad rope_theta or eps");
  CATQ_REQUIRE(a->act_quant == 0 || (a->act_quant == 1 && a->head_dim <= 128), CATQ_ERR_VALUE,
               "act_quant must be 0 or 1, and 1 needs head_dim 64 or 128 (fused attention)");
  return CATQ_OK;
}

// ------------------------------------------------------------------ kernels

__global__ __launch_bounds__(256) void rope_table_kernel(int64_t S, int d, double log2_theta,
                                                         float* cs, float* sn) {
  const int half = d / 2;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= S * half) return;
  const int64_t pos = i / half;
  const int f = (int)(i % half);
  const double inv = exp2(-(2.0 * f / d) * log2_theta);
  double s, c;
  sincos((double)pos * inv, &s, &c);
  cs[i] = (float)c;
  sn[i] = (float)s;
}

// One wavefront per (token, head) over the q and k heads.
__global__ __launch_bounds__(256) void qk_prep_fwd_kernel(const bf16* qkv, int64_t B, int64_t S,
                                                          int Hq, int Hkv, int d, int ld,
                                                          int qk_norm, float eps, const float* cs,
                                                          const float* sn, bf16* Qh, bf16* Kh,
                                                          bf16* Vh, float* rstd) {
  const int H = Hq + Hkv;
  const int Hall = Vh ? H + Hkv : H;
  const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (w >= B * S * Hall) return;
  const int64_t t = w / Hall;
  const int h = (int)(w % Hall);
  const int64_t b = t / S, s = t % S;
  const int half = d / 2;
  const bf16* src = qkv + t * ld + (int64_t)h * d;
  if (h >= H) {  // v head: head-major copy
    bf16* dst = Vh + ((b * Hkv + (h - H)) * S + s) * d;
    for (int i = lane; i < d; i += 64) dst[i] = src[i];
    return;
  }
  float x1[2], x2[2];
  const int np = (half + 63) / 64;
  float ss = 0.f;
  for (int p = 0; p < np; ++p) {
    const int i = lane + 64 * p;
    x1[p] = x2[p] = 0.f;
    if (i < half) {
      x1[p] = to_f(src[i]);
      x2[p] = to_f(src[i + half]);
    }
    ss = fmaf(x1[p], x1[p], fmaf(x2[p], x2[p], ss));
  }
  float r = 1.0f;
  if (qk_norm) {
    ss = wave_sum(ss);
    r = 1.0f / sqrtf(ss / (float)d + eps);
  }
  if (lane == 0) rstd[t * H + h] = r;
  bf16* dst = h < Hq ? Qh + ((b * Hq + h) * S + s) * d : Kh + ((b * Hkv + (h - Hq)) * S + s) * d;
  for (int p = 0; p < np; ++p) {
    const int i = lane + 64 * p;
    if (i >= half) continue;
    const float c = cs[s * half + i], sv = sn[s * half + i];
    const float a = x1[p] * r, bb = x2[p] * r;
    dst[i] = (bf16)(a * c - bb * sv);
    dst[i + half] = (bf16)(bb * c + a * sv);
  }
}

// W1.58A8 fake quantization of one (token, head) vector held by LPH lanes
// (16 values each, as stored: bf16): s = max|x|/127, x = bf16(rne(x/s)*s),
// clamped to +-127 codes; the same fp32 steps as catq_aux_act_quant.
__device__ __forceinline__ void head_act_quant(float (&x1)[8], float (&x2)[8], int LPH) {
  float m = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    x1[j] = (float)(bf16)x1[j];
    x2[j] = (float)(bf16)x2[j];
    m = fmaxf(m, fmaxf(fabsf(x1[j]), fabsf(x2[j])));
  }
  for (int k = LPH >> 1; k >= 1; k >>= 1) m = fmaxf(m, __shfl_xor(m, k, 64));
  const float s = m / 127.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    x1[j] = s > 0.f ? fminf(fmaxf(rintf(x1[j] / s), -127.f), 127.f) * s : 0.f;
    x2[j] = s > 0.f ? fminf(fmaxf(rintf(x2[j] / s), -127.f), 127.f) * s : 0.f;
  }
}

// Vectorised q/k preparation for head sizes with half % 8 == 0 and half/8 a
// power of two: LPH = half/8 lanes per (token, head), each lane owning
// elements i0..i0+7 of both rotation halves (two 16-byte loads and stores).
// a8: the stored Q, K and V heads are fake-quantized (W1.58A8).
__global__ __launch_bounds__(256) void qk_prep_fwd_vec_kernel(
    const bf16* qkv, int64_t B, int64_t S, int Hq, int Hkv, int d, int ld, int lph_log2,
    int qk_norm, float eps, const float* cs, const float* sn, bf16* Qh, bf16* Kh, bf16* Vh,
    float* rstd, int a8) {
  const int H = Hq + Hkv;
  const int Hall = Vh ? H + Hkv : H;
  const int LPH = 1 << lph_log2;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t unit = gid >> lph_log2;
  const int sub = (int)(gid & (LPH - 1));
  // whole units only: the grid covers units * LPH threads and LPH divides 64
  if (unit >= B * S * Hall) return;
  const int64_t t = unit / Hall;
  const int h = (int)(unit % Hall);
  const int64_t b = t / S, s = t % S;
  const int half = d / 2, i0 = sub * 8;
  const bf16* src = qkv + t * ld + (int64_t)h * d;
  if (h >= H) {  // v head: head-major copy
    bf16* dst = Vh + ((b * Hkv + (h - H)) * S + s) * d;
    if (a8) {
      float v1[8], v2[8];
      load8<bf16>(src + i0, v1);
      load8<bf16>(src + half + i0, v2);
      head_act_quant(v1, v2, LPH);
      store8<bf16>(dst + i0, v1);
      store8<bf16>(dst + half + i0, v2);
      return;
    }
    *reinterpret_cast<u32x4*>(dst + i0) = *reinterpret_cast<const u32x4*>(src + i0);
    *reinterpret_cast<u32x4*>(dst + half + i0) = *reinterpret_cast<const u32x4*>(src + half + i0);
    return;
  }
  float x1[8], x2[8];
  load8<bf16>(src + i0, x1);
  load8<bf16>(src + half + i0, x2);
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) ss = fmaf(x1[j], x1[j], fmaf(x2[j], x2[j], ss));
  float r = 1.0f;
  if (qk_norm) {
    for (int m = LPH >> 1; m >= 1; m >>= 1) ss += __shfl_xor(ss, m, 64);
    r = 1.0f / sqrtf(ss / (float)d + eps);
  }
  if (sub == 0) rstd[t * H + h] = r;
  float c[8], sv[8];
  load8<float>(cs + s * half + i0, c);
  load8<float>(sn + s * half + i0, sv);
  float o1[8], o2[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float a = x1[j] * r, bb = x2[j] * r;
    o1[j] = a * c[j] - bb * sv[j];
    o2[j] = bb * c[j] + a * sv[j];
  }
  bf16* dst = h < Hq ? Qh + ((b * Hq + h) * S + s) * d : Kh + ((b * Hkv + (h - Hq)) * S + s) * d;
  if (a8) head_act_quant(o1, o2, LPH);
  store8<bf16>(dst + i0, o1);
  store8<bf16>(dst + half + i0, o2);
}

// log2 of the lanes per head of the vectorised q/k kernels, or 0 when the
// layout does not allow them (half % 8, half/8 a power of two up to 64,
// 16-byte aligned rows).
static int qk_vec_lanes(int64_t d, int64_t ld, const void* qkv) {
  const int64_t half = d / 2;
  if (d % 16 != 0 || ld % 8 != 0 || !aligned16(qkv)) return 0;
  const int64_t lanes = half / 8;
  if (lanes < 2 || lanes > 64 || (lanes & (lanes - 1)) != 0) return 0;
  int lg = 0;
  while ((1 << lg) < lanes) ++lg;
  return lg;
}

template <int MAXC>
__global__ __launch_bounds__(256) void softmax_fwd_kernel(const float* Sc, int64_t S, bf16* P) {
  __shared__ float red[4];
  const int64_t row = blockIdx.x;  // (bh, i)
  const int64_t i = row % S;
  const float* src = Sc + row * S;
  bf16* dst = P + row * S;
  float v[MAXC];
  float mx = -INFINITY;
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int64_t j = threadIdx.x + 256 * c;
    v[c] = (j <= i) ? src[j] : -INFINITY;
    mx = fmaxf(mx, v[c]);
  }
  mx = wave_max(mx);
  const int wv = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[wv] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float sum = 0.f;
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int64_t j = threadIdx.x + 256 * c;
    v[c] = (j <= i) ? __expf(v[c] - mx) : 0.f;
    sum += v[c];
  }
  sum = wave_sum(sum);
  if ((threadIdx.x & 63) == 0) red[wv] = sum;
  __syncthreads();
  sum = red[0] + red[1] + red[2] + red[3];
  const float inv = 1.0f / sum;
  const int64_t lim = min(S, (i / 256 + 1) * 256);
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int64_t j = threadIdx.x + 256 * c;
    if (j < lim) dst[j] = (bf16)(v[c] * inv);
  }
}

template <int MAXC>
__global__ __launch_bounds__(256) void softmax_bwd_kernel(const bf16* P, const float* dP,
                                                          int64_t S, float scale, bf16* dS) {
  __shared__ float red[4];
  const int64_t row = blockIdx.x;
  const int64_t i = row % S;
  float p[MAXC], g[MAXC];
  float acc = 0.f;
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int64_t j = threadIdx.x + 256 * c;
    const bool ok = j <= i;
    p[c] = ok ? to_f(P[row * S + j]) : 0.f;
    g[c] = ok ? dP[row * S + j] : 0.f;
    acc = fmaf(p[c], g[c], acc);
  }
  acc = wave_sum(acc);
  const int wv = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[wv] = acc;
  __syncthreads();
  const float D = red[0] + red[1] + red[2] + red[3];
  const int64_t lim = min(S, (i / 256 + 1) * 256);
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int64_t j = threadIdx.x + 256 * c;
    if (j < lim) dS[row * S + j] = (bf16)(scale * p[c] * (g[c] - D));
  }
}

// One wavefront per (token, head) over q, k and v heads of d(qkv).
__global__ __launch_bounds__(256) void qk_prep_bwd_kernel(
    const bf16* qkv, const float* rstd, const float* cs, const float* sn, const float* dQ,
    const float* dKp, const float* dVp, int64_t B, int64_t S, int Hq, int Hkv, int d, int ld,
    int qk_norm, int per_kv, bf16* dqkv) {
  const int H = Hq + 2 * Hkv;
  const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (w >= B * S * H) return;
  const int64_t t = w / H;
  const int h = (int)(w % H);
  const int64_t b = t / S, s = t % S;
  const int half = d / 2;
  const int G = Hq / Hkv;
  const int np = (half + 63) / 64;
  bf16* dst = dqkv + t * ld + (int64_t)h * d;
  if (h >= Hq + Hkv) {  // v heads: sum over the q heads of the group
    const int kv = h - Hq - Hkv;
    for (int i = lane; i < d; i += 64) {
      float acc = 0.f;
      if (per_kv)
        for (int c = 0; c < per_kv; ++c) acc += dVp[(((c * B + b) * Hkv + kv) * S + s) * d + i];
      else
        for (int gq = 0; gq < G; ++gq) acc += dVp[((b * Hq + kv * G + gq) * S + s) * d + i];
      dst[i] = (bf16)acc;
    }
    return;
  }
  float g1[2], g2[2];
  for (int p = 0; p < np; ++p) {
    const int i = lane + 64 * p;
    g1[p] = g2[p] = 0.f;
    if (i >= half) continue;
    if (h < Hq) {
      const float* src = dQ + ((b * Hq + h) * S + s) * d;
      g1[p] = src[i];
      g2[p] = src[i + half];
    } else if (per_kv) {
      for (int c = 0; c < per_kv; ++c) {
        const float* src = dKp + (((c * B + b) * Hkv + (h - Hq)) * S + s) * d;
        g1[p] += src[i];
        g2[p] += src[i + half];
      }
    } else {
      const int kv = h - Hq;
      for (int gq = 0; gq < G; ++gq) {
        const float* src = dKp + ((b * Hq + kv * G + gq) * S + s) * d;
        g1[p] += src[i];
        g2[p] += src[i + half];
      }
    }
    // undo the rotation (transpose of the forward rotation)
    const float c = cs[s * half + i], sv = sn[s * half + i];
    const float a1 = g1[p] * c + g2[p] * sv;
    const float a2 = -g1[p] * sv + g2[p] * c;
    g1[p] = a1;
    g2[p] = a2;
  }
  const bf16* src = qkv + t * ld + (int64_t)h * d;
  if (qk_norm) {
    const float r = rstd[t * (Hq + Hkv) + h];
    float x1[2], x2[2];
    float dot = 0.f;
    for (int p = 0; p < np; ++p) {
      const int i = lane + 64 * p;
      x1[p] = x2[p] = 0.f;
      if (i < half) {
        x1[p] = to_f(src[i]);
        x2[p] = to_f(src[i + half]);
      }
      dot = fmaf(x1[p], g1[p], fmaf(x2[p], g2[p], dot));
    }
    dot = wave_sum(dot);
    const float coef = r * r * r * dot / (float)d;
    for (int p = 0; p < np; ++p) {
      g1[p] = r * g1[p] - x1[p] * coef;
      g2[p] = r * g2[p] - x2[p] * coef;
    }
  }
  for (int p = 0; p < np; ++p) {
    const int i = lane + 64 * p;
    if (i >= half) continue;
    dst[i] = (bf16)g1[p];
    dst[i + half] = (bf16)g2[p];
  }
}

// Vectorised backward of the q/k preparation (same lane layout as the forward).
__global__ __launch_bounds__(256) void qk_prep_bwd_vec_kernel(
    const bf16* qkv, const float* rstd, const float* cs, const float* sn, const float* dQ,
    const float* dKp, const float* dVp, int64_t B, int64_t S, int Hq, int Hkv, int d, int ld,
    int lph_log2, int qk_norm, int per_kv, bf16* dqkv) {
  const int H = Hq + 2 * Hkv;
  const int LPH = 1 << lph_log2;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t unit = gid >> lph_log2;
  const int sub = (int)(gid & (LPH - 1));
  if (unit >= B * S * H) return;
  const int64_t t = unit / H;
  const int h = (int)(unit % H);
  const int64_t b = t / S, s = t % S;
  const int half = d / 2, i0 = sub * 8;
  const int G = Hq / Hkv;
  bf16* dst = dqkv + t * ld + (int64_t)h * d;
  float g1[8], g2[8];
  auto gather = [&](const float* base_of_head0, int64_t head_stride, int nh) {
#pragma unroll
    for (int j = 0; j < 8; ++j) g1[j] = g2[j] = 0.f;
    for (int q = 0; q < nh; ++q) {
      const float* src = base_of_head0 + q * head_stride;
      float a[8], c[8];
      load8<float>(src + i0, a);
      load8<float>(src + half + i0, c);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        g1[j] += a[j];
        g2[j] += c[j];
      }
    }
  };
  if (h >= Hq + Hkv) {  // v heads: sum over the q heads of the group
    const int kv = h - Hq - Hkv;
    if (per_kv)
      gather(dVp + ((b * Hkv + kv) * S + s) * d, B * Hkv * S * d, per_kv);
    else
      gather(dVp + ((b * Hq + kv * G) * S + s) * d, S * d, G);
    store8<bf16>(dst + i0, g1);
    store8<bf16>(dst + half + i0, g2);
    return;
  }
  if (h < Hq)
    gather(dQ + ((b * Hq + h) * S + s) * d, 0, 1);
  else if (per_kv)
    gather(dKp + ((b * Hkv + (h - Hq)) * S + s) * d, B * Hkv * S * d, per_kv);
  else
    gather(dKp + ((b * Hq + (h - Hq) * G) * S + s) * d, S * d, G);
  {
    // undo the rotation (transpose of the forward rotation)
    float c[8], sv[8];
    load8<float>(cs + s * half + i0, c);
    load8<float>(sn + s * half + i0, sv);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float a1 = g1[j] * c[j] + g2[j] * sv[j];
      const float a2 = -g1[j] * sv[j] + g2[j] * c[j];
      g1[j] = a1;
      g2[j] = a2;
    }
  }
  if (qk_norm) {
    const bf16* src = qkv + t * ld + (int64_t)h * d;
    const float r = rstd[t * (Hq + Hkv) + h];
    float x1[8], x2[8];
    load8<bf16>(src + i0, x1);
    load8<bf16>(src + half + i0, x2);
    float dot = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) dot = fmaf(x1[j], g1[j], fmaf(x2[j], g2[j], dot));
    for (int m = LPH >> 1; m >= 1; m >>= 1) dot += __shfl_xor(dot, m, 64);
    const float coef = r * r * r * dot / (float)d;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      g1[j] = r * g1[j] - x1[j] * coef;
      g2[j] = r * g2[j] - x2[j] * coef;
    }
  }
  store8<bf16>(dst + i0, g1);
  store8<bf16>(dst + half + i0, g2);
}

static int row_chunks(int64_t S) {
  const int c = (int)((S + 255) / 256);
  return c <= 2 ? 2 : (c <= 4 ? 4 : (c <= 8 ? 8 : (c <= 16 ? 16 : 32)));
}

static void launch_softmax_fwd(const float* Sc, int64_t S, int64_t rows, bf16* P,
                               hipStream_t stream) {
  dim3 grid((unsigned)rows), block(256);
  switch (row_chunks(S)) {
    case 2: hipLaunchKernelGGL(softmax_fwd_kernel<2>, grid, block, 0, stream, Sc, S, P); break;
    case 4: hipLaunchKernelGGL(softmax_fwd_kernel<4>, grid, block, 0, stream, Sc, S, P); break;
    case 8: hipLaunchKernelGGL(softmax_fwd_kernel<8>, grid, block, 0, stream, Sc, S, P); break;
    case 16: hipLaunchKernelGGL(softmax_fwd_kernel<16>, grid, block, 0, stream, Sc, S, P); break;
    default: hipLaunchKernelGGL(softmax_fwd_kernel<32>, grid, block, 0, stream, Sc, S, P); break;
  }
}

static void launch_softmax_bwd(const bf16* P, const float* dP, int64_t S, int64_t rows,
                               float scale, bf16* dS, hipStream_t stream) {
  dim3 grid((unsigned)rows), block(256);
  switch (row_chunks(S)) {
    case 2: hipLaunchKernelGGL(softmax_bwd_kernel<2>, grid, block, 0, stream, P, dP, S, scale, dS); break;
    case 4: hipLaunchKernelGGL(softmax_bwd_kernel<4>, grid, block, 0, stream, P, dP, S, scale, dS); break;
    case 8: hipLaunchKernelGGL(softmax_bwd_kernel<8>, grid, block, 0, stream, P, dP, S, scale, dS); break;
    case 16: hipLaunchKernelGGL(softmax_bwd_kernel<16>, grid, block, 0, stream, P, dP, S, scale, dS); break;
    default: hipLaunchKernelGGL(softmax_bwd_kernel<32>, grid, block, 0, stream, P, dP, S, scale, dS); break;
  }
}

}  // namespace catq

using namespace catq;

extern "C" size_t catq_attn_saved_bytes(const catq_attn_desc* a) {
  if (check_desc(a) != CATQ_OK) return 0;
  return attn_layout(a).saved_total;
}

extern "C" size_t catq_attn_bwd_workspace_bytes(const catq_attn_desc* a) {
  if (check_desc(a) != CATQ_OK) return 0;
  return attn_layout(a).bwd_total;
}

extern "C" catq_status catq_aux_attention_fwd(const catq_attn_desc* a, const void* qkv, void* o,
                                              void* saved, size_t saved_bytes,
                                              hipStream_t stream) {
  clear_error();
  CATQ_TRY(check_desc(a));
  CATQ_REQUIRE(qkv && o && saved, CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(aligned16(qkv) && aligned16(o) && aligned16(saved), CATQ_ERR_ALIGN, "misaligned");
  const AttnLayout L = attn_layout(a);
  CATQ_REQUIRE(saved_bytes >= L.saved_total, CATQ_ERR_WORKSPACE,
               "saved buffer of %zu bytes needed", L.saved_total);
  char* sv = reinterpret_cast<char*>(saved);
  bf16* Qh = reinterpret_cast<bf16*>(sv + L.o_qh);
  bf16* Kh = reinterpret_cast<bf16*>(sv + L.o_kh);
  bf16* Vh = L.flash ? reinterpret_cast<bf16*>(sv + L.o_vh) : nullptr;
  bf16* P = reinterpret_cast<bf16*>(sv + L.o_p);
  float* rstd = reinterpret_cast<float*>(sv + L.o_rstd);
  float* cs = reinterpret_cast<float*>(sv + L.o_cos);
  float* sn = reinterpret_cast<float*>(sv + L.o_sin);
  float* Sc = reinterpret_cast<float*>(sv + L.o_sc);
  const int64_t half = L.d / 2;
  CATQ_TRACED(stream, "rope_table_kernel", 0.0, 8.0 * (double)L.S * half, L.S, half, 0,
              hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((L.S * half + 255) / 256)),
                                 dim3(256), 0, stream, L.S, (int)L.d,
                                 std::log2((double)a->rope_theta), cs, sn));
  CATQ_CHECK_LAUNCH("rope table");
  const int64_t nw = L.B * L.S * (L.Hq + L.Hkv + (L.flash ? L.Hkv : 0));
  const int lph = qk_vec_lanes(L.d, L.ld, qkv);
  // q, k (and v for the fused path) read once as bf16 and written once, plus the rope tables
  const double qby = 4.0 * (double)nw * L.d + 8.0 * (double)L.B * L.S * L.Hq * (L.d / 2);
  if (lph > 0) {
    const int64_t nt = nw << lph;
    CATQ_TRACED(stream, "qk_prep_fwd_vec_kernel", 0.0, qby, nw, L.d, 0,
                hipLaunchKernelGGL(qk_prep_fwd_vec_kernel, dim3((unsigned)((nt + 255) / 256)),
                                   dim3(256), 0, stream, (const bf16*)qkv, L.B, L.S, (int)L.Hq,
                                   (int)L.Hkv, (int)L.d, (int)L.ld, lph, a->qk_norm, a->eps, cs,
                                   sn, Qh, Kh, Vh, rstd, a->act_quant));
  } else {
    CATQ_REQUIRE(!a->act_quant, CATQ_ERR_VALUE,
                 "activation quantization needs the vectorised q/k path (head_dim 64 or 128, "
                 "16-byte aligned rows)");
    hipLaunchKernelGGL(qk_prep_fwd_kernel, dim3((unsigned)((nw + 3) / 4)), dim3(256), 0, stream,
                       (const bf16*)qkv, L.B, L.S, (int)L.Hq, (int)L.Hkv, (int)L.d, (int)L.ld,
                       a->qk_norm, a->eps, cs, sn, Qh, Kh, Vh, rstd);
  }
  CATQ_CHECK_LAUNCH("qk prep");
  if (L.flash) {
    FaArgs f;
    std::memset(&f, 0, sizeof(f));
    f.Q = Qh;
    f.K = Kh;
    f.V = Vh;
    f.O = reinterpret_cast<bf16*>(o);
    f.lse = reinterpret_cast<float*>(sv + L.o_lse);
    f.B = (int)L.B;
    f.S = (int)L.S;
    f.Hq = (int)L.Hq;
    f.Hkv = (int)L.Hkv;
    f.scale = (float)(1.0 / std::sqrt((double)L.d));
    f.c = (float)(1.4426950408889634 / std::sqrt((double)L.d));
    return flash_forward((int)L.d, f, stream);
  }
  // scores
  {
    GemmArgs g = gemm_args_default();
    g.A = Qh;
    g.B = Kh;
    g.C = Sc;
    g.M = L.S;
    g.N = L.S;
    g.K = L.d;
    g.lda = L.d;
    g.ldb = L.d;
    g.ldc = L.S;
    g.batch = (int32_t)(L.B * L.Hq);
    g.inner = (int32_t)L.Hq;
    g.a_so = L.Hq * L.S * L.d;
    g.a_si = L.S * L.d;
    g.b_so = L.Hkv * L.S * L.d;
    g.b_si = L.S * L.d;
    g.b_div = (int32_t)L.G;
    g.c_so = L.Hq * L.S * L.S;
    g.c_si = L.S * L.S;
    g.alpha = (float)(1.0 / std::sqrt((double)L.d));
    g.causal = 1;
    CATQ_TRY(gemm_run(g, 0, 0, CATQ_BF16, CATQ_F32, stream));
  }
  launch_softmax_fwd(Sc, L.S, L.B * L.Hq * L.S, P, stream);
  CATQ_CHECK_LAUNCH("softmax fwd");
  // O = P V
  {
    GemmArgs g = gemm_args_default();
    g.A = P;
    g.B = reinterpret_cast<const bf16*>(qkv) + (L.Hq + L.Hkv) * L.d;
    g.C = o;
    g.M = L.S;
    g.N = L.d;
    g.K = L.S;
    g.lda = L.S;
    g.ldb = L.ld;
    g.ldc = L.Hq * L.d;
    g.batch = (int32_t)(L.B * L.Hq);
    g.inner = (int32_t)L.Hq;
    g.a_so = L.Hq * L.S * L.S;
    g.a_si = L.S * L.S;
    g.b_so = L.S * L.ld;
    g.b_si = L.d;
    g.b_div = (int32_t)L.G;
    g.c_so = L.S * L.Hq * L.d;
    g.c_si = L.d;
    g.causal = 2;
    CATQ_TRY(gemm_run(g, 0, 1, CATQ_BF16, CATQ_BF16, stream));
  }
  return CATQ_OK;
}

extern "C" catq_status catq_aux_attention_bwd(const catq_attn_desc* a, const void* qkv,
                                              const void* o, const void* saved, const void* d_o,
                                              void* dqkv, void* workspace,
                                              size_t workspace_bytes, hipStream_t stream) {
  clear_error();
  CATQ_TRY(check_desc(a));
  CATQ_REQUIRE(qkv && o && saved && d_o && dqkv && workspace, CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(aligned16(qkv) && aligned16(o) && aligned16(saved) && aligned16(d_o) &&
                   aligned16(dqkv) && aligned16(workspace),
               CATQ_ERR_ALIGN, "misaligned");
  const AttnLayout L = attn_layout(a);
  CATQ_REQUIRE(workspace_bytes >= L.bwd_total, CATQ_ERR_WORKSPACE,
               "workspace of %zu bytes needed", L.bwd_total);
  const char* sv = reinterpret_cast<const char*>(saved);
  const bf16* Qh = reinterpret_cast<const bf16*>(sv + L.o_qh);
  const bf16* Kh = reinterpret_cast<const bf16*>(sv + L.o_kh);
  const bf16* P = reinterpret_cast<const bf16*>(sv + L.o_p);
  const float* rstd = reinterpret_cast<const float*>(sv + L.o_rstd);
  const float* cs = reinterpret_cast<const float*>(sv + L.o_cos);
  const float* sn = reinterpret_cast<const float*>(sv + L.o_sin);
  char* ws = reinterpret_cast<char*>(workspace);
  float* dP = reinterpret_cast<float*>(ws + L.o_dp);
  bf16* dS = reinterpret_cast<bf16*>(ws + L.o_ds);
  float* dQ = reinterpret_cast<float*>(ws + L.o_dq);
  float* dKp = reinterpret_cast<float*>(ws + L.o_dk);
  float* dVp = reinterpret_cast<float*>(ws + L.o_dv);
  if (L.flash) {
    FaArgs f;
    std::memset(&f, 0, sizeof(f));
    f.Q = Qh;
    f.K = Kh;
    f.V = reinterpret_cast<const bf16*>(sv + L.o_vh);
    f.O = const_cast<bf16*>(reinterpret_cast<const bf16*>(o));
    f.lse = const_cast<float*>(reinterpret_cast<const float*>(sv + L.o_lse));
    f.dO = reinterpret_cast<const bf16*>(d_o);
    f.Dsum = reinterpret_cast<float*>(ws + L.o_dsum);
    f.dQ = dQ;
    f.dK = dKp;
    f.dV = dVp;
    f.hsplit = L.hs;
    f.B = (int)L.B;
    f.S = (int)L.S;
    f.Hq = (int)L.Hq;
    f.Hkv = (int)L.Hkv;
    f.scale = (float)(1.0 / std::sqrt((double)L.d));
    f.c = (float)(1.4426950408889634 / std::sqrt((double)L.d));
    CATQ_TRY(flash_backward((int)L.d, f, stream));
  } else {
  const bf16* V = reinterpret_cast<const bf16*>(qkv) + (L.Hq + L.Hkv) * L.d;
  // dP = dO V^T
  {
    GemmArgs g = gemm_args_default();
    g.A = d_o;
    g.B = V;
    g.C = dP;
    g.M = L.S;
    g.N = L.S;
    g.K = L.d;
    g.lda = L.Hq * L.d;
    g.ldb = L.ld;
    g.ldc = L.S;
    g.batch = (int32_t)(L.B * L.Hq);
    g.inner = (int32_t)L.Hq;
    g.a_so = L.S * L.Hq * L.d;
    g.a_si = L.d;
    g.b_so = L.S * L.ld;
    g.b_si = L.d;
    g.b_div = (int32_t)L.G;
    g.c_so = L.Hq * L.S * L.S;
    g.c_si = L.S * L.S;
    g.causal = 1;
    CATQ_TRY(gemm_run(g, 0, 0, CATQ_BF16, CATQ_F32, stream));
  }
  launch_softmax_bwd(P, dP, L.S, L.B * L.Hq * L.S, (float)(1.0 / std::sqrt((double)L.d)), dS,
                     stream);
  CATQ_CHECK_LAUNCH("softmax bwd");
  // dQ = dS K
  {
    GemmArgs g = gemm_args_default();
    g.A = dS;
    g.B = Kh;
    g.C = dQ;
    g.M = L.S;
    g.N = L.d;
    g.K = L.S;
    g.lda = L.S;
    g.ldb = L.d;
    g.ldc = L.d;
    g.batch = (int32_t)(L.B * L.Hq);
    g.inner = (int32_t)L.Hq;
    g.a_so = L.Hq * L.S * L.S;
    g.a_si = L.S * L.S;
    g.b_so = L.Hkv * L.S * L.d;
    g.b_si = L.S * L.d;
    g.b_div = (int32_t)L.G;
    g.c_so = L.Hq * L.S * L.d;
    g.c_si = L.S * L.d;
    g.causal = 2;
    CATQ_TRY(gemm_run(g, 0, 1, CATQ_BF16, CATQ_F32, stream));
  }
  // dK (per q head) = dS^T Q ; dV (per q head) = P^T dO
  {
    GemmArgs g = gemm_args_default();
    g.A = dS;
    g.B = Qh;
    g.C = dKp;
    g.M = L.S;
    g.N = L.d;
    g.K = L.S;
    g.lda = L.S;
    g.ldb = L.d;
    g.ldc = L.d;
    g.batch = (int32_t)(L.B * L.Hq);
    g.inner = (int32_t)L.Hq;
    g.a_so = L.Hq * L.S * L.S;
    g.a_si = L.S * L.S;
    g.b_so = L.Hq * L.S * L.d;
    g.b_si = L.S * L.d;
    g.c_so = L.Hq * L.S * L.d;
    g.c_si = L.S * L.d;
    g.causal = 3;
    CATQ_TRY(gemm_run(g, 1, 1, CATQ_BF16, CATQ_F32, stream));
    g.A = P;
    g.B = d_o;
    g.C = dVp;
    g.ldb = L.Hq * L.d;
    g.b_so = L.S * L.Hq * L.d;
    g.b_si = L.d;
    CATQ_TRY(gemm_run(g, 1, 1, CATQ_BF16, CATQ_F32, stream));
  }
  }
  const int64_t nw = L.B * L.S * (L.Hq + 2 * L.Hkv);
  const int lph = qk_vec_lanes(L.d, L.ld, qkv) > 0 && aligned16(dqkv) ? qk_vec_lanes(L.d, L.ld, qkv)
                                                                     : 0;
  if (lph > 0) {
    const int64_t nt = nw << lph;
    // fp32 gradients in (q, k, v per kv head), bf16 q|k|v in, bf16 dq|dk|dv out
    const double bby = (double)nw * L.d * (4.0 + 2.0 + 2.0);
    CATQ_TRACED(stream, "qk_prep_bwd_vec_kernel", 0.0, bby, nw, L.d, 0,
                hipLaunchKernelGGL(qk_prep_bwd_vec_kernel, dim3((unsigned)((nt + 255) / 256)),
                                   dim3(256), 0, stream, (const bf16*)qkv, rstd, cs, sn,
                                   (const float*)dQ, (const float*)dKp, (const float*)dVp, L.B,
                                   L.S, (int)L.Hq, (int)L.Hkv, (int)L.d, (int)L.ld, lph,
                                   a->qk_norm, L.flash ? L.hs : 0, (bf16*)dqkv));
  } else {
    hipLaunchKernelGGL(qk_prep_bwd_kernel, dim3((unsigned)((nw + 3) / 4)), dim3(256), 0, stream,
                       (const bf16*)qkv, rstd, cs, sn, (const float*)dQ, (const float*)dKp,
                       (const float*)dVp, L.B, L.S, (int)L.Hq, (int)L.Hkv, (int)L.d, (int)L.ld,
                       a->qk_norm, L.flash ? L.hs : 0, (bf16*)dqkv);
  }
  CATQ_CHECK_LAUNCH("qk prep bwd");
  return CATQ_OK;
}
