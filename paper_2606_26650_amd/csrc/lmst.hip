// Learnable modulation + softened ternarisation kernels (gfx950).
//
//   lmst_fwd      group statistics (Eq. 3), modulation (Eq. 3-4), the branch
//                 of Eq. 6 (identity / transition f of Eq. 5 / hard Q of
//                 Eq. 2), fake weight alpha*T (Sec. 2.2: W ~ alpha*T, no mu),
//                 hard codes and group scales (App. B.2)
//   lmst_bwd      per-group gradients of the three learnable factors from
//                 dL/dW_fake
//   pack_ternary  2-bit storage of the codes
//   adamw         optimizer step on a factor array
//
// Work split: one lane owns 8 consecutive weights (one 16-byte bf16 load), so
// a group of g weights is g/8 adjacent lanes of one wavefront and every group
// reduction is a butterfly over those lanes.  The kernels stream W once and
// write W_fake once: they are bound by HBM bandwidth and VALU issue, not by
// any contraction.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "kernels.h"
#include "lmst_math.h"

namespace catq {

// ------------------------------------------------------------ lmst forward

struct FwdArgs {
  const void* W;
  const float* dmu;
  const float* dal;
  const float* dde;
  float* stats;
  void* Wf;
  int8_t* codes;
  uint8_t* packed;  // HARD: 2-bit codes, 8 per 16-bit word (pack layout)
  float* alpha_out;
  int64_t n_oct;  // number of 8-element runs
  int64_t s0, s1, s2;
  int32_t lg;     // log2(lanes per group)
  float delta0;
  StConst st;
  float inv_g;
};

template <typename WT>
__device__ __forceinline__ void group_stats_lanes(const float (&w)[8], int L, float inv_g,
                                                  float& mu0, float& alpha0) {
  // fixed order: (j, j+4), (j, j+2), (j, j+1) inside the 8, then a butterfly
  // over the L lanes with masks L/2, ..., 1 (all lanes end with the same sum)
  double a[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) a[j] = (double)w[j] + (double)w[j + 4];
  double b0 = a[0] + a[2], b1 = a[1] + a[3];
  double s = b0 + b1;
  for (int m = L >> 1; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
  mu0 = (float)(s * (double)inv_g);
  double dm = (double)mu0;
#pragma unroll
  for (int j = 0; j < 4; ++j) a[j] = fabs((double)w[j] - dm) + fabs((double)w[j + 4] - dm);
  b0 = a[0] + a[2];
  b1 = a[1] + a[3];
  double t = b0 + b1;
  for (int m = L >> 1; m >= 1; m >>= 1) t += __shfl_xor(t, m, 64);
  alpha0 = (float)(t * (double)inv_g);
}

// Each thread handles FWD_U octets spaced by the grid size, so a wave keeps
// FWD_U 16-byte loads of W (and their group scalars) in flight before it
// computes anything; consecutive lanes still take consecutive octets, and a
// group's lanes are always valid or invalid together (the grid size is a
// multiple of 256 and n_oct a multiple of the lanes per group).
constexpr int FWD_U = 4;

template <typename WT, typename OT, int MODE, bool STATS>
__global__ __launch_bounds__(256) void lmst_fwd_kernel(FwdArgs a) {
  const int64_t T = (int64_t)gridDim.x * blockDim.x;
  const int64_t o0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int L = 1 << a.lg;
  const int lane_in_g = (int)(o0 & (L - 1));
  float w[FWD_U][8];
  float st[FWD_U][2], fc[FWD_U][3];
#pragma unroll
  for (int u = 0; u < FWD_U; ++u) {
    const int64_t o = o0 + u * T;
    if (o < a.n_oct) load8<WT>(reinterpret_cast<const WT*>(a.W) + o * 8, w[u]);
  }
#pragma unroll
  for (int u = 0; u < FWD_U; ++u) {
    const int64_t o = o0 + u * T;
    if (o >= a.n_oct) continue;
    const int64_t grp = o >> a.lg;
    if (!STATS) {
      st[u][0] = a.stats[2 * grp];
      st[u][1] = a.stats[2 * grp + 1];
    }
    fc[u][0] = a.dmu[grp * a.s0];
    fc[u][1] = a.dal[grp * a.s1];
    fc[u][2] = a.dde[grp * a.s2];
  }
#pragma unroll
  for (int u = 0; u < FWD_U; ++u) {
    const int64_t o = o0 + u * T;
    if (o >= a.n_oct) continue;  // whole groups: all lanes of a group agree
    const int64_t grp = o >> a.lg;
    float mu0, alpha0;
    if (STATS) {
      group_stats_lanes<WT>(w[u], L, a.inv_g, mu0, alpha0);
      if (lane_in_g == 0) {
        a.stats[2 * grp] = mu0;
        a.stats[2 * grp + 1] = alpha0;
      }
    } else {
      mu0 = st[u][0];
      alpha0 = st[u][1];
    }
    GroupScalars gs = group_scalars(mu0, alpha0, fc[u][0], fc[u][1], fc[u][2], a.delta0);
    if (a.alpha_out && lane_in_g == 0) a.alpha_out[grp] = gs.alpha;

    float out[8];
    if (MODE == CATQ_IDENTITY) {
#pragma unroll
      for (int j = 0; j < 8; ++j) out[j] = w[u][j];
    } else if (MODE == CATQ_SOFT) {
      soft_values<8>(w[u], soft_group(gs, a.st), out);
    } else {  // HARD
      const HardThresh th = hard_thresh(gs.delta, gs.alpha_div);
      float cs[8];
      hard_codes8(w[u], gs.mu, th, cs);
      unsigned int lo = 0, hi = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float c = cs[j];
        out[j] = gs.alpha * c;
        unsigned int byte = (unsigned int)(int)c & 0xffu;
        if (j < 4)
          lo |= byte << (8 * j);
        else
          hi |= byte << (8 * (j - 4));
      }
      if (a.codes) {
        uint2 v;
        v.x = lo;
        v.y = hi;
        *reinterpret_cast<uint2*>(a.codes + o * 8) = v;
      }
      if (a.packed) {
        // element 8o + j -> bits 2j..2j+1 of the little-endian word at byte
        // 2o: code + 1 in {0, 1, 2}
        unsigned int word = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const unsigned int byte = j < 4 ? (lo >> (8 * j)) & 0xffu : (hi >> (8 * (j - 4))) & 0xffu;
          word |= (unsigned int)((int)(int8_t)byte + 1) << (2 * j);
        }
        *reinterpret_cast<unsigned short*>(a.packed + o * 2) = (unsigned short)word;
      }
    }
    if (a.Wf) store8<OT>(reinterpret_cast<OT*>(a.Wf) + o * 8, out);
  }
}

// SOFT branch with cached statistics, the launch a calibration repeats every
// soft step: one lane owns OCT octets (8 * OCT weights) of one group, so the
// group's constants are formed once per 8 * OCT weights; a group of g weights
// is g / (8 * OCT) adjacent lanes, and load u of lane i of a group reads octet
// u * (g / (8 * OCT)) + i, so every load instruction of a wave covers whole
// segments of 16 bytes per lane of a group.  Same arithmetic as
// lmst_fwd_kernel's SOFT branch (bit-identical fake weights).
template <typename WT, typename OT, int OCT>
__global__ __launch_bounds__(256) void lmst_soft_kernel(FwdArgs a) {
  constexpr int LOCT = OCT == 8 ? 3 : 2;
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= (a.n_oct >> LOCT)) return;
  const int lgl = a.lg - LOCT;              // log2(lanes per group)
  const int64_t grp = c >> lgl;
  const int li = (int)(c & ((1 << lgl) - 1));
  const int64_t base = (grp << (a.lg + 3)) + 8 * (int64_t)li;   // element of octet li
  const int64_t step = (int64_t)8 << lgl;                        // next octet of this lane
  float w[OCT][8];
#pragma unroll
  for (int u = 0; u < OCT; ++u)
    load8<WT>(reinterpret_cast<const WT*>(a.W) + base + u * step, w[u]);
  const GroupScalars gs = group_scalars(a.stats[2 * grp], a.stats[2 * grp + 1], a.dmu[grp * a.s0],
                                        a.dal[grp * a.s1], a.dde[grp * a.s2], a.delta0);
  if (a.alpha_out && li == 0) a.alpha_out[grp] = gs.alpha;
  const SoftGroup q = soft_group(gs, a.st);
#pragma unroll
  for (int u = 0; u < OCT; ++u) {
    float out[8];
    soft_values<8>(w[u], q, out);
    store8<OT>(reinterpret_cast<OT*>(a.Wf) + base + u * step, out);
  }
}

template <typename T>
static const char* tname() {
  return sizeof(T) == 2 ? "__bf16" : "float";
}

template <typename WT, typename OT, int MODE>
static void launch_fwd_mode(const FwdArgs& a, bool stats, dim3 grid, hipStream_t stream) {
  char tag[96];
  std::snprintf(tag, sizeof(tag), "lmst_fwd_kernel<%s, %s, %d, %s>", tname<WT>(), tname<OT>(),
                MODE, stats ? "true" : "false");
  // algorithmic bytes: W read once, W_fake / codes written once, per group
  // the three factors read (or one shared value) and the stats read or written
  const double n = (double)a.n_oct * 8.0;
  const double ng = n / (8.0 * (1 << a.lg));
  const double fac = 4.0 * ((a.s0 ? ng : 1) + (a.s1 ? ng : 1) + (a.s2 ? ng : 1));
  const double bytes = n * sizeof(WT) + (a.Wf ? n * sizeof(OT) : 0.0) + (a.codes ? n : 0.0) +
                       (a.packed ? n / 4.0 : 0.0) + fac + 8.0 * ng +
                       (a.alpha_out ? 4.0 * ng : 0.0);
  if (stats)
    CATQ_TRACED(stream, tag, 0.0, bytes, (int64_t)n, 0, 0,
                hipLaunchKernelGGL((lmst_fwd_kernel<WT, OT, MODE, true>), grid, dim3(256), 0,
                                   stream, a));
  else
    CATQ_TRACED(stream, tag, 0.0, bytes, (int64_t)n, 0, 0,
                hipLaunchKernelGGL((lmst_fwd_kernel<WT, OT, MODE, false>), grid, dim3(256), 0,
                                   stream, a));
}

template <typename WT, typename OT>
static void launch_fwd(const FwdArgs& a, int mode, bool stats, dim3 grid, hipStream_t stream) {
  if (mode == CATQ_IDENTITY)
    launch_fwd_mode<WT, OT, CATQ_IDENTITY>(a, stats, grid, stream);
  else if (mode == CATQ_SOFT)
    launch_fwd_mode<WT, OT, CATQ_SOFT>(a, stats, grid, stream);
  else
    launch_fwd_mode<WT, OT, CATQ_HARD>(a, stats, grid, stream);
}

template <typename WT, typename OT>
static void launch_soft(const FwdArgs& a, hipStream_t stream) {
  char tag[96];
  std::snprintf(tag, sizeof(tag), "lmst_soft_kernel<%s, %s>", tname<WT>(), tname<OT>());
  const double n = (double)a.n_oct * 8.0;
  const double ng = n / (8.0 * (1 << a.lg));
  const double fac = 4.0 * ((a.s0 ? ng : 1) + (a.s1 ? ng : 1) + (a.s2 ? ng : 1));
  const double bytes = n * sizeof(WT) + n * sizeof(OT) + fac + 8.0 * ng +
                       (a.alpha_out ? 4.0 * ng : 0.0);
  // 32 weights per lane (64 per lane measured slower: fewer waves in flight)
  const int64_t lanes = a.n_oct >> 2;
  CATQ_TRACED(stream, tag, 0.0, bytes, (int64_t)n, 0, 0,
              hipLaunchKernelGGL((lmst_soft_kernel<WT, OT, 4>),
                                 dim3((unsigned)((lanes + 255) / 256)), dim3(256), 0, stream, a));
}

catq_status check_lmst_params(const catq_lmst_params* p, int64_t d_in) {
  CATQ_REQUIRE(p != nullptr, CATQ_ERR_NULL, "params pointer is NULL");
  const int g = p->group_size;
  CATQ_REQUIRE(g >= 16 && g <= 512 && (g % 8) == 0 && (((g / 8) & (g / 8 - 1)) == 0),
               CATQ_ERR_VALUE, "group_size %d: must be 8 times a power of two in [16, 512]", g);
  CATQ_REQUIRE(d_in % g == 0, CATQ_ERR_SHAPE, "d_in %lld is not a multiple of group_size %d",
               (long long)d_in, g);
  CATQ_REQUIRE(p->mode >= CATQ_IDENTITY && p->mode <= CATQ_HARD, CATQ_ERR_VALUE, "bad mode %d",
               p->mode);
  CATQ_REQUIRE(std::isfinite(p->delta0) && p->delta0 > 0.0f, CATQ_ERR_VALUE,
               "delta0 must be finite and > 0");
  if (p->mode == CATQ_SOFT)
    CATQ_REQUIRE(std::isfinite(p->s) && p->s > 0.0f, CATQ_ERR_VALUE,
                 "SOFT mode needs a finite s > 0 (got %g)", (double)p->s);
  CATQ_REQUIRE(std::isfinite(p->s_bwd) && p->s_bwd >= 0.0f, CATQ_ERR_VALUE,
               "s_bwd must be finite and >= 0");
  for (int i = 0; i < 3; ++i)
    CATQ_REQUIRE(p->factor_stride[i] == 0 || p->factor_stride[i] == 1, CATQ_ERR_VALUE,
                 "factor_stride[%d] must be 0 or 1", i);
  return CATQ_OK;
}

static int ilog2(int v) {
  int r = 0;
  while ((1 << r) < v) ++r;
  return r;
}

// -------------------------------------------------------------- lmst bwd

struct BwdArgs {
  const float* G;     // nsplit partial sums, split i at G + i*split_stride
  int64_t split_stride;
  int32_t nsplit;
  float* G_out;       // optional: the summed G
  const void* W;
  const float* stats;
  const float* dmu;
  const float* dal;
  const float* dde;
  float* out[3];
  float* ws;  // [3][n_groups] for stride-0 factors
  int64_t n_oct, n_groups;
  int64_t s[3];
  int32_t lg;
  int32_t mode;
  int32_t ste;  // HARD with s_bwd == 0
  float delta0;
  StConst st;
};

// NS > 0: exactly NS split partials, all loads issued before any use;
// NS = 0: any count, folded in a loop.
template <typename WT, int NS>
__global__ __launch_bounds__(256) void lmst_bwd_kernel(BwdArgs a) {
  const int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (o >= a.n_oct) return;
  const int L = 1 << a.lg;
  const int64_t grp = o >> a.lg;
  const int lane_in_g = (int)(o & (L - 1));
  // the group's scalars first: their loads are in flight with the streams
  const float mu0 = a.stats[2 * grp], alpha0 = a.stats[2 * grp + 1];
  const float fmu = a.dmu[grp * a.s[0]], fal = a.dal[grp * a.s[1]], fde = a.dde[grp * a.s[2]];
  float w[8], G[8];
  load8<WT>(reinterpret_cast<const WT*>(a.W) + o * 8, w);
  // split-K partials of G, folded in split order (the same order and
  // rounding as a separate reduction pass)
  if constexpr (NS > 0) {
    float t[NS][8];
#pragma unroll
    for (int sp = 0; sp < NS; ++sp) load8<float>(a.G + sp * a.split_stride + o * 8, t[sp]);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      G[j] = t[0][j];
#pragma unroll
      for (int sp = 1; sp < NS; ++sp) G[j] += t[sp][j];
    }
  } else {
    load8<float>(a.G + o * 8, G);
    for (int sp = 1; sp < a.nsplit; ++sp) {
      float t[8];
      load8<float>(a.G + sp * a.split_stride + o * 8, t);
#pragma unroll
      for (int j = 0; j < 8; ++j) G[j] += t[j];
    }
  }
  if (a.G_out) store8<float>(a.G_out + o * 8, G);
  GroupScalars gs = group_scalars(mu0, alpha0, fmu, fal, fde, a.delta0);
  float ST = 0.f, SW = 0.f, S1 = 0.f, SD = 0.f;
  if (a.mode != CATQ_IDENTITY) {
    const float inv_a = 1.0f / gs.alpha_div;
    const float dz = gs.delta * a.st.c2s;
    const float ED = one_minus_exp_neg(gs.delta * a.st.s4, gs.delta * a.st.s4l);
    float hc[8];
    if (a.mode == CATQ_HARD) hard_codes8(w, gs.mu, hard_thresh(gs.delta, gs.alpha_div), hc);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      float xs = (w[j] - gs.mu) * inv_a;
      float fp, fwp, fdp;
      if (a.ste) {
        fwp = 1.0f;
        fdp = 0.0f;
        fp = 0.0f;
      } else {
        transition_parts_z(xs, a.st.c2s, dz, ED, fp, fwp, fdp);
      }
      float T = (a.mode == CATQ_HARD) ? hc[j] : fp;
      ST = fmaf(G[j], T, ST);
      float gf = G[j] * fwp;
      S1 += gf;
      SW = fmaf(gf, xs, SW);
      SD = fmaf(G[j], fdp, SD);
    }
  }
  for (int m = L >> 1; m >= 1; m >>= 1) {
    ST += __shfl_xor(ST, m, 64);
    SW += __shfl_xor(SW, m, 64);
    S1 += __shfl_xor(S1, m, 64);
    SD += __shfl_xor(SD, m, 64);
  }
  if (lane_in_g == 0) {
    // the constant factors of f (k2, soft only), f_W and f_Delta (sk4)
    const FacScale k = fac_scale(a.mode, a.ste, a.st);
    S1 *= k.w;
    SW *= k.w;
    SD *= k.d;
    ST *= k.f;
    float v[3];
    v[0] = alpha0 * (-S1);
    v[1] = alpha0 * (ST - SW);
    v[2] = a.delta0 * (gs.alpha * SD);
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      if (a.s[i] == 1)
        a.out[i][grp] = v[i];
      else
        a.ws[i * a.n_groups + grp] = v[i];
    }
  }
}

// Sum of the per-group contributions of shared (stride-0) factors, in a fixed
// order: thread t sums groups t, t+1024, ... in double, then a tree.
__global__ __launch_bounds__(1024) void shared_factor_reduce(const float* ws, int64_t n_groups,
                                                             int which, float* out) {
  __shared__ double red[1024];
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < n_groups; i += 1024) acc += (double)ws[which * n_groups + i];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = 512; s >= 1; s >>= 1) {
    if ((int)threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = (float)red[0];
}

catq_status finish_shared_factors(const int64_t* strides, int64_t n_groups, const float* ws,
                                  float* const* out, hipStream_t stream) {
  for (int i = 0; i < 3; ++i) {
    if (strides[i] == 0) {
      hipLaunchKernelGGL(shared_factor_reduce, dim3(1), dim3(1024), 0, stream, ws, n_groups, i,
                         out[i]);
      CATQ_CHECK_LAUNCH("shared factor reduction");
    }
  }
  return CATQ_OK;
}

catq_status launch_factor_grads(const float* G, int nsplit, int64_t split_stride, float* G_out,
                                const void* W, catq_dtype w_dtype, int64_t n_rows,
                                int64_t d_in, const float* stats, const float* d_mu,
                                const float* d_alpha, const float* d_delta,
                                const catq_lmst_params* p, float* g_mu, float* g_alpha,
                                float* g_delta, float* ws_shared, hipStream_t stream) {
  BwdArgs a;
  a.G = G;
  a.nsplit = nsplit > 1 ? nsplit : 1;
  a.split_stride = split_stride;
  a.G_out = G_out;
  a.W = W;
  a.stats = stats;
  a.dmu = d_mu;
  a.dal = d_alpha;
  a.dde = d_delta;
  a.out[0] = g_mu;
  a.out[1] = g_alpha;
  a.out[2] = g_delta;
  a.ws = ws_shared;
  const int64_t n = n_rows * d_in;
  a.n_oct = n / 8;
  a.n_groups = n / p->group_size;
  for (int i = 0; i < 3; ++i) a.s[i] = p->factor_stride[i];
  a.lg = ilog2(p->group_size / 8);
  a.mode = p->mode;
  a.ste = (p->mode == CATQ_HARD && p->s_bwd == 0.0f) ? 1 : 0;
  a.delta0 = p->delta0;
  const double s_use = (p->mode == CATQ_HARD) ? (double)p->s_bwd : (double)p->s;
  a.st = make_st(s_use > 0 ? s_use : 1.0);
  dim3 grid((unsigned)((a.n_oct + 255) / 256));
  const double nn = (double)n, ngd = (double)a.n_groups;
  const double bytes = nn * (4.0 * a.nsplit + (G_out ? 4.0 : 0.0) + (w_dtype == CATQ_BF16 ? 2.0 : 4.0)) +
                       ngd * (8.0 + 12.0 + 12.0);
  if (w_dtype == CATQ_BF16) {
    auto go = [&](auto kern) {
      CATQ_TRACED(stream, "lmst_bwd_kernel<__bf16>", 0.0, bytes, n, 0, 0,
                  hipLaunchKernelGGL(kern, grid, dim3(256), 0, stream, a));
    };
    if (a.nsplit == 1)
      go(lmst_bwd_kernel<bf16, 1>);
    else if (a.nsplit == 2)
      go(lmst_bwd_kernel<bf16, 2>);
    else if (a.nsplit == 4)
      go(lmst_bwd_kernel<bf16, 4>);
    else
      go(lmst_bwd_kernel<bf16, 0>);
  } else {
    CATQ_TRACED(stream, "lmst_bwd_kernel<float>", 0.0, bytes, n, 0, 0,
                hipLaunchKernelGGL((lmst_bwd_kernel<float, 0>), grid, dim3(256), 0, stream, a));
  }
  CATQ_CHECK_LAUNCH("factor gradients");
  for (int i = 0; i < 3; ++i) {
    if (a.s[i] == 0) {
      hipLaunchKernelGGL(shared_factor_reduce, dim3(1), dim3(1024), 0, stream, ws_shared,
                         a.n_groups, i, a.out[i]);
      CATQ_CHECK_LAUNCH("shared factor reduction");
    }
  }
  return CATQ_OK;
}

// ------------------------------------------------------------------ pack

__global__ __launch_bounds__(256) void pack_kernel(const int8_t* codes, int64_t n16,
                                                   int64_t n_bytes, uint8_t* packed) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < n16) {
    u32x4 v = *reinterpret_cast<const u32x4*>(codes + t * 16);
    unsigned int out = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      int c = (int)(int8_t)((v[i >> 2] >> (8 * (i & 3))) & 0xffu) + 1;
      unsigned int cc = (c >= 0 && c <= 2) ? (unsigned int)c : 3u;
      out |= cc << (2 * i);
    }
    *reinterpret_cast<unsigned int*>(packed + t * 4) = out;
  } else {
    // tail bytes (n_codes % 16 != 0)
    const int64_t b = n16 * 4 + (t - n16);
    if (b >= n_bytes) return;
    unsigned int out = 0;
    for (int j = 0; j < 4; ++j) {
      int c = (int)codes[b * 4 + j] + 1;
      unsigned int cc = (c >= 0 && c <= 2) ? (unsigned int)c : 3u;
      out |= cc << (2 * j);
    }
    packed[b] = (uint8_t)out;
  }
}

// ----------------------------------------------------------------- adamw

__global__ __launch_bounds__(256) void adamw_kernel(float* p, const float* g, float* m, float* v,
                                                    int64_t n, float lr, float b1, float c1,
                                                    float b2, float c2, float eps, float inv_bc1,
                                                    float inv_sqrt_bc2, float lo, float hi) {
  // c1 = 1 - beta1 and c2 = 1 - beta2 are formed in double on the host and
  // rounded once: 1 - (float)0.999 would be 1.3e-5 off 0.001.
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float gi = g[i];
  float mi = fmaf(b1, m[i], c1 * gi);
  float vi = fmaf(b2, v[i], c2 * gi * gi);
  m[i] = mi;
  v[i] = vi;
  float upd = (mi * inv_bc1) / (sqrtf(vi) * inv_sqrt_bc2 + eps);
  float np = p[i] - lr * upd;
  p[i] = fminf(fmaxf(np, lo), hi);
}

template <typename T>
__global__ __launch_bounds__(256) void add_kernel(const T* a, const T* b, T* y, int64_t n8) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n8) return;
  float x[8], z[8];
  load8<T>(a + i * 8, x);
  load8<T>(b + i * 8, z);
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] += z[j];
  store8<T>(y + i * 8, x);
}

}  // namespace catq

using namespace catq;

// =================================================================== C ABI

extern "C" catq_status catq_modulate_ternarize(const void* W, catq_dtype w_dtype, int64_t d_out,
                                               int64_t d_in, const float* d_mu,
                                               const float* d_alpha, const float* d_delta,
                                               const catq_lmst_params* p, float* stats,
                                               int32_t stats_mode, void* W_fake,
                                               catq_dtype wf_dtype, int8_t* codes,
                                               float* alpha_out, hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(W && d_mu && d_alpha && d_delta && stats, CATQ_ERR_NULL,
               "W, factors and stats must not be NULL");
  CATQ_REQUIRE(count_ok(d_out, d_in), CATQ_ERR_SHAPE,
               "d_out and d_in must be > 0 with d_out*d_in <= 2^38");
  CATQ_TRY(check_lmst_params(p, d_in));
  CATQ_REQUIRE(dtype_ok(w_dtype) && dtype_ok(wf_dtype), CATQ_ERR_DTYPE, "bad dtype");
  CATQ_REQUIRE(stats_mode == 0 || stats_mode == 1, CATQ_ERR_VALUE, "stats_mode must be 0 or 1");
  CATQ_REQUIRE(W_fake != nullptr || (p->mode == CATQ_HARD && codes != nullptr), CATQ_ERR_NULL,
               "W_fake may be NULL only in HARD mode with codes");
  CATQ_REQUIRE(codes == nullptr || p->mode == CATQ_HARD, CATQ_ERR_VALUE,
               "codes are produced only in HARD mode");
  CATQ_REQUIRE(aligned16(W) && aligned16(W_fake) && aligned16(codes) && aligned16(stats),
               CATQ_ERR_ALIGN, "W, W_fake, codes and stats must be 16-byte aligned");
  FwdArgs a;
  a.W = W;
  a.dmu = d_mu;
  a.dal = d_alpha;
  a.dde = d_delta;
  a.stats = stats;
  a.Wf = W_fake;
  a.codes = codes;
  a.packed = nullptr;
  a.alpha_out = alpha_out;
  a.n_oct = d_out * d_in / 8;
  a.s0 = p->factor_stride[0];
  a.s1 = p->factor_stride[1];
  a.s2 = p->factor_stride[2];
  a.lg = ilog2(p->group_size / 8);
  a.delta0 = p->delta0;
  a.st = make_st(p->mode == CATQ_SOFT ? (double)p->s : 1.0);
  a.inv_g = 1.0f / (float)p->group_size;
  const bool st = stats_mode == 0;
  if (p->mode == CATQ_SOFT && !st && p->group_size >= 32) {
    if (w_dtype == CATQ_BF16 && wf_dtype == CATQ_BF16)
      launch_soft<bf16, bf16>(a, stream);
    else if (w_dtype == CATQ_BF16)
      launch_soft<bf16, float>(a, stream);
    else if (wf_dtype == CATQ_BF16)
      launch_soft<float, bf16>(a, stream);
    else
      launch_soft<float, float>(a, stream);
    CATQ_CHECK_LAUNCH("modulate_ternarize");
    return CATQ_OK;
  }
  dim3 grid((unsigned)((a.n_oct + 256 * FWD_U - 1) / (256 * FWD_U)));
  if (w_dtype == CATQ_BF16 && wf_dtype == CATQ_BF16)
    launch_fwd<bf16, bf16>(a, p->mode, st, grid, stream);
  else if (w_dtype == CATQ_BF16)
    launch_fwd<bf16, float>(a, p->mode, st, grid, stream);
  else if (wf_dtype == CATQ_BF16)
    launch_fwd<float, bf16>(a, p->mode, st, grid, stream);
  else
    launch_fwd<float, float>(a, p->mode, st, grid, stream);
  CATQ_CHECK_LAUNCH("modulate_ternarize");
  return CATQ_OK;
}

extern "C" catq_status catq_ternarize_pack(const void* W, catq_dtype w_dtype, int64_t d_out,
                                           int64_t d_in, const float* d_mu, const float* d_alpha,
                                           const float* d_delta, const catq_lmst_params* p,
                                           float* stats, int32_t stats_mode, uint8_t* packed,
                                           float* alpha_out, hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(W && d_mu && d_alpha && d_delta && stats && packed, CATQ_ERR_NULL,
               "W, factors, stats and packed must not be NULL");
  CATQ_REQUIRE(count_ok(d_out, d_in), CATQ_ERR_SHAPE,
               "d_out and d_in must be > 0 with d_out*d_in <= 2^38");
  CATQ_TRY(check_lmst_params(p, d_in));
  CATQ_REQUIRE(p->mode == CATQ_HARD, CATQ_ERR_VALUE, "the packed codes are those of HARD mode");
  CATQ_REQUIRE(dtype_ok(w_dtype), CATQ_ERR_DTYPE, "bad dtype");
  CATQ_REQUIRE(stats_mode == 0 || stats_mode == 1, CATQ_ERR_VALUE, "stats_mode must be 0 or 1");
  CATQ_REQUIRE(aligned16(W) && aligned16(packed) && aligned16(stats), CATQ_ERR_ALIGN,
               "W, packed and stats must be 16-byte aligned");
  FwdArgs a;
  a.W = W;
  a.dmu = d_mu;
  a.dal = d_alpha;
  a.dde = d_delta;
  a.stats = stats;
  a.Wf = nullptr;
  a.codes = nullptr;
  a.packed = packed;
  a.alpha_out = alpha_out;
  a.n_oct = d_out * d_in / 8;
  a.s0 = p->factor_stride[0];
  a.s1 = p->factor_stride[1];
  a.s2 = p->factor_stride[2];
  a.lg = ilog2(p->group_size / 8);
  a.delta0 = p->delta0;
  a.st = make_st(1.0);
  a.inv_g = 1.0f / (float)p->group_size;
  dim3 grid((unsigned)((a.n_oct + 256 * FWD_U - 1) / (256 * FWD_U)));
  const bool st = stats_mode == 0;
  if (w_dtype == CATQ_BF16)
    launch_fwd_mode<bf16, bf16, CATQ_HARD>(a, st, grid, stream);
  else
    launch_fwd_mode<float, bf16, CATQ_HARD>(a, st, grid, stream);
  CATQ_CHECK_LAUNCH("ternarize_pack");
  return CATQ_OK;
}

extern "C" catq_status catq_pack_ternary(const int8_t* codes, int64_t d_out, int64_t d_in,
                                         uint8_t* packed, hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(codes && packed, CATQ_ERR_NULL, "codes and packed must not be NULL");
  CATQ_REQUIRE(count_ok(d_out, d_in), CATQ_ERR_SHAPE,
               "d_out and d_in must be > 0 with d_out*d_in <= 2^38");
  CATQ_REQUIRE(d_in % 4 == 0, CATQ_ERR_SHAPE, "d_in must be a multiple of 4");
  CATQ_REQUIRE(aligned16(codes) && aligned16(packed), CATQ_ERR_ALIGN,
               "codes and packed must be 16-byte aligned");
  const int64_t n = d_out * d_in;
  const int64_t n16 = n / 16;
  const int64_t n_bytes = n / 4;
  const int64_t threads = n16 + (n_bytes - n16 * 4);
  CATQ_TRACED(stream, "pack_kernel", 0.0, (double)n + (double)n_bytes, n, 0, 0,
              hipLaunchKernelGGL(pack_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256),
                                 0, stream, codes, n16, n_bytes, packed));
  CATQ_CHECK_LAUNCH("pack_ternary");
  return CATQ_OK;
}

extern "C" catq_status catq_aux_adamw(float* p, const float* grad, float* m, float* v, int64_t n,
                                      int64_t step, float lr, double beta1, double beta2,
                                      double eps, float lo, float hi, hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(p && grad && m && v, CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(count_ok(n) && step >= 1, CATQ_ERR_SHAPE, "n must be in [1, 2^38] and step >= 1");
  CATQ_REQUIRE(beta1 >= 0 && beta1 < 1 && beta2 >= 0 && beta2 < 1 && eps > 0 && lo <= hi,
               CATQ_ERR_VALUE, "bad optimizer hyper-parameters");
  const double bc1 = 1.0 - std::pow(beta1, (double)step);
  const double bc2 = 1.0 - std::pow(beta2, (double)step);
  hipLaunchKernelGGL(adamw_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, p,
                     grad, m, v, n, lr, (float)beta1, (float)(1.0 - beta1), (float)beta2,
                     (float)(1.0 - beta2), (float)eps, (float)(1.0 / bc1),
                     (float)(1.0 / std::sqrt(bc2)), lo, hi);
  CATQ_CHECK_LAUNCH("adamw");
  return CATQ_OK;
}

extern "C" catq_status catq_aux_add(const void* a, const void* b, void* y, catq_dtype dtype,
                                    int64_t n, hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(a && b && y, CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(count_ok(n) && n % 8 == 0, CATQ_ERR_SHAPE,
               "n must be a positive multiple of 8, at most 2^38");
  CATQ_REQUIRE(dtype_ok(dtype), CATQ_ERR_DTYPE, "bad dtype");
  CATQ_REQUIRE(aligned16(a) && aligned16(b) && aligned16(y), CATQ_ERR_ALIGN, "misaligned");
  const int64_t n8 = n / 8;
  dim3 grid((unsigned)((n8 + 255) / 256));
  if (dtype == CATQ_BF16)
    hipLaunchKernelGGL((add_kernel<bf16>), grid, dim3(256), 0, stream, (const bf16*)a,
                       (const bf16*)b, (bf16*)y, n8);
  else
    hipLaunchKernelGGL((add_kernel<float>), grid, dim3(256), 0, stream, (const float*)a,
                       (const float*)b, (float*)y, n8);
  CATQ_CHECK_LAUNCH("add");
  return CATQ_OK;
}
