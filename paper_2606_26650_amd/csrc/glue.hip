// Decoder-block pieces around the fake-ternary linears: RMSNorm, SwiGLU and the
// routing / permutation of the routed-expert MLP (gfx950).  All are streaming
// kernels bound by HBM bandwidth; rows are processed with 16-byte accesses.
#include <cmath>

#include "kernels.h"

namespace catq {

// ------------------------------------------------------------- block sums

template <int NT>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  if (l == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) s += red[i];
  __syncthreads();
  return s;
}

template <int NT>
__device__ __forceinline__ float block_max(float v, float* red) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  if (l == 0) red[w] = v;
  __syncthreads();
  float r = 0.f;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) r = fmaxf(r, red[i]);
  __syncthreads();
  return r;
}

// -------------------------------------------------- activation quantization
// Symmetric 8-bit absmax fake quantization (the W1.58A8 setting) of each
// group of `group` consecutive values of a row: s = max|x| / 127,
// q = round-half-even(x / s) clamped to [-127, 127] (0 when s = 0),
// y = bf16(q * s); every step in IEEE fp32.  One workgroup per (row, group):
// a pass for the maximum, a second (from L2) for the codes.  y may alias x.
template <typename XT>
__global__ __launch_bounds__(256) void act_quant_kernel(const XT* x, int64_t n, int64_t group,
                                                        bf16* y) {
  __shared__ float red[4];
  const int64_t off = (int64_t)blockIdx.x * n + (int64_t)blockIdx.y * group;
  const XT* xr = x + off;
  bf16* yr = y + off;
  const int64_t nc = group / 8;
  float m = 0.f;
  for (int64_t c = threadIdx.x; c < nc; c += 256) {
    float v[8];
    load8<XT>(xr + c * 8, v);
#pragma unroll
    for (int j = 0; j < 8; ++j) m = fmaxf(m, fabsf(v[j]));
  }
  m = block_max<256>(m, red);
  const float s = m / 127.0f;
  for (int64_t c = threadIdx.x; c < nc; c += 256) {
    float v[8];
    load8<XT>(xr + c * 8, v);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float q = s > 0.f ? fminf(fmaxf(rintf(v[j] / s), -127.f), 127.f) : 0.f;
      v[j] = q * s;
    }
    store8<bf16>(yr + c * 8, v);
  }
}

// ---------------------------------------------------------------- RMSNorm

template <typename XT>
__global__ __launch_bounds__(256) void rmsnorm_fwd_kernel(const XT* x, int64_t n, float eps,
                                                          bf16* y, float* rstd) {
  __shared__ float red[4];
  const int64_t row = blockIdx.x;
  const XT* xr = x + row * n;
  const int64_t nc = n / 8;
  float ss = 0.f;
  for (int64_t c = threadIdx.x; c < nc; c += 256) {
    float v[8];
    load8<XT>(xr + c * 8, v);
#pragma unroll
    for (int j = 0; j < 8; ++j) ss = fmaf(v[j], v[j], ss);
  }
  ss = block_sum<256>(ss, red);
  const float r = 1.0f / sqrtf(ss / (float)n + eps);
  if (threadIdx.x == 0 && rstd) rstd[row] = r;
  for (int64_t c = threadIdx.x; c < nc; c += 256) {
    float v[8];
    load8<XT>(xr + c * 8, v);
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] *= r;
    store8<bf16>(y + row * n + c * 8, v);
  }
}

template <typename XT>
__global__ __launch_bounds__(256) void rmsnorm_bwd_kernel(const XT* x, const float* rstd,
                                                          const bf16* dy, const bf16* dres,
                                                          int64_t n, bf16* dx) {
  __shared__ float red[4];
  const int64_t row = blockIdx.x;
  const int64_t nc = n / 8;
  float sd = 0.f;
  for (int64_t c = threadIdx.x; c < nc; c += 256) {
    float a[8], b[8];
    load8<XT>(x + row * n + c * 8, a);
    load8<bf16>(dy + row * n + c * 8, b);
#pragma unroll
    for (int j = 0; j < 8; ++j) sd = fmaf(a[j], b[j], sd);
  }
  sd = block_sum<256>(sd, red);
  const float r = rstd[row];
  const float coef = r * r * r * sd / (float)n;
  for (int64_t c = threadIdx.x; c < nc; c += 256) {
    float a[8], b[8], d[8];
    load8<XT>(x + row * n + c * 8, a);
    load8<bf16>(dy + row * n + c * 8, b);
    if (dres)
      load8<bf16>(dres + row * n + c * 8, d);
    else
#pragma unroll
      for (int j = 0; j < 8; ++j) d[j] = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) a[j] = fmaf(r, b[j], fmaf(-a[j], coef, d[j]));
    store8<bf16>(dx + row * n + c * 8, a);
  }
}

// ---------------------------------------------------------------- SwiGLU


__global__ __launch_bounds__(256) void swiglu_fwd_kernel(const bf16* gu, int64_t rows, int64_t F,
                                                         bf16* a) {
  const int64_t nc = F / 8;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * nc) return;
  const int64_t r = i / nc, c = i % nc;
  float g[8], u[8];
  load8<bf16>(gu + r * 2 * F + c * 8, g);
  load8<bf16>(gu + r * 2 * F + F + c * 8, u);
#pragma unroll
  for (int j = 0; j < 8; ++j) g[j] = swiglu1(g[j], u[j]);
  store8<bf16>(a + r * F + c * 8, g);
}

__global__ __launch_bounds__(256) void swiglu_bwd_kernel(const bf16* gu, const bf16* da,
                                                         int64_t rows, int64_t F, bf16* dgu) {
  const int64_t nc = F / 8;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * nc) return;
  const int64_t r = i / nc, c = i % nc;
  float g[8], u[8], d[8], dg[8], du[8];
  load8<bf16>(gu + r * 2 * F + c * 8, g);
  load8<bf16>(gu + r * 2 * F + F + c * 8, u);
  load8<bf16>(da + r * F + c * 8, d);
#pragma unroll
  for (int j = 0; j < 8; ++j) swiglu1_bwd(g[j], u[j], d[j], dg[j], du[j]);
  store8<bf16>(dgu + r * 2 * F + c * 8, dg);
  store8<bf16>(dgu + r * 2 * F + F + c * 8, du);
}

// ---------------------------------------------------------------- routing

// One wavefront per token: top-k of the E logits (largest first; equal values
// go to the lower expert id) and the softmax over the k selected logits.
__global__ __launch_bounds__(256) void moe_topk_kernel(const float* logits, int64_t T, int E,
                                                       int k, int32_t* ids, float* w) {
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= T) return;
  const int per = (E + 63) / 64;  // <= 16
  float v[16];
  for (int i = 0; i < 16; ++i) {
    const int e = lane + 64 * i;
    v[i] = (i < per && e < E) ? logits[t * E + e] : -INFINITY;
  }
  float sel[16];
  int sid[16];
  for (int j = 0; j < k; ++j) {
    // lane-local best (lowest id among equals), then across lanes
    float bv = -INFINITY;
    int be = 0x7fffffff;
    for (int i = 0; i < per; ++i) {
      const int e = lane + 64 * i;
      if (e < E && (v[i] > bv || (v[i] == bv && e < be))) {
        bv = v[i];
        be = e;
      }
    }
    for (int m = 32; m >= 1; m >>= 1) {
      const float ov = __shfl_xor(bv, m, 64);
      const int oe = __shfl_xor(be, m, 64);
      if (ov > bv || (ov == bv && oe < be)) {
        bv = ov;
        be = oe;
      }
    }
    sel[j] = bv;
    sid[j] = be;
    for (int i = 0; i < per; ++i)
      if (lane + 64 * i == be) v[i] = -INFINITY;
  }
  if (lane == 0) {
    const float mx = sel[0];
    float s = 0.f;
    float ex[16];
    for (int j = 0; j < k; ++j) {
      ex[j] = expf(sel[j] - mx);
      s += ex[j];
    }
    const float inv = 1.0f / s;
    for (int j = 0; j < k; ++j) {
      ids[t * k + j] = sid[j];
      w[t * k + j] = ex[j] * inv;
    }
  }
}

__global__ __launch_bounds__(256) void moe_count_kernel(const int32_t* ids, int64_t n,
                                                        int64_t* counts) {
  __shared__ float red[4];
  const int e = blockIdx.x;
  float c = 0.f;
  for (int64_t i = threadIdx.x; i < n; i += 256) c += (ids[i] == e) ? 1.f : 0.f;
  // counts up to 2^24 are exact in fp32
  c = block_sum<256>(c, red);
  if (threadIdx.x == 0) counts[e] = (int64_t)c;
}

__global__ void moe_offsets_kernel(const int64_t* counts, int E, int64_t* off) {
  if (threadIdx.x != 0) return;
  int64_t acc = 0;
  off[0] = 0;
  for (int e = 0; e < E; ++e) {
    acc += counts[e];
    off[e + 1] = acc;
  }
}

// Rank of every (token, slot) inside its expert, in token order.
__global__ __launch_bounds__(256) void moe_rank_kernel(const int32_t* ids, int64_t n,
                                                       const int64_t* off, int32_t* perm_row) {
  __shared__ int scan[256];
  const int e = blockIdx.x;
  int64_t base = off[e];
  for (int64_t c0 = 0; c0 < n; c0 += 256) {
    const int64_t i = c0 + threadIdx.x;
    const int f = (i < n && ids[i] == e) ? 1 : 0;
    scan[threadIdx.x] = f;
    __syncthreads();
    for (int s = 1; s < 256; s <<= 1) {
      const int v = (int)threadIdx.x >= s ? scan[threadIdx.x - s] : 0;
      __syncthreads();
      scan[threadIdx.x] += v;
      __syncthreads();
    }
    if (f) perm_row[i] = (int32_t)(base + scan[threadIdx.x] - 1);
    const int total = scan[255];
    __syncthreads();
    base += total;
  }
}

__global__ __launch_bounds__(256) void moe_gather_kernel(const bf16* x, const int32_t* perm,
                                                         int k, int64_t h, bf16* xg) {
  const int64_t tj = blockIdx.x;  // token*k + slot
  const int64_t t = tj / k;
  const int64_t dst = perm[tj];
  for (int64_t c = (int64_t)blockIdx.y * 256 + threadIdx.x; c < h / 8; c += (int64_t)gridDim.y * 256)
    *reinterpret_cast<u32x4*>(xg + dst * h + c * 8) =
        *reinterpret_cast<const u32x4*>(x + t * h + c * 8);
}

template <typename YT>
__global__ __launch_bounds__(256) void moe_combine_kernel(const bf16* yg, const int32_t* perm,
                                                          const float* w, const YT* res, int k,
                                                          int64_t h, YT* y) {
  const int64_t t = blockIdx.x;
  for (int64_t c = (int64_t)blockIdx.y * 256 + threadIdx.x; c < h / 8; c += (int64_t)gridDim.y * 256) {
    float acc[8];
    if (res)
      load8<YT>(res + t * h + c * 8, acc);
    else
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = 0.f;
    for (int s = 0; s < k; ++s) {
      const int64_t r = perm[t * k + s];
      const float ww = w[t * k + s];
      float v[8];
      load8<bf16>(yg + r * h + c * 8, v);
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = fmaf(ww, v[j], acc[j]);
    }
    store8<YT>(y + t * h + c * 8, acc);
  }
}

__global__ __launch_bounds__(256) void moe_combine_bwd_kernel(const bf16* dy, const int32_t* perm,
                                                              const float* w, int k, int64_t h,
                                                              bf16* dyg) {
  const int64_t tj = blockIdx.x;
  const int64_t t = tj / k;
  const int64_t r = perm[tj];
  const float ww = w[tj];
  for (int64_t c = (int64_t)blockIdx.y * 256 + threadIdx.x; c < h / 8; c += (int64_t)gridDim.y * 256) {
    float v[8];
    load8<bf16>(dy + t * h + c * 8, v);
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] *= ww;
    store8<bf16>(dyg + r * h + c * 8, v);
  }
}

__global__ __launch_bounds__(256) void moe_scatter_add_kernel(const bf16* dxg, const int32_t* perm,
                                                              int k, int64_t h, bf16* dx) {
  const int64_t t = blockIdx.x;
  for (int64_t c = (int64_t)blockIdx.y * 256 + threadIdx.x; c < h / 8; c += (int64_t)gridDim.y * 256) {
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < k; ++s) {
      const int64_t r = perm[t * k + s];
      float v[8];
      load8<bf16>(dxg + r * h + c * 8, v);
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] += v[j];
    }
    store8<bf16>(dx + t * h + c * 8, acc);
  }
}

static unsigned chunks_y(int64_t h) {
  const int64_t c = (h / 8 + 255) / 256;
  return (unsigned)(c < 1 ? 1 : c);
}

}  // namespace catq

using namespace catq;

extern "C" catq_status catq_aux_rmsnorm_fwd(const void* x, catq_dtype x_dtype, int64_t rows,
                                            int64_t n, float eps, void* y, float* rstd,
                                            hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(dtype_ok(x_dtype), CATQ_ERR_DTYPE, "bad dtype");
  CATQ_REQUIRE(x && y, CATQ_ERR_NULL, "x and y must not be NULL");
  CATQ_REQUIRE(count_ok(rows, n) && n % 8 == 0, CATQ_ERR_SHAPE,
               "need rows > 0, n a multiple of 8 and rows*n <= 2^38");
  CATQ_REQUIRE(eps >= 0, CATQ_ERR_VALUE, "eps must be >= 0");
  CATQ_REQUIRE(aligned16(x) && aligned16(y), CATQ_ERR_ALIGN, "misaligned");
  const double xs = x_dtype == CATQ_BF16 ? 2.0 : 4.0;
  const double by = (double)rows * n * (xs + 2.0) + (rstd ? 4.0 * rows : 0.0);
  if (x_dtype == CATQ_BF16)
    CATQ_TRACED(stream, "rmsnorm_fwd_kernel<__bf16>", 0.0, by, rows, n, 0,
                hipLaunchKernelGGL(rmsnorm_fwd_kernel<bf16>, dim3((unsigned)rows), dim3(256), 0,
                                   stream, (const bf16*)x, n, eps, (bf16*)y, rstd));
  else
    CATQ_TRACED(stream, "rmsnorm_fwd_kernel<float>", 0.0, by, rows, n, 0,
                hipLaunchKernelGGL(rmsnorm_fwd_kernel<float>, dim3((unsigned)rows), dim3(256), 0,
                                   stream, (const float*)x, n, eps, (bf16*)y, rstd));
  CATQ_CHECK_LAUNCH("rmsnorm fwd");
  return CATQ_OK;
}

extern "C" catq_status catq_aux_rmsnorm_bwd(const void* x, catq_dtype x_dtype, const float* rstd,
                                            const void* dy, const void* dres, int64_t rows,
                                            int64_t n, void* dx, hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(dtype_ok(x_dtype), CATQ_ERR_DTYPE, "bad dtype");
  CATQ_REQUIRE(x && rstd && dy && dx, CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(count_ok(rows, n) && n % 8 == 0, CATQ_ERR_SHAPE,
               "need rows > 0, n a multiple of 8 and rows*n <= 2^38");
  CATQ_REQUIRE(aligned16(x) && aligned16(dy) && aligned16(dres) && aligned16(dx), CATQ_ERR_ALIGN,
               "misaligned");
  const double xs = x_dtype == CATQ_BF16 ? 2.0 : 4.0;
  const double by = (double)rows * n * (xs + 2.0 + (dres ? 2.0 : 0.0) + 2.0) + 4.0 * rows;
  if (x_dtype == CATQ_BF16)
    CATQ_TRACED(stream, "rmsnorm_bwd_kernel<__bf16>", 0.0, by, rows, n, 0,
                hipLaunchKernelGGL(rmsnorm_bwd_kernel<bf16>, dim3((unsigned)rows), dim3(256), 0,
                                   stream, (const bf16*)x, rstd, (const bf16*)dy,
                                   (const bf16*)dres, n, (bf16*)dx));
  else
    CATQ_TRACED(stream, "rmsnorm_bwd_kernel<float>", 0.0, by, rows, n, 0,
                hipLaunchKernelGGL(rmsnorm_bwd_kernel<float>, dim3((unsigned)rows), dim3(256), 0,
                                   stream, (const float*)x, rstd, (const bf16*)dy,
                                   (const bf16*)dres, n, (bf16*)dx));
  CATQ_CHECK_LAUNCH("rmsnorm bwd");
  return CATQ_OK;
}

extern "C" catq_status catq_aux_act_quant(const void* x, catq_dtype x_dtype, int64_t rows,
                                          int64_t n, int64_t group, void* y,
                                          hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(rows >= 0, CATQ_ERR_SHAPE, "rows must be >= 0");
  if (rows == 0) return CATQ_OK;
  CATQ_REQUIRE(x && y, CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(dtype_ok(x_dtype), CATQ_ERR_DTYPE, "x must be bf16 or fp32");
  CATQ_REQUIRE(n > 0 && group > 0 && n % group == 0 && group % 8 == 0, CATQ_ERR_SHAPE,
               "group must be a multiple of 8 dividing n");
  CATQ_REQUIRE(rows <= INT32_MAX && n / group <= 65535 && count_ok(rows, n), CATQ_ERR_SHAPE,
               "too many rows or groups");
  CATQ_REQUIRE(aligned16(x) && aligned16(y), CATQ_ERR_ALIGN, "misaligned");
  CATQ_REQUIRE(x_dtype == CATQ_BF16 || x != y, CATQ_ERR_VALUE,
               "an fp32 input cannot be quantized in place (y is bf16)");
  const dim3 grid((unsigned)rows, (unsigned)(n / group));
  const double bytes = (double)rows * (double)n * (2.0 * dtype_size(x_dtype) + 2.0);
  if (x_dtype == CATQ_BF16)
    CATQ_TRACED(stream, "act_quant_kernel<bf16>", 0.0, bytes, rows, n, group,
                hipLaunchKernelGGL(act_quant_kernel<bf16>, grid, dim3(256), 0, stream,
                                   (const bf16*)x, n, group, (bf16*)y));
  else
    CATQ_TRACED(stream, "act_quant_kernel<float>", 0.0, bytes, rows, n, group,
                hipLaunchKernelGGL(act_quant_kernel<float>, grid, dim3(256), 0, stream,
                                   (const float*)x, n, group, (bf16*)y));
  CATQ_CHECK_LAUNCH("act quant");
  return CATQ_OK;
}

extern "C" catq_status catq_aux_swiglu_fwd(const void* gu, int64_t rows, int64_t F, void* a,
                                           hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(gu && a, CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(count_ok(rows, 2 * F) && F % 8 == 0, CATQ_ERR_SHAPE,
               "need rows > 0, F a multiple of 8 and rows*2F <= 2^38");
  CATQ_REQUIRE(aligned16(gu) && aligned16(a), CATQ_ERR_ALIGN, "misaligned");
  const int64_t n = rows * (F / 8);
  CATQ_TRACED(stream, "swiglu_fwd_kernel", 0.0, 6.0 * (double)rows * F, rows, F, 0,
              hipLaunchKernelGGL(swiglu_fwd_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256),
                                 0, stream, (const bf16*)gu, rows, F, (bf16*)a));
  CATQ_CHECK_LAUNCH("swiglu fwd");
  return CATQ_OK;
}

extern "C" catq_status catq_aux_swiglu_bwd(const void* gu, const void* da, int64_t rows, int64_t F,
                                           void* dgu, hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(gu && da && dgu, CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(count_ok(rows, 2 * F) && F % 8 == 0, CATQ_ERR_SHAPE,
               "need rows > 0, F a multiple of 8 and rows*2F <= 2^38");
  CATQ_REQUIRE(aligned16(gu) && aligned16(da) && aligned16(dgu), CATQ_ERR_ALIGN, "misaligned");
  const int64_t n = rows * (F / 8);
  CATQ_TRACED(stream, "swiglu_bwd_kernel", 0.0, 10.0 * (double)rows * F, rows, F, 0,
              hipLaunchKernelGGL(swiglu_bwd_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256),
                                 0, stream, (const bf16*)gu, (const bf16*)da, rows, F, (bf16*)dgu));
  CATQ_CHECK_LAUNCH("swiglu bwd");
  return CATQ_OK;
}

extern "C" size_t catq_aux_moe_route_workspace_bytes(int64_t T, int32_t E, int32_t k) {
  (void)T;
  (void)k;
  return round_up((size_t)(E > 0 ? E : 1) * sizeof(int64_t), 256);
}

extern "C" catq_status catq_aux_moe_route(const float* logits, int64_t T, int32_t E, int32_t k,
                                          int32_t* expert_ids, float* weights, int32_t* perm_row,
                                          int64_t* row_offsets, void* workspace,
                                          size_t workspace_bytes, hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(logits && expert_ids && weights && perm_row && row_offsets && workspace,
               CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(T > 0 && E > 0 && E <= 1024 && k >= 1 && k <= 16 && k <= E, CATQ_ERR_SHAPE,
               "need T > 0, 1 <= k <= min(16, E), E <= 1024");
  CATQ_REQUIRE(count_ok(T, k) && T * k < (int64_t)1 << 31 && count_ok(T, E), CATQ_ERR_SHAPE,
               "too many routed rows");
  CATQ_REQUIRE(workspace_bytes >= catq_aux_moe_route_workspace_bytes(T, E, k), CATQ_ERR_WORKSPACE,
               "workspace too small");
  int64_t* counts = reinterpret_cast<int64_t*>(workspace);
  hipLaunchKernelGGL(moe_topk_kernel, dim3((unsigned)((T + 3) / 4)), dim3(256), 0, stream, logits,
                     T, E, k, expert_ids, weights);
  CATQ_CHECK_LAUNCH("moe top-k");
  hipLaunchKernelGGL(moe_count_kernel, dim3((unsigned)E), dim3(256), 0, stream, expert_ids, T * k,
                     counts);
  CATQ_CHECK_LAUNCH("moe count");
  hipLaunchKernelGGL(moe_offsets_kernel, dim3(1), dim3(64), 0, stream, counts, E, row_offsets);
  CATQ_CHECK_LAUNCH("moe offsets");
  hipLaunchKernelGGL(moe_rank_kernel, dim3((unsigned)E), dim3(256), 0, stream, expert_ids, T * k,
                     row_offsets, perm_row);
  CATQ_CHECK_LAUNCH("moe rank");
  return CATQ_OK;
}

extern "C" catq_status catq_aux_moe_gather(const void* x, const int32_t* perm_row, int64_t T,
                                           int32_t k, int64_t h, void* xg, hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(x && perm_row && xg, CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(count_ok(T, k, h) && h % 8 == 0, CATQ_ERR_SHAPE,
               "need T, k, h > 0, h a multiple of 8 and T*k*h <= 2^38");
  CATQ_REQUIRE(aligned16(x) && aligned16(xg), CATQ_ERR_ALIGN, "misaligned");
  hipLaunchKernelGGL(moe_gather_kernel, dim3((unsigned)(T * k), chunks_y(h)), dim3(256), 0, stream,
                     (const bf16*)x, perm_row, k, h, (bf16*)xg);
  CATQ_CHECK_LAUNCH("moe gather");
  return CATQ_OK;
}

extern "C" catq_status catq_aux_moe_combine(const void* yg, const int32_t* perm_row,
                                            const float* weights, const void* res, int64_t T,
                                            int32_t k, int64_t h, void* y, catq_dtype y_dtype,
                                            hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(dtype_ok(y_dtype), CATQ_ERR_DTYPE, "bad dtype");
  CATQ_REQUIRE(yg && perm_row && weights && y, CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(count_ok(T, k, h) && h % 8 == 0, CATQ_ERR_SHAPE,
               "need T, k, h > 0, h a multiple of 8 and T*k*h <= 2^38");
  CATQ_REQUIRE(aligned16(yg) && aligned16(res) && aligned16(y), CATQ_ERR_ALIGN, "misaligned");
  if (y_dtype == CATQ_BF16)
    hipLaunchKernelGGL(moe_combine_kernel<bf16>, dim3((unsigned)T, chunks_y(h)), dim3(256), 0,
                       stream, (const bf16*)yg, perm_row, weights, (const bf16*)res, k, h,
                       (bf16*)y);
  else
    hipLaunchKernelGGL(moe_combine_kernel<float>, dim3((unsigned)T, chunks_y(h)), dim3(256), 0,
                       stream, (const bf16*)yg, perm_row, weights, (const float*)res, k, h,
                       (float*)y);
  CATQ_CHECK_LAUNCH("moe combine");
  return CATQ_OK;
}

extern "C" catq_status catq_aux_moe_combine_bwd(const void* dy, const int32_t* perm_row,
                                                const float* weights, int64_t T, int32_t k,
                                                int64_t h, void* dyg, hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(dy && perm_row && weights && dyg, CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(count_ok(T, k, h) && h % 8 == 0, CATQ_ERR_SHAPE,
               "need T, k, h > 0, h a multiple of 8 and T*k*h <= 2^38");
  CATQ_REQUIRE(aligned16(dy) && aligned16(dyg), CATQ_ERR_ALIGN, "misaligned");
  hipLaunchKernelGGL(moe_combine_bwd_kernel, dim3((unsigned)(T * k), chunks_y(h)), dim3(256), 0,
                     stream, (const bf16*)dy, perm_row, weights, k, h, (bf16*)dyg);
  CATQ_CHECK_LAUNCH("moe combine bwd");
  return CATQ_OK;
}

extern "C" catq_status catq_aux_moe_scatter_add(const void* dxg, const int32_t* perm_row, int64_t T,
                                                int32_t k, int64_t h, void* dx,
                                                hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(dxg && perm_row && dx, CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(count_ok(T, k, h) && h % 8 == 0, CATQ_ERR_SHAPE,
               "need T, k, h > 0, h a multiple of 8 and T*k*h <= 2^38");
  CATQ_REQUIRE(aligned16(dxg) && aligned16(dx), CATQ_ERR_ALIGN, "misaligned");
  hipLaunchKernelGGL(moe_scatter_add_kernel, dim3((unsigned)T, chunks_y(h)), dim3(256), 0, stream,
                     (const bf16*)dxg, perm_row, k, h, (bf16*)dx);
  CATQ_CHECK_LAUNCH("moe scatter add");
  return CATQ_OK;
}
