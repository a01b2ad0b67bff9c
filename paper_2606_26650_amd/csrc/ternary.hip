// Packed-ternary linear for deployment: Y = X · (alpha ⊙ T)ᵀ read straight
// from the 2-bit storage of the final ternarisation (App. B.2: ternary codes
// plus one scale per group, no zero point), so a decode step streams 2 bits
// per weight (+ 32 bits per group) from HBM instead of 16.
//
// Layout consumed (the one catq_pack_ternary writes): code c = T + 1 in
// {0, 1, 2}; byte b of row n holds elements 4b..4b+3, element 4b+j in bits
// 2j..2j+1; alpha fp32 [d_out][d_in / g].  Code 3 (invalid) contributes 0.
//
// gfx950 design.  One workgroup owns 16 (or 32) output rows and up to 16
// tokens; its waves split the rows' 128-code chunks round robin and are
// reduced through LDS in a fixed order (deterministic, no atomics).  Per chunk a lane loads
// 8 bytes (32 codes) of its row, turns them into four MFMA operands of bf16
// values 2T in {-2, 0, +2} with two byte-permute table lookups per four
// codes (the low byte of ±2 and 0 in bf16 is 0, so only the high byte needs
// a table), and issues four v_mfma_f32_16x16x32_bf16 against the matching
// 64 contiguous bytes of X.  The operand order is the natural k order, so X
// is loaded as is.  The chunk's 4 partial outputs per lane are scaled by
// alpha/2 (the factor 2 of the decode is exact) and accumulated in fp32.
// The scales of the workgroup's rows are staged in LDS once.

#include <type_traits>

#include "catq_internal.h"
#include "kernels.h"

namespace catq {
namespace {

struct TernArgs {
  const bf16* X;
  int64_t ldx, M;
  const uint8_t* P;
  const float* A;
  int64_t d_out, d_in, ldy;
  int32_t n_chunks;   // d_in / 128
  int32_t cpg_shift;  // log2(g / 128)
  void* Y;
};

// High byte of the bf16 value 2T for code c: c=0 -> -2 (0xC000), c=1 -> 0,
// c=2 -> +2 (0x4000), c=3 -> 0.
constexpr uint32_t kHiTab = 0x004000C0u;

// 16 codes (code i in bits 2i..2i+1 of w) -> 16 bf16 values 2T in k order:
// lo = codes 0..7, hi = codes 8..15.
__device__ __forceinline__ void decode16(uint32_t w, u32x4& lo, u32x4& hi) {
  const uint32_t h0 = __builtin_amdgcn_perm(0u, kHiTab, w & 0x03030303u);          // 0 4 8 12
  const uint32_t h1 = __builtin_amdgcn_perm(0u, kHiTab, (w >> 2) & 0x03030303u);   // 1 5 9 13
  const uint32_t h2 = __builtin_amdgcn_perm(0u, kHiTab, (w >> 4) & 0x03030303u);   // 2 6 10 14
  const uint32_t h3 = __builtin_amdgcn_perm(0u, kHiTab, (w >> 6) & 0x03030303u);   // 3 7 11 15
  // bytes 0 and 2 of each word are 0 (selector 0x0C); bytes 1 and 3 take the
  // high bytes of two consecutive codes (selector 0..3 from the second
  // operand, 4..7 from the first)
  lo.x = __builtin_amdgcn_perm(h1, h0, 0x040C000Cu);  // codes 0, 1
  lo.y = __builtin_amdgcn_perm(h3, h2, 0x040C000Cu);  // 2, 3
  lo.z = __builtin_amdgcn_perm(h1, h0, 0x050C010Cu);  // 4, 5
  lo.w = __builtin_amdgcn_perm(h3, h2, 0x050C010Cu);  // 6, 7
  hi.x = __builtin_amdgcn_perm(h1, h0, 0x060C020Cu);  // 8, 9
  hi.y = __builtin_amdgcn_perm(h3, h2, 0x060C020Cu);  // 10, 11
  hi.z = __builtin_amdgcn_perm(h1, h0, 0x070C030Cu);  // 12, 13
  hi.w = __builtin_amdgcn_perm(h3, h2, 0x070C030Cu);  // 14, 15
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// f(integral constant I) for I = 0 .. N-1, expanded at compile time (keeps
// register arrays indexed by constants even where the unroller gives up)
template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

template <typename OutT>
__device__ __forceinline__ void store1(OutT* p, float v);
template <>
__device__ __forceinline__ void store1<float>(float* p, float v) {
  *p = v;
}
template <>
__device__ __forceinline__ void store1<bf16>(bf16* p, float v) {
  *p = (bf16)v;
}

constexpr int kMaxChunks = 512;        // d_in <= 65536
constexpr int kBufferFlags = 0x00020000;  // raw buffer resource word 3 (gfx9 family)
constexpr int kOutOfRange = 0x40000000;   // offset past every slice this kernel builds

// One workgroup = one tile of 16 output rows x up to 16 tokens; grid
// (ceil(d_out / 16), ceil(M / 16)).  Its NW waves split the rows' 128-code
// chunks (wave w: chunks w, w + NW, ...; MAXC at most per batch) and are
// reduced through LDS in a fixed order.
//  * Every code load of a batch is issued at once (raw buffer loads over the
//    tile's rows: wave-uniform base and chunk offset, no address arithmetic
//    per chunk; rows past d_out get an out-of-range offset and read zeros).
//  * The tile's scales are staged in LDS ([chunk][row], alpha/2) by a
//    shift-indexed loop whose loads are all in flight together with the
//    codes.
//  * X comes from L2 two chunks ahead with buffer loads whose absent tokens
//    (15 of 16 lanes at one token) are out of range: no traffic, no branch.
// Dynamic LDS: n_chunks * 16 floats.
template <int NW, int MAXC, typename OutT>
__global__ __launch_bounds__(NW * 64) void ternary_gemv_kernel(TernArgs a) {
  extern __shared__ __align__(16) float s_alpha[];
  __shared__ float s_red[NW][16][17];  // [wave][token][row]
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches
  const int q = lane >> 4, c16 = lane & 15;
  const int64_t n0 = (int64_t)blockIdx.x * 16;
  const int64_t m0 = (int64_t)blockIdx.y * 16;
  const int nch = a.n_chunks;
  const int64_t row_bytes = a.d_in >> 2;

  const int tok_here = (int)min<int64_t>(16, a.M - m0);
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16*>(a.X + m0 * a.ldx), 0, (int)(tok_here * a.ldx * 2), kBufferFlags);
  const int xoff = c16 < tok_here ? (int)((c16 * a.ldx + 32 * q) * 2) : kOutOfRange;
  const int rows_here = (int)min<int64_t>(16, a.d_out - n0);
  const __amdgpu_buffer_rsrc_t pr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(a.P + n0 * row_bytes), 0, (int)(rows_here * row_bytes), kBufferFlags);
  const int poff = c16 < rows_here ? (int)(c16 * row_bytes + 8 * q) : kOutOfRange;
  const int my_chunks = wave < nch ? (nch - wave + NW - 1) / NW : 0;
  const int last = wave + NW * (my_chunks - 1);
  const int n_batches = (my_chunks + MAXC - 1) / MAXC;

  uint2 cw[MAXC];
  auto load_batch = [&](int b) {
    static_for<0, MAXC>([&](auto I) {
      const int ch = min(wave + NW * (b * MAXC + I()), last);   // past the last: unused
      cw[I()] = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(pr, poff, ch * 32, 0));
    });
  };
  auto load_x = [&](int ch, u32x4* xv) {
#pragma unroll
    for (int j = 0; j < 4; ++j) xv[j] = __builtin_amdgcn_raw_buffer_load_b128(xr, xoff + 16 * j, ch * 256, 0);
  };
  if (n_batches > 0) load_batch(0);
  u32x4 xv[3][4];
  if (n_batches > 0) {
    load_x(wave, xv[0]);
    load_x(min(wave + NW, last), xv[1]);
  }

  // scales: thread handles row tid % 16 and chunks tid / 16 + k (NW * 4),
  // all loads first, then the stores
  {
    constexpr int CPI = NW * 4;               // chunks per pass over the threads
    constexpr int KA = (kMaxChunks + CPI - 1) / CPI;
    const int r = tid & 15;
    const int64_t row = n0 + r;
    const float* arow = a.A + (row < a.d_out ? row : 0) * (int64_t)(nch >> a.cpg_shift);
    const bool rok = row < a.d_out;
    const int npass = (nch + CPI - 1) / CPI;
    for (int p0 = 0; p0 < npass; p0 += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int ch = (tid >> 4) + CPI * (p0 + u);
        v[u] = (rok && ch < nch) ? 0.5f * arow[ch >> a.cpg_shift] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int ch = (tid >> 4) + CPI * (p0 + u);
        if (ch < nch) s_alpha[ch * 16 + r] = v[u];
      }
    }
    (void)KA;
  }
  __syncthreads();

  f32x4 out = {0.f, 0.f, 0.f, 0.f};
  static_assert(MAXC % 3 == 0, "the three X buffers rotate in step across batches");
  for (int b = 0; b < n_batches; ++b) {
    if (b > 0) load_batch(b);
    static_for<0, MAXC>([&](auto I) {
      constexpr int i = I();
      const int k = b * MAXC + i;
      if (k >= my_chunks) return;                  // wave-uniform
      const int ch = wave + NW * k;
      // X two chunks ahead (clamped to the wave's last chunk)
      load_x(min(ch + 2 * NW, last), xv[(i + 2) % 3]);
      const u32x4* xa = xv[i % 3];
      u32x4 w0, w1, w2, w3;
      decode16(cw[i].x, w0, w1);
      decode16(cw[i].y, w2, w3);
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(w0), as_bf16x8(xa[0]), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(w1), as_bf16x8(xa[1]), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(w2), as_bf16x8(xa[2]), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(w3), as_bf16x8(xa[3]), acc, 0, 0, 0);
      // accumulator: rows 4q..4q+3 of the tile, token c16
      const f32x4 al = *reinterpret_cast<const f32x4*>(&s_alpha[ch * 16 + 4 * q]);
      out[0] += al[0] * acc[0];
      out[1] += al[1] * acc[1];
      out[2] += al[2] * acc[2];
      out[3] += al[3] * acc[3];
    });
  }

  // fixed-order reduction over the waves
#pragma unroll
  for (int r = 0; r < 4; ++r) s_red[wave][c16][4 * q + r] = out[r];
  __syncthreads();
  for (int i = tid; i < 256; i += NW * 64) {
    const int tok = i >> 4, r = i & 15;
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) sum += s_red[w][tok][r];
    if (tok < tok_here && r < rows_here)
      store1<OutT>(reinterpret_cast<OutT*>(a.Y) + (m0 + tok) * a.ldy + n0 + r, sum);
  }
}

template <int NW, int MAXC>
catq_status launch_tern(const TernArgs& a, catq_dtype y_dtype, hipStream_t stream) {
  const dim3 grid((unsigned)((a.d_out + 15) / 16), (unsigned)((a.M + 15) / 16));
  const size_t lds = (size_t)a.n_chunks * 16 * sizeof(float);
  const double flops = 2.0 * (double)a.M * (double)a.d_out * (double)a.d_in;
  const double bytes = (double)a.d_out * (double)a.d_in / 4.0 +
                       4.0 * (double)a.d_out * (double)(a.n_chunks >> a.cpg_shift) +
                       2.0 * (double)a.M * (double)a.d_in +
                       (double)a.M * (double)a.d_out * (y_dtype == CATQ_F32 ? 4.0 : 2.0);
  static char tag[64];
  snprintf(tag, sizeof tag, "ternary_gemv_kernel<%d, %d>", NW, MAXC);
  if (y_dtype == CATQ_F32) {
    CATQ_TRACED(stream, tag, flops, bytes, a.M, a.d_out, a.d_in,
                hipLaunchKernelGGL((ternary_gemv_kernel<NW, MAXC, float>), grid, dim3(NW * 64),
                                   lds, stream, a));
  } else {
    CATQ_TRACED(stream, tag, flops, bytes, a.M, a.d_out, a.d_in,
                hipLaunchKernelGGL((ternary_gemv_kernel<NW, MAXC, bf16>), grid, dim3(NW * 64),
                                   lds, stream, a));
  }
  CATQ_CHECK_LAUNCH("ternary_linear");
  return CATQ_OK;
}

}  // namespace
}  // namespace catq

extern "C" catq_status catq_ternary_linear(const void* X, int64_t M, int64_t ldx,
                                           const uint8_t* packed, const float* alpha,
                                           int64_t d_out, int64_t d_in, int32_t g, void* Y,
                                           catq_dtype y_dtype, int64_t ldy, hipStream_t stream) {
  using namespace catq;
  clear_error();
  CATQ_REQUIRE(M >= 0, CATQ_ERR_SHAPE, "M must be >= 0");
  if (M == 0) return CATQ_OK;
  CATQ_REQUIRE(X && packed && alpha && Y, CATQ_ERR_NULL, "X, packed, alpha and Y must not be NULL");
  CATQ_REQUIRE(count_ok(d_out, d_in), CATQ_ERR_SHAPE,
               "d_out and d_in must be > 0 with d_out*d_in <= 2^38");
  CATQ_REQUIRE(g >= 128 && g % 128 == 0 && ((g / 128) & (g / 128 - 1)) == 0, CATQ_ERR_VALUE,
               "g must be 128 times a power of two");
  CATQ_REQUIRE(d_in % g == 0, CATQ_ERR_SHAPE, "d_in (%lld) must be a multiple of g (%d)",
               (long long)d_in, g);
  CATQ_REQUIRE(d_in <= 128 * (int64_t)kMaxChunks, CATQ_ERR_SHAPE, "d_in must be <= %d",
               128 * kMaxChunks);
  CATQ_REQUIRE((d_out + 15) / 16 <= INT32_MAX && (M + 15) / 16 <= 65535, CATQ_ERR_SHAPE,
               "d_out or M too large for one launch");
  CATQ_REQUIRE(ldx >= d_in && ldx % 8 == 0 && ldx <= (1 << 24), CATQ_ERR_SHAPE,
               "ldx must be >= d_in, a multiple of 8 and <= 2^24");
  CATQ_REQUIRE(ldy >= d_out, CATQ_ERR_SHAPE, "ldy must be >= d_out");
  CATQ_REQUIRE(y_dtype == CATQ_F32 || y_dtype == CATQ_BF16, CATQ_ERR_DTYPE,
               "Y must be fp32 or bf16");
  CATQ_REQUIRE(aligned16(X) && aligned16(alpha) && (reinterpret_cast<uintptr_t>(packed) & 7) == 0 &&
                   (reinterpret_cast<uintptr_t>(Y) & 3) == 0,
               CATQ_ERR_ALIGN, "X and alpha must be 16-byte aligned, packed 8-byte, Y 4-byte");
  TernArgs a{};
  a.X = static_cast<const bf16*>(X);
  a.ldx = ldx;
  a.M = M;
  a.P = packed;
  a.A = alpha;
  a.d_out = d_out;
  a.d_in = d_in;
  a.ldy = ldy;
  a.n_chunks = (int32_t)(d_in / 128);
  a.cpg_shift = __builtin_ctz((unsigned)(g / 128));
  a.Y = Y;
  // few long waves: all of a wave's chunks (up to 21) in one batch
  if (a.n_chunks <= 42) return launch_tern<2, 21>(a, y_dtype, stream);
  if (a.n_chunks <= 84) return launch_tern<4, 21>(a, y_dtype, stream);
  if (a.n_chunks <= 168) return launch_tern<8, 21>(a, y_dtype, stream);
  return launch_tern<16, 21>(a, y_dtype, stream);
}
