// Packed-ternary linear for deployment: Y = X · (alpha ⊙ T)ᵀ read straight
// from the 2-bit storage of the final ternarisation (App. B.2: ternary codes
// plus one scale per group, no zero point), so a decode step streams 2 bits
// per weight (+ 32 bits per group) from HBM instead of 16.
//
// Layout consumed (the one catq_pack_ternary writes): code c = T + 1 in
// {0, 1, 2}; byte b of row n holds elements 4b..4b+3, element 4b+j in bits
// 2j..2j+1; alpha fp32 [d_out][d_in / g].  Code 3 (invalid) contributes 0.
//
// gfx950 design.  One workgroup owns R tiles of 16 output rows and up to 16
// tokens; its waves split the 128-code chunks round robin and are reduced
// through LDS in a fixed order (deterministic, no atomics).  Per chunk a lane
// loads 8 bytes (32 codes) of its row in each tile, turns them into four MFMA
// operands of bf16 values 2T in {-2, 0, +2} with two byte-permute table
// lookups per four codes (the low byte of +-2 and 0 in bf16 is 0, so only the
// high byte needs a table), and issues four v_mfma_f32_16x16x32_bf16 per tile
// against the matching 64 contiguous bytes of X, loaded once for all R tiles.
// The operand order is the natural k order, so X is loaded as is.  The chunk's
// 4 partial outputs per lane and tile are scaled by alpha/2 (the factor 2 of
// the decode is exact) and accumulated in fp32.  The scales of the
// workgroup's rows are staged in LDS once.
//
// Prefill-sized M takes a second kernel (ternary_gemm_kernel below) whose
// workgroups tile 128 rows x 64 or 128 tokens, so each code is decoded once
// per tile; the host picks the kernel by a fitted cost model.

#include <algorithm>
#include <cmath>
#include <cstdint>
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

// One workgroup = R tiles of 16 output rows (RT = 16 R rows) x up to 16
// tokens; grid (ceil(d_out / RT), ceil(M / 16)).  Its NW waves split the
// 128-code chunks (wave w: chunks w, w + NW, ...) and are reduced through LDS
// in a fixed order.
//  * X crosses the vector memory path once per chunk and wave and serves all
//    R tiles (at one token, 15 of the 16 token lanes read out of range: no
//    traffic, but the lanes still return data, so that return is shared);
//    with up to four tokens (XL) it is instead copied into LDS once.
//  * The codes and X of chunk k + D are issued while chunk k is multiplied:
//    a ring of D + 1 register slots keeps D chunks of every wave in flight.
//    Code loads are raw buffer loads over the tile's rows (wave-uniform base
//    and chunk offset; rows past d_out read zeros).
//  * The tile's scales ([chunk][row], alpha/2) are loaded first, coalesced
//    along each row (at most AMAX per thread, all in flight with the first D
//    chunks), and stored to LDS; the barrier before the products waits for
//    LDS only, not for the code loads in flight.  With one scale per chunk
//    and whole quads of chunks per row (VEC), a thread takes four
//    consecutive scales of a row per 16-byte load (AMAX / 4 loads).
// Dynamic LDS: n_chunks * (RT + 4) floats.
template <int NW, int R, int D, int AMAX, bool VEC, bool XL, typename OutT>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(4)))
void ternary_gemv_kernel(TernArgs a) {
  constexpr int RT = 16 * R;   // rows of the workgroup
  constexpr int AP = RT + 4;   // pitch of the staged scales (floats; 16-byte rows)
  constexpr int S = D + 1;     // register slots of the ring
  extern __shared__ __align__(16) float s_alpha[];
  // [wave][token][row] partial outputs; with X in LDS they reuse its space
  __shared__ float s_red_own[XL ? 1 : NW][16][RT + 1];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches
  const int q = lane >> 4, c16 = lane & 15;
  const int64_t n0 = (int64_t)blockIdx.x * RT;
  const int64_t m0 = (int64_t)blockIdx.y * 16;
  const int nch = a.n_chunks;
  const int64_t row_bytes = a.d_in >> 2;

  const int tok_here = (int)min<int64_t>(16, a.M - m0);
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16*>(a.X + m0 * a.ldx), 0, (int)(tok_here * a.ldx * 2), kBufferFlags);
  const int xoff = c16 < tok_here ? (int)((c16 * a.ldx + 32 * q) * 2) : kOutOfRange;
  // XL (at most four tokens): the workgroup's X rows are copied once into LDS
  // past the scales ([token][d_in] bf16, 16-byte slots, padded to whole
  // copies), before the scales are loaded, so that the wait for the scales
  // covers the copies; the ring then carries codes only, and the products
  // read X from LDS.  (Per chunk and wave, X loads cost as much as the codes
  // at one token, where 15 of 16 token lanes read nothing.)
  uint4* s_x = reinterpret_cast<uint4*>(s_alpha + a.n_chunks * AP);
  float (*s_red)[16][RT + 1] =
      XL ? reinterpret_cast<float (*)[16][RT + 1]>(s_x) : s_red_own;
  if constexpr (XL) {
    const i32x4_rsrc xb = buf_rsrc(a.X + m0 * a.ldx, (uint32_t)(tok_here * a.ldx * 2));
    const int row_slots = a.n_chunks * 16, slots = tok_here * row_slots;
    for (int i = wave; i * 64 < slots; i += NW) {
      const int sl = i * 64 + lane, t = sl / row_slots;
      const uint32_t off =
          sl < slots ? (uint32_t)(t * a.ldx * 2 + (sl - t * row_slots) * 16) : (uint32_t)kOutOfRange;
      dma16_buf(xb, off, 0u, s_x + i * 64);
    }
  }
  const int rows_here = (int)min<int64_t>(RT, a.d_out - n0);
  const __amdgpu_buffer_rsrc_t pr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(a.P + n0 * row_bytes), 0, (int)(rows_here * row_bytes), kBufferFlags);
  int poff[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int row = 16 * r + c16;
    poff[r] = row < rows_here ? (int)(row * row_bytes + 8 * q) : kOutOfRange;
  }
  const int my = wave < nch ? (nch - wave + NW - 1) / NW : 0;

  // scales: pair (row, chunk) = idx / nch, idx % nch (VEC: row and quad of
  // chunks, idx / (nch/4), idx % (nch/4)), consecutive threads along a row;
  // rows past d_out (and pairs past the tile) read zero through the buffer's
  // bound.  Loaded before the ring's first chunks and stored after them, so
  // both are in flight together.
  constexpr int NS = VEC ? (AMAX + 3) / 4 : AMAX;   // loads per thread
  constexpr int T = NW * 64;
  const int ng = nch >> a.cpg_shift;
  const int per_row = VEC ? nch >> 2 : nch;
  const __amdgpu_buffer_rsrc_t ar = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(a.A + n0 * ng), 0, rows_here * ng * 4, kBufferFlags);
  f32x4 av[NS];
#pragma unroll
  for (int u = 0; u < NS; ++u) {
    const int idx = tid + T * u;
    if constexpr (VEC) {
      av[u] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(ar, idx * 16, 0, 0));
    } else {
      const int r = idx / per_row, ch = idx - r * per_row;
      av[u][0] = __builtin_bit_cast(
          float, __builtin_amdgcn_raw_buffer_load_b32(ar, (r * ng + (ch >> a.cpg_shift)) * 4, 0, 0));
    }
  }
  __builtin_amdgcn_sched_barrier(0);   // (the scheduler keeps each phase in program order)

  // chunk of the wave's k-th: clamped to its last (the ring's loads past the
  // end re-read it; a wave without chunks reads chunk 0), never multiplied
  const int last = my > 0 ? wave + NW * (my - 1) : 0;
  uint2 cw[S][R];
  [[maybe_unused]] u32x4 xv[S][4];
  auto issue = [&](int k, auto slot_c) {
    constexpr int s = decltype(slot_c)::value;
    const int ch = min(wave + NW * k, last);
    if constexpr (!XL) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        xv[s][j] = __builtin_amdgcn_raw_buffer_load_b128(xr, xoff + 16 * j, ch * 256, 0);
    }
#pragma unroll
    for (int r = 0; r < R; ++r)
      cw[s][r] = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(pr, poff[r], ch * 32, 0));
  };
  static_for<0, D>([&](auto I) {
    issue(I(), I);
    __builtin_amdgcn_sched_barrier(0);   // (same load order as in the ring)
  });

#pragma unroll
  for (int u = 0; u < NS; ++u) {   // pairs past the tile: the unread pad column
    const int idx = tid + T * u;
    const int r = idx / per_row, c = idx - r * per_row;
    if constexpr (VEC) {
#pragma unroll
      for (int e = 0; e < 4; ++e) s_alpha[(4 * c + e) * AP + min(r, RT)] = 0.5f * av[u][e];
    } else {
      s_alpha[c * AP + min(r, RT)] = 0.5f * av[u][0];
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");

  f32x4 out[R];
#pragma unroll
  for (int r = 0; r < R; ++r) out[r] = f32x4{0.f, 0.f, 0.f, 0.f};
  // chunk k from slot k % S: four products per tile, scaled by the rows'
  // alpha/2 and accumulated
  auto compute = [&](int k, auto slot_c) {
    constexpr int i = decltype(slot_c)::value;
    const float* al = &s_alpha[(wave + NW * k) * AP + 4 * q];
    u32x4 xf[4];   // X of the chunk: lane (q, c16) holds token c16, k 32 q .. 32 q + 31
    if constexpr (XL) {
      const uint4* xp = s_x + min(c16, tok_here - 1) * (nch * 16) + (wave + NW * k) * 16 + 4 * q;
#pragma unroll
      for (int j = 0; j < 4; ++j) xf[j] = __builtin_bit_cast(u32x4, xp[j]);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) xf[j] = xv[i][j];
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      u32x4 w0, w1, w2, w3;
      decode16(cw[i][r].x, w0, w1);
      decode16(cw[i][r].y, w2, w3);
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(w0), as_bf16x8(xf[0]), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(w1), as_bf16x8(xf[1]), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(w2), as_bf16x8(xf[2]), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(w3), as_bf16x8(xf[3]), acc, 0, 0, 0);
      // accumulator: rows 16 r + 4q .. +3 of the workgroup, token c16
      const f32x4 sc = *reinterpret_cast<const f32x4*>(al + 16 * r);
#pragma unroll
      for (int e = 0; e < 4; ++e) out[r][e] += sc[e] * acc[e];
    }
  };
  // whole rounds of the ring without branches: chunk k + D issued into the
  // slot chunk k - 1 used, then chunk k multiplied
  const int full = my / S * S;
  for (int k0 = 0; k0 < full; k0 += S) {
    static_for<0, S>([&](auto I) {
      constexpr int i = I();
      issue(k0 + i + D, std::integral_constant<int, (i + D) % S>{});
      __builtin_amdgcn_sched_barrier(0);
      compute(k0 + i, I);
    });
  }
  // the last my - full (< S) chunks, already in flight
  static_for<0, S - 1>([&](auto I) {
    if (full + I() < my) compute(full + I(), I);
  });

  // fixed-order reduction over the waves (with X in LDS, once every wave has
  // finished reading it)
  if constexpr (XL) __syncthreads();
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int e = 0; e < 4; ++e) s_red[wave][c16][16 * r + 4 * q + e] = out[r][e];
  __syncthreads();
  for (int i = tid; i < 16 * RT; i += NW * 64) {
    const int tok = i / RT, r = i % RT;
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) sum += s_red[w][tok][r];
    if (tok < tok_here && r < rows_here)
      store1<OutT>(reinterpret_cast<OutT*>(a.Y) + (m0 + tok) * a.ldy + n0 + r, sum);
  }
}

// Prefill-sized M: one workgroup = a tile of 128 weight rows x TT tokens
// (TT = 128 or 64) on four waves (2 x 2, each 64 rows x TT/2 tokens), so a
// row's codes are decoded once per TT tokens instead of once per 16.  The
// 64-token tiles need fewer registers (three workgroups per compute unit
// instead of two) and give more workgroups on few rows.  Per 128-code chunk:
//  * the tile's X chunk (TT tokens x 128 k, bf16) arrives by direct copies
//    into a double-buffered LDS tile [token][16 slots of 8 k], slot s of
//    token t holding global slot s ^ (t & 15) (conflict-free fragment reads);
//  * a lane loads 32 bytes of codes of each of its two weight rows (one per
//    32-row block) and turns the half it needs of each word pair into two
//    MFMA operands (decode16 after one byte permute), in the natural k
//    order that the X fragments (16 bytes of a token row) share;
//  * eight k-steps of four v_mfma_f32_32x32x16_bf16 form the chunk's partial
//    products, which are scaled by the rows' alpha/2 (staged in LDS per
//    chunk) and accumulated in fp32, as in the decode kernel.
// The next chunk's copies, codes and scales are issued before the current
// chunk is multiplied.  Rows past d_out read zero codes and tokens past M
// zero X; neither is stored.  X offsets are 32-bit: 128 * ldx * 2 < 2^32.
constexpr int kGT = 128;

template <int TT, typename OutT>
__global__ __launch_bounds__(256, TT == 128 ? 2 : 3) void ternary_gemm_kernel(TernArgs a) {
  constexpr int CB = TT / 64;    // 32-token blocks per wave
  constexpr int NI = TT / 16;    // copy instructions per wave and chunk
  __shared__ __align__(16) uint4 s_x[2][TT * 16];   // [buffer][token * 16 + slot]
  __shared__ __align__(16) float s_al[2][kGT];      // [buffer][row]: alpha/2 of one chunk
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave & 1, wc = wave >> 1;  // 64-row and TT/2-token half of the tile
  const int h = lane >> 5, l32 = lane & 31;
  const int64_t n0 = (int64_t)blockIdx.x * kGT, m0 = (int64_t)blockIdx.y * TT;
  const int nch = a.n_chunks;
  const int64_t row_bytes = a.d_in >> 2;
  const int tok_here = (int)min<int64_t>(TT, a.M - m0);
  const int rows_here = (int)min<int64_t>(kGT, a.d_out - n0);
  const int ng = nch >> a.cpg_shift;

  // X copies: wave w fills tokens TT/4 w .. TT/4 (w + 1) - 1, four per instruction;
  // the lane's part of the offset repeats every four instructions (the
  // swizzle key is t & 15), the rest is uniform
  const i32x4_rsrc xr = buf_rsrc(a.X + m0 * a.ldx, (uint32_t)(tok_here * a.ldx * 2));
  uint32_t xl[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int tq = lane >> 4, slot = lane & 15;
    xl[j] = (uint32_t)(tq * a.ldx * 2) + (uint32_t)((slot ^ ((4 * j + tq) & 15)) * 16);
  }
  const uint32_t xlds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint4*)&s_x[0][0];
  const uint32_t xrow = (uint32_t)(a.ldx * 2);
  // codes of the lane's rows 64 wr + 32 rb + l32
  const __amdgpu_buffer_rsrc_t pr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(a.P + n0 * row_bytes), 0, (int)(rows_here * row_bytes), kBufferFlags);
  uint32_t poff[2];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) poff[rb] = (uint32_t)((64 * wr + 32 * rb + l32) * row_bytes);
  // scales: thread t < 128 takes row t of the tile
  const __amdgpu_buffer_rsrc_t ar = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(a.A + n0 * ng), 0, rows_here * ng * 4, kBufferFlags);
  const uint32_t aoff = (uint32_t)(min(tid, kGT - 1) * ng * 4);

  auto issue_x = [&](int c, int buf) {
#pragma unroll
    for (int i = 0; i < NI; ++i)
      dma16_lds(xr, xl[i & 3], (uint32_t)c * 256u + (uint32_t)(TT / 4 * wave + 4 * i) * xrow,
                xlds0 + (uint32_t)(buf * TT * 16 + (TT / 4 * wave + 4 * i) * 16) * 16u);
  };
  u32x4 cw[2][2], cn[2][2];  // codes of this chunk and of the next: [row block][16-byte half]
  auto load_codes = [&](int c, u32x4 (&dst)[2][2]) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        dst[rb][j] = __builtin_amdgcn_raw_buffer_load_b128(pr, (int)(poff[rb] + 16 * j), c * 32, 0);
  };
  auto load_alpha = [&](int c) {
    return __builtin_bit_cast(
        float, __builtin_amdgcn_raw_buffer_load_b32(ar, (int)(aoff + (uint32_t)(c >> a.cpg_shift) * 4u),
                                                    0, 0));
  };
  // vmcnt(0) as an s_waitcnt the compiler sees: the copies above are inline
  // assembly it does not count, so its own waits for the codes must know
  // that everything issued before has landed
  auto wait_all_vmem = [] { __builtin_amdgcn_s_waitcnt(0x0F70); };

  issue_x(0, 0);
  load_codes(0, cw);
  float av = load_alpha(0);
  wait_all_vmem();
  if (tid < kGT) s_al[0][tid] = 0.5f * av;
  __syncthreads();

  f32x16 out[2][CB];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) out[rb][cb][r] = 0.f;
  const uint32_t sel = h ? 0x07060302u : 0x05040100u;  // the lane's 16-bit half of two words
  int tr[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) tr[cb] = TT / 2 * wc + 32 * cb + l32;

  for (int c = 0; c < nch; ++c) {
    const int buf = c & 1;
    if (c + 1 < nch) {
      issue_x(c + 1, buf ^ 1);
      load_codes(c + 1, cn);
      av = load_alpha(c + 1);
    }
    const uint4* xt = s_x[buf];
    f32x16 acc[2][CB];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      bf16x8 A[2][2];  // [row block][k step of the pair]
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        const u32x4& q = cw[rb][p >> 1];
        const uint32_t t = __builtin_amdgcn_perm(q[(2 * p + 1) & 3], q[(2 * p) & 3], sel);
        u32x4 lo, hi;
        decode16(t, lo, hi);
        A[rb][0] = as_bf16x8(lo);
        A[rb][1] = as_bf16x8(hi);
      }
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int st = 2 * p + e;
        bf16x8 B[CB];
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
          B[cb] = __builtin_bit_cast(bf16x8, xt[tr[cb] * 16 + ((2 * st + h) ^ (tr[cb] & 15))]);
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int cb = 0; cb < CB; ++cb)
            acc[rb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                A[rb][e], B[cb], st == 0 ? f32x16{} : acc[rb][cb], 0, 0, 0);
      }
    }
    // out += (alpha/2 of the accumulator's rows) * acc; register r holds row
    // 8 (r / 4) + 4 h + r % 4 of its 32-row block
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const f32x4 sc =
            *reinterpret_cast<const f32x4*>(&s_al[buf][64 * wr + 32 * rb + 8 * qd + 4 * h]);
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            out[rb][cb][4 * qd + e] = fmaf(sc[e], acc[rb][cb][4 * qd + e], out[rb][cb][4 * qd + e]);
      }
    // the next chunk's copies, codes and scale have landed; this chunk's
    // buffers are free once every wave has passed the barrier
    wait_all_vmem();
    if (c + 1 < nch) {
      if (tid < kGT) s_al[buf ^ 1][tid] = 0.5f * av;
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int j = 0; j < 2; ++j) cw[rb][j] = cn[rb][j];
    }
    __syncthreads();
  }

  // Y[token][row]: lane column = token TT/2 wc + 32 cb + l32, register r = row
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int tok = tr[cb];
    if (tok >= tok_here) continue;
    OutT* yrow = reinterpret_cast<OutT*>(a.Y) + (m0 + tok) * a.ldy + n0;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 64 * wr + 32 * rb + 8 * (r >> 2) + 4 * h + (r & 3);
        if (row < rows_here) store1<OutT>(yrow + row, out[rb][cb][r]);
      }
  }
}

template <typename T>
struct OutTag {
  using type = T;
};

template <int NW, int R, int D, int AMAX>
catq_status launch_tern(const TernArgs& a, catq_dtype y_dtype, hipStream_t stream) {
  const bool vec = a.cpg_shift == 0 && a.n_chunks % 4 == 0;
  constexpr int RT = 16 * R;
  // every (row, chunk) scale pair of a tile has a thread slot, and the LDS
  // (scales + reduction) stays within 64 KB
  CATQ_REQUIRE((int64_t)a.n_chunks * RT <= (int64_t)AMAX * NW * 64 &&
                   (size_t)a.n_chunks * (RT + 4) * 4 + sizeof(float) * NW * 16 * (RT + 1) <= 65536,
               CATQ_ERR_SHAPE, "ternary_linear: no launch shape for d_in = %lld",
               (long long)a.d_in);
  const dim3 grid((unsigned)((a.d_out + RT - 1) / RT), (unsigned)((a.M + 15) / 16));
  const size_t lds_scales = (size_t)a.n_chunks * (RT + 4) * sizeof(float);
  // X in LDS for at most four tokens, where it fits beside the scales: whole
  // copies of 64 slots of 16 bytes
  // (the reduction's partial outputs then reuse the X space)
  const size_t red = sizeof(float) * NW * 16 * (RT + 1);
  const size_t lds_x = a.M <= 4 ? (size_t)((a.M * a.n_chunks * 16 + 63) / 64) * 64 * 16 : 0;
  const bool xl = lds_x > 0 && lds_scales + std::max(lds_x, red) <= 65536;
  const size_t lds = lds_scales + (xl ? std::max(lds_x, red) : 0);
  const double flops = 2.0 * (double)a.M * (double)a.d_out * (double)a.d_in;
  const double bytes = (double)a.d_out * (double)a.d_in / 4.0 +
                       4.0 * (double)a.d_out * (double)(a.n_chunks >> a.cpg_shift) +
                       2.0 * (double)a.M * (double)a.d_in +
                       (double)a.M * (double)a.d_out * (y_dtype == CATQ_F32 ? 4.0 : 2.0);
  static char tag[64];
  snprintf(tag, sizeof tag, "ternary_gemv_kernel<%d, %d, %d%s>", NW, R, D, xl ? ", x in lds" : "");
  auto launch = [&](auto vec_c, auto xl_c, auto out_c) {
    constexpr bool V = decltype(vec_c)::value, X = decltype(xl_c)::value;
    using OutT = typename decltype(out_c)::type;
    CATQ_TRACED(stream, tag, flops, bytes, a.M, a.d_out, a.d_in,
                hipLaunchKernelGGL((ternary_gemv_kernel<NW, R, D, AMAX, V, X, OutT>), grid,
                                   dim3(NW * 64), lds, stream, a));
  };
  auto with_out = [&](auto vec_c, auto xl_c) {
    if (y_dtype == CATQ_F32)
      launch(vec_c, xl_c, OutTag<float>{});
    else
      launch(vec_c, xl_c, OutTag<bf16>{});
  };
  using Tt = std::true_type;
  using Tf = std::false_type;
  if (vec) {
    if (xl) with_out(Tt{}, Tt{});
    else with_out(Tt{}, Tf{});
  } else {
    if (xl) with_out(Tf{}, Tt{});
    else with_out(Tf{}, Tf{});
  }
  CATQ_CHECK_LAUNCH("ternary_linear");
  return CATQ_OK;
}

// Which kernel: below 32 tokens always the decode kernel.  From there a
// cost model fitted to the kernels on MI355X picks the cheapest:
//  * tiled, TT tokens per tile: n_chunks x max(the chunk latency of a lone
//    workgroup, the workgroups on the fullest compute unit x what a unit
//    takes per workgroup and chunk); 1.45 / 1.23 us for 128-token tiles,
//    1.33 / 0.82 us for 64-token tiles;
//  * decode: ~7.5e-15 s per weight and token (rows over 64 chunks, whose
//    workgroups take eight waves, ~11e-15 s).
// 14B-shaped layers: gate|up tiled from 64 tokens, q|k|v and down from 256,
// o from 512; 64-token tiles for q|k|v and down at 256 tokens (53 against
// 66 us, 152 against 189) and gate|up at 64 (66 against 81), 128-token tiles
// from 512 (down 195 against 205, gate|up at 2048 839 against 1118 us).
// Returns 0 (decode), 64 or 128.
int pick_kernel(const TernArgs& a) {
  if (a.M < 32 || a.ldx > (1 << 23)) return 0;
  const double rows = (double)((a.d_out + kGT - 1) / kGT);
  auto tiled = [&](int tt, double lat, double thr) {
    const double wgs = rows * (double)((a.M + tt - 1) / tt);
    const double per = std::ceil(wgs / 256.0) * thr;
    return a.n_chunks * (per > lat ? per : lat);
  };
  const double t128 = tiled(128, 1.45, 1.23), t64 = tiled(64, 1.33, 0.82);
  const double decode =
      (double)a.M * (double)a.d_out * (double)a.d_in * (a.n_chunks > 64 ? 11e-9 : 7.5e-9);
  if (decode <= t128 && decode <= t64) return 0;
  return t64 < t128 ? 64 : 128;
}

template <int TT>
catq_status launch_tern_gemm(const TernArgs& a, catq_dtype y_dtype, hipStream_t stream) {
  const dim3 grid((unsigned)((a.d_out + kGT - 1) / kGT), (unsigned)((a.M + TT - 1) / TT));
  const double flops = 2.0 * (double)a.M * (double)a.d_out * (double)a.d_in;
  const double bytes = (double)grid.y * ((double)a.d_out * (double)a.d_in / 4.0 +
                                         4.0 * (double)a.d_out * (double)(a.n_chunks >> a.cpg_shift)) +
                       2.0 * (double)a.M * (double)a.d_in +
                       (double)a.M * (double)a.d_out * (y_dtype == CATQ_F32 ? 4.0 : 2.0);
  const char* tag = TT == 128 ? "ternary_gemm_kernel<128, 128>" : "ternary_gemm_kernel<128, 64>";
  if (y_dtype == CATQ_F32)
    CATQ_TRACED(stream, tag, flops, bytes, a.M, a.d_out, a.d_in,
                hipLaunchKernelGGL((ternary_gemm_kernel<TT, float>), grid, dim3(256), 0, stream, a));
  else
    CATQ_TRACED(stream, tag, flops, bytes, a.M, a.d_out, a.d_in,
                hipLaunchKernelGGL((ternary_gemm_kernel<TT, bf16>), grid, dim3(256), 0, stream, a));
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
  // Prefill-sized M: tiles of 128 rows x 64 or 128 tokens decode each code
  // once per tile (their X offsets need 128 * ldx * 2 < 2^32).
  switch (pick_kernel(a)) {
    case 128: return launch_tern_gemm<128>(a, y_dtype, stream);
    case 64: return launch_tern_gemm<64>(a, y_dtype, stream);
    default: break;
  }
  // What matters is the work of the fullest compute unit: the workgroups it gets,
  // ceil(workgroups / 256), times what one costs, R tiles of 16 rows plus the
  // X loads that serve all R (worth about 0.3 tile at one to four tokens,
  // whose other token lanes read nothing, and 1.5 tiles beyond).  Of R = 2..5
  // the least cost wins, ties to the larger R.  The 34816-row gate|up: R = 3
  // at one token (726 workgroups, at most 3 per unit; 18.4 us against 22.8
  // for R = 4), R = 5 at 16 tokens (26.4 against 29.2 for R = 3).  Rows
  // longer than 64 chunks take eight waves, their scales fewer rows.
  if (a.n_chunks <= 64) {
    const int64_t tiles = (d_out + 15) / 16, tok_tiles = (M + 15) / 16;
    const double x = M > 4 ? 1.5 : 0.3;
    int best_r = 2;
    double best = 1e300;
    for (int r = 2; r <= (a.n_chunks <= 51 ? 5 : 4); ++r) {
      const int64_t per_cu = ((tiles + r - 1) / r * tok_tiles + 255) / 256;
      const double cost = (double)per_cu * (r + x);
      if (cost <= best) best = cost, best_r = r;
    }
    switch (best_r) {
      case 5: return launch_tern<4, 5, 2, 16>(a, y_dtype, stream);
      case 4: return launch_tern<4, 4, 2, 16>(a, y_dtype, stream);
      case 3: return launch_tern<4, 3, 2, 16>(a, y_dtype, stream);
      default: return launch_tern<4, 2, 3, 16>(a, y_dtype, stream);
    }
  }
  if (a.n_chunks <= 256) return launch_tern<8, 2, 3, 16>(a, y_dtype, stream);
  return launch_tern<8, 1, 3, 16>(a, y_dtype, stream);
}
