// Matrix-core GEMMs of the fake-ternary linear layers and of attention (gfx950).
//
// The fake-ternary linears are the only dense contractions of the step
// (Sec. 2.4, Eq. 7: the window forward with alpha*T and its backward):
//   forward  Y  = X . W_fake^T      both operands contiguous along K
//   input    dX = dY . W_fake       W_fake contracted over its rows
//   weight   G  = dY^T . X          both operands contracted over tokens
// Two kernel templates, v_mfma_f32_32x32x16_bf16 with fp32 accumulation:
//   gemm_dma_kernel   operands straight into swizzled LDS tiles with buffer
//                     loads, K-major operands read with transpose loads; 256
//                     x 256 tiles on 16 waves (128 x 128 on 4 for small
//                     problems); dense, split-K, routed experts and the fused
//                     epilogues (SwiGLU forward/backward, factor gradients).
//                     It serves every projection of the calibration step.
//   gemm_bf16_kernel  register-staged tiles, operands contiguous along the
//                     output dimension transposed in registers with v_perm;
//                     the remaining shapes (unaligned extents, batched
//                     attention products of the unfused path).
// Both map workgroups to tiles so that neighbouring tiles share an XCD's L2
// (workgroups are dealt round-robin to the 8 XCDs).
#include <cmath>
#include <cstdio>
#include <cstring>
#include <type_traits>

#include "kernels.h"
#include "lmst_math.h"

namespace catq {

GemmArgs gemm_args_default() {
  GemmArgs a;
  std::memset(&a, 0, sizeof(a));  // every field, the epilogue arguments included
  a.A = a.B = a.R = nullptr;
  a.C = nullptr;
  a.M = a.N = a.K = 0;
  a.lda = a.ldb = a.ldc = a.ldr = 0;
  a.a_so = a.a_si = a.b_so = a.b_si = a.c_so = a.c_si = 0;
  a.a_div = a.b_div = a.c_div = a.inner = 1;
  a.batch = 1;
  a.alpha = 1.0f;
  a.causal = 0;
  a.group_off = nullptr;
  a.group_mode = 0;
  a.epi = 0;
  a.aux0 = a.aux1 = nullptr;
  a.ld_aux = 0;
  a.n_groups = 1;
  a.b_gs = a.c_gs = 0;
  a.max_rows_per_group = 0;
  return a;
}

// Internal launch record: GemmArgs plus split-K (blockIdx.z = split when > 1).
struct GemmLaunch {
  GemmArgs g;
  int32_t ksplit;
  int64_t kchunk;
  int64_t c_split_stride;
  int32_t tiles_m, tiles_n;
  int32_t group_m;  // tile rows per band of the tile walk (band_coords)
};

constexpr int LDS_PAD = 8;

__device__ __forceinline__ unsigned int perm(unsigned int hi_src, unsigned int lo_src,
                                             unsigned int sel) {
  return __builtin_amdgcn_perm(hi_src, lo_src, sel);
}

// Global -> register -> LDS staging of one operand tile (ROWS x BK, stored in
// LDS as [ROWS][BK + pad], K contiguous).
//   X_T = 0: the operand is contiguous along K; one item is a 16-byte chunk.
//   X_T = 1: the operand is contiguous along ROWS; one item is KR consecutive
//            K-rows x 8 ROWS (KR 16-byte loads), transposed in registers with
//            v_perm into 8 K-contiguous runs of KR elements.
template <int ROWS, int BK, int NT, int X_T>
struct TileLoader {
  static constexpr int KC = BK / 8;  // 16-byte chunks along K
  static constexpr int KR = (KC * (ROWS / 8) >= NT) ? 8 : ((BK / 4) * (ROWS / 8) >= NT ? 4 : 2);
  static constexpr int N_ITEMS = X_T == 0 ? ROWS * KC / NT : ((BK / KR) * (ROWS / 8)) / NT;
  static constexpr int N_REGS = X_T == 0 ? N_ITEMS : N_ITEMS * KR;
  static_assert(N_ITEMS >= 1, "tile too small for the thread count");
  static_assert(X_T == 0 ? (ROWS * KC) % NT == 0 : ((BK / KR) * (ROWS / 8)) % NT == 0,
                "uneven tile split");
  u32x4 r[N_REGS];

  // base points at element (row 0, k 0) of this operand for the current block;
  // rows are row0.., valid below row_lim; k runs k0.., valid below k_lim.
  __device__ __forceinline__ void load(const u16* __restrict__ base, int64_t ld, int64_t row0,
                                       int64_t row_lim, int64_t k0, int64_t k_lim, int tid) {
    const u32x4 z = {0u, 0u, 0u, 0u};
    if (X_T == 0) {
#pragma unroll
      for (int i = 0; i < N_ITEMS; ++i) {
        const int c = tid + i * NT;
        const int rr = c / KC, kc = c % KC;
        const int64_t row = row0 + rr, k = k0 + kc * 8;
        r[i] = (row < row_lim && k < k_lim)
                   ? *reinterpret_cast<const u32x4*>(base + row * ld + k)
                   : z;
      }
    } else {
#pragma unroll
      for (int i = 0; i < N_ITEMS; ++i) {
        const int b = tid + i * NT;
        const int kb = b / (ROWS / 8), mb = b % (ROWS / 8);
        const int64_t m = row0 + mb * 8;
        const bool mok = m < row_lim;
#pragma unroll
        for (int j = 0; j < KR; ++j) {
          const int64_t k = k0 + kb * KR + j;
          r[i * KR + j] = (mok && k < k_lim)
                              ? *reinterpret_cast<const u32x4*>(base + k * ld + m)
                              : z;
        }
      }
    }
  }

  __device__ __forceinline__ void store(u16* __restrict__ lds, int tid) const {
    constexpr int P = BK + LDS_PAD;
    if (X_T == 0) {
#pragma unroll
      for (int i = 0; i < N_ITEMS; ++i) {
        const int c = tid + i * NT;
        const int rr = c / KC, kc = c % KC;
        *reinterpret_cast<u32x4*>(lds + rr * P + kc * 8) = r[i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < N_ITEMS; ++i) {
        const int b = tid + i * NT;
        const int kb = b / (ROWS / 8), mb = b % (ROWS / 8);
        // r[i*KR + j] holds k = kb*KR + j for m = mb*8 + 0..7 (two per dword);
        // column mm becomes one K-contiguous run of KR elements.
#pragma unroll
        for (int mm = 0; mm < 8; ++mm) {
          const unsigned int sel = (mm & 1) ? 0x07060302u : 0x05040100u;
          const int dw = mm >> 1;
          u16* dst = lds + (mb * 8 + mm) * P + kb * KR;
          if (KR == 8) {
            u32x4 o;
#pragma unroll
            for (int p = 0; p < 4; ++p)
              o[p] = perm(r[i * KR + 2 * p + 1][dw], r[i * KR + 2 * p][dw], sel);
            *reinterpret_cast<u32x4*>(dst) = o;
          } else if (KR == 4) {
            uint2 o;
            o.x = perm(r[i * KR + 1][dw], r[i * KR + 0][dw], sel);
            o.y = perm(r[i * KR + 3][dw], r[i * KR + 2][dw], sel);
            *reinterpret_cast<uint2*>(dst) = o;
          } else {
            *reinterpret_cast<unsigned int*>(dst) = perm(r[i * KR + 1][dw], r[i * KR + 0][dw], sel);
          }
        }
      }
    }
  }
};

template <typename OutT>
__device__ __forceinline__ void store_out(OutT* p, float v);
template <>
__device__ __forceinline__ void store_out<float>(float* p, float v) {
  *p = v;
}
template <>
__device__ __forceinline__ void store_out<bf16>(bf16* p, float v) {
  *p = (bf16)v;
}

// tile id -> (tile row, tile column), walking bands of GROUP_M tile rows
// column by column (the A panels of a band stay in L2 while its B panels
// stream)
__device__ __forceinline__ void band_coords(int pid, int tiles_m, int tiles_n, int& pm, int& pn,
                                            int GROUP_M = 8) {
  const int in_group = GROUP_M * tiles_n;
  const int gid = pid / in_group;
  const int first = gid * GROUP_M;
  const int gsz = min(tiles_m - first, GROUP_M);
  const int r = pid % in_group;
  pm = first + r % gsz;
  pn = r / gsz;
}

__device__ __forceinline__ void tile_coords(int pid, int tiles_m, int tiles_n, int& pm, int& pn) {
  const int num = tiles_m * tiles_n;
  // keep neighbouring tiles on one XCD (round-robin dispatch over 8 XCDs)
  if ((num & 7) == 0) pid = (pid & 7) * (num >> 3) + (pid >> 3);
  band_coords(pid, tiles_m, tiles_n, pm, pn);
}

// One-dimensional grid over (K split, tile).  Workgroups are dealt to the 8
// XCDs round-robin; each XCD gets a contiguous range of (split, tile) ids, so
// with splits an XCD works through one K range (its operand panels are read
// by that XCD alone) and neighbouring tiles share its L2.
__device__ __forceinline__ void split_tile_coords(int lin, int tiles_m, int tiles_n, int ksplit,
                                                  int& pm, int& pn, int& z, int group_m) {
  const int T = tiles_m * tiles_n, num = T * ksplit;
  const int v = (num & 7) == 0 ? (lin & 7) * (num >> 3) + (lin >> 3) : lin;
  z = v / T;
  band_coords(v - z * T, tiles_m, tiles_n, pm, pn, group_m);
}

template <int BM, int BN, int BK, int WGM, int WGN, int A_T, int B_T, typename OutT, typename RT,
          bool HAS_R>
__global__ __launch_bounds__(WGM* WGN * 64) void gemm_bf16_kernel(GemmLaunch L) {
  constexpr int NT = WGM * WGN * 64;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  constexpr int P = BK + LDS_PAD;
  static_assert(FM >= 1 && FN >= 1 && BK % 16 == 0, "bad tile");
  __shared__ u16 sA[2][BM * P];
  __shared__ u16 sB[2][BN * P];

  const GemmArgs& g = L.g;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;

  int pm, pn, z = blockIdx.z;
  if (L.g.group_mode == 1) {
    // rows grouped by expert: blockIdx.x enumerates (m-tile, n-tile) over the
    // concatenation of every expert's m-tiles; walk the offsets to find ours
    const int t = blockIdx.x / L.tiles_n;
    pn = blockIdx.x % L.tiles_n;
    int acc_tiles = 0, e = 0;
    for (; e < L.g.n_groups; ++e) {
      const int64_t rows = L.g.group_off[e + 1] - L.g.group_off[e];
      const int nt = (int)((rows + BM - 1) / BM);
      if (t < acc_tiles + nt) break;
      acc_tiles += nt;
    }
    if (e >= L.g.n_groups) return;
    z = e;
    pm = t - acc_tiles;
  } else {
    tile_coords(blockIdx.x, L.tiles_m, L.tiles_n, pm, pn);
  }
  const int64_t m0 = (int64_t)pm * BM, n0 = (int64_t)pn * BN;

  // ---- operand bases, row limits and contraction range for this block
  const u16* Ab = reinterpret_cast<const u16*>(g.A);
  const u16* Bb = reinterpret_cast<const u16*>(g.B);
  int64_t a_row0 = m0;       // absolute row of A/C holding tile row 0
  int64_t row_lim = g.M;     // absolute rows of A/C below row_lim are valid
  int64_t kb = 0, ke = g.K;  // contraction range
  int64_t c_off = 0, r_off = 0;
  if (g.group_mode == 1) {
    const int64_t r0 = g.group_off[z], r1 = g.group_off[z + 1];
    if (m0 >= r1 - r0) return;
    a_row0 = r0 + m0;
    row_lim = r1;
    Bb += z * g.b_gs;
  } else if (g.group_mode == 2) {
    kb = g.group_off[z];
    ke = g.group_off[z + 1];
    c_off = z * g.c_gs;
  } else if (L.ksplit > 1) {
    kb = (int64_t)z * L.kchunk;
    ke = min(g.K, kb + L.kchunk);
    c_off = z * L.c_split_stride;
  } else {
    const int zo = z / g.inner, zi = z % g.inner;
    Ab += zo * g.a_so + (zi / g.a_div) * g.a_si;
    Bb += zo * g.b_so + (zi / g.b_div) * g.b_si;
    c_off = zo * g.c_so + (zi / g.c_div) * g.c_si;
    r_off = c_off;
  }
  if (g.causal == 1 && n0 >= m0 + BM) return;
  if (g.causal == 2) ke = min(ke, m0 + BM);
  if (g.causal == 3) kb = m0;  // BM is a multiple of BK

  TileLoader<BM, BK, NT, A_T> la;
  TileLoader<BN, BK, NT, B_T> lb;

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int64_t nk = ke > kb ? (ke - kb + BK - 1) / BK : 0;
  if (nk > 0) {
    la.load(Ab, g.lda, a_row0, row_lim, kb, ke, tid);
    lb.load(Bb, g.ldb, n0, g.N, kb, ke, tid);
    la.store(sA[0], tid);
    lb.store(sB[0], tid);
    __syncthreads();
  }
  for (int64_t kt = 0; kt < nk; ++kt) {
    const int buf = (int)(kt & 1);
    const bool more = kt + 1 < nk;
    if (more) {
      const int64_t k0 = kb + (kt + 1) * BK;
      la.load(Ab, g.lda, a_row0, row_lim, k0, ke, tid);
      lb.load(Bb, g.ldb, n0, g.N, k0, ke, tid);
    }
    const u16* pa = sA[buf] + (wm * WTM + (lane & 31)) * P + (lane >> 5) * 8;
    const u16* pb = sB[buf] + (wn * WTN + (lane & 31)) * P + (lane >> 5) * 8;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 fa[FM], fb[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        fa[i] = *reinterpret_cast<const bf16x8*>(pa + i * 32 * P + kk * 16);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        fb[j] = *reinterpret_cast<const bf16x8*>(pb + j * 32 * P + kk * 16);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      la.store(sA[buf ^ 1], tid);
      lb.store(sB[buf ^ 1], tid);
    }
    __syncthreads();
  }

  // ---- epilogue: 32x32 accumulator layout: acc[r] is row 8*(r/4) + 4*(lane/32) + r%4,
  // column lane%32 of the block
  OutT* C = reinterpret_cast<OutT*>(g.C) + c_off;
  const RT* R = HAS_R ? reinterpret_cast<const RT*>(g.R) + r_off : nullptr;
  const int64_t row_base = a_row0 - m0;  // grouped rows are absolute
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int64_t n = n0 + wn * WTN + j * 32 + (lane & 31);
      if (n >= g.N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t m = m0 + wm * WTM + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        const int64_t mrow = m + row_base;
        if (mrow >= row_lim) continue;
        float v = acc[i][j][r] * g.alpha;
        if (HAS_R) v += to_f(R[mrow * g.ldr + n]);
        store_out<OutT>(C + mrow * g.ldc + n, v);
      }
    }
  }
}

// four consecutive values <-> f32x4 (16-byte fp32 or 8-byte bf16 accesses)
__device__ __forceinline__ f32x4 load4f(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
__device__ __forceinline__ f32x4 load4f(const bf16* p) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
  f32x4 v;
  v[0] = __uint_as_float(u.x << 16);
  v[1] = __uint_as_float(u.x & 0xffff0000u);
  v[2] = __uint_as_float(u.y << 16);
  v[3] = __uint_as_float(u.y & 0xffff0000u);
  return v;
}
// 4 consecutive values kept as loaded (fp32: 16 B, bf16: 8 B), widened later
__device__ __forceinline__ f32x4 raw4(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
__device__ __forceinline__ uint2 raw4(const bf16* p) { return *reinterpret_cast<const uint2*>(p); }
__device__ __forceinline__ f32x4 widen4(f32x4 v) { return v; }
__device__ __forceinline__ f32x4 widen4(uint2 u) {
  f32x4 v;
  v[0] = __uint_as_float(u.x << 16);
  v[1] = __uint_as_float(u.x & 0xffff0000u);
  v[2] = __uint_as_float(u.y << 16);
  v[3] = __uint_as_float(u.y & 0xffff0000u);
  return v;
}
__device__ __forceinline__ void store4f(float* p, f32x4 v) { *reinterpret_cast<f32x4*>(p) = v; }
__device__ __forceinline__ void store4f(bf16* p, f32x4 v) {
  uint2 u;
  u.x = pack_bf16x2(v[0], v[1]);
  u.y = pack_bf16x2(v[2], v[3]);
  *reinterpret_cast<uint2*>(p) = u;
}

// ------------------------------------------- dense GEMM, direct to LDS
//
// Tiles move from global memory straight into LDS with buffer_load_dwordx4 ...
// lds (no register staging): each wave instruction fills 1 KB of LDS, lane l
// landing at base + 16 l.  Each operand is in one of two layouts:
//
// * K-contiguous ("nt", stored [rows][K]): a tile is ROWS x 64 bf16 =
//   ROWS*8 chunks of 16 B; chunk c of row r sits in slot r*8 + (c ^ ((r >> 1)
//   & 7)).  A 128-bit LDS read is served 16 lanes at a time over 64 four-byte
//   banks; the MFMA fragment read (16 consecutive rows at one chunk) then
//   covers all 16 bank groups once.  Rows past the matrix read as zero
//   (their results are never stored).
// * K-major ("km", stored [K][cols]): a tile is 64 rows of k x COLS bf16;
//   chunk c of row k sits in slot k*(COLS/8) + (c ^ (4*(k & 3))).  Fragments
//   come from two ds_read_b64_tr_b16 each: within a block of 16 lanes, lane i
//   receives element e of its 4 values from the lanes 4e..4e+3, column i mod 4
//   of their 8-byte rows.  When those four lanes point at row k0+e, columns
//   c0..c0+15, lane i gets column c0+i at rows k0..k0+3: the MFMA operand
//   (one column, consecutive k) without any transpose pass.  The XOR puts the
//   4 rows x 64 B that 32 lanes read in one cycle on 4 different 64-byte bank
//   windows.  COLS must divide the matrix extent.
//
// The swizzles are chosen through the global address each lane fetches.  Two
// LDS stages: the next tile is fetched while the current one is multiplied.
// Inside a tile the fragment reads of sub-step kk+1 are interleaved with the
// MFMAs of sub-step kk, and the first reads of the next tile overlap the last
// sub-step after the barrier.


// K-contiguous operand tile, ROWS x 64, for NW waves.  Buffer loads from the
// tile's first row: instructions i and i+2 differ only by 16 rows (a uniform
// offset), so a lane keeps two 32-bit offsets; rows past the matrix read as
// zero (their results are never stored).
template <int ROWS, int NW>
struct DmaOpNT {
  static constexpr int NI = ROWS / 8 / NW;  // 1 KB instructions per wave
  static constexpr int READS = 1;           // LDS reads per fragment
  static_assert(NI >= 2 && NI % 2 == 0, "tile too small for the wave count");
  const char* panel;     // byte address of the tile's first row (uniform)
  uint64_t bytes;        // bytes from panel to the end of the matrix
  uint32_t step;         // bytes between instructions i and i+2 (uniform)
  uint32_t voff[2];      // per lane, instructions of parity 0 and 1
  i32x4_rsrc rs;         // the tile's rows from the first k of its range
  int64_t k_first;
  __device__ __forceinline__ void init(const bf16* base, int64_t ld, int64_t row0, int64_t rows,
                                       int wave, int lane) {
    panel = reinterpret_cast<const char*>(base + row0 * ld);
    bytes = (uint64_t)(rows - row0) * (uint64_t)ld * 2;
    step = (uint32_t)(16 * ld * 2);
    const int rl = lane >> 3;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int blk = wave * NI + p;
      const int c = (lane & 7) ^ (((blk & 1) << 2) | (rl >> 1));
      voff[p] = (uint32_t)((blk * 8 + rl) * ld * 2 + c * 16);
    }
  }
  // tile row r holds matrix row half*(r & 1) + (row0 + r)/2 (row0 even):
  // gate and up rows of a fused [gate | up] weight taken in pairs (gate rows
  // past the end read up rows, up rows past the end read zero; neither is
  // stored)
  __device__ __forceinline__ void init_pairs(const bf16* base, int64_t ld, int64_t row0,
                                             int64_t half, int wave, int lane) {
    panel = reinterpret_cast<const char*>(base + (row0 >> 1) * ld);
    bytes = (uint64_t)(2 * half - (row0 >> 1)) * (uint64_t)ld * 2;
    step = (uint32_t)(8 * ld * 2);
    const int rl = lane >> 3;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int blk = wave * NI + p;
      const int c = (lane & 7) ^ (((blk & 1) << 2) | (rl >> 1));
      const int64_t mr = (rl & 1) * half + blk * 4 + (rl >> 1);
      voff[p] = (uint32_t)(mr * ld * 2 + c * 16);
    }
  }
  // one resource per tile, from the first k of the tile's contraction range
  // (the k offset of each copy goes in its scalar offset)
  __device__ __forceinline__ void bind(int64_t kb, int64_t) {
    const uint64_t b = (uint64_t)kb * 2;
    rs = buf_rsrc(panel + b, (uint32_t)min(bytes - b, (uint64_t)0xFFFFFFFFu));
    k_first = kb;
  }
  // (K-contiguous rows are whole: the contraction extent is a multiple of 64)
  __device__ __forceinline__ void issue(uint32_t lds, int64_t k0, int wave) const {
    const uint32_t ko = (uint32_t)(k0 - k_first) * 2;
#pragma unroll
    for (int i = 0; i < NI; ++i)
      dma16_lds(rs, voff[i & 1], ko + (uint32_t)(i >> 1) * step, lds + (wave * NI + i) * 1024);
  }
  // rows row0 .. row0+31 (lane: row row0 + lane%32), k = 16 kk + 8 (lane/32) .. +7
  __device__ __forceinline__ bf16x8 frag(const uint4* lds, int row0, int kk, int lane) const {
    const int cs = (kk * 2 + (lane >> 5)) ^ ((lane >> 1) & 7);
    return *reinterpret_cast<const bf16x8*>(&lds[(row0 + (lane & 31)) * 8 + cs]);
  }
};

// K-major operand tile, 64 x COLS, for NW waves.  Buffer loads from the
// tile's 64-row k slab; the swizzle repeats every P instructions, so a lane
// keeps P 32-bit offsets and the rest is a uniform offset.
template <int COLS, int NW>
struct DmaOpKM {
  static constexpr int CPR = COLS / 8;             // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;             // rows per 1 KB instruction
  static constexpr int NI = 64 * CPR / 64 / NW;    // instructions per wave
  static constexpr int P = RPI >= 4 ? 1 : 4 / RPI; // period of the swizzle in i
  static constexpr int READS = 2;
  static_assert(NI >= 1 && RPI >= 1 && NI % P == 0, "tile too small for the wave count");
  const char* panel;     // byte address of the tile's first column, row 0 (uniform)
  uint32_t ld2;          // row pitch in bytes
  uint32_t voff[P];      // per lane
  i32x4_rsrc rs;         // rows kb .. ke - 1 of the tile's columns
  int64_t k_first;
  __device__ __forceinline__ void init(const bf16* base, int64_t ld, int64_t col0, int64_t,
                                       int wave, int lane) {
    panel = reinterpret_cast<const char*>(base + col0);
    ld2 = (uint32_t)(ld * 2);
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int row = (wave * NI + p) * RPI + lane / CPR;
      const int c = (lane % CPR) ^ (4 * (row & 3));
      voff[p] = (uint32_t)(row * ld * 2 + c * 16);
    }
  }
  // one resource per tile over rows kb .. ke - 1 (rows at or past ke read as
  // zero; the host keeps (ke - kb + 64) * ld2 below 2^32)
  __device__ __forceinline__ void bind(int64_t kb, int64_t ke) {
    rs = buf_rsrc(panel + (uint64_t)kb * ld2, (uint32_t)((uint64_t)(ke - kb) * ld2));
    k_first = kb;
  }
  // rows k0 .. k0 + 63 of the range
  __device__ __forceinline__ void issue(uint32_t lds, int64_t k0, int wave) const {
    const uint32_t ko = (uint32_t)(k0 - k_first) * ld2;
#pragma unroll
    for (int i = 0; i < NI; ++i)
      dma16_lds(rs, voff[i % P], ko + (uint32_t)((i / P) * P * RPI) * ld2,
                lds + (wave * NI + i) * 1024);
  }
  // columns col0 .. col0+31 (lane: column col0 + lane%32), k = 16 kk + 8 (lane/32) .. +7
  __device__ __forceinline__ bf16x8 frag(const uint4* lds, int col0, int kk, int lane) const {
    const int blk = lane >> 4, s = lane & 15;
    const int col = col0 + 16 * (blk & 1) + 4 * (s & 3);
    u32x4 u;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int row = kk * 16 + 8 * (blk >> 1) + 4 * c + (s >> 2);
      const int chunk = (col >> 3) ^ (4 * (row & 3));
      const short* p = reinterpret_cast<const short*>(lds) + row * COLS + chunk * 8 + (col & 7);
      const lds_v4s v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) lds_v4s*)(p));
      u[2 * c] = (unsigned)(unsigned short)v[0] | ((unsigned)(unsigned short)v[1] << 16);
      u[2 * c + 1] = (unsigned)(unsigned short)v[2] | ((unsigned)(unsigned short)v[3] << 16);
    }
    return __builtin_bit_cast(bf16x8, u);
  }
};

// Rows grouped by expert (row range off[e] .. off[e+1]): the m-tiles of all
// experts concatenated.  Each wave finds, with a prefix sum of the experts'
// tile counts over its lanes (64 experts at a time), the expert and m-tile of
// concatenated tile t, and the total tile count.  Uniform across the wave.
__device__ __forceinline__ bool group_tile(const int64_t* off, int E, int t, int bm, int lane,
                                           int& e_out, int& pm_out, int& total_out) {
  int base = 0;
  bool found = false;
  for (int c0 = 0; c0 < E; c0 += 64) {
    const int e = c0 + lane;
    int nt = 0;
    if (e < E) nt = (int)((off[e + 1] - off[e] + bm - 1) / bm);
    int incl = nt;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int y = __shfl_up(incl, d, 64);
      if (lane >= d) incl += y;
    }
    const int chunk = __shfl(incl, 63, 64);
    if (!found && t < base + chunk) {
      const unsigned long long m = __ballot(base + incl > t);
      const int l = __builtin_ctzll(m);
      e_out = c0 + l;
      pm_out = t - base - __shfl(incl - nt, l, 64);
      found = true;
    }
    base += chunk;
  }
  total_out = base;
  return found;
}

template <int BM, int BN, int WGM, int WGN, bool AKM, bool BKM, typename OutT, typename RT,
          bool HAS_R, int EPI = 0, int SB = 2>
__global__ __launch_bounds__(WGM* WGN * 64, 1)
    __attribute__((amdgpu_waves_per_eu(1, (WGM * WGN + 3) / 4))) void gemm_dma_kernel(GemmLaunch L) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int NW = WGM * WGN;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  static_assert(FM >= 1 && FN >= 1 && FM * FN >= FM + FN, "bad tile");
  using OA = std::conditional_t<AKM, DmaOpKM<BM, NW>, DmaOpNT<BM, NW>>;
  using OB = std::conditional_t<BKM, DmaOpKM<BN, NW>, DmaOpNT<BN, NW>>;
  // one LDS allocation: the two stages of A, then the SB of B (the epilogue
  // stages the output through the first two stages' worth of it).  SB = 3
  // puts B's copies two k tiles ahead, for B streamed from HBM once (a large
  // weight, or an expert's weight used by one row tile)
  static_assert(SB == 2 || SB == 3, "two or three B stages");
  constexpr int LDS_SLOTS = 2 * (BM + BN) * 8;
  __shared__ uint4 smem[(2 * BM + SB * BN) * 8];
  auto sA = [&](int buf) { return smem + buf * (BM * 8); };
  auto sB = [&](int buf) { return smem + 2 * BM * 8 + buf * (BN * 8); };
  const GemmArgs& g = L.g;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  int pm = 0, pn = 0, z = 0;
  int64_t m0, m_lim = g.M;   // first row of A (rows) and C of the tile; rows below m_lim valid
  int64_t kb = 0, ke = g.K, c_off = 0;
  const bf16* Bb = reinterpret_cast<const bf16*>(g.B);
  if (g.group_mode == 1) {
    // rows grouped by expert; blocks past the experts' tiles leave at once
    // (uniformly: every wave computes the same search)
    const int t0 = (int)(blockIdx.x / L.tiles_n);
    int e = 0, pt = 0, tiles = 0;
    group_tile(g.group_off, g.n_groups, t0, BM, lane, e, pt, tiles);
    const int n_real = tiles * L.tiles_n;
    const int lin = blockIdx.x;
    if (lin >= n_real) return;
    // Each XCD (round-robin dispatch) takes a contiguous range of the real
    // tile ids, ordered expert by expert, then n-tile, then m-tile: the few
    // m-tiles of an expert that share one of its weight panels run back to
    // back on one L2, so each expert's weight is fetched about once.
    const int x = lin & 7, q = n_real >> 3, r = n_real & 7;
    const int v = x * q + min(x, r) + (lin >> 3);
    group_tile(g.group_off, g.n_groups, v / L.tiles_n, BM, lane, e, pt, tiles);
    const int64_t r0 = g.group_off[e];
    m_lim = g.group_off[e + 1];
    const int te = (int)((m_lim - r0 + BM - 1) / BM);              // the expert's m-tiles
    const int local = v - (v / L.tiles_n - pt) * L.tiles_n;        // id within the expert
    pn = local / te;
    m0 = r0 + (int64_t)(local - pn * te) * BM;
    Bb += (int64_t)e * g.b_gs;
  } else {
    split_tile_coords(blockIdx.x, L.tiles_m, L.tiles_n,
                      g.group_mode == 2 ? g.n_groups : L.ksplit, pm, pn, z, L.group_m);
    m0 = (int64_t)pm * BM;
    if (g.group_mode == 2) {
      // contraction grouped by expert (ragged): rows past the group's end
      // read as zero; an empty group writes a zero tile
      kb = g.group_off[z];
      ke = g.group_off[z + 1];
      c_off = (int64_t)z * g.c_gs;
    } else if (L.ksplit > 1) {
      kb = (int64_t)z * L.kchunk;
      ke = min(g.K, kb + L.kchunk);
      c_off = (int64_t)z * L.c_split_stride;
    }
  }
  const int64_t n0 = (int64_t)pn * BN;
  OA oa;
  OB ob;
  oa.init(reinterpret_cast<const bf16*>(g.A), g.lda, m0, m_lim, wave, lane);
  if constexpr (EPI == 1)
    ob.init_pairs(Bb, g.ldb, n0, g.N / 2, wave, lane);
  else
    ob.init(Bb, g.ldb, n0, g.N, wave, lane);
  oa.bind(kb, ke);
  ob.bind(kb, ke);
  // LDS byte address of the operand stages (uniform): A's two, then B's SB
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint4*)smem;
  bf16x8 fa[2][FM], fb[2][FN];
  // stages by index: A's is the k tile's parity, B's is carried along (kt % SB)
  auto ldfrag = [&](int ast, int bst, int kk, int slot) {
#pragma unroll
    for (int i = 0; i < FM; ++i) fa[slot][i] = oa.frag(sA(ast), wm * WTM + 32 * i, kk, lane);
#pragma unroll
    for (int j = 0; j < FN; ++j) fb[slot][j] = ob.frag(sB(bst), wn * WTN + 32 * j, kk, lane);
  };
  auto issueA = [&](int kt) {
    oa.issue(lds0 + (uint32_t)(kt & 1) * (BM * 128), kb + (int64_t)kt * 64, wave);
  };
  auto issueB = [&](int kt, int bst) {
    ob.issue(lds0 + 2 * BM * 128 + (uint32_t)bst * (BN * 128), kb + (int64_t)kt * 64, wave);
  };
  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  auto mfmas = [&](int slot) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[slot][i], fb[slot][j], acc[i][j], 0, 0, 0);
  };
  // the first FM+FN MFMAs each followed by one fragment's LDS reads, the rest back to back
  auto interleave = [&]() {
#pragma unroll
    for (int q = 0; q < FM; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, OA::READS, 0);
    }
#pragma unroll
    for (int q = 0; q < FN; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, OB::READS, 0);
    }
    if constexpr (FM * FN > FM + FN) __builtin_amdgcn_sched_group_barrier(0x008, FM * FN - (FM + FN), 0);
  };
  // one 64-deep tile: sub-steps 0..2 with the next sub-step's reads
  // interleaved, barrier, then sub-step 3 overlapped with the next tile's
  // first reads.  MORE is false only for the last tile (no branches inside
  // the steady-state body, so the interleaving spans it whole).
  const int nk = (int)((ke - kb + 63) / 64);
  auto tile = [&](int kt, int bst, auto more_c) {
    constexpr bool MORE = decltype(more_c)::value;
    const int bnext = bst + 1 == SB ? 0 : bst + 1;     // (kt + 1) % SB
    // copies of tile kt+1 (A; and B with two stages) or kt+2 (B, three
    // stages) into the stages tile kt-1 used; B's copies are issued last, so
    // with three stages waiting for all but B's newest finishes tile kt+1
    if (MORE) issueA(kt + 1);
    if (SB == 2 && MORE) issueB(kt + 1, bnext);
    const bool deep = SB == 3 && kt + 2 < nk;
    if (deep) issueB(kt + 2, bst == 0 ? SB - 1 : bst - 1);   // (kt + 2) % 3
#pragma unroll
    for (int kk = 0; kk < 3; ++kk) {
      ldfrag(kt & 1, bst, kk + 1, (kk & 1) ^ 1);
      mfmas(kk & 1);
      interleave();
    }
    if (deep)
      wait_vmem_n<OB::NI>();
    else
      wait_vmem();
    __syncthreads();
    if (MORE) ldfrag((kt + 1) & 1, bnext, 0, 0);
    mfmas(1);
    if (MORE) interleave();
  };
  // factor epilogue: the weights of a staged part (lane: row lane / 4 of
  // the part, 16 consecutive columns), loaded one part ahead; the first
  // part's during the last k tile
  [[maybe_unused]] uint2 epw[4];
  [[maybe_unused]] auto epi3_load = [&](int p) {
    if constexpr (EPI == 3) {
      constexpr int HP3 = 2, SR3 = 16;
      const int64_t mrow = m0 + wm * WTM + (p / HP3) * 32 + (p % HP3) * SR3;
      const int64_t wrow = (int64_t)z * g.M + min(mrow + (lane >> 2), m_lim - 1);
      const bf16* wsrc = reinterpret_cast<const bf16*>(g.fac.W) + wrow * g.fac.ldw + n0 +
                         wn * WTN + (lane & 3) * 16;
#pragma unroll
      for (int q = 0; q < 4; ++q) epw[q] = raw4(wsrc + 4 * q);
    }
  };
  if (nk > 0) {
    issueA(0);
    issueB(0, 0);
    if (SB == 3 && nk > 1) {
      issueB(1, 1);
      wait_vmem_n<OB::NI>();
    } else {
      wait_vmem();
    }
    __syncthreads();
    ldfrag(0, 0, 0, 0);
    int bst = 0;
    for (int kt = 0; kt < nk - 1; ++kt) {
      tile(kt, bst, std::true_type{});
      bst = bst + 1 == SB ? 0 : bst + 1;
    }
    if constexpr (EPI == 3) epi3_load(0);
    tile(nk - 1, bst, std::false_type{});
  } else if constexpr (EPI == 3) {
    epi3_load(0);
  }
  OutT* C = reinterpret_cast<OutT*>(g.C) + c_off;
  const RT* R = HAS_R ? reinterpret_cast<const RT*>(g.R) : nullptr;
  // Epilogue.  Every wave has passed the last barrier, so no LDS read of the
  // main loop is outstanding and each wave may reuse its own part of the
  // operand buffers: a 32-row slab of its tile goes to LDS row-major (pitch
  // WTN+8 floats, so the two row groups one store instruction touches fall on
  // different banks), then comes back as 4 consecutive columns per lane (16
  // lanes read one row) for vector global stores and residual loads.
  const bool vec = g.N % 4 == 0 && g.ldc % 4 == 0 && c_off % 4 == 0 && aligned16(C) &&
                   (!HAS_R || (g.ldr % 4 == 0 && aligned16(R)));
  if (vec) {
    constexpr int EP = WTN + 8;
    constexpr int LPR = WTN / 4, RPP = 64 / LPR;  // lanes per row, rows per pass
    // rows staged per LDS round trip: the whole 32-row slab when every wave's
    // share fits in the operand buffers, else half of it (16 waves; and the
    // factor epilogue, whose lane map takes 16-row parts)
    constexpr int SR = (EPI != 3 && NW * 32 * EP * 4 <= LDS_SLOTS * 16) ? 32 : 16;
    constexpr int NP = SR / RPP;                  // passes per staged part
    static_assert(NW * SR * EP * 4 <= LDS_SLOTS * 16, "epilogue staging");
    float* st = reinterpret_cast<float*>(smem) + wave * (SR * EP);
    // factor epilogue: the half-group sums of every tile row, past the staging
    // ([tile row][wave column block][term]; a 64-column block is half a group)
    [[maybe_unused]] float* fsum = reinterpret_cast<float*>(smem) + NW * SR * EP;
    static_assert(EPI != 3 || (BN % 128 == 0 && WTN == 64 &&
                               (NW * SR * EP + BM * WGN * 4) * 4 <= LDS_SLOTS * 16),
                  "factor epilogue layout");
    const int cc = (lane % LPR) * 4;
    const int64_t n = n0 + wn * WTN + cc;
    const int64_t n_c = min(n, g.N - 4);   // clamped column for the early loads
    // The parts' other inputs (residual, or gate and up of the forward, or
    // the weights) are loaded one part ahead: those of part p + 1 are in
    // flight while part p goes through LDS and out.  Rows clamped into the
    // matrix, the values of lanes outside it unused.
    constexpr int HP = 32 / SR, PARTS = FM * HP;
    using RawR = decltype(raw4((const RT*)nullptr));
    [[maybe_unused]] RawR rvb[2][NP];
    [[maybe_unused]] uint2 gvb[2][NP], uvb[2][NP];
    auto load_part = [&](int p, int slot) {
      const int64_t mr = m0 + wm * WTM + (p / HP) * 32 + (p % HP) * SR;
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        const int64_t m_c = min(mr + q * RPP + lane / LPR, m_lim - 1);
        if constexpr (EPI == 2) {
          const bf16* gu = reinterpret_cast<const bf16*>(g.aux0) + m_c * g.ld_aux;
          gvb[slot][q] = raw4(gu + n_c);
          uvb[slot][q] = raw4(gu + g.N + n_c);
        } else if constexpr (EPI == 0 && HAS_R) {
          rvb[slot][q] = raw4(R + m_c * g.ldr + n_c);
        }
      }
    };
    if constexpr (EPI == 3) {
      // Factor epilogue.  Lane l takes row l / 4 of each staged part and 16
      // consecutive columns, 16 (l % 4) .. +15 of the wave's 64 (which lie in
      // one half of a 128-weight group), over four 4-column passes: the row's
      // group scalars are the lane's own, its 16 weights arrive in four 8-byte
      // loads, and the four terms of the factor gradients are summed over the
      // lane's 16 weights, then over the row's 4 lanes.  G[m][n] of expert z,
      // or of the one dense problem (z = 0), unsplit, alpha 1.
      static_assert(WTN == 64 && SR == 16 && HP == 2, "factor epilogue lane map");
      constexpr int GPT = BN / 128;  // groups per tile row
      static_assert(BM * GPT <= NW * 64, "one reduced group per thread");
      const FacEpi& F = g.fac;
      const int rr = lane >> 2, cq = (lane & 3) * 16;
      const int64_t ncol = n0 + wn * WTN + cq;
      // The raw group scalars (mu0, alpha0 and the three factors) of a part's
      // row, loaded one part ahead, and those of the group this thread
      // reduces at the end, loaded with the last part: with a few k tiles
      // per tile (routed experts: ~256 rows) these loads' latency is
      // otherwise exposed.
      auto raw_scalars = [&](int64_t grp, float (&r)[5]) {
        r[0] = F.stats[2 * grp];
        r[1] = F.stats[2 * grp + 1];
        r[2] = F.dmu[grp * F.s[0]];
        r[3] = F.dal[grp * F.s[1]];
        r[4] = F.dde[grp * F.s[2]];
      };
      auto part_group = [&](int p) {
        const int64_t mrow = m0 + wm * WTM + (p / HP) * 32 + (p % HP) * SR;
        return ((int64_t)z * g.M + min(mrow + rr, m_lim - 1)) * (F.ldw >> 7) + (ncol >> 7);
      };
      const int ft = min(tid, BM * GPT - 1), frow = ft / GPT, fgt = ft % GPT;
      const int64_t fgrp = ((int64_t)z * g.M + m0 + frow) * (F.ldw >> 7) + (n0 >> 7) + fgt;
      float gsf[5], gsc[5], gsn[5];
      raw_scalars(part_group(0), gsc);
#pragma unroll
      for (int p = 0; p < PARTS; ++p) {
        const int i = p / HP, h = p % HP;
        const int64_t mrow = m0 + wm * WTM + i * 32 + h * SR;
        uint2 wv[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) wv[q] = epw[q];
        const GroupScalars gs = group_scalars(gsc[0], gsc[1], gsc[2], gsc[3], gsc[4], F.delta0);
        if (p + 1 < PARTS)
          raw_scalars(part_group(p + 1), gsn);
        else
          raw_scalars(fgrp, gsf);
        // the part's accumulator slab through this wave's staging area
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (row / SR == h) st[(row - h * SR) * EP + j * 32 + (lane & 31)] = acc[i][j][r];
          }
        // the next part's weights, in flight while this part is processed
        if (p + 1 < PARTS) epi3_load(p + 1);
        float sT = 0.f, s1 = 0.f, sW = 0.f, sD = 0.f;
        if (mrow + rr < m_lim && F.mode != CATQ_IDENTITY) {
          const float mu = gs.mu;
          // z = (w - mu) / alpha * c2s as one FMA per weight
          const float zk = F.st.c2s * __builtin_amdgcn_rcpf(gs.alpha_div), z0 = -mu * zk;
          const float dz = gs.delta * F.st.c2s;
          const float ed = one_minus_exp_neg(gs.delta * F.st.s4, gs.delta * F.st.s4l);
          // one pass: 4 weights (rotated into wv[0]) against 4 G values;
          // (HARD, STE: the straight-through estimator, hard mode only) are
          // launch constants, one loop per combination
          auto pass = [&](int q, auto hard_c, auto ste_c) {
            constexpr bool HARD = decltype(hard_c)::value, STE = decltype(ste_c)::value;
            const f32x4 v = *reinterpret_cast<const f32x4*>(st + rr * EP + cq + 4 * q);
            const f32x4 w = widen4(wv[0]);
            // the next pass's weights into wv[0] (registers rotated: no
            // dynamically indexed array)
            wv[0] = wv[1];
            wv[1] = wv[2];
            wv[2] = wv[3];
            float hc[4];
            if constexpr (HARD) {
              const float w4[4] = {w[0], w[1], w[2], w[3]};
              hard_codes_n<4>(w4, mu, hard_thresh(gs.delta, gs.alpha_div), hc);
            }
            float z[4], E[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              z[e] = fmaf(w[e], zk, z0);
              E[e] = 1.0f - __builtin_amdgcn_exp2f(-2.0f * fabsf(z[e]));
            }
            if constexpr (!STE) {
              // 1 - 2^(-2y) by its series below y = 0.09 (no cancellation),
              // only in passes where some lane of the wave has such a y
              bool small = false;
#pragma unroll
              for (int e = 0; e < 4; ++e) small |= fabsf(z[e]) < 0.09016844f;
              if (__any(small)) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                  const float y = fabsf(z[e]);
                  E[e] = y < 0.09016844f ? one_minus_exp2_neg2(y, 0.0f) : E[e];
                }
              }
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              float fp = 0.f, fwp = 1.f, fdp = 0.f;
              if constexpr (!STE) transition_parts_zE(z[e], dz, ed, E[e], fp, fwp, fdp);
              sT = fmaf(v[e], HARD ? hc[e] : fp, sT);
              const float gf = v[e] * fwp;
              s1 += gf;
              sW = fmaf(gf, z[e], sW);  // g f_W z: wz rescales per group
              sD = fmaf(v[e], fdp, sD);
            }
          };
          if (F.mode == CATQ_HARD && F.ste) {
#pragma unroll 1
            for (int q = 0; q < 4; ++q) pass(q, std::true_type{}, std::true_type{});
          } else if (F.mode == CATQ_HARD) {
#pragma unroll 1
            for (int q = 0; q < 4; ++q) pass(q, std::true_type{}, std::false_type{});
          } else {
#pragma unroll 1
            for (int q = 0; q < 4; ++q) pass(q, std::false_type{}, std::false_type{});
          }
        }
#pragma unroll
        for (int mk = 1; mk < 4; mk <<= 1) {
          sT += __shfl_xor(sT, mk, 64);
          s1 += __shfl_xor(s1, mk, 64);
          sW += __shfl_xor(sW, mk, 64);
          sD += __shfl_xor(sD, mk, 64);
        }
        if ((lane & 3) == 0) {
          // [tile row][wave column block][term]; the row's 64 columns of
          // this wave are half of one group
          float* d = fsum + ((int)(mrow - m0 + rr) * WGN + wn) * 4;
          d[0] = sT;
          d[1] = s1;
          d[2] = sW;
          d[3] = sD;
        }
        if (p + 1 < PARTS) {
#pragma unroll
          for (int k = 0; k < 5; ++k) gsc[k] = gsn[k];
        }
      }
      // both halves of each group in order, then the three factor gradients
      // (the separate factor-gradient kernel's formulas)
      __syncthreads();
      if (tid < BM * GPT) {
        const int row = frow, gt = fgt;
        const float* a0 = fsum + (row * WGN + 2 * gt) * 4;
        // the constant factors of f (k2, soft only), f_W and f_Delta (sk4)
        const FacScale k = fac_scale(F.mode, F.ste, F.st);
        const float sT = (a0[0] + a0[4]) * k.f, s1 = (a0[1] + a0[5]) * k.w;
        const float sW = (a0[2] + a0[6]) * k.wz, sD = (a0[3] + a0[7]) * k.d;
        const int64_t grp = fgrp;
        const float alpha0 = gsf[1];
        const GroupScalars gs = group_scalars(gsf[0], alpha0, gsf[2], gsf[3], gsf[4], F.delta0);
        float o[3];
        o[0] = alpha0 * (-s1);
        o[1] = alpha0 * (sT - sW);
        o[2] = F.delta0 * (gs.alpha * sD);
#pragma unroll
        for (int k = 0; k < 3; ++k) {
          if (F.s[k] == 1)
            F.out[k][grp] = o[k];
          else
            F.ws[k * F.n_groups + grp] = o[k];
        }
      }
    }
    // (the factor epilogue has its own loop above)
    if constexpr (EPI != 3) load_part(0, 0);
  #pragma unroll
    for (int p = 0; p < (EPI == 3 ? 0 : PARTS); ++p) {
      const int i = p / HP, h = p % HP;
      {
        const int64_t mrow = m0 + wm * WTM + i * 32 + h * SR;
        if (p + 1 < PARTS) load_part(p + 1, (p + 1) & 1);
        [[maybe_unused]] auto& rv = rvb[p & 1];
        [[maybe_unused]] auto& gv = gvb[p & 1];
        [[maybe_unused]] auto& uv = uvb[p & 1];
  #pragma unroll
        for (int j = 0; j < FN; ++j)
  #pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (row / SR == h) st[(row - h * SR) * EP + j * 32 + (lane & 31)] = acc[i][j][r];
          }
  #pragma unroll
        for (int q = 0; q < NP; ++q) {
          const int rr = q * RPP + lane / LPR;
          const int64_t m = mrow + rr;
          f32x4 v = *reinterpret_cast<const f32x4*>(st + rr * EP + cc);
          if (m < m_lim && n < g.N) {
            v *= g.alpha;
            if constexpr (EPI == 1) {
              // columns n..n+3 = gate_p, up_p, gate_p+1, up_p+1 (p = n/2), each
              // rounded as stored; gate|up back to [gate | up], a = SwiGLU
              const int64_t p = n >> 1, half = g.N >> 1;
              const float g0 = bf16_round_f(v[0]), u0 = bf16_round_f(v[1]);
              const float g1 = bf16_round_f(v[2]), u1 = bf16_round_f(v[3]);
              bf16* gu = reinterpret_cast<bf16*>(C) + m * g.ldc;
              *reinterpret_cast<unsigned*>(gu + p) = pack_bf16x2(g0, g1);
              *reinterpret_cast<unsigned*>(gu + half + p) = pack_bf16x2(u0, u1);
              bf16* ar = reinterpret_cast<bf16*>(g.aux0) + m * g.ld_aux;
              *reinterpret_cast<unsigned*>(ar + p) = pack_bf16x2(swiglu1(g0, u0), swiglu1(g1, u1));
            } else if constexpr (EPI == 2) {
              // v = d a[m][n..n+3] (rounded as stored); gate|up of the forward
              // from aux0, d[gate | up] to aux1
              const int64_t Fh = g.N;
              bf16* dgu = reinterpret_cast<bf16*>(g.aux1) + m * g.ld_aux;
              const f32x4 gg = widen4(gv[q]), uu = widen4(uv[q]);
              f32x4 dg, du;
  #pragma unroll
              for (int e = 0; e < 4; ++e) {
                float a_, b_;
                swiglu1_bwd(gg[e], uu[e], bf16_round_f(v[e]), a_, b_);
                dg[e] = a_;
                du[e] = b_;
              }
              store4f(dgu + n, dg);
              store4f(dgu + Fh + n, du);
            } else {
              if constexpr (HAS_R) v += widen4(rv[q]);
              store4f(C + m * g.ldc + n, v);
            }
          }
        }
      }
    }
  } else if constexpr (EPI == 0) {
    // (the fused epilogues run only where the host checked the vector path)
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int64_t n = n0 + wn * WTN + j * 32 + (lane & 31);
        if (n >= g.N) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t m = m0 + wm * WTM + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
          if (m >= m_lim) continue;
          float v = acc[i][j][r] * g.alpha;
          if (HAS_R) v += to_f(R[m * g.ldr + n]);
          store_out<OutT>(C + m * g.ldc + n, v);
        }
      }
    }
  }
#endif
}

// ------------------------------------------------------------- fp32 GEMM
// Plain LDS-tiled FMA kernel for fp32 problems (the fp32 single-linear
// workload); 64x64 tile, 16-deep K slices, 4x4 outputs per thread.
template <int A_T, int B_T>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmLaunch L) {
  const GemmArgs& g = L.g;
  __shared__ float sA[16][64 + 1];
  __shared__ float sB[16][64 + 1];
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  const int64_t m0 = (int64_t)blockIdx.y * 64, n0 = (int64_t)blockIdx.x * 64;
  const float* A = reinterpret_cast<const float*>(g.A);
  const float* B = reinterpret_cast<const float*>(g.B);
  int64_t kb = 0, ke = g.K, c_off = 0;
  if (L.ksplit > 1) {
    kb = (int64_t)blockIdx.z * L.kchunk;
    ke = min(g.K, kb + L.kchunk);
    c_off = blockIdx.z * L.c_split_stride;
  }
  float acc[4][4] = {};
  for (int64_t k0 = kb; k0 < ke; k0 += 16) {
    for (int e = threadIdx.x; e < 16 * 64; e += 256) {
      const int kk = e / 64, mm = e % 64;
      const int64_t k = k0 + kk, m = m0 + mm, n = n0 + mm;
      float va = 0.f, vb = 0.f;
      if (k < ke && m < g.M) va = A_T ? A[k * g.lda + m] : A[m * g.lda + k];
      if (k < ke && n < g.N) vb = B_T ? B[k * g.ldb + n] : B[n * g.ldb + k];
      sA[kk][mm] = va;
      sB[kk][mm] = vb;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = sA[kk][ty * 4 + i];
        b[i] = sB[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  float* C = reinterpret_cast<float*>(g.C) + c_off;
  const float* R = reinterpret_cast<const float*>(g.R);
  for (int i = 0; i < 4; ++i) {
    const int64_t m = m0 + ty * 4 + i;
    if (m >= g.M) continue;
    for (int j = 0; j < 4; ++j) {
      const int64_t n = n0 + tx * 4 + j;
      if (n >= g.N) continue;
      float v = acc[i][j] * g.alpha;
      if (R) v += R[m * g.ldr + n];
      C[m * g.ldc + n] = v;
    }
  }
}

// --------------------------------------------------------------- dispatch

template <typename T>
static const char* tname() {
  return sizeof(T) == 2 ? "__bf16" : "float";
}

// Algorithmic work of one GEMM launch: 2MNK per problem (half of it for the
// causal attention products), each operand read once and C written once.
static void gemm_work(const GemmLaunch& L, int out_bytes, double& flops, double& bytes) {
  const GemmArgs& g = L.g;
  // grouped problems: rows split among the groups (mode 1), or the
  // contraction split among them (mode 2, K = all groups' rows): either way
  // 2 M N K in total
  double nb = g.group_mode != 0 ? 1 : g.batch;
  double f = 2.0 * (double)g.M * (double)g.N * (double)g.K * nb;
  if (g.causal) f *= 0.5;
  flops = f;
  if (g.group_mode == 1)
    bytes = 2.0 * ((double)g.M * g.K + (double)g.n_groups * g.N * g.K) + (double)out_bytes * g.M * g.N;
  else if (g.group_mode == 2)
    bytes = 2.0 * ((double)g.K * g.M + (double)g.K * g.N) + (double)out_bytes * g.n_groups * g.M * g.N;
  else
    bytes = nb * (2.0 * ((double)g.M * g.K + (double)g.N * g.K) + (double)out_bytes * g.M * g.N);
}

template <int BM, int BN, int WGM, int WGN, int A_T, int B_T, typename OutT, typename RT>
static void launch_cfg(GemmLaunch& L, hipStream_t stream) {
  constexpr int BK = 64;
  const GemmArgs& g = L.g;
  // grouped rows: at most ceil(M/BM) + E m-tiles over all experts together
  L.tiles_m = g.group_mode == 1 ? (int)((g.M + BM - 1) / BM + g.n_groups)
                                : (int)((g.M + BM - 1) / BM);
  L.tiles_n = (int)((g.N + BN - 1) / BN);
  int zdim = g.group_mode == 2 ? g.n_groups
                               : (g.group_mode == 1 ? 1 : (L.ksplit > 1 ? L.ksplit : g.batch));
  dim3 grid((unsigned)(L.tiles_m * L.tiles_n), 1, (unsigned)zdim);
  dim3 block(WGM * WGN * 64);
  char tag[96];
  std::snprintf(tag, sizeof(tag), "gemm_bf16_kernel<%d, %d, %d, %d, %d, %d, %d, %s, %s, %s>", BM,
                BN, BK, WGM, WGN, A_T, B_T, tname<OutT>(), tname<RT>(), g.R ? "true" : "false");
  double flops, bytes;
  gemm_work(L, (int)sizeof(OutT), flops, bytes);
  if (g.R)
    CATQ_TRACED(stream, tag, flops, bytes, g.M, g.N, g.K,
                hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, BK, WGM, WGN, A_T, B_T, OutT, RT, true>),
                                   grid, block, 0, stream, L));
  else
    CATQ_TRACED(stream, tag, flops, bytes, g.M, g.N, g.K,
                hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, BK, WGM, WGN, A_T, B_T, OutT, RT, false>),
                                   grid, block, 0, stream, L));
}

template <int BM, int BN, int WGM, int WGN, bool AKM, bool BKM, typename OutT, typename RT,
          int EPI = 0, int SB = 2>
static void launch_dma(GemmLaunch& L, hipStream_t stream) {
  const GemmArgs& g = L.g;
  // Bands of the tile walk: 8 tile rows (of the 32 tiles in flight per XCD,
  // 8 x 4), but 2 (2 x 16) for the weight-gradient products, both operands
  // K-major: measured in the 14B-shaped calibration step, their launches
  // take 4.29 (8 rows), 4.21 (4), 4.16 (2) and 4.18 ms (1) per step, while
  // the other layouts are best at 8.
  L.group_m = AKM ? 2 : 8;
  // grouped rows: at most ceil(M/BM) + E m-tiles over all experts together
  L.tiles_m = (int)((g.M + BM - 1) / BM) + (g.group_mode == 1 ? g.n_groups : 0);
  L.tiles_n = (int)((g.N + BN - 1) / BN);
  dim3 grid((unsigned)(L.tiles_m * L.tiles_n * (g.group_mode == 2 ? g.n_groups : L.ksplit)));
  dim3 block(WGM * WGN * 64);
  char tag[112];
  std::snprintf(tag, sizeof(tag), "gemm_dma_kernel<%d, %d, %d, %d, %s%s, %s, %s, %s%s%s%s>", BM,
                BN, WGM, WGN, AKM ? "k" : "n", BKM ? "k" : "t", tname<OutT>(), tname<RT>(),
                g.R ? "true" : "false",
                EPI == 1 ? ", swiglu" : (EPI == 2 ? ", swiglu_bwd" : (EPI == 3 ? ", factor_grads" : "")),
                g.group_mode ? ", experts" : "", SB == 3 ? ", 3 B stages" : "");
  double flops, bytes;
  gemm_work(L, (int)sizeof(OutT), flops, bytes);
  if (EPI == 1) bytes += (double)g.M * (double)(g.N / 2) * 2.0;          // a written
  if (EPI == 2) bytes += (double)g.M * (double)g.N * 2.0 * 4.0 - (double)g.M * g.N * sizeof(OutT);
  if (EPI == 3) {  // W read instead of G written; per group stats, factors, gradients
    const double w = (double)g.n_groups * g.M * g.N;
    bytes += w * 2.0 - w * sizeof(OutT) + w / 128.0 * (8.0 + 12.0 + 12.0);
  }
  if (g.R)
    CATQ_TRACED(stream, tag, flops, bytes, g.M, g.N, g.K,
                hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WGM, WGN, AKM, BKM, OutT, RT, true, EPI, SB>),
                                   grid, block, 0, stream, L));
  else
    CATQ_TRACED(stream, tag, flops, bytes, g.M, g.N, g.K,
                hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WGM, WGN, AKM, BKM, OutT, RT, false, EPI, SB>),
                                   grid, block, 0, stream, L));
}

// The direct-to-LDS kernel serves dense bf16 problems with K (per split) a
// multiple of 64 and row pitches below 4M elements; a K-major operand also
// needs its tile extent to divide the matrix extent.
static bool dma_ok(const GemmLaunch& L, int a_t, int b_t, int bm, int bn) {
  const GemmArgs& g = L.g;
  // grouped: rows by expert with A K-contiguous, or the contraction by
  // expert with both operands K-major (ragged groups read zero past their end)
  const bool grouping = g.group_mode == 0 || (g.group_mode == 1 && a_t == 0) ||
                        (g.group_mode == 2 && a_t == 1 && b_t == 1);
  return grouping && g.causal == 0 && g.batch == 1 && (g.group_mode == 2 || g.K % 64 == 0) &&
         (L.ksplit <= 1 || L.kchunk % 64 == 0) && g.lda % 8 == 0 && g.ldb % 8 == 0 &&
         g.lda < (1 << 22) && g.ldb < (1 << 22) &&  // 32-bit buffer offsets within a tile
         // a K-major operand's resource spans its whole contraction range
         (a_t == 0 || (uint64_t)(g.K + 64) * (uint64_t)g.lda * 2 < (1ull << 32)) &&
         (b_t == 0 || (uint64_t)(g.K + 64) * (uint64_t)g.ldb * 2 < (1ull << 32)) &&
         aligned16(g.A) && aligned16(g.B) && (a_t == 0 || g.M % bm == 0) &&
         (b_t == 0 || g.N % bn == 0);
}

// A dense product on 256 x 256 tiles.  An unsplit forward product (both
// operands K-contiguous) takes three B stages, its weight's copies two k
// tiles ahead (bit-identical; in the 14B-shaped calibration step down 1.42
// -> 1.38 ms, q|k|v 0.434 -> 0.409 ms, o 0.308 -> 0.299 ms; no loss on the
// 1.7B-shaped block's smaller weights).
template <int A_T, int B_T, typename OutT, typename RT>
static void launch_dense256(GemmLaunch& L, hipStream_t stream) {
  if (A_T == 0 && B_T == 0 && L.ksplit <= 1)
    launch_dma<256, 256, 4, 4, false, false, OutT, RT, 0, 3>(L, stream);
  else
    launch_dma<256, 256, 4, 4, A_T == 1, B_T == 1, OutT, RT>(L, stream);
}

template <int A_T, int B_T, typename OutT, typename RT>
static void launch_bf16(GemmLaunch& L, hipStream_t stream) {
  const GemmArgs& g = L.g;
  if (g.group_mode == 1 && g.N >= 256 && dma_ok(L, A_T, B_T, 256, 256)) {
    // routed experts' rows: 256-row tiles on 16 waves, although each
    // expert's last tile is partly empty (with ~256 rows per expert, 128-row
    // tiles on 8 waves waste less but measured 25% slower).  In the forward
    // each expert's weight streams from HBM for about one row tile: three B
    // stages (copies two k tiles ahead; bit-identical; on the 235B-A22B-
    // shaped gate|up experts 1.17 -> 0.98 ms alone, 1.10 -> 1.09 ms in the
    // calibration step)
    if (A_T == 0 && B_T == 0)
      launch_dma<256, 256, 4, 4, false, false, OutT, RT, 0, 3>(L, stream);
    else
      launch_dma<256, 256, 4, 4, A_T == 1, B_T == 1, OutT, RT>(L, stream);
    return;
  }
  if (g.group_mode == 2 && dma_ok(L, A_T, B_T, 256, 256)) {
    launch_dma<256, 256, 4, 4, A_T == 1, B_T == 1, OutT, RT>(L, stream);
    return;
  }
  // the 256 x 256 tile from 160 tiles on (5/8 of the compute units busy in
  // one round still beats 128 x 128 tiles on 4 waves: the 2048 x 6144 weight
  // gradient over 8192 tokens, unsplit, takes 216 against 260 us)
  const int64_t t256 = ((g.M + 255) / 256) * ((g.N + 255) / 256) * L.ksplit;
  if (g.group_mode == 0 && g.M >= 256 && g.N >= 256 && t256 >= 160 &&
      dma_ok(L, A_T, B_T, 256, 256)) {
    // One workgroup of the 256 x 256 kernel fills a compute unit, so a last
    // round of a quarter to three quarters of the 256 units leaves the rest
    // idle (8192 x 5120 outputs: 640 tiles, 2.5 rounds).  Then the columns
    // past the last whole round go to the 128 x 128 kernel as a launch of
    // their own (two workgroups per unit, one round at most).  Both kernels
    // accumulate an output over K in the same order, so the bits do not
    // change; in the 14B-shaped calibration step the five such products
    // take 0.45 ms less.
    if (L.ksplit <= 1) {
      const int tm = (int)((g.M + 255) / 256), tn = (int)((g.N + 255) / 256);
      const int rem = (tm * tn) % 256;
      int h = 0;  // column tiles of the head: the most that make whole rounds
      if (rem >= 64 && rem <= 192)
        for (int c = tn - 1; c >= 1 && h == 0; --c)
          if ((tm * c) % 256 == 0) h = c;
      if (h > 0) {
        const int64_t nh = (int64_t)h * 256;
        GemmLaunch H = L, T = L;
        H.g.N = nh;
        T.g.N = g.N - nh;
        T.g.B = reinterpret_cast<const bf16*>(g.B) + (B_T ? nh : nh * g.ldb);
        T.g.C = reinterpret_cast<OutT*>(g.C) + nh;
        if (g.R) T.g.R = reinterpret_cast<const RT*>(g.R) + nh;
        const int64_t t128 = ((g.M + 127) / 128) * ((T.g.N + 127) / 128);
        if (t128 <= 512 && dma_ok(T, A_T, B_T, 128, 128)) {
          launch_dense256<A_T, B_T, OutT, RT>(H, stream);
          // the forward layout's split-off columns also take three B stages
          // (80 KB of LDS: two workgroups per unit still fit; 3-6% faster)
          if (A_T == 0 && B_T == 0)
            launch_dma<128, 128, 2, 2, false, false, OutT, RT, 0, 3>(T, stream);
          else
            launch_dma<128, 128, 2, 2, A_T == 1, B_T == 1, OutT, RT>(T, stream);
          return;
        }
      }
    }
    launch_dense256<A_T, B_T, OutT, RT>(L, stream);
    return;
  }
  if (g.group_mode == 0 && dma_ok(L, A_T, B_T, 128, 128)) {
    launch_dma<128, 128, 2, 2, A_T == 1, B_T == 1, OutT, RT>(L, stream);
    return;
  }
  int64_t rows = g.group_mode == 1 ? g.max_rows_per_group : g.M;
  if (rows <= 0) rows = g.M;
  // large output tiles for the big projections, 128x128 for thin problems
  if (rows >= 256 && g.N >= 256 && !(g.causal == 2 || g.causal == 3))
    launch_cfg<256, 256, 2, 4, A_T, B_T, OutT, RT>(L, stream);
  else
    launch_cfg<128, 128, 2, 2, A_T, B_T, OutT, RT>(L, stream);
}

template <typename OutT, typename RT>
static void launch_layout(GemmLaunch& L, int a_t, int b_t, hipStream_t stream) {
  if (a_t == 0 && b_t == 0) launch_bf16<0, 0, OutT, RT>(L, stream);
  else if (a_t == 0 && b_t == 1) launch_bf16<0, 1, OutT, RT>(L, stream);
  else if (a_t == 1 && b_t == 1) launch_bf16<1, 1, OutT, RT>(L, stream);
  else launch_bf16<1, 0, OutT, RT>(L, stream);
}

catq_status gemm_run_split(const GemmArgs& a, int a_t, int b_t, catq_dtype in_dtype,
                           catq_dtype c_dtype, int ksplit, int64_t c_split_stride,
                           hipStream_t stream, catq_dtype r_dtype) {
  GemmLaunch L;
  L.g = a;
  L.ksplit = ksplit > 1 ? ksplit : 1;
  L.kchunk = a.K;
  if (L.ksplit > 1) {
    CATQ_REQUIRE(a.group_mode == 0 && a.batch == 1 && a.causal == 0, CATQ_ERR_VALUE,
                 "split-K needs a dense unbatched problem");
    L.kchunk = (a.K + L.ksplit - 1) / L.ksplit;
    L.kchunk = (L.kchunk + 63) / 64 * 64;
    L.ksplit = (int)((a.K + L.kchunk - 1) / L.kchunk);
  }
  L.c_split_stride = c_split_stride;
  L.tiles_m = L.tiles_n = 0;
  if (a.M <= 0 || a.N <= 0 || a.K <= 0) return CATQ_OK;
  if (in_dtype == CATQ_F32) {
    CATQ_REQUIRE(c_dtype == CATQ_F32 && a.group_mode == 0 && a.batch == 1 && a.causal == 0 &&
                     (a.R == nullptr || r_dtype == CATQ_F32),
                 CATQ_ERR_DTYPE, "fp32 GEMM supports dense, unbatched fp32 problems only");
    dim3 grid((unsigned)((a.N + 63) / 64), (unsigned)((a.M + 63) / 64), (unsigned)L.ksplit);
    if (a_t == 0 && b_t == 0)
      hipLaunchKernelGGL((gemm_f32_kernel<0, 0>), grid, dim3(256), 0, stream, L);
    else if (a_t == 0 && b_t == 1)
      hipLaunchKernelGGL((gemm_f32_kernel<0, 1>), grid, dim3(256), 0, stream, L);
    else if (a_t == 1 && b_t == 1)
      hipLaunchKernelGGL((gemm_f32_kernel<1, 1>), grid, dim3(256), 0, stream, L);
    else
      hipLaunchKernelGGL((gemm_f32_kernel<1, 0>), grid, dim3(256), 0, stream, L);
    CATQ_CHECK_LAUNCH("gemm f32");
    return CATQ_OK;
  }
  CATQ_REQUIRE(in_dtype == CATQ_BF16, CATQ_ERR_DTYPE, "GEMM inputs must be bf16 or f32");
  if (c_dtype == CATQ_BF16) {
    CATQ_REQUIRE(a.R == nullptr || r_dtype == CATQ_BF16, CATQ_ERR_DTYPE,
                 "a bf16 output takes a bf16 residual");
    launch_layout<bf16, bf16>(L, a_t, b_t, stream);
  } else if (a.R != nullptr && r_dtype == CATQ_BF16) {
    launch_layout<float, bf16>(L, a_t, b_t, stream);
  } else {
    launch_layout<float, float>(L, a_t, b_t, stream);
  }
  CATQ_CHECK_LAUNCH("gemm bf16");
  return CATQ_OK;
}

catq_status gemm_run(const GemmArgs& a, int a_t, int b_t, catq_dtype in_dtype, catq_dtype c_dtype,
                     hipStream_t stream, catq_dtype r_dtype) {
  return gemm_run_split(a, a_t, b_t, in_dtype, c_dtype, 1, 0, stream, r_dtype);
}

catq_status gemm_run_epi(const GemmArgs& a, int a_t, int b_t, hipStream_t stream) {
  CATQ_REQUIRE(a.epi == 1 || a.epi == 2, CATQ_ERR_VALUE, "unknown fused epilogue");
  GemmLaunch L;
  L.g = a;
  L.ksplit = 1;
  L.kchunk = a.K;
  L.c_split_stride = 0;
  L.tiles_m = L.tiles_n = 0;
  if (a.M <= 0 || a.N <= 0 || a.K <= 0) return CATQ_OK;
  // the vector epilogue: 4 consecutive columns per lane, 4-byte (EPI 1) or
  // 8-byte (EPI 2) aligned rows of every output; and the shapes on which the
  // plain GEMM takes the same 256 x 256 kernel, so fused and unfused results
  // are the same bits
  const int64_t t256 = ((a.M + 255) / 256) * ((a.N + 255) / 256);
  const bool shape = t256 >= 160 && a.R == nullptr && a.alpha == 1.0f && a.N % 4 == 0 &&
                     a.ldc % 4 == 0 && a.ld_aux % 4 == 0 && aligned16(a.C) && aligned16(a.aux0) &&
                     (a.epi == 1 || aligned16(a.aux1));
  if (a.epi == 1) {
    // A [M][K] tokens (K-contiguous), B the fused weight [N][K]
    if (!(shape && a_t == 0 && b_t == 0 && a.M >= 256 && a.N >= 256 && dma_ok(L, 0, 0, 256, 256)))
      return CATQ_ERR_VALUE;
    // three B stages, as the plain forward products (bit-identical; 2.47 ->
    // 2.39 ms on the 14B-shaped gate|up in the calibration step)
    launch_dma<256, 256, 4, 4, false, false, bf16, bf16, 1, 3>(L, stream);
  } else {
    // dX-shaped: A = dY [M][K] (K-contiguous), B = W_fake [K][N] (K-major)
    if (!(shape && a_t == 0 && b_t == 1 && a.M >= 256 && a.N >= 256 && dma_ok(L, 0, 1, 256, 256)))
      return CATQ_ERR_VALUE;
    launch_dma<256, 256, 4, 4, false, true, bf16, bf16, 2>(L, stream);
  }
  CATQ_CHECK_LAUNCH("gemm fused epilogue");
  return CATQ_OK;
}

catq_status gemm_run_factor(const GemmArgs& a, hipStream_t stream) {
  CATQ_REQUIRE(a.epi == 3 && (a.group_mode == 2 || (a.group_mode == 0 && a.batch == 1 &&
                                                     a.causal == 0)),
               CATQ_ERR_VALUE, "not a factor-gradient launch");
  GemmLaunch L;
  L.g = a;
  L.ksplit = 1;
  L.kchunk = a.K;
  L.c_split_stride = 0;
  L.tiles_m = L.tiles_n = 0;
  // G [rows][d_in] (per expert, or one dense unsplit problem) from K-major
  // dY and X; whole 256 x 256 tiles (128-weight groups never straddle them),
  // C only as an aligned dummy
  const bool shape = a.M > 0 && a.N > 0 && a.M % 256 == 0 && a.N % 256 == 0 && a.alpha == 1.0f &&
                     a.R == nullptr && a.c_gs == 0 && a.ldc % 4 == 0 && aligned16(a.C) &&
                     a.fac.W != nullptr && (reinterpret_cast<uintptr_t>(a.fac.W) & 7) == 0 &&
                     a.fac.ldw == a.N && dma_ok(L, 1, 1, 256, 256);
  if (!shape) return CATQ_ERR_VALUE;
  if (a.group_mode == 0) {
    // A partial last round of a quarter to three quarters of the 256
    // compute units (5120 x 17408: 1360 tiles, 5.3 rounds): the columns past
    // the last whole round run as a 128 x 128 launch of their own (two
    // workgroups per unit, one round at most), with the weights, group
    // arrays and outputs taken from that column on (the row pitch of W, and
    // so the group numbering, stays the whole d_in)
    const int tm = (int)(a.M / 256), tn = (int)(a.N / 256);
    const int rem = (tm * tn) % 256;
    int h = 0;
    if (rem >= 64 && rem <= 192)
      for (int c = tn - 1; c >= 1 && h == 0; --c)
        if ((tm * c) % 256 == 0) h = c;
    if (h > 0) {
      const int64_t nh = (int64_t)h * 256, gsh = nh / 128;
      GemmLaunch H = L, T = L;
      H.g.N = nh;
      T.g.N = a.N - nh;
      T.g.B = reinterpret_cast<const bf16*>(a.B) + nh;
      FacEpi& F = T.g.fac;
      F.W = reinterpret_cast<const bf16*>(F.W) + nh;
      F.stats += 2 * gsh;
      F.dmu += gsh * F.s[0];
      F.dal += gsh * F.s[1];
      F.dde += gsh * F.s[2];
      for (int k = 0; k < 3; ++k)
        if (F.s[k] == 1) F.out[k] += gsh;
      if (F.ws != nullptr) F.ws += gsh;
      const int64_t t128 = (a.M / 128) * (T.g.N / 128);
      if (t128 <= 512 && dma_ok(T, 1, 1, 128, 128)) {
        launch_dma<256, 256, 4, 4, true, true, float, float, 3>(H, stream);
        launch_dma<128, 128, 2, 2, true, true, float, float, 3>(T, stream);
        CATQ_CHECK_LAUNCH("gemm factor epilogue");
        return CATQ_OK;
      }
    }
  }
  launch_dma<256, 256, 4, 4, true, true, float, float, 3>(L, stream);
  CATQ_CHECK_LAUNCH("gemm factor epilogue");
  return CATQ_OK;
}

int gemm_split_count(const GemmArgs& a, int ksplit) {
  if (ksplit <= 1) return 1;
  int64_t kchunk = (a.K + ksplit - 1) / ksplit;
  kchunk = (kchunk + 63) / 64 * 64;
  return (int)((a.K + kchunk - 1) / kchunk);
}

}  // namespace catq
