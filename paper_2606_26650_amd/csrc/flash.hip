// Fused causal grouped-query attention (forward and backward) on matrix cores
// (gfx950, v_mfma_f32_32x32x16_bf16), head dimension D in {64, 128}.
//
// Layout trick: every score tile is computed as S^T (keys x queries), so the
// 32x32 accumulator gives each lane ONE query column and 16 key rows.  The
// softmax over keys is then a reduction over the lane's own registers plus one
// exchange with lane^32, and the accumulator registers are directly the MFMA
// operand of the next product (P.V, dS.K, ...) once the other operand is read
// from LDS in the same key order (keys 4g..4g+3 and 8+4g..8+4g+3 of each
// 16-key slice, g = lane/32).
//
// Forward: one block = 4 wavefronts x 32 queries of one (batch, q head); key
// tiles of 64 stream through LDS (K as [key][d], V transposed as [d][key]);
// online softmax in base 2; O written token-major, and the per-query
// log-sum-exp (base 2) kept for the backward.
// Backward: dK/dV kernel (block = 128 keys of one kv head, four wavefronts
// accumulating dV and four dK, looping over the q heads of its group and the
// causal query tiles) and dQ kernel (block = 4 x 32 queries, looping over key
// tiles); P and dS are recomputed from the saved log-sum-exp and
// D = rowsum(dO * O).  No atomics: every output element is owned by one lane.
#include <cmath>

#include "kernels.h"

namespace catq {

namespace fa {

constexpr int BK = 64;   // keys (or queries) per streamed tile
constexpr int NT = 256;  // 4 wavefronts
constexpr int TP = BK + 4;  // pitch (elements) of transposed [d][64] tiles

template <int D>
struct Cfg {
  static constexpr int KP = D + 8;             // pitch of [row][d] tiles (16-byte rows)
  static constexpr int NCH = D / 8;            // 16-byte chunks per row
  static constexpr int ITEMS = (BK / 4) * NCH;  // 4-row x 8-column items per tile
  static constexpr int KS = D / 16;            // 16-wide slices of d
  static constexpr int DB = D / 32;            // 32-row blocks of d
};

// Registers of one 64 x D tile: each thread owns rows 4*kb4 .. 4*kb4+3 and
// columns 8*db .. 8*db+7 (db varies fastest across lanes: 16-byte loads of
// consecutive lanes are contiguous in a row).
template <int D>
struct Tile {
  u32x4 r[4];
  bool active;
  int kb4, db;
  __device__ __forceinline__ void load(const bf16* __restrict__ base, int64_t ld, int64_t row0,
                                       int64_t rows, int tid) {
    active = tid < Cfg<D>::ITEMS;
    db = tid % Cfg<D>::NCH;
    kb4 = tid / Cfg<D>::NCH;
    const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t row = row0 + 4 * kb4 + j;
      r[j] = (active && row < rows)
                 ? *reinterpret_cast<const u32x4*>(base + row * ld + 8 * db)
                 : z;
    }
  }
  // [row][KP] layout
  __device__ __forceinline__ void store_rows(u16* lds) const {
    if (!active) return;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *reinterpret_cast<u32x4*>(lds + (4 * kb4 + j) * Cfg<D>::KP + 8 * db) = r[j];
  }
  // [d][TP] layout, 4-element quads XOR-swizzled by (d >> 3) & 15
  __device__ __forceinline__ void store_transposed(u16* lds) const {
    if (!active) return;
#pragma unroll
    for (int mm = 0; mm < 8; ++mm) {
      const unsigned sel = (mm & 1) ? 0x07060302u : 0x05040100u;
      const int dw = mm >> 1;
      uint2 o;
      o.x = __builtin_amdgcn_perm(r[1][dw], r[0][dw], sel);
      o.y = __builtin_amdgcn_perm(r[3][dw], r[2][dw], sel);
      const int d = 8 * db + mm;
      const int q = kb4 ^ ((d >> 3) & 15);
      *reinterpret_cast<uint2*>(lds + d * TP + 4 * q) = o;
    }
  }
};

__device__ __forceinline__ bf16x8 frag_rows(const u16* lds, int row, int col, int pitch) {
  return *reinterpret_cast<const bf16x8*>(lds + row * pitch + col);
}

// Operand fragment from a transposed [d][TP] tile: row d, keys
// 16*slice + 4g .. +3 and 16*slice + 8 + 4g .. +3 (slice = 16-key slice index)
__device__ __forceinline__ bf16x8 frag_tr(const u16* lds, int d, int slice, int g) {
  const int s = (d >> 3) & 15;
  const int q1 = (4 * slice + g) ^ s, q2 = (4 * slice + 2 + g) ^ s;
  const uint2 a = *reinterpret_cast<const uint2*>(lds + d * TP + 4 * q1);
  const uint2 b = *reinterpret_cast<const uint2*>(lds + d * TP + 4 * q2);
  u32x4 v = {a.x, a.y, b.x, b.y};
  return __builtin_bit_cast(bf16x8, v);
}

// 8 accumulator values (regs 8h..8h+7 of a 32x32 block) -> bf16 operand
__device__ __forceinline__ bf16x8 pack8(const f32x16& a, int h) {
  u32x4 v;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = pack_bf16x2(a[8 * h + 2 * i], a[8 * h + 2 * i + 1]);
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

// row (within a 32-row accumulator block) of register r for lane group g
__device__ __forceinline__ int acc_row(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }

// Row-major 64 x D tiles filled by direct-to-LDS copies.  The 16-byte chunk
// c of row r sits at slot r*(D/8) + (c ^ tswz(r)).  For D = 128 the key
// ((r & 3) << 2) | ((r >> 2) & 3) puts both the 128-bit reads of 16
// consecutive rows at one chunk (fragments of K, Q, dO, V rows) and the
// transpose reads of 4 consecutive rows x 4 chunks (fragments of V^T, K^T,
// Q^T, dO^T) on 16 distinct bank groups; for D = 64 (8 chunks a row, two
// rows per 256-byte bank cycle) the key (r >> 1) & 7 does the former.
template <int D>
__device__ __forceinline__ int tswz(int r) {
  if constexpr (D == 128)
    return ((r & 3) << 2) | ((r >> 2) & 3);
  else
    return (r >> 1) & 7;
}

// 64 rows of D bf16 from row0 (rows at or past `rows` read the last row);
// all four wavefronts of the block take part.
template <int D>
__device__ __forceinline__ void dma_tile(const bf16* base, int64_t ld, int64_t row0, int64_t rows,
                                         uint4* lds, int wave, int lane) {
  constexpr int CPR = D / 8, RPI = 64 / CPR, NI = 64 / RPI / 4;
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int r = (wave * NI + i) * RPI + lane / CPR;
    const int c = (lane % CPR) ^ tswz<D>(r);
    dma16(base + min(row0 + r, rows - 1) * ld + c * 8, &lds[(wave * NI + i) * 64]);
  }
}

// The same 64 x D tile copy through a buffer resource: a lane keeps the byte
// offsets of its NI 16-byte chunks within a tile (rows past the sequence
// read as zero; their queries are masked), and each tile costs one resource
// and NI copies.
template <int D>
struct TileCopy {
  static constexpr int CPR = D / 8, RPI = 64 / CPR, NI = 64 / RPI / 4;
  uint32_t voff[NI];
  // wave: 0..3 within the four copying waves
  __device__ __forceinline__ void init(int64_t ld, int wave, int lane) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = (wave * NI + i) * RPI + lane / CPR;
      const int c = (lane % CPR) ^ tswz<D>(r);
      voff[i] = (uint32_t)((int64_t)r * ld * 2 + c * 16);
    }
  }
  __device__ __forceinline__ void issue(const bf16* base, int64_t ld, int row0, int rows, uint4* lds,
                                        int wave) const {
    const i32x4_rsrc rs = buf_rsrc(base + (int64_t)row0 * ld, (uint32_t)((int64_t)(rows - row0) * ld * 2));
#pragma unroll
    for (int i = 0; i < NI; ++i) dma16_buf(rs, voff[i], 0u, &lds[(wave * NI + i) * 64]);
  }
};

// Fragment of row `row`, 16-byte chunk `chunk` (8 consecutive columns).
template <int D>
__device__ __forceinline__ bf16x8 tfrag_row(const uint4* lds, int row, int chunk) {
  return *reinterpret_cast<const bf16x8*>(&lds[row * (D / 8) + (chunk ^ tswz<D>(row))]);
}

// Two independent 32-row accumulation chains over the D/16 slices of d:
// s[c] += (rows 32c + l32 of a swizzled row-major LDS tile) x b[t].  Each
// fragment is read PF slices ahead of its products, and a scheduling barrier
// that only vector and scalar ALU work may cross keeps it there: left alone,
// the scheduler sinks every read next to its product, and each slice then
// waits out the whole LDS latency.
template <int D, int PF>
__device__ __forceinline__ void chains2(const uint4* lds, const bf16x8 (&b)[D / 16], int l32,
                                        int g, f32x16 (&s)[2]) {
  constexpr int KS = D / 16, NB = PF + 1;
  bf16x8 fr[NB][2];
#pragma unroll
  for (int t = 0; t < PF; ++t) {
    fr[t][0] = tfrag_row<D>(lds, l32, 2 * t + g);
    fr[t][1] = tfrag_row<D>(lds, 32 + l32, 2 * t + g);
  }
#pragma unroll
  for (int t = 0; t < KS; ++t) {
    if (t + PF < KS) {
      fr[(t + PF) % NB][0] = tfrag_row<D>(lds, l32, 2 * (t + PF) + g);
      fr[(t + PF) % NB][1] = tfrag_row<D>(lds, 32 + l32, 2 * (t + PF) + g);
    }
    __builtin_amdgcn_sched_barrier(0x0406);
    s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[t % NB][0], b[t], s[0], 0, 0, 0);
    s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[t % NB][1], b[t], s[1], 0, 0, 0);
  }
}

// Transposed fragment: column col0 + lane%32, rows 16*slice + 4g + 0..3 then
// 16*slice + 8 + 4g + 0..3 (g = lane/32): the permuted key order of the
// score accumulators, read with two transpose loads.
template <int D>
__device__ __forceinline__ bf16x8 tfrag_tr(const uint4* lds, int col0, int slice, int lane) {
  const int blk = lane >> 4, s = lane & 15;
  const int col = col0 + 16 * (blk & 1) + 4 * (s & 3);
  u32x4 u;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int row = 16 * slice + 4 * (blk >> 1) + 8 * c + (s >> 2);
    const short* p = reinterpret_cast<const short*>(lds) + row * D +
                     (((col >> 3) ^ tswz<D>(row)) << 3) + (col & 7);
    const lds_v4s v = lds_read_tr16(p);
    u[2 * c] = (unsigned)(unsigned short)v[0] | ((unsigned)(unsigned short)v[1] << 16);
    u[2 * c + 1] = (unsigned)(unsigned short)v[2] | ((unsigned)(unsigned short)v[3] << 16);
  }
  return __builtin_bit_cast(bf16x8, u);
}

// Per-lane offsets (in bf16 elements) of the two transpose reads of
// tfrag_tr for each 32-column block i of a 64 x D tile.  The swizzle key of
// a row does not depend on its 16-row slice, so the reads of slice `slice`
// sit 16 * slice rows further: tr_read adds that as a constant.
template <int D>
struct TrOffsets {
  int o[D / 32][2];
  __device__ __forceinline__ void init(int lane) {
    const int blk = lane >> 4, s = lane & 15;
#pragma unroll
    for (int i = 0; i < D / 32; ++i)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int col = i * 32 + 16 * (blk & 1) + 4 * (s & 3);
        const int row = 4 * (blk >> 1) + 8 * c + (s >> 2);
        o[i][c] = row * D + (((col >> 3) ^ tswz<D>(row)) << 3) + (col & 7);
      }
  }
};

// tfrag_tr<D>(lds, 32 * i, slice, lane) from precomputed offsets
template <int D>
__device__ __forceinline__ bf16x8 tr_read(const uint4* lds, const TrOffsets<D>& t, int i,
                                          int slice) {
  const short* base = reinterpret_cast<const short*>(lds) + 16 * slice * D;
  u32x4 u;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const lds_v4s v = lds_read_tr16(base + t.o[i][c]);
    u[2 * c] = (unsigned)(unsigned short)v[0] | ((unsigned)(unsigned short)v[1] << 16);
    u[2 * c + 1] = (unsigned)(unsigned short)v[2] | ((unsigned)(unsigned short)v[3] << 16);
  }
  return __builtin_bit_cast(bf16x8, u);
}

}  // namespace fa

// ------------------------------------------------------------------ forward

template <int D>
__global__ __launch_bounds__(fa::NT, 2) void flash_fwd_kernel(FaArgs a) {
  using C = fa::Cfg<D>;
  constexpr int TW = 64 * D / 8;  // 16-byte slots of one 64 x D tile
  __shared__ uint4 sK[2][TW];
  __shared__ uint4 sV[2][TW];
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  // grid (B*Hq, query tiles): the longest causal rows are dispatched first
  const int qt = (int)gridDim.y - 1 - (int)blockIdx.y;
  const int h = blockIdx.x % a.Hq, b = blockIdx.x / a.Hq;
  const int kvh = h / (a.Hq / a.Hkv);
  const int q0 = qt * 128;
  const int qme = q0 + 32 * w + l32;  // this lane's query
  const bf16* Qb = a.Q + ((int64_t)(b * a.Hq + h) * a.S) * D;
  const bf16* Kb = a.K + ((int64_t)(b * a.Hkv + kvh) * a.S) * D;
  const bf16* Vb = a.V + ((int64_t)(b * a.Hkv + kvh) * a.S) * D;

  // Q fragments (operand B of S^T = K Q^T): lane holds query qme, d slice t
  bf16x8 qf[C::KS];
#pragma unroll
  for (int t = 0; t < C::KS; ++t) {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (qme < a.S) v = *reinterpret_cast<const u32x4*>(Qb + (int64_t)qme * D + 16 * t + 8 * g);
    qf[t] = __builtin_bit_cast(bf16x8, v);
  }
  f32x16 o[C::DB];
#pragma unroll
  for (int i = 0; i < C::DB; ++i) o[i] = fa::zero16();
  float m = -INFINITY, l = 0.f;  // running max (base-2 units) and sum

  const int q_last = min(q0 + 127, a.S - 1);
  const int nkt = q_last / fa::BK + 1;
  const int wave_first = q0 + 32 * w, wave_last = wave_first + 31;
  fa::TrOffsets<D> tro;
  tro.init(lane);
  // K and V rows by buffer copies (one set of lane offsets for both; rows
  // past the sequence read as zero, their keys are masked)
  fa::TileCopy<D> tcp;
  tcp.init(D, w, lane);
  auto issueK = [&](int buf, int k0) { tcp.issue(Kb, D, k0, a.S, sK[buf], w); };
  auto issueV = [&](int buf, int k0) { tcp.issue(Vb, D, k0, a.S, sV[buf], w); };
  // S^T of one key tile (K rows in `kl`) for the two 32-key blocks: two
  // independent accumulation chains, each fragment read one step ahead of
  // its products
  auto scores = [&](const uint4* kl, f32x16 (&s)[2]) {
    s[0] = fa::zero16();
    s[1] = fa::zero16();
    bf16x8 fr[2][2];
    fr[0][0] = fa::tfrag_row<D>(kl, l32, g);
    fr[0][1] = fa::tfrag_row<D>(kl, 32 + l32, g);
#pragma unroll
    for (int t = 0; t < C::KS; ++t) {
      if (t + 1 < C::KS) {
        fr[(t + 1) & 1][0] = fa::tfrag_row<D>(kl, l32, 2 * (t + 1) + g);
        fr[(t + 1) & 1][1] = fa::tfrag_row<D>(kl, 32 + l32, 2 * (t + 1) + g);
      }
      s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[t & 1][0], qf[t], s[0], 0, 0, 0);
      s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[t & 1][1], qf[t], s[1], 0, 0, 0);
    }
  };
  // Online softmax of one (masked) score tile, first half: the tile max of
  // the raw scores (the scale c > 0 commutes with it), the new running max
  // (msafe: 0 for a lane whose query lies past the sequence end, which sees
  // only masked keys) and the rescale factor of the old sums.  alpha == 1
  // exactly unless the running max moved: O is rescaled only when it moved
  // for some lane of the wave.
  auto tile_max = [&](f32x16 (&s)[2], float& msafe, float& alpha) {
    float mt = -INFINITY;
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s[sb][r]);
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float mn = fmaxf(m, mt * a.c);
    msafe = (mn == -INFINITY) ? 0.f : mn;
    alpha = __builtin_amdgcn_exp2f(m - msafe);
    const bool moved = mn != m;
    m = mn;
    if (__any(moved)) {
#pragma unroll
      for (int i = 0; i < C::DB; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[i][r] *= alpha;
    }
  };
  // second half: P = 2^(c s - m), packed as the bf16 operand of the
  // products, O^T += V^T P^T (V^T fragments by transpose reads of the V rows
  // in `vl`), l = alpha l + rowsum P
  auto accumulate = [&](f32x16 (&s)[2], const uint4* vl, float msafe, float alpha) {
    float rs = 0.f;
    bf16x8 pk[4];
#pragma unroll
    for (int sb = 0; sb < 2; ++sb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[sb][r], a.c, -msafe));
        s[sb][r] = p;
        rs += p;
      }
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) pk[2 * sb + hh] = fa::pack8(s[sb], hh);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int i = 0; i < C::DB; ++i)
        o[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa::tr_read<D>(vl, tro, i, j), pk[j], o[i], 0,
                                                       0, 0);
    rs += __shfl_xor(rs, 32, 64);
    l = l * alpha + rs;
  };

  // Software pipeline over key tiles: K runs one tile ahead of V, so while
  // the exponentials of tile kt run on the vector ALUs the scores of tile
  // kt+1 go to the matrix cores.  Prologue: K and V of tile 0, K of tile 1,
  // the scores of tile 0 (every wave reads tile 0: wave_last >= 31).
  issueK(0, 0);
  issueV(0, 0);
  if (nkt > 1) issueK(1, fa::BK);
  wait_vmem();
  __syncthreads();
  f32x16 sc[2];
  scores(sK[0], sc);
  // every wave has read K of tile 0 before tile 2 takes its buffer
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    const int k0 = kt * fa::BK, buf = kt & 1;
    // V of tile kt+1 into the buffer V of tile kt-1 left, K of tile kt+2
    // into that of tile kt (both read before the previous barrier)
    if (kt + 1 < nkt) issueV(buf ^ 1, k0 + fa::BK);
    if (kt + 2 < nkt) issueK(buf, k0 + 2 * fa::BK);
    if (k0 <= wave_last) {
      // A tile followed by another of the same wave lies wholly below the
      // wave's diagonal and inside the sequence (the next tile starts at or
      // before wave_last < S; tile starts are multiples of 64, wave starts
      // of 32): only the wave's last tile may need the causal / length mask.
      const bool next = kt + 1 < nkt && k0 + fa::BK <= wave_last;
      if (!next && (k0 + fa::BK - 1 > wave_first || k0 + fa::BK > a.S)) {
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = k0 + sb * 32 + fa::acc_row(r, g);
            if (key > qme || key >= a.S) sc[sb][r] = -INFINITY;
          }
      }
      float msafe, alpha;
      tile_max(sc, msafe, alpha);
      // One basic block: the next tile's scores beside this tile's
      // exponentials, then this tile's products.  On the wave's last tile
      // the scores read the other K buffer (a stale tile, or none filled
      // since) and are discarded: the wave skips every later tile.
      f32x16 sn[2];
      scores(sK[buf ^ 1], sn);
      accumulate(sc, sV[buf], msafe, alpha);
      sc[0] = sn[0];
      sc[1] = sn[1];
    }
    wait_vmem();
    __syncthreads();
  }
  if (qme < a.S) {
    const float inv = 1.0f / l;
    bf16* Ob = a.O + ((int64_t)b * a.S + qme) * (int64_t)(a.Hq * D) + (int64_t)h * D;
#pragma unroll
    for (int i = 0; i < C::DB; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) Ob[i * 32 + fa::acc_row(r, g)] = (bf16)(o[i][r] * inv);
    if (g == 0) a.lse[(int64_t)(b * a.Hq + h) * a.S + qme] = m + log2f(l);
  }
}

// D = rowsum(dO * O) per (batch, q head, query): D/8 lanes per row, each
// lane one 16-byte chunk of O and of dO.
template <int D>
__global__ __launch_bounds__(256) void flash_dsum_kernel(FaArgs a) {
  constexpr int LPR = D / 8;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = gid / LPR;  // (b*S + q)*Hq + h
  const int sub = (int)(gid % LPR);
  if (row >= (int64_t)a.B * a.S * a.Hq) return;  // whole rows: LPR divides 64
  const int h = (int)(row % a.Hq);
  const int64_t t = row / a.Hq;  // token b*S + q
  const int64_t off = t * (int64_t)(a.Hq * D) + (int64_t)h * D + 8 * sub;
  float o[8], d[8];
  load8<bf16>(a.O + off, o);
  load8<bf16>(a.dO + off, d);
  float acc = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) acc = fmaf(o[j], d[j], acc);
#pragma unroll
  for (int m = LPR >> 1; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 64);
  if (sub == 0) {
    const int64_t b = t / a.S, q = t % a.S;
    a.Dsum[(b * a.Hq + h) * a.S + q] = acc;
  }
}

// ------------------------------------------------------------- dK and dV
//
// Block = 8 wavefronts over 128 keys of one kv head.  Waves 0-3 accumulate
// dV and waves 4-7 dK, each for the 32 keys of slab w % 4.  Q and dO tiles of
// 64 queries stream into double-buffered swizzled row-major LDS tiles by
// direct copies (waves 0-3 copy Q, 4-7 dO, with the tile's log-sum-exp and
// D), one tile ahead.  Per tile the dV wave of a slab forms S^T and P
// (exponentials, mask) and hands P to the dK wave of the same slab through
// LDS, while that wave forms dP^T; the two waves hold P and dP in the same
// register layout (lane = key, registers = queries), so after one barrier
// the dK wave forms dS = P (dP - D) from P read back at its own lane.  The
// products with dO^T and Q^T take their operands by transpose reads of the
// row-major tiles.  Each wave holds one 32 x D accumulator set and issues 32
// MFMAs per tile (two independent 32-query chains for the scores, four
// accumulators for the products); two waves share a SIMD.

constexpr int DKDV_NT = 512;

template <int D, int ROLE>  // ROLE 0: dV, 1: dK
__device__ __forceinline__ void dkdv_waves(const FaArgs& a, uint4* sQ, uint4* sO, float* sL,
                                           float* sD, float* sP) {
  using C = fa::Cfg<D>;
  constexpr int TW = 64 * D / 8;  // 16-byte slots of one 64 x D tile
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int ks = __builtin_amdgcn_readfirstlane(tid >> 6) & 3;  // key slab of this wave
  // grid (B*Hkv*hsplit, key tiles): block chunk of a kv head takes its share
  // of the group's q heads and writes its own partial dK/dV
  const int chunk = blockIdx.x % a.hsplit, bk = blockIdx.x / a.hsplit;
  const int kt = blockIdx.y, kvh = bk % a.Hkv, b = bk / a.Hkv;
  const int G = a.Hq / a.Hkv, Gc = G / a.hsplit;
  const int k0 = kt * 128;
  const int wave_first = k0 + 32 * ks;  // queries below this see none of the wave's keys
  const int kme = wave_first + l32;     // this lane's key (column of S^T[q][key])
  // this lane's K row (dV waves: operand B of S^T = Q K^T) or V row (dK
  // waves: operand B of dP^T = dO V^T)
  const bf16* Rb = (ROLE == 0 ? a.K : a.V) + ((int64_t)(b * a.Hkv + kvh) * a.S) * D;
  bf16x8 rf[C::KS];
#pragma unroll
  for (int t = 0; t < C::KS; ++t) {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (kme < a.S) v = *reinterpret_cast<const u32x4*>(Rb + (int64_t)kme * D + 16 * t + 8 * g);
    rf[t] = __builtin_bit_cast(bf16x8, v);
  }
  f32x16 acc[C::DB];
#pragma unroll
  for (int i = 0; i < C::DB; ++i) acc[i] = fa::zero16();
  fa::TrOffsets<D> tro;
  tro.init(lane);
  fa::TileCopy<D> tcp;
  tcp.init(ROLE == 0 ? (int64_t)D : (int64_t)a.Hq * D, ks, lane);
  const int qt0 = k0 / fa::BK;
  const int nqt = (a.S + fa::BK - 1) / fa::BK;
  // P of this slab and a tile's 64 queries: [2 x 32-query blocks][4][64
  // lanes][4] floats (lane-major 16-byte chunks, no bank conflicts)
  float* P = sP + ks * (2 * 16 * 64);
  for (int gq = chunk * Gc; gq < (chunk + 1) * Gc; ++gq) {
    const int h = kvh * G + gq;
    const bf16* Qb = a.Q + ((int64_t)(b * a.Hq + h) * a.S) * D;
    const bf16* dOb = a.dO + (int64_t)b * a.S * (a.Hq * D) + (int64_t)h * D;
    // log-sum-exp (Q copiers) or D (dO copiers) of the head's queries; reads
    // past the sequence end land as zero
    const float* LDb = (ROLE == 0 ? a.lse : a.Dsum) + (int64_t)(b * a.Hq + h) * a.S;
    const i32x4_rsrc ld_rs = buf_rsrc(LDb, (uint32_t)a.S * 4u);
    // this wave's share of the copies of tile q0n into buffer buf
    auto issue = [&](int buf, int q0n) {
      if (ROLE == 0)
        tcp.issue(Qb, D, q0n, a.S, sQ + buf * TW, ks);
      else
        tcp.issue(dOb, (int64_t)a.Hq * D, q0n, a.S, sO + buf * TW, ks);
      if (ks == 0) dma4_buf(ld_rs, (uint32_t)(q0n + lane) * 4u, (ROLE == 0 ? sL : sD) + buf * 64);
    };
    // the first tile's copies; a tile's buffers are refilled only after the
    // barrier that ends the tile two before it
    issue(0, qt0 * fa::BK);
    wait_vmem();
    __syncthreads();
    for (int qt = qt0; qt < nqt; ++qt) {
      const int q0 = qt * fa::BK, buf = (qt - qt0) & 1;
      if (qt + 1 < nqt) issue(buf ^ 1, q0 + fa::BK);
      const uint4* tQ = sQ + buf * TW;
      const uint4* tO = sO + buf * TW;
      const float* tL = sL + buf * 64;
      const float* tD = sD + buf * 64;
      // a tile wholly before the slab's keys is skipped, but its copies and
      // barriers are kept (both waves of a slab skip alike)
      const bool active = q0 + fa::BK - 1 >= wave_first;
      // S^T[q][key] (dV waves) or dP^T[q][key] (dK waves) for the two 32-query
      // blocks: two independent accumulation chains
      f32x16 s[2];
      s[0] = fa::zero16();
      s[1] = fa::zero16();
      if (active) {
        fa::chains2<D, 2>(ROLE == 0 ? tQ : tO, rf, l32, g, s);
        if constexpr (ROLE == 0) {
          // P, rows = queries of this lane's registers; the causal / length
          // mask only on the 32 x 32 blocks that cross the slab's diagonal or
          // the sequence end (uniform)
#pragma unroll
          for (int qb = 0; qb < 2; ++qb) {
            const int qb0 = q0 + qb * 32;
            const bool masked = qb0 < wave_first + 31 || qb0 + 32 > a.S || wave_first + 31 >= a.S;
            if (masked) {
#pragma unroll
              for (int r = 0; r < 16; ++r) {
                const int qi = qb * 32 + fa::acc_row(r, g);
                const int q = q0 + qi;
                const float p = __builtin_amdgcn_exp2f(fmaf(s[qb][r], a.c, -tL[qi]));
                s[qb][r] = (q < kme || q >= a.S || kme >= a.S) ? 0.f : p;
              }
            } else {
#pragma unroll
              for (int r = 0; r < 16; ++r) {
                const int qi = qb * 32 + fa::acc_row(r, g);
                s[qb][r] = __builtin_amdgcn_exp2f(fmaf(s[qb][r], a.c, -tL[qi]));
              }
            }
#pragma unroll
            for (int c = 0; c < 4; ++c) {
              f32x4 v = {s[qb][4 * c], s[qb][4 * c + 1], s[qb][4 * c + 2], s[qb][4 * c + 3]};
              *reinterpret_cast<f32x4*>(P + ((qb * 4 + c) * 64 + lane) * 4) = v;
            }
          }
        } else {
          // dP - D while the dV waves form P
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int r = 0; r < 16; ++r) s[qb][r] -= tD[qb * 32 + fa::acc_row(r, g)];
        }
      }
      __syncthreads();
      if (active) {
        if constexpr (ROLE == 1) {
          // dS = P (dP - D)
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
              const f32x4 pv = *reinterpret_cast<const f32x4*>(P + ((qb * 4 + c) * 64 + lane) * 4);
#pragma unroll
              for (int e = 0; e < 4; ++e) s[qb][4 * c + e] *= pv[e];
            }
        }
        // dV[key][d] += P^T dO ; dK[key][d] += dS^T Q  (contraction over the
        // tile's queries, 16 at a time; dO^T and Q^T by transpose reads)
        const uint4* tsrc = ROLE == 0 ? tO : tQ;
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const bf16x8 pf = fa::pack8(s[qb], hh);
#pragma unroll
            for (int i = 0; i < C::DB; ++i)
              acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                  pf, fa::tr_read<D>(tsrc, tro, i, 2 * qb + hh), acc[i], 0, 0, 0);
          }
      }
      // the next tile's copies have landed; this tile's buffers and P are free
      wait_vmem();
      __syncthreads();
    }
  }
  // acc[i][r]: key row = 32 ks + acc_row(r, g) within the block, d column = 32 i + l32
  const int64_t part = (int64_t)chunk * a.B * a.Hkv * a.S * D;
  float* outb = (ROLE == 0 ? a.dV : a.dK) + part + ((int64_t)(b * a.Hkv + kvh) * a.S) * D;
  const float sc = ROLE == 0 ? 1.0f : a.scale;
#pragma unroll
  for (int i = 0; i < C::DB; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = wave_first + fa::acc_row(r, g);
      if (key < a.S) outb[(int64_t)key * D + 32 * i + l32] = acc[i][r] * sc;
    }
}

template <int D>
__global__ __launch_bounds__(DKDV_NT, 2) void flash_bwd_dkdv_kernel(FaArgs a) {
  constexpr int TW = 64 * D / 8;
  __shared__ uint4 sQ[2 * TW];  // Q tiles (row-major, swizzled), double-buffered
  __shared__ uint4 sO[2 * TW];  // dO tiles
  __shared__ __attribute__((aligned(16))) float sL[2 * 64], sD[2 * 64];
  __shared__ __attribute__((aligned(16))) float sP[4 * 2 * 16 * 64];  // P handed from dV to dK waves
  if (__builtin_amdgcn_readfirstlane(threadIdx.x >> 6) < 4)
    dkdv_waves<D, 0>(a, sQ, sO, sL, sD, sP);
  else
    dkdv_waves<D, 1>(a, sQ, sO, sL, sD, sP);
}

// ------------------------------------------------------------------- dQ

template <int D>
__global__ __launch_bounds__(fa::NT, 2) void flash_bwd_dq_kernel(FaArgs a) {
  using C = fa::Cfg<D>;
  constexpr int TW = 64 * D / 8;  // 16-byte slots of one 64 x D tile
  __shared__ uint4 sK[2][TW];
  __shared__ uint4 sV[2][TW];
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  // grid (B*Hq, query tiles): the longest causal rows are dispatched first
  const int qt = (int)gridDim.y - 1 - (int)blockIdx.y;
  const int h = blockIdx.x % a.Hq, b = blockIdx.x / a.Hq;
  const int kvh = h / (a.Hq / a.Hkv);
  const int q0 = qt * 128;
  const int qme = q0 + 32 * w + l32;
  const bf16* Qb = a.Q + ((int64_t)(b * a.Hq + h) * a.S) * D;
  const bf16* Kb = a.K + ((int64_t)(b * a.Hkv + kvh) * a.S) * D;
  const bf16* Vb = a.V + ((int64_t)(b * a.Hkv + kvh) * a.S) * D;
  const bf16* dOb = a.dO + (int64_t)b * a.S * (a.Hq * D) + (int64_t)h * D;
  bf16x8 qf[C::KS], of[C::KS];
#pragma unroll
  for (int t = 0; t < C::KS; ++t) {
    u32x4 qv = {0u, 0u, 0u, 0u}, ov = {0u, 0u, 0u, 0u};
    if (qme < a.S) {
      qv = *reinterpret_cast<const u32x4*>(Qb + (int64_t)qme * D + 16 * t + 8 * g);
      ov = *reinterpret_cast<const u32x4*>(dOb + (int64_t)qme * (a.Hq * D) + 16 * t + 8 * g);
    }
    qf[t] = __builtin_bit_cast(bf16x8, qv);
    of[t] = __builtin_bit_cast(bf16x8, ov);
  }
  const float lse = qme < a.S ? a.lse[(int64_t)(b * a.Hq + h) * a.S + qme] : 0.f;
  const float dsum = qme < a.S ? a.Dsum[(int64_t)(b * a.Hq + h) * a.S + qme] : 0.f;
  f32x16 dq[C::DB];
#pragma unroll
  for (int i = 0; i < C::DB; ++i) dq[i] = fa::zero16();
  const int q_last = min(q0 + 127, a.S - 1);
  const int nkt = q_last / fa::BK + 1;
  const int wave_last = q0 + 32 * w + 31;
  fa::TrOffsets<D> tro;
  tro.init(lane);
  // K and V tiles of 64 keys stream into swizzled row-major LDS tiles by
  // direct copies (rows past the sequence read the last row; their P is 0);
  // K^T fragments come from transpose reads of the same K tile
  auto issue = [&](int buf, int k0) {
    fa::dma_tile<D>(Kb, D, k0, a.S, sK[buf], w, lane);
    fa::dma_tile<D>(Vb, D, k0, a.S, sV[buf], w, lane);
  };
  issue(0, 0);
  wait_vmem();
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    const int k0 = kt * fa::BK, buf = kt & 1;
    // the next tile lands in the buffer every wave finished reading before
    // the previous barrier
    if (kt + 1 < nkt) issue(buf ^ 1, k0 + fa::BK);
    if (k0 <= wave_last) {
#pragma unroll
      for (int sb = 0; sb < 2; ++sb) {
        f32x16 s = fa::zero16(), dp = fa::zero16();
#pragma unroll
        for (int t = 0; t < C::KS; ++t) {
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              fa::tfrag_row<D>(sK[buf], sb * 32 + l32, 2 * t + g), qf[t], s, 0, 0, 0);
          dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              fa::tfrag_row<D>(sV[buf], sb * 32 + l32, 2 * t + g), of[t], dp, 0, 0, 0);
        }
        // causal / length mask only where the 32 x 32 block crosses the
        // wave's diagonal or the sequence end (uniform over the wave)
        const int kb0 = k0 + sb * 32;
        if (kb0 + 31 > q0 + 32 * w || kb0 + 32 > a.S || wave_last >= a.S) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = kb0 + fa::acc_row(r, g);
            float p = __builtin_amdgcn_exp2f(fmaf(s[r], a.c, -lse));
            if (key > qme || key >= a.S || qme >= a.S) p = 0.f;
            dp[r] = p * (dp[r] - dsum);
          }
        } else {
#pragma unroll
          for (int r = 0; r < 16; ++r)
            dp[r] = __builtin_amdgcn_exp2f(fmaf(s[r], a.c, -lse)) * (dp[r] - dsum);
        }
        // dQ^T[d][q] += K^T dS  (contraction over keys)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const bf16x8 df = fa::pack8(dp, hh);
#pragma unroll
          for (int i = 0; i < C::DB; ++i)
            dq[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                fa::tr_read<D>(sK[buf], tro, i, 2 * sb + hh), df, dq[i], 0, 0, 0);
        }
      }
    }
    wait_vmem();
    __syncthreads();
  }
  if (qme < a.S) {
    float* dQb = a.dQ + ((int64_t)(b * a.Hq + h) * a.S + qme) * D;
#pragma unroll
    for (int i = 0; i < C::DB; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) dQb[i * 32 + fa::acc_row(r, g)] = dq[i][r] * a.scale;
  }
}

// ------------------------------------------------------------------ launch

catq_status flash_forward(int D, FaArgs& a, hipStream_t stream) {
  dim3 grid((unsigned)(a.B * a.Hq), (unsigned)((a.S + 127) / 128)), block(fa::NT);
  const double f = 2.0 * 2.0 * (double)a.B * a.Hq * (double)a.S * a.S * D * 0.5;
  const double by = 2.0 * (double)a.B * a.S * D * (2.0 * a.Hq + 2.0 * a.Hkv) + 4.0 * a.B * a.Hq * a.S;
  if (D == 128)
    CATQ_TRACED(stream, "flash_fwd_kernel<128>", f, by, a.S, a.Hq, D,
                hipLaunchKernelGGL(flash_fwd_kernel<128>, grid, block, 0, stream, a));
  else
    CATQ_TRACED(stream, "flash_fwd_kernel<64>", f, by, a.S, a.Hq, D,
                hipLaunchKernelGGL(flash_fwd_kernel<64>, grid, block, 0, stream, a));
  CATQ_CHECK_LAUNCH("flash forward");
  return CATQ_OK;
}

catq_status flash_backward(int D, FaArgs& a, hipStream_t stream) {
  CATQ_REQUIRE(a.Hkv > 0 && a.Hq % a.Hkv == 0 && a.hsplit >= 1 && (a.Hq / a.Hkv) % a.hsplit == 0,
               CATQ_ERR_VALUE, "the q-head split must divide the group size");
  const int64_t rows = (int64_t)a.B * a.S * a.Hq;
  dim3 gs((unsigned)((rows * (D / 8) + 255) / 256));
  const double dby = (double)rows * (4.0 * D + 4.0);
  if (D == 128)
    CATQ_TRACED(stream, "flash_dsum_kernel<128>", 0.0, dby, rows, D, 0,
                hipLaunchKernelGGL(flash_dsum_kernel<128>, gs, dim3(256), 0, stream, a));
  else
    CATQ_TRACED(stream, "flash_dsum_kernel<64>", 0.0, dby, rows, D, 0,
                hipLaunchKernelGGL(flash_dsum_kernel<64>, gs, dim3(256), 0, stream, a));
  CATQ_CHECK_LAUNCH("flash dsum");
  const double half = 0.5 * 2.0 * (double)a.B * a.Hq * (double)a.S * a.S * D;
  dim3 gkv((unsigned)(a.B * a.Hkv * a.hsplit), (unsigned)((a.S + 127) / 128)), block(fa::NT);
  const dim3 block_kv(DKDV_NT);
  if (D == 128)
    CATQ_TRACED(stream, "flash_bwd_dkdv_kernel<128>", 4.0 * half, 0.0, a.S, a.Hkv, D,
                hipLaunchKernelGGL(flash_bwd_dkdv_kernel<128>, gkv, block_kv, 0, stream, a));
  else
    CATQ_TRACED(stream, "flash_bwd_dkdv_kernel<64>", 4.0 * half, 0.0, a.S, a.Hkv, D,
                hipLaunchKernelGGL(flash_bwd_dkdv_kernel<64>, gkv, block_kv, 0, stream, a));
  CATQ_CHECK_LAUNCH("flash dK dV");
  dim3 gq((unsigned)(a.B * a.Hq), (unsigned)((a.S + 127) / 128));
  if (D == 128)
    CATQ_TRACED(stream, "flash_bwd_dq_kernel<128>", 3.0 * half, 0.0, a.S, a.Hq, D,
                hipLaunchKernelGGL(flash_bwd_dq_kernel<128>, gq, block, 0, stream, a));
  else
    CATQ_TRACED(stream, "flash_bwd_dq_kernel<64>", 3.0 * half, 0.0, a.S, a.Hq, D,
                hipLaunchKernelGGL(flash_bwd_dq_kernel<64>, gq, block, 0, stream, a));
  CATQ_CHECK_LAUNCH("flash dQ");
  return CATQ_OK;
}

}  // namespace catq
