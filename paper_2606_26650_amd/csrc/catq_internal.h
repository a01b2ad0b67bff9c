// Internal helpers shared by the HIP sources of libcatq (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "catq.h"

namespace catq {

// ---- error reporting (thread-local message, see catq_last_error_message) ----
void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

#define CATQ_REQUIRE(cond, code, ...)      \
  do {                                     \
    if (!(cond)) {                         \
      ::catq::set_error(__VA_ARGS__);      \
      return (code);                       \
    }                                      \
  } while (0)

#define CATQ_CHECK_LAUNCH(what)                                                            \
  do {                                                                                     \
    hipError_t e_ = hipGetLastError();                                                     \
    if (e_ != hipSuccess) {                                                                \
      ::catq::set_error("%s: launch failed: %s", (what), hipGetErrorString(e_));           \
      return CATQ_ERR_HIP;                                                                 \
    }                                                                                      \
  } while (0)

#define CATQ_TRY(expr)                 \
  do {                                 \
    catq_status st_ = (expr);          \
    if (st_ != CATQ_OK) return st_;    \
  } while (0)

__host__ __device__ inline bool aligned16(const void* p) {
  return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}
inline bool dtype_ok(int d) { return d == CATQ_F32 || d == CATQ_BF16; }
inline size_t dtype_size(int d) { return d == CATQ_F32 ? 4 : 2; }
inline size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Element counts the library accepts: products of positive sizes that stay at
// or below 2^38 (more elements than any MI355X buffer holds), so the byte
// sizes, offsets and grid sizes derived from them cannot overflow.
constexpr int64_t MAX_ELEMS = int64_t(1) << 38;
inline bool count_ok(int64_t a, int64_t b = 1, int64_t c = 1, int64_t d = 1) {
  if (a <= 0 || b <= 0 || c <= 0 || d <= 0) return false;
  int64_t p;
  if (__builtin_mul_overflow(a, b, &p) || __builtin_mul_overflow(p, c, &p) ||
      __builtin_mul_overflow(p, d, &p))
    return false;
  return p <= MAX_ELEMS;
}

// ---- device-side types ----
typedef __bf16 bf16;
typedef unsigned short u16;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

__device__ __forceinline__ float bf16_lo(unsigned int w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(unsigned int w) { return __uint_as_float(w & 0xffff0000u); }

// Round-to-nearest-even float -> bf16 (hardware conversion on gfx950).
__device__ __forceinline__ unsigned short f2bf_bits(float f) {
  bf16 h = (bf16)f;
  return __builtin_bit_cast(unsigned short, h);
}
// Two floats -> two bf16 in one dword (lo in the low half), one packed
// conversion (the same rounding as f2bf_bits on each).
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
__device__ __forceinline__ unsigned int pack_bf16x2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(unsigned int, __builtin_convertvector(v, bf16x2));
}

// Load 8 consecutive elements (bf16 or fp32) as floats.
template <typename T>
__device__ __forceinline__ void load8(const T* p, float (&v)[8]);
template <>
__device__ __forceinline__ void load8<bf16>(const bf16* p, float (&v)[8]) {
  u32x4 u = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = bf16_lo(u[i]);
    v[2 * i + 1] = bf16_hi(u[i]);
  }
}
template <>
__device__ __forceinline__ void load8<float>(const float* p, float (&v)[8]) {
  f32x4 a = *reinterpret_cast<const f32x4*>(p);
  f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[i] = a[i];
    v[4 + i] = b[i];
  }
}

// SwiGLU of one (gate, up) pair and its backward; shared by the SwiGLU
// kernels and the GEMM epilogues that fuse them (identical results).
__device__ __forceinline__ float sigmoid_f(float g) { return 1.0f / (1.0f + __expf(-g)); }
__device__ __forceinline__ float swiglu1(float g, float u) { return g * sigmoid_f(g) * u; }
__device__ __forceinline__ void swiglu1_bwd(float g, float u, float d, float& dg, float& du) {
  const float sg = sigmoid_f(g);
  const float silu = g * sg;
  du = d * silu;
  dg = d * u * sg * (1.0f + g * (1.0f - sg));
}
__device__ __forceinline__ float bf16_round_f(float x) { return (float)(bf16)x; }

template <typename T>
__device__ __forceinline__ void store8(T* p, const float (&v)[8]);
template <>
__device__ __forceinline__ void store8<bf16>(bf16* p, const float (&v)[8]) {
  u32x4 u;
#pragma unroll
  for (int i = 0; i < 4; ++i) u[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
  *reinterpret_cast<u32x4*>(p) = u;
}
template <>
__device__ __forceinline__ void store8<float>(float* p, const float (&v)[8]) {
  f32x4 a, b;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    a[i] = v[i];
    b[i] = v[4 + i];
  }
  *reinterpret_cast<f32x4*>(p) = a;
  *reinterpret_cast<f32x4*>(p + 4) = b;
}

__device__ __forceinline__ float to_f(bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f(float x) { return x; }

// Wave-wide (64 lanes) reductions.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  return v;
}

// ------------------------------------------------ direct-to-LDS copies

// 16-byte global -> LDS copy, lane l landing at lds_base + 16*l.  Issued as
// inline assembly so that the compiler does not add conservative waits before
// every LDS read; the kernel waits (vmcnt) itself before the barrier that
// publishes the tile.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void* g, const void* lds_base) {
#if defined(__HIP_DEVICE_COMPILE__)
  const unsigned l = __builtin_amdgcn_readfirstlane(
      (unsigned)(uintptr_t)(__attribute__((address_space(3))) const void*)lds_base);
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(l), "v"(g)
               : "memory", "m0");
#endif
}

typedef int i32x4_rsrc __attribute__((ext_vector_type(4)));

// Buffer resource (uniform, SGPRs) for raw loads of `bytes` bytes from p:
// offsets at or past the end read as zero without touching memory.
__device__ __forceinline__ i32x4_rsrc buf_rsrc(const void* p, uint32_t bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)p;
  i32x4_rsrc r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xffffu));
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = 0x00020000;
  return r;
}

// 16-byte buffer -> LDS copy (lane l landing at lds_base + 16*l) from byte
// offset voff (per lane) + soff (uniform) of the resource.  One VGPR per
// lane instead of a 64-bit address; waits as for dma16.
__device__ __forceinline__ void dma16_buf(i32x4_rsrc rsrc, uint32_t voff, uint32_t soff,
                                          const void* lds_base) {
#if defined(__HIP_DEVICE_COMPILE__)
  const unsigned l = __builtin_amdgcn_readfirstlane(
      (unsigned)(uintptr_t)(__attribute__((address_space(3))) const void*)lds_base);
  const unsigned so = __builtin_amdgcn_readfirstlane(soff);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds" ::"s"(l), "v"(voff),
               "s"(rsrc), "s"(so)
               : "memory", "m0");
#endif
}
// The same with the LDS destination as a 32-bit LDS address (uniform), for
// kernels that form it once from their __shared__ array.
__device__ __forceinline__ void dma16_lds(i32x4_rsrc rsrc, uint32_t voff, uint32_t soff,
                                          uint32_t lds_addr) {
#if defined(__HIP_DEVICE_COMPILE__)
  const unsigned l = __builtin_amdgcn_readfirstlane(lds_addr);
  const unsigned so = __builtin_amdgcn_readfirstlane(soff);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds" ::"s"(l), "v"(voff),
               "s"(rsrc), "s"(so)
               : "memory", "m0");
#endif
}
// 4-byte buffer -> LDS copy (lane l landing at lds_base + 4*l) from byte
// offset voff of the resource; offsets past its size land as zero.
__device__ __forceinline__ void dma4_buf(i32x4_rsrc rsrc, uint32_t voff, const void* lds_base) {
#if defined(__HIP_DEVICE_COMPILE__)
  const unsigned l = __builtin_amdgcn_readfirstlane(
      (unsigned)(uintptr_t)(__attribute__((address_space(3))) const void*)lds_base);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds" ::"s"(l), "v"(voff),
               "s"(rsrc)
               : "memory", "m0");
#endif
}
#pragma clang diagnostic pop

// wait until at most N vector memory operations of this wave are in flight
// (loads complete in issue order: the N newest may still be outstanding)
template <int N>
__device__ __forceinline__ void wait_vmem_n() {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
#endif
}

__device__ __forceinline__ void wait_vmem() {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#endif
}

typedef short lds_v4s __attribute__((ext_vector_type(4)));

// ds_read_b64_tr_b16 from an LDS address given as a generic pointer into a
// __shared__ array.  Within a block of 16 lanes, output lane i receives
// element e from lanes 4e..4e+3, column i mod 4 of their 8-byte rows.
__device__ __forceinline__ lds_v4s lds_read_tr16(const void* p) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) lds_v4s*)(const_cast<void*>(p)));
#else
  return lds_v4s{0, 0, 0, 0};
#endif
}

}  // namespace catq
