// Internal launchers shared between the HIP translation units of libcatq.
#pragma once

#include "catq_internal.h"

namespace catq {

// ---------------------------------------------------------------- tracing
int trace_begin(hipStream_t stream, const char* tag, double flops, double bytes, int64_t M,
                int64_t N, int64_t K);
void trace_end(int slot, hipStream_t stream);

#define CATQ_TRACED(stream, tag, flops, bytes, M, N, K, launch)                   \
  do {                                                                           \
    const int slot_ = ::catq::trace_begin((stream), (tag), (flops), (bytes), (M), (N), (K)); \
    launch;                                                                      \
    ::catq::trace_end(slot_, (stream));                                          \
  } while (0)

// ------------------------------------------------------------------ LM + ST

// Factor gradients from G = dL/dW_fake (fp32, [n_rows][d_in]) for one weight
// matrix (or all experts' matrices stacked along rows).  `ws_shared` holds
// 3*n_groups floats and is used only when some factor stride is 0.
// The gradients of stride-0 (one per matrix) factors from their per-group
// terms in ws[k][n_groups] (fixed-order sum); stride-1 factors untouched.
catq_status finish_shared_factors(const int64_t* strides, int64_t n_groups, const float* ws,
                                  float* const* out, hipStream_t stream);
catq_status launch_factor_grads(const float* G, int nsplit, int64_t split_stride, float* G_out,
                                const void* W, catq_dtype w_dtype, int64_t n_rows, int64_t d_in,
                                const float* stats, const float* d_mu, const float* d_alpha,
                                const float* d_delta, const catq_lmst_params* p, float* g_mu,
                                float* g_alpha, float* g_delta, float* ws_shared,
                                hipStream_t stream);

catq_status check_lmst_params(const catq_lmst_params* p, int64_t d_in);

// -------------------------------------------------------------------- GEMM
//
// C[m][n] = alpha * sum_k A(m,k) B(n,k) (+ R[m][n])
//   A(m,k) = A[m*lda + k]   (a_t = 0, K contiguous)  or  A[k*lda + m]  (a_t = 1)
//   B(n,k) = B[n*ldb + k]   (b_t = 0, K contiguous)  or  B[k*ldb + n]  (b_t = 1)
// Batches: blockIdx.z = z, zo = z / inner, zi = z % inner; operand X is offset
// by zo*x_so + (zi / x_div)*x_si elements.
// Causal modes (square attention-score problems, rows = queries):
//   1  skip output tiles lying wholly above the diagonal (n0 >= m0 + BM)
//   2  contraction limited to k < m0 + BM          (P.V, dS.K)
//   3  contraction starts at k = m0 (rounded down)  (P^T.dO, dS^T.Q)
// Expert grouping through a device array off[E+1] (int64):
//   group_mode 1: rows of A and C grouped (row range off[e]..off[e+1]), B
//                 offset by e*b_gs; blockIdx.z = expert
//   group_mode 2: contraction grouped (k range off[e]..off[e+1]) ; C offset by
//                 e*c_gs; blockIdx.z = expert
// Per-launch constants of the transition function f at sharpness s (Eq. 5),
// formed on the host in double.
struct StConst {
  float c2s;   // 2 s log2(e):  q_a = 2^(-|x - D| * c2s)
  float s4;    // 4 s:          t = 4 s x
  float s4l;   // 4 s log2(e)
  float k2;    // 1 / tanh(s)   (f = (tanh a + tanh b) * k2 / 2)
  float sk4;   // 2 s / tanh(s) (f_W, f_D prefactor)
};

// Factor-gradient epilogue (EPI 3) of an unsplit weight gradient G (per
// expert, or one dense matrix): instead of G, the gradients of the three
// learnable factors of every 128-weight group of W (the reductions of
// Sec. 2.3), as the separate factor-gradient kernel computes them from G.
struct FacEpi {
  const void* W;          // bf16 weights [E][rows][ldw] (E = 1 when dense)
  int64_t ldw;            // row pitch of W (d_in; a column range of G keeps it)
  const float* stats;     // [n_groups][2] mu0, alpha0
  const float* dmu;
  const float* dal;
  const float* dde;
  float* out[3];          // per-group gradients (factor stride 1)
  float* ws;              // [3][n_groups] per-group terms of stride-0 factors
  int64_t n_groups;
  int64_t s[3];           // factor strides (1, or 0 = one value per matrix)
  int32_t mode, ste;
  float delta0;
  StConst st;
};

struct GemmArgs {
  const void* A;
  const void* B;
  void* C;
  const void* R;
  int64_t M, N, K;
  int64_t lda, ldb, ldc, ldr;
  int64_t a_so, a_si, b_so, b_si, c_so, c_si;
  int32_t a_div, b_div, c_div, inner;
  int32_t batch;
  float alpha;
  int32_t causal;
  const int64_t* group_off;
  int32_t group_mode;
  int32_t n_groups;
  int64_t b_gs, c_gs;
  int64_t max_rows_per_group;  // group_mode 1: bound used to size the grid
  // fused epilogues of the direct-to-LDS kernel (gemm_run_epi):
  //  1 (SwiGLU forward): B rows are the gate rows [0, N/2) and up rows
  //    [N/2, N) of a fused gate|up weight taken in (gate_j, up_j) pairs, so
  //    output columns 2j, 2j+1 hold gate_j, up_j; C receives them as
  //    [gate | up] (ldc) and aux0 the SwiGLU a [M][N/2] (ld_aux)
  //  2 (SwiGLU backward): C is the gradient of a [M][N]; aux0 holds the
  //    forward's [gate | up] [M][2N] and aux1 receives d[gate | up] (ld_aux);
  //    C itself is not written
  //  3 (factor gradients, group_mode 2, both operands K-major): see FacEpi;
  //    C is not written
  int32_t epi;
  void* aux0;
  void* aux1;
  int64_t ld_aux;
  FacEpi fac;
};

GemmArgs gemm_args_default();
// dtype of A, B (both bf16, or both f32); c_dtype of C; r_dtype of the residual R
// (a bf16 C takes a bf16 R; an fp32 C takes either).
catq_status gemm_run(const GemmArgs& a, int a_t, int b_t, catq_dtype in_dtype, catq_dtype c_dtype,
                     hipStream_t stream, catq_dtype r_dtype = CATQ_BF16);
// Split-K over the contraction (dense, unbatched): split i writes its partial
// product to C + i*c_split_stride.  Returns the number of splits actually used
// through gemm_split_count (chunks are multiples of 64).
catq_status gemm_run_split(const GemmArgs& a, int a_t, int b_t, catq_dtype in_dtype,
                           catq_dtype c_dtype, int ksplit, int64_t c_split_stride,
                           hipStream_t stream, catq_dtype r_dtype = CATQ_BF16);
int gemm_split_count(const GemmArgs& a, int ksplit);
// A dense bf16 GEMM with one of the fused epilogues above (a.epi).  Returns
// CATQ_ERR_VALUE without launching when the shape or layout does not fit
// the direct-to-LDS kernel's vector epilogue (the caller then runs the
// unfused pair of kernels).
catq_status gemm_run_epi(const GemmArgs& a, int a_t, int b_t, hipStream_t stream);
// Weight gradients reduced to factor gradients in the epilogue (a.epi = 3,
// a.fac filled; per expert with group_mode 2, or one dense problem with
// group_mode 0, never split); CATQ_ERR_VALUE when the shape is not eligible
// (then nothing was launched).
catq_status gemm_run_factor(const GemmArgs& a, hipStream_t stream);

// ---------------------------------------------------------- fused attention
struct FaArgs {
  const bf16* Q;      // [B][Hq][S][D]
  const bf16* K;      // [B][Hkv][S][D]
  const bf16* V;      // [B][Hkv][S][D]
  bf16* O;            // token-major [B*S][Hq*D]
  float* lse;         // [B][Hq][S], base 2
  const bf16* dO;     // token-major [B*S][Hq*D]
  float* Dsum;        // [B][Hq][S]
  float* dQ;          // [B][Hq][S][D]
  float* dK;          // [hsplit][B][Hkv][S][D]: partial sums over hsplit chunks of q heads
  float* dV;          // [hsplit][B][Hkv][S][D]
  int B, S, Hq, Hkv;
  int hsplit;         // blocks a kv head's q heads are split over (divides Hq/Hkv)
  float c;            // softmax scale * log2(e)
  float scale;        // softmax scale
};
catq_status flash_forward(int D, FaArgs& a, hipStream_t stream);
catq_status flash_backward(int D, FaArgs& a, hipStream_t stream);

}  // namespace catq
