// C ABI of the fake-ternary linear layer: forward, and backward to the input
// and to the learnable factors (Sec. 2.2-2.4).
#include "kernels.h"
#include "lmst_math.h"

namespace catq {

// Split of the token contraction of G = dY^T X.  A 256x256 tile holds a
// whole compute unit (128 KB of LDS), so the (N/256)x(K/256) tiles times the
// splits run in ceil(tiles * ks / 256) rounds, each as long as its share of
// the tokens (64 per iteration) plus the fixed cost of writing a 256x256
// fp32 partial (about 10 iterations, measured).  The factor-gradient pass
// then reads every partial once: N*K*4 bytes per split, about N*K/1.77e6
// iterations at the read rate it reaches.  The split with the least
// estimated total wins; each split keeps >= 1024 tokens.  (This picks the
// measured best of GEMM plus partial reads for every projection shape of
// the benchmarked block.)
static int choose_ksplit(int64_t M, int64_t N, int64_t K, int32_t n_experts) {
  if (n_experts > 1) return 1;
  constexpr int64_t kUnits = 256;      // compute units of the MI355X
  constexpr double kEpilogue = 10.0;   // partial write, in 64-token iterations
  constexpr double kRead = 1.77e6;     // weights whose partial one iteration reads back
  const int64_t tiles = ((N + 255) / 256) * ((K + 255) / 256);
  int best = 1;
  double best_cost = 0.0;
  for (int ks = 1; ks <= 64 && (ks == 1 || M / ks >= 1024); ks *= 2) {
    const int64_t rounds = (tiles * ks + kUnits - 1) / kUnits;
    const double cost = (double)rounds * ((double)M / (64.0 * ks) + kEpilogue) +
                        (double)ks * (double)N * (double)K / kRead;
    if (ks == 1 || cost < best_cost) {
      best = ks;
      best_cost = cost;
    }
  }
  return best;
}

static int splits_used(int64_t M, int64_t N, int64_t K, int32_t n_experts) {
  GemmArgs a = gemm_args_default();
  a.M = N;
  a.N = K;
  a.K = M;
  return gemm_split_count(a, choose_ksplit(M, N, K, n_experts));
}

static catq_status check_linear_common(const void* X, const void* W_fake, catq_dtype dtype,
                                       int64_t M, int64_t N, int64_t K, int32_t n_experts,
                                       const int64_t* row_offsets) {
  CATQ_REQUIRE(X && W_fake, CATQ_ERR_NULL, "X and W_fake must not be NULL");
  CATQ_REQUIRE(M > 0 && N > 0 && K > 0, CATQ_ERR_SHAPE, "M, N, K must be > 0");
  CATQ_REQUIRE(n_experts < 1 || (count_ok(M, K) && count_ok(M, N) && count_ok(n_experts, N, K)),
               CATQ_ERR_SHAPE, "M*K, M*N and n_experts*N*K must each be at most 2^38");
  CATQ_REQUIRE(dtype_ok(dtype), CATQ_ERR_DTYPE, "bad dtype");
  CATQ_REQUIRE(K % 8 == 0, CATQ_ERR_SHAPE, "K must be a multiple of 8");
  CATQ_REQUIRE(n_experts >= 1, CATQ_ERR_SHAPE, "n_experts must be >= 1");
  CATQ_REQUIRE(n_experts == 1 || row_offsets != nullptr, CATQ_ERR_NULL,
               "row_offsets required for n_experts > 1");
  CATQ_REQUIRE(n_experts == 1 || dtype == CATQ_BF16, CATQ_ERR_DTYPE,
               "routed experts run in bf16 only");
  return CATQ_OK;
}

}  // namespace catq

using namespace catq;

extern "C" size_t catq_workspace_size(int32_t which_call, int64_t M, int64_t N, int64_t K,
                                      int32_t n_experts) {
  // sizes the calls would reject need no workspace
  if (M <= 0 || N <= 0 || K <= 0 || n_experts < 1 || !count_ok(M, K) || !count_ok(M, N) ||
      !count_ok(n_experts, N, K))
    return 0;
  if (which_call == CATQ_WS_LINEAR_BWD) {
    const int64_t E = n_experts;
    const int ns = splits_used(M, N, K, n_experts);
    size_t g = round_up((size_t)(E * N * K) * 4 * (size_t)ns, 256);
    size_t shared = round_up((size_t)3 * (size_t)(E * N * K / 16) * 4, 256);
    return g + shared;
  }
  if (which_call == CATQ_WS_LOSS) return 4096 * sizeof(double);
  return 0;
}

extern "C" catq_status catq_fakeq_linear_fwd(const void* X, const void* W_fake, catq_dtype dtype,
                                             void* Y, catq_dtype y_dtype, int64_t M, int64_t N,
                                             int64_t K, int32_t n_experts,
                                             const int64_t* row_offsets, const void* residual,
                                             catq_dtype r_dtype, hipStream_t stream) {
  clear_error();
  CATQ_TRY(check_linear_common(X, W_fake, dtype, M, N, K, n_experts, row_offsets));
  CATQ_REQUIRE(Y != nullptr, CATQ_ERR_NULL, "Y must not be NULL");
  CATQ_REQUIRE(dtype_ok(y_dtype) && dtype_ok(r_dtype), CATQ_ERR_DTYPE, "bad y or residual dtype");
  CATQ_REQUIRE(dtype == CATQ_BF16 || (y_dtype == CATQ_F32 && r_dtype == CATQ_F32), CATQ_ERR_DTYPE,
               "fp32 inputs give an fp32 output and take an fp32 residual");
  CATQ_REQUIRE(y_dtype == CATQ_F32 || residual == nullptr || r_dtype == CATQ_BF16,
               CATQ_ERR_DTYPE, "a bf16 output takes a bf16 residual");
  CATQ_REQUIRE(residual == nullptr || n_experts == 1, CATQ_ERR_VALUE,
               "residual is supported for dense layers only");
  CATQ_REQUIRE(aligned16(X) && aligned16(W_fake) && aligned16(Y) && aligned16(residual),
               CATQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  GemmArgs a = gemm_args_default();
  a.A = X;
  a.B = W_fake;
  a.C = Y;
  a.R = residual;
  a.M = M;
  a.N = N;
  a.K = K;
  a.lda = K;
  a.ldb = K;
  a.ldc = N;
  a.ldr = N;
  if (n_experts > 1) {
    a.group_mode = 1;
    a.group_off = row_offsets;
    a.n_groups = n_experts;
    a.b_gs = N * K;
    a.max_rows_per_group = (M + n_experts - 1) / n_experts;
  }
  return gemm_run(a, 0, 0, dtype, y_dtype, stream, r_dtype);
}

extern "C" catq_status catq_fakeq_gateup_swiglu_fwd(const void* X, const void* W_fake, int64_t M,
                                                    int64_t F, int64_t K, void* gu, void* a,
                                                    hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(X && W_fake && gu && a, CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(count_ok(M, K) && count_ok(M, 2 * F) && count_ok(2 * F, K) && F % 8 == 0,
               CATQ_ERR_SHAPE,
               "M, K must be > 0 and F a positive multiple of 8");
  CATQ_REQUIRE(aligned16(X) && aligned16(W_fake) && aligned16(gu) && aligned16(a),
               CATQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  GemmArgs g = gemm_args_default();
  g.A = X;
  g.B = W_fake;
  g.C = gu;
  g.M = M;
  g.N = 2 * F;
  g.K = K;
  g.lda = K;
  g.ldb = K;
  g.ldc = 2 * F;
  g.epi = 1;
  g.aux0 = a;
  g.ld_aux = F;
  const catq_status st = gemm_run_epi(g, 0, 0, stream);
  if (st != CATQ_ERR_VALUE) return st;
  // not eligible for the fused epilogue: the GEMM, then the SwiGLU kernel
  clear_error();
  g.epi = 0;
  g.aux0 = nullptr;
  CATQ_TRY(gemm_run(g, 0, 0, CATQ_BF16, CATQ_BF16, stream));
  return catq_aux_swiglu_fwd(gu, M, F, a, stream);
}

extern "C" catq_status catq_fakeq_down_swiglu_bwd(const void* dY, const void* W_fake, int64_t M,
                                                  int64_t N, int64_t F, const void* gu, void* dgu,
                                                  void* da, hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(dY && W_fake && gu && dgu, CATQ_ERR_NULL, "NULL argument");
  CATQ_REQUIRE(count_ok(M, N) && count_ok(M, 2 * F) && count_ok(N, F) && F % 8 == 0,
               CATQ_ERR_SHAPE,
               "M, N must be > 0 and F a positive multiple of 8");
  CATQ_REQUIRE(aligned16(dY) && aligned16(W_fake) && aligned16(gu) && aligned16(dgu) &&
                   aligned16(da),
               CATQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  // d a = dY . W_fake (contraction over the N outputs; W_fake K-major)
  GemmArgs g = gemm_args_default();
  g.A = dY;
  g.B = W_fake;
  g.C = dgu;   // not written by the fused epilogue
  g.M = M;
  g.N = F;
  g.K = N;
  g.lda = N;
  g.ldb = F;
  g.ldc = F;
  g.epi = 2;
  g.aux0 = const_cast<void*>(gu);
  g.aux1 = dgu;
  g.ld_aux = 2 * F;
  const catq_status st = gemm_run_epi(g, 0, 1, stream);
  if (st != CATQ_ERR_VALUE) return st;
  // not eligible: d a into the caller's scratch, then the SwiGLU backward
  clear_error();
  CATQ_REQUIRE(da != nullptr, CATQ_ERR_NULL,
               "this shape needs the d a scratch buffer (bf16 [M][F])");
  g.epi = 0;
  g.C = da;
  g.aux0 = g.aux1 = nullptr;
  CATQ_TRY(gemm_run(g, 0, 1, CATQ_BF16, CATQ_BF16, stream));
  return catq_aux_swiglu_bwd(gu, da, M, F, dgu, stream);
}

extern "C" catq_status catq_fakeq_linear_bwd(
    const void* dY, const void* X, const void* W_fake, catq_dtype dtype, int64_t M, int64_t N,
    int64_t K, int32_t n_experts, const int64_t* row_offsets, const void* W, catq_dtype w_dtype,
    const float* stats, const float* d_mu, const float* d_alpha, const float* d_delta,
    const catq_lmst_params* p, void* dX, float* g_d_mu, float* g_d_alpha, float* g_d_delta,
    float* dW_fake, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  clear_error();
  CATQ_TRY(check_linear_common(X, W_fake, dtype, M, N, K, n_experts, row_offsets));
  // with no factor gradient and no dW_fake requested only dX is computed
  const bool want_g = g_d_mu || g_d_alpha || g_d_delta || dW_fake;
  CATQ_REQUIRE(dY && (want_g || dX), CATQ_ERR_NULL, "dY, and dX or the factor gradients, are required");
  CATQ_REQUIRE(N % 8 == 0, CATQ_ERR_SHAPE, "N must be a multiple of 8");
  if (!want_g) {
    CATQ_REQUIRE(aligned16(dY) && aligned16(X) && aligned16(W_fake) && aligned16(dX), CATQ_ERR_ALIGN,
                 "pointers must be 16-byte aligned");
  } else {
    CATQ_REQUIRE(W && stats && d_mu && d_alpha && d_delta && g_d_mu && g_d_alpha && g_d_delta,
                 CATQ_ERR_NULL, "W, stats, factors and all three factor-gradient outputs are required");
    CATQ_REQUIRE(dtype_ok(w_dtype), CATQ_ERR_DTYPE, "bad w_dtype");
    CATQ_TRY(check_lmst_params(p, K));
    CATQ_REQUIRE(aligned16(dY) && aligned16(X) && aligned16(W_fake) && aligned16(W) &&
                     aligned16(dX) && aligned16(dW_fake) && aligned16(workspace) && aligned16(stats),
                 CATQ_ERR_ALIGN, "pointers must be 16-byte aligned");
    const size_t need = catq_workspace_size(CATQ_WS_LINEAR_BWD, M, N, K, n_experts);
    CATQ_REQUIRE(workspace != nullptr && workspace_bytes >= need, CATQ_ERR_WORKSPACE,
                 "workspace of %zu bytes needed (got %zu)", need, workspace_bytes);
  }
  const int64_t E = n_experts;
  const int ns = splits_used(M, N, K, n_experts);
  const size_t g_bytes = round_up((size_t)(E * N * K) * 4 * (size_t)ns, 256);
  float* Gbuf = (dW_fake && ns == 1) ? dW_fake : reinterpret_cast<float*>(workspace);
  float* shared_ws = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) + g_bytes);


  // dX = dY . W_fake  (W_fake contracted over its rows: a K-major operand)
  if (dX) {
    GemmArgs a = gemm_args_default();
    a.A = dY;
    a.B = W_fake;
    a.C = dX;
    a.M = M;
    a.N = K;
    a.K = N;
    a.lda = N;
    a.ldb = K;
    a.ldc = K;
    if (n_experts > 1) {
      a.group_mode = 1;
      a.group_off = row_offsets;
      a.n_groups = n_experts;
      a.b_gs = N * K;
      a.max_rows_per_group = (M + n_experts - 1) / n_experts;
    }
    CATQ_TRY(gemm_run(a, 0, 1, dtype, dtype, stream));
  }
  if (!want_g) return CATQ_OK;
  // G = dY^T . X  (contraction over the tokens: both operands K-major), fp32.
  // Where every G element is final in one tile (experts, or a dense
  // gradient left unsplit), 128-weight groups, bf16 and no dW_fake asked
  // for, the factor gradients come out of the GEMM's epilogue and G never
  // reaches memory; CATQ_ERR_VALUE from the launch means the shape does not
  // fit that kernel, and the two-pass path below runs instead.
  auto factor_epilogue = [&](const GemmArgs& a) -> catq_status {
    if (!(dW_fake == nullptr && p->group_size == 128 && dtype == CATQ_BF16 &&
          w_dtype == CATQ_BF16))
      return CATQ_ERR_VALUE;
    GemmArgs f = a;
    f.epi = 3;
    f.c_gs = 0;  // C is only an aligned dummy
    FacEpi& fe = f.fac;
    fe.W = W;
    fe.ldw = K;
    fe.stats = stats;
    fe.dmu = d_mu;
    fe.dal = d_alpha;
    fe.dde = d_delta;
    fe.out[0] = g_d_mu;
    fe.out[1] = g_d_alpha;
    fe.out[2] = g_d_delta;
    fe.ws = shared_ws;
    fe.n_groups = E * N * K / 128;
    for (int i = 0; i < 3; ++i) fe.s[i] = p->factor_stride[i];
    fe.mode = p->mode;
    fe.ste = (p->mode == CATQ_HARD && p->s_bwd == 0.0f) ? 1 : 0;
    fe.delta0 = p->delta0;
    const double s_use = (p->mode == CATQ_HARD) ? (double)p->s_bwd : (double)p->s;
    fe.st = make_st(s_use > 0 ? s_use : 1.0);
    const catq_status st = gemm_run_factor(f, stream);
    if (st == CATQ_OK) return finish_shared_factors(fe.s, fe.n_groups, shared_ws, fe.out, stream);
    if (st == CATQ_ERR_VALUE) clear_error();
    return st;
  };
  {
    GemmArgs a = gemm_args_default();
    a.C = Gbuf;
    a.M = N;
    a.N = K;
    a.K = M;
    a.ldc = K;
    a.A = dY;
    a.B = X;
    a.lda = N;
    a.ldb = K;
    if (n_experts > 1) {
      a.group_mode = 2;
      a.group_off = row_offsets;
      a.n_groups = n_experts;
    }
    if (ns == 1) {
      const catq_status st = factor_epilogue(a);
      if (st != CATQ_ERR_VALUE) return st;
    }
    if (n_experts > 1) {
      a.c_gs = N * K;
      CATQ_TRY(gemm_run(a, 1, 1, dtype, CATQ_F32, stream));
    } else {
      CATQ_TRY(gemm_run_split(a, 1, 1, dtype, CATQ_F32, choose_ksplit(M, N, K, 1), N * K,
                              stream));
    }
  }
  // the factor kernel folds the split partials itself (and writes the summed
  // G when dW_fake is requested)
  float* G_out = (dW_fake && ns > 1) ? dW_fake : nullptr;
  return launch_factor_grads(Gbuf, ns, N * K, G_out, W, w_dtype, E * N, K, stats, d_mu, d_alpha,
                             d_delta, p, g_d_mu, g_d_alpha, g_d_delta, shared_ws, stream);
}
