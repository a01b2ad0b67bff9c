/*
 * catq.h -- C ABI of the CAT-Q calibration hot path on AMD Instinct MI355X (gfx950).
 *
 * One block-wise reconstruction step of CAT-Q (ternary post-training
 * quantisation of LLM weights):
 *   - learnable modulation (LM) of each weight group and of the ternary
 *     threshold (Sec. 2.2, Eq. 3-4),
 *   - softened ternarisation (ST) through the transition function f
 *     (Sec. 2.3, Eq. 5-6),
 *   - the fake-ternary linear layers of a decoder block,
 *   - the output-reconstruction loss against the full-precision block
 *     (Sec. 2.4, Eq. 7),
 *   - the backward pass to the activations and to the three learnable
 *     factors,
 *   - the final hard ternarisation (Eq. 2) and 2-bit packing of the
 *     ternary weights with their group scale (App. B.2).
 *
 * Conventions shared by every entry point
 *   Ownership   every pointer is a device pointer owned by the caller, unless
 *               the argument says "host".  The library keeps no pointer
 *               after a call returns and allocates no device memory.
 *   Streams     every call enqueues its work on `stream` (a hipStream_t; NULL
 *               is the null stream) and returns without synchronising.
 *   Errors      arguments are checked before anything is launched; on a bad
 *               argument nothing is launched, the call returns a non-zero
 *               catq_status and catq_last_error_message() (thread-local)
 *               explains it.  A failed launch returns CATQ_ERR_HIP.  Faults
 *               inside kernels surface at the caller's next synchronisation.
 *               NaN or Inf inside the data is not an error; it propagates.
 *   Determinism every result is bitwise reproducible run to run (no float
 *               atomics; fixed reduction orders).
 *   Layout      matrices are row-major.  A weight is [d_out][d_in] like a
 *               torch nn.Linear weight; activations are [rows][features].
 *               Every pointer must be 16-byte aligned.
 *   Groups      weights are quantised in groups of g consecutive elements of
 *               the row-major flattening (App. B.2, g = 128 by default);
 *               d_in must be a multiple of g, so a group is a g-wide slice of
 *               one row.  g is 8 times a power of two, 16 <= g <= 512.
 *   dtypes      CATQ_BF16 (bfloat16) or CATQ_F32 where allowed.
 */
#ifndef CATQ_H
#define CATQ_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CATQ_OK = 0,
  CATQ_ERR_NULL = 1,       /* a required pointer is NULL                       */
  CATQ_ERR_SHAPE = 2,      /* a size is <= 0, or sizes do not fit together     */
  CATQ_ERR_DTYPE = 3,      /* dtype not supported for this argument            */
  CATQ_ERR_VALUE = 4,      /* a scalar parameter is out of range               */
  CATQ_ERR_ALIGN = 5,      /* a pointer is not 16-byte aligned                 */
  CATQ_ERR_WORKSPACE = 6,  /* workspace missing or smaller than required       */
  CATQ_ERR_HIP = 7,        /* a HIP launch or runtime call failed              */
  /* never returned: they make every int32 value a valid catq_status, so a
     caller's out-of-range value is checked, not undefined (C++) */
  CATQ_STATUS_RANGE_MIN_ = INT32_MIN,
  CATQ_STATUS_RANGE_MAX_ = INT32_MAX
} catq_status;

typedef enum {
  CATQ_F32 = 0,
  CATQ_BF16 = 1,
  /* not dtypes: every int32 value is a valid catq_dtype, and the calls reject
     all but the two above with CATQ_ERR_DTYPE */
  CATQ_DTYPE_RANGE_MIN_ = INT32_MIN,
  CATQ_DTYPE_RANGE_MAX_ = INT32_MAX
} catq_dtype;

/* Branch of the softened-ternarisation schedule, Eq. 6. */
typedef enum {
  CATQ_IDENTITY = 0,  /* t = 0:            W_fake = W                          */
  CATQ_SOFT = 1,      /* 0 < t <= gamma:   W_fake = alpha * f(W_hat; s, Delta) */
  CATQ_HARD = 2       /* gamma < t <= 1:   W_fake = alpha * Q(W_hat; Delta)    */
} catq_mode;

/* Parameters of one LM+ST evaluation (Eq. 3-6).  Passed by host pointer. */
typedef struct {
  int32_t group_size;        /* g, see "Groups" above                                  */
  int32_t mode;              /* catq_mode                                              */
  float delta0;              /* Delta0 of Eq. 4 (paper default 0.5); > 0, finite       */
  float s;                   /* sharpness of f in SOFT mode, s = (t/gamma)*s0; > 0     */
  float s_bwd;               /* HARD mode backward: derivatives of f at s_bwd stand in
                                for the hard step (s_bwd = 0: straight-through,
                                f_W = 1, f_Delta = 0); >= 0                            */
  int64_t factor_stride[3];  /* d_mu, d_alpha, d_Delta: 1 = one value per group,
                                0 = one value shared by every group                    */
} catq_lmst_params;

/*
 * catq_modulate_ternarize -- LM (Eq. 3-4) and ST (Eq. 5-6) of one weight
 * matrix, and the hard ternary codes and group scales of Eq. 2 (App. B.2).
 *
 * Per group j (stats [j] = {mu0, alpha0}):
 *   mu0 = mean(W), alpha0 = mean|W - mu0|        (float64 sums in a fixed
 *        order, rounded to fp32; only when stats_mode == 0)
 *   mu = mu0 + d_mu*alpha0, alpha = d_alpha*alpha0, Delta = d_Delta*Delta0
 *        (each rounded once to fp32)
 * Per element: W_hat = (W - mu)/alpha and
 *   IDENTITY  W_fake = W
 *   SOFT      W_fake = alpha * f(W_hat; s, Delta),
 *             f(x; s, D) = [tanh(s(x-D)) + tanh(s(x+D))] / (2 tanh s)   (Eq. 5)
 *   HARD      code = +1 if W - mu > Delta*alpha, -1 if W - mu < -Delta*alpha,
 *             else 0 (decided exactly in float64; a tie gives 0),
 *             W_fake = alpha * code
 * alpha is replaced by max(alpha, FLT_MIN) as a divisor (constant groups).
 *
 *   W          [d_out][d_in], w_dtype bf16 or f32
 *   d_mu, d_alpha, d_delta   fp32 factors, n_groups = d_out*d_in/g values
 *              each (or 1 when that factor's stride is 0)
 *   p          host pointer to the parameters
 *   stats      fp32 [n_groups][2]; stats_mode 0 computes and writes them,
 *              1 reads them (as written by an earlier call on the same W)
 *   W_fake     [d_out][d_in] in wf_dtype (bf16 or f32); may be NULL only in
 *              HARD mode when `codes` is given
 *   codes      int8 [d_out][d_in] in {-1,0,1}; HARD mode only; may be NULL
 *   alpha_out  fp32 [n_groups] group scales alpha; may be NULL
 * Errors: NULL W/factors/stats/p, W_fake NULL when required, codes outside
 * HARD, d_in % g, g out of range, s <= 0 or non-finite in SOFT, delta0 <= 0,
 * s_bwd < 0, bad mode or dtypes, misaligned pointers.
 */
catq_status catq_modulate_ternarize(const void* W, catq_dtype w_dtype, int64_t d_out, int64_t d_in,
                                    const float* d_mu, const float* d_alpha, const float* d_delta,
                                    const catq_lmst_params* p, float* stats, int32_t stats_mode,
                                    void* W_fake, catq_dtype wf_dtype, int8_t* codes,
                                    float* alpha_out, hipStream_t stream);

/*
 * catq_fakeq_linear_fwd -- the fake-ternary linear layer of the window
 * forward (Sec. 2.4, Eq. 7): Y[M][N] = X[M][K] . W_fake[N][K]^T (+ residual),
 * fp32 accumulation, output rounded to y_dtype.
 *
 *   dtype        dtype of X and W_fake: CATQ_BF16 (matrix-core path) or
 *                CATQ_F32 (then Y and the residual are fp32 too)
 *   y_dtype      dtype of Y (bf16 or f32)
 *   n_experts    1 for a dense layer (row_offsets NULL).  For routed experts
 *                (E = n_experts > 1) W_fake is [E][N][K] and the rows of X and
 *                Y are grouped by expert: rows [row_offsets[e], row_offsets[e+1])
 *                belong to expert e.  row_offsets is a device int64 [E+1] array
 *                with row_offsets[0] = 0, non-decreasing, row_offsets[E] = M.
 *   residual     optional [M][N] array of r_dtype added to the product (a
 *                residual connection fused into the store; an fp32 residual
 *                stream keeps the small difference between the fake-ternary
 *                and the full-precision block outputs above bf16 rounding);
 *                NULL for none.  Dense layers only; a bf16 Y takes a bf16
 *                residual.
 * Requires K % 8 == 0; M, N, K > 0.
 */
catq_status catq_fakeq_linear_fwd(const void* X, const void* W_fake, catq_dtype dtype, void* Y,
                                  catq_dtype y_dtype, int64_t M, int64_t N, int64_t K,
                                  int32_t n_experts, const int64_t* row_offsets,
                                  const void* residual, catq_dtype r_dtype, hipStream_t stream);

/*
 * catq_fakeq_linear_bwd -- backward of the fake-ternary linear layer to its
 * input and to the learnable factors of its weight: the gradient of the
 * reconstruction loss of Eq. 7 (Sec. 2.4) taken through the softened
 * ternarisation of Eq. 5-6 (Sec. 2.3; in the hard branch, the derivatives of
 * the last soft sharpness stand in for the step) and the modulation of
 * Eq. 3-4 (Sec. 2.2).  Only the three factors are learned; W is frozen.
 *
 *   dX[M][K]      = dY[M][N] . W_fake[N][K]            (NULL: not computed)
 *   G[N][K]       = dY^T . X  (= dL/dW_fake, fp32)     (into dW_fake if given,
 *                                                        else into workspace)
 *   per group, with f_W, f_Delta the partial derivatives of f at (W_hat; s, Delta)
 *   (HARD mode: T = code, derivatives at s_bwd; IDENTITY: all zero):
 *     dL/dd_mu    = -alpha0 * sum G f_W
 *     dL/dd_alpha =  alpha0 * (sum G T - sum G f_W W_hat)
 *     dL/dd_Delta =  Delta0 * alpha * sum G f_Delta
 *   written (overwritten) to g_d_mu, g_d_alpha, g_d_delta; a factor with
 *   stride 0 receives one value, the sum over all groups.
 *
 *   dY, X, W_fake   as in catq_fakeq_linear_fwd (same dtype, same expert
 *                   grouping through n_experts / row_offsets)
 *   W, w_dtype      the frozen full-precision weight ([E][N][K] for experts)
 *   stats           fp32 [n_groups][2] from catq_modulate_ternarize
 *   d_mu, d_alpha, d_delta, p   the factors and parameters of the forward
 *   workspace       device scratch of at least
 *                   catq_workspace_size(CATQ_WS_LINEAR_BWD, M, N, K, n_experts)
 *                   bytes (may be NULL when that size is 0)
 * With g_d_mu, g_d_alpha, g_d_delta and dW_fake all NULL only dX is computed
 * (W, w_dtype, stats, the factors, p and the workspace are then not read);
 * a caller can so run the input-gradient half and the weight-gradient half
 * (dX NULL) on two streams.  Otherwise all three gradient outputs are
 * required.
 * Where G needs no split of the token contraction (routed experts, or a
 * dense shape the library leaves unsplit) and bf16 operands, 128-weight
 * groups and no dW_fake are given, the factor gradients are reduced inside
 * the G product and G is not stored; they then agree with the two-pass
 * result up to the order of the fp32 sums (deterministic either way).
 * Requires N % 8 == 0 and K % 8 == 0.
 */
catq_status catq_fakeq_linear_bwd(const void* dY, const void* X, const void* W_fake,
                                  catq_dtype dtype, int64_t M, int64_t N, int64_t K,
                                  int32_t n_experts, const int64_t* row_offsets, const void* W,
                                  catq_dtype w_dtype, const float* stats, const float* d_mu,
                                  const float* d_alpha, const float* d_delta,
                                  const catq_lmst_params* p, void* dX, float* g_d_mu,
                                  float* g_d_alpha, float* g_d_delta, float* dW_fake,
                                  void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * catq_block_recon_loss -- the reconstruction loss of Eq. 7 as a mean over
 * the n outputs of the window:
 *   loss = (1/n) sum_i (Y_q[i] - Y_fp[i])^2          -> fp32 scalar at `loss`
 *   dY_q[i] = 2 (Y_q[i] - Y_fp[i]) / n               -> dy_dtype (NULL: skipped)
 * Y_q and Y_fp (both of `dtype`) are the window outputs with fake-ternary and
 * with full-precision weights on the same calibration input.  The sum is
 * reduced in a fixed order (fp32 within 8 elements, float64 beyond).
 * workspace >= catq_workspace_size(CATQ_WS_LOSS, n, 1, 1, 1) bytes.
 * Requires n % 8 == 0.
 */
catq_status catq_block_recon_loss(const void* Y_q, const void* Y_fp, catq_dtype dtype, int64_t n,
                                  float* loss, void* dY_q, catq_dtype dy_dtype, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream);

/*
 * catq_block_recon_loss_noalloc -- catq_block_recon_loss without a workspace
 * argument and without any allocation, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same kernels, same arguments otherwise, same bits.
 * Its partial sums live in a library-owned file-scope device array of 1024
 * doubles (8 KiB; each GPU the library runs on holds one copy until the
 * process ends); every n accepted by catq_block_recon_loss needs at most 1024
 * partials, and each partial is written before it is read, so nothing has to
 * be cleared between calls.  Calls that overlap on one GPU (two streams, or
 * two host threads) share that array and race: issue them in order.
 * Errors as catq_block_recon_loss (no CATQ_ERR_WORKSPACE); CATQ_ERR_HIP if
 * the array's device address cannot be obtained.
 */
catq_status catq_block_recon_loss_noalloc(const void* Y_q, const void* Y_fp, catq_dtype dtype,
                                          int64_t n, float* loss, void* dY_q, catq_dtype dy_dtype,
                                          hipStream_t stream);

/*
 * catq_pack_ternary -- 2-bit storage of ternary codes for deployment
 * (App. B.2: T in {-1,0,+1} plus the group scale alpha, zero-point free).
 * Code c = T + 1 in {0,1,2}; byte b of row r holds elements 4b..4b+3 of that
 * row, element 4b+j in bits 2j..2j+1 (least significant first).
 *   codes   int8 [d_out][d_in]    packed  uint8 [d_out][d_in/4]
 * Requires d_in % 4 == 0.  A code outside {-1,0,1} is stored as 3 (invalid).
 */
catq_status catq_pack_ternary(const int8_t* codes, int64_t d_out, int64_t d_in, uint8_t* packed,
                              hipStream_t stream);

/*
 * catq_ternarize_pack -- the final hard ternarisation (Eq. 2 on the modulated
 * weights of Eq. 3-4) written straight to the 2-bit storage above (App. B.2),
 * with the group scales: the codes of catq_modulate_ternarize in HARD mode,
 * packed as catq_pack_ternary packs them, in one pass over W (no int8 codes
 * and no W_fake in memory).
 *   W, w_dtype, d_out, d_in, d_mu, d_alpha, d_delta, stats, stats_mode
 *              as for catq_modulate_ternarize
 *   p          host pointer; p->mode must be CATQ_HARD
 *   packed     uint8 [d_out][d_in/4], written
 *   alpha_out  fp32 [n_groups] group scales alpha; may be NULL
 * Errors: NULL W/factors/stats/packed/p, mode other than HARD, d_in % g,
 * g out of range, delta0 <= 0, bad w_dtype, misaligned pointers.
 */
catq_status catq_ternarize_pack(const void* W, catq_dtype w_dtype, int64_t d_out, int64_t d_in,
                                const float* d_mu, const float* d_alpha, const float* d_delta,
                                const catq_lmst_params* p, float* stats, int32_t stats_mode,
                                uint8_t* packed, float* alpha_out, hipStream_t stream);

/* catq_ternary_linear -- deployment-side linear layer on that storage:
 *   Y[m][n] = sum_k X[m][k] * alpha[n][k / g] * T[n][k]
 * i.e. Y = X (alpha * T)^T with the ternary weights and group scales of the
 * final ternarisation (App. B.2: T plus one scale per group, no zero point),
 * reading 2 bits per weight.  Code 3 (invalid) contributes 0.
 *   X       bf16 [M][ldx] (row-major; d_in <= ldx <= 2^24, ldx % 8 == 0)
 *   packed  uint8 [d_out][d_in/4] in the layout above
 *   alpha   fp32 [d_out][d_in/g]
 *   Y       y_dtype (fp32 or bf16) [M][ldy], ldy >= d_out; written, not
 *           accumulated
 * g is the group size (128 times a power of two, dividing d_in); d_in <= 65536.
 * M = 0 is a no-op.  Accumulation in fp32 in a fixed order (bitwise
 * deterministic for a given shape).  Decode-sized M re-reads the codes per
 * 16 tokens; from 32 tokens on, where it is estimated cheaper, a kernel of
 * 128-row x 64- or 128-token tiles decodes each code once per tile (same
 * per-chunk fp32 scaling, so the same error bound).  X and alpha 16-byte
 * aligned, packed 8-byte, Y 4-byte. */
catq_status catq_ternary_linear(const void* X, int64_t M, int64_t ldx, const uint8_t* packed,
                                const float* alpha, int64_t d_out, int64_t d_in, int32_t g,
                                void* Y, catq_dtype y_dtype, int64_t ldy, hipStream_t stream);

/* Fused variants for the SwiGLU MLP of a decoder block (a4 and a8 with the
 * SwiGLU of a5 / a7 in the GEMM epilogue; same results as the unfused calls).
 *
 * catq_fakeq_gateup_swiglu_fwd -- the fused gate|up projection and its SwiGLU:
 *   gu = X W_fake^T, a = silu(gate) * up
 *   X bf16 [M][K], W_fake bf16 [2F][K] (gate rows, then up rows), gu bf16
 *   [M][2F] ([gate | up]), a bf16 [M][F]; F % 8 == 0.
 * catq_fakeq_down_swiglu_bwd -- input gradient of the down projection with
 * the SwiGLU backward:  d a = dY W_fake, then d gate = d a * up * silu'(gate),
 * d up = d a * silu(gate), written as d[gate | up]:
 *   dY bf16 [M][N], W_fake bf16 [N][F], gu bf16 [M][2F] (the forward's),
 *   dgu bf16 [M][2F] out; da bf16 [M][F] is scratch used only for shapes the
 *   fused epilogue does not take (may be NULL otherwise; then such a shape is
 *   CATQ_ERR_NULL).  F % 8 == 0.  16-byte aligned pointers. */
catq_status catq_fakeq_gateup_swiglu_fwd(const void* X, const void* W_fake, int64_t M, int64_t F,
                                         int64_t K, void* gu, void* a, hipStream_t stream);
catq_status catq_fakeq_down_swiglu_bwd(const void* dY, const void* W_fake, int64_t M, int64_t N,
                                       int64_t F, const void* gu, void* dgu, void* da,
                                       hipStream_t stream);

/* Workspace sizes, in bytes, for the calls that take a workspace. */
enum { CATQ_WS_LINEAR_BWD = 0, CATQ_WS_LOSS = 1 };
size_t catq_workspace_size(int32_t which_call, int64_t M, int64_t N, int64_t K, int32_t n_experts);

const char* catq_status_string(catq_status s);
/* Detail of the last failure on the calling thread ("" if none). */
const char* catq_last_error_message(void);

/* ===================================================================== *
 * Auxiliary entry points: the rest of the decoder block around the fake-
 * ternary linears (the paper uses its host models' blocks unchanged).
 * Same conventions as above.  bf16 activations unless stated.
 * ===================================================================== */

/* y = x / sqrt(mean(x^2) + eps) per row of length n (unit weight); x of
 * x_dtype (bf16 or fp32), y bf16, rstd fp32 [rows] (may be NULL). */
catq_status catq_aux_rmsnorm_fwd(const void* x, catq_dtype x_dtype, int64_t rows, int64_t n,
                                 float eps, void* y, float* rstd, hipStream_t stream);
/* dx = rstd*dy - x*rstd^3*sum(dy*x)/n (+ dres if not NULL); x of x_dtype,
 * dy, dres and dx bf16. */
catq_status catq_aux_rmsnorm_bwd(const void* x, catq_dtype x_dtype, const float* rstd,
                                 const void* dy, const void* dres, int64_t rows, int64_t n,
                                 void* dx, hipStream_t stream);

/* W1.58A8 activation fake quantization (Sec. 3: all intermediate
 * activations but the softmax output are quantized to 8 bits; the quantizer
 * is not specified -- this is symmetric absmax per group): for each group of
 * `group` consecutive values of a row, s = max|x|/127, q = round-half-even
 * (x/s) clamped to [-127, 127] (0 when s = 0), y = bf16(q*s), all in IEEE
 * fp32.  x [rows][n] of x_dtype (bf16 or fp32), y bf16 [rows][n]; y may be x
 * when x is bf16.  group divides n and is a multiple of 8.  rows = 0 is a
 * no-op.  The backward is straight-through (no call needed). */
catq_status catq_aux_act_quant(const void* x, catq_dtype x_dtype, int64_t rows, int64_t n,
                               int64_t group, void* y, hipStream_t stream);

/* Attention geometry for the q/k/v buffer produced by the fused q|k|v linear. */
typedef struct {
  int32_t batch, seq, n_q, n_kv, head_dim;
  int32_t qk_norm;     /* per-head RMSNorm on q and k before the rotary embedding */
  float rope_theta;    /* rotary base; pairs (i, i + d/2) rotate by pos*theta^(-2i/d) */
  float eps;           /* RMSNorm epsilon of the q/k norms */
  int32_t act_quant;   /* 1: Q, K, V of the attention products fake-quantized to 8 bits
                          per (token, head) as in catq_aux_act_quant (W1.58A8; the softmax
                          output is not); needs head_dim 64 or 128.  0: off */
} catq_attn_desc;

/*
 * Causal grouped-query softmax attention on qkv [batch*seq][(n_q + 2 n_kv) d]
 * (q heads, then k heads, then v heads), output o [batch*seq][n_q d].
 * The forward keeps what the backward needs (and its own scratch) in `saved`,
 * at least catq_attn_saved_bytes(a) bytes; the backward takes the forward's
 * output o, needs a scratch workspace of catq_attn_bwd_workspace_bytes(a)
 * bytes and writes dqkv in the layout of qkv.  qkv, o, d_o and dqkv are bf16.
 * Head dims 64 and 128 run fused (flash) kernels that keep only the per-query
 * log-sum-exp; 256 runs score matrices through the GEMM kernel.
 */
size_t catq_attn_saved_bytes(const catq_attn_desc* a);
size_t catq_attn_bwd_workspace_bytes(const catq_attn_desc* a);
catq_status catq_aux_attention_fwd(const catq_attn_desc* a, const void* qkv, void* o, void* saved,
                                   size_t saved_bytes, hipStream_t stream);
catq_status catq_aux_attention_bwd(const catq_attn_desc* a, const void* qkv, const void* o,
                                   const void* saved, const void* d_o, void* dqkv,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/* SwiGLU on gu [rows][2F] (gate | up): a = silu(gate) * up, [rows][F]. */
catq_status catq_aux_swiglu_fwd(const void* gu, int64_t rows, int64_t F, void* a,
                                hipStream_t stream);
catq_status catq_aux_swiglu_bwd(const void* gu, const void* da, int64_t rows, int64_t F,
                                void* dgu, hipStream_t stream);

/*
 * Routed experts.  logits fp32 [T][E] (router left unquantised, App. B.2).
 * catq_aux_moe_route: top-k per token (largest first, ties to the lower id),
 *   weights = softmax over the k selected logits (fp32 [T][k]), expert ids
 *   int32 [T][k], row_offsets int64 [E+1], and for each (token, slot) its row
 *   in the expert-grouped order, perm_row int32 [T][k] (tokens in order
 *   inside each expert).  Requires k <= 16, E <= 1024.
 * catq_aux_moe_gather: xg[perm_row[t][j]] = x[t]          ([T*k][h])
 * catq_aux_moe_combine: y[t] = res[t] + sum_j w[t][j] * yg[perm_row[t][j]]
 *   (res and y of y_dtype, bf16 or fp32; res may be NULL)
 * catq_aux_moe_combine_bwd: dyg[perm_row[t][j]] = w[t][j] * dy[t]
 * catq_aux_moe_scatter_add: dx[t] = sum_j dxg[perm_row[t][j]]
 */
catq_status catq_aux_moe_route(const float* logits, int64_t T, int32_t E, int32_t k,
                               int32_t* expert_ids, float* weights, int32_t* perm_row,
                               int64_t* row_offsets, void* workspace, size_t workspace_bytes,
                               hipStream_t stream);
size_t catq_aux_moe_route_workspace_bytes(int64_t T, int32_t E, int32_t k);
catq_status catq_aux_moe_gather(const void* x, const int32_t* perm_row, int64_t T, int32_t k,
                                int64_t h, void* xg, hipStream_t stream);
catq_status catq_aux_moe_combine(const void* yg, const int32_t* perm_row, const float* weights,
                                 const void* res, int64_t T, int32_t k, int64_t h, void* y,
                                 catq_dtype y_dtype, hipStream_t stream);
catq_status catq_aux_moe_combine_bwd(const void* dy, const int32_t* perm_row, const float* weights,
                                     int64_t T, int32_t k, int64_t h, void* dyg,
                                     hipStream_t stream);
catq_status catq_aux_moe_scatter_add(const void* dxg, const int32_t* perm_row, int64_t T, int32_t k,
                                     int64_t h, void* dx, hipStream_t stream);

/*
 * AdamW on one factor array (fp32 [n]): m, v moments updated in place,
 * p -= lr * mhat / (sqrt(vhat) + eps), no weight decay; then clamped to
 * [lo, hi] (the constraints -1 < d_mu < 1, d_alpha > 0, d_Delta > 0 of Sec. 2.2).
 * step is 1-based.  beta1, beta2 and eps are taken in double: the kernel's
 * 1 - beta and the bias corrections are formed from them in double and
 * rounded once to fp32 (1 - (float)0.999 would miss 0.001 by 1.3e-5).
 */
catq_status catq_aux_adamw(float* p, const float* grad, float* m, float* v, int64_t n,
                           int64_t step, float lr, double beta1, double beta2, double eps, float lo,
                           float hi, hipStream_t stream);

/* Elementwise y = a + b (bf16 or f32), n % 8 == 0. */
catq_status catq_aux_add(const void* a, const void* b, void* y, catq_dtype dtype, int64_t n,
                         hipStream_t stream);

/* ===================================================================== *
 * Launch tracing (measurement aid).  While enabled, the library records a
 * pair of HIP events around each of its kernel launches, on the launch
 * stream, with the kernel's tag (its function and template arguments) and
 * the algorithmic work of that launch.  Process-global, one host thread.
 * ===================================================================== */
typedef struct {
  char tag[96];   /* kernel function and template arguments                 */
  double flops;   /* algorithmic floating-point operations of the launch     */
  double bytes;   /* algorithmic HBM bytes (each operand read/written once)  */
  int64_t M, N, K;
  float ms;       /* event-measured duration (filled by catq_trace_get)      */
} catq_trace_rec;

/* Create `capacity` event pairs and start recording (host memory only). */
catq_status catq_trace_enable(int32_t capacity);
void catq_trace_pause(int32_t paused);
void catq_trace_reset(void);
int32_t catq_trace_count(void);
/* Waits for record i's stop event and returns the record with its duration. */
catq_status catq_trace_get(int32_t i, catq_trace_rec* out);
void catq_trace_disable(void);

#ifdef __cplusplus
}
#endif
#endif /* CATQ_H */
