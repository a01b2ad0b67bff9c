// Output-reconstruction loss of Eq. 7 (mean of squared differences over the
// window output) and its gradient.  Two deterministic passes: a fixed grid of
// blocks accumulates fixed slices (fp32 per 8 elements, float64 per thread and
// across the block), then one block folds the per-block partials in order.
#include "kernels.h"

namespace catq {

constexpr int LOSS_BLOCKS = 1024;
constexpr int LOSS_THREADS = 256;

template <typename T, typename DT>
__global__ __launch_bounds__(LOSS_THREADS) void loss_partial_kernel(const T* yq, const T* yfp,
                                                                    int64_t n8, float scale,
                                                                    DT* dy, double* partial) {
  __shared__ double red[LOSS_THREADS];
  double acc = 0.0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n8; i += stride) {
    float a[8], b[8];
    load8<T>(yq + i * 8, a);
    load8<T>(yfp + i * 8, b);
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float d = a[j] - b[j];
      s = fmaf(d, d, s);
      a[j] = d * scale;
    }
    acc += (double)s;
    if (dy) store8<DT>(dy + i * 8, a);
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = LOSS_THREADS / 2; s >= 1; s >>= 1) {
    if ((int)threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) partial[blockIdx.x] = red[0];
}

__global__ __launch_bounds__(LOSS_THREADS) void loss_final_kernel(const double* partial, int nb,
                                                                  double inv_n, float* loss) {
  __shared__ double red[LOSS_THREADS];
  double acc = 0.0;
  for (int i = threadIdx.x; i < nb; i += LOSS_THREADS) acc += partial[i];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = LOSS_THREADS / 2; s >= 1; s >>= 1) {
    if ((int)threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) loss[0] = (float)(red[0] * inv_n);
}

}  // namespace catq

using namespace catq;

extern "C" catq_status catq_block_recon_loss(const void* Y_q, const void* Y_fp, catq_dtype dtype,
                                             int64_t n, float* loss, void* dY_q,
                                             catq_dtype dy_dtype, void* workspace,
                                             size_t workspace_bytes, hipStream_t stream) {
  clear_error();
  CATQ_REQUIRE(dtype_ok(dy_dtype), CATQ_ERR_DTYPE, "bad dy dtype");
  CATQ_REQUIRE(Y_q && Y_fp && loss, CATQ_ERR_NULL, "Y_q, Y_fp and loss must not be NULL");
  CATQ_REQUIRE(n > 0 && n % 8 == 0, CATQ_ERR_SHAPE, "n must be a positive multiple of 8");
  CATQ_REQUIRE(dtype_ok(dtype), CATQ_ERR_DTYPE, "bad dtype");
  CATQ_REQUIRE(aligned16(Y_q) && aligned16(Y_fp) && aligned16(dY_q) && aligned16(workspace),
               CATQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  const size_t need = catq_workspace_size(CATQ_WS_LOSS, n, 1, 1, 1);
  CATQ_REQUIRE(workspace && workspace_bytes >= need, CATQ_ERR_WORKSPACE,
               "workspace of %zu bytes needed", need);
  const int64_t n8 = n / 8;
  int nb = (int)((n8 + LOSS_THREADS - 1) / LOSS_THREADS);
  if (nb > LOSS_BLOCKS) nb = LOSS_BLOCKS;
  const float scale = (float)(2.0 / (double)n);
  double* partial = reinterpret_cast<double*>(workspace);
  dim3 g(nb), b(LOSS_THREADS);
  const double lby = (double)n * ((dtype == CATQ_BF16 ? 4.0 : 8.0) + (dY_q ? (dy_dtype == CATQ_BF16 ? 2.0 : 4.0) : 0.0));
  CATQ_TRACED(stream, "loss_partial_kernel", 0.0, lby, n, 0, 0, {
    if (dtype == CATQ_BF16 && dy_dtype == CATQ_BF16)
      hipLaunchKernelGGL((loss_partial_kernel<bf16, bf16>), g, b, 0, stream, (const bf16*)Y_q,
                         (const bf16*)Y_fp, n8, scale, (bf16*)dY_q, partial);
    else if (dtype == CATQ_BF16)
      hipLaunchKernelGGL((loss_partial_kernel<bf16, float>), g, b, 0, stream, (const bf16*)Y_q,
                         (const bf16*)Y_fp, n8, scale, (float*)dY_q, partial);
    else if (dy_dtype == CATQ_BF16)
      hipLaunchKernelGGL((loss_partial_kernel<float, bf16>), g, b, 0, stream, (const float*)Y_q,
                         (const float*)Y_fp, n8, scale, (bf16*)dY_q, partial);
    else
      hipLaunchKernelGGL((loss_partial_kernel<float, float>), g, b, 0, stream, (const float*)Y_q,
                         (const float*)Y_fp, n8, scale, (float*)dY_q, partial);
  });
  CATQ_CHECK_LAUNCH("recon loss");
  hipLaunchKernelGGL(loss_final_kernel, dim3(1), dim3(LOSS_THREADS), 0, stream, partial, nb,
                     1.0 / (double)n, loss);
  CATQ_CHECK_LAUNCH("recon loss final");
  return CATQ_OK;
}
