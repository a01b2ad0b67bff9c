// Output-reconstruction loss of Eq. 7 (mean of squared differences over the
// window output) and its gradient.  Two deterministic passes: a fixed grid of
// blocks accumulates fixed slices (fp32 per 8 elements, float64 per thread and
// across the block), then one block folds the per-block partials in order.
#include <mutex>

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

// Partials of the allocation-free entry point: one double per block of the
// first pass (at most LOSS_BLOCKS), file-scope device memory held by each GPU
// until the process ends.  Host code must not use this name as an address:
// its device address comes from hipGetSymbolAddress, per device.
static __device__ __align__(256) double scratch[LOSS_BLOCKS];

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex scratch_mu;
double* scratch_ptr[MAX_DEVICES] = {};

// Device address of `scratch` on the current device, resolved once per
// device with that device current.
catq_status scratch_address(double** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  CATQ_REQUIRE(e == hipSuccess, CATQ_ERR_HIP, "hipGetDevice failed: %s", hipGetErrorString(e));
  CATQ_REQUIRE(dev >= 0 && dev < MAX_DEVICES, CATQ_ERR_HIP, "device %d beyond %d", dev,
               MAX_DEVICES);
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    CATQ_REQUIRE(e == hipSuccess && p, CATQ_ERR_HIP, "hipGetSymbolAddress(scratch) failed: %s",
                 hipGetErrorString(e));
    scratch_ptr[dev] = static_cast<double*>(p);
  }
  *out = scratch_ptr[dev];
  return CATQ_OK;
}

catq_status check_loss_args(const void* Y_q, const void* Y_fp, catq_dtype dtype, int64_t n,
                            float* loss, void* dY_q, catq_dtype dy_dtype) {
  CATQ_REQUIRE(dtype_ok(dy_dtype), CATQ_ERR_DTYPE, "bad dy dtype");
  CATQ_REQUIRE(Y_q && Y_fp && loss, CATQ_ERR_NULL, "Y_q, Y_fp and loss must not be NULL");
  CATQ_REQUIRE(count_ok(n) && n % 8 == 0, CATQ_ERR_SHAPE,
               "n must be a positive multiple of 8, at most 2^38");
  CATQ_REQUIRE(dtype_ok(dtype), CATQ_ERR_DTYPE, "bad dtype");
  CATQ_REQUIRE(aligned16(Y_q) && aligned16(Y_fp) && aligned16(dY_q), CATQ_ERR_ALIGN,
               "pointers must be 16-byte aligned");
  return CATQ_OK;
}

// Number of first-pass blocks (= partials) for n outputs.
int loss_blocks(int64_t n) {
  const int64_t n8 = n / 8;
  int64_t nb = (n8 + LOSS_THREADS - 1) / LOSS_THREADS;
  return (int)(nb > LOSS_BLOCKS ? LOSS_BLOCKS : nb);
}

// Both passes, the partials in `partial` (nb doubles, each written by the
// first pass before the second reads it).
catq_status launch_loss(const void* Y_q, const void* Y_fp, catq_dtype dtype, int64_t n,
                        float* loss, void* dY_q, catq_dtype dy_dtype, double* partial,
                        hipStream_t stream) {
  const int64_t n8 = n / 8;
  const int nb = loss_blocks(n);
  const float scale = (float)(2.0 / (double)n);
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

}  // namespace

}  // namespace catq

using namespace catq;

extern "C" catq_status catq_block_recon_loss(const void* Y_q, const void* Y_fp, catq_dtype dtype,
                                             int64_t n, float* loss, void* dY_q,
                                             catq_dtype dy_dtype, void* workspace,
                                             size_t workspace_bytes, hipStream_t stream) {
  clear_error();
  CATQ_TRY(check_loss_args(Y_q, Y_fp, dtype, n, loss, dY_q, dy_dtype));
  CATQ_REQUIRE(aligned16(workspace), CATQ_ERR_ALIGN, "pointers must be 16-byte aligned");
  const size_t need = catq_workspace_size(CATQ_WS_LOSS, n, 1, 1, 1);
  CATQ_REQUIRE(workspace && workspace_bytes >= need, CATQ_ERR_WORKSPACE,
               "workspace of %zu bytes needed", need);
  return launch_loss(Y_q, Y_fp, dtype, n, loss, dY_q, dy_dtype,
                     reinterpret_cast<double*>(workspace), stream);
}

extern "C" catq_status catq_block_recon_loss_noalloc(const void* Y_q, const void* Y_fp,
                                                     catq_dtype dtype, int64_t n, float* loss,
                                                     void* dY_q, catq_dtype dy_dtype,
                                                     hipStream_t stream) {
  clear_error();
  CATQ_TRY(check_loss_args(Y_q, Y_fp, dtype, n, loss, dY_q, dy_dtype));
  const int nb = loss_blocks(n);
  CATQ_REQUIRE(nb <= LOSS_BLOCKS, CATQ_ERR_SHAPE,
               "%d partial sums exceed the %d of the library's scratch", nb, LOSS_BLOCKS);
  double* partial = nullptr;
  CATQ_TRY(scratch_address(&partial));
  return launch_loss(Y_q, Y_fp, dtype, n, loss, dY_q, dy_dtype, partial, stream);
}
