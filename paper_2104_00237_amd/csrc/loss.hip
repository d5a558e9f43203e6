// Loss kernels: forward value and gradient in one pass.  Sums are taken in a
// fixed order in float64, so the loss is deterministic.
//
//   cross-entropy  loss = mean_b (logsumexp(z_b) - z_{b,y_b});  dz = (softmax - onehot) / B
//   squared error  loss = mean (y - t)^2;                        dy = 2 (y - t) / numel

#include "common.h"

namespace opfuse {

// Fixed-shape tree reduction of one double per thread over a 256-thread block.
__device__ double block_sum256(double v, double* sh) {
  sh[threadIdx.x] = v;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s) sh[threadIdx.x] += sh[threadIdx.x + s];
    __syncthreads();
  }
  return sh[0];
}

// One workgroup; thread t owns rows t, t+256, ...
__global__ __launch_bounds__(256) void xent_kernel(const float* __restrict__ z,
                                                   const int64_t* __restrict__ labels, int64_t B,
                                                   int64_t C, int64_t ld, float* loss, float* dz) {
  __shared__ double sh[256];
  double part = 0.0;
  const float invB = 1.0f / (float)B;
  for (int64_t b = threadIdx.x; b < B; b += 256) {
    const float* row = z + b * ld;
    float mx = row[0];
    for (int64_t c = 1; c < C; ++c) mx = fmaxf(mx, row[c]);
    float se = 0.f;
    for (int64_t c = 0; c < C; ++c) se += expf(row[c] - mx);
    const float lse = mx + logf(se);
    const int64_t y = labels[b];
    const bool ok = y >= 0 && y < C;
    part += ok ? (double)(lse - row[y]) : (double)NAN;
    for (int64_t c = 0; c < C; ++c) {
      const float p = expf(row[c] - lse);
      dz[b * ld + c] = ((c == y) ? p - 1.f : p) * invB;
    }
  }
  const double tot = block_sum256(part, sh);
  if (threadIdx.x == 0) *loss = (float)(tot / (double)B);
}

hipError_t launch_xent(const float* z, const int64_t* labels, int64_t B, int64_t C, int64_t ld,
                       float* loss, float* dz, hipStream_t stream) {
  hipLaunchKernelGGL(xent_kernel, dim3(1), dim3(256), 0, stream, z, labels, B, C, ld, loss, dz);
  return hipGetLastError();
}

constexpr int MSE_BLOCKS = 512;

size_t mse_ws_bytes(int64_t, int64_t) { return MSE_BLOCKS * sizeof(double); }

__global__ __launch_bounds__(256) void mse_partial_kernel(const float* __restrict__ y,
                                                          const float* __restrict__ t, int64_t M,
                                                          int64_t D, int64_t ld, float* dy,
                                                          double* part) {
  __shared__ double sh[256];
  const int64_t n = M * D;
  const float scale = 2.0f / (float)n;
  double acc = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int64_t r = i / D, c = i % D;
    const float d = y[r * ld + c] - t[i];
    dy[r * ld + c] = d * scale;
    acc += (double)d * (double)d;
  }
  const double s = block_sum256(acc, sh);
  if (threadIdx.x == 0) part[blockIdx.x] = s;
}

__global__ __launch_bounds__(256) void mse_final_kernel(const double* part, int nb, int64_t n,
                                                        float* loss) {
  __shared__ double sh[256];
  double acc = 0.0;
  for (int i = threadIdx.x; i < nb; i += 256) acc += part[i];
  const double s = block_sum256(acc, sh);
  if (threadIdx.x == 0) *loss = (float)(s / (double)n);
}

hipError_t launch_mse(const float* y, const float* t, int64_t M, int64_t D, int64_t ld,
                      float* loss, float* dy, void* ws, hipStream_t stream) {
  double* part = (double*)ws;
  hipLaunchKernelGGL(mse_partial_kernel, dim3(MSE_BLOCKS), dim3(256), 0, stream, y, t, M, D, ld,
                     dy, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(mse_final_kernel, dim3(1), dim3(256), 0, stream, (const double*)part,
                     MSE_BLOCKS, M * D, loss);
  return hipGetLastError();
}

}  // namespace opfuse
