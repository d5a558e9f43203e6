// 2x2 max-pool, stride 2, NHWC, with the window position of the first maximum
// (row-major window order, strict >) kept for the backward pass.  The
// backward scatters each pooled gradient to that position and can apply the
// ReLU mask of the pool's input (the ReLU output feeding the pool: the
// derivative there is 1 exactly where that output is > 0).
//
// Global average pool over the spatial positions of an NHWC map ([N, P, C],
// P = H*W): y[n,c] = (sum over p in order of x[n,p,c]) / P; the backward
// spreads dy[n,c] / P to every position, with the same optional ReLU mask.

#include "common.h"

namespace opfuse {

__global__ __launch_bounds__(256) void maxpool_fwd_kernel(const float* __restrict__ x, int64_t N,
                                                          int64_t H, int64_t W, int64_t C,
                                                          float* __restrict__ y,
                                                          uint8_t* __restrict__ arg) {
  const int64_t Ho = H / 2, Wo = W / 2;
  const int64_t total = N * Ho * Wo * C;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * 256) {
    const int64_t c = i % C, t = i / C;
    const int64_t wo = t % Wo, t2 = t / Wo, ho = t2 % Ho, n = t2 / Ho;
    const int64_t base = ((n * H + 2 * ho) * W + 2 * wo) * C + c;
    const float v0 = x[base], v1 = x[base + C], v2 = x[base + W * C], v3 = x[base + W * C + C];
    float best = v0;
    uint8_t a = 0;
    if (v1 > best) { best = v1; a = 1; }
    if (v2 > best) { best = v2; a = 2; }
    if (v3 > best) { best = v3; a = 3; }
    y[i] = best;
    arg[i] = a;
  }
}

__global__ __launch_bounds__(256) void maxpool_bwd_kernel(const float* __restrict__ dy,
                                                          const uint8_t* __restrict__ arg,
                                                          const float* __restrict__ mask_src,
                                                          int64_t N, int64_t H, int64_t W,
                                                          int64_t C, float* __restrict__ dx) {
  const int64_t Ho = H / 2, Wo = W / 2;
  const int64_t total = N * Ho * Wo * C;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * 256) {
    const int64_t c = i % C, t = i / C;
    const int64_t wo = t % Wo, t2 = t / Wo, ho = t2 % Ho, n = t2 / Ho;
    const int64_t base = ((n * H + 2 * ho) * W + 2 * wo) * C + c;
    const int64_t off[4] = {base, base + C, base + W * C, base + W * C + C};
    const int a = arg[i];
    const float g = dy[i];
    for (int k = 0; k < 4; ++k) {
      float v = (k == a) ? g : 0.f;
      if (mask_src && k == a && !(mask_src[off[k]] > 0.f)) v = 0.f;
      dx[off[k]] = v;
    }
  }
}

// One thread per (n, c): consecutive threads read consecutive channels.
__global__ __launch_bounds__(256) void avgpool_fwd_kernel(const float* __restrict__ x, int64_t N,
                                                          int64_t P, int64_t C,
                                                          float* __restrict__ y) {
  const int64_t total = N * C;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * 256) {
    const int64_t c = i % C, n = i / C;
    const float* src = x + n * P * C + c;
    float s = 0.f;
    for (int64_t p = 0; p < P; ++p) s = __fadd_rn(s, src[p * C]);
    y[i] = __fdiv_rn(s, (float)P);
  }
}

__global__ __launch_bounds__(256) void avgpool_bwd_kernel(const float* __restrict__ dy,
                                                          const float* __restrict__ mask_src,
                                                          int64_t N, int64_t P, int64_t C,
                                                          float* __restrict__ dx) {
  const int64_t total = N * P * C;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * 256) {
    const int64_t c = i % C, n = i / (P * C);
    float v = __fdiv_rn(dy[n * C + c], (float)P);
    if (mask_src && !(mask_src[i] > 0.f)) v = 0.f;
    dx[i] = v;
  }
}

static unsigned blocks_for(int64_t n) {
  const int64_t b = (n + 255) / 256;
  return (unsigned)(b < 65536 ? (b > 0 ? b : 1) : 65536);
}

hipError_t launch_maxpool_fwd(const float* x, int64_t N, int64_t H, int64_t W, int64_t C,
                              float* y, uint8_t* arg, hipStream_t s) {
  hipLaunchKernelGGL(maxpool_fwd_kernel, dim3(blocks_for(N * (H / 2) * (W / 2) * C)), dim3(256),
                     0, s, x, N, H, W, C, y, arg);
  return hipGetLastError();
}

hipError_t launch_maxpool_bwd(const float* dy, const uint8_t* arg, const float* mask_src,
                              int64_t N, int64_t H, int64_t W, int64_t C, float* dx,
                              hipStream_t s) {
  hipLaunchKernelGGL(maxpool_bwd_kernel, dim3(blocks_for(N * (H / 2) * (W / 2) * C)), dim3(256),
                     0, s, dy, arg, mask_src, N, H, W, C, dx);
  return hipGetLastError();
}

hipError_t launch_avgpool_fwd(const float* x, int64_t N, int64_t P, int64_t C, float* y,
                              hipStream_t s) {
  hipLaunchKernelGGL(avgpool_fwd_kernel, dim3(blocks_for(N * C)), dim3(256), 0, s, x, N, P, C, y);
  return hipGetLastError();
}

hipError_t launch_avgpool_bwd(const float* dy, const float* mask_src, int64_t N, int64_t P,
                              int64_t C, float* dx, hipStream_t s) {
  hipLaunchKernelGGL(avgpool_bwd_kernel, dim3(blocks_for(N * P * C)), dim3(256), 0, s, dy,
                     mask_src, N, P, C, dx);
  return hipGetLastError();
}

}  // namespace opfuse
