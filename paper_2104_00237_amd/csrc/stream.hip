// HBM streaming probes: the read, copy and in-place read-modify-write rates
// (one array, or three updated side by side)
// this device achieves with plain coalesced 128-bit accesses, and the
// three-array rate in the 4-byte column layout of the merged backward kernel.  They give the achievable ceiling
// that the parameter-bound kernels (the fused and merged updates, which
// stream W and the optimizer state once) are measured against, beside the
// published 8 TB/s.  Not part of the paper's method.
//
// Each thread moves UNROLL float4s per pass, all loads issued before any use,
// so a workgroup of 256 threads has UNROLL * 4 KiB in flight; the grid strides
// over the buffer.  Loads and stores are non-temporal: the data is touched
// once and should not displace anything in the caches.

#include <algorithm>

#include "common.h"

namespace opfuse {

namespace {

constexpr int kStreamUnroll = 8;
typedef float v4f __attribute__((ext_vector_type(4)));  // a native vector: non-temporal builtins take it

template <int U>
__global__ __launch_bounds__(256) void stream_read_kernel(const v4f* __restrict__ src,
                                                          int64_t n4, float* __restrict__ sink) {
  const int64_t stride = (int64_t)gridDim.x * 256 * U;
  float acc = 0.f;
  int64_t i = (int64_t)blockIdx.x * 256 * U + threadIdx.x;
  for (; i + (U - 1) * 256 < n4; i += stride) {
    v4f v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(src + i + u * 256);
#pragma unroll
    for (int u = 0; u < U; ++u) acc += (v[u].x + v[u].y) + (v[u].z + v[u].w);
  }
  for (int u = 0; u < U; ++u) {
    const int64_t j = i + u * 256;
    if (j < n4) {
      const v4f t = src[j];
      acc += (t.x + t.y) + (t.z + t.w);
    }
  }
  // The sum is stored only if it equals a value it practically never takes;
  // the branch keeps the loads live without a store per thread.
  if (acc == 1.2345678e-30f) sink[0] = acc;
}

template <int U>
__global__ __launch_bounds__(256) void stream_copy_kernel(const v4f* __restrict__ src,
                                                          v4f* __restrict__ dst, int64_t n4) {
  const int64_t stride = (int64_t)gridDim.x * 256 * U;
  int64_t i = (int64_t)blockIdx.x * 256 * U + threadIdx.x;
  for (; i + (U - 1) * 256 < n4; i += stride) {
    v4f v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(src + i + u * 256);
#pragma unroll
    for (int u = 0; u < U; ++u) __builtin_nontemporal_store(v[u], dst + i + u * 256);
  }
  for (int u = 0; u < U; ++u) {
    const int64_t j = i + u * 256;
    if (j < n4) dst[j] = src[j];
  }
}

// In place: every element read, incremented and written back.
template <int U>
__global__ __launch_bounds__(256) void stream_rmw_kernel(v4f* __restrict__ dst, int64_t n4) {
  const int64_t stride = (int64_t)gridDim.x * 256 * U;
  int64_t i = (int64_t)blockIdx.x * 256 * U + threadIdx.x;
  for (; i + (U - 1) * 256 < n4; i += stride) {
    v4f v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(dst + i + u * 256);
#pragma unroll
    for (int u = 0; u < U; ++u) __builtin_nontemporal_store(v[u] + 1.f, dst + i + u * 256);
  }
  for (int u = 0; u < U; ++u) {
    const int64_t j = i + u * 256;
    if (j < n4) dst[j] = dst[j] + 1.f;
  }
}

// Three arrays of n3 float4s in place, element i of all three in the same
// pass (the pattern of an update that reads W, m and v and writes them back).
template <int U>
__global__ __launch_bounds__(256) void stream_rmw3_kernel(v4f* __restrict__ a, int64_t n3) {
  v4f* __restrict__ b = a + n3;
  v4f* __restrict__ c = b + n3;
  const int64_t stride = (int64_t)gridDim.x * 256 * U;
  int64_t i = (int64_t)blockIdx.x * 256 * U + threadIdx.x;
  for (; i + (U - 1) * 256 < n3; i += stride) {
    v4f va[U], vb[U], vc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      va[u] = __builtin_nontemporal_load(a + i + u * 256);
      vb[u] = __builtin_nontemporal_load(b + i + u * 256);
      vc[u] = __builtin_nontemporal_load(c + i + u * 256);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      __builtin_nontemporal_store(va[u] + 1.f, a + i + u * 256);
      __builtin_nontemporal_store(vb[u] + 1.f, b + i + u * 256);
      __builtin_nontemporal_store(vc[u] + 1.f, c + i + u * 256);
    }
  }
  for (int u = 0; u < U; ++u) {
    const int64_t j = i + u * 256;
    if (j < n3) {
      a[j] = a[j] + 1.f;
      b[j] = b[j] + 1.f;
      c[j] = c[j] + 1.f;
    }
  }
}

}  // namespace

// Three arrays of rows of kColRow floats, read and written in 4-byte accesses
// in the layout of a 32 x 32 fp32 MFMA accumulator: a workgroup owns 128
// columns (4 wavefronts x 32) of a range of rows, walked in chunks of 32 rows;
// a lane holds its column at rows 8 j + 4 h + e (j, e < 4; h: the wavefront
// half).  This is how the merged backward kernel moves W, m and v, so its rate
// is that kernel's streaming ceiling.
constexpr int kColRow = 8192;

__device__ __forceinline__ int col_acc_row(int i, int h) { return (i >> 2) * 8 + h * 4 + (i & 3); }

__global__ __launch_bounds__(256) void stream_rmw3_columns_kernel(float* __restrict__ a,
                                                                  int64_t rows, int nr) {
  float* __restrict__ b = a + rows * kColRow;
  float* __restrict__ c = b + rows * kColRow;
  const int lane = threadIdx.x & 63, h = lane >> 5;
  const int64_t col = (int64_t)blockIdx.x * 128 + (threadIdx.x >> 6) * 32 + (lane & 31);
  const int64_t r0 = (int64_t)blockIdx.y * nr;
  const int64_t r1 = r0 + nr < rows ? r0 + nr : rows;
  for (int64_t n0 = r0; n0 < r1; n0 += 32) {   // rows is a multiple of 32
    float va[16], vb[16], vc[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int64_t o = (n0 + col_acc_row(i, h)) * kColRow + col;
      va[i] = a[o]; vb[i] = b[o]; vc[i] = c[o];
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int64_t o = (n0 + col_acc_row(i, h)) * kColRow + col;
      a[o] = va[i] + 1.f; b[o] = vb[i] + 1.f; c[o] = vc[i] + 1.f;
    }
  }
}

hipError_t hbm_stream_launch(int mode, const float* src, float* dst, int64_t n, int blocks,
                             hipStream_t stream) {
  if (mode == 4) {
    // the merged kernel's grid: 64 column strips x up to 8 row ranges
    const int64_t rows = n / 3 / kColRow;
    const int64_t chunks = rows / 32;
    const int ranges = (int)std::min<int64_t>(8, chunks);
    const int nr = (int)((chunks + ranges - 1) / ranges) * 32;
    hipLaunchKernelGGL(stream_rmw3_columns_kernel, dim3(kColRow / 128, ranges), dim3(256), 0,
                       stream, dst, rows, nr);
    return hipGetLastError();
  }
  const int64_t n4 = n / 4;
  if (blocks <= 0) blocks = 2048;  // 8 workgroups per compute unit
  if (mode == 0)
    hipLaunchKernelGGL(stream_read_kernel<kStreamUnroll>, dim3(blocks), dim3(256), 0, stream,
                       reinterpret_cast<const v4f*>(src), n4, dst);
  else if (mode == 2)
    hipLaunchKernelGGL(stream_rmw_kernel<kStreamUnroll>, dim3(blocks), dim3(256), 0, stream,
                       reinterpret_cast<v4f*>(dst), n4);
  else if (mode == 3)
    hipLaunchKernelGGL(stream_rmw3_kernel<kStreamUnroll / 2>, dim3(blocks), dim3(256), 0, stream,
                       reinterpret_cast<v4f*>(dst), n4 / 3);
  else
    hipLaunchKernelGGL(stream_copy_kernel<kStreamUnroll>, dim3(blocks), dim3(256), 0, stream,
                       reinterpret_cast<const v4f*>(src), reinterpret_cast<v4f*>(dst), n4);
  return hipGetLastError();
}

}  // namespace opfuse
