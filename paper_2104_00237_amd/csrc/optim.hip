// Element-wise optimizer kernels.
//
// multi_update: the eager third stage (Fig. 1(b)) -- one launch updates many
// tensors, each workgroup taking one 4096-element chunk of one tensor, with
// 128-bit loads of w, g, m, v and stores of w, m, v (read and reset of the
// gradient by the optimizer, Section 3 "Baseline").  It also serves the
// element-wise fused update of a single tensor (bias / norm parameters, and
// the forward-fusion flush).
//
// rows_update: the gradient is given as rows to be summed (per-row partial
// gradients); each thread owns one element, sums its column over the rows in
// row order and applies the update, so the gradient vector is never stored.

#include <algorithm>

#include "common.h"

namespace opfuse {

constexpr int MT_MAX = 48;
constexpr int MT_CHUNK = 4096;  // elements per workgroup: 256 threads x 4 x 4

struct MTEntry {
  of_param p;
  const float* g;
  int64_t chunk0;  // first chunk index of this tensor
  int vec;         // 128-bit paths allowed
};

struct MTArgs {
  int n;
  MTEntry e[MT_MAX];
};

__global__ __launch_bounds__(256) void multi_update_kernel(MTArgs a, OptK o) {
  opt_prepare(o);
  const int64_t chunk = blockIdx.x;
  int t = 0;
  while (t + 1 < a.n && a.e[t + 1].chunk0 <= chunk) ++t;
  const MTEntry& E = a.e[t];
  const int64_t base = (chunk - E.chunk0) * MT_CHUNK;
  const int64_t numel = E.p.numel;
  if (E.vec) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t i = base + ((int64_t)u * 256 + threadIdx.x) * 4;
      if (i + 3 < numel) {
        update4(o, E.p, ld4(E.g + i), i);
      } else {
        for (int64_t k = i; k < numel && k < i + 4; ++k) update1(o, E.p, E.g[k], k);
      }
    }
  } else {
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int64_t i = base + (int64_t)u * 256 + threadIdx.x;
      if (i < numel) update1(o, E.p, E.g[i], i);
    }
  }
}

hipError_t launch_multi_update(int n, const of_param* params, const float* const* grads,
                               const OptK& o, hipStream_t stream) {
  for (int s = 0; s < n; s += MT_MAX) {
    MTArgs a;
    a.n = std::min(MT_MAX, n - s);
    int64_t chunks = 0;
    for (int i = 0; i < a.n; ++i) {
      const of_param& p = params[s + i];
      MTEntry& E = a.e[i];
      E.p = p;
      E.g = grads[s + i];
      E.chunk0 = chunks;
      E.vec = aligned16(p.w) && aligned16(p.m) && aligned16(E.g) &&
              (o.kind == OF_OPT_SGD || aligned16(p.v)) &&
              (p.w_bf16 == nullptr || ((uintptr_t)p.w_bf16 & 7u) == 0);
      chunks += (p.numel + MT_CHUNK - 1) / MT_CHUNK;
    }
    hipLaunchKernelGGL(multi_update_kernel, dim3((unsigned)chunks), dim3(256), 0, stream, a, o);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

__global__ __launch_bounds__(256) void rows_update_kernel(of_param p, const float* __restrict__ g,
                                                          int64_t rows, int64_t ld, OptK o) {
  opt_prepare(o);
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= p.numel) return;
  // The optimizer state is loaded before the row sum, and the loads of 32
  // rows are issued before their (in-order) accumulation: the kernel is a
  // chain of load round trips, as few as possible.
  const OptState1 st = opt_load1(o, p, i);
  float s = g[i];
  for (int64_t r0 = 1; r0 < rows; r0 += 32) {
    float v[32];
#pragma unroll
    for (int k = 0; k < 32; ++k) v[k] = r0 + k < rows ? g[(r0 + k) * ld + i] : 0.f;
#pragma unroll
    for (int k = 0; k < 32; ++k)
      if (r0 + k < rows) s = __fadd_rn(s, v[k]);
  }
  opt_apply1(o, p, st, s, i);
}

hipError_t launch_rows_update(const of_param& p, const float* g, int64_t rows, int64_t ld,
                              const OptK& o, hipStream_t stream) {
  const unsigned blocks = (unsigned)((p.numel + 255) / 256);
  hipLaunchKernelGGL(rows_update_kernel, dim3(blocks), dim3(256), 0, stream, p, g, rows, ld, o);
  return hipGetLastError();
}

// ------------------------------------------------ global-norm clipping
// Pass 1: workgroup b sums the squares of its grid-stride share of the
// gradients of up to CLIP_MAX tensors in float64, in a fixed order (per-lane
// accumulators, then a fixed tree), and writes (first launch) or adds (later
// launches, stream-ordered) its partial.  A row-partial gradient's element is
// its rows summed in row order in fp32, as the rows-mode update sums them.
// Pass 2: one workgroup sums the CLIP_WG partials with a fixed tree and
// writes the factor (and the norm).

constexpr int CLIP_MAX = 32;
constexpr int CLIP_WG = OF_CLIP_WS_BYTES / 8;   // partials, one per workgroup
static_assert(CLIP_WG == 256, "one partial per workgroup of the sum pass");

struct ClipEntry {
  const float* g;
  int64_t numel, rows, ld;
  int vec;   // a 16-byte aligned vector gradient
};

struct ClipArgs {
  int n, accumulate;
  ClipEntry e[CLIP_MAX];
};

__device__ __forceinline__ double wg_sum256(double x, double* red) {
  const int tid = threadIdx.x;
  red[tid] = x;
  __syncthreads();
#pragma unroll
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) red[tid] = red[tid] + red[tid + w];
    __syncthreads();
  }
  return red[0];
}

__global__ __launch_bounds__(256) void grad_sumsq_kernel(ClipArgs a, double* __restrict__ partial) {
  __shared__ double red[256];
  const int64_t lane = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * 256;
  double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
  for (int t = 0; t < a.n; ++t) {
    const ClipEntry& E = a.e[t];
    if (E.rows == 1 && E.vec) {
      for (int64_t i = lane * 4; i < E.numel; i += stride * 4) {
        if (i + 3 < E.numel) {
          const float4 v = ld4(E.g + i);
          s0 += (double)v.x * (double)v.x;
          s1 += (double)v.y * (double)v.y;
          s2 += (double)v.z * (double)v.z;
          s3 += (double)v.w * (double)v.w;
        } else {
          for (int64_t k = i; k < E.numel; ++k) s0 += (double)E.g[k] * (double)E.g[k];
        }
      }
    } else if (E.rows == 1) {
      for (int64_t i = lane; i < E.numel; i += stride) s0 += (double)E.g[i] * (double)E.g[i];
    } else {
      for (int64_t i = lane; i < E.numel; i += stride) {
        float x = E.g[i];
        for (int64_t r = 1; r < E.rows; ++r) x = __fadd_rn(x, E.g[r * E.ld + i]);
        s0 += (double)x * (double)x;
      }
    }
  }
  const double tot = wg_sum256((s0 + s1) + (s2 + s3), red);
  if (threadIdx.x == 0) partial[blockIdx.x] = a.accumulate ? partial[blockIdx.x] + tot : tot;
}

__global__ __launch_bounds__(256) void clip_finish_kernel(const double* __restrict__ partial,
                                                          float max_norm, float* scale,
                                                          float* norm) {
  __shared__ double red[256];
  const double tot = wg_sum256(partial[threadIdx.x], red);
  if (threadIdx.x == 0) {
    const double nrm = sqrt(tot);
    const double f = (double)max_norm / (nrm + 1e-6);
    scale[0] = (float)(f > 1.0 ? 1.0 : f);   // NaN stays NaN
    if (norm) norm[0] = (float)nrm;
  }
}

hipError_t launch_grad_clip(int n, const of_grad_ref* grads, float max_norm, float* scale,
                            float* norm, double* partial, hipStream_t stream) {
  for (int b = 0; b < n; b += CLIP_MAX) {
    ClipArgs a;
    a.n = std::min(CLIP_MAX, n - b);
    a.accumulate = b > 0;
    for (int i = 0; i < a.n; ++i) {
      const of_grad_ref& g = grads[b + i];
      ClipEntry& E = a.e[i];
      E.g = g.g;
      E.numel = g.numel;
      E.rows = g.rows;
      E.ld = g.ld ? g.ld : g.numel;
      E.vec = g.rows == 1 && aligned16(g.g);
    }
    hipLaunchKernelGGL(grad_sumsq_kernel, dim3(CLIP_WG), dim3(256), 0, stream, a, partial);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(clip_finish_kernel, dim3(1), dim3(256), 0, stream, partial, max_norm, scale,
                     norm);
  return hipGetLastError();
}

__global__ void step_advance_kernel(int64_t* step, int64_t delta) {
  if (threadIdx.x == 0) *step += delta;
}

hipError_t launch_step_advance(int64_t* step_dev, int64_t delta, hipStream_t stream) {
  hipLaunchKernelGGL(step_advance_kernel, dim3(1), dim3(64), 0, stream, step_dev, delta);
  return hipGetLastError();
}

}  // namespace opfuse
