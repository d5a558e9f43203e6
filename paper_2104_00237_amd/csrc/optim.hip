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
  // loads of 8 rows are issued before their (in-order) accumulation
  float s = g[i];
  for (int64_t r0 = 1; r0 < rows; r0 += 8) {
    float v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = r0 + k < rows ? g[(r0 + k) * ld + i] : 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if (r0 + k < rows) s = __fadd_rn(s, v[k]);
  }
  update1(o, p, s, i);
}

hipError_t launch_rows_update(const of_param& p, const float* g, int64_t rows, int64_t ld,
                              const OptK& o, hipStream_t stream) {
  const unsigned blocks = (unsigned)((p.numel + 255) / 256);
  hipLaunchKernelGGL(rows_update_kernel, dim3(blocks), dim3(256), 0, stream, p, g, rows, ld, o);
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
