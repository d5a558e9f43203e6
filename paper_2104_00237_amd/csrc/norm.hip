// LayerNorm over the last dimension (biased variance, eps inside the square
// root), its backward, and two small element-wise helpers (sum of rows, add).
//
// Forward: one wavefront per row; mean, then the variance of the centred
// values, then y = (x - mean) * rstd * gamma + beta; mean and rstd are kept
// for the backward.  y is stored as fp32, or (yb) as its bf16 rounding (round
// to nearest even) when only a bf16-operand contraction reads it: the same
// value the contraction would round it to, in half the bytes.
// Backward, per row: with xh = (x - mean) * rstd and g = dy * gamma,
//   dx = rstd * (g - mean(g) - xh * mean(g * xh))  (+ the residual gradient);
// the parameter gradients sum dy * xh and dy over the rows.  They are written
// as per-row-group partials [G, D], which the element-wise fused update sums
// in group order while it applies the optimizer, so the gradient vector of
// gamma and beta is never stored (or of_reduce_rows materialises it).

#include <algorithm>
#include <initializer_list>

#include "common.h"

namespace opfuse {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = __fadd_rn(v, __shfl_xor(v, o, 64));
  return v;
}

__global__ __launch_bounds__(256) void ln_fwd_kernel(const float* __restrict__ x, int64_t M,
                                                     int64_t D, const float* __restrict__ gamma,
                                                     const float* __restrict__ beta, float eps,
                                                     float* __restrict__ y,
                                                     uint16_t* __restrict__ yb,
                                                     float* __restrict__ mean,
                                                     float* __restrict__ rstd) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const float* xr = x + row * D;
  float s = 0.f;
  for (int64_t j = lane; j < D; j += 64) s = __fadd_rn(s, xr[j]);
  const float mu = __fdiv_rn(wave_sum(s), (float)D);
  float q = 0.f;
  for (int64_t j = lane; j < D; j += 64) {
    const float d = __fsub_rn(xr[j], mu);
    q = __fmaf_rn(d, d, q);
  }
  const float var = __fdiv_rn(wave_sum(q), (float)D);
  const float rs = __fdiv_rn(1.f, __fsqrt_rn(__fadd_rn(var, eps)));
  for (int64_t j = lane; j < D; j += 64) {
    const float o = __fmaf_rn(__fmul_rn(__fsub_rn(xr[j], mu), rs), gamma[j], beta[j]);
    if (yb) yb[row * D + j] = f32_to_bf16(o);
    else y[row * D + j] = o;
  }
  if (lane == 0) {
    mean[row] = mu;
    rstd[row] = rs;
  }
}

__global__ __launch_bounds__(256) void ln_bwd_dx_kernel(
    const float* __restrict__ dy, const float* __restrict__ x, const float* __restrict__ mean,
    const float* __restrict__ rstd, const float* __restrict__ gamma, const float* __restrict__ dres,
    int64_t M, int64_t D, float* __restrict__ dx) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const float* xr = x + row * D;
  const float* dr = dy + row * D;
  const float mu = mean[row], rs = rstd[row];
  float s1 = 0.f, s2 = 0.f;
  for (int64_t j = lane; j < D; j += 64) {
    const float xh = __fmul_rn(__fsub_rn(xr[j], mu), rs);
    const float g = __fmul_rn(dr[j], gamma[j]);
    s1 = __fadd_rn(s1, g);
    s2 = __fmaf_rn(g, xh, s2);
  }
  const float c1 = __fdiv_rn(wave_sum(s1), (float)D);
  const float c2 = __fdiv_rn(wave_sum(s2), (float)D);
  float* o = dx + row * D;
  const float* rr = dres ? dres + row * D : nullptr;
  for (int64_t j = lane; j < D; j += 64) {
    const float xh = __fmul_rn(__fsub_rn(xr[j], mu), rs);
    const float g = __fmul_rn(dr[j], gamma[j]);
    float v = __fmul_rn(rs, __fsub_rn(__fsub_rn(g, c1), __fmul_rn(xh, c2)));
    if (rr) v = __fadd_rn(rr[j], v);
    o[j] = v;
  }
}

// Parameter-gradient partials: workgroup (column block, row group) sums its
// rows in order for 256 columns.
__global__ __launch_bounds__(256) void ln_bwd_param_kernel(
    const float* __restrict__ dy, const float* __restrict__ x, const float* __restrict__ mean,
    const float* __restrict__ rstd, int64_t M, int64_t D, int64_t rows_per_group,
    float* __restrict__ dgamma_rows, float* __restrict__ dbeta_rows) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t grp = blockIdx.y;
  if (j >= D) return;
  const int64_t r0 = grp * rows_per_group, r1 = std::min(M, r0 + rows_per_group);
  float sg = 0.f, sb = 0.f;
  // loads of 16 rows are issued before their (in-order) accumulation; the
  // row statistics are the same for every lane
  for (int64_t rb = r0; rb < r1; rb += 16) {
    float d[16], xv[16], mu[16], rs[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int64_t r = rb + k;
      const bool ok = r < r1;
      d[k] = ok ? dy[r * D + j] : 0.f;
      xv[k] = ok ? x[r * D + j] : 0.f;
      mu[k] = ok ? mean[r] : 0.f;
      rs[k] = ok ? rstd[r] : 0.f;
    }
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      if (rb + k < r1) {
        const float xh = __fmul_rn(__fsub_rn(xv[k], mu[k]), rs[k]);
        sg = __fmaf_rn(d[k], xh, sg);
        sb = __fadd_rn(sb, d[k]);
      }
    }
  }
  dgamma_rows[grp * D + j] = sg;
  dbeta_rows[grp * D + j] = sb;
}

// Row held in registers: lane j owns the float4 columns 4*(j + 64*c), c < NPL
// (D a multiple of 4, D <= 256*NPL, 16-byte aligned rows).  Same arithmetic
// as the scalar kernels above in a different summation order.
template <int NPL>
__global__ __launch_bounds__(256) void ln_fwd_vec_kernel(const float* __restrict__ x, int64_t M,
                                                         int64_t D, const float* __restrict__ gamma,
                                                         const float* __restrict__ beta, float eps,
                                                         float* __restrict__ y,
                                                         uint16_t* __restrict__ yb,
                                                         float* __restrict__ mean,
                                                         float* __restrict__ rstd) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const float* xr = x + row * D;
  float4 v[NPL];
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < NPL; ++c) {
    const int64_t j = 4 * (lane + 64 * c);
    v[c] = j < D ? ld4(xr + j) : make_float4(0.f, 0.f, 0.f, 0.f);
    s = __fadd_rn(s, __fadd_rn(__fadd_rn(v[c].x, v[c].y), __fadd_rn(v[c].z, v[c].w)));
  }
  const float mu = __fdiv_rn(wave_sum(s), (float)D);
  float q = 0.f;
#pragma unroll
  for (int c = 0; c < NPL; ++c) {
    const int64_t j = 4 * (lane + 64 * c);
    if (j < D) {
      const float a = __fsub_rn(v[c].x, mu), b = __fsub_rn(v[c].y, mu);
      const float e = __fsub_rn(v[c].z, mu), f = __fsub_rn(v[c].w, mu);
      q = __fmaf_rn(a, a, q); q = __fmaf_rn(b, b, q);
      q = __fmaf_rn(e, e, q); q = __fmaf_rn(f, f, q);
    }
  }
  const float var = __fdiv_rn(wave_sum(q), (float)D);
  const float rs = __fdiv_rn(1.f, __fsqrt_rn(__fadd_rn(var, eps)));
#pragma unroll
  for (int c = 0; c < NPL; ++c) {
    const int64_t j = 4 * (lane + 64 * c);
    if (j < D) {
      const float4 g = ld4(gamma + j), b = ld4(beta + j);
      const float4 o = make_float4(__fmaf_rn(__fmul_rn(__fsub_rn(v[c].x, mu), rs), g.x, b.x),
                                   __fmaf_rn(__fmul_rn(__fsub_rn(v[c].y, mu), rs), g.y, b.y),
                                   __fmaf_rn(__fmul_rn(__fsub_rn(v[c].z, mu), rs), g.z, b.z),
                                   __fmaf_rn(__fmul_rn(__fsub_rn(v[c].w, mu), rs), g.w, b.w));
      if (yb) st_bf16x4(yb + row * D + j, o);
      else st4(y + row * D + j, o);
    }
  }
  if (lane == 0) {
    mean[row] = mu;
    rstd[row] = rs;
  }
}

template <int NPL>
__global__ __launch_bounds__(256) void ln_bwd_dx_vec_kernel(
    const float* __restrict__ dy, const float* __restrict__ x, const float* __restrict__ mean,
    const float* __restrict__ rstd, const float* __restrict__ gamma, const float* __restrict__ dres,
    int64_t M, int64_t D, float* __restrict__ dx) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const float mu = mean[row], rs = rstd[row];
  float xh[NPL][4], g[NPL][4];
  float4 rv[NPL];   // the residual gradient, loaded before the row sums
#pragma unroll
  for (int c = 0; c < NPL; ++c) {
    const int64_t j = 4 * (lane + 64 * c);
    rv[c] = dres && j < D ? ld4(dres + row * D + j) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int c = 0; c < NPL; ++c) {
    const int64_t j = 4 * (lane + 64 * c);
    const float4 xv = j < D ? ld4(x + row * D + j) : make_float4(0.f, 0.f, 0.f, 0.f);
    const float4 dv = j < D ? ld4(dy + row * D + j) : make_float4(0.f, 0.f, 0.f, 0.f);
    const float4 gm = j < D ? ld4(gamma + j) : make_float4(0.f, 0.f, 0.f, 0.f);
    const float xa[4] = {xv.x, xv.y, xv.z, xv.w}, da[4] = {dv.x, dv.y, dv.z, dv.w};
    const float ga[4] = {gm.x, gm.y, gm.z, gm.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      xh[c][e] = __fmul_rn(__fsub_rn(xa[e], mu), rs);
      g[c][e] = __fmul_rn(da[e], ga[e]);
      s1 = __fadd_rn(s1, g[c][e]);
      s2 = __fmaf_rn(g[c][e], xh[c][e], s2);
    }
  }
  const float c1 = __fdiv_rn(wave_sum(s1), (float)D);
  const float c2 = __fdiv_rn(wave_sum(s2), (float)D);
#pragma unroll
  for (int c = 0; c < NPL; ++c) {
    const int64_t j = 4 * (lane + 64 * c);
    if (j < D) {
      float o[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        o[e] = __fmul_rn(rs, __fsub_rn(__fsub_rn(g[c][e], c1), __fmul_rn(xh[c][e], c2)));
      if (dres) {
        const float4 r = rv[c];
        o[0] = __fadd_rn(r.x, o[0]); o[1] = __fadd_rn(r.y, o[1]);
        o[2] = __fadd_rn(r.z, o[2]); o[3] = __fadd_rn(r.w, o[3]);
      }
      st4(dx + row * D + j, make_float4(o[0], o[1], o[2], o[3]));
    }
  }
}

int64_t ln_partial_rows(int64_t M) { return std::min<int64_t>(64, std::max<int64_t>(1, (M + 63) / 64)); }

// Register-resident variant: D a multiple of 4, at most 2048, 16-byte aligned.
static int ln_npl(int64_t D, std::initializer_list<const void*> ptrs) {
  if (D % 4 != 0 || D > 2048) return 0;
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return 0;
  return D <= 256 ? 1 : D <= 512 ? 2 : D <= 1024 ? 4 : 8;
}

hipError_t launch_ln_fwd(const float* x, int64_t M, int64_t D, const float* gamma,
                         const float* beta, float eps, float* y, uint16_t* yb, float* mean,
                         float* rstd, hipStream_t s) {
  const dim3 g((unsigned)((M + 3) / 4));
  // a bf16 row of D (a multiple of 4) elements is stored 4 at a time: 8-byte aligned base
  const int npl = (yb && ((uintptr_t)yb & 7u)) ? 0 : ln_npl(D, {x, gamma, beta, y});
  switch (npl) {
    case 1: hipLaunchKernelGGL(ln_fwd_vec_kernel<1>, g, dim3(256), 0, s, x, M, D, gamma, beta, eps, y, yb, mean, rstd); return hipGetLastError();
    case 2: hipLaunchKernelGGL(ln_fwd_vec_kernel<2>, g, dim3(256), 0, s, x, M, D, gamma, beta, eps, y, yb, mean, rstd); return hipGetLastError();
    case 4: hipLaunchKernelGGL(ln_fwd_vec_kernel<4>, g, dim3(256), 0, s, x, M, D, gamma, beta, eps, y, yb, mean, rstd); return hipGetLastError();
    case 8: hipLaunchKernelGGL(ln_fwd_vec_kernel<8>, g, dim3(256), 0, s, x, M, D, gamma, beta, eps, y, yb, mean, rstd); return hipGetLastError();
    default: break;
  }
  hipLaunchKernelGGL(ln_fwd_kernel, dim3((unsigned)((M + 3) / 4)), dim3(256), 0, s, x, M, D, gamma,
                     beta, eps, y, yb, mean, rstd);
  return hipGetLastError();
}

hipError_t launch_ln_bwd(const float* dy, const float* x, const float* mean, const float* rstd,
                         const float* gamma, const float* dres, int64_t M, int64_t D, float* dx,
                         float* dgamma_rows, float* dbeta_rows, hipStream_t s) {
  if (dx) {
    const dim3 g((unsigned)((M + 3) / 4));
    switch (ln_npl(D, {dy, x, gamma, dres, dx})) {
      case 1: hipLaunchKernelGGL(ln_bwd_dx_vec_kernel<1>, g, dim3(256), 0, s, dy, x, mean, rstd, gamma, dres, M, D, dx); break;
      case 2: hipLaunchKernelGGL(ln_bwd_dx_vec_kernel<2>, g, dim3(256), 0, s, dy, x, mean, rstd, gamma, dres, M, D, dx); break;
      case 4: hipLaunchKernelGGL(ln_bwd_dx_vec_kernel<4>, g, dim3(256), 0, s, dy, x, mean, rstd, gamma, dres, M, D, dx); break;
      case 8: hipLaunchKernelGGL(ln_bwd_dx_vec_kernel<8>, g, dim3(256), 0, s, dy, x, mean, rstd, gamma, dres, M, D, dx); break;
      default:
        hipLaunchKernelGGL(ln_bwd_dx_kernel, g, dim3(256), 0, s, dy, x, mean, rstd, gamma, dres, M, D, dx);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (dgamma_rows) {
    const int64_t G = ln_partial_rows(M);
    const int64_t rpg = (M + G - 1) / G;
    hipLaunchKernelGGL(ln_bwd_param_kernel, dim3((unsigned)((D + 255) / 256), (unsigned)G),
                       dim3(256), 0, s, dy, x, mean, rstd, M, D, rpg, dgamma_rows, dbeta_rows);
    return hipGetLastError();
  }
  return hipSuccess;
}

__global__ __launch_bounds__(256) void reduce_rows_kernel(const float* __restrict__ src,
                                                          int64_t rows, int64_t ld, int64_t n,
                                                          float* __restrict__ dst) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  // loads of 32 rows are issued before their (in-order) accumulation
  float s = src[i];
  for (int64_t r0 = 1; r0 < rows; r0 += 32) {
    float v[32];
#pragma unroll
    for (int k = 0; k < 32; ++k) v[k] = r0 + k < rows ? src[(r0 + k) * ld + i] : 0.f;
#pragma unroll
    for (int k = 0; k < 32; ++k)
      if (r0 + k < rows) s = __fadd_rn(s, v[k]);
  }
  dst[i] = s;
}

hipError_t launch_reduce_rows(const float* src, int64_t rows, int64_t ld, int64_t n, float* dst,
                              hipStream_t s) {
  hipLaunchKernelGGL(reduce_rows_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src,
                     rows, ld, n, dst);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void add_kernel(const float* __restrict__ a,
                                                  const float* __restrict__ b, int64_t n, int vec,
                                                  float* __restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  if (vec) {
    const int64_t n4 = n / 4;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride) {
      const float4 x = ld4(a + 4 * i), y = ld4(b + 4 * i);
      st4(out + 4 * i, make_float4(__fadd_rn(x.x, y.x), __fadd_rn(x.y, y.y), __fadd_rn(x.z, y.z),
                                   __fadd_rn(x.w, y.w)));
    }
    for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride)
      out[i] = __fadd_rn(a[i], b[i]);
  } else {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride)
      out[i] = __fadd_rn(a[i], b[i]);
  }
}

hipError_t launch_add(const float* a, const float* b, int64_t n, float* out, hipStream_t s) {
  const int vec = aligned16(a) && aligned16(b) && aligned16(out);
  const int64_t work = vec ? (n + 3) / 4 : n;
  const unsigned blocks = (unsigned)std::min<int64_t>(4096, std::max<int64_t>(1, (work + 255) / 256));
  hipLaunchKernelGGL(add_kernel, dim3(blocks), dim3(256), 0, s, a, b, n, vec, out);
  return hipGetLastError();
}

}  // namespace opfuse
