// Depthwise 3x3 convolution (one filter per channel, stride 1 or 2, zero pad 1),
// NHWC activations, filter [3,3,C] (tap-major, channels contiguous), bias [C].
// These layers have few parameters and little arithmetic per byte, so every
// kernel here is bound by HBM traffic, not by the matrix cores: consecutive
// lanes take consecutive channels (coalesced 256-byte wave accesses).  The
// forward, the stride-1 data gradient and the filter gradient walk columns of
// a few rows with the 3x3 window in registers, so a row step loads only the
// new window rows; the stride-2 data gradient (at most four taps per input
// pixel) takes one pixel per thread.
//
// Filter gradient: dW[ky,kx,c] = sum over (n,h,w) of dy[n,h,w,c] *
// x[n,h+ky-1,w+kx-1,c], db[c] = sum of dy[n,h,w,c].  Pass 1 splits the output
// pixels, in units of one column over up to 16 rows, over S slices; each
// workgroup takes CB channels (CB from 16, 32, 48, 64, whichever pads C least;
// one channel per thread group, or CB / 4 channel quads when C % 4 == 0 and
// the tensors are 16-byte aligned) and writes the ten per-channel sums of its
// slice, each the in-order sum of 16 unit streams that both kernels partition
// and order alike.  S is sized so that the grid fills the chip.
// Pass 2 adds the S slices of each sum: L lanes (a power of two up to 64) take
// consecutive runs of slices, each in slice order, and the run sums are added
// in lane order; it then either writes dW / db (eager) or applies the
// optimizer to W, b and their history right there (backward-fusion: the
// filter gradient is never stored; the parameter's state is loaded before the
// slices are summed).  Both passes are deterministic: the two pass-1 kernels
// take the same operations in the same order for every element, so the bits
// do not depend on which one runs (that is, on the pointers' alignment), and
// the fused pass applies the same per-element update as the eager optimizer
// kernel, so eager and fused give the same bits.

#include <algorithm>

#include "common.h"

namespace opfuse {

constexpr int DW_CB_MAX = 64;  // channels per workgroup in pass 1, at most
constexpr int DW_TAPS = 10;    // nine filter taps + the bias sum

// Input [N,H,W,C]; output [N,Ho,Wo,C] with Ho = (H - 1) / S + 1 for the
// stride S (1 or 2, zero padding 1), a template parameter of the kernels.
struct DwShape {
  int N, H, W, C;
  int Ho, Wo;
};

// dx[n,h,w,c] = sum over the taps (ky, kx) with h + 1 - ky = S ho and
// w + 1 - kx = S wo (0 <= ho < Ho, 0 <= wo < Wo) of dy[n,ho,wo,c] * W[ky,kx,c],
// times the previous layer's activation derivative (ReLU: its saved output > 0).
template <int S>
__global__ __launch_bounds__(256) void dw_dgrad_kernel(const float* __restrict__ dy,
                                                       const float* __restrict__ w,
                                                       const float* __restrict__ prev,
                                                       int act_prev, float* __restrict__ dx,
                                                       DwShape s, int total) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const int c = i % s.C, p = i / s.C;
  const int col = p % s.W, t = p / s.W, row = t % s.H, n = t / s.H;
  float acc = 0.f;
#pragma unroll
  for (int ky = 0; ky < 3; ++ky) {
    const int th = row - ky + 1;
    if (th < 0 || th % S) continue;
    const int hh = th / S;
    if (hh >= s.Ho) continue;
#pragma unroll
    for (int kx = 0; kx < 3; ++kx) {
      const int tw = col - kx + 1;
      if (tw < 0 || tw % S) continue;
      const int ww = tw / S;
      if (ww >= s.Wo) continue;
      acc = __fmaf_rn(dy[((n * s.Ho + hh) * s.Wo + ww) * s.C + c], w[(ky * 3 + kx) * s.C + c], acc);
    }
  }
  dx[i] = act_prev == OF_ACT_NONE ? acc : __fmul_rn(acc, act_grad(act_prev, prev[i]));
}

// Pass 1: workgroup (channel block, slice) sums its slice's output pixels for
// cb channels (4 * cb threads).  The pixels are taken in units: one column wo
// of one image over up to DW_SEG consecutive output rows, unit
// u = (n * Wo + wo) * nseg + seg.  A slice's units are split into 16 streams
// (stream j takes the slice's units j, j + 16, j + 32, ... in order) whose sums
// are then added in stream order: the same partition and order as the
// four-channel kernel below, so a shape gives the same bits whichever of the
// two runs.  Thread (channel, sub) keeps the streams sub, sub + 4, sub + 8 and
// sub + 12.  The stream sums meet in LDS, [16][10][cb] floats.
//
// Within a unit the rows are walked top to bottom with the window's three
// input rows of three taps held in registers, so each row step loads only the
// input rows it has not seen yet (one at stride 1, two at stride 2) and the
// output gradient, instead of all nine taps.
constexpr int DW_SEG = 16;

__device__ __forceinline__ float dwv_load(const float* p, float) { return *p; }
__device__ __forceinline__ float4 dwv_load(const float* p, float4) { return ld4(p); }
__device__ __forceinline__ float dwv_fma(float a, float b, float c) { return __fmaf_rn(a, b, c); }
__device__ __forceinline__ float4 dwv_fma(float4 a, float4 b, float4 c) {
  return make_float4(__fmaf_rn(a.x, b.x, c.x), __fmaf_rn(a.y, b.y, c.y), __fmaf_rn(a.z, b.z, c.z),
                     __fmaf_rn(a.w, b.w, c.w));
}
__device__ __forceinline__ float dwv_add(float a, float b) { return __fadd_rn(a, b); }
__device__ __forceinline__ float4 dwv_add(float4 a, float4 b) {
  return make_float4(__fadd_rn(a.x, b.x), __fadd_rn(a.y, b.y), __fadd_rn(a.z, b.z),
                     __fadd_rn(a.w, b.w));
}
__device__ __forceinline__ void dwv_zero(float& v) { v = 0.f; }
__device__ __forceinline__ void dwv_zero(float4& v) { v = make_float4(0.f, 0.f, 0.f, 0.f); }

// Unit u's contribution to the ten sums of channel c (V = float) or of the
// channel quad from c (V = float4).  A tap outside the input (zero padding)
// contributes nothing, as in the forward.
template <int S, class V>
__device__ __forceinline__ void dw_wgrad_unit(const float* __restrict__ dy,
                                              const float* __restrict__ x, const DwShape& s,
                                              int nseg, int u, int c, V (&acc)[DW_TAPS]) {
  const int seg = u % nseg, t = u / nseg, wo = t % s.Wo, n = t / s.Wo;
  const int h0 = seg * DW_SEG, h1 = min(s.Ho, h0 + DW_SEG);
  bool cv[3];
  int wc[3];
#pragma unroll
  for (int kx = 0; kx < 3; ++kx) {
    const int ww = wo * S + kx - 1;
    cv[kx] = ww >= 0 && ww < s.W;
    wc[kx] = cv[kx] ? ww : 0;
  }
  V win[3][3];
  bool rv[3];
  auto load_row = [&](int hh, V (&r)[3], bool& ok) {
    ok = hh >= 0 && hh < s.H;
    const float* base = x + ((int64_t)n * s.H + (ok ? hh : 0)) * s.W * s.C + c;
#pragma unroll
    for (int kx = 0; kx < 3; ++kx) {
      if (ok && cv[kx]) r[kx] = dwv_load(base + (int64_t)wc[kx] * s.C, V{});
      else dwv_zero(r[kx]);
    }
  };
  load_row(h0 * S - 1, win[0], rv[0]);
  load_row(h0 * S, win[1], rv[1]);
  load_row(h0 * S + 1, win[2], rv[2]);
  for (int ho = h0; ho < h1; ++ho) {
    if (ho > h0) {
      if (S == 1) {
#pragma unroll
        for (int kx = 0; kx < 3; ++kx) {
          win[0][kx] = win[1][kx];
          win[1][kx] = win[2][kx];
        }
        rv[0] = rv[1];
        rv[1] = rv[2];
        load_row(ho + 1, win[2], rv[2]);
      } else {
#pragma unroll
        for (int kx = 0; kx < 3; ++kx) win[0][kx] = win[2][kx];
        rv[0] = rv[2];
        load_row(2 * ho, win[1], rv[1]);
        load_row(2 * ho + 1, win[2], rv[2]);
      }
    }
    const V g = dwv_load(dy + (((int64_t)n * s.Ho + ho) * s.Wo + wo) * s.C + c, V{});
#pragma unroll
    for (int ky = 0; ky < 3; ++ky)
#pragma unroll
      for (int kx = 0; kx < 3; ++kx)
        if (rv[ky] && cv[kx]) acc[ky * 3 + kx] = dwv_fma(g, win[ky][kx], acc[ky * 3 + kx]);
    acc[9] = dwv_add(acc[9], g);
  }
}

// The 16 stream sums of each of the 10 * cb outputs, added in stream order.
__device__ __forceinline__ void dw_slice_sums(const float* red, int cb, int c0, int C,
                                              float* __restrict__ part_row) {
  for (int j = threadIdx.x; j < DW_TAPS * cb; j += blockDim.x) {
    const int k = j / cb, l = j % cb;
    float v = red[k * cb + l];
#pragma unroll
    for (int u = 1; u < 16; ++u) v = __fadd_rn(v, red[(u * DW_TAPS + k) * cb + l]);
    if (c0 + l < C) part_row[(int64_t)k * C + c0 + l] = v;
  }
}

template <int S>
__global__ __launch_bounds__(256) void dw_wgrad_partial_kernel(const float* __restrict__ dy,
                                                               const float* __restrict__ x,
                                                               float* __restrict__ part,
                                                               DwShape s, int per_slice, int cb,
                                                               int nseg) {
  extern __shared__ float red[];   // [16][DW_TAPS][cb]
  const int cl = threadIdx.x % cb, sub = threadIdx.x / cb;
  const int c = blockIdx.x * cb + cl;
  const int U = s.N * s.Wo * nseg;  // units
  const int u0 = blockIdx.y * per_slice, u1 = min(U, u0 + per_slice);
  float acc[4][DW_TAPS];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int k = 0; k < DW_TAPS; ++k) acc[j][k] = 0.f;
  if (c < s.C) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      for (int u = u0 + sub + 4 * j; u < u1; u += 16)
        dw_wgrad_unit<S, float>(dy, x, s, nseg, u, c, acc[j]);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int k = 0; k < DW_TAPS; ++k) red[((sub + 4 * j) * DW_TAPS + k) * cb + cl] = acc[j][k];
  __syncthreads();
  dw_slice_sums(red, cb, blockIdx.x * cb, s.C, part + (int64_t)blockIdx.y * DW_TAPS * s.C);
}

// ---- four-channel variants (C % 4 == 0, 16-byte aligned tensors): one thread
// per channel quad, 128-bit loads and stores; every element takes the same
// arithmetic, in the same order, as in the one-channel kernels above.
__device__ __forceinline__ float4 fma4(float4 a, float4 b, float4 c) {
  return make_float4(__fmaf_rn(a.x, b.x, c.x), __fmaf_rn(a.y, b.y, c.y), __fmaf_rn(a.z, b.z, c.z),
                     __fmaf_rn(a.w, b.w, c.w));
}

template <int S>
__global__ __launch_bounds__(256) void dw_dgrad4_kernel(const float* __restrict__ dy,
                                                        const float* __restrict__ w,
                                                        const float* __restrict__ prev,
                                                        int act_prev, float* __restrict__ dx,
                                                        DwShape s, int quads) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= quads) return;
  const int Cq = s.C >> 2;
  const int c = (i % Cq) * 4, p = i / Cq;
  const int col = p % s.W, t = p / s.W, row = t % s.H, n = t / s.H;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int ky = 0; ky < 3; ++ky) {
    const int th = row - ky + 1;
    if (th < 0 || th % S) continue;
    const int hh = th / S;
    if (hh >= s.Ho) continue;
#pragma unroll
    for (int kx = 0; kx < 3; ++kx) {
      const int tw = col - kx + 1;
      if (tw < 0 || tw % S) continue;
      const int ww = tw / S;
      if (ww >= s.Wo) continue;
      acc = fma4(ld4(dy + ((n * s.Ho + hh) * s.Wo + ww) * s.C + c), ld4(w + (ky * 3 + kx) * s.C + c), acc);
    }
  }
  if (act_prev != OF_ACT_NONE) {
    const float4 pv = ld4(prev + (int64_t)i * 4);
    acc = make_float4(__fmul_rn(acc.x, act_grad(act_prev, pv.x)), __fmul_rn(acc.y, act_grad(act_prev, pv.y)),
                      __fmul_rn(acc.z, act_grad(act_prev, pv.z)), __fmul_rn(acc.w, act_grad(act_prev, pv.w)));
  }
  st4(dx + (int64_t)i * 4, acc);
}

// Pass 1, four channels per thread: cb / 4 channel quads x 16 unit streams
// per workgroup.
template <int S>
__global__ __launch_bounds__(256) void dw_wgrad_partial4_kernel(const float* __restrict__ dy,
                                                                const float* __restrict__ x,
                                                                float* __restrict__ part,
                                                                DwShape s, int per_slice, int cb,
                                                                int nseg) {
  extern __shared__ float red[];   // [16][DW_TAPS][cb]
  const int nq = cb / 4;
  const int q = threadIdx.x % nq, sub = threadIdx.x / nq;
  const int c = blockIdx.x * cb + q * 4;
  const int U = s.N * s.Wo * nseg;  // units
  const int u0 = blockIdx.y * per_slice, u1 = min(U, u0 + per_slice);
  float4 acc[DW_TAPS];
#pragma unroll
  for (int k = 0; k < DW_TAPS; ++k) acc[k] = make_float4(0.f, 0.f, 0.f, 0.f);
  if (c < s.C) {
    for (int u = u0 + sub; u < u1; u += 16) dw_wgrad_unit<S, float4>(dy, x, s, nseg, u, c, acc);
  }
#pragma unroll
  for (int k = 0; k < DW_TAPS; ++k) {
    float* r = red + (sub * DW_TAPS + k) * cb + q * 4;
    r[0] = acc[k].x;
    r[1] = acc[k].y;
    r[2] = acc[k].z;
    r[3] = acc[k].w;
  }
  __syncthreads();
  dw_slice_sums(red, cb, blockIdx.x * cb, s.C, part + (int64_t)blockIdx.y * DW_TAPS * s.C);
}

// ---- column sweeps for the forward (strides 1 and 2) and the stride-1 data
// gradient: one thread per unit (a column of one image over a few rows of the
// output it writes) and channel (V = float) or channel quad (V = float4).  The filter is read once per unit and the window's three rows of
// three taps stay in registers, so each output row loads only the rows it has
// not seen (one, or two for the stride-2 forward) instead of nine taps.
// Each output sums its in-range taps in (ky, kx) order, then adds the bias
// (forward) or applies the previous layer's activation derivative (data
// gradient), the same operations as the per-pixel stride-2 data gradient.
__device__ __forceinline__ float dwv_act(int act, float z) { return act_fwd(act, z); }
__device__ __forceinline__ float4 dwv_act(int act, float4 z) {
  return make_float4(act_fwd(act, z.x), act_fwd(act, z.y), act_fwd(act, z.z), act_fwd(act, z.w));
}
__device__ __forceinline__ float dwv_dact(float acc, int act, const float* p, float) {
  return act == OF_ACT_NONE ? acc : __fmul_rn(acc, act_grad(act, *p));
}
__device__ __forceinline__ float4 dwv_dact(float4 acc, int act, const float* p, float4) {
  if (act == OF_ACT_NONE) return acc;
  const float4 v = ld4(p);
  return make_float4(__fmul_rn(acc.x, act_grad(act, v.x)), __fmul_rn(acc.y, act_grad(act, v.y)),
                     __fmul_rn(acc.z, act_grad(act, v.z)), __fmul_rn(acc.w, act_grad(act, v.w)));
}
__device__ __forceinline__ void dwv_store(float* p, float v) { *p = v; }
__device__ __forceinline__ void dwv_store(float* p, float4 v) { st4(p, v); }

template <int S, class V>
__global__ __launch_bounds__(256) void dw_fwd_sweep_kernel(const float* __restrict__ x,
                                                           const float* __restrict__ w,
                                                           const float* __restrict__ b,
                                                           float* __restrict__ y, DwShape s,
                                                           int act, int seg_rows, int nseg, int nq,
                                                           int total) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  constexpr int VW = sizeof(V) / sizeof(float);
  const int c = (i % nq) * VW, u = i / nq;
  const int seg = u % nseg, t = u / nseg, wo = t % s.Wo, n = t / s.Wo;
  const int h0 = seg * seg_rows, h1 = min(s.Ho, h0 + seg_rows);
  V wk[9], bb;
#pragma unroll
  for (int k = 0; k < 9; ++k) wk[k] = dwv_load(w + k * s.C + c, V{});
  if (b) bb = dwv_load(b + c, V{});
  else dwv_zero(bb);
  bool cv[3];
  int wc[3];
#pragma unroll
  for (int kx = 0; kx < 3; ++kx) {
    const int ww = wo * S + kx - 1;
    cv[kx] = ww >= 0 && ww < s.W;
    wc[kx] = cv[kx] ? ww : 0;
  }
  auto load_row = [&](int hh, V (&r)[3], bool& ok) {
    ok = hh >= 0 && hh < s.H;
    const float* base = x + ((int64_t)n * s.H + (ok ? hh : 0)) * s.W * s.C + c;
#pragma unroll
    for (int kx = 0; kx < 3; ++kx) {
      if (ok && cv[kx]) r[kx] = dwv_load(base + (int64_t)wc[kx] * s.C, V{});
      else dwv_zero(r[kx]);
    }
  };
  V win[3][3], nx[2][3];
  bool rv[3], nv[2];
  load_row(h0 * S - 1, win[0], rv[0]);
  load_row(h0 * S, win[1], rv[1]);
  load_row(h0 * S + 1, win[2], rv[2]);
  for (int ho = h0; ho < h1; ++ho) {
    // the next output row's new input rows are requested before this row's sums
    if (ho + 1 < h1) {
      if (S == 1) {
        load_row(ho + 2, nx[0], nv[0]);
      } else {
        load_row(2 * ho + 2, nx[0], nv[0]);
        load_row(2 * ho + 3, nx[1], nv[1]);
      }
    }
    V acc;
    dwv_zero(acc);
#pragma unroll
    for (int ky = 0; ky < 3; ++ky)
#pragma unroll
      for (int kx = 0; kx < 3; ++kx)
        if (rv[ky] && cv[kx]) acc = dwv_fma(win[ky][kx], wk[ky * 3 + kx], acc);
    if (b) acc = dwv_add(acc, bb);
    dwv_store(y + (((int64_t)n * s.Ho + ho) * s.Wo + wo) * s.C + c, dwv_act(act, acc));
    if (ho + 1 < h1) {
#pragma unroll
      for (int kx = 0; kx < 3; ++kx) {
        if (S == 1) {
          win[0][kx] = win[1][kx];
          win[1][kx] = win[2][kx];
          win[2][kx] = nx[0][kx];
        } else {
          win[0][kx] = win[2][kx];
          win[1][kx] = nx[0][kx];
          win[2][kx] = nx[1][kx];
        }
      }
      if (S == 1) {
        rv[0] = rv[1];
        rv[1] = rv[2];
        rv[2] = nv[0];
      } else {
        rv[0] = rv[2];
        rv[1] = nv[0];
        rv[2] = nv[1];
      }
    }
  }
}

// Stride 1: dx[n,h,w,c] = sum over (ky, kx) of dy[n,h+1-ky,w+1-kx,c] * W[ky,kx,c];
// window row ky holds dy row h + 1 - ky, column kx dy column w + 1 - kx.
template <class V>
__global__ __launch_bounds__(256) void dw_dgrad_sweep_kernel(const float* __restrict__ dy,
                                                             const float* __restrict__ w,
                                                             const float* __restrict__ prev,
                                                             int act_prev, float* __restrict__ dx,
                                                             DwShape s, int seg_rows, int nseg,
                                                             int nq, int total) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  constexpr int VW = sizeof(V) / sizeof(float);
  const int c = (i % nq) * VW, u = i / nq;
  const int seg = u % nseg, t = u / nseg, col = t % s.W, n = t / s.W;
  const int h0 = seg * seg_rows, h1 = min(s.H, h0 + seg_rows);
  V wk[9];
#pragma unroll
  for (int k = 0; k < 9; ++k) wk[k] = dwv_load(w + k * s.C + c, V{});
  bool cv[3];
  int wc[3];
#pragma unroll
  for (int kx = 0; kx < 3; ++kx) {
    const int ww = col + 1 - kx;
    cv[kx] = ww >= 0 && ww < s.Wo;
    wc[kx] = cv[kx] ? ww : 0;
  }
  auto load_row = [&](int hh, V (&r)[3], bool& ok) {
    ok = hh >= 0 && hh < s.Ho;
    const float* base = dy + ((int64_t)n * s.Ho + (ok ? hh : 0)) * s.Wo * s.C + c;
#pragma unroll
    for (int kx = 0; kx < 3; ++kx) {
      if (ok && cv[kx]) r[kx] = dwv_load(base + (int64_t)wc[kx] * s.C, V{});
      else dwv_zero(r[kx]);
    }
  };
  V win[3][3], nx[3];
  bool rv[3], nv;
  load_row(h0 + 1, win[0], rv[0]);
  load_row(h0, win[1], rv[1]);
  load_row(h0 - 1, win[2], rv[2]);
  for (int h = h0; h < h1; ++h) {
    // the next row's new dy row is requested before this row's sums
    if (h + 1 < h1) load_row(h + 2, nx, nv);
    V acc;
    dwv_zero(acc);
#pragma unroll
    for (int ky = 0; ky < 3; ++ky)
#pragma unroll
      for (int kx = 0; kx < 3; ++kx)
        if (rv[ky] && cv[kx]) acc = dwv_fma(win[ky][kx], wk[ky * 3 + kx], acc);
    const int64_t o = (((int64_t)n * s.H + h) * s.W + col) * s.C + c;
    dwv_store(dx + o, dwv_dact(acc, act_prev, prev + o, V{}));
    if (h + 1 < h1) {
#pragma unroll
      for (int kx = 0; kx < 3; ++kx) {
        win[2][kx] = win[1][kx];
        win[1][kx] = win[0][kx];
        win[0][kx] = nx[kx];
      }
      rv[2] = rv[1];
      rv[1] = rv[0];
      rv[0] = nv;
    }
  }
}

struct DwReduce {
  const float* part;
  int S, C;
  int lanes;    // L: lanes per output element (a power of two, at most 64)
  // eager
  float* dw;
  float* db;
  int accumulate;
  // fused
  int fused;
  of_param W, b;
  const float* gW;
  const float* gb;
};

// Pass 2: L consecutive lanes per filter element (and bias element).
__global__ __launch_bounds__(256) void dw_wgrad_reduce_kernel(DwReduce r, OptK o) {
  if (r.fused) opt_prepare(o);
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int L = r.lanes;
  const int j = (int)(t / L), lane = (int)(t % L);
  const bool live = j < DW_TAPS * r.C;
  const int k = live ? j / r.C : 0, c = live ? j % r.C : 0;
  const bool bias = k == 9;
  const bool want = live && (bias ? (r.fused ? r.b.w != nullptr : r.db != nullptr) : true);
  const int off = bias ? c : j;
  // the lead lane loads the parameter's state while the slices are summed
  OptState1 st{0.f, 0.f, 0.f};
  if (r.fused && want && lane == 0) st = opt_load1(o, bias ? r.b : r.W, off);
  // lane l sums slices [l * SG, (l + 1) * SG) in order, 8 loads in flight
  const int SG = (r.S + L - 1) / L;
  const int kb = min(r.S, lane * SG), ke = min(r.S, kb + SG);
  const int64_t ld = (int64_t)DW_TAPS * r.C;
  float g = 0.f;
  if (want) {
    for (int s0 = kb; s0 < ke; s0 += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = s0 + u < ke ? r.part[(s0 + u) * ld + j] : 0.f;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (s0 + u < ke) g = s0 + u == kb ? v[u] : __fadd_rn(g, v[u]);
    }
  }
  // the run sums, added in lane order (the whole group stays within a wave)
  if (L > 1) {
    const int lead = (threadIdx.x & 63) & ~(L - 1);
    float tot = __shfl(g, lead);
    for (int u = 1; u < L; ++u) {
      const float e = __shfl(g, lead + u);
      if (u * SG < r.S) tot = __fadd_rn(tot, e);
    }
    g = tot;
  }
  if (!want || lane != 0) return;
  if (!r.fused) {
    float* dst = bias ? r.db + c : r.dw + j;
    *dst = r.accumulate ? __fadd_rn(*dst, g) : g;
    return;
  }
  const float* gp = bias ? r.gb : r.gW;
  if (gp) g = __fadd_rn(g, gp[off]);
  opt_apply1(o, bias ? r.b : r.W, st, g, off);
}

namespace {
int dw_stride(const of_conv_desc& d) { return d.stride > 1 ? (int)d.stride : 1; }
int64_t dw_out(int64_t n, int S) { return (n - 1) / S + 1; }
int64_t dw_out_pixels(const of_conv_desc& d) {
  return d.N * dw_out(d.H, dw_stride(d)) * dw_out(d.W, dw_stride(d));
}
// Channels per pass-1 workgroup: the width of 64, 48, 32, 16 that pads C
// least (ties to the wider).
int dw_cb(const of_conv_desc& d) {
  int best = DW_CB_MAX;
  int64_t best_pad = -1;
  for (int cb = DW_CB_MAX; cb >= 16; cb -= 16) {
    const int64_t pad = (d.C + cb - 1) / cb * cb - d.C;
    if (best_pad < 0 || pad < best_pad) best = cb, best_pad = pad;
  }
  return best;
}
// Units of pass 1 (one column of one image over up to DW_SEG output rows).
int dw_nseg(const of_conv_desc& d) { return (int)((dw_out(d.H, dw_stride(d)) + DW_SEG - 1) / DW_SEG); }
int64_t dw_units(const of_conv_desc& d) { return d.N * dw_out(d.W, dw_stride(d)) * dw_nseg(d); }
// Unit slices of pass 1: enough workgroups for about 1024 threads per compute
// unit, each slice at least one unit per stream.
int dw_slices(const of_conv_desc& d) {
  const int64_t U = dw_units(d);
  const int cb = dw_cb(d);
  const int64_t nblk = (d.C + cb - 1) / cb;
  const int64_t want = std::max<int64_t>(1, (256 * 1024 / (4 * cb)) / nblk);
  return (int)std::max<int64_t>(1, std::min<int64_t>((U + 15) / 16, want));
}
// Rows per thread of the forward and stride-1 data-gradient sweeps (measured on
// MI355X over MobileNetV2's 17 depthwise layers at batch 32: the forward 0.315 ms
// one pixel per thread, 0.285 with 4 rows, 0.271 with 8; the data gradient
// fastest at 2, where it ties the one-pixel kernel).
constexpr int DW_FWD_SEG = 8;
constexpr int DW_DGRAD_SEG = 2;
// Lanes per element of pass 2: runs of about 4 slices, at most a wave.
int dw_lanes(int S) {
  int L = 1;
  while (L < 64 && L * 8 <= S) L *= 2;
  return L;
}
DwShape dw_shape(const of_conv_desc& d) {
  const int S = dw_stride(d);
  return DwShape{(int)d.N, (int)d.H, (int)d.W, (int)d.C, (int)dw_out(d.H, S), (int)dw_out(d.W, S)};
}
}  // namespace

size_t dw_workspace_bytes(const of_conv_desc& d) {
  return (size_t)dw_slices(d) * DW_TAPS * (size_t)d.C * sizeof(float);
}

hipError_t launch_dw_fwd(const of_conv_desc& d, const float* x, const float* w, const float* b,
                         float* y, hipStream_t stream) {
  // one thread per unit (an output column over up to DW_FWD_SEG rows) and channel (quad)
  const int seg_rows = DW_FWD_SEG;
  const int64_t Ho = dw_out(d.H, dw_stride(d));
  const int nseg = (int)((Ho + seg_rows - 1) / seg_rows);
  const int64_t units = d.N * dw_out(d.W, dw_stride(d)) * nseg;
  const bool quad = d.C % 4 == 0 && aligned16(x) && aligned16(w) && aligned16(b) && aligned16(y);
  const int nq = (int)(quad ? d.C / 4 : d.C);
  const int total = (int)(units * nq);
  const dim3 grid((total + 255) / 256);
  const float* bias = d.has_bias ? b : nullptr;
  const bool two = dw_stride(d) == 2;
  if (quad) {
    if (two)
      hipLaunchKernelGGL((dw_fwd_sweep_kernel<2, float4>), grid, dim3(256), 0, stream, x, w, bias,
                         y, dw_shape(d), (int)d.act, seg_rows, nseg, nq, total);
    else
      hipLaunchKernelGGL((dw_fwd_sweep_kernel<1, float4>), grid, dim3(256), 0, stream, x, w, bias,
                         y, dw_shape(d), (int)d.act, seg_rows, nseg, nq, total);
  } else {
    if (two)
      hipLaunchKernelGGL((dw_fwd_sweep_kernel<2, float>), grid, dim3(256), 0, stream, x, w, bias,
                         y, dw_shape(d), (int)d.act, seg_rows, nseg, nq, total);
    else
      hipLaunchKernelGGL((dw_fwd_sweep_kernel<1, float>), grid, dim3(256), 0, stream, x, w, bias,
                         y, dw_shape(d), (int)d.act, seg_rows, nseg, nq, total);
  }
  return hipGetLastError();
}

hipError_t launch_dw_dgrad(const of_conv_desc& d, const float* dy, const float* w,
                           const float* prev, int act_prev, float* dx, hipStream_t stream) {
  const bool quad = d.C % 4 == 0 && aligned16(dy) && aligned16(w) && aligned16(prev) &&
                    aligned16(dx);
  if (dw_stride(d) == 1) {
    // one thread per unit (an input column over up to DW_DGRAD_SEG rows) and channel (quad)
    const int seg_rows = DW_DGRAD_SEG;
    const int nseg = (int)((d.H + seg_rows - 1) / seg_rows);
    const int nq = (int)(quad ? d.C / 4 : d.C);
    const int total = (int)(d.N * d.W * nseg * nq);
    const dim3 grid((total + 255) / 256);
    if (quad)
      hipLaunchKernelGGL(dw_dgrad_sweep_kernel<float4>, grid, dim3(256), 0, stream, dy, w, prev,
                         act_prev, dx, dw_shape(d), seg_rows, nseg, nq, total);
    else
      hipLaunchKernelGGL(dw_dgrad_sweep_kernel<float>, grid, dim3(256), 0, stream, dy, w, prev,
                         act_prev, dx, dw_shape(d), seg_rows, nseg, nq, total);
    return hipGetLastError();
  }
  // stride 2: one thread per input element (quad); each takes at most four taps
  const int total = (int)(d.N * d.H * d.W * d.C);
  if (quad) {
    const int quads = total / 4;
    hipLaunchKernelGGL(dw_dgrad4_kernel<2>, dim3((quads + 255) / 256), dim3(256), 0, stream, dy, w,
                       prev, act_prev, dx, dw_shape(d), quads);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(dw_dgrad_kernel<2>, dim3((total + 255) / 256), dim3(256), 0, stream, dy, w,
                     prev, act_prev, dx, dw_shape(d), total);
  return hipGetLastError();
}

hipError_t launch_dw_wgrad(const of_conv_desc& d, const float* dy, const float* x, float* dw,
                           float* db, int accumulate, const of_param* W, const of_param* b,
                           const float* gW, const float* gb, const OptK* o, void* ws,
                           hipStream_t stream) {
  const int nsl = dw_slices(d);   // unit slices of pass 1
  const int64_t U = dw_units(d);
  const int per = (int)((U + nsl - 1) / nsl);
  const int nseg = dw_nseg(d);
  const int cb = dw_cb(d);
  const int nblk = (int)((d.C + cb - 1) / cb);
  const size_t lds = (size_t)16 * DW_TAPS * cb * sizeof(float);
  float* part = static_cast<float*>(ws);
  const bool two = dw_stride(d) == 2;
  const dim3 grid(nblk, nsl), block(4 * cb);
  if (d.C % 4 == 0 && aligned16(dy) && aligned16(x)) {
    if (two)
      hipLaunchKernelGGL(dw_wgrad_partial4_kernel<2>, grid, block, lds, stream, dy, x, part,
                         dw_shape(d), per, cb, nseg);
    else
      hipLaunchKernelGGL(dw_wgrad_partial4_kernel<1>, grid, block, lds, stream, dy, x, part,
                         dw_shape(d), per, cb, nseg);
  } else {
    if (two)
      hipLaunchKernelGGL(dw_wgrad_partial_kernel<2>, grid, block, lds, stream, dy, x, part,
                         dw_shape(d), per, cb, nseg);
    else
      hipLaunchKernelGGL(dw_wgrad_partial_kernel<1>, grid, block, lds, stream, dy, x, part,
                         dw_shape(d), per, cb, nseg);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  DwReduce r{};
  r.part = part;
  r.S = nsl;
  r.C = (int)d.C;
  r.lanes = dw_lanes(nsl);
  r.dw = dw;
  r.db = db;
  r.accumulate = accumulate;
  r.fused = o != nullptr;
  if (W) r.W = *W;
  if (b) r.b = *b;
  r.gW = gW;
  r.gb = gb;
  const int64_t n = (int64_t)DW_TAPS * d.C * r.lanes;
  hipLaunchKernelGGL(dw_wgrad_reduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                     stream, r, o ? *o : OptK{});
  return hipGetLastError();
}

}  // namespace opfuse
