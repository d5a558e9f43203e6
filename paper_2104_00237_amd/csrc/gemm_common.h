// Device helpers shared by the fp32 and bf16 contraction kernels: buffer
// loads with out-of-range masking, the epilogues (plain, data gradient,
// weight gradient, backward-fusion update) and the split-reduction pass.
#pragma once

#include <algorithm>

#include "common.h"

namespace opfuse {

// ------------------------------------------------------------ operand tiles
// Operand loads are buffer loads: an offset outside the buffer returns 0, so a
// masked element is loaded from an out-of-range offset instead of being
// branched around.  Every thread issues the same loads every chunk, which lets
// the compiler keep several chunks in flight (its wait counters stay exact).
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOOB = 0x80000000u;  // beyond num_records: reads as 0

// `base` must be the same in every lane (a tile origin): buffer descriptors
// live in scalar registers.  Reading it from the first lane says so to the
// compiler, which otherwise may not prove it and wraps every load in a loop
// over the distinct values.
__device__ __forceinline__ rsrc_t make_rsrc(const void* base) {
  const uint64_t a = (uint64_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  void* ub = (void*)(((uint64_t)hi << 32) | lo);
  // raw buffer, stride 0, 2^31-1 bytes addressable from `base`
  return __builtin_amdgcn_make_buffer_rsrc(ub, (short)0, 0x7fffffff, 0x00020000);
}
// Descriptor of `base + off` elements, or of nothing when `base` is NULL (an
// optional state tensor): every load through it reads 0 and every store is
// dropped, without touching memory.
__device__ __forceinline__ rsrc_t make_rsrc_opt(const float* base, int64_t off) {
  if (base == nullptr) return __builtin_amdgcn_make_buffer_rsrc((void*)nullptr, (short)0, 0, 0x00020000);
  return make_rsrc(base + off);
}
__device__ __forceinline__ float4 bload4(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ float bload1(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

// ------------------------------------------------------------ tile order
// Workgroups are dispatched to the 8 XCDs (each with its own L2) round-robin
// by linear workgroup index.  Tiles are renumbered so that each XCD owns one
// rectangular block of the output (the 8 blocks tile the grid), so an XCD's L2
// fetches only the operand rows and columns of its block instead of nearly
// all of both operands.  Grids whose tile counts do not factor that way keep
// the plain order.  Every tile is still computed exactly once.
__device__ __forceinline__ void xcd_tile(int& tx, int& ty, int group = 0) {
  const int gx = gridDim.x, gy = gridDim.y;
  tx = blockIdx.x;
  ty = blockIdx.y;
  if ((gx * gy) % 8 != 0) return;
  // 8 = sx * sy blocks with sx | gx and sy | gy; prefer the squarest blocks
  int sx = 0, best = 1 << 30;
  for (int c = 1; c <= 8; c *= 2) {
    const int r = 8 / c;
    if (gx % c || gy % r) continue;
    const int bw = gx / c, bh = gy / r;
    const int score = bw > bh ? bw - bh : bh - bw;
    if (score < best) { best = score; sx = c; }
  }
  if (sx == 0) return;
  const int sy = 8 / sx, bw = gx / sx, bh = gy / sy;
  const int lin = blockIdx.x + gx * blockIdx.y;
  const int xcd = lin & 7, j = lin >> 3;            // j < bw * bh
  if (group > 0 && bh % group == 0) {
    // strips of `group` block rows, each walked column by column: the tiles an
    // XCD runs at once form squares that share their operand panels in L2
    const int strip = j / (group * bw), k = j % (group * bw);
    tx = (xcd % sx) * bw + k / group;
    ty = (xcd / sx) * bh + strip * group + k % group;
    return;
  }
  tx = (xcd % sx) * bw + j % bw;
  ty = (xcd / sx) * bh + j / bw;
}

// ------------------------------------------------------------ carried update
// Run by the workgroups of the z-slices from c.z0 on, grid-stride over the
// carried tensors.  Each element gets the same operations as in the eager
// optimizer pass (vector gradients) or the rows-mode update (row partials).
// NT: threads per workgroup of the launch the update rides on.
template <int NT = 256>
__device__ __forceinline__ void carry_update(const CarryArgs& c) {
  OptK o = c.opt;
  opt_prepare(o);
  const int64_t slice = (int64_t)gridDim.x * gridDim.y;
  const int64_t u = ((int64_t)blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x;
  const int64_t U = (int64_t)c.cz * slice;
  // (unrolled: the tensors are indexed statically, so the arguments stay in
  // scalar registers instead of being copied to per-lane scratch)
#pragma unroll
  for (int k = 0; k < OF_CARRY_MAX; ++k) {
    const CarryTensor& T = c.t[k];
    if (T.p.w == nullptr) continue;
    const int64_t n = T.p.numel;
    if (T.rows == 1) {
      for (int64_t i = (u * NT + threadIdx.x) * 4; i < n; i += U * NT * 4) {
        if (T.vec && i + 3 < n) {
          update4(o, T.p, ld4(T.g + i), i);
        } else {
          for (int64_t e = i; e < n && e < i + 4; ++e) update1(o, T.p, T.g[e], e);
        }
      }
    } else {
      for (int64_t i = u * NT + threadIdx.x; i < n; i += U * NT) {
        float s = T.g[i];
        for (int64_t r0 = 1; r0 < T.rows; r0 += 8) {
          float v[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) v[q] = r0 + q < T.rows ? T.g[(r0 + q) * T.ld + i] : 0.f;
#pragma unroll
          for (int q = 0; q < 8; ++q)
            if (r0 + q < T.rows) s = __fadd_rn(s, v[q]);
        }
        update1(o, T.p, s, i);
      }
    }
  }
}

// z-slices of carry workgroups for a contraction whose slice has `slice`
// workgroups: about one workgroup per 256 work items (a float4 of a vector
// gradient, an element of a rows gradient), at most 256 workgroups.
inline int carry_slices(const CarryArgs& c, int64_t slice) {
  int64_t items = 0;
  for (int k = 0; k < OF_CARRY_MAX; ++k) {
    const CarryTensor& T = c.t[k];
    if (T.p.w == nullptr) continue;
    items += T.rows == 1 ? (T.p.numel + 3) / 4 : T.p.numel;
  }
  if (items == 0) return 0;
  const int64_t want = std::min<int64_t>(256, (items + 255) / 256);
  return (int)((want + slice - 1) / slice);
}

// ----------------------------------------------------------------- epilogues
// c[0..n) are the results for (p, q..q+n-1).  vec: 128-bit memory paths allowed
// (bit 0: out/z/prev/res, bit 1: parameter arrays); only used when n == 4.
// A residual R (ea.res: a forward's skip connection, or the gradient a data
// gradient's skip connection adds) is added last, rounded once: the value a
// separate element-wise addition of the two stored tensors gives.
template <int EPI>
__device__ __forceinline__ void epilogue(const EpiArgs& ea, int p, int q, const float (&c)[4],
                                         int n, const float* bias, int vec) {
  if (EPI == EPI_FWD || EPI == EPI_FWD_FF) {
    float zv[4];
    for (int e = 0; e < 4; ++e) zv[e] = (bias && e < n) ? __fadd_rn(c[e], bias[e]) : c[e];
    const int64_t oy = (int64_t)p * ea.ldo + q, oz = (int64_t)p * ea.ldz + q;
    const int64_t orr = (int64_t)p * ea.ldr + q;
    if (n == 4 && (vec & 1)) {
      if (ea.z) st4(ea.z + oz, make_float4(zv[0], zv[1], zv[2], zv[3]));
      float4 y = make_float4(act_fwd(ea.act, zv[0]), act_fwd(ea.act, zv[1]),
                             act_fwd(ea.act, zv[2]), act_fwd(ea.act, zv[3]));
      if (ea.res) {
        const float4 r = ld4(ea.res + orr);
        y.x = __fadd_rn(y.x, r.x); y.y = __fadd_rn(y.y, r.y);
        y.z = __fadd_rn(y.z, r.z); y.w = __fadd_rn(y.w, r.w);
      }
      if (ea.yb) st_bf16x4(ea.yb + oy, y);
      else st4(ea.out + oy, y);
    } else {
      for (int e = 0; e < n; ++e) {
        if (ea.z) ea.z[oz + e] = zv[e];
        float y = act_fwd(ea.act, zv[e]);
        if (ea.res) y = __fadd_rn(y, ea.res[orr + e]);
        if (ea.yb) ea.yb[oy + e] = f32_to_bf16(y);
        else ea.out[oy + e] = y;
      }
    }
  } else if (EPI == EPI_DGRAD) {
    const int64_t oo = (int64_t)p * ea.ldo + q, op = (int64_t)p * ea.ldp + q;
    const int64_t orr = (int64_t)p * ea.ldr + q;
    if (n == 4 && (vec & 1)) {
      float4 r = make_float4(c[0], c[1], c[2], c[3]);
      if (ea.act != OF_ACT_NONE) {
        const float4 s = ld4(ea.prev + op);
        r.x = __fmul_rn(r.x, act_grad(ea.act, s.x));
        r.y = __fmul_rn(r.y, act_grad(ea.act, s.y));
        r.z = __fmul_rn(r.z, act_grad(ea.act, s.z));
        r.w = __fmul_rn(r.w, act_grad(ea.act, s.w));
      }
      if (ea.res) {
        const float4 t = ld4(ea.res + orr);
        r.x = __fadd_rn(r.x, t.x); r.y = __fadd_rn(r.y, t.y);
        r.z = __fadd_rn(r.z, t.z); r.w = __fadd_rn(r.w, t.w);
      }
      st4(ea.out + oo, r);
    } else {
      for (int e = 0; e < n; ++e) {
        float r = c[e];
        if (ea.act != OF_ACT_NONE) r = __fmul_rn(r, act_grad(ea.act, ea.prev[op + e]));
        if (ea.res) r = __fadd_rn(r, ea.res[orr + e]);
        ea.out[oo + e] = r;
      }
    }
  } else if (EPI == EPI_WGRAD) {
    const int64_t oo = (int64_t)p * ea.ldo + q;
    if (n == 4 && (vec & 1)) {
      float4 r = make_float4(c[0], c[1], c[2], c[3]);
      if (ea.accumulate) {
        const float4 o = ld4(ea.out + oo);
        r.x = __fadd_rn(o.x, r.x); r.y = __fadd_rn(o.y, r.y);
        r.z = __fadd_rn(o.z, r.z); r.w = __fadd_rn(o.w, r.w);
      }
      st4(ea.out + oo, r);
    } else {
      for (int e = 0; e < n; ++e)
        ea.out[oo + e] = ea.accumulate ? __fadd_rn(ea.out[oo + e], c[e]) : c[e];
    }
  } else if (EPI == EPI_WGRAD_BF) {
    const int64_t oo = (int64_t)p * ea.ldo + q;
    if (n == 4 && (vec & 2)) {
      float4 g = make_float4(c[0], c[1], c[2], c[3]);
      if (ea.gW) {
        const float4 e = ld4(ea.gW + oo);
        g.x = __fadd_rn(e.x, g.x); g.y = __fadd_rn(e.y, g.y);
        g.z = __fadd_rn(e.z, g.z); g.w = __fadd_rn(e.w, g.w);
      }
      update4(ea.opt, ea.W, g, oo);
    } else {
      for (int e = 0; e < n; ++e) {
        const float g = ea.gW ? __fadd_rn(ea.gW[oo + e], c[e]) : c[e];
        update1(ea.opt, ea.W, g, oo + e);
      }
    }
  }
}

// Bias gradient of output row p (wgrad): store / accumulate, or update the bias.
template <int EPI>
__device__ __forceinline__ void bias_epilogue(const EpiArgs& ea, int p, float g) {
  if (EPI == EPI_WGRAD) {
    ea.db[p] = ea.accumulate ? __fadd_rn(ea.db[p], g) : g;
  } else if (EPI == EPI_WGRAD_BF) {
    update1(ea.opt, ea.b, ea.gb ? __fadd_rn(ea.gb[p], g) : g, p);
  }
}

// Backward-fusion items of the reduction passes load the parameter's state
// (and a shared parameter's pending gradient) before they sum the partials,
// so that the update does not wait for one more memory round trip at the end.
struct BfPre {
  OptState4 st;
  float4 e;
};

__device__ __forceinline__ BfPre bf_preload(const EpiArgs& ea, int64_t oo) {
  BfPre b;
  b.st = opt_load4(ea.opt, ea.W, oo);
  b.e = ea.gW ? ld4(ea.gW + oo) : make_float4(0.f, 0.f, 0.f, 0.f);
  return b;
}

// The vector backward-fusion epilogue on a preloaded state: the same
// operations as epilogue<EPI_WGRAD_BF> on an item of four.
__device__ __forceinline__ void bf_apply(const EpiArgs& ea, const BfPre& b, const float (&c)[4],
                                         int64_t oo) {
  float4 g = make_float4(c[0], c[1], c[2], c[3]);
  if (ea.gW) {
    g.x = __fadd_rn(b.e.x, g.x); g.y = __fadd_rn(b.e.y, g.y);
    g.z = __fadd_rn(b.e.z, g.z); g.w = __fadd_rn(b.e.w, g.w);
  }
  opt_apply4(ea.opt, ea.W, b.st, g, oo);
}

// Sum the split partials in split order, then run the epilogue.
template <int EPI>
__device__ __forceinline__ void split_reduce_body(int P, int Q, int S, EpiArgs& ea,
                                                  const float* __restrict__ partial, int vec_epi,
                                                  int with_db) {
  if (EPI == EPI_WGRAD_BF) opt_prepare(ea.opt);
  const int nq4 = (Q + 3) / 4;
  const int64_t total = (int64_t)P * nq4;
  const int64_t PQ = (int64_t)P * Q;
  for (int64_t idx = blockIdx.x * 256 + threadIdx.x; idx < total; idx += (int64_t)gridDim.x * 256) {
    const int p = (int)(idx / nq4), q = (int)(idx % nq4) * 4;
    const int n = min(4, Q - q);
    float c[4] = {0.f, 0.f, 0.f, 0.f};
    const float* src = partial + (int64_t)p * Q + q;
    const int64_t oo = (int64_t)p * ea.ldo + q;
    const bool pre = EPI == EPI_WGRAD_BF && n == 4 && (vec_epi & 2);
    BfPre bp;
    if (pre) bp = bf_preload(ea, oo);
    // The loads of 8 splits are issued before they are added in split order,
    // so a long split list is not one dependent chain of loads.
    if (n == 4 && (Q & 3) == 0) {
      float4 s = ld4(src);
      for (int k0 = 1; k0 < S; k0 += 8) {
        float4 t[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          t[u] = k0 + u < S ? ld4(src + (int64_t)(k0 + u) * PQ) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (k0 + u < S) {
            s.x = __fadd_rn(s.x, t[u].x); s.y = __fadd_rn(s.y, t[u].y);
            s.z = __fadd_rn(s.z, t[u].z); s.w = __fadd_rn(s.w, t[u].w);
          }
        }
      }
      c[0] = s.x; c[1] = s.y; c[2] = s.z; c[3] = s.w;
    } else {
      float s4[4];
      for (int e = 0; e < n; ++e) s4[e] = src[e];
      for (int k0 = 1; k0 < S; k0 += 8) {
        float t[8][4];
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            t[u][e] = (k0 + u < S && e < n) ? src[(int64_t)(k0 + u) * PQ + e] : 0.f;
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (k0 + u < S)
            for (int e = 0; e < n; ++e) s4[e] = __fadd_rn(s4[e], t[u][e]);
      }
      for (int e = 0; e < n; ++e) c[e] = s4[e];
    }
    if (pre) {
      bf_apply(ea, bp, c, oo);
      continue;
    }
    const float* bias = nullptr;
    if ((EPI == EPI_FWD || EPI == EPI_FWD_FF) && ea.bias) bias = ea.bias + q;
    epilogue<EPI == EPI_FWD_FF ? EPI_FWD : EPI>(ea, p, q, c, n, bias, vec_epi);
  }
  if (with_db) {
    const float* dbp = partial + (int64_t)S * PQ;
    for (int p = blockIdx.x * 256 + threadIdx.x; p < P; p += gridDim.x * 256) {
      float s = dbp[p];
      for (int k0 = 1; k0 < S; k0 += 8) {
        float t[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) t[u] = k0 + u < S ? dbp[(int64_t)(k0 + u) * P + p] : 0.f;
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (k0 + u < S) s = __fadd_rn(s, t[u]);
      }
      bias_epilogue<EPI>(ea, p, s);
    }
  }
}

// Long split lists: G = 8 consecutive lanes (one wave holds whole groups)
// share each float4 item of the output.  Lane j sums the splits
// j*SG .. (j+1)*SG - 1 in split order (SG = ceil(S / 8)); the group's first
// lane then adds the 8 sums in lane order and runs the epilogue.  A single
// thread per item would wait for S / 8 load latencies in a row.  The order
// is fixed, so every ordering that shares a tiling still gets the same bits.
// The bias-gradient partials are summed the same way.
template <int EPI>
__device__ __forceinline__ void split_reduce_coop_body(int P, int Q, int S, EpiArgs& ea,
                                                       const float* __restrict__ partial,
                                                       int vec_epi, int with_db) {
  if (EPI == EPI_WGRAD_BF) opt_prepare(ea.opt);
  const int nq4 = (Q + 3) / 4;
  const int64_t total = (int64_t)P * nq4;
  const int64_t PQ = (int64_t)P * Q;
  const int lane = threadIdx.x & 63, j = lane & 7, lead = lane & ~7;
  const int SG = (S + 7) / 8;
  const int kb = min(S, j * SG), ke = min(S, kb + SG);
  const int64_t groups = (int64_t)gridDim.x * 32;
  // lanes [0, 4): this lane's partial sums of the item's (up to) 4 elements
  auto lane_sum = [&](const float* src, int n, bool v4, float (&acc)[4]) {
    for (int e = 0; e < 4; ++e) acc[e] = 0.f;
    for (int k0 = kb; k0 < ke; k0 += 8) {
      float4 t[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int k = k0 + u;
        if (k < ke) {
          const float* a = src + (int64_t)k * PQ;
          t[u] = v4 ? ld4(a) : make_float4(a[0], n > 1 ? a[1] : 0.f, n > 2 ? a[2] : 0.f,
                                           n > 3 ? a[3] : 0.f);
        } else {
          t[u] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (k0 + u < ke) {
          acc[0] = __fadd_rn(acc[0], t[u].x); acc[1] = __fadd_rn(acc[1], t[u].y);
          acc[2] = __fadd_rn(acc[2], t[u].z); acc[3] = __fadd_rn(acc[3], t[u].w);
        }
      }
    }
  };
  for (int64_t idx = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 3; idx < total; idx += groups) {
    const int p = (int)(idx / nq4), q = (int)(idx % nq4) * 4;
    const int n = min(4, Q - q);
    const int64_t oo = (int64_t)p * ea.ldo + q;
    const bool pre = EPI == EPI_WGRAD_BF && n == 4 && (vec_epi & 2) && j == 0;
    BfPre bp;
    if (pre) bp = bf_preload(ea, oo);
    float acc[4];
    lane_sum(partial + (int64_t)p * Q + q, n, n == 4 && (Q & 3) == 0, acc);
    float c[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      c[e] = __shfl(acc[e], lead);
#pragma unroll
      for (int g = 1; g < 8; ++g) c[e] = __fadd_rn(c[e], __shfl(acc[e], lead + g));
    }
    if (pre) {
      bf_apply(ea, bp, c, oo);
    } else if (j == 0) {
      const float* bias = nullptr;
      if ((EPI == EPI_FWD || EPI == EPI_FWD_FF) && ea.bias) bias = ea.bias + q;
      epilogue<EPI == EPI_FWD_FF ? EPI_FWD : EPI>(ea, p, q, c, n, bias, vec_epi);
    }
  }
  if (with_db) {
    const float* dbp = partial + (int64_t)S * PQ;
    for (int64_t p = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 3; p < P; p += groups) {
      float acc = 0.f;
      for (int k0 = kb; k0 < ke; k0 += 8) {
        float t[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) t[u] = k0 + u < ke ? dbp[(int64_t)(k0 + u) * P + p] : 0.f;
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (k0 + u < ke) acc = __fadd_rn(acc, t[u]);
      }
      float s = __shfl(acc, lead);
#pragma unroll
      for (int g = 1; g < 8; ++g) s = __fadd_rn(s, __shfl(acc, lead + g));
      if (j == 0) bias_epilogue<EPI>(ea, (int)p, s);
    }
  }
}

}  // namespace opfuse
