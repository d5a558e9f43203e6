// bf16-operand contractions of a linear layer on the CDNA4 matrix cores
// (v_mfma_f32_32x32x16_bf16), with the same epilogues as the fp32 kernels:
// plain forward, data gradient, weight gradient, and the weight gradient with
// the optimizer applied in its epilogue (backward-fusion).
//
// Operands stay in their storage type in HBM: fp32 activations and gradients
// are rounded to bf16 (round to nearest even) as they are staged into LDS,
// which is the same value as rounding them just before the product; an
// activation that only these contractions read may be stored as that bf16
// rounding by its producer and is then read as stored (the forward's X, the
// weight gradient's X); a weight operand is read from its bf16 shadow when one
// is given (half the bytes), else rounded from the fp32 master.  Products of
// bf16 values are exact in fp32 and the sums accumulate in fp32.  A forward
// may store its output Y as bf16 as well (for a consumer of the same kind).
//
// LDS layout: each operand tile is stored as BR/8 planes of [BX][8] bf16, so
// the 8 consecutive reduction elements a lane feeds one MFMA are one 16-byte
// read.  A tile element (x, r) lives at plane r/8, row x, slot r%8.  Loads are
// grouped in quads along the contiguous index (4 reduction elements of one
// row, or 4 rows by 4 output columns when the output index is contiguous), so
// every LDS store writes 4 bf16 (8 bytes) along the reduction index.
//
// The reduction runs in chunks of BR with double-buffered LDS and one barrier
// per chunk; the next chunk's global loads are issued before the current
// chunk's MFMAs.  A grid-level split of the reduction writes fp32 partials that
// a second kernel sums in split order before the epilogue (deterministic; the
// eager and backward-fusion weight gradients share the tiling rule).

#include <algorithm>
#include <cstdio>
#include <cstdlib>

#include "gemm_common.h"

namespace opfuse {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float float2_t __attribute__((ext_vector_type(2)));
typedef float floatx16_t __attribute__((ext_vector_type(16)));

template <int BP_, int BQ_, int BR_, int WP_, int WQ_, int NS_>
struct BTile {
  static constexpr int BP = BP_, BQ = BQ_, BR = BR_, WP = WP_, WQ = WQ_;
  static constexpr int NS = NS_;   // operand chunks in the register ring
  static constexpr int NW = WP * WQ, NT = 64 * NW;
  static_assert(NW == 4 || NW == 8, "a workgroup is 4 or 8 wavefronts");
  static_assert(BR % 16 == 0, "whole MFMA reduction steps");
  static constexpr int WTP = BP / WP, WTQ = BQ / WQ;
  static constexpr int TP = WTP / 32, TQ = WTQ / 32;
  static_assert(TP >= 1 && TQ >= 1 && WTP % 32 == 0 && WTQ % 32 == 0, "32x32 blocks");
  // Plane strides in bf16 elements, padded by 8 (16 bytes) against bank conflicts.
  static constexpr int PLA = BP * 8 + 8, PLB = BQ * 8 + 8;
  static constexpr int STAGE = (BR / 8) * (PLA + PLB);          // bf16 elements per stage
  static constexpr int SM_MAIN = 2 * STAGE * 2;                  // bytes, two stages
  // The fp32 accumulators are staged through LDS for the epilogue in NPASS
  // bands of PR rows, each band at most 64 KB with rows padded by 4 floats.
  static constexpr int LDC = BQ + 4;
  static constexpr int NPASS = (BP * LDC * 4 <= 65536)       ? 1
                               : ((BP / 2) * LDC * 4 <= 65536) ? 2
                               : ((BP / 4) * LDC * 4 <= 65536) ? 4 : 8;
  static constexpr int PR = BP / NPASS;
  static_assert(PR % 32 == 0, "a band holds whole 32-row MFMA blocks");
  static constexpr int SM_C = PR * LDC * 4;                      // bytes
  static constexpr int SMX = SM_MAIN > SM_C ? SM_MAIN : SM_C;
  static_assert(SMX <= 160 * 1024, "LDS per workgroup");
};

using BT128x128 = BTile<128, 128, 32, 2, 2, 4>;
using BT64x64 = BTile<64, 64, 32, 2, 2, 4>;
// Eight wavefronts (two per SIMD, each on a 64x64 sub-tile) share one A tile
// over 256 output columns, so each A byte fetched feeds twice the outputs.
using BT128x256 = BTile<128, 256, 64, 2, 4, 2>;
#ifdef OPFUSE_TUNING
using BT128x128R64 = BTile<128, 128, 64, 2, 2, 2>;
using BT128x256R32 = BTile<128, 256, 32, 2, 4, 4>;
using BT256x128 = BTile<256, 128, 32, 4, 2, 4>;
using BT256x256W8 = BTile<256, 256, 32, 2, 4, 2>;
using BT256x256W4 = BTile<256, 256, 32, 2, 2, 2>;
enum BTileId { BTI_64x64 = 0, BTI_128x128, BTI_128x256, BTI_128x128R64, BTI_128x256R32,
               BTI_256x128, BTI_256x256W8, BTI_256x256W4, BTI_COUNT };
static const int kBTileBP[BTI_COUNT] = {64, 128, 128, 128, 128, 256, 256, 256};
static const int kBTileBQ[BTI_COUNT] = {64, 128, 256, 128, 256, 128, 256, 256};
static const int kBTileBR[BTI_COUNT] = {32, 32, 64, 64, 32, 32, 32, 32};
#else
enum BTileId { BTI_64x64 = 0, BTI_128x128, BTI_128x256, BTI_COUNT };
static const int kBTileBP[BTI_COUNT] = {64, 128, 128};
static const int kBTileBQ[BTI_COUNT] = {64, 128, 256};
static const int kBTileBR[BTI_COUNT] = {32, 32, 64};
#endif

// Two fp32 values to packed bf16, round to nearest even (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t cvt2(float a, float b) {
  const float2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ uint2 pack_bf16x4(float a, float b, float c, float d) {
  return make_uint2(cvt2(a, b), cvt2(c, d));
}

// Row of a plane that tile row x is stored in: the low two bits are XORed
// with bits 4-5, so the four 8-byte stores of a transposed 4x4 item (rows
// 4l+k of lane l) spread over all bank groups instead of every 4th lane
// colliding; the rows a wave reads for one MFMA stay one contiguous block.
__device__ __forceinline__ int swz(int x) { return x ^ ((x >> 4) & 3); }

__device__ __forceinline__ uint2 bload8(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}
__device__ __forceinline__ uint32_t bload_u16(rsrc_t r, uint32_t off) {
  return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}

// One operand tile (BX output rows x BR reduction elements) in flight between
// its global loads and its LDS store.  RC: the reduction index is contiguous
// in memory.  BF: the source holds bf16 (else fp32).  VEC: 128-bit (fp32) or
// 64-bit (bf16) loads are allowed: aligned base, strides a multiple of 4
// elements and the contiguous extent ending on a quad boundary (for a bf16
// source with a contiguous reduction index: 16-byte aligned, strides and
// extent multiples of 8, loaded as 128-bit octets).
// An item is a quad along r (RC) or a 4 x 4 block (r, x) (not RC).
template <int BX, int BR, bool RC, bool BF, bool VEC, int NT>
struct BLoad {
  // A bf16 source with a contiguous reduction index moves 8 elements (one
  // 16-byte load, one 16-byte LDS store) per item when vector loads are allowed.
  static constexpr bool W8 = RC && BF && VEC;
  static constexpr int QW = W8 ? 8 : 4;          // reduction elements per RC item
  static constexpr int NQ = RC ? BX * (BR / QW) : (BR / 4) * (BX / 4);  // items
  static constexpr int PER = (NQ + NT - 1) / NT;
  static constexpr int NV = RC ? 1 : 4;          // vectors per item
  static constexpr int PL = BX * 8 + 8;          // plane stride (bf16 elements)
  // raw data: fp32 float4, bf16 quads (as uint2) or bf16 octets (as uint4)
  float4 f[BF ? 1 : PER][BF ? 1 : NV];
  uint2 h[(BF && !W8) ? PER : 1][(BF && !W8) ? NV : 1];
  uint4 o[W8 ? PER : 1];

  __device__ __forceinline__ static void coords(int idx, int& x, int& r) {
    if (RC) { x = idx / (BR / QW); r = (idx % (BR / QW)) * QW; }
    else    { r = (idx / (BX / 4)) * 4; x = (idx % (BX / 4)) * 4; }
  }

  __device__ __forceinline__ void load(const void* tensor, int64_t s_x, int64_t s_r, int x0,
                                       int r0, int nx, int nr, int tid) {
    constexpr int ES = BF ? 2 : 4;
    const rsrc_t rs = make_rsrc((const char*)tensor + ((int64_t)x0 * s_x + (int64_t)r0 * s_r) * ES);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int idx = tid + i * NT;
      int x, r;
      coords(idx, x, r);
      const bool live = (NQ % NT == 0) || idx < NQ;
      if constexpr (W8) {
        // vector loads of a bf16 operand need the reduction extent to be a
        // multiple of 8, so an octet is whole or absent
        const bool ok = live && x < nx && r < nr;
        const uint32_t off = ok ? (uint32_t)((x * s_x + r) * 2) : kOOB;
        o[i] = __builtin_bit_cast(uint4, bload4(rs, off));
        continue;
      }
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        // vector j: RC -> the quad (x, r..r+3); else the quad (x..x+3, r+j)
        const int vx = x, vr = RC ? r : r + j;
        if constexpr (VEC) {
          const bool ok = live && vx < nx && vr < nr;
          const uint32_t off = ok ? (uint32_t)((vx * s_x + vr * s_r) * ES) : kOOB;
          if constexpr (BF) h[i][j] = bload8(rs, off);
          else f[i][j] = bload4(rs, off);
        } else {
          float e[4];
          uint32_t u[4];
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const int xx = RC ? vx : vx + k, rr = RC ? vr + k : vr;
            const bool ok = live && xx < nx && rr < nr;
            const uint32_t off = ok ? (uint32_t)((xx * s_x + rr * s_r) * ES) : kOOB;
            if constexpr (BF) u[k] = bload_u16(rs, off);
            else e[k] = bload1(rs, off);
          }
          if constexpr (BF) h[i][j] = make_uint2(u[0] | (u[1] << 16), u[2] | (u[3] << 16));
          else f[i][j] = make_float4(e[0], e[1], e[2], e[3]);
        }
      }
    }
  }

  // Element k (0..3) of vector j of item i: bf16 bits, or the fp32 value.
  __device__ __forceinline__ uint32_t bits(int i, int j, int k) const {
    const uint32_t w = (k < 2) ? h[i][j].x : h[i][j].y;
    return (k & 1) ? (w >> 16) : (w & 0xffffu);
  }
  __device__ __forceinline__ float val(int i, int j, int k) const {
    return k == 0 ? f[i][j].x : k == 1 ? f[i][j].y : k == 2 ? f[i][j].z : f[i][j].w;
  }

  __device__ __forceinline__ void store(uint16_t* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int idx = tid + i * NT;
      if (NQ % NT != 0 && idx >= NQ) continue;
      int x, r;
      coords(idx, x, r);
      const int plane = r >> 3, slot = r & 7;   // slot is 0 or 4
      if constexpr (W8) {
        *reinterpret_cast<uint4*>(&lds[plane * PL + swz(x) * 8]) = o[i];
      } else if (RC) {
        uint2 q;
        if constexpr (BF) q = h[i][0];
        else q = pack_bf16x4(f[i][0].x, f[i][0].y, f[i][0].z, f[i][0].w);
        *reinterpret_cast<uint2*>(&lds[plane * PL + swz(x) * 8 + slot]) = q;
      } else {
        // transpose the 4 x 4 block: row x+k gets elements k of vectors 0..3
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          uint2 q;
          if constexpr (BF)
            q = make_uint2(bits(i, 0, k) | (bits(i, 1, k) << 16),
                           bits(i, 2, k) | (bits(i, 3, k) << 16));
          else
            q = pack_bf16x4(val(i, 0, k), val(i, 1, k), val(i, 2, k), val(i, 3, k));
          *reinterpret_cast<uint2*>(&lds[plane * PL + swz(x + k) * 8 + slot]) = q;
        }
      }
    }
  }

  // Column sums of the fp32 values (the A operand of a weight gradient is dZ:
  // its sums over the reduction are the bias gradient).  Not RC only.
  __device__ __forceinline__ void colsum(float (&acc)[PER][4]) const {
    if constexpr (!BF && !RC) {
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        acc[i][0] = __fadd_rn(acc[i][0], __fadd_rn(__fadd_rn(__fadd_rn(f[i][0].x, f[i][1].x), f[i][2].x), f[i][3].x));
        acc[i][1] = __fadd_rn(acc[i][1], __fadd_rn(__fadd_rn(__fadd_rn(f[i][0].y, f[i][1].y), f[i][2].y), f[i][3].y));
        acc[i][2] = __fadd_rn(acc[i][2], __fadd_rn(__fadd_rn(__fadd_rn(f[i][0].z, f[i][1].z), f[i][2].z), f[i][3].z));
        acc[i][3] = __fadd_rn(acc[i][3], __fadd_rn(__fadd_rn(__fadd_rn(f[i][0].w, f[i][1].w), f[i][2].w), f[i][3].w));
      }
    }
  }
};

// Operand roles per contraction (see the fp32 kernels): forward A = X (RC),
// B = W (RC); data gradient A = dZ (RC), B = W (output-contiguous); weight
// gradient A = dZ, B = X (both output-contiguous).
template <class T, int EPI, bool VA, bool VB, bool BBF, bool ABF>
__global__ __launch_bounds__(T::NT) void gemm_bf16_kernel(GemmProblem pr, EpiArgs ea, int r_split,
                                                        float* partial, int vec_epi) {
  if (EPI == EPI_WGRAD_BF) opt_prepare(ea.opt);
  constexpr bool A_RC = (EPI == EPI_FWD || EPI == EPI_DGRAD);
  constexpr bool B_RC = (EPI == EPI_FWD);
  constexpr bool WG = (EPI == EPI_WGRAD || EPI == EPI_WGRAD_BF);
  __shared__ __attribute__((aligned(16))) unsigned char smem_raw[T::SMX];
  uint16_t* smem = reinterpret_cast<uint16_t*>(smem_raw);
  if constexpr (EPI == EPI_FWD) {
    if ((int)blockIdx.z < ea.carry.cz) {
      carry_update<T::NT>(ea.carry);  // a later operator's update rides on this launch
      return;
    }
  }

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wp = wave % T::WP, wq = wave / T::WP;
  int tx, ty;
  xcd_tile(tx, ty, pr.group);
  const int p0 = tx * T::BP, q0 = ty * T::BQ;
  const int split = (int)blockIdx.z - ea.carry.cz, S = (int)gridDim.z - ea.carry.cz;
  const int rbeg = split * r_split;
  const int rend = min(pr.R, rbeg + r_split);
  const int nch = (rend - rbeg + T::BR - 1) / T::BR;
  const bool do_db = WG && ea.with_db && ty == 0;

  static_assert(!ABF || EPI == EPI_FWD, "a bf16 A operand only in a forward");
  using LA = BLoad<T::BP, T::BR, A_RC, ABF, VA, T::NT>;
  using LB = BLoad<T::BQ, T::BR, B_RC, BBF, VB, T::NT>;
  constexpr int NS = T::NS;
  LA la[NS];
  LB lb[NS];
  float dbs[LA::PER][4];
#pragma unroll
  for (int i = 0; i < LA::PER; ++i) dbs[i][0] = dbs[i][1] = dbs[i][2] = dbs[i][3] = 0.f;

  floatx16_t acc[T::TP][T::TQ];
#pragma unroll
  for (int i = 0; i < T::TP; ++i)
#pragma unroll
    for (int j = 0; j < T::TQ; ++j)
#pragma unroll
      for (int k = 0; k < 16; ++k) acc[i][j][k] = 0.f;

  const int np = pr.P - p0, nq = pr.Q - q0;
  // Register ring of NS chunks: chunk c+NS-1 is requested before chunk c is
  // staged and multiplied; chunks past the end load nothing (every offset is
  // out of range) and are skipped.
  auto issue = [&](int slot, int c) {
    const int r0 = rbeg + c * T::BR;
    const int nr = c < nch ? rend - r0 : 0;
    la[slot].load(pr.A, pr.a_sp, pr.a_sr, p0, r0, np, nr, tid);
    lb[slot].load(pr.B, pr.b_sq, pr.b_sr, q0, r0, nq, nr, tid);
  };

  constexpr int SA = (T::BR / 8) * T::PLA;   // A part of a stage
#pragma unroll
  for (int s = 0; s < NS - 1; ++s) {
    issue(s, s);
    __builtin_amdgcn_sched_barrier(0);  // chunk 0 stays the oldest load
  }
  for (int c0 = 0; c0 < nch; c0 += NS) {
#pragma unroll
   for (int s = 0; s < NS; ++s) {
    const int c = c0 + s;
    issue((s + NS - 1) % NS, c + NS - 1);
    uint16_t* buf = smem + (c & 1) * T::STAGE;
    if (c < nch) {
      la[s].store(buf, tid);
      lb[s].store(buf + SA, tid);
      if (do_db) la[s].colsum(dbs);
    }
    __syncthreads();
    if (c >= nch) continue;
    const uint16_t* a_s = buf;
    const uint16_t* b_s = buf + SA;
#pragma unroll
    for (int ks = 0; ks < T::BR / 16; ++ks) {
      const int plane = 2 * ks + (lane >> 5);
      bf16x8_t a[T::TP], b[T::TQ];
#pragma unroll
      for (int i = 0; i < T::TP; ++i)
        a[i] = *reinterpret_cast<const bf16x8_t*>(
            &a_s[plane * T::PLA + swz(wp * T::WTP + i * 32 + (lane & 31)) * 8]);
#pragma unroll
      for (int j = 0; j < T::TQ; ++j)
        b[j] = *reinterpret_cast<const bf16x8_t*>(
            &b_s[plane * T::PLB + swz(wq * T::WTQ + j * 32 + (lane & 31)) * 8]);
#pragma unroll
      for (int i = 0; i < T::TP; ++i)
#pragma unroll
        for (int j = 0; j < T::TQ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
   }
  }
  __syncthreads();

  // Stage the accumulators through LDS in row-major order, one band of PR
  // rows at a time (MFMA 32x32 layout: lane holds column lane%32 and rows
  // 8*(k/4) + 4*(lane/32) + k%4), and run the epilogue on each band.
  float* Cs = reinterpret_cast<float*>(smem_raw);
  constexpr int NQ4 = T::BQ / 4;
  constexpr int ITEMS = T::PR * NQ4;
  constexpr int EPT = (ITEMS + T::NT - 1) / T::NT;
#pragma unroll
  for (int h = 0; h < T::NPASS; ++h) {
    if (h) __syncthreads();   // the previous band has been read
#pragma unroll
    for (int i = 0; i < T::TP; ++i) {
      const int rb = wp * T::WTP + i * 32 - h * T::PR;   // block's first row in the band
      if (rb < 0 || rb >= T::PR) continue;
#pragma unroll
      for (int j = 0; j < T::TQ; ++j)
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          const int p = rb + (k >> 2) * 8 + (lane >> 5) * 4 + (k & 3);
          const int q = wq * T::WTQ + j * 32 + (lane & 31);
          Cs[p * T::LDC + q] = acc[i][j][k];
        }
    }
    __syncthreads();

    if constexpr (EPI == EPI_WGRAD_BF) {
      if (S == 1 && (vec_epi & 2) && (pr.Q & 3) == 0) {
        // Backward-fusion without a split: the W, m, v of a group of items are
        // requested together, then updated and stored.  Item by item, each
        // item's loads would wait behind the previous item's stores (they may
        // alias), one memory latency per item.  Same arithmetic as update4.
        constexpr int G = EPT < 2 ? EPT : 2;
        const int64_t org = (int64_t)(p0 + h * T::PR) * ea.ldo + q0;
        const rsrc_t rw = make_rsrc(ea.W.w + org);
        const rsrc_t rm = make_rsrc_opt(ea.W.m, org);
        const rsrc_t rv = ea.opt.kind != OF_OPT_SGD ? make_rsrc(ea.W.v + org) : rm;
#pragma unroll
        for (int e0 = 0; e0 < EPT; e0 += G) {
          float4 pw[G], pm[G], pv[G];
#pragma unroll
          for (int u = 0; u < G; ++u) {
            const int idx = tid + (e0 + u) * T::NT;
            const int p = idx / NQ4, q = (idx % NQ4) * 4;
            const bool ok = e0 + u < EPT && idx < ITEMS && p0 + h * T::PR + p < pr.P &&
                            q0 + q < pr.Q;
            const uint32_t off = ok ? (uint32_t)((p * ea.ldo + q) * 4) : kOOB;
            pw[u] = bload4(rw, off);
            pm[u] = bload4(rm, off);
            pv[u] = bload4(rv, off);
          }
#pragma unroll
          for (int u = 0; u < G; ++u) {
            const int idx = tid + (e0 + u) * T::NT;
            if (e0 + u >= EPT || idx >= ITEMS) break;
            const int p = idx / NQ4, q = (idx % NQ4) * 4;
            const int gp = p0 + h * T::PR + p, gq = q0 + q;
            if (gp >= pr.P || gq >= pr.Q) continue;
            const int64_t oo = (int64_t)gp * ea.ldo + gq;
            float4 g = *reinterpret_cast<const float4*>(&Cs[p * T::LDC + q]);
            if (ea.gW) {
              const float4 e = ld4(ea.gW + oo);
              g.x = __fadd_rn(e.x, g.x); g.y = __fadd_rn(e.y, g.y);
              g.z = __fadd_rn(e.z, g.z); g.w = __fadd_rn(e.w, g.w);
            }
            float4 w = pw[u], m = pm[u], v = pv[u];
            opt_update(ea.opt, w.x, g.x, m.x, v.x);
            opt_update(ea.opt, w.y, g.y, m.y, v.y);
            opt_update(ea.opt, w.z, g.z, m.z, v.z);
            opt_update(ea.opt, w.w, g.w, m.w, v.w);
            st4(ea.W.w + oo, w);
            if (ea.W.m) st4(ea.W.m + oo, m);
            if (ea.opt.kind != OF_OPT_SGD) st4(ea.W.v + oo, v);
            if (ea.W.w_bf16) st_bf16x4(ea.W.w_bf16 + oo, w);
          }
        }
        continue;
      }
    }
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const int idx = tid + e * T::NT;
      if (ITEMS % T::NT != 0 && idx >= ITEMS) break;
      const int p = idx / NQ4, q = (idx % NQ4) * 4;
      const int gp = p0 + h * T::PR + p, gq = q0 + q;
      if (gp >= pr.P || gq >= pr.Q) continue;
      const float4 cv = *reinterpret_cast<const float4*>(&Cs[p * T::LDC + q]);
      const float c[4] = {cv.x, cv.y, cv.z, cv.w};
      const int n = min(4, pr.Q - gq);
      if (S > 1) {
        float* dst = partial + ((int64_t)split * pr.P + gp) * pr.Q + gq;
        if (n == 4 && (pr.Q & 3) == 0) st4(dst, cv);
        else for (int k = 0; k < n; ++k) dst[k] = c[k];
      } else {
        const float* bias = (EPI == EPI_FWD && ea.bias) ? ea.bias + gq : nullptr;
        epilogue<EPI>(ea, gp, gq, c, n, bias, vec_epi);
      }
    }
  }

  if (do_db) {
    // Bias gradient: per-thread column sums, then summed over the threads that
    // hold the same columns, in thread order.
    __syncthreads();
    constexpr int RQ = T::BR / 4;           // threads per column quad
    float* red = reinterpret_cast<float*>(smem_raw);  // [RQ][BP]
#pragma unroll
    for (int i = 0; i < LA::PER; ++i) {
      const int idx = tid + i * T::NT;
      if (idx < LA::NQ) {
        const int rq = idx / (T::BP / 4), x = (idx % (T::BP / 4)) * 4;
        for (int k = 0; k < 4; ++k) red[rq * T::BP + x + k] = dbs[i][k];
      }
    }
    __syncthreads();
    if (tid < T::BP && p0 + tid < pr.P) {
      float s = red[tid];
      for (int rq = 1; rq < RQ; ++rq) s = __fadd_rn(s, red[rq * T::BP + tid]);
      if (S > 1) partial[(int64_t)S * pr.P * pr.Q + (int64_t)split * pr.P + p0 + tid] = s;
      else bias_epilogue<EPI>(ea, p0 + tid, s);
    }
  }
}

template <int EPI>
__global__ __launch_bounds__(256) void split_reduce_bf16_kernel(int P, int Q, int S, EpiArgs ea,
                                                                const float* __restrict__ partial,
                                                                int vec_epi, int with_db) {
  split_reduce_body<EPI>(P, Q, S, ea, partial, vec_epi, with_db);
}

// --------------------------------------------------------------- host side
struct BCfg {
  int tile, S, r_split;
  int cz = 0;   // z-slices of carried-update workgroups after the splits
};

static int64_t bntiles(int t, int P, int Q) {
  return (int64_t)((P + kBTileBP[t] - 1) / kBTileBP[t]) * ((Q + kBTileBQ[t] - 1) / kBTileBQ[t]);
}

// 128x256 eight-wave tiles for large outputs (at least 512 of them) and, in
// a forward, for long reductions (at least 128 tiles, 2048 or more reduction
// elements); else 128x128 tiles when the output has enough of them, else
// 64x64.  The reduction is split until there are about 256 workgroups, and
// for a forward until no split spans more than 2048 elements (at least 4
// chunks per split).  Gradients keep whole reductions on the wide tiles:
// backward-fusion runs them beside each other on two streams, where fewer,
// split workgroups lose what they gain alone (measured on MI355X).  The eager
// and backward-fusion weight gradients share this rule.
static BCfg bselect_default(int kind, int P, int Q, int R) {
  const int64_t nw = bntiles(BTI_128x256, P, Q);
  const bool wide = nw >= 512 || (kind == EPI_FWD && nw >= 128 && R >= 2048);
  const int t = wide                                    ? BTI_128x256
                : bntiles(BTI_128x128, P, Q) >= 64      ? BTI_128x128
                                                        : BTI_64x64;
  const int BR = kBTileBR[t];
  const int64_t nt = bntiles(t, P, Q);
  int S = (int)std::max<int64_t>(1, (256 + nt - 1) / nt);
  // A forward with a long reduction splits further, to at most 2048 elements
  // per split (measured on MI355X at 4096 tokens).  The gradients keep the
  // plain rule: backward-fusion runs them beside each other on two streams,
  // where the extra workgroups and second passes cost more than they save.
  if (kind == EPI_FWD)
    while (S < 8 && (R + S - 1) / S > 2048) S *= 2;
  S = std::min(S, std::min(8, std::max(1, R / (4 * BR))));
  int r_split = (((R + S - 1) / S) + BR - 1) / BR * BR;
  S = (R + r_split - 1) / r_split;
  return BCfg{t, S, r_split};
}

#ifdef OPFUSE_TUNING
// Tuning builds only: OPFUSE_BF16_CFG="tile,S" overrides the bf16 tiling;
// OPFUSE_BF16_WG_S=S the split of the weight gradients alone.
static BCfg bselect(int kind, int P, int Q, int R) {
  const char* e = getenv("OPFUSE_BF16_CFG");
  const char* wgs = getenv("OPFUSE_BF16_WG_S");
  if (!e && wgs && (kind == EPI_WGRAD || kind == EPI_WGRAD_BF)) {
    BCfg c = bselect_default(kind, P, Q, R);
    const int S = std::max(1, atoi(wgs)), BR = kBTileBR[c.tile];
    c.r_split = ((R + S - 1) / S + BR - 1) / BR * BR;
    c.S = (R + c.r_split - 1) / c.r_split;
    return c;
  }
  if (!e) return bselect_default(kind, P, Q, R);
  int t = 1, S = 1;
  sscanf(e, "%d,%d", &t, &S);
  t = std::max(0, std::min(t, (int)BTI_COUNT - 1));
  S = std::max(1, S);
  const int BR = kBTileBR[t];
  const int r_split = ((R + S - 1) / S + BR - 1) / BR * BR;
  return BCfg{t, (R + r_split - 1) / r_split, r_split};
}
#else
static BCfg bselect(int kind, int P, int Q, int R) { return bselect_default(kind, P, Q, R); }
#endif

size_t gemm_bf16_workspace_bytes(int kind, int P, int Q, int R) {
  const BCfg c = bselect(kind, P, Q, R);
  if (c.S <= 1) return 0;
  return (size_t)c.S * ((size_t)P * Q + P) * sizeof(float);
}

template <class T, int EPI, bool VA, bool VB>
static hipError_t blaunch_v(const BCfg& c, const GemmProblem& pr, const EpiArgs& ea, void* ws,
                            int vec_epi, hipStream_t s) {
  dim3 grid((pr.P + T::BP - 1) / T::BP, (pr.Q + T::BQ - 1) / T::BQ, c.S + c.cz);
  if constexpr (EPI == EPI_FWD) {
    if (pr.a_bf16) {
      if (!pr.b_bf16) return hipErrorInvalidValue;
      hipLaunchKernelGGL((gemm_bf16_kernel<T, EPI, VA, VB, true, true>), grid, dim3(T::NT), 0, s,
                         pr, ea, c.r_split, (float*)ws, vec_epi);
      return hipGetLastError();
    }
  }
  if (pr.b_bf16)
    hipLaunchKernelGGL((gemm_bf16_kernel<T, EPI, VA, VB, true, false>), grid, dim3(T::NT), 0, s, pr,
                       ea, c.r_split, (float*)ws, vec_epi);
  else
    hipLaunchKernelGGL((gemm_bf16_kernel<T, EPI, VA, VB, false, false>), grid, dim3(T::NT), 0, s, pr,
                       ea, c.r_split, (float*)ws, vec_epi);
  return hipGetLastError();
}

template <class T, int EPI>
static hipError_t blaunch_t(const BCfg& c, const GemmProblem& pr, const EpiArgs& ea, void* ws,
                            int vec_ops, int vec_epi, hipStream_t s) {
  switch (vec_ops) {
    case 3: return blaunch_v<T, EPI, true, true>(c, pr, ea, ws, vec_epi, s);
    case 1: return blaunch_v<T, EPI, true, false>(c, pr, ea, ws, vec_epi, s);
    case 2: return blaunch_v<T, EPI, false, true>(c, pr, ea, ws, vec_epi, s);
    default: return blaunch_v<T, EPI, false, false>(c, pr, ea, ws, vec_epi, s);
  }
}

template <int EPI>
static hipError_t blaunch_kind(const BCfg& c, const GemmProblem& pr, const EpiArgs& ea, void* ws,
                               int vec_ops, int vec_epi, hipStream_t s) {
  switch (c.tile) {
    case BTI_128x128: return blaunch_t<BT128x128, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
    case BTI_128x256: return blaunch_t<BT128x256, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
#ifdef OPFUSE_TUNING
    case BTI_128x128R64: return blaunch_t<BT128x128R64, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
    case BTI_128x256R32: return blaunch_t<BT128x256R32, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
    case BTI_256x128: return blaunch_t<BT256x128, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
    case BTI_256x256W8: return blaunch_t<BT256x256W8, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
    case BTI_256x256W4: return blaunch_t<BT256x256W4, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
#endif
    default: return blaunch_t<BT64x64, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
  }
}

static int bvec_flags(const GemmProblem& pr, int kind, const EpiArgs& ea, int* vec_epi) {
  const bool a_rc = (kind == EPI_FWD || kind == EPI_DGRAD);
  const bool b_rc = (kind == EPI_FWD);
  // fp32 quads: 16-byte aligned rows; bf16 quads: 8-byte aligned rows; bf16
  // octets (a bf16 operand whose reduction index is contiguous): 16-byte
  // aligned rows and a reduction extent that is a multiple of 8
  const int ga = pr.a_bf16 && a_rc ? 8 : 4, gb = pr.b_bf16 && b_rc ? 8 : 4;
  const bool a_al = pr.a_bf16 && !a_rc ? (((uintptr_t)pr.A & 7u) == 0) : aligned16(pr.A);
  const bool va = a_al && ((pr.a_sr == 1 ? pr.a_sp : pr.a_sr) % ga == 0) &&
                  ((a_rc ? pr.R : pr.P) % ga == 0);
  const bool b_al = pr.b_bf16 && !b_rc ? (((uintptr_t)pr.B & 7u) == 0) : aligned16(pr.B);
  const bool vb = b_al && ((pr.b_sr == 1 ? pr.b_sq : pr.b_sr) % gb == 0) &&
                  ((b_rc ? pr.R : pr.Q) % gb == 0);
  int ve = 0;
  if (aligned16(ea.out) && ea.ldo % 4 == 0 && (ea.z == nullptr || (aligned16(ea.z) && ea.ldz % 4 == 0)) &&
      (ea.yb == nullptr || ((uintptr_t)ea.yb & 7u) == 0) &&
      (ea.res == nullptr || (aligned16(ea.res) && ea.ldr % 4 == 0)) &&
      (ea.prev == nullptr || (aligned16(ea.prev) && ea.ldp % 4 == 0)))
    ve |= 1;
  if (kind == EPI_WGRAD_BF && aligned16(ea.W.w) && aligned16(ea.W.m) && ea.ldo % 4 == 0 &&
      (ea.opt.kind == OF_OPT_SGD || aligned16(ea.W.v)) && (ea.gW == nullptr || aligned16(ea.gW)) &&
      (ea.W.w_bf16 == nullptr || ((uintptr_t)ea.W.w_bf16 & 7u) == 0))
    ve |= 2;
  *vec_epi = ve;
  return (va ? 1 : 0) | (vb ? 2 : 0);
}

hipError_t gemm_bf16_launch(int kind, const GemmProblem& pr_in, const EpiArgs& ea_in, void* ws,
                            hipStream_t stream) {
  GemmProblem pr = pr_in;
#ifdef OPFUSE_TUNING
  // Tuning builds only: read a forward's A operand as bf16 (timing only).
  if (kind == EPI_FWD && getenv("OPFUSE_TUNE_ABF")) pr.a_bf16 = 1;
  if (getenv("OPFUSE_BF16_GROUP")) pr.group = atoi(getenv("OPFUSE_BF16_GROUP"));
#endif
  if ((pr.a_bf16 && kind != EPI_FWD) || pr.conv) return hipErrorInvalidValue;
  BCfg c = bselect(kind, pr.P, pr.Q, pr.R);
  EpiArgs ea = ea_in;
  ea.carry.cz = 0;
  if (ea.carry.t[0].p.w) {
    if (kind != EPI_FWD) return hipErrorInvalidValue;  // only a forward carries an update
    c.cz = carry_slices(ea.carry, bntiles(c.tile, pr.P, pr.Q));
    ea.carry.cz = c.cz;
  }
  int vec_epi = 0;
  const int vec_ops = bvec_flags(pr, kind, ea, &vec_epi);
  const int with_db = (kind == EPI_WGRAD || kind == EPI_WGRAD_BF) && ea.with_db;
  hipError_t e;
  switch (kind) {
    case EPI_FWD: e = blaunch_kind<EPI_FWD>(c, pr, ea, ws, vec_ops, vec_epi, stream); break;
    case EPI_DGRAD: e = blaunch_kind<EPI_DGRAD>(c, pr, ea, ws, vec_ops, vec_epi, stream); break;
    case EPI_WGRAD: e = blaunch_kind<EPI_WGRAD>(c, pr, ea, ws, vec_ops, vec_epi, stream); break;
    case EPI_WGRAD_BF: e = blaunch_kind<EPI_WGRAD_BF>(c, pr, ea, ws, vec_ops, vec_epi, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess || c.S <= 1) return e;
  const int64_t work = (int64_t)pr.P * ((pr.Q + 3) / 4);
  const int blocks = (int)std::min<int64_t>(2048, std::max<int64_t>(1, (work + 255) / 256));
  const dim3 g(blocks);
  switch (kind) {
    case EPI_FWD:
      hipLaunchKernelGGL(split_reduce_bf16_kernel<EPI_FWD>, g, dim3(256), 0, stream, pr.P, pr.Q,
                         c.S, ea, (const float*)ws, vec_epi, 0);
      break;
    case EPI_DGRAD:
      hipLaunchKernelGGL(split_reduce_bf16_kernel<EPI_DGRAD>, g, dim3(256), 0, stream, pr.P, pr.Q,
                         c.S, ea, (const float*)ws, vec_epi, 0);
      break;
    case EPI_WGRAD:
      hipLaunchKernelGGL(split_reduce_bf16_kernel<EPI_WGRAD>, g, dim3(256), 0, stream, pr.P, pr.Q,
                         c.S, ea, (const float*)ws, vec_epi, with_db);
      break;
    case EPI_WGRAD_BF:
      hipLaunchKernelGGL(split_reduce_bf16_kernel<EPI_WGRAD_BF>, g, dim3(256), 0, stream, pr.P,
                         pr.Q, c.S, ea, (const float*)ws, vec_epi, with_db);
      break;
  }
  return hipGetLastError();
}

}  // namespace opfuse
