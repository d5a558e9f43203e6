// fp32 MFMA contractions of a linear layer, with the optimizer fused into
// their prologue (forward-fusion) or epilogue (backward-fusion).
//
// One tiled kernel computes C[P,Q] = sum_r A(p,r) B(q,r) on the CDNA matrix
// cores (v_mfma_f32_32x32x2_f32).  A workgroup of 4 wavefronts owns a BP x BQ
// output tile; wavefronts split it WP x WQ and, when WR > 1, also split each
// reduction chunk (their partial tiles are summed in wave order).  Operand
// tiles go global -> registers -> LDS ([r][x] layout, double buffered); the
// next chunk's global loads are issued before the current chunk's MFMAs.
// A forward or data gradient on 32x32 tiles can instead load its operands
// straight into the matrix-core registers (gemm_direct_kernel, which runs
// v_mfma_f32_16x16x4_f32 on 16x16 sub-blocks).
// A grid-level split of the reduction (gridDim.z > 1) writes partial tiles to
// the workspace and a second kernel sums them in split order and runs the
// epilogue, so every result is deterministic and the same shape always uses
// the same tiling whatever the epilogue is.
//
// The three contractions of a linear layer (X [M,K], W [N,K], dZ [M,N]):
//   forward  C[m,n] = sum_k X[m,k] W[n,k]    P=M Q=N R=K  A,B reduction-contiguous
//   dgrad    C[m,k] = sum_n dZ[m,n] W[n,k]   P=M Q=K R=N  A red.-contig., B output-contig.
//   wgrad    C[n,k] = sum_m dZ[m,n] X[m,k]   P=N Q=K R=M  A,B output-contiguous
//
// Forward-fusion (Appendix B.1, Alg. 2): the B operand of the forward is W.
// When M fits one row tile (gridDim.x == 1) each W element is loaded by
// exactly one workgroup; that workgroup loads W, the pending gradient and the
// history, applies the update, writes them back, and puts the updated value
// into LDS for the MFMAs (Fig. 2: the update's write is merged with the next
// forward's read).  The bias update is done once per column tile by the
// split-0 workgroup.
//
// Backward-fusion (Appendix B.2, Alg. 3): the output of the wgrad is dW; its
// epilogue loads W and the history, applies the update with the accumulated
// tile as the gradient and writes them back; dW is never stored (Fig. 2: the
// gradient accumulation is merged with the optimizer's read).  The bias
// gradient is the column sum of the A tiles (dZ) the workgroups of column
// tile 0 already stage in LDS.

#include <algorithm>
#include <type_traits>
#include <cstdio>
#include <cstdlib>

#include "gemm_common.h"

namespace opfuse {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

template <int BP_, int BQ_, int BR_, int WP_, int WQ_, int WR_, int NS_, int PAD_ = 4>
struct Tile {
  static constexpr int BP = BP_, BQ = BQ_, BR = BR_, WP = WP_, WQ = WQ_, WR = WR_;
  // LDS row padding of the operand tiles (floats).  4 keeps rows 16-byte
  // aligned for the vector stores of output-contiguous operands; a tile whose
  // operands are both reduction-contiguous (stored one float at a time) may
  // take 2, which spreads its transposing stores over all 64 banks.
  static constexpr int PAD = PAD_;
  static constexpr int NS = NS_;  // operand chunks in the register ring
  static_assert(WP * WQ * WR == 4, "a workgroup is 4 wavefronts");
  static constexpr int WTP = BP / WP, WTQ = BQ / WQ;   // wavefront tile
  static constexpr int TP = WTP / 32, TQ = WTQ / 32;   // 32x32 MFMA blocks per wavefront
  static_assert(TP >= 1 && TQ >= 1 && WTP % 32 == 0 && WTQ % 32 == 0, "32x32 blocks");
  static constexpr int RW = BR / WR;                    // chunk rows per wavefront
  static_assert(RW % 2 == 0 && BR % 4 == 0, "k pairs");
  static constexpr int LDA = BP + PAD, LDB = BQ + PAD;
  static constexpr int LDC = (WR * BP * (BQ + 4) * 4 <= 60 * 1024) ? BQ + 4 : BQ;
  static constexpr int SM_MAIN = 2 * BR * (LDA + LDB);
  static constexpr int SM_C = WR * BP * LDC;
  static constexpr int SMX = SM_MAIN > SM_C ? SM_MAIN : SM_C;  // floats
  static_assert(SMX * 4 <= 64 * 1024, "LDS per workgroup");
};

// Tile menu (P x Q per workgroup, reduction chunk, wavefront split).
using T32x32 = Tile<32, 32, 32, 1, 1, 4, 4>;
using T64x32 = Tile<64, 32, 32, 2, 1, 2, 4>;
using T64x64 = Tile<64, 64, 16, 2, 2, 1, 4>;
using T128x64 = Tile<128, 64, 16, 2, 2, 1, 4>;
using T128x128 = Tile<128, 128, 16, 2, 2, 1, 3>;
using T256x32 = Tile<256, 32, 16, 4, 1, 1, 3>;
// 64 rows x 128 columns with the reduction layout of T64x32 (32-deep chunks,
// each halved between two wavefronts): every output element takes the same
// MFMA sequence as on T64x32, so results are identical to it bit for bit.
using T64x128 = Tile<64, 128, 32, 1, 2, 2, 4, 2>;

// TI_32x32D, TI_32x32D8: 32x32 blocks with operands loaded straight into the
// matrix-core registers by 4 or 8 wavefronts (gemm_direct_kernel; forward and
// data gradient of linear layers only, the LDS-staged 32x32 tile elsewhere).
enum TileId {
  TI_32x32 = 0, TI_64x32, TI_64x64, TI_128x64, TI_128x128, TI_256x32,
  TI_32x32D, TI_32x32D8, TI_64x128, TI_COUNT
};
static const int kTileBP[TI_COUNT] = {32, 64, 64, 128, 128, 256, 32, 32, 64};
static const int kTileBQ[TI_COUNT] = {32, 32, 64, 64, 128, 32, 32, 32, 128};
static const int kTileBR[TI_COUNT] = {32, 32, 16, 16, 16, 16, 32, 32, 32};


// A BX (output dim) x BR (reduction) tile of one operand, held in registers as
// float4s between its global load and its LDS store.  RC: the reduction index
// is contiguous in memory (else the output index is).  `base` points at the
// tile's first element; nx / nr are the valid extents from there (<= 0: none).
// vec: 128-bit loads (base 16B aligned, strides and both extents' ends
// multiples of 4 along the contiguous index).
template <int BX, int BR, bool RC, bool VEC, int PAD = 4>
struct TileLoad {
  static constexpr int NV = BX * BR / 4;
  static constexpr int PER = (NV + 255) / 256;
  float4 v[PER];

  __device__ __forceinline__ void load(const float* tensor, const GemmProblem&, int64_t s_x,
                                       int64_t s_r, int x0, int r0, int nx, int nr, int tid) {
    const rsrc_t rs = make_rsrc(tensor + (int64_t)x0 * s_x + (int64_t)r0 * s_r);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int idx = tid + i * 256;
      int x, r;
      if (RC) { x = idx / (BR / 4); r = (idx % (BR / 4)) * 4; }
      else    { r = idx / (BX / 4); x = (idx % (BX / 4)) * 4; }
      const bool live = NV % 256 == 0 || idx < NV;
      if constexpr (VEC) {
        const bool ok = live && x < nx && r < nr;
        const uint32_t off = ok ? (uint32_t)((x * s_x + r * s_r) * 4) : kOOB;
        v[i] = bload4(rs, off);
      } else {
        float e[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int xx = RC ? x : x + k, rr = RC ? r + k : r;
          const bool ok = live && xx < nx && rr < nr;
          e[k] = bload1(rs, ok ? (uint32_t)((xx * s_x + rr * s_r) * 4) : kOOB);
        }
        v[i] = make_float4(e[0], e[1], e[2], e[3]);
      }
    }
  }

  __device__ __forceinline__ void store(float* lds, int tid) const {
    constexpr int LD = BX + PAD;
    static_assert(RC || PAD % 4 == 0, "float4 stores need 16-byte aligned rows");
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int idx = tid + i * 256;
      if (NV % 256 == 0 || idx < NV) {
        if (RC) {
          const int x = idx / (BR / 4), r = (idx % (BR / 4)) * 4;
          lds[(r + 0) * LD + x] = v[i].x;
          lds[(r + 1) * LD + x] = v[i].y;
          lds[(r + 2) * LD + x] = v[i].z;
          lds[(r + 3) * LD + x] = v[i].w;
        } else {
          const int r = idx / (BX / 4), x = (idx % (BX / 4)) * 4;
          *reinterpret_cast<float4*>(&lds[r * LD + x]) = v[i];
        }
      }
    }
  }
};

// Convolution operands gathered from NHWC tensors / KRSC filters.  Element
// (x, r) of the tile is tensor element (x0 + x, r0 + r) of the implicit GEMM
// operand; its offset is formed from the convolution geometry, and elements in
// the zero padding (or past the operand) read from an out-of-range offset.
// VEC: the channel count along the contiguous index is a multiple of 4, so a
// float4 never straddles two filter taps.
enum GatherKind { G_FWD_A = 1, G_DGRAD_A = 2, G_WGRAD_B = 3, G_DGRAD_B = 4 };

template <int KIND>
__device__ __forceinline__ int64_t gather_off(const GemmProblem& g, int x, int r, bool& ok) {
  // FWD_A: x = m, r = k = (tap, c).  DGRAD_A: x = m, r = k = (tap, co).
  // WGRAD_B: x = k = (tap, c), r = m.  DGRAD_B: x = c, r = k = (tap, co).
  if constexpr (KIND == G_DGRAD_B) {
    const int tap = fdiv(r, g.dCout), co = r - tap * g.cCout;
    return ((int64_t)co * 9 + tap) * g.cC + x;
  } else {
    const int m = (KIND == G_WGRAD_B) ? r : x;
    const int k = (KIND == G_WGRAD_B) ? x : r;
    const int ch = (KIND == G_DGRAD_A) ? g.cCout : g.cC;
    const FastDiv& fch = (KIND == G_DGRAD_A) ? g.dCout : g.dC;
    const int t = fdiv(m, g.dW), w = m - t * g.cW;
    const int n = fdiv(t, g.dH), h = t - n * g.cH;
    const int tap = fdiv(k, fch), c = k - tap * ch;
    const int rr = tap / 3, ss = tap - 3 * rr;
    const int hi = (KIND == G_DGRAD_A) ? h + 1 - rr : h + rr - 1;
    const int wi = (KIND == G_DGRAD_A) ? w + 1 - ss : w + ss - 1;
    ok = ok && hi >= 0 && hi < g.cH && wi >= 0 && wi < g.cW;
    return (((int64_t)n * g.cH + hi) * g.cW + wi) * ch + c;
  }
}

template <int BX, int BR, bool RC, bool VEC, int KIND>
struct GatherLoad : TileLoad<BX, BR, RC, VEC> {
  using Base = TileLoad<BX, BR, RC, VEC>;
  using Base::v;
  __device__ __forceinline__ void load(const float* tensor, const GemmProblem& g, int64_t, int64_t,
                                       int x0, int r0, int nx, int nr, int tid) {
    const rsrc_t rs = make_rsrc(tensor);
#pragma unroll
    for (int i = 0; i < Base::PER; ++i) {
      const int idx = tid + i * 256;
      int x, r;
      if (RC) { x = idx / (BR / 4); r = (idx % (BR / 4)) * 4; }
      else    { r = idx / (BX / 4); x = (idx % (BX / 4)) * 4; }
      const bool live = idx < Base::NV;
      if constexpr (VEC) {
        bool ok = live && x < nx && r < nr;
        const int64_t o = gather_off<KIND>(g, x0 + x, r0 + r, ok);
        v[i] = bload4(rs, ok ? (uint32_t)(o * 4) : kOOB);
      } else {
        float e[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int xx = RC ? x : x + k, rr = RC ? r + k : r;
          bool ok = live && xx < nx && rr < nr;
          const int64_t o = gather_off<KIND>(g, x0 + xx, r0 + rr, ok);
          e[k] = bload1(rs, ok ? (uint32_t)(o * 4) : kOOB);
        }
        v[i] = make_float4(e[0], e[1], e[2], e[3]);
      }
    }
  }
};

// Forward-fusion B operand: W tile (reduction-contiguous) with its pending
// update.  load() issues the loads of W, g, m, v; apply() runs after the
// previous chunk's MFMAs, updates, writes back and stages the new W in LDS.
// `off` is relative to the tile's first element (row stride ldw).
template <int BX, int BR, bool VEC>
struct FFTileLoad {
  static constexpr int NV = BX * BR / 4;
  static constexpr int PER = (NV + 255) / 256;
  float4 w[PER], g[PER], m[PER], v[PER];
  int valid[PER];  // bit e set: element e of the float4 is inside the matrix
  int64_t base;    // element index of the tile origin in W

  __device__ __forceinline__ void load(const EpiArgs& ea, int64_t ldw, int x0, int r0, int nx,
                                       int nr, int tid) {
    const bool adam = ea.opt.kind != OF_OPT_SGD;
    base = (int64_t)x0 * ldw + r0;
    const rsrc_t rw = make_rsrc(ea.W.w + base), rg = make_rsrc(ea.gW + base);
    const rsrc_t rm = make_rsrc_opt(ea.W.m, base);
    const rsrc_t rv = adam ? make_rsrc(ea.W.v + base) : rm;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int idx = tid + i * 256;
      const int x = idx / (BR / 4), r = (idx % (BR / 4)) * 4;
      const bool live = idx < NV && x < nx;
      if constexpr (VEC) {
        const bool ok = live && r < nr;
        valid[i] = ok ? 0xf : 0;
        const uint32_t off = ok ? (uint32_t)((x * ldw + r) * 4) : kOOB;
        w[i] = bload4(rw, off);
        g[i] = bload4(rg, off);
        m[i] = bload4(rm, off);
        v[i] = bload4(rv, off);
      } else {
        float ew[4], eg[4], em[4], ev[4];
        valid[i] = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const bool ok = live && r + k < nr;
          valid[i] |= ok ? (1 << k) : 0;
          const uint32_t off = ok ? (uint32_t)((x * ldw + r + k) * 4) : kOOB;
          ew[k] = bload1(rw, off);
          eg[k] = bload1(rg, off);
          em[k] = bload1(rm, off);
          ev[k] = bload1(rv, off);
        }
        w[i] = make_float4(ew[0], ew[1], ew[2], ew[3]);
        g[i] = make_float4(eg[0], eg[1], eg[2], eg[3]);
        m[i] = make_float4(em[0], em[1], em[2], em[3]);
        v[i] = make_float4(ev[0], ev[1], ev[2], ev[3]);
      }
    }
  }

  // owner: this workgroup writes the updated values (to ea.Wout when set, else
  // in place); every workgroup feeds them to its MFMAs.
  __device__ __forceinline__ void apply(const EpiArgs& ea, int64_t ldw, float* lds, int tid,
                                        bool owner) {
    constexpr int LD = BX + 4;
    const bool adam = ea.opt.kind != OF_OPT_SGD;
    const of_param& out = ea.Wout.w ? ea.Wout : ea.W;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int idx = tid + i * 256;
      if (idx >= NV) continue;
      const int x = idx / (BR / 4), r = (idx % (BR / 4)) * 4;
      const int64_t o = base + (int64_t)x * ldw + r;
      float* pw = reinterpret_cast<float*>(&w[i]);
      float* pg = reinterpret_cast<float*>(&g[i]);
      float* pm = reinterpret_cast<float*>(&m[i]);
      float* pv = reinterpret_cast<float*>(&v[i]);
      if (valid[i] == 0xf && ((uintptr_t)(out.w + o) & 15u) == 0) {
        for (int e = 0; e < 4; ++e) opt_update(ea.opt, pw[e], pg[e], pm[e], pv[e]);
        if (owner) {
          st4(out.w + o, w[i]);
          if (out.m) st4(out.m + o, m[i]);
          if (adam) st4(out.v + o, v[i]);
          if (out.w_bf16) st_bf16x4(out.w_bf16 + o, w[i]);
        }
      } else if (valid[i]) {
        for (int e = 0; e < 4; ++e) {
          if (valid[i] & (1 << e)) {
            opt_update(ea.opt, pw[e], pg[e], pm[e], pv[e]);
            if (owner) {
              out.w[o + e] = pw[e];
              if (out.m) out.m[o + e] = pm[e];
              if (adam) out.v[o + e] = pv[e];
              if (out.w_bf16) out.w_bf16[o + e] = f32_to_bf16(pw[e]);
            }
          }
        }
      }
      lds[(r + 0) * LD + x] = w[i].x;
      lds[(r + 1) * LD + x] = w[i].y;
      lds[(r + 2) * LD + x] = w[i].z;
      lds[(r + 3) * LD + x] = w[i].w;
    }
  }
};

// -------------------------------------------------------------------- kernel
// VECS: bit 0 -- 128-bit loads of A allowed, bit 1 -- of B.
template <class T, int EPI, int VECS, bool CONV>
__global__ __launch_bounds__(256) void gemm_kernel(GemmProblem pr, EpiArgs ea, int r_split,
                                                   float* partial, int vec_epi) {
  constexpr bool VA = (VECS & 1) != 0, VB = (VECS & 2) != 0;
  constexpr bool A_RC = (EPI == EPI_FWD || EPI == EPI_FWD_FF || EPI == EPI_DGRAD);
  constexpr bool B_RC = (EPI == EPI_FWD || EPI == EPI_FWD_FF);
  constexpr bool WG = (EPI == EPI_WGRAD || EPI == EPI_WGRAD_BF);
  // Forward-fusion also keeps the updated bias slice of its column tile.
  constexpr int SMEM = T::SMX + (EPI == EPI_FWD_FF ? T::BQ : 0);
  static_assert(SMEM * 4 <= 160 * 1024, "LDS per workgroup");
  static_assert(EPI != EPI_FWD_FF || T::PAD == 4, "the fused forward stages W with a pad of 4");
  __shared__ __attribute__((aligned(16))) float smem[SMEM];
  if constexpr (EPI == EPI_FWD) {
    if ((int)blockIdx.z < ea.carry.cz) {
      carry_update(ea.carry);  // a later operator's update rides on this launch
      return;
    }
  }

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wp = wave % T::WP, wq = (wave / T::WP) % T::WQ, wr = wave / (T::WP * T::WQ);
  int tx, ty;
  xcd_tile(tx, ty);
  const int p0 = tx * T::BP, q0 = ty * T::BQ;
  const int split = (int)blockIdx.z - ea.carry.cz, S = (int)gridDim.z - ea.carry.cz;
  const int rbeg = split * r_split;
  const int rend = min(pr.R, rbeg + r_split);
  const int nch = (rend - rbeg + T::BR - 1) / T::BR;
  const bool do_db = WG && ea.with_db && ty == 0;
  // forward-fusion: the workgroup that writes the updated W tile (all of them
  // when each W tile has one row tile; row tile 0 when it goes to Wout)
  const bool ff_owner = ea.Wout.w == nullptr || p0 == 0;

  // Buffer b (0/1) of the A and B tiles: A at b*STAGE, B at b*STAGE + BR*LDA.
  constexpr int STAGE = T::BR * (T::LDA + T::LDB);
  constexpr int BOFF = T::BR * T::LDA;
  float* bias_s = smem + T::SMX;  // valid for forward-fusion only

  floatx16 acc[T::TP][T::TQ];
#pragma unroll
  for (int i = 0; i < T::TP; ++i)
#pragma unroll
    for (int j = 0; j < T::TQ; ++j)
#pragma unroll
      for (int k = 0; k < 16; ++k) acc[i][j][k] = 0.f;

  // Epilogue operands of small tiles are loaded during the main loop so their
  // latency hides behind it: the parameter and history tile of backward-fusion
  // (this workgroup is their only reader and writer) and the previous layer's
  // saved tensor of the data gradient.  They are issued after the first
  // operand chunks, which are then not queued behind them.  Thread t handles
  // the float4 items t, t+256, ... of the tile in row-major order.
  constexpr int NQ4 = T::BQ / 4;
  constexpr int ITEMS = T::BP * NQ4;
  constexpr int EPT = (ITEMS + 255) / 256;
  constexpr bool PREF_BF = (EPI == EPI_WGRAD_BF) && EPT <= 2;
  constexpr bool PREF_DG = (EPI == EPI_DGRAD) && EPT <= 4;
  constexpr int NPF = (PREF_BF || PREF_DG) ? EPT : 1;
  float4 pf_w[NPF], pf_m[NPF], pf_v[NPF];
  const bool pref = (PREF_BF && S == 1 && (vec_epi & 2) && ea.gW == nullptr) ||
                    (PREF_DG && S == 1 && (vec_epi & 1) && ea.act != OF_ACT_NONE &&
                     ea.res == nullptr);
  auto prefetch = [&]() {
    if constexpr (PREF_BF || PREF_DG) {
      if (pref) {
        const int64_t ld = PREF_BF ? ea.ldo : ea.ldp;
        const int64_t org = (int64_t)p0 * ld + q0;
        const rsrc_t r0 = make_rsrc(PREF_BF ? ea.W.w + org : ea.prev + org);
        const rsrc_t r1 = PREF_BF ? make_rsrc_opt(ea.W.m, org) : make_rsrc(ea.prev + org);
        const rsrc_t r2 = (PREF_BF && ea.opt.kind != OF_OPT_SGD) ? make_rsrc(ea.W.v + org) : r1;
#pragma unroll
        for (int e = 0; e < EPT; ++e) {
          const int idx = tid + e * 256;
          const int p = idx / NQ4, q = (idx % NQ4) * 4;
          const bool ok = idx < ITEMS && p0 + p < pr.P && q0 + q + 3 < pr.Q;
          const uint32_t off = ok ? (uint32_t)((p * ld + q) * 4) : kOOB;
          pf_w[e] = bload4(r0, off);
          if constexpr (PREF_BF) {
            pf_m[e] = bload4(r1, off);
            pf_v[e] = bload4(r2, off);
          }
        }
      }
    }
  };

  // Register ring of NS operand chunks: the loads of chunk c+NS-1 are issued
  // before chunk c is stored to LDS and multiplied, so NS-1 chunks are in
  // flight per workgroup.  The loop runs to a multiple of NS; chunks past the
  // end load nothing (every offset out of range) and skip the MFMAs.
  // Forward-fusion holds four arrays per stage and keeps a two-stage ring.
  constexpr int NS = (EPI == EPI_FWD_FF) ? 2 : T::NS;
  using ALoad = std::conditional_t<
      CONV && (EPI == EPI_FWD || EPI == EPI_FWD_FF || EPI == EPI_DGRAD),
      GatherLoad<T::BP, T::BR, true, VA, EPI == EPI_DGRAD ? G_DGRAD_A : G_FWD_A>,
      TileLoad<T::BP, T::BR, A_RC, VA, T::PAD>>;
  using BLoad = std::conditional_t<
      CONV && EPI == EPI_DGRAD, GatherLoad<T::BQ, T::BR, false, VB, G_DGRAD_B>,
      std::conditional_t<CONV && WG, GatherLoad<T::BQ, T::BR, false, VB, G_WGRAD_B>,
                         TileLoad<T::BQ, T::BR, B_RC, VB, T::PAD>>>;
  ALoad la[NS];
  BLoad lb[(EPI == EPI_FWD_FF) ? 1 : NS];
  FFTileLoad<T::BQ, T::BR, VB> lf[(EPI == EPI_FWD_FF) ? NS : 1];
  const int64_t ldw = pr.b_sq;  // FF: W row stride (= K)
  const int np = pr.P - p0, nq = pr.Q - q0;

  float dbsum = 0.f;

  auto issue = [&](int slot, int c) {
    const int r0 = rbeg + c * T::BR;
    const int nr = c < nch ? rend - r0 : 0;
    la[slot].load(pr.A, pr, pr.a_sp, pr.a_sr, p0, r0, np, nr, tid);
    if constexpr (EPI == EPI_FWD_FF)
      lf[slot].load(ea, ldw, q0, r0, nq, nr, tid);
    else
      lb[slot].load(pr.B, pr, pr.b_sq, pr.b_sr, q0, r0, nq, nr, tid);
  };

  // One chunk's MFMAs on the operands in LDS buffer `buf`.
  auto mfma_chunk = [&](const float* buf) {
    const float* a_s = buf;
    const float* b_s = buf + BOFF;
#pragma unroll
    for (int kk = 0; kk < T::RW; kk += 2) {
      const int r = wr * T::RW + kk + (lane >> 5);
      float a[T::TP], b[T::TQ];
#pragma unroll
      for (int i = 0; i < T::TP; ++i)
        a[i] = a_s[r * T::LDA + wp * T::WTP + i * 32 + (lane & 31)];
#pragma unroll
      for (int j = 0; j < T::TQ; ++j)
        b[j] = b_s[r * T::LDB + wq * T::WTQ + j * 32 + (lane & 31)];
#pragma unroll
      for (int i = 0; i < T::TP; ++i)
#pragma unroll
        for (int j = 0; j < T::TQ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  };

  // Pipelined main loop (every contraction but the fused forward, whose W
  // tiles are updated between load and staging): the matrix cores stay fed
  // across chunks, which matters most where one wavefront per SIMD has
  // nothing else to hide latency behind.
  //  * every operand of chunk c is read from LDS first, into registers of
  //    its own, so one LDS latency is exposed per chunk rather than one per
  //    pair of reduction rows;
  //  * chunk c+1 is stored to the other LDS buffer, and chunk c+NS's global
  //    loads are issued, between chunk c's MFMAs;
  //  * one barrier per chunk: buffer c&1 is written again (chunk c+2) only
  //    after every wavefront passed the barrier that follows its reads.
  // The MFMA sequence of each output, and the order of the bias-gradient
  // sums, are those of the loop further below.
  constexpr bool PIPE = (EPI != EPI_FWD_FF);
  if constexpr (PIPE) {
    constexpr int KS = T::RW / 2;
    constexpr int NM = KS * T::TP * T::TQ;                  // MFMAs per chunk
    constexpr int NLD = (VA ? 1 : 4) * ALoad::PER + (VB ? 1 : 4) * BLoad::PER;  // global loads
    constexpr int NST = (A_RC ? 2 : 1) * ALoad::PER + (B_RC ? 2 : 1) * BLoad::PER;  // LDS stores
    constexpr int NG = NM >= 8 ? NM / 4 - 1 : 1;           // interleave groups
    constexpr int GL = (NLD + NG - 1) / NG, GS = (NST + NG - 1) / NG;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      issue(s, s);
      __builtin_amdgcn_sched_barrier(0);
    }
    prefetch();
    if (EPI == EPI_WGRAD_BF) opt_prepare(ea.opt);
    la[0].store(smem, tid);
    lb[0].store(smem + BOFF, tid);
    __syncthreads();
    // Chunk c from slot s (s == c % NS, a constant after unrolling).
    auto chunk = [&](const int c, const int s) {
      const float* a_s = smem + (c & 1) * STAGE;
      const float* b_s = a_s + BOFF;
      float a[KS][T::TP], b[KS][T::TQ];
#pragma unroll
      for (int k = 0; k < KS; ++k) {
        const int r = wr * T::RW + 2 * k + (lane >> 5);
#pragma unroll
        for (int i = 0; i < T::TP; ++i)
          a[k][i] = a_s[r * T::LDA + wp * T::WTP + i * 32 + (lane & 31)];
#pragma unroll
        for (int j = 0; j < T::TQ; ++j)
          b[k][j] = b_s[r * T::LDB + wq * T::WTQ + j * 32 + (lane & 31)];
      }
      if (do_db && tid < T::BP) {
        // Column sums of dZ for this tile's output rows, in reduction order.
#pragma unroll 4
        for (int r = 0; r < T::BR; ++r) dbsum = __fadd_rn(dbsum, a_s[r * T::LDA + tid]);
      }
      __builtin_amdgcn_sched_barrier(0);
      issue(s, c + NS);   // slot s held chunk c, already in LDS
      float* nbuf = smem + ((c + 1) & 1) * STAGE;
      la[(s + 1) % NS].store(nbuf, tid);
      lb[(s + 1) % NS].store(nbuf + BOFF, tid);
#pragma unroll
      for (int k = 0; k < KS; ++k)
#pragma unroll
        for (int i = 0; i < T::TP; ++i)
#pragma unroll
          for (int j = 0; j < T::TQ; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[k][i], b[k][j], acc[i][j], 0, 0, 0);
      // 4 MFMAs, then a share of the global loads and of the LDS stores, in
      // each group; the last MFMAs cover the stores' completion before the
      // barrier and, after it, the next chunk's LDS reads
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        __builtin_amdgcn_sched_group_barrier(0x008, NM >= 8 ? 4 : NM, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, GL, 0);
        __builtin_amdgcn_sched_group_barrier(0x200, GS, 0);
      }
      if constexpr (NM >= 8) __builtin_amdgcn_sched_group_barrier(0x008, NM - 4 * NG, 0);
      __syncthreads();
    };
    // Whole rounds of NS chunks without a branch between them, so each
    // chunk's LDS reads can start among the previous chunk's last MFMAs; then
    // the remainder.
    const int nfull = nch / NS * NS;
    for (int c0 = 0; c0 < nfull; c0 += NS) {
#pragma unroll
      for (int s = 0; s < NS; ++s) chunk(c0 + s, s);
    }
#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
      if (nfull + s < nch) chunk(nfull + s, s);
  }

  // In-order prologue (the scheduling barriers keep chunk 0 oldest), so the
  // loop waits for one chunk at a time instead of draining the ring.
#pragma unroll
  for (int s = 0; s < NS - 1; ++s) {
    if constexpr (PIPE) break;
    issue(s, s);
    __builtin_amdgcn_sched_barrier(0);
  }
  if constexpr (!PIPE) {
    prefetch();
    // (after the loads above are in flight, so their latency hides this)
    if (EPI == EPI_FWD_FF || EPI == EPI_WGRAD_BF) opt_prepare(ea.opt);
  }

  for (int c0 = 0; c0 < (PIPE ? 0 : nch); c0 += NS) {
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const int c = c0 + s;
      issue((s + NS - 1) % NS, c + NS - 1);
      float* buf = smem + (c & 1) * STAGE;
      la[s].store(buf, tid);
      if constexpr (EPI == EPI_FWD_FF) {
        if (c < nch) lf[s].apply(ea, ldw, buf + BOFF, tid, ff_owner);
      } else {
        lb[s].store(buf + BOFF, tid);
      }
      __syncthreads();
      if (c < nch) {
        const float* a_s = buf;
        mfma_chunk(buf);
        if (do_db && tid < T::BP) {
          // Column sums of dZ for this tile's output rows, in reduction order.
#pragma unroll 4
          for (int r = 0; r < T::BR; ++r) dbsum = __fadd_rn(dbsum, a_s[r * T::LDA + tid]);
        }
      }
    }
  }
  // Every wavefront is done with the operand buffers before they are reused.
  __syncthreads();

  // Stage the accumulators (MFMA 32x32 layout: lane holds column lane%32 and
  // rows 8*(k/4) + 4*(lane/32) + k%4) through LDS in row-major order.
  float* Cs = smem;
#pragma unroll
  for (int i = 0; i < T::TP; ++i)
#pragma unroll
    for (int j = 0; j < T::TQ; ++j)
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const int p = wp * T::WTP + i * 32 + (k >> 2) * 8 + (lane >> 5) * 4 + (k & 3);
        const int q = wq * T::WTQ + j * 32 + (lane & 31);
        Cs[(wr * T::BP + p) * T::LDC + q] = acc[i][j][k];
      }

  // Forward-fusion bias: the split-0 workgroups compute the update; it is
  // written once per column tile (by row tile 0 when the update goes to a
  // second buffer set, else by the only row tile).
  const bool ff_bias = (EPI == EPI_FWD_FF) && ea.b.w != nullptr;
  if (ff_bias && split == 0 && tid < T::BQ && q0 + tid < pr.Q) {
    const int i = q0 + tid;
    const bool adam = ea.opt.kind != OF_OPT_SGD;
    float w = ea.b.w[i], m = ea.b.m ? ea.b.m[i] : 0.f, v = adam ? ea.b.v[i] : 0.f;
    opt_update(ea.opt, w, ea.gb[i], m, v);
    if (ff_owner) {
      const of_param& out = ea.bout.w ? ea.bout : ea.b;
      out.w[i] = w;
      if (out.m) out.m[i] = m;
      if (adam) out.v[i] = v;
      if (out.w_bf16) out.w_bf16[i] = f32_to_bf16(w);
    }
    bias_s[tid] = w;
  }
  __syncthreads();

  const float* bias_base = nullptr;
  if (EPI == EPI_FWD) bias_base = ea.bias;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int idx = tid + e * 256;
    if (idx >= ITEMS) break;
    const int p = idx / NQ4, q = (idx % NQ4) * 4;
    const int gp = p0 + p, gq = q0 + q;
    if (gp >= pr.P || gq >= pr.Q) continue;
    float c[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float s = Cs[p * T::LDC + q + e];
#pragma unroll
      for (int w2 = 1; w2 < T::WR; ++w2) s = __fadd_rn(s, Cs[(w2 * T::BP + p) * T::LDC + q + e]);
      c[e] = s;
    }
    const int n = min(4, pr.Q - gq);
    if (S > 1) {
      float* dst = partial + ((int64_t)split * pr.P + gp) * pr.Q + gq;
      if (n == 4 && (pr.Q & 3) == 0) st4(dst, make_float4(c[0], c[1], c[2], c[3]));
      else for (int e = 0; e < n; ++e) dst[e] = c[e];
    } else if (pref && n == 4) {
      if constexpr (PREF_BF) {
        // backward-fusion with the parameter tile already in registers
        float4 w = pf_w[e], m = pf_m[e], v = pf_v[e];
        opt_update(ea.opt, w.x, c[0], m.x, v.x);
        opt_update(ea.opt, w.y, c[1], m.y, v.y);
        opt_update(ea.opt, w.z, c[2], m.z, v.z);
        opt_update(ea.opt, w.w, c[3], m.w, v.w);
        const int64_t oo = (int64_t)gp * ea.ldo + gq;
        st4(ea.W.w + oo, w);
        if (ea.W.m) st4(ea.W.m + oo, m);
        if (ea.opt.kind != OF_OPT_SGD) st4(ea.W.v + oo, v);
        if (ea.W.w_bf16) st_bf16x4(ea.W.w_bf16 + oo, w);
      } else if constexpr (PREF_DG) {
        const float4 sv = pf_w[e];
        const float4 r = make_float4(__fmul_rn(c[0], act_grad(ea.act, sv.x)),
                                     __fmul_rn(c[1], act_grad(ea.act, sv.y)),
                                     __fmul_rn(c[2], act_grad(ea.act, sv.z)),
                                     __fmul_rn(c[3], act_grad(ea.act, sv.w)));
        st4(ea.out + (int64_t)gp * ea.ldo + gq, r);
      }
    } else {
      const float* bias = nullptr;
      if (EPI == EPI_FWD && bias_base) bias = bias_base + gq;
      if (EPI == EPI_FWD_FF && ff_bias) bias = bias_s + q;
      epilogue<EPI>(ea, gp, gq, c, n, bias, vec_epi);
    }
  }
  if (do_db && tid < T::BP && p0 + tid < pr.P) {
    if (S > 1) partial[(int64_t)S * pr.P * pr.Q + (int64_t)split * pr.P + p0 + tid] = dbsum;
    else bias_epilogue<EPI>(ea, p0 + tid, dbsum);
  }
}

// ------------------------------------------------------- direct 32x32 tiles
// One 32x32 output block per workgroup of NW wavefronts, for the forward and
// the data gradient.  Operands go from memory straight into the MFMA operand
// registers (no LDS staging).  Each wave runs v_mfma_f32_16x16x4_f32 on the
// 2x2 sub-blocks of 16x16.  The waves split the reduction into blocks of 16
// elements and wave w takes blocks w, w+NW, w+2NW, ... of its split; lane
// (row, g), g = lane/16, holds elements 16b+4g .. 16b+4g+3 of rows row and
// row+16 of A and of B, and MFMA step e pairs element e of the four groups
// (the same pairing for A and B, so every product of a block is summed
// exactly once).  Four lanes share each row, so a 128-bit load reads 64
// contiguous bytes per row.  A reduction-contiguous operand takes one 128-bit
// load per row and block, the other kind four 32-bit loads that are coalesced
// across the lanes.  NS blocks are in flight per wave.  The NW partial tiles
// are summed in wave order through LDS before the epilogue.
template <int EPI, int NW, int NS, int VECS>
__global__ __launch_bounds__(64 * NW) void gemm_direct_kernel(GemmProblem pr, EpiArgs ea,
                                                              int r_split, float* partial,
                                                              int vec_epi) {
  static_assert(EPI == EPI_FWD || EPI == EPI_DGRAD, "forward and data gradient only");
  static_assert(NW >= 4 && NW <= 16 && NS >= 2, "shape");
  constexpr bool VA = (VECS & 1) != 0, VB = (VECS & 2) != 0;
  constexpr bool B_RC = (EPI == EPI_FWD);  // dgrad: W is output-contiguous
  constexpr int KB = 16;                   // reduction elements per block
  __shared__ __attribute__((aligned(16))) float Cs[NW * 32 * 32];
  if constexpr (EPI == EPI_FWD) {
    if ((int)blockIdx.z < ea.carry.cz) {
      carry_update(ea.carry);  // a later operator's update rides on this launch
      return;
    }
  }

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int tx, ty;
  xcd_tile(tx, ty);
  const int p0 = tx * 32, q0 = ty * 32;
  const int split = (int)blockIdx.z - ea.carry.cz, S = (int)gridDim.z - ea.carry.cz;
  const int rbeg = split * r_split;
  const int rend = min(pr.R, rbeg + r_split);
  const int np = pr.P - p0, nq = pr.Q - q0;

  // Epilogue item of thread tid < 256: row ep, columns eq .. eq+3 of the block.
  // The data gradient loads its saved tensor (for act') before the main loop.
  const int ep = tid >> 3, eq = (tid & 7) * 4;
  const bool pref = EPI == EPI_DGRAD && S == 1 && (vec_epi & 1) && ea.act != OF_ACT_NONE &&
                    ea.res == nullptr;
  float4 pf = make_float4(0.f, 0.f, 0.f, 0.f);
  if (pref) {
    const bool ok = tid < 256 && ep < np && eq + 3 < nq;
    const rsrc_t rp = make_rsrc(ea.prev + (int64_t)p0 * ea.ldp + q0);
    pf = bload4(rp, ok ? (uint32_t)((ep * ea.ldp + eq) * 4) : kOOB);
  }

  const int row = lane & 15, grp = lane >> 4;
  const int nr = rend - rbeg;
  const int nblk = (nr + KB - 1) / KB;
  const int myblk = nblk > wave ? (nblk - wave + NW - 1) / NW : 0;
  const rsrc_t rsa = make_rsrc(pr.A + (int64_t)p0 * pr.a_sp + (int64_t)rbeg * pr.a_sr);
  const rsrc_t rsb = make_rsrc(pr.B + (int64_t)q0 * pr.b_sq + (int64_t)rbeg * pr.b_sr);
  auto ld = [&](const rsrc_t& rs, int64_t s_x, int64_t s_r, bool rc, bool vec, int x, int nx,
                int r) -> float4 {
    if (rc && vec) {
      const bool ok = x < nx && r < nr;
      return bload4(rs, ok ? (uint32_t)((x * s_x + r) * 4) : kOOB);
    }
    float e[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const bool ok = x < nx && r + k < nr;
      e[k] = bload1(rs, ok ? (uint32_t)((x * s_x + (r + k) * s_r) * 4) : kOOB);
    }
    return make_float4(e[0], e[1], e[2], e[3]);
  };
  float4 ra[NS][2], rb[NS][2];  // [slot][row half]
  auto dload = [&](int slot, int i) {
    const int r = KB * (wave + NW * i) + 4 * grp;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      ra[slot][hh] = ld(rsa, pr.a_sp, pr.a_sr, true, VA, row + 16 * hh, np, r);
      rb[slot][hh] = ld(rsb, pr.b_sq, pr.b_sr, B_RC, VB, row + 16 * hh, nq, r);
    }
  };

  floatx4 acc[2][2];  // sub-block (row half of A, row half of B)
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[a][b][k] = 0.f;
  // Blocks past this wave's last one load nothing (every offset out of range).
  // The prologue issues the blocks in order (the scheduling barriers keep it
  // so): the loop head then waits only for the oldest block, not for the whole
  // ring, which it would if block 0 were issued last.
#pragma unroll
  for (int s = 0; s < NS - 1; ++s) {
    dload(s, s);
    __builtin_amdgcn_sched_barrier(0);
  }
  for (int i0 = 0; i0 < myblk; i0 += NS) {
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const int i = i0 + s;
      dload((s + NS - 1) % NS, i + NS - 1);
      if (i < myblk) {
        const float av[2][4] = {{ra[s][0].x, ra[s][0].y, ra[s][0].z, ra[s][0].w},
                                {ra[s][1].x, ra[s][1].y, ra[s][1].z, ra[s][1].w}};
        const float bv[2][4] = {{rb[s][0].x, rb[s][0].y, rb[s][0].z, rb[s][0].w},
                                {rb[s][1].x, rb[s][1].y, rb[s][1].z, rb[s][1].w}};
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b)
              acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[a][e], bv[b][e], acc[a][b], 0, 0, 0);
      }
    }
  }

  // Partial tile of wave w at Cs[w][32][32] (MFMA 16x16 layout: lane holds
  // column lane%16 and rows 4*(lane/16) + k of its sub-block).
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int k = 0; k < 4; ++k)
        Cs[(wave * 32 + 16 * a + 4 * grp + k) * 32 + 16 * b + row] = acc[a][b][k];
  __syncthreads();
  if (tid >= 256) return;
  const int gp = p0 + ep, gq = q0 + eq;
  if (gp >= pr.P || gq >= pr.Q) return;
  float4 sum = *reinterpret_cast<const float4*>(Cs + ep * 32 + eq);
#pragma unroll
  for (int w = 1; w < NW; ++w) {
    const float4 t = *reinterpret_cast<const float4*>(Cs + (w * 32 + ep) * 32 + eq);
    sum.x = __fadd_rn(sum.x, t.x); sum.y = __fadd_rn(sum.y, t.y);
    sum.z = __fadd_rn(sum.z, t.z); sum.w = __fadd_rn(sum.w, t.w);
  }
  const float c[4] = {sum.x, sum.y, sum.z, sum.w};
  const int n = min(4, pr.Q - gq);
  if (S > 1) {
    float* dst = partial + ((int64_t)split * pr.P + gp) * pr.Q + gq;
    if (n == 4 && (pr.Q & 3) == 0) st4(dst, sum);
    else for (int e = 0; e < n; ++e) dst[e] = c[e];
  } else if (pref && n == 4) {
    const float4 r = make_float4(__fmul_rn(c[0], act_grad(ea.act, pf.x)),
                                 __fmul_rn(c[1], act_grad(ea.act, pf.y)),
                                 __fmul_rn(c[2], act_grad(ea.act, pf.z)),
                                 __fmul_rn(c[3], act_grad(ea.act, pf.w)));
    st4(ea.out + (int64_t)gp * ea.ldo + gq, r);
  } else {
    const float* bias = (EPI == EPI_FWD && ea.bias) ? ea.bias + gq : nullptr;
    epilogue<EPI>(ea, gp, gq, c, n, bias, vec_epi);
  }
}

// Sum the split partials (8 lanes per output item for long split lists),
// then run the epilogue.
template <int EPI>
__global__ __launch_bounds__(256) void split_reduce_coop_kernel(int P, int Q, int S, EpiArgs ea,
                                                                const float* __restrict__ partial,
                                                                int vec_epi, int with_db) {
  split_reduce_coop_body<EPI>(P, Q, S, ea, partial, vec_epi, with_db);
}

// Sum the split partials in split order, then run the epilogue.
template <int EPI>
__global__ __launch_bounds__(256) void split_reduce_kernel(int P, int Q, int S, EpiArgs ea,
                                                           const float* __restrict__ partial,
                                                           int vec_epi, int with_db) {
  split_reduce_body<EPI>(P, Q, S, ea, partial, vec_epi, with_db);
}


// --------------------------------------------------------------- host side
struct GemmCfg {
  int tile;
  int S;        // grid-level reduction splits
  int r_split;  // reduction elements per split (multiple of the tile's BR)
  int cz = 0;   // z-slices of carried-update workgroups after the splits
};

static int64_t ntiles(int t, int P, int Q) {
  return (int64_t)((P + kTileBP[t] - 1) / kTileBP[t]) * ((Q + kTileBQ[t] - 1) / kTileBQ[t]);
}

// Tiling by contraction kind and shape (measured on MI355X):
//   * the eager and backward-fusion weight gradients share one rule, so their
//     accumulated sums are identical;
//   * forward-fusion needs one row tile to cover all of M (each W element is
//     loaded, updated and written by exactly one workgroup); the plain forward
//     uses that same tiling while M <= 64 and its own faster one above.
static GemmCfg make_cfg(int t, int P, int Q, int R, int64_t target_ctas, int max_s) {
  const int BR = kTileBR[t];
  const int64_t nt = ntiles(t, P, Q);
  int S = (int)std::max<int64_t>(1, (target_ctas + nt - 1) / nt);
  const int maxS = std::max(1, R / (4 * BR));  // at least 4 chunks per split
  S = std::min(S, std::min(maxS, max_s));
  int r_split = (((R + S - 1) / S) + BR - 1) / BR * BR;
  S = (R + r_split - 1) / r_split;
  return GemmCfg{t, S, r_split};
}

static int ff_tile(int P) { return P <= 32 ? TI_32x32 : TI_64x32; }

static GemmCfg select_cfg_default(int kind, int P, int Q, int R) {
  // The forward and the fused forward of at most 64 rows share one tiling (the
  // same tile, splits and split length), so their results are bit-identical;
  // about 1024 workgroups (measured on MI355X at 64 x 8192 x 8192: fused
  // forward 416 us with 4 splits, 435 us with 2).  One row tile covers the M
  // rows, so the update can be written in place.  A fused forward of more
  // rows writes its update to a second buffer set (every row tile computes it,
  // row tile 0 stores it) and takes the plain forward's tiling.
  if (kind == EPI_FWD_FF)
    return P <= 64 ? make_cfg(ff_tile(P), P, Q, R, 1024, 8) : select_cfg_default(EPI_FWD, P, Q, R);
  if (kind == EPI_FWD && P <= 64) {
    GemmCfg c = make_cfg(ff_tile(P), P, Q, R, 1024, 8);
    // Between 33 and 64 rows, with enough columns to fill the chip: 64x128
    // tiles with the same splits, whose sums equal the 64x32 tile's bit for
    // bit; a third of the operand loads per flop (measured on MI355X at
    // 64 x 8192 x 8192: 108 against 115 us).
    if (P > 32 && ntiles(TI_64x128, P, Q) * c.S >= 256) c.tile = TI_64x128;
    return c;
  }
  if (kind == EPI_WGRAD || kind == EPI_WGRAD_BF) {
    // A short reduction onto a huge output (an 8192 x 8192 layer at 64 rows):
    // whole reductions on 64x64 tiles (measured on MI355X: plain 115 us, fused with
    // Adam 356 us; 127 / 366 us on 128x128 tiles).
    if (R <= 128 && ntiles(TI_128x128, P, Q) >= 1024) return make_cfg(TI_64x64, P, Q, R, 1, 1);
    if (R <= 1024 && ntiles(TI_32x32, P, Q) >= 512) return make_cfg(TI_32x32, P, Q, R, 1, 1);
    // A very long reduction onto few outputs (the pixel rows of a 1x1
    // convolution, 65k-400k rows onto a few hundred weights): up to 256
    // splits, on 64x32 tiles when P > 32 so that the B operand is read once per
    // 64 output rows (measured on MI355X at 401408 x 96 x 16: 70 us, 139 us
    // with 32x32 tiles and at most 64 splits).
    if (R >= 65536) return make_cfg(P > 32 ? TI_64x32 : TI_32x32, P, Q, R, 1024, 256);
    // Many tiles over a moderate reduction (a 1x1 head of 1280 x 320 over 1568
    // rows): 64x32 tiles, split to about 2048 workgroups (31.9 us, 42.5 us
    // unsplit on 32x32 tiles).
    if (R >= 1024 && ntiles(TI_32x32, P, Q) >= 256) return make_cfg(TI_64x32, P, Q, R, 2048, 16);
  }
  // Tall, narrow products (a 1x1 convolution as a linear over 16k-400k pixel
  // rows onto at most 256 channels): narrow tiles, whole reductions.  The
  // 128x128 tile the rule below would pick leaves most of each tile empty
  // (measured on MI355X, forward / data gradient: 401408 x 16 x 32 121 / 98 us
  // on 128x128, 36 us on 256x32 / 36 us on 64x32; 100352 x 144 x 24 71 / 65 us,
  // 39 / 23 us).
  if ((kind == EPI_FWD || kind == EPI_DGRAD) && P >= 16384 && Q <= 256) {
    if (kind == EPI_FWD)
      return make_cfg(P >= 65536 ? TI_256x32 : (Q <= 32 ? TI_32x32 : TI_64x64), P, Q, R, 1, 1);
    return make_cfg(Q <= 32 ? TI_64x32 : TI_64x64, P, Q, R, 1, 1);
  }
  if (P <= 64 && ntiles(TI_64x64, P, Q) >= 64) return make_cfg(TI_64x64, P, Q, R, 1024, 8);
  // Larger outputs: the biggest tile that still gives one workgroup per CU; no
  // reduction split (each split costs a second kernel, ~4 us back to back).
  // A forward or data gradient that lands on 32x32 tiles loads its operands
  // straight into the matrix-core registers (its A operand is reduction-
  // contiguous; measured faster there, slower for the weight gradient).
  const int order[4] = {TI_128x128, TI_128x64, TI_64x64, TI_32x32};
  for (int i = 0; i < 4; ++i)
    if (ntiles(order[i], P, Q) >= 256) {
      const bool direct = order[i] == TI_32x32 && (kind == EPI_FWD || kind == EPI_DGRAD);
      return make_cfg(direct ? TI_32x32D : order[i], P, Q, R, 256, 16);
    }
  // Fewer than 256 blocks of 32x32 (a narrow classifier, a short batch): a
  // forward or data gradient takes direct 32x32 tiles, unsplit while the
  // reduction is short (its second pass would cost more than the split saves).
  if (kind == EPI_FWD || kind == EPI_DGRAD)
    return make_cfg(TI_32x32D, P, Q, R, R <= 1024 ? 1 : 64, 16);
  // A weight gradient of few tiles over a short reduction (a classifier, a
  // narrow layer) stays in one pass: splitting 256 rows in two saved less than
  // the second pass costs (mlp8x1024's 10 x 1024 classifier: 7.0 + 5.7 us).
  if (R <= 1024) return make_cfg(TI_32x32, P, Q, R, 1, 1);
  return make_cfg(TI_32x32, P, Q, R, 1024, 64);
}

// Convolutions: the tile and reduction split that minimise a cost model fitted
// to measured implicit-GEMM times on MI355X (the VGG-11 layer shapes, within 2%
// of the best measured choice in total).  A workgroup alone runs its tile at
// kEff of a CU's fp32 matrix rate; kConc workgroups share a CU; a split adds a
// second pass (fixed cost plus reading and writing the partials).  The rule
// depends on (P, Q, R) only, so the eager and backward-fusion weight gradients
// still share their tiling.
static GemmCfg select_cfg_conv(int P, int Q, int R) {
  // A first layer of at most 32 filters over few input channels (a 3-channel
  // image stem: 3x3x3 = 27 reduction elements) at 65k pixels or more: its
  // forward takes 256x32 tiles, its weight gradient 32x32 tiles split over the
  // pixels (measured on MI355X at 32 x 112 x 112 x 3 -> 32: forward 90 -> 62 us,
  // weight gradient 99 -> 62 us).
  if (R <= 32 && Q <= 32 && P >= 65536) return make_cfg(TI_256x32, P, Q, R, 1, 1);
  if (Q <= 32 && P <= 32 && R >= 65536) return make_cfg(TI_32x32, P, Q, R, 256, 256);
  static const double kEff[6] = {0.489, 0.283, 0.617, 0.488, 0.714, 0.765};
  static const int kConc[6] = {1, 4, 3, 4, 2, 1};
  static const int kSplits[8] = {1, 2, 4, 8, 16, 32, 64, 128};
  const double cu_rate = 157.3e12 / 256;  // fp32 matrix flop/s per CU
  double best = 1e30;
  GemmCfg pick{TI_32x32, 1, (R + 31) / 32 * 32};
  for (int t = 0; t < 6; ++t) {
    const int BR = kTileBR[t];
    for (int S : kSplits) {
      if (S > 1 && R / S < 2 * BR) continue;
      const int r_split = ((R + S - 1) / S + BR - 1) / BR * BR;
      const int Se = (R + r_split - 1) / r_split;
      const double W = (double)ntiles(t, P, Q) * Se;
      const double per = (double)kTileBP[t] * kTileBQ[t] * r_split * 2 / (kEff[t] * cu_rate) * 1e6;
      double T = per * std::max(1.0, W / (256.0 * kConc[t]));
      if (Se > 1) T += 1.97 + (double)P * Q * Se * 8 / 5e12 * 1e6;
      if (T < best) {
        best = T;
        pick = GemmCfg{t, Se, r_split};
      }
    }
  }
  return pick;
}

static GemmCfg select_cfg_any(int kind, int P, int Q, int R, int conv) {
  return conv ? select_cfg_conv(P, Q, R) : select_cfg_default(kind, P, Q, R);
}

#ifdef OPFUSE_TUNING
// Tuning builds only: OPFUSE_CFG="tile,S" overrides the tiling of every contraction.
static GemmCfg select_cfg(int kind, int P, int Q, int R, int conv) {
  const char* e = getenv("OPFUSE_CFG");
  if (!e) return select_cfg_any(kind, P, Q, R, conv);
  int t = 0, S = 1;
  sscanf(e, "%d,%d", &t, &S);
  return make_cfg(t, P, Q, R, (int64_t)S * ntiles(t, P, Q), S);
}
#else
static GemmCfg select_cfg(int kind, int P, int Q, int R, int conv) {
  return select_cfg_any(kind, P, Q, R, conv);
}
#endif

size_t gemm_workspace_bytes(int kind, int P, int Q, int R, int conv) {
  const GemmCfg c = select_cfg(kind, P, Q, R, conv);
  if (c.S <= 1) return 0;
  return (size_t)c.S * ((size_t)P * Q + P) * sizeof(float);
}

template <class T, int EPI>
static hipError_t launch_t(const GemmCfg& c, const GemmProblem& pr, const EpiArgs& ea, void* ws,
                           int vec_ops, int vec_epi, hipStream_t stream) {
  dim3 grid((pr.P + T::BP - 1) / T::BP, (pr.Q + T::BQ - 1) / T::BQ, c.S + c.cz);
  if (pr.conv) {
    // convolutions: 128-bit gathers per operand (the channel counts differ)
    switch (vec_ops) {
      case 3: hipLaunchKernelGGL((gemm_kernel<T, EPI, 3, true>), grid, dim3(256), 0, stream, pr, ea, c.r_split, (float*)ws, vec_epi); break;
      case 2: hipLaunchKernelGGL((gemm_kernel<T, EPI, 2, true>), grid, dim3(256), 0, stream, pr, ea, c.r_split, (float*)ws, vec_epi); break;
      case 1: hipLaunchKernelGGL((gemm_kernel<T, EPI, 1, true>), grid, dim3(256), 0, stream, pr, ea, c.r_split, (float*)ws, vec_epi); break;
      default: hipLaunchKernelGGL((gemm_kernel<T, EPI, 0, true>), grid, dim3(256), 0, stream, pr, ea, c.r_split, (float*)ws, vec_epi);
    }
    return hipGetLastError();
  }
  // 128-bit operand loads only when both operands allow them.
  if (vec_ops == 3)
    hipLaunchKernelGGL((gemm_kernel<T, EPI, 3, false>), grid, dim3(256), 0, stream, pr, ea,
                       c.r_split, (float*)ws, vec_epi);
  else
    hipLaunchKernelGGL((gemm_kernel<T, EPI, 0, false>), grid, dim3(256), 0, stream, pr, ea,
                       c.r_split, (float*)ws, vec_epi);
  return hipGetLastError();
}

template <int EPI, int NW, int NS>
static hipError_t launch_direct(const GemmCfg& c, const GemmProblem& pr, const EpiArgs& ea,
                                void* ws, int vec_ops, int vec_epi, hipStream_t stream) {
  dim3 grid((pr.P + 31) / 32, (pr.Q + 31) / 32, c.S + c.cz);
  // The data gradient's B operand (W) is output-contiguous and never takes
  // 128-bit loads, so only A's flag matters there.
  const int v = EPI == EPI_FWD ? (vec_ops == 3 ? 3 : 0) : (vec_ops & 1);
  if (v == 3)
    hipLaunchKernelGGL((gemm_direct_kernel<EPI, NW, NS, 3>), grid, dim3(64 * NW), 0, stream, pr,
                       ea, c.r_split, (float*)ws, vec_epi);
  else if (v == 1)
    hipLaunchKernelGGL((gemm_direct_kernel<EPI, NW, NS, 1>), grid, dim3(64 * NW), 0, stream, pr,
                       ea, c.r_split, (float*)ws, vec_epi);
  else
    hipLaunchKernelGGL((gemm_direct_kernel<EPI, NW, NS, 0>), grid, dim3(64 * NW), 0, stream, pr,
                       ea, c.r_split, (float*)ws, vec_epi);
  return hipGetLastError();
}

template <int EPI>
static hipError_t launch_kind(const GemmCfg& c, const GemmProblem& pr, const EpiArgs& ea, void* ws,
                              int vec_ops, int vec_epi, hipStream_t s) {
  switch (c.tile) {
    case TI_32x32: return launch_t<T32x32, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
    case TI_64x32: return launch_t<T64x32, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
    case TI_64x64: return launch_t<T64x64, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
    case TI_128x64: return launch_t<T128x64, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
    case TI_128x128:
      // gemm_launch gives a fused forward 128x64 instead (LDS for the bias row).
      if constexpr (EPI == EPI_FWD_FF) return hipErrorInvalidValue;
      else return launch_t<T128x128, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
    case TI_256x32: return launch_t<T256x32, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
    case TI_64x128:
      // the plain forward of linear layers only (its fused counterpart keeps
      // T64x32, whose sums it reproduces)
      if constexpr (EPI == EPI_FWD) {
        if (pr.conv) return hipErrorInvalidValue;
        dim3 grid((pr.P + 63) / 64, (pr.Q + 127) / 128, c.S + c.cz);
        if (vec_ops == 3)
          hipLaunchKernelGGL((gemm_kernel<T64x128, EPI, 3, false>), grid, dim3(256), 0, s, pr, ea,
                             c.r_split, (float*)ws, vec_epi);
        else
          hipLaunchKernelGGL((gemm_kernel<T64x128, EPI, 0, false>), grid, dim3(256), 0, s, pr, ea,
                             c.r_split, (float*)ws, vec_epi);
        return hipGetLastError();
      }
      return hipErrorInvalidValue;
    case TI_32x32D:
    case TI_32x32D8:
      // direct loads exist for the linear forward and data gradient; the same
      // tiling through LDS otherwise
      if constexpr (EPI == EPI_FWD || EPI == EPI_DGRAD) {
        if (!pr.conv) {
          if (c.tile == TI_32x32D) return launch_direct<EPI, 4, 4>(c, pr, ea, ws, vec_ops, vec_epi, s);
          return launch_direct<EPI, 8, 4>(c, pr, ea, ws, vec_ops, vec_epi, s);
        }
      }
      return launch_t<T32x32, EPI>(c, pr, ea, ws, vec_ops, vec_epi, s);
  }
  return hipErrorInvalidValue;
}

// Split counts from which 8 lanes share each output item of the reduction pass.
constexpr int kCoopSplits = 16;

template <int EPI>
static hipError_t launch_reduce(const GemmCfg& c, const GemmProblem& pr, const EpiArgs& ea,
                                void* ws, int vec_epi, int with_db, hipStream_t s) {
  const int64_t work = (int64_t)pr.P * ((pr.Q + 3) / 4);
  if (c.S >= kCoopSplits) {
    const int64_t lanes = std::max<int64_t>(work, with_db ? pr.P : 0) * 8;
    const int blocks = (int)std::min<int64_t>(2048, std::max<int64_t>(1, (lanes + 255) / 256));
    hipLaunchKernelGGL((split_reduce_coop_kernel<EPI>), dim3(blocks), dim3(256), 0, s, pr.P, pr.Q,
                       c.S, ea, (const float*)ws, vec_epi, with_db);
    return hipGetLastError();
  }
  const int blocks = (int)std::min<int64_t>(2048, std::max<int64_t>(1, (work + 255) / 256));
  hipLaunchKernelGGL((split_reduce_kernel<EPI>), dim3(blocks), dim3(256), 0, s, pr.P, pr.Q, c.S,
                     ea, (const float*)ws, vec_epi, with_db);
  return hipGetLastError();
}

static int vec_flags(const GemmProblem& pr, int kind, const EpiArgs& ea, int* vec_epi) {
  // Operand tiles: 128-bit loads need a 16B-aligned base and a row stride that
  // keeps every row 16B aligned.
  // The contiguous extent must also end on a float4 boundary (a float4 is
  // either wholly inside the operand or wholly masked).
  const bool a_rc = (kind == EPI_FWD || kind == EPI_FWD_FF || kind == EPI_DGRAD);
  const bool b_rc = (kind == EPI_FWD || kind == EPI_FWD_FF);
  bool va = aligned16(pr.A) && ((pr.a_sr == 1 ? pr.a_sp : pr.a_sr) % 4 == 0) &&
            ((a_rc ? pr.R : pr.P) % 4 == 0);
  bool vb = aligned16(pr.B) && ((pr.b_sr == 1 ? pr.b_sq : pr.b_sr) % 4 == 0) &&
            ((b_rc ? pr.R : pr.Q) % 4 == 0);
  if (pr.conv) {
    // gathers: a float4 stays within one filter tap when the channel count along
    // the contiguous index is a multiple of 4
    const bool cin4 = pr.cC % 4 == 0, cout4 = pr.cCout % 4 == 0;
    if (kind == EPI_FWD || kind == EPI_FWD_FF) { va = aligned16(pr.A) && cin4; vb = aligned16(pr.B) && cin4; }
    if (kind == EPI_DGRAD) { va = aligned16(pr.A) && cout4; vb = aligned16(pr.B) && cin4; }
    if (kind == EPI_WGRAD || kind == EPI_WGRAD_BF) {
      va = aligned16(pr.A) && cout4;
      vb = aligned16(pr.B) && cin4;
    }
  }
  if (kind == EPI_FWD_FF)
    vb = vb && aligned16(ea.W.w) && aligned16(ea.W.m) && aligned16(ea.gW) &&
         (ea.opt.kind == OF_OPT_SGD || aligned16(ea.W.v)) &&
         aligned16(ea.Wout.w) && aligned16(ea.Wout.m) &&
         (ea.opt.kind == OF_OPT_SGD || aligned16(ea.Wout.v)) &&
         (ea.W.w_bf16 == nullptr || ((uintptr_t)ea.W.w_bf16 & 7u) == 0);
  int ve = 0;
  if (aligned16(ea.out) && ea.ldo % 4 == 0 && (ea.z == nullptr || (aligned16(ea.z) && ea.ldz % 4 == 0)) &&
      (ea.prev == nullptr || (aligned16(ea.prev) && ea.ldp % 4 == 0)) &&
      (ea.res == nullptr || (aligned16(ea.res) && ea.ldr % 4 == 0)))
    ve |= 1;
  if (kind == EPI_WGRAD_BF && aligned16(ea.W.w) && aligned16(ea.W.m) && ea.ldo % 4 == 0 &&
      (ea.opt.kind == OF_OPT_SGD || aligned16(ea.W.v)) && (ea.gW == nullptr || aligned16(ea.gW)) &&
      (ea.W.w_bf16 == nullptr || ((uintptr_t)ea.W.w_bf16 & 7u) == 0))
    ve |= 2;
  *vec_epi = ve;
  return (va ? 1 : 0) | (vb ? 2 : 0);
}

hipError_t gemm_launch(int kind, const GemmProblem& pr, const EpiArgs& ea_in, void* ws,
                       hipStream_t stream) {
  GemmCfg c = select_cfg(kind, pr.P, pr.Q, pr.R, pr.conv);
  // The 128x128 tile leaves no LDS for forward-fusion's bias row; a fused
  // forward given it takes 128x64 with the same splits (the same reduction
  // ranges and workspace).
  if (kind == EPI_FWD_FF && c.tile == TI_128x128) c.tile = TI_128x64;
  EpiArgs ea = ea_in;
  ea.carry.cz = 0;
  if (ea.carry.t[0].p.w) {
    if (kind != EPI_FWD) return hipErrorInvalidValue;  // only a forward carries an update
    c.cz = carry_slices(ea.carry, ntiles(c.tile, pr.P, pr.Q));
    ea.carry.cz = c.cz;
  }
  int vec_epi = 0;
  const int vec_ops = vec_flags(pr, kind, ea, &vec_epi);
  const bool wg = (kind == EPI_WGRAD || kind == EPI_WGRAD_BF);
  const int with_db = wg && ea.with_db;
  hipError_t e;
  switch (kind) {
    case EPI_FWD: e = launch_kind<EPI_FWD>(c, pr, ea, ws, vec_ops, vec_epi, stream); break;
    case EPI_FWD_FF: e = launch_kind<EPI_FWD_FF>(c, pr, ea, ws, vec_ops, vec_epi, stream); break;
    case EPI_DGRAD: e = launch_kind<EPI_DGRAD>(c, pr, ea, ws, vec_ops, vec_epi, stream); break;
    case EPI_WGRAD: e = launch_kind<EPI_WGRAD>(c, pr, ea, ws, vec_ops, vec_epi, stream); break;
    case EPI_WGRAD_BF: e = launch_kind<EPI_WGRAD_BF>(c, pr, ea, ws, vec_ops, vec_epi, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess || c.S <= 1) return e;
  EpiArgs er = ea;
  // the bias the split-0 workgroups have updated (written to bout when set)
  if (kind == EPI_FWD_FF) er.bias = ea.bout.w ? ea.bout.w : ea.b.w;
  switch (kind) {
    case EPI_FWD: return launch_reduce<EPI_FWD>(c, pr, er, ws, vec_epi, 0, stream);
    case EPI_FWD_FF: return launch_reduce<EPI_FWD_FF>(c, pr, er, ws, vec_epi, 0, stream);
    case EPI_DGRAD: return launch_reduce<EPI_DGRAD>(c, pr, er, ws, vec_epi, 0, stream);
    case EPI_WGRAD: return launch_reduce<EPI_WGRAD>(c, pr, er, ws, vec_epi, with_db, stream);
    case EPI_WGRAD_BF: return launch_reduce<EPI_WGRAD_BF>(c, pr, er, ws, vec_epi, with_db, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace opfuse
