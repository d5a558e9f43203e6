// Backward-fusion with the data gradient merged into the update's read of W
// (Section 3 "Backward-Fusion": the two consecutive reads of a parameter, by
// the input-gradient computation and by the optimizer, become one read).
//
// For a linear layer with few token rows (M <= 64; X [M,K], W [N,K],
// dZ [M,N]) one kernel streams W once:
//   - a workgroup owns a strip of 128 columns of W and a range of NR rows,
//     which it walks in chunks of 32 rows;
//   - each chunk's W, m, v (and an extra gradient of earlier uses) are loaded
//     straight into registers in the layout of the weight-gradient
//     accumulator of v_mfma_f32_32x32x2_f32;
//   - the same registers are the B operand of the data-gradient partial
//     dX_s[m,k] += sum_n dZ[m,n] W_old[n,k] (the reduction over the chunk's
//     rows is taken in the accumulator's row order), so dX uses the old W as
//     the dependency rule after Alg. 3 requires;
//   - the weight gradient dW = dZ^T X of the chunk (reduction over the M
//     rows; X's fragment stays in registers for the whole kernel) is the
//     gradient of the update, which writes W, m, v back; dW is never stored.
// The row ranges' partials dX_s go to a workspace [S, M, K] and a second
// kernel sums them in range order and applies the previous layer's
// activation derivative, so the result is deterministic.
//
// Per parameter and step this moves R W, m, v and W W, m, v (24 B for Adam)
// instead of the separate data gradient's extra read of W (28 B).

#include <mutex>

#include "gemm_common.h"

namespace opfuse {

typedef float floatx16 __attribute__((ext_vector_type(16)));

namespace {

constexpr int MG_BK = 128;   // W columns per workgroup: 4 wavefronts x 32
constexpr int MG_BN = 32;    // W rows per chunk
constexpr int MG_LDZ = MG_BN + 1;  // LDS row pitch of the dZ chunk (floats)

struct MergedArgs {
  const float* dz; int64_t ldz;
  const float* x; int64_t ldx;
  of_param W; const float* gW;
  of_param b; const float* gb;
  OptK opt;
  float* part;       // [S, M, K] data-gradient partials; NULL: no data gradient
  int M, N, K, NR;   // NR: rows per range (a multiple of MG_BN)
  int dz_vec;        // dZ rows 16-byte aligned with N a multiple of 4
};

// Row (within a 32-row block) of accumulator element i of a lane in half h
// of the wavefront: elements 4j..4j+3 are rows 8j + 4h .. 8j + 4h + 3.
__device__ __forceinline__ int acc_row(int i, int h) { return (i >> 2) * 8 + h * 4 + (i & 3); }

__device__ __forceinline__ void bstore1(rsrc_t r, uint32_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, off, 0, 0);
}

// One chunk's parameter fragment: element i of a lane is row n0 + acc_row(i, h)
// and column kcol of W (and of m, v, gW).
// HAS_G: an extra gradient is added (the fragment holds it too).
template <bool HAS_G>
struct ParFrag {
  float w[16], m[16], v[16], g[HAS_G ? 16 : 1];

  __device__ __forceinline__ void load(const MergedArgs& a, int n0, int n_end, int h, int kcol,
                                       bool kok, bool adam) {
    const int64_t base = (int64_t)n0 * a.K;
    const rsrc_t rw = make_rsrc(a.W.w + base);
    const rsrc_t rm = make_rsrc_opt(a.W.m, base);   // no m: reads 0
    const rsrc_t rv = adam ? make_rsrc(a.W.v + base) : rm;
    const rsrc_t rg = HAS_G ? make_rsrc(a.gW + base) : rm;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int n = acc_row(i, h);
      const bool ok = kok && n0 + n < n_end;
      const uint32_t off = ok ? (uint32_t)((n * a.K + kcol) * 4) : kOOB;
      w[i] = bload1(rw, off);
      m[i] = bload1(rm, off);
      v[i] = adam ? bload1(rv, off) : 0.f;
      if constexpr (HAS_G) g[i] = bload1(rg, off);
    }
  }
};

// dZ[0:64, n0:n0+32] through registers into LDS ([m][n], pitch MG_LDZ);
// rows >= M and columns >= n_end read as 0.
struct DzChunk {
  float4 r[2];

  __device__ __forceinline__ void load(const MergedArgs& a, int n0, int n_end, int tid) {
    const rsrc_t rz = make_rsrc(a.dz + n0);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int idx = tid + 256 * q, m = idx >> 3, j = (idx & 7) * 4;
      if (a.dz_vec) {
        const bool ok = m < a.M && n0 + j < n_end;
        r[q] = bload4(rz, ok ? (uint32_t)((m * a.ldz + j) * 4) : kOOB);
      } else {
        float e[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const bool ok = m < a.M && n0 + j + t < n_end;
          e[t] = bload1(rz, ok ? (uint32_t)((m * a.ldz + j + t) * 4) : kOOB);
        }
        r[q] = make_float4(e[0], e[1], e[2], e[3]);
      }
    }
  }

  __device__ __forceinline__ void store(float* lds, int tid) const {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int idx = tid + 256 * q, m = idx >> 3, j = (idx & 7) * 4;
      float* p = lds + m * MG_LDZ + j;
      p[0] = r[q].x;
      p[1] = r[q].y;
      p[2] = r[q].z;
      p[3] = r[q].w;
    }
  }
};

// Everything a workgroup keeps across chunks.
template <int MB>
struct MergedState {
  int tid, h, c, kcol, n_end;
  bool kok, adam, do_dx, do_db;
  int mpairs;
  OptK o;
  float xf[32];        // X[2s + h][kcol]: B operand of every chunk's weight gradient
  floatx16 accd[MB];   // data-gradient partial, rows mb*32 + acc_row(i, h), column kcol
  DzChunk zr;
};

// One chunk of rows n0..n0+31 whose W fragment is `cu` and whose dZ is in LDS
// buffer `zc`; the next chunk's loads go to `nx` and `zr` first (when `more`),
// so they are in flight while this chunk computes.
template <int MB, bool HAS_G>
__device__ __forceinline__ void merged_chunk(const MergedArgs& a, MergedState<MB>& st,
                                             const ParFrag<HAS_G>& cu, ParFrag<HAS_G>& nx, int n0,
                                             const float* zc, float* zn) {
  const int h = st.h, c = st.c;
  const int n1 = n0 + MG_BN;
  const bool more = n1 < st.n_end;
  if (more) {
    st.zr.load(a, n1, st.n_end, st.tid);
    nx.load(a, n1, st.n_end, h, st.kcol, st.kok, st.adam);
  }

  // Data-gradient partial with the old W: reduction slot h of step s is
  // chunk row acc_row(s, h), the row the W fragment's element s holds.
  if (st.do_dx) {
#pragma unroll
    for (int s = 0; s < 16; ++s) {
      const int n = acc_row(s, h);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        st.accd[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(zc[(mb * 32 + c) * MG_LDZ + n], cu.w[s],
                                                          st.accd[mb], 0, 0, 0);
    }
  }

  // Weight gradient of the chunk: dW[n][kcol] = sum_m dZ[m][n] X[m][kcol].
  floatx16 accw;
#pragma unroll
  for (int i = 0; i < 16; ++i) accw[i] = 0.f;
#pragma unroll
  for (int s = 0; s < 32; ++s) {
    if (s < st.mpairs)
      accw = __builtin_amdgcn_mfma_f32_32x32x2f32(zc[(2 * s + h) * MG_LDZ + c], st.xf[s], accw, 0,
                                                  0, 0);
  }

  // Bias: db[n] = sum over rows of dZ, in row order (strip 0 only).
  if (st.do_db && st.tid < MG_BN && n0 + st.tid < st.n_end) {
    float s = zc[st.tid];
    for (int m = 1; m < a.M; ++m) s = __fadd_rn(s, zc[m * MG_LDZ + st.tid]);
    if (a.gb) s = __fadd_rn(s, a.gb[n0 + st.tid]);
    update1(st.o, a.b, s, n0 + st.tid);
  }

  // The update, from the registers: W, m, v written back, dW never stored.
  {
    const int64_t base = (int64_t)n0 * a.K;
    const rsrc_t rw = make_rsrc(a.W.w + base);
    const rsrc_t rm = make_rsrc_opt(a.W.m, base);   // no m: stores dropped
    const rsrc_t rv = st.adam ? make_rsrc(a.W.v + base) : rm;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int n = acc_row(i, h);
      const bool ok = st.kok && n0 + n < st.n_end;
      const uint32_t off = ok ? (uint32_t)((n * a.K + st.kcol) * 4) : kOOB;
      float w = cu.w[i], m = cu.m[i], v = cu.v[i];
      float g = accw[i];
      if constexpr (HAS_G) g = __fadd_rn(g, cu.g[i]);
      opt_update(st.o, w, g, m, v);
      bstore1(rw, off, w);
      bstore1(rm, off, m);
      if (st.adam) bstore1(rv, off, v);
    }
  }

  if (more) st.zr.store(zn, st.tid);
  __syncthreads();
}

// MB: 32-row blocks of token rows (1: M <= 32, 2: M <= 64).  Two workgroups
// per compute unit (at most 256 registers per lane) unless the fragments also
// hold an extra gradient.
template <int MB, bool HAS_G>
__global__ __launch_bounds__(256, HAS_G ? 1 : 2) void merged_bwd_kernel(MergedArgs a) {
  __shared__ float dzc[2][64 * MG_LDZ];
  MergedState<MB> st;
  st.tid = threadIdx.x;
  const int lane = st.tid & 63, wave = st.tid >> 6;
  st.h = lane >> 5;
  st.c = lane & 31;
  st.kcol = blockIdx.x * MG_BK + wave * 32 + st.c;
  st.kok = st.kcol < a.K;
  const int n_beg = blockIdx.y * a.NR;
  st.n_end = min(a.N, n_beg + a.NR);
  st.adam = a.opt.kind != OF_OPT_SGD;
  st.do_dx = a.part != nullptr;
  st.do_db = a.b.w != nullptr && blockIdx.x == 0;
  st.mpairs = (a.M + 1) >> 1;

  ParFrag<HAS_G> fa, fb;
  if (n_beg < st.n_end) {
    st.zr.load(a, n_beg, st.n_end, st.tid);
    fa.load(a, n_beg, st.n_end, st.h, st.kcol, st.kok, st.adam);
  }
  {
    const rsrc_t rx = make_rsrc(a.x);
#pragma unroll
    for (int s = 0; s < 32; ++s) {
      const int m = 2 * s + st.h;
      st.xf[s] = bload1(rx, (st.kok && m < a.M) ? (uint32_t)((m * a.ldx + st.kcol) * 4) : kOOB);
    }
  }
  st.o = a.opt;
  opt_prepare(st.o);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int i = 0; i < 16; ++i) st.accd[mb][i] = 0.f;

  st.zr.store(dzc[0], st.tid);
  __syncthreads();
  // Chunks alternate between the two fragments and the two LDS buffers.
  for (int n0 = n_beg; n0 < st.n_end; n0 += 2 * MG_BN) {
    merged_chunk<MB, HAS_G>(a, st, fa, fb, n0, dzc[0], dzc[1]);
    if (n0 + MG_BN < st.n_end)
      merged_chunk<MB, HAS_G>(a, st, fb, fa, n0 + MG_BN, dzc[1], dzc[0]);
  }

  if (st.do_dx) {
    const rsrc_t rp = make_rsrc(a.part + (int64_t)blockIdx.y * a.M * a.K);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int m = mb * 32 + acc_row(i, st.h);
        const bool ok = st.kok && m < a.M;
        bstore1(rp, ok ? (uint32_t)((m * a.K + st.kcol) * 4) : kOOB, st.accd[mb][i]);
      }
  }
}

// dX[m,k] = (sum over ranges s, in order, of part[s,m,k]) * act'(prev[m,k]).
__global__ __launch_bounds__(256) void merged_dx_kernel(const float* __restrict__ part, int S,
                                                        int M, int K, const float* __restrict__ prev,
                                                        int64_t ldp, int act, float* __restrict__ dx,
                                                        int64_t ldx) {
  const int64_t MK = (int64_t)M * K;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < MK; e += (int64_t)gridDim.x * 256) {
    float s = part[e];
    for (int q0 = 1; q0 < S; q0 += 8) {
      float v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = q0 + q < S ? part[(q0 + q) * MK + e] : 0.f;
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (q0 + q < S) s = __fadd_rn(s, v[q]);
    }
    const int64_t m = e / K, k = e - m * K;
    if (act != OF_ACT_NONE) s = __fmul_rn(s, act_grad(act, prev[m * ldp + k]));
    dx[m * ldx + k] = s;
  }
}

}  // namespace

// Row ranges for an M x N x K layer: about two workgroups per compute unit
// (512 in all) and `per` whole chunks of MG_BN rows per range.  A W of more
// than 64 MB (streamed from HBM) keeps the partials (S * M * K) at most an
// eighth of W; a smaller one stays in the caches and takes as many ranges as
// the workgroup target asks (a 1024 x 1024 layer would otherwise run on 16
// workgroups).
void merged_plan(int M, int N, int K, int* S, int* per) {
  const int strips = (K + MG_BK - 1) / MG_BK;
  const int chunks = (N + MG_BN - 1) / MG_BN;
  int s = std::max(1, (512 + strips - 1) / strips);
  if ((int64_t)N * K * 4 > (64LL << 20)) s = std::min(s, std::max(1, N / (8 * M)));
  s = std::min(s, chunks);
  *per = (chunks + s - 1) / s;
  *S = (chunks + *per - 1) / *per;
}

// Partials buffer of the no-allocation entry point (of_linear_bwd_merged_static),
// for callers that cannot allocate (graph capture, serving loops).  32 MiB
// holds the partials of every layer of at most 64 rows whose W has up to
// 65536 columns (an 8192 x 8192 layer at 64 rows needs 16 MiB).  Each device
// the library runs on holds its own copy until the process ends; every call on
// a device shares it, so calls that overlap on one device race.  The partials
// need no clearing: every element read is written earlier in the same call.
constexpr size_t kMergedScratchBytes = OF_MERGED_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) float merged_scratch[kMergedScratchBytes / sizeof(float)];

size_t merged_scratch_bytes() { return kMergedScratchBytes; }

// In host code `merged_scratch` names a host-side stand-in, not device memory:
// its device address comes from the runtime, per device, with that device
// current, on the first call there.
hipError_t merged_scratch_ptr(float** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(merged_scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = static_cast<float*>(addr[dev]);
  return hipSuccess;
}

size_t merged_workspace_bytes(int M, int N, int K) {
  int S, per;
  merged_plan(M, N, K, &S, &per);
  return (size_t)S * M * K * sizeof(float);
}

hipError_t merged_bwd_launch(const MergedLaunch& L, hipStream_t stream) {
  MergedArgs a;
  a.dz = L.dz; a.ldz = L.ldz;
  a.x = L.x; a.ldx = L.ldx;
  a.W = L.W; a.gW = L.gW;
  a.b = L.b; a.gb = L.gb;
  a.opt = L.opt;
  a.M = L.M; a.N = L.N; a.K = L.K;
  int S, per;
  merged_plan(L.M, L.N, L.K, &S, &per);
  a.NR = per * MG_BN;
  a.part = L.dx ? L.part : nullptr;
  a.dz_vec = aligned16(L.dz) && L.ldz % 4 == 0 && L.N % 4 == 0;
  const dim3 grid((L.K + MG_BK - 1) / MG_BK, S);
  const bool g = L.gW != nullptr;
  if (L.M <= 32) {
    if (g) hipLaunchKernelGGL((merged_bwd_kernel<1, true>), grid, dim3(256), 0, stream, a);
    else   hipLaunchKernelGGL((merged_bwd_kernel<1, false>), grid, dim3(256), 0, stream, a);
  } else {
    if (g) hipLaunchKernelGGL((merged_bwd_kernel<2, true>), grid, dim3(256), 0, stream, a);
    else   hipLaunchKernelGGL((merged_bwd_kernel<2, false>), grid, dim3(256), 0, stream, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !L.dx) return e;
  const int64_t MK = (int64_t)L.M * L.K;
  const int blocks = (int)std::min<int64_t>((MK + 255) / 256, 2048);
  hipLaunchKernelGGL(merged_dx_kernel, dim3(blocks), dim3(256), 0, stream, L.part, S, L.M, L.K,
                     L.prev, L.ldx, L.act_prev, L.dx, L.ldx);
  return hipGetLastError();
}

}  // namespace opfuse
