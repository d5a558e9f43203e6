// Internal declarations shared by the opfuse HIP sources (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/opfuse.h"

namespace opfuse {

// Optimizer hyperparameters as the kernels consume them.  The step-dependent
// bias corrections are computed in float64 on the host when the step is given
// by value, else by opt_prepare() in the kernel from the device step counter
// (the same arithmetic, so both give the same bits).
struct OptK {
  int kind;          // of_opt_kind
  float lr, wd, mom;
  float b1, b2, eps;
  float omb1, omb2;  // 1 - beta1, 1 - beta2
  float decay;       // 1 - lr * wd  (AdamW)
  int64_t step;
  const int64_t* step_dev;
  float step_size;   // lr / (1 - beta1^t)
  float rsqrt_bc2;   // 1 / sqrt(1 - beta2^t)
  int prepared;      // step_size / rsqrt_bc2 already set (step given by value)
  const float* gscale_dev;  // optional gradient scale in device memory
  float gscale;      // the scale in use (1 unless read from gscale_dev)
};

OptK make_optk(const of_opt& o);

// beta^t by binary exponentiation in float64: a fixed sequence of correctly
// rounded multiplications, so the host and every kernel get the same value.
__host__ __device__ inline double pow_steps(double b, int64_t t) {
  double r = 1.0;
  while (t > 0) {
    if (t & 1) r *= b;
    b *= b;
    t >>= 1;
  }
  return r;
}

// The Adam bias corrections of update t, in float64, rounded once to float.
__host__ __device__ inline void opt_constants(OptK& o, int64_t t) {
  const double bc1 = 1.0 - pow_steps((double)o.b1, t);
  const double bc2 = 1.0 - pow_steps((double)o.b2, t);
  o.step_size = (float)((double)o.lr / bc1);
  o.rsqrt_bc2 = (float)(1.0 / sqrt(bc2));
}

// Kernels call this before their first update: with a step given by value the
// host has already set the constants; with a device step counter they are
// computed here, from the step the kernel reads when it runs.
// A gradient scale given by address is read here too.
__device__ __forceinline__ void opt_prepare(OptK& o) {
  if (o.gscale_dev) o.gscale = *o.gscale_dev;
  if (o.kind != OF_OPT_ADAM && o.kind != OF_OPT_ADAMW) return;   // no step-dependent constants
  if (o.prepared) return;
  opt_constants(o, *o.step_dev);
}

// The one per-element update used by every kernel that changes a parameter
// (Appendix A, Alg. 1: theta_t = theta_{t-1} + pi(...)).  All operations are
// explicitly rounded (the sources are also built with -ffp-contract=off), so
// the same gradient gives the same bits in every ordering and kernel.
// __fsqrt_rn is the hardware square root (within 1 ulp, the same instruction
// everywhere); no divisor is a bare square root, which the compiler could turn
// into a reciprocal-square-root product in some kernels only.
__device__ __forceinline__ void opt_update(const OptK& o, float& w, float g, float& m, float& v) {
  g = __fmul_rn(g, o.gscale);   // the gradient scale (exact when it is 1)
  if (o.kind == OF_OPT_SGD) {
    // Momentum policy pi_2 with coupled weight decay.
    const float gp = __fmaf_rn(o.wd, w, g);
    m = __fmaf_rn(o.mom, m, gp);
    w = __fmaf_rn(-o.lr, m, w);
  } else if (o.kind == OF_OPT_ADAGRAD) {
    // v: running sum of squared gradients.
    const float gp = __fmaf_rn(o.wd, w, g);
    v = __fmaf_rn(gp, gp, v);
    w = __fsub_rn(w, __fdiv_rn(__fmul_rn(o.lr, gp), __fadd_rn(__fsqrt_rn(v), o.eps)));
  } else if (o.kind == OF_OPT_RMSPROP) {
    // v: decaying average of squared gradients (decay b2); m: momentum buffer.
    const float gp = __fmaf_rn(o.wd, w, g);
    v = __fmaf_rn(o.b2, v, __fmul_rn(__fmul_rn(o.omb2, gp), gp));
    const float step = __fdiv_rn(gp, __fadd_rn(__fsqrt_rn(v), o.eps));
    if (o.mom != 0.f) {
      m = __fmaf_rn(o.mom, m, step);
      w = __fmaf_rn(-o.lr, m, w);
    } else {
      w = __fmaf_rn(-o.lr, step, w);
    }
  } else if (o.kind == OF_OPT_ADADELTA) {
    // v: decaying average of squared gradients; m: of squared updates (decay b2).
    const float gp = __fmaf_rn(o.wd, w, g);
    v = __fmaf_rn(o.b2, v, __fmul_rn(__fmul_rn(o.omb2, gp), gp));
    // sqrt((m + eps) / (v + eps)) rather than a quotient of square roots: a
    // division by a bare hardware square root may be rewritten as a product
    // with a reciprocal square root in some kernels and not in others
    const float delta =
        __fmul_rn(__fsqrt_rn(__fdiv_rn(__fadd_rn(m, o.eps), __fadd_rn(v, o.eps))), gp);
    m = __fmaf_rn(o.b2, m, __fmul_rn(__fmul_rn(o.omb2, delta), delta));
    w = __fmaf_rn(-o.lr, delta, w);
  } else {
    float gp = g;
    if (o.kind == OF_OPT_ADAMW) {
      w = __fmul_rn(w, o.decay);
    } else {
      gp = __fmaf_rn(o.wd, w, g);
    }
    m = __fmaf_rn(o.b1, m, __fmul_rn(o.omb1, gp));
    v = __fmaf_rn(o.b2, v, __fmul_rn(__fmul_rn(o.omb2, gp), gp));
    const float denom = __fadd_rn(__fmul_rn(__fsqrt_rn(v), o.rsqrt_bc2), o.eps);
    w = __fsub_rn(w, __fdiv_rn(__fmul_rn(o.step_size, m), denom));
  }
}

// float -> bfloat16 bits, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_round(float f) {
  return __uint_as_float(((uint32_t)f32_to_bf16(f)) << 16);
}

// Derivative of the forward activation, evaluated from the saved tensor the
// dgrad epilogue receives: Y for ReLU (Y > 0 exactly when Z > 0), Z for GELU.
__device__ __forceinline__ float act_grad(int act, float saved) {
  if (act == OF_ACT_RELU) return saved > 0.f ? 1.f : 0.f;
  if (act == OF_ACT_GELU) {
    const float cdf = 0.5f * (1.f + erff(saved * 0.70710678118654752f));
    const float pdf = 0.39894228040143268f * expf(-0.5f * saved * saved);
    return cdf + saved * pdf;
  }
  return 1.f;
}

__device__ __forceinline__ float act_fwd(int act, float z) {
  if (act == OF_ACT_RELU) return z > 0.f ? z : 0.f;
  if (act == OF_ACT_GELU) return z * (0.5f * (1.f + erff(z * 0.70710678118654752f)));
  return z;
}

__device__ __forceinline__ float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ void st4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }

__device__ __forceinline__ void st_bf16x4(uint16_t* p, float4 w) {
  const uint32_t lo = (uint32_t)f32_to_bf16(w.x) | ((uint32_t)f32_to_bf16(w.y) << 16);
  const uint32_t hi = (uint32_t)f32_to_bf16(w.z) | ((uint32_t)f32_to_bf16(w.w) << 16);
  *reinterpret_cast<uint2*>(p) = make_uint2(lo, hi);
}

// A parameter element's optimizer state (weight and history), loaded apart
// from its update so that a kernel can issue these loads before the gradient
// they wait for is ready.  P.m may be NULL for an optimizer that keeps no m
// (Adagrad, RMSprop without momentum): it is then neither read nor written;
// v is read and written for every optimizer but SGD.
struct OptState4 { float4 w, m, v; };
struct OptState1 { float w, m, v; };

__device__ __forceinline__ OptState4 opt_load4(const OptK& o, const of_param& P, int64_t off) {
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
  return OptState4{ld4(P.w + off), P.m ? ld4(P.m + off) : z,
                   o.kind != OF_OPT_SGD ? ld4(P.v + off) : z};
}

__device__ __forceinline__ OptState1 opt_load1(const OptK& o, const of_param& P, int64_t off) {
  return OptState1{P.w[off], P.m ? P.m[off] : 0.f, o.kind != OF_OPT_SGD ? P.v[off] : 0.f};
}

// Apply the update with gradient g to a loaded state and store it back.
__device__ __forceinline__ float4 opt_apply4(const OptK& o, const of_param& P, OptState4 s,
                                             float4 g, int64_t off) {
  opt_update(o, s.w.x, g.x, s.m.x, s.v.x);
  opt_update(o, s.w.y, g.y, s.m.y, s.v.y);
  opt_update(o, s.w.z, g.z, s.m.z, s.v.z);
  opt_update(o, s.w.w, g.w, s.m.w, s.v.w);
  st4(P.w + off, s.w);
  if (P.m) st4(P.m + off, s.m);
  if (o.kind != OF_OPT_SGD) st4(P.v + off, s.v);
  if (P.w_bf16) st_bf16x4(P.w_bf16 + off, s.w);
  return s.w;
}

__device__ __forceinline__ float opt_apply1(const OptK& o, const of_param& P, OptState1 s, float g,
                                            int64_t off) {
  opt_update(o, s.w, g, s.m, s.v);
  P.w[off] = s.w;
  if (P.m) P.m[off] = s.m;
  if (o.kind != OF_OPT_SGD) P.v[off] = s.v;
  if (P.w_bf16) P.w_bf16[off] = f32_to_bf16(s.w);
  return s.w;
}

// Update 4 consecutive parameter elements at `off` (all valid, 16B aligned).
__device__ __forceinline__ float4 update4(const OptK& o, const of_param& P, float4 g, int64_t off) {
  return opt_apply4(o, P, opt_load4(o, P, off), g, off);
}

__device__ __forceinline__ float update1(const OptK& o, const of_param& P, float g, int64_t off) {
  return opt_apply1(o, P, opt_load1(o, P, off), g, off);
}

inline bool aligned16(const void* p) { return (((uintptr_t)p) & 15u) == 0; }

// ---------------------------------------------------------------- GEMM API
// C[P,Q] = sum_r A(p,r) B(q,r) with
//   A(p,r) = A[p*a_sp + r*a_sr], one of a_sp / a_sr equal to 1,
//   B(q,r) = B[q*b_sq + r*b_sr], one of b_sq / b_sr equal to 1.

enum EpiKind {
  EPI_FWD = 0,        // y = act(c + bias), z = c + bias
  EPI_FWD_FF = 1,     // forward-fusion: B tiles (W) are updated while loaded
  EPI_DGRAD = 2,      // dx = c * act'(prev)
  EPI_WGRAD = 3,      // dw = c (or +=), db = column sums of A (or +=)
  EPI_WGRAD_BF = 4,   // backward-fusion: update W (and b) from c (and sums)
};

// Convolutions (3x3, stride 1, zero padding 1, NHWC activations, [Cout,3,3,C]
// filters) run as implicit GEMMs: conv != 0 selects gathered operand addressing
// instead of the strides above.
//   forward  C[m, co]   = sum_k X~(m, k) W[co, k]     m=(n,h,w), k=(r,s,c)
//   dgrad    C[m, c]    = sum_k dY~(m, k) W~(c, k)    k=(r,s,co): dY at (h+1-r, w+1-s)
//   wgrad    C[co, k]   = sum_m dY[m, co] X~(k, m)
// Division by a fixed divisor d as a multiply-high and a shift (the
// round-up method of Granlund and Montgomery): for 0 <= n < 2^31,
// n / d == (umulhi(n, m) + n) >> s with s = ceil(log2 d) and
// m = floor(2^32 (2^s - d) / d) + 1.  Set on the host by make_fastdiv().
struct FastDiv {
  uint32_t d, m, s;
};

inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t s = 0;
  while ((1ull << s) < d) ++s;
  const uint64_t m = ((1ull << 32) * ((1ull << s) - d)) / d + 1;
  return FastDiv{d, (uint32_t)m, s};
}

__device__ __forceinline__ int fdiv(int n, const FastDiv& f) {
  const uint32_t t = __umulhi((uint32_t)n, f.m);
  return (int)((t + (uint32_t)n) >> f.s);
}

struct GemmProblem {
  const float* A; int64_t a_sp, a_sr;
  const float* B; int64_t b_sq, b_sr;
  int P, Q, R;
  int conv;                     // 0: strided operands; 1: convolution gathers
  int cN, cH, cW, cC, cCout;    // convolution geometry (input N, H, W, C; Cout)
  int a_bf16, b_bf16;           // bf16 kernels: the operand is stored as bf16 (else fp32)
  FastDiv dW, dH, dC, dCout;    // convolution: divisors of the gather index arithmetic
  int group = 0;                // tile order within an XCD's block: 0 rows of the block, g > 0 strips of g tile rows
};

// Updates carried by a contraction launch (forward-fusion of later
// operators): the workgroups of the z-slices from z0 on apply the optimizer to
// up to OF_CARRY_MAX tensors instead of computing tiles.  A tensor's gradient
// is one vector (rows == 1) or `rows` row partials of stride `ld`, summed in
// row order.
struct CarryTensor {
  of_param p;           // p.w == nullptr: no tensor
  const float* g;
  int64_t rows, ld;
  int vec;              // 128-bit paths allowed (vector gradients)
};
struct CarryArgs {
  CarryTensor t[OF_CARRY_MAX];
  OptK opt;
  int cz;               // leading z-slices that apply the update (dispatched first,
                        // so they run beside the contraction); 0: nothing carried
};

struct EpiArgs {
  // outputs
  float* out; int64_t ldo;      // y (FWD), dx (DGRAD), dw (WGRAD)
  float* z; int64_t ldz;        // FWD: pre-activation (optional)
  uint16_t* yb;                 // FWD (bf16 kernels): y stored as bf16 here, out unused
  const float* res; int64_t ldr;   // FWD: added to y; DGRAD: added to dx (may be NULL)
  const float* prev; int64_t ldp;  // DGRAD: saved tensor of the previous layer
  int act;                      // FWD: activation; DGRAD: previous layer's activation
  int accumulate;               // WGRAD
  // bias
  const float* bias;            // FWD: bias to add (may be NULL)
  float* db;                    // WGRAD: bias gradient out (may be NULL)
  // parameters being updated (FWD_FF: W is the B operand; WGRAD_BF: W is the output)
  of_param W;                   // W.w etc.
  const float* gW;              // FWD_FF: pending gradient; WGRAD_BF: extra gradient (shared use)
  of_param b;                   // FF / BF bias parameter (b.w NULL if none)
  // FF with many readers of each W tile (a convolution): every workgroup reads
  // W, b and their history from the fields above and computes the update;
  // only the workgroups of row tile 0 write it, to these (a second buffer
  // set).  Wout.w == NULL: the update is written in place (one row tile).
  of_param Wout, bout;
  const float* gb;              // FF: pending bias gradient; BF: extra bias gradient
  int with_db;                  // WGRAD: db != NULL; WGRAD_BF: b.w != NULL
  OptK opt;
  CarryArgs carry;              // FWD: a later operator's update (carry.cz == 0: none)
};

size_t gemm_workspace_bytes(int kind, int P, int Q, int R, int conv = 0);
hipError_t gemm_launch(int kind, const GemmProblem& pr, const EpiArgs& ea, void* ws,
                       hipStream_t stream);
// bf16-operand contractions (operands rounded to bf16, fp32 accumulation);
// kinds EPI_FWD, EPI_DGRAD, EPI_WGRAD, EPI_WGRAD_BF; strided operands only.
size_t gemm_bf16_workspace_bytes(int kind, int P, int Q, int R);
hipError_t gemm_bf16_launch(int kind, const GemmProblem& pr, const EpiArgs& ea, void* ws,
                            hipStream_t stream);

// Backward-fusion of a linear layer with at most 64 token rows whose data
// gradient is merged into the update's read of W (fp32 operands).
struct MergedLaunch {
  const float* dz; int64_t ldz;     // dZ [M, ldz]
  const float* x; int64_t ldx;      // X [M, ldx]; also the row stride of prev and dx
  of_param W; const float* gW;      // gW: extra gradient of earlier uses (or NULL)
  of_param b; const float* gb;      // b.w == NULL: no bias
  OptK opt;
  const float* prev; int act_prev;  // the previous layer's saved tensor and activation
  float* dx;                        // NULL: no data gradient
  float* part;                      // workspace: merged_workspace_bytes(M, N, K)
  int M, N, K;
};
constexpr int kMergedMaxM = 64;
hipError_t hbm_stream_launch(int mode, const float* src, float* dst, int64_t n, int blocks,
                             hipStream_t stream);
size_t merged_workspace_bytes(int M, int N, int K);
hipError_t merged_bwd_launch(const MergedLaunch& L, hipStream_t stream);
// The library-owned partials buffer of of_linear_bwd_merged_static: its size,
// and its address on the current device (looked up once per device).
size_t merged_scratch_bytes();
hipError_t merged_scratch_ptr(float** ptr);

// ------------------------------------------------------ depthwise 3x3 conv
size_t dw_workspace_bytes(const of_conv_desc& d);
hipError_t launch_dw_fwd(const of_conv_desc& d, const float* x, const float* w, const float* b,
                         float* y, hipStream_t stream);
hipError_t launch_dw_dgrad(const of_conv_desc& d, const float* dy, const float* w,
                           const float* prev, int act_prev, float* dx, hipStream_t stream);
// o == NULL: eager (writes or adds dw, db); else backward-fusion of W and b.
hipError_t launch_dw_wgrad(const of_conv_desc& d, const float* dy, const float* x, float* dw,
                           float* db, int accumulate, const of_param* W, const of_param* b,
                           const float* gW, const float* gb, const OptK* o, void* ws,
                           hipStream_t stream);

// ------------------------------------------------------ elementwise / losses
hipError_t launch_multi_update(int n, const of_param* params, const float* const* grads,
                               const OptK& o, hipStream_t stream);
hipError_t launch_rows_update(const of_param& p, const float* g, int64_t rows, int64_t ld,
                              const OptK& o, hipStream_t stream);
hipError_t launch_step_advance(int64_t* step_dev, int64_t delta, hipStream_t stream);
hipError_t launch_grad_clip(int n, const of_grad_ref* grads, float max_norm, float* scale,
                            float* norm, double* partial, hipStream_t stream);
hipError_t launch_maxpool_fwd(const float* x, int64_t N, int64_t H, int64_t W, int64_t C,
                              float* y, uint8_t* arg, hipStream_t s);
hipError_t launch_maxpool_bwd(const float* dy, const uint8_t* arg, const float* mask_src,
                              int64_t N, int64_t H, int64_t W, int64_t C, float* dx,
                              hipStream_t s);
hipError_t launch_avgpool_fwd(const float* x, int64_t N, int64_t P, int64_t C, float* y,
                              hipStream_t s);
hipError_t launch_avgpool_bwd(const float* dy, const float* mask_src, int64_t N, int64_t P,
                              int64_t C, float* dx, hipStream_t s);
int64_t ln_partial_rows(int64_t M);
// y: fp32 output, or NULL when yb (the output rounded to bf16) is given.
hipError_t launch_ln_fwd(const float* x, int64_t M, int64_t D, const float* gamma,
                         const float* beta, float eps, float* y, uint16_t* yb, float* mean,
                         float* rstd, hipStream_t s);
hipError_t launch_ln_bwd(const float* dy, const float* x, const float* mean, const float* rstd,
                         const float* gamma, const float* dres, int64_t M, int64_t D, float* dx,
                         float* dgamma_rows, float* dbeta_rows, hipStream_t s);
hipError_t launch_reduce_rows(const float* src, int64_t rows, int64_t ld, int64_t n, float* dst,
                              hipStream_t s);
hipError_t launch_add(const float* a, const float* b, int64_t n, float* out, hipStream_t s);
hipError_t launch_xent(const float* z, const int64_t* labels, int64_t B, int64_t C, int64_t ld,
                       float* loss, float* dz, hipStream_t stream);
size_t mse_ws_bytes(int64_t M, int64_t D);
hipError_t launch_mse(const float* y, const float* t, int64_t M, int64_t D, int64_t ld,
                      float* loss, float* dy, void* ws, hipStream_t stream);

}  // namespace opfuse
