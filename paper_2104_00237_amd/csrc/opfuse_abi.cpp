// C ABI of the opfuse library: argument validation (before any HIP call),
// dispatch to the kernel launchers, thread-local error text.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <unordered_map>

#include "common.h"

using namespace opfuse;

namespace {

thread_local std::string g_err;

of_status fail(of_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

of_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return OF_OK;
  return fail(OF_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool al4(const void* p) { return (((uintptr_t)p) & 3u) == 0; }

#define REQUIRE(cond, st, ...)                   \
  do {                                           \
    if (!(cond)) return fail(st, __VA_ARGS__);   \
  } while (0)

of_status check_opt(const of_opt* o) {
  REQUIRE(o != nullptr, OF_EINVAL, "opt is NULL");
  REQUIRE(o->kind >= OF_OPT_SGD && o->kind <= OF_OPT_ADADELTA, OF_EINVAL,
          "opt->kind %d is not an of_opt_kind", (int)o->kind);
  REQUIRE(o->step_dev != nullptr || o->step >= 1, OF_EINVAL, "opt->step must be >= 1 (got %lld)",
          (long long)o->step);
  REQUIRE((((uintptr_t)o->step_dev) & 7u) == 0, OF_EALIGN, "opt->step_dev must be 8-byte aligned");
  REQUIRE((((uintptr_t)o->grad_scale) & 3u) == 0, OF_EALIGN,
          "opt->grad_scale must be 4-byte aligned");
  REQUIRE(std::isfinite(o->lr) && std::isfinite(o->weight_decay), OF_EINVAL,
          "opt->lr / weight_decay must be finite");
  if (o->kind != OF_OPT_SGD) {
    REQUIRE(o->beta1 >= 0.f && o->beta1 < 1.f && o->beta2 >= 0.f && o->beta2 < 1.f, OF_EINVAL,
            "opt->beta1 / beta2 must be in [0, 1)");
  }
  if (o->kind == OF_OPT_ADAGRAD || o->kind == OF_OPT_RMSPROP || o->kind == OF_OPT_ADADELTA) {
    REQUIRE(o->eps > 0.f && std::isfinite(o->eps), OF_EINVAL,
            "opt->eps must be > 0 for Adagrad, RMSprop and Adadelta");
  }
  return OF_OK;
}

// Whether the optimizer keeps the m tensor (Adagrad and RMSprop without
// momentum do not; their m may be NULL and is then never touched).
bool uses_m(const of_opt& o) {
  return !(o.kind == OF_OPT_ADAGRAD || (o.kind == OF_OPT_RMSPROP && o.momentum == 0.f));
}

of_status check_param(const of_param* p, const char* name, int64_t numel, const of_opt& opt,
                      bool need_w) {
  const int kind = opt.kind;
  REQUIRE(p != nullptr, OF_EINVAL, "%s is NULL", name);
  REQUIRE(p->numel == numel, OF_EINVAL, "%s->numel is %lld, expected %lld", name,
          (long long)p->numel, (long long)numel);
  if (need_w) REQUIRE(p->w != nullptr, OF_EINVAL, "%s->w is NULL", name);
  if (uses_m(opt)) REQUIRE(p->m != nullptr, OF_EINVAL, "%s->m is NULL", name);
  if (kind != OF_OPT_SGD)
    REQUIRE(p->v != nullptr, OF_EINVAL, "%s->v is NULL (every optimizer but SGD needs v)", name);
  REQUIRE(al4(p->w) && al4(p->m) && al4(p->v), OF_EALIGN, "%s arrays must be 4-byte aligned", name);
  REQUIRE((((uintptr_t)p->w_bf16) & 1u) == 0, OF_EALIGN, "%s->w_bf16 must be 2-byte aligned", name);
  return OF_OK;
}

// Validates `c` and fills `out` (z0 is left to the launcher).
of_status make_carry(const of_carry* c, CarryArgs* out) {
  memset(out, 0, sizeof(*out));
  if (c == nullptr) return OF_OK;
  REQUIRE(c->n >= 1 && c->n <= OF_CARRY_MAX, OF_EINVAL, "next->n is %d, not in [1, %d]",
          (int)c->n, OF_CARRY_MAX);
  of_status st = check_opt(&c->opt);
  if (st != OF_OK) return st;
  for (int k = 0; k < c->n; ++k) {
    char name[24];
    snprintf(name, sizeof(name), "next->t[%d]", k);
    const of_param& P = c->t[k];
    REQUIRE(P.numel >= 1, OF_EINVAL, "%s.numel must be >= 1", name);
    if ((st = check_param(&P, name, P.numel, c->opt, true)) != OF_OK) return st;
    REQUIRE(c->g[k] != nullptr, OF_EINVAL, "next->g[%d] is NULL", k);
    REQUIRE(al4(c->g[k]), OF_EALIGN, "next->g[%d] must be 4-byte aligned", k);
    REQUIRE(c->rows[k] >= 1, OF_EINVAL, "next->rows[%d] must be >= 1", k);
    CarryTensor& T = out->t[k];
    T.p = P;
    T.g = c->g[k];
    T.rows = c->rows[k];
    T.ld = P.numel;
    T.vec = T.rows == 1 && aligned16(T.p.w) && aligned16(T.p.m) && aligned16(T.g) &&
            (c->opt.kind == OF_OPT_SGD || aligned16(T.p.v)) &&
            (T.p.w_bf16 == nullptr || (((uintptr_t)T.p.w_bf16) & 7u) == 0);
  }
  out->opt = make_optk(c->opt);
  return OF_OK;
}

of_status check_linear(const of_linear_desc* d) {
  REQUIRE(d != nullptr, OF_EINVAL, "desc is NULL");
  REQUIRE(d->M >= 1 && d->N >= 1 && d->K >= 1, OF_EINVAL, "M, N, K must be >= 1 (got %lld %lld %lld)",
          (long long)d->M, (long long)d->N, (long long)d->K);
  REQUIRE(d->M < (1LL << 31) && d->N < (1LL << 31) && d->K < (1LL << 31), OF_EUNSUPPORTED,
          "M, N, K must be < 2^31");
  REQUIRE(d->ldx == 0 || d->ldx >= d->K, OF_EINVAL, "ldx must be 0 or >= K");
  REQUIRE(d->ldy == 0 || d->ldy >= d->N, OF_EINVAL, "ldy must be 0 or >= N");
  REQUIRE(d->act == OF_ACT_NONE || d->act == OF_ACT_RELU || d->act == OF_ACT_GELU, OF_EINVAL,
          "act %d is not an of_act", (int)d->act);
  REQUIRE(d->dtype == OF_F32 || d->dtype == OF_BF16, OF_EINVAL, "dtype %d is not an of_dtype",
          (int)d->dtype);
  REQUIRE((d->io & ~(OF_IO_X_BF16 | OF_IO_Y_BF16)) == 0, OF_EINVAL,
          "io %d has bits other than OF_IO_X_BF16 | OF_IO_Y_BF16", (int)d->io);
  REQUIRE(d->io == 0 || d->dtype == OF_BF16, OF_EINVAL,
          "bf16 storage of X or Y (io %d) needs dtype OF_BF16", (int)d->io);
  // Operand tiles are read through buffer descriptors based at the tile's
  // first element, with 32-bit byte offsets against a 2^31-1-byte range.  An
  // offset never exceeds the size of the operand matrix it reads from, so every
  // operand (X [M, ldx], W [N, K], Y / Z / dZ [M, ldy], float32 in memory) must
  // stay below 2 GiB; larger shapes would read zeros or wrapped data.
  const int64_t lx = d->ldx ? d->ldx : d->K, ly = d->ldy ? d->ldy : d->N;
  constexpr int64_t kMaxOperandBytes = (1LL << 31) - 16;
  constexpr int64_t kMaxElems = kMaxOperandBytes / 4;
  // (written as divisions: M, N, K < 2^31 but ldx and ldy are unbounded so far)
  REQUIRE(lx <= kMaxElems / d->M && d->K <= kMaxElems / d->N && ly <= kMaxElems / d->M,
          OF_EUNSUPPORTED,
          "operand too large: X [%lld x %lld], W [%lld x %lld] and Y [%lld x %lld] must each be "
          "< 2 GiB (32-bit buffer offsets)",
          (long long)d->M, (long long)lx, (long long)d->N, (long long)d->K, (long long)d->M,
          (long long)ly);
  return OF_OK;
}

// A bf16 shadow of W is only meaningful when the contraction takes bf16 operands.
of_status check_shadow(const of_linear_desc* d, const of_param* W) {
  REQUIRE(d->dtype == OF_BF16 || W == nullptr || W->w_bf16 == nullptr, OF_EINVAL,
          "W->w_bf16 is set but the descriptor's dtype is OF_F32");
  return OF_OK;
}

int64_t ldx_of(const of_linear_desc* d) { return d->ldx ? d->ldx : d->K; }
int64_t ldy_of(const of_linear_desc* d) { return d->ldy ? d->ldy : d->N; }

int kind_of(int32_t op) {
  return op == OF_LINEAR_FWD ? EPI_FWD : op == OF_LINEAR_BWD_DATA ? EPI_DGRAD : EPI_WGRAD;
}

size_t ws_needed(const of_linear_desc* d, int kind) {
  const int M = (int)d->M, N = (int)d->N, K = (int)d->K;
  if (d->dtype == OF_BF16) {
    // bf16 forward-fusion runs its update as a pre-pass, then the plain forward
    switch (kind) {
      case EPI_FWD: case EPI_FWD_FF: return gemm_bf16_workspace_bytes(EPI_FWD, M, N, K);
      case EPI_DGRAD: return gemm_bf16_workspace_bytes(kind, M, K, N);
      default: return gemm_bf16_workspace_bytes(kind, N, K, M);
    }
  }
  switch (kind) {
    case EPI_FWD: case EPI_FWD_FF:
      // one query serves both forwards
      return std::max(gemm_workspace_bytes(EPI_FWD, M, N, K), gemm_workspace_bytes(EPI_FWD_FF, M, N, K));
    case EPI_DGRAD: return gemm_workspace_bytes(kind, M, K, N);
    default: return gemm_workspace_bytes(kind, N, K, M);
  }
}

of_status check_ws(const of_linear_desc* d, int kind, const void* ws, size_t ws_bytes) {
  const size_t need = ws_needed(d, kind);
  REQUIRE(ws_bytes >= need, OF_EWORKSPACE, "workspace of %zu bytes is smaller than the %zu needed",
          ws_bytes, need);
  REQUIRE(need == 0 || ws != nullptr, OF_EWORKSPACE, "workspace is NULL");
  REQUIRE(ws == nullptr || (((uintptr_t)ws) & 15u) == 0, OF_EALIGN, "workspace must be 16-byte aligned");
  return OF_OK;
}

EpiArgs empty_epi() {
  EpiArgs e;
  memset(&e, 0, sizeof(e));
  return e;
}

hipEvent_t side_event() {
  // One event per thread and device: a wait enqueued by hipStreamWaitEvent is
  // bound to the record made before it, so re-recording later is safe.
  thread_local std::unordered_map<int, hipEvent_t> events;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  auto it = events.find(dev);
  if (it != events.end()) return it->second;
  hipEvent_t ev = nullptr;
  if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) return nullptr;
  events[dev] = ev;
  return ev;
}

// Contraction on the fp32 or the bf16 matrix-core path, by the descriptor's dtype.
hipError_t gemm_dispatch(const of_linear_desc* d, int kind, const GemmProblem& pr,
                         const EpiArgs& ea, void* ws, hipStream_t s) {
  return d->dtype == OF_BF16 ? gemm_bf16_launch(kind, pr, ea, ws, s)
                             : gemm_launch(kind, pr, ea, ws, s);
}

// The weight operand: the bf16 shadow when the operands are bf16 and it exists.
void set_weight_operand(const of_linear_desc* d, const of_param* W, GemmProblem& pr) {
  if (d->dtype == OF_BF16 && W->w_bf16) {
    pr.B = reinterpret_cast<const float*>(W->w_bf16);
    pr.b_bf16 = 1;
  } else {
    pr.B = W->w;
  }
}

bool x_bf16(const of_linear_desc* d) { return (d->io & OF_IO_X_BF16) != 0; }
bool y_bf16(const of_linear_desc* d) { return (d->io & OF_IO_Y_BF16) != 0; }

// Alignment of X's storage: 4 bytes for fp32, 2 for bf16 (OF_IO_X_BF16).
bool x_aligned(const of_linear_desc* d, const float* x) {
  return (((uintptr_t)x) & (x_bf16(d) ? 1u : 3u)) == 0;
}

// Launch helpers shared by the entry points (arguments already validated).
of_status run_fwd(const of_linear_desc* d, const float* x, const of_param* W, const float* b,
                  float* z, float* y, void* ws, hipStream_t s, const CarryArgs* carry = nullptr,
                  const float* res = nullptr) {
  GemmProblem pr{x, ldx_of(d), 1, nullptr, d->K, 1, (int)d->M, (int)d->N, (int)d->K};
  set_weight_operand(d, W, pr);
  pr.a_bf16 = x_bf16(d) ? 1 : 0;
  EpiArgs ea = empty_epi();
  ea.ldo = ldy_of(d);
  if (y_bf16(d)) ea.yb = reinterpret_cast<uint16_t*>(y);
  else ea.out = y;
  ea.res = res; ea.ldr = ldy_of(d);
  ea.z = z; ea.ldz = ldy_of(d);
  ea.act = d->act;
  ea.bias = d->has_bias ? b : nullptr;
  if (carry) ea.carry = *carry;
  return hip_status(gemm_dispatch(d, EPI_FWD, pr, ea, ws, s), "of_linear_fwd launch");
}

of_status run_dgrad(const of_linear_desc* d, const float* dz, const of_param* W, const float* prev,
                    int32_t act_prev, float* dx, void* ws, hipStream_t s,
                    const float* res = nullptr) {
  // dX[m,k] = sum_n dZ[m,n] W[n,k]: A = dZ (reduction-contiguous), B(k, n) = W[n*K + k].
  GemmProblem pr{dz, ldy_of(d), 1, nullptr, 1, d->K, (int)d->M, (int)d->K, (int)d->N};
  set_weight_operand(d, W, pr);
  EpiArgs ea = empty_epi();
  ea.out = dx; ea.ldo = ldx_of(d);
  ea.prev = prev; ea.ldp = ldx_of(d);
  ea.act = act_prev;
  ea.res = res; ea.ldr = ldx_of(d);
  return hip_status(gemm_dispatch(d, EPI_DGRAD, pr, ea, ws, s), "dgrad launch");
}

GemmProblem wgrad_problem(const of_linear_desc* d, const float* dz, const float* x) {
  // dW[n,k] = sum_m dZ[m,n] X[m,k]: A(n, m) = dZ[m*ldy + n], B(k, m) = X[m*ldx + k].
  GemmProblem pr{dz, 1, ldy_of(d), x, 1, ldx_of(d), (int)d->N, (int)d->K, (int)d->M};
  pr.b_bf16 = x_bf16(d) ? 1 : 0;   // X stored as bf16 is read as stored
  return pr;
}

of_status check_act_prev(int32_t act_prev, const float* prev) {
  REQUIRE(act_prev == OF_ACT_NONE || act_prev == OF_ACT_RELU || act_prev == OF_ACT_GELU, OF_EINVAL,
          "act_prev %d is not an of_act", (int)act_prev);
  REQUIRE(act_prev == OF_ACT_NONE || prev != nullptr, OF_EINVAL,
          "prev is NULL but act_prev needs the previous layer's saved tensor");
  REQUIRE(al4(prev), OF_EALIGN, "prev must be 4-byte aligned");
  return OF_OK;
}

of_status check_conv(const of_conv_desc* d) {
  REQUIRE(d != nullptr, OF_EINVAL, "desc is NULL");
  REQUIRE(d->N >= 1 && d->H >= 1 && d->W >= 1 && d->C >= 1 && d->Cout >= 1, OF_EINVAL,
          "N, H, W, C, Cout must be >= 1");
  REQUIRE(d->N * d->H * d->W < (1LL << 31) && 9 * d->C * d->Cout < (1LL << 31), OF_EUNSUPPORTED,
          "convolution too large for 32-bit indexing");
  REQUIRE(d->N * d->H * d->W * std::max(d->C, d->Cout) * 4 < (1LL << 31), OF_EUNSUPPORTED,
          "activation tensors must be < 2 GiB");
  REQUIRE(d->act == OF_ACT_NONE || d->act == OF_ACT_RELU, OF_EUNSUPPORTED,
          "convolutions support OF_ACT_NONE and OF_ACT_RELU");
  REQUIRE(d->stride == 0 || d->stride == 1, OF_EUNSUPPORTED,
          "3x3 convolutions run with stride 1 (got stride %d)", (int)d->stride);
  return OF_OK;
}

GemmProblem conv_problem(const of_conv_desc* d, int kind, const float* a, const float* b) {
  const int NHW = (int)(d->N * d->H * d->W), C = (int)d->C, Co = (int)d->Cout;
  GemmProblem pr{};
  pr.conv = 1;
  pr.cN = (int)d->N; pr.cH = (int)d->H; pr.cW = (int)d->W; pr.cC = C; pr.cCout = Co;
  pr.dW = make_fastdiv((uint32_t)d->W); pr.dH = make_fastdiv((uint32_t)d->H);
  pr.dC = make_fastdiv((uint32_t)C); pr.dCout = make_fastdiv((uint32_t)Co);
  pr.A = a; pr.B = b;
  if (kind == EPI_FWD) {          // A = x gathered, B = W [Cout, 9C]
    pr.P = NHW; pr.Q = Co; pr.R = 9 * C; pr.b_sq = 9 * C; pr.b_sr = 1;
  } else if (kind == EPI_DGRAD) { // A = dy gathered, B = W gathered
    pr.P = NHW; pr.Q = C; pr.R = 9 * Co;
  } else {                        // A = dy [NHW, Cout], B = x gathered
    pr.P = Co; pr.Q = 9 * C; pr.R = NHW; pr.a_sp = 1; pr.a_sr = Co;
  }
  return pr;
}

size_t conv_ws(const of_conv_desc* d, int kind) {
  const GemmProblem pr = conv_problem(d, kind, nullptr, nullptr);
  return gemm_workspace_bytes(kind, pr.P, pr.Q, pr.R, 1);
}

of_status check_conv_ws(const of_conv_desc* d, int kind, const void* ws, size_t ws_bytes) {
  const size_t need = conv_ws(d, kind);
  REQUIRE(ws_bytes >= need, OF_EWORKSPACE, "workspace of %zu bytes is smaller than the %zu needed",
          ws_bytes, need);
  REQUIRE(need == 0 || ws != nullptr, OF_EWORKSPACE, "workspace is NULL");
  REQUIRE(ws == nullptr || (((uintptr_t)ws) & 15u) == 0, OF_EALIGN, "workspace must be 16-byte aligned");
  return OF_OK;
}

}  // namespace

namespace opfuse {
OptK make_optk(const of_opt& o) {
  OptK k;
  k.kind = o.kind;
  k.lr = o.lr;
  k.wd = o.weight_decay;
  k.mom = o.momentum;
  k.b1 = o.beta1;
  k.b2 = o.beta2;
  k.eps = o.eps;
  k.omb1 = (float)(1.0 - (double)o.beta1);
  k.omb2 = (float)(1.0 - (double)o.beta2);
  k.decay = (float)(1.0 - (double)o.lr * (double)o.weight_decay);
  k.step = o.step;
  k.step_dev = o.step_dev;
  k.gscale_dev = o.grad_scale;
  k.gscale = 1.f;
  k.step_size = 0.f;
  k.rsqrt_bc2 = 0.f;
  k.prepared = 0;
  if (o.step_dev == nullptr && o.kind != OF_OPT_SGD) {
    opt_constants(k, o.step);
    k.prepared = 1;
  }
  return k;
}
}  // namespace opfuse

extern "C" {

int of_version(void) { return OF_VERSION; }

const char* of_last_error(void) { return g_err.c_str(); }

// The merged backward's supported descriptors.
of_status check_merged(const of_linear_desc* d) {
  REQUIRE(d->dtype == OF_F32, OF_EUNSUPPORTED, "of_linear_bwd_merged takes fp32 operands only");
  REQUIRE(d->M <= kMergedMaxM, OF_EUNSUPPORTED, "of_linear_bwd_merged needs M <= %d (got %lld)",
          kMergedMaxM, (long long)d->M);
  REQUIRE(d->K <= (1LL << 22) && ldx_of(d) <= (1LL << 22) && ldy_of(d) <= (1LL << 22),
          OF_EUNSUPPORTED, "of_linear_bwd_merged needs K, ldx and ldy <= 2^22");
  return OF_OK;
}

size_t of_linear_workspace_size(const of_linear_desc* d, int32_t op) {
  if (check_linear(d) != OF_OK) return 0;
  if (op < OF_LINEAR_FWD || op > OF_LINEAR_BWD_MERGED) {
    fail(OF_EINVAL, "op %d is not an of_linear_op", (int)op);
    return 0;
  }
  if (op == OF_LINEAR_BWD_MERGED) {
    if (check_merged(d) != OF_OK) return 0;
    return merged_workspace_bytes((int)d->M, (int)d->N, (int)d->K);
  }
  return ws_needed(d, kind_of(op));
}

of_status of_linear_fwd(const of_linear_desc* d, const float* x, const of_param* W, const float* b,
                        float* z, float* y, void* ws, size_t ws_bytes, void* stream) {
  return of_linear_fwd_carry(d, x, W, b, z, y, nullptr, ws, ws_bytes, stream);
}

namespace {
// of_linear_fwd_carry and of_linear_fwd_res (res: residual or NULL).
of_status fwd_entry(const of_linear_desc* d, const float* x, const of_param* W, const float* b,
                    const float* res, float* z, float* y, const of_carry* next, void* ws,
                    size_t ws_bytes, void* stream) {
  of_status st = check_linear(d);
  if (st != OF_OK) return st;
  if (res) {
    // read once per element by the thread that writes it: in place is safe,
    // any other overlap with y or z is not
    const int64_t bytes = (d->M - 1) * ldy_of(d) * 4 + d->N * 4;
    const int64_t ybytes = (d->M - 1) * ldy_of(d) * (y_bf16(d) ? 2 : 4) + d->N * (y_bf16(d) ? 2 : 4);
    auto apart = [&](const void* o, int64_t ob) {
      const uintptr_t a = (uintptr_t)res, c = (uintptr_t)o;
      return o == nullptr || a + (uintptr_t)bytes <= c || c + (uintptr_t)ob <= a;
    };
    REQUIRE(al4(res), OF_EALIGN, "res must be 4-byte aligned");
    REQUIRE((res == y && !y_bf16(d)) || apart(y, ybytes), OF_EINVAL,
            "res must be y itself (fp32 Y) or not overlap it");
    REQUIRE(apart(z, bytes), OF_EINVAL, "res must not overlap z");
  }
  REQUIRE(x && W && W->w && y, OF_EINVAL, "x, W, W->w and y are required");
  REQUIRE(W->numel == d->N * d->K, OF_EINVAL, "W->numel must be N*K");
  REQUIRE(!d->has_bias || b, OF_EINVAL, "has_bias is set but b is NULL");
  REQUIRE(d->act != OF_ACT_GELU || z, OF_EINVAL, "GELU needs z (its derivative reads Z)");
  REQUIRE(al4(W->w) && al4(b) && al4(z), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  REQUIRE(x_aligned(d, x), OF_EALIGN, "x must be %d-byte aligned", x_bf16(d) ? 2 : 4);
  REQUIRE((((uintptr_t)y) & (y_bf16(d) ? 1u : 3u)) == 0, OF_EALIGN, "y must be %d-byte aligned",
          y_bf16(d) ? 2 : 4);
  REQUIRE((((uintptr_t)W->w_bf16) & 1u) == 0, OF_EALIGN, "W->w_bf16 must be 2-byte aligned");
  REQUIRE(!x_bf16(d) || W->w_bf16, OF_EINVAL,
          "X stored as bf16 (OF_IO_X_BF16) needs the weight's bf16 shadow W->w_bf16");
  if ((st = check_shadow(d, W)) != OF_OK) return st;
  if ((st = check_ws(d, EPI_FWD, ws, ws_bytes)) != OF_OK) return st;
  CarryArgs carry;
  if ((st = make_carry(next, &carry)) != OF_OK) return st;
  return run_fwd(d, x, W, b, z, y, ws, (hipStream_t)stream, next ? &carry : nullptr, res);
}
}  // namespace

of_status of_linear_fwd_carry(const of_linear_desc* d, const float* x, const of_param* W,
                              const float* b, float* z, float* y, const of_carry* next,
                              void* ws, size_t ws_bytes, void* stream) {
  return fwd_entry(d, x, W, b, nullptr, z, y, next, ws, ws_bytes, stream);
}

of_status of_linear_fwd_res(const of_linear_desc* d, const float* x, const of_param* W,
                            const float* b, const float* res, float* z, float* y,
                            const of_carry* next, void* ws, size_t ws_bytes, void* stream) {
  REQUIRE(res != nullptr, OF_EINVAL, "res is required (of_linear_fwd_carry has none)");
  return fwd_entry(d, x, W, b, res, z, y, next, ws, ws_bytes, stream);
}

// Largest M whose forward-fusion can write its update in place: the M rows
// fit one row tile, so each W element has one reader.
constexpr int64_t kFusedForwardMaxRows = 64;

of_status of_linear_fwd_fused(const of_linear_desc* d, const float* x, const of_param* W,
                              const of_param* W_out, const float* gW, const of_param* b,
                              const of_param* b_out, const float* gb, const of_opt* opt,
                              float* z, float* y, void* ws, size_t ws_bytes, void* stream) {
  if (opt == nullptr) return of_linear_fwd(d, x, W, b ? b->w : nullptr, z, y, ws, ws_bytes, stream);
  of_status st = check_linear(d);
  if (st != OF_OK) return st;
  if ((st = check_opt(opt)) != OF_OK) return st;
  REQUIRE(x && y && gW, OF_EINVAL, "x, y and gW are required");
  if ((st = check_param(W, "W", d->N * d->K, *opt, true)) != OF_OK) return st;
  if (d->has_bias) {
    if ((st = check_param(b, "b", d->N, *opt, true)) != OF_OK) return st;
    REQUIRE(gb != nullptr, OF_EINVAL, "has_bias is set but gb is NULL");
  }
  REQUIRE(d->act != OF_ACT_GELU || z, OF_EINVAL, "GELU needs z");
  REQUIRE(al4(x) && al4(gW) && al4(gb) && al4(z) && al4(y), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  if ((st = check_shadow(d, W)) != OF_OK) return st;
  REQUIRE(d->dtype == OF_F32, OF_EUNSUPPORTED,
          "of_linear_fwd_fused takes fp32 operands: with bf16 operands every row tile would "
          "read the fp32 weight, gradient and history (16 B per element) in place of the 2-byte "
          "shadow; apply the pending update with of_linear_fwd_carry or "
          "of_elementwise_fused_update instead");
  if (W_out) {
    // every row tile reads the current set while row tile 0 writes the new one
    if ((st = check_param(W_out, "W_out", d->N * d->K, *opt, true)) != OF_OK) return st;
    REQUIRE(W_out->w != W->w && (W->m == nullptr || W_out->m != W->m) &&
                (W->v == nullptr || W_out->v != W->v),
            OF_EINVAL, "W_out must not share buffers with W");
    REQUIRE(!d->has_bias || b_out, OF_EINVAL, "W_out is set and has_bias: b_out is required");
    if (d->has_bias) {
      if ((st = check_param(b_out, "b_out", d->N, *opt, true)) != OF_OK) return st;
      REQUIRE(b_out->w != b->w && (b->m == nullptr || b_out->m != b->m) &&
                  (b->v == nullptr || b_out->v != b->v),
              OF_EINVAL, "b_out must not share buffers with b");
    }
  } else {
    REQUIRE(d->M <= kFusedForwardMaxRows, OF_EUNSUPPORTED,
            "in-place forward-fusion needs the M rows in one row tile (M <= %lld, got %lld): "
            "pass W_out (and b_out) to have the update written to a second buffer set",
            (long long)kFusedForwardMaxRows, (long long)d->M);
    REQUIRE(b_out == nullptr, OF_EINVAL, "b_out without W_out");
  }
  if ((st = check_ws(d, EPI_FWD_FF, ws, ws_bytes)) != OF_OK) return st;
  GemmProblem pr{x, ldx_of(d), 1, W->w, d->K, 1, (int)d->M, (int)d->N, (int)d->K};
  EpiArgs ea = empty_epi();
  ea.out = y; ea.ldo = ldy_of(d);
  ea.z = z; ea.ldz = ldy_of(d);
  ea.act = d->act;
  ea.W = *W;
  if (W_out) ea.Wout = *W_out;
  ea.gW = gW;
  if (d->has_bias) {
    ea.b = *b;
    ea.gb = gb;
    if (W_out) ea.bout = *b_out;
  }
  ea.opt = make_optk(*opt);
  return hip_status(gemm_launch(EPI_FWD_FF, pr, ea, ws, (hipStream_t)stream),
                    "of_linear_fwd_fused launch");
}

namespace {
// of_linear_bwd_data and of_linear_bwd_data_res (res: residual gradient or NULL).
of_status bwd_data_entry(const of_linear_desc* d, const float* dz, const of_param* W,
                         const float* prev, int32_t act_prev, const float* res, float* dx,
                         void* ws, size_t ws_bytes, void* stream) {
  of_status st = check_linear(d);
  if (st != OF_OK) return st;
  if (res) {
    // read once per element by the thread that writes it: in place is safe
    const int64_t bytes = ((d->M - 1) * ldx_of(d) + d->K) * 4;
    const uintptr_t a = (uintptr_t)res, c = (uintptr_t)dx;
    REQUIRE(al4(res), OF_EALIGN, "res must be 4-byte aligned");
    REQUIRE(res == dx || dx == nullptr || a + (uintptr_t)bytes <= c || c + (uintptr_t)bytes <= a,
            OF_EINVAL, "res must be dx itself or not overlap it");
  }
  REQUIRE(dz && W && W->w && dx, OF_EINVAL, "dz, W, W->w and dx are required");
  REQUIRE(W->numel == d->N * d->K, OF_EINVAL, "W->numel must be N*K");
  if ((st = check_act_prev(act_prev, prev)) != OF_OK) return st;
  REQUIRE(al4(dz) && al4(W->w) && al4(dx), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  REQUIRE((((uintptr_t)W->w_bf16) & 1u) == 0, OF_EALIGN, "W->w_bf16 must be 2-byte aligned");
  if ((st = check_shadow(d, W)) != OF_OK) return st;
  if ((st = check_ws(d, EPI_DGRAD, ws, ws_bytes)) != OF_OK) return st;
  return run_dgrad(d, dz, W, prev, act_prev, dx, ws, (hipStream_t)stream, res);
}
}  // namespace

of_status of_linear_bwd_data(const of_linear_desc* d, const float* dz, const of_param* W,
                             const float* prev, int32_t act_prev, float* dx, void* ws,
                             size_t ws_bytes, void* stream) {
  return bwd_data_entry(d, dz, W, prev, act_prev, nullptr, dx, ws, ws_bytes, stream);
}

of_status of_linear_bwd_data_res(const of_linear_desc* d, const float* dz, const of_param* W,
                                 const float* prev, int32_t act_prev, const float* res,
                                 float* dx, void* ws, size_t ws_bytes, void* stream) {
  REQUIRE(res != nullptr, OF_EINVAL, "res is required (of_linear_bwd_data has none)");
  return bwd_data_entry(d, dz, W, prev, act_prev, res, dx, ws, ws_bytes, stream);
}

of_status of_linear_bwd_weight(const of_linear_desc* d, const float* dz, const float* x, float* dw,
                               float* db, int32_t accumulate, void* ws, size_t ws_bytes,
                               void* stream) {
  of_status st = check_linear(d);
  if (st != OF_OK) return st;
  REQUIRE(dz && x && dw, OF_EINVAL, "dz, x and dw are required");
  REQUIRE(al4(dz) && al4(dw) && al4(db), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  REQUIRE(x_aligned(d, x), OF_EALIGN, "x must be %d-byte aligned", x_bf16(d) ? 2 : 4);
  if ((st = check_ws(d, EPI_WGRAD, ws, ws_bytes)) != OF_OK) return st;
  EpiArgs ea = empty_epi();
  ea.out = dw; ea.ldo = d->K;
  ea.db = db;
  ea.with_db = db != nullptr;
  ea.accumulate = accumulate ? 1 : 0;
  return hip_status(gemm_dispatch(d, EPI_WGRAD, wgrad_problem(d, dz, x), ea, ws, (hipStream_t)stream),
                    "of_linear_bwd_weight launch");
}

of_status of_linear_bwd_fused(const of_linear_desc* d, const float* dz, const float* x,
                              const of_param* W, const of_param* b, const float* gW_partial,
                              const float* gb_partial, const of_opt* opt, const float* prev,
                              int32_t act_prev, float* dx_prev, void* ws, size_t ws_bytes,
                              void* ws_update, size_t ws_update_bytes, void* stream,
                              void* update_stream) {
  of_status st = check_linear(d);
  if (st != OF_OK) return st;
  if ((st = check_opt(opt)) != OF_OK) return st;
  REQUIRE(dz && x, OF_EINVAL, "dz and x are required");
  if ((st = check_param(W, "W", d->N * d->K, *opt, true)) != OF_OK) return st;
  if (b) {
    if ((st = check_param(b, "b", d->N, *opt, true)) != OF_OK) return st;
  }
  REQUIRE(al4(dz) && al4(gW_partial) && al4(gb_partial) && al4(dx_prev), OF_EALIGN,
          "fp32 pointers must be 4-byte aligned");
  REQUIRE(x_aligned(d, x), OF_EALIGN, "x must be %d-byte aligned", x_bf16(d) ? 2 : 4);
  if (dx_prev) {
    if ((st = check_act_prev(act_prev, prev)) != OF_OK) return st;
    if ((st = check_ws(d, EPI_DGRAD, ws, ws_bytes)) != OF_OK) return st;
  }
  if ((st = check_shadow(d, W)) != OF_OK) return st;
  if ((st = check_ws(d, EPI_WGRAD_BF, ws_update, ws_update_bytes)) != OF_OK) return st;
  const hipStream_t s = (hipStream_t)stream;
  hipStream_t su = s;
  hipEvent_t ev = nullptr;
  if (update_stream != nullptr && update_stream != stream) {
    ev = side_event();
    REQUIRE(ev != nullptr, OF_EHIP, "could not create the side-stream event");
    su = (hipStream_t)update_stream;
  }
  if (dx_prev) {
    // Data gradient first, with the old W (the dependency rule after Alg. 3).
    if ((st = run_dgrad(d, dz, W, prev, act_prev, dx_prev, ws, s)) != OF_OK) return st;
  }
  if (ev) {
    if ((st = hip_status(hipEventRecord(ev, s), "hipEventRecord")) != OF_OK) return st;
    if ((st = hip_status(hipStreamWaitEvent(su, ev, 0), "hipStreamWaitEvent")) != OF_OK) return st;
  }
  EpiArgs ea = empty_epi();
  ea.ldo = d->K;
  ea.W = *W;
  ea.gW = gW_partial;
  if (b) { ea.b = *b; ea.gb = gb_partial; }
  ea.with_db = b != nullptr;
  ea.opt = make_optk(*opt);
  return hip_status(gemm_dispatch(d, EPI_WGRAD_BF, wgrad_problem(d, dz, x), ea, ws_update, su),
                    "of_linear_bwd_fused launch");
}

namespace {
// Shared by of_linear_bwd_merged (caller workspace) and
// of_linear_bwd_merged_static (library scratch: use_scratch, ws unused).
of_status merged_entry(const of_linear_desc* d, const float* dz, const float* x,
                       const of_param* W, const of_param* b, const float* gW_partial,
                       const float* gb_partial, const of_opt* opt, const float* prev,
                       int32_t act_prev, float* dx_prev, void* ws, size_t ws_bytes,
                       void* stream, bool use_scratch) {
  of_status st = check_linear(d);
  if (st != OF_OK) return st;
  if ((st = check_merged(d)) != OF_OK) return st;
  if ((st = check_opt(opt)) != OF_OK) return st;
  REQUIRE(dz && x, OF_EINVAL, "dz and x are required");
  if ((st = check_param(W, "W", d->N * d->K, *opt, true)) != OF_OK) return st;
  if (b) {
    if ((st = check_param(b, "b", d->N, *opt, true)) != OF_OK) return st;
  }
  REQUIRE(al4(dz) && al4(x) && al4(gW_partial) && al4(gb_partial) && al4(dx_prev) && al4(prev),
          OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  if ((st = check_shadow(d, W)) != OF_OK) return st;
  const size_t need = merged_workspace_bytes((int)d->M, (int)d->N, (int)d->K);
  float* part = static_cast<float*>(ws);
  if (dx_prev) {
    if ((st = check_act_prev(act_prev, prev)) != OF_OK) return st;
    if (use_scratch) {
      REQUIRE(need <= merged_scratch_bytes(), OF_EUNSUPPORTED,
              "of_linear_bwd_merged_static: this shape needs %zu bytes of partials, more than "
              "the library's %zu-byte scratch (use of_linear_bwd_merged with a workspace)",
              need, merged_scratch_bytes());
      if ((st = hip_status(merged_scratch_ptr(&part), "of_linear_bwd_merged_static scratch")) !=
          OF_OK)
        return st;
    } else {
      REQUIRE(ws_bytes >= need, OF_EWORKSPACE,
              "workspace of %zu bytes is smaller than the %zu needed", ws_bytes, need);
      REQUIRE(ws != nullptr, OF_EWORKSPACE, "workspace is NULL");
      REQUIRE((((uintptr_t)ws) & 15u) == 0, OF_EALIGN, "workspace must be 16-byte aligned");
    }
  }
  MergedLaunch L;
  L.dz = dz; L.ldz = ldy_of(d);
  L.x = x; L.ldx = ldx_of(d);
  L.W = *W; L.gW = gW_partial;
  if (b) { L.b = *b; } else { memset(&L.b, 0, sizeof(L.b)); }
  L.gb = b ? gb_partial : nullptr;
  L.opt = make_optk(*opt);
  L.prev = prev; L.act_prev = act_prev;
  L.dx = dx_prev;
  L.part = part;
  L.M = (int)d->M; L.N = (int)d->N; L.K = (int)d->K;
  return hip_status(merged_bwd_launch(L, (hipStream_t)stream),
                    use_scratch ? "of_linear_bwd_merged_static launch" : "of_linear_bwd_merged launch");
}
}  // namespace

of_status of_linear_bwd_merged(const of_linear_desc* d, const float* dz, const float* x,
                               const of_param* W, const of_param* b, const float* gW_partial,
                               const float* gb_partial, const of_opt* opt, const float* prev,
                               int32_t act_prev, float* dx_prev, void* ws, size_t ws_bytes,
                               void* stream) {
  return merged_entry(d, dz, x, W, b, gW_partial, gb_partial, opt, prev, act_prev, dx_prev, ws,
                      ws_bytes, stream, false);
}

of_status of_linear_bwd_merged_static(const of_linear_desc* d, const float* dz, const float* x,
                                      const of_param* W, const of_param* b,
                                      const float* gW_partial, const float* gb_partial,
                                      const of_opt* opt, const float* prev, int32_t act_prev,
                                      float* dx_prev, void* stream) {
  return merged_entry(d, dz, x, W, b, gW_partial, gb_partial, opt, prev, act_prev, dx_prev,
                      nullptr, 0, stream, true);
}

of_status of_hbm_stream(int32_t mode, const float* src, float* dst, int64_t n, int32_t blocks,
                        void* stream) {
  REQUIRE(mode == OF_STREAM_READ || mode == OF_STREAM_COPY || mode == OF_STREAM_RMW ||
              mode == OF_STREAM_RMW3 || mode == OF_STREAM_RMW3_COLUMNS,
          OF_EINVAL, "mode %d is not an OF_STREAM_* mode", (int)mode);
  const bool rmw = mode == OF_STREAM_RMW || mode == OF_STREAM_RMW3 ||
                   mode == OF_STREAM_RMW3_COLUMNS;
  REQUIRE(mode != OF_STREAM_RMW3_COLUMNS || (n > 0 && n % (3LL * 8192 * 32) == 0), OF_EINVAL,
          "OF_STREAM_RMW3_COLUMNS: n must be a positive multiple of 3 * 8192 * 32 (three "
          "arrays of whole 32-row chunks of 8192-float rows; got %lld)", (long long)n);
  REQUIRE(dst && (src || rmw), OF_EINVAL,
          "dst is required, and src unless the mode is a read-modify-write");
  REQUIRE(n >= 4 && n % 4 == 0, OF_EINVAL, "n must be a positive multiple of 4 (got %lld)",
          (long long)n);
  REQUIRE(mode != OF_STREAM_RMW3 || n % 12 == 0, OF_EINVAL,
          "OF_STREAM_RMW3: n must be a multiple of 12 (three arrays of float4s; got %lld)",
          (long long)n);
  REQUIRE(blocks >= 0 && blocks <= 65535, OF_EINVAL, "blocks must be in [0, 65535]");
  if (rmw)
    REQUIRE(aligned16(dst), OF_EALIGN, "dst must be 16-byte aligned");
  else
    REQUIRE(aligned16(src) && (mode == OF_STREAM_READ ? al4(dst) : aligned16(dst)), OF_EALIGN,
            "src (and dst when copying) must be 16-byte aligned");
  return hip_status(hbm_stream_launch(mode, src, dst, n, blocks, (hipStream_t)stream),
                    "of_hbm_stream launch");
}

size_t of_conv_workspace_size(const of_conv_desc* d, int32_t op) {
  if (check_conv(d) != OF_OK) return 0;
  if (op < OF_CONV_FWD || op > OF_CONV_BWD_WEIGHT) {
    fail(OF_EINVAL, "op %d is not an of_conv_op", (int)op);
    return 0;
  }
  const int kind = op == OF_CONV_FWD ? EPI_FWD : op == OF_CONV_BWD_DATA ? EPI_DGRAD : EPI_WGRAD;
  return conv_ws(d, kind);
}

of_status of_conv_fwd(const of_conv_desc* d, const float* x, const of_param* W, const float* b,
                      float* y, void* ws, size_t ws_bytes, void* stream) {
  return of_conv_fwd_carry(d, x, W, b, y, nullptr, ws, ws_bytes, stream);
}

of_status of_conv_fwd_carry(const of_conv_desc* d, const float* x, const of_param* W,
                            const float* b, float* y, const of_carry* next, void* ws,
                            size_t ws_bytes, void* stream) {
  of_status st = check_conv(d);
  if (st != OF_OK) return st;
  REQUIRE(x && W && W->w && y, OF_EINVAL, "x, W, W->w and y are required");
  REQUIRE(W->numel == 9 * d->C * d->Cout, OF_EINVAL, "W->numel must be Cout*9*C");
  REQUIRE(!d->has_bias || b, OF_EINVAL, "has_bias is set but b is NULL");
  REQUIRE(al4(x) && al4(W->w) && al4(b) && al4(y), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  if ((st = check_conv_ws(d, EPI_FWD, ws, ws_bytes)) != OF_OK) return st;
  EpiArgs ea = empty_epi();
  if ((st = make_carry(next, &ea.carry)) != OF_OK) return st;
  ea.out = y; ea.ldo = d->Cout;
  ea.act = d->act;
  ea.bias = d->has_bias ? b : nullptr;
  return hip_status(gemm_launch(EPI_FWD, conv_problem(d, EPI_FWD, x, W->w), ea, ws,
                                (hipStream_t)stream), "of_conv_fwd launch");
}

of_status of_conv_fwd_fused(const of_conv_desc* d, const float* x, const of_param* W,
                            const of_param* W_out, const float* gW, const of_param* b,
                            const of_param* b_out, const float* gb, const of_opt* opt, float* y,
                            void* ws, size_t ws_bytes, void* stream) {
  of_status st = check_conv(d);
  if (st != OF_OK) return st;
  if ((st = check_opt(opt)) != OF_OK) return st;
  REQUIRE(x && y && gW, OF_EINVAL, "x, y and gW are required");
  const int64_t nw = 9 * d->C * d->Cout;
  if ((st = check_param(W, "W", nw, *opt, true)) != OF_OK) return st;
  if ((st = check_param(W_out, "W_out", nw, *opt, true)) != OF_OK) return st;
  REQUIRE(W->w_bf16 == nullptr && W_out->w_bf16 == nullptr, OF_EINVAL,
          "convolutions take fp32 filters (no bf16 shadow)");
  // every workgroup reads the old generation while row tile 0 writes the new one
  REQUIRE(W_out->w != W->w && (W->m == nullptr || W_out->m != W->m) &&
          (W->v == nullptr || W_out->v != W->v), OF_EINVAL,
          "W_out must not share buffers with W");
  REQUIRE(!d->has_bias || (b && b_out && gb), OF_EINVAL, "has_bias needs b, b_out and gb");
  if (d->has_bias) {
    if ((st = check_param(b, "b", d->Cout, *opt, true)) != OF_OK) return st;
    if ((st = check_param(b_out, "b_out", d->Cout, *opt, true)) != OF_OK) return st;
    REQUIRE(b_out->w != b->w && (b->m == nullptr || b_out->m != b->m) &&
            (b->v == nullptr || b_out->v != b->v), OF_EINVAL,
            "b_out must not share buffers with b");
  }
  REQUIRE(al4(x) && al4(y) && al4(gW) && al4(gb), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  if ((st = check_conv_ws(d, EPI_FWD, ws, ws_bytes)) != OF_OK) return st;
  EpiArgs ea = empty_epi();
  ea.out = y; ea.ldo = d->Cout;
  ea.act = d->act;
  ea.W = *W; ea.Wout = *W_out; ea.gW = gW;
  if (d->has_bias) { ea.b = *b; ea.bout = *b_out; ea.gb = gb; }
  ea.opt = make_optk(*opt);
  return hip_status(gemm_launch(EPI_FWD_FF, conv_problem(d, EPI_FWD, x, W->w), ea, ws,
                                (hipStream_t)stream), "of_conv_fwd_fused launch");
}

of_status of_conv_bwd_data(const of_conv_desc* d, const float* dy, const of_param* W,
                           const float* prev, int32_t act_prev, float* dx, void* ws,
                           size_t ws_bytes, void* stream) {
  of_status st = check_conv(d);
  if (st != OF_OK) return st;
  REQUIRE(dy && W && W->w && dx, OF_EINVAL, "dy, W, W->w and dx are required");
  REQUIRE(W->numel == 9 * d->C * d->Cout, OF_EINVAL, "W->numel must be Cout*9*C");
  if ((st = check_act_prev(act_prev, prev)) != OF_OK) return st;
  REQUIRE(act_prev != OF_ACT_GELU, OF_EUNSUPPORTED, "convolutions support ReLU only");
  REQUIRE(al4(dy) && al4(W->w) && al4(dx), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  if ((st = check_conv_ws(d, EPI_DGRAD, ws, ws_bytes)) != OF_OK) return st;
  EpiArgs ea = empty_epi();
  ea.out = dx; ea.ldo = d->C;
  ea.prev = prev; ea.ldp = d->C;
  ea.act = act_prev;
  return hip_status(gemm_launch(EPI_DGRAD, conv_problem(d, EPI_DGRAD, dy, W->w), ea, ws,
                                (hipStream_t)stream), "of_conv_bwd_data launch");
}

of_status of_conv_bwd_weight(const of_conv_desc* d, const float* dy, const float* x, float* dw,
                             float* db, int32_t accumulate, void* ws, size_t ws_bytes,
                             void* stream) {
  of_status st = check_conv(d);
  if (st != OF_OK) return st;
  REQUIRE(dy && x && dw, OF_EINVAL, "dy, x and dw are required");
  REQUIRE(al4(dy) && al4(x) && al4(dw) && al4(db), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  if ((st = check_conv_ws(d, EPI_WGRAD, ws, ws_bytes)) != OF_OK) return st;
  EpiArgs ea = empty_epi();
  ea.out = dw; ea.ldo = 9 * d->C;
  ea.db = db;
  ea.with_db = db != nullptr;
  ea.accumulate = accumulate ? 1 : 0;
  return hip_status(gemm_launch(EPI_WGRAD, conv_problem(d, EPI_WGRAD, dy, x), ea, ws,
                                (hipStream_t)stream), "of_conv_bwd_weight launch");
}

of_status of_conv_wgrad_fused(const of_conv_desc* d, const float* dy, const float* x,
                              const of_param* W, const of_param* b, const float* gW_partial,
                              const float* gb_partial, const of_opt* opt, void* ws,
                              size_t ws_bytes, void* stream) {
  of_status st = check_conv(d);
  if (st != OF_OK) return st;
  if ((st = check_opt(opt)) != OF_OK) return st;
  REQUIRE(dy && x, OF_EINVAL, "dy and x are required");
  if ((st = check_param(W, "W", 9 * d->C * d->Cout, *opt, true)) != OF_OK) return st;
  if (b) {
    if ((st = check_param(b, "b", d->Cout, *opt, true)) != OF_OK) return st;
  }
  REQUIRE(al4(dy) && al4(x) && al4(gW_partial) && al4(gb_partial), OF_EALIGN,
          "fp32 pointers must be 4-byte aligned");
  if ((st = check_conv_ws(d, EPI_WGRAD_BF, ws, ws_bytes)) != OF_OK) return st;
  EpiArgs ea = empty_epi();
  ea.ldo = 9 * d->C;
  ea.W = *W;
  ea.gW = gW_partial;
  if (b) { ea.b = *b; ea.gb = gb_partial; }
  ea.with_db = b != nullptr;
  ea.opt = make_optk(*opt);
  return hip_status(gemm_launch(EPI_WGRAD_BF, conv_problem(d, EPI_WGRAD_BF, dy, x), ea, ws,
                                (hipStream_t)stream), "of_conv_wgrad_fused launch");
}

namespace {
of_status check_dw(const of_conv_desc* d) {
  REQUIRE(d != nullptr, OF_EINVAL, "desc is NULL");
  REQUIRE(d->N >= 1 && d->H >= 1 && d->W >= 1 && d->C >= 1, OF_EINVAL,
          "N, H, W, C must be >= 1");
  REQUIRE(d->Cout == d->C, OF_EINVAL, "a depthwise convolution needs Cout == C (got %lld, %lld)",
          (long long)d->Cout, (long long)d->C);
  REQUIRE(d->N * d->H * d->W * d->C < (1LL << 31), OF_EUNSUPPORTED,
          "activation tensors must have < 2^31 elements");
  REQUIRE(d->act == OF_ACT_NONE || d->act == OF_ACT_RELU, OF_EUNSUPPORTED,
          "depthwise convolutions support OF_ACT_NONE and OF_ACT_RELU");
  REQUIRE(d->stride >= 0 && d->stride <= 2, OF_EUNSUPPORTED,
          "depthwise convolutions run with stride 1 or 2 (got %d)", (int)d->stride);
  return OF_OK;
}

of_status check_dw_ws(const of_conv_desc* d, const void* ws, size_t ws_bytes) {
  const size_t need = dw_workspace_bytes(*d);
  REQUIRE(ws_bytes >= need, OF_EWORKSPACE, "workspace of %zu bytes is smaller than the %zu needed",
          ws_bytes, need);
  REQUIRE(ws != nullptr, OF_EWORKSPACE, "workspace is NULL");
  REQUIRE((((uintptr_t)ws) & 15u) == 0, OF_EALIGN, "workspace must be 16-byte aligned");
  return OF_OK;
}
}  // namespace

size_t of_dwconv_workspace_size(const of_conv_desc* d) {
  if (check_dw(d) != OF_OK) return 0;
  return dw_workspace_bytes(*d);
}

of_status of_dwconv_fwd(const of_conv_desc* d, const float* x, const float* W, const float* b,
                        float* y, void* stream) {
  of_status st = check_dw(d);
  if (st != OF_OK) return st;
  REQUIRE(x && W && y, OF_EINVAL, "x, W and y are required");
  REQUIRE(!d->has_bias || b, OF_EINVAL, "has_bias is set but b is NULL");
  REQUIRE(al4(x) && al4(W) && al4(b) && al4(y), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  return hip_status(launch_dw_fwd(*d, x, W, b, y, (hipStream_t)stream), "of_dwconv_fwd launch");
}

of_status of_dwconv_bwd_data(const of_conv_desc* d, const float* dy, const float* W,
                             const float* prev, int32_t act_prev, float* dx, void* stream) {
  of_status st = check_dw(d);
  if (st != OF_OK) return st;
  REQUIRE(dy && W && dx, OF_EINVAL, "dy, W and dx are required");
  REQUIRE(act_prev == OF_ACT_NONE || act_prev == OF_ACT_RELU, OF_EUNSUPPORTED,
          "act_prev must be OF_ACT_NONE or OF_ACT_RELU");
  REQUIRE(act_prev == OF_ACT_NONE || prev, OF_EINVAL, "act_prev needs prev");
  REQUIRE(al4(dy) && al4(W) && al4(prev) && al4(dx), OF_EALIGN,
          "fp32 pointers must be 4-byte aligned");
  return hip_status(launch_dw_dgrad(*d, dy, W, prev, act_prev, dx, (hipStream_t)stream),
                    "of_dwconv_bwd_data launch");
}

of_status of_dwconv_bwd_weight(const of_conv_desc* d, const float* dy, const float* x, float* dw,
                               float* db, int32_t accumulate, void* ws, size_t ws_bytes,
                               void* stream) {
  of_status st = check_dw(d);
  if (st != OF_OK) return st;
  REQUIRE(dy && x && dw, OF_EINVAL, "dy, x and dw are required");
  REQUIRE(accumulate == 0 || accumulate == 1, OF_EINVAL, "accumulate must be 0 or 1");
  REQUIRE(al4(dy) && al4(x) && al4(dw) && al4(db), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  if ((st = check_dw_ws(d, ws, ws_bytes)) != OF_OK) return st;
  return hip_status(launch_dw_wgrad(*d, dy, x, dw, db, accumulate, nullptr, nullptr, nullptr,
                                    nullptr, nullptr, ws, (hipStream_t)stream),
                    "of_dwconv_bwd_weight launch");
}

of_status of_dwconv_wgrad_fused(const of_conv_desc* d, const float* dy, const float* x,
                                const of_param* W, const of_param* b, const float* gW_partial,
                                const float* gb_partial, const of_opt* opt, void* ws,
                                size_t ws_bytes, void* stream) {
  of_status st = check_dw(d);
  if (st != OF_OK) return st;
  if ((st = check_opt(opt)) != OF_OK) return st;
  REQUIRE(dy && x, OF_EINVAL, "dy and x are required");
  if ((st = check_param(W, "W", 9 * d->C, *opt, true)) != OF_OK) return st;
  if (b) {
    if ((st = check_param(b, "b", d->C, *opt, true)) != OF_OK) return st;
  }
  REQUIRE(al4(dy) && al4(x) && al4(gW_partial) && al4(gb_partial), OF_EALIGN,
          "fp32 pointers must be 4-byte aligned");
  if ((st = check_dw_ws(d, ws, ws_bytes)) != OF_OK) return st;
  const OptK o = make_optk(*opt);
  return hip_status(launch_dw_wgrad(*d, dy, x, nullptr, nullptr, 0, W, b, gW_partial,
                                    b ? gb_partial : nullptr, &o, ws, (hipStream_t)stream),
                    "of_dwconv_wgrad_fused launch");
}

of_status of_maxpool2x2_fwd(const float* x, int64_t N, int64_t H, int64_t W, int64_t C, float* y,
                            uint8_t* argmax, void* stream) {
  REQUIRE(x && y && argmax, OF_EINVAL, "x, y and argmax are required");
  REQUIRE(N >= 1 && H >= 2 && W >= 2 && C >= 1 && H % 2 == 0 && W % 2 == 0, OF_EINVAL,
          "N, C >= 1 and H, W even and >= 2 are required");
  REQUIRE(al4(x) && al4(y), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  return hip_status(launch_maxpool_fwd(x, N, H, W, C, y, argmax, (hipStream_t)stream),
                    "of_maxpool2x2_fwd launch");
}

of_status of_maxpool2x2_bwd(const float* dy, const uint8_t* argmax, const float* mask_src,
                            int64_t N, int64_t H, int64_t W, int64_t C, float* dx, void* stream) {
  REQUIRE(dy && argmax && dx, OF_EINVAL, "dy, argmax and dx are required");
  REQUIRE(N >= 1 && H >= 2 && W >= 2 && C >= 1 && H % 2 == 0 && W % 2 == 0, OF_EINVAL,
          "N, C >= 1 and H, W even and >= 2 are required");
  REQUIRE(al4(dy) && al4(dx) && al4(mask_src), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  return hip_status(launch_maxpool_bwd(dy, argmax, mask_src, N, H, W, C, dx, (hipStream_t)stream),
                    "of_maxpool2x2_bwd launch");
}

of_status of_avgpool_fwd(const float* x, int64_t N, int64_t P, int64_t C, float* y, void* stream) {
  REQUIRE(x && y, OF_EINVAL, "x and y are required");
  REQUIRE(N >= 1 && P >= 1 && C >= 1, OF_EINVAL, "N, P and C must be >= 1");
  REQUIRE(N <= (1LL << 40) / P / C, OF_EUNSUPPORTED, "N * P * C must be < 2^40");
  REQUIRE(al4(x) && al4(y), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  return hip_status(launch_avgpool_fwd(x, N, P, C, y, (hipStream_t)stream), "of_avgpool_fwd launch");
}

of_status of_avgpool_bwd(const float* dy, const float* mask_src, int64_t N, int64_t P, int64_t C,
                         float* dx, void* stream) {
  REQUIRE(dy && dx, OF_EINVAL, "dy and dx are required");
  REQUIRE(N >= 1 && P >= 1 && C >= 1, OF_EINVAL, "N, P and C must be >= 1");
  REQUIRE(N <= (1LL << 40) / P / C, OF_EUNSUPPORTED, "N * P * C must be < 2^40");
  REQUIRE(al4(dy) && al4(dx) && al4(mask_src), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  return hip_status(launch_avgpool_bwd(dy, mask_src, N, P, C, dx, (hipStream_t)stream),
                    "of_avgpool_bwd launch");
}

of_status of_elementwise_fused_update(const of_param* p, const float* g, int64_t g_rows,
                                      int64_t g_ld, const of_opt* opt, void* stream) {
  of_status st = check_opt(opt);
  if (st != OF_OK) return st;
  REQUIRE(p != nullptr && p->numel >= 1, OF_EINVAL, "p is NULL or p->numel < 1");
  if ((st = check_param(p, "p", p->numel, *opt, true)) != OF_OK) return st;
  REQUIRE(g != nullptr, OF_EINVAL, "g is NULL");
  REQUIRE(al4(g), OF_EALIGN, "g must be 4-byte aligned");
  REQUIRE(g_rows >= 1, OF_EINVAL, "g_rows must be >= 1");
  REQUIRE(g_ld == 0 || g_ld >= p->numel, OF_EINVAL, "g_ld must be 0 or >= numel");
  const OptK ok = make_optk(*opt);
  const hipStream_t s = (hipStream_t)stream;
  if (g_rows == 1) {
    const float* gs[1] = {g};
    return hip_status(launch_multi_update(1, p, gs, ok, s), "of_elementwise_fused_update launch");
  }
  return hip_status(launch_rows_update(*p, g, g_rows, g_ld ? g_ld : p->numel, ok, s),
                    "of_elementwise_fused_update launch");
}

of_status of_optimizer_step(int32_t n, const of_param* params, const float* const* grads,
                            const of_opt* opt, void* stream) {
  of_status st = check_opt(opt);
  if (st != OF_OK) return st;
  REQUIRE(n >= 1 && params && grads, OF_EINVAL, "n >= 1, params and grads are required");
  for (int32_t i = 0; i < n; ++i) {
    char name[32];
    snprintf(name, sizeof(name), "params[%d]", (int)i);
    REQUIRE(params[i].numel >= 1, OF_EINVAL, "%s.numel < 1", name);
    if ((st = check_param(&params[i], name, params[i].numel, *opt, true)) != OF_OK) return st;
    REQUIRE(grads[i] != nullptr, OF_EINVAL, "grads[%d] is NULL", (int)i);
    REQUIRE(al4(grads[i]), OF_EALIGN, "grads[%d] must be 4-byte aligned", (int)i);
  }
  return hip_status(launch_multi_update(n, params, grads, make_optk(*opt), (hipStream_t)stream),
                    "of_optimizer_step launch");
}

of_status of_grad_clip_scale(int32_t n, const of_grad_ref* grads, float max_norm, float* scale,
                             float* norm, void* ws, size_t ws_bytes, void* stream) {
  REQUIRE(n >= 1 && grads != nullptr, OF_EINVAL, "n >= 1 and grads are required");
  REQUIRE(std::isfinite(max_norm) && max_norm > 0.f, OF_EINVAL,
          "max_norm must be finite and > 0 (got %g)", (double)max_norm);
  REQUIRE(scale != nullptr, OF_EINVAL, "scale is NULL");
  REQUIRE(al4(scale) && (norm == nullptr || al4(norm)), OF_EALIGN,
          "scale / norm must be 4-byte aligned");
  REQUIRE(ws != nullptr && ws_bytes >= OF_CLIP_WS_BYTES, OF_EWORKSPACE,
          "workspace of %d bytes required (got %zu)", (int)OF_CLIP_WS_BYTES, ws_bytes);
  REQUIRE((((uintptr_t)ws) & 7u) == 0, OF_EALIGN, "ws must be 8-byte aligned");
  for (int32_t i = 0; i < n; ++i) {
    const of_grad_ref& g = grads[i];
    REQUIRE(g.g != nullptr, OF_EINVAL, "grads[%d].g is NULL", (int)i);
    REQUIRE(al4(g.g), OF_EALIGN, "grads[%d].g must be 4-byte aligned", (int)i);
    REQUIRE(g.numel >= 1 && g.rows >= 1, OF_EINVAL, "grads[%d]: numel and rows must be >= 1",
            (int)i);
    REQUIRE(g.ld == 0 || g.ld >= g.numel, OF_EINVAL, "grads[%d].ld must be 0 or >= numel",
            (int)i);
  }
  return hip_status(launch_grad_clip(n, grads, max_norm, scale, norm, (double*)ws,
                                     (hipStream_t)stream),
                    "of_grad_clip_scale launch");
}

of_status of_step_advance(int64_t* step_dev, int64_t delta, void* stream) {
  REQUIRE(step_dev != nullptr, OF_EINVAL, "step_dev is NULL");
  REQUIRE((((uintptr_t)step_dev) & 7u) == 0, OF_EALIGN, "step_dev must be 8-byte aligned");
  return hip_status(launch_step_advance(step_dev, delta, (hipStream_t)stream),
                    "of_step_advance launch");
}

of_status of_xent_fwd_bwd(const float* logits, const int64_t* labels, int64_t B, int64_t C,
                          int64_t ld, float* loss, float* dlogits, void* stream) {
  REQUIRE(logits && labels && loss && dlogits, OF_EINVAL, "logits, labels, loss, dlogits are required");
  REQUIRE(B >= 1 && C >= 1, OF_EINVAL, "B and C must be >= 1");
  REQUIRE(ld == 0 || ld >= C, OF_EINVAL, "ld must be 0 or >= C");
  REQUIRE(al4(logits) && al4(loss) && al4(dlogits) && (((uintptr_t)labels) & 7u) == 0, OF_EALIGN,
          "misaligned pointer");
  return hip_status(launch_xent(logits, labels, B, C, ld ? ld : C, loss, dlogits, (hipStream_t)stream),
                    "of_xent_fwd_bwd launch");
}

of_status of_layernorm_fwd(const float* x, int64_t M, int64_t D, const float* gamma,
                           const float* beta, float eps, float* y, float* mean, float* rstd,
                           void* stream) {
  REQUIRE(x && gamma && beta && y && mean && rstd, OF_EINVAL,
          "x, gamma, beta, y, mean and rstd are required");
  REQUIRE(M >= 1 && D >= 1, OF_EINVAL, "M and D must be >= 1");
  REQUIRE(std::isfinite(eps) && eps > 0.f, OF_EINVAL, "eps must be finite and > 0");
  REQUIRE(al4(x) && al4(gamma) && al4(beta) && al4(y) && al4(mean) && al4(rstd), OF_EALIGN,
          "fp32 pointers must be 4-byte aligned");
  return hip_status(launch_ln_fwd(x, M, D, gamma, beta, eps, y, nullptr, mean, rstd,
                                  (hipStream_t)stream),
                    "of_layernorm_fwd launch");
}

of_status of_layernorm_fwd_bf16(const float* x, int64_t M, int64_t D, const float* gamma,
                                const float* beta, float eps, uint16_t* y, float* mean,
                                float* rstd, void* stream) {
  REQUIRE(x && gamma && beta && y && mean && rstd, OF_EINVAL,
          "x, gamma, beta, y, mean and rstd are required");
  REQUIRE(M >= 1 && D >= 1, OF_EINVAL, "M and D must be >= 1");
  REQUIRE(std::isfinite(eps) && eps > 0.f, OF_EINVAL, "eps must be finite and > 0");
  REQUIRE(al4(x) && al4(gamma) && al4(beta) && al4(mean) && al4(rstd), OF_EALIGN,
          "fp32 pointers must be 4-byte aligned");
  REQUIRE((((uintptr_t)y) & 1u) == 0, OF_EALIGN, "y (bf16) must be 2-byte aligned");
  return hip_status(launch_ln_fwd(x, M, D, gamma, beta, eps, nullptr, y, mean, rstd,
                                  (hipStream_t)stream),
                    "of_layernorm_fwd_bf16 launch");
}

int64_t of_layernorm_partial_rows(int64_t M) { return M >= 1 ? ln_partial_rows(M) : 0; }

of_status of_layernorm_bwd(const float* dy, const float* x, const float* mean, const float* rstd,
                           const float* gamma, const float* dres, int64_t M, int64_t D, float* dx,
                           float* dgamma_rows, float* dbeta_rows, void* stream) {
  REQUIRE(dy && x && mean && rstd, OF_EINVAL, "dy, x, mean and rstd are required");
  REQUIRE(!dgamma_rows == !dbeta_rows, OF_EINVAL,
          "dgamma_rows and dbeta_rows are given together or both NULL");
  REQUIRE(dx || dgamma_rows, OF_EINVAL, "nothing to compute: dx and the partials are all NULL");
  REQUIRE(!dx || gamma, OF_EINVAL, "gamma is required for dx");
  REQUIRE(M >= 1 && D >= 1, OF_EINVAL, "M and D must be >= 1");
  REQUIRE(!dx || (dx != dy && dx != x), OF_EINVAL,
          "dx must not alias dy or x (both are read again)");
  REQUIRE(al4(dy) && al4(x) && al4(mean) && al4(rstd) && al4(gamma) && al4(dres) && al4(dx) &&
              al4(dgamma_rows) && al4(dbeta_rows),
          OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  return hip_status(launch_ln_bwd(dy, x, mean, rstd, gamma, dres, M, D, dx, dgamma_rows,
                                  dbeta_rows, (hipStream_t)stream),
                    "of_layernorm_bwd launch");
}

of_status of_reduce_rows(const float* src, int64_t rows, int64_t ld, int64_t n, float* dst,
                         void* stream) {
  REQUIRE(src && dst, OF_EINVAL, "src and dst are required");
  REQUIRE(rows >= 1 && n >= 1, OF_EINVAL, "rows and n must be >= 1");
  if (ld == 0) ld = n;
  REQUIRE(ld >= n, OF_EINVAL, "ld must be 0 or >= n");
  REQUIRE(al4(src) && al4(dst), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  return hip_status(launch_reduce_rows(src, rows, ld, n, dst, (hipStream_t)stream),
                    "of_reduce_rows launch");
}

of_status of_add(const float* a, const float* b, int64_t n, float* out, void* stream) {
  REQUIRE(a && b && out, OF_EINVAL, "a, b and out are required");
  REQUIRE(n >= 1, OF_EINVAL, "n must be >= 1");
  REQUIRE(al4(a) && al4(b) && al4(out), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  return hip_status(launch_add(a, b, n, out, (hipStream_t)stream), "of_add launch");
}

size_t of_mse_workspace_size(int64_t M, int64_t D) { return mse_ws_bytes(M, D); }

of_status of_mse_fwd_bwd(const float* y, const float* t, int64_t M, int64_t D, int64_t ld,
                         float* loss, float* dy, void* ws, size_t ws_bytes, void* stream) {
  REQUIRE(y && t && loss && dy, OF_EINVAL, "y, t, loss and dy are required");
  REQUIRE(M >= 1 && D >= 1, OF_EINVAL, "M and D must be >= 1");
  REQUIRE(ld == 0 || ld >= D, OF_EINVAL, "ld must be 0 or >= D");
  REQUIRE(al4(y) && al4(t) && al4(loss) && al4(dy), OF_EALIGN, "fp32 pointers must be 4-byte aligned");
  const size_t need = mse_ws_bytes(M, D);
  REQUIRE(ws_bytes >= need && ws != nullptr, OF_EWORKSPACE, "workspace of %zu bytes is smaller than %zu",
          ws_bytes, need);
  REQUIRE((((uintptr_t)ws) & 7u) == 0, OF_EALIGN, "workspace must be 8-byte aligned");
  return hip_status(launch_mse(y, t, M, D, ld ? ld : D, loss, dy, ws, (hipStream_t)stream),
                    "of_mse_fwd_bwd launch");
}

}  // extern "C"
