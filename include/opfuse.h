/*
 * opfuse.h -- optimizer fusion on AMD Instinct MI355X (gfx950), C ABI.
 *
 * Implements the hot path of "Optimizer Fusion: Efficient Training with Better
 * Locality and Parallelism" (Jiang et al., arXiv 2104.00237):
 *
 *   - backward-fusion (Section 3 "Backward-Fusion", Appendix B.2, Alg. 3): the
 *     weight-gradient contraction dW = dZ^T X applies the optimizer to W and
 *     its history in its epilogue; dW is never written to memory;
 *   - forward-fusion (Section 3 "Forward-Fusion", Appendix B.1, Alg. 2): the
 *     pending update is applied while the next forward contraction loads its
 *     W tiles; the updated tile is written back and fed to the matrix cores;
 *   - the eager three-stage path (Section 1, Fig. 1(b)): forward, backward
 *     writing every gradient, then one multi-tensor optimizer launch.
 *
 * Conventions for every entry point:
 *   - Pointers named x, y, w, ... are DEVICE pointers owned by the caller.
 *     The library never allocates, frees or retains them after returning.
 *   - Work is enqueued asynchronously on `stream` (a hipStream_t passed as
 *     void*; NULL is the null stream).  Device faults surface at the caller's
 *     next synchronisation.
 *   - Arguments are validated synchronously before any HIP call; on failure
 *     nothing is enqueued and a status other than OF_OK is returned, with a
 *     message in of_last_error() (thread-local).
 *   - Layouts are row-major.  A linear layer has X [M,K] (row stride ldx),
 *     W [N,K], bias [N], Z/Y [M,N] (row stride ldy).  A convolution has NHWC
 *     activations and [Cout,3,3,Cin] filters.
 *   - Any size is accepted (ragged tails are masked); 128-bit memory paths are
 *     used when a pointer is 16-byte aligned and its row stride is a multiple
 *     of 4 elements.  fp32 pointers must be 4-byte aligned (else OF_EALIGN).
 *   - Entry points that take a workspace need at least the bytes the matching
 *     *_workspace_size query returns (else OF_EWORKSPACE).  The workspace holds
 *     split-reduction partials only; it needs no initialisation and may be
 *     reused by later calls on the same stream.
 *   - Calls that touch the same parameter on different streams race unless the
 *     caller orders them (except inside of_linear_bwd_fused, see there).
 */
#ifndef OPFUSE_H
#define OPFUSE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OF_VERSION 1

typedef enum of_status {
  OF_OK = 0,
  OF_EINVAL = 1,        /* null required pointer, non-positive size, bad enum, step < 1 */
  OF_EUNSUPPORTED = 2,  /* valid but unsupported combination (dtype / activation / shape) */
  OF_EALIGN = 3,        /* pointer not aligned to its element size */
  OF_EWORKSPACE = 4,    /* workspace smaller than the query returns */
  OF_EHIP = 5           /* a HIP launch failed; of_last_error() has the HIP error text */
} of_status;

typedef enum of_dtype { OF_F32 = 0, OF_BF16 = 1 } of_dtype;

/* Activation applied to Z in a forward epilogue; its derivative is applied
 * in the dgrad epilogue of the NEXT layer (see of_linear_bwd_data). */
typedef enum of_act { OF_ACT_NONE = 0, OF_ACT_RELU = 1, OF_ACT_GELU = 2 } of_act;

/*
 * Optimizer policy pi (Appendix A, Alg. 1).  `step` is the 1-based index t of
 * the update being applied; the caller owns and increments it.  Bias
 * corrections 1 - beta^t are computed in float64 (beta^t by binary
 * exponentiation): by the library at the call when `step` is given by value,
 * by each updating kernel from *step_dev otherwise -- the same arithmetic, so
 * both give identical results.
 *
 *   OF_OPT_SGD    momentum (Appendix A, Eq. for pi_2) with coupled weight decay:
 *                   g' = g + wd*w;  m = momentum*m + g';  w -= lr*m
 *                 (m starts at 0, dampening 0, no Nesterov; momentum 0 is pi_1)
 *   OF_OPT_ADAM   Adam with coupled L2 weight decay g' = g + wd*w:
 *                   m = b1 m + (1-b1) g';  v = b2 v + (1-b2) g'^2
 *                   w -= (lr/(1-b1^t)) * m / (sqrt(v)/sqrt(1-b2^t) + eps)
 *   OF_OPT_ADAMW  w *= (1 - lr*wd), then the Adam step on the raw g.
 *   The other optimizers of the paper's comparison (Section 4, "Various Models
 *   and Optimizers", Fig. 7), with coupled weight decay g' = g + wd*w:
 *   OF_OPT_ADAGRAD   v += g'^2;  w -= lr * g' / (sqrt(v) + eps)
 *                    (v starts at 0; m is not used but must be given)
 *   OF_OPT_RMSPROP   v = beta2 v + (1-beta2) g'^2;  s = g' / (sqrt(v) + eps)
 *                    momentum == 0: w -= lr * s;  else m = momentum m + s, w -= lr * m
 *                    (beta2 is the smoothing constant alpha)
 *   OF_OPT_ADADELTA  v = beta2 v + (1-beta2) g'^2
 *                    d = sqrt((m + eps) / (v + eps)) * g'
 *                    m = beta2 m + (1-beta2) d^2;  w -= lr * d
 *                    (beta2 is the decay rate rho; m accumulates squared updates)
 *   All of them keep v (and m), so every entry point takes them as for Adam.
 *
 * Every kernel that updates a parameter uses one shared per-element update
 * with explicitly rounded operations, so all orderings compute bit-identical
 * values from identical gradients.
 */
typedef enum of_opt_kind {
  OF_OPT_SGD = 0, OF_OPT_ADAM = 1, OF_OPT_ADAMW = 2,
  OF_OPT_ADAGRAD = 3, OF_OPT_RMSPROP = 4, OF_OPT_ADADELTA = 5
} of_opt_kind;

typedef struct of_opt {
  int32_t kind;
  float lr;
  float weight_decay;
  float momentum;   /* SGD, RMSprop */
  float beta1;      /* Adam / AdamW */
  float beta2;      /* Adam / AdamW; RMSprop alpha; Adadelta rho */
  float eps;
  int64_t step;     /* >= 1; ignored when step_dev is not NULL */
  /* Optional device address of the step, read by the kernels when they run
   * (for launches captured once and replayed, e.g. in a HIP graph; see
   * of_step_advance).  The value there must be >= 1 when they run. */
  const int64_t* step_dev;
  /* Optional device address of a gradient scale, read by the kernels when they
   * run: every gradient element is multiplied by it (rounded to fp32) before
   * the update uses it.  NULL means 1, which leaves every result bit-identical
   * to an unscaled update.  of_grad_clip_scale writes the factor for
   * global-norm clipping; only orderings that update after the whole backward
   * pass (eager, forward-fusion) can use that factor (Table 1). */
  const float* grad_scale;
} of_opt;

/*
 * A trainable tensor theta with its history (Fig. 2, "History").
 *   w       fp32 master values [numel]
 *   m       SGD momentum buffer, Adam first moment, RMSprop momentum buffer or
 *           Adadelta squared-update average [numel]; required, except for Adagrad
 *           and RMSprop with momentum 0, which keep no m: there it may be NULL
 *           and is then neither read nor written
 *   v       Adam second moment, or the squared-gradient state of Adagrad,
 *           RMSprop and Adadelta [numel] (required unless SGD, ignored for SGD)
 *   w_bf16  optional bf16 copy of w (round to nearest even), rewritten by every
 *           update when not NULL; it is the matmul operand when dtype is OF_BF16
 */
typedef struct of_param {
  float* w;
  float* m;
  float* v;
  uint16_t* w_bf16;
  int64_t numel;
} of_param;

/*
 * Pending updates carried by a forward launch (forward-fusion of later
 * operators, Appendix B.1, Alg. 2): n tensors (1 <= n <= OF_CARRY_MAX), each
 * with its pending gradient g[i], updated with `opt` by extra workgroups of
 * the forward's kernel.  A gradient is one vector of numel elements
 * (rows[i] == 1) or rows[i] row partials [rows, numel] summed in row order (a
 * LayerNorm parameter's gradient).  Every element gets exactly the
 * operations of of_optimizer_step (vector) or of_elementwise_fused_update
 * (rows), so results are bit-identical to those passes.  The carried tensors
 * must not overlap each other or anything the forward reads or writes.
 */
#define OF_CARRY_MAX 4
typedef struct of_carry {
  int32_t n;
  of_param t[OF_CARRY_MAX];
  const float* g[OF_CARRY_MAX];
  int64_t rows[OF_CARRY_MAX];
  of_opt opt;
} of_carry;

/*
 * Storage of a bf16-operand layer's activations (of_linear_desc.io, bit flags;
 * dtype OF_BF16 only, 0 otherwise).  A tensor that only bf16-operand
 * contractions read can be kept as its bf16 rounding (uint16 bit patterns,
 * round to nearest even): the value the contraction would round the fp32
 * tensor to, so results are bit-identical, with half the bytes moved.
 *   OF_IO_X_BF16  X [M, ldx] is stored as bf16: the forward's and the weight
 *                 gradient's `x` point to it (pass it cast to the pointer
 *                 type; 2-byte aligned).  The forward then needs W->w_bf16.
 *   OF_IO_Y_BF16  the forward stores Y = act(Z) as bf16 [M, ldy] into `y`
 *                 (cast; 2-byte aligned); Z, when requested, stays fp32.
 */
enum { OF_IO_X_BF16 = 1, OF_IO_Y_BF16 = 2 };

typedef struct of_linear_desc {
  int64_t M, N, K;   /* rows, output features, input features (all >= 1) */
  int64_t ldx;       /* row stride of X in elements; 0 means K */
  int64_t ldy;       /* row stride of Y, Z, dZ in elements; 0 means N */
  int32_t dtype;     /* matmul operand type: OF_F32, or OF_BF16 (operands rounded to bf16, fp32 accumulate) */
  int32_t act;       /* of_act applied in the forward epilogue */
  int32_t has_bias;  /* 1: bias [N] added in the forward */
  int32_t io;        /* OF_IO_* flags (bf16 storage of X and Y); 0: fp32 */
} of_linear_desc;

typedef struct of_conv_desc {
  int64_t N, H, W, C;  /* input batch, height, width, channels (NHWC) */
  int64_t Cout;        /* output channels; filter is [Cout,3,3,C], zero pad 1 */
  int32_t act;         /* of_act applied in the forward epilogue (NONE or RELU) */
  int32_t has_bias;
  int32_t stride;      /* 0 or 1: stride 1; 2: stride 2 (depthwise only), output
                          [N, (H-1)/2+1, (W-1)/2+1, C] */
} of_conv_desc;

/* Which call a workspace query is for. */
typedef enum of_linear_op {
  OF_LINEAR_FWD = 0,        /* of_linear_fwd, of_linear_fwd_fused */
  OF_LINEAR_BWD_DATA = 1,   /* of_linear_bwd_data, the dgrad half of of_linear_bwd_fused */
  OF_LINEAR_BWD_WEIGHT = 2, /* of_linear_bwd_weight, the wgrad half of of_linear_bwd_fused */
  OF_LINEAR_BWD_MERGED = 3  /* of_linear_bwd_merged (0 when the descriptor is unsupported there) */
} of_linear_op;

typedef enum of_conv_op {
  OF_CONV_FWD = 0, OF_CONV_BWD_DATA = 1, OF_CONV_BWD_WEIGHT = 2
} of_conv_op;

/* ---------------------------------------------------------------- basics */

/* OF_VERSION of the built library. */
int of_version(void);

/* Message for the last non-OF_OK status returned on this thread ("" if none). */
const char* of_last_error(void);

/* Bytes of workspace `op` needs for `d` (0 if none); 0 and OF_EINVAL in
 * of_last_error() for an invalid descriptor. */
size_t of_linear_workspace_size(const of_linear_desc* d, int32_t op);

/* ------------------------------------------------------- linear layers */

/*
 * Plain forward (Fig. 1(a), the forward node of a linear layer):
 *   Z = X W^T + b,  Y = act(Z).
 * x: [M, ldx] fp32 (OF_F32) or fp32 rounded to bf16 on load (OF_BF16), or
 * bf16 as stored (OF_IO_X_BF16).
 * W: W->w is read for OF_F32, W->w_bf16 for OF_BF16.  b: [N] or NULL when
 * !has_bias.  z: [M, ldy] fp32, optional (needed by GELU's derivative);
 * y: [M, ldy] fp32 (bf16 with OF_IO_Y_BF16), required.  Workspace:
 * OF_LINEAR_FWD.
 */
of_status of_linear_fwd(const of_linear_desc* d, const float* x, const of_param* W,
                        const float* b, float* z, float* y, void* ws, size_t ws_bytes,
                        void* stream);

/*
 * Forward-fusion forward (Section 3 "Forward-Fusion"; Appendix B.1, Alg. 2;
 * the purple frame of Fig. 2): the optimizer of W (and b) runs on the pending
 * gradients gW [N,K] (gb [N]) with `opt` while the W tiles are loaded for the
 * contraction, and Y = act(X W'^T + b') is computed from the updated values
 * W', b'.  Each element's update is written exactly once:
 *   W_out == NULL: in place into W (and b).  Needs the M rows in one row tile
 *     of the contraction (M <= 64), so each W element has one reader;
 *     otherwise OF_EUNSUPPORTED.
 *   W_out != NULL: into the second buffer set W_out (and b_out; both sets of
 *     the same sizes and optimizer, no buffer shared).  Any M: every row tile
 *     computes the update of its W tile in registers from W (the set is only
 *     read), and the first row tile stores it to W_out, which the caller makes
 *     the current set afterwards (the two sets alternate step by step).
 * fp32 operands only (dtype OF_F32; OF_EUNSUPPORTED otherwise: with bf16
 * operands every row tile would read the fp32 weight, gradient and history,
 * 16 B per element, where the contraction reads the 2-byte shadow).
 * opt == NULL means nothing is pending (the first iteration): identical to
 * of_linear_fwd, and W_out, b_out are ignored.  b/gb (and b_out): NULL when
 * !has_bias.  Workspace: OF_LINEAR_FWD.
 */
of_status of_linear_fwd_fused(const of_linear_desc* d, const float* x, const of_param* W,
                              const of_param* W_out, const float* gW, const of_param* b,
                              const of_param* b_out, const float* gb, const of_opt* opt,
                              float* z, float* y, void* ws, size_t ws_bytes, void* stream);

/*
 * of_linear_fwd whose launch also applies a later operator's pending update
 * (forward-fusion): `next` is applied by extra workgroups of the same kernel,
 * overlapping the contraction, so the later operator's forward finds its
 * parameters updated without a launch of its own.  next == NULL: identical to
 * of_linear_fwd.  Y is bit-identical to of_linear_fwd's, and the carried
 * tensors to a separate update pass.
 */
of_status of_linear_fwd_carry(const of_linear_desc* d, const float* x, const of_param* W,
                              const float* b, float* z, float* y, const of_carry* next,
                              void* ws, size_t ws_bytes, void* stream);

/*
 * of_linear_fwd_carry with a residual connection added in the epilogue:
 *   Y = act(X W^T + b) + R
 * (a pre-LN transformer block's h = x + proj(v) and y = h + fc2(g); an
 * inverted-residual block's input added to its projection).  The sum is
 * rounded once, so Y equals of_linear_fwd followed by of_add, bit for bit,
 * without storing and re-reading the branch output.  res: [M, ldy] fp32,
 * required, 4-byte aligned; it may be y itself (fp32 Y, in place) and must
 * not overlap y otherwise, nor z.  next may be NULL.
 */
of_status of_linear_fwd_res(const of_linear_desc* d, const float* x, const of_param* W,
                            const float* b, const float* res, float* z, float* y,
                            const of_carry* next, void* ws, size_t ws_bytes, void* stream);

/*
 * Data gradient with the OLD weights (the dependency rule after Alg. 3):
 *   dX = (dZ W) * act_prev'(prev)
 * dz: [M, ldy].  prev: the previous layer's saved tensor, [M, ldx]: its Y for
 * OF_ACT_RELU (the mask is Y > 0, equal to Z > 0), its Z for OF_ACT_GELU,
 * NULL for OF_ACT_NONE.  dx: [M, ldx] fp32.  Workspace: OF_LINEAR_BWD_DATA.
 */
of_status of_linear_bwd_data(const of_linear_desc* d, const float* dz, const of_param* W,
                             const float* prev, int32_t act_prev, float* dx, void* ws,
                             size_t ws_bytes, void* stream);

/*
 * of_linear_bwd_data with the gradient of a skip connection added in the
 * epilogue: dX = (dZ W_old) * act_prev'(prev) + R (R is not multiplied by the
 * activation's derivative: the skip connection bypasses it), e.g. the input
 * gradient of an inverted-residual block, whose input also feeds the block's
 * output.  Rounded once, so equal bit for bit to of_linear_bwd_data followed
 * by of_add.  res: [M, ldx] fp32, required, 4-byte aligned; it may be dx
 * itself and must not overlap it otherwise.  Backward-fusion pairs it with
 * of_linear_bwd_fused with dx_prev == NULL (the update only).
 */
of_status of_linear_bwd_data_res(const of_linear_desc* d, const float* dz, const of_param* W,
                                 const float* prev, int32_t act_prev, const float* res,
                                 float* dx, void* ws, size_t ws_bytes, void* stream);

/*
 * Eager weight gradient (Fig. 1(b); the gradient is materialised and later
 * read and reset by the optimizer, Section 3 "Baseline"):
 *   dW = dZ^T X [N,K],  db = sum over rows of dZ [N] (db may be NULL).
 * accumulate = 1 adds into dw/db (a parameter used more than once).  x: the
 * forward's X [M, ldx], fp32, or bf16 as stored with OF_IO_X_BF16.
 * Workspace: OF_LINEAR_BWD_WEIGHT.
 */
of_status of_linear_bwd_weight(const of_linear_desc* d, const float* dz, const float* x,
                               float* dw, float* db, int32_t accumulate, void* ws,
                               size_t ws_bytes, void* stream);

/*
 * Backward-fusion for one linear layer (Section 3 "Backward-Fusion";
 * Appendix B.2, Alg. 3 and the dependency rule after it):
 *   1. if dx_prev != NULL: dX = (dZ W_old) * act_prev'(prev) on `stream`
 *      (exactly of_linear_bwd_data);
 *   2. the weight-gradient contraction dZ^T X, whose epilogue adds gW_partial
 *      (gradient of earlier uses of a shared W, or NULL), applies `opt` to W
 *      and its history and writes W, m, v (and w_bf16); dW is never stored.
 *      With b != NULL the bias gradient sum(dZ) (+ gb_partial) updates b the
 *      same way inside the same kernel.
 * Step 2 runs after step 1 in stream order, so step 1 always reads the old W.
 * If update_stream != NULL, step 2 is enqueued on update_stream after an
 * event recorded on `stream` behind step 1, and `stream` continues at once
 * (the overlap of updating with back-propagation, Section 3); the caller must
 * then order later reads of W and b after update_stream.  The two halves use
 * workspaces ws (OF_LINEAR_BWD_DATA) and ws_update (OF_LINEAR_BWD_WEIGHT),
 * which must not overlap when update_stream != NULL.  x as in
 * of_linear_bwd_weight (bf16 with OF_IO_X_BF16).
 */
of_status of_linear_bwd_fused(const of_linear_desc* d, const float* dz, const float* x,
                              const of_param* W, const of_param* b, const float* gW_partial,
                              const float* gb_partial, const of_opt* opt, const float* prev,
                              int32_t act_prev, float* dx_prev, void* ws, size_t ws_bytes,
                              void* ws_update, size_t ws_update_bytes, void* stream,
                              void* update_stream);

/*
 * Backward-fusion with the data gradient merged into the update's read of W
 * (Section 3 "Backward-Fusion": the parameter reads of the input-gradient
 * computation and of the optimizer are merged into one).  Computes what
 * of_linear_bwd_fused computes, in one pass over W, m, v:
 *   dX = (dZ W_old) * act_prev'(prev)   (if dx_prev != NULL)
 *   W, m, v <- update(W, dZ^T X (+ gW_partial), m, v)
 *   b, m, v <- update(b, sum over rows of dZ (+ gb_partial), ...)  (if b != NULL)
 * Each W element is read once, used by the data gradient (old value, so the
 * dependency rule after Alg. 3 holds within the kernel) and by the update, and
 * written once; dW is never stored.  The data gradient is summed over row
 * ranges of W in a fixed order, so results are deterministic, but they are
 * rounded differently from of_linear_bwd_fused's (not bit-identical to it).
 * Supported: dtype OF_F32, M <= 64 (the parameter-bound case), K, ldx and ldy
 * <= 2^22; otherwise OF_EUNSUPPORTED.
 * Arguments as in of_linear_bwd_fused; prev and dx_prev have row stride ldx.
 * ws: at least of_linear_workspace_size(d, OF_LINEAR_BWD_MERGED) bytes when
 * dx_prev != NULL (the data-gradient partials), else may be NULL.  Everything
 * is enqueued on `stream`.
 */
of_status of_linear_bwd_merged(const of_linear_desc* d, const float* dz, const float* x,
                               const of_param* W, const of_param* b, const float* gW_partial,
                               const float* gb_partial, const of_opt* opt, const float* prev,
                               int32_t act_prev, float* dx_prev, void* ws, size_t ws_bytes,
                               void* stream);

/*
 * of_linear_bwd_merged without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Arguments, results and errors as in
 * of_linear_bwd_merged; the data-gradient partials go to a buffer the library
 * holds in device memory: OF_MERGED_STATIC_SCRATCH_BYTES per device, kept
 * until the process ends.  A shape whose partials need more
 * (of_linear_workspace_size(d, OF_LINEAR_BWD_MERGED) above that; e.g. more
 * than 65536 columns at 64 rows) returns OF_EUNSUPPORTED before any launch.
 * No call allocates or frees memory.  Every call on one device shares the
 * buffer: calls that overlap on a device (different streams or threads
 * without ordering between them) race and must not be issued.  The buffer's
 * device address is looked up on the first call made on each device.
 */
#define OF_MERGED_STATIC_SCRATCH_BYTES (32u << 20)
of_status of_linear_bwd_merged_static(const of_linear_desc* d, const float* dz, const float* x,
                                      const of_param* W, const of_param* b,
                                      const float* gW_partial, const float* gb_partial,
                                      const of_opt* opt, const float* prev, int32_t act_prev,
                                      float* dx_prev, void* stream);

/* ------------------------------------------------- convolution layers */
/*
 * 3x3 convolutions (cross-correlation, stride 1, zero padding 1) as implicit
 * GEMMs: x [N,H,W,C] NHWC, filter W [Cout,3,3,C] (KRSC), bias [Cout],
 * y / dy [N,H,W,Cout].  Workspace: of_conv_workspace_size(d, op).
 */
size_t of_conv_workspace_size(const of_conv_desc* d, int32_t op);

/* Forward node of a convolution layer (Fig. 1(a)): y = act(conv(x, W) + b). */
of_status of_conv_fwd(const of_conv_desc* d, const float* x, const of_param* W, const float* b,
                      float* y, void* ws, size_t ws_bytes, void* stream);

/* of_conv_fwd carrying a later operator's pending update, as of_linear_fwd_carry. */
of_status of_conv_fwd_carry(const of_conv_desc* d, const float* x, const of_param* W,
                            const float* b, float* y, const of_carry* next, void* ws,
                            size_t ws_bytes, void* stream);

/*
 * Data gradient with the OLD filter (the dependency rule after Alg. 3):
 *   dx = conv_transpose(dy, W) * act_prev'(prev),  dx [N,H,W,C];
 * prev: the previous layer's saved output [N,H,W,C] (ReLU: mask prev > 0), or
 * NULL with OF_ACT_NONE.
 */
/*
 * Forward-fusion of a convolution in the filter-tile prologue (Section 3
 * "Forward-Fusion", Appendix B.1, Alg. 2): y = act(conv(x, W_new) + b_new),
 * where (W_new, m, v) = update(W, gW, m, v) and likewise for b.
 * A filter tile is read by every workgroup of the launch's pixel rows, so the
 * update is not written in place: every workgroup reads W, b and their history
 * (the old generation, unchanged by the call) and computes the update in
 * registers; the workgroups of the first pixel-row tile write the new values to
 * W_out and b_out (a second buffer set of the same sizes, not sharing any
 * buffer with W and b).  The caller then uses W_out / b_out as the parameters
 * (the two sets alternate from step to step).  Every element gets the
 * arithmetic of of_optimizer_step, and the contraction is the one of_conv_fwd
 * runs, so y and the new parameters are bit-identical to an update pass
 * followed by of_conv_fwd.  Workspace: of_conv_workspace_size(d, OF_CONV_FWD).
 */
of_status of_conv_fwd_fused(const of_conv_desc* d, const float* x, const of_param* W,
                            const of_param* W_out, const float* gW, const of_param* b,
                            const of_param* b_out, const float* gb, const of_opt* opt, float* y,
                            void* ws, size_t ws_bytes, void* stream);

of_status of_conv_bwd_data(const of_conv_desc* d, const float* dy, const of_param* W,
                           const float* prev, int32_t act_prev, float* dx, void* ws,
                           size_t ws_bytes, void* stream);

/* Eager filter gradient: dw [Cout,3,3,C] = sum over n,h,w of dy (x) im2col(x);
 * db [Cout] = sum of dy (db may be NULL); accumulate = 1 adds. */
of_status of_conv_bwd_weight(const of_conv_desc* d, const float* dy, const float* x, float* dw,
                             float* db, int32_t accumulate, void* ws, size_t ws_bytes,
                             void* stream);

/*
 * Backward-fusion for a convolution layer (Section 3 "Backward-Fusion";
 * Appendix B.2, Alg. 3): the implicit-GEMM filter-gradient contraction whose
 * epilogue adds gW_partial (may be NULL), applies `opt` (e.g. SGD with
 * momentum, Appendix A) to W and its history and writes them; the filter
 * gradient is never stored.  With b != NULL the bias gradient sum(dy)
 * (+ gb_partial) updates b in the same kernel.  The caller runs the data
 * gradient (of_conv_bwd_data) first: it needs the old W.
 */
of_status of_conv_wgrad_fused(const of_conv_desc* d, const float* dy, const float* x,
                              const of_param* W, const of_param* b, const float* gW_partial,
                              const float* gb_partial, const of_opt* opt, void* ws,
                              size_t ws_bytes, void* stream);

/* ------------------------------------------- depthwise 3x3 convolutions */
/*
 * The small-parameter layers where the paper sees its largest gains
 * (Appendix C, "Various Models and Optimizers", Fig. 6: speedup against
 * parameters per layer; MobileNetV2 in Fig. 3 and Table 2): one 3x3 filter
 * per channel (channel multiplier 1), zero padding 1, stride 1 or 2
 * (d->stride).  Descriptor: of_conv_desc with Cout == C.  x, dx, prev are the
 * input [N,H,W,C] NHWC; y, dy the output [N,Ho,Wo,C] with Ho = (H-1)/S + 1,
 * Wo = (W-1)/S + 1 for stride S (H, W at stride 1); so
 *   y[n,ho,wo,c] = b[c] + sum over ky, kx < 3 of
 *                  x[n, S ho + ky - 1, S wo + kx - 1, c] W[ky,kx,c]
 * (out-of-range input pixels are zero).  The filter W is [3,3,C] (tap-major, channels contiguous);
 * the bias is [C].  act is OF_ACT_NONE or OF_ACT_RELU.  All pointers are
 * device memory owned by the caller.  Errors: OF_EINVAL for NULL or
 * inconsistent arguments (Cout != C), OF_EUNSUPPORTED for tensors of 2^31
 * elements or more, OF_EALIGN for misaligned pointers, OF_EWORKSPACE for a
 * short workspace; nothing is launched then.
 */

/* Bytes of workspace the filter-gradient calls need (0 for an invalid desc). */
size_t of_dwconv_workspace_size(const of_conv_desc* d);

/* Forward node: y[n,h,w,c] = act(b[c] + sum over taps of
 * x[n,h+ky-1,w+kx-1,c] * W[ky,kx,c]). */
of_status of_dwconv_fwd(const of_conv_desc* d, const float* x, const float* W, const float* b,
                        float* y, void* stream);

/* Data gradient with the OLD filter: dx[n,h,w,c] = (sum over taps of
 * dy[n,h-ky+1,w-kx+1,c] * W[ky,kx,c]) * act_prev'(prev); act_prev is
 * OF_ACT_NONE (prev may be NULL) or OF_ACT_RELU (mask prev > 0). */
of_status of_dwconv_bwd_data(const of_conv_desc* d, const float* dy, const float* W,
                             const float* prev, int32_t act_prev, float* dx, void* stream);

/* Eager filter gradient: dw[ky,kx,c] = sum over n,h,w of dy[n,h,w,c] *
 * x[n,h+ky-1,w+kx-1,c]; db[c] = sum of dy (db may be NULL); accumulate = 1
 * adds to dw / db.  Deterministic (fixed slice order). */
of_status of_dwconv_bwd_weight(const of_conv_desc* d, const float* dy, const float* x, float* dw,
                               float* db, int32_t accumulate, void* ws, size_t ws_bytes,
                               void* stream);

/* Backward-fusion (Section 3 "Backward-Fusion", Alg. 3): the filter and bias
 * gradients of of_dwconv_bwd_weight (+ gW_partial / gb_partial when given) are
 * applied by `opt` to W, b and their history in the reduction's last pass and
 * never stored.  The result is bit-identical to of_dwconv_bwd_weight followed
 * by of_optimizer_step.  The caller runs of_dwconv_bwd_data first (old W). */
of_status of_dwconv_wgrad_fused(const of_conv_desc* d, const float* dy, const float* x,
                                const of_param* W, const of_param* b, const float* gW_partial,
                                const float* gb_partial, const of_opt* opt, void* ws,
                                size_t ws_bytes, void* stream);

/*
 * Support operators.  The paper defines none of the calls below (max-pool,
 * losses, LayerNorm, row sums, add): they complete the synthetic workloads'
 * forward and backward passes around the fused layers, and follow the usual
 * definitions stated with each.
 *
 * 2x2 max-pool, stride 2 (H, W even): y [N,H/2,W/2,C]; argmax [N,H/2,W/2,C]
 * holds the window position 0..3 of the first maximum in row-major window
 * order (ties keep the earlier position).
 */
of_status of_maxpool2x2_fwd(const float* x, int64_t N, int64_t H, int64_t W, int64_t C, float* y,
                            uint8_t* argmax, void* stream);

/*
 * Backward of the max-pool: dx [N,H,W,C] gets dy at each window's argmax and 0
 * elsewhere; with mask_src != NULL (the pool input, a ReLU output) the value
 * at the argmax is kept only where mask_src > 0 (the ReLU derivative).
 */
of_status of_maxpool2x2_bwd(const float* dy, const uint8_t* argmax, const float* mask_src,
                            int64_t N, int64_t H, int64_t W, int64_t C, float* dx, void* stream);

/*
 * Global average pool (MobileNetV2's head; a support operator): x [N, P, C]
 * (an NHWC map with P = H*W positions), y [N, C]:
 *   y[n,c] = (sum over p = 0 .. P-1, in order, of x[n,p,c]) / P.
 * Backward: dx[n,p,c] = dy[n,c] / P, set to 0 where mask_src (the pool input,
 * a ReLU output, [N, P, C]; may be NULL) is not > 0.  Errors: OF_EINVAL,
 * OF_EUNSUPPORTED (N*P*C >= 2^40), OF_EALIGN, before any launch.
 */
of_status of_avgpool_fwd(const float* x, int64_t N, int64_t P, int64_t C, float* y, void* stream);
of_status of_avgpool_bwd(const float* dy, const float* mask_src, int64_t N, int64_t P, int64_t C,
                         float* dx, void* stream);

/* ------------------------------------------------ elementwise optimizer */

/*
 * Fused elementwise update of one tensor (bias / norm parameters, and the
 * forward-fusion flush; Section 3, the optimizer reads and resets the
 * accumulated gradient):
 *   g_rows == 1: gradient g[numel];
 *   g_rows  > 1: g is [g_rows, numel] with row stride g_ld (0 means numel),
 *                and the gradient is the sum of the rows, taken in row order
 *                inside the kernel; it is never stored.
 */
of_status of_elementwise_fused_update(const of_param* p, const float* g, int64_t g_rows,
                                      int64_t g_ld, const of_opt* opt, void* stream);

/*
 * Eager optimizer stage (Fig. 1(b) stage 3; one launch for the element-wise
 * work of many tensors, in the manner of fused multi-tensor optimizers,
 * Appendix A): for i < n, params[i] is updated with grads[i] [params[i].numel].
 * params and grads are HOST arrays of n entries holding device pointers.
 */
of_status of_optimizer_step(int32_t n, const of_param* params, const float* const* grads,
                            const of_opt* opt, void* stream);

/*
 * Global-norm gradient clipping factor (the global-information step that
 * forward-fusion allows and backward-fusion does not: Appendix B.1, Table 1).
 * Over the gradients of n tensors,
 *   norm  = sqrt(sum over every element e of every tensor of g[e]^2)
 *   scale = max_norm / (norm + 1e-6), capped at 1  (NaN norm: NaN; infinite: 0)
 * and writes scale, and norm when `norm` is not NULL (one fp32 each, device
 * memory), in stream order.  Pass `scale` as of_opt.grad_scale to the updates
 * that consume these gradients.
 * A gradient is a vector [numel] (rows == 1) or row partials [rows, ld]
 * (row stride ld >= numel, 0 meaning numel) whose element is the sum of its
 * rows in row order in fp32 -- exactly the value the rows-mode update uses.
 * Squares are summed in float64, in a fixed order (deterministic); the
 * result matches the float64 definition to about 1e-15 relative.
 * grads: HOST array of n entries holding device pointers; n >= 1.
 * ws: device workspace of at least OF_CLIP_WS_BYTES bytes, 8-byte aligned.
 * max_norm must be > 0 and finite.
 */
typedef struct of_grad_ref {
  const float* g;
  int64_t numel;   /* >= 1 */
  int64_t rows;    /* >= 1 */
  int64_t ld;      /* row stride of row partials in elements; 0 means numel */
} of_grad_ref;

#define OF_CLIP_WS_BYTES 2048

of_status of_grad_clip_scale(int32_t n, const of_grad_ref* grads, float max_norm, float* scale,
                             float* norm, void* ws, size_t ws_bytes, void* stream);

/*
 * Adds `delta` to the device step counter *step_dev in stream order (one
 * thread; part of the host ordering state a captured training step replays:
 * Alg. 2 / Alg. 3 count the updates per parameter).
 */
of_status of_step_advance(int64_t* step_dev, int64_t delta, void* stream);

/* ------------------------------------------------------------- losses */

/*
 * Softmax cross-entropy, forward and backward in one launch (a support
 * operator, not defined by the paper):
 *   loss = mean_b (logsumexp(z_b) - z_{b,label_b});  dz = (softmax(z) - onehot)/B.
 * logits: [B, C] row stride ld (0 means C); labels: int64 [B] in [0, C)
 * (out-of-range labels give loss NaN); loss: one fp32 on the device; dlogits:
 * [B, ld].
 */
of_status of_xent_fwd_bwd(const float* logits, const int64_t* labels, int64_t B, int64_t C,
                          int64_t ld, float* loss, float* dlogits, void* stream);

/* ------------------------------------------------------ LayerNorm, add */

/*
 * LayerNorm over the last dimension (the normalisation of the Transformer
 * blocks the paper trains, Appendix C; a support operator whose formula the
 * paper does not give): biased variance over D, eps inside
 * the square root,
 *   y = (x - mean) / sqrt(var + eps) * gamma + beta.
 * x, y: [M, D] contiguous fp32; gamma, beta: [D]; mean, rstd: [M] outputs
 * (1 / sqrt(var + eps)), kept for the backward.
 */
of_status of_layernorm_fwd(const float* x, int64_t M, int64_t D, const float* gamma,
                           const float* beta, float eps, float* y, float* mean, float* rstd,
                           void* stream);

/*
 * of_layernorm_fwd with y stored as bf16 [M, D] (uint16 bit patterns, each the
 * fp32 result rounded to the nearest bf16, ties to even), for an output that
 * only bf16-operand contractions read (a transformer block's LN outputs feed
 * its QKV and FC1 linears): the value such a contraction rounds an fp32 y to,
 * in half the bytes.  mean and rstd are
 * fp32 as in of_layernorm_fwd, bit-identical to it.  y must be 2-byte aligned.
 */
of_status of_layernorm_fwd_bf16(const float* x, int64_t M, int64_t D, const float* gamma,
                                const float* beta, float eps, uint16_t* y, float* mean,
                                float* rstd, void* stream);

/* Number of row groups G of the parameter-gradient partials of
 * of_layernorm_bwd for M rows (1 <= G <= 64). */
int64_t of_layernorm_partial_rows(int64_t M);

/*
 * LayerNorm backward.  With xh = (x - mean) * rstd and g = dy * gamma:
 *   dx = dres + rstd * (g - mean_D(g) - xh * mean_D(g * xh))
 * (dres: optional [M, D] gradient added in, e.g. the residual branch; NULL
 * for none; it may alias dx).  The parameter gradients are written as per
 * row-group partial sums dgamma_rows, dbeta_rows: [G, D] with
 * G = of_layernorm_partial_rows(M), row g holding the sums over rows
 * [g*ceil(M/G), (g+1)*ceil(M/G)) of dy * xh and dy.  Pass them to
 * of_elementwise_fused_update with g_rows = G (backward- or forward-fusion:
 * the gradient vector is never stored) or to of_reduce_rows (eager).
 * dx must not alias dy or x.
 * The two halves may be computed by separate calls, e.g. on two streams
 * (both only read dy and x): dx == NULL computes only the partials (gamma and
 * dres are then not read and may be NULL); dgamma_rows == dbeta_rows == NULL
 * computes only dx.  Results are bit-identical to one call.  OF_EINVAL if
 * all three outputs are NULL or only one of the partials is.
 */
of_status of_layernorm_bwd(const float* dy, const float* x, const float* mean, const float* rstd,
                           const float* gamma, const float* dres, int64_t M, int64_t D, float* dx,
                           float* dgamma_rows, float* dbeta_rows, void* stream);

/* dst[i] = sum over r = 0 .. rows-1, in order, of src[r*ld + i], i < n
 * (ld = 0 means n): materialises a gradient given as row partials. */
of_status of_reduce_rows(const float* src, int64_t rows, int64_t ld, int64_t n, float* dst,
                         void* stream);

/* out = a + b element-wise over n fp32 values (the residual connections of
 * a Transformer block); out may alias a or b. */
of_status of_add(const float* a, const float* b, int64_t n, float* out, void* stream);

/*
 * Mean squared error, forward and backward (a support operator, not defined
 * by the paper):
 *   loss = mean over all M*D elements of (y - t)^2;  dy = 2 (y - t) / (M*D).
 * y: [M, ld], t: [M, D] contiguous, dy: [M, ld]; loss: one fp32 on the device.
 * ws: at least of_mse_workspace_size(M, D) bytes.
 */
size_t of_mse_workspace_size(int64_t M, int64_t D);
of_status of_mse_fwd_bwd(const float* y, const float* t, int64_t M, int64_t D, int64_t ld,
                         float* loss, float* dy, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------- measurement */

/*
 * HBM streaming probe (not part of the paper's method): the read rate
 * (OF_STREAM_READ: src is read, dst receives at most one float), the copy
 * rate (OF_STREAM_COPY: dst = src) or the in-place read-modify-write rate
 * (OF_STREAM_RMW: dst[i] += 1, src unused and may be NULL; the access pattern
 * of an optimizer update, which reads W, m, v and writes them back; with
 * OF_STREAM_RMW3 dst is three consecutive arrays of n/3 floats, n a multiple
 * of 12, and each thread updates the same index of all three together, as
 * an update of W, m and v does) this
 * device reaches with coalesced 128-bit non-temporal accesses, the achievable
 * ceiling beside the published peak for the kernels that stream parameters
 * and optimizer state.  src, dst: n floats of device memory, 16-byte aligned
 * (dst: 4-byte aligned for a read), n a positive multiple of 4; blocks:
 * workgroups of 256 threads (0: 2048).
 * OF_STREAM_RMW3_COLUMNS: as OF_STREAM_RMW3 (n a multiple of 3 * 8192 * 32:
 * three arrays of rows of 8192 floats in whole 32-row chunks), but in the
 * access pattern of of_linear_bwd_merged's W, m, v: 4-byte accesses, a
 * workgroup per 128 columns of a range of rows (at most 8 ranges), a lane
 * per column holding 16 rows of each 32-row chunk in the layout of a 32 x 32
 * fp32 MFMA accumulator; `blocks` is ignored.  That kernel's streaming
 * ceiling.  Errors: OF_EINVAL, OF_EALIGN before any launch.
 */
enum { OF_STREAM_READ = 0, OF_STREAM_COPY = 1, OF_STREAM_RMW = 2, OF_STREAM_RMW3 = 3,
       OF_STREAM_RMW3_COLUMNS = 4 };
of_status of_hbm_stream(int32_t mode, const float* src, float* dst, int64_t n, int32_t blocks,
                        void* stream);

#ifdef __cplusplus
}
#endif

#endif /* OPFUSE_H */
