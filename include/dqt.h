/*
 * dqt.h -- C ABI of libdqt, the training step of a DQT linear layer on
 * AMD MI355X (gfx950).
 *
 * Direct Quantized Training (Zhao et al., "Direct Quantized Training of
 * Language Models with Stochastic Rounding", arXiv 2412.04787) keeps every
 * weight matrix on an n-bit integer grid for the whole of training: the
 * weight is W~ = q * alpha with integer codes q in [qmin, qmax] and one fp32
 * scale per tensor (Sec. 3.2, Eq. 2-4; alpha = 1/s of Eq. 3, fixed after
 * initialisation).  A step is
 *   1. quantise the activations to 8 bits per token       (Sec. 3.2, BitNet),
 *   2. forward  Y  = X~ W~^T                               (Sec. 3.2),
 *   3. backward dX = dY W~ and dW = dY^T X~                (Sec. 3.2, no STE),
 *   4. direct update q <- Clip(SR(q - lr * dW / alpha))    (Sec. 3.1 Eq. 1,
 *                                                           Sec. 3.2 Eq. 5).
 *
 * Conventions for every entry point:
 *  - Tensor pointers are DEVICE pointers unless marked "host".  The caller
 *    owns every buffer; the library never allocates or frees memory on these
 *    calls and holds no mutable global state (except the static scratch of
 *    dqt_linear_fwd_batch_noalloc, and the launch timer while one runs: it
 *    creates and frees its events at start and stop), so calls on different
 *    streams or devices may run concurrently (as long as their buffers
 *    differ).
 *  - Layouts are row-major.  W is [d_out, d_in] (nn.Linear); X is [M, d_in];
 *    Y and dY are [M, d_out].  M is the number of tokens.
 *  - `stream` is a hipStream_t (NULL = the legacy default stream).  Every
 *    device entry point is asynchronous on that stream.
 *  - All arguments are checked before anything is enqueued; on an error
 *    nothing is launched and the status says why.  A launch failure reported
 *    by the runtime returns DQT_ERR_HIP.  Faults during execution surface at
 *    the caller's next synchronisation.  Nothing throws or aborts.
 *  - Shapes: d_in and d_out are multiples of 16 and at least 16; M >= 0 (any
 *    value, M = 0 is a no-op except that dW is then written as zeros).
 *    Base pointers must be 16-byte aligned.
 *  - Non-finite values in X or dY are not checked.
 *  - Workspaces (dqt_linear_fwd / dqt_linear_bwd and their batches) are
 *    caller-owned device buffers of at least the size the matching
 *    *_workspace() call returns.  Their contents on entry do not matter:
 *    the first 256 bytes hold the library's tile counters, which every call
 *    clears on its stream before the kernels that use them.  Calls that
 *    share a workspace must not run concurrently.
 */
#ifndef DQT_H
#define DQT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DQT_OK = 0,
  DQT_ERR_NULL = 1,        /* a required pointer is NULL                      */
  DQT_ERR_SHAPE = 2,       /* a dimension is negative, too small or unaligned */
  DQT_ERR_ALIGN = 3,       /* a base pointer is not 16-byte aligned           */
  DQT_ERR_DTYPE = 4,       /* a dtype is not allowed in that position         */
  DQT_ERR_RANGE = 5,       /* qmin/qmax/alpha/lr out of range                 */
  DQT_ERR_WORKSPACE = 6,   /* workspace missing or smaller than required      */
  DQT_ERR_UNSUPPORTED = 7, /* a valid but unimplemented combination          */
  DQT_ERR_HIP = 8          /* the HIP runtime reported an error               */
} dqt_status;

typedef enum {
  DQT_F32 = 0,        /* IEEE binary32                                        */
  DQT_BF16 = 1,       /* bfloat16                                             */
  DQT_I8 = 2,         /* int8                                                 */
  DQT_FP8E4M3 = 3,    /* OCP E4M3 ("fn": bias 7, max 448, no inf)             */
  DQT_TERNARY2 = 4,   /* packed 2-bit ternary weight codes, see dqt_weight    */
  DQT_INT4 = 5,       /* packed 4-bit weight codes, see dqt_weight            */
  DQT_INT3 = 6        /* packed 3-bit weight codes, see dqt_weight            */
} dqt_dtype;

/*
 * Weight descriptor (Sec. 3.2).
 *   d_out, d_in: multiples of 16, 16 <= d_out, 16 <= d_in <= 65536 (the
 *          int8 forward's int32 sums stay exact: |acc| <= 128 * 128 * 65536
 *          = 2^30); else DQT_ERR_SHAPE.
 *   wfmt = DQT_TERNARY2: q in {-1, 0, 1}; weight (n, k) is stored as the
 *          2-bit code q + 1 in byte n * (d_in / 4) + k / 4, bit offset
 *          2 * (k % 4).  Code 3 is never written and must not appear.
 *          Requires qmin = -1, qmax = 1.
 *   wfmt = DQT_I8: one int8 code per weight, [d_out, d_in] row-major.
 *          Requires -128 <= qmin < qmax <= 127 (Eq. 3 gives -2^(n-1) ..
 *          2^(n-1) - 1; a symmetric -127..127 grid is also allowed).
 *   wfmt = DQT_INT4: the n-bit grids of Eq. 3 for n <= 4 (n = 2, 3, 4:
 *          -2..1, -4..3, -8..7) in 4-bit two's-complement nibbles: weight
 *          (n, k) at byte n * (d_in / 2) + k / 2, low nibble for even k.
 *          Requires -8 <= qmin < qmax <= 7.  The forward and dX expand the
 *          nibbles to int8 or e4m3 / bf16 in the workspace; the updates work
 *          on the nibbles in place.
 *   wfmt = DQT_INT3: the n = 3 grid of Eq. 3 (-4..3) at 3 bits per weight:
 *          each group of 8 weights (n, 8 g .. 8 g + 7) is a 24-bit
 *          little-endian word in bytes n * (3 d_in / 8) + 3 g .. + 2, weight
 *          8 g + j at bits 3 j (two's complement).  Requires
 *          -4 <= qmin < qmax <= 3.  The forward and dX expand the fields to
 *          int8 or e4m3 / bf16 in the workspace; the updates work on the
 *          packed bytes in place.
 *   alpha: dequantisation scale, the weight's real value is q * alpha
 *          (alpha = 1/s, Eq. 3).  Finite and > 0.  Fixed for the life of the
 *          tensor: the library never recomputes it (Sec. 3.2 skips Eq. 2-4
 *          after initialisation).
 *   tensor_id: separates the random streams of different tensors in
 *          dqt_sr_update.
 */
typedef struct {
  int32_t d_out;
  int32_t d_in;
  int32_t wfmt;       /* dqt_dtype: DQT_TERNARY2, DQT_INT3, DQT_INT4 or DQT_I8 */
  int32_t qmin;
  int32_t qmax;
  float alpha;
  uint32_t tensor_id;
  uint32_t reserved;  /* must be 0 */
} dqt_weight;

/*
 * Per-token activation quantisation (Sec. 3.2: inputs and activations are
 * quantised to 8 bits following BitNet).  For each row m of X [M, K]:
 *   g_m = max(max_k |x_mk|, 1e-5)
 *   act_q = DQT_I8:      Xq = clamp(rint(x * fl(127/g_m)), -128, 127),
 *                        xdq[m] = fl(g_m / 127)
 *   act_q = DQT_FP8E4M3: Xq = e4m3_rne_saturate(x * fl(448/g_m)),
 *                        xdq[m] = fl(g_m / 448)
 * Each product and quotient is one correctly rounded fp32 operation.
 *   X:   [M, K], x_t = DQT_F32 or DQT_BF16.   (input)
 *   Xq:  [M, K] int8 or e4m3 bytes.           (output)
 *   xdq: [M] fp32 dequantisation scales.      (output)
 * K must be a multiple of 16; M at most 2^28.
 */
dqt_status dqt_act_quant(const void* X, int32_t x_t, int64_t M, int32_t K,
                         int32_t act_q, void* Xq, float* xdq, void* stream);

/*
 * RMSNorm of each token, then the per-token activation quantisation of
 * dqt_act_quant applied to its output, in one launch: the normalised row
 * never reaches memory.  (In a LLaMA block the q/k/v and gate/up linears
 * take RMSNorm outputs, and Sec. 3.2 quantises the linears' inputs to 8
 * bits; the norm itself is the block's, not the paper's.)  For each row m of
 * X [M, K], every operation one correctly rounded fp32 operation:
 *   s_m  = sum over k of fl(x_mk * x_mk), in this order: lane l = 0..63 adds
 *          the squares of the chunks of 8 consecutive elements l, l + 64,
 *          l + 128, ... (each chunk's elements in order) into a sum starting
 *          at 0; then for d = 32, 16, 8, 4, 2, 1 every lane sum s_l becomes
 *          s_l + s_(l xor d); s_m is the result
 *   r_m  = 1 / sqrt(s_m / K + eps)
 *   y_mk = (x_mk * r_m) * gamma_k
 *   Xq, xdq: dqt_act_quant of y (act_q = DQT_I8 or DQT_FP8E4M3).
 *   X: [M, K], x_t = DQT_F32 or DQT_BF16; gamma: [K] fp32; eps: finite, > 0.
 *   Xq: [M, K] codes; xdq: [M] scales; rinv: NULL or [M] fp32, receives r_m
 *   (for the norm's backward).  K a multiple of 16, M at most 2^28.
 */
dqt_status dqt_rmsnorm_act_quant(const void* X, int32_t x_t, const float* gamma,
                                 float eps, int64_t M, int32_t K, int32_t act_q,
                                 void* Xq, float* xdq, float* rinv, void* stream);

/*
 * Backward of the RMSNorm in front of a group of linears, for training a
 * model built of DQT layers (the norm is the model's, not the paper's; its
 * forward is dqt_rmsnorm_act_quant, whose rinv this takes).  The linears' dX
 * pass straight through the activation quantiser, so the norm's output
 * gradient is their sum.  For each row m of X [M, K], in fp32:
 *   dn_mk = sum over i of dY_i[m, k]          (i = 0 .. n_dy - 1 in order)
 *   g_mk  = dn_mk gamma_k,  c_m = (sum over k of g_mk x_mk) / K
 *   dX_mk = r_m g_mk - x_mk r_m^3 c_m         (rounded to bf16)
 *   gpart[b, k] = sum over the rows m of block b of dn_mk x_mk r_m
 * so that the gradient of gamma is the sum of gpart over b (the caller
 * sums).  Block b takes rows 4 b .. 4 b + 3, then those blocks * 4 further on.
 *   n_dy: 1 .. 4; dY: host array of n_dy device pointers to [M, K] bf16.
 *   X: [M, K], x_t = DQT_BF16; gamma: [K] fp32; rinv: [M] fp32.
 *   dX: [M, K] bf16 (output, aliasing no input); gpart: [blocks, K] fp32
 *   (output); blocks: 1 .. 65536.  K: a multiple of 16, at most 8192.
 * Errors: DQT_ERR_NULL, DQT_ERR_SHAPE, DQT_ERR_DTYPE, DQT_ERR_ALIGN.
 */
dqt_status dqt_rmsnorm_backward(int32_t n_dy, const void* const* dY, const void* X, int32_t x_t,
                                const float* gamma, const float* rinv, int64_t M, int32_t K,
                                void* dX, float* gpart, int32_t blocks, void* stream);

/* Bytes of device workspace for the fastest form of dqt_linear_fwd on this
 * weight: the 256 counter bytes, plus, for ternary, 3-bit and 4-bit codes,
 * d_out * d_in bytes the codes are expanded into (int8 or e4m3 bytes, or
 * FP4 E2M1 values at half a byte each for ternary codes against e4m3
 * activations).  Ternary codes with d_in a multiple of 64 also run from the
 * packed codes, expanded in registers, with the 256 counter bytes alone: a
 * smaller workspace than this selects that form (same results for int8
 * activations, bit for bit; within the e4m3 forward's tolerance otherwise).
 * Depends only on the descriptor. */
size_t dqt_linear_fwd_workspace(const dqt_weight* w);

/*
 * Forward of a DQT linear (Sec. 3.2):  Y = X~ W~^T, i.e.
 *   acc[m, n] = sum_k Xq[m, k] * q[n, k]     (int32, exact, for int8 codes;
 *                                             fp32 MFMA sum for e4m3 codes)
 *   Y[m, n]   = fl(fl(acc) * fl(xdq[m] * alpha)), cast to y_t (RNE).
 *   w, Wq: weight descriptor (host) and codes (device).
 *   X:     [M, d_in] (x_t = DQT_F32/DQT_BF16), or NULL when Xq/xdq already
 *          hold this input's quantised form (several linears sharing one
 *          input quantise it once with dqt_act_quant).
 *   act_q: DQT_I8 or DQT_FP8E4M3 (e4m3 needs wfmt = DQT_TERNARY2, DQT_INT3
 *          or DQT_INT4, whose values e4m3 holds exactly).
 *   Xq, xdq: [M, d_in] codes and [M] scales; written when X != NULL, read
 *          otherwise.  Keep them for dqt_linear_bwd.
 *   Y:     [M, d_out], y_t = DQT_F32 or DQT_BF16.  (output)
 *   ws, ws_bytes: device workspace of dqt_linear_fwd_workspace() bytes, or
 *          of at least the 256 counter bytes for ternary codes with d_in a
 *          multiple of 64 (see dqt_linear_fwd_workspace); DQT_ERR_WORKSPACE
 *          when smaller.
 */
dqt_status dqt_linear_fwd(const dqt_weight* w, const void* Wq,
                          const void* X, int32_t x_t, int64_t M, int32_t act_q,
                          void* Xq, float* xdq,
                          void* Y, int32_t y_t,
                          void* ws, size_t ws_bytes, void* stream);

/* Bytes of device workspace dqt_linear_bwd needs for this weight and M.
 * Depends only on (d_out, d_in, M) and covers every dtype combination:
 * fp32 split-reduction partials, the weights unpacked to bf16 (dX) and the
 * dequantised activation X~ in bf16 (dW). */
size_t dqt_linear_bwd_workspace(const dqt_weight* w, int64_t M);

/*
 * Backward of a DQT linear (Sec. 3.2).  The gradient is taken with respect to
 * the quantised weight W~ itself (no straight-through estimator on weights);
 * the activation quantiser is treated as the identity (BitNet convention):
 *   dX[m, k] = alpha * sum_n dY[m, n] * q[n, k]          cast to dx_t
 *   dW[n, k] = sum_m dY[m, n] * X~[m, k]                 fp32
 * with X~[m, k] = cast_xt(fl(value(Xq[m, k]) * xdq[m])), the dequantised
 * activation in the environment dtype xt_t (DQT_F32 or DQT_BF16).
 * Products of bf16 operands are summed in fp32 by the matrix cores; with
 * xt_t = DQT_F32 the operands are fp32 (dY must then be DQT_F32).
 *   dY: [M, d_out], dy_t = DQT_F32 or DQT_BF16.
 *   dX: [M, d_in] or NULL (skipped); dx_t = DQT_F32 or DQT_BF16.
 *   dW: [d_out, d_in] fp32 or NULL (skipped); overwritten, never accumulated.
 *   ws, ws_bytes: device workspace of at least dqt_linear_bwd_workspace()
 *   bytes.  Results do not depend on timing: the split reduction over tokens
 *   is summed in a fixed order.
 */
dqt_status dqt_linear_bwd(const dqt_weight* w, const void* Wq,
                          const void* Xq, int32_t act_q, const float* xdq,
                          const void* dY, int32_t dy_t, int64_t M, int32_t xt_t,
                          void* dX, int32_t dx_t, float* dW,
                          void* ws, size_t ws_bytes, void* stream);

/*
 * Direct stochastic-rounding update (Sec. 3.1 Eq. 1 and Sec. 3.2 Eq. 5),
 * in place on Wq.  In grid units the optimiser target W' = W~ - lr * dW is
 * x = q + delta with delta = -fl(c * dW), c = fl(lr / alpha) (formed once on
 * the host).  Eq. 1 rounds x to floor(x) with probability ceil(x) - x and to
 * ceil(x) otherwise; the result is clipped to [qmin, qmax] and stored back.
 * Random bits for element i = n * d_in + k (32 bits, exact 2^-32
 * resolution): U(i) = P16(i) << 16 | S16(i), where P16/S16 are 16-bit halves
 * of Philox4x32-10 (Salmon et al., SC'11) with key (lo32(seed), hi32(seed))
 * and counter (lo32(i >> 3), hi32(i >> 3) | s << 31, step, tensor_id),
 * s = 0 for P16 and 1 for S16; element i takes output word (i & 7) >> 1, low
 * half for even i, high half for odd i.  The move away from q's side
 * happens iff U < ceil(p * 2^32) where p is the distance of x from the grid
 * point on q's side.
 *   dW:  [d_out, d_in] fp32.  A non-finite entry leaves its weight unchanged
 *        and is counted in counters[1].
 *   lr:  finite, >= 0.
 *   counters: NULL, or device uint64[2] to which the number of changed
 *        weights and of non-finite gradient entries are ADDED.
 * Each thread owns whole bytes of Wq, so the update has no write races and
 * is bit-reproducible for a given (seed, step, tensor_id).
 */
dqt_status dqt_sr_update(const dqt_weight* w, void* Wq, const float* dW,
                         float lr, uint64_t seed, uint32_t step,
                         unsigned long long* counters, void* stream);

/*
 * Batches.  One call runs the same step for up to DQT_MAX_BATCH linears that
 * share the token count M and the dtypes (e.g. the seven linears of a
 * transformer block), as one launch per stage, so that the tiles of every
 * linear fill the GPU together.  Results are those of the single-linear calls
 * above; only the split of the dW reduction over tokens (a fixed function of
 * the batch's shapes) may differ, which changes dW by fp32 rounding only.
 * Linears may share Xq/xdq (the same input); the activation X~ is then
 * formed once.  All weights of a batch must have the same wfmt.
 */
#define DQT_MAX_BATCH 8

typedef struct {
  const dqt_weight* w;  /* descriptor (host pointer)                          */
  void* Wq;             /* codes (device); dqt_sr_update_batch updates them    */
  const void* Xq;       /* [M, d_in] quantised input (dqt_act_quant)           */
  const float* xdq;     /* [M] its per-token scales                            */
  void* Y;              /* forward output [M, d_out]                           */
  const void* dY;       /* upstream gradient [M, d_out]                        */
  void* dX;             /* input gradient [M, d_in], or NULL to skip           */
  float* dW;            /* weight gradient [d_out, d_in] fp32, or NULL to skip */
} dqt_linear_io;

/* Workspace bytes of the fastest form of dqt_linear_fwd_batch (see
 * dqt_linear_fwd_workspace: the sum over the linears, counters once);
 * depends only on the descriptors. */
size_t dqt_linear_fwd_batch_workspace(int32_t n, const dqt_linear_io* io);

/* Forward of n linears (see dqt_linear_fwd; inputs already quantised).
 * Uses w, Wq, Xq, xdq, Y of each entry. */
dqt_status dqt_linear_fwd_batch(int32_t n, const dqt_linear_io* io, int64_t M,
                                int32_t act_q, int32_t y_t,
                                void* ws, size_t ws_bytes, void* stream);

/*
 * The forward of n linears (dqt_linear_fwd_batch) without a workspace
 * argument, for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation.  The
 * call allocates nothing: its scratch (the tile counters, plus the operand
 * bytes of dqt_linear_fwd_batch_workspace() when they fit; ternary codes
 * whose expansion does not fit run from the packed codes) is a static device
 * array of DQT_NOALLOC_SCRATCH_BYTES that each GPU the library runs on holds
 * until the process ends; its address is looked up on a device's first call.
 * Calls on one GPU share that array, so calls that overlap in time on one
 * GPU (different streams, or threads without ordering) race and must not be
 * made; the counters are cleared by every call on its stream.
 *   Arguments and results: those of dqt_linear_fwd_batch.
 *   Errors: those of dqt_linear_fwd_batch; DQT_ERR_WORKSPACE when the
 *   smallest workspace of the batch exceeds DQT_NOALLOC_SCRATCH_BYTES
 *   (nothing is launched); DQT_ERR_HIP when the array's address cannot be
 *   found.
 */
#define DQT_NOALLOC_SCRATCH_BYTES (32u << 20)

dqt_status dqt_linear_fwd_batch_noalloc(int32_t n, const dqt_linear_io* io, int64_t M,
                                        int32_t act_q, int32_t y_t, void* stream);

/* Workspace bytes of dqt_linear_bwd_batch; depends only on the descriptors'
 * shapes and M. */
size_t dqt_linear_bwd_batch_workspace(int32_t n, const dqt_linear_io* io,
                                      int64_t M);

/* Backward of n linears (see dqt_linear_bwd).  Uses w, Wq, Xq, xdq, dY, dX,
 * dW of each entry; dX and dW may be NULL per entry. */
dqt_status dqt_linear_bwd_batch(int32_t n, const dqt_linear_io* io, int64_t M,
                                int32_t act_q, int32_t dy_t, int32_t xt_t,
                                int32_t dx_t, void* ws, size_t ws_bytes,
                                void* stream);

/* Activation quantisation (see dqt_act_quant) of n inputs with the same M
 * and dtypes in one launch.  Entry s quantises X [M, K] into Xq and xdq. */
typedef struct {
  const void* X;        /* [M, K] input (device)                               */
  void* Xq;             /* [M, K] codes (device, output)                       */
  float* xdq;           /* [M] scales (device, output)                         */
  int32_t K;            /* row length, a multiple of 16                        */
  int32_t reserved;     /* must be 0                                           */
} dqt_act_io;

dqt_status dqt_act_quant_batch(int32_t n, const dqt_act_io* io, int32_t x_t,
                               int64_t M, int32_t act_q, void* stream);

/* Direct SR update of n weight tensors in one launch (see dqt_sr_update);
 * uses w, Wq, dW of each entry.  Each tensor draws from its own stream
 * (tensor_id); counters, when given, receive the totals over all tensors. */
dqt_status dqt_sr_update_batch(int32_t n, const dqt_linear_io* io, float lr,
                               uint64_t seed, uint32_t step,
                               unsigned long long* counters, void* stream);

/*
 * Direct SR update of any number of weight tensors in one launch (Sec. 3.2:
 * Eq. 5 is applied to every weight matrix of the model at every step), with
 * the per-tensor fractions of changed weights of Sec. 5.2 counted in the
 * same pass.  The tensors are described by a table in device memory:
 *   dqt_sr_table_bytes(n):  bytes of the table of n tensors (64 per tensor).
 *   dqt_sr_table_build (host): validates entries io[0 .. n-1] (w, Wq, dW;
 *          one code format; the checks of dqt_sr_update_batch) and writes
 *          the table into the host buffer `table` of table_bytes bytes.  The
 *          caller copies it to device memory; the copy stays valid for as
 *          long as the descriptors and the Wq / dW addresses do not change,
 *          so it is built once and reused every step.
 *   dqt_sr_update_table: the update of every tensor of io (checked again,
 *          as by dqt_sr_table_build), reading the tensors from `table`, the
 *          device copy of dqt_sr_table_build(n, io); results are those of
 *          dqt_sr_update on each tensor with its own tensor_id (the step size
 *          fl(lr / alpha) is formed on the device by the same correctly
 *          rounded fp32 division).
 *          counters: NULL, or device uint64[2] (changed, non-finite; ADDED).
 *          per_tensor: NULL, or device uint64[2 n]; entry 2 s (2 s + 1)
 *          receives the changed (non-finite) count of tensor s (ADDED).
 *   Errors: DQT_ERR_SHAPE (n < 1), DQT_ERR_NULL, DQT_ERR_ALIGN (16 bytes
 *   for the table, 8 for the counters), DQT_ERR_WORKSPACE (host buffer too
 *   small), DQT_ERR_UNSUPPORTED (mixed code formats), DQT_ERR_RANGE, and
 *   the weight checks of dqt_sr_update.
 */
size_t dqt_sr_table_bytes(int32_t n);
dqt_status dqt_sr_table_build(int32_t n, const dqt_linear_io* io, void* table,
                              size_t table_bytes);
dqt_status dqt_sr_update_table(int32_t n, const dqt_linear_io* io, const void* table,
                               float lr, uint64_t seed, uint32_t step,
                               unsigned long long* counters,
                               unsigned long long* per_tensor, void* stream);

/*
 * Analysis variants of the direct update (Sec. 5).  The paper contrasts SR
 * with a deterministic rounding that drops small updates, and intervenes in
 * the smallest 20 % of each step's updates, keeping those codes or forcing
 * them to change.  With delta = -fl(fl(lr / alpha) * dW) as in
 * dqt_sr_update and x = q + delta:
 *   DQT_UPD_SR            the plain update (dqt_sr_update_batch);
 *   DQT_UPD_NEAREST       x rounded to the nearest grid value, ties to even;
 *   DQT_UPD_FORCE_REMAIN  codes in the bottom set keep their value,
 *   DQT_UPD_FORCE_CHANGE  codes in the bottom set take x rounded away from q
 *                         (ceil for delta > 0, floor for delta < 0);
 *   every other code (and every code under DQT_UPD_SR) takes the plain
 *   update with its draws, then all are clipped to [qmin, qmax].
 * The bottom set of a tensor is {key <= tau}: key is the fp32 bit pattern of
 * |fl(fl(lr / alpha) * dW)| as an unsigned integer (a non-finite dW ranks
 * above every finite one), tau the k-th smallest key, k = floor(frac * n) in double
 * (n = d_out * d_in < 2^32; ties at tau may enlarge the set; k = 0 leaves it
 * empty).  A non-finite dW keeps its code and is counted in counters[1].
 *   frac: in [0, 1] (used by the two force modes).
 *   ws, ws_bytes: dqt_update_variant_workspace(n) bytes for the force modes
 *   (the exact selection's state); NULL / 0 allowed for the other modes.
 * Uses w, Wq (updated in place) and dW of each entry of io.
 */
#define DQT_UPD_SR 0
#define DQT_UPD_NEAREST 1
#define DQT_UPD_FORCE_REMAIN 2
#define DQT_UPD_FORCE_CHANGE 3

size_t dqt_update_variant_workspace(int32_t n);

dqt_status dqt_update_variant_batch(int32_t n, const dqt_linear_io* io, float lr,
                                    uint64_t seed, uint32_t step, int32_t mode,
                                    float frac, unsigned long long* counters,
                                    void* ws, size_t ws_bytes, void* stream);

/*
 * The deterministic control of Sec. 5.1 read literally: instead of the
 * stochastic rounding of Eq. 5, the updated real-valued matrix W' = W~ -
 * lr dW (W~ = q alpha) is absmax-quantised afresh, i.e. Eq. 3-4 with the
 * maximum of |W'| in place of the mean, which gives the tensor a new scale
 * every step.  Per tensor, every operation one correctly rounded fp32
 * operation:
 *   W'_i   = q_i alpha - lr dW_i        (a non-finite dW_i is read as 0 and
 *                                        counted in counters[1])
 *   m      = max_i |W'_i|;  s' = qmax / m;  alpha' = m / qmax
 *   q'_i   = Clip(rint(W'_i s'), qmin, qmax)     (rint: ties to even)
 * with m = 0 giving q' = 0 and alpha' = alpha.  The codes are updated in
 * place and alpha' of tensor l is written to alpha_out[l] (device fp32 [n]);
 * the caller adopts it (the descriptor's alpha) for the next step.
 *   counters: NULL, or device uint64[2] (changed, non-finite; ADDED).
 *   ws, ws_bytes: dqt_absmax_requant_workspace(n) bytes of device memory.
 * Uses w, Wq, dW of each of the n (1..DQT_MAX_BATCH) entries of io.
 */
size_t dqt_absmax_requant_workspace(int32_t n);
dqt_status dqt_absmax_requant_batch(int32_t n, const dqt_linear_io* io, float lr,
                                    float* alpha_out, unsigned long long* counters,
                                    void* ws, size_t ws_bytes, void* stream);

/*
 * AdamW with direct stochastic rounding.  The paper trains DQT with AdamW
 * modified to round stochastically (Sec. 4.1): the optimiser's target W'
 * (Sec. 3.2) is the AdamW step with decoupled weight decay and bias
 * correction, and the new code is Clip(SR(W' / alpha)) (Eq. 1 and 5 in grid
 * units, the draws of dqt_sr_update).  The paper gives no further detail;
 * this library fixes, per element, in fp32 with round-to-nearest-even after
 * every operation (no fused multiply-add; sqrt and division correctly
 * rounded):
 *   m' = b1 m + ob1 g,   v' = b2 v + (ob2 g) g,
 *   u  = m' / (sqrt(v') k2 + eps),   delta = -(cu u + cd q),   x = q + delta,
 * with per-call constants formed in double and rounded once to fp32:
 *   b1 = beta1, b2 = beta2, ob1 = 1 - b1, ob2 = 1 - b2,
 *   k2 = 1 / sqrt(1 - b2^t), cu = lr / (alpha (1 - b1^t)), cd = lr wd,
 * t = step, b^t by binary exponentiation (low bit first) in double.
 * An element whose gradient is non-finite or whose delta is NaN keeps its
 * code, m and v and is counted in counters[1].
 */
typedef struct {
  float lr;             /* >= 0, finite                                         */
  float beta1, beta2;   /* in [0, 1)                                            */
  float eps;            /* > 0, finite                                          */
  float weight_decay;   /* >= 0, finite (decoupled: W' includes -lr wd W~)      */
} dqt_adamw;

/* One tensor.  Wq (codes), m and v ([d_out, d_in] fp32, both zero before
 * the first step) are updated in place; dW: [d_out, d_in] fp32.  step >= 1
 * is AdamW's t and keys the draws as in dqt_sr_update.  counters: NULL, or
 * device uint64[2] to which the changed and non-finite counts are ADDED.
 * Errors: DQT_ERR_NULL, DQT_ERR_ALIGN (16 bytes), DQT_ERR_RANGE (a
 * hyper-parameter out of range, step 0, or a non-finite cu). */
dqt_status dqt_adamw_sr_update(const dqt_weight* w, void* Wq, const float* dW,
                               float* m, float* v, const dqt_adamw* hp,
                               uint64_t seed, uint32_t step,
                               unsigned long long* counters, void* stream);

/* n tensors of one code format in one launch; uses w, Wq, dW of each entry
 * of io, and m[l], v[l] (host arrays of n device pointers). */
dqt_status dqt_adamw_sr_update_batch(int32_t n, const dqt_linear_io* io,
                                     float* const* m, float* const* v,
                                     const dqt_adamw* hp, uint64_t seed,
                                     uint32_t step, unsigned long long* counters,
                                     void* stream);

/*
 * Backward and direct SR update of n linears in one call (Sec. 3.2: the
 * update of Eq. 5 consumes dW of the backward), with dW never written to the
 * caller's memory: the dW product's epilogue updates the 8 codes of each
 * group of 8 consecutive weights of a row as it forms their gradients; when
 * the dW reduction over tokens is split, the kernel that sums the partials
 * does.  With the environment variable DQT_SR_EPILOGUE=staged, dW is
 * instead staged in the workspace and a streaming pass updates the codes
 * (same dW bits, same codes); the workspace query reads it too.  The codes and counters equal those of dqt_linear_bwd_batch
 * writing dW followed by dqt_sr_update_batch on that dW, bit for bit; dX is
 * formed from the codes as they were before the update.
 *   io: uses w, Wq (updated in place), Xq, xdq, dY, dX of each entry; dX may
 *       be NULL per entry; every dW must be NULL (DQT_ERR_UNSUPPORTED
 *       otherwise: use the two calls to keep dW).
 *   dy_t, xt_t: DQT_BF16 only (the matrix-core path); other values return
 *       DQT_ERR_UNSUPPORTED.  dx_t: DQT_F32 or DQT_BF16.
 *   lr, seed, step, counters: as dqt_sr_update_batch.
 *   ws, ws_bytes: at least dqt_linear_bwd_batch_workspace(n, io, M) bytes.
 *   M = 0: dW is zero, which moves no weight; nothing is launched.
 */
dqt_status dqt_linear_bwd_sr_batch(int32_t n, const dqt_linear_io* io, int64_t M,
                                   int32_t act_q, int32_t dy_t, int32_t xt_t,
                                   int32_t dx_t, float lr, uint64_t seed,
                                   uint32_t step, unsigned long long* counters,
                                   void* ws, size_t ws_bytes, void* stream);

/*
 * Helpers (not on the timed path).
 */

/* The 32-bit draws U(i), i = i0 .. i0 + n - 1, of dqt_sr_update, written to
 * device out[n].  For checking the random stream. */
dqt_status dqt_debug_rng(uint64_t seed, uint32_t step, uint32_t tensor_id,
                         uint64_t i0, int64_t n, uint32_t* out, void* stream);

/* AbsMean initial quantisation on the host (Sec. 3.2, Eq. 2-4):
 *   AbsMean = mean |W0| (sum in fp64, index order), s = qmax / AbsMean,
 *   q = clip(rint(W0 * s), qmin, qmax) with the product in fp64,
 *   alpha = fl32(AbsMean / qmax).
 * W0: host fp32 [n]; q: host int8 [n] (output); alpha: host (output).
 * Returns DQT_ERR_RANGE when AbsMean is 0 or not finite. */
dqt_status dqt_absmean_init(const float* W0, int64_t n, int32_t qmin,
                            int32_t qmax, int8_t* q, float* alpha);

/* Host packing of ternary codes into the DQT_TERNARY2 layout and back.
 * q: host int8 [rows, cols] in {-1, 0, 1}; packed: host uint8 [rows, cols/4];
 * cols must be a multiple of 4.  pack returns DQT_ERR_RANGE (and stops) on a
 * value outside {-1, 0, 1}. */
dqt_status dqt_pack_ternary(const int8_t* q, int64_t rows, int64_t cols,
                            uint8_t* packed);
dqt_status dqt_unpack_ternary(const uint8_t* packed, int64_t rows,
                              int64_t cols, int8_t* q);

/* Host packing of codes in [-8, 7] into the DQT_INT4 layout and back.
 * q: host int8 [rows, cols]; packed: host uint8 [rows, cols/2]; cols must be
 * even.  pack returns DQT_ERR_RANGE (and stops) on a value outside [-8, 7]. */
dqt_status dqt_pack_int4(const int8_t* q, int64_t rows, int64_t cols, uint8_t* packed);
dqt_status dqt_unpack_int4(const uint8_t* packed, int64_t rows, int64_t cols, int8_t* q);

/* Host packing of codes in [-4, 3] into the DQT_INT3 layout and back.
 * q: host int8 [rows, cols]; packed: host uint8 [rows, 3 cols / 8]; cols a
 * multiple of 8.  pack returns DQT_ERR_RANGE (and stops) on a value outside
 * [-4, 3]. */
dqt_status dqt_pack_int3(const int8_t* q, int64_t rows, int64_t cols, uint8_t* packed);
dqt_status dqt_unpack_int3(const uint8_t* packed, int64_t rows, int64_t cols, int8_t* q);

/* ------------------------------------------------------------ measurement
 * Launch timer: the durations of the library's GEMM kernel launches (the
 * forward, dX and dW products, alone or in one launch), without the passes
 * around them, for a caller that measures a kernel against its roofline.
 * Not for graph capture: the events are recorded when a launch is issued.
 *
 *   dqt_launch_timer_start(max_launches): creates 2 * max_launches events
 *          (1 <= max_launches <= DQT_LAUNCH_TIMER_MAX; else DQT_ERR_SHAPE) on
 *          the current device; from then on every GEMM kernel launch, in
 *          issue order, is bracketed by the next pair, recorded on the call's
 *          stream, until max_launches are taken (later launches run
 *          untimed).  One timer per process: DQT_ERR_UNSUPPORTED while one
 *          runs.  Timed launches must run on the device current at start.
 *   dqt_launch_timer_stop(ms, max, count): waits for the recorded pairs,
 *          writes the first min(max, *count) durations (milliseconds, host
 *          float[max]) to ms, the number of timed launches to *count, and
 *          frees the events.  DQT_ERR_UNSUPPORTED when no timer runs;
 *          DQT_ERR_NULL / DQT_ERR_SHAPE for bad arguments (the timer keeps
 *          running); DQT_ERR_HIP if an event fails (the events are freed).
 */
#define DQT_LAUNCH_TIMER_MAX 65536
dqt_status dqt_launch_timer_start(int32_t max_launches);
dqt_status dqt_launch_timer_stop(float* ms, int32_t max, int32_t* count);

/* A plain streaming read of `bytes` bytes of device memory (one pass, 16-byte
 * non-temporal loads over a fixed grid of DQT_READ_STREAM_SINK_WORDS / 4
 * blocks): the read rate this chip achieves, which the streaming kernels
 * (SR update, AdamW) are compared with.
 *   src:   device, 16-byte aligned; bytes a multiple of 16 (DQT_ERR_SHAPE),
 *          0 does nothing.
 *   sink:  device uint32[DQT_READ_STREAM_SINK_WORDS], 16-byte aligned:
 *          receives xors of the data read (so no read is elided).
 *   Asynchronous on `stream`; DQT_ERR_NULL / DQT_ERR_ALIGN for bad pointers.
 */
#define DQT_READ_STREAM_SINK_WORDS 32768
dqt_status dqt_read_stream(const void* src, size_t bytes, uint32_t* sink, void* stream);

/* Human-readable name of a status code (static storage). */
const char* dqt_status_string(int32_t status);

/* Library version as MAJOR * 10000 + MINOR * 100 + PATCH. */
int32_t dqt_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DQT_H */
