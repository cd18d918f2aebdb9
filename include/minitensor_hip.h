/*
 * libminitensor_hip: MI355X (gfx950) kernels for the dense layer and the
 * broadcasting matmul of MiniTensor, with their reverse-mode gradients.
 *
 * Operations (MiniTensor paper):
 *   Sec. 3.1, Eq. (1)   matmul Y = X W^T, and the NumPy/PyTorch broadcasting
 *                       rule (left-pad with singleton dims, virtually expand
 *                       size-1 dims without materialising them).
 *   Sec. 3.2, Eq. (4)   matmul pullbacks  Xbar += Ybar W,  Wbar += Ybar^T X;
 *                       add pullback      xbar += zbar (summed over the axes
 *                       an input was broadcast along).
 *   Sec. 3.3, Eq. (5)   Dense(x; W, b) = x W^T + 1 b^T.
 *   Sec. 3.5            gradient buffers exist only when a backward needs them
 *                       (here: a null output pointer skips its work).
 *
 * Conventions for every entry point
 *   - Tensors are described by mt_tensor: a device pointer, a dtype, a rank
 *     and per-dim sizes and strides counted in ELEMENTS (not bytes).
 *   - The caller owns every buffer. No entry point allocates device memory.
 *     Workspace, where an entry point takes one, is caller-supplied device
 *     memory; its required size comes from the matching *_workspace call.
 *     A NULL workspace (or one that is too small) selects a slower variant
 *     that needs none, so workspace only ever buys speed (the convolution,
 *     whose unfolded input lives there, is the one exception).
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     All device work is enqueued on it asynchronously; results are visible
 *     after the caller synchronises that stream.
 *   - Every argument is validated on the host before any HIP call. On failure
 *     the call returns a non-zero mt_status, enqueues nothing, leaves every
 *     output untouched and records a message for mt_last_error() (per
 *     thread). A failed launch returns MT_ERR_HIP with HIP's error string.
 *     Device faults surface at the caller's next synchronisation. No C++
 *     exception or abort crosses this interface.
 *   - Outputs must not overlap any input or each other (MT_ERR_ALIAS).
 *   - Results are deterministic: no floating-point atomics are used, so the
 *     same call on the same inputs returns bit-identical outputs.
 *   - Floating point: fp32 operands are multiplied and accumulated in fp32
 *     (matrix cores, v_mfma_f32_32x32x2_f32). bf16 operands are multiplied
 *     exactly and accumulated in fp32 (v_mfma_f32_32x32x16_bf16). Every
 *     output, bias and bias gradient is fp32.
 */
#ifndef MINITENSOR_HIP_H
#define MINITENSOR_HIP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MT_MAX_DIMS 8

typedef enum { MT_F32 = 0, MT_BF16 = 1 } mt_dtype;

typedef enum {
  MT_OK = 0,
  MT_ERR_NULL = 1,        /* a required pointer is NULL */
  MT_ERR_NDIM = 2,        /* rank outside what the operation accepts */
  MT_ERR_SHAPE = 3,       /* sizes do not match / do not broadcast */
  MT_ERR_DTYPE = 4,       /* unsupported dtype or dtype combination */
  MT_ERR_LAYOUT = 5,      /* strides the kernels cannot address */
  MT_ERR_ALIAS = 6,       /* an output overlaps an input or another output */
  MT_ERR_WORKSPACE = 7,   /* workspace pointer given with a bad size/alignment */
  MT_ERR_HIP = 8,         /* the HIP runtime reported an error */
  MT_ERR_INVALID = 9      /* any other invalid argument (flags, negative size) */
} mt_status;

/* A strided view of device memory. Sizes and strides are in elements. */
typedef struct {
  void* data;
  int32_t dtype;                 /* mt_dtype */
  int32_t ndim;                  /* 0..MT_MAX_DIMS */
  int64_t shape[MT_MAX_DIMS];
  int64_t stride[MT_MAX_DIMS];
} mt_tensor;

/* Flags. */
#define MT_ACCUMULATE 1u   /* out += result (the "+=" of the pullbacks, Sec. 3.2);
                              default: out = result */
#define MT_REDUCE_INTO 2u  /* mt_matmul: c may have the shape of the full result
                              summed over some batch axes (the un-broadcast shape
                              of an operand); the sum is folded into the product */
#define MT_CONV_REUSE_UNFOLD 4u  /* mt_conv2d_bwd: the start of ws still holds the
                              unfolded input that mt_conv2d_fwd wrote there for the
                              same x, w, stride and padding (the forward's workspace
                              passed again, untouched since); dw then skips the
                              unfolding. The backward overwrites it (when dx is
                              asked), so it serves one backward. Ignored where the
                              forward may have gathered the image instead (the
                              layouts listed under mt_conv2d_fwd, C a multiple
                              of 32): the backward then never reads the unfolded
                              input, or unfolds it itself. */

/* ------------------------------------------------------------------ linear
 * mt_linear_fwd: Y = X W^T + 1 b^T (Eq. (5); with b == NULL, Eq. (1)).
 *   x [M, K]  f32 or bf16          w [N, K] same dtype as x
 *   b [N]     f32, or NULL          y [M, N] f32
 * Matrix operands may have any row pitch (stride[0] >= inner size) but their
 * inner dim must be contiguous (stride[1] == 1; MT_ERR_LAYOUT otherwise).
 * b must be contiguous. M, N or K may be 0 (K == 0 writes y = b or 0).
 */
mt_status mt_linear_fwd(const mt_tensor* x, const mt_tensor* w, const mt_tensor* b,
                        const mt_tensor* y, void* stream);

/* mt_linear_bwd: gradients of Eq. (5) from the upstream gradient dY:
 *   dx [M, K] = dY W        (Eq. (4))       f32, or NULL to skip
 *   dw [N, K] = dY^T X      (Eq. (4))       f32, or NULL to skip
 *   db [N]    = 1^T dY      (add pullback)  f32, or NULL to skip
 *   x [M, K], w [N, K], dy [M, N] share one dtype (f32 or bf16); x may be
 *   NULL when dw is NULL and w may be NULL when dx is NULL.
 * flags: MT_ACCUMULATE adds into dx/dw/db instead of overwriting.
 * ws/ws_bytes: optional workspace (size from mt_linear_bwd_workspace); used
 * for split reductions of db and split-K partial sums of dx / dw when their
 * output tiles under-fill the GPU.
 * With dw and db both requested, db is summed inside the dW product from the
 * dY tiles it reads (db is the column sum of that product's left operand
 * dY^T), so dY is streamed once; db alone runs a column-sum pass over dY.
 */
mt_status mt_linear_bwd(const mt_tensor* x, const mt_tensor* w, const mt_tensor* dy,
                        const mt_tensor* dx, const mt_tensor* dw, const mt_tensor* db,
                        uint32_t flags, void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes mt_linear_bwd can use for these arguments (0 if none). */
mt_status mt_linear_bwd_workspace(const mt_tensor* x, const mt_tensor* w, const mt_tensor* dy,
                                  const mt_tensor* dx, const mt_tensor* dw, const mt_tensor* db,
                                  size_t* bytes);

/* mt_linear_bwd_noalloc: mt_linear_bwd for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc). It takes no workspace: the split-K partials and db
 * row-slice sums go to a fixed scratch array inside the library, one per GPU
 * (MT_NOALLOC_SCRATCH_BYTES, held from the first call on that GPU until the
 * process ends). The call allocates nothing; it runs the same kernels with
 * the same plan as mt_linear_bwd given a workspace of the size
 * mt_linear_bwd_workspace reports, so the results are bit-identical to that.
 *   Arguments, flags and errors as mt_linear_bwd; in addition
 *   MT_ERR_WORKSPACE (nothing enqueued) when these sizes need more scratch
 *   than MT_NOALLOC_SCRATCH_BYTES, and MT_ERR_INVALID when `stream` does not
 *   belong to the current device.
 *   Every call on one GPU shares that GPU's scratch array: calls that overlap
 *   in time on one GPU (other streams, other threads) race and must be
 *   ordered by the caller. Nothing in the array needs to start at zero.
 */
#define MT_NOALLOC_SCRATCH_BYTES (32u << 20)
mt_status mt_linear_bwd_noalloc(const mt_tensor* x, const mt_tensor* w, const mt_tensor* dy,
                                const mt_tensor* dx, const mt_tensor* dw, const mt_tensor* db,
                                uint32_t flags, void* stream);

/* ------------------------------------------ dense layer + nonlinearity
 * Nonlinearities of Sec. 3.3 ("Nonlinearities"): ReLU, Sigmoid, Tanh, GELU
 * (z Phi(z) with the standard normal CDF Phi, not its tanh approximation).
 * Their derivatives: ReLU 1{z > 0}, Sigmoid s (1 - s), Tanh 1 - tanh^2,
 * GELU Phi(z) + z phi(z). Evaluated in fp32 with the device library's
 * expf / tanhf / erff.
 */
#define MT_ACT_NONE 0
#define MT_ACT_RELU 1
#define MT_ACT_SIGMOID 2
#define MT_ACT_TANH 3
#define MT_ACT_GELU 4

/* mt_linear_act_fwd: y = act(Z), Z = X W^T + 1 b^T (Eq. (5) followed by a
 * nonlinearity), fused into the product's epilogue: the biased accumulators
 * go through act in registers and Z is never re-read.
 *   x, w, b, y as for mt_linear_fwd; act: one of MT_ACT_*;
 *   z [M, N] f32 or NULL: receives the pre-activation Z (the pullback of
 *   act needs it; mt_act_bwd takes it). Any row pitch, inner dim contiguous.
 * Errors as mt_linear_fwd, plus MT_ERR_INVALID for an unknown act and
 * MT_ERR_ALIAS when z overlaps an input or y.
 */
mt_status mt_linear_act_fwd(const mt_tensor* x, const mt_tensor* w, const mt_tensor* b,
                            int32_t act, const mt_tensor* z, const mt_tensor* y, void* stream);

/* mt_act_bwd: the pullback of y = act(z) (chain rule, Sec. 3.2 Eq. (3)), with
 * the bias gradient of the dense layer before it folded into the same pass:
 *   dz = dy * act'(z)                      elementwise
 *   db = 1^T dz  (sum over rows)           the add pullback through the
 *                                          broadcast bias (Sec. 3.1, 3.2)
 *   z  [M, N] f32 (the saved pre-activation)
 *   dy [M, N] f32 or bf16; dz [M, N] the same dtype as dy (bf16: rounded to
 *   nearest even from the fp32 product); db [N] f32 or NULL, summed from the
 *   fp32 products before any rounding.
 * Matrices: any row pitch, inner dim contiguous. flags: MT_ACCUMULATE adds
 * into dz and db. ws: optional (mt_act_bwd_workspace), row-slice sums of db.
 * dz then feeds mt_linear_bwd as its dy, with db = NULL there.
 */
mt_status mt_act_bwd(int32_t act, const mt_tensor* z, const mt_tensor* dy, const mt_tensor* dz,
                     const mt_tensor* db, uint32_t flags, void* ws, size_t ws_bytes,
                     void* stream);
mt_status mt_act_bwd_workspace(int32_t act, const mt_tensor* z, const mt_tensor* dy,
                               const mt_tensor* dz, const mt_tensor* db, size_t* bytes);

/* ------------------------------------------------------------------ loss
 * mt_mse_loss: mean squared error (Sec. 3.3, "Losses") over all N elements
 * and its gradient:
 *   loss = (1/N) sum_i (pred_i - target_i)^2     (a 1-element f32 tensor, or NULL)
 *   dpred = 2 (pred - target) / N                 (pred's shape, or NULL)
 * pred, target, dpred: f32, contiguous, one shape. At least one output.
 * The sum runs in fp32 per block in a fixed order, then over blocks in
 * block order: deterministic. ws: optional (mt_mse_loss_workspace).
 */
mt_status mt_mse_loss(const mt_tensor* pred, const mt_tensor* target, const mt_tensor* loss,
                      const mt_tensor* dpred, void* ws, size_t ws_bytes, void* stream);
mt_status mt_mse_loss_workspace(const mt_tensor* pred, const mt_tensor* target, size_t* bytes);

/* ------------------------------------------------------------ optimizers
 * In-place parameter updates (Sec. 3.3, "Optimizers") for n parameter
 * tensors at once (arrays of n descriptors; element i of each array belongs
 * to parameter i). Every tensor is f32 and contiguous, and the tensors of
 * one parameter share its shape. Parameters and states are read and
 * overwritten; no updated tensor may overlap another tensor of the call.
 * Up to 32 tensors go into one kernel launch. Arithmetic is fp32.
 *
 * mt_sgd_step, Eq. (9):
 *   v <- momentum v + g + weight_decay theta;   theta <- theta - lr v
 */
mt_status mt_sgd_step(int32_t n, const mt_tensor* params, const mt_tensor* grads,
                      const mt_tensor* velocity, float lr, float momentum, float weight_decay,
                      void* stream);

/* mt_adam_step, Eq. (10), at step t = `step` (>= 1, counted by the caller):
 *   m <- b1 m + (1 - b1) g;  v <- b2 v + (1 - b2) g^2;
 *   theta <- theta - lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps)
 * The bias corrections 1 / (1 - b^t) are formed in double on the host.
 * Needs 0 <= b1, b2 < 1 and eps >= 0 (MT_ERR_INVALID otherwise).
 */
mt_status mt_adam_step(int32_t n, const mt_tensor* params, const mt_tensor* grads,
                       const mt_tensor* exp_avg, const mt_tensor* exp_avg_sq, float lr, float beta1,
                       float beta2, float eps, int64_t step, void* stream);

/* mt_rmsprop_step: an exponential average of squared gradients, the step
 * scaled by (v + eps)^(-1/2) as the paper states it (eps inside the root):
 *   v <- alpha v + (1 - alpha) g^2;   theta <- theta - lr g / sqrt(v + eps)
 */
mt_status mt_rmsprop_step(int32_t n, const mt_tensor* params, const mt_tensor* grads,
                          const mt_tensor* sq_avg, float lr, float alpha, float eps, void* stream);

/* ----------------------------------------------------------- convolution
 * 2-D convolution of Sec. 3.3 Eq. (6), batched, with stride (stride_h,
 * stride_w) and zero padding (pad_h, pad_w), 0-based indices:
 *   y[n][c][i][j] = sum_{c', u, v} w[c][c'][u][v] x[n][c'][i sh + u - ph][j sw + v - pw] + b[c]
 *   (x read as 0 outside the image), Ho = (H + 2 ph - KH) / sh + 1, likewise Wo.
 * Shapes are given in [N][C][H][W] order whatever the memory layout:
 *   x  [N, C, H, W]    f32, any strides (read through them)
 *   w  [CO, C, KH, KW] f32; the taps of one output channel contiguous, either
 *                      as [C][KH][KW] (the usual layout) or channels-last
 *                      [KH][KW][C]; any pitch between output channels
 *   b  [CO] f32 or NULL;  y [N, CO, Ho, Wo] f32 channels-last contiguous
 *                      (memory order N, Ho, Wo, CO)
 * The convolution runs as a product of the unfolded input U (a row per output
 * pixel, a column per tap) with the flattened weights on the matrix cores.
 * Where x is channels-last (c stride 1, the other strides multiples of 4, a
 * 16-byte aligned base), w is channels-last and C is a multiple of 32 (the
 * weight gradient: of 4), with y, w and b allowing 16-byte accesses, the
 * product's loads gather U's entries from x directly and U is never formed.
 * Otherwise U is unfolded into the caller's workspace, which is REQUIRED for
 * that path (MT_ERR_WORKSPACE without it; N Ho Wo x round_up(C KH KW, 4)
 * floats at its start). After U (or from the start) the workspace holds the
 * partial tiles of a split contraction or of the stream-K schedule (the
 * tile-major K-stages shared evenly by one block per CU, cut tiles summed by
 * a fixed-order pass) that products with a ragged last wave of tiles take;
 * those are optional: a shorter workspace runs one tile per block. Sizes
 * from the *_workspace calls. The backward's dx is one product
 * gathering dy where the convolution has stride 1, CO is a multiple of 32 and
 * dx is channels-last (16-byte aligned); with strides up to the window size
 * (KH >= sh, KW >= sw) it is one such product per sub-pixel phase of the
 * stride; otherwise it goes through dU = dY Wf in the workspace and a fold.
 * fp32 only.
 */
mt_status mt_conv2d_fwd(const mt_tensor* x, const mt_tensor* w, const mt_tensor* b,
                        const mt_tensor* y, int32_t stride_h, int32_t stride_w, int32_t pad_h,
                        int32_t pad_w, void* ws, size_t ws_bytes, void* stream);
mt_status mt_conv2d_fwd_workspace(const mt_tensor* x, const mt_tensor* w, const mt_tensor* b,
                                  const mt_tensor* y, int32_t stride_h, int32_t stride_w,
                                  int32_t pad_h, int32_t pad_w, size_t* bytes);

/* mt_conv2d_bwd: the pullbacks of Eq. (6) from dy (the matmul pullbacks of
 * Eq. (4) through the unfolded form, and the add pullback for b):
 *   dx[n][c'][h][x] = sum of dy[n][c][i][j] w[c][c'][u][v] over the (c, i, j, u, v)
 *                     with h = i sh + u - ph, x = j sw + v - pw   (NULL to skip)
 *   dw[c][c'][u][v] = sum over (n, i, j) of dy[n][c][i][j] x[n][c'][i sh + u - ph][j sw + v - pw]
 *   db[c]           = sum over (n, i, j) of dy[n][c][i][j]
 *   dy [N, CO, Ho, Wo] channels-last contiguous; dx [N, C, H, W] contiguous,
 *   channels-last or [N][C][H][W]; dw the shape of w with its taps in w's
 *   order; db [CO]. x and w are needed for their shapes (and x's data for
 *   dw, w's data for dx). flags: MT_ACCUMULATE, MT_CONV_REUSE_UNFOLD. The input gradient is a
 *   gather over the taps that read each element: no atomics, deterministic. With dw and db
 *   both requested, db is summed inside the dW product (the column sums of dY^T, its first
 *   operand); db alone runs a column-sum pass over dy.
 */
mt_status mt_conv2d_bwd(const mt_tensor* x, const mt_tensor* w, const mt_tensor* dy,
                        const mt_tensor* dx, const mt_tensor* dw, const mt_tensor* db,
                        int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                        uint32_t flags, void* ws, size_t ws_bytes, void* stream);
mt_status mt_conv2d_bwd_workspace(const mt_tensor* x, const mt_tensor* w, const mt_tensor* dy,
                                  const mt_tensor* dx, const mt_tensor* dw, const mt_tensor* db,
                                  int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                  size_t* bytes);

/* -------------------------------------------------------------- matmul
 * mt_matmul: C = A @ B with NumPy/PyTorch matmul semantics (Eq. (1) per
 * batch element, batch dims broadcast per Sec. 3.1):
 *   - a and b have rank >= 1; a 1-D a is treated as [1, K] and a 1-D b as
 *     [K, 1], the added dim being dropped from the result;
 *   - the batch dims (all but the last two) broadcast; a broadcast dim may
 *     have any stride (including 0);
 *   - the two matrix dims of each operand must have one of them contiguous:
 *     stride[-1] == 1 (row-major) or stride[-2] == 1 (a transposed view);
 *   - a and b share one dtype (f32 or bf16); c is f32, row-major contiguous,
 *     with exactly the result shape, or, with MT_REDUCE_INTO, that shape
 *     summed over some batch axes (leading axes dropped, kept axes of size
 *     1), i.e. the gradient of a broadcast operand.
 * flags: MT_ACCUMULATE, MT_REDUCE_INTO.
 * ws/ws_bytes: optional workspace (size from mt_matmul_workspace) for split-K
 * partial sums when the output tiles alone under-fill the GPU (e.g. a
 * gradient summed over broadcast axes, whose sum runs inside the product).
 */
mt_status mt_matmul(const mt_tensor* a, const mt_tensor* b, const mt_tensor* c, uint32_t flags,
                    void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes mt_matmul can use for these arguments (0 if none). */
mt_status mt_matmul_workspace(const mt_tensor* a, const mt_tensor* b, const mt_tensor* c,
                              uint32_t flags, size_t* bytes);

/* mt_reduce_broadcast_grad: the add pullback through a broadcast (Sec. 3.1,
 * Sec. 3.2): grad_in = grad_out summed over every axis along which an input
 * of grad_in's shape was broadcast to grad_out's shape. grad_in's shape,
 * left-padded with ones, must equal grad_out's shape except for dims of
 * size 1. grad_out: f32, any strides. grad_in: f32, row-major contiguous.
 * flags: MT_ACCUMULATE. ws: optional (mt_reduce_broadcast_grad_workspace).
 */
mt_status mt_reduce_broadcast_grad(const mt_tensor* grad_out, const mt_tensor* grad_in,
                                   uint32_t flags, void* ws, size_t ws_bytes, void* stream);

mt_status mt_reduce_broadcast_grad_workspace(const mt_tensor* grad_out, const mt_tensor* grad_in,
                                             size_t* bytes);

/* ------------------------------------------------------- workspace query
 * mt_workspace_bytes: the workspace size of one call, by operation, with the
 * same tensors the call takes (NULL where the call allows it), for callers
 * that size workspaces generically. It equals the matching *_workspace
 * entry point's answer. args, in order:
 *   MT_OP_MATMUL, MT_OP_MATMUL_REDUCE_INTO   {a, b, c}         (flags 0 / MT_REDUCE_INTO)
 *   MT_OP_LINEAR_FWD                         {x, w, b, y}      (always 0)
 *   MT_OP_LINEAR_BWD                         {x, w, dy, dx, dw, db}
 *   MT_OP_REDUCE_BROADCAST_GRAD              {grad_out, grad_in}
 *   MT_OP_MSE_LOSS                           {pred, target}
 * The nonlinearity pullback and the convolution take non-tensor arguments:
 * use mt_act_bwd_workspace / mt_conv2d_*_workspace. Returns SIZE_MAX for an
 * unknown op, a wrong count or invalid tensors (message in mt_last_error()).
 * Host-only.
 */
#define MT_OP_MATMUL 0
#define MT_OP_MATMUL_REDUCE_INTO 1
#define MT_OP_LINEAR_FWD 2
#define MT_OP_LINEAR_BWD 3
#define MT_OP_REDUCE_BROADCAST_GRAD 4
#define MT_OP_MSE_LOSS 5
size_t mt_workspace_bytes(int32_t op, const mt_tensor* const* args, int32_t nargs);

/* ------------------------------------------------- host-only shape helpers
 * No GPU needed; results are exact. Shapes are arrays of int64 sizes.
 * mt_broadcast_shape: the broadcast of two shapes (Sec. 3.1).
 * mt_matmul_shape:    the result shape of mt_matmul for operand shapes a, b.
 * *nout receives the rank, out[] (room for MT_MAX_DIMS) the sizes.
 */
mt_status mt_broadcast_shape(int32_t na, const int64_t* a, int32_t nb, const int64_t* b,
                             int32_t* nout, int64_t* out);
mt_status mt_matmul_shape(int32_t na, const int64_t* a, int32_t nb, const int64_t* b,
                          int32_t* nout, int64_t* out);

/* Testing and tuning knobs, for tests and measurements only: each setting
 * is process-wide and applies to every later call from any thread (the
 * values are atomics, so setting one while calls run is safe, but which of
 * those calls see it is unspecified; a production caller leaves them at
 * their defaults). Returns 0 = accepted, -1 = unknown key, -2 = value out of
 * range. Keys: "cfg" GEMM tile
 * configuration (-1 = automatic; register-staged tiles 0 = 256x256,
 * 1 = 256x128, 2 = 128x256, 3 = 128x128, 4 = 64x64, 5 = 256x256 with 8 waves;
 * tiles streamed straight into an LDS ring 6 = 256x256 with 8 waves,
 * 7 = 256x256 with 4 waves, 8 = 256x128, 9 = 128x256, 10 = 128x128,
 * 11 = 128x128 with 8 waves, 12 = 128x128 with 8 waves and 64-deep fp32
 * K-stages (bf16 maps it to 10), 13 = 256x192, 14 = 256x96 (K-contiguous B
 * only, else 8), 15 = 64x384 (13-15: fp32 operands without 16-byte aligned
 * rows only, else 8; bf16 10); fp32 operands that do not allow 16-byte loads
 * run on tiles 6, 8, 9, 10 and 13-15 with 4-byte lanes (11 and 12 map to 10),
 * else at 128x128 or 64x64; bf16 ones at 128x128 or 64x64); "vec1"
 * (1 = force the narrow-load kernels); "splits" (0..4096, split-K count for
 * mt_linear_bwd's dw, 0 = automatic); "parts" (0..4096, row slices of the db
 * and broadcast-gradient reductions, 0 = automatic); "krot" (1 = the default:
 * blocks of the 256x256 DMA tile start their K loop at a stage that depends
 * on their XCD and wrap around; 0 = every block starts at k = 0); "persist"
 * (1 = the default: plain products of whole 256x256 tiles, more tiles
 * than CUs, no accumulate, run on a grid of one block per CU that walks the
 * plain grid's tiles, bf16 dW with db's column sums included, fp32 dW never;
 * 0 = the plain grid; the two give identical bits);
 * convolution: "conv_gather" (1 = the default: products gather the image
 * where the layout allows; 0 = always unfold), "stream_k" (gathered 256x256
 * forward and input-gradient products: 0 never, 1 = the default: when the
 * last round of blocks would be ragged, 2 always), "sk_blocks" (0..65535
 * stream-K blocks, 0 = one per CU), "phase_grid" (strided input gradient:
 * 0 a launch per sub-pixel phase, 1 = the default: one grid when large,
 * 2 always one grid). Results stay within the documented accuracy for
 * every setting. */
int mt_debug_set(const char* key, int64_t value);

/* Static description of a status code. */
const char* mt_status_str(mt_status s);
/* Message describing this thread's last failed call ("" if none). */
const char* mt_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MINITENSOR_HIP_H */
