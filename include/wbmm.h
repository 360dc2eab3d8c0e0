/*
 * wbmm.h — C ABI of the MI355X (gfx950) WBMM library.
 *
 * Windowed Batch Matrix Multiplication (WBMM), from "WBMM: Windowed Batch
 * Matrix Multiplication for Efficient Large Receptive Field Convolution":
 * the input X[B,C,H,W] is cut into non-overlapping w x w windows; each window,
 * flattened row-major to a d = w*w vector, is multiplied by a per-channel
 * d x d matrix M_c built from a relative-position table T[C,(2w-1)^2]
 * (Sec. 3.4 and Alg. 1; eq. index_computation; eq. index_select):
 *
 *   I[i, j] = (h_i - h_j + w - 1) * (2w - 1) + (w_i - w_j + w - 1)
 *   M_c[i, j] = T[c, I[i, j]]
 *   Y_window = X_window * M_c        (row vector times matrix, Theorem 3.2:
 *                                     i = input position, j = output position)
 *
 * M_c is never stored in memory: the kernels build its blocks on the fly from
 * T in on-chip memory (the tiled scheme the paper names as future work in its
 * Limitations section).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All tensor pointers are DEVICE pointers, owned by the caller, dense and
 *   contiguous.  x, y, dy, dx are NCHW in `dtype`.  table is [C, (2w-1)^2] in
 *   `dtype`, row-major over (dh, dw) = input - output offsets.
 * - dtable is always float32 [C, (2w-1)^2] and is OVERWRITTEN (not
 *   accumulated into), whatever `dtype` is.
 * - H and W need not be multiples of w: the map is zero-padded at the bottom
 *   and right up to window multiples and the outputs are cropped back to
 *   H x W (Sec. 3.4.1, "Handling Arbitrary Input Sizes").
 * - 16-bit inputs are multiplied on the matrix cores with float32
 *   accumulation; every output element is rounded once (nearest-even) from
 *   its float32 sum.  float32 inputs use float32 matrix-core products.
 * - Work is enqueued on `stream` (a hipStream_t passed as void*, NULL = the
 *   default stream).  Calls are asynchronous: nothing is synchronised, and the
 *   caller must keep every buffer alive until the stream has passed the work.
 * - The library keeps no state and allocates no memory; calls are
 *   thread-safe.  Every argument is validated on the host before any GPU work
 *   is enqueued; errors are returned, never printed, never fatal.
 * - Supported window sizes: 1 <= w <= 16.  w = 7 and w = 14 are the sizes the
 *   paper uses; the others run the same kernels.
 * - Pointers must be aligned to their element size.  Outputs must not
 *   overlap inputs (WBMM_ERR_INVALID_ARG).
 */
#ifndef WBMM_H
#define WBMM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  WBMM_F32 = 0,  /* float32 storage and float32 products          */
  WBMM_BF16 = 1, /* bfloat16 storage, float32 accumulation        */
  WBMM_F16 = 2   /* IEEE half storage, float32 accumulation       */
} wbmm_dtype;

typedef enum {
  WBMM_OK = 0,
  WBMM_ERR_INVALID_ARG = 1, /* null pointer, non-positive size, overlap,
                               misalignment, too-small workspace, overflow */
  WBMM_ERR_UNSUPPORTED = 2, /* window size or dtype without a kernel       */
  WBMM_ERR_HIP = 3,         /* the HIP runtime refused the launch          */
  WBMM_ERR_SCRATCH = 4      /* wbmm_backward_noalloc: the shape needs more
                               scratch than the library's static buffer   */
} wbmm_status;

/* Forward pass, Alg. 1: y = WBMM(x; table, w).
 * x, y: [B,C,H,W] in dtype; table: [C,(2w-1)^2] in dtype. */
wbmm_status wbmm_forward(const void *x, const void *table, void *y,
                         int64_t B, int64_t C, int64_t H, int64_t W, int w,
                         wbmm_dtype dtype, void *stream);

/* Gradient with respect to the input for upstream gradient dy: per window,
 * dx = dy * M_c^T.  The paper does not write the backward pass out; this is
 * the chain rule applied to the per-window product Y_b = X_b M of Alg. 1 and
 * Theorem 3.2 (row-vector convention, i = input, j = output), with padded
 * positions (Sec. "Handling Arbitrary Input Sizes") receiving nothing.
 * Because I[j,i] = (2w-1)^2 - 1 - I[i,j] (eq. index_computation), M_c^T is
 * the matrix of the reversed table, so this runs the forward kernels with the
 * table read back to front.  dy, dx: [B,C,H,W] in dtype. */
wbmm_status wbmm_backward_input(const void *dy, const void *table, void *dx,
                                int64_t B, int64_t C, int64_t H, int64_t W,
                                int w, wbmm_dtype dtype, void *stream);

/* Size in bytes of the device workspace wbmm_backward_table needs for this
 * shape (0 when none is needed).  Returns 0 for invalid arguments as well;
 * wbmm_backward_table reports those. */
size_t wbmm_backward_table_workspace_bytes(int64_t B, int64_t C, int64_t H,
                                           int64_t W, int w,
                                           wbmm_dtype dtype);

/* Gradient with respect to the table:
 *   dtable[c, k] = sum over images, windows and (input i, output j) pairs with
 *                  I[i, j] = k of x[.., i] * dy[.., j]
 * i.e. the per-window products X^T dY scattered back onto the table through
 * the index of eq. index_select (M_c = T[c, I]).  The paper states that
 * during training the gradients flow through the table and M is rebuilt on
 * every forward pass (Sec. "Inference Caching Mechanism"); the formula is the
 * chain rule on Alg. 1 and Theorem 3.2.  x, dy: [B,C,H,W] in dtype; dtable:
 * float32 [C,(2w-1)^2], overwritten.
 *
 * workspace: device buffer of at least wbmm_backward_table_workspace_bytes()
 * bytes (may be NULL when that is 0), 4-byte aligned.  When a channel's
 * windows are split into several slabs, each slab writes its partial table
 * gradient there ([slabs, C, (2w-1)^2] float32) and a second kernel, enqueued
 * on the same stream, sums the partials into dtable.  The workspace may hold
 * anything on entry and is left holding partial sums; calls that can run
 * concurrently must not share one.
 *
 * The reduction has a fixed order (slab partials are summed in slab order):
 * the result is bitwise reproducible for a given shape. */
wbmm_status wbmm_backward_table(const void *x, const void *dy, float *dtable,
                                void *workspace, size_t workspace_bytes,
                                int64_t B, int64_t C, int64_t H, int64_t W,
                                int w, wbmm_dtype dtype, void *stream);

/* Size in bytes of the device workspace wbmm_backward needs for this shape;
 * equal to wbmm_backward_table_workspace_bytes() (same use and rules). */
size_t wbmm_backward_workspace_bytes(int64_t B, int64_t C, int64_t H, int64_t W,
                                     int w, wbmm_dtype dtype);

/* Both gradients in one pass (the input gradient of wbmm_backward_input and
 * the table gradient of wbmm_backward_table, the chain rule on Alg. 1 and
 * Theorem 3.2 for the training mode of Sec. "Inference Caching Mechanism",
 * where gradients flow through the table): every window of x and dy is
 * read once.  Results equal those of the two separate calls bit for bit.
 * x, dy, dx: [B,C,H,W] in dtype; table: [C,(2w-1)^2] in dtype; dtable: float32
 * [C,(2w-1)^2], overwritten.  dx and dtable must not overlap any input, each
 * other or the workspace.  workspace / workspace_bytes: as for
 * wbmm_backward_table (any contents on entry; no concurrent sharing). */
wbmm_status wbmm_backward(const void *x, const void *dy, const void *table,
                          void *dx, float *dtable, void *workspace,
                          size_t workspace_bytes, int64_t B, int64_t C,
                          int64_t H, int64_t W, int w, wbmm_dtype dtype,
                          void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the fused
 * backward of wbmm_backward (the same kernels, the same results bit for bit)
 * with its table-gradient scratch -- the per-slab partial sums that
 * wbmm_backward keeps in the caller's workspace -- held in a static device
 * buffer of this library instead.  No workspace argument;
 * x, dy, table, dx, dtable and every other argument as for wbmm_backward.
 *
 * - The buffer holds WBMM_NOALLOC_SCRATCH_BYTES (4 MiB) per device; each
 *   device the library runs on keeps its own copy until the process ends.
 *   A shape whose scratch would exceed it (wbmm_backward_workspace_bytes()
 *   greater than that) is rejected with WBMM_ERR_SCRATCH before any GPU
 *   work is enqueued.
 * - The call allocates nothing: no hipMalloc, no hipFree, no allocating
 *   library routine.  The first call on a device looks up the buffer's device
 *   address (hipGetSymbolAddress, with that device current) and keeps it.
 * - A call writes the partial sums before it reads them, so nothing carries
 *   over between calls and the buffer is never cleared.
 * - All calls on one device share that device's buffer: calls that overlap
 *   in time on one GPU (on different streams, or from different threads
 *   without ordering) race and give wrong results.  Serialise them. */
#define WBMM_NOALLOC_SCRATCH_BYTES ((size_t)4 << 20)
wbmm_status wbmm_backward_noalloc(const void *x, const void *dy,
                                  const void *table, void *dx, float *dtable,
                                  int64_t B, int64_t C, int64_t H, int64_t W,
                                  int w, wbmm_dtype dtype, void *stream);

/* ---- Hierarchical (global + local) form (Sec. "Hierarchical Window
 * Reparameterization" and the appendix algorithms of its training and
 * inference modes).  Global windows of w_g = 2 wl, each split into 2 x 2
 * local sub-windows of wl x wl; two tables: table_g [C,(2 w_g - 1)^2] and
 * table_l [C,(2 wl - 1)^2], in dtype.  Per global window
 *   y = x M_fused,  M_fused = M_g + diag_blocks(M_l, M_l, M_l, M_l) + 2 I,
 * which equals the training form x M_g + x + x_sub M_l + x_sub.  The fused
 * matrix is never built: the kernel adds the local blocks and the identity
 * as extra matrix-core products of the w_g kernel.  1 <= wl <= 8.
 * Same conventions as above (device pointers, NCHW, zero padding at the
 * bottom/right to multiples of w_g, outputs cropped). */
wbmm_status wbmm_hier_forward(const void *x, const void *table_g,
                              const void *table_l, void *y, int64_t B,
                              int64_t C, int64_t H, int64_t W, int wl,
                              wbmm_dtype dtype, void *stream);

/* dx = dy M_fused^T (both tables read back to front). */
wbmm_status wbmm_hier_backward_input(const void *dy, const void *table_g,
                                     const void *table_l, void *dx, int64_t B,
                                     int64_t C, int64_t H, int64_t W, int wl,
                                     wbmm_dtype dtype, void *stream);

/* Workspace for wbmm_hier_backward: enough for the two table gradients run
 * one after the other and for both computed in one pass (both tables' slab
 * partials); same rules as for wbmm_backward_table (any contents on entry,
 * no concurrent sharing). */
size_t wbmm_hier_backward_workspace_bytes(int64_t B, int64_t C, int64_t H,
                                          int64_t W, int wl, wbmm_dtype dtype);

/* All gradients of the hierarchical form: dx as wbmm_hier_backward_input
 * (bit for bit); dtable_g = the table gradient with windows 2 wl, dtable_l =
 * the table gradient with windows wl (the local sub-windows of the padded
 * global windows are the wl windows of the map); both float32, overwritten.
 * One launch on `stream` where the channel-stream pass applies (2 wl >= 10;
 * H and W multiples of 2 wl, a power of two of at most 16 windows per map
 * row, windows per image a multiple or a divisor of 16; 4-byte aligned
 * tensors; C at most the device's compute units); otherwise the input
 * gradient, then the two table gradients in one launch or two.  Outputs must not overlap inputs, each
 * other or the workspace. */
wbmm_status wbmm_hier_backward(const void *x, const void *dy,
                               const void *table_g, const void *table_l,
                               void *dx, float *dtable_g, float *dtable_l,
                               void *workspace, size_t workspace_bytes,
                               int64_t B, int64_t C, int64_t H, int64_t W,
                               int wl, wbmm_dtype dtype, void *stream);

/* ---- Cached-matrix (dense) form, for any window w_h x w_w with
 * 1 <= w_h, w_w <= 16 (Alg. 1 with the matrix built once, eq. index_select;
 * the paper's cached variant).  Positions inside a window are row-major,
 * p = h * w_w + x, d = w_h * w_w.  M is [C, d, d] in dtype, M[c][i][j] with
 * i the input and j the output position; any matrix may be given (it need
 * not come from a table), so rectangular windows, fused matrices and cached
 * matrices share these calls.  Same tensor conventions as above. */

/* m[c][i][j] = table[c][I(i, j)], table [C,(2 w_h - 1)(2 w_w - 1)] with
 * I = (h_i - h_j + w_h - 1)(2 w_w - 1) + (x_i - x_j + w_w - 1). */
wbmm_status wbmm_build_matrix(const void *table, void *m, int64_t C, int wh,
                              int ww, wbmm_dtype dtype, void *stream);

/* y_window = x_window * m[c] per w_h x w_w window. */
wbmm_status wbmm_dense_forward(const void *x, const void *m, void *y,
                               int64_t B, int64_t C, int64_t H, int64_t W,
                               int wh, int ww, wbmm_dtype dtype, void *stream);

/* dx_window = dy_window * m[c]^T. */
wbmm_status wbmm_dense_backward_input(const void *dy, const void *m, void *dx,
                                      int64_t B, int64_t C, int64_t H,
                                      int64_t W, int wh, int ww,
                                      wbmm_dtype dtype, void *stream);

/* dm[c] = sum over images and windows of x_window^T dy_window: float32
 * [C, d, d], overwritten. */
wbmm_status wbmm_dense_backward_matrix(const void *x, const void *dy, float *dm,
                                       int64_t B, int64_t C, int64_t H,
                                       int64_t W, int wh, int ww,
                                       wbmm_dtype dtype, void *stream);

/* dtable[c][k] = sum of dm[c][i][j] over the pairs with I(i, j) = k (the
 * adjoint of wbmm_build_matrix), in a fixed order; float32, overwritten. */
wbmm_status wbmm_bin_matrix(const float *dm, float *dtable, int64_t C, int wh,
                            int ww, void *stream);

/* Static description of a status code (never NULL). */
const char *wbmm_status_string(wbmm_status s);

/* Host-only: writes the d*d int32 relative position index I[i][j]
 * (eq. index_computation) that the kernels evaluate arithmetically, row-major,
 * d = w*w, into caller-owned host memory.  No GPU work. */
wbmm_status wbmm_relative_index(int w, int32_t *out_host);

/* Library version, e.g. "0.1.0". */
const char *wbmm_version(void);

#ifdef __cplusplus
}
#endif

#endif /* WBMM_H */
