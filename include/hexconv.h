/*
 * hexconv.h -- C ABI of libhexconv: hexagonal convolution and pooling on
 * MI355X (gfx950).
 *
 * The operations are those of HexagDLy (Steppa & Holch, arXiv:1903.01814,
 * Sec. 2), computed directly by HIP kernels:
 *
 *  Addressing (Sec. 2.1, Fig. 1): hexagonally sampled data in a rectangular
 *  tensor whose columns are columns of vertically adjacent pixels, every
 *  second column shifted by half a pitch so that rows line up.  Rows count
 *  top to bottom, columns left to right.  Convention fixed here: the odd
 *  columns (1, 3, ...) are the ones lying half a pitch lower in the
 *  hexagonal array.  Blank tensor cells hold whatever the caller put there
 *  and are computed on like any other value.
 *
 *  Kernel of size k (Sec. 2.2): the centre pixel plus k layers of neighbours,
 *  T = 1 + 3k(k+1) taps.  Taps are numbered column by column (column offset
 *  -k .. k), each column top to bottom; a weight belongs to one physical
 *  direction, the same for both column parities.  hex_tap_table gives the
 *  (column, row) offsets per centre-column parity.
 *
 *  Padding and stride (Sec. 2.3, Fig. 4): kernels are centred on tensor
 *  elements only and taps outside the tensor read zero.  A stride s takes
 *  equal steps of s pitches along the three lattice axes from the top-left
 *  element: output (i, j) is centred on input row s*i + (j odd ? s/2 : 0)
 *  (integer division), column s*j.  The output uses the same addressing.
 *  W_out = (W-1)/s + 1; all output columns get the length of the shortest
 *  one (H_out from hex_out_shape).
 *
 *  Pooling (Sec. 2.4): the same windows, padding and stride with a max or an
 *  average.  Conventions fixed here: padded taps count as zeros in both; the
 *  average divides by T; the max keeps the first maximal tap in tap order.
 *
 * Conventions for every entry point:
 *  - H and W are always the INPUT sizes; output sizes come from
 *    hex_out_shape.
 *  - Tensors are dense NCHW device pointers: x[N][C_in][H][W],
 *    y[N][C_out][H_out][W_out], w[C_out][C_in][T] (same dtype as x), bias
 *    [C_out] (dtype of x).  Pointers must be 16-byte aligned.  dw and db are
 *    float32 whatever the input dtype.
 *  - The caller owns and allocates every buffer, including workspaces.  The
 *    library never allocates, frees or synchronises; it only enqueues
 *    kernels on `stream` (a hipStream_t; NULL = the default stream).
 *  - Outputs are fully overwritten, never accumulated into.
 *  - Arguments are validated on the host before anything is enqueued; a
 *    rejected call returns a negative hex_status and enqueues nothing.
 *  - N = 0 is a valid empty batch and batch-shaped buffers may then be NULL:
 *    forward, backward-data and pooling calls return HEX_OK and enqueue
 *    nothing; hexconv_bwd_weight writes zeros to dw (and db).  When the
 *    input is too small for any output (H_out = 0), forward calls write
 *    nothing and gradient calls write zeros.
 *  - bf16 paths read bf16, accumulate in float32 and round outputs to
 *    nearest-even.  The ReLU flag applies max(0, .) before rounding.
 *  - No function throws; all are safe to call from C.
 */
#ifndef HEXCONV_H
#define HEXCONV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    HEX_OK = 0,
    HEX_ERR_INVALID_ARG = -1, /* null pointer, bad size, k, stride, dtype */
    HEX_ERR_UNSUPPORTED = -2, /* valid request the library does not implement */
    HEX_ERR_LAUNCH = -3       /* a kernel launch reported an error */
} hex_status;

typedef enum { HEX_F32 = 0, HEX_BF16 = 1 } hex_dtype;

typedef enum { HEX_POOL_MAX = 0, HEX_POOL_AVG = 1 } hex_pool_mode;

enum { HEX_FLAG_RELU = 1 };

#define HEX_MAX_K 8      /* largest kernel size accepted */
#define HEX_MAX_STRIDE 8 /* largest stride accepted (in the plane and along z) */
#define HEX_MAX_KZ 4     /* largest half-depth of a 3-D window (2*4+1 planes) */

/* Number of taps of a size-k kernel, 1 + 3k(k+1) (Sec. 2.2); negative
 * hex_status for k outside [0, HEX_MAX_K]. */
int hex_num_taps(int k);

/* Output size of an H x W input under a size-k kernel and stride s
 * (Sec. 2.3).  Every window is centred on a tensor element and padding
 * supplies the taps that fall outside, so the size depends on the stride
 * only: k is validated (0 .. HEX_MAX_K) and otherwise does not change the
 * result.  H_out may be 0 when H is too small for the odd output columns.
 * H_out and W_out are host pointers.  Returns a hex_status. */
int hex_out_shape(int H, int W, int k, int stride, int *H_out, int *W_out);

/* Tap offsets of a size-k kernel for a centre element in a column of the
 * given parity (0 even, 1 odd): tap t reads element (r + drow[t],
 * c + dcol[t]).  dcol and drow are host arrays of hex_num_taps(k) ints.
 * Returns a hex_status. */
int hex_tap_table(int k, int parity, int *dcol, int *drow);

/*
 * Forward convolution (Sec. 2.3):
 *   y[n][co][i][j] = bias[co] + sum_ci sum_t w[co][ci][t] * x[n][ci][p_t]
 * where p_t is tap t of the window centred on output (i, j), and x reads 0
 * outside the tensor.  bias may be NULL.  flags: HEX_FLAG_RELU.
 */
int hexconv_fwd(const void *x, const void *w, const void *bias, void *y,
                int N, int C_in, int C_out, int H, int W, int k, int stride,
                hex_dtype dt, int flags, void *stream);

/*
 * Gradient of the forward map with respect to x (adjoint of hexconv_fwd
 * without bias).  The paper's layers are meant to sit inside CNN models
 * that are trained by gradient descent (Sec. 2.4, and the networks trained
 * in Sec. 4); this is the data half of that backward pass:
 *   dx[n][ci][p] = sum over (co, i, j, t) with p_t(i, j) = p of
 *                  w[co][ci][t] * dy[n][co][i][j].
 * dy is [N][C_out][H_out][W_out]; dx is [N][C_in][H][W] in dtype dt.
 */
int hexconv_bwd_data(const void *dy, const void *w, void *dx, int N, int C_in,
                     int C_out, int H, int W, int k, int stride, hex_dtype dt,
                     void *stream);

/* Bytes of device workspace hexconv_bwd_weight needs for these sizes
 * (0 for invalid arguments). */
size_t hexconv_bwd_weight_workspace(int N, int C_in, int C_out, int H, int W,
                                    int k, int stride, hex_dtype dt);

/*
 * Gradient with respect to the weights and bias, the parameter half of the
 * backward pass of a hexagonal convolution layer trained inside a CNN
 * (Sec. 2.4; the trained networks of Sec. 4):
 *   dw[co][ci][t] = sum_n sum_(i,j) dy[n][co][i][j] * x[n][ci][p_t(i, j)]
 *   db[co]        = sum_n sum_(i,j) dy[n][co][i][j]          (db nullable)
 * dw and db are float32 device buffers.  ws is a device workspace of at
 * least hexconv_bwd_weight_workspace(...) bytes (may be NULL when that is
 * 0).  The reduction order is fixed, so results are deterministic.
 */
int hexconv_bwd_weight(const void *x, const void *dy, float *dw, float *db,
                       void *ws, size_t ws_bytes, int N, int C_in, int C_out,
                       int H, int W, int k, int stride, hex_dtype dt,
                       void *stream);

/* Bytes of device workspace hexconv_bwd needs for these sizes (0 for
 * invalid arguments). */
size_t hexconv_bwd_workspace(int N, int C_in, int C_out, int H, int W, int k,
                             int stride, hex_dtype dt);

/*
 * Both gradients of one convolution layer in one call (Sec. 2.4: the
 * backward pass of a hexagonal layer): the results of hexconv_bwd_data
 * (written to dx) and of hexconv_bwd_weight (dw, db), for the same
 * arguments.  dx may be NULL (first layer: no data gradient); w may then be
 * NULL too.  db is nullable.  ws: at least hexconv_bwd_workspace(...) bytes.
 * Where a fused kernel exists for the shape (float32 or bfloat16, one or
 * two input channels, at most 32 output channels, stride 1) dy is read from
 * memory once for both results; otherwise the two gradients are computed one
 * after the other.  Every argument is checked
 * before anything is enqueued.  Deterministic, like hexconv_bwd_weight.
 */
int hexconv_bwd(const void *x, const void *dy, const void *w, void *dx,
                float *dw, float *db, void *ws, size_t ws_bytes, int N,
                int C_in, int C_out, int H, int W, int k, int stride,
                hex_dtype dt, void *stream);

/*
 * hexconv_bwd without a workspace argument, for callers that cannot
 * allocate device memory: code being captured into a HIP graph, tight
 * serving loops, harnesses that forbid allocation.  Same arguments,
 * results and checks as hexconv_bwd (results bit-identical to it), minus
 * ws and ws_bytes: the workspace lives in a static device array of the
 * library, HEX_NOALLOC_SCRATCH_BYTES bytes per GPU, which each GPU the
 * library runs on holds until the process ends.  A shape whose workspace
 * (hexconv_bwd_workspace) exceeds that size is rejected with
 * HEX_ERR_UNSUPPORTED before anything is enqueued.  The call allocates and
 * frees nothing.  Every call on one GPU shares that GPU's array, so calls
 * that overlap on one GPU (on different streams, or from several threads)
 * race and must be serialised by the caller; calls on one stream are
 * ordered and safe.  HEX_ERR_LAUNCH if the array's device address cannot be
 * obtained.
 */
#define HEX_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int hexconv_bwd_noalloc(const void *x, const void *dy, const void *w, void *dx, float *dw,
                        float *db, int N, int C_in, int C_out, int H, int W, int k,
                        int stride, hex_dtype dt, void *stream);

/*
 * Pooling (Sec. 2.4) over the windows of hexconv_fwd, per channel:
 *   max: y = value of the first maximal tap (padding counts as 0);
 *   avg: y = (sum of the T tap values, padding 0) / T.
 * argmax_tap (nullable, uint8 [N][C][H_out][W_out]) receives the winning
 * tap index for HEX_POOL_MAX; it is not written for HEX_POOL_AVG.
 */
int hexpool_fwd(const void *x, void *y, uint8_t *argmax_tap, int N, int C,
                int H, int W, int k, int stride, hex_pool_mode mode,
                hex_dtype dt, void *stream);

/*
 * Pooling gradient, the backward pass of the pooling layer of Sec. 2.4 as
 * used in the trained networks of Sec. 4: max routes dy[o] to the element
 * its argmax tap points at (dropped when that tap is padding; argmax_tap required); avg shares
 * dy[o] / T over the in-tensor taps.  When relu_y is not NULL (the ReLU
 * output that fed the pool, [N][C][H][W], dtype dt) the result is
 * multiplied by [relu_y > 0].  dx is [N][C][H][W].
 */
int hexpool_bwd(const void *dy, const uint8_t *argmax_tap, const void *relu_y,
                void *dx, int N, int C, int H, int W, int k, int stride,
                hex_pool_mode mode, hex_dtype dt, void *stream);

/*
 * Three-dimensional operations (Sec. 2.4: hexagonal layout in the x-y plane,
 * equidistant samples along z, e.g. the time slices of a hexagonal camera).
 * Conventions fixed here (the paper gives no further detail):
 *  - tensors are dense NCDHW: x[N][C_in][D][H][W], D planes along z, each
 *    an H x W plane in the addressing above;
 *  - a window of size (k, kz) is the size-k hexagon in the plane times the
 *    2kz+1 planes dz = -kz .. kz around the centre plane (0 <= kz <=
 *    HEX_MAX_KZ); taps are numbered dz-major (dz ascending), the hexagonal
 *    taps in hex_tap_table order inside; w[C_out][C_in][2kz+1][T];
 *  - padding and stride follow the 2-D rule along z too: windows are
 *    centred on real planes only, planes outside the tensor read zero, and
 *    output plane l is centred on input plane stride_z * l, so
 *    D_out = (D - 1) / stride_z + 1 (1 <= stride_z <= HEX_MAX_STRIDE);
 *  - pooling takes the maximum or the average over the (2kz+1) * T taps,
 *    padded taps counting as zeros; the average divides by (2kz+1) * T; the
 *    maximum keeps the first maximal tap, whose index (dz + kz) * T + t is
 *    written to a uint16 argmax.
 * Every other convention (ownership, alignment, asynchrony, validation,
 * empty batches, bf16 rounding, fp32 weight gradients, the ReLU flag) is
 * that of the 2-D entry points.  H, W and D are input sizes.
 */

/* Output size of a D x H x W input (Sec. 2.3 in the plane, the same rule
 * along z): D_out = (D - 1) / stride_z + 1; H_out, W_out as
 * hex_out_shape.  Host pointers.  Returns a hex_status. */
int hex_out_shape3d(int D, int H, int W, int k, int kz, int stride, int stride_z, int *D_out,
                    int *H_out, int *W_out);

/*
 * 3-D forward convolution (Sec. 2.4):
 *   y[n][co][l][i][j] = bias[co] + sum_ci sum_dz sum_t
 *       w[co][ci][dz+kz][t] * x[n][ci][stride_z*l + dz][p_t(i, j)]
 * x reads 0 outside the tensor.  y is [N][C_out][D_out][H_out][W_out].
 * bias may be NULL; flags: HEX_FLAG_RELU.
 */
int hexconv3d_fwd(const void *x, const void *w, const void *bias, void *y, int N, int C_in,
                  int C_out, int D, int H, int W, int k, int kz, int stride, int stride_z,
                  hex_dtype dt, int flags, void *stream);

/* Gradient of hexconv3d_fwd with respect to x (its adjoint without bias;
 * the data half of the backward pass of a 3-D layer inside a trained CNN,
 * Sec. 2.4).  dy is [N][C_out][D_out][H_out][W_out], dx [N][C_in][D][H][W]. */
int hexconv3d_bwd_data(const void *dy, const void *w, void *dx, int N, int C_in, int C_out, int D,
                       int H, int W, int k, int kz, int stride, int stride_z, hex_dtype dt,
                       void *stream);

/* Bytes of device workspace hexconv3d_bwd_weight needs (0 for invalid
 * arguments). */
size_t hexconv3d_bwd_weight_workspace(int N, int C_in, int C_out, int D, int H, int W, int k,
                                      int kz, int stride, int stride_z, hex_dtype dt);

/* Gradient with respect to the weights and bias (Sec. 2.4, the parameter
 * half of a 3-D layer's backward pass):
 *   dw[co][ci][dz+kz][t] = sum over (n, l, i, j) of
 *       dy[n][co][l][i][j] * x[n][ci][stride_z*l + dz][p_t(i, j)]
 *   db[co] = sum of dy[n][co] (nullable)
 * float32 dw [C_out][C_in][2kz+1][T] and db; deterministic; ws as for
 * hexconv_bwd_weight. */
int hexconv3d_bwd_weight(const void *x, const void *dy, float *dw, float *db, void *ws,
                         size_t ws_bytes, int N, int C_in, int C_out, int D, int H, int W, int k,
                         int kz, int stride, int stride_z, hex_dtype dt, void *stream);

/* 3-D pooling (Sec. 2.4: pooling built like the convolutions, same
 * padding and striding) per channel over the (k, kz) windows: max or
 * average as stated above.  argmax (nullable, uint16
 * [N][C][D_out][H_out][W_out]) receives (dz + kz) * T + t of the winning
 * tap for HEX_POOL_MAX. */
int hexpool3d_fwd(const void *x, void *y, uint16_t *argmax, int N, int C, int D, int H, int W,
                  int k, int kz, int stride, int stride_z, hex_pool_mode mode, hex_dtype dt,
                  void *stream);

/* Gradient of hexpool3d_fwd: max routes dy to the element of its argmax tap
 * (dropped when that tap is padding; argmax required), average shares dy /
 * ((2kz+1) T) over the in-tensor taps; times [relu_y > 0] when relu_y
 * ([N][C][D][H][W]) is given.  dx is [N][C][D][H][W]. */
int hexpool3d_bwd(const void *dy, const uint16_t *argmax, const void *relu_y, void *dx, int N,
                  int C, int D, int H, int W, int k, int kz, int stride, int stride_z,
                  hex_pool_mode mode, hex_dtype dt, void *stream);

/* Static description of a hex_status value. */
const char *hex_status_string(int status);

/* For diagnosis: the HIP runtime's description of the error behind the last
 * HEX_ERR_LAUNCH returned on the calling thread ("" if there was none).
 * Static string, never NULL. */
const char *hex_last_launch_error(void);

/*
 * Kernel timing, for profiling (not part of the paper's operations).
 * Between hexconv_timing_begin() and hexconv_timing_end(), every kernel the
 * library launches carries a pair of HIP events that the runtime records at
 * the start and at the end of that kernel's own execution, on the stream it
 * is launched on (so the dispatch is not counted).  hexconv_timing_end()
 * stops recording, waits
 * for the recorded events and reports, per kernel (by the kernel's function
 * name, template arguments dropped, in order of first launch), the number
 * of launches and their summed GPU time in milliseconds.
 *   names:    caller-owned, max_kernels * HEX_TIMING_NAME_LEN chars; entry i
 *             at names + i * HEX_TIMING_NAME_LEN, NUL-terminated
 *   counts, total_ms: caller-owned arrays of max_kernels
 *   n_kernels: receives the number of entries filled (at most max_kernels;
 *             further kernels are dropped)
 * Recording allocates events on the host side of every launch: do not
 * enable it while a HIP graph is being captured, nor from several threads
 * at once.  Returns HEX_ERR_INVALID_ARG for NULL outputs or max_kernels < 1,
 * HEX_ERR_LAUNCH if an event could not be waited for.
 */
#define HEX_TIMING_NAME_LEN 64
int hexconv_timing_begin(void);
int hexconv_timing_end(int max_kernels, char *names, int *counts, double *total_ms,
                       int *n_kernels);

#ifdef __cplusplus
}
#endif

#endif /* HEXCONV_H */
