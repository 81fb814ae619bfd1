/*
 * hexoracle.c -- fp64 CPU reference for hexagonal convolution and pooling.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow definition that the GPU
 * library is checked against.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it; the product path never does.  It
 * shares no code, header or table with the GPU library.
 *
 * Everything follows the definitions in HexagDLy (Steppa & Holch,
 * arXiv:1903.01814), Sec. 2:
 *
 *  Addressing (Sec. 2.1, Fig. 1).  A hexagonal array is rotated until
 *  neighbouring pixels line up vertically, so the pixels fall into columns;
 *  every second column is then moved up by half a pixel pitch so that all
 *  columns share one set of rows.  Tensor element (r, c) counts rows top to
 *  bottom and columns left to right.  Reading adopted (the figure is not
 *  available): the odd columns c = 1, 3, ... are the ones that sit half a pitch
 *  lower in the hexagonal array ("odd-q").  Axial coordinates of element
 *  (r, c) are q = c, s = r - floor(c/2); two pixels are neighbours iff their
 *  axial difference is one of (+-1,0), (0,+-1), (1,-1), (-1,1), and the number
 *  of neighbour steps between them is max(|dq|, |ds|, |dq+ds|).
 *
 *  Kernel of size k (Sec. 2.2).  The centre pixel plus k layers of
 *  neighbours: every axial offset (dq, ds) with hex distance <= k.  Taps are
 *  numbered in canonical order: dq ascending, then ds ascending.  Weight
 *  layout w[C_out][C_in][T].
 *
 *  Padding (Sec. 2.3).  A kernel is only ever centred on a real tensor
 *  element; taps falling outside the tensor read zero.
 *
 *  Stride (Sec. 2.3, Fig. 4).  Steps of equal length s along the three
 *  lattice axes, starting at the top-left element: the kernel centres are the
 *  axial points s*(Q, S).  The output is again stored in the same addressing,
 *  so output element (i, j) has axial (Q, S) = (j, i - floor(j/2)) and its
 *  centre sits at input axial (s*Q, s*S).  Output column j exists while its
 *  centre column s*j < W; all output columns get the length of the shortest
 *  one (steps that would make columns of unequal length are dropped).
 *
 *  Pooling (Sec. 2.4).  Same windows, padding and stride; max or average over
 *  the T taps of the window.  Readings adopted: padded taps take part as
 *  zeros in both the max and the average, the average divides by T, and the
 *  max keeps the first maximal tap in canonical order (strict comparison).
 *
 * All arithmetic is in double.  Loops run in the order of the definitions;
 * OpenMP only splits independent output elements across threads.
 */
#include <stdlib.h>
#include <string.h>
#include <limits.h>

#define ORACLE_OK 0
#define ORACLE_BAD (-1)

/* ---------------------------------------------------------------- geometry */

static long floordiv(long a, long b)
{
    long q = a / b;
    if ((a % b != 0) && ((a < 0) != (b < 0)))
        q -= 1;
    return q;
}

static long labs_(long a) { return a < 0 ? -a : a; }

/* offset (r, c) -> axial (q, s) */
static void to_axial(long r, long c, long *q, long *s)
{
    *q = c;
    *s = r - floordiv(c, 2);
}

/* axial (q, s) -> offset (r, c) */
static void to_offset(long q, long s, long *r, long *c)
{
    *c = q;
    *r = s + floordiv(q, 2);
}

static long hex_distance(long dq, long ds)
{
    long a = labs_(dq), b = labs_(ds), e = labs_(dq + ds);
    long m = a > b ? a : b;
    return m > e ? m : e;
}

/* Number of taps of a size-k kernel, by enumeration. */
int oracle_num_taps(int k)
{
    if (k < 0)
        return ORACLE_BAD;
    int n = 0;
    for (long dq = -k; dq <= k; dq++)
        for (long ds = -k; ds <= k; ds++)
            if (hex_distance(dq, ds) <= k)
                n++;
    return n;
}

/* Axial tap offsets of a size-k kernel in canonical order (dq, then ds). */
int oracle_taps(int k, int *dq_out, int *ds_out)
{
    if (k < 0)
        return ORACLE_BAD;
    int n = 0;
    for (long dq = -k; dq <= k; dq++)
        for (long ds = -k; ds <= k; ds++)
            if (hex_distance(dq, ds) <= k) {
                dq_out[n] = (int)dq;
                ds_out[n] = (int)ds;
                n++;
            }
    return n;
}

/* Tensor element reached from element (r, c) by the axial step (dq, ds). */
void oracle_step(int r, int c, int dq, int ds, int *r_out, int *c_out)
{
    long q, s, rr, cc;
    to_axial(r, c, &q, &s);
    to_offset(q + dq, s + ds, &rr, &cc);
    *r_out = (int)rr;
    *c_out = (int)cc;
}

/* Axial coordinates of the kernel centre for output element (i, j). */
static void centre_axial(long i, long j, int stride, long *q, long *s)
{
    long Q, S;
    to_axial(i, j, &Q, &S);
    *q = stride * Q;
    *s = stride * S;
}

/* Input tensor element on which output (i, j) is centred. */
void oracle_centre(int i, int j, int stride, int *r_out, int *c_out)
{
    long q, s, r, c;
    centre_axial(i, j, stride, &q, &s);
    to_offset(q, s, &r, &c);
    *r_out = (int)r;
    *c_out = (int)c;
}

/* Output size for an H x W input under stride s (independent of k). */
int oracle_out_shape(int H, int W, int stride, int *Ho, int *Wo)
{
    if (H < 1 || W < 1 || stride < 1)
        return ORACLE_BAD;
    long wo = 0;
    for (;;) {
        int r, c;
        oracle_centre(0, (int)wo, stride, &r, &c);
        if (c >= W)
            break;
        wo++;
    }
    long ho = LONG_MAX;
    for (long j = 0; j < wo; j++) {
        long cnt = 0;
        for (;;) {
            int r, c;
            oracle_centre((int)cnt, (int)j, stride, &r, &c);
            if (r >= H)
                break;
            cnt++;
        }
        if (cnt < ho)
            ho = cnt;
    }
    *Ho = (int)ho;
    *Wo = (int)wo;
    return ORACLE_OK;
}

/* Value of input plane `plane` (H x W) at axial (q, s); zero outside. */
static double tap_value(const double *plane, int H, int W, long q, long s,
                        int *inside)
{
    long r, c;
    to_offset(q, s, &r, &c);
    if (r < 0 || r >= H || c < 0 || c >= W) {
        *inside = 0;
        return 0.0;
    }
    *inside = 1;
    return plane[r * (long)W + c];
}

typedef struct {
    int T;
    int *dq, *ds;
} taps_t;

static int taps_make(int k, taps_t *tp)
{
    tp->T = oracle_num_taps(k);
    if (tp->T < 1)
        return ORACLE_BAD;
    tp->dq = (int *)malloc(sizeof(int) * tp->T);
    tp->ds = (int *)malloc(sizeof(int) * tp->T);
    oracle_taps(k, tp->dq, tp->ds);
    return ORACLE_OK;
}

static void taps_free(taps_t *tp)
{
    free(tp->dq);
    free(tp->ds);
}

/* ------------------------------------------------------------ convolution */

/* y[n][co][i][j] = b[co] + sum_ci sum_t w[co][ci][t] * x[n][ci][centre + tap t] */
static double conv_fwd_one(const double *x, const double *w, const double *b,
                           const taps_t *tp, long n, long co, long i, long j,
                           int Ci, int H, int W, int stride)
{
    long q0, s0;
    centre_axial(i, j, stride, &q0, &s0);
    double acc = b ? b[co] : 0.0;
    for (long ci = 0; ci < Ci; ci++) {
        const double *plane = x + (n * Ci + ci) * (long)H * W;
        for (int t = 0; t < tp->T; t++) {
            int inside;
            double v = tap_value(plane, H, W, q0 + tp->dq[t], s0 + tp->ds[t],
                                 &inside);
            if (inside)
                acc += w[(co * Ci + ci) * tp->T + t] * v;
        }
    }
    return acc;
}

int oracle_conv_fwd(const double *x, const double *w, const double *b,
                    double *y, int N, int Ci, int Co, int H, int W, int k,
                    int stride)
{
    int Ho, Wo;
    taps_t tp;
    if (N < 0 || Ci < 1 || Co < 1 || oracle_out_shape(H, W, stride, &Ho, &Wo)
        || taps_make(k, &tp))
        return ORACLE_BAD;
#pragma omp parallel for collapse(2) schedule(static)
    for (long n = 0; n < N; n++)
        for (long co = 0; co < Co; co++)
            for (long i = 0; i < Ho; i++)
                for (long j = 0; j < Wo; j++)
                    y[((n * Co + co) * Ho + i) * Wo + j] = conv_fwd_one(
                        x, w, b, &tp, n, co, i, j, Ci, H, W, stride);
    taps_free(&tp);
    return ORACLE_OK;
}

/* Selected outputs only: idx[] are flat indices into y[N][Co][Ho][Wo]. */
int oracle_conv_fwd_at(const double *x, const double *w, const double *b,
                       const long *idx, long nidx, double *out, int N, int Ci,
                       int Co, int H, int W, int k, int stride)
{
    int Ho, Wo;
    taps_t tp;
    if (N < 0 || Ci < 1 || Co < 1 || oracle_out_shape(H, W, stride, &Ho, &Wo)
        || taps_make(k, &tp))
        return ORACLE_BAD;
    long total = (long)N * Co * Ho * Wo;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(| : bad)
    for (long e = 0; e < nidx; e++) {
        long f = idx[e];
        if (f < 0 || f >= total) {
            bad = 1;
            continue;
        }
        long j = f % Wo, i = (f / Wo) % Ho, co = (f / ((long)Wo * Ho)) % Co,
             n = f / ((long)Wo * Ho * Co);
        out[e] = conv_fwd_one(x, w, b, &tp, n, co, i, j, Ci, H, W, stride);
    }
    taps_free(&tp);
    return bad ? ORACLE_BAD : ORACLE_OK;
}

/*
 * Gradient with respect to x, as the plain adjoint of the forward sum: every
 * product w[co][ci][t] * x[n][ci][centre(i,j) + tap t] of the forward pass
 * sends dy[n][co][i][j] * w[co][ci][t] back to that input element.
 */
int oracle_conv_bwd_data(const double *dy, const double *w, double *dx, int N,
                         int Ci, int Co, int H, int W, int k, int stride)
{
    int Ho, Wo;
    taps_t tp;
    if (N < 0 || Ci < 1 || Co < 1 || oracle_out_shape(H, W, stride, &Ho, &Wo)
        || taps_make(k, &tp))
        return ORACLE_BAD;
    memset(dx, 0, sizeof(double) * (size_t)N * Ci * H * W);
#pragma omp parallel for schedule(static)
    for (long n = 0; n < N; n++)
        for (long co = 0; co < Co; co++)
            for (long i = 0; i < Ho; i++)
                for (long j = 0; j < Wo; j++) {
                    double g = dy[((n * Co + co) * Ho + i) * Wo + j];
                    long q0, s0;
                    centre_axial(i, j, stride, &q0, &s0);
                    for (long ci = 0; ci < Ci; ci++)
                        for (int t = 0; t < tp.T; t++) {
                            long r, c;
                            to_offset(q0 + tp.dq[t], s0 + tp.ds[t], &r, &c);
                            if (r < 0 || r >= H || c < 0 || c >= W)
                                continue;
                            dx[((n * Ci + ci) * H + r) * W + c] +=
                                g * w[(co * Ci + ci) * tp.T + t];
                        }
                }
    taps_free(&tp);
    return ORACLE_OK;
}

/*
 * Selected elements of dx: for input element (n, ci, r, c), collect every
 * (output, tap) pair of the forward pass that reads it, by testing all output
 * elements whose centre lies near (r, c).
 */
int oracle_conv_bwd_data_at(const double *dy, const double *w, const long *idx,
                            long nidx, double *out, int N, int Ci, int Co,
                            int H, int W, int k, int stride)
{
    int Ho, Wo;
    taps_t tp;
    if (N < 0 || Ci < 1 || Co < 1 || oracle_out_shape(H, W, stride, &Ho, &Wo)
        || taps_make(k, &tp))
        return ORACLE_BAD;
    long total = (long)N * Ci * H * W;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 4) reduction(| : bad)
    for (long e = 0; e < nidx; e++) {
        long f = idx[e];
        if (f < 0 || f >= total) {
            bad = 1;
            continue;
        }
        long c = f % W, r = (f / W) % H, ci = (f / ((long)W * H)) % Ci,
             n = f / ((long)W * H * Ci);
        double acc = 0.0;
        for (long i = 0; i < Ho; i++)
            for (long j = 0; j < Wo; j++) {
                int rc, cc;
                oracle_centre((int)i, (int)j, stride, &rc, &cc);
                /* |dq| <= k columns; |drow| <= |ds| + |floor(dq/2)| + 1 <= 2k+1 */
                if (labs_(cc - c) > k || labs_(rc - r) > 2 * k + 1)
                    continue;
                long q0, s0;
                centre_axial(i, j, stride, &q0, &s0);
                for (int t = 0; t < tp.T; t++) {
                    long rr, cq;
                    to_offset(q0 + tp.dq[t], s0 + tp.ds[t], &rr, &cq);
                    if (rr != r || cq != c)
                        continue;
                    for (long co = 0; co < Co; co++)
                        acc += dy[((n * Co + co) * Ho + i) * Wo + j] *
                               w[(co * Ci + ci) * tp.T + t];
                }
            }
        out[e] = acc;
    }
    taps_free(&tp);
    return bad ? ORACLE_BAD : ORACLE_OK;
}

/* dw[co][ci][t] = sum_n sum_(i,j) dy[n][co][i][j] * x[n][ci][centre + tap t] */
static double conv_dw_one(const double *x, const double *dy, const taps_t *tp,
                          long co, long ci, int t, int N, int Ci, int Co,
                          int H, int W, int Ho, int Wo, int stride)
{
    double acc = 0.0;
    for (long n = 0; n < N; n++) {
        const double *plane = x + (n * Ci + ci) * (long)H * W;
        for (long i = 0; i < Ho; i++)
            for (long j = 0; j < Wo; j++) {
                long q0, s0;
                int inside;
                centre_axial(i, j, stride, &q0, &s0);
                double v = tap_value(plane, H, W, q0 + tp->dq[t],
                                     s0 + tp->ds[t], &inside);
                if (inside)
                    acc += dy[((n * Co + co) * Ho + i) * Wo + j] * v;
            }
    }
    return acc;
}

int oracle_conv_bwd_weight(const double *x, const double *dy, double *dw,
                           double *db, int N, int Ci, int Co, int H, int W,
                           int k, int stride)
{
    int Ho, Wo;
    taps_t tp;
    if (N < 0 || Ci < 1 || Co < 1 || oracle_out_shape(H, W, stride, &Ho, &Wo)
        || taps_make(k, &tp))
        return ORACLE_BAD;
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (long co = 0; co < Co; co++)
        for (long ci = 0; ci < Ci; ci++)
            for (int t = 0; t < tp.T; t++)
                dw[(co * Ci + ci) * tp.T + t] = conv_dw_one(
                    x, dy, &tp, co, ci, t, N, Ci, Co, H, W, Ho, Wo, stride);
    if (db) {
        for (long co = 0; co < Co; co++) {
            double acc = 0.0;
            for (long n = 0; n < N; n++)
                for (long i = 0; i < Ho; i++)
                    for (long j = 0; j < Wo; j++)
                        acc += dy[((n * Co + co) * Ho + i) * Wo + j];
            db[co] = acc;
        }
    }
    taps_free(&tp);
    return ORACLE_OK;
}

/* Selected elements of dw: idx[] are flat indices into dw[Co][Ci][T]. */
int oracle_conv_bwd_weight_at(const double *x, const double *dy,
                              const long *idx, long nidx, double *out, int N,
                              int Ci, int Co, int H, int W, int k, int stride)
{
    int Ho, Wo;
    taps_t tp;
    if (N < 0 || Ci < 1 || Co < 1 || oracle_out_shape(H, W, stride, &Ho, &Wo)
        || taps_make(k, &tp))
        return ORACLE_BAD;
    long total = (long)Co * Ci * tp.T;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (long e = 0; e < nidx; e++) {
        long f = idx[e];
        if (f < 0 || f >= total) {
            bad = 1;
            continue;
        }
        int t = (int)(f % tp.T);
        long ci = (f / tp.T) % Ci, co = f / ((long)tp.T * Ci);
        out[e] = conv_dw_one(x, dy, &tp, co, ci, t, N, Ci, Co, H, W, Ho, Wo,
                             stride);
    }
    taps_free(&tp);
    return bad ? ORACLE_BAD : ORACLE_OK;
}

/* ---------------------------------------------------------------- pooling */

#define ORACLE_POOL_MAX 0
#define ORACLE_POOL_AVG 1

int oracle_pool_fwd(const double *x, double *y, int *argmax, int N, int C,
                    int H, int W, int k, int stride, int mode)
{
    int Ho, Wo;
    taps_t tp;
    if (N < 0 || C < 1 || (mode != ORACLE_POOL_MAX && mode != ORACLE_POOL_AVG)
        || oracle_out_shape(H, W, stride, &Ho, &Wo) || taps_make(k, &tp))
        return ORACLE_BAD;
#pragma omp parallel for collapse(2) schedule(static)
    for (long n = 0; n < N; n++)
        for (long ch = 0; ch < C; ch++) {
            const double *plane = x + (n * C + ch) * (long)H * W;
            for (long i = 0; i < Ho; i++)
                for (long j = 0; j < Wo; j++) {
                    long q0, s0;
                    centre_axial(i, j, stride, &q0, &s0);
                    double best = 0.0, sum = 0.0;
                    int arg = 0;
                    for (int t = 0; t < tp.T; t++) {
                        int inside;
                        double v = tap_value(plane, H, W, q0 + tp.dq[t],
                                             s0 + tp.ds[t], &inside);
                        sum += v;
                        if (t == 0 || v > best) {
                            best = v;
                            arg = t;
                        }
                    }
                    long o = ((n * C + ch) * Ho + i) * Wo + j;
                    y[o] = mode == ORACLE_POOL_MAX ? best : sum / tp.T;
                    if (argmax)
                        argmax[o] = arg;
                }
        }
    taps_free(&tp);
    return ORACLE_OK;
}

/*
 * Pool gradient.  Max: each output's gradient goes to the element its
 * argmax tap points at (dropped when that tap is padding).  Average: each
 * output's gradient is shared out as dy/T over every in-tensor tap.  When
 * relu_y is given (the ReLU output that fed the pool), the result is
 * multiplied by [relu_y > 0].
 */
int oracle_pool_bwd(const double *dy, const int *argmax, const double *relu_y,
                    double *dx, int N, int C, int H, int W, int k, int stride,
                    int mode)
{
    int Ho, Wo;
    taps_t tp;
    if (N < 0 || C < 1 || (mode != ORACLE_POOL_MAX && mode != ORACLE_POOL_AVG)
        || (mode == ORACLE_POOL_MAX && !argmax)
        || oracle_out_shape(H, W, stride, &Ho, &Wo) || taps_make(k, &tp))
        return ORACLE_BAD;
    memset(dx, 0, sizeof(double) * (size_t)N * C * H * W);
    int bad = 0;
#pragma omp parallel for collapse(2) schedule(static) reduction(| : bad)
    for (long n = 0; n < N; n++)
        for (long ch = 0; ch < C; ch++) {
            double *plane = dx + (n * C + ch) * (long)H * W;
            for (long i = 0; i < Ho; i++)
                for (long j = 0; j < Wo; j++) {
                    long o = ((n * C + ch) * Ho + i) * Wo + j;
                    long q0, s0;
                    centre_axial(i, j, stride, &q0, &s0);
                    for (int t = 0; t < tp.T; t++) {
                        double g;
                        if (mode == ORACLE_POOL_MAX) {
                            if (argmax[o] < 0 || argmax[o] >= tp.T)
                                bad = 1;
                            if (t != argmax[o])
                                continue;
                            g = dy[o];
                        } else {
                            g = dy[o] / tp.T;
                        }
                        long r, c;
                        to_offset(q0 + tp.dq[t], s0 + tp.ds[t], &r, &c);
                        if (r < 0 || r >= H || c < 0 || c >= W)
                            continue;
                        plane[r * W + c] += g;
                    }
                }
        }
    if (relu_y) {
        long total = (long)N * C * H * W;
        for (long e = 0; e < total; e++)
            if (!(relu_y[e] > 0.0))
                dx[e] = 0.0;
    }
    taps_free(&tp);
    return bad ? ORACLE_BAD : ORACLE_OK;
}

/* ------------------------------------------------------ three dimensions */

/*
 * Three-dimensional operations (Sec. 2.4, "Software Functionalities"): the
 * x-y planes are hexagonal, in the addressing above, and the samples along
 * z are equidistant (e.g. the time slices of a hexagonal camera).  The paper
 * gives no further detail; readings adopted:
 *  - tensors x[N][C][D][H][W]: D planes along z, each an H x W hexagonal
 *    plane;
 *  - a kernel of size (k, kz) is the size-k hexagonal window in the plane
 *    times the 2kz+1 planes dz = -kz .. kz around the centre plane; taps are
 *    numbered dz-major (dz ascending), the hexagonal taps in canonical order
 *    inside; weights w[C_out][C_in][2kz+1][T];
 *  - padding and stride follow the 2-D rule along z as well: windows are
 *    centred on real planes only and planes outside the tensor read zero;
 *    the centres are the planes sz*l, l = 0, 1, ... while sz*l < D, so
 *    D_out = floor((D-1)/sz) + 1 (equal steps from the first plane);
 *  - pooling: maximum or average over the (2kz+1)*T taps, padded taps
 *    counting as zeros; the average divides by (2kz+1)*T; the maximum keeps
 *    the first maximal tap in the order above, its index (dz+kz)*T + t.
 */

int oracle_out_shape3d(int D, int H, int W, int stride, int stride_z, int *Do,
                       int *Ho, int *Wo)
{
    if (D < 1 || stride_z < 1 || oracle_out_shape(H, W, stride, Ho, Wo))
        return ORACLE_BAD;
    long l = 0;
    while ((long)stride_z * l < D)
        l++;
    *Do = (int)l;
    return ORACLE_OK;
}

typedef struct {
    int N, Ci, Co, D, H, W, Do, Ho, Wo, kz, Z, stride, stride_z;
    taps_t tp;
} shape3d_t;

static int shape3d_make(int N, int Ci, int Co, int D, int H, int W, int k,
                        int kz, int stride, int stride_z, shape3d_t *sh)
{
    if (N < 0 || Ci < 1 || Co < 1 || kz < 0 ||
        oracle_out_shape3d(D, H, W, stride, stride_z, &sh->Do, &sh->Ho, &sh->Wo)
        || taps_make(k, &sh->tp))
        return ORACLE_BAD;
    sh->N = N;
    sh->Ci = Ci;
    sh->Co = Co;
    sh->D = D;
    sh->H = H;
    sh->W = W;
    sh->kz = kz;
    sh->Z = 2 * kz + 1;
    sh->stride = stride;
    sh->stride_z = stride_z;
    return ORACLE_OK;
}

/* plane z of channel ch of image n in x[N][C][D][H][W] */
static const double *plane3d(const double *x, const shape3d_t *sh, long n,
                             long ch, long C, long z)
{
    return x + ((n * C + ch) * sh->D + z) * (long)sh->H * sh->W;
}

/* y[n][co][l][i][j] = b[co] + sum_ci sum_dz sum_t w[co][ci][dz][t] * x[n][ci][sz*l+dz][centre + tap t] */
static double conv3d_fwd_one(const double *x, const double *w, const double *b,
                             const shape3d_t *sh, long n, long co, long l,
                             long i, long j)
{
    long q0, s0;
    centre_axial(i, j, sh->stride, &q0, &s0);
    const long z0 = (long)sh->stride_z * l;
    const int T = sh->tp.T;
    double acc = b ? b[co] : 0.0;
    for (long ci = 0; ci < sh->Ci; ci++)
        for (long dz = -sh->kz; dz <= sh->kz; dz++) {
            const long z = z0 + dz;
            if (z < 0 || z >= sh->D)
                continue;
            const double *plane = plane3d(x, sh, n, ci, sh->Ci, z);
            for (int t = 0; t < T; t++) {
                int inside;
                double v = tap_value(plane, sh->H, sh->W, q0 + sh->tp.dq[t],
                                     s0 + sh->tp.ds[t], &inside);
                if (inside)
                    acc += w[((co * sh->Ci + ci) * sh->Z + (dz + sh->kz)) * T + t] * v;
            }
        }
    return acc;
}

int oracle_conv3d_fwd(const double *x, const double *w, const double *b,
                      double *y, int N, int Ci, int Co, int D, int H, int W,
                      int k, int kz, int stride, int stride_z)
{
    shape3d_t sh;
    if (shape3d_make(N, Ci, Co, D, H, W, k, kz, stride, stride_z, &sh))
        return ORACLE_BAD;
    const long Do = sh.Do, Ho = sh.Ho, Wo = sh.Wo;
#pragma omp parallel for collapse(3) schedule(static)
    for (long n = 0; n < N; n++)
        for (long co = 0; co < Co; co++)
            for (long l = 0; l < Do; l++)
                for (long i = 0; i < Ho; i++)
                    for (long j = 0; j < Wo; j++)
                        y[(((n * Co + co) * Do + l) * Ho + i) * Wo + j] =
                            conv3d_fwd_one(x, w, b, &sh, n, co, l, i, j);
    taps_free(&sh.tp);
    return ORACLE_OK;
}

/*
 * Gradient with respect to x: the adjoint of the forward sum -- every
 * product w[co][ci][dz][t] * x[n][ci][sz*l+dz][centre(i,j) + tap t] sends
 * dy[n][co][l][i][j] * w[co][ci][dz][t] back to that input element.
 */
int oracle_conv3d_bwd_data(const double *dy, const double *w, double *dx,
                           int N, int Ci, int Co, int D, int H, int W, int k,
                           int kz, int stride, int stride_z)
{
    shape3d_t sh;
    if (shape3d_make(N, Ci, Co, D, H, W, k, kz, stride, stride_z, &sh))
        return ORACLE_BAD;
    const long Do = sh.Do, Ho = sh.Ho, Wo = sh.Wo;
    const int T = sh.tp.T;
    memset(dx, 0, sizeof(double) * (size_t)N * Ci * D * H * W);
#pragma omp parallel for schedule(static)
    for (long n = 0; n < N; n++)
        for (long co = 0; co < Co; co++)
            for (long l = 0; l < Do; l++)
                for (long i = 0; i < Ho; i++)
                    for (long j = 0; j < Wo; j++) {
                        const double g = dy[(((n * Co + co) * Do + l) * Ho + i) * Wo + j];
                        long q0, s0;
                        centre_axial(i, j, stride, &q0, &s0);
                        for (long ci = 0; ci < Ci; ci++)
                            for (long dz = -kz; dz <= kz; dz++) {
                                const long z = (long)stride_z * l + dz;
                                if (z < 0 || z >= D)
                                    continue;
                                for (int t = 0; t < T; t++) {
                                    long r, c;
                                    to_offset(q0 + sh.tp.dq[t], s0 + sh.tp.ds[t], &r, &c);
                                    if (r < 0 || r >= H || c < 0 || c >= W)
                                        continue;
                                    dx[(((n * Ci + ci) * D + z) * H + r) * W + c] +=
                                        g * w[((co * Ci + ci) * sh.Z + (dz + kz)) * T + t];
                                }
                            }
                    }
    taps_free(&sh.tp);
    return ORACLE_OK;
}

/* dw[co][ci][dz][t] = sum_n sum_(l,i,j) dy[n][co][l][i][j] * x[n][ci][sz*l+dz][centre + tap t];
 * db[co] = sum_n sum_(l,i,j) dy[n][co][l][i][j] */
int oracle_conv3d_bwd_weight(const double *x, const double *dy, double *dw,
                             double *db, int N, int Ci, int Co, int D, int H,
                             int W, int k, int kz, int stride, int stride_z)
{
    shape3d_t sh;
    if (shape3d_make(N, Ci, Co, D, H, W, k, kz, stride, stride_z, &sh))
        return ORACLE_BAD;
    const long Do = sh.Do, Ho = sh.Ho, Wo = sh.Wo;
    const int T = sh.tp.T, Z = sh.Z;
#pragma omp parallel for collapse(3) schedule(dynamic, 1)
    for (long co = 0; co < Co; co++)
        for (long ci = 0; ci < Ci; ci++)
            for (long zt = 0; zt < (long)Z * T; zt++) {
                const long dz = zt / T - kz;
                const int t = (int)(zt % T);
                double acc = 0.0;
                for (long n = 0; n < N; n++)
                    for (long l = 0; l < Do; l++) {
                        const long z = (long)stride_z * l + dz;
                        if (z < 0 || z >= D)
                            continue;
                        const double *plane = plane3d(x, &sh, n, ci, Ci, z);
                        for (long i = 0; i < Ho; i++)
                            for (long j = 0; j < Wo; j++) {
                                long q0, s0;
                                int inside;
                                centre_axial(i, j, stride, &q0, &s0);
                                double v = tap_value(plane, H, W, q0 + sh.tp.dq[t],
                                                     s0 + sh.tp.ds[t], &inside);
                                if (inside)
                                    acc += dy[(((n * Co + co) * Do + l) * Ho + i) * Wo + j] * v;
                            }
                    }
                dw[(co * Ci + ci) * (long)Z * T + zt] = acc;
            }
    if (db) {
        for (long co = 0; co < Co; co++) {
            double acc = 0.0;
            for (long n = 0; n < N; n++)
                for (long e = 0; e < Do * Ho * Wo; e++)
                    acc += dy[(n * Co + co) * Do * Ho * Wo + e];
            db[co] = acc;
        }
    }
    taps_free(&sh.tp);
    return ORACLE_OK;
}

int oracle_pool3d_fwd(const double *x, double *y, int *argmax, int N, int C,
                      int D, int H, int W, int k, int kz, int stride,
                      int stride_z, int mode)
{
    shape3d_t sh;
    if ((mode != ORACLE_POOL_MAX && mode != ORACLE_POOL_AVG) ||
        shape3d_make(N, C, C, D, H, W, k, kz, stride, stride_z, &sh))
        return ORACLE_BAD;
    const long Do = sh.Do, Ho = sh.Ho, Wo = sh.Wo;
    const int T = sh.tp.T;
#pragma omp parallel for collapse(3) schedule(static)
    for (long n = 0; n < N; n++)
        for (long ch = 0; ch < C; ch++)
            for (long l = 0; l < Do; l++)
                for (long i = 0; i < Ho; i++)
                    for (long j = 0; j < Wo; j++) {
                        long q0, s0;
                        centre_axial(i, j, stride, &q0, &s0);
                        double best = 0.0, sum = 0.0;
                        int arg = 0, first = 1;
                        for (long dz = -kz; dz <= kz; dz++) {
                            const long z = (long)stride_z * l + dz;
                            for (int t = 0; t < T; t++) {
                                double v = 0.0;
                                if (z >= 0 && z < D) {
                                    int inside;
                                    v = tap_value(plane3d(x, &sh, n, ch, C, z), H, W,
                                                  q0 + sh.tp.dq[t], s0 + sh.tp.ds[t], &inside);
                                }
                                sum += v;
                                if (first || v > best) {
                                    best = v;
                                    arg = (int)((dz + kz) * T + t);
                                    first = 0;
                                }
                            }
                        }
                        const long o = (((n * C + ch) * Do + l) * Ho + i) * Wo + j;
                        y[o] = mode == ORACLE_POOL_MAX ? best : sum / ((double)sh.Z * T);
                        if (argmax)
                            argmax[o] = arg;
                    }
    taps_free(&sh.tp);
    return ORACLE_OK;
}

/*
 * 3-D pool gradient.  Max: each output's gradient goes to the element its
 * argmax tap points at (dropped when that tap is padding).  Average: dy /
 * ((2kz+1) T) to every in-tensor tap.  relu_y (nullable) masks the result
 * by [relu_y > 0].
 */
int oracle_pool3d_bwd(const double *dy, const int *argmax, const double *relu_y,
                      double *dx, int N, int C, int D, int H, int W, int k,
                      int kz, int stride, int stride_z, int mode)
{
    shape3d_t sh;
    if ((mode != ORACLE_POOL_MAX && mode != ORACLE_POOL_AVG) ||
        (mode == ORACLE_POOL_MAX && !argmax) ||
        shape3d_make(N, C, C, D, H, W, k, kz, stride, stride_z, &sh))
        return ORACLE_BAD;
    const long Do = sh.Do, Ho = sh.Ho, Wo = sh.Wo;
    const int T = sh.tp.T;
    const long ZT = (long)sh.Z * T;
    memset(dx, 0, sizeof(double) * (size_t)N * C * D * H * W);
    int bad = 0;
#pragma omp parallel for collapse(2) schedule(static) reduction(| : bad)
    for (long n = 0; n < N; n++)
        for (long ch = 0; ch < C; ch++)
            for (long l = 0; l < Do; l++)
                for (long i = 0; i < Ho; i++)
                    for (long j = 0; j < Wo; j++) {
                        const long o = (((n * C + ch) * Do + l) * Ho + i) * Wo + j;
                        long q0, s0;
                        centre_axial(i, j, stride, &q0, &s0);
                        if (mode == ORACLE_POOL_MAX && (argmax[o] < 0 || argmax[o] >= ZT))
                            bad = 1;
                        for (long zt = 0; zt < ZT; zt++) {
                            double g;
                            if (mode == ORACLE_POOL_MAX) {
                                if (zt != argmax[o])
                                    continue;
                                g = dy[o];
                            } else {
                                g = dy[o] / (double)ZT;
                            }
                            const long z = (long)stride_z * l + zt / T - kz;
                            const int t = (int)(zt % T);
                            long r, c;
                            to_offset(q0 + sh.tp.dq[t], s0 + sh.tp.ds[t], &r, &c);
                            if (z < 0 || z >= D || r < 0 || r >= H || c < 0 || c >= W)
                                continue;
                            dx[(((n * C + ch) * D + z) * H + r) * W + c] += g;
                        }
                    }
    if (relu_y) {
        const long total = (long)N * C * D * H * W;
        for (long e = 0; e < total; e++)
            if (!(relu_y[e] > 0.0))
                dx[e] = 0.0;
    }
    taps_free(&sh.tp);
    return bad ? ORACLE_BAD : ORACLE_OK;
}

/* Threads the OpenMP runtime will use for the parallel loops above. */
int oracle_threads(void)
{
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            n = omp_get_num_threads();
#endif
        }
    }
    return n;
}

/* Sets the number of threads later parallel loops use (n >= 1); used to
 * time the reference on one core.  No effect on results. */
int oracle_set_threads(int n)
{
    if (n < 1)
        return ORACLE_BAD;
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    omp_set_num_threads(n);
#endif
    return ORACLE_OK;
}
