/* Drives the fp64 oracle (oracle/hexoracle.c) over 2-D and 3-D cases for a
 * build with AddressSanitizer and UndefinedBehaviorSanitizer: every entry
 * point at several kernel sizes, strides and ragged shapes, including the
 * sampled variants and argmax-driven pooling gradients.  Exit status 0 when
 * every call returned success (the sanitizers abort on a finding). */
#include <stdio.h>
#include <stdlib.h>

int oracle_num_taps(int k);
int oracle_out_shape(int H, int W, int stride, int *Ho, int *Wo);
int oracle_out_shape3d(int D, int H, int W, int s, int sz, int *Do, int *Ho, int *Wo);
int oracle_conv_fwd(const double *x, const double *w, const double *b, double *y, int N, int Ci,
                    int Co, int H, int W, int k, int stride);
int oracle_conv_fwd_at(const double *x, const double *w, const double *b, const long *idx,
                       long nidx, double *out, int N, int Ci, int Co, int H, int W, int k,
                       int stride);
int oracle_conv_bwd_data(const double *dy, const double *w, double *dx, int N, int Ci, int Co,
                         int H, int W, int k, int stride);
int oracle_conv_bwd_data_at(const double *dy, const double *w, const long *idx, long nidx,
                            double *out, int N, int Ci, int Co, int H, int W, int k, int stride);
int oracle_conv_bwd_weight(const double *x, const double *dy, double *dw, double *db, int N,
                           int Ci, int Co, int H, int W, int k, int stride);
int oracle_conv_bwd_weight_at(const double *x, const double *dy, const long *idx, long nidx,
                              double *out, int N, int Ci, int Co, int H, int W, int k, int stride);
int oracle_pool_fwd(const double *x, double *y, int *argmax, int N, int C, int H, int W, int k,
                    int stride, int mode);
int oracle_pool_bwd(const double *dy, const int *argmax, const double *relu_y, double *dx, int N,
                    int C, int H, int W, int k, int stride, int mode);
int oracle_conv3d_fwd(const double *x, const double *w, const double *b, double *y, int N,
                      int Ci, int Co, int D, int H, int W, int k, int kz, int s, int sz);
int oracle_conv3d_bwd_data(const double *dy, const double *w, double *dx, int N, int Ci, int Co,
                           int D, int H, int W, int k, int kz, int s, int sz);
int oracle_conv3d_bwd_weight(const double *x, const double *dy, double *dw, double *db, int N,
                             int Ci, int Co, int D, int H, int W, int k, int kz, int s, int sz);
int oracle_pool3d_fwd(const double *x, double *y, int *argmax, int N, int C, int D, int H, int W,
                      int k, int kz, int s, int sz, int mode);
int oracle_pool3d_bwd(const double *dy, const int *argmax, const double *relu_y, double *dx,
                      int N, int C, int D, int H, int W, int k, int kz, int s, int sz, int mode);

static double *rnd(long n)
{
    double *p = malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    for (long i = 0; i < n; i++)
        p[i] = (double)rand() / RAND_MAX - 0.5;
    return p;
}

#define CHECK(call)                                                                           \
    do {                                                                                      \
        if ((call) != 0) {                                                                    \
            fprintf(stderr, "failed: %s\n", #call);                                           \
            return 1;                                                                         \
        }                                                                                     \
    } while (0)

int main(void)
{
    static const int cases[][5] = {{9, 8, 1, 1, 0}, {7, 11, 2, 1, 0}, {12, 13, 1, 2, 0},
                                   {5, 5, 2, 3, 0}, {17, 9, 3, 4, 0}, {1, 7, 1, 1, 0},
                                   {6, 1, 2, 1, 0}, {20, 22, 5, 5, 0}, {25, 27, 8, 8, 0}};
    for (unsigned c = 0; c < sizeof(cases) / sizeof(cases[0]); c++) {
        const int H = cases[c][0], W = cases[c][1], k = cases[c][2], s = cases[c][3];
        const int N = 2, Ci = 3, Co = 2, T = oracle_num_taps(k);
        int Ho, Wo;
        CHECK(oracle_out_shape(H, W, s, &Ho, &Wo));
        const long nx = (long)N * Ci * H * W, ny = (long)N * Co * Ho * Wo, nw = (long)Co * Ci * T;
        double *x = rnd(nx), *w = rnd(nw), *b = rnd(Co), *y = rnd(ny), *dy = rnd(ny),
               *dx = rnd(nx), *dw = rnd(nw), *db = rnd(Co), *out = rnd(8);
        long idx[3] = {0, ny > 1 ? ny / 2 : 0, ny > 0 ? ny - 1 : 0};
        if (ny > 0) {
            CHECK(oracle_conv_fwd(x, w, b, y, N, Ci, Co, H, W, k, s));
            CHECK(oracle_conv_fwd_at(x, w, b, idx, 3, out, N, Ci, Co, H, W, k, s));
        }
        CHECK(oracle_conv_bwd_data(dy, w, dx, N, Ci, Co, H, W, k, s));
        long idxx[3] = {0, nx / 2, nx - 1};
        CHECK(oracle_conv_bwd_data_at(dy, w, idxx, 3, out, N, Ci, Co, H, W, k, s));
        CHECK(oracle_conv_bwd_weight(x, dy, dw, db, N, Ci, Co, H, W, k, s));
        long idxw[2] = {0, nw - 1};
        CHECK(oracle_conv_bwd_weight_at(x, dy, idxw, 2, out, N, Ci, Co, H, W, k, s));
        int *am = malloc(sizeof(int) * (size_t)(ny > 0 ? ny : 1));
        double *yp = rnd((long)N * Ci * Ho * Wo), *dyp = rnd((long)N * Ci * Ho * Wo);
        int *amp = malloc(sizeof(int) * (size_t)(N * Ci * Ho * Wo + 1));
        for (int mode = 0; mode < 2; mode++) {
            CHECK(oracle_pool_fwd(x, yp, amp, N, Ci, H, W, k, s, mode));
            CHECK(oracle_pool_bwd(dyp, amp, x, dx, N, Ci, H, W, k, s, mode));
        }
        free(x); free(w); free(b); free(y); free(dy); free(dx); free(dw); free(db); free(out);
        free(am); free(yp); free(dyp); free(amp);
    }
    static const int c3[][7] = {{4, 6, 7, 1, 1, 1, 1}, {5, 9, 8, 2, 2, 2, 1}, {1, 5, 5, 1, 2, 1, 1},
                                {7, 8, 9, 0, 4, 1, 3}, {6, 12, 12, 3, 1, 3, 2}};
    for (unsigned c = 0; c < sizeof(c3) / sizeof(c3[0]); c++) {
        const int D = c3[c][0], H = c3[c][1], W = c3[c][2], k = c3[c][3], kz = c3[c][4];
        const int s = c3[c][5], sz = c3[c][6];
        const int N = 2, Ci = 2, Co = 3, T = oracle_num_taps(k), Z = 2 * kz + 1;
        int Do, Ho, Wo;
        CHECK(oracle_out_shape3d(D, H, W, s, sz, &Do, &Ho, &Wo));
        const long nx = (long)N * Ci * D * H * W, ny = (long)N * Co * Do * Ho * Wo;
        const long nw = (long)Co * Ci * Z * T, np = (long)N * Ci * Do * Ho * Wo;
        double *x = rnd(nx), *w = rnd(nw), *b = rnd(Co), *y = rnd(ny), *dy = rnd(ny),
               *dx = rnd(nx), *dw = rnd(nw), *db = rnd(Co), *yp = rnd(np), *dyp = rnd(np);
        int *amp = malloc(sizeof(int) * (size_t)(np + 1));
        CHECK(oracle_conv3d_fwd(x, w, b, y, N, Ci, Co, D, H, W, k, kz, s, sz));
        CHECK(oracle_conv3d_bwd_data(dy, w, dx, N, Ci, Co, D, H, W, k, kz, s, sz));
        CHECK(oracle_conv3d_bwd_weight(x, dy, dw, db, N, Ci, Co, D, H, W, k, kz, s, sz));
        for (int mode = 0; mode < 2; mode++) {
            CHECK(oracle_pool3d_fwd(x, yp, amp, N, Ci, D, H, W, k, kz, s, sz, mode));
            CHECK(oracle_pool3d_bwd(dyp, amp, x, dx, N, Ci, D, H, W, k, kz, s, sz, mode));
        }
        free(x); free(w); free(b); free(y); free(dy); free(dx); free(dw); free(db); free(yp);
        free(dyp); free(amp);
    }
    printf("oracle sanitized run ok\n");
    return 0;
}
