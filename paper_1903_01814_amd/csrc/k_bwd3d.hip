// k_bwd3d.hip -- data gradient of a three-dimensional layer (hexagonal
// planes stacked along z, Sec. 2.4) with few input channels, float32, plane
// stride 1 and in-plane stride 1, k <= 2:
//
//   dx[n][ci][e](p) = sum_co sum_dz sum_t w[co][ci][dz][t] * dy[n][co][e + kz - dz](p - tap t)
//
// (dz = 0 .. 2kz indexes the planes -kz .. kz; in the plane the adjoint is
// the point-reflected kernel, t <-> T-1-t).  A block owns one band of rows
// of one sample and a range of dx planes [e_lo, e_hi).  It walks the dy
// planes d that reach those planes (d = e_lo - kz .. e_hi + kz - 1 inside
// the volume) in order and stages each one's window once, all C_out
// channels, in the sheared layout of shear.h (a tap is a fixed offset).  A
// dy plane d feeds the 2kz + 1 dx planes d - kz .. d + kz, which a thread
// holds for its pixels in a register ring: slot s is plane d - kz + s and
// takes the weights w[co][ci][s].  After plane d, slot 0 (plane d - kz) has
// every contribution: it is stored when it belongs to the block, and the
// ring shifts by one.  Every dy element is read from HBM once per plane
// chunk (plus the 2kz planes a chunk shares with its neighbours).
//
// Thread = (column, strip of R = 2 rows) of the band; the weights of an
// output channel are read with scalar loads (block-uniform addresses): read
// from LDS, even as broadcasts, they took two thirds of the LDS bandwidth
// that bounds the channel loop (c6 data gradient 110 -> 89 us).  The next
// plane is loaded into registers while the current one is computed.  One
// plane ahead, and
// at most 8 staged window rows per thread (the block takes extra threads,
// idle in the products, to get there), keep the kernel at about 90
// registers: five waves per SIMD instead of two with two planes ahead of 12
// rows each (215 registers; c6 data gradient 145 -> 110 us).
#include <algorithm>

#include "hexdev.h"
#include "kernels.h"
#include "shear.h"

namespace hexk {
namespace {

using namespace hexgeom;

constexpr int kMaxThreads3 = 512;

struct Bwd3Args {
    int TR;        // rows per band
    int nbands;    // bands per plane
    int EC;        // dx planes per block
    int nchunks;   // plane chunks per (sample, band)
    int P, CS;     // sheared column pitch, floats per staged channel
    FastDiv fdlr;  // division by TR + 2K (window rows)
};

template <int K, int KZ, int CI, int R, int U>
__global__ __launch_bounds__(kMaxThreads3) void bwd_data3d_smallc_k(
    const float *__restrict__ dy, const float *__restrict__ w, float *__restrict__ dx,
    ConvShape sh, Bwd3Args a)
{
    constexpr int T = num_taps(K);
    constexpr int Z = 2 * KZ + 1;
    extern __shared__ float ds3[];
    const int W = sh.W, H = sh.H, D = sh.D, Co = sh.Co;
    const size_t HW = static_cast<size_t>(H) * W;

    int blk = blockIdx.x;
    const int chunk = blk % a.nchunks;
    blk /= a.nchunks;
    const int band = blk % a.nbands;
    const int n = blk / a.nbands;
    const int r0 = band * a.TR;
    const int rows = min(a.TR, H - r0);
    const int e_lo = chunk * a.EC, e_hi = min(D, e_lo + a.EC);
    const int dlo = max(0, e_lo - KZ), dhi = min(D, e_hi + KZ);

    const ShearTile tl{r0 - K, -K, a.TR + 2 * K, W + 2 * K, a.P, a.CS};
    const int c = threadIdx.x % W, strip = threadIdx.x / W;
    const bool active = strip * R < rows; // threadIdx.x < W * ceil(TR / R)
    const int a0 = active ? tl.addr(r0 + strip * R, c) : 0;

    // dy plane d of every output channel (one "channel" per C_out)
    const float *img = dy + static_cast<size_t>(n) * Co * D * HW;
    auto load_plane = [&](ShearPrefetch<U> &p, int d) {
        d = min(d, dhi - 1); // past the last plane: reload it (never committed)
        p.load3(img, D * HW, HW, static_cast<long>(d) * static_cast<long>(HW), 1, 0, 1, Co, H, W,
                tl, a.TR + 2 * K, a.fdlr);
    };

    float acc[Z][CI][R];
#pragma unroll
    for (int s = 0; s < Z; ++s)
#pragma unroll
        for (int ci = 0; ci < CI; ++ci)
#pragma unroll
            for (int r = 0; r < R; ++r)
                acc[s][ci][r] = 0.f;

    auto store_slot0 = [&](int e) {
        if (!active || e < e_lo || e >= e_hi)
            return;
#pragma unroll
        for (int ci = 0; ci < CI; ++ci) {
            float *dst = dx + ((static_cast<size_t>(n) * CI + ci) * D + e) * HW +
                         static_cast<size_t>(r0 + strip * R) * W + c;
#pragma unroll
            for (int r = 0; r < R; ++r)
                if (strip * R + r < rows)
                    dst[static_cast<size_t>(r) * W] = acc[0][ci][r];
        }
    };
    auto shift = [&]() {
#pragma unroll
        for (int s = 0; s + 1 < Z; ++s)
#pragma unroll
            for (int ci = 0; ci < CI; ++ci)
#pragma unroll
                for (int r = 0; r < R; ++r)
                    acc[s][ci][r] = acc[s + 1][ci][r];
#pragma unroll
        for (int ci = 0; ci < CI; ++ci)
#pragma unroll
            for (int r = 0; r < R; ++r)
                acc[Z - 1][ci][r] = 0.f;
    };

    // one dy plane: stage it, request the next plane into the same
    // registers, add its contributions to the ring, retire slot 0
    auto plane_step = [&](ShearPrefetch<U> &p, int d) {
        __syncthreads(); // the previous plane's reads are done
        p.commit(ds3);
        __syncthreads();
        load_plane(p, d + 1);
        if (active) {
            for (int co = 0; co < Co; ++co) {
                const float *src = ds3 + co * a.CS + a0;
                int t0 = 0;
#pragma unroll
                for (int dq = -K; dq <= K; ++dq) {
                    const int len = 2 * K + 1 - (dq < 0 ? -dq : dq);
                    const int dslo = dq < 0 ? -K - dq : -K;
                    const float *col = src + dq * a.P + dslo;
                    float v[R + 2 * K];
#pragma unroll
                    for (int j = 0; j < R + 2 * K; ++j)
                        if (j < R + len - 1)
                            v[j] = col[j];
#pragma unroll
                    for (int u = 0; u < 2 * K + 1; ++u) {
                        if (u < len) {
                            const int tr = t0 + u; // position in the reflected row
#pragma unroll
                            for (int ci = 0; ci < CI; ++ci) {
                                const float *wc = w + static_cast<size_t>(co * CI + ci) * Z * T;
#pragma unroll
                                for (int s = 0; s < Z; ++s) {
                                    const float wv = wc[s * T + (T - 1 - tr)];
#pragma unroll
                                    for (int r = 0; r < R; ++r)
                                        acc[s][ci][r] += wv * v[r + u];
                                }
                            }
                        }
                    }
                    t0 += len;
                }
            }
        }
        store_slot0(d - KZ);
        shift();
    };

    // the ring starts at dx planes dlo - kz .. dlo + kz
    ShearPrefetch<U> pa;
    load_plane(pa, dlo);
    for (int d = dlo; d < dhi; ++d)
        plane_step(pa, d);
    // planes dhi - kz .. dhi - 1 have no further dy plane inside the range
#pragma unroll
    for (int s = 0; s < KZ; ++s) {
        store_slot0(dhi - KZ + s);
        shift();
    }
}

inline int cdiv(long x, long y) { return static_cast<int>((x + y - 1) / y); }

constexpr size_t kLds3 = 64 * 1024;

struct Bwd3Plan {
    Bwd3Args a;
    int R, U, threads, grid;
    size_t lds;
    bool ok;
};

Bwd3Plan plan_bwd3(const ConvShape &sh)
{
    Bwd3Plan pl{};
    pl.ok = false;
    if (sh.s != 1 || sh.sz != 1 || (sh.k != 1 && sh.k != 2) || sh.kz > 2 ||
        (sh.Ci != 1 && sh.Ci != 2) || sh.W % 4 != 0 || sh.W > 256 || sh.Co > 64 || sh.N < 1)
        return pl;
    const int K = sh.k;
    Bwd3Args &a = pl.a;
    // rows per band and per thread: about 2 blocks' worth of threads per band
    a.TR = 8;
    pl.R = 2; // two rows per thread: each weight read serves two outputs
    if (sh.W * cdiv(a.TR, pl.R) > kMaxThreads3)
        return pl;
    pl.threads = cdiv(sh.W * cdiv(a.TR, pl.R), 64) * 64;
    a.nbands = cdiv(sh.H, a.TR);
    a.P = a.TR + 2 * K + 1;
    a.CS = (sh.W + 2 * K) * a.P;
    a.fdlr = make_fastdiv(static_cast<uint32_t>(a.TR + 2 * K));
    pl.lds = sizeof(float) * static_cast<size_t>(sh.Co) * a.CS;
    if (pl.lds > kLds3)
        return pl;
    // staging rows per thread (ShearPrefetch): one 4-column group per thread
    const int groups = ShearPrefetch<1>::groups(sh.W + 2 * K);
    if (groups > pl.threads)
        return pl;
    // staging rows per thread: more threads (idle in the products) until a
    // thread stages at most 8 window rows (92 registers at k = 1, against
    // 143 for 12 rows)
    auto rows_per_thread = [&](int nt) {
        return cdiv(static_cast<long>(sh.Co) * (a.TR + 2 * K), nt / groups);
    };
    while (rows_per_thread(pl.threads) > 8 && pl.threads + 64 <= kMaxThreads3)
        pl.threads += 64;
    const int rpt = rows_per_thread(pl.threads);
    pl.U = rpt <= 4 ? 4 : rpt <= 8 ? 8 : rpt <= 12 ? 12 : 0;
    if (pl.U == 0)
        return pl;
    // plane chunks: about four blocks per compute unit in all
    const long base = static_cast<long>(sh.N) * a.nbands;
    a.nchunks = std::max(1, std::min(sh.D, cdiv(4L * device_cus(), base)));
    a.EC = cdiv(sh.D, a.nchunks);
    a.nchunks = cdiv(sh.D, a.EC);
    const long grid = base * a.nchunks;
    if (grid > (1L << 31) - 1)
        return pl;
    pl.grid = static_cast<int>(grid);
    pl.ok = true;
    return pl;
}

template <int K, int KZ, int CI, int R>
hipError_t launch_bwd3_u(const Bwd3Plan &pl, const float *dy, const float *w, float *dx,
                         const ConvShape &sh, hipStream_t st)
{
#define HEX_B3(UV)                                                                           \
    HEX_LAUNCH((bwd_data3d_smallc_k<K, KZ, CI, R, UV>), dim3(pl.grid), dim3(pl.threads),     \
               pl.lds, st, dy, w, dx, sh, pl.a)
    if (pl.U == 4)
        HEX_B3(4);
    else if (pl.U == 8)
        HEX_B3(8);
    else
        HEX_B3(12);
#undef HEX_B3
    return hipGetLastError();
}

template <int K, int KZ>
hipError_t launch_bwd3_k(const Bwd3Plan &pl, const float *dy, const float *w, float *dx,
                         const ConvShape &sh, hipStream_t st)
{
    if (sh.Ci == 1)
        return pl.R == 1 ? launch_bwd3_u<K, KZ, 1, 1>(pl, dy, w, dx, sh, st)
                         : launch_bwd3_u<K, KZ, 1, 2>(pl, dy, w, dx, sh, st);
    return pl.R == 1 ? launch_bwd3_u<K, KZ, 2, 1>(pl, dy, w, dx, sh, st)
                     : launch_bwd3_u<K, KZ, 2, 2>(pl, dy, w, dx, sh, st);
}

} // namespace

bool smallc3d_f32_bwd_data_ok(const ConvShape &sh) { return plan_bwd3(sh).ok; }

hipError_t smallc3d_f32_bwd_data(const float *dy, const float *w, float *dx, const ConvShape &sh,
                                 hipStream_t st)
{
    const Bwd3Plan pl = plan_bwd3(sh);
    if (!pl.ok)
        return hipErrorInvalidValue;
    if (sh.k == 1) {
        if (sh.kz == 0)
            return launch_bwd3_k<1, 0>(pl, dy, w, dx, sh, st);
        if (sh.kz == 1)
            return launch_bwd3_k<1, 1>(pl, dy, w, dx, sh, st);
        return launch_bwd3_k<1, 2>(pl, dy, w, dx, sh, st);
    }
    if (sh.kz == 0)
        return launch_bwd3_k<2, 0>(pl, dy, w, dx, sh, st);
    if (sh.kz == 1)
        return launch_bwd3_k<2, 1>(pl, dy, w, dx, sh, st);
    return launch_bwd3_k<2, 2>(pl, dy, w, dx, sh, st);
}

} // namespace hexk
