// k_bwd3d.hip -- data gradient of a three-dimensional layer (hexagonal
// planes stacked along z, Sec. 2.4) with few input channels, float32 or
// bfloat16 data (float32 arithmetic), plane stride 1 and in-plane stride 1,
// k <= 2:
//
//   dx[n][ci][e](p) = sum_co sum_dz sum_t w[co][ci][dz][t] * dy[n][co][e + kz - dz](p - tap t)
//
// (dz = 0 .. 2kz indexes the planes -kz .. kz; in the plane the adjoint is
// the point-reflected kernel, t <-> T-1-t).  A block owns one band of rows
// of one sample and a range of dx planes [e_lo, e_hi).  It walks the dy
// planes d that reach those planes (d = e_lo - kz .. e_hi + kz - 1 inside
// the volume) in order and stages each one's window once, in groups of as
// many output channels as 64 KB of LDS hold, in the sheared layout of
// shear.h (a tap is a fixed offset).  A
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
// group is loaded into registers while the current one is computed.  One
// group ahead, and at most 8 staged window rows per thread (the block takes
// extra threads,
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
    int CC, nck;   // output channels staged at a time, such groups per plane
    int P, CS;     // sheared column pitch, floats per staged channel
    FastDiv fdlr;  // division by TR + 2K (window rows)
};

constexpr int kR3 = 2; // rows per thread: each weight read serves two outputs

template <typename TT, int K, int KZ, int CI, int U, bool GRP>
__global__ __launch_bounds__(kMaxThreads3) void bwd_data3d_smallc_k(
    const TT *__restrict__ dy, const TT *__restrict__ w, TT *__restrict__ dx, ConvShape sh,
    Bwd3Args a)
{
    constexpr int T = num_taps(K);
    constexpr int Z = 2 * KZ + 1;
    constexpr int R = kR3;
    static_assert(CI == 1 || CI == 2, "one or two input channels");
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

    // one group (the whole of C_out) compiled as a constant where it fits
    const int nck = GRP ? a.nck : 1, CC = GRP ? a.CC : Co;
    const ShearTile tl{r0 - K, -K, a.TR + 2 * K, W + 2 * K, a.P, a.CS};
    const int c = threadIdx.x % W, strip = threadIdx.x / W;
    const bool active = strip * R < rows; // threadIdx.x < W * ceil(TR / R)
    const int a0 = active ? tl.addr(r0 + strip * R, c) : 0;

    // dy plane d of output channels c0 .. c0 + CC - 1 (one staged "channel"
    // per output channel)
    const TT *img = dy + static_cast<size_t>(n) * Co * D * HW;
    auto load_group = [&](ShearPrefetch<U> &p, int d, int g) {
        if (d >= dhi) { // past the last step: reload it (never committed)
            d = dhi - 1;
            g = nck - 1;
        }
        const int c0 = g * CC;
        p.load3(img + static_cast<size_t>(c0) * D * HW, D * HW, HW,
                static_cast<long>(d) * static_cast<long>(HW), 1, 0, 1, min(CC, Co - c0), H, W,
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
            TT *dst = dx + ((static_cast<size_t>(n) * CI + ci) * D + e) * HW +
                      static_cast<size_t>(r0 + strip * R) * W + c;
#pragma unroll
            for (int r = 0; r < R; ++r)
                if (strip * R + r < rows)
                    dst[static_cast<size_t>(r) * W] = from_f<TT>(acc[0][ci][r]);
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

    // one group of output channels of dy plane d: stage it, request the
    // next group (or the next plane's first) into the same registers, add
    // its contributions to the ring; after the plane's last group retire
    // slot 0
    auto group_step = [&](ShearPrefetch<U> &p, int d, int g) {
        __syncthreads(); // the previous group's reads are done
        p.commit(ds3);
        __syncthreads();
        const bool last = g + 1 == nck;
        load_group(p, last ? d + 1 : d, last ? 0 : g + 1);
        const int c0 = g * CC, cn = min(CC, Co - c0);
        if (active) {
            // products of staged channel cl with its weights: wt(ci, m) is
            // value m of the Z T weights of (this output channel, ci)
            auto channel = [&](int cl, auto wt) __attribute__((always_inline)) {
                const float *src = ds3 + cl * a.CS + a0;
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
#pragma unroll
                                for (int s = 0; s < Z; ++s) {
                                    const float wv = wt(ci, s * T + (T - 1 - tr));
#pragma unroll
                                    for (int r = 0; r < R; ++r)
                                        acc[s][ci][r] += wv * v[r + u];
                                }
                            }
                        }
                    }
                    t0 += len;
                }
            };
            constexpr int L = CI * Z * T; // weights per output channel (odd for CI = 1)
            if constexpr (sizeof(TT) == sizeof(float)) {
                for (int cl = 0; cl < cn; ++cl) {
                    const float *w0 = w + static_cast<size_t>(c0 + cl) * L;
                    const float *w1 = w0 + (CI - 1) * Z * T;
                    channel(cl, [&](int ci, int m) { return (ci == 0 ? w0 : w1)[m]; });
                }
            } else {
                // bfloat16: output channels in pairs from an even one (c0 is
                // even), so that every weight is at a compile-time offset
                // from an even element and needs no select
                int cl = 0;
                for (; cl + 1 < cn; cl += 2) {
                    const WEven<TT> we(w, static_cast<uint32_t>((c0 + cl) * L));
                    channel(cl, [&](int ci, int m) { return we(ci * Z * T + m); });
                    channel(cl + 1, [&](int ci, int m) { return we(L + ci * Z * T + m); });
                }
                if (cl < cn) {
                    const WEven<TT> we(w, static_cast<uint32_t>((c0 + cl) * L));
                    channel(cl, [&](int ci, int m) { return we(ci * Z * T + m); });
                }
            }
        }
        if (last) {
            store_slot0(d - KZ);
            shift();
        }
    };

    // the ring starts at dx planes dlo - kz .. dlo + kz
    ShearPrefetch<U> pa;
    load_group(pa, dlo, 0);
    for (int d = dlo; d < dhi; ++d)
        for (int g = 0; g < nck; ++g)
            group_step(pa, d, g);
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
    int U, threads, grid;
    size_t lds;
    bool ok;
};

Bwd3Plan plan_bwd3(const ConvShape &sh)
{
    Bwd3Plan pl{};
    pl.ok = false;
    if (sh.s != 1 || sh.sz != 1 || (sh.k != 1 && sh.k != 2) || sh.kz > 2 ||
        (sh.Ci != 1 && sh.Ci != 2) || sh.W % 4 != 0 || sh.W > 256 || sh.N < 1)
        return pl;
    const int K = sh.k;
    Bwd3Args &a = pl.a;
    a.TR = 8; // rows per band
    if (sh.W * cdiv(a.TR, kR3) > kMaxThreads3)
        return pl;
    pl.threads = cdiv(sh.W * cdiv(a.TR, kR3), 64) * 64;
    a.nbands = cdiv(sh.H, a.TR);
    a.P = a.TR + 2 * K + 1;
    a.CS = (sh.W + 2 * K) * a.P;
    a.fdlr = make_fastdiv(static_cast<uint32_t>(a.TR + 2 * K));
    // output channels staged at a time: as many as the LDS budget holds,
    // balanced over the groups of a plane
    // (an even number when there are several groups: bfloat16 weights are
    // read for pairs of output channels from an even one)
    const size_t per_ch = sizeof(float) * static_cast<size_t>(a.CS);
    const int cmax = static_cast<int>(kLds3 / per_ch) & ~1;
    if (cmax < 2)
        return pl;
    a.nck = cdiv(sh.Co, cmax);
    a.CC = a.nck == 1 ? sh.Co : (cdiv(sh.Co, a.nck) + 1) & ~1;
    pl.lds = per_ch * a.CC;
    // staging rows per thread (ShearPrefetch): one 4-column group per thread
    const int groups = ShearPrefetch<1>::groups(sh.W + 2 * K);
    if (groups > pl.threads)
        return pl;
    // staging rows per thread: more threads (idle in the products) until a
    // thread stages at most 8 window rows (92 registers at k = 1, against
    // 143 for 12 rows)
    auto rows_per_thread = [&](int nt) {
        return cdiv(static_cast<long>(a.CC) * (a.TR + 2 * K), nt / groups);
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

template <typename TT, int K, int KZ, int CI>
hipError_t launch_bwd3_u(const Bwd3Plan &pl, const TT *dy, const TT *w, TT *dx,
                         const ConvShape &sh, hipStream_t st)
{
#define HEX_B3(UV)                                                                           \
    do {                                                                                     \
        if (pl.a.nck > 1)                                                                    \
            HEX_LAUNCH((bwd_data3d_smallc_k<TT, K, KZ, CI, UV, true>), dim3(pl.grid),        \
                       dim3(pl.threads), pl.lds, st, dy, w, dx, sh, pl.a);                   \
        else                                                                                 \
            HEX_LAUNCH((bwd_data3d_smallc_k<TT, K, KZ, CI, UV, false>), dim3(pl.grid),       \
                       dim3(pl.threads), pl.lds, st, dy, w, dx, sh, pl.a);                   \
    } while (0)
    if (pl.U == 4)
        HEX_B3(4);
    else if (pl.U == 8)
        HEX_B3(8);
    else
        HEX_B3(12);
#undef HEX_B3
    return hipGetLastError();
}

template <typename TT, int K, int KZ>
hipError_t launch_bwd3_k(const Bwd3Plan &pl, const TT *dy, const TT *w, TT *dx,
                         const ConvShape &sh, hipStream_t st)
{
    return sh.Ci == 1 ? launch_bwd3_u<TT, K, KZ, 1>(pl, dy, w, dx, sh, st)
                      : launch_bwd3_u<TT, K, KZ, 2>(pl, dy, w, dx, sh, st);
}

template <typename TT>
hipError_t launch_bwd3(const Bwd3Plan &pl, const TT *dy, const TT *w, TT *dx,
                       const ConvShape &sh, hipStream_t st)
{
    if (sh.k == 1) {
        if (sh.kz == 0)
            return launch_bwd3_k<TT, 1, 0>(pl, dy, w, dx, sh, st);
        if (sh.kz == 1)
            return launch_bwd3_k<TT, 1, 1>(pl, dy, w, dx, sh, st);
        return launch_bwd3_k<TT, 1, 2>(pl, dy, w, dx, sh, st);
    }
    if (sh.kz == 0)
        return launch_bwd3_k<TT, 2, 0>(pl, dy, w, dx, sh, st);
    if (sh.kz == 1)
        return launch_bwd3_k<TT, 2, 1>(pl, dy, w, dx, sh, st);
    return launch_bwd3_k<TT, 2, 2>(pl, dy, w, dx, sh, st);
}

} // namespace

bool smallc3d_bwd_data_ok(const ConvShape &sh) { return plan_bwd3(sh).ok; }

hipError_t smallc3d_bwd_data(const void *dy, const void *w, void *dx, const ConvShape &sh,
                             Dtype d, hipStream_t st)
{
    const Bwd3Plan pl = plan_bwd3(sh);
    if (!pl.ok)
        return hipErrorInvalidValue;
    if (d == F32)
        return launch_bwd3(pl, static_cast<const float *>(dy), static_cast<const float *>(w),
                           static_cast<float *>(dx), sh, st);
    return launch_bwd3(pl, static_cast<const bf16raw *>(dy), static_cast<const bf16raw *>(w),
                       static_cast<bf16raw *>(dx), sh, st);
}

} // namespace hexk
