// k_bwd_f32.hip -- both gradients of a float32 layer with few input
// channels (camera images) in one pass over dy.
//
//   dx[n][ci][p] = sum_co sum_t w[co][ci][T-1-t] * dy[n][co][p + tap t]
//   dw[co][ci][t] = sum_n sum_p dy[n][co][p] * x[n][ci][p + tap t]
//   db[co]        = sum_n sum_p dy[n][co][p]
// (stride 1: the data gradient is the convolution of dy with the
// point-reflected kernel, t <-> T-1-t).
//
// A tile is TR = 8 full-width rows of one image.  All C_out planes of dy and
// the C_in planes of x are staged into LDS in the sheared column-major layout
// (shear.h): element (r, c) of the window at (c - c_lo) * P + (r - r_lo) -
// (floor(c/2) - floor(c_lo/2)), P = TR + 2k + 1, so that a tap (dq, ds) is
// the parity-free offset dq * P + ds and a column is a run of consecutive
// words.  TR and k are compile-time constants, so every offset inside a tile
// is an instruction immediate.  The k halo columns are zeroed once per block;
// rows outside the image are staged as zeros.  The next tile's loads are in
// flight in registers while the current one is computed.
//
// Weight gradient on the fp32 matrix cores (v_mfma_f32_16x16x4f32,
// a = A[lane % 16][lane / 16], b = B[lane / 16][lane % 16]): M = output
// channels, N = (ci, t) plus a ones column for db, K = pixels, 4 consecutive
// rows of one column per step.  Lanes without a channel or a tap read from a
// plane of zeros, the bias column from a plane of ones, so the inner loop has
// no selects.  Accumulators stay in registers for the whole kernel; each
// block writes one partial sum per output element (reduced in a fixed order).
//
// Data gradient on the VALU: thread = (column, group of CG output channels),
// all TR rows of the column; each tap column (fixed dq) is a run of
// consecutive words, loaded once per channel and reused by all its taps.  The
// channel groups' partial sums are added in LDS in a fixed order.
#include <algorithm>
#include <type_traits>

#include "hexdev.h"
#include "kernels.h"
#include "shear.h" // FastDiv

namespace hexk {
namespace {

using namespace hexgeom;

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 512;   // 8 waves per block, one block per compute unit
constexpr int kDxThreads = 256; // waves 0-3: data gradient; waves 4-7: weight gradient
constexpr int kDwWaves = 4;
constexpr int kTR = 8;          // rows per tile

template <int K> struct Geo {
    static constexpr int LR = kTR + 2 * K; // window rows
    static constexpr int P = LR + 1;       // column pitch
    // word of window element (r_local = r - r0, c) relative to the channel
    // base: (c + K) * P + (r_local + K) - floor(c/2) + floor(-K/2)
    __host__ __device__ static constexpr int colbase(int c) { return (c + K) * P - (c >> 1) - 1; }
};

struct BwdTiling {
    int W4;            // float4 groups per row
    int CS;            // LDS words per x channel and per constant plane
    int CSD;           // LDS words per dy channel
    int xo, zo, oo;    // LDS offsets: x planes, zeros plane, ones plane
    int G;             // output-channel groups of the data gradient
    int CG;            // output channels per group (G * CG >= C_out)
    int tiles_per_img, ntiles;
    int per;           // tiles per block: block b walks tiles [b * per, b * per + per)
    int nitems;        // float4 staging items per tile
    int dxp;           // LDS offset of the data-gradient partials
    int wl;            // LDS offset of the reflected weights
    int dummy;         // LDS offset of a 4-word sink for dead staging items
    FastDiv fdw4, fdlr;
};

// Where the staging items of a thread go: item i = tid + u * kThreads is
// (channel, window row, float4 column group).  Its LDS word and its element
// offset inside the image do not depend on the tile, so they are computed
// once (pk: LDS word | window row << 16 | dy item << 24 | live << 25).
template <int K, int U> struct StageMap {
    int pk[U], goff[U];

    __device__ __forceinline__ void init(const ConvShape &sh, const BwdTiling &bt)
    {
        using G = Geo<K>;
        const int HW = sh.H * sh.W;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = threadIdx.x + u * kThreads;
            const int q = static_cast<int>(fdiv(static_cast<uint32_t>(i), bt.fdw4));
            const int c4 = i - q * bt.W4;
            const int ch = static_cast<int>(fdiv(static_cast<uint32_t>(q), bt.fdlr));
            const int rr = q - ch * G::LR;
            const bool live = i < bt.nitems;
            const bool isdy = ch < sh.Co;
            const int base = isdy ? ch * bt.CSD : bt.xo + (ch - sh.Co) * bt.CS;
            const int dst = live ? base + G::colbase(4 * c4) + rr : bt.dummy;
            pk[u] = dst | (rr << 16) | (isdy ? 1 << 24 : 0) | (live ? 1 << 25 : 0);
            goff[u] = (isdy ? ch : ch - sh.Co) * HW + rr * sh.W + 4 * c4;
        }
    }
};

// One tile's dy and x rows in registers, as loaded (4 elements per item:
// a float4, or 8 bytes of bf16).  Every load is issued (items outside the
// image read a valid address) and okm records which hold image data; the
// others are replaced by zeros when committed.  Loads that are always
// issued keep the count of loads in flight fixed, so a commit waits only
// for its own buffer.
template <typename TT, int U> struct StageBuf {
    typedef typename std::conditional<sizeof(TT) == 4, float4, uint2>::type Raw;
    Raw v[U];
    uint32_t okm;

    __device__ __forceinline__ static float4 widen(const float4 &q) { return q; }
    __device__ __forceinline__ static float4 widen(const uint2 &q)
    {
        return make_float4(__uint_as_float(q.x << 16), __uint_as_float(q.x & 0xffff0000u),
                           __uint_as_float(q.y << 16), __uint_as_float(q.y & 0xffff0000u));
    }

    template <int K>
    __device__ __forceinline__ void load(const StageMap<K, U> &m, const TT *__restrict__ x,
                                         const TT *__restrict__ dy, const ConvShape &sh, int n,
                                         int r0)
    {
        const size_t HW = static_cast<size_t>(sh.H) * sh.W;
        // row r0 - K of image n, channel 0: items add their offsets to it
        const long rofs = static_cast<long>(r0 - K) * sh.W;
        const TT *dyn = dy + static_cast<size_t>(n) * sh.Co * HW + rofs;
        const TT *xn = x + static_cast<size_t>(n) * sh.Ci * HW + rofs;
        const int rlo = K - r0, rhi = sh.H - r0 + K; // window rows inside the image
        okm = 0;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int rr = (m.pk[u] >> 16) & 0xff;
            const bool ok = ((m.pk[u] >> 25) & 1) && rr >= rlo && rr < rhi;
            const TT *b = ((m.pk[u] >> 24) & 1) ? dyn : xn;
            v[u] = *reinterpret_cast<const Raw *>(ok ? b + m.goff[u] : x);
            okm |= ok ? 1u << u : 0u;
        }
    }

    // columns 4c4 .. 4c4+3 of a row sit at +0, +P, +2P-1, +3P-1
    template <int K>
    __device__ __forceinline__ void commit(const StageMap<K, U> &m, float *__restrict__ lds) const
    {
        using G = Geo<K>;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const float4 q = ((okm >> u) & 1) ? widen(v[u]) : make_float4(0.f, 0.f, 0.f, 0.f);
            float *d = lds + (m.pk[u] & 0xffff);
            d[0] = q.x;
            d[G::P] = q.y;
            d[2 * G::P - 1] = q.z;
            d[3 * G::P - 1] = q.w;
        }
    }
};

// CGT: output channels per data-gradient group when fixed at compile time
// (the channel loop is then unrolled), 0 for a loop over bt.CG.
template <typename TT, int K, int CI, int MT, int NT, int CGT, int U>
__global__ __launch_bounds__(kThreads) void bwd_smallc_k(
    const TT *__restrict__ x, const TT *__restrict__ dy, const TT *__restrict__ w,
    TT *__restrict__ dx, float *__restrict__ part, ConvShape sh, BwdTiling bt, int do_dx)
{
    using Gm = Geo<K>;
    constexpr int T = num_taps(K);
    constexpr int J = CI * T; // tap columns; column J is the bias column
    constexpr int P = Gm::P;
    extern __shared__ __align__(16) float lds[];
    float *dxp = lds + bt.dxp; // [G][CI][TR][W]
    float *wl = lds + bt.wl;   // [C_out + 1][CI][T], reflected taps; row C_out = 0
    const int W = sh.W, Co = sh.Co;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const bool dxrole = wave < kDwWaves;

    // reflected weights (at most 3 per thread: (C_out + 1) * C_in * T <= 33 *
    // 38 < 3 * kThreads, from C_out <= 32 and C_in * T + 1 <= 64), read
    // before the tile loads so that waiting for them does not wait for the
    // tiles; without the data gradient w is not read (it may be NULL)
    const int nwl = (Co + 1) * CI * T;
    float wreg[3];
#pragma unroll
    for (int u = 0; u < 3; ++u) {
        const int e = tid + u * kThreads;
        const int co = e / (CI * T), rem = e - co * (CI * T);
        const int ci = rem / T, t = rem - ci * T;
        wreg[u] = (do_dx != 0 && e < nwl && co < Co)
                      ? to_f(w[(static_cast<size_t>(co) * CI + ci) * T + (T - 1 - t)])
                      : 0.f;
    }

    // the first two tiles' loads are in flight during the one-time set-up
    StageMap<K, U> map;
    map.init(sh, bt);
    StageBuf<TT, U> sa, sb;
    const int tpi = bt.tiles_per_img;
    // a contiguous run of tiles (consecutive row bands of one image): the
    // halo rows a tile shares with the previous one were fetched by this
    // block, so they come from this XCD's L2 rather than from HBM
    const int t_begin = blockIdx.x * bt.per;
    const int t_end = min(t_begin + bt.per, bt.ntiles);
    // Every step issues the same loads (a tile past this block's run reloads
    // its last one, from L2, and is never committed), so the wait before a
    // commit only covers the loads of that buffer and not the newer ones.
    auto load_tile = [&](StageBuf<TT, U> &b, int t) {
        t = min(t, t_end - 1);
        const int n = t / tpi;
        b.load(map, x, dy, sh, n, (t - n * tpi) * kTR);
    };
    // issued in this order (the scheduler may not swap them): the steady
    // state has the older buffer's loads first as well, so the waits before
    // a commit are the same on the loop's entry and back edge
    load_tile(sa, t_begin);
    __builtin_amdgcn_sched_barrier(0);
    load_tile(sb, t_begin + 1);
    __builtin_amdgcn_sched_barrier(0);

    // ---- data gradient role: thread = (channel group g, column c), all TR
    // rows of the column, CG output channels
    const bool dxthr = dxrole && do_dx != 0 && tid < bt.G * W;
    const int g = dxthr ? tid / W : 0;
    const int c = dxthr ? tid - g * W : 0;
    const int cbase = Gm::colbase(c) + K; // word of (row r0, column c)
    // ---- weight gradient role: operands of this lane (word offsets from a
    // pixel); lanes without a channel or a tap read a plane of zeros, the
    // bias column a plane of ones
    const int m = lane & 15, kq = lane >> 4;
    int abase[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
        abase[i] = i * 16 + m < Co ? (i * 16 + m) * bt.CSD : bt.zo;
    int bbase[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int col = j * 16 + m;
        bbase[j] = col == J ? bt.oo : bt.zo;
        if (col < J) {
            const int ci = col / T, t = col - ci * T;
            int dq = 0, ds = 0;
            tap_axial(K, t, dq, ds);
            bbase[j] = bt.xo + ci * bt.CS + dq * P + ds;
        }
    }
    // K-steps of this wave: pixel quads (column c0w + 2i, rows 4 * (dw & 1) + 0..3)
    const int dwv = wave - kDwWaves;
    const int c0w = (dwv >> 1) & 1;
    const int p0 = Gm::colbase(c0w) + K + 4 * (dwv & 1) + kq;
    constexpr int PSTEP = 2 * P - 1; // two columns further
    const int nsteps = (W - c0w + 1) / 2;
    floatx4 acc[2][MT][NT];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NT; ++j)
                acc[h][i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    auto kstep = [&](int i, int h) {
        const int pa = p0 + i * PSTEP;
        float a[MT], b[NT];
#pragma unroll
        for (int ii = 0; ii < MT; ++ii)
            a[ii] = lds[abase[ii] + pa];
#pragma unroll
        for (int j = 0; j < NT; ++j)
            b[j] = lds[bbase[j] + pa];
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
            for (int ii = 0; ii < MT; ++ii)
                acc[h][ii][j] =
                    __builtin_amdgcn_mfma_f32_16x16x4f32(a[ii], b[j], acc[h][ii][j], 0, 0, 0);
    };

    // once per block: zero halo columns of every channel, the zeros plane,
    // the ones plane, the reflected weights (no global load inside the tile
    // loop: it would wait for the prefetches issued before it)
    {
        const int nch = Co + CI;
        for (int e = tid; e < nch * 2 * K * Gm::LR; e += kThreads) {
            const int rr = e % Gm::LR, rest = e / Gm::LR;
            const int side = rest % (2 * K), ch = rest / (2 * K);
            const int cc = side < K ? side - K : W + side - K;
            const int base = ch < Co ? ch * bt.CSD : bt.xo + (ch - Co) * bt.CS;
            lds[base + Gm::colbase(cc) + rr] = 0.f;
        }
        for (int e = tid; e < bt.CS; e += kThreads) {
            lds[bt.zo + e] = 0.f;
            lds[bt.oo + e] = 1.f;
        }
#pragma unroll
        for (int u = 0; u < 3; ++u)
            if (tid + u * kThreads < nwl)
                wl[tid + u * kThreads] = wreg[u];
    }

    // One tile: stage it, start the loads of the tile two steps ahead into
    // the same registers, then the two roles work on the window at the same
    // time (VALU and matrix cores of each SIMD).  Rows past the image are
    // zeros, so a short last tile needs no masking.
    auto tile_step = [&](StageBuf<TT, U> &buf, int tile) {
        const int n = tile / tpi;
        const int r0 = (tile - n * tpi) * kTR;
        const int rows = min(kTR, sh.H - r0);
        buf.commit(map, lds);
        __syncthreads(); // tile staged (and, the first time, the constants)
        load_tile(buf, tile + 2);
        if (dxrole) {
            if (dxthr) {
                float gacc[CI][kTR];
#pragma unroll
                for (int ci = 0; ci < CI; ++ci)
#pragma unroll
                    for (int r = 0; r < kTR; ++r)
                        gacc[ci][r] = 0.f;
                // one output channel's contribution (all taps, all CI)
                auto chan = [&](int cc) {
                    // CGT >= bt.CG: groups of CGT still cover every channel once
                    const int co = g * (CGT > 0 ? CGT : bt.CG) + cc;
                    const bool ok = co < Co;
                    const float *src = lds + (ok ? co : 0) * bt.CSD + cbase;
                    const float *wc = wl + (ok ? co : Co) * CI * T;
                    int t0 = 0;
#pragma unroll
                    for (int dq = -K; dq <= K; ++dq) {
                        const int len = 2 * K + 1 - (dq < 0 ? -dq : dq);
                        const int dslo = dq < 0 ? -K - dq : -K;
                        const float *col = src + dq * P + dslo;
                        float v[kTR + 2 * K];
#pragma unroll
                        for (int j = 0; j < kTR + 2 * K; ++j)
                            if (j < kTR + len - 1)
                                v[j] = col[j];
#pragma unroll
                        for (int u = 0; u < 2 * K + 1; ++u) {
                            if (u < len) {
#pragma unroll
                                for (int ci = 0; ci < CI; ++ci) {
                                    const float wv = wc[ci * T + t0 + u];
#pragma unroll
                                    for (int r = 0; r < kTR; ++r)
                                        gacc[ci][r] += wv * v[r + u];
                                }
                            }
                        }
                        t0 += len;
                    }
                };
                if constexpr (CGT > 0) {
#pragma unroll
                    for (int cc = 0; cc < CGT; ++cc)
                        chan(cc);
                } else {
#pragma unroll 1
                    for (int cc = 0; cc < bt.CG; ++cc)
                        chan(cc);
                }
#pragma unroll
                for (int ci = 0; ci < CI; ++ci)
#pragma unroll
                    for (int r = 0; r < kTR; ++r)
                        dxp[((g * CI + ci) * kTR + r) * W + c] = gacc[ci][r];
            }
        } else {
            int i = 0;
            for (; i + 1 < nsteps; i += 2) {
                kstep(i, 0);
                kstep(i + 1, 1);
            }
            if (i < nsteps)
                kstep(i, 0);
        }
        __syncthreads(); // partials written; every read of the window done
        // dx: the groups' partials added in a fixed order, 16-byte stores.
        // Exactly CI stores per thread (CI * TR * W / 4 <= CI * kThreads for
        // W <= 256); a thread past the end repeats the last element's store
        // (same value, same address), so the count of stores in flight is
        // fixed and the loads issued before them are not waited for.
        if (do_dx != 0) {
            const int perp4 = rows * W / 4;
#pragma unroll
            for (int u = 0; u < CI; ++u) {
                const int e4 = min(tid + u * kThreads, CI * perp4 - 1);
                {
                    const int ci = e4 >= perp4 ? 1 : 0;
                    const int rem = 4 * (e4 - ci * perp4);
                    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
                    for (int gg = 0; gg < bt.G; ++gg) {
                        const float *q = dxp + (gg * CI + ci) * kTR * W + rem;
                        s.x += q[0];
                        s.y += q[1];
                        s.z += q[2];
                        s.w += q[3];
                    }
                    TT *dst = dx + (static_cast<size_t>(n) * CI + ci) * sh.H * W +
                              static_cast<size_t>(r0) * W + rem;
                    if constexpr (sizeof(TT) == 4) {
                        *reinterpret_cast<float4 *>(dst) = s;
                    } else {
                        *reinterpret_cast<uint2 *>(dst) = make_uint2(
                            from_f<bf16raw>(s.x) | (uint32_t(from_f<bf16raw>(s.y)) << 16),
                            from_f<bf16raw>(s.z) | (uint32_t(from_f<bf16raw>(s.w)) << 16));
                    }
                }
            }
        }
    };

    // two register buffers, so the loop is unrolled by two; no exit between
    // the two halves (a path from the first half back to the loop head would
    // make the waits before its commit cover the other buffer's loads)
    int tile = t_begin;
    for (; tile + 1 < t_end; tile += 2) {
        tile_step(sa, tile);
        tile_step(sb, tile + 1);
    }
    if (tile < t_end)
        tile_step(sa, tile);

    // sum the accumulator sets and the weight-gradient waves in a fixed
    // order; one partial per output element (chunked layout)
    __syncthreads();
    float *red = lds; // [kDwWaves][MT * 16][NT * 16]
    if (!dxrole) {
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NT; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    red[((dwv * MT + i) * 16 + 4 * kq + q) * (NT * 16) + j * 16 + m] =
                        acc[0][i][j][q] + acc[1][i][j][q];
    }
    __syncthreads();
    constexpr int Jt = J + 1;
    for (int e = tid; e < Co * Jt; e += kThreads) {
        const int row = e / Jt, col = e - row * Jt;
        float s = 0.f;
#pragma unroll
        for (int wv = 0; wv < kDwWaves; ++wv)
            s += red[(wv * MT * 16 + row) * (NT * 16) + col];
        part[part_index(e, blockIdx.x, gridDim.x)] = s;
    }
}

inline int cdiv(long a, long b) { return static_cast<int>((a + b - 1) / b); }

constexpr size_t kLdsMax = 160 * 1024;

int bwd_nt(const ConvShape &sh)
{
    const int nt = cdiv(sh.Ci * sh.T + 1, 16);
    return nt <= 1 ? 1 : (nt <= 2 ? 2 : 4);
}

BwdTiling bwd_tiling(const ConvShape &sh)
{
    BwdTiling bt;
    const int LR = kTR + 2 * sh.k, P = LR + 1, LC = sh.W + 2 * sh.k;
    bt.W4 = sh.W / 4;
    bt.CS = LC * P;
    // dy channel stride == 2 mod 32: the 16 channels x 4 rows of an A
    // fragment fall in distinct banks of each half-wave
    bt.CSD = (bt.CS + 29) / 32 * 32 + 2;
    bt.xo = sh.Co * bt.CSD;
    bt.zo = bt.xo + sh.Ci * bt.CS;
    bt.oo = bt.zo + bt.CS;
    bt.G = std::max(1, std::min(sh.Co, kDxThreads / sh.W));
    bt.CG = cdiv(sh.Co, bt.G);
    bt.tiles_per_img = cdiv(sh.H, kTR);
    bt.ntiles = bt.tiles_per_img * sh.N;
    bt.per = cdiv(bt.ntiles, std::max(1, device_cus()));
    bt.nitems = (sh.Co + sh.Ci) * LR * bt.W4;
    bt.dxp = bt.oo + bt.CS;
    bt.wl = bt.dxp + bt.G * sh.Ci * kTR * sh.W;
    bt.dummy = bt.wl + (sh.Co + 1) * sh.Ci * sh.T;
    bt.fdw4 = make_fastdiv(static_cast<uint32_t>(bt.W4));
    bt.fdlr = make_fastdiv(static_cast<uint32_t>(LR));
    return bt;
}

int bwd_u(const BwdTiling &bt) { return cdiv(bt.nitems, kThreads); }

// register buffers per dtype: fp32 items are 16 bytes, bf16 items 8
int bwd_umax(Dtype d) { return d == F32 ? 8 : 12; }

size_t bwd_lds(const ConvShape &sh, const BwdTiling &bt)
{
    const int P = kTR + 2 * sh.k + 1;
    const size_t main = sizeof(float) * (static_cast<size_t>(bt.dummy) + 3 * P + 1);
    const size_t red = sizeof(float) * kDwWaves * cdiv(sh.Co, 16) * 16 * bwd_nt(sh) * 16;
    return std::max(main, red);
}

// Persistent grid: at most one block per compute unit, each walking a
// contiguous run of tiles (bt.per of them).
int bwd_grid(const BwdTiling &bt) { return cdiv(bt.ntiles, bt.per); }

template <typename TT, int K, int CI, int NT>
void launch_bwd(int MT, int U, const BwdTiling &bt, const ConvShape &sh, size_t lds,
                hipStream_t st, const TT *x, const TT *dy, const TT *w, TT *dx, float *part,
                int do_dx)
{
    const dim3 grid(bwd_grid(bt));
#define HEX_B2(MTV, CGV, UV)                                                                  \
    HEX_LAUNCH((bwd_smallc_k<TT, K, CI, MTV, NT, CGV, UV>), grid, dim3(kThreads), lds, st, x, dy, \
               w, dx, part, sh, bt, do_dx)
    // fp32 (the camera layers) unrolls channel groups of 2, 3 or 4
#define HEX_B(MTV, UV)                                                                        \
    do {                                                                                     \
        if constexpr (sizeof(TT) == 4) {                                                     \
            if (bt.CG <= 2) HEX_B2(MTV, 2, UV);                                              \
            else if (bt.CG == 3) HEX_B2(MTV, 3, UV);                                         \
            else if (bt.CG == 4) HEX_B2(MTV, 4, UV);                                         \
            else HEX_B2(MTV, 0, UV);                                                         \
        } else {                                                                             \
            HEX_B2(MTV, 0, UV);                                                              \
        }                                                                                    \
    } while (0)
#define HEX_B_U(MTV)                                                                          \
    do {                                                                                     \
        if (U <= 4) {                                                                        \
            HEX_B(MTV, 4);                                                                   \
        } else if (U <= 8) {                                                                 \
            HEX_B(MTV, 8);                                                                   \
        } else {                                                                             \
            if constexpr (sizeof(TT) == 2)                                                   \
                HEX_B(MTV, 12);                                                              \
        }                                                                                    \
    } while (0)
    if (MT == 1)
        HEX_B_U(1);
    else
        HEX_B_U(2);
#undef HEX_B_U
#undef HEX_B
#undef HEX_B2
}

template <typename TT>
hipError_t bwd_fused_t(const TT *x, const TT *dy, const TT *w, TT *dx, float *dw, float *db,
                       void *ws, const ConvShape &sh, hipStream_t st)
{
    const BwdTiling bt = bwd_tiling(sh);
    const int nparts = bwd_grid(bt);
    const int MT = cdiv(sh.Co, 16);
    const int U = bwd_u(bt);
    float *part = static_cast<float *>(ws);
    const size_t lds = bwd_lds(sh, bt);
    const int do_dx = dx != nullptr ? 1 : 0;
    if (sh.k == 1) {
        if (sh.Ci == 1)
            launch_bwd<TT, 1, 1, 1>(MT, U, bt, sh, lds, st, x, dy, w, dx, part, do_dx); // J + 1 = 8
        else
            launch_bwd<TT, 1, 2, 1>(MT, U, bt, sh, lds, st, x, dy, w, dx, part, do_dx); // 15
    } else if (sh.k == 2) {
        if (sh.Ci == 1)
            launch_bwd<TT, 2, 1, 2>(MT, U, bt, sh, lds, st, x, dy, w, dx, part, do_dx); // 20
        else
            launch_bwd<TT, 2, 2, 4>(MT, U, bt, sh, lds, st, x, dy, w, dx, part, do_dx); // 39
    } else {
        launch_bwd<TT, 3, 1, 4>(MT, U, bt, sh, lds, st, x, dy, w, dx, part, do_dx); // 38
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    return reduce_chunked(part, nparts, sh.Co, sh.Ci * sh.T, dw, db, st);
}

} // namespace

bool smallc_bwd_fused_ok(const ConvShape &sh, Dtype d)
{
    if (sh.s != 1 || sh.k < 1 || sh.k > 3 || sh.Ci > 2 || sh.Co > 32 || sh.W % 4 != 0 ||
        sh.W > kDxThreads || sh.Ci * sh.T + 1 > 64)
        return false;
    const BwdTiling bt = bwd_tiling(sh);
    return bt.CG <= 8 && bwd_u(bt) <= bwd_umax(d) && bwd_lds(sh, bt) <= kLdsMax;
}

size_t smallc_bwd_fused_workspace(const ConvShape &sh)
{
    const BwdTiling bt = bwd_tiling(sh);
    return sizeof(float) * static_cast<size_t>(bwd_grid(bt)) * kPartChunk *
           part_chunks(sh.Co * (sh.Ci * sh.T + 1));
}

hipError_t smallc_bwd_fused(const void *x, const void *dy, const void *w, void *dx, float *dw,
                            float *db, void *ws, const ConvShape &sh, Dtype d, hipStream_t st)
{
    if (d == F32)
        return bwd_fused_t(static_cast<const float *>(x), static_cast<const float *>(dy),
                           static_cast<const float *>(w), static_cast<float *>(dx), dw, db, ws,
                           sh, st);
    return bwd_fused_t(static_cast<const bf16raw *>(x), static_cast<const bf16raw *>(dy),
                       static_cast<const bf16raw *>(w), static_cast<bf16raw *>(dx), dw, db, ws, sh,
                       st);
}

} // namespace hexk
