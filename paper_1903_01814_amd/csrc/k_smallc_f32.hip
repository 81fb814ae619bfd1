// k_smallc_f32.hip -- float32-arithmetic kernels for few input channels at
// stride 1 (camera images: C_in*T <= 64); the data is float32 or bfloat16
// (converted while it is staged, results rounded when they are stored).
//
// All three kernels stage their input tile (all channels, one batched pass)
// into the sheared LDS layout of shear.h, where a hexagonal tap (dq, ds) is
// the constant offset dq*P + ds from its centre for both column parities.
// The forward and weight-gradient kernels are persistent: each block walks a
// strided list of tiles and loads the next tile's input into registers while
// it computes and stores the current one (weights are loaded once).
//
// Forward: implicit GEMM on the fp32 matrix cores.  For 16 consecutive
// pixels of a tile, D[pixel][co] = sum_k A[pixel][k] * B[k][co] with
// k = (ci, tap): A is read from LDS at centre + offset(k), B (weights) stays
// in registers.  v_mfma_f32_16x16x4_f32 lane layout:
//   a = A[lane % 16][lane / 16], b = B[lane / 16][lane % 16],
//   d[j] = D[4 * (lane / 16) + j][lane % 16],
// so each lane stores 4 consecutive pixels of one channel (16-byte store).
//
// Backward-data: at stride 1 the adjoint is a forward convolution of dy
// with the point-reflected kernel (tap t <-> T-1-t) and C_in/C_out swapped.
// With one or two output channels it is a matrix-vector product, so it runs
// on the VALU: each thread owns R consecutive rows of one column; the
// neighbourhood columns are contiguous runs in the sheared layout, read
// once per input channel and reused by all taps of that column.  The
// weights are block-uniform and come by scalar loads (bfloat16 ones as
// aligned 32-bit words, hexdev.h).
//
// Weight gradient: D[co][(ci,t)] = sum_pixels dy[co][p] * x[ci][p + tap t]
// on the fp32 matrix cores with the pixels as the contraction index, so the
// reduction over pixels happens inside the MFMA; an extra B column of ones
// yields db.  Per-block partial sums are written to the workspace and added
// in a fixed order by k_reduce.hip (deterministic).
#include <algorithm>

#include "hexdev.h"
#include "kernels.h"
#include "shear.h"

namespace hexk {
namespace {

using namespace hexgeom;

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kFwdMT = 5; // 16-pixel M-tiles per wave and forward tile (tiles <= 320 pixels)

// Blocks are handed to the 8 XCDs round-robin; give each XCD a contiguous
// range of tiles so neighbouring tiles (shared halo rows) meet in one L2.
__device__ __forceinline__ int xcd_remap(int b, int nb)
{
    constexpr int X = 8;
    const int per = nb / X, rem = nb % X;
    const int xcd = b % X, idx = b / X;
    return xcd * per + min(xcd, rem) + idx;
}

// Tiling of the output plane (= input plane at stride 1) into TR x TW tiles.
struct Tiling {
    int TR, TW, tiles_c, tiles_per_img, ntiles, P, CS;
    FastDiv fdw;  // division by TW
    FastDiv fdtr; // division by TR
    FastDiv fdlr; // division by TR + 2k (staged window rows)
};

struct TileOrigin {
    int n, r0, c0, rows, cols;
};

__device__ __forceinline__ TileOrigin tile_of(int b, const Tiling &tg, const ConvShape &sh)
{
    TileOrigin o;
    o.n = b / tg.tiles_per_img;
    const int tt = b - o.n * tg.tiles_per_img;
    const int tr = tt / tg.tiles_c;
    o.r0 = tr * tg.TR;
    o.c0 = (tt - tr * tg.tiles_c) * tg.TW;
    o.rows = min(tg.TR, sh.H - o.r0);
    o.cols = min(tg.TW, sh.W - o.c0);
    return o;
}

__device__ __forceinline__ ShearTile window_of(const TileOrigin &o, const Tiling &tg, int K)
{
    return ShearTile{o.r0 - K, o.c0 - K, o.rows + 2 * K, o.cols + 2 * K, tg.P, tg.CS};
}

// Row-major copy of a tile of `nch` planes (no halo) staged through
// registers: dst[ch * dstride + pr * TW + pc].  Work split: one 4-column group
// per thread, (channel, row) pairs strided by blockDim / groups.  Requires
// W % 4 == 0 (so TW, the tile's columns and every group of 4 lie inside the
// row): each item is one 16-byte (fp32) or 8-byte (bf16) load and, dstride
// being even, two 8-byte LDS writes.
template <int U> struct PlainPrefetch {
    float v[U][4];
    int da[U];

    __host__ __device__ static int groups(int TW) { return (TW + 3) / 4; }
    __host__ __device__ static int rows_per_thread(int nch, int TR, int TW, int nt)
    {
        const int rstep = nt / groups(TW);
        return rstep > 0 ? (nch * TR + rstep - 1) / rstep : 1 << 30;
    }

    template <typename T>
    __device__ __forceinline__ void load(const T *__restrict__ src, size_t src_plane, int nch,
                                         int W, const TileOrigin &o, int TW, int dstride,
                                         const FastDiv &fdtr, int TR)
    {
        const int ng = groups(TW);
        const int rstep = blockDim.x / ng;
        const int g = threadIdx.x % ng, fr0 = threadIdx.x / ng;
        const int pc = 4 * g;
        const int total = nch * TR;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int fr = fr0 + u * rstep;
            const int ch = static_cast<int>(fdiv(static_cast<uint32_t>(fr), fdtr));
            const int pr = fr - ch * TR;
            const bool ok = fr0 < rstep && fr < total && pr < o.rows && pc < o.cols;
            da[u] = ok ? ch * dstride + pr * TW + pc : -1;
            // items without data read the plane's first group (always valid)
            const T *p =
                src + (ok ? ch * src_plane + static_cast<size_t>(o.r0 + pr) * W + o.c0 + pc : 0);
            Vec4Load<T>::load(p, v[u]);
        }
    }

    __device__ __forceinline__ void commit(float *__restrict__ dst) const
    {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (da[u] >= 0) {
                *reinterpret_cast<float2 *>(dst + da[u]) = make_float2(v[u][0], v[u][1]);
                *reinterpret_cast<float2 *>(dst + da[u] + 2) = make_float2(v[u][2], v[u][3]);
            }
        }
    }
};

// --------------------------------------------------------------- forward

// D3: three-dimensional layer.  A tile's "image" index then runs over
// (sample, output plane) pairs (sh.N = samples x output planes here), and
// the staged channels are the 2 kz + 1 planes around the centre plane of
// every input channel (ch = ci * Z + dz), so the contraction runs over
// (ci, dz, t) -- exactly the order of w[C_out][C_in][2kz+1][T].
template <typename TT, int K, int KS, int U, bool D3>
__global__ __launch_bounds__(kThreads) void fwd_smallc_k(
    const TT *__restrict__ x, const TT *__restrict__ w, const TT *__restrict__ bias,
    TT *__restrict__ y, ConvShape sh, int relu, Tiling tg)
{
    // W % 4 == 0 (smallc_fwd_ok): every 4-pixel group of a tile row is whole
    constexpr int T = num_taps(K);
    extern __shared__ float xs[];
    const int NCH = D3 ? sh.Ci * sh.Z : sh.Ci; // staged channels
    float *wt = xs + NCH * tg.CS; // [16][NCH * T + 1]: this block's weights, bias last
    const size_t HW = static_cast<size_t>(sh.H) * sh.W;
    const int J = NCH * T;

    // input channel 0 of the tile's sample, the output plane's index, and the
    // staging of a tile's window (all planes around the output plane)
    auto stage = [&](ShearPrefetch<U> &p, const TileOrigin &o) {
        if constexpr (D3) {
            const int n = o.n / sh.Do, dd = o.n - n * sh.Do;
            const int d0 = dd * sh.sz - sh.kz; // plane of dz = 0
            p.load3(x + static_cast<size_t>(n) * sh.Ci * sh.D * HW, sh.D * HW, HW,
                    static_cast<long>(d0) * static_cast<long>(HW), sh.Z, max(0, -d0),
                    min(sh.Z, sh.D - d0), NCH, sh.H, sh.W, window_of(o, tg, K), tg.TR + 2 * K,
                    tg.fdlr);
        } else {
            p.load(x + static_cast<size_t>(o.n) * sh.Ci * HW, HW, sh.Ci, sh.H, sh.W,
                   window_of(o, tg, K), tg.TR + 2 * K, tg.fdlr);
        }
    };
    // first element of output plane (sample, channel co, plane) of a tile
    auto out_plane = [&](const TileOrigin &o, int co) -> size_t {
        if constexpr (D3) {
            const int n = o.n / sh.Do, dd = o.n - n * sh.Do;
            return ((static_cast<size_t>(n) * sh.Co + co) * sh.Do + dd) * HW;
        } else {
            return (static_cast<size_t>(o.n) * sh.Co + co) * HW;
        }
    };

    // the first tile's loads are in flight while the weights are staged
    ShearPrefetch<U> pf;
    int t = blockIdx.x;
    if (t < tg.ntiles)
        stage(pf, tile_of(t, tg, sh));

    // The block's weights (16 output channels) and biases: one coalesced
    // pass into LDS.  Every block reads the same few lines, so per-lane
    // gathers from global memory would queue on them.
    for (int e = threadIdx.x; e < 16 * (J + 1); e += blockDim.x) {
        const int r = e / (J + 1), col = e - r * (J + 1);
        const int cog = blockIdx.y * 16 + r;
        float v = 0.f;
        if (cog < sh.Co)
            v = col < J ? to_f(w[static_cast<size_t>(cog) * J + col])
                        : (bias != nullptr ? to_f(bias[cog]) : 0.f);
        wt[e] = v;
    }

    // per-lane tap offsets
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int m = lane & 15, kq = lane >> 4;
    const int co = blockIdx.y * 16 + m; // B and D column of this lane
    int off[KS]; // LDS offset of k from the centre (may be negative)
    bool kval[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const int kk = kq + 4 * s;
        off[s] = 0;
        kval[s] = kk < J;
        if (kval[s]) {
            const int ci = kk / T, tap = kk - ci * T;
            int dq = 0, ds = 0;
            tap_axial(K, tap, dq, ds);
            off[s] = ci * tg.CS + dq * tg.P + ds;
        }
    }

    // The pixel slots of this lane's M-tiles (mt = wave + kWaves * i; tiles
    // hold at most kFwdMT * kWaves * 16 slots) do not depend on the tile:
    // window address of the A row (its sheared offset is the same for every
    // tile, the column origin being even), the slot's row and column, and
    // the output offset of the lane's four D rows.  Computed once, so the
    // products of a tile are LDS reads, matrix-core steps and stores.
    const int Kh = (-K) >> 1; // floor(-K / 2)
    const int cen0 = K * tg.P + K + Kh; // slot (0, 0)
    int cen[kFwdMT], prc[kFwdMT], qoff[kFwdMT], qrc[kFwdMT];
#pragma unroll
    for (int i = 0; i < kFwdMT; ++i) {
        const int mt = wave + kWaves * i;
        const int p = mt * 16 + m;
        const int pr = static_cast<int>(fdiv(p, tg.fdw));
        const int pc = p - pr * tg.TW;
        cen[i] = (pc + K) * tg.P + pr + K - ((pc >> 1) - Kh);
        prc[i] = (pr << 16) | pc;
        const int q0 = mt * 16 + 4 * kq;
        const int qr = static_cast<int>(fdiv(q0, tg.fdw));
        const int qc = q0 - qr * tg.TW;
        qoff[i] = qr * sh.W + qc;
        qrc[i] = (qr << 16) | qc;
    }

    float bw[KS], bco = 0.f;
    bool have_w = false;
    for (; t < tg.ntiles; t += gridDim.x) {
        const TileOrigin o = tile_of(t, tg, sh);
        __syncthreads(); // previous tile's reads of xs are done (and the weights staged)
        if (!have_w) {
#pragma unroll
            for (int s = 0; s < KS; ++s)
                bw[s] = kval[s] ? wt[m * (J + 1) + kq + 4 * s] : 0.f;
            bco = wt[m * (J + 1) + J];
            have_w = true;
        }
        pf.commit(xs);
        __syncthreads();
        const int tn = t + gridDim.x;
        if (tn < tg.ntiles)
            stage(pf, tile_of(tn, tg, sh));

        const int ntile = (o.rows * tg.TW + 15) / 16;
        TT *yb = y + out_plane(o, co) + static_cast<size_t>(o.r0) * sh.W + o.c0;
#pragma unroll
        for (int i = 0; i < kFwdMT; ++i) {
            if (wave + kWaves * i >= ntile) // wave-uniform
                break;
            // A row: slots outside the tile read the taps of slot 0, inside
            // the window (their results are not stored); K columns past the
            // taps (off = 0) are replaced by 0
            const bool pv = (prc[i] >> 16) < o.rows && (prc[i] & 0xffff) < o.cols;
            const int ca = pv ? cen[i] : cen0;
            float a[KS];
#pragma unroll
            for (int s = 0; s < KS; ++s)
                a[s] = xs[ca + off[s]];
            floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < KS; ++s)
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(kval[s] ? a[s] : 0.f, bw[s], acc, 0,
                                                           0, 0);
            // D rows of this lane: slots q0..q0+3, one tile row (TW % 4 == 0,
            // and W % 4 == 0 puts all four inside the tile or none)
            if (co >= sh.Co || (qrc[i] >> 16) >= o.rows || (qrc[i] & 0xffff) >= o.cols)
                continue;
            float v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                v[j] = acc[j] + bco;
                if (relu)
                    v[j] = fmaxf(v[j], 0.f);
            }
            TT *dst = yb + qoff[i];
            if constexpr (sizeof(TT) == 4) {
                *reinterpret_cast<float4 *>(dst) = make_float4(v[0], v[1], v[2], v[3]);
            } else {
                const uint32_t lo = from_f<bf16raw>(v[0]) | (uint32_t(from_f<bf16raw>(v[1])) << 16);
                const uint32_t hi = from_f<bf16raw>(v[2]) | (uint32_t(from_f<bf16raw>(v[3])) << 16);
                *reinterpret_cast<uint2 *>(dst) = make_uint2(lo, hi);
            }
        }
    }
}

// --------------------------------------------------------- backward-data

// dx[n][oc][p] = sum_ic sum_u w[ic][oc][T-1-u] * dy[n][ic][p + tap u]
// (ic runs over C_out, oc over C_in).  Thread = column c, rows
// [strip*R, strip*R + R) of the tile; one output channel per block.
template <typename TT, int K, int R>
__global__ __launch_bounds__(kThreads) void bwd_data_f32_k(
    const TT *__restrict__ dy, const TT *__restrict__ w, TT *__restrict__ dx, ConvShape sh,
    Tiling tg, int ic_chunk, int vec4)
{
    constexpr int T = num_taps(K);
    extern __shared__ float ds_[];
    const TileOrigin o = tile_of(xcd_remap(blockIdx.x, gridDim.x), tg, sh);
    const ShearTile tl = window_of(o, tg, K);
    const int cs = tl.chan_stride();
    const int oc = blockIdx.y;
    const int ICN = sh.Co, OCN = sh.Ci;
    const size_t HW = static_cast<size_t>(sh.H) * sh.W;

    const int lc = threadIdx.x % tg.TW, strip = threadIdx.x / tg.TW;
    const int S = tg.TR / R;
    const bool active = strip < S && lc < o.cols && strip * R < o.rows;
    // centre address of the strip's first row (valid for active threads)
    const int a0 = active ? tl.addr(o.r0 + strip * R, o.c0 + lc) : 0;

    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r)
        acc[r] = 0.f;

    for (int ic0 = 0; ic0 < ICN; ic0 += ic_chunk) {
        const int icn = min(ic_chunk, ICN - ic0);
        if (ic0 > 0)
            __syncthreads();
        stage_shear<8>(ds_, dy + (static_cast<size_t>(o.n) * ICN + ic0) * HW, HW, icn, sh.H,
                       sh.W, tl, tg.TR + 2 * K, tg.fdlr, vec4 != 0);
        __syncthreads();
        if (!active)
            continue;
        for (int icl = 0; icl < icn; ++icl) {
            const int ic = ic0 + icl;
            const typename WRow<TT>::type wr(w, static_cast<uint32_t>((ic * OCN + oc) * T));
            const float *src = ds_ + icl * cs + a0;
            int t0 = 0;
#pragma unroll
            for (int dq = -K; dq <= K; ++dq) {
                const int len = 2 * K + 1 - (dq < 0 ? -dq : dq);
                const int dslo = dq < 0 ? -K - dq : -K;
                const float *col = src + dq * tg.P + dslo;
                float v[R + 2 * K];
#pragma unroll
                for (int j = 0; j < R + 2 * K; ++j)
                    if (j < R + len - 1)
                        v[j] = col[j];
#pragma unroll
                for (int u = 0; u < 2 * K + 1; ++u) {
                    if (u < len) {
                        const float wv = wr(T - 1 - (t0 + u));
#pragma unroll
                        for (int r = 0; r < R; ++r)
                            acc[r] += wv * v[r + u];
                    }
                }
                t0 += len;
            }
        }
    }
    if (!active)
        return;
    TT *dst = dx + (static_cast<size_t>(o.n) * OCN + oc) * HW + o.c0 + lc;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int row = strip * R + r;
        if (row < o.rows)
            dst[static_cast<size_t>(o.r0 + row) * sh.W] = from_f<TT>(acc[r]);
    }
}

// -------------------------------------------------------- weight gradient

// D3: three-dimensional layer, tiles over (sample, output plane) pairs with
// the 2kz + 1 input planes around each output plane staged as channels
// (ch = ci * Z + dz), so that column (ch, t) is dw[co][ci][dz][t].
template <typename TT, int K, int NT, int UX, int UD, bool D3>
__global__ __launch_bounds__(kThreads) void wgrad_f32_k(
    const TT *__restrict__ x, const TT *__restrict__ dy, float *__restrict__ part, ConvShape sh,
    Tiling tg, int dstride)
{
    constexpr int T = num_taps(K);
    extern __shared__ float lds[];
    const int b = blockIdx.x; // partial slot
    const int NCH = D3 ? sh.Ci * sh.Z : sh.Ci; // staged x channels
    float *xs = lds;                      // [NCH][CS]
    float *dys = xs + NCH * tg.CS;        // [16][dstride], pitch TW
    float *red = dys + 16 * dstride;      // [kWaves][16][NT * 16]
    const int mt = blockIdx.y;            // 16 output channels
    const int nco = min(16, sh.Co - mt * 16);
    const size_t HW = static_cast<size_t>(sh.H) * sh.W;

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int m = lane & 15, kq = lane >> 4;
    const int J = NCH * T; // tap columns; column J is the bias column
    int off[NT];  // LDS offset of the tap from the centre (may be negative)
    int kind[NT]; // 0: tap column, 1: ones (bias column), 2: unused
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int col = j * 16 + m;
        off[j] = 0;
        kind[j] = col < J ? 0 : (col == J ? 1 : 2);
        if (col < J) {
            const int ci = col / T, t = col - ci * T;
            int dq = 0, ds = 0;
            tap_axial(K, t, dq, ds);
            off[j] = ci * tg.CS + dq * tg.P + ds;
        }
    }
    const bool arow = m < nco; // A row (output channel) present

    floatx4 acc[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j)
        acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};

    ShearPrefetch<UX> px;
    PlainPrefetch<UD> pd;
    // a tile's x window (every plane around its output plane) and dy rows
    auto stage = [&](const TileOrigin &o) {
        if constexpr (D3) {
            const int n = o.n / sh.Do, dd = o.n - n * sh.Do;
            const int d0 = dd * sh.sz - sh.kz;
            px.load3(x + static_cast<size_t>(n) * sh.Ci * sh.D * HW, sh.D * HW, HW,
                     static_cast<long>(d0) * static_cast<long>(HW), sh.Z, max(0, -d0),
                     min(sh.Z, sh.D - d0), NCH, sh.H, sh.W, window_of(o, tg, K), tg.TR + 2 * K,
                     tg.fdlr);
            pd.load(dy + ((static_cast<size_t>(n) * sh.Co + mt * 16) * sh.Do + dd) * HW,
                    sh.Do * HW, nco, sh.W, o, tg.TW, dstride, tg.fdtr, tg.TR);
        } else {
            px.load(x + static_cast<size_t>(o.n) * sh.Ci * HW, HW, sh.Ci, sh.H, sh.W,
                    window_of(o, tg, K), tg.TR + 2 * K, tg.fdlr);
            pd.load(dy + (static_cast<size_t>(o.n) * sh.Co + mt * 16) * HW, HW, nco, sh.W, o,
                    tg.TW, dstride, tg.fdtr, tg.TR);
        }
    };
    // this lane's first pixel slot (K-step ks = wave) and its row and
    // column in the tile; later K-steps move 16 slots on.  Window addresses
    // are relative to the tile's window, the same for every tile (the
    // column origin is even).
    const int Kh = (-K) >> 1; // floor(-K / 2)
    const int p_first = wave * 4 + kq;
    const int pr_first = static_cast<int>(fdiv(p_first, tg.fdw));
    const int pc_first = p_first - pr_first * tg.TW;
    int t = b;
    if (t < tg.ntiles)
        stage(tile_of(t, tg, sh));
    for (; t < tg.ntiles; t += gridDim.x) {
        const TileOrigin o = tile_of(t, tg, sh);
        __syncthreads();
        px.commit(xs);
        pd.commit(dys);
        __syncthreads();
        const int tn = t + gridDim.x;
        if (tn < tg.ntiles)
            stage(tile_of(tn, tg, sh));
        const int nslot = o.rows * tg.TW;
        const int nks = (nslot + 3) / 4;
        int p = p_first, pr = pr_first, pc = pc_first;
        for (int ks = wave; ks < nks; ks += kWaves) {
            const bool pv = pr < o.rows && pc < o.cols;
            // reads issued unconditionally (clamped addresses), then masked
            float a = dys[(pv && arow) ? m * dstride + p : 0];
            a = (pv && arow) ? a : 0.f;
            const int centre = pv ? (pc + K) * tg.P + pr + K - ((pc >> 1) - Kh) : 0;
            float bx[NT];
#pragma unroll
            for (int j = 0; j < NT; ++j)
                bx[j] = xs[(pv && kind[j] == 0) ? centre + off[j] : 0];
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                const float bv = !pv ? 0.f : (kind[j] == 0 ? bx[j] : (kind[j] == 1 ? 1.f : 0.f));
                acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bv, acc[j], 0, 0, 0);
            }
            p += 4 * kWaves;
            pc += 4 * kWaves;
            while (pc >= tg.TW) {
                pc -= tg.TW;
                ++pr;
            }
        }
    }
    // sum the waves' D tiles in a fixed order, write this block's partial
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q)
            red[(wave * 16 + 4 * kq + q) * (NT * 16) + j * 16 + m] = acc[j][q];
    __syncthreads();
    const int Jt = J + 1;
    for (int e = threadIdx.x; e < 16 * Jt; e += kThreads) {
        const int row = e / Jt, col = e - row * Jt;
        float s = 0.f;
        for (int wv = 0; wv < kWaves; ++wv)
            s += red[(wv * 16 + row) * (NT * 16) + col];
        const int cog = mt * 16 + row;
        if (row < nco)
            part[(static_cast<size_t>(cog) * Jt + col) * gridDim.x + b] = s;
    }
}

inline int cdiv(long a, long b) { return static_cast<int>((a + b - 1) / b); }

constexpr size_t kLdsLimit = 64 * 1024;

// sheared column stride for a window of LR rows
int shear_pitch(int LR) { return LR + 1; }

// Output tiles: full rows when W <= 128, else 128-column tiles; about
// `target` pixels per block.
Tiling make_tiling(const ConvShape &sh, int target)
{
    Tiling tg;
    tg.TW = std::min(sh.W, 128);
    tg.TW = (tg.TW + 3) / 4 * 4; // 16-byte aligned rows within the tile
    tg.TR = std::max(1, std::min(sh.H, target / tg.TW));
    tg.tiles_c = cdiv(sh.W, tg.TW);
    tg.tiles_per_img = tg.tiles_c * cdiv(sh.H, tg.TR);
    tg.ntiles = tg.tiles_per_img * sh.N;
    tg.P = shear_pitch(tg.TR + 2 * sh.k);
    tg.CS = (tg.TW + 2 * sh.k) * tg.P;
    tg.fdw = make_fastdiv(static_cast<uint32_t>(tg.TW));
    tg.fdtr = make_fastdiv(static_cast<uint32_t>(tg.TR));
    tg.fdlr = make_fastdiv(static_cast<uint32_t>(tg.TR + 2 * sh.k));
    return tg;
}

size_t shear_bytes(const ConvShape &sh, const Tiling &tg, int nch)
{
    return sizeof(float) * static_cast<size_t>(nch) * (tg.TW + 2 * sh.k) * tg.P;
}

// staged input window plus the block's weights and biases
size_t fwd_lds(const ConvShape &sh, const Tiling &tg)
{
    const int nch = sh.Ci * sh.Z; // staged channels (planes around the centre in 3-D)
    return shear_bytes(sh, tg, nch) + sizeof(float) * 16 * (nch * sh.T + 1);
}

// The forward tiles (sample, output plane) pairs as images: a 2-D layer has
// one plane per sample.
ConvShape fwd_view(const ConvShape &sh)
{
    ConvShape e = sh;
    e.N = sh.N * sh.Do;
    return e;
}

int wgrad_nt(const ConvShape &sh)
{
    const int NT = cdiv(sh.Ci * sh.Z * sh.T + 1, 16);
    return NT <= 1 ? 1 : (NT <= 2 ? 2 : 4);
}

int wgrad_dstride(const Tiling &tg)
{
    // >= TR*TW and == 2 mod 32: conflict-free A reads (16 channels x 4 pixels)
    const int need = tg.TR * tg.TW;
    return (need + 29) / 32 * 32 + 2;
}

size_t wgrad_lds(const ConvShape &sh, const Tiling &tg)
{
    return shear_bytes(sh, tg, sh.Ci * sh.Z) +
           sizeof(float) * (16 * static_cast<size_t>(wgrad_dstride(tg)) +
                            kWaves * 16 * wgrad_nt(sh) * 16);
}

constexpr int kFwdTarget = 320;
constexpr int kWgradTarget = 320;
constexpr int kBwdR = 4;
constexpr int kFwdBlocks = 1024;   // persistent grid caps
// weight gradient: persistent blocks per CU, as many as LDS holds up to this
// cap (c6 weight gradient: 138 us at 2 per CU, 111 us at 4)
constexpr int kWgradPerCu = 4;
constexpr size_t kLdsPerCu = 160 * 1024;

// prefetch depth (float4 per thread) for a sheared window, 0 if too deep
int shear_depth(const ConvShape &sh, const Tiling &tg, int nch)
{
    if (ShearPrefetch<1>::groups(tg.TW + 2 * sh.k) > kThreads)
        return 0;
    const int r = ShearPrefetch<1>::rows_per_thread(nch, tg.TR + 2 * sh.k, tg.TW + 2 * sh.k,
                                                    kThreads);
    return r <= 1 ? 1 : r <= 2 ? 2 : r <= 4 ? 4 : r <= 8 ? 8 : 0;
}

int plain_depth(const Tiling &tg, int nch)
{
    if (PlainPrefetch<1>::groups(tg.TW) > kThreads)
        return 0;
    const int r = PlainPrefetch<1>::rows_per_thread(nch, tg.TR, tg.TW, kThreads);
    return r <= 2 ? 2 : r <= 4 ? 4 : r <= 8 ? 8 : r <= 12 ? 12 : 0;
}

Tiling bwd_tiling(const ConvShape &sh)
{
    Tiling tg;
    tg.TW = std::min(sh.W, 64);
    const int S = std::max(1, kThreads / tg.TW);
    tg.TR = S * kBwdR;
    tg.tiles_c = cdiv(sh.W, tg.TW);
    tg.tiles_per_img = tg.tiles_c * cdiv(sh.H, tg.TR);
    tg.ntiles = tg.tiles_per_img * sh.N;
    tg.P = shear_pitch(tg.TR + 2 * sh.k);
    tg.CS = (tg.TW + 2 * sh.k) * tg.P;
    tg.fdw = make_fastdiv(static_cast<uint32_t>(tg.TW));
    tg.fdtr = make_fastdiv(static_cast<uint32_t>(tg.TR));
    tg.fdlr = make_fastdiv(static_cast<uint32_t>(tg.TR + 2 * sh.k));
    return tg;
}

int bwd_ic_chunk(const ConvShape &sh, const Tiling &tg)
{
    const size_t per = shear_bytes(sh, tg, 1);
    const int fit = static_cast<int>(std::max<size_t>(1, (48 * 1024) / per));
    return std::min(sh.Co, fit);
}

} // namespace

// ------------------------------------------------------------- launchers

bool smallc_fwd_ok(const ConvShape &sh)
{
    const int nch = sh.Ci * sh.Z;
    if (sh.s != 1 || sh.k < 1 || sh.k > 3 || nch * sh.T > 64 || sh.W % 4 != 0)
        return false;
    const ConvShape e = fwd_view(sh);
    const Tiling tg = make_tiling(e, kFwdTarget);
    return fwd_lds(e, tg) <= kLdsLimit && shear_depth(e, tg, nch) > 0 &&
           tg.TR * tg.TW <= kFwdMT * kWaves * 16 && tg.TW < (1 << 15) && tg.TR < (1 << 15);
}

namespace {
template <typename TT>
hipError_t smallc_fwd_t(const TT *x, const TT *w, const TT *b, TT *y, const ConvShape &sh0,
                        bool relu, hipStream_t st)
{
    const ConvShape sh = fwd_view(sh0);
    const int nch = sh.Ci * sh.Z;
    const bool d3 = sh.D != 1 || sh.Z != 1;
    const Tiling tg = make_tiling(sh, kFwdTarget);
    const int KS = cdiv(nch * sh.T, 4);
    const int U = shear_depth(sh, tg, nch);
    dim3 grid(std::min(tg.ntiles, kFwdBlocks), cdiv(sh.Co, 16));
    const size_t lds = fwd_lds(sh, tg);
#define HEX_FWD_SC(KV, KSV, UV)                                                              \
    do {                                                                                     \
        if (d3)                                                                              \
            HEX_LAUNCH((fwd_smallc_k<TT, KV, KSV, UV, true>), grid, dim3(kThreads), lds, st, \
                       x, w, b, y, sh, relu ? 1 : 0, tg);                                 \
        else                                                                                 \
            HEX_LAUNCH((fwd_smallc_k<TT, KV, KSV, UV, false>), grid, dim3(kThreads), lds,    \
                       st, x, w, b, y, sh, relu ? 1 : 0, tg);                             \
    } while (0)
#define HEX_FWD_SC_U(KV, KSV)                                                                \
    do {                                                                                     \
        if (U == 1) HEX_FWD_SC(KV, KSV, 1);                                                  \
        else if (U == 2) HEX_FWD_SC(KV, KSV, 2);                                             \
        else if (U == 4) HEX_FWD_SC(KV, KSV, 4);                                             \
        else HEX_FWD_SC(KV, KSV, 8);                                                         \
    } while (0)
    if (sh.k == 1) {
        if (KS <= 2) HEX_FWD_SC_U(1, 2);
        else if (KS <= 4) HEX_FWD_SC_U(1, 4);
        else if (KS <= 6) HEX_FWD_SC_U(1, 6);
        else if (KS <= 8) HEX_FWD_SC_U(1, 8);
        else HEX_FWD_SC_U(1, 16);
    } else if (sh.k == 2) {
        if (KS <= 5) HEX_FWD_SC_U(2, 5);
        else if (KS <= 10) HEX_FWD_SC_U(2, 10);
        else HEX_FWD_SC_U(2, 16);
    } else {
        HEX_FWD_SC_U(3, 10); // 37 taps of one input channel (nch * T <= 64)
    }
#undef HEX_FWD_SC_U
#undef HEX_FWD_SC
    return hipGetLastError();
}
} // namespace

hipError_t smallc_fwd(const void *x, const void *w, const void *b, void *y, const ConvShape &sh,
                      Dtype d, bool relu, hipStream_t st)
{
    if (d == F32)
        return smallc_fwd_t(static_cast<const float *>(x), static_cast<const float *>(w),
                            static_cast<const float *>(b), static_cast<float *>(y), sh, relu, st);
    return smallc_fwd_t(static_cast<const bf16raw *>(x), static_cast<const bf16raw *>(w),
                        static_cast<const bf16raw *>(b), static_cast<bf16raw *>(y), sh, relu, st);
}

bool smallc_bwd_data_ok(const ConvShape &sh)
{
    return sh.s == 1 && sh.k >= 1 && sh.k <= 3 && sh.Ci <= 4 &&
           shear_bytes(sh, bwd_tiling(sh), 1) <= kLdsLimit;
}

namespace {
template <typename TT>
hipError_t smallc_bwd_data_t(const TT *dy, const TT *w, TT *dx, const ConvShape &sh,
                             hipStream_t st)
{
    const Tiling tg = bwd_tiling(sh);
    const int ic_chunk = bwd_ic_chunk(sh, tg);
    const size_t lds = shear_bytes(sh, tg, ic_chunk);
    const int vec4 = (sh.W % 4 == 0) ? 1 : 0;
    dim3 grid(tg.ntiles, sh.Ci);
    if (sh.k == 1)
        HEX_LAUNCH((bwd_data_f32_k<TT, 1, kBwdR>), grid, dim3(kThreads), lds, st, dy, w, dx,
                   sh, tg, ic_chunk, vec4);
    else if (sh.k == 2)
        HEX_LAUNCH((bwd_data_f32_k<TT, 2, kBwdR>), grid, dim3(kThreads), lds, st, dy, w, dx,
                   sh, tg, ic_chunk, vec4);
    else
        HEX_LAUNCH((bwd_data_f32_k<TT, 3, kBwdR>), grid, dim3(kThreads), lds, st, dy, w, dx,
                   sh, tg, ic_chunk, vec4);
    return hipGetLastError();
}
} // namespace

hipError_t smallc_bwd_data(const void *dy, const void *w, void *dx, const ConvShape &sh, Dtype d,
                           hipStream_t st)
{
    if (d == F32)
        return smallc_bwd_data_t(static_cast<const float *>(dy), static_cast<const float *>(w),
                                 static_cast<float *>(dx), sh, st);
    return smallc_bwd_data_t(static_cast<const bf16raw *>(dy), static_cast<const bf16raw *>(w),
                             static_cast<bf16raw *>(dx), sh, st);
}

namespace {
int wgrad_grid(const ConvShape &sh, const Tiling &tg)
{
    const int per_cu = std::max(
        1, std::min(kWgradPerCu, static_cast<int>(kLdsPerCu / std::max<size_t>(1, wgrad_lds(sh, tg)))));
    return std::min(tg.ntiles, device_cus() * per_cu);
}
} // namespace

// (2-D shapes have Z = 1 and one plane per sample; the tiles of a 3-D
// shape are (sample, output plane) pairs: fwd_view)
bool smallc_wgrad_ok(const ConvShape &sh0)
{
    const ConvShape sh = fwd_view(sh0);
    const int nch = sh.Ci * sh.Z;
    if (sh.s != 1 || sh.k < 1 || sh.k > 3 || nch * sh.T + 1 > 64 || sh.W % 4 != 0)
        return false;
    const Tiling tg = make_tiling(sh, kWgradTarget);
    return wgrad_lds(sh, tg) <= kLdsLimit && shear_depth(sh, tg, nch) > 0 &&
           plain_depth(tg, 16) > 0;
}

size_t smallc_wgrad_workspace(const ConvShape &sh0)
{
    const ConvShape sh = fwd_view(sh0);
    const Tiling tg = make_tiling(sh, kWgradTarget);
    return sizeof(float) * static_cast<size_t>(wgrad_grid(sh, tg)) * sh.Co *
           (sh.Ci * sh.Z * sh.T + 1);
}

namespace {
template <typename TT>
hipError_t smallc_wgrad_t(const TT *x, const TT *dy, float *dw, float *db, void *ws,
                          const ConvShape &sh0, hipStream_t st)
{
    const ConvShape sh = fwd_view(sh0);
    const int nch = sh.Ci * sh.Z;
    const bool d3 = sh.D != 1 || sh.Z != 1;
    const Tiling tg = make_tiling(sh, kWgradTarget);
    const int nparts = wgrad_grid(sh, tg);
    const int NT = wgrad_nt(sh);
    const int UX = shear_depth(sh, tg, nch);
    const int UD = plain_depth(tg, 16);
    const int dstride = wgrad_dstride(tg);
    float *part = static_cast<float *>(ws);
    dim3 grid(nparts, cdiv(sh.Co, 16));
    const size_t lds = wgrad_lds(sh, tg);
#define HEX_WG(KV, NTV, UXV, UDV)                                                            \
    do {                                                                                     \
        if (d3)                                                                              \
            HEX_LAUNCH((wgrad_f32_k<TT, KV, NTV, UXV, UDV, true>), grid, dim3(kThreads), lds,\
                       st, x, dy, part, sh, tg, dstride);                                    \
        else                                                                                 \
            HEX_LAUNCH((wgrad_f32_k<TT, KV, NTV, UXV, UDV, false>), grid, dim3(kThreads), lds,\
                       st, x, dy, part, sh, tg, dstride);                                    \
    } while (0)
#define HEX_WG_UD(KV, NTV, UXV)                                                              \
    do {                                                                                     \
        if (UD <= 4) HEX_WG(KV, NTV, UXV, 4);                                                \
        else if (UD <= 8) HEX_WG(KV, NTV, UXV, 8);                                           \
        else HEX_WG(KV, NTV, UXV, 12);                                                       \
    } while (0)
#define HEX_WG_UX(KV, NTV)                                                                   \
    do {                                                                                     \
        if (UX <= 2) HEX_WG_UD(KV, NTV, 2);                                                  \
        else if (UX <= 4) HEX_WG_UD(KV, NTV, 4);                                             \
        else HEX_WG_UD(KV, NTV, 8);                                                          \
    } while (0)
    if (sh.k == 1) {
        if (NT == 1) HEX_WG_UX(1, 1);
        else if (NT == 2) HEX_WG_UX(1, 2);
        else HEX_WG_UX(1, 4);
    } else if (sh.k == 2) {
        if (NT == 1) HEX_WG_UX(2, 1);
        else if (NT == 2) HEX_WG_UX(2, 2);
        else HEX_WG_UX(2, 4);
    } else {
        HEX_WG_UX(3, 4); // 37 taps of one input channel plus the bias column
    }
#undef HEX_WG_UX
#undef HEX_WG_UD
#undef HEX_WG
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    return reduce_partials(part, nparts, sh.Co, nch * sh.T, dw, db, st);
}
} // namespace

hipError_t smallc_wgrad(const void *x, const void *dy, float *dw, float *db, void *ws,
                        const ConvShape &sh, Dtype d, hipStream_t st)
{
    if (d == F32)
        return smallc_wgrad_t(static_cast<const float *>(x), static_cast<const float *>(dy), dw,
                              db, ws, sh, st);
    return smallc_wgrad_t(static_cast<const bf16raw *>(x), static_cast<const bf16raw *>(dy), dw,
                          db, ws, sh, st);
}

} // namespace hexk
