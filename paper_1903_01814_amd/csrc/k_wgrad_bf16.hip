// k_wgrad_bf16.hip -- bf16 weight gradient on the matrix cores.
//
//   dw[co][(ci, t)] = sum_{n, p} dy[n][co][p] * x[n][ci][p + tap t]
//   db[co]          = sum_{n, p} dy[n][co][p]
// GEMM with M = co, N = (ci, t) (ci-major, as in the weight layout) and the
// pixels as the contraction index, on v_mfma_f32_16x16x32_bf16:
//   a[i] = A[lane % 16][8 * (lane / 16) + i]  -- dy of channel co at 8
//          consecutive pixels of one row: one 16-byte LDS read;
//   b[i] = B[8 * (lane / 16) + i][lane % 16] -- x of (ci, t) at the same 8
//          pixels moved by tap t: 8 two-byte LDS reads, whose row offset
//          alternates with the pixels' column parity.
// The reduction over pixels happens inside the MFMA.  Blocks are persistent
// over full-width pixel tiles of one image and keep their accumulators in
// registers; each block writes one partial sum per output element, laid out
// in chunks of 64 elements so that both the writes and the fixed-order
// reduction (reduce_chunked) are contiguous.
//
// Block = 4 waves; a block owns 4 channel tiles (64 co) x NB column tiles
// (grid.y enumerates the (co, column) groups); wave w owns column tiles
// w, w + 4, ... of the group (NBW = NB / 4 per wave).  A column group's
// columns span only a few input channels (ci-major, T taps each), and only
// those are staged: at k = 3 with 64 input channels each of the 6 groups
// stages 14 channels instead of 64, which also leaves room for two-row tiles
// (16 x 64 -> 64 x 128 x 128: 721 -> 222 us).
#include <algorithm>

#include "hexdev.h"
#include "kernels.h"

namespace hexk {
namespace {

using namespace hexgeom;

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short shortx8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;
constexpr int kMB = 4;          // channel tiles (of 16 co) per block
constexpr int kXO = 8;          // slot column of plane column 0 in the x window

struct WgTiling {
    int TR, npix_max;       // rows per pixel tile (full width), pixels per tile
    int ntiles;             // pixel tiles over the whole batch
    int tiles_per_img;
    int LCP, XCS;           // x tile: slots per row, slots per channel
    int DP;                 // dy tile pitch (bf16 per channel)
    int J, Jt;              // taps columns Ci*T, plus bias column
    int ncol_tiles;         // ceil(J / 16)
    int NB;                 // column tiles per block
    int NCI;                // x channels a column group needs at most
    int mgroups, ngroups;   // grid.y = mgroups * ngroups
    int nparts;             // partial slots (= grid.x)
};

// SV: the stride when it is 1 (compile-time), else 0 (the stride of sh).
// At stride s output pixel (i, j) is centred on input row s i + (j & 1)
// floor(s / 2), column s j: the x window of a tile of TR output rows spans
// s (TR - 1) + floor(s / 2) + 2K + 1 input rows, and element e of a run of 8
// pixels sits s e columns after the first (odd pixels floor(s / 2) rows down).
template <int K, int NBW, int SV>
__global__ __launch_bounds__(kThreads) void wgrad_bf16_k(
    const bf16raw *__restrict__ x, const bf16raw *__restrict__ dy, float *__restrict__ part,
    ConvShape sh, WgTiling tg)
{
    constexpr int T = num_taps(K);
    extern __shared__ __align__(16) bf16raw lds[];
    bf16raw *xs = lds;                                        // [NCI][XCS]
    bf16raw *ds_ = lds + static_cast<size_t>(tg.NCI) * tg.XCS; // [64][DP]

    const int H = sh.H, W = sh.W, Wo = sh.Wo;
    const int S = SV ? SV : sh.s, SH = S >> 1;
    const size_t HW = static_cast<size_t>(H) * W;
    const size_t HWo = static_cast<size_t>(sh.Ho) * Wo;
    const int mg = blockIdx.y % tg.mgroups, ngp = blockIdx.y / tg.mgroups;
    const int co_blk = mg * kMB * 16;
    const int nco = min(kMB * 16, sh.Co - co_blk);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int m = lane & 15, kq = lane >> 4;

    // the columns (ci, t) of this block's column group span input channels
    // ci_lo .. ci_lo + nci - 1: only those are staged
    const int ci_lo = (ngp * tg.NB * 16) / T;
    const int nci = min(tg.NCI, sh.Ci - ci_lo);
    // this lane's B columns: (ci, t) and the two parity offsets (in slots)
    int boff0[NBW], boff1[NBW], bch[NBW];
    bool bval[NBW];
#pragma unroll
    for (int j = 0; j < NBW; ++j) {
        const int ntl = ngp * tg.NB + wave + 4 * j; // column tile
        const int col = ntl * 16 + m;
        bval[j] = (wave + 4 * j) < tg.NB && ntl < tg.ncol_tiles && col < tg.J;
        const int ci = bval[j] ? col / T : 0, t = bval[j] ? col - ci * T : 0;
        int dq = 0, ds = 0;
        tap_axial(K, t, dq, ds);
        bch[j] = bval[j] ? ci - ci_lo : 0;
        boff0[j] = tap_drow(dq, ds, 0) * tg.LCP + dq;
        boff1[j] = (tap_drow(dq, ds, S & 1) + SH) * tg.LCP + dq;
    }
    floatx4 acc[kMB][NBW];
#pragma unroll
    for (int i = 0; i < kMB; ++i)
#pragma unroll
        for (int j = 0; j < NBW; ++j)
            acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    float dbs = 0.f; // partial db of channel tile `wave` (first column group only)

    for (int tile = blockIdx.x; tile < tg.ntiles; tile += gridDim.x) {
        const int n = tile / tg.tiles_per_img;
        const int r0 = (tile - n * tg.tiles_per_img) * tg.TR; // first output row
        const int rows = min(tg.TR, sh.Ho - r0);
        const int npix = rows * Wo;
        __syncthreads(); // previous tile's LDS reads are done
        // x window input rows S r0 - K .. S (r0 + rows - 1) + SH + K; plane
        // column c sits at slot column c + kXO (16-byte aligned), the K halo
        // columns on each side hold zeros
        {
            const int LR = S * (rows - 1) + SH + 2 * K + 1;
            const int cols8 = W / 8;          // 16-byte column groups of a row
            const int items = nci * LR * cols8;
            for (int it0 = threadIdx.x; it0 < items; it0 += 4 * kThreads) {
                uint4 v[4];
                int dst[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int it = it0 + u * kThreads;
                    const bool live = it < items;
                    const int g = live ? it % cols8 : 0;
                    const int rest = live ? it / cols8 : 0;
                    const int rr = rest % LR, ci = rest / LR;
                    const int r = S * r0 - K + rr;
                    const bool ok = live && r >= 0 && r < H;
                    dst[u] = live ? ci * tg.XCS + rr * tg.LCP + kXO + 8 * g : -1;
                    const uint4 q = *reinterpret_cast<const uint4 *>(
                        x + (ok ? (static_cast<size_t>(n) * sh.Ci + ci_lo + ci) * HW + static_cast<size_t>(r) * W + 8 * g
                                : 0));
                    v[u] = ok ? q : make_uint4(0, 0, 0, 0);
                }
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (dst[u] >= 0)
                        *reinterpret_cast<uint4 *>(xs + dst[u]) = v[u];
            }
            const int hitems = nci * LR * 2 * K;
            for (int e = threadIdx.x; e < hitems; e += kThreads) {
                const int side = e % (2 * K);
                const int rest = e / (2 * K);
                const int rr = rest % LR, ci = rest / LR;
                const int cc = side < K ? kXO - K + side : kXO + W + side - K;
                xs[ci * tg.XCS + rr * tg.LCP + cc] = 0;
            }
        }
        // dy tile: channels co_blk .. co_blk+nco-1, pixels r0*Wo .. r0*Wo+npix-1
        {
            const int n8 = npix / 8;
            const int items = nco * n8;
            for (int it0 = threadIdx.x; it0 < items; it0 += 4 * kThreads) {
                uint4 v[4];
                int dst[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int it = it0 + u * kThreads;
                    const bool live = it < items;
                    const int c = live ? it / n8 : 0, g = live ? it - c * n8 : 0;
                    dst[u] = live ? c * tg.DP + 8 * g : -1;
                    v[u] = *reinterpret_cast<const uint4 *>(
                        dy + (live ? (static_cast<size_t>(n) * sh.Co + co_blk + c) * HWo +
                                         static_cast<size_t>(r0) * Wo + 8 * g
                                   : 0));
                }
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (dst[u] >= 0)
                        *reinterpret_cast<uint4 *>(ds_ + dst[u]) = v[u];
            }
        }
        __syncthreads();

        const int nks = (npix + 31) / 32;
        for (int ks = 0; ks < nks; ++ks) {
            const int p = ks * 32 + 8 * kq; // first pixel of this lane's group of 8
            const bool pv = p < npix;       // groups never straddle rows (Wo % 8 == 0)
            const int pr = pv ? p / Wo : 0, pc = pv ? p - pr * Wo : 0;
            // slot of the centre of pixel (pr, pc) in the x window (window
            // row S pr + K, column S pc; pc is even)
            const int s0 = (S * pr + K) * tg.LCP + S * pc + kXO;
            bf16x8 a[kMB];
#pragma unroll
            for (int i = 0; i < kMB; ++i) {
                const int c = i * 16 + m;
                const uint4 q = *reinterpret_cast<const uint4 *>(ds_ + ((pv && c < nco) ? c * tg.DP + p : 0));
                a[i] = __builtin_bit_cast(bf16x8, (pv && c < nco) ? q : make_uint4(0, 0, 0, 0));
            }
            if (ngp == 0) {
#pragma unroll
                for (int i = 0; i < kMB; ++i)
                    if (i == wave)
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            dbs += static_cast<float>(a[i][e]);
            }
#pragma unroll
            for (int j = 0; j < NBW; ++j) {
                // pixel pc + e is odd for odd e (pc is even)
                const bf16raw *b0 = xs + bch[j] * tg.XCS + s0 + boff0[j];
                const bf16raw *b1 = xs + bch[j] * tg.XCS + s0 + boff1[j];
                shortx8 bs;
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    bs[e] = static_cast<short>((e & 1) ? b1[S * e] : b0[S * e]);
                const bool ok = pv && bval[j];
                const bf16x8 b = __builtin_bit_cast(bf16x8, ok ? bs : shortx8{0, 0, 0, 0, 0, 0, 0, 0});
#pragma unroll
                for (int i = 0; i < kMB; ++i)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b, acc[i][j], 0, 0, 0);
            }
        }
    }

    // partial sums of this block: element e = co * Jt + col, chunked layout
    // part_index(e, slot): chunked layout
    const size_t slot = blockIdx.x;
#pragma unroll
    for (int i = 0; i < kMB; ++i) {
#pragma unroll
        for (int j = 0; j < NBW; ++j) {
            if (!bval[j])
                continue;
            const int col = (ngp * tg.NB + wave + 4 * j) * 16 + m;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int co = co_blk + i * 16 + 4 * kq + q;
                if (co >= sh.Co)
                    continue;
                const size_t e = static_cast<size_t>(co) * tg.Jt + col;
                part[part_index(static_cast<int>(e), static_cast<int>(slot), tg.nparts)] = acc[i][j][q];
            }
        }
    }
    if (ngp == 0) {
        // db: wave w holds channel tile w; sum its 4 lane groups (kq)
        __shared__ float dred[kMB][64];
        dred[wave][lane] = dbs;
        __syncthreads();
        if (threadIdx.x < kMB * 16) {
            const int i = threadIdx.x / 16, mm = threadIdx.x % 16;
            const float s = (dred[i][mm] + dred[i][mm + 16]) + (dred[i][mm + 32] + dred[i][mm + 48]);
            const int co = co_blk + i * 16 + mm;
            if (co < sh.Co) {
                const size_t e = static_cast<size_t>(co) * tg.Jt + tg.J;
                part[part_index(static_cast<int>(e), static_cast<int>(slot), tg.nparts)] = s;
            }
        }
    }
}

inline int cdiv(long a, long b) { return static_cast<int>((a + b - 1) / b); }

constexpr int kWgBlocks = 512; // persistent blocks (x grid.y groups)

// x window rows of a tile of TR output rows
int wg_win_rows(const ConvShape &sh, int TR) { return sh.s * (TR - 1) + sh.s / 2 + 2 * sh.k + 1; }

size_t wg_lds_bytes(const ConvShape &sh, int TR, int NCI)
{
    const long LCP = sh.W + 2 * kXO;
    const long XCS = static_cast<long>(wg_win_rows(sh, TR)) * LCP + 8;
    const long DP = static_cast<long>(TR) * sh.Wo + 8;
    return sizeof(bf16raw) * static_cast<size_t>(NCI * XCS + kMB * 16 * DP);
}

// input channels spanned by NB column tiles (16 columns each, ci-major with T
// taps per channel) starting anywhere
int wg_nci(const ConvShape &sh, int NB)
{
    return std::min(sh.Ci, (NB * 16 - 1) / sh.T + 2);
}

constexpr size_t kWgLdsTarget = 80 * 1024;  // two blocks per CU
constexpr size_t kWgLdsMax = 150 * 1024;    // one block per CU

WgTiling wg_tiling(const ConvShape &sh, int NBW)
{
    WgTiling tg;
    // tallest full-width tile of at most 256 pixels within the LDS target
    const int NCI = wg_nci(sh, 4 * NBW);
    int TR = std::max(1, std::min(sh.Ho, 256 / std::max(1, sh.Wo)));
    while (TR > 1 && wg_lds_bytes(sh, TR, NCI) > kWgLdsTarget)
        --TR;
    tg.NCI = NCI;
    tg.TR = TR;
    tg.npix_max = tg.TR * sh.Wo;
    tg.tiles_per_img = cdiv(sh.Ho, tg.TR);
    tg.ntiles = tg.tiles_per_img * sh.N;
    tg.LCP = sh.W + 2 * kXO;
    tg.XCS = wg_win_rows(sh, tg.TR) * tg.LCP + 8;
    tg.DP = tg.npix_max + 8;
    tg.J = sh.Ci * sh.T;
    tg.Jt = tg.J + 1;
    tg.ncol_tiles = cdiv(tg.J, 16);
    tg.NB = 4 * NBW;
    tg.mgroups = cdiv(sh.Co, kMB * 16);
    tg.ngroups = cdiv(tg.ncol_tiles, tg.NB);
    tg.nparts = std::max(1, std::min(tg.ntiles, kWgBlocks / (tg.mgroups * tg.ngroups)));
    return tg;
}

// column tiles per wave: as few column groups as 7 tiles per wave allow,
// split evenly between the groups
int wg_nbw(const ConvShape &sh)
{
    const int ncol = cdiv(sh.Ci * sh.T, 16);
    const int groups = cdiv(ncol, 4 * 7);
    return cdiv(ncol, 4 * groups);
}

size_t wg_lds(const ConvShape &sh, const WgTiling &tg) { return wg_lds_bytes(sh, tg.TR, tg.NCI); }

} // namespace

bool bf16_wgrad_ok(const ConvShape &sh)
{
    if (sh.s < 1 || sh.k < 1 || sh.k > 3 || sh.W % 8 != 0 || sh.W > 256 || sh.Ho < 1 ||
        sh.Wo % 8 != 0)
        return false;
    return wg_lds(sh, wg_tiling(sh, wg_nbw(sh))) <= kWgLdsMax;
}

size_t bf16_wgrad_workspace(const ConvShape &sh)
{
    const WgTiling tg = wg_tiling(sh, wg_nbw(sh));
    const size_t E = static_cast<size_t>(sh.Co) * tg.Jt;
    return sizeof(float) * static_cast<size_t>(part_chunks(static_cast<int>(E))) * kPartChunk *
           tg.nparts;
}

hipError_t bf16_wgrad(const void *x, const void *dy, float *dw, float *db, void *ws,
                      const ConvShape &sh, hipStream_t st)
{
    const int nbw = wg_nbw(sh);
    const WgTiling tg = wg_tiling(sh, nbw);
    dim3 grid(tg.nparts, tg.mgroups * tg.ngroups);
    const size_t lds = wg_lds(sh, tg);
    const bf16raw *xp = static_cast<const bf16raw *>(x);
    const bf16raw *dp = static_cast<const bf16raw *>(dy);
    float *part = static_cast<float *>(ws);
#define HEX_WG_S(KV, NV, SV)                                                                 \
    HEX_LAUNCH((wgrad_bf16_k<KV, NV, SV>), grid, dim3(kThreads), lds, st, xp, dp, part, sh, tg)
#define HEX_WG(KV, NV)                                                                       \
    do {                                                                                     \
        if (sh.s == 1) HEX_WG_S(KV, NV, 1); else HEX_WG_S(KV, NV, 0);                        \
    } while (0)
#define HEX_WG_N(KV)                                                                         \
    do {                                                                                     \
        switch (nbw) {                                                                       \
        case 1: HEX_WG(KV, 1); break;                                                        \
        case 2: HEX_WG(KV, 2); break;                                                        \
        case 3: HEX_WG(KV, 3); break;                                                        \
        case 4: HEX_WG(KV, 4); break;                                                        \
        case 5: HEX_WG(KV, 5); break;                                                        \
        case 6: HEX_WG(KV, 6); break;                                                        \
        default: HEX_WG(KV, 7); break;                                                       \
        }                                                                                    \
    } while (0)
    if (sh.k == 1)
        HEX_WG_N(1);
    else if (sh.k == 2)
        HEX_WG_N(2);
    else
        HEX_WG_N(3);
#undef HEX_WG_N
#undef HEX_WG
#undef HEX_WG_S
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    return reduce_chunked(part, tg.nparts, sh.Co, tg.J, dw, db, st);
}

} // namespace hexk
