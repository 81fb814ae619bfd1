// k_mfma_gen.hip -- bf16 convolutions on the matrix cores at any stride and
// for kernel sizes up to 3, where the stride-1 kernels of k_mfma_bf16.hip do
// not apply (strides above 1, 37 taps at k = 3).
//
// Both kernels are implicit GEMMs on v_mfma_f32_32x32x16_bf16 (lane layout:
// a[i] = A[lane % 32][8 * (lane / 32) + i], b[i] = B[8 * (lane / 32) + i]
// [lane % 32], d[r] = D[8 * (r / 4) + 4 * (lane / 32) + r % 4][lane % 32]):
// the 32 rows of A are 32 destination pixels, the contraction runs over
// (tap, 16 channels) per K-step, the 32 columns of B over 32 destination
// channels, and a block covers 64 destination channels.
//
// Forward (Sec. 2.3, stride lattice of Fig. 4): a block computes a tile of
// full-width output rows.  The input window of the tile (rows s i0 - k ..,
// columns -k .., zero outside the tensor) is staged channel-last in LDS,
// 32 input channels at a time, so an A fragment is one 16-byte LDS read at
// the slot of the pixel's centre plus the tap's offset (one window row
// further for odd tap columns when the centre column is odd).
//
// Data gradient (the adjoint, a transposed lattice gather): input pixel p
// receives from tap t only when p - d_t is a kernel centre, i.e. when the
// axial coordinates of p - d_t are multiples of s.  The pixels of a tile are
// sorted into the s * s classes of their axial coordinates modulo s; within
// a class exactly the taps congruent to it are live, and for a live tap the
// source output sits at a fixed axial offset -- a row offset that alternates
// with the column parity, as in the forward.  Every 32-pixel group holds one
// class, so its K-loop visits only its own taps and no product is wasted.
// dy is staged channel-last like the forward's input, the results go through
// LDS and leave as whole rows.
//
// In both, the weights of a group of taps for the block's 64 destination
// channels and one 32-channel chunk of the contraction are gathered from
// global memory into LDS per stage, so any number of taps fits.  Slot and
// weight rows are 40 bf16 (80 bytes, an odd multiple of 16: conflict-free
// 16-byte fragment reads of 32 consecutive rows).
#include <algorithm>

#include "hexdev.h"
#include "kernels.h"

namespace hexk {
namespace {

using namespace hexgeom;

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kGThreads = 256; // 4 waves
constexpr int kCK = 32;        // contraction channels per staged chunk
constexpr int kCP = kCK + 8;   // bf16 per LDS slot / weight row
constexpr int kNB = 64;        // destination channels per block
constexpr int kMG = 2;         // 32-pixel groups per wave and round

struct GenArgs {
    int N;
    int Cs, Cd;       // contraction (source) and destination channels
    int Hs, Ws;       // source planes (x for the forward, dy for the data gradient)
    int Hd, Wd;       // destination planes (y, dx)
    int s;            // stride
    int TR;           // destination rows per tile
    int tiles;        // tiles per image
    int WR, WC;       // window rows and slots per row
    int coff;         // window column of source column 0
    int split;        // window columns stored by residue mod split (the forward's stride)
    int WCs;          // slots per residue class; a window row holds RP = split * WCs slots
    int RP;
    int TG;           // taps per weight stage (kTG)
    int win_off;      // byte offsets in LDS: window, weights, output staging
    int wgt_off;
    int out_off;
    int OP;           // output staging pitch (bf16 per destination channel)
    int nblk;         // destination-channel blocks of 64
    int relu;
    int CW;           // contraction channels held by the window (32, 64 or 128)
    int SP;           // bf16 per window slot (CW + 8)
    int resident;     // every stage's weights held in LDS for the block's life
    int ntot;         // tiles in the batch (N * tiles)
};

__device__ __forceinline__ uint32_t lo16(uint32_t v) { return v & 0xffffu; }
__device__ __forceinline__ uint32_t hi16(uint32_t v) { return v >> 16; }

// Rows [g_r0, g_r0 + nrows) of CW channels of one image (src points at the
// first plane; planes HW apart, rows of Wsrc elements, Wsrc a multiple of 8)
// into window rows 0 .. nrows-1: source column c goes to slot column c +
// coff (if below WC), slots of SP bf16, 8 channels per 16-byte vector.
// Rows outside [0, Hsrc) and the slot columns holding no source column are
// zero.  Two items per thread per round, all their loads issued first.
__device__ __forceinline__ void stage_window(bf16raw *__restrict__ win,
                                             const bf16raw *__restrict__ src, size_t HW,
                                             int Hsrc, int Wsrc, int g_r0, int nrows, int WC,
                                             int coff, int CW, int SP, int split, int WCs,
                                             int RP)
{
    constexpr int U = 2;
    const int ngl = __builtin_ctz(CW >> 3); // log2 of the 8-channel groups
    const int ncol8 = Wsrc >> 3;
    const int items = (nrows * ncol8) << ngl;
    for (int it0 = threadIdx.x; it0 < items; it0 += U * kGThreads) {
        uint4 v[U][8];
        int slot0[U], ncopy[U], grp[U];
#pragma unroll
        for (int h = 0; h < U; ++h) {
            const int it = it0 + h * kGThreads;
            const int g = it & ((1 << ngl) - 1), rest = it >> ngl;
            const int ch = rest % ncol8, rr = rest / ncol8;
            const int r = g_r0 + rr, col0 = 8 * ch;
            const bool live = it < items && col0 + coff < WC;
            const bool rin = live && r >= 0 && r < Hsrc;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                v[h][e] = rin ? *reinterpret_cast<const uint4 *>(src + (8 * g + e) * HW +
                                                                 static_cast<size_t>(r) * Wsrc + col0)
                              : make_uint4(0, 0, 0, 0);
            slot0[h] = rr * RP;                // + column map of col0 + coff + px
            ncopy[h] = live ? min(8, WC - col0 - coff) : 0;
            grp[h] = (col0 + coff) | (g << 20); // window column of px 0, channel group
        }
#pragma unroll
        for (int h = 0; h < U; ++h) {
            const int g = grp[h] >> 20, c0w = grp[h] & 0xfffff;
            // window column c lives at slot column (c % split) WCs + c / split
            int cq = c0w / split, cr = c0w - (c0w / split) * split;
#pragma unroll
            for (int px = 0; px < 8; ++px) {
                if (px >= ncopy[h])
                    break;
                const int scol = cr * WCs + cq;
                if (++cr == split) {
                    cr = 0;
                    ++cq;
                }
                uint32_t q[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const uint32_t a = reinterpret_cast<const uint32_t *>(&v[h][2 * j])[px >> 1];
                    const uint32_t b = reinterpret_cast<const uint32_t *>(&v[h][2 * j + 1])[px >> 1];
                    q[j] = (px & 1) ? (hi16(a) | (b & 0xffff0000u)) : (lo16(a) | (b << 16));
                }
                *reinterpret_cast<uint4 *>(win + (slot0[h] + scol) * SP + 8 * g) =
                    make_uint4(q[0], q[1], q[2], q[3]);
            }
        }
    }
    // slot columns without a source column: [0, coff) and [Wsrc + coff, WC)
    const int right = max(0, WC - Wsrc - coff);
    const int side = coff + right;
    const int zitems = (nrows * side) << ngl;
    for (int it = threadIdx.x; it < zitems; it += kGThreads) {
        const int g = it & ((1 << ngl) - 1), rest = it >> ngl;
        const int sc = rest % side, rr = rest / side;
        const int col = sc < coff ? sc : Wsrc + coff + (sc - coff);
        const int scol = (col % split) * WCs + col / split;
        *reinterpret_cast<uint4 *>(win + (rr * RP + scol) * SP + 8 * g) = make_uint4(0, 0, 0, 0);
    }
}

// Weights of one stage -- taps [t0, t0 + kTG) of one 32-channel chunk of
// the contraction, for the block's 64 destination channels -- in LDS as
// wl[tt * kTB + n * kCP + kc] (kTB = 64 rows of kCP plus a pad of 8, so the
// tap blocks start on different banks):
//   forward (DG = false): n = output channel d0 + n, kc = input channel c0 + kc,
//     value w[d0 + n][c0 + kc][t0 + tt];
//   data gradient (DG = true): n = input channel d0 + n, kc = output channel
//     c0 + kc, value w[c0 + kc][d0 + n][t0 + tt].
// Zero for destination channels past Cd and taps past T.  w is
// [Cout][Cin][T].  Thread mapping: tap tt = tid % 8, channel octet kc0 =
// 8 ((tid / 8) % 4), rows n = tid / 32 + 8 j (j < 8); a thread gathers the
// eight channels kc0 .. kc0 + 7 of each of its rows (loads one stride apart:
// T elements in the forward, C_in T in the data gradient), packs them into
// 16 bytes and writes them with one LDS store.  Eight consecutive lanes read
// eight consecutive taps, one 16-byte run.  load() issues every load of the
// thread (while the previous stage computes); store() writes them.
constexpr int kTG = 8;                      // taps per stage
constexpr int kTB = kNB * kCP + 8;          // bf16 per tap block in LDS

template <bool DG> struct WgtRegs {
    uint4 v[8]; // row j: channels kc0 .. kc0 + 7

    __device__ __forceinline__ void load(const bf16raw *__restrict__ w, int T, int Cs, int Cd,
                                         int d0, int c0, int t0)
    {
        const int tt = threadIdx.x & 7, kc0 = 8 * ((threadIdx.x >> 3) & 3);
        const int nb = threadIdx.x >> 5;
        const bool tv = t0 + tt < T;
        const int t = tv ? t0 + tt : T - 1;            // clamped: valid address, value dropped
        const size_t cstride = DG ? static_cast<size_t>(Cd) * T : static_cast<size_t>(T);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int n = nb + 8 * j;
            const bool nv = tv && d0 + n < Cd;
            const int d = nv ? d0 + n : Cd - 1;
            const bf16raw *p = DG ? w + (static_cast<size_t>(c0 + kc0) * Cd + d) * T + t
                                  : w + (static_cast<size_t>(d) * Cs + c0 + kc0) * T + t;
            uint32_t q[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t lo = p[(2 * i) * cstride];
                const uint32_t hi = p[(2 * i + 1) * cstride];
                q[i] = nv ? (lo | (hi << 16)) : 0u;
            }
            v[j] = make_uint4(q[0], q[1], q[2], q[3]);
        }
    }

    __device__ __forceinline__ void store(bf16raw *__restrict__ wl) const
    {
        const int tt = threadIdx.x & 7, kc0 = 8 * ((threadIdx.x >> 3) & 3);
        const int nb = threadIdx.x >> 5;
#pragma unroll
        for (int j = 0; j < 8; ++j)
            *reinterpret_cast<uint4 *>(wl + tt * kTB + (nb + 8 * j) * kCP + kc0) = v[j];
    }
};

// Slot offset of axial tap (dq, ds) from a forward centre: row ds + dq/2
// (floor), plus one more row for odd dq when the centre column is odd.
__device__ __forceinline__ int fwd_tap_off(int dq, int ds, int WC)
{
    return (ds + floor_half(dq)) * WC + dq;
}

// Slot column offset of window column c (>= 0) in a window split by column
// residue mod s: (c % s) WCs + c / s.
__device__ __forceinline__ int tap_col(int c, int s, int WCs) { return (c % s) * WCs + c / s; }

// Accumulate one K-step (16 channels at window channel cl + 16 h) for the
// wave's groups: A at window slot slot[m], B for both 32-channel halves of
// the block.
template <int MG>
__device__ __forceinline__ void kstep(floatx16 (&acc)[MG][2], const bf16raw *__restrict__ win,
                                      const bf16raw *__restrict__ wrow, const int (&slot)[MG],
                                      int ng, int h, int kh, int SP, int cl)
{
    const bf16x8 b0 = *reinterpret_cast<const bf16x8 *>(wrow + h * 16);
    const bf16x8 b1 = *reinterpret_cast<const bf16x8 *>(wrow + 32 * kCP + h * 16);
#pragma unroll
    for (int m = 0; m < MG; ++m) {
        if (m >= ng)
            break;
        const bf16x8 a =
            *reinterpret_cast<const bf16x8 *>(win + slot[m] * SP + cl + h * 16 + 8 * kh);
        acc[m][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b0, acc[m][0], 0, 0, 0);
        acc[m][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b1, acc[m][1], 0, 0, 0);
    }
}

// Stage weights: every stage at once (resident, once per block) or one
// stage into the single buffer.  Stage st = (chunk st / NTG, taps
// (st % NTG) * kTG ..).
constexpr int kStageElems = kTG * kTB; // bf16 per stage in LDS

template <bool DG>
__device__ __forceinline__ void stage_all_weights(bf16raw *__restrict__ wl,
                                                  const bf16raw *__restrict__ w, int T, int NTG,
                                                  int nst, int Cs, int Cd, int d0)
{
    for (int st = 0; st < nst; ++st) {
        WgtRegs<DG> r;
        r.load(w, T, Cs, Cd, d0, (st / NTG) * kCK, (st % NTG) * kTG);
        r.store(wl + st * kStageElems);
    }
}

// ---------------------------------------------------------------- forward
// Persistent blocks: block b keeps destination block db = b % nblk (output
// channels 64 db ..) and walks the tiles b / nblk, + gridDim / nblk, ...; a
// tile is (image n, output rows i0 .. i0 + rows - 1, all W_out columns).
// Pixel p of the tile (row-major) is in group p / 32; wave w owns groups w,
// w + 4 (tiles hold at most 256 pixels).  Per tile the stages run over
// (32-channel chunk, 8 taps); the window holds CW channels and is staged
// when a stage starts a new window's worth of channels; streamed weights of
// the next stage (of this tile or the next) load during the current one.
template <int K>
__global__ __launch_bounds__(kGThreads) void conv_gen_fwd_k(const bf16raw *__restrict__ x,
                                                            const bf16raw *__restrict__ w,
                                                            const bf16raw *__restrict__ bias,
                                                            bf16raw *__restrict__ y, GenArgs a)
{
    constexpr int T = num_taps(K);
    constexpr TapTable<K> tab{};
    constexpr int NTG = (T + kTG - 1) / kTG;
    extern __shared__ __align__(16) unsigned char smem[];
    bf16raw *win = reinterpret_cast<bf16raw *>(smem + a.win_off);
    bf16raw *wl = reinterpret_cast<bf16raw *>(smem + a.wgt_off);
    bf16raw *outl = reinterpret_cast<bf16raw *>(smem + a.out_off);

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n32 = lane & 31, kh = lane >> 5;
    const int db = blockIdx.x % a.nblk, tstep = gridDim.x / a.nblk;
    const int d0 = db * kNB;
    const int s = a.s;
    const int nst = (a.Cs / kCK) * NTG;
    const size_t HWs = static_cast<size_t>(a.Hs) * a.Ws;
    const size_t HWd = static_cast<size_t>(a.Hd) * a.Wd;
    const int nd = min(kNB, a.Cd - d0);
    float bv[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int d = d0 + j * 32 + n32;
        bv[j] = (bias != nullptr && d < a.Cd) ? to_f(bias[d]) : 0.f;
    }

    WgtRegs<false> wr;
    if (a.resident)
        stage_all_weights<false>(wl, w, T, NTG, nst, a.Cs, a.Cd, d0);
    else
        wr.load(w, T, a.Cs, a.Cd, d0, 0, 0);

    for (int tb = blockIdx.x / a.nblk; tb < a.ntot; tb += tstep) {
        const int n = tb / a.tiles, i0 = (tb - n * a.tiles) * a.TR;
        const int rows = min(a.TR, a.Hd - i0);
        const int M = rows * a.Wd;
        const int ngroups = (M + 31) >> 5;
        const int r_lo = s * i0 - K; // window row 0

        // this lane's pixel (A row) per group: window slot of its centre and
        // the extra row of odd tap columns when the centre column is odd
        int slot0[kMG], podd[kMG];
        int ng = 0;
#pragma unroll
        for (int m = 0; m < kMG; ++m) {
            const int g = wave + 4 * m;
            if (g < ngroups)
                ng = m + 1;
            const int p = min(g * 32 + n32, M - 1); // clamped: valid, never stored
            const int i = i0 + p / a.Wd, j = p % a.Wd;
            const int rc = s * i + (j & 1) * (s >> 1), cc = s * j;
            // window column cc + coff + dq = s j + coff + dq sits at slot
            // column j + tap_col(dq) (the window is split by column mod s)
            slot0[m] = (rc - r_lo) * a.RP + j;
            podd[m] = (cc & 1) ? a.RP : 0;
        }
        floatx16 acc[kMG][2];
#pragma unroll
        for (int m = 0; m < kMG; ++m)
            acc[m][0] = acc[m][1] = floatx16{};

        for (int st = 0; st < nst; ++st) {
            const int c0 = (st / NTG) * kCK, t0 = (st % NTG) * kTG;
            const int cw0 = c0 - c0 % a.CW; // first channel of the window
            __syncthreads(); // the previous stage's (or tile's) readers are done
            if (c0 == cw0 && t0 == 0)
                stage_window(win, x + (static_cast<size_t>(n) * a.Cs + cw0) * HWs, HWs, a.Hs,
                             a.Ws, r_lo, a.WR, a.WC, a.coff, a.CW, a.SP, a.split, a.WCs, a.RP);
            if (!a.resident)
                wr.store(wl);
            __syncthreads();
            if (!a.resident && (st + 1 < nst || tb + tstep < a.ntot)) {
                const int sn = st + 1 < nst ? st + 1 : 0; // next stage, maybe the next tile's
                wr.load(w, T, a.Cs, a.Cd, d0, (sn / NTG) * kCK, (sn % NTG) * kTG);
            }
            if (ng == 0)
                continue;
            const bf16raw *wst = a.resident ? wl + st * kStageElems : wl;
            const int ntap = min(kTG, T - t0);
            for (int tt = 0; tt < ntap; ++tt) {
                const int t = t0 + tt;
                const int dq = tab.dq[t], ds = tab.ds[t];
                const int off = fwd_tap_off(dq, ds, a.RP) - dq + tap_col(dq + a.coff, s, a.WCs);
                int slot[kMG];
#pragma unroll
                for (int m = 0; m < kMG; ++m)
                    slot[m] = slot0[m] + off + ((dq & 1) ? podd[m] : 0);
                const bf16raw *wrow = wst + tt * kTB + n32 * kCP + 8 * kh;
                kstep<kMG>(acc, win, wrow, slot, ng, 0, kh, a.SP, c0 - cw0);
                kstep<kMG>(acc, win, wrow, slot, ng, 1, kh, a.SP, c0 - cw0);
            }
        }

        // epilogue: bias, ReLU, bf16 into LDS [channel][pixel], then whole rows
        __syncthreads();
#pragma unroll
        for (int m = 0; m < kMG; ++m) {
            if (m >= ng)
                break;
            const int g = wave + 4 * m;
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                bf16raw *orow = outl + (j * 32 + n32) * a.OP + g * 32 + 4 * kh;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float v[4];
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        v[r] = acc[m][j][4 * q + r] + bv[j];
                        if (a.relu)
                            v[r] = fmaxf(v[r], 0.f);
                    }
                    bf16raw o[4];
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        o[r] = from_f<bf16raw>(v[r]);
                    // pixels g*32 + 8q + 4kh + 0..3 (rows padded to 32-pixel groups)
                    *reinterpret_cast<uint2 *>(orow + 8 * q) =
                        make_uint2(o[0] | (static_cast<uint32_t>(o[1]) << 16),
                                   o[2] | (static_cast<uint32_t>(o[3]) << 16));
                }
            }
        }
        __syncthreads();
        bf16raw *ybase =
            y + (static_cast<size_t>(n) * a.Cd + d0) * HWd + static_cast<size_t>(i0) * a.Wd;
        if ((a.Wd & 7) == 0) { // then every row of the tile starts on 16 bytes
            const int nv = M >> 3;
            for (int e = threadIdx.x; e < nd * nv; e += kGThreads) {
                const int d = e / nv, v = e - d * nv;
                const bf16raw *src = outl + d * a.OP + 8 * v;
                const uint2 lo = *reinterpret_cast<const uint2 *>(src);
                const uint2 hi = *reinterpret_cast<const uint2 *>(src + 4);
                *reinterpret_cast<uint4 *>(ybase + d * HWd + 8 * v) =
                    make_uint4(lo.x, lo.y, hi.x, hi.y);
            }
        } else {
            for (int e = threadIdx.x; e < nd * M; e += kGThreads) {
                const int d = e / M, p = e - d * M;
                ybase[d * HWd + p] = outl[d * a.OP + p];
            }
        }
    }
}

// ---------------------------------------------------------- data gradient
// Block: tile (image n, input rows r0 .. r0 + TR - 1 with TR a multiple of
// s, all W columns) x destination block db (input channels 64 db ..).  The
// tile's pixels are sorted into classes (a, b) = (c mod s, (r - floor(c/2))
// mod s), class index a s + b; class (a, b) holds, per column c = a + s v
// (v < nv(a) = ceil((W - a) / s)), the TR / s rows with that axial residue:
// element e = u nv + v.  Groups of 32 class elements are numbered class by
// class; round q gives wave w the groups 8 q + w + 4 m, m < kMG.
struct DgClass {
    int a, b, nv, size, g0; // residues, columns, elements, first group
};

// v mod s and v / s for the small offsets of a tap against a class residue
// (|v| < 2 s + 4): a few subtractions instead of a division
__device__ __forceinline__ void small_divmod(int v, int s, int &q, int &r)
{
    q = 0;
    while (v < 0) {
        v += s;
        --q;
    }
    while (v >= s) {
        v -= s;
        ++q;
    }
    r = v;
}

__device__ __forceinline__ DgClass dg_class_of_group(int g, int s, int W, int TR)
{
    int g0 = 0;
    for (int cl = 0; cl < s * s; ++cl) {
        const int a = cl / s, b = cl - (cl / s) * s;
        const int nv = (W - a + s - 1) / s;
        const int size = (TR / s) * nv;
        const int ng = (size + 31) >> 5;
        if (g < g0 + ng)
            return DgClass{a, b, nv, size, g0};
        g0 += ng;
    }
    return DgClass{0, 0, 0, 0, g0}; // past the last group: empty
}

// input pixel (row, column) of class element e
__device__ __forceinline__ void dg_pixel(const DgClass &k, int e, int s, int r0, int &r, int &c)
{
    const int u = e / k.nv, v = e - (e / k.nv) * k.nv;
    c = k.a + s * v;
    const int rs = floordiv(k.b + floor_half(c) - r0, s); // first row of this residue at or after r0
    r = r0 + (k.b + floor_half(c) - r0) - s * rs + s * u;
}

template <int K>
__global__ __launch_bounds__(kGThreads) void conv_gen_dgrad_k(const bf16raw *__restrict__ dy,
                                                              const bf16raw *__restrict__ w,
                                                              bf16raw *__restrict__ dx, GenArgs a,
                                                              int ngroups_total)
{
    constexpr int T = num_taps(K);
    constexpr int NTG = (T + kTG - 1) / kTG;
    extern __shared__ __align__(16) unsigned char smem[];
    bf16raw *win = reinterpret_cast<bf16raw *>(smem + a.win_off);
    bf16raw *wl = reinterpret_cast<bf16raw *>(smem + a.wgt_off);
    bf16raw *outl = reinterpret_cast<bf16raw *>(smem + a.out_off);

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n32 = lane & 31, kh = lane >> 5;
    const int db = blockIdx.x % a.nblk, tstep = gridDim.x / a.nblk;
    const int d0 = db * kNB;
    const int s = a.s;
    const int nst = (a.Cs / kCK) * NTG;
    const size_t HWs = static_cast<size_t>(a.Hs) * a.Ws;
    const size_t HWd = static_cast<size_t>(a.Hd) * a.Wd;
    const int nd = min(kNB, a.Cd - d0);
    const int nrounds = (ngroups_total + 4 * kMG - 1) / (4 * kMG);
    const bool alias = a.out_off == a.win_off; // single round only
    const bool whole = a.CW == a.Cs;            // the window holds every channel

    WgtRegs<true> wr;
    if (a.resident)
        stage_all_weights<true>(wl, w, T, NTG, nst, a.Cs, a.Cd, d0);
    else
        wr.load(w, T, a.Cs, a.Cd, d0, 0, 0);

    for (int tb = blockIdx.x / a.nblk; tb < a.ntot; tb += tstep) {
        const int n = tb / a.tiles, r0 = (tb - n * a.tiles) * a.TR;
        // window row 0 = output row i_lo = floor((r0 - K - s/2) / s)
        const int i_lo = floordiv(r0 - K - (s >> 1), s);

        for (int rd = 0; rd < nrounds; ++rd) {
            // this wave's groups in this round: one class each
            DgClass cls[kMG];
            int slot0[kMG], peven[kMG], pix[kMG];
            int ng = 0;
#pragma unroll
            for (int m = 0; m < kMG; ++m) {
                const int g = rd * 4 * kMG + wave + 4 * m;
                cls[m] = dg_class_of_group(g, s, a.Wd, a.TR);
                // the class is the wave's: keep it in scalar registers
                cls[m].a = __builtin_amdgcn_readfirstlane(cls[m].a);
                cls[m].b = __builtin_amdgcn_readfirstlane(cls[m].b);
                cls[m].nv = __builtin_amdgcn_readfirstlane(cls[m].nv);
                cls[m].size = __builtin_amdgcn_readfirstlane(cls[m].size);
                cls[m].g0 = __builtin_amdgcn_readfirstlane(cls[m].g0);
                const int e0 = (g - cls[m].g0) * 32;
                const bool live = g < ngroups_total;
                if (live)
                    ng = m + 1;
                int r = r0, c = 0;
                if (live)
                    dg_pixel(cls[m], min(e0 + n32, cls[m].size - 1), s, r0, r, c);
                // tile position of this lane's A row (-1 past the class's end)
                pix[m] = (live && e0 + n32 < cls[m].size) ? (r - r0) * a.Wd + c : -1;
                // axial (q, sa) = (c, r - floor(c/2)); class residues (a, b):
                // c_s = (c - a) / s, sa_s = (sa - b) / s (exact)
                const int cs = (c - cls[m].a) / s;
                const int sas = floordiv(r - floor_half(c) - cls[m].b, s);
                // source output (i, j) of a live tap: j = c_s - dQ, i = sa_s - dS + floor(j/2)
                slot0[m] = (sas + floor_half(cs) - i_lo) * a.RP + cs + a.coff;
                peven[m] = (cs & 1) ? 0 : a.RP; // one row less for odd dQ at even c_s
            }
            // taps that reach each group's class, once per round: lane t
            // (t < T) tests tap t against the class residues; the ballot is
            // the group's tap mask (wave-uniform), and the lane keeps the
            // tap's slot offset for the K-steps to read back
            uint64_t tmask[kMG];
            int tdel[kMG], todd[kMG];
            {
                int dq = 0, ds = 0;
                if (lane < T)
                    tap_axial(K, lane, dq, ds);
#pragma unroll
                for (int m = 0; m < kMG; ++m) {
                    const int vq = dq - cls[m].a, vs = ds - cls[m].b;
                    const int dQ = floordiv(vq, s), dS = floordiv(vs, s);
                    const bool match = lane < T && m < ng && vq == dQ * s && vs == dS * s;
                    tmask[m] = __ballot(match);
                    tdel[m] = -(dS + floor_half(dQ)) * a.RP - dQ;
                    todd[m] = dQ & 1;
                }
            }
            floatx16 acc[kMG][2];
#pragma unroll
            for (int m = 0; m < kMG; ++m)
                acc[m][0] = acc[m][1] = floatx16{};

            for (int st = 0; st < nst; ++st) {
                const int c0 = (st / NTG) * kCK, t0 = (st % NTG) * kTG;
                const int cw0 = c0 - c0 % a.CW;
                __syncthreads();
                if (c0 == cw0 && t0 == 0 && (!whole || rd == 0))
                    stage_window(win, dy + (static_cast<size_t>(n) * a.Cs + cw0) * HWs, HWs,
                                 a.Hs, a.Ws, i_lo, a.WR, a.WC, a.coff, a.CW, a.SP, a.split,
                                 a.WCs, a.RP);
                if (!a.resident)
                    wr.store(wl);
                __syncthreads();
                if (!a.resident &&
                    (st + 1 < nst || rd + 1 < nrounds || tb + tstep < a.ntot)) {
                    const int sn = st + 1 < nst ? st + 1 : 0;
                    wr.load(w, T, a.Cs, a.Cd, d0, (sn / NTG) * kCK, (sn % NTG) * kTG);
                }
                if (ng == 0)
                    continue;
                const bf16raw *wst = a.resident ? wl + st * kStageElems : wl;
                const int ntap = min(kTG, T - t0);
                const int cl = c0 - cw0;
                const uint64_t smask = ((uint64_t(1) << ntap) - 1) << t0; // ntap <= 8
#pragma unroll
                for (int m = 0; m < kMG; ++m) {
                    // this stage's taps of the group's class, one at a time
                    uint64_t bits = tmask[m] & smask;
                    while (bits != 0) {
                        const int t = static_cast<int>(__builtin_ctzll(bits));
                        bits &= bits - 1;
                        const int del = __builtin_amdgcn_readlane(tdel[m], t);
                        const int odd = __builtin_amdgcn_readlane(todd[m], t);
                        const int slot = slot0[m] + del - (odd ? peven[m] : 0);
                        const bf16raw *wrow = wst + (t - t0) * kTB + n32 * kCP + 8 * kh;
                        const bf16x8 b0 = *reinterpret_cast<const bf16x8 *>(wrow);
                        const bf16x8 b1 = *reinterpret_cast<const bf16x8 *>(wrow + 32 * kCP);
                        const bf16x8 b2 = *reinterpret_cast<const bf16x8 *>(wrow + 16);
                        const bf16x8 b3 = *reinterpret_cast<const bf16x8 *>(wrow + 32 * kCP + 16);
                        const bf16raw *ap = win + slot * a.SP + cl + 8 * kh;
                        const bf16x8 x0 = *reinterpret_cast<const bf16x8 *>(ap);
                        const bf16x8 x1 = *reinterpret_cast<const bf16x8 *>(ap + 16);
                        acc[m][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x0, b0, acc[m][0], 0, 0, 0);
                        acc[m][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x0, b1, acc[m][1], 0, 0, 0);
                        acc[m][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x1, b2, acc[m][0], 0, 0, 0);
                        acc[m][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x1, b3, acc[m][1], 0, 0, 0);
                    }
                }
            }
            // this round's results into the LDS tile [channel][row-major pixel]
            if (alias)
                __syncthreads(); // the tile overlays the window (single round)
#pragma unroll
            for (int m = 0; m < kMG; ++m) {
                if (m >= ng)
                    break;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    // D row 8 (r / 4) + 4 kh + r % 4 is the A row of that lane
                    const int p = __shfl(pix[m], 8 * (r >> 2) + 4 * kh + (r & 3), 64);
                    if (p < 0)
                        continue;
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        outl[(j * 32 + n32) * a.OP + p] = from_f<bf16raw>(acc[m][j][r]);
                }
            }
        }
        __syncthreads();
        const int M = a.TR * a.Wd; // TR divides H: whole tiles
        bf16raw *xbase =
            dx + (static_cast<size_t>(n) * a.Cd + d0) * HWd + static_cast<size_t>(r0) * a.Wd;
        const int nv = M >> 3; // W % 8 == 0
        for (int e = threadIdx.x; e < nd * nv; e += kGThreads) {
            const int d = e / nv, v = e - d * nv;
            const bf16raw *src = outl + d * a.OP + 8 * v;
            const uint2 lo = *reinterpret_cast<const uint2 *>(src);
            const uint2 hi = *reinterpret_cast<const uint2 *>(src + 4);
            *reinterpret_cast<uint4 *>(xbase + d * HWd + 8 * v) = make_uint4(lo.x, lo.y, hi.x, hi.y);
        }
    }
}

inline int cdiv(long a, long b) { return static_cast<int>((a + b - 1) / b); }

constexpr size_t kGenLds = 160 * 1024; // one block per CU (registers allow no more)

size_t align256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

// Output staging pitch: the tile's pixels padded to whole 32-pixel groups,
// plus 4 (rows 8 mod 16 bytes apart for the 8-byte writes).
int out_pitch(int M) { return ((M + 31) & ~31) + 4; }

// LDS offsets of a plan -- window (WR x WC slots of SP bf16), output
// staging (overlaying the window when `alias`), weights (every stage when
// resident, else one) -- if they fit.
bool finish_plan(GenArgs &a, int M, bool alias, int nst, size_t &lds)
{
    const size_t win = align256(sizeof(bf16raw) * static_cast<size_t>(a.WR) * a.RP * a.SP);
    const size_t out = align256(sizeof(bf16raw) * static_cast<size_t>(kNB) * out_pitch(M));
    const size_t wgt = sizeof(bf16raw) * static_cast<size_t>(a.resident ? nst : 1) * kStageElems;
    const size_t base = alias ? std::max(win, out) : win + out;
    if (base + wgt > kGenLds)
        return false;
    a.TG = kTG;
    a.win_off = 0;
    a.out_off = alias ? 0 : static_cast<int>(win);
    a.wgt_off = static_cast<int>(base);
    a.OP = out_pitch(M);
    lds = base + wgt;
    return true;
}

// Window channel counts to try, widest first: divisors of Cs among 128, 64, 32.
int window_channels(int Cs, int idx)
{
    static const int cand[3] = {128, 64, 32};
    int found = 0;
    for (int c : cand)
        if (c <= Cs && Cs % c == 0) {
            if (found == idx)
                return c;
            ++found;
        }
    return 0;
}

// Persistent grid: as many blocks per destination block as CUs, at most one
// per tile.
int persistent_blocks(const GenArgs &a)
{
    const int per_db = std::max(1, std::min(a.ntot, device_cus() / std::max(1, a.nblk)));
    return per_db * a.nblk;
}

bool plan_fwd(const ConvShape &sh, GenArgs &a, size_t &lds)
{
    if (sh.k < 1 || sh.k > 3 || sh.Ci % kCK != 0 || sh.W % 8 != 0 || sh.Wo > 256 || sh.Ho < 1 ||
        sh.D != 1)
        return false;
    a = GenArgs{};
    a.N = sh.N;
    a.Cs = sh.Ci;
    a.Cd = sh.Co;
    a.Hs = sh.H;
    a.Ws = sh.W;
    a.Hd = sh.Ho;
    a.Wd = sh.Wo;
    a.s = sh.s;
    a.coff = sh.k;
    a.WC = sh.s * (sh.Wo - 1) + 2 * sh.k + 1;
    a.split = sh.s;
    a.WCs = cdiv(a.WC, sh.s);
    a.RP = a.split * a.WCs;
    a.nblk = cdiv(sh.Co, kNB);
    const int nst = (sh.Ci / kCK) * cdiv(sh.T, kTG);
    // the tallest tile of at most 256 pixels, then the widest window, then
    // resident weights
    for (int TR = std::max(1, std::min(sh.Ho, 256 / sh.Wo)); TR >= 1; --TR) {
        a.TR = TR;
        a.WR = sh.s * (TR - 1) + (sh.s >> 1) + 2 * sh.k + 1;
        a.tiles = cdiv(sh.Ho, TR);
        a.ntot = sh.N * a.tiles;
        for (int ci = 0; window_channels(sh.Ci, ci) > 0; ++ci) {
            a.CW = window_channels(sh.Ci, ci);
            a.SP = a.CW + 8;
            for (int res = 1; res >= 0; --res) {
                a.resident = res;
                if (finish_plan(a, TR * sh.Wo, true, nst, lds))
                    return true;
            }
        }
    }
    return false;
}

// groups of 32 class elements of a tile of TR rows
int dg_groups(int s, int W, int TR)
{
    int g = 0;
    for (int cl = 0; cl < s * s; ++cl) {
        const int a = cl / s;
        const int nv = (W - a + s - 1) / s;
        g += ((TR / s) * nv + 31) / 32;
    }
    return g;
}

bool plan_dgrad(const ConvShape &sh, GenArgs &a, size_t &lds, int &ngroups)
{
    if (sh.k < 1 || sh.k > 3 || sh.Co % kCK != 0 || sh.W % 8 != 0 || sh.Wo % 8 != 0 ||
        sh.W > 256 || sh.Ho < 1 || sh.D != 1 || sh.H % sh.s != 0)
        return false;
    a = GenArgs{};
    a.N = sh.N;
    a.Cs = sh.Co;
    a.Cd = sh.Ci;
    a.Hs = sh.Ho;
    a.Ws = sh.Wo;
    a.Hd = sh.H;
    a.Wd = sh.W;
    a.s = sh.s;
    a.coff = sh.k;
    a.WC = sh.Wo + 2 * sh.k;
    a.split = 1;
    a.WCs = a.WC;
    a.RP = a.WC;
    a.nblk = cdiv(sh.Ci, kNB);
    const int nst = (sh.Co / kCK) * cdiv(sh.T, kTG);
    // tiles of TR input rows, a multiple of s dividing H, at most 256 pixels
    // where possible; then the widest window, then resident weights
    for (int TR = sh.s * std::max(1, 256 / (sh.s * sh.W)); TR >= sh.s; TR -= sh.s) {
        if (sh.H % TR != 0)
            continue;
        a.TR = TR;
        const int i_lo = -((sh.k + (sh.s >> 1) + sh.s - 1) / sh.s); // floor((-k - s/2) / s)
        const int i_hi = (TR - 1 + sh.k) / sh.s;                     // floor((TR - 1 + k) / s)
        a.WR = i_hi - i_lo + 1;
        a.tiles = sh.H / TR;
        a.ntot = sh.N * a.tiles;
        ngroups = dg_groups(sh.s, sh.W, TR);
        const bool single = ngroups <= 4 * kMG;
        for (int ci = 0; window_channels(sh.Co, ci) > 0; ++ci) {
            a.CW = window_channels(sh.Co, ci);
            a.SP = a.CW + 8;
            for (int res = 1; res >= 0; --res) {
                a.resident = res;
                if (finish_plan(a, TR * sh.W, single, nst, lds))
                    return true;
            }
        }
    }
    return false;
}

} // namespace

bool bf16_gen_fwd_ok(const ConvShape &sh)
{
    GenArgs a;
    size_t lds = 0;
    return plan_fwd(sh, a, lds);
}

bool bf16_gen_dgrad_ok(const ConvShape &sh)
{
    GenArgs a;
    size_t lds = 0;
    int ng = 0;
    return plan_dgrad(sh, a, lds, ng);
}

hipError_t bf16_gen_fwd(const void *x, const void *w, const void *bias, void *y,
                        const ConvShape &sh, bool relu, hipStream_t st)
{
    GenArgs a;
    size_t lds = 0;
    if (!plan_fwd(sh, a, lds))
        return hipErrorInvalidConfiguration;
    a.relu = relu ? 1 : 0;
    dim3 grid(persistent_blocks(a));
#define HEX_GF(KV)                                                                           \
    HEX_LAUNCH((conv_gen_fwd_k<KV>), grid, dim3(kGThreads), lds, st,                        \
               static_cast<const bf16raw *>(x), static_cast<const bf16raw *>(w),             \
               static_cast<const bf16raw *>(bias), static_cast<bf16raw *>(y), a)
    if (sh.k == 1)
        HEX_GF(1);
    else if (sh.k == 2)
        HEX_GF(2);
    else
        HEX_GF(3);
#undef HEX_GF
    return hipGetLastError();
}

hipError_t bf16_gen_dgrad(const void *dy, const void *w, void *dx, const ConvShape &sh,
                          hipStream_t st)
{
    GenArgs a;
    size_t lds = 0;
    int ngroups = 0;
    if (!plan_dgrad(sh, a, lds, ngroups))
        return hipErrorInvalidConfiguration;
    dim3 grid(persistent_blocks(a));
#define HEX_GD(KV)                                                                           \
    HEX_LAUNCH((conv_gen_dgrad_k<KV>), grid, dim3(kGThreads), lds, st,                      \
               static_cast<const bf16raw *>(dy), static_cast<const bf16raw *>(w),            \
               static_cast<bf16raw *>(dx), a, ngroups)
    if (sh.k == 1)
        HEX_GD(1);
    else if (sh.k == 2)
        HEX_GD(2);
    else
        HEX_GD(3);
#undef HEX_GD
    return hipGetLastError();
}

} // namespace hexk
