// k_mfma_bf16.hip -- bf16 convolutions on the matrix cores (fp32 accumulate)
// for input channel counts that are a multiple of 32, at stride 1.
//
// Implicit GEMM for the forward pass and, with the point-reflected kernel
// and the channel roles swapped, for the stride-1 data gradient:
//   D[pixel][oc] = sum_{t, ic} A[pixel][(t, ic)] * B[(t, ic)][oc]
//   forward:        A = x at pixel + tap t,  B[(t, ic)][oc] = w[oc][ic][t]
//   data gradient:  A = dy at pixel + tap t, B[(t, ic)][oc] = w[ic][oc][T-1-t]
// The contraction index runs over taps, then input channels, so the 8 A
// values of a lane are 8 consecutive channels of one pixel.
//
// Common to both kernels below: the input window of a pixel tile (full-width
// rows plus k halo rows, k zero columns on each side) is staged channel-last
// in LDS from contiguous 8-pixel chunks of the NCHW planes through an 8x8
// register transpose, so an A fragment is one 16-byte LDS read and a tap is
// a fixed slot offset (one window row further for odd tap columns when the
// pixel's column is odd).  The weights of a block's output channels are
// copied once from global memory (16-byte coalesced loads) into LDS as
// [oc][t][ic], where a B fragment is one 16-byte read, and then held in
// registers or kept resident in LDS.  Results get bias, ReLU and round-to-
// nearest-even in registers, go through LDS as [oc][pixel], and leave as
// contiguous 16-byte stores.  LDS pitches follow measured bank behaviour of
// gfx950: 16-byte fragment reads of 32 rows are conflict-free at a row pitch
// that is an odd multiple of 16 bytes, of 16 rows at 32 mod 64 bytes;
// 8-byte writes of 16 or 32 rows at 8 mod 16 bytes.
//
// conv_bf16_wide32_k (preferred): v_mfma_f32_32x32x16_bf16, one block of 8
// waves per CU, each block a contiguous run of row tiles, the next tile's
// rows prefetched into registers while the current one is computed, the A
// fragments of the next two K-steps in flight.  Where LDS holds it, the
// window is a ring of TR + 2K rows kept from tile to tile of an image (a
// tile after the first stages only its TR new rows) and the results are
// staged in a region of their own.  The 32x32 instruction keeps the matrix
// cores at about 2 PFLOP/s with one or two waves per SIMD, where the 16x16
// one needs more waves than the registers allow.
// conv_bf16_wide_k (fallback for other channel counts): 16x16x32, 4 waves,
// two blocks per CU, pixel tiles handed out so that the blocks of one XCD
// work on neighbouring tiles at the same time.
#include <algorithm>
#include <type_traits>

#include "hexdev.h"
#include "kernels.h"

namespace hexk {
namespace {

using namespace hexgeom;

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kXcd = 8;

struct WideArgs {
    int N, H, W;
    int IC, OC;         // channels of the kernel's input and output tensors
    int KS;             // K-steps: T * IC / 32
    int TR, ntr;        // rows per pixel tile, pixel tiles per image
    int ptiles;         // pixel tiles in the batch
    int nocc;           // output-channel chunks
    int spx;            // tile slots per XCD (per chunk)
    int nslots;         // tile slots per chunk (= 8 * spx)
    int LCP, CS;        // input window: slots per row, bf16 per slot
    int OP;             // output staging pitch (bf16 per channel)
    int WP;             // weight row pitch in LDS (bf16 per output channel)
    int tile_off;       // byte offset of the tile region in LDS
    int vec_out;        // 16-byte output stores allowed
    int wgroups;        // channel groups whose weights are copied per pass (registers mode)
    int per_block;      // pixel tiles per block (prefetching kernel)
    int ring;           // 32x32 kernel: window rows kept from tile to tile of an image
    int out_off;        // 32x32 kernel: byte offset of the output staging in LDS
};

__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel)
{
    return __builtin_amdgcn_perm(hi, lo, sel);
}

typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// two floats -> two bf16 (round to nearest even) in one dword, lo first;
// gfx950 converts a pair in one instruction
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2{lo, hi}, bf16x2));
}

// Copy the weights of kernel-output channels [o_lo, o_lo + nrow) into LDS
// as wl[ocl * WP + t * IC + ic] (zero for channels >= OC).  Every load of a
// thread is issued before the first LDS write, so the copy costs about one
// memory latency.
//   forward, w[oc][ic][t]: the rows form one contiguous run whose length
//     and start are multiples of 32 elements (IC % 32 == 0): 16-byte loads,
//     8 consecutive (ic, t) per load;
//   data gradient, w[ic][oc][t] (ic = the convolution's output channel):
//     one run of nrow * T elements per ic, read element by element.
template <int T, bool REFLECT, int NTHR = kThreads>
__device__ __forceinline__ void stage_weights(bf16raw *__restrict__ wl, const bf16raw *__restrict__ w,
                                              int o_lo, int nrow, int IC, int OC, int WP)
{
    const int nval = max(0, min(nrow, OC - o_lo)); // rows that exist
    constexpr int U = 8;
    if constexpr (!REFLECT) {
        const int per = IC * T;                     // elements per row, a multiple of 32
        const int nchunk = nrow * per / 8;
        const int nvchunk = nval * per / 8;
        const bf16raw *src = w + static_cast<size_t>(o_lo) * per;
        for (int q0 = threadIdx.x; q0 < nchunk; q0 += U * NTHR) {
            uint4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int q = q0 + u * NTHR;
                v[u] = q < nvchunk ? *reinterpret_cast<const uint4 *>(src + 8 * static_cast<size_t>(q))
                                   : make_uint4(0, 0, 0, 0);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int q = q0 + u * NTHR;
                if (q >= nchunk)
                    break;
                const int ocl = (8 * q) / per;      // a chunk never straddles two rows
                const int rem = 8 * q - ocl * per;
                int ic = rem / T, t = rem - (rem / T) * T;
                bf16raw *dst = wl + ocl * WP;
                const bf16raw *e = reinterpret_cast<const bf16raw *>(&v[u]);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    dst[t * IC + ic] = e[j];
                    if (++t == T) {
                        t = 0;
                        ++ic;
                    }
                }
            }
        }
    } else {
        const int run = nrow * T;                   // per ic
        const int vrun = nval * T;
        const int total = IC * run;
        for (int e0 = threadIdx.x; e0 < total; e0 += U * NTHR) {
            bf16raw v[U];
            int dsti[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int e = e0 + u * NTHR;
                const int ic = e / run;
                const int rest = e - ic * run;
                const int ocl = rest / T, tn = rest - (rest / T) * T;
                const bool ok = e < total && rest < vrun;
                v[u] = ok ? w[(static_cast<size_t>(ic) * OC + o_lo) * T + rest] : bf16raw(0);
                dsti[u] = e < total ? ocl * WP + (T - 1 - tn) * IC + ic : -1;
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (dsti[u] >= 0)
                    wl[dsti[u]] = v[u];
        }
    }
}

// Input window of a pixel tile (rows r0-K .. r0+rows+K-1 of one image, all
// IC channels), staged channel-last into LDS at slot ((r - r0 + K) * LCP +
// c + K).  The rows inside the image are one contiguous run of each NCHW
// plane; a work item is one 8-channel group of one 8-element chunk of that
// run (chunks aligned to 8 elements), consecutive items take consecutive
// channel groups.  load() reads U items of this thread (items it0 + h *
// 256) into registers, commit() transposes them (8 x 8 bf16) into 8 pixel
// slots; zero_halo() clears the K columns on each side and the window rows
// outside the image.
struct WideWindow {
    int e_lo, e_hi, e_al, items, rbase, ra, rb, rows;
    __device__ __forceinline__ WideWindow(int K, int H, int W, int IC, int r0, int rows_)
    {
        rows = rows_;
        rbase = r0 - K;
        ra = max(r0 - K, 0);
        rb = min(r0 + rows_ + K, H);
        e_lo = ra * W;
        e_hi = rb * W;
        e_al = e_lo & ~7;
        items = (IC >> 3) * ((e_hi - e_al + 7) >> 3);
    }
};

template <int K, int U, int NTHR = kThreads> struct WideTileRegs {
    uint4 v[U][8];
    int eb[U], cg[U];

    __device__ __forceinline__ void load(const bf16raw *__restrict__ src, const WideWindow &wd,
                                         int HW, int IC, int it0)
    {
        const int ncg = IC >> 3;
#pragma unroll
        for (int h = 0; h < U; ++h) {
            const int it = it0 + h * NTHR;
            const bool live = it < wd.items;
            const int ch = live ? it / ncg : 0;
            cg[h] = live ? it - ch * ncg : 0;
            // e_al + 8*ch is a multiple of 8 below e_hi <= H*W (a multiple
            // of 8): all 8 elements lie inside the plane
            const int e0 = wd.e_al + 8 * ch;
#pragma unroll
            for (int j = 0; j < 8; ++j)
                v[h][j] = *reinterpret_cast<const uint4 *>(
                    src + static_cast<size_t>(cg[h] * 8 + j) * HW + e0);
            eb[h] = live ? e0 : -1;
        }
    }

    __device__ __forceinline__ void commit(bf16raw *__restrict__ tl, const WideWindow &wd, int W,
                                           int LCP, int CS) const
    {
#pragma unroll
        for (int h = 0; h < U; ++h) {
            if (eb[h] < 0)
                continue;
            // the 8 pixels eb..eb+7 cross at most one row end (W >= 8); slot =
            // window-relative element + 2K per row end crossed + K
            const int r = eb[h] / W;
            const int c = eb[h] - r * W;
            const int base = (eb[h] - wd.rbase * W) + (r - wd.rbase) * 2 * K + K;
#pragma unroll
            for (int px = 0; px < 8; ++px) {
                const int e = eb[h] + px;
                const int brk = (c + px >= W) ? 1 : 0;
                const uint32_t sel = (px & 1) ? 0x07060302u : 0x05040100u;
                uint32_t w4[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const uint32_t lo = reinterpret_cast<const uint32_t *>(&v[h][2 * q])[px >> 1];
                    const uint32_t hi = reinterpret_cast<const uint32_t *>(&v[h][2 * q + 1])[px >> 1];
                    w4[q] = perm(hi, lo, sel);
                }
                const int slot = base + px + brk * 2 * K;
                if (e >= wd.e_lo && e < wd.e_hi)
                    *reinterpret_cast<uint4 *>(tl + static_cast<size_t>(slot) * CS + cg[h] * 8) =
                        make_uint4(w4[0], w4[1], w4[2], w4[3]);
            }
        }
    }
};

template <int K, int NTHR = kThreads>
__device__ __forceinline__ void zero_halo(bf16raw *__restrict__ tl, const WideWindow &wd, int W,
                                          int IC, int LCP, int CS)
{
    const int LR = wd.rows + 2 * K;
    const int v8 = IC >> 3; // 16-byte vectors per slot holding data
    const int side = LR * 2 * K;
    const int nlo = wd.ra - wd.rbase;                 // window rows above the image
    const int out_rows = nlo + (wd.rbase + LR - wd.rb); // ... plus below it
    const int total = (side + out_rows * LCP) * v8;
    for (int e = threadIdx.x; e < total; e += NTHR) {
        const int s = e / v8, q = e - s * v8;
        int slot;
        if (s < side) {
            const int rr = s / (2 * K), j = s - rr * 2 * K;
            slot = rr * LCP + (j < K ? j : W + j);
        } else {
            const int s2 = s - side;
            const int orow = s2 / LCP, c = s2 - orow * LCP;
            const int rr = orow < nlo ? orow : (wd.rb - wd.rbase) + (orow - nlo);
            slot = rr * LCP + c;
        }
        *reinterpret_cast<uint4 *>(tl + static_cast<size_t>(slot) * CS + q * 8) = make_uint4(0, 0, 0, 0);
    }
}

// Whole window, U items per thread per round.
template <int K, int U>
__device__ __forceinline__ void stage_tile(bf16raw *__restrict__ tl, const bf16raw *__restrict__ src,
                                           int H, int W, int IC, int r0, int rows, int LCP, int CS)
{
    const WideWindow wd(K, H, W, IC, r0, rows);
    for (int it0 = threadIdx.x; it0 < wd.items; it0 += U * kThreads) {
        WideTileRegs<K, U> g;
        g.load(src, wd, H * W, IC, it0);
        g.commit(tl, wd, W, LCP, CS);
    }
    zero_halo<K>(tl, wd, W, IC, LCP, CS);
}

// Ring window of the 32x32 kernel.  The window of a tile (rows r0 - K ..
// r0 + TR + K - 1) lives in R = TR + 2K ring rows of LCP slots, image row r
// in ring row (r + K) mod R, so the next tile of the same image finds its
// first 2K rows already there and stages only its TR new ones; the first
// tile of an image (or of a block) stages the whole window.  Staged rows
// inside the image [rlo, rhi) are items of one 8-channel group of one
// 8-element chunk (chunks aligned to 8 elements, as for the full window),
// one per thread.
struct RingRows {
    int e_lo, e_hi, e_al, items;
    __device__ __forceinline__ RingRows(int W, int IC, int rlo, int rhi)
    {
        e_lo = rlo * W;
        e_hi = max(rhi, rlo) * W;
        e_al = e_lo & ~7;
        items = e_hi > e_lo ? (IC >> 3) * ((e_hi - e_al + 7) >> 3) : 0;
    }
};

template <int NTHR> struct RingRegs {
    uint4 v[8];
    int eb, cg;

    __device__ __forceinline__ void load(const bf16raw *__restrict__ src, const RingRows &rw,
                                         int HW, int IC)
    {
        const int ncg = IC >> 3;
        const int it = threadIdx.x;
        const bool live = it < rw.items;
        const int ch = live ? it / ncg : 0;
        cg = live ? it - ch * ncg : 0;
        // e_al + 8*ch is a multiple of 8 below H*W: all 8 elements lie in
        // the plane (and item 0 of an empty range reads chunk 0)
        const int e0 = live ? rw.e_al + 8 * ch : 0;
#pragma unroll
        for (int j = 0; j < 8; ++j)
            v[j] = *reinterpret_cast<const uint4 *>(src + static_cast<size_t>(cg * 8 + j) * HW + e0);
        eb = live ? e0 : -1;
    }

    __device__ __forceinline__ void commit(bf16raw *__restrict__ tl, const RingRows &rw, int K,
                                           int W, int R, int LCP, int CS) const
    {
        if (eb < 0)
            return;
        // the 8 pixels eb..eb+7 cross at most one row end (W >= 8)
        const int r = eb / W, c = eb - r * W;
        int rr = (r + K) % R;
        const int rr1 = rr + 1 == R ? 0 : rr + 1;
#pragma unroll
        for (int px = 0; px < 8; ++px) {
            const int e = eb + px;
            const bool brk = c + px >= W;
            const uint32_t sel = (px & 1) ? 0x07060302u : 0x05040100u;
            uint32_t w4[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t lo = reinterpret_cast<const uint32_t *>(&v[2 * q])[px >> 1];
                const uint32_t hi = reinterpret_cast<const uint32_t *>(&v[2 * q + 1])[px >> 1];
                w4[q] = perm(hi, lo, sel);
            }
            const int slot = (brk ? rr1 * LCP + c + px - W : rr * LCP + c + px) + K;
            if (e >= rw.e_lo && e < rw.e_hi)
                *reinterpret_cast<uint4 *>(tl + static_cast<size_t>(slot) * CS + cg * 8) =
                    make_uint4(w4[0], w4[1], w4[2], w4[3]);
        }
    }
};

// Zeros for the ring window: with cols, the K side columns of all R ring
// rows; and the ring rows of image rows [slo, shi) outside the image.
template <int NTHR>
__device__ __forceinline__ void ring_zero(bf16raw *__restrict__ tl, bool cols, int slo, int shi,
                                          int K, int H, int W, int IC, int R, int LCP, int CS)
{
    const int v8 = IC >> 3;
    const int side = cols ? R * 2 * K : 0;
    const int nlo = max(0, min(shi, 0) - slo);     // rows above the image
    const int nhi = max(0, shi - max(slo, H));     // rows below it
    const int total = (side + (nlo + nhi) * LCP) * v8;
    for (int e = threadIdx.x; e < total; e += NTHR) {
        const int s = e / v8, q = e - s * v8;
        int slot;
        if (s < side) {
            const int rr = s / (2 * K), j = s - rr * 2 * K;
            slot = rr * LCP + (j < K ? j : W + j);
        } else {
            const int s2 = s - side;
            const int o = s2 / LCP, c = s2 - o * LCP;
            const int r = o < nlo ? slo + o : max(slo, H) + (o - nlo);
            slot = ((r + K) % R) * LCP + c;
        }
        *reinterpret_cast<uint4 *>(tl + static_cast<size_t>(slot) * CS + q * 8) = make_uint4(0, 0, 0, 0);
    }
}

// Epilogue of a pixel tile, first half: bias, ReLU and bf16 rounding of
// this wave's MT x NT accumulator tiles into LDS as [oc][pixel] with pitch
// OP (OP = 4 mod 8: the 8-byte writes of 16 channel rows hit distinct
// banks).  Rows of pixels past the tile's end hold garbage, never stored.
template <int NT, int PW, int MT>
__device__ __forceinline__ void wide_epilogue(bf16raw *__restrict__ outl, int OP,
                                              const floatx4 (&acc)[MT][NT], const float (&bv)[NT],
                                              int ocl0, int pg, int m, int kq, int relu)
{
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int ocl = ocl0 + j * 16 + m;
#pragma unroll
        for (int i = 0; i < MT; ++i) {
            const int q0 = (pg + PW * i) * 16 + 4 * kq;
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                v[r] = acc[i][j][r] + bv[j];
                if (relu)
                    v[r] = fmaxf(v[r], 0.f);
            }
            *reinterpret_cast<uint2 *>(outl + ocl * OP + q0) =
                make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
        }
    }
}

// Second half: 16-byte stores of noc channel rows of npix pixels (npix % 8
// == 0) from the LDS tile (row pitch OP, rows 8-byte aligned) to y_base +
// ocl * HW.  Every thread issues exactly NST stores (NV = 16-byte vectors per
// full row); lanes past the end repeat a valid vector -- the same data to the
// same address -- so the number of outstanding memory operations is known at
// compile time and a later wait for loads does not wait for these stores.
template <int NST, int NV, int NTHR = kThreads>
__device__ __forceinline__ void wide_store(bf16raw *__restrict__ y_base, size_t HW,
                                           const bf16raw *__restrict__ outl, int OP, int noc,
                                           int npix)
{
    const int nvec = npix >> 3;
#pragma unroll
    for (int st = 0; st < NST; ++st) {
        const int e = threadIdx.x + st * NTHR;
        const int ocl = min(e / NV, noc - 1);
        const int v8 = min(e - (e / NV) * NV, nvec - 1);
        const bf16raw *src = outl + ocl * OP + v8 * 8;
        const uint2 lo = *reinterpret_cast<const uint2 *>(src);
        const uint2 hi = *reinterpret_cast<const uint2 *>(src + 4);
        *reinterpret_cast<uint4 *>(y_base + static_cast<size_t>(ocl) * HW + v8 * 8) =
            make_uint4(lo.x, lo.y, hi.x, hi.y);
    }
}

// Scalar variant for tiles whose rows do not start on 8-element boundaries.
template <int NTHR = kThreads>
__device__ __forceinline__ void wide_store_scalar(bf16raw *__restrict__ y_base, size_t HW,
                                                  const bf16raw *__restrict__ outl, int OP,
                                                  int noc, int npix)
{
    for (int e = threadIdx.x; e < noc * npix; e += NTHR) {
        const int ocl = e / npix, p = e - ocl * npix;
        y_base[static_cast<size_t>(ocl) * HW + p] = outl[ocl * OP + p];
    }
}

// One K-step for the wave's MT pixel tiles and NT channel tiles: the tap
// (dq, ds) of step ks, read at each A row's centre slot plus the tap's slot
// offset (one window row further for odd tap columns when the lane's pixel
// column is odd).  Rows past the tile's last pixel read a clamped, valid
// centre; their results are never stored.
template <int K, int NT, int MT>
__device__ __forceinline__ void wide_kstep(floatx4 (&acc)[MT][NT], const bf16x8 (&bq)[NT],
                                           const unsigned char *__restrict__ tlb,
                                           const int (&adr)[MT], int oddoff, int t, int icoff,
                                           int rowb, int slotb)
{
    int dq = 0, ds = 0;
    tap_axial(K, t, dq, ds);
    const int toff = (ds + floor_half(dq)) * rowb + dq * slotb + icoff + ((dq & 1) ? oddoff : 0);
    uint4 qa[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
        qa[i] = *reinterpret_cast<const uint4 *>(tlb + adr[i] + toff);
#pragma unroll
    for (int i = 0; i < MT; ++i) {
        const bf16x8 av = __builtin_bit_cast(bf16x8, qa[i]);
#pragma unroll
        for (int j = 0; j < NT; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bq[j], acc[i][j], 0, 0, 0);
    }
}

// KS > 0: B fragments of all KS K-steps held in registers; KS == 0: read
// from the LDS-resident weights every K-step (a.KS K-steps).
// Wave w: pixel group w % PW (pixel tiles w % PW + PW * i, i < MT) and
// output-channel group w / PW (NT tiles of 16 channels).
template <int K, int KS, int NT, int PW, int MT, bool REFLECT>
__global__ __launch_bounds__(kThreads, KS > 0 ? 2 : 1) void conv_bf16_wide_k(
    const bf16raw *__restrict__ xin, const bf16raw *__restrict__ w, const bf16raw *__restrict__ bias,
    bf16raw *__restrict__ y, WideArgs a, int relu)
{
    constexpr int T = num_taps(K);
    constexpr bool WL = KS == 0;
    constexpr int OG = kWaves / PW;
    constexpr int OCB = OG * NT * 16;
    constexpr int ICB = WL ? 1 : KS / T; // 32-channel blocks per tap (registers mode)
    extern __shared__ __align__(16) unsigned char smem[];
    bf16raw *wl = reinterpret_cast<bf16raw *>(smem);
    bf16raw *tl = reinterpret_cast<bf16raw *>(smem + a.tile_off);

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int m = lane & 15, kq = lane >> 4;
    const int pg = wave % PW, og = wave / PW;

    // persistent work: a fixed channel chunk and strided pixel-tile slots
    const int b = blockIdx.x;
    const int xcd = b % kXcd, jj = b / kXcd;
    const int occ = jj % a.nocc, sj = jj / a.nocc;
    const int slot0 = xcd * a.spx + sj;
    const int oc_base = occ * OCB;
    const bool wave_live = oc_base + og * NT * 16 < a.OC;

    // ---- weights
    bf16x8 bfr[WL ? 1 : KS][NT];
    if constexpr (WL) {
        stage_weights<T, REFLECT>(wl, w, oc_base, OCB, a.IC, a.OC, a.WP);
    } else {
        // through the tile region: all channel groups at once if they fit
        // (a.wgroups == OG), else one group at a time
        for (int g = 0; g < OG; g += a.wgroups) {
            __syncthreads();
            stage_weights<T, REFLECT>(tl, w, oc_base + g * NT * 16, a.wgroups * NT * 16, a.IC,
                                      a.OC, a.WP);
            __syncthreads();
            if (og >= g && og < g + a.wgroups) {
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
#pragma unroll
                    for (int j = 0; j < NT; ++j)
                        bfr[ks][j] = *reinterpret_cast<const bf16x8 *>(
                            tl + ((og - g) * NT * 16 + j * 16 + m) * a.WP + ks * 32 + 8 * kq);
            }
        }
    }

    const int H = a.H, W = a.W;
    const int HW = H * W;
    const int rowb = a.LCP * a.CS * 2; // bytes per window row
    const int slotb = a.CS * 2;        // bytes per slot
    const unsigned char *tlb = reinterpret_cast<const unsigned char *>(tl);
    float bv[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int oc = oc_base + og * NT * 16 + j * 16 + m;
        bv[j] = (bias != nullptr && oc < a.OC) ? to_f(bias[oc]) : 0.f;
    }

    for (int pt = slot0; pt < a.ptiles; pt += a.nslots) {
        const int n = pt / a.ntr;
        const int r0 = (pt - n * a.ntr) * a.TR;
        const int rows = min(a.TR, H - r0);
        const int npix = rows * W;

        __syncthreads(); // the previous tile's (or the weight copy's) LDS reads are done
        stage_tile<K, (KS >= 14) ? 1 : 2>(tl, xin + static_cast<size_t>(n) * a.IC * HW, H, W, a.IC, r0, rows, a.LCP,
                      a.CS);
        __syncthreads();

        // centre-slot byte address of this lane's A row in each tile (W is
        // even and tiles start on multiples of 16 pixels, so the column
        // parity of the lane's pixel is the parity of m)
        int adr[MT];
#pragma unroll
        for (int i = 0; i < MT; ++i) {
            const int p = min((pg + PW * i) * 16 + m, npix - 1);
            const int pr = p / W, pc = p - pr * W;
            adr[i] = ((pr + K) * a.LCP + pc + K) * slotb + kq * 16;
        }
        const int oddoff = (m & 1) ? rowb : 0;
        floatx4 acc[MT][NT];
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NT; ++j)
                acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

        if (wave_live) {
            if constexpr (WL) {
                const int icb = a.IC >> 5;
                const bf16raw *wrow = wl + (og * NT * 16 + m) * a.WP + 8 * kq;
                for (int ks = 0; ks < a.KS; ++ks) {
                    const int t = ks / icb;
                    bf16x8 bq[NT];
#pragma unroll
                    for (int j = 0; j < NT; ++j)
                        bq[j] = *reinterpret_cast<const bf16x8 *>(wrow + j * 16 * a.WP + ks * 32);
                    wide_kstep<K, NT, MT>(acc, bq, tlb, adr, oddoff, t, (ks - t * icb) * 64,
                                          rowb, slotb);
                }
            } else {
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    // bound the scheduler's hoisting of fragment loads to one
                    // K-step (the weights already hold most registers)
                    __builtin_amdgcn_sched_barrier(0);
                    wide_kstep<K, NT, MT>(acc, bfr[ks], tlb, adr, oddoff, ks / ICB,
                                          (ks % ICB) * 64, rowb, slotb);
                }
            }
        }

        // epilogue: bias, ReLU, bf16 into LDS as [oc][pixel], then 16-byte stores
        __syncthreads();
        bf16raw *outl = tl;
        if (wave_live)
            wide_epilogue<NT, PW, MT>(outl, a.OP, acc, bv, og * NT * 16, pg, m, kq, relu);
        __syncthreads();
        const int noc = min(OCB, a.OC - oc_base);
        bf16raw *ybase =
            y + (static_cast<size_t>(n) * a.OC + oc_base) * HW + static_cast<size_t>(r0) * W;
        if (a.vec_out)
            wide_store<(OCB * PW * MT * 2 + kThreads - 1) / kThreads, PW * MT * 2>(ybase, HW, outl,
                                                                                  a.OP, noc, npix);
        else
            wide_store_scalar(ybase, HW, outl, a.OP, noc, npix);
    }
}

// ---------------------------------------------------------------------------
// 32x32x16 kernel.  v_mfma_f32_32x32x16_bf16 (lane layout checked on the
// device): a[i] = A[lane % 32][8 * (lane / 32) + i],
// b[i] = B[8 * (lane / 32) + i][lane % 32],
// d[r] = D[8 * (r / 4) + 4 * (lane / 32) + r % 4][lane % 32].
// A = 32 pixels x 16 channels of one tap (one 16-byte LDS read per lane),
// B = 16 channels x 32 output channels, D = 32 pixels x 32 output channels:
// each lane ends with 4 runs of 4 consecutive pixels of one channel.
// K-step ks covers tap ks / (IC/16) and channels 16 * (ks % (IC/16)) + 0..15.
//
// One block of 8 waves per CU (two waves per SIMD): wave w computes output
// channels 32 * (w / PW) .. +31 for pixel tiles (w % PW) + PW * i, i < MT,
// of 32 pixels each.  Block b owns the contiguous pixel tiles
// [b * per, (b + 1) * per) -- consecutive row tiles, whose shared halo rows
// the same CU has just read and finds in its L2 -- and loads the next tile's
// window into registers while it computes the current one.  The weights of
// the block's channels are held in registers (KS > 0: KS K-steps) or stay
// resident in LDS (KS == 0, for long contractions: a.KS K-steps).
constexpr int kThreads32 = 512;

template <int K, int KS, bool WL, int OG, int PW, int MT, bool REFLECT>
__global__ __launch_bounds__(kThreads32) void conv_bf16_wide32_k(
    const bf16raw *__restrict__ xin, const bf16raw *__restrict__ w, const bf16raw *__restrict__ bias,
    bf16raw *__restrict__ y, WideArgs a, int relu)
{
    static_assert(OG * PW == kThreads32 / 64, "8 waves");
    constexpr int T = num_taps(K);
    static_assert(KS % T == 0, "whole 16-channel blocks per tap");
    constexpr int ICB = KS / T; // 16-channel blocks per tap
    constexpr int OCB = OG * 32;
    constexpr int PIX = PW * MT * 32;
    extern __shared__ __align__(16) unsigned char smem[];
    bf16raw *wl = reinterpret_cast<bf16raw *>(smem);
    bf16raw *tl = reinterpret_cast<bf16raw *>(smem + a.tile_off);

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n32 = lane & 31, kh = lane >> 5;
    const int pg = wave % PW, og = wave / PW;

    // block -> (channel chunk, run of tiles); the chunks of one run are 8
    // blocks apart, i.e. on the same XCD, and share its L2
    const int xcd = blockIdx.x % kXcd, jj = blockIdx.x / kXcd;
    const int occ = jj % a.nocc;
    const int slot = (jj / a.nocc) * kXcd + xcd;
    const int oc_base = occ * OCB;
    const int OCc = min(OCB, a.OC - oc_base); // channels of this chunk
    const bool wave_live = og * 32 < OCc;
    const int t_begin = slot * a.per_block;
    const int t_end = min(t_begin + a.per_block, a.ptiles);
    if (t_begin >= t_end)
        return; // the whole block

    // ---- weights
    bf16x8 bfr[WL ? 1 : KS];
    (void)bfr;
    if constexpr (WL) {
        stage_weights<T, REFLECT, kThreads32>(wl, w, oc_base, OCB, a.IC, a.OC, a.WP);
    } else {
        for (int g = 0; g < OG; g += a.wgroups) {
            __syncthreads();
            stage_weights<T, REFLECT, kThreads32>(tl, w, oc_base + g * 32, a.wgroups * 32, a.IC,
                                                  a.OC, a.WP);
            __syncthreads();
            if (og >= g && og < g + a.wgroups) {
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    bfr[ks] = *reinterpret_cast<const bf16x8 *>(
                        tl + ((og - g) * 32 + n32) * a.WP + ks * 16 + 8 * kh);
            }
        }
    }
    float bv;
    {
        const int oc = oc_base + og * 32 + n32;
        bv = (bias != nullptr && oc < a.OC) ? to_f(bias[oc]) : 0.f;
    }

    const int H = a.H, W = a.W;
    const int HW = H * W;
    const int rowb = a.LCP * a.CS * 2;
    const int slotb = a.CS * 2;
    const unsigned char *tlb = reinterpret_cast<const unsigned char *>(tl);
    // W even, tiles on multiples of 32: a lane's pixel column has the parity of n32
    const int podd = n32 & 1;
    const bf16raw *wrow = wl + (og * 32 + n32) * a.WP + 8 * kh;
    const int R = a.TR + 2 * K; // ring rows

    // tile pt stages image rows [slo, shi): the whole window for the first
    // tile of an image or of the block (every tile without the ring), else
    // the TR rows after the previous window
    auto staged = [&](int pt, int &slo, int &shi) {
        const int n = pt / a.ntr, r0 = (pt - n * a.ntr) * a.TR;
        const bool whole = !a.ring || pt == t_begin || r0 == 0;
        slo = whole ? r0 - K : r0 + K;
        shi = r0 + a.TR + K;
    };
    RingRegs<kThreads32> g;
    {
        int slo, shi;
        staged(t_begin, slo, shi);
        const int n = t_begin / a.ntr;
        g.load(xin + static_cast<size_t>(n) * a.IC * HW,
               RingRows(W, a.IC, max(slo, 0), min(shi, H)), HW, a.IC);
    }
    for (int pt = t_begin; pt < t_end; ++pt) {
        const int n = pt / a.ntr;
        const int r0 = (pt - n * a.ntr) * a.TR;
        const int rows = min(a.TR, H - r0);
        const int npix = rows * W;
        int slo, shi;
        staged(pt, slo, shi);

        __syncthreads(); // the previous tile's (or the weight copy's) LDS reads are done
        g.commit(tl, RingRows(W, a.IC, max(slo, 0), min(shi, H)), K, W, R, a.LCP, a.CS);
        ring_zero<kThreads32>(tl, slo == r0 - K, slo, shi, K, H, W, a.IC, R, a.LCP, a.CS);
        __syncthreads();
        if (pt + 1 < t_end) {
            int slo2, shi2;
            staged(pt + 1, slo2, shi2);
            const int n2 = (pt + 1) / a.ntr;
            g.load(xin + static_cast<size_t>(n2) * a.IC * HW,
                   RingRows(W, a.IC, max(slo2, 0), min(shi2, H)), HW, a.IC);
        }

        // A rows (pixels): column part of the slot address, and the ring row
        // offsets of the image rows d - K from the pixel's row (d = 0 .. 2K),
        // plain and one row further for odd pixel columns (taps with odd dq);
        // pixels past the tile read a clamped valid centre, their results
        // are never stored
        int colb[MT], ro[MT][2 * K + 1], rop[MT][2 * K + 1];
#pragma unroll
        for (int i = 0; i < MT; ++i) {
            const int p = min((pg + PW * i) * 32 + n32, npix - 1);
            const int pr = p / W, pc = p - pr * W;
            colb[i] = (pc + K) * slotb + kh * 16;
            // image row pr + d - K of the tile is ring row (rb + d) mod R
            const int rb = (r0 + pr) % R;
            // (rb + d + 1 < 2R: R = TR + 2K > 2K); computed, not selected
            // from ro, which would put ro in scratch memory
#pragma unroll
            for (int d = 0; d <= 2 * K; ++d) {
                const int rr = rb + d, rq = rr + podd;
                ro[i][d] = (rr >= R ? rr - R : rr) * rowb;
                rop[i][d] = (rq >= R ? rq - R : rq) * rowb;
            }
        }
        floatx16 acc[MT];
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[i][r] = 0.f;

        if (wave_live) {
            // the tap and channel block of K-step ks are compile-time
            // constants once the loop is unrolled
            auto fetch_a = [&](uint4(&q)[MT], int ks) {
                const int t = ks / ICB;
                constexpr TapTable<K> tt;
                const int dq = tt.dq[t], ds = tt.ds[t];
                const int d = K + ds + floor_half(dq); // row of even columns, + K
                const int toff = dq * slotb + (ks % ICB) * 32;
#pragma unroll
                for (int i = 0; i < MT; ++i)
                    q[i] = *reinterpret_cast<const uint4 *>(
                        tlb + ((dq & 1) ? rop[i][d] : ro[i][d]) + colb[i] + toff);
            };
            auto fetch_b = [&](int ks) -> bf16x8 {
                if constexpr (WL)
                    return *reinterpret_cast<const bf16x8 *>(wrow + ks * 16);
                else
                    return bfr[ks];
            };
            // fragments of the next DEPTH - 1 K-steps in flight
            constexpr int DEPTH = 3;
            uint4 qa[DEPTH][MT];
            bf16x8 qb[DEPTH];
#pragma unroll
            for (int d = 0; d < DEPTH - 1 && d < KS; ++d) {
                fetch_a(qa[d], d);
                qb[d] = fetch_b(d);
            }
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                if (ks + DEPTH - 1 < KS) {
                    fetch_a(qa[(ks + DEPTH - 1) % DEPTH], ks + DEPTH - 1);
                    qb[(ks + DEPTH - 1) % DEPTH] = fetch_b(ks + DEPTH - 1);
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int i = 0; i < MT; ++i)
                    acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8, qa[ks % DEPTH][i]), qb[ks % DEPTH], acc[i], 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
            }
        }

        // epilogue: bias, ReLU, bf16 into LDS as [oc][pixel] (pitch OP = 4 mod
        // 8: conflict-free 8-byte writes), then 16-byte stores.  Without the
        // ring the staging overlays the window.
        if (!a.ring)
            __syncthreads();
        bf16raw *outl = reinterpret_cast<bf16raw *>(smem + a.out_off);
        if (wave_live) {
            const int ocl = og * 32 + n32;
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int gq = 0; gq < 4; ++gq) {
                    const int q0 = (pg + PW * i) * 32 + 8 * gq + 4 * kh;
                    float v[4];
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        v[r] = acc[i][4 * gq + r] + bv;
                        if (relu)
                            v[r] = fmaxf(v[r], 0.f);
                    }
                    *reinterpret_cast<uint2 *>(outl + ocl * a.OP + q0) =
                        make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
                }
        }
        __syncthreads();
        bf16raw *ybase =
            y + (static_cast<size_t>(n) * a.OC + oc_base) * HW + static_cast<size_t>(r0) * W;
        if (a.vec_out)
            wide_store<(OCB * PIX / 8 + kThreads32 - 1) / kThreads32, PIX / 8, kThreads32>(
                ybase, HW, outl, a.OP, OCc, npix);
        else
            wide_store_scalar<kThreads32>(ybase, HW, outl, a.OP, OCc, npix);
    }
}

// ---------------------------------------------------------------------------
// Pipelined 32x32x16 kernel for one-row pixel tiles: k = 1, 32 or 64
// channels in, at most 64 out, rows of 64 < W <= 128 pixels (W % 8 == 0).
// The kernel above runs every phase of a tile (commit of the staged rows,
// products, epilogue, stores) one after another with all 8 waves; here two
// roles share each SIMD and one barrier per tile:
//   waves 0-3 compute: wave w takes output channels 32 (w / 2) .. +31 of the
//     row's pixel tiles (w % 2) and (w % 2) + 2 (32 pixels each) with the
//     block's weights in registers, and write the tile's results to one of
//     two LDS output buffers;
//   waves 4-7 stage and store: while tile j is computed they transpose the
//     row that tile j + 1 adds to the window into the ring's spare row and
//     store tile j - 1's results from the other output buffer; input rows
//     are requested two at a time, two tiles before the first is needed.
// The window is a ring of 2K + 2 rows (image row r at ring row (r + K) mod
// (2K + 2)): the row being written is never one being read.  Blocks walk
// runs of at most 32 consecutive rows of one image; a run's first window is
// staged before its first tile.  The staging steps of a run are unrolled,
// so register buffers have fixed names, and the input pointer is not
// declared restrict: with it the compiler moves the prefetch loads down to
// their first use, across the barriers.
// Measured (64 x 64 channels, 128 x 128 rows, 64 images): forward 78-79 us
// against 85-91 us for the kernel above, data gradient 84-85 against 89-93;
// with the products skipped the memory traffic alone takes 73 us, with the
// memory traffic skipped the rest 51 us.
struct PipeArgs {
    int N, H, W, IC, OC;
    int run_rows, runs_per_img, nruns;
    int LCP, CS, OP, WP;
    int out_off; // byte offset of the two output buffers in LDS
};

constexpr int kPipeThreads = 512;
constexpr int kPipeStageThreads = 256; // waves 4-7
constexpr int kPipeBurst = 2;          // input rows requested together (4: no faster)
constexpr int kPipeMaxRows = 32;       // rows per run (the staging steps are unrolled)

// One staged item: 4 channels of 8 consecutive pixels of one input row, a
// 16-byte load from each of 4 planes.  Every staging thread owns one item of
// every row (items past the row's end repeat its last item, rows outside the
// image are read at a valid row and committed as zeros), so loads and
// commits happen on every thread without conditions and the compiler's
// memory-counter waits stay exact.
template <int K, int IC> struct PipeItem {
    uint4 v[4];
    int zero;

    __device__ __forceinline__ void load(const bf16raw *img, size_t HW, int H, int W, int x, int it)
    {
        constexpr int NQ = IC / 4;
        const int itc = min(it, (W / 8) * NQ - 1);
        const int ch = itc / NQ, cq = itc - ch * NQ;
        const int xr = min(max(x, 0), H - 1);
        zero = (x < 0 || x >= H) ? 1 : 0;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            v[j] = *reinterpret_cast<const uint4 *>(img + static_cast<size_t>(cq * 4 + j) * HW +
                                                    xr * W + 8 * ch);
    }

    // transpose into 8 pixel slots of ring row (x + K) mod (2K + 2)
    __device__ __forceinline__ void commit(bf16raw *__restrict__ ring, int W, int LCP, int CS, int x,
                                           int it) const
    {
        constexpr int NQ = IC / 4;
        constexpr int R = 2 * K + 2;
        const int itc = min(it, (W / 8) * NQ - 1);
        const int ch = itc / NQ, cq = itc - ch * NQ;
        const int s0 = ((x + K) % R) * LCP + K + 8 * ch;
#pragma unroll
        for (int px = 0; px < 8; ++px) {
            const uint32_t sel = (px & 1) ? 0x07060302u : 0x05040100u;
            const uint32_t a0 = reinterpret_cast<const uint32_t *>(&v[0])[px >> 1];
            const uint32_t a1 = reinterpret_cast<const uint32_t *>(&v[1])[px >> 1];
            const uint32_t a2 = reinterpret_cast<const uint32_t *>(&v[2])[px >> 1];
            const uint32_t a3 = reinterpret_cast<const uint32_t *>(&v[3])[px >> 1];
            const uint32_t lo = zero ? 0u : perm(a1, a0, sel);
            const uint32_t hi = zero ? 0u : perm(a3, a2, sel);
            *reinterpret_cast<uint2 *>(ring + static_cast<size_t>(s0 + px) * CS + cq * 4) =
                make_uint2(lo, hi);
        }
    }
};

// f(std::integral_constant<int, J>) for J = I, I + 1, ... < N while f
// returns true, as nested conditionals (no loop)
template <int I, int N, typename F> __device__ __forceinline__ void nested_steps(F &&f)
{
    if constexpr (I < N) {
        if (f(std::integral_constant<int, I>{}))
            nested_steps<I + 1, N>(f);
    }
}

// 16-byte stores of one output row (OC channels x W pixels) from an LDS
// output buffer: exactly 4 per staging thread (64 x 128 pixels at most);
// threads past the end repeat the last vector (same data, same address), so
// the count of outstanding memory operations is fixed at compile time.
__device__ __forceinline__ void pipe_store(bf16raw *__restrict__ yb, size_t HW,
                                           const bf16raw *__restrict__ ob, int OP, int OC, int W,
                                           int tid)
{
    const int nv = W / 8, total = OC * nv;
#pragma unroll
    for (int st = 0; st < 4; ++st) {
        const int e = min(tid + st * kPipeStageThreads, total - 1);
        const int oc = e / nv, v8 = e - oc * nv;
        const bf16raw *src = ob + oc * OP + v8 * 8;
        const uint2 lo = *reinterpret_cast<const uint2 *>(src);
        const uint2 hi = *reinterpret_cast<const uint2 *>(src + 4);
        *reinterpret_cast<uint4 *>(yb + static_cast<size_t>(oc) * HW + v8 * 8) =
            make_uint4(lo.x, lo.y, hi.x, hi.y);
    }
}

template <int K, int IC, bool REFLECT>
__global__ __launch_bounds__(kPipeThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void
conv_bf16_pipe_k(const bf16raw *xin, const bf16raw *__restrict__ w,
                 const bf16raw *__restrict__ bias, bf16raw *__restrict__ y, PipeArgs a, int relu)
{
    constexpr int T = num_taps(K);
    constexpr int ICB = IC / 16; // 16-channel blocks per tap
    constexpr int KS = T * ICB;
    constexpr int R = 2 * K + 2;
    constexpr int MT = 2, PW = 2;
    extern __shared__ __align__(16) unsigned char smem[];
    bf16raw *ring = reinterpret_cast<bf16raw *>(smem);
    bf16raw *outb = reinterpret_cast<bf16raw *>(smem + a.out_off);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int H = a.H, W = a.W;
    const size_t HW = static_cast<size_t>(H) * W;
    const int obuf = 64 * a.OP; // bf16 per output buffer

    // weights through the ring region into the computing waves' registers
    stage_weights<T, REFLECT, kPipeThreads>(ring, w, 0, 64, IC, a.OC, a.WP);
    __syncthreads();

    if (wave >= 4) {
        // ---- staging and storing waves
        const int tid = threadIdx.x - 4 * 64;
        __syncthreads(); // the computing waves hold the weights: the ring is free
        // zero the K side columns of every ring row (never written again)
        for (int e = tid; e < R * 2 * K * (IC / 8); e += kPipeStageThreads) {
            const int s = e / (IC / 8), q = e - s * (IC / 8);
            const int rr = s / (2 * K), jc = s - rr * 2 * K;
            const int slot = rr * a.LCP + (jc < K ? jc : W + jc);
            *reinterpret_cast<uint4 *>(ring + static_cast<size_t>(slot) * a.CS + q * 8) =
                make_uint4(0, 0, 0, 0);
        }
        // tile j (j >= 1) adds row rb + j + K; the rows of tiles BU m + 1 ..
        // BU (m + 1) ("burst" m) are requested together, when tile BU m + 1
        // is committed (one tile after the last of burst m - 1), into
        // register buffer m % 2.  Rows past the run repeat its last row, which
        // then lands, unchanged, on the ring row it already occupies.
        constexpr int BU = kPipeBurst;
        PipeItem<K, IC> buf[2][BU];
        for (int ru = blockIdx.x; ru < a.nruns; ru += gridDim.x) {
            const int n = ru / a.runs_per_img;
            const int rb = (ru - n * a.runs_per_img) * a.run_rows;
            const int nt = min(a.run_rows, H - rb);
            const int xlast = rb + nt - 1 + K;
            const bf16raw *img = xin + static_cast<size_t>(n) * IC * HW;
            auto row_of = [&](int jt) { return min(rb + jt + K, xlast); };
            auto load_burst = [&](PipeItem<K, IC>(&b)[BU], int m) {
#pragma unroll
                for (int q = 0; q < BU; ++q)
                    b[q].load(img, HW, H, W, row_of(BU * m + 1 + q), tid);
            };
            auto store_row = [&](int jt) {
                pipe_store(y + static_cast<size_t>(n) * a.OC * HW + static_cast<size_t>(rb + jt) * W,
                           HW, outb + (jt & 1) * obuf, a.OP, a.OC, W, tid);
            };
            // the first window (rows rb - K .. rb + K)
            {
                PipeItem<K, IC> pw[2 * K + 1];
#pragma unroll
                for (int rr = 0; rr <= 2 * K; ++rr)
                    pw[rr].load(img, HW, H, W, rb - K + rr, tid);
#pragma unroll
                for (int rr = 0; rr <= 2 * K; ++rr)
                    pw[rr].commit(ring, W, a.LCP, a.CS, rb - K + rr, tid);
            }
            load_burst(buf[0], 0);
            __syncthreads(); // the run's first window is in place
            // step 0: request burst 1, commit tile 1's row
            load_burst(buf[1], 1);
            buf[0][0].commit(ring, W, a.LCP, a.CS, row_of(1), tid);
            __syncthreads();
            // steps 1 .. nt - 1, unrolled and nested (a step runs only after
            // the previous one), so every buffer index is a constant and the
            // memory-counter waits see one path: a commit waits only for its
            // own burst, never for the burst just requested or the stores
            nested_steps<1, kPipeMaxRows>([&](auto jc) -> bool {
                constexpr int j = decltype(jc)::value;
                if (j >= nt)
                    return false;
                if constexpr (j % BU == 0)
                    load_burst(buf[(j / BU + 1) % 2], j / BU + 1);
                buf[(j / BU) % 2][j % BU].commit(ring, W, a.LCP, a.CS, row_of(j + 1), tid);
                store_row(j - 1);
                __syncthreads();
                return true;
            });
            store_row(nt - 1);
            __syncthreads(); // the last results are read before the next run writes them
        }
        return;
    }

    // ---- computing waves
    const int n32 = lane & 31, kh = lane >> 5;
    const int pg = wave & 1, og = wave >> 1;
    const int ocl = og * 32 + n32;
    const bool wave_live = og * 32 < a.OC;
    bf16x8 bfr[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
        bfr[ks] = *reinterpret_cast<const bf16x8 *>(ring + ocl * a.WP + ks * 16 + 8 * kh);
    const float bv = (bias != nullptr && ocl < a.OC) ? to_f(bias[ocl]) : 0.f;
    __syncthreads(); // weights read
    const int slotb = a.CS * 2, rowb = a.LCP * slotb;
    const unsigned char *ringb = reinterpret_cast<const unsigned char *>(ring);
    int colb[MT], podd[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) {
        const int pc = min((pg + PW * i) * 32 + n32, W - 1);
        colb[i] = (pc + K) * slotb + kh * 16;
        podd[i] = pc & 1;
    }
    for (int ru = blockIdx.x; ru < a.nruns; ru += gridDim.x) {
        const int n = ru / a.runs_per_img;
        const int rb = (ru - n * a.runs_per_img) * a.run_rows;
        const int nt = min(a.run_rows, H - rb);
        (void)n;
        __syncthreads(); // the run's first window is in place
        for (int j = 0; j < nt; ++j) {
            const int rc = rb + j;
            // ring row offsets of image rows rc + d - K (d = 0 .. 2K), plain
            // and one row further for odd pixel columns (odd tap columns)
            int ro[2 * K + 1], rop[MT][2 * K + 1];
#pragma unroll
            for (int d = 0; d <= 2 * K; ++d) {
                const int rr = (rc + d) % R;
                ro[d] = rr * rowb;
#pragma unroll
                for (int i = 0; i < MT; ++i) {
                    const int rq = rr + podd[i];
                    rop[i][d] = (rq >= R ? rq - R : rq) * rowb;
                }
            }
            floatx16 acc[MT];
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    acc[i][r] = 0.f;
            if (wave_live) {
                auto fetch_a = [&](uint4(&q)[MT], int ks) {
                    const int t = ks / ICB;
                    constexpr TapTable<K> tt;
                    const int dq = tt.dq[t], ds = tt.ds[t];
                    const int d = K + ds + floor_half(dq);
                    const int toff = dq * slotb + (ks % ICB) * 32;
#pragma unroll
                    for (int i = 0; i < MT; ++i)
                        q[i] = *reinterpret_cast<const uint4 *>(
                            ringb + ((dq & 1) ? rop[i][d] : ro[d]) + colb[i] + toff);
                };
                constexpr int DEPTH = 3;
                uint4 qa[DEPTH][MT];
#pragma unroll
                for (int d = 0; d < DEPTH - 1 && d < KS; ++d)
                    fetch_a(qa[d], d);
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    if (ks + DEPTH - 1 < KS)
                        fetch_a(qa[(ks + DEPTH - 1) % DEPTH], ks + DEPTH - 1);
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int i = 0; i < MT; ++i)
                        acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            __builtin_bit_cast(bf16x8, qa[ks % DEPTH][i]), bfr[ks], acc[i], 0, 0, 0);
                    __builtin_amdgcn_sched_barrier(0);
                }
                // bias, ReLU, bf16 into output buffer j % 2 as [oc][pixel]
                bf16raw *ob = outb + (j & 1) * obuf;
#pragma unroll
                for (int i = 0; i < MT; ++i)
#pragma unroll
                    for (int gq = 0; gq < 4; ++gq) {
                        const int q0 = (pg + PW * i) * 32 + 8 * gq + 4 * kh;
                        float v[4];
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            v[r] = acc[i][4 * gq + r] + bv;
                            if (relu)
                                v[r] = fmaxf(v[r], 0.f);
                        }
                        *reinterpret_cast<uint2 *>(ob + ocl * a.OP + q0) =
                            make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
                    }
            }
            __syncthreads();
        }
        __syncthreads(); // matches the staging waves' barrier after the run's last stores
    }
}

inline int cdiv(long a, long b) { return static_cast<int>((a + b - 1) / b); }

constexpr size_t kLds2 = 80 * 1024;  // two blocks per CU
constexpr size_t kLds1 = 160 * 1024; // one block per CU

// A kernel configuration.
//   E32 = 1: 32x32x16 kernel, 8 waves, OG channel groups of 32 x PW pixel
//            groups, MT tiles of 32 pixels per wave;
//   E32 = 0: 16x16x32 kernel, 4 waves, NT channel tiles of 16 x PW pixel
//            groups, MT tiles of 16 pixels per wave.
//   KSR = K-steps held in registers (0: weights resident in LDS).
struct WideCfg {
    int E32, NT, PW, MT, KSR; // KSR: K-steps held in registers, 0 = weights in LDS
    int WLK;                  // E32 with weights in LDS: instantiated K-step count
    int waves() const { return E32 ? 8 : kWaves; }
    int OCB() const { return E32 ? (waves() / PW) * 32 : (waves() / PW) * NT * 16; }
    int pix() const { return PW * MT * (E32 ? 32 : 16); }
};

struct WidePlan {
    WideCfg cfg;
    WideArgs a;
    size_t lds;
    int grid;
    bool ok;
};

// Row pitch (bf16) of LDS-resident weights whose 16-byte B fragments are
// read by 16 (E32 = 0) or 32 (E32 = 1) consecutive rows without bank
// conflicts: 32 mod 64 bytes, respectively an odd multiple of 16 bytes.
int resident_pitch(int Kc, bool e32)
{
    if (e32) {
        int p = (Kc + 7) / 8 * 8;
        if ((p / 8) % 2 == 0)
            p += 8;
        return p;
    }
    int p = (Kc + 15) / 16 * 16;
    if ((p / 16) % 2 == 0)
        p += 16;
    return p;
}

// Configurations with an instantiated kernel (see dispatch_wide).
bool instantiated(int k, const WideCfg &c)
{
    if (c.E32) {
        if (c.NT != 1)
            return false;
        if (c.PW == 4 && c.MT == 2) // 64 channels
            return (c.KSR == 0 && k == 2 && c.WLK == 38) ||
                   (k == 1 && (c.KSR == 14 || c.KSR == 28));
        if (c.PW == 2 && c.MT == 2) // 128 channels
            return k == 1 && c.KSR == 28;
        if (c.PW == 8 && c.MT == 1) // 32 channels, weights in LDS
            return c.KSR == 0 && ((k == 2 && c.WLK == 76) || (k == 1 && c.WLK == 56));
        return false;
    }
    if (c.NT == 2 && c.PW == 2 && c.MT == 4)
        return k == 1 && (c.KSR == 7 || c.KSR == 14);
    return c.KSR == 0 && c.NT == 2 && c.PW == 4 && c.MT == 4;
}

bool plan_cfg(const ConvShape &sh, int IC, int OC, const WideCfg &c, WidePlan &pl)
{
    if (sh.W > c.pix())
        return false;
    WideArgs a{};
    a.N = sh.N;
    a.H = sh.H;
    a.W = sh.W;
    a.IC = IC;
    a.OC = OC;
    a.KS = sh.T * IC / (c.E32 ? 16 : 32);
    a.TR = std::min(sh.H, c.pix() / sh.W);
    // 16-byte output rows need tile origins on 8-element boundaries
    while (a.TR > 1 && (a.TR * sh.W) % 8 != 0)
        --a.TR;
    a.ntr = cdiv(sh.H, a.TR);
    a.ptiles = sh.N * a.ntr;
    a.nocc = cdiv(OC, c.OCB());
    a.vec_out = ((a.TR * sh.W) % 8 == 0) ? 1 : 0;
    a.LCP = sh.W + 2 * sh.k;
    // slot pitch: odd multiple of 16 bytes for 32-row fragment reads,
    // 32 mod 64 bytes for 16-row ones
    a.CS = c.E32 ? IC + 8 : IC + 16;
    a.OP = c.pix() + 4; // 8 mod 16 bytes: conflict-free 8-byte epilogue writes
    const size_t tile_in = 2ull * (a.TR + 2 * sh.k) * a.LCP * a.CS;
    const size_t tile_out = 2ull * c.OCB() * a.OP;
    const int og = c.waves() / c.PW;
    const bool two_per_cu = !c.E32 && c.KSR > 0;
    const size_t limit = two_per_cu ? kLds2 : kLds1;
    // 32x32 kernel: the input window and the output staging side by side
    // (the window rows carry over from tile to tile) if LDS holds both,
    // else the staging overlays the window
    auto layout = [&](bool ring, size_t &lds) {
        const size_t in_r = (tile_in + 255) / 256 * 256;
        const size_t tiles = ring ? in_r + tile_out : std::max(tile_in, tile_out);
        if (c.KSR > 0) {
            a.WP = sh.T * IC;
            a.tile_off = 0;
            const size_t wgroup = 2ull * (c.OCB() / og) * a.WP; // bytes per channel group
            a.wgroups = (wgroup * og <= tiles) ? og : 1;
            lds = std::max(tiles, wgroup * a.wgroups);
        } else {
            a.WP = resident_pitch(sh.T * IC, c.E32 != 0);
            a.tile_off = static_cast<int>((2ull * c.OCB() * a.WP + 255) / 256 * 256);
            a.wgroups = 1;
            lds = a.tile_off + tiles;
        }
        a.ring = ring ? 1 : 0;
        a.out_off = a.tile_off + (ring ? static_cast<int>(in_r) : 0);
        return lds <= limit;
    };
    size_t lds = 0;
    if (!(c.E32 && layout(true, lds)) && !layout(false, lds))
        return false;
    if (c.E32) {
        // staged window items of one tile: at most one per thread
        const int slack = (sh.W % 8 == 0) ? 0 : 1;
        const long items = static_cast<long>(IC / 8) *
                           ((static_cast<long>(a.TR + 2 * sh.k) * sh.W + 7) / 8 + slack);
        if (items > kThreads32)
            return false;
        // runs of consecutive tiles, 8 * nocc blocks per round of XCDs
        const int runs = std::max(1, std::min(device_cus() / a.nocc, a.ptiles));
        a.per_block = cdiv(a.ptiles, runs);
        const int nrun = cdiv(a.ptiles, a.per_block);
        pl.grid = cdiv(nrun, kXcd) * kXcd * a.nocc; // blocks past the last run exit at once
    } else {
        const int per_cu = c.KSR > 0 ? 2 : 1;
        const int want = std::max(1, device_cus() * per_cu / (kXcd * a.nocc));
        a.spx = std::max(1, std::min(want, cdiv(a.ptiles, kXcd)));
        a.nslots = kXcd * a.spx;
        pl.grid = a.nslots * a.nocc;
    }
    pl.cfg = c;
    pl.a = a;
    pl.lds = lds;
    pl.ok = true;
    return true;
}

WidePlan plan_wide(const ConvShape &sh, int IC, int OC)
{
    WidePlan pl{};
    pl.ok = false;
    const int KS32 = sh.T * IC / 16, KS16 = sh.T * IC / 32;
    const WideCfg cands[] = {
        {1, 1, 2, 2, KS32, 0}, // 32x32: 128 channels, weights in registers
        {1, 1, 4, 2, KS32, 0}, // 32x32: 64 channels, weights in registers
        {1, 1, 4, 2, 0, KS32}, // 32x32: 64 channels, weights in LDS
        {1, 1, 8, 1, 0, KS32}, // 32x32: 32 channels, weights in LDS
        {0, 2, 2, 4, KS16, 0}, // 16x16 fallbacks
        {0, 2, 4, 4, 0, 0},
    };
    for (const WideCfg &c : cands) {
        if (c.E32 && c.PW == 2 && OC <= 64)
            continue; // 128-channel blocks only for more than 64 channels
        if (!instantiated(sh.k, c))
            continue;
        if (plan_cfg(sh, IC, OC, c, pl))
            return pl;
    }
    return pl;
}

template <int K, int KS, int NT, int PW, int MT, bool R>
hipError_t launch_wide(const WidePlan &pl, const bf16raw *x, const bf16raw *w, const bf16raw *b,
                       bf16raw *y, bool relu, hipStream_t st)
{
    HEX_LAUNCH((conv_bf16_wide_k<K, KS, NT, PW, MT, R>), dim3(pl.grid), dim3(kThreads),
                       pl.lds, st, x, w, b, y, pl.a, relu ? 1 : 0);
    return hipGetLastError();
}

template <int K, int KS, bool WL, int OG, int PW, int MT, bool R>
hipError_t launch_wide32(const WidePlan &pl, const bf16raw *x, const bf16raw *w,
                         const bf16raw *b, bf16raw *y, bool relu, hipStream_t st)
{
    HEX_LAUNCH((conv_bf16_wide32_k<K, KS, WL, OG, PW, MT, R>), dim3(pl.grid),
                       dim3(kThreads32), pl.lds, st, x, w, b, y, pl.a, relu ? 1 : 0);
    return hipGetLastError();
}

template <bool R>
hipError_t dispatch_wide(const WidePlan &pl, int k, const bf16raw *x, const bf16raw *w,
                         const bf16raw *b, bf16raw *y, bool relu, hipStream_t st)
{
    const WideCfg &c = pl.cfg;
    if (c.E32) {
        if (c.PW == 8)
            return k == 1 ? launch_wide32<1, 56, true, 1, 8, 1, R>(pl, x, w, b, y, relu, st)
                          : launch_wide32<2, 76, true, 1, 8, 1, R>(pl, x, w, b, y, relu, st);
        if (c.PW == 2)
            return launch_wide32<1, 28, false, 4, 2, 2, R>(pl, x, w, b, y, relu, st);
        if (c.KSR == 0)
            return launch_wide32<2, 38, true, 2, 4, 2, R>(pl, x, w, b, y, relu, st);
        if (c.KSR == 14)
            return launch_wide32<1, 14, false, 2, 4, 2, R>(pl, x, w, b, y, relu, st);
        return launch_wide32<1, 28, false, 2, 4, 2, R>(pl, x, w, b, y, relu, st);
    }
    if (c.KSR == 0)
        return k == 1 ? launch_wide<1, 0, 2, 4, 4, R>(pl, x, w, b, y, relu, st)
                      : launch_wide<2, 0, 2, 4, 4, R>(pl, x, w, b, y, relu, st);
    if (c.KSR == 7)
        return launch_wide<1, 7, 2, 2, 4, R>(pl, x, w, b, y, relu, st);
    return launch_wide<1, 14, 2, 2, 4, R>(pl, x, w, b, y, relu, st);
}

bool pipe_plan(const ConvShape &sh, int IC, int OC, PipeArgs &a, size_t &lds, int &grid)
{
    if (sh.s != 1 || sh.k != 1 || (IC != 32 && IC != 64) || OC < 1 || OC > 64 || sh.W % 8 != 0 ||
        sh.W <= 64 || sh.W > 128 || sh.N < 1 || sh.H < 1)
        return false;
    const int K = sh.k;
    a.N = sh.N;
    a.H = sh.H;
    a.W = sh.W;
    a.IC = IC;
    a.OC = OC;
    a.LCP = sh.W + 2 * K;
    a.CS = IC + 8;  // odd multiple of 16 bytes: conflict-free 32-row fragment reads
    a.OP = 128 + 4; // 8 mod 16 bytes: conflict-free 8-byte epilogue writes
    a.WP = sh.T * IC;
    const size_t ring = 2ull * (2 * K + 2) * a.LCP * a.CS;
    a.out_off = static_cast<int>((ring + 255) / 256 * 256);
    lds = std::max(static_cast<size_t>(a.out_off) + 2ull * 2 * 64 * a.OP, 2ull * 64 * a.WP);
    if (lds > kLds1)
        return false;
    const int cus = device_cus();
    a.runs_per_img = std::max(cdiv(sh.H, kPipeMaxRows), std::min(sh.H, cdiv(cus, sh.N)));
    a.run_rows = cdiv(sh.H, a.runs_per_img);
    a.runs_per_img = cdiv(sh.H, a.run_rows);
    a.nruns = sh.N * a.runs_per_img;
    grid = std::min(a.nruns, cus);
    return true;
}

template <bool R>
hipError_t launch_pipe(const PipeArgs &a, size_t lds, int grid, const bf16raw *x, const bf16raw *w,
                       const bf16raw *b, bf16raw *y, bool relu, hipStream_t st)
{
    if (a.IC == 64)
        HEX_LAUNCH((conv_bf16_pipe_k<1, 64, R>), dim3(grid), dim3(kPipeThreads), lds, st, x, w, b, y,
                   a, relu ? 1 : 0);
    else
        HEX_LAUNCH((conv_bf16_pipe_k<1, 32, R>), dim3(grid), dim3(kPipeThreads), lds, st, x, w, b, y,
                   a, relu ? 1 : 0);
    return hipGetLastError();
}

} // namespace

bool bf16_wide_ok(const ConvShape &sh, int IC, int OC)
{
    if (sh.s != 1 || (sh.k != 1 && sh.k != 2) || IC % 32 != 0 || IC > 128 || sh.W % 2 != 0 ||
        sh.W < 8 || (static_cast<long>(sh.H) * sh.W) % 8 != 0)
        return false;
    return plan_wide(sh, IC, OC).ok;
}

hipError_t bf16_wide_conv(const void *in, const void *w, const void *bias, void *out,
                          const ConvShape &sh, bool reflect, bool relu, hipStream_t st)
{
    const int IC = reflect ? sh.Co : sh.Ci;
    const int OC = reflect ? sh.Ci : sh.Co;
    {
        PipeArgs pa{};
        size_t lds = 0;
        int grid = 0;
        if (pipe_plan(sh, IC, OC, pa, lds, grid)) {
            const bf16raw *x = static_cast<const bf16raw *>(in);
            const bf16raw *wp = static_cast<const bf16raw *>(w);
            bf16raw *y = static_cast<bf16raw *>(out);
            if (reflect)
                return launch_pipe<true>(pa, lds, grid, x, wp, nullptr, y, false, st);
            return launch_pipe<false>(pa, lds, grid, x, wp, static_cast<const bf16raw *>(bias), y,
                                      relu, st);
        }
    }
    const WidePlan pl = plan_wide(sh, IC, OC);
    if (!pl.ok)
        return hipErrorInvalidValue;
    const bf16raw *x = static_cast<const bf16raw *>(in);
    const bf16raw *wp = static_cast<const bf16raw *>(w);
    bf16raw *y = static_cast<bf16raw *>(out);
    if (reflect)
        return dispatch_wide<true>(pl, sh.k, x, wp, nullptr, y, false, st);
    return dispatch_wide<false>(pl, sh.k, x, wp, static_cast<const bf16raw *>(bias), y, relu, st);
}

} // namespace hexk
