// k_wgrad32.hip -- bf16 weight and bias gradient on the matrix cores for
// input and output channel counts that are multiples of 32, at stride 1:
//   dw[co][ci][t] = sum_{n, p} dy[n][co][p] * x[n][ci][p + tap t]
//   db[co]        = sum_{n, p} dy[n][co][p]
// One GEMM per tap, D_t[co][ci] = sum_p dy[co][p] * x[ci][p + tap t], with
// the pixels as the contraction index, on v_mfma_f32_32x32x16_bf16:
//   a[i] = A[lane % 32][8 * (lane / 32) + i]: dy of channel co at 8 pixels,
//   b[i] = B[8 * (lane / 32) + i][lane % 32]: x of channel ci at the same 8
//          pixels moved by tap t,
//   d[r] = D[8 * (r / 4) + 4 * (lane / 32) + r % 4][lane % 32].
//
// Pixel order.  A tap's row offset depends on the column parity of the
// centre (offset-column addressing, Sec. 2.1), so the contraction runs over
// runs of 8 pixels of one row and one column parity: the tiles of x and dy
// are stored in LDS with every row split into its even and its odd columns
// (split index j = column / 2, rows padded to WS, a multiple of 8).  For a
// centre of parity p in split position j, tap (dq, ds) reads row +
// drow(p, dq, ds), parity (p + dq) & 1, split position j + ((p + dq) >> 1):
// the same offset for all 8 pixels of a run, and for all lanes (one tap per
// GEMM).  The split position moves by s = (p + dq) >> 1 in {-1, 0, 1}
// elements; s = 0 is one aligned 16-byte read, s = +-1 one aligned 16-byte
// read plus one 4-byte read and four byte-aligns, all fixed at compile time.
// A K-step (16 pixels) is two runs of the same parity.  Zero pads around
// the split rows and zero rows outside the image give the padding taps.
//
// Work split.  One block of 8 waves per CU (two per SIMD) owns a contiguous
// run of pixel tiles (full-width rows) and has two kinds of wave that meet
// at the two barriers of every tile: waves 4-7 stage the next tile in
// registers while the others compute and write it to LDS between the
// barriers; waves 0-3 compute.  They run separate loops, so the staging
// registers and the accumulators are never live in the same wave (each of
// the two may use 256).  Computing wave w owns one 32-channel block of ci,
// a group of taps (compile-time; one loop per group, so each group's
// accumulators keep their registers) and every 32-channel block of co in
// the pass (at most two), so each B fragment feeds one product per co block
// and no two waves add to the same output; the wave of the first ci block
// and the last (smallest) tap group also sums dy for db.  K-steps go in
// pairs with the A fragments alternating between two register sets, and
// every tap's B fragment of the next K-step is requested right after that
// tap's products.  Each block writes its accumulators to its own partial
// slot exactly as they sit in the registers (one 64-lane register = 64
// contiguous floats, whole 256-byte lines), and a final kernel adds the
// slots in a fixed order and scatters the sums to dw[co][ci][t] and db --
// deterministic.
#include <algorithm>
#include <type_traits>

#include "hexdev.h"
#include "kernels.h"
#include "shear.h"

namespace hexk {
namespace {

using namespace hexgeom;

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kP = 256;      // producer threads: waves 4..7 stage the next tile
constexpr int kT = 2 * kP;   // threads per block: waves 0..3 compute, 4..7 stage
constexpr int kWaves = 4;    // computing waves, one per SIMD
constexpr int kRegChunk = 64; // floats per partial chunk (one register of a wave)
constexpr int kMaxRounds = 32; // staging items per thread at most

struct Wg32Args {
    int N, H, W, CI, CO;
    int co0, COT;  // this pass covers output channels co0 .. co0 + CO - 1 of COT
    int WS;        // split row length of one parity (elements), multiple of 8
    int XS;        // x split segment: 8 zero pad + WS + 8 zero pad
    int TR, ntr, ptiles, per_block;
    int dyc;       // dy LDS pitch per channel (elements)
    int xc;        // x LDS pitch per channel (elements)
    int x_off;     // element offset of the x region in LDS
    int nparts;    // partial slots (= blocks)
    int nchunk;    // partial chunks per slot: tiles * 16 + db chunks
    int items_x, items_dy; // staging items of a full tile
    int cpr;       // staging chunks per image row
    FastDiv fcpr, fxr, ftr; // division by cpr, TR + 2K, TR
    // regular staging (Wg32RegsR): channel blocks per row (0: general
    // staging), channels per round, log2 of the chunks per row
    int rg, rpu, lcpr;
};

__device__ __forceinline__ int udiv(int n, const FastDiv &f)
{
    return static_cast<int>(fdiv(static_cast<uint32_t>(n), f));
}

__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel)
{
    return __builtin_amdgcn_perm(hi, lo, sel);
}
__device__ __forceinline__ uint32_t align2(uint32_t hi, uint32_t lo)
{
    return __builtin_amdgcn_alignbyte(hi, lo, 2); // (hi:lo) >> 16
}

// The thread index behind an empty asm: an item's address arithmetic is
// then redone at every tile instead of being hoisted out of the tile loop,
// where it would hold about eight registers per item for the whole kernel.
__device__ __forceinline__ int opaque_tid()
{
    int t = threadIdx.x;
    asm volatile("" : "+v"(t));
    return t;
}

// Staged window of one pixel tile: rows r0 - K .. r0 + TR + K - 1 of x and
// rows r0 .. r0 + TR - 1 of dy; rows outside the image or past the tile end
// (dy) are zero.  Item: one CW-column chunk of one row of one channel.
template <int K, int CW, int U> struct Wg32Regs {
    typedef typename std::conditional<CW == 8, uint4, uint2>::type Chunk;
    Chunk v[U];
    uint32_t okm; // bit u: item u holds image data (else it stages zeros)

    // Every load is issued unconditionally (rows outside the image read row
    // 0 of the plane, items past the end read item 0) so that none waits for
    // another; okm says which to keep.
    __device__ __forceinline__ void load(const bf16raw *__restrict__ x,
                                         const bf16raw *__restrict__ dy, const Wg32Args &a,
                                         int n, int r0, int rows)
    {
        const size_t HW = static_cast<size_t>(a.H) * a.W;
        const int XR = a.TR + 2 * K;
        const int total = a.items_x + a.items_dy;
        const int tid = opaque_tid() - kP;
        okm = 0;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int it0 = tid + u * kP;
            const int it = it0 < total ? it0 : 0;
            int ch, c, r;
            bool ok;
            const bf16raw *src;
            if (it < a.items_x) {
                const int rest = udiv(it, a.fcpr);
                c = it - rest * a.cpr;
                ch = udiv(rest, a.fxr);
                const int rr = rest - ch * XR;
                r = r0 - K + rr;
                ok = r >= 0 && r < a.H;
                src = x + (static_cast<size_t>(n) * a.CI + ch) * HW;
            } else {
                const int i2 = it - a.items_x;
                const int rest = udiv(i2, a.fcpr);
                c = i2 - rest * a.cpr;
                ch = udiv(rest, a.ftr);
                const int rr = rest - ch * a.TR;
                r = r0 + rr;
                ok = rr < rows;
                src = dy + (static_cast<size_t>(n) * a.COT + a.co0 + ch) * HW;
            }
            ok = ok && it0 < total;
            v[u] = *reinterpret_cast<const Chunk *>(src + static_cast<size_t>(ok ? r : 0) * a.W + c * CW);
            okm |= ok ? (1u << u) : 0u;
        }
    }

    // even columns of the chunk to parity 0, odd to parity 1
    __device__ __forceinline__ void commit(bf16raw *__restrict__ lds, const Wg32Args &a) const
    {
        const int XR = a.TR + 2 * K;
        const int total = a.items_x + a.items_dy;
        constexpr uint32_t E = 0x05040100u, O = 0x07060302u;
        const int tid = opaque_tid() - kP;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int it = tid + u * kP;
            if (it >= total)
                continue;
            int c, off0, off1;
            if (it < a.items_x) {
                const int rest = udiv(it, a.fcpr);
                c = it - rest * a.cpr;
                const int ch = udiv(rest, a.fxr), rr = rest - ch * XR;
                const int b = a.x_off + ch * a.xc + (rr * 2) * a.XS + 8 + c * (CW / 2);
                off0 = b;
                off1 = b + a.XS;
            } else {
                const int i2 = it - a.items_x;
                const int rest = udiv(i2, a.fcpr);
                c = i2 - rest * a.cpr;
                const int ch = udiv(rest, a.ftr), rr = rest - ch * a.TR;
                const int b = ch * a.dyc + (rr * 2) * a.WS + c * (CW / 2);
                off0 = b;
                off1 = b + a.WS;
            }
            const bool ok = (okm >> u) & 1u;
            if constexpr (CW == 8) {
                const uint4 q = ok ? v[u] : make_uint4(0, 0, 0, 0);
                *reinterpret_cast<uint2 *>(lds + off0) = make_uint2(perm(q.y, q.x, E), perm(q.w, q.z, E));
                *reinterpret_cast<uint2 *>(lds + off1) = make_uint2(perm(q.y, q.x, O), perm(q.w, q.z, O));
            } else {
                const uint2 q = ok ? v[u] : make_uint2(0, 0);
                *reinterpret_cast<uint32_t *>(lds + off0) = perm(q.y, q.x, E);
                *reinterpret_cast<uint32_t *>(lds + off1) = perm(q.y, q.x, O);
            }
        }
    }
};

// Regular staging, for 16-byte chunks where the chunks per row (cpr, a
// power of two) divide the staging threads and both channel counts (x and
// this pass's dy) are G times rpu = kP / cpr.  Thread tid stages chunk
// tid % cpr of channel tid / cpr (relative) in every round; round u covers
// rpu channels of one row: x window row u / G, channels (u % G) * rpu, for
// u < rx = (TR + 2K) G, then dy row u / G - (TR + 2K).  Where a round reads
// and writes is then the same for the whole block and a compile-time
// multiple of a few strides: per item one load, and at the commit one
// address add, four permutes and two LDS writes.
template <int K, int U, int G> struct Wg32RegsR {
    uint4 v[U];
    uint32_t okm; // bit u: round u holds image data (the same for all threads)

    __device__ __forceinline__ void load(const bf16raw *__restrict__ x,
                                         const bf16raw *__restrict__ dy, const Wg32Args &a,
                                         int n, int r0, int rows)
    {
        const size_t HW = static_cast<size_t>(a.H) * a.W;
        const int tid = static_cast<int>(threadIdx.x) - kP;
        const uint32_t voff = static_cast<uint32_t>((tid >> a.lcpr) * HW +
                                                    (tid & ((1 << a.lcpr) - 1)) * 8);
        const int XR = a.TR + 2 * K, rx = XR * G, rt = rx + a.TR * G;
        const int RH = a.rpu * a.H * a.W; // elements between the channel blocks of a row
        const bf16raw *xn = x + static_cast<size_t>(n) * a.CI * HW;
        const bf16raw *xw = xn + static_cast<ptrdiff_t>(r0 - K) * a.W;
        // dy round u reads row u / G - XR: the base takes XR rows off
        const bf16raw *yw = dy + (static_cast<size_t>(n) * a.COT + a.co0) * HW +
                            static_cast<ptrdiff_t>(r0 - XR) * a.W;
        // rounds in the image: x rows lo .. hi - 1 of the window, dy rows
        // below the tile's end
        const int lo = max(0, K - r0), hi = min(XR, a.H - r0 + K);
        uint32_t m = 0;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int rr = u / G;
            const bool ok = u < rx ? (rr >= lo && rr < hi) : (u < rt && rr - XR < rows);
            m |= ok ? (1u << u) : 0u;
        }
        okm = __builtin_amdgcn_readfirstlane(m);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int ro = (u / G) * a.W + (u % G) * RH; // offset from the base
            const bf16raw *src = ((okm >> u) & 1u) ? (u < rx ? xw : yw) + ro : xn;
            v[u] = *reinterpret_cast<const uint4 *>(src + voff);
        }
    }

    // even columns of the chunk to parity 0, odd to parity 1.  Without
    // branches: rounds outside the image write zeros (a select), rounds past
    // the tile's last one write to this lane's 16 bytes of the sink region at
    // the end of LDS.  (With a branch per round the staging waves issued
    // about 600 scalar instructions and 150 branches per tile, and the
    // commit took about 3 us of every tile while the computing waves waited.)
    __device__ __forceinline__ void commit(bf16raw *__restrict__ lds, const Wg32Args &a) const
    {
        constexpr uint32_t E = 0x05040100u, O = 0x07060302u;
        const int tid = static_cast<int>(threadIdx.x) - kP;
        const int j = tid >> a.lcpr, c4 = (tid & ((1 << a.lcpr) - 1)) * 4;
        const int XR = a.TR + 2 * K, rx = XR * G, rt = rx + a.TR * G;
        const int bx = a.x_off + j * a.xc + 8 + c4;
        const int by = j * a.dyc + c4 - XR * 2 * a.WS; // dy round u: row u / G - XR
        const int sx = a.rpu * a.xc, sy = a.rpu * a.dyc;
        const int sink = a.x_off + a.CI * a.xc + (threadIdx.x & 63) * 8;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool isx = u < rx;
            const int rr = u / G, cb = u % G;
            const int offx = bx + rr * 2 * a.XS + cb * sx;
            const int offy = by + rr * 2 * a.WS + cb * sy;
            const bool live = u < rt;
            const int off0 = live ? (isx ? offx : offy) : sink;
            const int off1 = live ? off0 + (isx ? a.XS : a.WS) : sink + 4;
            const bool ok = (okm >> u) & 1u;
            const uint4 q = v[u];
            const uint32_t e0 = ok ? perm(q.y, q.x, E) : 0u, e1 = ok ? perm(q.w, q.z, E) : 0u;
            const uint32_t o0 = ok ? perm(q.y, q.x, O) : 0u, o1 = ok ? perm(q.w, q.z, O) : 0u;
            *reinterpret_cast<uint2 *>(lds + off0) = make_uint2(e0, e1);
            *reinterpret_cast<uint2 *>(lds + off1) = make_uint2(o0, o1);
        }
    }
};

// B fragment as read from LDS: the 16-byte aligned chunk holding the run
// and, for a run shifted by one split position, the neighbouring 4 bytes.
// The byte-aligns that form the fragment are left to the product that uses
// it, so waiting for the read does not come right after issuing it.
struct BRaw {
    uint4 c;
    uint32_t e;
};

template <int S> __device__ __forceinline__ BRaw read_shifted(const bf16raw *__restrict__ p)
{
    BRaw r;
    r.c = *reinterpret_cast<const uint4 *>(p);
    if constexpr (S == 0) {
        r.e = 0;
    } else {
        // the offset behind an empty asm: merged with the chunk into one
        // 4-byte aligned 20-byte load, the read would become three
        int off = S == 1 ? 8 : -2;
        asm("" : "+v"(off));
        r.e = *reinterpret_cast<const uint32_t *>(p + off);
    }
    return r;
}

// the 8 split elements starting S (-1, 0, 1) positions after the chunk
template <int S> __device__ __forceinline__ bf16x8 frag_shifted(const BRaw &r)
{
    const uint4 c0 = r.c;
    if constexpr (S == 0)
        return __builtin_bit_cast(bf16x8, c0);
    else if constexpr (S == 1)
        return __builtin_bit_cast(bf16x8, make_uint4(align2(c0.y, c0.x), align2(c0.z, c0.y),
                                                     align2(c0.w, c0.z), align2(r.e, c0.w)));
    else
        return __builtin_bit_cast(bf16x8, make_uint4(align2(c0.x, r.e), align2(c0.y, c0.x),
                                                     align2(c0.z, c0.y), align2(c0.w, c0.z)));
}

// Where the runs of a K-step start.  Lanes kh = 0 / 1 take runs 2q and
// 2q + 1 of K-step q; run i lies in window row i / rpr at split position
// 8 * (i % rpr).  Kept as element offsets of the run in a dy channel
// (rows of 2 * WS) and in an x channel (rows of 2 * XS), advanced one
// K-step (16 split positions) at a time.
struct WgRun {
    int j0, ao, xo;
    __device__ __forceinline__ void init(int kh, int WS, int XS)
    {
        j0 = ao = xo = 8 * kh;
        wrap(WS, XS);
    }
    __device__ __forceinline__ void wrap(int WS, int XS)
    {
        // a split row holds at least one run, so two steps suffice
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            if (j0 >= WS) {
                j0 -= WS;
                ao += WS;          // + 2 WS - WS
                xo += 2 * XS - WS;
            }
        }
    }
    __device__ __forceinline__ void next(int WS, int XS)
    {
        j0 += 16;
        ao += 16;
        xo += 16;
        wrap(WS, XS);
    }
};

// A fragments (dy of each co block) of the runs at r, column parity P.
template <int P, int NCB>
__device__ __forceinline__ void wg_fetchA(bf16x8 (&a)[NCB], const bf16raw *__restrict__ dyb,
                                          int dyblk, int WS, const WgRun &r)
{
    const bf16raw *p = dyb + P * WS + r.ao;
#pragma unroll
    for (int c = 0; c < NCB; ++c)
        a[c] = *reinterpret_cast<const bf16x8 *>(p + c * dyblk);
}

// Split-position shift of tap t for centres of parity P: -1, 0 or 1.
template <int K, int P> __device__ __forceinline__ constexpr int tap_shift(int t)
{
    constexpr TapTable<K> tt;
    return floor_half(P + tt.dq[t]);
}

// Offset of tap t's B runs from the runs of A in an x channel: window row
// K + drow, column parity (P + dq) & 1 (the same for the whole block).
template <int K, int P> __device__ __forceinline__ int tap_xoff(int t, int XS)
{
    constexpr TapTable<K> tt;
    const int dq = tt.dq[t], ds = tt.ds[t];
    return ((K + tap_drow(dq, ds, P)) * 2 + ((P + dq) & 1)) * XS;
}

// B fragment of tap t for the runs at xr (x moved by the tap), as read.
template <int K, int P>
__device__ __forceinline__ BRaw wg_readB(int t, const bf16raw *__restrict__ xr, int toff)
{
    const int sh = tap_shift<K, P>(t);
    const bf16raw *base = xr + toff;
    if (sh == 0)
        return read_shifted<0>(base);
    if (sh == 1)
        return read_shifted<1>(base);
    return read_shifted<-1>(base);
}

template <int K, int P> __device__ __forceinline__ bf16x8 wg_fragB(int t, const BRaw &r)
{
    const int sh = tap_shift<K, P>(t);
    if (sh == 0)
        return frag_shifted<0>(r);
    if (sh == 1)
        return frag_shifted<1>(r);
    return frag_shifted<-1>(r);
}

// One K-step: the products of every tap with the A fragments a, each
// followed by the request for that tap's B fragment at the runs xr of the
// next K-step, so a fragment has the rest of a K-step's products to arrive.
template <int K, int P, int T0, int NT, int NCB, int TPG>
__device__ __forceinline__ void wg_kstep(floatx16 (&acc)[NCB][TPG], float (&dbs)[NCB],
                                         bool do_db, const bf16x8 (&a)[NCB], BRaw (&b)[NT],
                                         const bf16raw *__restrict__ xr, const int (&toff)[NT])
{
    if (do_db) {
#pragma unroll
        for (int c = 0; c < NCB; ++c)
#pragma unroll
            for (int e = 0; e < 8; ++e)
                dbs[c] += static_cast<float>(a[c][e]);
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const bf16x8 bf = wg_fragB<K, P>(T0 + t, b[t]);
#pragma unroll
        for (int c = 0; c < NCB; ++c)
            acc[c][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[c], bf, acc[c][t], 0, 0, 0);
        b[t] = wg_readB<K, P>(T0 + t, xr, toff[t]);
        // keep the read here, a tap's products ahead of its use
        __builtin_amdgcn_sched_barrier(0);
    }
}

// All K-steps of column parity P for taps [T0, T1), two per loop turn so
// that the A fragments alternate between two register sets; the next
// K-step's A fragments are requested before this one's products.
template <int K, int P, int T0, int T1, int NCB, int TPG>
__device__ __forceinline__ void wg_parity(floatx16 (&acc)[NCB][TPG], float (&dbs)[NCB],
                                          bool do_db, const bf16raw *__restrict__ dyb, int dyblk,
                                          const bf16raw *__restrict__ xb, int WS, int XS, int nq,
                                          int kh)
{
    // nq >= 1: a tile holds at least one K-step (the planner pairs runs)
    constexpr int NT = T1 - T0;
    int toff[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
        toff[t] = tap_xoff<K, P>(T0 + t, XS);
    WgRun r;
    r.init(kh, WS, XS);
    bf16x8 a0[NCB], a1[NCB];
    wg_fetchA<P, NCB>(a0, dyb, dyblk, WS, r);
    BRaw b[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
        b[t] = wg_readB<K, P>(T0 + t, xb + r.xo, toff[t]);
    // pairs of K-steps with no exit between them (an exit there would let
    // the compiler sink the B requests below the products); the last
    // K-step requests its own runs again
    int q = 0;
    for (; q + 2 <= nq; q += 2) {
        r.next(WS, XS);
        wg_fetchA<P, NCB>(a1, dyb, dyblk, WS, r);
        wg_kstep<K, P, T0, NT, NCB, TPG>(acc, dbs, do_db, a0, b, xb + r.xo, toff);
        WgRun rn = r;
        rn.next(WS, XS);
        const bool more = q + 2 < nq;
        r.j0 = more ? rn.j0 : r.j0;
        r.ao = more ? rn.ao : r.ao;
        r.xo = more ? rn.xo : r.xo;
        wg_fetchA<P, NCB>(a0, dyb, dyblk, WS, r);
        wg_kstep<K, P, T0, NT, NCB, TPG>(acc, dbs, do_db, a1, b, xb + r.xo, toff);
    }
    if (q < nq)
        wg_kstep<K, P, T0, NT, NCB, TPG>(acc, dbs, do_db, a0, b, xb + r.xo, toff);
}

// A computing wave of ci block ib and tap group GI (taps T0 .. T1 - 1) over
// the block's run of tiles: both barriers of every tile, the products of
// both column parities, then its accumulators to the block's partial slot.
// One instantiation per group keeps each group's registers its own.
template <int K, int NIB, int NCB, int TPG, int GI>
__device__ __forceinline__ void wg_consume(const bf16raw *__restrict__ lds, float *__restrict__ part,
                                           const Wg32Args &a, int ib, int t_begin, int t_end)
{
    constexpr int T = num_taps(K);
    constexpr int T0 = GI * TPG;
    constexpr int T1 = (T0 + TPG < T) ? T0 + TPG : T;
    constexpr int NT = T1 > T0 ? T1 - T0 : 0;
    const int lane = threadIdx.x & 63, n32 = lane & 31, kh = lane >> 5;
    const int slot = blockIdx.x;

    floatx16 acc[NCB][TPG];
#pragma unroll
    for (int c = 0; c < NCB; ++c)
#pragma unroll
        for (int i = 0; i < TPG; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[c][i][r] = 0.f;
    float dbs[NCB];
#pragma unroll
    for (int c = 0; c < NCB; ++c)
        dbs[c] = 0.f;
    // the db sums go to the last tap group, which has the fewest taps
    constexpr int G = (T + TPG - 1) / TPG;
    const bool do_db = ib == 0 && GI == G - 1;
    const bf16raw *dyb = lds + n32 * a.dyc;
    const int dyblk = 32 * a.dyc; // next co block
    const bf16raw *xb = lds + a.x_off + (ib * 32 + n32) * a.xc + 8;
    const int rpr = a.WS >> 3; // runs per split row
    // K-steps: pairs of runs of one parity; run i = (row i / rpr, split
    // position 8 * (i % rpr)); lanes kh = 0 / 1 take runs 2q / 2q + 1
    const int nq = (a.TR * rpr) >> 1;
    for (int pt = t_begin; pt < t_end; ++pt) {
        __syncthreads();
        __syncthreads(); // tile pt is in LDS
        if constexpr (NT > 0) {
            wg_parity<K, 0, T0, T1, NCB, TPG>(acc, dbs, do_db, dyb, dyblk, xb, a.WS, a.XS, nq,
                                              kh);
            wg_parity<K, 1, T0, T1, NCB, TPG>(acc, dbs, do_db, dyb, dyblk, xb, a.WS, a.XS, nq,
                                              kh);
        }
    }

    // partial slot of this block: tile (t, ib, cb) -> chunks (tile * 16 + r),
    // one 64-float chunk per accumulator register, lanes in order
#pragma unroll
    for (int c = 0; c < NCB; ++c) {
#pragma unroll
        for (int i = 0; i < NT; ++i) {
            const int tile = ((T0 + i) * NIB + ib) * NCB + c;
#pragma unroll
            for (int r = 0; r < 16; ++r)
                part[part_index(tile * 16 * kRegChunk + r * kRegChunk + lane, slot, a.nparts)] =
                    acc[c][i][r];
        }
    }
    if (do_db) {
        const int base = T * NIB * NCB * 16 * kRegChunk; // db after the tiles
#pragma unroll
        for (int c = 0; c < NCB; ++c) {
            // lanes n32 and n32 + 32 hold the same channel
            const float s = dbs[c] + __shfl_xor(dbs[c], 32, 64);
            if (kh == 0)
                part[part_index(base + c * 32 + n32, slot, a.nparts)] = s;
        }
    }
}

template <int K, int NIB, int NCB, int TPG, int GI, int G>
__device__ __forceinline__ void wg_consume_group(int g, const bf16raw *__restrict__ lds,
                                                 float *__restrict__ part, const Wg32Args &a,
                                                 int ib, int t_begin, int t_end)
{
    if constexpr (GI < G) {
        if (g == GI)
            wg_consume<K, NIB, NCB, TPG, GI>(lds, part, a, ib, t_begin, t_end);
        else
            wg_consume_group<K, NIB, NCB, TPG, GI + 1, G>(g, lds, part, a, ib, t_begin, t_end);
    }
}

// Waves: NIB ci blocks x G = 4 / NIB tap groups; NCB co blocks per wave.
template <int K, int NIB, int NCB, int CW, int U, int RG>
__global__ __launch_bounds__(kT) __attribute__((amdgpu_waves_per_eu(2, 2))) void wgrad32_k(
    const bf16raw *__restrict__ x, const bf16raw *__restrict__ dy, float *__restrict__ part,
    Wg32Args a)
{
    constexpr int T = num_taps(K);
    constexpr int G = kWaves / NIB;
    constexpr int TPG = (T + G - 1) / G; // taps per group
    extern __shared__ __align__(16) bf16raw lds[];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const bool producer = wave >= kWaves;
    const int ib = wave % NIB, g = wave / NIB;
    const int slot = blockIdx.x;

    // zero the whole LDS once: pads and unused split positions stay zero
    {
        const int total = (a.x_off + a.CI * a.xc) / 8;
        for (int e = threadIdx.x; e < total; e += kT)
            reinterpret_cast<uint4 *>(lds)[e] = make_uint4(0, 0, 0, 0);
    }

    const int t_begin = slot * a.per_block;
    const int t_end = min(t_begin + a.per_block, a.ptiles);

    // Staging waves: hold the next tile in registers while the computing
    // waves work on the current one from LDS, and write it to LDS between
    // the two barriers of every tile.  Both kinds of wave pass the same
    // barriers; the two loops keep the staging registers and the
    // accumulators out of each other's way.
    if (producer) {
        typename std::conditional<(RG > 0), Wg32RegsR<K, U, RG>, Wg32Regs<K, CW, U>>::type regs;
        if (t_begin < t_end) {
            const int n = t_begin / a.ntr, r0 = (t_begin - n * a.ntr) * a.TR;
            regs.load(x, dy, a, n, r0, min(a.TR, a.H - r0));
        }
        for (int pt = t_begin; pt < t_end; ++pt) {
            __syncthreads(); // previous tile's reads done (and the LDS clear)
            regs.commit(lds, a);
            __syncthreads();
            if (pt + 1 < t_end) {
                const int n = (pt + 1) / a.ntr, r0 = (pt + 1 - n * a.ntr) * a.TR;
                regs.load(x, dy, a, n, r0, min(a.TR, a.H - r0));
            }
        }
        return;
    }

    wg_consume_group<K, NIB, NCB, TPG, 0, G>(g, lds, part, a, ib, t_begin, t_end);
}

// Sum the slots of every partial position in a fixed order and scatter to
// dw[co][ci][t] / db[co].  Block = 64 positions x kRedSlices slot slices;
// each thread adds every kRedSlices-th slot, issuing kRedBatch loads before
// adding any, then the slices are added by a fixed tree in LDS.
constexpr int kRedSlices = 16;
constexpr int kRedBatch = 16; // slots per thread whose loads are in flight together

__global__ __launch_bounds__(kRegChunk * kRedSlices) void wgrad32_reduce_k(
    const float *__restrict__ part, int nparts, int npos, int CI, int CO, int co0, int T,
    float *__restrict__ dw, float *__restrict__ db)
{
    __shared__ float red[kRedSlices][kRegChunk];
    const int el = threadIdx.x % kRegChunk, sl = threadIdx.x / kRegChunk;
    const int pos = blockIdx.x * kRegChunk + el;
    float acc = 0.f;
    if (pos < npos) {
        for (int p0 = 0; p0 < nparts; p0 += kRedSlices * kRedBatch) {
            float v[kRedBatch];
#pragma unroll
            for (int u = 0; u < kRedBatch; ++u) {
                const int p = p0 + sl + u * kRedSlices;
                v[u] = p < nparts ? part[part_index(pos, p, nparts)] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < kRedBatch; ++u)
                acc += v[u];
        }
    }
    red[sl][el] = acc;
    for (int half = kRedSlices / 2; half > 0; half >>= 1) {
        __syncthreads();
        if (sl < half)
            red[sl][el] += red[sl + half][el];
    }
    if (sl != 0 || pos >= npos)
        return;
    const float v = red[0][el];
    const int NIB = CI >> 5, NCB = CO >> 5;
    const int ntile_pos = T * NIB * NCB * 16 * kRegChunk;
    if (pos < ntile_pos) {
        const int tile = pos / (16 * kRegChunk);
        const int r = (pos / kRegChunk) % 16, lane = pos % kRegChunk;
        const int cb = tile % NCB, ib = (tile / NCB) % NIB, t = tile / (NCB * NIB);
        const int co = co0 + cb * 32 + 8 * (r / 4) + 4 * (lane / 32) + r % 4;
        const int ci = ib * 32 + lane % 32;
        dw[(static_cast<size_t>(co) * CI + ci) * T + t] = v;
    } else if (db != nullptr) {
        db[co0 + pos - ntile_pos] = v;
    }
}

inline int cdiv(long a, long b) { return static_cast<int>((a + b - 1) / b); }

constexpr size_t kLdsMax = 160 * 1024;

// Most staging items per thread (prefetch registers: 16 or 8 bytes each);
// every variant holds 32 next to its accumulators without scratch spills
// (the compiler's resource report).
constexpr int kMaxItems = kMaxRounds;

// Most 32-channel co blocks per wave next to its taps' accumulators (each
// block and tap one 16-register tile, at most 192 registers): k = 1 splits
// 7 taps over 4 / NIB groups, k = 2 splits 19.  0: not supported.
constexpr int max_ncb(int K, int NIB)
{
    return K == 1 ? (NIB <= 2 ? 2 : 1) : (NIB == 1 ? 2 : NIB == 2 ? 1 : 0);
}

// LDS bytes: dy, then x
// (plus 1 KB after x: the regular staging's sink for unused rounds, 16
// bytes per lane)
size_t wg32_lds(const Wg32Args &a)
{
    return 2ull * (a.x_off + static_cast<size_t>(a.CI) * a.xc) + 1024;
}

// tiling of the pass over output channels co0 .. co0 + CO - 1 for a given
// rows-per-tile; false if it does not fit
bool wg32_args(const ConvShape &sh, int co0, int CO, int TR, Wg32Args &a)
{
    a.N = sh.N;
    a.H = sh.H;
    a.W = sh.W;
    a.CI = sh.Ci;
    a.CO = CO;
    a.co0 = co0;
    a.COT = sh.Co;
    a.WS = cdiv((sh.W + 1) / 2, 8) * 8;
    a.XS = a.WS + 16;
    a.TR = TR;
    if ((a.TR * (a.WS / 8)) % 2 != 0)
        return false; // K-steps pair runs of one parity
    a.ntr = cdiv(sh.H, a.TR);
    a.ptiles = sh.N * a.ntr;
    // pitches: odd multiples of 16 bytes (32-row fragment reads)
    a.dyc = a.TR * 2 * a.WS + 8;
    if ((a.dyc / 8) % 2 == 0)
        a.dyc += 8;
    a.xc = (a.TR + 2 * sh.k) * 2 * a.XS + 8;
    if ((a.xc / 8) % 2 == 0)
        a.xc += 8;
    a.x_off = CO * a.dyc;
    if (wg32_lds(a) > kLdsMax)
        return false;
    const int CW = (sh.W % 8 == 0) ? 8 : 4;
    a.cpr = sh.W / CW;
    a.items_x = sh.Ci * (a.TR + 2 * sh.k) * a.cpr;
    a.items_dy = CO * a.TR * a.cpr;
    a.fcpr = make_fastdiv(static_cast<uint32_t>(a.cpr));
    a.fxr = make_fastdiv(static_cast<uint32_t>(a.TR + 2 * sh.k));
    a.ftr = make_fastdiv(static_cast<uint32_t>(a.TR));
    // regular staging: 16-byte chunks, a power-of-two chunk count per row
    // dividing the staging threads, x and dy each G = 2 or 4 rounds of
    // channels per row, offsets within 31 bits
    a.rg = a.rpu = a.lcpr = 0;
    if (CW == 8 && a.cpr <= kP && (a.cpr & (a.cpr - 1)) == 0) {
        const int rpu = kP / a.cpr;
        const int g = sh.Ci / rpu;
        if (sh.Ci == CO && sh.Ci % rpu == 0 && (g == 2 || g == 4) &&
            static_cast<long>(sh.Ci) * sh.H * sh.W < (1L << 31)) {
            a.rg = g;
            a.rpu = rpu;
            while ((1 << a.lcpr) < a.cpr)
                ++a.lcpr;
        }
    }
    return true;
}

int wg32_U(const Wg32Args &a) { return cdiv(a.items_x + a.items_dy, kP); }

bool wg32_plan(const ConvShape &sh, int co0, int CO, Wg32Args &a)
{
    const int NIB = sh.Ci / 32, NCB = CO / 32;
    const int C = NIB * NCB;
    if (NCB > max_ncb(sh.k, NIB))
        return false;
    // Tile height (at most 512 pixels a tile) that fits LDS and the staging
    // registers and stages the fewest rows per image: x rows with their
    // halo plus dy rows, over all tiles of the image (rows past the image
    // are computed but not real, so a ragged last tile costs a whole one);
    // ties go to the taller tile.
    int best = 0;
    long best_rows = 0;
    for (int TR = std::min(sh.H, std::max(1, 512 / sh.W)); TR >= 1; --TR) {
        if (!wg32_args(sh, co0, CO, TR, a) || wg32_U(a) > kMaxItems)
            continue;
        const long rows = static_cast<long>(a.ntr) *
                          (static_cast<long>(TR + 2 * sh.k) * sh.Ci + static_cast<long>(TR) * CO);
        if (best == 0 || rows < best_rows) {
            best = TR;
            best_rows = rows;
        }
    }
    if (best == 0 || !wg32_args(sh, co0, CO, best, a))
        return false;
    const int blocks = std::max(1, std::min(device_cus(), a.ptiles));
    a.per_block = cdiv(a.ptiles, blocks);
    a.nparts = cdiv(a.ptiles, a.per_block);
    a.nchunk = sh.T * C * 16 + cdiv(CO, kRegChunk);
    return true;
}

// Calls f(co0, CO, args) for every pass; false if some pass has no plan.
template <typename F> bool wg32_passes(const ConvShape &sh, F &&f)
{
    if (sh.s != 1 || (sh.k != 1 && sh.k != 2) || sh.Ci % 32 != 0 || sh.Co % 32 != 0 ||
        sh.W % 4 != 0)
        return false;
    const int nib = sh.Ci / 32;
    if (nib != 1 && nib != 2 && nib != 4)
        return false;
    for (int co0 = 0; co0 < sh.Co;) {
        // two 32-channel co blocks per pass where a tile fits, else one
        Wg32Args a{};
        int nb = std::min(max_ncb(sh.k, nib), (sh.Co - co0) / 32);
        while (nb > 0 && !wg32_plan(sh, co0, 32 * nb, a))
            --nb;
        if (nb == 0 || !f(a))
            return false;
        co0 += 32 * nb;
    }
    return true;
}

template <int K, int NIB, int NCB, int CW, int RG>
void launch_w32_cw(int U, const Wg32Args &a, size_t lds, hipStream_t st, const bf16raw *x,
                   const bf16raw *dy, float *part)
{
    if constexpr (NCB <= max_ncb(K, NIB)) {
#define HEX_W32(UV)                                                                          \
    HEX_LAUNCH((wgrad32_k<K, NIB, NCB, CW, UV, RG>), dim3(a.nparts), dim3(kT), lds, st, x,   \
               dy, part, a)
        static_assert(kMaxItems == 32, "staging variants: 8, 16, 24, 32 items");
        if (U <= 8)
            HEX_W32(8);
        else if (U <= 16)
            HEX_W32(16);
        else if (U <= 24)
            HEX_W32(24);
        else
            HEX_W32(32);
#undef HEX_W32
    }
}

template <int K, int NIB>
void launch_w32_nib(int NCB, bool cw8, int U, const Wg32Args &a, size_t lds, hipStream_t st,
                    const bf16raw *x, const bf16raw *dy, float *part)
{
    // regular staging needs C_in == this pass's C_out: one co block with one
    // ci block, two with two
    bool done = false;
    if constexpr (NIB <= 2) {
        if (NCB == NIB && a.rg == 2) {
            launch_w32_cw<K, NIB, NIB, 8, 2>(U, a, lds, st, x, dy, part);
            done = true;
        } else if (NCB == NIB && a.rg == 4) {
            launch_w32_cw<K, NIB, NIB, 8, 4>(U, a, lds, st, x, dy, part);
            done = true;
        }
    }
    if (done)
        return;
    if (NCB == 1) {
        if (cw8) launch_w32_cw<K, NIB, 1, 8, 0>(U, a, lds, st, x, dy, part);
        else launch_w32_cw<K, NIB, 1, 4, 0>(U, a, lds, st, x, dy, part);
    } else {
        if (cw8) launch_w32_cw<K, NIB, 2, 8, 0>(U, a, lds, st, x, dy, part);
        else launch_w32_cw<K, NIB, 2, 4, 0>(U, a, lds, st, x, dy, part);
    }
}

template <int K>
void launch_w32(int NIB, int NCB, bool cw8, int U, const Wg32Args &a, size_t lds,
                hipStream_t st, const bf16raw *x, const bf16raw *dy, float *part)
{
    if (NIB == 1)
        launch_w32_nib<K, 1>(NCB, cw8, U, a, lds, st, x, dy, part);
    else if (NIB == 2)
        launch_w32_nib<K, 2>(NCB, cw8, U, a, lds, st, x, dy, part);
    else
        launch_w32_nib<K, 4>(NCB, cw8, U, a, lds, st, x, dy, part);
}

} // namespace

int bf16_wgrad32_passes(const ConvShape &sh)
{
    int n = 0;
    if (!wg32_passes(sh, [&](const Wg32Args &) {
            ++n;
            return true;
        }))
        return 0;
    return n;
}

// One partial buffer serves every pass: the passes run in stream order.
size_t bf16_wgrad32_workspace(const ConvShape &sh)
{
    size_t need = 0;
    if (!wg32_passes(sh, [&](const Wg32Args &a) {
            need = std::max(need, sizeof(float) * static_cast<size_t>(a.nchunk) * kRegChunk *
                                      a.nparts);
            return true;
        }))
        return 0;
    return need;
}

hipError_t bf16_wgrad32(const void *x, const void *dy, float *dw, float *db, void *ws,
                        const ConvShape &sh, hipStream_t st)
{
    const bf16raw *xp = static_cast<const bf16raw *>(x);
    const bf16raw *dp = static_cast<const bf16raw *>(dy);
    float *part = static_cast<float *>(ws);
    hipError_t err = hipSuccess;
    const bool ok = wg32_passes(sh, [&](const Wg32Args &a) {
        const int NIB = sh.Ci / 32, NCB = a.CO / 32;
        const int C = NIB * NCB;
        const int U = wg32_U(a);
        const bool cw8 = sh.W % 8 == 0;
        const size_t lds = wg32_lds(a);
        if (sh.k == 1)
            launch_w32<1>(NIB, NCB, cw8, U, a, lds, st, xp, dp, part);
        else
            launch_w32<2>(NIB, NCB, cw8, U, a, lds, st, xp, dp, part);
        err = hipGetLastError();
        if (err != hipSuccess)
            return false;
        const int npos = sh.T * C * 16 * kRegChunk + a.CO;
        HEX_LAUNCH(wgrad32_reduce_k, dim3(cdiv(npos, kRegChunk)), dim3(kRegChunk * kRedSlices), 0, st, part,
                           a.nparts, npos, sh.Ci, a.CO, a.co0, sh.T, dw, db);
        err = hipGetLastError();
        return err == hipSuccess;
    });
    if (!ok && err == hipSuccess)
        return hipErrorInvalidValue;
    return err;
}

} // namespace hexk
