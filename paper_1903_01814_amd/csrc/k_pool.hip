// k_pool.hip -- hexagonal max / mean pooling, forward and backward, for
// kernel sizes k <= 3 and strides 1 to 4 (Sec. 2.4: the pool window is the
// size-k hexagon, padded like the convolution; stride as in Sec. 2.3).
//
// Forward: persistent blocks walk groups of NP planes, loading the next
// group into registers while the current one is reduced and stored.  A
// group's NP whole input planes are staged into LDS with a zero border
// (k rows above and below, a 16-byte pad left and right of every row), so a
// tap never needs a bounds check and padded taps read 0 (they take part in
// the max and the mean).  Each thread then reduces the T taps of one output
// from LDS: the strict "v > best" scan in canonical tap order keeps the
// first maximal tap, whose index is the uint8 argmax.  With an even stride
// every centre column is even, so the tap offsets are compile-time.
//
// Backward: scatter in tap phases.  dx of NP planes is accumulated in fp32
// in LDS; in phase t every output whose argmax is t (mean pooling: every
// output) adds its dy to the input pixel under tap t.  Two outputs with the
// same tap never reach the same pixel, so a phase needs no atomics, and the
// phases run in tap order -- each pixel receives its contributions in the
// same order as a gather over taps would add them, so the result is
// deterministic and independent of the thread layout.  Contributions through
// taps outside the input are dropped.  Mean pooling divides the sum by T;
// the ReLU mask [relu_in > 0] is applied last.
#include <algorithm>

#include "hexdev.h"
#include "kernels.h"
#include "shear.h"

namespace hexk {
namespace {

using namespace hexgeom;

constexpr int kPoolThreads = 256;

struct PoolArgs {
    int nplanes, H, W, Ho, Wo;
    int NP;      // planes per block
    int pitch;   // LDS row pitch (elements) of a staged input plane
    int LR;      // LDS rows of a staged input plane (H + 2k)
    FastDiv fwo; // division by Wo
    FastDiv fho; // division by Ho * Wo
    FastDiv fho_rows; // division by Ho
    FastDiv fw;  // division by W
    FastDiv fh;  // division by H
    FastDiv fcr; // division by the 16-byte chunks of an input row
};

// centre of output (i, j) (stride S)
template <int S> __device__ __forceinline__ int centre_r(int i, int j)
{
    return S * i + (j & 1) * (S / 2);
}

// Interior rows of a group of NP planes in 16-byte chunks, U per thread; the
// planes are contiguous in x, so chunk it is x[group start + VEC * it].
// Every load is issued (the index clamped) so that their count is fixed.
// (a native vector type: copies of the uint4 struct become memcpys that keep
// the array in scratch memory)
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
template <typename TT, int K, int U> struct PoolStage {
    static constexpr int VEC = 16 / sizeof(TT);
    u32x4 v[U];

    __device__ __forceinline__ void load(const TT *__restrict__ x, const PoolArgs &a, int g)
    {
        const int np = min(a.NP, a.nplanes - g * a.NP);
        const int items = np * a.H * (a.W / VEC);
        const TT *src = x + static_cast<size_t>(g) * a.NP * a.H * a.W;
#pragma clang loop unroll(full)
        for (int u = 0; u < U; ++u) {
            const int it = threadIdx.x + u * kPoolThreads;
            v[u] = *reinterpret_cast<const u32x4 *>(src + static_cast<size_t>(min(it, items - 1)) * VEC);
        }
    }

    // into LDS rows K .. K + H - 1 of each plane, after the 16-byte left pad
    __device__ __forceinline__ void commit(TT *__restrict__ lds, const PoolArgs &a, int g) const
    {
        const int np = min(a.NP, a.nplanes - g * a.NP);
        const int cpr = a.W / VEC;
        const int items = np * a.H * cpr;
        const int plane_l = a.LR * a.pitch;
#pragma clang loop unroll(full)
        for (int u = 0; u < U; ++u) {
            const int it = threadIdx.x + u * kPoolThreads;
            if (it < items) {
                const int rowi = static_cast<int>(fdiv(static_cast<uint32_t>(it), a.fcr));
                const int ch = it - rowi * cpr;
                const int pl = static_cast<int>(fdiv(static_cast<uint32_t>(rowi), a.fh));
                const int r = rowi - pl * a.H;
                *reinterpret_cast<u32x4 *>(lds + pl * plane_l + (r + K) * a.pitch + VEC + ch * VEC) = v[u];
            }
        }
    }
};

// ARG: write the argmax tap (max pooling).  U: 16-byte chunks per thread of
// a group of NP planes.  Persistent blocks walk the plane groups g =
// blockIdx.x, + gridDim.x, ...; the next group's chunks are loaded into
// registers right after the current group is written to LDS, so every block
// has a load in flight while it reduces and stores.
template <typename TT, int MODE, int K, int S, bool ARG, int U>
__global__ __launch_bounds__(kPoolThreads) void pool_fwd_k(const TT *__restrict__ x,
                                                           TT *__restrict__ y,
                                                           uint8_t *__restrict__ am, PoolArgs a)
{
    constexpr int T = num_taps(K);
    constexpr int VEC = 16 / sizeof(TT); // elements per 16 bytes = left pad
    extern __shared__ __align__(16) unsigned char smem[];
    TT *lds = reinterpret_cast<TT *>(smem);
    const int H = a.H, W = a.W;
    const int plane_l = a.LR * a.pitch;
    const int ngroups = (a.nplanes + a.NP - 1) / a.NP;

    // zero border, once: whole rows above / below, one 16-byte chunk left
    // and right; the group's rows never overwrite it
    {
        const int vrow = a.pitch / VEC; // 16-byte chunks per LDS row
        const int per_plane = 2 * K * vrow + 2 * H;
        for (int e = threadIdx.x; e < a.NP * per_plane; e += kPoolThreads) {
            const int pl = e / per_plane, q = e - pl * per_plane;
            int off;
            if (q < 2 * K * vrow) {
                const int rr = q / vrow, v = q - rr * vrow;
                const int row = rr < K ? rr : H + rr; // rows 0..K-1 and H+K..H+2K-1
                off = row * a.pitch + v * VEC;
            } else {
                const int q2 = q - 2 * K * vrow;
                const int row = K + (q2 >> 1);
                off = row * a.pitch + ((q2 & 1) ? VEC + W : 0);
            }
            *reinterpret_cast<uint4 *>(lds + pl * plane_l + off) = make_uint4(0, 0, 0, 0);
        }
    }

    PoolStage<TT, K, U> stg;

    // thread -> output column j (fixed) and every rpp-th output row of the
    // group's planes (rows of consecutive planes follow each other)
    const int Wo = a.Wo, Ho = a.Ho;
    const int HWo = Ho * Wo;
    const int rpp = kPoolThreads / Wo; // output rows per pass (Wo <= 256)
    const int j = threadIdx.x % Wo;
    const int row0 = threadIdx.x / Wo;
    const int cc = S * j;
    const int par = (S % 2 == 0) ? 0 : (cc & 1);
    const int halfs = (j & 1) * (S / 2);
    constexpr TapTable<K> tt;

    // k = 1, stride 2, bfloat16, even W_out: a thread takes the outputs j
    // and j + 1 (j even) of a row.  Their centres are (2i, 2j) and
    // (2i + 1, 2j + 2), and their 14 taps lie in input columns 2j - 2 ..
    // 2j + 3 and rows 2i - 1 .. 2i + 2: eight aligned 32-bit LDS reads (two
    // columns each) instead of fourteen 16-bit ones, and one 32-bit store.
    constexpr bool PAIRS = K == 1 && S == 2 && sizeof(TT) == 2;
    const bool pairs = PAIRS && Wo % 2 == 0;
    auto pool_pairs = [&](int g) __attribute__((always_inline)) {
        const int npair = Wo / 2;
        const int rpp2 = kPoolThreads / npair; // Wo <= 256: at least one row per pass
        const int jp = threadIdx.x % npair, prow0 = threadIdx.x / npair;
        if (prow0 >= rpp2)
            return;
        const int j2 = 2 * jp;
        const int p0 = g * a.NP;
        const int np = min(a.NP, a.nplanes - p0);
        TT *yb = y + static_cast<size_t>(p0) * HWo;
        uint8_t *ab = am != nullptr ? am + static_cast<size_t>(p0) * HWo : nullptr;
        int pl = static_cast<int>(fdiv(static_cast<uint32_t>(prow0), a.fho_rows));
        int i = prow0 - pl * Ho;
        for (int row = prow0; row < np * Ho; row += rpp2) {
            // word (two columns) c2 of window row rr: rows 2i - 1 + rr,
            // columns 2j - 2 + 2 c2 and 2j - 1 + 2 c2
            const uint32_t *wrow = reinterpret_cast<const uint32_t *>(
                lds + pl * plane_l + (2 * i - 1 + K) * a.pitch + VEC + j2 * 2 - 2);
            const int wp = a.pitch / 2; // words per LDS row
            float v[4][6];
            auto take = [&](int rr, int c2) {
                const uint32_t q = wrow[rr * wp + c2];
                v[rr][2 * c2] = __uint_as_float(q << 16);
                v[rr][2 * c2 + 1] = __uint_as_float(q & 0xffff0000u);
            };
            take(0, 0); take(1, 0);
            take(0, 1); take(1, 1); take(2, 1);
            take(1, 2); take(2, 2); take(3, 2);
            float res[2];
            int arg[2] = {0, 0};
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                // centre of output j + h: window row 1 + h, column 2 + 2h
                float best = 0.f, sum = 0.f;
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    const int dr = tap_drow(tt.dq[t], tt.ds[t], 0);
                    const float val = v[1 + h + dr][2 + 2 * h + tt.dq[t]];
                    if (MODE == 0) {
                        if (t == 0 || val > best) {
                            best = val;
                            if (ARG)
                                arg[h] = t;
                        }
                    } else {
                        sum += val;
                    }
                }
                res[h] = MODE == 0 ? best : sum / static_cast<float>(T);
            }
            const int o = row * Wo + j2; // plane-major, even
            *reinterpret_cast<uint32_t *>(yb + o) =
                static_cast<uint32_t>(from_f<TT>(res[0])) |
                (static_cast<uint32_t>(from_f<TT>(res[1])) << 16);
            if (ARG)
                *reinterpret_cast<uint16_t *>(ab + o) =
                    static_cast<uint16_t>(arg[0] | (arg[1] << 8));
            i += rpp2;
            while (i >= Ho) {
                i -= Ho;
                ++pl;
            }
        }
    };

    if (blockIdx.x < ngroups)
        stg.load(x, a, blockIdx.x);
    for (int g = blockIdx.x; g < ngroups; g += gridDim.x) {
        __syncthreads(); // the previous group's LDS reads are done (and the border)
        stg.commit(lds, a, g);
        __syncthreads();
        if (g + static_cast<int>(gridDim.x) < ngroups)
            stg.load(x, a, g + gridDim.x);
        if constexpr (PAIRS) {
            if (pairs) {
                pool_pairs(g);
                continue;
            }
        }
        if (row0 < rpp) { // spare threads: only the staging and the barriers
            const int p0 = g * a.NP;
            const int np = min(a.NP, a.nplanes - p0);
            TT *yb = y + static_cast<size_t>(p0) * HWo;
            uint8_t *ab = am != nullptr ? am + static_cast<size_t>(p0) * HWo : nullptr;
            int pl = static_cast<int>(fdiv(static_cast<uint32_t>(row0), a.fho_rows));
            int i = row0 - pl * Ho;
            for (int row = row0; row < np * Ho; row += rpp) {
                const int rc = S * i + halfs;
                const TT *cen = lds + pl * plane_l + (rc + K) * a.pitch + VEC + cc;
                float best = 0.f, sum = 0.f;
                int arg = 0;
    #pragma unroll
                for (int t = 0; t < T; ++t) {
                    const int dr = par ? tap_drow(tt.dq[t], tt.ds[t], 1) : tap_drow(tt.dq[t], tt.ds[t], 0);
                    const float val = to_f(cen[dr * a.pitch + tt.dq[t]]);
                    if (MODE == 0) {
                        if (t == 0 || val > best) {
                            best = val;
                            if (ARG)
                                arg = t;
                        }
                    } else {
                        sum += val;
                    }
                }
                const int o = row * Wo + j; // plane-major: pl * HWo + i * Wo + j
                if (MODE == 0) {
                    yb[o] = from_f<TT>(best);
                    if (ARG)
                        ab[o] = static_cast<uint8_t>(arg);
                } else {
                    yb[o] = from_f<TT>(sum / static_cast<float>(T));
                }
                i += rpp;
                while (i >= Ho) {
                    i -= Ho;
                    ++pl;
                }
            }
        }
    }
}

// OPT: outputs per thread held in registers across the tap phases.  Every
// global read of a block is issued before its first wait -- the outputs' dy
// and argmax (indices clamped, so the count is fixed) and the first
// kPoolBwdPrefetch 16-byte relu_y chunks of each thread -- so a block makes
// one round trip to memory instead of one per output and per chunk.
constexpr int kPoolBwdPrefetch = 4;

// relu_y and dx are not restrict-qualified: without a mask the relu_y reads
// go to dx (same shape; the values are not used), so that their count is
// fixed and the wait before the tap phases covers dy and the argmax only.
template <typename TT, int MODE, int K, int S, int OPT>
__global__ __launch_bounds__(kPoolThreads) void pool_bwd_k(const TT *__restrict__ dy,
                                                           const uint8_t *__restrict__ am,
                                                           const TT *relu_y, TT *dx, PoolArgs a)
{
    constexpr int T = num_taps(K);
    constexpr int VEC = 16 / sizeof(TT); // W is a multiple of VEC
    constexpr int RUP = kPoolBwdPrefetch;
    extern __shared__ __align__(16) float acc[]; // [np][H][W]
    const int p0 = blockIdx.x * a.NP;
    const int np = min(a.NP, a.nplanes - p0);
    const int H = a.H, W = a.W;
    const int HW = H * W;
    const int HWo = a.Ho * a.Wo;
    const int nout = np * HWo;
    const int nchunk = np * HW / VEC;
    const size_t go0 = static_cast<size_t>(p0) * HWo;
    const size_t g0 = static_cast<size_t>(p0) * HW;

    TT gv[OPT];
    uint8_t tv[OPT];
#pragma unroll
    for (int u = 0; u < OPT; ++u) {
        const int e = min(static_cast<int>(threadIdx.x) + u * kPoolThreads, nout - 1);
        gv[u] = dy[go0 + e];
        tv[u] = (MODE == 0) ? am[go0 + e] : 0;
    }
    const bool relu = relu_y != nullptr;
    const TT *rsrc = relu ? relu_y : dx;
    u32x4 rv[RUP];
#pragma unroll
    for (int u = 0; u < RUP; ++u) {
        const int c = min(static_cast<int>(threadIdx.x) + u * kPoolThreads, nchunk - 1);
        rv[u] = *reinterpret_cast<const u32x4 *>(rsrc + g0 + static_cast<size_t>(c) * VEC);
    }

    for (int e = threadIdx.x * 4; e < np * HW; e += kPoolThreads * 4)
        *reinterpret_cast<float4 *>(acc + e) = make_float4(0.f, 0.f, 0.f, 0.f);

    // this thread's outputs: centre, plane offset, dy and (max pooling) the
    // one pixel its gradient goes to -- under its argmax tap, -1 where that
    // tap lies outside the input
    constexpr TapTable<K> tt;
    float g[OPT];
    int tap[OPT], base[OPT], rc_[OPT], cc_[OPT], tgt[OPT];
#pragma unroll
    for (int u = 0; u < OPT; ++u) {
        const int e = threadIdx.x + u * kPoolThreads;
        const bool live = e < nout;
        const int ee = live ? e : 0;
        const int pl = static_cast<int>(fdiv(static_cast<uint32_t>(ee), a.fho));
        const int o = ee - pl * HWo;
        const int i = static_cast<int>(fdiv(static_cast<uint32_t>(o), a.fwo));
        const int j = o - i * a.Wo;
        rc_[u] = centre_r<S>(i, j);
        cc_[u] = S * j;
        base[u] = pl * HW;
        g[u] = to_f(gv[u]);
        tap[u] = !live ? -1 : (MODE == 0) ? static_cast<int>(tv[u]) : T; // T: every tap
        tgt[u] = -1;
        if (MODE == 0) {
            const int par = (S % 2 == 0) ? 0 : (cc_[u] & 1);
            int dr = 0, dc = 0;
#pragma unroll
            for (int t = 0; t < T; ++t) {
                const bool hit = tap[u] == t;
                dr = hit ? (par ? tap_drow(tt.dq[t], tt.ds[t], 1) : tap_drow(tt.dq[t], tt.ds[t], 0)) : dr;
                dc = hit ? tt.dq[t] : dc;
            }
            const int r = rc_[u] + dr, c = cc_[u] + dc;
            const bool in = tap[u] >= 0 && tap[u] < T && r >= 0 && r < H && c >= 0 && c < W;
            tgt[u] = in ? base[u] + r * W + c : -1;
        }
    }
    __syncthreads();

#pragma unroll
    for (int t = 0; t < T; ++t) {
        float cur[OPT];
        int ad[OPT];
        bool on[OPT];
#pragma unroll
        for (int u = 0; u < OPT; ++u) {
            if (MODE == 0) {
                on[u] = tap[u] == t && tgt[u] >= 0;
                ad[u] = tgt[u];
            } else {
                const int par = (S % 2 == 0) ? 0 : (cc_[u] & 1);
                const int r = rc_[u] + (par ? tap_drow(tt.dq[t], tt.ds[t], 1) : tap_drow(tt.dq[t], tt.ds[t], 0));
                const int c = cc_[u] + tt.dq[t];
                on[u] = tap[u] == T && r >= 0 && r < H && c >= 0 && c < W;
                ad[u] = base[u] + r * W + c;
            }
            cur[u] = acc[on[u] ? ad[u] : 0];
        }
        // two outputs never reach one pixel in the same phase, so the reads
        // of a phase (all issued, unused ones from element 0) may all
        // precede its writes
#pragma unroll
        for (int u = 0; u < OPT; ++u)
            if (on[u])
                acc[ad[u]] = cur[u] + g[u];
        __syncthreads(); // phase t complete before phase t+1 touches the same pixels
    }

    // dx of the block's planes (contiguous in memory), VEC pixels per chunk
    auto emit = [&](int c, const u32x4 &rr) {
        const int e0 = c * VEC;
        const TT *rt = reinterpret_cast<const TT *>(&rr);
        TT ov[VEC];
#pragma unroll
        for (int q = 0; q < VEC; q += 4) {
            const float4 v4 = *reinterpret_cast<const float4 *>(acc + e0 + q);
            const float vv[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                float v = vv[h];
                if (MODE == 1)
                    v = v / static_cast<float>(T);
                if (relu && !(to_f(rt[q + h]) > 0.f))
                    v = 0.f;
                ov[q + h] = from_f<TT>(v);
            }
        }
        *reinterpret_cast<u32x4 *>(dx + g0 + e0) = *reinterpret_cast<const u32x4 *>(ov);
    };
#pragma unroll
    for (int u = 0; u < RUP; ++u) {
        const int c = threadIdx.x + u * kPoolThreads;
        if (c < nchunk)
            emit(c, rv[u]);
    }
    for (int c = threadIdx.x + RUP * kPoolThreads; c < nchunk; c += kPoolThreads) {
        u32x4 rr = {0u, 0u, 0u, 0u};
        if (relu)
            rr = *reinterpret_cast<const u32x4 *>(relu_y + g0 + static_cast<size_t>(c) * VEC);
        emit(c, rr);
    }
}

inline int cdiv(long a, long b) { return static_cast<int>((a + b - 1) / b); }

constexpr size_t kPoolLds = 48 * 1024;
constexpr size_t kLdsPerCu = 160 * 1024;
constexpr int kPoolMaxU = 12; // staged 16-byte chunks per thread at most (forward)

PoolArgs pool_args(const ConvShape &sh, int esz)
{
    PoolArgs a{};
    a.nplanes = sh.N * sh.Ci;
    a.H = sh.H;
    a.W = sh.W;
    a.Ho = sh.Ho;
    a.Wo = sh.Wo;
    const int vec = 16 / esz;
    a.pitch = sh.W + 2 * vec;
    a.LR = sh.H + 2 * sh.k;
    a.fwo = make_fastdiv(static_cast<uint32_t>(std::max(1, sh.Wo)));
    a.fho = make_fastdiv(static_cast<uint32_t>(std::max(1, sh.Ho * sh.Wo)));
    a.fho_rows = make_fastdiv(static_cast<uint32_t>(std::max(1, sh.Ho)));
    a.fw = make_fastdiv(static_cast<uint32_t>(sh.W));
    a.fh = make_fastdiv(static_cast<uint32_t>(sh.H));
    a.fcr = make_fastdiv(static_cast<uint32_t>(std::max(1, sh.W / vec)));
    return a;
}

size_t fwd_plane_bytes(const PoolArgs &a, int esz) { return static_cast<size_t>(a.LR) * a.pitch * esz; }

int bwd_opt(const PoolArgs &a, int np) { return cdiv(static_cast<long>(np) * a.Ho * a.Wo, kPoolThreads); }

} // namespace

bool pool_fast_ok(const ConvShape &sh, Dtype dt)
{
    const int esz = dt == F32 ? 4 : 2;
    // the 16-byte pad left and right of a staged row holds the k-column halo
    if (sh.k > 3 || sh.k > 16 / esz || sh.s < 1 || sh.s > 4 || sh.W % (16 / esz) != 0 ||
        sh.Ho == 0 || sh.Wo > kPoolThreads)
        return false;
    const PoolArgs a = pool_args(sh, esz);
    // one plane must fit; the backward holds up to 16 outputs per thread
    return fwd_plane_bytes(a, esz) <= kPoolLds &&
           sizeof(float) * static_cast<size_t>(sh.H) * sh.W <= kPoolLds &&
           bwd_opt(a, 1) <= 16;
}

hipError_t pool_fwd_fast(const void *x, void *y, uint8_t *am, const ConvShape &sh, int mode,
                         Dtype dt, hipStream_t st)
{
    const int esz = dt == F32 ? 4 : 2;
    PoolArgs a = pool_args(sh, esz);
    // planes per group: LDS budget and about 4 outputs per thread (measured
    // on the 40x40 -> 20x20 pools: 2 planes per group beat 1, 5 and 10);
    // chunks per thread within the instantiated staging depths
    const int by_lds = static_cast<int>(kPoolLds / fwd_plane_bytes(a, esz));
    const int by_work = std::max(1, (4 * kPoolThreads) / std::max(1, sh.Ho * sh.Wo));
    a.NP = std::max(1, std::min(by_lds, by_work));
    const int cpr = sh.W / (16 / esz);
    while (a.NP > 1 && a.NP * sh.H * cpr > kPoolMaxU * kPoolThreads)
        --a.NP;
    const int U = cdiv(static_cast<long>(a.NP) * sh.H * cpr, kPoolThreads);
    const size_t lds = fwd_plane_bytes(a, esz) * a.NP;
    // persistent blocks: as many as fit on a CU (threads and LDS), or one per group
    const int groups = cdiv(a.nplanes, a.NP);
    const int per_cu = std::max(1, std::min(8, static_cast<int>(kLdsPerCu / std::max<size_t>(lds, 1))));
    const int grid = std::max(1, std::min(groups, device_cus() * per_cu));
#define HEX_PF_U(TT, M, KV, SV, ARGV)                                                        \
    do {                                                                                     \
        if (U <= 1) HEX_LAUNCH((pool_fwd_k<TT, M, KV, SV, ARGV, 1>), dim3(grid),             \
                               dim3(kPoolThreads), lds, st, static_cast<const TT *>(x),      \
                               static_cast<TT *>(y), am, a);                                 \
        else if (U <= 2) HEX_LAUNCH((pool_fwd_k<TT, M, KV, SV, ARGV, 2>), dim3(grid),        \
                                    dim3(kPoolThreads), lds, st, static_cast<const TT *>(x), \
                                    static_cast<TT *>(y), am, a);                            \
        else if (U <= 4) HEX_LAUNCH((pool_fwd_k<TT, M, KV, SV, ARGV, 4>), dim3(grid),        \
                                    dim3(kPoolThreads), lds, st, static_cast<const TT *>(x), \
                                    static_cast<TT *>(y), am, a);                            \
        else HEX_LAUNCH((pool_fwd_k<TT, M, KV, SV, ARGV, kPoolMaxU>), dim3(grid),            \
                        dim3(kPoolThreads), lds, st, static_cast<const TT *>(x),             \
                        static_cast<TT *>(y), am, a);                                        \
    } while (0)
#define HEX_PF(TT, M, KV, SV)                                                                \
    do {                                                                                     \
        if (am != nullptr)                                                                   \
            HEX_PF_U(TT, M, KV, SV, true);                                                   \
        else                                                                                 \
            HEX_PF_U(TT, M, KV, SV, false);                                                  \
    } while (0)
#define HEX_PF_KS(TT, M)                                                                     \
    do {                                                                                     \
        if (sh.s == 1) {                                                                     \
            if (sh.k == 0) HEX_PF(TT, M, 0, 1);                                              \
            else if (sh.k == 1) HEX_PF(TT, M, 1, 1);                                         \
            else if (sh.k == 2) HEX_PF(TT, M, 2, 1);                                         \
            else HEX_PF(TT, M, 3, 1);                                                        \
        }                                                                                    \
        else if (sh.s == 2) {                                                                \
            if (sh.k == 0) HEX_PF(TT, M, 0, 2);                                              \
            else if (sh.k == 1) HEX_PF(TT, M, 1, 2);                                         \
            else if (sh.k == 2) HEX_PF(TT, M, 2, 2);                                         \
            else HEX_PF(TT, M, 3, 2);                                                        \
        }                                                                                    \
        else if (sh.s == 3) {                                                                \
            if (sh.k == 0) HEX_PF(TT, M, 0, 3);                                              \
            else if (sh.k == 1) HEX_PF(TT, M, 1, 3);                                         \
            else if (sh.k == 2) HEX_PF(TT, M, 2, 3);                                         \
            else HEX_PF(TT, M, 3, 3);                                                        \
        }                                                                                    \
        else {                                                                               \
            if (sh.k == 0) HEX_PF(TT, M, 0, 4);                                              \
            else if (sh.k == 1) HEX_PF(TT, M, 1, 4);                                         \
            else if (sh.k == 2) HEX_PF(TT, M, 2, 4);                                         \
            else HEX_PF(TT, M, 3, 4);                                                        \
        }                                                                                    \
    } while (0)
    if (dt == F32) {
        if (mode == 0) HEX_PF_KS(float, 0); else HEX_PF_KS(float, 1);
    } else {
        if (mode == 0) HEX_PF_KS(bf16raw, 0); else HEX_PF_KS(bf16raw, 1);
    }
#undef HEX_PF_KS
#undef HEX_PF
#undef HEX_PF_U
    return hipGetLastError();
}

hipError_t pool_bwd_fast(const void *dy, const uint8_t *am, const void *relu_y, void *dx,
                         const ConvShape &sh, int mode, Dtype dt, hipStream_t st)
{
    const int esz = dt == F32 ? 4 : 2;
    PoolArgs a = pool_args(sh, esz);
    const size_t plane = sizeof(float) * static_cast<size_t>(sh.H) * sh.W;
    const int by_lds = static_cast<int>(kPoolLds / plane);
    // up to 4 outputs per thread (measured: 8 and 16 were slower at the
    // 48x48 and 24x24 stride-2 pools)
    const int by_opt = std::max(1, (4 * kPoolThreads) / std::max(1, sh.Ho * sh.Wo));
    a.NP = std::max(1, std::min(by_lds, by_opt));
    const int opt = bwd_opt(a, a.NP);
    const int grid = cdiv(a.nplanes, a.NP);
    const size_t lds = plane * a.NP;
#define HEX_PB(TT, M, KV, SV, OV)                                                            \
    HEX_LAUNCH((pool_bwd_k<TT, M, KV, SV, OV>), dim3(grid), dim3(kPoolThreads), lds,         \
                       st, static_cast<const TT *>(dy), am, static_cast<const TT *>(relu_y), \
                       static_cast<TT *>(dx), a)
#define HEX_PB_O(TT, M, KV, SV)                                                              \
    do {                                                                                     \
        if (opt <= 1) HEX_PB(TT, M, KV, SV, 1);                                              \
        else if (opt <= 2) HEX_PB(TT, M, KV, SV, 2);                                         \
        else if (opt <= 4) HEX_PB(TT, M, KV, SV, 4);                                         \
        else if (opt <= 8) HEX_PB(TT, M, KV, SV, 8);                                         \
        else HEX_PB(TT, M, KV, SV, 16);                                                      \
    } while (0)
#define HEX_PB_KS(TT, M)                                                                     \
    do {                                                                                     \
        if (sh.s == 1) {                                                                     \
            if (sh.k == 0) HEX_PB_O(TT, M, 0, 1);                                            \
            else if (sh.k == 1) HEX_PB_O(TT, M, 1, 1);                                       \
            else if (sh.k == 2) HEX_PB_O(TT, M, 2, 1);                                       \
            else HEX_PB_O(TT, M, 3, 1);                                                      \
        }                                                                                    \
        else if (sh.s == 2) {                                                                \
            if (sh.k == 0) HEX_PB_O(TT, M, 0, 2);                                            \
            else if (sh.k == 1) HEX_PB_O(TT, M, 1, 2);                                       \
            else if (sh.k == 2) HEX_PB_O(TT, M, 2, 2);                                       \
            else HEX_PB_O(TT, M, 3, 2);                                                      \
        }                                                                                    \
        else if (sh.s == 3) {                                                                \
            if (sh.k == 0) HEX_PB_O(TT, M, 0, 3);                                            \
            else if (sh.k == 1) HEX_PB_O(TT, M, 1, 3);                                       \
            else if (sh.k == 2) HEX_PB_O(TT, M, 2, 3);                                       \
            else HEX_PB_O(TT, M, 3, 3);                                                      \
        }                                                                                    \
        else {                                                                               \
            if (sh.k == 0) HEX_PB_O(TT, M, 0, 4);                                            \
            else if (sh.k == 1) HEX_PB_O(TT, M, 1, 4);                                       \
            else if (sh.k == 2) HEX_PB_O(TT, M, 2, 4);                                       \
            else HEX_PB_O(TT, M, 3, 4);                                                      \
        }                                                                                    \
    } while (0)
    if (dt == F32) {
        if (mode == 0) HEX_PB_KS(float, 0); else HEX_PB_KS(float, 1);
    } else {
        if (mode == 0) HEX_PB_KS(bf16raw, 0); else HEX_PB_KS(bf16raw, 1);
    }
#undef HEX_PB_KS
#undef HEX_PB_O
#undef HEX_PB
    return hipGetLastError();
}

} // namespace hexk
