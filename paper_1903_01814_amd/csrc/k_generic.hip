// k_generic.hip -- kernels that handle every kernel size, stride, channel
// count and dtype.  The shape-specialised kernels in the other files take
// over for the common cases; these remain the path for everything else.
//
// Conv forward: one output pixel per thread, a 2-D output tile per block,
// the input region of the tile (with its k-wide halo, zero outside the
// tensor) and the block's weights staged in LDS as float, a few input
// channels per pair of barriers.
// Conv backward-data: gather form -- each input pixel looks up, per tap, the
// output whose window reads it (a lattice test for strides > 1); the weights
// of a few output channels at a time are staged in LDS as float.
// Weight gradient: per-chunk partial sums in a fixed tree order, then the
// fixed-order reduction over chunks of k_reduce.hip (deterministic).
// Pool forward / backward: one output (input) element per thread.
#include <algorithm>

#include "generic_plan.h"
#include "hexdev.h"
#include "kernels.h"
#include "stage.h"

namespace hexk {
namespace {

using namespace hexgeom;

using plan::kThreads;
using plan::region_cols;
using plan::region_rows;
// Channels per block (plan::chan_block): output channels (forward) or input
// channels (data gradient), 8, 32 or 64.
constexpr int kTapGroup = 8;  // taps accumulated per pass (weight gradient)
constexpr int kWgCoBlock = 8; // output channels per block (weight gradient, >= 32 channels)

// Depth: every kernel here also serves the three-dimensional operations
// (x[N][C][D][H][W], a window of 2kz+1 planes around the centre plane
// sz*l, planes outside the tensor reading zero); a 2-D call is the case
// D = D_out = 1, kz = 0.  An input channel ci and a plane offset dz form one
// "pair" p = ci*Z + dz_index (Z = 2kz+1), so the weights w[C_out][C_in][Z][T]
// are w[C_out][pairs][T] and each pair is staged like one 2-D input channel.

// Plane of pair p for output plane l of image n (nullptr: a padding plane).
template <typename T>
__device__ __forceinline__ const T *pair_plane(const T *x, const ConvShape &sh, int n, int p, int l)
{
    const int ci = p / sh.Z, dzi = p - ci * sh.Z;
    const int z = sh.sz * l + dzi - sh.kz;
    if (z < 0 || z >= sh.D)
        return nullptr;
    return x + ((static_cast<size_t>(n) * sh.Ci + ci) * sh.D + z) * (static_cast<size_t>(sh.H) * sh.W);
}

// G pairs per stage: their regions and weights are staged between one pair
// of barriers, and each tap's CB weights are read as broadcast 16-byte LDS
// vectors.  blockIdx.x = output plane l * tiles + tile.
template <typename T, int CB>
__global__ __launch_bounds__(kThreads) void conv_fwd_generic_k(
    const T *__restrict__ x, const T *__restrict__ w, const T *__restrict__ b,
    T *__restrict__ y, ConvShape sh, int relu, int TI, int TJ, int tiles_j, int G)
{
    extern __shared__ __align__(16) float region[];
    __shared__ TapLds tl;
    fill_taps(tl, sh.k);

    const int tiles = gridDim.x / sh.Do;
    const int l = blockIdx.x / tiles;
    const int tile = blockIdx.x - l * tiles;
    const int n = blockIdx.y;
    const int co0 = blockIdx.z * CB;
    const int ti0 = (tile / tiles_j) * TI;
    const int tj0 = (tile % tiles_j) * TJ;
    const int r_lo = sh.s * ti0 - sh.k;
    const int c_lo = sh.s * tj0 - sh.k;
    const int RH = region_rows(TI, sh.k, sh.s);
    const int RW = region_cols(TJ, sh.k, sh.s);
    const int RF = plan::region_floats(TI, TJ, sh.k, sh.s);
    float *wl = region + static_cast<size_t>(G) * RF; // [G][T][CB]

    const int li = threadIdx.x / TJ, lj = threadIdx.x % TJ;
    const int i = ti0 + li, j = tj0 + lj;
    const bool active = threadIdx.x < TI * TJ && i < sh.Ho && j < sh.Wo;
    int rr = 0, cc = 0, par = 0;
    if (active) {
        rr = centre_row(i, j, sh.s) - r_lo;
        cc = centre_col(j, sh.s) - c_lo;
        par = centre_col(j, sh.s) & 1;
    }

    float acc[CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
        acc[cb] = (b != nullptr && co0 + cb < sh.Co) ? to_f(b[co0 + cb]) : 0.f;

    const int P = sh.Ci * sh.Z;
    const int TCB = sh.T * CB;
    for (int p0 = 0; p0 < P; p0 += G) {
        const int ng = min(G, P - p0);
        __syncthreads();
        for (int g = 0; g < ng; ++g) {
            const T *plane = pair_plane(x, sh, n, p0 + g, l);
            // a padding plane stages zeros (no row is inside)
            stage_window<8>(region + static_cast<size_t>(g) * RF, plane != nullptr ? plane : x,
                            plane != nullptr ? sh.H : 0, sh.W, r_lo, c_lo, RH, RW);
        }
        // weights of output channels co0 .. co0 + CB - 1 (clamped to the
        // last one; those accumulators are never stored)
        for (int e = threadIdx.x; e < ng * TCB; e += kThreads) {
            const int cb = e % CB, rest = e / CB;
            const int g = rest / sh.T, t = rest - g * sh.T;
            const int co = min(co0 + cb, sh.Co - 1);
            wl[e] = to_f(w[(static_cast<size_t>(co) * P + p0 + g) * sh.T + t]);
        }
        __syncthreads();
        if (active) {
            for (int g = 0; g < ng; ++g) {
                const float *rg = region + static_cast<size_t>(g) * RF;
                const float *wg = wl + g * TCB;
                for (int t = 0; t < sh.T; ++t) {
                    const float v = rg[(rr + tl.drow[par][t]) * RW + cc + tl.dq[t]];
                    const float4 *w4 = reinterpret_cast<const float4 *>(wg + t * CB);
#pragma unroll
                    for (int q = 0; q < CB / 4; ++q) {
                        const float4 ww = w4[q];
                        acc[4 * q] += ww.x * v;
                        acc[4 * q + 1] += ww.y * v;
                        acc[4 * q + 2] += ww.z * v;
                        acc[4 * q + 3] += ww.w * v;
                    }
                }
            }
        }
    }
    if (!active)
        return;
    const size_t HWo = static_cast<size_t>(sh.Ho) * sh.Wo;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
        const int co = co0 + cb;
        if (co >= sh.Co)
            break;
        float v = acc[cb];
        if (relu)
            v = fmaxf(v, 0.f);
        y[((static_cast<size_t>(n) * sh.Co + co) * sh.Do + l) * HWo + static_cast<size_t>(i) * sh.Wo + j] =
            from_f<T>(v);
    }
}

// CC output channels per stage: their weights (one plane offset) for the
// block's CB input channels are staged in LDS as float [CC][T][CB] between
// one pair of barriers and read as broadcast 16-byte vectors.
// blockIdx.x = input plane z * pixel blocks + pixel block.
template <typename T, int CB>
__global__ __launch_bounds__(kThreads) void conv_bwd_data_generic_k(
    const T *__restrict__ dy, const T *__restrict__ w, T *__restrict__ dx, ConvShape sh, int CC)
{
    extern __shared__ __align__(16) float wl[];
    __shared__ TapLds tl;
    fill_taps(tl, sh.k);

    const int pblocks = gridDim.x / sh.D;
    const int z = blockIdx.x / pblocks;
    const int p = (blockIdx.x - z * pblocks) * kThreads + threadIdx.x;
    const int n = blockIdx.y;
    const int ci0 = blockIdx.z * CB;
    const bool active = p < sh.H * sh.W;
    const int r = active ? p / sh.W : 0, c = active ? p % sh.W : 0;
    const size_t HWo = static_cast<size_t>(sh.Ho) * sh.Wo;
    const int P = sh.Ci * sh.Z;

    float acc[CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
        acc[cb] = 0.f;

    const int TCB = sh.T * CB;
    for (int dzi = 0; dzi < sh.Z; ++dzi) {
        // the output plane whose window reads plane z at offset dz (block-uniform)
        const int zc = z - (dzi - sh.kz);
        if (zc < 0 || zc % sh.sz != 0 || zc / sh.sz >= sh.Do)
            continue;
        const int l = zc / sh.sz;
        for (int co0 = 0; co0 < sh.Co; co0 += CC) {
            const int nc = min(CC, sh.Co - co0);
            __syncthreads(); // previous stage read (and the tap table written)
            for (int e = threadIdx.x; e < nc * TCB; e += kThreads) {
                const int cb = e % CB, rest = e / CB;
                const int q = rest / sh.T, t = rest - q * sh.T;
                const int ci = min(ci0 + cb, sh.Ci - 1); // clamped: never stored
                wl[e] = to_f(w[(static_cast<size_t>(co0 + q) * P + ci * sh.Z + dzi) * sh.T + t]);
            }
            __syncthreads();
            if (!active)
                continue;
            for (int t = 0; t < sh.T; ++t) {
                int i = 0, j = 0;
                if (!source_output(r, c, tl.dq[t], tl.ds[t], sh.s, sh.Ho, sh.Wo, i, j))
                    continue;
                const T *dyo = dy + ((static_cast<size_t>(n) * sh.Co + co0) * sh.Do + l) * HWo +
                               static_cast<size_t>(i) * sh.Wo + j;
                for (int q = 0; q < nc; ++q) {
                    const float g = to_f(dyo[static_cast<size_t>(q) * sh.Do * HWo]);
                    const float4 *w4 = reinterpret_cast<const float4 *>(wl + (q * sh.T + t) * CB);
#pragma unroll
                    for (int v = 0; v < CB / 4; ++v) {
                        const float4 ww = w4[v];
                        acc[4 * v] += ww.x * g;
                        acc[4 * v + 1] += ww.y * g;
                        acc[4 * v + 2] += ww.z * g;
                        acc[4 * v + 3] += ww.w * g;
                    }
                }
            }
        }
    }
    if (!active)
        return;
    const size_t HW = static_cast<size_t>(sh.H) * sh.W;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
        const int ci = ci0 + cb;
        if (ci >= sh.Ci)
            break;
        dx[((static_cast<size_t>(n) * sh.Ci + ci) * sh.D + z) * HW + p] = from_f<T>(acc[cb]);
    }
}

// Block = (pixel chunk, CO output channels, one input channel): per output
// pixel the dy of the block's output channels and the x under one group of
// (plane offset, tap) pairs feed CO x kTapGroup accumulators.  Sums over
// the block's threads: a fixed xor-shuffle tree per wave, then the waves in
// order.  Pixels run over (n, l, i, j); taps tt = dz_index * T + t.
template <typename T, int CO>
__global__ __launch_bounds__(kThreads) void wgrad_partial_generic_k(
    const T *__restrict__ x, const T *__restrict__ dy, float *__restrict__ part, ConvShape sh,
    int chunk)
{
    constexpr int NV = CO * kTapGroup + CO; // tap sums, then bias sums
    constexpr int kWavesG = kThreads / 64;
    __shared__ TapLds tl;
    __shared__ float red[kWavesG][NV];
    fill_taps(tl, sh.k);
    __syncthreads();

    const int co0 = blockIdx.y * CO, ci = blockIdx.z;
    const long HWo = static_cast<long>(sh.Ho) * sh.Wo;
    const long DHWo = HWo * sh.Do;
    const long total = DHWo * sh.N;
    const long begin = static_cast<long>(blockIdx.x) * chunk;
    const long end = min(begin + chunk, total);
    const size_t HW = static_cast<size_t>(sh.H) * sh.W;
    const bool do_bias = (ci == 0);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int TT = sh.Z * sh.T;
    const size_t Jt = static_cast<size_t>(sh.Ci) * TT + 1;

    for (int tg = 0; tg < TT; tg += kTapGroup) {
        float acc[CO][kTapGroup];
        float accb[CO];
#pragma unroll
        for (int q = 0; q < CO; ++q) {
            accb[q] = 0.f;
#pragma unroll
            for (int u = 0; u < kTapGroup; ++u)
                acc[q][u] = 0.f;
        }
        for (long e = begin + threadIdx.x; e < end; e += kThreads) {
            const int n = static_cast<int>(e / DHWo);
            const long rem = e - static_cast<long>(n) * DHWo;
            const int l = static_cast<int>(rem / HWo);
            const int o = static_cast<int>(rem - static_cast<long>(l) * HWo);
            const int i = o / sh.Wo, j = o % sh.Wo;
            float g[CO];
#pragma unroll
            for (int q = 0; q < CO; ++q)
                g[q] = co0 + q < sh.Co
                           ? to_f(dy[(static_cast<size_t>(n) * sh.Co + co0 + q) * DHWo + rem])
                           : 0.f;
            const int rc = centre_row(i, j, sh.s), cc = centre_col(j, sh.s);
            const int par = cc & 1;
            const T *img = x + static_cast<size_t>(n * sh.Ci + ci) * sh.D * HW;
#pragma unroll
            for (int u = 0; u < kTapGroup; ++u) {
                const int tt = tg + u;
                float v = 0.f;
                if (tt < TT) {
                    const int dzi = tt / sh.T, t = tt - dzi * sh.T;
                    const int z = sh.sz * l + dzi - sh.kz;
                    const int r = rc + tl.drow[par][t], c = cc + tl.dq[t];
                    if (z >= 0 && z < sh.D && r >= 0 && r < sh.H && c >= 0 && c < sh.W)
                        v = to_f(img[z * HW + static_cast<size_t>(r) * sh.W + c]);
                }
#pragma unroll
                for (int q = 0; q < CO; ++q)
                    acc[q][u] += g[q] * v;
            }
            if (tg == 0) {
#pragma unroll
                for (int q = 0; q < CO; ++q)
                    accb[q] += g[q];
            }
        }
        // wave sums (fixed xor tree), lane 0 to LDS
#pragma unroll
        for (int q = 0; q < CO; ++q) {
#pragma unroll
            for (int u = 0; u <= kTapGroup; ++u) {
                float v = u < kTapGroup ? acc[q][u] : accb[q];
#pragma unroll
                for (int m = 32; m > 0; m >>= 1)
                    v += __shfl_xor(v, m, 64);
                if (lane == 0)
                    red[wave][u < kTapGroup ? q * kTapGroup + u : CO * kTapGroup + q] = v;
            }
        }
        __syncthreads();
        // partial layout [e][chunk], e = co * (Ci*Z*T + 1) + col
        for (int idx = threadIdx.x; idx < NV; idx += kThreads) {
            float v = red[0][idx];
#pragma unroll
            for (int wv = 1; wv < kWavesG; ++wv)
                v += red[wv][idx];
            if (idx < CO * kTapGroup) {
                const int q = idx / kTapGroup, tt = tg + idx % kTapGroup;
                if (co0 + q < sh.Co && tt < TT)
                    part[((co0 + q) * Jt + static_cast<size_t>(ci) * TT + tt) * gridDim.x +
                         blockIdx.x] = v;
            } else {
                const int q = idx - CO * kTapGroup;
                if (tg == 0 && do_bias && co0 + q < sh.Co)
                    part[((co0 + q) * Jt + Jt - 1) * gridDim.x + blockIdx.x] = v;
            }
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(kThreads) void fill_zero_k(float *__restrict__ a, int na,
                                                        float *__restrict__ b, int nb)
{
    const int e = blockIdx.x * kThreads + threadIdx.x;
    if (e < na)
        a[e] = 0.f;
    else if (b != nullptr && e < na + nb)
        b[e - na] = 0.f;
}

// One output element per thread; argmax index dz_index * T + t (AM: uint8_t
// for 2-D calls, uint16_t for 3-D ones).
template <typename T, int MODE, typename AM>
__global__ __launch_bounds__(kThreads) void pool_fwd_generic_k(
    const T *__restrict__ x, T *__restrict__ y, AM *__restrict__ am,
    ConvShape sh, long total)
{
    __shared__ TapLds tl;
    fill_taps(tl, sh.k);
    __syncthreads();
    const long HWo = static_cast<long>(sh.Ho) * sh.Wo;
    const long DHWo = HWo * sh.Do;
    const size_t HW = static_cast<size_t>(sh.H) * sh.W;
    for (long e = static_cast<long>(blockIdx.x) * kThreads + threadIdx.x; e < total;
         e += static_cast<long>(gridDim.x) * kThreads) {
        const long plane = e / DHWo;
        const long rem = e - plane * DHWo;
        const int l = static_cast<int>(rem / HWo);
        const int o = static_cast<int>(rem - static_cast<long>(l) * HWo);
        const int i = o / sh.Wo, j = o % sh.Wo;
        const int rc = centre_row(i, j, sh.s), cc = centre_col(j, sh.s);
        const int par = cc & 1;
        float best = 0.f, sum = 0.f;
        int arg = 0;
        for (int dzi = 0; dzi < sh.Z; ++dzi) {
            const int z = sh.sz * l + dzi - sh.kz;
            const bool zin = z >= 0 && z < sh.D;
            const T *src = x + (plane * sh.D + (zin ? z : 0)) * HW;
            for (int t = 0; t < sh.T; ++t) {
                const int r = rc + tl.drow[par][t], c = cc + tl.dq[t];
                const float v = (zin && r >= 0 && r < sh.H && c >= 0 && c < sh.W)
                                    ? to_f(src[static_cast<size_t>(r) * sh.W + c])
                                    : 0.f;
                sum += v;
                if ((dzi == 0 && t == 0) || v > best) {
                    best = v;
                    arg = dzi * sh.T + t;
                }
            }
        }
        if (MODE == 0) {
            y[e] = from_f<T>(best);
            if (am != nullptr)
                am[e] = static_cast<AM>(arg);
        } else {
            y[e] = from_f<T>(sum / static_cast<float>(sh.Z * sh.T));
        }
    }
}

// One input element per thread: gathers from every output whose window
// holds it (plane lattice, then the hexagonal lattice test).
template <typename T, int MODE, typename AM>
__global__ __launch_bounds__(kThreads) void pool_bwd_generic_k(
    const T *__restrict__ dy, const AM *__restrict__ am,
    const T *__restrict__ relu_y, T *__restrict__ dx, ConvShape sh, long total)
{
    __shared__ TapLds tl;
    fill_taps(tl, sh.k);
    __syncthreads();
    const long HW = static_cast<long>(sh.H) * sh.W;
    const long DHW = HW * sh.D;
    const size_t HWo = static_cast<size_t>(sh.Ho) * sh.Wo;
    for (long e = static_cast<long>(blockIdx.x) * kThreads + threadIdx.x; e < total;
         e += static_cast<long>(gridDim.x) * kThreads) {
        const long plane = e / DHW;
        const long rem = e - plane * DHW;
        const int z = static_cast<int>(rem / HW);
        const int p = static_cast<int>(rem - static_cast<long>(z) * HW);
        const int r = p / sh.W, c = p % sh.W;
        float acc = 0.f;
        for (int dzi = 0; dzi < sh.Z; ++dzi) {
            const int zc = z - (dzi - sh.kz);
            if (zc < 0 || zc % sh.sz != 0 || zc / sh.sz >= sh.Do)
                continue;
            const int l = zc / sh.sz;
            for (int t = 0; t < sh.T; ++t) {
                int i = 0, j = 0;
                if (!source_output(r, c, tl.dq[t], tl.ds[t], sh.s, sh.Ho, sh.Wo, i, j))
                    continue;
                const size_t o = (plane * sh.Do + l) * HWo + static_cast<size_t>(i) * sh.Wo + j;
                if (MODE == 0) {
                    if (static_cast<int>(am[o]) == dzi * sh.T + t)
                        acc += to_f(dy[o]);
                } else {
                    acc += to_f(dy[o]);
                }
            }
        }
        if (MODE == 1)
            acc = acc / static_cast<float>(sh.Z * sh.T);
        if (relu_y != nullptr && !(to_f(relu_y[e]) > 0.f))
            acc = 0.f;
        dx[e] = from_f<T>(acc);
    }
}

inline int cdiv(long a, long b) { return static_cast<int>((a + b - 1) / b); }

// output channels per weight-gradient block: narrow layers keep one channel
// per block (more blocks, a cheaper block-wide sum)
int wgrad_co_block(int Co) { return Co >= 32 ? kWgCoBlock : 1; }

int wgrad_generic_chunks(const ConvShape &sh, int &chunk)
{
    const long total = static_cast<long>(sh.N) * sh.Do * sh.Ho * sh.Wo;
    const long pairs = static_cast<long>(cdiv(sh.Co, wgrad_co_block(sh.Co))) * sh.Ci;
    long nchunks = (2048 + pairs - 1) / pairs;
    nchunks = std::max(1L, std::min(nchunks, (total + 255) / 256));
    nchunks = std::min(nchunks, 65535L);
    chunk = static_cast<int>((total + nchunks - 1) / nchunks);
    if (chunk < 1)
        chunk = 1;
    return static_cast<int>((total + chunk - 1) / chunk);
}

} // namespace

bool conv_fwd_generic_ok(const ConvShape &sh)
{
    return plan::plan_fwd(sh.Ci * sh.Z, sh.Co, sh.k, sh.s).ok;
}

bool conv_bwd_data_generic_ok(const ConvShape &sh)
{
    return plan::plan_bwd_data(sh.Ci, sh.Co, sh.k).ok;
}

hipError_t conv_fwd_generic(const void *x, const void *w, const void *b, void *y,
                            const ConvShape &sh, Dtype dt, bool relu, hipStream_t st)
{
    // (input channel, plane offset) pairs are staged like 2-D input channels
    const plan::FwdPlan p = plan::plan_fwd(sh.Ci * sh.Z, sh.Co, sh.k, sh.s);
    if (!p.ok)
        return hipErrorInvalidConfiguration; // the ABI checks the plan first
    const int TI = p.TI, TJ = p.TJ, cb = p.cb, G = p.G;
    const size_t lds = p.lds;
    const int tiles_i = cdiv(sh.Ho, TI), tiles_j = cdiv(sh.Wo, TJ);
    dim3 grid(tiles_i * tiles_j * sh.Do, sh.N, cdiv(sh.Co, cb));
#define HEX_FWD_G(TT, CBV)                                                                   \
    HEX_LAUNCH((conv_fwd_generic_k<TT, CBV>), grid, dim3(kThreads), lds, st, (const TT *)x, \
               (const TT *)w, (const TT *)b, (TT *)y, sh, relu ? 1 : 0, TI, TJ, tiles_j, G)
#define HEX_FWD_CB(TT)                                                                       \
    do {                                                                                     \
        if (cb == 8) HEX_FWD_G(TT, 8);                                                       \
        else if (cb == 32) HEX_FWD_G(TT, 32);                                                \
        else HEX_FWD_G(TT, 64);                                                              \
    } while (0)
    if (dt == F32)
        HEX_FWD_CB(float);
    else
        HEX_FWD_CB(bf16raw);
#undef HEX_FWD_CB
#undef HEX_FWD_G
    return hipGetLastError();
}

hipError_t conv_bwd_data_generic(const void *dy, const void *w, void *dx, const ConvShape &sh,
                                 Dtype dt, hipStream_t st)
{
    const plan::BwdDataPlan p = plan::plan_bwd_data(sh.Ci, sh.Co, sh.k);
    if (!p.ok)
        return hipErrorInvalidConfiguration; // the ABI checks the plan first
    const int cb = p.cb, CC = p.CC;
    const size_t lds = p.lds;
    dim3 grid(cdiv(static_cast<long>(sh.H) * sh.W, kThreads) * sh.D, sh.N, cdiv(sh.Ci, cb));
#define HEX_BD_G(TT, CBV)                                                                    \
    HEX_LAUNCH((conv_bwd_data_generic_k<TT, CBV>), grid, dim3(kThreads), lds, st,            \
               (const TT *)dy, (const TT *)w, (TT *)dx, sh, CC)
#define HEX_BD_CB(TT)                                                                        \
    do {                                                                                     \
        if (cb == 8) HEX_BD_G(TT, 8);                                                        \
        else if (cb == 32) HEX_BD_G(TT, 32);                                                 \
        else HEX_BD_G(TT, 64);                                                               \
    } while (0)
    if (dt == F32)
        HEX_BD_CB(float);
    else
        HEX_BD_CB(bf16raw);
#undef HEX_BD_CB
#undef HEX_BD_G
    return hipGetLastError();
}

size_t wgrad_generic_workspace(const ConvShape &sh)
{
    int chunk;
    const int nchunks = wgrad_generic_chunks(sh, chunk);
    return sizeof(float) * static_cast<size_t>(nchunks) *
           (static_cast<size_t>(sh.Co) * sh.Ci * sh.Z * sh.T + sh.Co);
}

hipError_t wgrad_generic(const void *x, const void *dy, float *dw, float *db, void *ws,
                         const ConvShape &sh, Dtype dt, hipStream_t st)
{
    int chunk;
    const int nchunks = wgrad_generic_chunks(sh, chunk);
    float *part = static_cast<float *>(ws);
    const int cob = wgrad_co_block(sh.Co);
    dim3 grid(nchunks, cdiv(sh.Co, cob), sh.Ci);
#define HEX_WGG(TT, COV)                                                                     \
    HEX_LAUNCH((wgrad_partial_generic_k<TT, COV>), grid, dim3(kThreads), 0, st,              \
               (const TT *)x, (const TT *)dy, part, sh, chunk)
    if (dt == F32) {
        if (cob == 1) HEX_WGG(float, 1); else HEX_WGG(float, kWgCoBlock);
    } else {
        if (cob == 1) HEX_WGG(bf16raw, 1); else HEX_WGG(bf16raw, kWgCoBlock);
    }
#undef HEX_WGG
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    return reduce_partials(part, nchunks, sh.Co, sh.Ci * sh.Z * sh.T, dw, db, st);
}

hipError_t fill_zero_f32(float *dw, float *db, const ConvShape &sh, hipStream_t st)
{
    const long EW = static_cast<long>(sh.Co) * sh.Ci * sh.Z * sh.T;
    HEX_LAUNCH(fill_zero_k, dim3(cdiv(EW + sh.Co, kThreads)), dim3(kThreads), 0, st, dw,
                       static_cast<int>(EW), db, sh.Co);
    return hipGetLastError();
}

hipError_t pool_fwd_generic(const void *x, void *y, void *am, const ConvShape &sh, int mode,
                            Dtype dt, bool am16, hipStream_t st)
{
    const long total = static_cast<long>(sh.N) * sh.Ci * sh.Do * sh.Ho * sh.Wo;
    const int blocks = std::max(1, std::min(cdiv(total, kThreads), 65535 * 16));
#define HEX_POOL_FWD(T, M, A)                                                                \
    HEX_LAUNCH((pool_fwd_generic_k<T, M, A>), dim3(blocks), dim3(kThreads), 0, st,           \
               (const T *)x, (T *)y, (A *)am, sh, total)
#define HEX_POOL_FWD_A(T, M)                                                                 \
    do {                                                                                     \
        if (am16) HEX_POOL_FWD(T, M, uint16_t); else HEX_POOL_FWD(T, M, uint8_t);            \
    } while (0)
    if (dt == F32) {
        if (mode == 0) HEX_POOL_FWD_A(float, 0); else HEX_POOL_FWD(float, 1, uint8_t);
    } else {
        if (mode == 0) HEX_POOL_FWD_A(bf16raw, 0); else HEX_POOL_FWD(bf16raw, 1, uint8_t);
    }
#undef HEX_POOL_FWD_A
#undef HEX_POOL_FWD
    return hipGetLastError();
}

hipError_t pool_bwd_generic(const void *dy, const void *am, const void *relu_y, void *dx,
                            const ConvShape &sh, int mode, Dtype dt, bool am16, hipStream_t st)
{
    const long total = static_cast<long>(sh.N) * sh.Ci * sh.D * sh.H * sh.W;
    const int blocks = std::max(1, std::min(cdiv(total, kThreads), 65535 * 16));
#define HEX_POOL_BWD(T, M, A)                                                                \
    HEX_LAUNCH((pool_bwd_generic_k<T, M, A>), dim3(blocks), dim3(kThreads), 0, st,           \
               (const T *)dy, (const A *)am, (const T *)relu_y, (T *)dx, sh, total)
#define HEX_POOL_BWD_A(T, M)                                                                 \
    do {                                                                                     \
        if (am16) HEX_POOL_BWD(T, M, uint16_t); else HEX_POOL_BWD(T, M, uint8_t);            \
    } while (0)
    if (dt == F32) {
        if (mode == 0) HEX_POOL_BWD_A(float, 0); else HEX_POOL_BWD(float, 1, uint8_t);
    } else {
        if (mode == 0) HEX_POOL_BWD_A(bf16raw, 0); else HEX_POOL_BWD(bf16raw, 1, uint8_t);
    }
#undef HEX_POOL_BWD_A
#undef HEX_POOL_BWD
    return hipGetLastError();
}

} // namespace hexk
