// k_mfma_bf16.hip -- bf16 convolutions on the matrix cores (fp32 accumulate).
//
// Implicit GEMM for the forward pass and, with the point-reflected kernel
// and the channel roles swapped, for the stride-1 data gradient:
//   D[pixel][oc] = sum_{t, ic} A[pixel][(t, ic)] * B[(t, ic)][oc]
//   forward:        A = x at pixel + tap t,  B[(t, ic)][oc] = w[oc][ic][t]
//   data gradient:  A = dy at pixel + tap t, B[(t, ic)][oc] = w[ic][oc][T-1-t]
// v_mfma_f32_16x16x32_bf16, lane layout (checked on the device):
//   a[i] = A[lane % 16][8 * (lane / 16) + i], b[i] = B[8 * (lane / 16) + i][lane % 16],
//   d[j] = D[4 * (lane / 16) + j][lane % 16].
// K runs over taps, then input channels in blocks of 32, so each lane's 8
// A values are 8 consecutive channels of one pixel: the input tile is kept
// channel-last in LDS (one 16-byte read per A fragment), pixel slots
// row-major with the k-wide zero halo; a tap is one of two fixed slot offsets
// chosen by the column parity of the lane's pixel.  The tile is staged from
// NCHW through registers with an 8x8 bf16 transpose.
//
// Block: full-width tile of TR rows, 64 output channels (grid.y covers more),
// 4 waves = 2 channel halves x 2 pixel halves; each wave accumulates up to 8
// pixel tiles x 2 channel tiles.  Weights (B) are held in registers, KC
// K-steps at a time.  The result goes through LDS so that global stores are
// contiguous 16-byte rows.
#include <algorithm>

#include "hexdev.h"
#include "kernels.h"

namespace hexk {
namespace {

using namespace hexgeom;

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;
constexpr int kMT = 8; // pixel tiles (of 16) per wave
constexpr int kOCB = 64; // output channels per block

struct WideTiling {
    int TR, npix_max, LCP, CS; // LCP: slots per LDS row; CS: bf16 per pixel slot
    int ntiles;              // tiles per image
    int IC, OC, KS;          // input / output channels, K-steps (32 each)
};

__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel)
{
    return __builtin_amdgcn_perm(hi, lo, sel);
}

// Stage a full-width window (rows r0-K .. r0+rows+K-1, columns -K .. W+K-1)
// of IC channels into LDS, channel-last: element (r, c, ic) at
// (((r - r_lo) * LCP + c - c_lo) * CS + ic).  Work item = (8-channel group, window row, 8-column
// group): 8 loads of 16 bytes, an 8x8 transpose, 8 stores of 16 bytes.
struct WideWindow {
    int r_lo, c_lo, LR, LC;
    __device__ __forceinline__ int slot(int r, int c, int LCP) const
    {
        return (r - r_lo) * LCP + (c - c_lo);
    }
};

__device__ __forceinline__ void stage_wide(bf16raw *__restrict__ lds, const bf16raw *__restrict__ src,
                                           size_t HW, int H, int W, int IC, const WideWindow &tl,
                                           int LCP, int CS)
{
    const int a8 = (tl.c_lo >= 0 ? tl.c_lo : tl.c_lo - 7) / 8 * 8;
    const int ng = (tl.c_lo + tl.LC - a8 + 7) / 8;
    const int items = (IC / 8) * tl.LR * ng;
    for (int it0 = threadIdx.x; it0 < items; it0 += 2 * kThreads) {
        uint4 in[2][8];
        int cq[2], rq[2], gq[2];
        bool live[2], rowok[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int it = it0 + h * kThreads;
            live[h] = it < items;
            const int g = it % ng;
            const int rest = it / ng;
            const int rr = rest % tl.LR;
            const int cg = rest / tl.LR;
            cq[h] = cg;
            rq[h] = rr;
            gq[h] = g;
            const int r = tl.r_lo + rr;
            const int c = a8 + 8 * g;
            rowok[h] = live[h] && r >= 0 && r < H && c >= 0 && c + 7 < W;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const bf16raw *p =
                    src + (rowok[h] ? (static_cast<size_t>(cg * 8 + j) * HW + static_cast<size_t>(r) * W + c)
                                    : 0);
                in[h][j] = *reinterpret_cast<const uint4 *>(p);
            }
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            if (!live[h])
                continue;
            const int c = a8 + 8 * gq[h];
            const int r = tl.r_lo + rq[h];
#pragma unroll
            for (int px = 0; px < 8; ++px) {
                const int cc = c + px;
                if (cc < tl.c_lo || cc >= tl.c_lo + tl.LC)
                    continue;
                const uint32_t sel = (px & 1) ? 0x07060302u : 0x05040100u;
                uint4 o;
                // channel pair (2e, 2e+1) of pixel px: dword px/2 of rows 2e, 2e+1
                uint32_t w4[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t lo = reinterpret_cast<const uint32_t *>(&in[h][2 * e])[px >> 1];
                    const uint32_t hi = reinterpret_cast<const uint32_t *>(&in[h][2 * e + 1])[px >> 1];
                    w4[e] = perm(hi, lo, sel);
                }
                o.x = rowok[h] ? w4[0] : 0u;
                o.y = rowok[h] ? w4[1] : 0u;
                o.z = rowok[h] ? w4[2] : 0u;
                o.w = rowok[h] ? w4[3] : 0u;
                *reinterpret_cast<uint4 *>(lds + static_cast<size_t>(tl.slot(r, cc, LCP)) * CS +
                                           cq[h] * 8) = o;
            }
        }
    }
}

template <int K, int KC, bool REFLECT>
__global__ __launch_bounds__(kThreads, 2) void conv_bf16_wide_k(
    const bf16raw *__restrict__ xin, const bf16raw *__restrict__ w, const bf16raw *__restrict__ bias,
    bf16raw *__restrict__ y, ConvShape sh, int relu, WideTiling tg)
{
    constexpr int T = num_taps(K);
    extern __shared__ __align__(16) bf16raw lds[];
    const int H = sh.H, W = sh.W;
    const size_t HW = static_cast<size_t>(H) * W;
    const int IC = tg.IC, OC = tg.OC;
    const int n = blockIdx.x / tg.ntiles;
    const int r0 = (blockIdx.x - n * tg.ntiles) * tg.TR;
    const int rows = min(tg.TR, H - r0);
    const int npix = rows * W;
    const WideWindow tl{r0 - K, -K, rows + 2 * K, W + 2 * K};
    const int oc_blk = blockIdx.y * kOCB;

    stage_wide(lds, xin + static_cast<size_t>(n) * IC * HW, HW, H, W, IC, tl, tg.LCP, tg.CS);

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int m = lane & 15, kq = lane >> 4;
    const int ph = wave & 1;        // pixel half
    const int oh = wave >> 1;       // output-channel half (32 channels)
    const int ntile = (npix + 15) / 16;

    // centre slots and column parity of this lane's A rows
    int cen[kMT];
    bool pv[kMT], podd[kMT];
#pragma unroll
    for (int i = 0; i < kMT; ++i) {
        const int mt = ph + 2 * i;
        const int p = mt * 16 + m;
        pv[i] = mt < ntile && p < npix;
        const int pr = pv[i] ? p / W : 0, pc = pv[i] ? p - pr * W : 0;
        cen[i] = tl.slot(r0 + pr, pc, tg.LCP);
        podd[i] = (pc & 1) != 0;
    }
    floatx4 acc[kMT][2];
#pragma unroll
    for (int i = 0; i < kMT; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
            acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    __syncthreads();

    const int icb = IC / 32; // K-steps per tap
    for (int s0 = 0; s0 < tg.KS; s0 += KC) {
        // B fragments for K-steps s0 .. s0+KC-1 and this wave's 2 channel tiles
        bf16x8 bfr[KC][2];
#pragma unroll
        for (int s = 0; s < KC; ++s) {
            const int ks = s0 + s;
            const int t = ks / icb;
            const int ic0 = (ks - t * icb) * 32 + 8 * kq;
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int oc = oc_blk + oh * 32 + j * 16 + m;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    bf16raw v = 0;
                    if (ks < tg.KS && oc < OC) {
                        const int ic = ic0 + e;
                        v = REFLECT ? w[(static_cast<size_t>(ic) * OC + oc) * T + (T - 1 - t)]
                                    : w[(static_cast<size_t>(oc) * IC + ic) * T + t];
                    }
                    bfr[s][j][e] = __builtin_bit_cast(__bf16, v);
                }
            }
        }
#pragma unroll
        for (int s = 0; s < KC; ++s) {
            const int ks = s0 + s;
            if (ks >= tg.KS)
                break;
            const int t = ks / icb;
            const int ic0 = (ks - t * icb) * 32 + 8 * kq;
            int dq = 0, ds = 0;
            tap_axial(K, t, dq, ds);
            const int off0 = tap_drow(dq, ds, 0) * tg.LCP + dq;
            const int off1 = tap_drow(dq, ds, 1) * tg.LCP + dq;
            uint4 qa[kMT];
#pragma unroll
            for (int i = 0; i < kMT; ++i) {
                // every read issued (slot 0 for padding lanes), then masked
                const int sl = pv[i] ? cen[i] + (podd[i] ? off1 : off0) : 0;
                qa[i] = *reinterpret_cast<const uint4 *>(lds + static_cast<size_t>(sl) * tg.CS + ic0);
            }
#pragma unroll
            for (int i = 0; i < kMT; ++i) {
                const uint4 q = pv[i] ? qa[i] : make_uint4(0, 0, 0, 0);
                const bf16x8 a = __builtin_bit_cast(bf16x8, q);
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bfr[s][j], acc[i][j], 0, 0, 0);
            }
        }
    }

    // epilogue: bias, ReLU, bf16 into LDS [oc][pixel], then contiguous stores
    __syncthreads();
    const int opitch = tg.npix_max + 8;
    bf16raw *outl = lds;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int ocl = oh * 32 + j * 16 + m;
        const int oc = oc_blk + ocl;
        const float bv = (bias != nullptr && oc < OC) ? to_f(bias[oc]) : 0.f;
#pragma unroll
        for (int i = 0; i < kMT; ++i) {
            const int mt = ph + 2 * i;
            const int q0 = mt * 16 + 4 * kq;
            if (mt >= ntile)
                continue;
            uint32_t pk[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                float v0 = acc[i][j][2 * h] + bv, v1 = acc[i][j][2 * h + 1] + bv;
                if (relu) {
                    v0 = fmaxf(v0, 0.f);
                    v1 = fmaxf(v1, 0.f);
                }
                pk[h] = static_cast<uint32_t>(from_f<bf16raw>(v0)) |
                        (static_cast<uint32_t>(from_f<bf16raw>(v1)) << 16);
            }
            *reinterpret_cast<uint2 *>(outl + ocl * opitch + q0) = make_uint2(pk[0], pk[1]);
        }
    }
    __syncthreads();
    const int nvec = (npix + 7) / 8;
    const int noc = min(kOCB, OC - oc_blk);
    for (int e = threadIdx.x; e < noc * nvec; e += kThreads) {
        const int ocl = e / nvec, v8 = e - ocl * nvec;
        const int p = v8 * 8;
        bf16raw *dst = y + (static_cast<size_t>(n) * OC + oc_blk + ocl) * HW + static_cast<size_t>(r0) * W + p;
        const bf16raw *srcp = outl + ocl * opitch + p;
        if (p + 7 < npix) {
            *reinterpret_cast<uint4 *>(dst) = *reinterpret_cast<const uint4 *>(srcp);
        } else {
            for (int q = 0; q < npix - p; ++q)
                dst[q] = srcp[q];
        }
    }
}

inline int cdiv(long a, long b) { return static_cast<int>((a + b - 1) / b); }

constexpr int kKC = 7; // K-steps whose B fragments are held at once

WideTiling wide_tiling(const ConvShape &sh, int IC, int OC)
{
    WideTiling tg;
    // rows per block: at most 2 * kMT pixel tiles of 16
    tg.TR = std::max(1, std::min(sh.H, (2 * kMT * 16) / sh.W));
    tg.npix_max = tg.TR * sh.W;
    tg.LCP = sh.W + 2 * sh.k;
    tg.CS = IC + 8; // 16-byte aligned pixel vectors, staggered banks
    tg.ntiles = cdiv(sh.H, tg.TR);
    tg.IC = IC;
    tg.OC = OC;
    tg.KS = sh.T * IC / 32;
    return tg;
}

size_t wide_lds_bytes(const ConvShape &sh, const WideTiling &tg)
{
    const size_t in = sizeof(bf16raw) * static_cast<size_t>(tg.TR + 2 * sh.k) * tg.LCP * tg.CS;
    const size_t out = sizeof(bf16raw) * static_cast<size_t>(kOCB) * (tg.npix_max + 8);
    return std::max(in, out);
}

} // namespace

bool bf16_wide_ok(const ConvShape &sh, int IC, int OC)
{
    if (sh.s != 1 || (sh.k != 1 && sh.k != 2) || IC % 32 != 0 || sh.W % 8 != 0 ||
        sh.W > 2 * kMT * 16)
        return false;
    const WideTiling tg = wide_tiling(sh, IC, OC);
    return wide_lds_bytes(sh, tg) <= 80 * 1024;
}

hipError_t bf16_wide_conv(const void *in, const void *w, const void *bias, void *out,
                          const ConvShape &sh, bool reflect, bool relu, hipStream_t st)
{
    const int IC = reflect ? sh.Co : sh.Ci;
    const int OC = reflect ? sh.Ci : sh.Co;
    const WideTiling tg = wide_tiling(sh, IC, OC);
    dim3 grid(tg.ntiles * sh.N, cdiv(OC, kOCB));
    const size_t lds = wide_lds_bytes(sh, tg);
    const bf16raw *x = static_cast<const bf16raw *>(in);
    const bf16raw *wp = static_cast<const bf16raw *>(w);
    const bf16raw *bp = static_cast<const bf16raw *>(bias);
    bf16raw *y = static_cast<bf16raw *>(out);
#define HEX_WIDE(KV, RV)                                                                     \
    hipLaunchKernelGGL((conv_bf16_wide_k<KV, kKC, RV>), grid, dim3(kThreads), lds, st, x, wp, \
                       bp, y, sh, relu ? 1 : 0, tg)
    if (sh.k == 1) {
        if (reflect) HEX_WIDE(1, true); else HEX_WIDE(1, false);
    } else {
        if (reflect) HEX_WIDE(2, true); else HEX_WIDE(2, false);
    }
#undef HEX_WIDE
    return hipGetLastError();
}

} // namespace hexk
