// shear.h -- the sheared LDS tile layout and its staging routine.
//
// A block stages a window of input rows [r_lo, r_lo+LR) x columns
// [c_lo, c_lo+LC) of one or more channel planes.  Element (r, c) of a
// channel is stored at
//     addr(r, c) = (c - c_lo) * P + (r - r_lo) - (floor(c/2) - floor(c_lo/2)),
// i.e. column-major with every column shifted up by floor(c/2): the row
// index inside a column becomes the axial coordinate s = r - floor(c/2).
// In axial coordinates a tap (dq, ds) is a plain translation, so the tap of
// a centre stored at address a sits at a + dq*P + ds whatever the centre's
// column parity -- no parity-dependent addressing remains in the inner
// loops.  P >= LR + 1 keeps the columns apart.
//
// Window cells outside the H x W plane are written as zeros (the padding
// of the convolution).
#pragma once

#include "hexdev.h"

namespace hexk {

struct ShearTile {
    int r_lo, c_lo, LR, LC, P;
    int CS; // floats per channel (>= LC * P; fixed for all tiles of a launch)
    __device__ __forceinline__ int addr(int r, int c) const
    {
        return (c - c_lo) * P + (r - r_lo) - ((c >> 1) - (c_lo >> 1));
    }
    __host__ __device__ __forceinline__ int chan_stride() const { return CS; }
};

// Division by a block-uniform positive divisor d for numerators < 2^31
// (multiply-high method; magic numbers computed on the host).
struct FastDiv {
    uint32_t d, m, l;
};

inline FastDiv make_fastdiv(uint32_t d)
{
    uint32_t l = 0;
    while ((1u << l) < d)
        ++l;
    const uint64_t m = ((uint64_t(1) << 32) * ((uint64_t(1) << l) - d)) / d + 1;
    return FastDiv{d, static_cast<uint32_t>(m), l};
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv &f)
{
    return (__umulhi(f.m, n) + n) >> f.l;
}

template <typename T> struct Vec4Load;
template <> struct Vec4Load<float> {
    __device__ __forceinline__ static void load(const float *p, float v[4])
    {
        const float4 q = *reinterpret_cast<const float4 *>(p);
        v[0] = q.x;
        v[1] = q.y;
        v[2] = q.z;
        v[3] = q.w;
    }
};
template <> struct Vec4Load<bf16raw> {
    __device__ __forceinline__ static void load(const bf16raw *p, float v[4])
    {
        const uint2 q = *reinterpret_cast<const uint2 *>(p);
        v[0] = __uint_as_float(q.x << 16);
        v[1] = __uint_as_float(q.x & 0xffff0000u);
        v[2] = __uint_as_float(q.y << 16);
        v[3] = __uint_as_float(q.y & 0xffff0000u);
    }
};

// Stage `nch` channel planes (plane stride `src_plane` elements, row stride
// W) into dst[ch * chan_stride + addr(r, c)] for the window rows
// r_lo .. r_lo + LRmax - 1 (rows past the block's own window land in the
// unused slack of each column and are never read as taps).  Each thread
// owns one 4-column group and walks (channel, row) pairs; every batch of U
// loads is issued before any is consumed (addresses of out-of-plane rows
// are clamped to the plane start and the values replaced by zero), so the
// loads overlap.  Groups entirely outside the plane are written as zeros
// without loads.  Requires the window origin column c_lo + K to be a
// multiple of 4 when `vec4` (W % 4 == 0) for whole-group loads.  Call from
// all threads of the block.
template <int U, typename T>
__device__ __forceinline__ void stage_shear(float *__restrict__ dst, const T *__restrict__ src,
                                            size_t src_plane, int nch, int H, int W,
                                            const ShearTile &tl, int LRmax, const FastDiv &fdlr,
                                            bool vec4)
{
    const int nt = blockDim.x;
    const int a4 = (tl.c_lo >= 0 ? tl.c_lo : tl.c_lo - 3) / 4 * 4; // floor to multiple of 4
    const int ng = (tl.c_lo + tl.LC - a4 + 3) / 4;
    const int gp = ng < nt ? ng : nt; // groups handled per pass
    const int rstep = nt / gp;
    const int fr0 = threadIdx.x / gp;
    if (fr0 >= rstep)
        return;
    const int cs = tl.chan_stride();
    const int total = nch * LRmax;
    const int P = tl.P;
    for (int g = threadIdx.x % gp; g < ng; g += gp) {
        const int c = a4 + 4 * g;
        const bool inside = vec4 && c >= 0 && c + 3 < W;
        const bool outside = c + 3 < 0 || c >= W;
        // LDS offsets of the group's 4 columns relative to column c (c even)
        const int base_c = (c - tl.c_lo) * P - ((c >> 1) - (tl.c_lo >> 1));
        const int o1 = P, o2 = 2 * P - 1, o3 = 3 * P - 1;
        bool wcol[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            wcol[j] = (c + j >= tl.c_lo) && (c + j < tl.c_lo + tl.LC);
        // the three cases are separate loops so each batch is straight-line
        if (inside) {
            for (int fb = fr0; fb < total; fb += rstep * U) {
                float v[U][4];
                int da[U]; // may be negative (address of a halo column group)
                bool okr[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int fr = fb + u * rstep;
                    const int ch = static_cast<int>(fdiv(static_cast<uint32_t>(fr), fdlr));
                    const int rr = fr - ch * LRmax;
                    const int r = tl.r_lo + rr;
                    okr[u] = fr < total && r >= 0 && r < H;
                    da[u] = ch * cs + base_c + rr;
                    const T *p = src + (okr[u] ? ch * src_plane + static_cast<size_t>(r) * W + c : 0);
                    Vec4Load<T>::load(p, v[u]);
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    if (fb + u * rstep < total) {
                        float *d = dst + da[u];
                        const float z0 = okr[u] ? v[u][0] : 0.f, z1 = okr[u] ? v[u][1] : 0.f;
                        const float z2 = okr[u] ? v[u][2] : 0.f, z3 = okr[u] ? v[u][3] : 0.f;
                        if (wcol[0]) d[0] = z0;
                        if (wcol[1]) d[o1] = z1;
                        if (wcol[2]) d[o2] = z2;
                        if (wcol[3]) d[o3] = z3;
                    }
                }
            }
        } else if (outside) {
            for (int fr = fr0; fr < total; fr += rstep) {
                const int ch = static_cast<int>(fdiv(static_cast<uint32_t>(fr), fdlr));
                float *d = dst + ch * cs + base_c + (fr - ch * LRmax);
                if (wcol[0]) d[0] = 0.f;
                if (wcol[1]) d[o1] = 0.f;
                if (wcol[2]) d[o2] = 0.f;
                if (wcol[3]) d[o3] = 0.f;
            }
        } else {
            for (int fb = fr0; fb < total; fb += rstep * U) {
                float v[U][4];
                int da[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int fr = fb + u * rstep;
                    const int ch = static_cast<int>(fdiv(static_cast<uint32_t>(fr), fdlr));
                    const int rr = fr - ch * LRmax;
                    const int r = tl.r_lo + rr;
                    const bool ok = fr < total && r >= 0 && r < H;
                    da[u] = ch * cs + base_c + rr;
                    const T *row = src + (ok ? ch * src_plane + static_cast<size_t>(r) * W : 0);
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const bool okj = ok && c + j >= 0 && c + j < W;
                        const float t = to_f(row[okj ? c + j : 0]);
                        v[u][j] = okj ? t : 0.f;
                    }
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    if (fb + u * rstep < total) {
                        float *d = dst + da[u];
                        if (wcol[0]) d[0] = v[u][0];
                        if (wcol[1]) d[o1] = v[u][1];
                        if (wcol[2]) d[o2] = v[u][2];
                        if (wcol[3]) d[o3] = v[u][3];
                    }
                }
            }
        }
    }
}

// dst[ch * dst_plane + pr * pitch + pc] = plane ch at (r0 + pr, c0 + pc) for
// pr < rows, pc < cols (no halo; every element is inside the plane).  Rows
// are walked up to `rows_max` (fdr divides by it) so that the flattened
// (channel, row) index needs no loop.  Same batching as stage_shear.
template <int U, typename T>
__device__ __forceinline__ void stage_plain(float *__restrict__ dst, int dst_plane, int pitch,
                                            const T *__restrict__ src, size_t src_plane, int nch,
                                            int W, int r0, int c0, int rows, int cols,
                                            int rows_max, const FastDiv &fdr, bool vec4)
{
    const int nt = blockDim.x;
    const int ng = (cols + 3) / 4;
    const int gp = ng < nt ? ng : nt;
    const int rstep = nt / gp;
    const int fr0 = threadIdx.x / gp;
    if (fr0 >= rstep)
        return;
    const int total = nch * rows_max;
    for (int g = threadIdx.x % gp; g < ng; g += gp) {
        const int pc = 4 * g;
        const bool full = vec4 && pc + 3 < cols;
        for (int fb = fr0; fb < total; fb += rstep * U) {
            float v[U][4];
            int da[U];
            if (full) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int fr = fb + u * rstep;
                    const int ch = static_cast<int>(fdiv(static_cast<uint32_t>(fr), fdr));
                    const int pr = fr - ch * rows_max;
                    const bool ok = fr < total && pr < rows;
                    da[u] = ok ? ch * dst_plane + pr * pitch + pc : -1;
                    Vec4Load<T>::load(
                        src + (ok ? ch * src_plane + static_cast<size_t>(r0 + pr) * W + c0 + pc : 0),
                        v[u]);
                }
            } else {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int fr = fb + u * rstep;
                    const int ch = static_cast<int>(fdiv(static_cast<uint32_t>(fr), fdr));
                    const int pr = fr - ch * rows_max;
                    const bool ok = fr < total && pr < rows;
                    da[u] = ok ? ch * dst_plane + pr * pitch + pc : -1;
                    const T *row =
                        src + (ok ? ch * src_plane + static_cast<size_t>(r0 + pr) * W + c0 : 0);
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        v[u][j] = to_f(row[(ok && pc + j < cols) ? pc + j : 0]);
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (da[u] >= 0) {
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        if (pc + j < cols)
                            dst[da[u] + j] = v[u][j];
                }
            }
        }
    }
}


// Register-staged copy of a sheared window, for software pipelining: load()
// issues the global loads of a window into registers (up to U float4 per
// thread), commit() writes them to LDS later -- so the loads of the next
// tile overlap the compute and stores of the current one.  The work split
// is that of stage_shear; the launcher checks fits().
template <int U> struct ShearPrefetch {
    float v[U][4];
    int da[U];    // LDS address of the group's first column (may be negative)
    bool live[U]; // row to be written
    bool okr[U];  // row inside the plane (else zeros)
    int base_c, c;
    bool wcol[4];
    int P;

    // column groups of a window of LCmax columns (upper bound) and the rows
    // each thread covers; the launcher checks groups <= threads, rows <= U
    __host__ __device__ static int groups(int LCmax) { return (LCmax + 3) / 4 + 1; }
    __host__ __device__ static int rows_per_thread(int nch, int LRmax, int LCmax, int nt)
    {
        const int rstep = nt / groups(LCmax);
        return rstep > 0 ? (nch * LRmax + rstep - 1) / rstep : 1 << 30;
    }

    // Requires ceil(window columns / 4) + 1 <= blockDim.x (one column group
    // per thread) and W % 4 == 0 (whole 4-column groups are inside or outside
    // the plane).
    template <typename T>
    __device__ __forceinline__ void load(const T *__restrict__ src, size_t src_plane, int nch,
                                         int H, int W, const ShearTile &tl, int LRmax,
                                         const FastDiv &fdlr)
    {
        const int nt = blockDim.x;
        const int a4 = (tl.c_lo >= 0 ? tl.c_lo : tl.c_lo - 3) / 4 * 4;
        const int ng = (tl.c_lo + tl.LC - a4 + 3) / 4;
        const int rstep = nt / ng;
        const int g = threadIdx.x % ng;
        const int fr0 = threadIdx.x / ng;
        const int cs = tl.chan_stride();
        const int total = nch * LRmax;
        P = tl.P;
        c = a4 + 4 * g;
        base_c = (c - tl.c_lo) * P - ((c >> 1) - (tl.c_lo >> 1));
#pragma unroll
        for (int j = 0; j < 4; ++j)
            wcol[j] = (c + j >= tl.c_lo) && (c + j < tl.c_lo + tl.LC);
        const bool inside = c >= 0 && c + 3 < W;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int fr = fr0 + u * rstep;
            live[u] = fr0 < rstep && fr < total;
            const int ch = static_cast<int>(fdiv(static_cast<uint32_t>(fr), fdlr));
            const int rr = fr - ch * LRmax;
            const int r = tl.r_lo + rr;
            okr[u] = live[u] && inside && r >= 0 && r < H;
            da[u] = ch * cs + base_c + rr;
            Vec4Load<T>::load(src + (okr[u] ? ch * src_plane + static_cast<size_t>(r) * W + c : 0),
                              v[u]);
        }
    }

    // Three-dimensional variant: staged channel ch = ci * Z + dz is plane
    // d0 + dz of input channel ci (channel stride chan_plane, plane stride
    // plane); planes dz outside [dz_lo, dz_hi) lie outside the volume and
    // are staged as zeros.  img is channel 0, plane 0 of the sample (a valid
    // address; z_off = d0 * plane is added only for loaded rows).
    template <typename T>
    __device__ __forceinline__ void load3(const T *__restrict__ img, size_t chan_plane,
                                          size_t plane, long z_off, int Z, int dz_lo, int dz_hi,
                                          int nch, int H, int W, const ShearTile &tl, int LRmax,
                                          const FastDiv &fdlr)
    {
        const int nt = blockDim.x;
        const int a4 = (tl.c_lo >= 0 ? tl.c_lo : tl.c_lo - 3) / 4 * 4;
        const int ng = (tl.c_lo + tl.LC - a4 + 3) / 4;
        const int rstep = nt / ng;
        const int g = threadIdx.x % ng;
        const int fr0 = threadIdx.x / ng;
        const int cs = tl.chan_stride();
        const int total = nch * LRmax;
        P = tl.P;
        c = a4 + 4 * g;
        base_c = (c - tl.c_lo) * P - ((c >> 1) - (tl.c_lo >> 1));
#pragma unroll
        for (int j = 0; j < 4; ++j)
            wcol[j] = (c + j >= tl.c_lo) && (c + j < tl.c_lo + tl.LC);
        const bool inside = c >= 0 && c + 3 < W;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int fr = fr0 + u * rstep;
            live[u] = fr0 < rstep && fr < total;
            const int ch = static_cast<int>(fdiv(static_cast<uint32_t>(fr), fdlr));
            const int rr = fr - ch * LRmax;
            const int r = tl.r_lo + rr;
            const int ci = ch / Z, dz = ch - ci * Z;
            okr[u] = live[u] && inside && r >= 0 && r < H && dz >= dz_lo && dz < dz_hi;
            da[u] = ch * cs + base_c + rr;
            Vec4Load<T>::load(img + (okr[u] ? static_cast<long>(ci * chan_plane + dz * plane) +
                                                  z_off + static_cast<long>(r) * W + c
                                            : 0),
                              v[u]);
        }
    }

    __device__ __forceinline__ void commit(float *__restrict__ dst) const
    {
        const int o1 = P, o2 = 2 * P - 1, o3 = 3 * P - 1;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (live[u]) {
                float *d = dst + da[u];
                if (wcol[0]) d[0] = okr[u] ? v[u][0] : 0.f;
                if (wcol[1]) d[o1] = okr[u] ? v[u][1] : 0.f;
                if (wcol[2]) d[o2] = okr[u] ? v[u][2] : 0.f;
                if (wcol[3]) d[o3] = okr[u] ? v[u][3] : 0.f;
            }
        }
    }
};

} // namespace hexk
