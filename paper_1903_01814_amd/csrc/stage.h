// stage.h -- global -> LDS staging helpers.
//
// Each thread issues a batch of U independent global loads into registers
// before writing any of them to LDS, so a block keeps U loads per thread in
// flight instead of waiting out one memory latency per element.
#pragma once

#include "hexdev.h"

namespace hexk {

// dst[rr * LC + cc] = plane[(r_lo + rr) * W + (c_lo + cc)] for rr < LR,
// cc < LC, zero outside the H x W plane.  All threads of the block call it.
template <int U, typename T>
__device__ __forceinline__ void stage_window(float *__restrict__ dst, const T *__restrict__ plane,
                                             int H, int W, int r_lo, int c_lo, int LR, int LC)
{
    const int nt = blockDim.x;
    if (LC <= nt) {
        // fixed column per thread, rows strided: no division in the loop
        const int rstep = nt / LC;
        const int cc = threadIdx.x % LC;
        const int rr0 = threadIdx.x / LC;
        if (rr0 >= rstep)
            return;
        const int c = c_lo + cc;
        const bool cin = c >= 0 && c < W;
        for (int rb = rr0; rb < LR; rb += rstep * U) {
            float v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int rr = rb + u * rstep;
                const int r = r_lo + rr;
                v[u] = (rr < LR && cin && r >= 0 && r < H)
                           ? to_f(plane[static_cast<size_t>(r) * W + c])
                           : 0.f;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int rr = rb + u * rstep;
                if (rr < LR)
                    dst[rr * LC + cc] = v[u];
            }
        }
    } else {
        const int total = LR * LC;
        for (int base = threadIdx.x; base < total; base += nt * U) {
            float v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int e = base + u * nt;
                const int rr = e / LC, cc = e - rr * LC;
                const int r = r_lo + rr, c = c_lo + cc;
                v[u] = (e < total && r >= 0 && r < H && c >= 0 && c < W)
                           ? to_f(plane[static_cast<size_t>(r) * W + c])
                           : 0.f;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int e = base + u * nt;
                if (e < total)
                    dst[e] = v[u];
            }
        }
    }
}

// dst[row * dst_stride + i] = src[row * src_stride + i] for row < nrows,
// i < len (each source row contiguous).
template <int U, typename T>
__device__ __forceinline__ void stage_rows(float *__restrict__ dst, int dst_stride,
                                           const T *__restrict__ src, size_t src_stride,
                                           int nrows, int len)
{
    const int nt = blockDim.x;
    const int total = nrows * len;
    for (int base = threadIdx.x; base < total; base += nt * U) {
        float v[U];
        int row[U], col[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int e = base + u * nt;
            row[u] = e / len;
            col[u] = e - row[u] * len;
            v[u] = e < total ? to_f(src[row[u] * src_stride + col[u]]) : 0.f;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int e = base + u * nt;
            if (e < total)
                dst[row[u] * dst_stride + col[u]] = v[u];
        }
    }
}

} // namespace hexk
