// hexdev.h -- device-side helpers shared by the kernels: dtype conversion,
// tap tables in LDS, launch-shape helpers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hexgeom.h"

namespace hexk {

using bf16raw = uint16_t; // bfloat16 bits

__device__ __forceinline__ float to_f(float v) { return v; }
__device__ __forceinline__ float to_f(bf16raw v)
{
    return __uint_as_float(static_cast<uint32_t>(v) << 16);
}

template <typename T> __device__ __forceinline__ T from_f(float f);
template <> __device__ __forceinline__ float from_f<float>(float f) { return f; }
// float32 -> bfloat16, round to nearest even (gfx950 converts in hardware;
// NaN stays NaN)
template <> __device__ __forceinline__ bf16raw from_f<bf16raw>(float f)
{
    return __builtin_bit_cast(bf16raw, static_cast<__bf16>(f));
}

// Block-uniform reads of one row of weights (row length odd, element m a
// compile-time constant after unrolling), for scalar loads.  float rows are
// read directly.  A bfloat16 element comes from the aligned 32-bit word that
// holds it (there is no 16-bit scalar load; the array must be 4-byte
// aligned, and the ABI requires 16).  The row start passes through an empty
// asm so that the compiler cannot learn its parity: where it could, it split
// the address into a base and an immediate offset that were each 2 mod 4,
// and the scalar load read the wrong word.  With the parity unknown, element
// m is a select between its word for an even and for an odd row start, both
// at word offsets fixed at compile time; with an odd row length both words
// hold an element of the array.
struct WRowF32 {
    const float *p;
    __device__ __forceinline__ WRowF32(const float *w, uint32_t e0) : p(w + e0) {}
    __device__ __forceinline__ float operator()(int m) const { return p[m]; }
};

struct WRowBf16 {
    const uint32_t *wb; // word holding element 0 of the row
    uint32_t odd;       // element 0 is the word's high half
    __device__ __forceinline__ WRowBf16(const bf16raw *w, uint32_t e0)
    {
        asm volatile("" : "+s"(e0));
        wb = reinterpret_cast<const uint32_t *>(w) + (e0 >> 1);
        odd = e0 & 1u;
    }
    __device__ __forceinline__ static uint32_t half(uint32_t v, int hi)
    {
        return hi ? (v & 0xffff0000u) : (v << 16);
    }
    __device__ __forceinline__ float operator()(int m) const
    {
        const uint32_t ev = half(wb[m >> 1], m & 1);
        const uint32_t ov = half(wb[(m + 1) >> 1], (m + 1) & 1);
        return __uint_as_float(odd ? ov : ev);
    }
};

template <typename T> struct WRow;
template <> struct WRow<float> { using type = WRowF32; };
template <> struct WRow<bf16raw> { using type = WRowBf16; };

// Block-uniform reads at compile-time offsets from an even element index e
// (scalar loads; the offset a constant after unrolling).  With e even, a
// bfloat16 element's word and half follow from the offset alone, so no
// select is needed; e passes through an empty asm for the reason given at
// WRowBf16.  Every word read holds an element of the array.
template <typename T> struct WEven;
template <> struct WEven<float> {
    const float *p;
    __device__ __forceinline__ WEven(const float *w, uint32_t e) : p(w + e) {}
    __device__ __forceinline__ float operator()(int off) const { return p[off]; }
};
template <> struct WEven<bf16raw> {
    const uint32_t *wb;
    __device__ __forceinline__ WEven(const bf16raw *w, uint32_t e)
    {
        asm volatile("" : "+s"(e));
        wb = reinterpret_cast<const uint32_t *>(w) + (e >> 1);
    }
    __device__ __forceinline__ float operator()(int off) const
    {
        const uint32_t v = wb[off >> 1];
        return __uint_as_float((off & 1) ? (v & 0xffff0000u) : (v << 16));
    }
};

// Per-block tap table in LDS: column offset, and row offset per centre
// parity, for every tap of a size-k kernel.
struct TapLds {
    int8_t dq[hexgeom::num_taps(8)];
    int8_t ds[hexgeom::num_taps(8)];
    int8_t drow[2][hexgeom::num_taps(8)];
};

__device__ __forceinline__ void fill_taps(TapLds &tl, int k)
{
    const int T = hexgeom::num_taps(k);
    for (int t = threadIdx.x; t < T; t += blockDim.x) {
        int dq = 0, ds = 0;
        hexgeom::tap_axial(k, t, dq, ds);
        tl.dq[t] = static_cast<int8_t>(dq);
        tl.ds[t] = static_cast<int8_t>(ds);
        tl.drow[0][t] = static_cast<int8_t>(hexgeom::tap_drow(dq, ds, 0));
        tl.drow[1][t] = static_cast<int8_t>(hexgeom::tap_drow(dq, ds, 1));
    }
}

} // namespace hexk
