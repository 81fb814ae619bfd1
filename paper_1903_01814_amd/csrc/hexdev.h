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
