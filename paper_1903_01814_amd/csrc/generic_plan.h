// generic_plan.h -- launch plans of the generic convolution kernels
// (k_generic.hip): tile shape, channels per block and LDS bytes per block.
//
// Host arithmetic only (it also compiles with a plain C++ compiler, so the
// plans can be checked without a GPU).  A plan either fits the LDS a
// generic block may use (kGenericLdsLimit) or says it does not; the C ABI
// turns the latter into HEX_ERR_UNSUPPORTED before anything is enqueued.
#pragma once

#include <stddef.h>

#include "hexgeom.h"

namespace hexk {
namespace plan {

constexpr size_t kGenericLdsLimit = 64 * 1024; // LDS per generic block
constexpr size_t kGenericStageLds = 40 * 1024; // several channels per stage up to this
constexpr size_t kWeightLds = 32 * 1024;       // staged float weights of one channel
constexpr int kThreads = 256;                  // threads per generic block

// Input region read by a TI x TJ tile of outputs: rows s(TI-1) + floor(s/2)
// + 2k + 1 (the odd output columns sit floor(s/2) rows lower), columns
// s(TJ-1) + 2k + 1.
HEX_HD constexpr int region_rows(int TI, int k, int s) { return s * (TI - 1) + (s >> 1) + 2 * k + 1; }
HEX_HD constexpr int region_cols(int TJ, int k, int s) { return s * (TJ - 1) + 2 * k + 1; }
// floats of one staged region, rounded up to 16 bytes
HEX_HD constexpr int region_floats(int TI, int TJ, int k, int s)
{
    return (region_rows(TI, k, s) * region_cols(TJ, k, s) + 3) & ~3;
}

// Channels per block (output channels in the forward, input channels in
// the data gradient) for a layer of C such channels and T taps: 64, 32 or
// 8, the largest whose float weights per staged channel stay within
// kWeightLds (every staged input element, or loaded dy element, feeds that
// many accumulators).
inline int chan_block(int C, int T)
{
    if (C >= 64 && sizeof(float) * static_cast<size_t>(T) * 64 <= kWeightLds)
        return 64;
    if (C >= 32 && sizeof(float) * static_cast<size_t>(T) * 32 <= kWeightLds)
        return 32;
    return 8;
}

struct FwdPlan {
    bool ok;
    int TI, TJ; // output tile per block (TI * TJ <= kThreads)
    int cb;     // output channels per block
    int G;      // input channels staged per pair of barriers
    size_t lds; // dynamic LDS bytes per block
};

// Forward: the first tile (largest first) whose region plus the block's
// weights of one input channel fit in `limit`; then as many input channels
// per stage as fit in kGenericStageLds (at most 8).
inline FwdPlan plan_fwd(int Ci, int Co, int k, int s, size_t limit = kGenericLdsLimit)
{
    static const int cand[][2] = {{8, 32}, {16, 16}, {4, 64}, {8, 16}, {4, 32},
                                  {4, 16}, {2, 16}, {1, 16}, {1, 8}};
    FwdPlan p{false, 0, 0, 0, 0, 0};
    const int T = hexgeom::num_taps(k);
    p.cb = chan_block(Co, T);
    const size_t wbytes = sizeof(float) * static_cast<size_t>(T) * p.cb;
    for (const auto &c : cand) {
        const size_t per_ch = sizeof(float) * static_cast<size_t>(region_floats(c[0], c[1], k, s)) + wbytes;
        if (per_ch > limit)
            continue;
        p.TI = c[0];
        p.TJ = c[1];
        size_t G = kGenericStageLds / per_ch;
        if (G > 8)
            G = 8;
        if (G > static_cast<size_t>(Ci))
            G = static_cast<size_t>(Ci);
        if (G < 1)
            G = 1;
        p.G = static_cast<int>(G);
        p.lds = per_ch * G;
        p.ok = p.lds <= limit;
        return p;
    }
    return p;
}

struct BwdDataPlan {
    bool ok;
    int cb;     // input channels per block
    int CC;     // output channels whose weights are staged per pass
    size_t lds; // dynamic LDS bytes per block
};

// Data gradient: the weights of CC output channels for the block's cb input
// channels per stage, CC as large as kGenericStageLds allows.
inline BwdDataPlan plan_bwd_data(int Ci, int Co, int k, size_t limit = kGenericLdsLimit)
{
    BwdDataPlan p{false, 0, 0, 0};
    const int T = hexgeom::num_taps(k);
    p.cb = chan_block(Ci, T);
    const size_t per_co = sizeof(float) * static_cast<size_t>(T) * p.cb;
    size_t CC = kGenericStageLds / per_co;
    if (CC > static_cast<size_t>(Co))
        CC = static_cast<size_t>(Co);
    if (CC < 1)
        CC = 1;
    p.CC = static_cast<int>(CC);
    p.lds = per_co * CC;
    p.ok = p.lds <= limit;
    return p;
}

} // namespace plan
} // namespace hexk
