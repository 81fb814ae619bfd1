// hexgeom.h -- hexagonal-grid geometry shared by host code and kernels.
//
// Offset-column addressing of HexagDLy (arXiv:1903.01814, Sec. 2.1): odd
// columns sit half a pitch lower.  A size-k kernel (Sec. 2.2) has 2k+1
// columns; the column at offset dq (-k..k) holds 2k+1-|dq| taps whose axial
// row offsets ds run from max(-k, -k-dq) to min(k, k-dq).  In tensor terms a
// tap (dq, ds) read from a centre in a column of parity p lands on
//     column + dq,   row + ds + floor(dq/2) + p*(dq & 1),
// so the row offset of the odd-dq columns depends on the centre's parity.
// Stride s (Sec. 2.3): output (i, j) is centred on input
//     row s*i + (j & 1) * (s/2),   column s*j.
#pragma once

#ifdef __HIPCC__
#include <hip/hip_runtime.h>
#define HEX_HD __host__ __device__ __forceinline__
#else
#define HEX_HD inline
#endif

namespace hexgeom {

HEX_HD constexpr int num_taps(int k) { return 1 + 3 * k * (k + 1); }

HEX_HD constexpr int iabs(int v) { return v < 0 ? -v : v; }

// floor(a / 2) for any sign (arithmetic shift)
HEX_HD constexpr int floor_half(int a) { return a >> 1; }

// first axial row offset of column dq
HEX_HD constexpr int col_ds_lo(int k, int dq) { return dq < 0 ? -k - dq : -k; }

HEX_HD constexpr int col_len(int k, int dq) { return 2 * k + 1 - iabs(dq); }

// column offset and axial row offset of tap t (canonical order)
HEX_HD constexpr void tap_axial(int k, int t, int &dq, int &ds)
{
    int q = -k;
    int rem = t;
    while (rem >= col_len(k, q)) {
        rem -= col_len(k, q);
        ++q;
    }
    dq = q;
    ds = col_ds_lo(k, q) + rem;
}

// The taps of a size-K kernel as compile-time tables (tap_axial evaluated
// by the compiler; index with constants so the values fold into the code).
template <int K> struct TapTable {
    int dq[num_taps(K)];
    int ds[num_taps(K)];
    constexpr TapTable() : dq(), ds()
    {
        for (int t = 0; t < num_taps(K); ++t)
            tap_axial(K, t, dq[t], ds[t]);
    }
};

// tensor row offset of axial tap (dq, ds) for a centre column of parity p
HEX_HD constexpr int tap_drow(int dq, int ds, int p)
{
    return ds + floor_half(dq) + p * (dq & 1);
}

// index of the tap with the opposite displacement (-dq, -ds)
HEX_HD constexpr int reflect_tap(int k, int t) { return num_taps(k) - 1 - t; }

HEX_HD constexpr int centre_row(int i, int j, int s) { return s * i + (j & 1) * (s >> 1); }
HEX_HD constexpr int centre_col(int j, int s) { return s * j; }

HEX_HD constexpr void out_shape(int H, int W, int s, int &Ho, int &Wo)
{
    Wo = (W - 1) / s + 1;
    int even = (H - 1) / s + 1;
    int odd_span = H - 1 - (s >> 1);
    int odd = odd_span >= 0 ? odd_span / s + 1 : 0;
    Ho = (Wo >= 2 && odd < even) ? odd : even;
}

// floor division by a positive divisor
HEX_HD constexpr int floordiv(int a, int b)
{
    return a >= 0 ? a / b : -((-a + b - 1) / b);
}

// Output whose window reads input (r, c) through tap (dq, ds), if any:
// the centre is (r, c) moved by (-dq, -ds) in axial coordinates, which must
// be a lattice point s*(Q, S) with output (i, j) = (S + floor(Q/2), Q) in
// range.
HEX_HD constexpr bool source_output(int r, int c, int dq, int ds, int s,
                                    int Ho, int Wo, int &i, int &j)
{
    const int cq = c - dq;                     // centre column (= axial q)
    const int cs = r - floor_half(c) - ds;     // centre axial s
    if (cq < 0 || cq % s != 0)
        return false;
    const int Q = cq / s;
    if (Q >= Wo)
        return false;
    if (cs % s != 0)
        return false;
    const int S = floordiv(cs, s);
    const int ii = S + floor_half(Q);
    if (ii < 0 || ii >= Ho)
        return false;
    i = ii;
    j = Q;
    return true;
}

} // namespace hexgeom
