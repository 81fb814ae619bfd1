// Drives the library's host geometry (csrc/hexgeom.h: tap tables, output
// shape, source-output lattice test) and the generic kernels' launch plans
// (csrc/generic_plan.h) over every kernel size and stride the ABI accepts,
// for a build with AddressSanitizer and UndefinedBehaviorSanitizer.  It also
// checks two properties on the way: every tap lies within k columns and k
// rows, and each (input element, tap) pair with a source output is read by
// that output's window.
#include <cstdio>
#include <cstdlib>
#include <initializer_list>

#include "generic_plan.h"
#include "hexgeom.h"

int main()
{
    using namespace hexgeom;
    for (int k = 0; k <= 8; ++k) {
        const int T = num_taps(k);
        for (int t = 0; t < T; ++t) {
            int dq = 0, ds = 0;
            tap_axial(k, t, dq, ds);
            for (int p = 0; p < 2; ++p) {
                const int dr = tap_drow(dq, ds, p);
                if (dq < -k || dq > k || dr < -k || dr > k) {
                    std::fprintf(stderr, "tap out of range k=%d t=%d\n", k, t);
                    return 1;
                }
            }
        }
        for (int s = 1; s <= 8; ++s) {
            for (int H = 1; H <= 19; H += 3)
                for (int W = 1; W <= 19; W += 2) {
                    int Ho = 0, Wo = 0;
                    out_shape(H, W, s, Ho, Wo);
                    // every output's window reads the element its tap points at
                    for (int r = 0; r < H; ++r)
                        for (int c = 0; c < W; ++c)
                            for (int t = 0; t < T; ++t) {
                                int dq = 0, ds = 0, i = 0, j = 0;
                                tap_axial(k, t, dq, ds);
                                if (!source_output(r, c, dq, ds, s, Ho, Wo, i, j))
                                    continue;
                                const int rc = centre_row(i, j, s), cc = centre_col(j, s);
                                if (rc + tap_drow(dq, ds, cc & 1) != r || cc + dq != c) {
                                    std::fprintf(stderr, "lattice mismatch\n");
                                    return 1;
                                }
                            }
                }
            for (int C : {1, 8, 31, 32, 64, 65, 512}) {
                if (!hexk::plan::plan_fwd(C, C, k, s).ok || !hexk::plan::plan_bwd_data(C, C, k).ok) {
                    std::fprintf(stderr, "plan does not fit k=%d s=%d C=%d\n", k, s, C);
                    return 1;
                }
            }
        }
    }
    std::printf("geometry sanitized run ok\n");
    return 0;
}
