// plan_query.cpp -- exposes the generic kernels' launch plans
// (paper_1903_01814_amd/csrc/generic_plan.h, host arithmetic only) to the
// CPU tests through a C interface.  Built with g++ by the tests.
#include "generic_plan.h"

extern "C" {

// out: ok, TI, TJ, cb, G, lds
void plan_fwd_query(int Ci, int Co, int k, int s, long limit, long *out)
{
    const hexk::plan::FwdPlan p = hexk::plan::plan_fwd(Ci, Co, k, s, static_cast<size_t>(limit));
    out[0] = p.ok;
    out[1] = p.TI;
    out[2] = p.TJ;
    out[3] = p.cb;
    out[4] = p.G;
    out[5] = static_cast<long>(p.lds);
}

// out: ok, cb, CC, lds
void plan_bwd_data_query(int Ci, int Co, int k, long limit, long *out)
{
    const hexk::plan::BwdDataPlan p = hexk::plan::plan_bwd_data(Ci, Co, k, static_cast<size_t>(limit));
    out[0] = p.ok;
    out[1] = p.cb;
    out[2] = p.CC;
    out[3] = static_cast<long>(p.lds);
}

long plan_lds_limit(void) { return static_cast<long>(hexk::plan::kGenericLdsLimit); }
}
