// k_reduce.hip -- deterministic reduction of weight-gradient partial sums.
//
// The weight-gradient kernels leave one partial sum per (output element,
// partial slot) in the workspace, laid out [e][slot] with
// e = co * (C_in*T + 1) + col: col < C_in*T is dw[co][col], col == C_in*T is
// db[co].  One block per element sums its slots in a fixed order (strided
// per thread, then a fixed LDS tree), so results do not depend on timing.
#include "hexdev.h"
#include "kernels.h"

namespace hexk {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void reduce_partials_k(
    const float *__restrict__ part, int nparts, int J, float *__restrict__ dw,
    float *__restrict__ db)
{
    __shared__ float red[kThreads];
    const int e = blockIdx.x;
    const float *src = part + static_cast<size_t>(e) * nparts;
    float s = 0.f;
    for (int p = threadIdx.x; p < nparts; p += kThreads)
        s += src[p];
    red[threadIdx.x] = s;
    for (int half = kThreads / 2; half > 0; half >>= 1) {
        __syncthreads();
        if (threadIdx.x < half)
            red[threadIdx.x] += red[threadIdx.x + half];
    }
    if (threadIdx.x == 0) {
        const int Jt = J + 1;
        const int co = e / Jt, col = e % Jt;
        if (col < J)
            dw[static_cast<size_t>(co) * J + col] = red[0];
        else if (db != nullptr)
            db[co] = red[0];
    }
}

} // namespace

hipError_t reduce_partials(const float *part, int nparts, int Co, int J, float *dw, float *db,
                           hipStream_t st)
{
    const int E = Co * (J + 1);
    hipLaunchKernelGGL(reduce_partials_k, dim3(E), dim3(kThreads), 0, st, part, nparts, J, dw,
                       db);
    return hipGetLastError();
}

} // namespace hexk
