// k_reduce.hip -- deterministic reduction of weight-gradient partial sums.
//
// The weight-gradient kernels leave one partial sum per (output element,
// partial slot) in the workspace, with e = co * (C_in*T + 1) + col:
// col < C_in*T is dw[co][col], col == C_in*T is db[co].  Two layouts:
//  - [e][slot] (reduce_partials): one wave per element sums its slots;
//  - chunked, part_index() in kernels.h (reduce_chunked): chunks of 64
//    elements, each slot's 64 values contiguous, so a block writing its
//    partials and the reduction reading them both touch whole lines.
// Either way the slots are summed in a fixed order (strided per thread,
// then a fixed tree), so results do not depend on timing.
#include "hexdev.h"
#include "kernels.h"

namespace hexk {
namespace {

// [e][slot] layout: one wave per element; each lane sums a strided subset of
// the slots (four interleaved accumulators), then a butterfly over the wave.
__global__ __launch_bounds__(64) void reduce_partials_k(const float *__restrict__ part, int nparts,
                                                       int J, float *__restrict__ dw,
                                                       float *__restrict__ db)
{
    const int e = blockIdx.x;
    const int lane = threadIdx.x;
    const float *src = part + static_cast<size_t>(e) * nparts;
    float s[4] = {0.f, 0.f, 0.f, 0.f};
    int p = lane;
    for (; p + 192 < nparts; p += 256) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
            s[u] += src[p + 64 * u];
    }
    for (; p < nparts; p += 64)
        s[0] += src[p];
    float v = (s[0] + s[1]) + (s[2] + s[3]);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        v += __shfl_xor(v, off, 64);
    if (lane == 0) {
        const int Jt = J + 1;
        const int co = e / Jt, col = e % Jt;
        if (col < J)
            dw[static_cast<size_t>(co) * J + col] = v;
        else if (db != nullptr)
            db[co] = v;
    }
}

constexpr int kRedSlices = 16; // slot slices per chunk block (1024 threads)
constexpr int kRedBatch = 16;  // slots per thread whose loads are in flight together

// Chunked layout: one block per chunk of 64 elements; thread (slice sl,
// element el) adds slots sl, sl + 16, sl + 32, ... of its element, issuing
// the loads of 16 slots before adding any (one memory latency per 256
// slots), then the 16 slices are added by a fixed tree.  The order of the
// additions depends only on nparts, so results are reproducible.
__global__ __launch_bounds__(kPartChunk * kRedSlices) void reduce_chunked_k(
    const float *__restrict__ part, int nparts, int E, int J, float *__restrict__ dw,
    float *__restrict__ db)
{
    __shared__ float red[kRedSlices][kPartChunk];
    const int chunk = blockIdx.x;
    const int el = threadIdx.x % kPartChunk, sl = threadIdx.x / kPartChunk;
    const float *src = part + static_cast<size_t>(chunk) * nparts * kPartChunk + el;
    float acc = 0.f;
    for (int p0 = 0; p0 < nparts; p0 += kRedSlices * kRedBatch) {
        float v[kRedBatch];
#pragma unroll
        for (int u = 0; u < kRedBatch; ++u) {
            const int p = p0 + sl + u * kRedSlices;
            v[u] = p < nparts ? src[static_cast<size_t>(p) * kPartChunk] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kRedBatch; ++u)
            acc += v[u];
    }
    red[sl][el] = acc;
    for (int half = kRedSlices / 2; half > 0; half >>= 1) {
        __syncthreads();
        if (sl < half)
            red[sl][el] += red[sl + half][el];
    }
    if (sl == 0) {
        const int e = chunk * kPartChunk + el;
        if (e < E) {
            const int Jt = J + 1, co = e / Jt, col = e - co * Jt;
            if (col < J)
                dw[static_cast<size_t>(co) * J + col] = red[0][el];
            else if (db != nullptr)
                db[co] = red[0][el];
        }
    }
}

} // namespace

hipError_t reduce_chunked(const float *part, int nparts, int Co, int J, float *dw, float *db,
                          hipStream_t st)
{
    const int E = Co * (J + 1);
    HEX_LAUNCH(reduce_chunked_k, dim3((E + kPartChunk - 1) / kPartChunk),
                       dim3(kPartChunk * kRedSlices), 0, st, part, nparts, E, J, dw, db);
    return hipGetLastError();
}

hipError_t reduce_partials(const float *part, int nparts, int Co, int J, float *dw, float *db,
                           hipStream_t st)
{
    const int E = Co * (J + 1);
    HEX_LAUNCH(reduce_partials_k, dim3(E), dim3(64), 0, st, part, nparts, J, dw, db);
    return hipGetLastError();
}

} // namespace hexk
