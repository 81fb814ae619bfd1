// kernels.h -- host-side launchers of the HIP kernels (internal).
//
// Every launcher assumes its arguments were validated by the C ABI layer
// (hexconv_abi.cpp): sizes positive, k and stride in range, shapes
// consistent, pointers non-null where required.  Launchers enqueue on the
// given stream and return the launch status.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hexk {

// Optional per-launch timing (hexconv_timing_begin / hexconv_timing_end):
// when enabled, each launch made through HEX_LAUNCH carries a HIP event pair
// that the runtime records at the start and at the end of that kernel's own
// execution (hipExtLaunchKernelGGL), so the dispatch of the launch is not
// counted; otherwise the launch is a plain one and the cost is one relaxed
// atomic load.
struct KTimer {
    explicit KTimer(const char *kernel);
    ~KTimer();
    KTimer(const KTimer &) = delete;
    KTimer &operator=(const KTimer &) = delete;
    bool active() const { return a_ != nullptr; }
    hipEvent_t start() const { return a_; }
    hipEvent_t stop() const { return b_; }

  private:
    const char *name_;
    hipEvent_t a_, b_;
};

// The launchers report hipGetLastError() after their launches; the
// thread's error state is cleared first, so that a status left by an
// earlier runtime call of the caller (or of another library on the same
// thread) is not taken for a failure of this launch.
#define HEX_LAUNCH(kern, grid, block, shm, st, ...)                                          \
    do {                                                                                     \
        (void)hipGetLastError();                                                             \
        ::hexk::KTimer hex_kt_(#kern);                                                       \
        if (hex_kt_.active())                                                                \
            hipExtLaunchKernelGGL(kern, grid, block, shm, st, hex_kt_.start(), hex_kt_.stop(), \
                                  0, __VA_ARGS__);                                           \
        else                                                                                 \
            hipLaunchKernelGGL(kern, grid, block, shm, st, __VA_ARGS__);                     \
    } while (0)

enum Dtype { F32 = 0, BF16 = 1 };

// Sizes of one call.  Three-dimensional calls add D planes along z, a
// window of Z = 2kz+1 planes and a plane stride sz (D_out output planes);
// 2-D calls have D = Do = Z = sz = 1, kz = 0.  Only the generic kernels
// read the depth fields; the specialised kernels are chosen for 2-D calls
// only.
struct ConvShape {
    int N, Ci, Co, H, W, k, s, Ho, Wo, T;
    int D, Do, kz, Z, sz;
};

// Sum weight-gradient partials laid out [e][slot], e = co*(J+1) + col
// (col < J: dw[co][col]; col == J: db[co], skipped when db is null), in a
// fixed order.  J = C_in * T.
hipError_t reduce_partials(const float *part, int nparts, int Co, int J, float *dw, float *db,
                           hipStream_t st);

// Compute units of the current device (queried once per device).
int device_cus();

// Chunked partial-sum layout: element e (e = co * (C_in*T + 1) + col) of
// partial slot `slot` lives at part_index(e, slot, nparts); reduced by
// reduce_chunked.  Workspace: part_chunks(E) * kPartChunk * nparts floats.
constexpr int kPartChunk = 64;
__host__ __device__ inline size_t part_index(int e, int slot, int nparts)
{
    return (static_cast<size_t>(e / kPartChunk) * nparts + slot) * kPartChunk + e % kPartChunk;
}
inline int part_chunks(int E) { return (E + kPartChunk - 1) / kPartChunk; }
hipError_t reduce_chunked(const float *part, int nparts, int Co, int J, float *dw, float *db,
                          hipStream_t st);

// ---- generic kernels: any k, stride, channel count and dtype -----------
// whether the launch plan of the generic forward / data gradient fits the
// LDS of a block (checked by the ABI before anything is enqueued)
bool conv_fwd_generic_ok(const ConvShape &sh);
bool conv_bwd_data_generic_ok(const ConvShape &sh);
hipError_t conv_fwd_generic(const void *x, const void *w, const void *b,
                            void *y, const ConvShape &sh, Dtype dt, bool relu,
                            hipStream_t st);
hipError_t conv_bwd_data_generic(const void *dy, const void *w, void *dx,
                                 const ConvShape &sh, Dtype dt,
                                 hipStream_t st);
size_t wgrad_generic_workspace(const ConvShape &sh);
hipError_t wgrad_generic(const void *x, const void *dy, float *dw, float *db,
                         void *ws, const ConvShape &sh, Dtype dt,
                         hipStream_t st);
// dw (and db if not null) := 0
hipError_t fill_zero_f32(float *dw, float *db, const ConvShape &sh, hipStream_t st);
// argmax: uint8_t per output (am16 false) or uint16_t (am16 true, the 3-D
// entry points), index dz_index * T + t
hipError_t pool_fwd_generic(const void *x, void *y, void *am,
                            const ConvShape &sh, int mode, Dtype dt, bool am16,
                            hipStream_t st);
hipError_t pool_bwd_generic(const void *dy, const void *am,
                            const void *relu_y, void *dx, const ConvShape &sh,
                            int mode, Dtype dt, bool am16, hipStream_t st);

// ---- pooling, k <= 3, stride 1 to 4, rows of whole 16-byte chunks -----
bool pool_fast_ok(const ConvShape &sh, Dtype dt);
hipError_t pool_fwd_fast(const void *x, void *y, uint8_t *am, const ConvShape &sh, int mode,
                         Dtype dt, hipStream_t st);
hipError_t pool_bwd_fast(const void *dy, const uint8_t *am, const void *relu_y, void *dx,
                         const ConvShape &sh, int mode, Dtype dt, hipStream_t st);

// ---- few input channels (C_in*T <= 64), stride 1, fp32 or bf16 data,
// fp32 arithmetic --------------------------------------------------------
bool smallc_fwd_ok(const ConvShape &sh);
hipError_t smallc_fwd(const void *x, const void *w, const void *b, void *y, const ConvShape &sh,
                      Dtype d, bool relu, hipStream_t st);
bool smallc_bwd_data_ok(const ConvShape &sh);
hipError_t smallc_bwd_data(const void *dy, const void *w, void *dx, const ConvShape &sh, Dtype d,
                           hipStream_t st);
// Data gradient of a 3-D layer with 1 or 2 input channels, float32 or
// bfloat16, plane and in-plane stride 1, k <= 2, kz <= 2, W % 4 == 0
// (k_bwd3d.hip).
bool smallc3d_bwd_data_ok(const ConvShape &sh);
hipError_t smallc3d_bwd_data(const void *dy, const void *w, void *dx, const ConvShape &sh,
                             Dtype d, hipStream_t st);
bool smallc_wgrad_ok(const ConvShape &sh);
size_t smallc_wgrad_workspace(const ConvShape &sh);
hipError_t smallc_wgrad(const void *x, const void *dy, float *dw, float *db, void *ws,
                        const ConvShape &sh, Dtype d, hipStream_t st);
// both gradients in one pass over dy (C_in <= 2, C_out <= 32), fp32 or bf16
bool smallc_bwd_fused_ok(const ConvShape &sh, Dtype d);
size_t smallc_bwd_fused_workspace(const ConvShape &sh);
hipError_t smallc_bwd_fused(const void *x, const void *dy, const void *w, void *dx, float *dw,
                            float *db, void *ws, const ConvShape &sh, Dtype d, hipStream_t st);

// ---- bf16 matrix-core convolution, input channels a multiple of 32 -----
// forward (reflect = false: IC = C_in, OC = C_out) or stride-1 data
// gradient (reflect = true: IC = C_out, OC = C_in)
bool bf16_wide_ok(const ConvShape &sh, int IC, int OC);
hipError_t bf16_wide_conv(const void *in, const void *w, const void *bias, void *out,
                          const ConvShape &sh, bool reflect, bool relu, hipStream_t st);

// ---- bf16 matrix-core convolution at any stride, k <= 3 ------------------
// forward: C_in % 32 == 0, W % 8 == 0, W_out <= 256; data gradient (the
// transposed lattice gather): C_out % 32 == 0, W and W_out % 8 == 0,
// W <= 256, H a multiple of the stride
bool bf16_gen_fwd_ok(const ConvShape &sh);
hipError_t bf16_gen_fwd(const void *x, const void *w, const void *bias, void *y,
                        const ConvShape &sh, bool relu, hipStream_t st);
bool bf16_gen_dgrad_ok(const ConvShape &sh);
hipError_t bf16_gen_dgrad(const void *dy, const void *w, void *dx, const ConvShape &sh,
                          hipStream_t st);

// ---- bf16 32x32 matrix-core weight gradient (C_in, C_out multiples of 32) --
// output-channel passes the kernel needs for this shape (0: not supported)
int bf16_wgrad32_passes(const ConvShape &sh);
size_t bf16_wgrad32_workspace(const ConvShape &sh);
hipError_t bf16_wgrad32(const void *x, const void *dy, float *dw, float *db, void *ws,
                        const ConvShape &sh, hipStream_t st);

// ---- bf16 matrix-core weight gradient (k <= 3, W and W_out % 8 == 0) ---
bool bf16_wgrad_ok(const ConvShape &sh);
size_t bf16_wgrad_workspace(const ConvShape &sh);
hipError_t bf16_wgrad(const void *x, const void *dy, float *dw, float *db, void *ws,
                      const ConvShape &sh, hipStream_t st);

} // namespace hexk
