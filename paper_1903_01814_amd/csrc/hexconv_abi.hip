// hexconv_abi.hip -- the extern "C" entry points declared in hexconv.h:
// argument validation (host only, before anything is enqueued), choice of
// kernel per shape regime, and launch-status mapping.
#include <atomic>
#include <mutex>
#include <stdint.h>
#include <string>
#include <vector>
#include <stdlib.h>
#include <string.h>

#include "../../include/hexconv.h"
#include "hexgeom.h"
#include "kernels.h"

namespace hexk {

int device_cus()
{
    constexpr int kMaxDev = 64;
    static std::atomic<int> cache[kMaxDev];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0)
        return 256;
    if (dev < kMaxDev) {
        const int c = cache[dev].load(std::memory_order_relaxed);
        if (c > 0)
            return c;
    }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        cus = 256;
    if (dev < kMaxDev)
        cache[dev].store(cus, std::memory_order_relaxed);
    return cus;
}

// ---- per-launch timing --------------------------------------------------

namespace {

std::atomic<bool> g_timing{false};
std::mutex g_timing_mu;

struct TimedLaunch {
    std::string name;
    hipEvent_t a, b;
};
std::vector<TimedLaunch> g_timed;

// "(name<args>)" or "name<args>" -> "name"
std::string kernel_base_name(const char *s)
{
    std::string n;
    for (; *s == '(' || *s == ' '; ++s) {
    }
    for (; *s != '\0' && *s != '<' && *s != '(' && *s != ')' && *s != ' ' && *s != ','; ++s)
        n.push_back(*s);
    return n;
}

} // namespace

KTimer::KTimer(const char *kernel) : name_(kernel), a_(nullptr), b_(nullptr)
{
    if (!g_timing.load(std::memory_order_relaxed))
        return;
    if (hipEventCreate(&a_) != hipSuccess) {
        a_ = nullptr;
        return;
    }
    if (hipEventCreate(&b_) != hipSuccess) {
        (void)hipEventDestroy(a_);
        a_ = nullptr;
        return;
    }
    // the launch itself records the pair (see HEX_LAUNCH)
}

KTimer::~KTimer()
{
    if (a_ == nullptr)
        return;
    std::lock_guard<std::mutex> lock(g_timing_mu);
    g_timed.push_back(TimedLaunch{kernel_base_name(name_), a_, b_});
}

} // namespace hexk

namespace {

using hexk::ConvShape;
using hexk::Dtype;

constexpr long kMaxElems = (1L << 31) - 1; // per tensor, int32-indexable planes

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool dtype_ok(int dt) { return dt == HEX_F32 || dt == HEX_BF16; }

size_t dtype_bytes(int dt) { return dt == HEX_F32 ? 4 : 2; }

// Shape checks shared by every op.  Fills `sh`.  C_in/C_out both = C for pools.
int check_shape(int N, int Ci, int Co, int H, int W, int k, int stride, int dt, ConvShape &sh)
{
    if (N < 0 || Ci < 1 || Co < 1 || H < 1 || W < 1)
        return HEX_ERR_INVALID_ARG;
    if (k < 0 || k > HEX_MAX_K || stride < 1 || stride > HEX_MAX_STRIDE)
        return HEX_ERR_INVALID_ARG;
    if (!dtype_ok(dt))
        return HEX_ERR_INVALID_ARG;
    if (H > 65535 || W > 65535 || N > 65535 || Ci > 65535 || Co > 65535)
        return HEX_ERR_UNSUPPORTED;
    const long hw = static_cast<long>(H) * W;
    if (hw * N > kMaxElems / Ci || hw * N > kMaxElems / Co)
        return HEX_ERR_UNSUPPORTED;
    if (static_cast<long>(Co) * Ci * hexgeom::num_taps(k) > kMaxElems)
        return HEX_ERR_UNSUPPORTED;
    sh.N = N;
    sh.Ci = Ci;
    sh.Co = Co;
    sh.H = H;
    sh.W = W;
    sh.k = k;
    sh.s = stride;
    sh.T = hexgeom::num_taps(k);
    hexgeom::out_shape(H, W, stride, sh.Ho, sh.Wo);
    sh.D = sh.Do = sh.Z = sh.sz = 1;
    sh.kz = 0;
    return HEX_OK;
}

// Shape checks of the three-dimensional entry points: the 2-D checks of the
// plane, then the planes (D), the window depth (kz) and the plane stride.
int check_shape3d(int N, int Ci, int Co, int D, int H, int W, int k, int kz, int stride,
                  int stride_z, int dt, ConvShape &sh)
{
    if (D < 1 || kz < 0 || kz > HEX_MAX_KZ || stride_z < 1 || stride_z > HEX_MAX_STRIDE)
        return HEX_ERR_INVALID_ARG;
    int rc = check_shape(N, Ci, Co, H, W, k, stride, dt, sh);
    if (rc != HEX_OK)
        return rc;
    if (D > 65535)
        return HEX_ERR_UNSUPPORTED;
    const long dhw = static_cast<long>(D) * H * W;
    if (dhw * N > kMaxElems / Ci || dhw * N > kMaxElems / Co)
        return HEX_ERR_UNSUPPORTED;
    if (static_cast<long>(Co) * Ci * (2 * kz + 1) * sh.T > kMaxElems)
        return HEX_ERR_UNSUPPORTED;
    sh.D = D;
    sh.kz = kz;
    sh.Z = 2 * kz + 1;
    sh.sz = stride_z;
    sh.Do = (D - 1) / stride_z + 1;
    return HEX_OK;
}

int ptrs_ok(std::initializer_list<const void *> required, std::initializer_list<const void *> optional)
{
    for (const void *p : required)
        if (p == nullptr || !aligned16(p))
            return HEX_ERR_INVALID_ARG;
    for (const void *p : optional)
        if (p != nullptr && !aligned16(p))
            return HEX_ERR_INVALID_ARG;
    return HEX_OK;
}

// HIP status of the last failed launch on this thread (hex_last_launch_error)
thread_local hipError_t g_last_launch_error = hipSuccess;

int launched(hipError_t e)
{
    if (e == hipSuccess)
        return HEX_OK;
    g_last_launch_error = e;
    return HEX_ERR_LAUNCH;
}

// HEXCONV_PATH=generic forces the generic kernels (used by tests to compare
// the specialised kernels against them).
bool force_generic()
{
    const char *v = getenv("HEXCONV_PATH");
    return v != nullptr && strcmp(v, "generic") == 0;
}

// Weight-gradient kernel family for a shape; the workspace query and the
// call must agree, so both go through this choice.
enum class WgradPath { Generic, Fused, Small, Bf16Mfma32, Bf16Mfma };

WgradPath wgrad_path(const ConvShape &sh, Dtype d)
{
    if (force_generic())
        return WgradPath::Generic;
    // where the fused backward applies, it is also the fastest weight
    // gradient with its data-gradient waves off (fp32 1 -> 16 channels, 40x40,
    // k = 2: 18 -> 13 us; bf16 1 -> 32 channels, 48x48, N = 512: 69 -> 59 us
    // at k = 2, 66 -> 38 us at k = 1)
    if (hexk::smallc_bwd_fused_ok(sh, d))
        return WgradPath::Fused;
    const bool small = hexk::smallc_wgrad_ok(sh);
    if (d == hexk::F32)
        return small ? WgradPath::Small : WgradPath::Generic;
    // bf16 with few input channels: the small-channel kernel stages x once
    // per 16 output channels, so it wins only for one such block at k <= 2
    // (1 -> 16 channels, 40x40, N = 256: 27 -> 18 us at k = 1, 26 -> 23 us
    // at k = 2; 32 or 64 output channels and k = 3 favour the bf16 kernels)
    if (small && sh.Co <= 16 && sh.k <= 2)
        return WgradPath::Small;
    // several passes re-read x once per pass: then the single-pass kernel,
    // where it applies, is the faster one
    const int passes = hexk::bf16_wgrad32_passes(sh);
    if (passes == 1 || (passes > 1 && !hexk::bf16_wgrad_ok(sh)))
        return WgradPath::Bf16Mfma32;
    if (hexk::bf16_wgrad_ok(sh))
        return WgradPath::Bf16Mfma;
    return small ? WgradPath::Small : WgradPath::Generic;
}

// Fused data + weight gradient (hexconv_bwd) for this shape?
bool bwd_fused(const ConvShape &sh, Dtype d)
{
    return !force_generic() && hexk::smallc_bwd_fused_ok(sh, d);
}

size_t wgrad_workspace(const ConvShape &sh, Dtype d)
{
    switch (wgrad_path(sh, d)) {
    case WgradPath::Fused:
        return hexk::smallc_bwd_fused_workspace(sh);
    case WgradPath::Small:
        return hexk::smallc_wgrad_workspace(sh);
    case WgradPath::Bf16Mfma32:
        return hexk::bf16_wgrad32_workspace(sh);
    case WgradPath::Bf16Mfma:
        return hexk::bf16_wgrad_workspace(sh);
    default:
        return hexk::wgrad_generic_workspace(sh);
    }
}

// Every check of hexconv_bwd's arguments but the workspace, so that a bad
// argument enqueues nothing; `need` receives the workspace bytes.
int bwd_check(const void *x, const void *dy, const void *w, const void *dx, const float *dw,
              const float *db, int N, int Ci, int Co, int H, int W, int k, int stride, int dt,
              ConvShape &sh, size_t &need)
{
    int rc = check_shape(N, Ci, Co, H, W, k, stride, dt, sh);
    if (rc != HEX_OK)
        return rc;
    if ((rc = ptrs_ok({dw}, {x, dy, w, dx, db})) != HEX_OK)
        return rc;
    const bool empty = (N == 0 || sh.Ho == 0);
    if (!empty && (x == nullptr || dy == nullptr))
        return HEX_ERR_INVALID_ARG;
    if (dx != nullptr && w == nullptr)
        return HEX_ERR_INVALID_ARG;
    const Dtype d = static_cast<Dtype>(dt);
    need = empty ? 0
                 : (bwd_fused(sh, d) ? hexk::smallc_bwd_fused_workspace(sh) : wgrad_workspace(sh, d));
    return HEX_OK;
}

} // namespace

// Scratch memory of hexconv_bwd_noalloc: one copy of this array per GPU,
// held until the process ends, shared by every such call on that GPU.  On
// the host the name only stands for the symbol: host code uses the device
// address of the current GPU's copy, obtained once per device by
// scratch_ptr(), never the name itself.
static __device__ __align__(256) unsigned char scratch[HEX_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_dev[kMaxScratchDevices];

// Device address of the current GPU's scratch array (looked up on the
// first call on each device), or nullptr if it cannot be obtained.
void *scratch_ptr()
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxScratchDevices)
        return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_dev[dev] == nullptr) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
            return nullptr;
        g_scratch_dev[dev] = p;
    }
    return g_scratch_dev[dev];
}

} // namespace

extern "C" {

int hex_num_taps(int k)
{
    if (k < 0 || k > HEX_MAX_K)
        return HEX_ERR_INVALID_ARG;
    return hexgeom::num_taps(k);
}

int hex_out_shape(int H, int W, int k, int stride, int *H_out, int *W_out)
{
    if (H < 1 || W < 1 || k < 0 || k > HEX_MAX_K || stride < 1 || stride > HEX_MAX_STRIDE ||
        H_out == nullptr || W_out == nullptr)
        return HEX_ERR_INVALID_ARG;
    int ho = 0, wo = 0;
    hexgeom::out_shape(H, W, stride, ho, wo);
    *H_out = ho;
    *W_out = wo;
    return HEX_OK;
}

int hex_tap_table(int k, int parity, int *dcol, int *drow)
{
    if (k < 0 || k > HEX_MAX_K || (parity != 0 && parity != 1) || dcol == nullptr ||
        drow == nullptr)
        return HEX_ERR_INVALID_ARG;
    const int T = hexgeom::num_taps(k);
    for (int t = 0; t < T; ++t) {
        int dq = 0, ds = 0;
        hexgeom::tap_axial(k, t, dq, ds);
        dcol[t] = dq;
        drow[t] = hexgeom::tap_drow(dq, ds, parity);
    }
    return HEX_OK;
}

int hexconv_fwd(const void *x, const void *w, const void *bias, void *y, int N, int C_in,
                int C_out, int H, int W, int k, int stride, hex_dtype dt, int flags, void *stream)
{
    ConvShape sh;
    int rc = check_shape(N, C_in, C_out, H, W, k, stride, dt, sh);
    if (rc != HEX_OK)
        return rc;
    if ((flags & ~HEX_FLAG_RELU) != 0)
        return HEX_ERR_INVALID_ARG;
    if (N == 0)
        return HEX_OK; // empty batch: buffers may be NULL
    if ((rc = ptrs_ok({x, w, y}, {bias})) != HEX_OK)
        return rc;
    if (sh.Ho == 0)
        return HEX_OK;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const bool relu = (flags & HEX_FLAG_RELU) != 0;
    const Dtype d = static_cast<Dtype>(dt);
    if (!force_generic()) {
        if (hexk::smallc_fwd_ok(sh))
            return launched(hexk::smallc_fwd(x, w, bias, y, sh, d, relu, st));
        if (d == hexk::BF16 && hexk::bf16_wide_ok(sh, sh.Ci, sh.Co))
            return launched(hexk::bf16_wide_conv(x, w, bias, y, sh, false, relu, st));
        if (d == hexk::BF16 && hexk::bf16_gen_fwd_ok(sh))
            return launched(hexk::bf16_gen_fwd(x, w, bias, y, sh, relu, st));
    }
    if (!hexk::conv_fwd_generic_ok(sh))
        return HEX_ERR_UNSUPPORTED;
    return launched(hexk::conv_fwd_generic(x, w, bias, y, sh, d, relu, st));
}

int hexconv_bwd_data(const void *dy, const void *w, void *dx, int N, int C_in, int C_out, int H,
                     int W, int k, int stride, hex_dtype dt, void *stream)
{
    ConvShape sh;
    int rc = check_shape(N, C_in, C_out, H, W, k, stride, dt, sh);
    if (rc != HEX_OK)
        return rc;
    if (N == 0)
        return HEX_OK; // empty batch: buffers may be NULL
    if ((rc = ptrs_ok({w, dx}, {dy})) != HEX_OK)
        return rc;
    if (dy == nullptr && sh.Ho > 0)
        return HEX_ERR_INVALID_ARG;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const Dtype d = static_cast<Dtype>(dt);
    if (!force_generic() && sh.Ho > 0) {
        // bf16 with 32 or more output channels: the matrix-core kernel
        // before the small-channel one (1 -> 64 channels, 48x48, k = 2:
        // 29 against 59 us)
        if (d == hexk::BF16 && hexk::bf16_wide_ok(sh, sh.Co, sh.Ci))
            return launched(hexk::bf16_wide_conv(dy, w, nullptr, dx, sh, true, false, st));
        if (hexk::smallc_bwd_data_ok(sh))
            return launched(hexk::smallc_bwd_data(dy, w, dx, sh, d, st));
        if (d == hexk::BF16 && hexk::bf16_gen_dgrad_ok(sh))
            return launched(hexk::bf16_gen_dgrad(dy, w, dx, sh, st));
    }
    if (!hexk::conv_bwd_data_generic_ok(sh))
        return HEX_ERR_UNSUPPORTED;
    return launched(hexk::conv_bwd_data_generic(dy, w, dx, sh, d, st));
}

size_t hexconv_bwd_weight_workspace(int N, int C_in, int C_out, int H, int W, int k, int stride,
                                    hex_dtype dt)
{
    ConvShape sh;
    if (check_shape(N, C_in, C_out, H, W, k, stride, dt, sh) != HEX_OK)
        return 0;
    if (N == 0 || sh.Ho == 0)
        return 0;
    return wgrad_workspace(sh, static_cast<Dtype>(dt));
}

int hexconv_bwd_weight(const void *x, const void *dy, float *dw, float *db, void *ws,
                       size_t ws_bytes, int N, int C_in, int C_out, int H, int W, int k,
                       int stride, hex_dtype dt, void *stream)
{
    ConvShape sh;
    int rc = check_shape(N, C_in, C_out, H, W, k, stride, dt, sh);
    if (rc != HEX_OK)
        return rc;
    if ((rc = ptrs_ok({dw}, {x, dy, db, ws})) != HEX_OK)
        return rc;
    const bool empty = (N == 0 || sh.Ho == 0);
    if (!empty && (x == nullptr || dy == nullptr))
        return HEX_ERR_INVALID_ARG;
    const Dtype d = static_cast<Dtype>(dt);
    const size_t need = empty ? 0 : wgrad_workspace(sh, d);
    if (need > 0 && (ws == nullptr || ws_bytes < need))
        return HEX_ERR_INVALID_ARG;
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (empty)
        return launched(hexk::fill_zero_f32(dw, db, sh, st));
    switch (wgrad_path(sh, d)) {
    case WgradPath::Fused: // no data gradient: w is not read
        return launched(hexk::smallc_bwd_fused(x, dy, nullptr, nullptr, dw, db, ws, sh, d, st));
    case WgradPath::Small:
        return launched(hexk::smallc_wgrad(x, dy, dw, db, ws, sh, d, st));
    case WgradPath::Bf16Mfma32:
        return launched(hexk::bf16_wgrad32(x, dy, dw, db, ws, sh, st));
    case WgradPath::Bf16Mfma:
        return launched(hexk::bf16_wgrad(x, dy, dw, db, ws, sh, st));
    default:
        return launched(hexk::wgrad_generic(x, dy, dw, db, ws, sh, d, st));
    }
}

size_t hexconv_bwd_workspace(int N, int C_in, int C_out, int H, int W, int k, int stride,
                             hex_dtype dt)
{
    ConvShape sh;
    if (check_shape(N, C_in, C_out, H, W, k, stride, dt, sh) != HEX_OK)
        return 0;
    if (N == 0 || sh.Ho == 0)
        return 0;
    const Dtype d = static_cast<Dtype>(dt);
    return bwd_fused(sh, d) ? hexk::smallc_bwd_fused_workspace(sh) : wgrad_workspace(sh, d);
}

// hexconv_bwd after its checks: ws holds at least the workspace the shape
// needs (ws_bytes of it).
static int bwd_run(const void *x, const void *dy, const void *w, void *dx, float *dw, float *db,
                   void *ws, size_t ws_bytes, const ConvShape &sh, hex_dtype dt, void *stream)
{
    hipStream_t st = static_cast<hipStream_t>(stream);
    const Dtype d = static_cast<Dtype>(dt);
    const bool empty = (sh.N == 0 || sh.Ho == 0);
    if (!empty && bwd_fused(sh, d))
        return launched(hexk::smallc_bwd_fused(x, dy, w, dx, dw, db, ws, sh, d, st));
    if (dx != nullptr && sh.N > 0) {
        const int rc = hexconv_bwd_data(dy, w, dx, sh.N, sh.Ci, sh.Co, sh.H, sh.W, sh.k, sh.s, dt,
                                        stream);
        if (rc != HEX_OK)
            return rc;
    }
    return hexconv_bwd_weight(x, dy, dw, db, ws, ws_bytes, sh.N, sh.Ci, sh.Co, sh.H, sh.W, sh.k,
                              sh.s, dt, stream);
}

int hexconv_bwd(const void *x, const void *dy, const void *w, void *dx, float *dw, float *db,
                void *ws, size_t ws_bytes, int N, int C_in, int C_out, int H, int W, int k,
                int stride, hex_dtype dt, void *stream)
{
    ConvShape sh;
    size_t need = 0;
    int rc = bwd_check(x, dy, w, dx, dw, db, N, C_in, C_out, H, W, k, stride, dt, sh, need);
    if (rc != HEX_OK)
        return rc;
    if ((rc = ptrs_ok({}, {ws})) != HEX_OK)
        return rc;
    if (need > 0 && (ws == nullptr || ws_bytes < need))
        return HEX_ERR_INVALID_ARG;
    return bwd_run(x, dy, w, dx, dw, db, ws, ws_bytes, sh, dt, stream);
}

int hexconv_bwd_noalloc(const void *x, const void *dy, const void *w, void *dx, float *dw,
                        float *db, int N, int C_in, int C_out, int H, int W, int k, int stride,
                        hex_dtype dt, void *stream)
{
    ConvShape sh;
    size_t need = 0;
    int rc = bwd_check(x, dy, w, dx, dw, db, N, C_in, C_out, H, W, k, stride, dt, sh, need);
    if (rc != HEX_OK)
        return rc;
    if (need > HEX_NOALLOC_SCRATCH_BYTES)
        return HEX_ERR_UNSUPPORTED;
    void *ws = nullptr;
    if (need > 0 && (ws = scratch_ptr()) == nullptr)
        return HEX_ERR_LAUNCH;
    return bwd_run(x, dy, w, dx, dw, db, ws, need > 0 ? HEX_NOALLOC_SCRATCH_BYTES : 0, sh, dt,
                   stream);
}

int hexpool_fwd(const void *x, void *y, uint8_t *argmax_tap, int N, int C, int H, int W, int k,
                int stride, hex_pool_mode mode, hex_dtype dt, void *stream)
{
    ConvShape sh;
    int rc = check_shape(N, C, C, H, W, k, stride, dt, sh);
    if (rc != HEX_OK)
        return rc;
    if (mode != HEX_POOL_MAX && mode != HEX_POOL_AVG)
        return HEX_ERR_INVALID_ARG;
    if (N == 0)
        return HEX_OK; // empty batch: buffers may be NULL
    if ((rc = ptrs_ok({x, y}, {argmax_tap})) != HEX_OK)
        return rc;
    if (sh.Ho == 0)
        return HEX_OK;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const Dtype d = static_cast<Dtype>(dt);
    uint8_t *am = mode == HEX_POOL_MAX ? argmax_tap : nullptr;
    if (!force_generic() && hexk::pool_fast_ok(sh, d))
        return launched(hexk::pool_fwd_fast(x, y, am, sh, mode, d, st));
    return launched(hexk::pool_fwd_generic(x, y, am, sh, mode, d, false, st));
}

int hexpool_bwd(const void *dy, const uint8_t *argmax_tap, const void *relu_y, void *dx, int N,
                int C, int H, int W, int k, int stride, hex_pool_mode mode, hex_dtype dt,
                void *stream)
{
    ConvShape sh;
    int rc = check_shape(N, C, C, H, W, k, stride, dt, sh);
    if (rc != HEX_OK)
        return rc;
    if (mode != HEX_POOL_MAX && mode != HEX_POOL_AVG)
        return HEX_ERR_INVALID_ARG;
    if (N == 0)
        return HEX_OK; // empty batch: buffers may be NULL
    if ((rc = ptrs_ok({dx}, {dy, argmax_tap, relu_y})) != HEX_OK)
        return rc;
    if (sh.Ho > 0 && (dy == nullptr || (mode == HEX_POOL_MAX && argmax_tap == nullptr)))
        return HEX_ERR_INVALID_ARG;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const Dtype d = static_cast<Dtype>(dt);
    if (!force_generic() && sh.Ho > 0 && hexk::pool_fast_ok(sh, d))
        return launched(hexk::pool_bwd_fast(dy, argmax_tap, relu_y, dx, sh, mode, d, st));
    return launched(hexk::pool_bwd_generic(dy, argmax_tap, relu_y, dx, sh, mode, d, false, st));
}

// ------------------------------------------------------- three dimensions

int hex_out_shape3d(int D, int H, int W, int k, int kz, int stride, int stride_z, int *D_out,
                    int *H_out, int *W_out)
{
    if (D < 1 || kz < 0 || kz > HEX_MAX_KZ || stride_z < 1 || stride_z > HEX_MAX_STRIDE ||
        D_out == nullptr)
        return HEX_ERR_INVALID_ARG;
    const int rc = hex_out_shape(H, W, k, stride, H_out, W_out);
    if (rc != HEX_OK)
        return rc;
    *D_out = (D - 1) / stride_z + 1;
    return HEX_OK;
}

int hexconv3d_fwd(const void *x, const void *w, const void *bias, void *y, int N, int C_in,
                  int C_out, int D, int H, int W, int k, int kz, int stride, int stride_z,
                  hex_dtype dt, int flags, void *stream)
{
    ConvShape sh;
    int rc = check_shape3d(N, C_in, C_out, D, H, W, k, kz, stride, stride_z, dt, sh);
    if (rc != HEX_OK)
        return rc;
    if ((flags & ~HEX_FLAG_RELU) != 0)
        return HEX_ERR_INVALID_ARG;
    if (N == 0)
        return HEX_OK;
    if ((rc = ptrs_ok({x, w, y}, {bias})) != HEX_OK)
        return rc;
    if (sh.Ho == 0)
        return HEX_OK;
    // few input channels: the small-channel forward with the 2kz + 1 planes
    // around each output plane staged as extra input channels
    if (!force_generic() && hexk::smallc_fwd_ok(sh))
        return launched(hexk::smallc_fwd(x, w, bias, y, sh, static_cast<Dtype>(dt),
                                         (flags & HEX_FLAG_RELU) != 0,
                                         static_cast<hipStream_t>(stream)));
    if (!hexk::conv_fwd_generic_ok(sh))
        return HEX_ERR_UNSUPPORTED;
    return launched(hexk::conv_fwd_generic(x, w, bias, y, sh, static_cast<Dtype>(dt),
                                           (flags & HEX_FLAG_RELU) != 0,
                                           static_cast<hipStream_t>(stream)));
}

int hexconv3d_bwd_data(const void *dy, const void *w, void *dx, int N, int C_in, int C_out, int D,
                       int H, int W, int k, int kz, int stride, int stride_z, hex_dtype dt,
                       void *stream)
{
    ConvShape sh;
    int rc = check_shape3d(N, C_in, C_out, D, H, W, k, kz, stride, stride_z, dt, sh);
    if (rc != HEX_OK)
        return rc;
    if (N == 0)
        return HEX_OK;
    if ((rc = ptrs_ok({w, dx}, {dy})) != HEX_OK)
        return rc;
    if (dy == nullptr && sh.Ho > 0)
        return HEX_ERR_INVALID_ARG;
    if (!force_generic() && sh.Ho > 0 && hexk::smallc3d_bwd_data_ok(sh))
        return launched(hexk::smallc3d_bwd_data(dy, w, dx, sh, static_cast<Dtype>(dt),
                                                static_cast<hipStream_t>(stream)));
    if (!hexk::conv_bwd_data_generic_ok(sh))
        return HEX_ERR_UNSUPPORTED;
    return launched(hexk::conv_bwd_data_generic(dy, w, dx, sh, static_cast<Dtype>(dt),
                                                static_cast<hipStream_t>(stream)));
}

namespace {
// 3-D weight gradient: the small-channel kernel with the planes around each
// output plane staged as channels where it applies, else the generic one
bool wgrad3d_smallc(const ConvShape &sh)
{
    return !force_generic() && hexk::smallc_wgrad_ok(sh);
}

size_t wgrad3d_workspace(const ConvShape &sh)
{
    return wgrad3d_smallc(sh) ? hexk::smallc_wgrad_workspace(sh)
                              : hexk::wgrad_generic_workspace(sh);
}
} // namespace

size_t hexconv3d_bwd_weight_workspace(int N, int C_in, int C_out, int D, int H, int W, int k,
                                      int kz, int stride, int stride_z, hex_dtype dt)
{
    ConvShape sh;
    if (check_shape3d(N, C_in, C_out, D, H, W, k, kz, stride, stride_z, dt, sh) != HEX_OK)
        return 0;
    if (N == 0 || sh.Ho == 0)
        return 0;
    return wgrad3d_workspace(sh);
}

int hexconv3d_bwd_weight(const void *x, const void *dy, float *dw, float *db, void *ws,
                         size_t ws_bytes, int N, int C_in, int C_out, int D, int H, int W, int k,
                         int kz, int stride, int stride_z, hex_dtype dt, void *stream)
{
    ConvShape sh;
    int rc = check_shape3d(N, C_in, C_out, D, H, W, k, kz, stride, stride_z, dt, sh);
    if (rc != HEX_OK)
        return rc;
    if ((rc = ptrs_ok({dw}, {x, dy, db, ws})) != HEX_OK)
        return rc;
    const bool empty = (N == 0 || sh.Ho == 0);
    if (!empty && (x == nullptr || dy == nullptr))
        return HEX_ERR_INVALID_ARG;
    const size_t need = empty ? 0 : wgrad3d_workspace(sh);
    if (need > 0 && (ws == nullptr || ws_bytes < need))
        return HEX_ERR_INVALID_ARG;
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (empty)
        return launched(hexk::fill_zero_f32(dw, db, sh, st));
    if (wgrad3d_smallc(sh))
        return launched(
            hexk::smallc_wgrad(x, dy, dw, db, ws, sh, static_cast<Dtype>(dt), st));
    return launched(hexk::wgrad_generic(x, dy, dw, db, ws, sh, static_cast<Dtype>(dt), st));
}

int hexpool3d_fwd(const void *x, void *y, uint16_t *argmax, int N, int C, int D, int H, int W,
                  int k, int kz, int stride, int stride_z, hex_pool_mode mode, hex_dtype dt,
                  void *stream)
{
    ConvShape sh;
    int rc = check_shape3d(N, C, C, D, H, W, k, kz, stride, stride_z, dt, sh);
    if (rc != HEX_OK)
        return rc;
    if (mode != HEX_POOL_MAX && mode != HEX_POOL_AVG)
        return HEX_ERR_INVALID_ARG;
    if (N == 0)
        return HEX_OK;
    if ((rc = ptrs_ok({x, y}, {argmax})) != HEX_OK)
        return rc;
    if (sh.Ho == 0)
        return HEX_OK;
    return launched(hexk::pool_fwd_generic(x, y, mode == HEX_POOL_MAX ? argmax : nullptr, sh,
                                           mode, static_cast<Dtype>(dt), true,
                                           static_cast<hipStream_t>(stream)));
}

int hexpool3d_bwd(const void *dy, const uint16_t *argmax, const void *relu_y, void *dx, int N,
                  int C, int D, int H, int W, int k, int kz, int stride, int stride_z,
                  hex_pool_mode mode, hex_dtype dt, void *stream)
{
    ConvShape sh;
    int rc = check_shape3d(N, C, C, D, H, W, k, kz, stride, stride_z, dt, sh);
    if (rc != HEX_OK)
        return rc;
    if (mode != HEX_POOL_MAX && mode != HEX_POOL_AVG)
        return HEX_ERR_INVALID_ARG;
    if (N == 0)
        return HEX_OK;
    if ((rc = ptrs_ok({dx}, {dy, argmax, relu_y})) != HEX_OK)
        return rc;
    if (sh.Ho > 0 && (dy == nullptr || (mode == HEX_POOL_MAX && argmax == nullptr)))
        return HEX_ERR_INVALID_ARG;
    return launched(hexk::pool_bwd_generic(dy, argmax, relu_y, dx, sh, mode,
                                           static_cast<Dtype>(dt), true,
                                           static_cast<hipStream_t>(stream)));
}

int hexconv_timing_begin(void)
{
    std::lock_guard<std::mutex> lock(hexk::g_timing_mu);
    for (auto &t : hexk::g_timed) {
        (void)hipEventDestroy(t.a);
        (void)hipEventDestroy(t.b);
    }
    hexk::g_timed.clear();
    hexk::g_timing.store(true);
    return HEX_OK;
}

int hexconv_timing_end(int max_kernels, char *names, int *counts, double *total_ms,
                       int *n_kernels)
{
    hexk::g_timing.store(false);
    if (max_kernels < 1 || names == nullptr || counts == nullptr || total_ms == nullptr ||
        n_kernels == nullptr)
        return HEX_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lock(hexk::g_timing_mu);
    std::vector<std::string> order;
    int rc = HEX_OK;
    *n_kernels = 0;
    for (auto &t : hexk::g_timed) {
        float ms = 0.f;
        if (hipEventSynchronize(t.b) != hipSuccess || hipEventElapsedTime(&ms, t.a, t.b) != hipSuccess)
            rc = HEX_ERR_LAUNCH;
        (void)hipEventDestroy(t.a);
        (void)hipEventDestroy(t.b);
        int i = 0;
        while (i < static_cast<int>(order.size()) && order[i] != t.name)
            ++i;
        if (i == static_cast<int>(order.size())) {
            if (i >= max_kernels)
                continue;
            order.push_back(t.name);
            char *dst = names + static_cast<size_t>(i) * HEX_TIMING_NAME_LEN;
            strncpy(dst, t.name.c_str(), HEX_TIMING_NAME_LEN - 1);
            dst[HEX_TIMING_NAME_LEN - 1] = '\0';
            counts[i] = 0;
            total_ms[i] = 0.0;
        }
        counts[i] += 1;
        total_ms[i] += ms;
    }
    hexk::g_timed.clear();
    *n_kernels = static_cast<int>(order.size());
    return rc;
}

const char *hex_last_launch_error(void)
{
    return g_last_launch_error == hipSuccess ? "" : hipGetErrorString(g_last_launch_error);
}

const char *hex_status_string(int status)
{
    switch (status) {
    case HEX_OK:
        return "HEX_OK";
    case HEX_ERR_INVALID_ARG:
        return "HEX_ERR_INVALID_ARG: invalid argument";
    case HEX_ERR_UNSUPPORTED:
        return "HEX_ERR_UNSUPPORTED: valid request not implemented by the library";
    case HEX_ERR_LAUNCH:
        return "HEX_ERR_LAUNCH: kernel launch failed";
    default:
        return "unknown hex_status";
    }
}

} // extern "C"
