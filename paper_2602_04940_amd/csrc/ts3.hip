// Host side of the C ABI declared in include/ts3.h: validation, the state
// object and its device buffers, the call-order state machine, and kernel
// dispatch over the supported (dtype, C, M) shapes.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/ts3.h"
#include "ts3_pass1.h"
#include "ts3_pass1pc.h"
#include "ts3_pass1pcw.h"
#include "ts3_pass1pcp.h"
#include "ts3_pass2pc.h"
#include "ts3_backward.h"
#include "ts3_pass2.h"
#include "ts3_small.h"
#include "ts3_rt.h"
#include "ts3_pass2sf.h"

using namespace ts3;

namespace {

thread_local std::string g_err;

ts3_status fail(ts3_status s, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
ts3_status fail(ts3_status s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

#define HIP_TRY(expr)                                                                          \
    do {                                                                                       \
        hipError_t e_ = (expr);                                                                \
        if (e_ != hipSuccess)                                                                  \
            return fail(e_ == hipErrorOutOfMemory ? TS3_ERR_OUT_OF_MEMORY : TS3_ERR_HIP,       \
                        "%s failed: %s", #expr, hipGetErrorString(e_));                        \
    } while (0)

#define LAUNCH_CHECK(what)                                                                     \
    do {                                                                                       \
        hipError_t e_ = hipGetLastError();                                                     \
        if (e_ != hipSuccess) return fail(TS3_ERR_HIP, "%s launch: %s", what, hipGetErrorString(e_)); \
    } while (0)

constexpr int ATTN_LDS_MAX = 160 * 1024;
constexpr size_t PASS2_LDS_MAX = 160 * 1024;

enum Phase { PH_RESET = 0, PH_ACCUM = 1, PH_FINAL = 2, PH_ATTEND = 3 };

// Kernel entry points for one (dtype, C, M) instantiation, or the
// runtime-shape kernels (rt) for the other multiples of 16.  The pass entry
// points take C and M, which only the runtime-shape ones read.
struct Kernels {
    void (*pass1)(const void *, int64_t, int64_t, int32_t, int32_t, int32_t, int32_t, int32_t, const void *,
                  const float *, float *, hipStream_t);
    hipError_t (*pass2)(const void *, int64_t, int32_t, int32_t, int32_t, const void *, const float *, const void *,
                        void *, hipStream_t);
    // Backward (float32 storage only; NULL for bfloat16).
    void (*bw_head)(const float *, const float *, int64_t, int64_t, int32_t, int32_t, int32_t, const float *,
                    const float *, float *, hipStream_t);
    void (*bw_dx)(const float *, const float *, int64_t, int32_t, const float *, const float *, const float *,
                  const float *, const float *, const float *, const float *, float, float *, float *,
                  hipStream_t);
    void (*bw_dw2)(const float *, const float *, int64_t, int64_t, int32_t, int32_t, int32_t, float *,
                   hipStream_t);
    // Pass 1 in the projected form (bfloat16, C = 128, head width 16): x, n,
    // span0, Q, nspan, H, W2', b2', W1 fragments, partials [span][H][M][17].
    void (*pass1p)(const void *, int64_t, int64_t, int32_t, int32_t, int32_t, const void *, const float *,
                   const void *, float *, hipStream_t) = nullptr;
    // Pass 2 in the slice-state form (bfloat16, head width 16): x, n, W2', b2',
    // s'^T fragments, W3^T fragments, b3, out.  NULL where it does not apply.
    hipError_t (*pass2sf)(const void *, int64_t, const void *, const float *, const void *, const void *,
                          const float *, void *, hipStream_t) = nullptr;
    bool rt = false;  // operands in the runtime-shape layouts (k_prep_w2_rt, k_prep_z_rt)
};

template <typename T, int C, int M>
void launch_pass1(const void *x, int64_t n, int64_t span0, int32_t Q, int32_t nspan, int32_t H, int32_t, int32_t,
                  const void *w2p, const float *b2s, float *partials, hipStream_t st) {
    if constexpr (sizeof(T) == 2 && C == 256) {
        // Wide rows: two heads per workgroup, two producer and two consumer
        // waves per head (H is even for every wide shape check_desc accepts).
        hipLaunchKernelGGL((k_slice_accumulate_pcw<C, M>), dim3(nspan * (H / 2)), dim3(512), 0, st,
                           (const bf16_t *)x, n, span0, Q, nspan, H, (const bf16_t *)w2p, b2s, partials);
    } else if constexpr (sizeof(T) == 2 && M >= 32 && C == 128) {
        // Two heads per workgroup whenever H is even (independently of the
        // span count, so that every tiling sums a span the same way); the one
        // odd case, H = 1, takes the generic kernel.
        if (H % 2 == 0)
            hipLaunchKernelGGL((k_slice_accumulate_pc<C, M>), dim3(nspan * (H / 2)), dim3(512), 0, st,
                               (const bf16_t *)x, n, span0, Q, nspan, H, (const bf16_t *)w2p, b2s, partials);
        else
            hipLaunchKernelGGL((k_slice_accumulate<T, C, M>), dim3(nspan * H), dim3(256), 0, st,
                               (const T *)x, n, span0, Q, nspan, H, (const T *)w2p, b2s, partials);
    } else {
        hipLaunchKernelGGL((k_slice_accumulate<T, C, M>), dim3(nspan * H), dim3(256), 0, st,
                           (const T *)x, n, span0, Q, nspan, H, (const T *)w2p, b2s, partials);
    }
}

// Compute units of the current device, looked up once per device.
int device_cu_count() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (dev < 0 || dev >= 64) {
        int c = 0;
        return hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && c > 0 ? c : 256;
    }
    int c = cache[dev].load(std::memory_order_relaxed);
    if (c <= 0) {
        if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || c <= 0) c = 256;
        cache[dev].store(c, std::memory_order_relaxed);
    }
    return c;
}


template <typename T, int C, int M>
hipError_t launch_pass2(const void *x, int64_t n, int32_t H, int32_t, int32_t, const void *w2p, const float *b2s,
                        const void *zp, void *out, hipStream_t st) {
    using Cfg = Pass2Cfg<T, C, M>;
    const int64_t nblk = (n + Cfg::POINTS_PER_WG - 1) / Cfg::POINTS_PER_WG;
    if constexpr (sizeof(T) == 2 && C == 256) {
        // Producer and consumer waves, heads streamed through LDS, persistent
        // workgroups of 128-point blocks.  (At C = 128 the same kernel ran
        // 22% slower than the eight-wave one below: the producer's softmax is
        // twice as large against its MFMAs.)
        using PCfg = Pass2PCCfg<C, M>;
        const int64_t blocks = (n + PCfg::POINTS_PER_WG - 1) / PCfg::POINTS_PER_WG;
        const int64_t grid = std::min<int64_t>(blocks, device_cu_count());
        if (grid > 0)
            hipLaunchKernelGGL((k_deslice_pc<C, M>), dim3((unsigned)grid), dim3(512), 0, st, (const bf16_t *)x, n, H,
                               (const bf16_t *)w2p, b2s, (const bf16_t *)zp, (bf16_t *)out);
        return hipSuccess;
    } else if constexpr (sizeof(T) == 2 && C <= 128) {
        using WCfg = Pass2W8Cfg<T, C, M>;
        const size_t lds = WCfg::lds_bytes(H);
        // The kernel's static LDS is a property of its code (thread-safe init).
        static const size_t static_lds = [] {
            hipFuncAttributes fa{};
            return hipFuncGetAttributes(&fa, (const void *)k_deslice_w8<T, C, M>) == hipSuccess
                       ? fa.sharedSizeBytes : PASS2_LDS_MAX;
        }();
        if (lds + static_lds <= PASS2_LDS_MAX) {
            // Granted on every call: the attribute may be per device, and the
            // call costs microseconds against a launch of a million points.
            if (hipFuncSetAttribute((const void *)k_deslice_w8<T, C, M>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                    (int)lds) != hipSuccess)
                return hipGetLastError();
            // At most P2_MAX_ITERS blocks per workgroup and launch (the kernel
            // records slow-path blocks in a 64-bit mask); larger calls are
            // split, which changes no result: every point is decoded alone.
            const int64_t cus = device_cu_count();
            const int64_t span = cus * P2_MAX_ITERS * WCfg::POINTS_PER_WG;
            for (int64_t off = 0; off < n; off += span) {
                const int64_t m = std::min<int64_t>(span, n - off);
                const int64_t wblk = (m + WCfg::POINTS_PER_WG - 1) / WCfg::POINTS_PER_WG;
                const int64_t grid = std::min<int64_t>(wblk, cus);
                hipLaunchKernelGGL((k_deslice_w8<T, C, M>), dim3((unsigned)grid), dim3(64 * WCfg::WAVES), lds, st,
                                   (const T *)x + off * C, m, H, (const T *)w2p, b2s, (const T *)zp,
                                   (T *)out + off * C);
            }
            return hipSuccess;
        }
        // Every supported 16-bit shape fits the staged kernel's LDS (H*dh = C
        // bounds H*M*C); a shape that does not has no decoding kernel.
        return hipErrorInvalidConfiguration;
    } else {
        hipLaunchKernelGGL((k_deslice<T, C, M>), dim3((unsigned)nblk), dim3(256), 0, st, (const T *)x, n, H,
                           (const T *)w2p, b2s, (const T *)zp, (T *)out);
        return hipSuccess;
    }
}

template <int C, int M>
void launch_bw_head(const float *x, const float *g, int64_t n, int64_t span0, int32_t Q, int32_t nspan,
                    int32_t H, const float *w2p, const float *b2s, float *partials, hipStream_t st) {
    const int64_t places = (int64_t)BW_XCDS * ((nspan + BW_XCDS - 1) / BW_XCDS) * H;
    hipLaunchKernelGGL((k_bw_head<C, M>), dim3((unsigned)places), dim3(512), 0, st, x, g, n, span0, Q, nspan, H,
                       w2p, b2s, partials);
}

template <int C, int M>
void launch_bw_dw2(const float *x, const float *dzs, int64_t n, int64_t span0, int32_t Q, int32_t nspan, int32_t H,
                   float *partials, hipStream_t st) {
    const int64_t places = (int64_t)BW_XCDS * ((nspan + BW_XCDS - 1) / BW_XCDS) * H;
    hipLaunchKernelGGL((k_bw_dw2<C, M>), dim3((unsigned)places), dim3(512), 0, st, x, dzs, n, span0, Q, nspan, H,
                       partials);
}

constexpr int BW_DX_TILES_PER_WAVE = 4;  // each L2 A fragment serves four 16-point tiles

template <int C, int M>
void launch_bw_dx(const float *x, const float *g, int64_t n, int32_t H, const float *w2p, const float *b2s,
                  const float *W2, const float *Z, const float *dsr, const float *dsT, const float *dd,
                  float inv_tau, float *dx, float *dzs, hipStream_t st) {
    constexpr int NT = BW_DX_TILES_PER_WAVE;
    hipLaunchKernelGGL((k_bw_dx<C, M, NT>), dim3((unsigned)((n + 64 * NT - 1) / (64 * NT))), dim3(256), 0, st, x, g,
                       n, H, w2p, b2s, W2, Z, dsr, dsT, dd, inv_tau, dx, dzs);
}

template <int C, int M>
void launch_pass1p(const void *x, int64_t n, int64_t span0, int32_t Q, int32_t nspan, int32_t H, const void *w2p,
                   const float *b2s, const void *w1p, float *partials, hipStream_t st) {
    hipLaunchKernelGGL((k_slice_accumulate_pcp<C, M>), dim3(nspan * (H / 2)), dim3(PCP_THREADS), 0, st, (const bf16_t *)x,
                       n, span0, Q, nspan, H, (const bf16_t *)w2p, b2s, (const bf16_t *)w1p, partials);
}

template <int C, int M>
hipError_t launch_pass2sf(const void *x, int64_t n, const void *w2p, const float *b2s, const void *sf,
                          const void *w3f, const float *b3, void *out, hipStream_t st) {
    using Cfg = Pass2SFCfg<C, M>;
    // At most P2_MAX_ITERS blocks per workgroup and launch (the kernel records
    // fallback blocks in a 64-bit mask); larger calls are split, which changes
    // no result: every point is decoded alone.
    const int64_t cus = device_cu_count();
    const int64_t span = cus * P2_MAX_ITERS * Cfg::POINTS_PER_WG;
    for (int64_t off = 0; off < n; off += span) {
        const int64_t m = std::min<int64_t>(span, n - off);
        const int64_t blocks = (m + Cfg::POINTS_PER_WG - 1) / Cfg::POINTS_PER_WG;
        const int64_t grid = std::min<int64_t>(blocks, cus);
        hipLaunchKernelGGL((k_deslice_sf<C, M>), dim3((unsigned)grid), dim3(512), 0, st,
                           (const bf16_t *)x + off * C, m, (const bf16_t *)w2p, b2s, (const bf16_t *)sf,
                           (const bf16_t *)w3f, b3, (bf16_t *)out + off * C);
    }
    return hipSuccess;
}

template <typename T, int C, int M> Kernels make_kernels() {
    if constexpr (C > 128 && sizeof(T) == 4)
        return Kernels{nullptr, nullptr, nullptr, nullptr, nullptr};  // float32 rows of 1 KB: no pass-1 kernel
    else if constexpr (sizeof(T) == 4)
        return Kernels{&launch_pass1<T, C, M>, &launch_pass2<T, C, M>, &launch_bw_head<C, M>, &launch_bw_dx<C, M>,
                       &launch_bw_dw2<C, M>};
    else if constexpr (C == 128 && M % 32 == 0)
        return Kernels{&launch_pass1<T, C, M>, &launch_pass2<T, C, M>, nullptr, nullptr, nullptr,
                       &launch_pass1p<C, M>, &launch_pass2sf<C, M>};
    else if constexpr (C <= 128 && M % 32 == 0)
        return Kernels{&launch_pass1<T, C, M>, &launch_pass2<T, C, M>, nullptr, nullptr, nullptr, nullptr,
                       &launch_pass2sf<C, M>};
    else
        return Kernels{&launch_pass1<T, C, M>, &launch_pass2<T, C, M>, nullptr, nullptr, nullptr};
}

// Launches of at most RT_MAX_WGS workgroups (larger calls are split into
// span or point ranges, which changes no result).
constexpr int64_t RT_MAX_WGS = 1 << 22;

template <typename T>
void launch_pass1_rt(const void *x, int64_t n, int64_t span0, int32_t Q, int32_t nspan, int32_t H, int32_t C,
                     int32_t M, const void *w2r, const float *b2s, float *partials, hipStream_t st) {
    const size_t lds = (size_t)RT_PTS * (C + M) * 4;
    const int64_t per_span = (int64_t)H * ((C + 63) / 64);
    const int64_t batch = std::max<int64_t>(1, RT_MAX_WGS / per_span);
    for (int64_t s0 = 0; s0 < nspan; s0 += batch) {
        const int64_t ns = std::min<int64_t>(batch, nspan - s0);
        hipLaunchKernelGGL(k_slice_accumulate_rt<T>, dim3((unsigned)(ns * per_span)), dim3(256), lds, st,
                           (const T *)x + s0 * Q * C, n - s0 * Q, span0 + s0, Q, H, C, M, (const T *)w2r, b2s,
                           partials);
    }
}
template <typename T>
hipError_t launch_pass2_rt(const void *x, int64_t n, int32_t H, int32_t C, int32_t M, const void *w2r,
                           const float *b2s, const void *zr, void *out, hipStream_t st) {
    const size_t lds = (size_t)RT_PTS * (C + M) * 4;
    for (int64_t p0 = 0; p0 < n; p0 += RT_MAX_WGS * RT_PTS) {
        const int64_t np = std::min<int64_t>(RT_MAX_WGS * RT_PTS, n - p0);
        hipLaunchKernelGGL(k_deslice_rt<T>, dim3((unsigned)((np + RT_PTS - 1) / RT_PTS)), dim3(256), lds, st,
                           (const T *)x + p0 * C, np, H, C, M, (const T *)w2r, b2s, (const T *)zr,
                           (T *)out + p0 * C);
    }
    return hipSuccess;
}

bool find_kernels(int dtype, int C, int M, Kernels *k) {
#define TS3_SHAPE(CC, MM)                                                                      \
    if (C == CC && M == MM) {                                                                  \
        *k = dtype == TS3_BF16 ? make_kernels<bf16_t, CC, MM>() : make_kernels<float, CC, MM>(); \
        return k->pass1 != nullptr;                                                            \
    }
    TS3_SHAPE(64, 16)
    TS3_SHAPE(64, 32)
    TS3_SHAPE(128, 16)
    TS3_SHAPE(128, 32)
    TS3_SHAPE(128, 64)
    TS3_SHAPE(256, 64)
#undef TS3_SHAPE
    return false;
}

// The tuned kernels for (dtype, C, M), else the runtime-shape ones when C and
// M are multiples of 16 within their limits.
bool find_any_kernels(int dtype, int C, int M, Kernels *k) {
    if (find_kernels(dtype, C, M, k)) return true;
    if (C % 16 != 0 || M % 16 != 0 || C > RT_MAX_C || M > RT_MAX_M) return false;
    *k = dtype == TS3_BF16 ? Kernels{&launch_pass1_rt<bf16_t>, &launch_pass2_rt<bf16_t>, nullptr, nullptr, nullptr}
                           : Kernels{&launch_pass1_rt<float>, &launch_pass2_rt<float>, nullptr, nullptr, nullptr};
    k->rt = true;
    return true;
}

// Elements of the prepared W2' and Z buffers (fragment order, or rows for
// the runtime-shape kernels).
int64_t w2p_elems(const ts3_desc &d) { return (int64_t)d.H * d.M * d.C; }
int64_t zp_elems(const ts3_desc &d, bool rt) {
    const int KM = d.M >= 32 ? d.M / 32 : 1;
    return rt ? (int64_t)d.H * d.M * d.C : (int64_t)d.H * (d.C / 16) * KM * 512;
}

}  // namespace

struct ts3_state {
    ts3_desc desc;
    Kernels k;
    int esize;          // bytes per io element
    int64_t nspan_max;  // spans the partial buffer holds
    int64_t E;          // floats per (span, head-block) partial row group: H*M*(C+1)
    int64_t nrun_max;
    // device buffers
    float *partials = nullptr, *runs = nullptr, *s_raw = nullptr, *dsum = nullptr, *s = nullptr,
          *s1 = nullptr, *Z = nullptr, *b2s = nullptr, *b3 = nullptr;
    // backward: dZ, ds_raw [H][M][C], ds_raw transposed [H][C][M], dd [H][M], dW2^T [H][M][C]
    float *bdZ = nullptr, *bdsr = nullptr, *bdsT = nullptr, *bdd = nullptr, *bdW2T = nullptr;
    // backward: dz [H][points][M] of one tile, allocated by the first backward
    // whose tile needs more than it holds
    float *bdz = nullptr;
    int64_t bdz_points = 0;
    void *w2p = nullptr, *zp = nullptr;
    // slice-state form of pass 2: s'^T and W3^T fragments, valid after attention
    // (not after a state injected as Z)
    void *sfp = nullptr, *w3p = nullptr;
    bool sf_ready = false;
    int64_t bytes = 0;
    // host bookkeeping
    std::vector<uint8_t> span_written;
    int64_t span_hi = 0;
    int phase = PH_RESET;
    bool w2_ready = false;
    bool partials_fwd = false;  // the partial buffer holds pass-1 span sums (not a backward's)
    const float *W2 = nullptr, *b2 = nullptr, *W1 = nullptr;
    // projected pass 1 (k.pass1p and head width 16): the partials and the
    // folded sums hold t = sum w (x W1) ([H][M][16]) instead of s_raw = sum w x
    bool proj = false;
    int rowc = 0;  // columns of a partial row before its d entry: dh if proj, else C
    void *w1p = nullptr;
    // Second stream for ts3_layer_forward (default priority): consecutive
    // tiles and chunks alternate between it and the caller's stream, so one
    // launch's last partial round of workgroups overlaps the next launch's
    // first.
    hipStream_t aux = nullptr;
    hipEvent_t ev_fork = nullptr, ev_join = nullptr;
};

namespace {

ts3_status check_desc(const ts3_desc *d) {
    if (!d) return fail(TS3_ERR_INVALID_ARG, "desc is NULL");
    if (d->C <= 0 || d->H <= 0 || d->M <= 0 || d->dh <= 0)
        return fail(TS3_ERR_INVALID_ARG, "C, H, M, dh must be positive (got %d, %d, %d, %d)", d->C, d->H,
                    d->M, d->dh);
    if ((int64_t)d->H * d->dh != d->C)
        return fail(TS3_ERR_UNSUPPORTED, "H*dh (%d*%d) must equal C (%d)", d->H, d->dh, d->C);
    if (d->io_dtype != TS3_FP32 && d->io_dtype != TS3_BF16)
        return fail(TS3_ERR_INVALID_ARG, "io_dtype %d is not TS3_FP32 or TS3_BF16", d->io_dtype);
    if (d->accum != TS3_ACCUM_FP32 && d->accum != TS3_ACCUM_FP64)
        return fail(TS3_ERR_INVALID_ARG, "accum %d is not TS3_ACCUM_FP32 or TS3_ACCUM_FP64", d->accum);
    if (!(d->temperature > 0.f)) return fail(TS3_ERR_INVALID_ARG, "temperature must be > 0");
    if (!(d->eps >= 0.f) || std::isinf(d->eps)) return fail(TS3_ERR_INVALID_ARG, "eps must be finite and >= 0");
    if (d->group_span <= 0 || d->group_span > (1 << 30))
        return fail(TS3_ERR_INVALID_ARG, "group_span must be in [1, 2^30] (got %lld)",
                    (long long)d->group_span);
    if (d->max_points < 0) return fail(TS3_ERR_INVALID_ARG, "max_points must be >= 0");
    if (d->H > 4096 || d->dh > 256) return fail(TS3_ERR_UNSUPPORTED, "H <= 4096 and dh <= 256 required");
    Kernels k;
    if (!find_any_kernels(d->io_dtype, d->C, d->M, &k))
        return fail(TS3_ERR_UNSUPPORTED, "no kernel for C=%d, M=%d (C and M must be multiples of 16 with "
                    "C <= %d and M <= %d)", d->C, d->M, RT_MAX_C, RT_MAX_M);
    if ((5 * d->M * d->dh + d->M * d->M) * 4 > ATTN_LDS_MAX)
        return fail(TS3_ERR_UNSUPPORTED, "token attention needs (5*M*dh + M*M) floats <= 160 KiB of LDS");
    if (d->C == 256 && d->H % 2 != 0)  // implied by the LDS bound at M = 64; the wide pass 1 pairs heads
        return fail(TS3_ERR_UNSUPPORTED, "C=256 needs an even head count");
    const int64_t nspan = (d->max_points + d->group_span - 1) / d->group_span;
    if (nspan * (int64_t)d->H > (int64_t)INT32_MAX)
        return fail(TS3_ERR_UNSUPPORTED, "too many spans: raise group_span");
    return TS3_OK;
}

ts3_status check_weights_w2(const ts3_weights *w) {
    if (!w) return fail(TS3_ERR_INVALID_ARG, "weights is NULL");
    if (!w->W2) return fail(TS3_ERR_INVALID_ARG, "W2 is NULL");
    return TS3_OK;
}

ts3_status prep_w2(ts3_state *st, const ts3_weights *w, hipStream_t stream) {
    const ts3_desc &d = st->desc;
    const float scale = (float)(1.4426950408889634 / (double)d.temperature);
    const int64_t total = w2p_elems(d);
    const int grid = (int)std::min<int64_t>((total + 255) / 256, 4096);
    const int grid2 = std::max(grid, (d.H * d.M + 255) / 256);
    if (st->k.rt && d.io_dtype == TS3_BF16)
        hipLaunchKernelGGL(k_prep_w2_rt<bf16_t>, dim3(grid2), dim3(256), 0, stream, w->W2, w->b2, scale, d.C, d.H,
                           d.M, (bf16_t *)st->w2p, st->b2s);
    else if (st->k.rt)
        hipLaunchKernelGGL(k_prep_w2_rt<float>, dim3(grid2), dim3(256), 0, stream, w->W2, w->b2, scale, d.C, d.H,
                           d.M, (float *)st->w2p, st->b2s);
    else if (d.io_dtype == TS3_BF16)
        hipLaunchKernelGGL(k_prep_w2<bf16_t>, dim3(grid2), dim3(256), 0, stream, w->W2, w->b2, scale, d.C,
                           d.H, d.M, (bf16_t *)st->w2p, st->b2s);
    else
        hipLaunchKernelGGL(k_prep_w2<float>, dim3(grid2), dim3(256), 0, stream, w->W2, w->b2, scale, d.C,
                           d.H, d.M, (float *)st->w2p, st->b2s);
    LAUNCH_CHECK("prep_w2");
    if (st->proj && w->W1) {  // the W1 fragments of the projected pass 1
        const int64_t nw1 = (int64_t)d.C * d.C;
        hipLaunchKernelGGL(k_prep_w1, dim3((unsigned)std::min<int64_t>((nw1 + 255) / 256, 1024)), dim3(256), 0,
                           stream, w->W1, d.C, d.H, (bf16_t *)st->w1p);
        LAUNCH_CHECK("prep_w1");
        st->W1 = w->W1;
    }
    st->W2 = w->W2;
    st->b2 = w->b2;
    st->w2_ready = true;
    return TS3_OK;
}

ts3_status prep_z(ts3_state *st, hipStream_t stream) {
    const ts3_desc &d = st->desc;
    const int64_t total = zp_elems(d, st->k.rt);
    const int grid = (int)std::min<int64_t>((total + 255) / 256, 4096);
    if (st->k.rt && d.io_dtype == TS3_BF16)
        hipLaunchKernelGGL(k_prep_z_rt<bf16_t>, dim3(grid), dim3(256), 0, stream, st->Z, st->b3, d.C, d.H, d.M,
                           (bf16_t *)st->zp);
    else if (st->k.rt)
        hipLaunchKernelGGL(k_prep_z_rt<float>, dim3(grid), dim3(256), 0, stream, st->Z, st->b3, d.C, d.H, d.M,
                           (float *)st->zp);
    else if (d.io_dtype == TS3_BF16)
        hipLaunchKernelGGL(k_prep_z<bf16_t>, dim3(grid), dim3(256), 0, stream, st->Z, st->b3, d.C, d.H, d.M,
                           (bf16_t *)st->zp);
    else
        hipLaunchKernelGGL(k_prep_z<float>, dim3(grid), dim3(256), 0, stream, st->Z, st->b3, d.C, d.H, d.M,
                           (float *)st->zp);
    LAUNCH_CHECK("prep_z");
    return TS3_OK;
}

bool same_w2(const ts3_state *st, const ts3_weights *w) { return w->W2 == st->W2 && w->b2 == st->b2; }

}  // namespace

extern "C" {

const char *ts3_status_string(ts3_status s) {
    switch (s) {
        case TS3_OK: return "ok";
        case TS3_ERR_INVALID_ARG: return "invalid argument";
        case TS3_ERR_BAD_STATE: return "call out of order";
        case TS3_ERR_OUT_OF_MEMORY: return "out of device memory";
        case TS3_ERR_HIP: return "HIP runtime error";
        case TS3_ERR_UNSUPPORTED: return "unsupported shape";
    }
    return "unknown status";
}

const char *ts3_last_error(void) { return g_err.c_str(); }

ts3_status ts3_state_free(ts3_state *st) {
    if (!st) return TS3_OK;
    hipError_t e = hipDeviceSynchronize();
    void *bufs[] = {st->partials, st->runs, st->s_raw, st->dsum, st->s,    st->s1,    st->Z,
                    st->b2s,      st->b3,   st->w2p,   st->zp,   st->bdZ,  st->bdsr,  st->bdsT,
                    st->bdd,      st->bdW2T, st->bdz,  st->sfp,  st->w3p,   st->w1p};
    for (void *b : bufs)
        if (b) (void)hipFree(b);
    if (st->ev_fork) (void)hipEventDestroy(st->ev_fork);
    if (st->ev_join) (void)hipEventDestroy(st->ev_join);
    if (st->aux) (void)hipStreamDestroy(st->aux);
    delete st;
    if (e != hipSuccess) return fail(TS3_ERR_HIP, "hipDeviceSynchronize: %s", hipGetErrorString(e));
    return TS3_OK;
}

namespace {
// The second stream and its two events, made with the state so that
// ts3_layer_forward creates nothing.
ts3_status make_aux(ts3_state *st) {
    HIP_TRY(hipStreamCreateWithFlags(&st->aux, hipStreamNonBlocking));
    HIP_TRY(hipEventCreateWithFlags(&st->ev_fork, hipEventDisableTiming));
    HIP_TRY(hipEventCreateWithFlags(&st->ev_join, hipEventDisableTiming));
    return TS3_OK;
}
}  // namespace

ts3_status ts3_state_create(const ts3_desc *desc, ts3_state **out) {
    if (!out) return fail(TS3_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    ts3_status s = check_desc(desc);
    if (s != TS3_OK) return s;
    ts3_state *st = new (std::nothrow) ts3_state();
    if (!st) return fail(TS3_ERR_OUT_OF_MEMORY, "host allocation failed");
    st->desc = *desc;
    find_any_kernels(desc->io_dtype, desc->C, desc->M, &st->k);
    const ts3_desc &d = st->desc;
    st->esize = d.io_dtype == TS3_BF16 ? 2 : 4;
    st->nspan_max = std::max<int64_t>(1, (d.max_points + d.group_span - 1) / d.group_span);
    st->proj = st->k.pass1p && d.H * 16 == d.C;
    st->rowc = st->proj ? 16 : d.C;
    st->E = (int64_t)d.H * d.M * (st->rowc + 1);
    st->nrun_max = (st->nspan_max + FOLD - 1) / FOLD;
    const int64_t HM = (int64_t)d.H * d.M;
    struct Req {
        void **p;
        int64_t bytes;
    } reqs[] = {
        {(void **)&st->partials, st->nspan_max * st->E * 4},
        {(void **)&st->runs, st->nrun_max * st->E * 8},  // float or double run sums
        {(void **)&st->s_raw, HM * d.C * 4},
        {(void **)&st->dsum, HM * 4},
        {(void **)&st->s, HM * d.dh * 4},
        {(void **)&st->s1, HM * d.dh * 4},
        {(void **)&st->Z, HM * d.C * 4},
        {(void **)&st->b2s, HM * 4},
        {(void **)&st->b3, (int64_t)d.C * 4},
        {&st->w2p, w2p_elems(d) * st->esize},
        {&st->zp, zp_elems(d, st->k.rt) * st->esize},
        {(void **)&st->bdZ, HM * d.C * 4},
        {(void **)&st->bdsr, HM * d.C * 4},
        {(void **)&st->bdsT, HM * d.C * 4},
        {(void **)&st->bdd, HM * 4},
        {(void **)&st->bdW2T, HM * d.C * 4},
        // slice-state pass 2 (head width 16 only; empty otherwise)
        {&st->sfp, d.H * 16 == d.C && st->k.pass2sf ? HM * 16 * 2 : 0},
        {&st->w3p, d.H * 16 == d.C && st->k.pass2sf ? (int64_t)d.C * d.C * 2 : 0},
        {&st->w1p, st->proj ? (int64_t)d.C * d.C * 4 : 0},  // W1 fragments [2][H][C/32][64][8]
    };
    if (d.H * 16 != d.C) st->k.pass2sf = nullptr;
    for (auto &r : reqs) {
        if (r.bytes == 0) continue;
        hipError_t e = hipMalloc(r.p, (size_t)r.bytes);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            ts3_state_free(st);
            return fail(e == hipErrorOutOfMemory ? TS3_ERR_OUT_OF_MEMORY : TS3_ERR_HIP,
                        "hipMalloc(%lld bytes): %s", (long long)r.bytes, hipGetErrorString(e));
        }
        st->bytes += r.bytes;
    }
    st->span_written.assign((size_t)st->nspan_max, 0);
    s = make_aux(st);
    if (s != TS3_OK) {
        ts3_state_free(st);
        return s;
    }
    *out = st;
    return TS3_OK;
}

ts3_status ts3_state_bytes(const ts3_state *st, int64_t *bytes) {
    if (!st || !bytes) return fail(TS3_ERR_INVALID_ARG, "NULL argument");
    *bytes = st->bytes;
    return TS3_OK;
}

ts3_status ts3_state_reset(ts3_state *st, void *stream) {
    (void)stream;
    if (!st) return fail(TS3_ERR_INVALID_ARG, "state is NULL");
    std::fill(st->span_written.begin(), st->span_written.end(), 0);
    st->span_hi = 0;
    st->phase = PH_RESET;
    st->w2_ready = false;
    st->partials_fwd = false;
    st->W2 = st->b2 = nullptr;
    return TS3_OK;
}

ts3_status ts3_slice_accumulate(ts3_state *st, const ts3_weights *w, const void *x_tile, int64_t n_tile,
                                int64_t point_offset, void *stream) {
    if (!st) return fail(TS3_ERR_INVALID_ARG, "state is NULL");
    ts3_status s = check_weights_w2(w);
    if (s != TS3_OK) return s;
    if (st->phase != PH_RESET && st->phase != PH_ACCUM)
        return fail(TS3_ERR_BAD_STATE, "accumulate after finalize: call ts3_state_reset first");
    if (n_tile < 0 || point_offset < 0) return fail(TS3_ERR_INVALID_ARG, "negative size or offset");
    if (n_tile == 0) return TS3_OK;
    if (!x_tile) return fail(TS3_ERR_INVALID_ARG, "x_tile is NULL");
    if (((uintptr_t)x_tile & 15) != 0) return fail(TS3_ERR_INVALID_ARG, "x_tile must be 16-byte aligned");
    const ts3_desc &d = st->desc;
    const int64_t Q = d.group_span;
    if (point_offset % Q != 0)
        return fail(TS3_ERR_INVALID_ARG, "point_offset %lld is not a multiple of group_span %lld",
                    (long long)point_offset, (long long)Q);
    if (point_offset + n_tile > d.max_points)
        return fail(TS3_ERR_INVALID_ARG, "tile end %lld exceeds max_points %lld",
                    (long long)(point_offset + n_tile), (long long)d.max_points);
    if (st->proj && !w->W1) return fail(TS3_ERR_INVALID_ARG, "W1 is NULL (this layer accumulates projected sums)");
    if (st->w2_ready && !same_w2(st, w))
        return fail(TS3_ERR_INVALID_ARG, "W2/b2 differ from the ones recorded at the first accumulate");
    if (st->w2_ready && st->proj && w->W1 != st->W1)
        return fail(TS3_ERR_INVALID_ARG, "W1 differs from the one recorded at the first accumulate");
    const int64_t span0 = point_offset / Q;
    const int64_t nspan = (n_tile + Q - 1) / Q;
    const bool ragged = n_tile % Q != 0;
    for (int64_t i = span0; i < span0 + nspan; ++i)
        if (st->span_written[(size_t)i])
            return fail(TS3_ERR_INVALID_ARG, "tile overlaps span %lld accumulated earlier", (long long)i);
    // A ragged (short) last span must hold the mesh's last point: no written span may follow it.
    if (ragged && span0 + nspan < st->span_hi)
        return fail(TS3_ERR_INVALID_ARG, "a tile ending inside a span must be the mesh's last tile");
    for (int64_t i = 0; i < span0; ++i)
        if (st->span_written[(size_t)i] == 2)
            return fail(TS3_ERR_INVALID_ARG, "a tile ending inside a span was accumulated before this one");
    hipStream_t hs = (hipStream_t)stream;
    if (!st->w2_ready) {
        s = prep_w2(st, w, hs);
        if (s != TS3_OK) return s;
    }
    if (st->proj)
        st->k.pass1p(x_tile, n_tile, span0, (int32_t)Q, (int32_t)nspan, d.H, st->w2p, st->b2s, st->w1p, st->partials,
                     hs);
    else
        st->k.pass1(x_tile, n_tile, span0, (int32_t)Q, (int32_t)nspan, d.H, d.C, d.M, st->w2p, st->b2s, st->partials,
                hs);
    LAUNCH_CHECK("slice_accumulate");
    for (int64_t i = span0; i < span0 + nspan; ++i) st->span_written[(size_t)i] = 1;
    if (ragged) st->span_written[(size_t)(span0 + nspan - 1)] = 2;
    st->span_hi = std::max(st->span_hi, span0 + nspan);
    st->phase = PH_ACCUM;
    st->partials_fwd = true;
    return TS3_OK;
}

}  // extern "C"

namespace {

// Ordered fold of the first nspan span partials into main [H*M*C] and the
// column C entries into col [H*M] (the forward's fold kernels).
template <typename T>
ts3_status fold_partials_t(ts3_state *st, int64_t nspan, int rowc, float *main, float *col, hipStream_t hs) {
    const int64_t E = (int64_t)st->desc.H * st->desc.M * (rowc + 1);
    const int64_t nrun = (nspan + FOLD - 1) / FOLD;
    const unsigned gx = (unsigned)((E + 255) / 256);
    T *runs = reinterpret_cast<T *>(st->runs);
    hipLaunchKernelGGL(k_fold_runs<T>, dim3(gx, (unsigned)nrun), dim3(256), 0, hs, st->partials, E, nspan, runs);
    LAUNCH_CHECK("fold_runs");
    hipLaunchKernelGGL(k_fold_final<T>, dim3(gx), dim3(256), 0, hs, runs, E, nrun, rowc, main, col);
    LAUNCH_CHECK("fold_final");
    return TS3_OK;
}

// rowc: columns of a partial row before its last (d-like) entry.
ts3_status fold_partials(ts3_state *st, int64_t nspan, int rowc, float *main, float *col, hipStream_t hs) {
    return st->desc.accum == TS3_ACCUM_FP64 ? fold_partials_t<double>(st, nspan, rowc, main, col, hs)
                                            : fold_partials_t<float>(st, nspan, rowc, main, col, hs);
}

}  // namespace

extern "C" {

ts3_status ts3_slice_finalize(ts3_state *st, const ts3_weights *w, void *stream) {
    if (!st) return fail(TS3_ERR_INVALID_ARG, "state is NULL");
    if (!w || !w->W1) return fail(TS3_ERR_INVALID_ARG, "weights or W1 is NULL");
    if (st->phase != PH_RESET && st->phase != PH_ACCUM)
        return fail(TS3_ERR_BAD_STATE, "finalize needs a reset or accumulating state");
    const ts3_desc &d = st->desc;
    hipStream_t hs = (hipStream_t)stream;
    const int64_t E = st->E;
    const int64_t nspan = std::max<int64_t>(st->span_hi, 1);
    // Spans below span_hi that no tile wrote contribute zero.
    for (int64_t i = 0; i < nspan; ++i) {
        if (st->span_written[(size_t)i]) continue;
        int64_t j = i;
        while (j < nspan && !st->span_written[(size_t)j]) ++j;
        const int64_t cnt = (j - i) * E;
        hipLaunchKernelGGL(k_zero, dim3((unsigned)std::min<int64_t>((cnt + 255) / 256, 65535)), dim3(256), 0,
                           hs, st->partials + i * E, cnt);
        LAUNCH_CHECK("zero spans");
        i = j;
    }
    const ts3_status s = fold_partials(st, nspan, st->rowc, st->s_raw, st->dsum, hs);
    if (s != TS3_OK) return s;
    if (st->proj)
        hipLaunchKernelGGL(k_finalize_proj, dim3(d.H), dim3(256), 0, hs, st->s_raw, st->dsum, w->b1, d.H, d.M, d.eps,
                           st->s);
    else
        hipLaunchKernelGGL(k_finalize, dim3(d.H * d.M), dim3(64), 0, hs, st->s_raw, st->dsum, w->W1, w->b1, d.C,
                           d.H, d.M, d.dh, d.eps, st->s);
    LAUNCH_CHECK("finalize");
    st->phase = PH_FINAL;
    return TS3_OK;
}

ts3_status ts3_token_attention(ts3_state *st, const ts3_weights *w, void *stream) {
    if (!st) return fail(TS3_ERR_INVALID_ARG, "state is NULL");
    if (!w || !w->Wq || !w->Wk || !w->Wv || !w->W3)
        return fail(TS3_ERR_INVALID_ARG, "weights, Wq, Wk, Wv or W3 is NULL");
    if (st->phase != PH_FINAL) return fail(TS3_ERR_BAD_STATE, "token_attention needs a finalized state");
    const ts3_desc &d = st->desc;
    hipStream_t hs = (hipStream_t)stream;
    const size_t lds = (size_t)(5 * d.M * d.dh + d.M * d.M) * 4;
    if (lds > 64 * 1024)
        HIP_TRY(hipFuncSetAttribute((const void *)k_attention, hipFuncAttributeMaxDynamicSharedMemorySize,
                                    ATTN_LDS_MAX));
    // Z's columns in blocks of 64 over as many workgroups per head
    const int zb = d.C % 64 == 0 ? d.C / 64 : 1;
    hipLaunchKernelGGL(k_attention, dim3(d.H, zb), dim3(256), lds, hs, st->s, w->Wq, w->Wk, w->Wv, w->W3, d.C, d.H,
                       d.M, d.dh, st->s1, st->Z);
    LAUNCH_CHECK("attention");
    if (w->b3)
        HIP_TRY(hipMemcpyAsync(st->b3, w->b3, (size_t)d.C * 4, hipMemcpyDeviceToDevice, hs));
    else
        hipLaunchKernelGGL(k_zero, dim3(1), dim3(256), 0, hs, st->b3, (int64_t)d.C);
    LAUNCH_CHECK("b3");
    ts3_status s = prep_z(st, hs);  // folds b3 into the prepared Z
    if (s != TS3_OK) return s;
    st->sf_ready = false;
    if (st->k.pass2sf && st->sfp && st->w3p) {
        // operands of the slice-state pass 2: s'^T and W3^T fragments
        const int64_t nsf = (int64_t)d.H * d.M * 16, nw3 = (int64_t)d.C * d.C;
        hipLaunchKernelGGL(k_prep_sf<bf16_t>, dim3((unsigned)std::min<int64_t>((nsf + 255) / 256, 1024)), dim3(256),
                           0, hs, st->s1, d.H, d.M, (bf16_t *)st->sfp);
        hipLaunchKernelGGL(k_prep_w3f<bf16_t>, dim3((unsigned)std::min<int64_t>((nw3 + 255) / 256, 1024)),
                           dim3(256), 0, hs, w->W3, d.C, (bf16_t *)st->w3p);
        LAUNCH_CHECK("prep_sf");
        st->sf_ready = true;
    }
    st->phase = PH_ATTEND;
    return TS3_OK;
}

ts3_status ts3_deslice(const ts3_state *st, const ts3_weights *w, const void *x_chunk, int64_t n_chunk,
                       void *out_chunk, void *stream) {
    if (!st) return fail(TS3_ERR_INVALID_ARG, "state is NULL");
    ts3_status s = check_weights_w2(w);
    if (s != TS3_OK) return s;
    if (st->phase != PH_ATTEND) return fail(TS3_ERR_BAD_STATE, "deslice needs the cached state (attention)");
    if (!same_w2(st, w)) return fail(TS3_ERR_INVALID_ARG, "W2/b2 differ from the ones recorded for this state");
    if (n_chunk < 0) return fail(TS3_ERR_INVALID_ARG, "negative n_chunk");
    if (n_chunk == 0) return TS3_OK;
    if (!x_chunk || !out_chunk) return fail(TS3_ERR_INVALID_ARG, "x_chunk or out_chunk is NULL");
    if (((uintptr_t)x_chunk & 15) || ((uintptr_t)out_chunk & 15))
        return fail(TS3_ERR_INVALID_ARG, "x_chunk and out_chunk must be 16-byte aligned");
    const ts3_desc &d = st->desc;
    if (n_chunk > ((int64_t)INT32_MAX) * 64) return fail(TS3_ERR_INVALID_ARG, "n_chunk too large for one launch");
    const hipError_t le =
        st->k.pass2sf && st->sf_ready
            ? st->k.pass2sf(x_chunk, n_chunk, st->w2p, st->b2s, st->sfp, st->w3p, st->b3, out_chunk,
                            (hipStream_t)stream)
            : st->k.pass2(x_chunk, n_chunk, d.H, d.C, d.M, st->w2p, st->b2s, st->zp, out_chunk, (hipStream_t)stream);
    if (le != hipSuccess) return fail(TS3_ERR_HIP, "deslice LDS setup: %s", hipGetErrorString(le));
    LAUNCH_CHECK("deslice");
    return TS3_OK;
}

namespace {

// The second stream starts after everything enqueued on `main` so far.
ts3_status fork_aux(ts3_state *st, hipStream_t main, bool *forked) {
    HIP_TRY(hipEventRecord(st->ev_fork, main));
    HIP_TRY(hipStreamWaitEvent(st->aux, st->ev_fork, 0));
    *forked = true;
    return TS3_OK;
}

// Later work on `main` waits for everything enqueued on the second stream
// (also after an error, so nothing is left running unordered).
ts3_status join_aux(ts3_state *st, hipStream_t main, ts3_status s) {
    hipError_t e = hipEventRecord(st->ev_join, st->aux);
    if (e == hipSuccess) e = hipStreamWaitEvent(main, st->ev_join, 0);
    if (e != hipSuccess && s == TS3_OK) return fail(TS3_ERR_HIP, "stream join: %s", hipGetErrorString(e));
    return s;
}

}  // namespace

ts3_status ts3_layer_forward(ts3_state *st, const ts3_weights *w, const void *x, int64_t N, int64_t tile,
                             int64_t chunk, void *out, void *stream) {
    if (!st) return fail(TS3_ERR_INVALID_ARG, "state is NULL");
    if (N < 0 || tile <= 0 || chunk <= 0) return fail(TS3_ERR_INVALID_ARG, "N >= 0, tile > 0, chunk > 0 required");
    if (tile % st->desc.group_span != 0)
        return fail(TS3_ERR_INVALID_ARG, "tile %lld is not a multiple of group_span %lld", (long long)tile,
                    (long long)st->desc.group_span);
    if (N > 0 && (!x || !out)) return fail(TS3_ERR_INVALID_ARG, "x or out is NULL");
    ts3_status s = ts3_state_reset(st, stream);
    if (s == TS3_OK) s = check_weights_w2(w);
    const char *xb = (const char *)x;
    char *ob = (char *)out;
    const int64_t row = (int64_t)st->desc.C * st->esize;
    hipStream_t main = (hipStream_t)stream;
    // W2' is prepared once on the caller's stream, before either stream reads it.
    if (s == TS3_OK) s = prep_w2(st, w, main);
    // Pass-1 tiles write disjoint group partials and pass-2 chunks disjoint
    // output rows, so each loop runs its launches alternately on the caller's
    // stream and the second one, forked from and joined back into the caller's.
    bool forked = false;
    if (s == TS3_OK && N > tile) s = fork_aux(st, main, &forked);
    for (int64_t t0 = 0, i = 0; s == TS3_OK && t0 < N; t0 += tile, ++i)
        s = ts3_slice_accumulate(st, w, xb + t0 * row, std::min(tile, N - t0), t0, (i & 1) ? st->aux : main);
    if (forked) s = join_aux(st, main, s);
    if (s == TS3_OK) s = ts3_slice_finalize(st, w, stream);
    if (s == TS3_OK) s = ts3_token_attention(st, w, stream);
    forked = false;
    if (s == TS3_OK && N > chunk) s = fork_aux(st, main, &forked);
    for (int64_t c0 = 0, i = 0; s == TS3_OK && c0 < N; c0 += chunk, ++i)
        s = ts3_deslice(st, w, xb + c0 * row, std::min(chunk, N - c0), ob + c0 * row, (i & 1) ? st->aux : main);
    if (forked) s = join_aux(st, main, s);
    return s;
}


ts3_status ts3_layer_backward(ts3_state *st, const ts3_weights *w, const void *x, const void *g, int64_t N,
                              int64_t tile, void *dx, const ts3_grads *gr, void *stream) {
    if (!st) return fail(TS3_ERR_INVALID_ARG, "state is NULL");
    if (!w || !w->W2 || !w->W1 || !w->Wq || !w->Wk || !w->Wv || !w->W3)
        return fail(TS3_ERR_INVALID_ARG, "weights or a weight matrix is NULL");
    if (!gr || !gr->dW2 || !gr->db2 || !gr->dW1 || !gr->db1 || !gr->dWq || !gr->dWk || !gr->dWv || !gr->dW3 ||
        !gr->db3)
        return fail(TS3_ERR_INVALID_ARG, "grads or one of its pointers is NULL");
    const ts3_desc &d = st->desc;
    if (d.io_dtype != TS3_FP32 || !st->k.bw_head || !st->k.bw_dx)
        return fail(TS3_ERR_UNSUPPORTED, "the backward is built for float32 storage with C in {64, 128} and "
                    "M in {16, 32, 64}");
    if (N <= 0 || tile <= 0) return fail(TS3_ERR_INVALID_ARG, "N > 0 and tile > 0 required");
    if (tile % d.group_span != 0)
        return fail(TS3_ERR_INVALID_ARG, "tile %lld is not a multiple of group_span %lld", (long long)tile,
                    (long long)d.group_span);
    if (N > d.max_points) return fail(TS3_ERR_INVALID_ARG, "N exceeds max_points");
    if (!x || !g || !dx) return fail(TS3_ERR_INVALID_ARG, "x, g or dx is NULL");
    if (((uintptr_t)x & 15) || ((uintptr_t)g & 15) || ((uintptr_t)dx & 15))
        return fail(TS3_ERR_INVALID_ARG, "x, g and dx must be 16-byte aligned");
    const int64_t Q = d.group_span;
    const int64_t nspan_all = (N + Q - 1) / Q;
    if (st->phase != PH_ATTEND || st->span_hi != nspan_all)
        return fail(TS3_ERR_BAD_STATE, "backward needs the state of the forward over the same %lld points",
                    (long long)N);
    if (!same_w2(st, w)) return fail(TS3_ERR_INVALID_ARG, "W2/b2 differ from the ones of the forward");
    hipStream_t hs = (hipStream_t)stream;
    const float inv_tau = 1.f / d.temperature;
    const int64_t HM = (int64_t)d.H * d.M;
    const float *xf = (const float *)x, *gf = (const float *)g;
    const float *w2p = (const float *)st->w2p;
    const int64_t nt_max = std::min(tile, N);
    if (st->bdz_points < nt_max) {
        // dz of one tile, [H][points][M]; kept by the state for later calls
        if (st->bdz) {
            HIP_TRY(hipStreamSynchronize(hs));
            (void)hipFree(st->bdz);
            st->bdz = nullptr;
            st->bytes -= st->bdz_points * HM * 4;
            st->bdz_points = 0;
        }
        const size_t bytes = (size_t)(nt_max * HM * 4);
        hipError_t e = hipMalloc((void **)&st->bdz, bytes);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            st->bdz = nullptr;
            return fail(e == hipErrorOutOfMemory ? TS3_ERR_OUT_OF_MEMORY : TS3_ERR_HIP,
                        "hipMalloc(%zu bytes) for the backward's dz: %s", bytes, hipGetErrorString(e));
        }
        st->bdz_points = nt_max;
        st->bytes += (int64_t)bytes;
    }
    // dZ = sum_i w_i^T g_i (its column C, sum_i w_i, is not needed)
    st->partials_fwd = false;  // the backward passes reuse the span partial buffer
    for (int64_t t0 = 0; t0 < N; t0 += tile) {
        const int64_t nt = std::min(tile, N - t0);
        st->k.bw_head(xf + t0 * d.C, gf + t0 * d.C, nt, t0 / Q, (int32_t)Q, (int32_t)((nt + Q - 1) / Q), d.H, w2p,
                      st->b2s, st->partials, hs);
        LAUNCH_CHECK("backward dZ pass");
    }
    ts3_status s = fold_partials(st, nspan_all, d.C, st->bdZ, st->bdd, hs);
    if (s != TS3_OK) return s;
    // token side: ds_raw, dd and the Linear1 / attention / Linear3 gradients
    const size_t lds = (size_t)(2 * d.M * d.C + 10 * d.M * d.dh + 2 * d.M * d.M) * 4;
    if (lds > (size_t)ATTN_LDS_MAX) return fail(TS3_ERR_UNSUPPORTED, "token backward needs %zu bytes of LDS", lds);
    HIP_TRY(hipFuncSetAttribute((const void *)k_bw_token, hipFuncAttributeMaxDynamicSharedMemorySize, ATTN_LDS_MAX));
    hipLaunchKernelGGL(k_bw_token, dim3(d.H), dim3(256), lds, hs, st->s_raw, st->dsum, st->s, st->s1, st->bdZ,
                       w->W1, w->Wq, w->Wk, w->Wv, w->W3, d.C, d.H, d.M, d.dh, d.eps, st->bdsr, st->bdsT, st->bdd,
                       gr->dW1, gr->db1, gr->dWq, gr->dWk, gr->dWv, gr->dW3, gr->db3);
    LAUNCH_CHECK("token backward");
    // Per tile: dx (which stores dz), then the tile's span partials of dW2^T
    // and db2 from the stored dz.
    for (int64_t t0 = 0; t0 < N; t0 += tile) {
        const int64_t nt = std::min(tile, N - t0);
        st->k.bw_dx(xf + t0 * d.C, gf + t0 * d.C, nt, d.H, w2p, st->b2s, w->W2, st->Z, st->bdsr, st->bdsT, st->bdd,
                    inv_tau, (float *)dx + t0 * d.C, st->bdz, hs);
        LAUNCH_CHECK("backward dx pass");
        st->k.bw_dw2(xf + t0 * d.C, st->bdz, nt, t0 / Q, (int32_t)Q, (int32_t)((nt + Q - 1) / Q), d.H,
                     st->partials, hs);
        LAUNCH_CHECK("backward dW2 pass");
    }
    s = fold_partials(st, nspan_all, d.C, st->bdW2T, gr->db2, hs);
    if (s != TS3_OK) return s;
    hipLaunchKernelGGL(k_bw_transpose_w2, dim3((unsigned)std::min<int64_t>((d.C * HM + 255) / 256, 4096)), dim3(256),
                       0, hs, st->bdW2T, d.C, (int)HM, gr->dW2);
    LAUNCH_CHECK("dW2 transpose");
    return TS3_OK;
}

ts3_status ts3_state_projected(const ts3_state *st, int32_t *projected) {
    if (!st || !projected) return fail(TS3_ERR_INVALID_ARG, "NULL argument");
    *projected = st->proj ? 1 : 0;
    return TS3_OK;
}

ts3_status ts3_state_get(const ts3_state *st, int32_t which, float *host_dst, int64_t n, void *stream) {
    if (!st || !host_dst) return fail(TS3_ERR_INVALID_ARG, "NULL argument");
    const ts3_desc &d = st->desc;
    const int64_t HM = (int64_t)d.H * d.M;
    const float *src = nullptr;
    int64_t size = 0;
    int need = PH_FINAL;
    switch (which) {
        case TS3_S_RAW:
            if (st->proj) return fail(TS3_ERR_UNSUPPORTED, "this state accumulates projected sums: read TS3_T_RAW");
            src = st->s_raw;
            size = HM * d.C;
            break;
        case TS3_T_RAW:
            if (!st->proj) return fail(TS3_ERR_UNSUPPORTED, "this state accumulates unprojected sums: read TS3_S_RAW");
            src = st->s_raw;
            size = HM * 16;
            break;
        case TS3_D: src = st->dsum; size = HM; break;
        case TS3_S: src = st->s; size = HM * d.dh; break;
        case TS3_S1: src = st->s1; size = HM * d.dh; need = PH_ATTEND; break;
        case TS3_ZP: src = st->Z; size = HM * d.C; need = PH_ATTEND; break;
        default: return fail(TS3_ERR_INVALID_ARG, "unknown buffer %d", which);
    }
    if (n != size) return fail(TS3_ERR_INVALID_ARG, "buffer %d holds %lld floats, not %lld", which,
                                (long long)size, (long long)n);
    if (st->phase < need) return fail(TS3_ERR_BAD_STATE, "buffer %d is not computed yet", which);
    hipStream_t hs = (hipStream_t)stream;
    HIP_TRY(hipMemcpyAsync(host_dst, src, (size_t)size * 4, hipMemcpyDeviceToHost, hs));
    HIP_TRY(hipStreamSynchronize(hs));
    return TS3_OK;
}

ts3_status ts3_state_get_spans(const ts3_state *st, int64_t span0, int64_t nspan, float *host_dst, int64_t n,
                               void *stream) {
    if (!st || !host_dst) return fail(TS3_ERR_INVALID_ARG, "NULL argument");
    if (span0 < 0 || nspan <= 0 || span0 + nspan > st->nspan_max)
        return fail(TS3_ERR_INVALID_ARG, "spans [%lld, %lld) outside the state's %lld spans", (long long)span0,
                    (long long)(span0 + nspan), (long long)st->nspan_max);
    if (n != nspan * st->E)
        return fail(TS3_ERR_INVALID_ARG, "%lld spans hold %lld floats, not %lld", (long long)nspan,
                    (long long)(nspan * st->E), (long long)n);
    if (!st->partials_fwd) return fail(TS3_ERR_BAD_STATE, "no pass-1 span partials (reset, or a backward ran)");
    for (int64_t i = span0; i < span0 + nspan; ++i)
        if (!st->span_written[(size_t)i])
            return fail(TS3_ERR_BAD_STATE, "span %lld has not been accumulated", (long long)i);
    hipStream_t hs = (hipStream_t)stream;
    HIP_TRY(hipMemcpyAsync(host_dst, st->partials + span0 * st->E, (size_t)n * 4, hipMemcpyDeviceToHost, hs));
    HIP_TRY(hipStreamSynchronize(hs));
    return TS3_OK;
}

ts3_status ts3_state_set(ts3_state *st, const ts3_weights *w, int32_t which, const float *host_src, int64_t n,
                         const float *host_b3, void *stream) {
    if (!st || !host_src) return fail(TS3_ERR_INVALID_ARG, "NULL argument");
    ts3_status s = check_weights_w2(w);
    if (s != TS3_OK) return s;
    if (which != TS3_ZP) return fail(TS3_ERR_INVALID_ARG, "only TS3_ZP can be set");
    const ts3_desc &d = st->desc;
    const int64_t size = (int64_t)d.H * d.M * d.C;
    if (n != size) return fail(TS3_ERR_INVALID_ARG, "Z holds %lld floats, not %lld", (long long)size, (long long)n);
    hipStream_t hs = (hipStream_t)stream;
    HIP_TRY(hipMemcpyAsync(st->Z, host_src, (size_t)size * 4, hipMemcpyHostToDevice, hs));
    std::vector<float> b3(d.C, 0.f);
    if (host_b3) std::memcpy(b3.data(), host_b3, (size_t)d.C * 4);
    HIP_TRY(hipMemcpyAsync(st->b3, b3.data(), (size_t)d.C * 4, hipMemcpyHostToDevice, hs));
    s = prep_z(st, hs);
    if (s == TS3_OK) s = prep_w2(st, w, hs);
    if (s != TS3_OK) return s;
    HIP_TRY(hipStreamSynchronize(hs));
    st->sf_ready = false;  // an injected Z need not factor as s' W3: decode in the cached-Z form
    st->phase = PH_ATTEND;
    return TS3_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Layer forward without allocation (ts3_layer_forward_noalloc).  Every buffer
// the layer needs beyond x, out and the weights lives in one file-scope device
// array.  Its device address is looked up once per device; host code uses only
// that address, never the array's name, which in host code is a stand-in and
// not a device pointer.
namespace {

constexpr size_t SCRATCH_BYTES = size_t(64) << 20;
constexpr int SCRATCH_MAX_DEVICES = 64;
static __device__ __align__(256) unsigned char scratch[SCRATCH_BYTES];

std::once_flag g_scratch_once[SCRATCH_MAX_DEVICES];
void *g_scratch_ptr[SCRATCH_MAX_DEVICES];
hipError_t g_scratch_err[SCRATCH_MAX_DEVICES];

// The current device's copy of the array (each device holds its own).
ts3_status scratch_base(void **out) {
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= SCRATCH_MAX_DEVICES)
        return fail(TS3_ERR_UNSUPPORTED, "device %d: the no-allocation path serves devices 0..%d", dev,
                    SCRATCH_MAX_DEVICES - 1);
    std::call_once(g_scratch_once[dev], [dev] {
        g_scratch_err[dev] = hipGetSymbolAddress(&g_scratch_ptr[dev], HIP_SYMBOL(scratch));
    });
    if (g_scratch_err[dev] != hipSuccess)
        return fail(TS3_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                    hipGetErrorString(g_scratch_err[dev]));
    *out = g_scratch_ptr[dev];
    return TS3_OK;
}

// Byte layout of the scratch array for one call (each region 256-aligned).
struct ScratchLayout {
    size_t partials, runs, s_raw, dsum, s, s1, Z, b2s, b3, w2p, zp, sfp, w3p, w1p, total;
};

ScratchLayout scratch_layout(const ts3_desc &d, int64_t N, int64_t tile) {
    auto up = [](size_t b) { return (b + 255) & ~size_t(255); };
    const int64_t HM = (int64_t)d.H * d.M;
    Kernels k;
    find_any_kernels(d.io_dtype, d.C, d.M, &k);
    const bool proj = k.pass1p && d.H * 16 == d.C;  // the projected pass 1, as for a state
    const int64_t E = HM * ((proj ? 16 : d.C) + 1);
    const int64_t Q = d.group_span;
    const int64_t tile_spans = (std::min<int64_t>(tile, std::max<int64_t>(N, 1)) + Q - 1) / Q;
    // An empty mesh still folds one (zero) span.
    const int64_t nrun = (std::max<int64_t>((N + Q - 1) / Q, 1) + FOLD - 1) / FOLD;
    const int esize = d.io_dtype == TS3_BF16 ? 2 : 4;
    ScratchLayout L{};
    size_t at = 0;
    auto take = [&](size_t &field, size_t bytes) { field = at; at += up(bytes); };
    take(L.partials, (size_t)(tile_spans * E) * 4);
    take(L.runs, (size_t)(nrun * E) * (d.accum == TS3_ACCUM_FP64 ? 8 : 4));
    take(L.s_raw, (size_t)(HM * d.C) * 4);
    take(L.dsum, (size_t)HM * 4);
    take(L.s, (size_t)(HM * d.dh) * 4);
    take(L.s1, (size_t)(HM * d.dh) * 4);
    take(L.Z, (size_t)(HM * d.C) * 4);
    take(L.b2s, (size_t)HM * 4);
    take(L.b3, (size_t)d.C * 4);
    take(L.w2p, (size_t)w2p_elems(d) * esize);
    take(L.zp, (size_t)zp_elems(d, k.rt) * esize);
    const bool sf = k.pass2sf && d.H * 16 == d.C;  // the slice-state pass 2, as for a state
    take(L.sfp, sf ? (size_t)HM * 16 * 2 : 0);
    take(L.w3p, sf ? (size_t)d.C * d.C * 2 : 0);
    take(L.w1p, proj ? (size_t)d.C * d.C * 4 : 0);
    L.total = at;
    return L;
}

template <typename T>
void fold_tile(const float *partials, int64_t E, int64_t g0, int64_t ns, void *runs, hipStream_t hs) {
    const int64_t r_first = g0 / FOLD, r_last = (g0 + ns - 1) / FOLD;
    hipLaunchKernelGGL(k_fold_runs_tile<T>, dim3((unsigned)((E + 255) / 256), (unsigned)(r_last - r_first + 1)),
                       dim3(256), 0, hs, partials, E, g0, ns, (T *)runs);
}

}  // namespace

extern "C" {

ts3_status ts3_layer_forward_noalloc(const ts3_desc *desc, const ts3_weights *w, const void *x, int64_t N,
                                     int64_t tile, int64_t chunk, void *out, void *stream) {
    ts3_status s = check_desc(desc);
    if (s != TS3_OK) return s;
    s = check_weights_w2(w);
    if (s != TS3_OK) return s;
    if (!w->W1 || !w->Wq || !w->Wk || !w->Wv || !w->W3)
        return fail(TS3_ERR_INVALID_ARG, "W1, Wq, Wk, Wv or W3 is NULL");
    const ts3_desc &d = *desc;
    if (N < 0 || tile <= 0 || chunk <= 0) return fail(TS3_ERR_INVALID_ARG, "N >= 0, tile > 0, chunk > 0 required");
    if (tile % d.group_span != 0)
        return fail(TS3_ERR_INVALID_ARG, "tile %lld is not a multiple of group_span %lld", (long long)tile,
                    (long long)d.group_span);
    if (N > 0 && (!x || !out)) return fail(TS3_ERR_INVALID_ARG, "x or out is NULL");
    if (((uintptr_t)x & 15) || ((uintptr_t)out & 15))
        return fail(TS3_ERR_INVALID_ARG, "x and out must be 16-byte aligned");
    if (N > ((int64_t)INT32_MAX) * 64) return fail(TS3_ERR_INVALID_ARG, "N too large");
    const ScratchLayout lay = scratch_layout(d, N, tile);
    if (lay.total > SCRATCH_BYTES)
        return fail(TS3_ERR_INVALID_ARG,
                    "this call needs %llu bytes of scratch (span partials of one %lld-point tile and the run sums "
                    "of %lld points); the fixed maximum is %llu bytes: use fewer points, smaller tiles or a "
                    "larger group_span, or ts3_layer_forward",
                    (unsigned long long)lay.total, (long long)tile, (long long)N,
                    (unsigned long long)SCRATCH_BYTES);
    void *base = nullptr;
    s = scratch_base(&base);
    if (s != TS3_OK) return s;
    unsigned char *b = (unsigned char *)base;
    // A state on the host stack whose device buffers are regions of the array;
    // it owns nothing and is never freed.
    ts3_state st;
    st.desc = d;
    find_any_kernels(d.io_dtype, d.C, d.M, &st.k);
    st.esize = d.io_dtype == TS3_BF16 ? 2 : 4;
    st.proj = st.k.pass1p && d.H * 16 == d.C;
    st.rowc = st.proj ? 16 : d.C;
    st.E = (int64_t)d.H * d.M * (st.rowc + 1);
    st.w1p = st.proj ? b + lay.w1p : nullptr;
    st.partials = (float *)(b + lay.partials);
    st.runs = (float *)(b + lay.runs);
    st.s_raw = (float *)(b + lay.s_raw);
    st.dsum = (float *)(b + lay.dsum);
    st.s = (float *)(b + lay.s);
    st.s1 = (float *)(b + lay.s1);
    st.Z = (float *)(b + lay.Z);
    st.b2s = (float *)(b + lay.b2s);
    st.b3 = (float *)(b + lay.b3);
    st.w2p = b + lay.w2p;
    st.zp = b + lay.zp;
    if (st.k.pass2sf && d.H * 16 == d.C) {
        st.sfp = b + lay.sfp;
        st.w3p = b + lay.w3p;
    } else {
        st.k.pass2sf = nullptr;
    }
    hipStream_t hs = (hipStream_t)stream;
    const int64_t Q = d.group_span;
    const int64_t E = st.E;
    const int64_t nspan = std::max<int64_t>((N + Q - 1) / Q, 1);
    const int64_t nrun = (nspan + FOLD - 1) / FOLD;
    s = prep_w2(&st, w, hs);
    if (s != TS3_OK) return s;
    if (N == 0) {  // an empty mesh: the one span is zero
        hipLaunchKernelGGL(k_zero, dim3((unsigned)((E + 255) / 256)), dim3(256), 0, hs, st.partials, E);
        LAUNCH_CHECK("zero span");
        if (d.accum == TS3_ACCUM_FP64) fold_tile<double>(st.partials, E, 0, 1, st.runs, hs);
        else fold_tile<float>(st.partials, E, 0, 1, st.runs, hs);
        LAUNCH_CHECK("fold");
    }
    // Pass 1 tile by tile on the caller's stream: the tile's spans go to the
    // start of the partial region, then into their runs.
    for (int64_t t0 = 0; t0 < N; t0 += tile) {
        const int64_t nt = std::min(tile, N - t0);
        const int64_t ns = (nt + Q - 1) / Q;
        if (st.proj)
            st.k.pass1p((const char *)x + t0 * d.C * st.esize, nt, 0, (int32_t)Q, (int32_t)ns, d.H, st.w2p, st.b2s,
                        st.w1p, st.partials, hs);
        else
            st.k.pass1((const char *)x + t0 * d.C * st.esize, nt, 0, (int32_t)Q, (int32_t)ns, d.H, d.C, d.M,
                       st.w2p, st.b2s, st.partials, hs);
        LAUNCH_CHECK("slice_accumulate");
        if (d.accum == TS3_ACCUM_FP64) fold_tile<double>(st.partials, E, t0 / Q, ns, st.runs, hs);
        else fold_tile<float>(st.partials, E, t0 / Q, ns, st.runs, hs);
        LAUNCH_CHECK("fold");
    }
    const unsigned gx = (unsigned)((E + 255) / 256);
    if (d.accum == TS3_ACCUM_FP64)
        hipLaunchKernelGGL(k_fold_final<double>, dim3(gx), dim3(256), 0, hs, (const double *)st.runs, E, nrun,
                           st.rowc, st.s_raw, st.dsum);
    else
        hipLaunchKernelGGL(k_fold_final<float>, dim3(gx), dim3(256), 0, hs, (const float *)st.runs, E, nrun,
                           st.rowc, st.s_raw, st.dsum);
    LAUNCH_CHECK("fold_final");
    if (st.proj)
        hipLaunchKernelGGL(k_finalize_proj, dim3(d.H), dim3(256), 0, hs, st.s_raw, st.dsum, w->b1, d.H, d.M, d.eps,
                           st.s);
    else
        hipLaunchKernelGGL(k_finalize, dim3(d.H * d.M), dim3(64), 0, hs, st.s_raw, st.dsum, w->W1, w->b1, d.C, d.H,
                           d.M, d.dh, d.eps, st.s);
    LAUNCH_CHECK("finalize");
    st.phase = PH_FINAL;
    s = ts3_token_attention(&st, w, stream);
    if (s != TS3_OK) return s;
    for (int64_t c0 = 0; s == TS3_OK && c0 < N; c0 += chunk)
        s = ts3_deslice(&st, w, (const char *)x + c0 * d.C * st.esize, std::min(chunk, N - c0),
                        (char *)out + c0 * d.C * st.esize, stream);
    return s;
}

}  // extern "C"

#include "ts3_stack.h"
