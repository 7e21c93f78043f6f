// Host side of the MonarchAttention C ABI (include/monarch_attn.h): argument
// checks, the per-device workspace, dispatch of the half-step kernels by
// (dtype, d, padded m, padded b), and optional per-launch HIP-event timing.
//
// Launch order for T steps (paper, Implementation paragraph of Sec. 3; R is
// updated before L in every step):
//   T == 1 : R(first, final) -> apply
//   T >= 2 : R(first) -> L -> [R -> L] x (T - 2) -> R(final) -> apply
// "first" reads alpha_R straight from Q with c_R = 1 (L^(0) = I); "final" also
// forms Y; apply is the last L half-step fused with O = sum_k L Y.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "ma_kernels.hpp"
#include "../../include/monarch_attn.h"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

int pad16(int64_t x) { return (int)((x + 15) / 16 * 16); }

size_t elem_bytes(int32_t dtype) { return dtype == MA_F32 ? 4 : 2; }

int check_shape(int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype)
{
    if (dtype != MA_F32 && dtype != MA_BF16 && dtype != MA_F16) return fail(MA_EINVAL, "unknown dtype %d", dtype);
    if (m < 1 || b < 1 || N < 1 || d < 1) return fail(MA_EINVAL, "N, d, m, b must be >= 1");
    if (m * b != N) return fail(MA_EINVAL, "N (%lld) != m (%lld) * b (%lld)", (long long)N, (long long)m, (long long)b);
    if (T < 1) return fail(MA_EINVAL, "T must be >= 1 (got %d)", T);
    if (T > 64) return fail(MA_EUNSUPPORTED, "T > 64 is not supported (got %d)", T);
    if (m > 128 || b > 128) return fail(MA_EUNSUPPORTED, "m and b must be <= 128 (got m=%lld, b=%lld)", (long long)m, (long long)b);
    if (d != 64 && d != 128) return fail(MA_EUNSUPPORTED, "d must be 64 or 128 (got %lld)", (long long)d);
    if (dtype == MA_F32 && ((int64_t)pad16(m) * d > 8192 || (int64_t)pad16(b) * d > 8192))
        return fail(MA_EUNSUPPORTED, "fp32 needs 16*ceil(m/16)*d <= 8192 and 16*ceil(b/16)*d <= 8192");
    return MA_OK;
}

size_t workspace_bytes(int64_t BH, int64_t N, int64_t d, int32_t dtype)
{
    // alpha_R, alpha_L, Y in the element type; c_R, c_L in fp32; 256-byte aligned pieces.
    const size_t st = ((size_t)BH * N * d * elem_bytes(dtype) + 255) / 256 * 256;
    const size_t cs = ((size_t)BH * N * sizeof(float) + 255) / 256 * 256;
    return 3 * st + 2 * cs;
}

struct Workspace {
    void *ptr = nullptr;
    size_t bytes = 0;
};

constexpr int kMaxDevices = 64;
std::mutex g_ws_mutex;
Workspace g_ws[kMaxDevices];

// ---- per-launch timing ----
constexpr int kMaxLaunches = 2 * 64 + 2;
struct Timing {
    bool enabled = false;
    bool ready = false;
    int nlaunch = 0;
    int kind[kMaxLaunches];
    hipEvent_t ev[2 * kMaxLaunches];
    bool created = false;
};
std::mutex g_timing_mutex;
Timing g_timing;

bool overlaps(const void *a, size_t na, const void *b, size_t nb)
{
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

struct Launcher {
    hipStream_t stream;
    bool timed;
    int n = 0;

    template <typename F> int run(int kind, F &&launch)
    {
        if (timed) {
            if (n >= kMaxLaunches) return fail(MA_EHIP, "too many launches to time");
            if (hipEventRecord(g_timing.ev[2 * n], stream) != hipSuccess) return fail(MA_EHIP, "hipEventRecord failed");
        }
        launch();
        if (timed) {
            g_timing.kind[n] = kind;
            if (hipEventRecord(g_timing.ev[2 * n + 1], stream) != hipSuccess) return fail(MA_EHIP, "hipEventRecord failed");
        }
        ++n;
        return MA_OK;
    }
};

struct Bufs {
    const void *q, *k, *v;
    void *out;
    void *aR, *aL, *Y;
    float *cR, *cL;
};

template <typename T, int NB, int D, bool RG>
int launch_r(Launcher &L, const Bufs &B, ma::HeadDims hd, int64_t BH, bool first, bool final_)
{
    constexpr int W = ma::Split<NB / 16>::W;
    hd.units = BH * hd.m;
    const dim3 grid((unsigned)hd.units), block(64 * W);
    const T *q = (const T *)B.q, *k = (const T *)B.k, *v = (const T *)B.v;
    const T *aR = (const T *)B.aR;
    T *aL = (T *)B.aL, *Y = (T *)B.Y;
    const int kind = final_ ? 2 : 0;
    if (first && final_)
        return L.run(kind, [&] { hipLaunchKernelGGL((ma::r_half_step<T, NB, D, true, true, RG>), grid, block, 0, L.stream, q, k, v, aR, B.cR, aL, B.cL, Y, hd); });
    if (first)
        return L.run(kind, [&] { hipLaunchKernelGGL((ma::r_half_step<T, NB, D, true, false, RG>), grid, block, 0, L.stream, q, k, v, aR, B.cR, aL, B.cL, Y, hd); });
    if (final_)
        return L.run(kind, [&] { hipLaunchKernelGGL((ma::r_half_step<T, NB, D, false, true, RG>), grid, block, 0, L.stream, q, k, v, aR, B.cR, aL, B.cL, Y, hd); });
    return L.run(kind, [&] { hipLaunchKernelGGL((ma::r_half_step<T, NB, D, false, false, RG>), grid, block, 0, L.stream, q, k, v, aR, B.cR, aL, B.cL, Y, hd); });
}

template <typename T, int NM, int D, bool RG>
int launch_l(Launcher &L, const Bufs &B, ma::HeadDims hd, int64_t BH, bool apply)
{
    constexpr int W = ma::Split<NM / 16>::W;
    hd.units = BH * hd.b;
    const dim3 grid((unsigned)hd.units), block(64 * W);
    const T *q = (const T *)B.q;
    const T *aL = (const T *)B.aL, *Y = (const T *)B.Y;
    if (apply)
        return L.run(3, [&] { hipLaunchKernelGGL((ma::monarch_apply<T, NM, D, RG>), grid, block, 0, L.stream, q, aL, B.cL, Y, (T *)B.out, hd); });
    return L.run(1, [&] { hipLaunchKernelGGL((ma::l_half_step<T, NM, D, RG>), grid, block, 0, L.stream, q, aL, B.cL, (T *)B.aR, B.cR, hd); });
}

template <typename T, int D, int NB>
int dispatch_r(Launcher &L, const Bufs &B, ma::HeadDims hd, int64_t BH, bool first, bool final_)
{
    if constexpr (std::is_same<T, float>::value && NB * D > 8192) {
        return fail(MA_EUNSUPPORTED, "fp32 tile too large");
    } else {
        return hd.b != NB ? launch_r<T, NB, D, true>(L, B, hd, BH, first, final_)
                         : launch_r<T, NB, D, false>(L, B, hd, BH, first, final_);
    }
}

template <typename T, int D, int NM>
int dispatch_l(Launcher &L, const Bufs &B, ma::HeadDims hd, int64_t BH, bool apply)
{
    if constexpr (std::is_same<T, float>::value && NM * D > 8192) {
        return fail(MA_EUNSUPPORTED, "fp32 tile too large");
    } else {
        return hd.m != NM ? launch_l<T, NM, D, true>(L, B, hd, BH, apply)
                         : launch_l<T, NM, D, false>(L, B, hd, BH, apply);
    }
}

template <typename T, int D>
int r_step(Launcher &L, const Bufs &B, ma::HeadDims hd, int64_t BH, bool first, bool final_)
{
    switch (pad16(hd.b)) {
    case 16: return dispatch_r<T, D, 16>(L, B, hd, BH, first, final_);
    case 32: return dispatch_r<T, D, 32>(L, B, hd, BH, first, final_);
    case 48: return dispatch_r<T, D, 64>(L, B, hd, BH, first, final_);
    case 64: return dispatch_r<T, D, 64>(L, B, hd, BH, first, final_);
    default: return dispatch_r<T, D, 128>(L, B, hd, BH, first, final_);
    }
}

template <typename T, int D>
int l_step(Launcher &L, const Bufs &B, ma::HeadDims hd, int64_t BH, bool apply)
{
    switch (pad16(hd.m)) {
    case 16: return dispatch_l<T, D, 16>(L, B, hd, BH, apply);
    case 32: return dispatch_l<T, D, 32>(L, B, hd, BH, apply);
    case 48: return dispatch_l<T, D, 64>(L, B, hd, BH, apply);
    case 64: return dispatch_l<T, D, 64>(L, B, hd, BH, apply);
    default: return dispatch_l<T, D, 128>(L, B, hd, BH, apply);
    }
}

template <typename T, int D>
int run_all(Launcher &L, const Bufs &B, ma::HeadDims hd, int64_t BH, int T_)
{
    int rc;
    for (int t = 1; t <= T_; ++t) {
        const bool first = (t == 1), last = (t == T_);
        if ((rc = r_step<T, D>(L, B, hd, BH, first, last)) != MA_OK) return rc;
        if ((rc = l_step<T, D>(L, B, hd, BH, last)) != MA_OK) return rc;
    }
    return MA_OK;
}

template <typename T>
int run_dtype(Launcher &L, const Bufs &B, ma::HeadDims hd, int64_t BH, int64_t d, int T_)
{
    return d == 64 ? run_all<T, 64>(L, B, hd, BH, T_) : run_all<T, 128>(L, B, hd, BH, T_);
}

}  // namespace

extern "C" {

const char *monarch_attn_last_error(void) { return g_err; }

int monarch_attn_check(int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype)
{
    g_err[0] = '\0';
    return check_shape(N, d, m, b, T, dtype);
}

size_t monarch_attn_workspace_bytes(int64_t B, int64_t H, int64_t N, int64_t d, int64_t m, int64_t b,
                                    int32_t T, int32_t dtype)
{
    if (B < 1 || H < 1 || check_shape(N, d, m, b, T, dtype) != MA_OK) return 0;
    return workspace_bytes(B * H, N, d, dtype);
}

int monarch_attn_release_workspace(void)
{
    g_err[0] = '\0';
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return fail(MA_EHIP, "hipGetDevice failed");
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    if (g_ws[dev].ptr) {
        if (hipDeviceSynchronize() != hipSuccess || hipFree(g_ws[dev].ptr) != hipSuccess)
            return fail(MA_EHIP, "freeing the workspace failed");
    }
    g_ws[dev] = Workspace{};
    return MA_OK;
}

int monarch_attn_timing_enable(int32_t flag)
{
    g_err[0] = '\0';
    std::lock_guard<std::mutex> lock(g_timing_mutex);
    if (flag && !g_timing.created) {
        for (int i = 0; i < 2 * kMaxLaunches; ++i) {
            if (hipEventCreate(&g_timing.ev[i]) != hipSuccess) return fail(MA_EHIP, "hipEventCreate failed");
        }
        g_timing.created = true;
    }
    g_timing.enabled = flag != 0;
    g_timing.ready = false;
    return MA_OK;
}

int32_t monarch_attn_timing_read(float *ms, int32_t *kind, int32_t cap)
{
    g_err[0] = '\0';
    std::lock_guard<std::mutex> lock(g_timing_mutex);
    if (!g_timing.ready) {
        fail(MA_EINVAL, "no timed call to read");
        return -1;
    }
    const int n = g_timing.nlaunch;
    if (hipEventSynchronize(g_timing.ev[2 * n - 1]) != hipSuccess) {
        fail(MA_EHIP, "hipEventSynchronize failed");
        return -1;
    }
    for (int i = 0; i < n && i < cap; ++i) {
        float t = 0.f;
        if (hipEventElapsedTime(&t, g_timing.ev[2 * i], g_timing.ev[2 * i + 1]) != hipSuccess) {
            fail(MA_EHIP, "hipEventElapsedTime failed");
            return -1;
        }
        if (ms) ms[i] = t;
        if (kind) kind[i] = g_timing.kind[i];
    }
    return n;
}

int monarch_attn_fwd(const void *q, const void *k, const void *v, void *out, int64_t B, int64_t H, int64_t N,
                     int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype, void *stream)
{
    g_err[0] = '\0';
    if (!q || !k || !v || !out) return fail(MA_EINVAL, "null tensor pointer");
    if (B < 1 || H < 1) return fail(MA_EINVAL, "B and H must be >= 1");
    int rc = check_shape(N, d, m, b, T, dtype);
    if (rc != MA_OK) return rc;
    if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)out) & 15u)
        return fail(MA_EINVAL, "q, k, v and out must be 16-byte aligned");
    const int64_t BH = B * H;
    if (BH * (int64_t)(m > b ? m : b) > (int64_t)0x7fffffff) return fail(MA_EUNSUPPORTED, "too many heads for one grid");
    const size_t tensor_bytes = (size_t)BH * N * d * elem_bytes(dtype);
    if (overlaps(out, tensor_bytes, q, tensor_bytes) || overlaps(out, tensor_bytes, k, tensor_bytes) ||
        overlaps(out, tensor_bytes, v, tensor_bytes))
        return fail(MA_EINVAL, "out must not overlap q, k or v");

    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return fail(MA_EHIP, "hipGetDevice failed");
    const size_t need = workspace_bytes(BH, N, d, dtype);
    void *ws = nullptr;
    {
        std::lock_guard<std::mutex> lock(g_ws_mutex);
        Workspace &w = g_ws[dev];
        if (w.bytes < need) {
            if (w.ptr) {
                if (hipDeviceSynchronize() != hipSuccess) return fail(MA_EHIP, "hipDeviceSynchronize failed");
                (void)hipFree(w.ptr);
                w = Workspace{};
            }
            void *p = nullptr;
            if (hipMalloc(&p, need) != hipSuccess) {
                (void)hipGetLastError();
                return fail(MA_ENOMEM, "hipMalloc of %zu workspace bytes failed", need);
            }
            w.ptr = p;
            w.bytes = need;
        }
        ws = w.ptr;
    }

    const size_t st = ((size_t)BH * N * d * elem_bytes(dtype) + 255) / 256 * 256;
    const size_t cs = ((size_t)BH * N * sizeof(float) + 255) / 256 * 256;
    char *base = (char *)ws;
    Bufs bufs{q, k, v, out, base, base + st, base + 2 * st, (float *)(base + 3 * st), (float *)(base + 3 * st + cs)};
    ma::HeadDims hd{(int)m, (int)b, (float)(1.4426950408889634 / std::sqrt((double)d)), 0};

    std::unique_lock<std::mutex> tlock(g_timing_mutex);
    Launcher L{(hipStream_t)stream, g_timing.enabled};
    if (!L.timed) tlock.unlock();
    (void)hipGetLastError();  // clear a stale error so the check below is ours
    switch (dtype) {
    case MA_F32: rc = run_dtype<float>(L, bufs, hd, BH, d, T); break;
    case MA_BF16: rc = run_dtype<__bf16>(L, bufs, hd, BH, d, T); break;
    default: rc = run_dtype<_Float16>(L, bufs, hd, BH, d, T); break;
    }
    if (L.timed) {
        g_timing.nlaunch = L.n;
        g_timing.ready = (rc == MA_OK && L.n > 0);
    }
    if (rc != MA_OK) return rc;
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(MA_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
    return MA_OK;
}

}  // extern "C"
