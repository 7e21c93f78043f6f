// Launch helpers and shape dispatch, instantiated once per element type in
// dispatch_{bf16,f16,f32}.hip (split so the kernels compile in parallel).
//
// Launch order for T steps (paper, Implementation paragraph of Sec. 3; R is
// updated before L in every step), one launch per half-step:
//   T == 1 : R(first, final) -> apply
//   T >= 2 : R(first) -> L -> [R -> L] x (T - 2) -> R(final) -> apply
// "first" reads alpha_R straight from Q with c_R = 1 (L^(0) = I); "final" also
// forms Y; apply is the last L half-step fused with O = sum_k L Y.
// The single-launch path runs the same sequence inside monarch_persistent.
#pragma once

#include <type_traits>

#include "host_common.hpp"
#include "ma_kernels.hpp"

namespace ma_host {

template <typename T> ma::Bufs<T> typed(const CallBufs &B)
{
    return ma::Bufs<T>{(const T *)B.q, (const T *)B.k, (const T *)B.v, (T *)B.out, (T *)B.aR, (T *)B.aL, (T *)B.Y,
                       B.cR, B.cL};
}

template <typename F> int launched(F &&f)
{
    f();
    return MA_OK;
}

template <typename T, int NB, int D, bool RG>
int launch_r(Launcher &L, const CallBufs &B, ma::HeadDims hd, int64_t BH, bool first, bool final_)
{
    constexpr int W = ma::Split<NB / 16>::W;
    hd.units = BH * hd.m;
    const dim3 grid((unsigned)hd.units), block(64 * W);
    const ma::Bufs<T> p = typed<T>(B);
    const int kind = final_ ? kRFinal : kR;
    if (first && final_)
        return L.run(kind, [&] { return launched([&] { hipLaunchKernelGGL((ma::r_half_step<T, NB, D, true, true, RG>), grid, block, 0, L.stream, p, hd); }); });
    if (first)
        return L.run(kind, [&] { return launched([&] { hipLaunchKernelGGL((ma::r_half_step<T, NB, D, true, false, RG>), grid, block, 0, L.stream, p, hd); }); });
    if (final_)
        return L.run(kind, [&] { return launched([&] { hipLaunchKernelGGL((ma::r_half_step<T, NB, D, false, true, RG>), grid, block, 0, L.stream, p, hd); }); });
    return L.run(kind, [&] { return launched([&] { hipLaunchKernelGGL((ma::r_half_step<T, NB, D, false, false, RG>), grid, block, 0, L.stream, p, hd); }); });
}

template <typename T, int NM, int D, bool RG>
int launch_l(Launcher &L, const CallBufs &B, ma::HeadDims hd, int64_t BH, bool apply)
{
    constexpr int W = ma::Split<NM / 16>::W;
    hd.units = BH * hd.b;
    const dim3 grid((unsigned)hd.units), block(64 * W);
    const ma::Bufs<T> p = typed<T>(B);
    if (apply)
        return L.run(kApply, [&] { return launched([&] { hipLaunchKernelGGL((ma::monarch_apply<T, NM, D, RG>), grid, block, 0, L.stream, p, hd); }); });
    return L.run(kL, [&] { return launched([&] { hipLaunchKernelGGL((ma::l_half_step<T, NM, D, RG>), grid, block, 0, L.stream, p, hd); }); });
}

template <typename T, int D, int NB>
int dispatch_r(Launcher &L, const CallBufs &B, ma::HeadDims hd, int64_t BH, bool first, bool final_)
{
    if constexpr (std::is_same<T, float>::value && NB * D > 8192) {
        return fail(MA_EUNSUPPORTED, "fp32 tile too large");
    } else {
        return hd.b != NB ? launch_r<T, NB, D, true>(L, B, hd, BH, first, final_)
                          : launch_r<T, NB, D, false>(L, B, hd, BH, first, final_);
    }
}

template <typename T, int D, int NM>
int dispatch_l(Launcher &L, const CallBufs &B, ma::HeadDims hd, int64_t BH, bool apply)
{
    if constexpr (std::is_same<T, float>::value && NM * D > 8192) {
        return fail(MA_EUNSUPPORTED, "fp32 tile too large");
    } else {
        return hd.m != NM ? launch_l<T, NM, D, true>(L, B, hd, BH, apply)
                          : launch_l<T, NM, D, false>(L, B, hd, BH, apply);
    }
}

// Tile size (16, 32, 64 or 128 rows) used for a block of n <= 128 rows.
inline int tile_rows(int n)
{
    const int p = pad16(n);
    return p <= 16 ? 16 : p <= 32 ? 32 : p <= 64 ? 64 : 128;
}

template <typename T, int D>
int r_step(Launcher &L, const CallBufs &B, ma::HeadDims hd, int64_t BH, bool first, bool final_)
{
    switch (tile_rows(hd.b)) {
    case 16: return dispatch_r<T, D, 16>(L, B, hd, BH, first, final_);
    case 32: return dispatch_r<T, D, 32>(L, B, hd, BH, first, final_);
    case 64: return dispatch_r<T, D, 64>(L, B, hd, BH, first, final_);
    default: return dispatch_r<T, D, 128>(L, B, hd, BH, first, final_);
    }
}

template <typename T, int D>
int l_step(Launcher &L, const CallBufs &B, ma::HeadDims hd, int64_t BH, bool apply)
{
    switch (tile_rows(hd.m)) {
    case 16: return dispatch_l<T, D, 16>(L, B, hd, BH, apply);
    case 32: return dispatch_l<T, D, 32>(L, B, hd, BH, apply);
    case 64: return dispatch_l<T, D, 64>(L, B, hd, BH, apply);
    default: return dispatch_l<T, D, 128>(L, B, hd, BH, apply);
    }
}

template <typename T, int D>
int run_half_steps(Launcher &L, const CallBufs &B, ma::HeadDims hd, int64_t BH, int T_)
{
    int rc;
    for (int t = 1; t <= T_; ++t) {
        const bool first = (t == 1), last = (t == T_);
        if ((rc = r_step<T, D>(L, B, hd, BH, first, last)) != MA_OK) return rc;
        if ((rc = l_step<T, D>(L, B, hd, BH, last)) != MA_OK) return rc;
    }
    return MA_OK;
}

// ---- single launch ----
// Returns MA_EUNSUPPORTED (nothing enqueued) when the cooperative launch is
// not possible, so that the caller can fall back to the half-step launches.
template <typename T, int NT, int D, bool RGB, bool RGM>
int launch_persistent(Launcher &L, const CallBufs &B, ma::HeadDims hd, const CallDims &c)
{
    using P = ma::Persistent<T, NT, NT, D, RGB, RGM>;
    auto kern = ma::monarch_persistent<T, NT, NT, D, RGB, RGM>;
    static int per_cu = -1;  // co-resident workgroups per CU, queried once
    if (per_cu < 0) {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kern, 64 * P::W, 0) != hipSuccess) {
            (void)hipGetLastError();
            nb = 0;
        }
        per_cu = nb;
    }
    if (per_cu < 1 || c.num_cus < 1) return fail(MA_EUNSUPPORTED, "single launch: no co-resident workgroups");
    // no more workgroups per XCD than the units of one phase on that XCD
    const int64_t heads_per_xcd = (c.BH + 7) / 8;
    const int64_t units = heads_per_xcd * (hd.m > hd.b ? hd.m : hd.b);
    const int64_t cap = (int64_t)per_cu * c.num_cus;
    const unsigned grid = (unsigned)(units * 8 < cap ? units * 8 : cap);
    ma::Bufs<T> p = typed<T>(B);
    int64_t BH = c.BH;
    int T_ = c.T;
    ma::SyncState ss{B.sync, B.error, B.state_stride, B.c_stride, 0u};
    void *args[] = {&p, &hd, &BH, &T_, &ss};
    return L.run(kPersistent, [&]() -> int {
        if (hipMemsetAsync(B.sync, 0, kSyncWords * sizeof(unsigned), L.stream) != hipSuccess)
            return fail(MA_EHIP, "hipMemsetAsync of the synchronisation counters failed");
        const hipError_t e = hipLaunchCooperativeKernel((const void *)kern, dim3(grid), dim3(64 * P::W), args, 0, L.stream);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(MA_EUNSUPPORTED, "cooperative launch failed: %s", hipGetErrorString(e));
        }
        return MA_OK;
    });
}

template <typename T, int D, int NT>
int dispatch_persistent(Launcher &L, const CallBufs &B, ma::HeadDims hd, const CallDims &c)
{
    if constexpr (std::is_same<T, float>::value && NT * D > 8192) {
        return fail(MA_EUNSUPPORTED, "fp32 tile too large");
    } else {
        const bool rgb = hd.b != NT, rgm = hd.m != NT;
        if (rgb && rgm) return launch_persistent<T, NT, D, true, true>(L, B, hd, c);
        if (rgb) return launch_persistent<T, NT, D, true, false>(L, B, hd, c);
        if (rgm) return launch_persistent<T, NT, D, false, true>(L, B, hd, c);
        return launch_persistent<T, NT, D, false, false>(L, B, hd, c);
    }
}

template <typename T, int D>
int run_persistent(Launcher &L, const CallBufs &B, ma::HeadDims hd, const CallDims &c)
{
    if (tile_rows(hd.m) != tile_rows(hd.b)) return fail(MA_EUNSUPPORTED, "single launch needs m and b in one tile class");
    switch (tile_rows(hd.b)) {
    case 16: return dispatch_persistent<T, D, 16>(L, B, hd, c);
    case 32: return dispatch_persistent<T, D, 32>(L, B, hd, c);
    case 64: return dispatch_persistent<T, D, 64>(L, B, hd, c);
    default: return dispatch_persistent<T, D, 128>(L, B, hd, c);
    }
}

template <typename T, int D> int run_call_d(Launcher &L, const CallBufs &B, const CallDims &c, int path)
{
    ma::HeadDims hd{c.m, c.b, c.s_log2e, 0};
    if (path == kSingle) {
        // only on request: measured slower than the half-steps at every shape tried
        if (B.copies < c.T) return fail(MA_EUNSUPPORTED, "single launch supports T <= %d", kMaxSingleT);
        return run_persistent<T, D>(L, B, hd, c);
    }
    return run_half_steps<T, D>(L, B, hd, c.BH, c.T);
}

template <typename T> int run_call_impl(Launcher &L, const CallBufs &B, const CallDims &c, int path)
{
    return c.d == 64 ? run_call_d<T, 64>(L, B, c, path) : run_call_d<T, 128>(L, B, c, path);
}

}  // namespace ma_host
