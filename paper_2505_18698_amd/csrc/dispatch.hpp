// Launch helpers and shape dispatch, instantiated once per element type in
// dispatch_{bf16,f16,f32}.hip (split so the kernels compile in parallel).
//
// Launch order for T steps (paper, Implementation paragraph of Sec. 3; R is
// updated before L in every step), one launch per half-step:
//   T == 1 : R(first, final) -> apply
//   T >= 2 : R(first) -> L -> [R -> L] x (T - 2) -> R(final) -> apply
// "first" reads alpha_R straight from Q with c_R = 1 (L^(0) = I); "final" also
// forms Y; apply is the last L half-step fused with O = sum_k L Y.
// For small heads monarch_fused_head runs the same sequence in one workgroup
// per head, with the states in LDS.
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

// ---- one workgroup per head ----
template <typename T, bool RGB, bool RGM> int launch_fused(Launcher &L, const CallBufs &B, ma::HeadDims hd, const CallDims &c)
{
    using U = ma::FusedHead<T, RGB, RGM>;
    // one workgroup per compute unit (its LDS holds one), each looping over heads
    const int64_t grid = c.BH < c.num_cus ? c.BH : c.num_cus;
    hd.units = c.BH;
    const ma::Bufs<T> p = typed<T>(B);
    const int64_t BH = c.BH;
    const int T_ = c.T;
    return L.run(kFused, [&] {
        return launched([&] {
            hipLaunchKernelGGL((ma::monarch_fused_head<T, RGB, RGM>), dim3((unsigned)grid), dim3(64 * U::NW), 0,
                               L.stream, p, hd, BH, T_);
        });
    });
}

template <typename T> int run_fused(Launcher &L, const CallBufs &B, ma::HeadDims hd, const CallDims &c)
{
    if constexpr (sizeof(T) != 2) {
        return fail(MA_EUNSUPPORTED, "the fused kernel needs 16-bit elements");
    } else {
        const bool rgb = hd.b != 16, rgm = hd.m != 16;
        if (rgb && rgm) return launch_fused<T, true, true>(L, B, hd, c);
        if (rgb) return launch_fused<T, true, false>(L, B, hd, c);
        if (rgm) return launch_fused<T, false, true>(L, B, hd, c);
        return launch_fused<T, false, false>(L, B, hd, c);
    }
}

template <typename T> int run_call_impl(Launcher &L, const CallBufs &B, const CallDims &c, int path)
{
    const int32_t dtype = std::is_same<T, float>::value ? MA_F32 : std::is_same<T, __bf16>::value ? MA_BF16 : MA_F16;
    ma::HeadDims hd{c.m, c.b, c.s_log2e, 0};
    if (path == kFusedHead && !fused_applies(dtype, c.d, c.m, c.b))
        return fail(MA_EUNSUPPORTED, "the fused kernel needs bf16/fp16, d = 64 and m, b <= 16");
    if (uses_fused(path, dtype, c.d, c.m, c.b)) return run_fused<T>(L, B, hd, c);
    return c.d == 64 ? run_half_steps<T, 64>(L, B, hd, c.BH, c.T) : run_half_steps<T, 128>(L, B, hd, c.BH, c.T);
}

}  // namespace ma_host
