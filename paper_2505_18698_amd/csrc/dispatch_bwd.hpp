// Launches of the gradient (monarch_attn_bwd): the forward half-steps again
// with every step's states kept, then the reverse sweep of backward.hpp.
// Instantiated once per element type in dispatch_{bf16,f16,f32}.hip.
#pragma once

#include "backward.hpp"
#include "dispatch.hpp"

namespace ma_host {

// ---- gradient ----
template <typename T, int S, int D, bool LAST, bool LENS>
int launch_l_bwd(Launcher &L, const ma::BwdBufs<T> &p, const ma::BwdDims &dm, int64_t BH)
{
    const dim3 grid((unsigned)(BH * dm.b)), block(ma::bwd::Geo<S, D, sizeof(T) == 2>::NTH);
    return L.run(kBwdL, [&] {
        return launched([&] {
            if constexpr (ma::bwd::two_per_cu(S, D, sizeof(T)))
                hipLaunchKernelGGL((ma::bwd::l_bwd2<T, S, D, LAST, LENS>), grid, block, 0, L.stream, p, dm);
            else
                hipLaunchKernelGGL((ma::bwd::l_bwd<T, S, D, LAST, LENS>), grid, block, 0, L.stream, p, dm);
        });
    });
}

template <typename T, int S, int D, bool FIRST, bool LAST, bool LENS>
int launch_r_bwd(Launcher &L, const ma::BwdBufs<T> &p, const ma::BwdDims &dm, int64_t BH)
{
    const dim3 grid((unsigned)(BH * dm.m)), block(ma::bwd::Geo<S, D, sizeof(T) == 2>::NTH);
    return L.run(kBwdR, [&] {
        return launched([&] {
            if constexpr (ma::bwd::two_per_cu(S, D, sizeof(T)))
                hipLaunchKernelGGL((ma::bwd::r_bwd2<T, S, D, FIRST, LAST, LENS>), grid, block, 0, L.stream, p, dm);
            else
                hipLaunchKernelGGL((ma::bwd::r_bwd<T, S, D, FIRST, LAST, LENS>), grid, block, 0, L.stream, p, dm);
        });
    });
}

// One launch of the L-update gradient of a step, on tiles of S >= m rows (and
// of the R-update gradient, S >= b): each kernel takes the tile of its own
// dimension.  128-row tiles at D = 128 hold 16-bit unit tiles (16-bit
// elements only, the only ones the forward takes at that size).
template <typename T, int D, bool LENS>
int l_bwd_step(Launcher &L, const ma::BwdBufs<T> &p, const ma::BwdDims &dm, int64_t BH, bool last)
{
    switch (tile_rows(dm.m)) {
    case 16: return last ? launch_l_bwd<T, 16, D, true, LENS>(L, p, dm, BH) : launch_l_bwd<T, 16, D, false, LENS>(L, p, dm, BH);
    case 32: return last ? launch_l_bwd<T, 32, D, true, LENS>(L, p, dm, BH) : launch_l_bwd<T, 32, D, false, LENS>(L, p, dm, BH);
    case 64: return last ? launch_l_bwd<T, 64, D, true, LENS>(L, p, dm, BH) : launch_l_bwd<T, 64, D, false, LENS>(L, p, dm, BH);
    default:
        if constexpr (D == 128 && std::is_same<T, float>::value) {  // the forward takes no such fp32 shape
            return fail(MA_EUNSUPPORTED, "fp32 128-row blocks need d <= 96");
        } else {
            return last ? launch_l_bwd<T, 128, D, true, LENS>(L, p, dm, BH)
                        : launch_l_bwd<T, 128, D, false, LENS>(L, p, dm, BH);
        }
    }
}

template <typename T, int S, int D, bool LENS>
int r_bwd_tile(Launcher &L, const ma::BwdBufs<T> &p, const ma::BwdDims &dm, int64_t BH, bool first, bool last)
{
    if (first)
        return last ? launch_r_bwd<T, S, D, true, true, LENS>(L, p, dm, BH)
                    : launch_r_bwd<T, S, D, true, false, LENS>(L, p, dm, BH);
    return last ? launch_r_bwd<T, S, D, false, true, LENS>(L, p, dm, BH)
                : launch_r_bwd<T, S, D, false, false, LENS>(L, p, dm, BH);
}

template <typename T, int D, bool LENS>
int r_bwd_step(Launcher &L, const ma::BwdBufs<T> &p, const ma::BwdDims &dm, int64_t BH, bool first, bool last)
{
    switch (tile_rows(dm.b)) {
    case 16: return r_bwd_tile<T, 16, D, LENS>(L, p, dm, BH, first, last);
    case 32: return r_bwd_tile<T, 32, D, LENS>(L, p, dm, BH, first, last);
    case 64: return r_bwd_tile<T, 64, D, LENS>(L, p, dm, BH, first, last);
    default:
        if constexpr (D == 128 && std::is_same<T, float>::value) {  // the forward takes no such fp32 shape
            return fail(MA_EUNSUPPORTED, "fp32 128-row blocks need d <= 96");
        } else {
            return r_bwd_tile<T, 128, D, LENS>(L, p, dm, BH, first, last);
        }
    }
}

// The reverse sweep, t = T .. 1: the L update of step t, then its R update.
// LENS: per-sequence lengths (instantiations of their own).
template <typename T, int D, bool LENS> int bwd_sweep_impl(Launcher &L, const BwdCallBufs &B, const CallDims &c)
{
    ma::BwdDims dm{c.m, c.b, c.n, c.d, (float)(1.0 / std::sqrt((double)c.d))};
    dm.lens = B.lens;
    dm.H = (int)c.H;
    ma::BwdBufs<T> p{(const T *)B.q, (const T *)B.k, (const T *)B.v, (const T *)B.dout, nullptr, nullptr,
                     (const T *)B.Y, nullptr, nullptr, B.dQ, B.dK, (T *)B.dq, (T *)B.dk, (T *)B.dv, B.daL, B.dcL,
                     B.dY, B.daR, B.dcR};
    int rc;
    for (int t = c.T; t >= 1; --t) {
        const bool first = t == 1, last = t == c.T;
        p.aL = (const T *)(B.aL + (size_t)(t - 1) * B.st);
        p.cL = B.cL + (size_t)(t - 1) * B.cst;
        p.aR = first ? nullptr : (const T *)(B.aR + (size_t)(t - 2) * B.st);
        p.cR = first ? nullptr : B.cR + (size_t)(t - 2) * B.cst;
        if ((rc = l_bwd_step<T, D, LENS>(L, p, dm, c.BH, last)) != MA_OK) return rc;
        if ((rc = r_bwd_step<T, D, LENS>(L, p, dm, c.BH, first, last)) != MA_OK) return rc;
    }
    return MA_OK;
}

template <typename T, int D> int bwd_sweep(Launcher &L, const BwdCallBufs &B, const CallDims &c)
{
    return B.lens ? bwd_sweep_impl<T, D, true>(L, B, c) : bwd_sweep_impl<T, D, false>(L, B, c);
}

// The forward half-steps again, each step's states to buffers of their own,
// then the reverse sweep.  States with rows of d elements; every (m, b, d) the
// forward takes.
template <typename T, int D> int run_bwd_d(Launcher &L, const BwdCallBufs &B, const CallDims &c)
{
    ma::HeadDims hd{c.m, c.b, c.n, c.d, c.s_log2e, 0};
    hd.T = c.T;
    hd.lens = B.lens;  // the recompute takes the same per-sequence lengths
    hd.H = (int)c.H;
    int rc;
    for (int t = 1; t <= c.T; ++t) {
        hd.t = t;
        const bool first = t == 1, last = t == c.T;
        const CallBufs r{B.q, B.k, B.v, nullptr,
                         first ? nullptr : B.aR + (size_t)(t - 2) * B.st, B.aL + (size_t)(t - 1) * B.st, B.Y,
                         first ? nullptr : B.cR + (size_t)(t - 2) * B.cst, B.cL + (size_t)(t - 1) * B.cst, nullptr,
                         nullptr};
        if ((rc = r_step<T, D>(L, r, hd, c.BH, c.num_cus, first, last)) != MA_OK) return rc;
        if (last) break;
        const CallBufs l{B.q, B.k, B.v, nullptr, B.aR + (size_t)(t - 1) * B.st, B.aL + (size_t)(t - 1) * B.st, B.Y,
                         B.cR + (size_t)(t - 1) * B.cst, B.cL + (size_t)(t - 1) * B.cst, nullptr, nullptr};
        if ((rc = l_step<T, D>(L, l, hd, c.BH, c.num_cus, false)) != MA_OK) return rc;
    }
    return bwd_sweep<T, D>(L, B, c);
}

template <typename T> int run_bwd_impl(Launcher &L, const BwdCallBufs &B, const CallDims &c)
{
    switch (tile_d(c.d)) {
    case 64: return run_bwd_d<T, 64>(L, B, c);
    case 96: return run_bwd_d<T, 96>(L, B, c);
    default: return run_bwd_d<T, 128>(L, B, c);
    }
}

}  // namespace ma_host
