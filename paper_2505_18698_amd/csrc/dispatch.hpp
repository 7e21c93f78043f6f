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

#include <cmath>
#include <mutex>
#include <type_traits>
#include <unordered_map>

#include "grouped.hpp"
#include "host_common.hpp"
#include "ma_kernels.hpp"

namespace ma_host {

template <typename T> ma::Bufs<T> typed(const CallBufs &B)
{
    return ma::Bufs<T>{(const T *)B.q, (const T *)B.k, (const T *)B.v, (T *)B.out, (T *)B.aR, (T *)B.aL, (T *)B.Y,
                       B.cR, B.cL, B.obj_part};
}

template <typename F> int launched(F &&f)
{
    f();
    return MA_OK;
}

// Workgroups of `kern` (at `threads` threads) resident on one compute unit,
// queried once per kernel.
inline int resident_per_cu(const void *kern, int threads)
{
    static std::mutex mu;
    static std::unordered_map<const void *, int> cache;
    std::lock_guard<std::mutex> lock(mu);
    auto it = cache.find(kern);
    if (it != cache.end()) return it->second;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kern, threads, 0) != hipSuccess || n < 1) {
        (void)hipGetLastError();
        n = 1;
    }
    cache.emplace(kern, n);
    return n;
}

// Grid of a half-step launch: every unit once, at most one workgroup per
// resident slot (the workgroups loop over units).
inline dim3 unit_grid(const void *kern, int threads, int64_t units, int num_cus)
{
    const int64_t cap = (int64_t)resident_per_cu(kern, threads) * num_cus;
    return dim3((unsigned)(units < cap ? units : cap));
}

template <typename T, int NB, int D, bool FIRST, bool FINAL, bool RG, bool LENS>
int launch_r1(Launcher &L, const CallBufs &B, ma::HeadDims hd, int64_t BH, int num_cus)
{
    constexpr int W = ma::Split<NB / 16>::W;
    auto kern = ma::r_half_step<T, NB, D, FIRST, FINAL, RG, LENS>;
    hd.units = BH * hd.m;
    const dim3 grid = unit_grid((const void *)kern, 64 * W, hd.units, num_cus), block(64 * W);
    const ma::Bufs<T> p = typed<T>(B);
    return L.run(FINAL ? kRFinal : kR,
                 [&] { return launched([&] { hipLaunchKernelGGL(kern, grid, block, 0, L.stream, p, hd); }); });
}

template <typename T, int NB, int D, bool RG, bool LENS = false>
int launch_r(Launcher &L, const CallBufs &B, ma::HeadDims hd, int64_t BH, int num_cus, bool first, bool final_)
{
    if (first && final_) return launch_r1<T, NB, D, true, true, RG, LENS>(L, B, hd, BH, num_cus);
    if (first) return launch_r1<T, NB, D, true, false, RG, LENS>(L, B, hd, BH, num_cus);
    if (final_) return launch_r1<T, NB, D, false, true, RG, LENS>(L, B, hd, BH, num_cus);
    return launch_r1<T, NB, D, false, false, RG, LENS>(L, B, hd, BH, num_cus);
}

template <typename T, int NM, int D, bool RG, bool LENS = false>
int launch_l(Launcher &L, const CallBufs &B, ma::HeadDims hd, int64_t BH, int num_cus, bool apply)
{
    constexpr int W = ma::Split<NM / 16>::W;
    hd.units = BH * hd.b;
    const ma::Bufs<T> p = typed<T>(B);
    const dim3 block(64 * W);
    if (apply) {
        auto kern = ma::monarch_apply<T, NM, D, RG, LENS>;
        const dim3 grid = unit_grid((const void *)kern, 64 * W, hd.units, num_cus);
        return L.run(kApply, [&] { return launched([&] { hipLaunchKernelGGL(kern, grid, block, 0, L.stream, p, hd); }); });
    }
    auto kern = ma::l_half_step<T, NM, D, RG, LENS>;
    const dim3 grid = unit_grid((const void *)kern, 64 * W, hd.units, num_cus);
    return L.run(kL, [&] { return launched([&] { hipLaunchKernelGGL(kern, grid, block, 0, L.stream, p, hd); }); });
}

template <typename T, int D, int NB>
int dispatch_r(Launcher &L, const CallBufs &B, ma::HeadDims hd, int64_t BH, int nc, bool first, bool final_)
{
    if constexpr (std::is_same<T, float>::value && NB * D > 8192) {
        return fail(MA_EUNSUPPORTED, "fp32 tile too large");
    } else {
        // masked softmax over i when the tile is padded or the last block is
        // short; per-sequence lengths have instantiations of their own
        if (hd.lens) return launch_r<T, NB, D, true, true>(L, B, hd, BH, nc, first, final_);
        const bool ragged = hd.b != NB || hd.n != hd.m * hd.b;
        return ragged ? launch_r<T, NB, D, true>(L, B, hd, BH, nc, first, final_)
                      : launch_r<T, NB, D, false>(L, B, hd, BH, nc, first, final_);
    }
}

template <typename T, int D, int NM>
int dispatch_l(Launcher &L, const CallBufs &B, ma::HeadDims hd, int64_t BH, int nc, bool apply)
{
    if constexpr (std::is_same<T, float>::value && NM * D > 8192) {
        return fail(MA_EUNSUPPORTED, "fp32 tile too large");
    } else {
        if (hd.lens) return launch_l<T, NM, D, true, true>(L, B, hd, BH, nc, apply);
        return hd.m != NM ? launch_l<T, NM, D, true>(L, B, hd, BH, nc, apply)
                          : launch_l<T, NM, D, false>(L, B, hd, BH, nc, apply);
    }
}

template <typename T, int D>
int r_step(Launcher &L, const CallBufs &B, ma::HeadDims hd, int64_t BH, int nc, bool first, bool final_)
{
    switch (tile_rows(hd.b)) {
    case 16: return dispatch_r<T, D, 16>(L, B, hd, BH, nc, first, final_);
    case 32: return dispatch_r<T, D, 32>(L, B, hd, BH, nc, first, final_);
    case 64: return dispatch_r<T, D, 64>(L, B, hd, BH, nc, first, final_);
    default: return dispatch_r<T, D, 128>(L, B, hd, BH, nc, first, final_);
    }
}

template <typename T, int D>
int l_step(Launcher &L, const CallBufs &B, ma::HeadDims hd, int64_t BH, int nc, bool apply)
{
    switch (tile_rows(hd.m)) {
    case 16: return dispatch_l<T, D, 16>(L, B, hd, BH, nc, apply);
    case 32: return dispatch_l<T, D, 32>(L, B, hd, BH, nc, apply);
    case 64: return dispatch_l<T, D, 64>(L, B, hd, BH, nc, apply);
    default: return dispatch_l<T, D, 128>(L, B, hd, BH, nc, apply);
    }
}

template <typename T, int D>
int run_half_steps(Launcher &L, const CallBufs &B, ma::HeadDims hd, const CallDims &c)
{
    int rc;
    hd.T = c.T;
    for (int t = 1; t <= c.T; ++t) {
        const bool first = (t == 1), last = (t == c.T);
        hd.t = t;
        if ((rc = r_step<T, D>(L, B, hd, c.BH, c.num_cus, first, last)) != MA_OK) return rc;
        if ((rc = l_step<T, D>(L, B, hd, c.BH, c.num_cus, last)) != MA_OK) return rc;
    }
    return MA_OK;
}

// ---- one workgroup per head ----
template <typename T, bool RGB, bool RGM, bool LENS = false>
int launch_fused(Launcher &L, const CallBufs &B, ma::HeadDims hd, const CallDims &c)
{
    using U = ma::FusedHead<T, RGB, RGM, LENS>;
    // one workgroup per compute unit (its LDS holds one), each looping over heads
    const int64_t grid = c.BH < c.num_cus ? c.BH : c.num_cus;
    hd.units = c.BH;
    const ma::Bufs<T> p = typed<T>(B);
    const int64_t BH = c.BH;
    const int T_ = c.T;
    return L.run(kFused, [&] {
        return launched([&] {
            hipLaunchKernelGGL((ma::monarch_fused_head<T, RGB, RGM, LENS>), dim3((unsigned)grid), dim3(64 * U::NW), 0,
                               L.stream, p, hd, BH, T_);
        });
    });
}

template <typename T> int run_fused(Launcher &L, const CallBufs &B, ma::HeadDims hd, const CallDims &c)
{
    if constexpr (sizeof(T) != 2) {
        return fail(MA_EUNSUPPORTED, "the fused kernel needs 16-bit elements");
    } else {
        if (hd.lens) return launch_fused<T, true, true, true>(L, B, hd, c);
        const bool rgb = hd.b != 16 || hd.n != hd.m * hd.b, rgm = hd.m != 16;
        if (rgb && rgm) return launch_fused<T, true, true>(L, B, hd, c);
        if (rgb) return launch_fused<T, true, false>(L, B, hd, c);
        if (rgm) return launch_fused<T, false, true>(L, B, hd, c);
        return launch_fused<T, false, false>(L, B, hd, c);
    }
}

// ---- one workgroup per (head, group of residue classes) ----

// Workgroups of `kern` resident per CU at `lds` bytes of dynamic LDS, with
// the kernel allowed that much LDS (set once per kernel).
inline int resident_per_cu_lds(const void *kern, int threads, int lds)
{
    static std::mutex mu;
    static std::unordered_map<const void *, int> attr;                // LDS bytes allowed so far
    static std::unordered_map<uint64_t, int> cache;                    // (kernel, lds) -> workgroups
    std::lock_guard<std::mutex> lock(mu);
    int &allowed = attr[kern];
    if (allowed < lds) {
        if (hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds) != hipSuccess) {
            (void)hipGetLastError();
            return 0;
        }
        allowed = lds;
    }
    const uint64_t key = (uint64_t)(uintptr_t)kern * 1000003u + (uint64_t)lds;
    auto it = cache.find(key);
    if (it != cache.end()) return it->second;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kern, threads, lds) != hipSuccess) {
        (void)hipGetLastError();
        n = 0;
    }
    cache.emplace(key, n);
    return n;
}

constexpr int kMaxLds = 160 * 1024;

// Classes per workgroup: the largest G (at most 16 and at most b) whose LDS
// fits and that still gives every compute unit a workgroup, unless that G
// needs more rounds of resident workgroups than the next larger one (then
// that one); if no G fills the device, the smallest that fits.  A unit's R
// half-steps stream all of the head's K and V whatever G is, so a second
// round costs about a whole unit, and fewer, larger groups move fewer bytes.
template <typename U> int group_size(const void *kern, int64_t BH, int b, int num_cus)
{
    const int cand[5] = {16, 8, 4, 2, 1};
    int prev = 0;
    int64_t prev_rounds = 0;
    for (int i = 0; i < 5; ++i) {
        const int G = cand[i] < b ? cand[i] : b;
        if (G == prev || U::lds_bytes(G) > kMaxLds) continue;
        const int per_cu = resident_per_cu_lds(kern, U::NTH, U::lds_bytes(G));
        if (per_cu < 1) continue;
        const int64_t units = BH * ((b + G - 1) / G), slots = (int64_t)per_cu * num_cus;
        const int64_t rounds = (units + slots - 1) / slots;
        if (units >= num_cus) return prev && prev_rounds < rounds ? prev : G;
        prev = G;
        prev_rounds = rounds;
    }
    return prev;
}

template <typename T, int NB, int NM, bool RG, bool YG>
int launch_group(Launcher &L, const CallBufs &B, ma::HeadDims hd, const CallDims &c, int G)
{
    using U = ma::FusedGroup<T, NB, NM, 64, RG, YG>;
    auto kern = ma::monarch_fused_group<T, NB, NM, 64, RG, YG>;
    if (G < 1) return fail(MA_EUNSUPPORTED, "the grouped kernel's LDS does not fit");
    const int lds = U::lds_bytes(G);
    const int per_cu = resident_per_cu_lds((const void *)kern, U::NTH, lds);
    if (per_cu < 1) return fail(MA_EUNSUPPORTED, "the grouped kernel cannot be resident with %d bytes of LDS", lds);
    const int groups = (c.b + G - 1) / G;
    const int64_t units = c.BH * groups;
    if (units > 0x7fffffff) return fail(MA_EUNSUPPORTED, "too many units for one grid");
    const int64_t cap = (int64_t)per_cu * c.num_cus;
    const int64_t grid = units < cap ? units : cap;
    const int xcd_perm = units % 8 == 0 ? 1 : 0;
    hd.units = units;
    const ma::Bufs<T> p = typed<T>(B);
    const int T_ = c.T;
    return L.run(kGroup, [&] {
        return launched([&] {
            hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(U::NTH), (unsigned)lds, L.stream, p, hd, G, groups,
                               units, xcd_perm, T_);
        });
    });
}

template <typename T, int NB, int NM, bool RG, bool YG> int group_size_of(const CallDims &c)
{
    using U = ma::FusedGroup<T, NB, NM, 64, RG, YG>;
    return group_size<U>((const void *)ma::monarch_fused_group<T, NB, NM, 64, RG, YG>, c.BH, c.b, c.num_cus);
}

// Full tiles: Y through O where that allows larger groups than Y in LDS
// (fewer groups stream K and V), else Y in LDS (no round trip of Y).
template <typename T, int NB, int NM> int dispatch_group_rg(Launcher &L, const CallBufs &B, ma::HeadDims hd, const CallDims &c)
{
    const bool rg = c.b != NB || c.m != NM || c.n != c.m * c.b;
    if (rg) return launch_group<T, NB, NM, true, false>(L, B, hd, c, group_size_of<T, NB, NM, true, false>(c));
    const int g_lds = group_size_of<T, NB, NM, false, false>(c), g_out = group_size_of<T, NB, NM, false, true>(c);
    return g_out > g_lds ? launch_group<T, NB, NM, false, true>(L, B, hd, c, g_out)
                         : launch_group<T, NB, NM, false, false>(L, B, hd, c, g_lds);
}

template <typename T, int NB> int dispatch_group_m(Launcher &L, const CallBufs &B, ma::HeadDims hd, const CallDims &c)
{
    switch (tile_rows(c.m)) {
    case 16: return dispatch_group_rg<T, NB, 16>(L, B, hd, c);
    case 32: return dispatch_group_rg<T, NB, 32>(L, B, hd, c);
    default: return dispatch_group_rg<T, NB, 64>(L, B, hd, c);
    }
}

template <typename T> int run_group(Launcher &L, const CallBufs &B, ma::HeadDims hd, const CallDims &c)
{
    if constexpr (sizeof(T) != 2) {
        return fail(MA_EUNSUPPORTED, "the grouped kernel needs 16-bit elements");
    } else {
        // (b <= 32: grouped_applies)
        return tile_rows(c.b) == 16 ? dispatch_group_m<T, 16>(L, B, hd, c) : dispatch_group_m<T, 32>(L, B, hd, c);
    }
}

template <typename T, int D> int launch_exact(Launcher &L, const CallBufs &B, float *lse, int64_t BH, int n, int d)
{
    const ma::Bufs<T> p = typed<T>(B);
    const int64_t grid = BH * ((n + 63) / 64);
    if (grid > 0x7fffffff) return fail(MA_EUNSUPPORTED, "too many query blocks for one grid");
    const float s_log2e = (float)(1.4426950408889634 / std::sqrt((double)d));
    return L.run(kExact, [&] {
        return launched([&] {
            hipLaunchKernelGGL((ma::exact_attention<T, D>), dim3((unsigned)grid), dim3(256), 0, L.stream, p, lse, n, d,
                               s_log2e);
        });
    });
}

template <typename T> int run_exact_impl(Launcher &L, const CallBufs &B, float *lse, int64_t BH, int n, int d)
{
    switch (tile_d(d)) {
    case 64: return launch_exact<T, 64>(L, B, lse, BH, n, d);
    case 96: return launch_exact<T, 96>(L, B, lse, BH, n, d);
    default: return launch_exact<T, 128>(L, B, lse, BH, n, d);
    }
}

template <typename T> int run_call_impl(Launcher &L, const CallBufs &B, const CallDims &c, int path)
{
    const int32_t dtype = std::is_same<T, float>::value ? MA_F32 : std::is_same<T, __bf16>::value ? MA_BF16 : MA_F16;
    ma::HeadDims hd{c.m, c.b, c.n, c.d, c.s_log2e, 0};
    hd.lens = B.lens;
    hd.H = (int)c.H;
    hd.colnorm = 1;
    hd.rev = B.rev;
    // the grouped kernel takes neither lengths nor the objective nor pre-padding
    const int fam = family_of(path, dtype, c.d, c.m, c.b, B.lens != nullptr || B.rev, B.obj != nullptr);
    if (fam == kFamNone)
        return fail(MA_EUNSUPPORTED, path == kFusedHead
                                         ? "the one-workgroup-per-head kernel needs bf16/fp16, d <= 64 and m, b <= 16"
                                         : "the grouped kernel needs bf16/fp16, d <= 64, m <= 64, b <= 32, no lengths, "
                                           "no pre-padding and no objective");
    int rc;
    if (fam == kFamFused) {
        rc = run_fused<T>(L, B, hd, c);
    } else if (fam == kFamGroup) {
        rc = run_group<T>(L, B, hd, c);
    } else {
        switch (tile_d(c.d)) {
        case 64: rc = run_half_steps<T, 64>(L, B, hd, c); break;
        case 96: rc = run_half_steps<T, 96>(L, B, hd, c); break;
        default: rc = run_half_steps<T, 128>(L, B, hd, c); break;
        }
    }
    if (rc != MA_OK || !B.obj) return rc;
    const int64_t units = c.BH * c.T;  // one (head, step) per thread
    const float *part = B.obj_part;
    float *obj = B.obj;
    const int b = c.b;
    return L.run(kObjSum, [&] {
        return launched([&] {
            hipLaunchKernelGGL(ma::objective_sum, dim3((unsigned)((units + 255) / 256)), dim3(256), 0, L.stream, part,
                               obj, units, b);
        });
    });
}

}  // namespace ma_host
