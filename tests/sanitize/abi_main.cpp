// Driver of the C ABI's host code for the AddressSanitizer /
// UndefinedBehaviorSanitizer build (tests/test_sanitizers.py): monarch_attn.hip
// compiled for the host only and linked with stand-ins for the per-dtype
// dispatch units (which hold the kernels and are never reached here).  Every
// call below must fail, or finish, in the argument checks before any HIP call:
// malformed and unsupported shapes, null, misaligned and overlapping
// pointers, head counts at the grid limit and beyond int64, the shape
// queries and workspace sizes, and the empty calls that return at once.
#include <cstdint>
#include <cstdio>
#include <cstring>

#include "../../paper_2505_18698_amd/csrc/host_common.hpp"

namespace ma_host {
#define MA_STANDIN(T)                                                                                     \
    template <> int run_call<T>(Launcher &, const CallBufs &, const CallDims &, int)                      \
    {                                                                                                     \
        return fail(MA_EHIP, "stand-in dispatch reached");                                               \
    }                                                                                                     \
    template <> int run_exact<T>(Launcher &, const CallBufs &, float *, int64_t, int, int)                \
    {                                                                                                     \
        return fail(MA_EHIP, "stand-in dispatch reached");                                               \
    }                                                                                                     \
    template <> int run_bwd<T>(Launcher &, const BwdCallBufs &, const CallDims &)                         \
    {                                                                                                     \
        return fail(MA_EHIP, "stand-in dispatch reached");                                               \
    }
MA_STANDIN(float)
MA_STANDIN(__bf16)
MA_STANDIN(_Float16)
}  // namespace ma_host

static int fails = 0;

static void expect(bool cond, const char *what)
{
    if (!cond) {
        std::fprintf(stderr, "FAILED: %s (%s)\n", what, monarch_attn_last_error());
        ++fails;
    }
}

int main()
{
    char *F = reinterpret_cast<char *>(uintptr_t(1) << 20);  // aligned, never dereferenced
    char *O = F + (uintptr_t(1) << 24);
    const int64_t big = INT64_MAX;
    // malformed (MA_EINVAL) and unsupported (MA_EUNSUPPORTED) forward calls
    expect(monarch_attn_fwd(nullptr, F, F, O, 1, 1, 256, 64, 16, 16, 1, 1, nullptr) == MA_EINVAL, "null q");
    expect(monarch_attn_fwd(F, F, F, O, -1, 1, 256, 64, 16, 16, 1, 1, nullptr) == MA_EINVAL, "B < 0");
    expect(monarch_attn_fwd(F, F, F, O, 1, 1, 257, 64, 16, 16, 1, 1, nullptr) == MA_EINVAL, "N > m b");
    expect(monarch_attn_fwd(F, F, F, O, 1, 1, 256, 64, 16, 16, 0, 1, nullptr) == MA_EINVAL, "T = 0");
    expect(monarch_attn_fwd(F, F, F, O, 1, 1, 256, 64, 16, 16, 1, 9, nullptr) == MA_EINVAL, "dtype");
    expect(monarch_attn_fwd(F + 2, F, F, O, 1, 1, 256, 64, 16, 16, 1, 1, nullptr) == MA_EINVAL, "misaligned");
    expect(monarch_attn_fwd(F, F, F, F + 64, 1, 1, 256, 64, 16, 16, 1, 1, nullptr) == MA_EINVAL, "overlap");
    expect(monarch_attn_fwd(F, F, F, O, 1, 1, 256, 136, 16, 16, 1, 1, nullptr) == MA_EUNSUPPORTED, "d > 128");
    expect(monarch_attn_fwd(F, F, F, O, 1, 1, 512, 64, 2, 256, 1, 1, nullptr) == MA_EUNSUPPORTED, "b > 128");
    expect(monarch_attn_fwd(F, F, F, O, 1, 1, 256, 64, 16, 16, 65, 0, nullptr) == MA_EUNSUPPORTED, "T > 64");
    expect(monarch_attn_fwd(F, F, F, O, 1, 1, 256, 64, 16, 16, MONARCH_ATTN_MAX_T_16BIT + 1, 1, nullptr) ==
               MA_EUNSUPPORTED,
           "16-bit T cap");
    expect(monarch_attn_fwd(F, F, F, O, int64_t(1) << 24, int64_t(1) << 24, 256, 64, 16, 16, 1, 1, nullptr) ==
               MA_EUNSUPPORTED,
           "grid limit");
    expect(monarch_attn_fwd(F, F, F, O, big, big, 256, 64, 16, 16, 1, 1, nullptr) == MA_EUNSUPPORTED,
           "B H beyond int64");
    expect(monarch_attn_fwd(F, F, F, O, 1, 1, big, 64, 1, 128, 1, 1, nullptr) == MA_EINVAL, "huge N");
    expect(monarch_attn_fwd(F, F, F, O, 1, 1, 256, big, 16, 16, 1, 1, nullptr) == MA_EUNSUPPORTED, "huge d");
    // the other entry points
    expect(monarch_attn_fwd_varlen(F, F, F, O, nullptr, 1, 1, 256, 64, 16, 16, 1, 1, nullptr) == MA_EINVAL,
           "varlen null lens");
    expect(monarch_attn_fwd_objective(F, F, F, O, nullptr, 1, 1, 256, 64, 16, 16, 1, 1, nullptr) == MA_EINVAL,
           "objective null obj");
    expect(monarch_attn_fwd_prepad(F, F, F, O, reinterpret_cast<const int32_t *>(F + 2), 1, 1, 250, 64, 16, 16, 1,
                                   1, nullptr) == MA_EINVAL,
           "prepad misaligned lens");
    expect(monarch_attn_fwd_prepad(F, F, F, O, nullptr, 1, 1, 240, 64, 16, 16, 1, 1, nullptr) == MA_EINVAL,
           "prepad m != ceil(N / b)");
    expect(monarch_attn_exact_fwd(F, F, F, O, reinterpret_cast<float *>(F + 2), 1, 1, 256, 64, 1, nullptr) ==
               MA_EINVAL,
           "exact misaligned lse");
    expect(monarch_attn_bwd(F, F, F, F, O, O, O, 1, 1, 256, 64, 16, 16, 1, 1, nullptr) == MA_EINVAL,
           "bwd overlapping outputs");
    expect(monarch_attn_bwd(F, F, F, F, O, O + (1 << 20), O + (2 << 20), 1, 1, 256, 64, 16, 16, 33, 0, nullptr) ==
               MA_EUNSUPPORTED,
           "bwd T > 32");
    // calls with nothing to compute return at once
    expect(monarch_attn_fwd(nullptr, nullptr, nullptr, nullptr, 0, 4, 256, 64, 16, 16, 2, 1, nullptr) == MA_OK,
           "empty batch");
    expect(monarch_attn_fwd(nullptr, nullptr, nullptr, nullptr, 2, 4, 0, 64, 0, 16, 2, 1, nullptr) == MA_OK,
           "empty sequence");
    // queries
    expect(monarch_attn_check(16384, 64, 128, 128, 2, 1) == MA_OK, "check 16K");
    expect(monarch_attn_check(16384, 128, 128, 128, 2, 0) == MA_EUNSUPPORTED, "check fp32 tile");
    expect(monarch_attn_bwd_check(1024, 64, 32, 32, MONARCH_ATTN_MAX_T_16BIT_BWD + 1, 1) == MA_EUNSUPPORTED,
           "bwd check 16-bit T cap");
    expect(monarch_attn_workspace_bytes(1, 16, 16384, 64, 128, 128, 2, 1) > 0, "workspace bytes");
    expect(monarch_attn_workspace_bytes(1, 1, big, 64, 128, 128, 2, 1) == 0, "workspace of a bad shape");
    expect(monarch_attn_bwd_workspace_bytes(1, 16, 16384, 64, 128, 128, 2, 1) > 0, "bwd workspace bytes");
    expect(monarch_attn_set_path(7) == -1, "unknown path");
    expect(monarch_attn_set_path(1) == 0 && monarch_attn_set_path(0) == 1, "path round trip");
    expect(std::strlen(monarch_attn_build_id()) == 16, "build id");
    // the schedule a forward call runs (ma_host::family_of): automatic,
    // then forced; 16-bit types are 1 (bf16) and 2 (fp16), fp32 is 0
    using namespace ma_host;
    expect(family_of(kAuto, MA_BF16, 64, 14, 14, false, false) == kFamFused, "auto: ViT heads in one workgroup");
    expect(family_of(kAuto, MA_F16, 64, 16, 16, false, false) == kFamFused, "auto: 16 x 16 in one workgroup");
    expect(family_of(kAuto, MA_BF16, 64, 32, 32, false, false) == kFamGroup, "auto: 32 x 32 grouped");
    expect(family_of(kAuto, MA_BF16, 48, 17, 8, false, false) == kFamGroup, "auto: m = 17 grouped");
    expect(family_of(kAuto, MA_BF16, 64, 33, 32, false, false) == kFamHalf, "auto: m = 33 half-steps");
    expect(family_of(kAuto, MA_BF16, 64, 16, 33, false, false) == kFamHalf, "auto: b = 33 half-steps");
    expect(family_of(kAuto, MA_BF16, 72, 16, 16, false, false) == kFamHalf, "auto: d = 72 half-steps");
    expect(family_of(kAuto, MA_F32, 64, 16, 16, false, false) == kFamHalf, "auto: fp32 half-steps");
    expect(family_of(kAuto, MA_BF16, 64, 32, 32, true, false) == kFamHalf, "auto: lengths half-steps");
    expect(family_of(kAuto, MA_BF16, 64, 14, 14, true, false) == kFamFused, "auto: lengths, small heads fused");
    expect(family_of(kAuto, MA_BF16, 64, 32, 32, false, true) == kFamHalf, "auto: objective half-steps");
    expect(family_of(kAuto, MA_BF16, 64, 128, 128, false, false) == kFamHalf, "auto: 16K half-steps");
    expect(family_of(kHalfSteps, MA_BF16, 64, 14, 14, false, false) == kFamHalf, "forced half-steps");
    expect(family_of(kFusedHead, MA_BF16, 64, 17, 16, false, false) == kFamNone, "forced fused, m = 17");
    expect(family_of(kGrouped, MA_BF16, 64, 64, 32, false, false) == kFamGroup, "forced grouped, m = 64");
    expect(family_of(kGrouped, MA_BF16, 64, 8, 33, false, false) == kFamNone, "forced grouped, b = 33");
    expect(family_of(kGrouped, MA_F32, 64, 16, 16, false, false) == kFamNone, "forced grouped, fp32");
    if (fails) return 1;
    std::printf("ABI sanitizer run: ok\n");
    return 0;
}
