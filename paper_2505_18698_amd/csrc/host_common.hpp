// Host-side pieces shared by the C ABI (monarch_attn.hip) and the per-dtype
// dispatch units (dispatch_*.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/monarch_attn.h"

namespace ma_host {

// Record a failure for monarch_attn_last_error() and return `code`.
int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));

inline int pad16(int64_t x) { return (int)((x + 15) / 16 * 16); }

// Tile size (16, 32, 64 or 128 rows) the kernels use for a block of n <= 128 rows.
inline int tile_rows(int64_t n)
{
    const int p = pad16(n);
    return p <= 16 ? 16 : p <= 32 ? 32 : p <= 64 ? 64 : 128;
}

// Kernel kinds reported by the timing interface.
enum Kind { kR = 0, kL = 1, kRFinal = 2, kApply = 3, kFused = 4, kObjSum = 5, kExact = 6, kBwdL = 7, kBwdR = 8,
            kGroup = 9 };

// Per-launch HIP events around every kernel when timing is enabled.
constexpr int kMaxLaunches = 2 * 64 + 2;
struct Timing {
    bool enabled = false;
    bool ready = false;
    int nlaunch = 0;
    int kind[kMaxLaunches];
    hipEvent_t ev[2 * kMaxLaunches];
    bool created = false;
};
extern Timing g_timing;

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
        const int rc = launch();
        if (rc != MA_OK) return rc;
        if (timed) {
            g_timing.kind[n] = kind;
            if (hipEventRecord(g_timing.ev[2 * n + 1], stream) != hipSuccess) return fail(MA_EHIP, "hipEventRecord failed");
        }
        ++n;
        return MA_OK;
    }
};

// Untyped tensors and states of one call (the states are null on the fused
// path; obj_part and obj are null unless the objective is requested).
struct CallBufs {
    const void *q, *k, *v;
    void *out;
    void *aR, *aL, *Y;
    float *cR, *cL;
    float *obj_part;  // [B*H][T][b] shares (workspace)
    float *obj;       // [B*H][T] result (caller's)
    const int *lens = nullptr;  // [B] real rows per batch element (device), or null
    int rev = 0;                // pre-padded sequences (HeadDims::rev)
};

struct CallDims {
    int64_t BH;
    int64_t H;  // heads per batch element
    int m, b, n, d, T;  // n: rows per head, (m - 1) * b < n <= m * b
    float s_log2e;
    int num_cus;  // compute units of the device
};

// Path selection (monarch_attn_set_path): 0 = automatic; 1 = one launch per
// half-step; 2 = one workgroup per head (or MA_EUNSUPPORTED); 3 = one
// workgroup per (head, group of residue classes) (or MA_EUNSUPPORTED).
enum Path { kAuto = 0, kHalfSteps = 1, kFusedHead = 2, kGrouped = 3 };

// The kernel family that runs a forward call.
enum Family { kFamHalf = 0, kFamFused = 1, kFamGroup = 2, kFamNone = -1 };

// Tile width of the kernels for head dimension d (columns d..D-1 are zero).
inline int tile_d(int64_t d) { return d <= 64 ? 64 : d <= 96 ? 96 : 128; }

// The fused one-workgroup-per-head kernel holds Q, K and all states of a head
// in LDS: 16-bit elements, d <= 64, m and b at most 16.
inline bool fused_applies(int32_t dtype, int64_t d, int64_t m, int64_t b)
{
    return (dtype == MA_BF16 || dtype == MA_F16) && d <= 64 && m <= 16 && b <= 16;
}

// The one-workgroup-per-(head, group of classes) kernel keeps the states of
// its classes in LDS: 16-bit elements, d <= 64, m at most 64, b at most 32,
// and neither per-sequence lengths nor the objective.
inline bool grouped_applies(int32_t dtype, int64_t d, int64_t m, int64_t b, bool lens, bool obj)
{
    return (dtype == MA_BF16 || dtype == MA_F16) && d <= 64 && m <= 64 && b <= 32 && !lens && !obj;
}

// The family that runs a call under `path` (kFamNone: the forced path does
// not take the shape).  Automatic: the one-workgroup-per-head kernel where it
// applies; else the grouped kernel where it applies with m <= 32 (measured
// faster than the half-steps there at 16 and 192 heads and T = 1, 2, apart
// from 24-row blocks at T = 1 with many heads, up to 15% slower; with more
// blocks every group streams more of K and V); else the half-steps.  All
// families give the same bits.
inline int family_of(int path, int32_t dtype, int64_t d, int64_t m, int64_t b, bool lens, bool obj)
{
    switch (path) {
    case kHalfSteps: return kFamHalf;
    case kFusedHead: return fused_applies(dtype, d, m, b) ? kFamFused : kFamNone;
    case kGrouped: return grouped_applies(dtype, d, m, b, lens, obj) ? kFamGroup : kFamNone;
    default:
        if (fused_applies(dtype, d, m, b)) return kFamFused;
        if (grouped_applies(dtype, d, m, b, lens, obj) && m <= 32) return kFamGroup;
        return kFamHalf;
    }
}

// Enqueue the whole forward pass for one element type (defined per dtype).
template <typename T> int run_call(Launcher &L, const CallBufs &B, const CallDims &c, int path);

// Buffers of one gradient call: the caller's tensors, the states of every
// step of the recomputed forward pass (alpha_R and c_R of steps 2..T, alpha_L
// and c_L of steps 1..T, `st` bytes resp. `cst` floats apart, and Y), and the
// fp32 gradients of the states and accumulators of dQ, dK.
struct BwdCallBufs {
    const void *q, *k, *v, *dout;
    void *dq, *dk, *dv;
    char *aR, *aL;
    void *Y;
    float *cR, *cL;
    size_t st, cst;
    float *dQ, *dK, *daL, *dcL, *dY, *daR, *dcR;
    const int *lens = nullptr;  // [B] real rows per batch element (device), or null
};

// Enqueue the gradient (forward recompute, then the reverse sweep) for one element type.
template <typename T> int run_bwd(Launcher &L, const BwdCallBufs &B, const CallDims &c);

// Enqueue exact softmax attention (with the row logsumexps when lse != null).
template <typename T> int run_exact(Launcher &L, const CallBufs &B, float *lse, int64_t BH, int n, int d);

}  // namespace ma_host
