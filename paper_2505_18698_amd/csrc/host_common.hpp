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

// Kernel kinds reported by the timing interface.
enum Kind { kR = 0, kL = 1, kRFinal = 2, kApply = 3, kPersistent = 4 };

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

// Untyped tensors, states and the single-launch synchronisation area of one call.
struct CallBufs {
    const void *q, *k, *v;
    void *out;
    void *aR, *aL, *Y;
    float *cR, *cL;
    unsigned *sync;     // zeroed counters for the single-launch path (kSyncWords words)
    int *error;         // host-visible flag written by the single-launch path
    int copies;         // per-iteration copies of alpha_R, alpha_L, c_R, c_L in the workspace
    int64_t state_stride, c_stride;  // elements / floats between two copies
};
constexpr int kSyncWords = 16 + 16 * 8;
// The single launch keeps one copy of every state per iteration; above this T
// it is not used (and the workspace holds a single copy).
constexpr int kMaxSingleT = 8;

struct CallDims {
    int64_t BH;
    int m, b, d, T;
    float s_log2e;
    int num_cus;
};

// Path selection: 0 = single launch when it applies, else one launch per
// half-step; 1 = one launch per half-step; 2 = single launch or MA_EUNSUPPORTED.
enum Path { kAuto = 0, kHalfSteps = 1, kSingle = 2 };

// Enqueue the whole forward pass for one element type (defined per dtype).
template <typename T> int run_call(Launcher &L, const CallBufs &B, const CallDims &c, int path);

}  // namespace ma_host
