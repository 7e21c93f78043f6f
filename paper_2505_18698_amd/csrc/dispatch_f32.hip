// Kernels and dispatch for element type float.
#include "dispatch.hpp"

namespace ma_host {
template <> int run_call<float>(Launcher &L, const CallBufs &B, const CallDims &c, int path)
{
    return run_call_impl<float>(L, B, c, path);
}
template <> int run_exact<float>(Launcher &L, const CallBufs &B, float *lse, int64_t BH, int n, int d)
{
    return run_exact_impl<float>(L, B, lse, BH, n, d);
}
}  // namespace ma_host
