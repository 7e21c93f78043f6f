// Kernels and dispatch for element type float.
#include "dispatch.hpp"
#include "dispatch_bwd.hpp"

namespace ma_host {
template <> int run_call<float>(Launcher &L, const CallBufs &B, const CallDims &c, int path)
{
    return run_call_impl<float>(L, B, c, path);
}
template <> int run_exact<float>(Launcher &L, const CallBufs &B, float *lse, int64_t BH, int n, int d)
{
    return run_exact_impl<float>(L, B, lse, BH, n, d);
}
template <> int run_bwd<float>(Launcher &L, const BwdCallBufs &B, const CallDims &c)
{
    return run_bwd_impl<float>(L, B, c);
}
}  // namespace ma_host
