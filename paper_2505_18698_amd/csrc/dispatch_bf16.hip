// Kernels and dispatch for element type __bf16.
#include "dispatch.hpp"
#include "dispatch_bwd.hpp"

namespace ma_host {
template <> int run_call<__bf16>(Launcher &L, const CallBufs &B, const CallDims &c, int path)
{
    return run_call_impl<__bf16>(L, B, c, path);
}
template <> int run_exact<__bf16>(Launcher &L, const CallBufs &B, float *lse, int64_t BH, int n, int d)
{
    return run_exact_impl<__bf16>(L, B, lse, BH, n, d);
}
template <> int run_bwd<__bf16>(Launcher &L, const BwdCallBufs &B, const CallDims &c)
{
    return run_bwd_impl<__bf16>(L, B, c);
}
}  // namespace ma_host
