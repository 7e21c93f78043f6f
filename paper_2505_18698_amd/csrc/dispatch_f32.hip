// Kernels and dispatch for element type float.
#include "dispatch.hpp"

namespace ma_host {
template <> int run_call<float>(Launcher &L, const CallBufs &B, const CallDims &c, int path)
{
    return run_call_impl<float>(L, B, c, path);
}
}  // namespace ma_host
