// Kernels and dispatch for element type _Float16.
#include "dispatch.hpp"

namespace ma_host {
template <> int run_call<_Float16>(Launcher &L, const CallBufs &B, const CallDims &c, int path)
{
    return run_call_impl<_Float16>(L, B, c, path);
}
}  // namespace ma_host
