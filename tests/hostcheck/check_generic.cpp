// Host-side checks of launch plans whose kernels have no address walk yet
// (test infrastructure; see check_main.cpp): a non-empty grid, a workgroup
// within the hardware limit and LDS within a CU.
#include "check.hpp"

namespace hostcheck {

void check_generic(const cliff::LaunchPlan& p)
{
    if (p.grid < 1 || p.grid >= (1ll << 31)) fail("kind %d: grid of %lld", p.kind, (long long)p.grid);
    if (p.block < 64 || p.block > 1024 || p.block % 64)
        fail("kind %d: workgroup of %lld threads", p.kind, (long long)p.block);
    if (p.lds_bytes < 0 || p.lds_bytes > 160 * 1024)
        fail("kind %d: %lld LDS bytes", p.kind, (long long)p.lds_bytes);
}

}  // namespace hostcheck
