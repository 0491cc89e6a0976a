// Host-only stand-ins for the kernel launchers, so that the C-ABI layer (forge_api.cpp) can be
// built with g++ and AddressSanitizer for the boundary tests.  Those tests never reach a
// launch (validation stops at the device check on a machine without a GPU); every stub
// fails loudly if one is reached anyway.
#include <cstdio>
#include <cstdlib>

#include "forge_internal.h"

namespace forge_impl {

[[noreturn]] static void unreachable(const char *what)
{
    std::fprintf(stderr, "launch stub reached: %s\n", what);
    std::abort();
}

TileShape tile_shape(int) { unreachable("tile_shape"); }
hipError_t launch_fused(const Args &, int, hipStream_t) { unreachable("launch_fused"); }
hipError_t launch_fused_group(const Args *, int, int, hipStream_t) { unreachable("launch_fused_group"); }
hipError_t launch_fused_rule(const Args *, int, int, int, hipStream_t) { unreachable("launch_fused_rule"); }
hipError_t launch_fused_wfp8(const Args *, int, int, hipStream_t) { unreachable("launch_fused_wfp8"); }
hipError_t launch_wgrad(const Args &, int, hipStream_t) { unreachable("launch_wgrad"); }
hipError_t launch_adamw(const Args &, int, int, hipStream_t) { unreachable("launch_adamw"); }
hipError_t launch_dx(const DxSeg *, int, uint16_t *, int, int, hipStream_t) { unreachable("launch_dx"); }
int device_cu_count() { unreachable("device_cu_count"); }
hipError_t scratch_address(void **) { unreachable("scratch_address"); }

}  // namespace forge_impl
