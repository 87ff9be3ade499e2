// Launchers for the host-only sanitizer build of the C entry points
// (tests/test_sanitizers.py): they launch nothing, count their calls and
// report a launch error, so an argument the checks wrongly accept shows up
// as ATTN_ELAUNCH and as a nonzero count.
#include <stddef.h>
#include <stdint.h>

#include "attn_params.h"

static int g_launches = 0;

namespace h15 {

int launch_fwd(const Params&, int, int, int, int, void*, bool) { return ++g_launches, 1; }
int launch_probe_fill(float*, float*, uint32_t*, size_t, void*) { return ++g_launches, 1; }
int launch_decode(const DecParams&, int, int, int, int, void*, bool) { return ++g_launches, 1; }
// the built-in decode workspace: the library's stated size, no address
size_t scratch_capacity() { return (size_t)16 << 20; }
int scratch_address(void*, void**) { return ++g_launches, 1; }

}  // namespace h15

extern "C" int h15_stub_launches(void) { return g_launches; }
