// Launch stubs for the host-only sanitizer build of the C ABI layer: the
// argument checks run as in the library, and a call that passes them counts
// here instead of launching anything (no GPU, no HIP runtime call).
#include "gdn_launch.h"

namespace gdn {

int g_stub_launches = 0;

hipError_t launch_decode(const DecodeArgs&, hipStream_t) {
    ++g_stub_launches;
    return hipSuccess;
}

hipError_t launch_prefill(const PrefillArgs&, hipStream_t) {
    ++g_stub_launches;
    return hipSuccess;
}

}  // namespace gdn
