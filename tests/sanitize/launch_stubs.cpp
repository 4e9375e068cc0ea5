// Launch stubs for the host-only sanitizer build of the ABI layer: every
// device launch aborts, so a validation failure that still reached a launch
// ends the run.  Only conv_channels_per_thread (a constant the validation
// reads) returns normally.
#include <cstdio>
#include <cstdlib>

#include "sf_launch.hpp"

namespace sf {
[[noreturn]] static void launched(const char *what) {
    std::fprintf(stderr, "unexpected launch: %s\n", what);
    std::abort();
}
hipError_t launch_kernel(int, int, int, const SegArgs &, hipStream_t, hipEvent_t, hipEvent_t) { launched("launch_kernel"); }
hipError_t launch_kernel_vg(int, int, int, const SegArgs &, hipStream_t, hipEvent_t, hipEvent_t) {
    launched("launch_kernel_vg");
}
hipError_t launch_state_copy(const float *, float *, int64_t, hipStream_t) { launched("launch_state_copy"); }
int conv_channels_per_thread() { return 8; }
hipError_t launch_conv(bool, const ConvArgs &, hipStream_t, hipEvent_t, hipEvent_t) { launched("launch_conv"); }
hipError_t launch_gdn_phase(int, const GdnArgs &, int, hipStream_t, hipEvent_t, hipEvent_t) {
    launched("launch_gdn_phase");
}
}  // namespace sf
