// Launchers of a host-only build of the library (no device code): every
// launch reports that no device is present, so an entry point that reaches a
// launch returns NA_ERR_HIP.  Linked with na_api.cpp into the sanitizer build
// of libna.so that the CPU test suite loads through NA_LIBRARY.
#include "na_launch.h"

namespace na {

hipError_t launch_forward(const Geo&, int, int, int, int, const void*, const void*, const void*,
                          void*, float*, float, hipStream_t) {
    return hipErrorNoDevice;
}

hipError_t launch_backward(const Geo&, int, int, int, int, const void*, const void*, const void*,
                           const void*, const float*, const void*, void*, void*, void*, float,
                           hipStream_t) {
    return hipErrorNoDevice;
}

hipError_t launch_unfused(const UGeo&, int, int, int, const void*, const void*, void*, float*,
                          float, hipStream_t) {
    return hipErrorNoDevice;
}

hipError_t launch_debug_windows(int, const int*, const int*, const int*, const int*, int*, int*,
                                int*, hipStream_t) {
    return hipErrorNoDevice;
}

}  // namespace na
