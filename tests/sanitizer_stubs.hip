// Launcher stubs for the sanitizer build of libags's host code (test
// infrastructure): that build leaves out the file of the step, finalize,
// correction and update kernels, and the host-side tests it runs never
// reach a launch.
#include "ags_internal.h"

namespace ags {

hipError_t launch_step(const StepArgs&, ags_dtype, int, bool, hipStream_t, KernelEvents) {
    return hipErrorInvalidDeviceFunction;
}
hipError_t launch_finalize(const StepArgs&, int, hipStream_t, KernelEvents) {
    return hipErrorInvalidDeviceFunction;
}
hipError_t launch_update(const UpdateArgs&, ags_dtype, hipStream_t, KernelEvents) {
    return hipErrorInvalidDeviceFunction;
}
hipError_t launch_correct(const UpdateArgs&, ags_dtype, hipStream_t, KernelEvents) {
    return hipErrorInvalidDeviceFunction;
}
hipError_t launch_set_lr(DevState*, float, hipStream_t) {
    return hipErrorInvalidDeviceFunction;
}

}  // namespace ags
