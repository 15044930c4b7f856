// Stand-ins for the kernel launchers, linked instead of the kernels into the
// sanitized build of the C ABI's host code (tests/abi_sanitizer_driver.c):
// every case that driver runs must be settled by validation, so any call
// here is counted and reported as a failure.
#include "zpp_launch.h"

extern "C" {
int zpp_test_launches = 0;
}

namespace zpp {

namespace {
hipError_t reached() {
    ++zpp_test_launches;
    return hipErrorNotSupported;
}
}  // namespace

hipError_t launch_adam(float *, float *, float *, const float *, uint16_t *, size_t,
                       const AdamConsts &, bool, hipStream_t) {
    return reached();
}
hipError_t launch_refresh(uint16_t *, const uint16_t *, size_t, bool, hipStream_t) {
    return reached();
}
hipError_t launch_quantize(const uint16_t *, size_t, uint32_t, int8_t *, float *, bool,
                           hipStream_t) {
    return reached();
}
hipError_t launch_quantize_copy(const uint16_t *, size_t, uint32_t, int8_t *, float *, uint16_t *,
                                bool, hipStream_t) {
    return reached();
}
hipError_t launch_fused(float *, float *, float *, const float *, uint16_t *, uint16_t *, int8_t *,
                        float *, size_t, uint32_t, const AdamConsts &, bool, hipStream_t) {
    return reached();
}
hipError_t launch_gather(const GatherShards &, uint32_t, size_t, uint32_t, size_t, uint16_t *,
                         bool, hipStream_t) {
    return reached();
}
hipError_t launch_quantize_i4(const float *, size_t, uint32_t, uint8_t *, float *, bool,
                              hipStream_t) {
    return reached();
}
hipError_t launch_dequant_reduce_i4(const uint8_t *const *, const float *const *, uint32_t, size_t,
                                    uint32_t, float, float *, bool, hipStream_t) {
    return reached();
}
hipError_t launch_fused_receive(float *, float *, float *, const uint8_t *const *,
                                const float *const *, uint32_t, uint32_t, float, uint16_t *,
                                uint16_t *, int8_t *, float *, size_t, uint32_t,
                                const AdamConsts &, bool, hipStream_t) {
    return reached();
}
hipError_t launch_receive_adam(float *, float *, float *, const uint8_t *const *,
                               const float *const *, uint32_t, uint32_t, float, uint16_t *, size_t,
                               const AdamConsts &, bool, hipStream_t) {
    return reached();
}

hipError_t launch_quantize_i4_il(const float *, size_t, uint32_t, uint32_t, uint32_t, uint8_t *,
                                 float *, bool, hipStream_t) {
    return reached();
}
hipError_t launch_dequant_reduce_i4_il(const uint8_t *, const float *, uint32_t, size_t, uint32_t,
                                       float, float *, bool, hipStream_t) {
    return reached();
}
hipError_t launch_receive_adam_il(float *, float *, float *, const uint8_t *, const float *,
                                  uint32_t, uint32_t, float, uint16_t *, size_t, const AdamConsts &,
                                  bool, hipStream_t) {
    return reached();
}
hipError_t launch_fused_receive_il(float *, float *, float *, const uint8_t *, const float *,
                                   uint32_t, uint32_t, float, uint16_t *, uint16_t *, int8_t *,
                                   float *, size_t, uint32_t, const AdamConsts &, bool,
                                   hipStream_t) {
    return reached();
}

}  // namespace zpp
