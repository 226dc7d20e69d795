// Host-only stand-ins for the kernel launchers of the shard library, so that
// its host code (argument checks, layouts, the host plan, the host packer)
// can be built and run under AddressSanitizer and UndefinedBehaviorSanitizer
// on a machine without a GPU.  Every launcher reports "not supported"; the
// sanitizer driver never reaches one.
#include "bdl_launch.h"

namespace bdl {

hipError_t launch_dec_main(const DecArgs&, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_dec_epi(const DecArgs&, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_prep(const PrepArgs&, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_shrink(const FwdArgs&, int, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_gemm(const FwdArgs&, int, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_gemm_big(const FwdArgs&, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_gemm_mid(const FwdArgs&, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_mid_epi(const FwdArgs&, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_pack_adapter(uint16_t*, uint16_t*, const uint16_t*, int, int, const int*, int, int, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_pack_rows(const uint16_t*, uint16_t*, int, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_set_slots(int*, float*, int*, const SlotBatch&, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_pack_int4(const uint8_t*, const uint16_t*, uint32_t*, uint16_t*, int, int, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_mlp_pack(const float*, const float*, uint16_t*, int, int, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t static_scratch_init(int) { return hipErrorNotSupported; }
void* static_scratch(int) { return nullptr; }

}  // namespace bdl
