// Kernel launchers for a host-only build of the library's C ABI (the
// sanitizer test in test_c_abi.py): the host-only entry points it exercises
// never launch a kernel, so every launcher here just reports failure. The
// declarations come from the library's internal header, so a signature that
// drifts fails to compile.
#include "lamb_internal.h"

namespace lamb_mi355x {

hipError_t launch_moments(const StepKind &, const TensorDesc *, const int32_t *, int32_t,
                          Partial *, int32_t, int32_t, uint32_t *, const uint32_t *, int32_t,
                          const StepArgs &, hipStream_t) {
    return hipErrorNotSupported;
}

hipError_t launch_finalize(NormKind, const TensorDesc *, int32_t, const Partial *, const SegDesc *,
                           int32_t, const SegRange *, Partial *, const FinalizeArgs &, float *,
                           double *, double *, uint32_t *, hipStream_t) {
    return hipErrorNotSupported;
}

hipError_t launch_apply(const StepKind &, const TensorDesc *, const int32_t *, int32_t,
                        const float *, int32_t, int32_t, uint32_t *, const uint32_t *, int32_t,
                        int32_t *, Partial *, const StepArgs &, hipStream_t) {
    return hipErrorNotSupported;
}

hipError_t launch_totals(NormKind, const Partial *, const SegDesc *, int32_t, const SegRange *,
                         int32_t, Partial *, double *, uint32_t *, const uint32_t *, int32_t,
                         hipStream_t) {
    return hipErrorNotSupported;
}

hipError_t launch_scale(NormKind, const double *, int32_t, const FinalizeArgs &, float *,
                        double *, double *, uint32_t *, hipStream_t) {
    return hipErrorNotSupported;
}

hipError_t launch_finite(bool, const TensorDesc *, const ChunkDesc *, int32_t, uint32_t *,
                         const uint32_t *, float, hipStream_t) {
    return hipErrorNotSupported;
}

hipError_t launch_fused(const StepKind &, int, const TensorDesc *, const ChunkDesc *, int32_t,
                        int32_t, uint64_t *, uint32_t *, uint32_t *, bool, int32_t *,
                        const StepArgs &, const FinalizeArgs &, double *, double *,
                        const double *, float *, uint64_t *, hipStream_t) {
    return hipErrorNotSupported;
}

hipError_t fused_blocks_per_cu(const StepKind &, int, int *) { return hipErrorNotSupported; }

}  // namespace lamb_mi355x
