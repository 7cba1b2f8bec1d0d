// Host-side helpers of the C ABI (defined in lamb_api.cpp) that every source
// file implementing entry points of include/lamb_mi355x.h uses: error
// reporting, validation of tensor tables and hyperparameters, and the
// per-step kernel scalars. Not installed.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "lamb_internal.h"
#include "lamb_mi355x.h"

namespace lamb_mi355x {

constexpr int64_t kMaxChunkElems = int64_t(1) << 30;
constexpr int64_t kMaxNumel = int64_t(1) << 40;  // elements per tensor

// Records the calling thread's error detail (lamb_last_error) and returns
// `status`.
lamb_status fail(lamb_status status, const char *fmt, ...)
    __attribute__((format(printf, 2, 3)));
lamb_status fail_hip(hipError_t err, const char *what);

// chunk_elems as lamb_plan_create takes it: 0 picks the default.
lamb_status resolve_chunk_elems(int32_t requested, int32_t *out);

// A buffer of the tensor table, for the overlap check.
struct BufferRange {
    uintptr_t lo, hi;
    int32_t tensor;
    const char *what;
};

// Validates a table of blocks (as lamb_plan_create documents) using the
// caller's room for 4 * n ranges, which it leaves sorted; allocates nothing.
lamb_status check_table(const lamb_tensor *tensors, int32_t n_tensors, lamb_grad_dtype g_dtype,
                        bool needs_v, BufferRange *ranges, int32_t *n_ranges);

// Validates one step's hyperparameters before any HIP call; `plan` may be
// null (a planless step), otherwise the variant must match its algorithm.
lamb_status check_hparams(const lamb_plan *plan, const lamb_hparams *hp,
                          const int32_t *nonfinite_out);

// fp32 kernel scalars, kernel choice and finalize scalars of a validated step.
StepArgs step_args(const lamb_hparams &hp);
StepKind step_kind(const lamb_hparams &hp, lamb_grad_dtype g_dtype);
FinalizeArgs finalize_args(const lamb_hparams &hp);

}  // namespace lamb_mi355x
