// Host-side helpers shared by the C-ABI entry points: error reporting and
// plan validation.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "plan_data.h"

namespace tsp {

// Record a failure for talaria_sp_last_error() and return `code`.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Return the plan behind `plan` if it is a valid plan, else record EINVAL.
const PlanData* checked_plan(const talaria_sp_plan* plan, int* status);

// Map a HIP launch status to TALARIA_SP_OK / TALARIA_SP_EHIP.
int launch_status(const char* what);

// The kernels move bf16 rows and partials in 16-byte vectors.
inline bool aligned16(const void* a) { return ((uintptr_t)a & 15u) == 0; }

}  // namespace tsp

#if defined(__HIPCC__)
#include <hip/hip_runtime.h>
namespace tsp {
// Merge the split partials of a plan (f16 normalised outputs, fp32 base-2
// LSE) into out / lse (no-op when nothing is split).  Defined with the
// prefill kernel.
int launch_combine(const PlanData& p, const _Float16* part_o, const float* part_lse,
                   uint16_t* out, float* lse, hipStream_t st);
}  // namespace tsp
#endif

