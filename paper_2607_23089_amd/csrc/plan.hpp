// Launch planning of the row-softmax library (plan.hip): what the template
// dispatch and the C ABI (rowsm.hip) need from the launcher.  Each plan_*
// call fills a Plan for one call's shape, dtypes, pointer alignments and
// config overrides, and returns ROWSM_OK or ROWSM_EINVAL when the requested
// family or override cannot take that shape; it launches nothing.
#pragma once

#include <stdint.h>

#include "launch.hpp"

namespace rowsm {

// Compute-unit count of the current device (cached per device; 256 when no
// device can be queried).
int cu_count();

int dtype_bytes(int dt);  // 4 for ROWSM_F32, 2 for ROWSM_BF16
bool dtype_ok(int dt);    // ROWSM_F32 or ROWSM_BF16

// Forward plan for mode kPlain, kFused or kLog over rows x cols, x at address
// xa and y at ya (alignment only), on a device of cus compute units; inplace
// (y == x) excludes the forms whose blocks exchange partial results.
int plan_for(int64_t rows, int64_t cols, int in_dt, int out_dt, uintptr_t xa, uintptr_t ya,
             const rowsm_config* cfg, int cus, int mode, bool inplace, Plan* p);

// Backward plan: ia is the alignment of the inputs y and dy together, dxa of
// the output dx; inplace (dx == y or dx == dy) as plan_for().
int plan_backward(int64_t rows, int64_t cols, int in_dt, int out_dt, uintptr_t ia,
                  uintptr_t dxa, const rowsm_config* cfg, int cus, bool inplace, Plan* p);

// Grouped top-2 plan over ngroups groups of g scores at address sa.
int plan_moe(int64_t ngroups, int64_t g, int in_dt, uintptr_t sa, const rowsm_config* cfg,
             int cus, Plan* p);

// A group size the grouped top-2 kernels take: a power of two in [2, 64].
bool moe_group_ok(int64_t g);

}  // namespace rowsm
