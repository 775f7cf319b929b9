// MoE group score, fp32 scores.
#include "launch_moe.hpp"

namespace rowsm {
int launch_moe_f32(const Call& c, int out_dt) { return launch_moe_in<F32>(c, out_dt); }
}  // namespace rowsm
