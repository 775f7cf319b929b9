// MoE group score, bf16 scores.
#include "launch_moe.hpp"

namespace rowsm {
int launch_moe_bf16(const Call& c, int out_dt) { return launch_moe_in<BF16>(c, out_dt); }
}  // namespace rowsm
