// MoE group-score launcher: dispatch on the group size G (2..64), the vector
// width and the groups per lane.  A Call carries the scores in x, the group
// scores in y, the number of groups in rows and G in cols; Plan::lpr is the
// lanes per group and Plan::rpl the groups per lane.  Instantiated once per
// input dtype (launch_moe_<dtype>.hip).
#pragma once

#include "group_top2.hpp"
#include "launch.hpp"

namespace rowsm {

template <typename In, typename Out, int VW, int G, int RPL>
bool try_moe(const Call& c, int* status) {
  if constexpr (G % VW == 0 && G / VW <= kWave) {
    if (c.cols == G && c.p.rpl == RPL) {
      group_top2_kernel<In, Out, VW, G / VW, RPL>
          <<<dim3((unsigned)c.p.grid), dim3(c.p.block), 0, c.st>>>(
              static_cast<const typename In::storage*>(c.x),
              static_cast<typename Out::storage*>(c.y), c.rows);
      *status = hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
      return true;
    }
  }
  return false;
}

template <typename In, typename Out, int VW, int G>
bool try_moe_rpl(const Call& c, int* status) {
  return try_moe<In, Out, VW, G, 1>(c, status) || try_moe<In, Out, VW, G, 2>(c, status) ||
         try_moe<In, Out, VW, G, 4>(c, status) || try_moe<In, Out, VW, G, 8>(c, status);
}

template <typename In, typename Out, int VW, int MODE>
struct MoeLaunch {
  static int run(const Call& c) {
    int status = ROWSM_EINVAL;
    (void)(try_moe_rpl<In, Out, VW, 2>(c, &status) || try_moe_rpl<In, Out, VW, 4>(c, &status) ||
           try_moe_rpl<In, Out, VW, 8>(c, &status) || try_moe_rpl<In, Out, VW, 16>(c, &status) ||
           try_moe_rpl<In, Out, VW, 32>(c, &status) || try_moe_rpl<In, Out, VW, 64>(c, &status));
    return status;
  }
};

// Input dtype fixed by the translation unit; output dtype and vector width
// at run time.
template <typename In>
int launch_moe_in(const Call& c, int out_dt) {
  auto out = [&](auto out_tag) -> int {
    using Out = decltype(out_tag);
    constexpr int V16 = 16 / In::bytes, V8 = 8 / In::bytes;
    if (c.p.vw == 1) return MoeLaunch<In, Out, 1, kMoe>::run(c);
    if (c.p.vw == V8) return MoeLaunch<In, Out, V8, kMoe>::run(c);
    if (c.p.vw == V16) return MoeLaunch<In, Out, V16, kMoe>::run(c);
    return ROWSM_EINVAL;
  };
  return out_dt == ROWSM_F32 ? out(F32{}) : out(BF16{});
}

}  // namespace rowsm
