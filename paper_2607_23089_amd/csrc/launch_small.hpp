// Small-row family launcher: the (lanes per row, rows per lane) dispatch.
// Instantiated once per output form (launch_small_<form>.hip).
#pragma once

#include "launch.hpp"
#include "small_row.hpp"

namespace rowsm {

template <typename In, typename Out, int VW, int MODE>
struct SmallLaunch {
  static int run(const Call& c) {
    const Plan& p = c.p;
    auto xp = static_cast<const typename In::storage*>(c.x);
    auto yp = static_cast<typename Out::storage*>(c.y);
    // The fused form is compiled for 4 rows per lane only.
#define ROWSM_SMALL_CASE(L, R)                                                        \
    if constexpr (MODE != kFused || R == 4) {                                         \
      if (p.lpr == L && p.rpl == R) {                                                 \
        small_row_kernel<In, Out, VW, L, R, MODE>                                     \
            <<<dim3((unsigned)p.grid), dim3(p.block), 0, c.st>>>(xp, yp, c.rows, c.cols, c.fz); \
        return hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;               \
      }                                                                               \
    }
#define ROWSM_SMALL_L(L) \
    ROWSM_SMALL_CASE(L, 1) ROWSM_SMALL_CASE(L, 2) ROWSM_SMALL_CASE(L, 4) ROWSM_SMALL_CASE(L, 8)
    ROWSM_SMALL_L(1) ROWSM_SMALL_L(2) ROWSM_SMALL_L(4) ROWSM_SMALL_L(8) ROWSM_SMALL_L(16)
    ROWSM_SMALL_L(32)
#undef ROWSM_SMALL_L
#undef ROWSM_SMALL_CASE
    return ROWSM_EINVAL;
  }
};

template <int MODE>
int launch_small(const Call& c, int in_dt, int out_dt) {
  return dispatch<SmallLaunch, MODE>(c, in_dt, out_dt);
}

}  // namespace rowsm
