// Two-pass large-row family launcher: dispatch on the tile depth U.
// Instantiated once per output form (launch_large_<form>.hip).
#pragma once

#include "large_row.hpp"
#include "launch.hpp"

namespace rowsm {

template <typename In, typename Out, int VW, int MODE>
struct LargeLaunch {
  static int run(const Call& c) {
    auto xp = static_cast<const typename In::storage*>(c.x);
    auto yp = static_cast<typename Out::storage*>(c.y);
    const dim3 g((unsigned)c.p.grid), b(c.p.block);
    if (c.p.u == 2)
      large_row_kernel<In, Out, VW, 2, MODE><<<g, b, 0, c.st>>>(xp, yp, c.rows, c.cols, c.fz);
    else if (c.p.u == 4)
      large_row_kernel<In, Out, VW, 4, MODE><<<g, b, 0, c.st>>>(xp, yp, c.rows, c.cols, c.fz);
    else if (c.p.u == 8)
      large_row_kernel<In, Out, VW, 8, MODE><<<g, b, 0, c.st>>>(xp, yp, c.rows, c.cols, c.fz);
    else
      return ROWSM_EINVAL;
    return hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
  }
};

template <int MODE>
int launch_large(const Call& c, int in_dt, int out_dt) {
  return dispatch<LargeLaunch, MODE>(c, in_dt, out_dt);
}

}  // namespace rowsm
