// Two-pass large-row family launcher: one block per row (p.stream == 1, grid
// p.grid), or p.stream blocks per row that exchange their (max, sum) pairs
// through the split form's workspace; dispatch on the tile depth U.
// Instantiated once per output form (launch_large_<form>.hip).
#pragma once

#include "large_row.hpp"
#include "launch.hpp"
#include "split_launch.hpp"

namespace rowsm {

template <typename In, typename Out, int VW, int U, int MODE>
int launch_large_u(const Call& c) {
  auto kern = large_row_kernel<In, Out, VW, U, MODE>;
  auto xp = static_cast<const typename In::storage*>(c.x);
  auto yp = static_cast<typename Out::storage*>(c.y);
  if (c.p.stream <= 1) {
    (void)hipGetLastError();
    kern<<<dim3((unsigned)c.p.grid), dim3(c.p.block), 0, c.st>>>(xp, yp, c.rows, c.cols, 1,
                                                                  SplitWorkspace{}, 0, c.fz);
    return hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
  }
  return launch_exchanging(c, kern, c.p.stream, [&](unsigned grid, SplitWorkspace ws,
                                                    uint32_t tag0) {
    kern<<<dim3(grid), dim3(c.p.block), 0, c.st>>>(xp, yp, c.rows, c.cols, c.p.stream, ws, tag0,
                                                  c.fz);
  });
}

template <typename In, typename Out, int VW, int MODE>
struct LargeLaunch {
  static int run(const Call& c) {
    if (c.p.u == 2) return launch_large_u<In, Out, VW, 2, MODE>(c);
    if (c.p.u == 4) return launch_large_u<In, Out, VW, 4, MODE>(c);
    if (c.p.u == 8) return launch_large_u<In, Out, VW, 8, MODE>(c);
    return ROWSM_EINVAL;
  }
};

template <int MODE>
int launch_large(const Call& c, int in_dt, int out_dt) {
  return dispatch<LargeLaunch, MODE>(c, in_dt, out_dt);
}

}  // namespace rowsm
