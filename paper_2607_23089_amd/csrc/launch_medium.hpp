// Medium-row family launcher: dispatch on the compile-time slot count and
// the packed/unpacked form.  Instantiated once per output form
// (launch_medium_<form>.hip).
#pragma once

#include <type_traits>
#include <utility>

#include "launch.hpp"
#include "medium_row.hpp"

namespace rowsm {

template <typename In, typename Out, int VW, int NV, bool PACKED, int MODE>
bool try_medium(const Call& c, int* status) {
  // Slot counts the planner can choose: fused rows hold at most 32 values
  // per lane (the column indices are live too), the others 64.
  constexpr bool compiled =
      PACKED ? (MODE != kFused && std::is_same<In, BF16>::value && VW == 8 && NV >= 9 &&
                NV <= 24)
             : (NV * VW <= (MODE == kFused ? 32 : 64) && NV <= 16);
  if constexpr (compiled) {
    if (c.p.nv == NV && c.p.packed == PACKED) {
      medium_row_kernel<In, Out, VW, NV, PACKED, MODE>
          <<<dim3((unsigned)c.p.grid), dim3(c.p.block), 0, c.st>>>(
              static_cast<const typename In::storage*>(c.x),
              static_cast<typename Out::storage*>(c.y), c.rows, c.cols, c.p.wpr, c.fz);
      *status = hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
      return true;
    }
  }
  return false;
}

template <typename In, typename Out, int VW, bool PACKED, int MODE, int... NVs>
int medium_nv(const Call& c, std::integer_sequence<int, NVs...>) {
  int status = ROWSM_EINVAL;
  (void)(try_medium<In, Out, VW, NVs + 1, PACKED, MODE>(c, &status) || ...);
  return status;
}

template <typename In, typename Out, int VW, int MODE>
struct MediumLaunch {
  static int run(const Call& c) {
    if (c.p.packed)
      return medium_nv<In, Out, VW, true, MODE>(c, std::make_integer_sequence<int, 24>{});
    return medium_nv<In, Out, VW, false, MODE>(c, std::make_integer_sequence<int, 16>{});
  }
};

template <int MODE>
int launch_medium(const Call& c, int in_dt, int out_dt) {
  return dispatch<MediumLaunch, MODE>(c, in_dt, out_dt);
}

}  // namespace rowsm
