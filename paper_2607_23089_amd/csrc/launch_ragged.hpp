// Launcher of the medium kernel for rows of a width that is not a multiple
// of the vector width (ragged_row.hpp): the full 16-byte vector width of the
// dtype pair, dispatch on the compile-time slot count.  Instantiated once
// per output form (launch_ragged_<form>.hip).
#pragma once

#include <utility>

#include "launch.hpp"
#include "ragged_row.hpp"

namespace rowsm {

// Values per lane of the ragged kernels: at most 40 (about 100 VGPRs at the
// cap, within the 1024-thread launch bound's 128).
template <typename In, typename Out>
constexpr int ragged_cap() {
  return 40;
}

template <typename In, typename Out, int VW, int NV, int MODE>
bool try_ragged(const Call& c, int* status) {
  if constexpr (NV * VW <= ragged_cap<In, Out>()) {
    if (c.p.nv == NV) {
      ragged_row_kernel<In, Out, VW, NV, MODE>
          <<<dim3((unsigned)c.p.grid), dim3(c.p.block), 0, c.st>>>(
              static_cast<const typename In::storage*>(c.x),
              static_cast<typename Out::storage*>(c.y), c.rows, c.cols, c.p.wpr);
      *status = hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
      return true;
    }
  }
  return false;
}

template <typename In, typename Out, int MODE, int... NVs>
int ragged_nv(const Call& c, std::integer_sequence<int, NVs...>) {
  constexpr int VW = 16 / (In::bytes > Out::bytes ? In::bytes : Out::bytes);
  int status = ROWSM_EINVAL;
  if (c.p.vw != VW) return status;
  (void)(try_ragged<In, Out, VW, NVs + 1, MODE>(c, &status) || ...);
  return status;
}

template <int MODE>
int launch_ragged(const Call& c, int in_dt, int out_dt) {
  constexpr auto seq = std::make_integer_sequence<int, 16>{};
  if (in_dt == ROWSM_F32 && out_dt == ROWSM_F32) return ragged_nv<F32, F32, MODE>(c, seq);
  if (in_dt == ROWSM_F32) return ragged_nv<F32, BF16, MODE>(c, seq);
  if (out_dt == ROWSM_F32) return ragged_nv<BF16, F32, MODE>(c, seq);
  return ragged_nv<BF16, BF16, MODE>(c, seq);
}

}  // namespace rowsm
