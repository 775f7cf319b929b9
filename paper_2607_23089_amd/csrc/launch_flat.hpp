// Launcher of the flat short-row kernel (flat_row.hpp): the full 16-byte
// vector width of the dtype pair, dispatch on the lanes per row and elements
// per lane of the row phase.  Instantiated once per output form and for the
// backward (launch_flat_<form>.hip; for the backward c.x is y, c.dy is dy and
// c.y is dx).
#pragma once

#include "flat_row.hpp"
#include "launch.hpp"

namespace rowsm {

template <typename In, typename Out, int VW, int LPR, int E, int MODE>
bool try_flat(const Call& c, int* status) {
  if (c.p.lpr != LPR || c.p.nv != E) return false;
  // vectors per lane of a tile (c.p.rpl): 4, or 2 for bf16 to bf16
  constexpr bool kTwo = In::bytes == 2 && Out::bytes == 2;
  const int slots = kTwo && c.p.rpl == 2 ? 2 : kFlatSlots;
  if (c.p.rpl != slots) return false;
  const int G = (slots * kWave * VW - (VW - 1)) / c.cols;
  if (G < 1) return false;
  if constexpr (MODE == kBackward) {
    const auto yp = static_cast<const typename In::storage*>(c.x);
    const auto dyp = static_cast<const typename In::storage*>(c.dy);
    const auto dxp = static_cast<typename Out::storage*>(c.y);
    if (slots == 2) {
      if constexpr (kTwo)
        bwd_flat_kernel<In, Out, VW, LPR, E, 2><<<dim3((unsigned)c.p.grid), dim3(kWave), 0, c.st>>>(
            yp, dyp, dxp, c.rows, c.cols, G);
    } else {
      bwd_flat_kernel<In, Out, VW, LPR, E, kFlatSlots>
          <<<dim3((unsigned)c.p.grid), dim3(kWave), 0, c.st>>>(yp, dyp, dxp, c.rows, c.cols, G);
    }
  } else {
    const auto xp = static_cast<const typename In::storage*>(c.x);
    const auto yp = static_cast<typename Out::storage*>(c.y);
    if (slots == 2) {
      if constexpr (kTwo)
        flat_row_kernel<In, Out, VW, LPR, E, MODE, 2>
            <<<dim3((unsigned)c.p.grid), dim3(kWave), 0, c.st>>>(xp, yp, c.rows, c.cols, G);
    } else {
      flat_row_kernel<In, Out, VW, LPR, E, MODE, kFlatSlots>
          <<<dim3((unsigned)c.p.grid), dim3(kWave), 0, c.st>>>(xp, yp, c.rows, c.cols, G);
    }
  }
  *status = hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
  return true;
}

// (lanes per row, elements per lane): LPR = max(8, pow2 >= cols / 8) up to 64,
// 4 for rows of at most 16 columns, E the power of two >= cols / LPR
// (flat_row_shape() in plan.hip).
template <typename In, typename Out, int MODE>
int flat_pair(const Call& c) {
  constexpr int VW = 16 / (In::bytes > Out::bytes ? In::bytes : Out::bytes);
  int status = ROWSM_EINVAL;
  if (c.p.vw != VW || c.p.block != kWave) return status;
  (void)(try_flat<In, Out, VW, 8, 2, MODE>(c, &status) ||
         try_flat<In, Out, VW, 8, 4, MODE>(c, &status) ||
         try_flat<In, Out, VW, 8, 8, MODE>(c, &status) ||
         try_flat<In, Out, VW, 16, 8, MODE>(c, &status) ||
         try_flat<In, Out, VW, 32, 8, MODE>(c, &status) ||
         try_flat<In, Out, VW, 64, 8, MODE>(c, &status) ||
         try_flat<In, Out, VW, 64, 16, MODE>(c, &status) ||
         try_flat<In, Out, VW, 4, 4, MODE>(c, &status));
  return status;
}

template <int MODE>
int launch_flat(const Call& c, int in_dt, int out_dt) {
  if (in_dt == ROWSM_F32 && out_dt == ROWSM_F32) return flat_pair<F32, F32, MODE>(c);
  if (in_dt == ROWSM_F32) return flat_pair<F32, BF16, MODE>(c);
  if (out_dt == ROWSM_F32) return flat_pair<BF16, F32, MODE>(c);
  return flat_pair<BF16, BF16, MODE>(c);
}

}  // namespace rowsm
