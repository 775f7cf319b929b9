// Softmax-backward launchers, one per family (launch_bwd_<family>.hip).  A
// backward Call carries y in x, dy in dy and dx in y.
#pragma once

#include <utility>

#include "backward_row.hpp"
#include "launch.hpp"
#include "split_launch.hpp"

namespace rowsm {

template <typename In>
struct BwdPtrs {
  const typename In::storage* y;
  const typename In::storage* dy;
};

template <typename In>
inline BwdPtrs<In> bwd_inputs(const Call& c) {
  return {static_cast<const typename In::storage*>(c.x),
          static_cast<const typename In::storage*>(c.dy)};
}

// Compile-time slot counts of the register-resident forms: a lane holds at
// most 128 bytes of each input (NV * VW * In::bytes), and at most 16 slots.
template <typename In, int VW, int NV>
constexpr bool bwd_nv_compiled() {
  return NV >= 1 && NV <= 16 && NV * VW * In::bytes <= 128;
}

template <typename In, typename Out, int VW, int MODE>
struct BwdSmallLaunch {
  static int run(const Call& c) {
    const Plan& p = c.p;
    const BwdPtrs<In> in = bwd_inputs<In>(c);
    auto dxp = static_cast<typename Out::storage*>(c.y);
#define ROWSM_BWD_SMALL_CASE(L, R)                                                    \
    if (p.lpr == L && p.rpl == R) {                                                   \
      bwd_small_kernel<In, Out, VW, L, R><<<dim3((unsigned)p.grid), dim3(p.block), 0, c.st>>>( \
          in.y, in.dy, dxp, c.rows, c.cols);                                          \
      return hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;                 \
    }
#define ROWSM_BWD_SMALL_L(L) \
    ROWSM_BWD_SMALL_CASE(L, 1) ROWSM_BWD_SMALL_CASE(L, 2) ROWSM_BWD_SMALL_CASE(L, 4) \
    ROWSM_BWD_SMALL_CASE(L, 8)
    ROWSM_BWD_SMALL_L(1) ROWSM_BWD_SMALL_L(2) ROWSM_BWD_SMALL_L(4) ROWSM_BWD_SMALL_L(8)
    ROWSM_BWD_SMALL_L(16) ROWSM_BWD_SMALL_L(32)
#undef ROWSM_BWD_SMALL_L
#undef ROWSM_BWD_SMALL_CASE
    return ROWSM_EINVAL;
  }
};

template <typename In, typename Out, int VW, int NV>
bool try_bwd_medium(const Call& c, int* status) {
  if constexpr (bwd_nv_compiled<In, VW, NV>()) {
    if (c.p.nv == NV) {
      const BwdPtrs<In> in = bwd_inputs<In>(c);
      bwd_medium_kernel<In, Out, VW, NV><<<dim3((unsigned)c.p.grid), dim3(c.p.block), 0, c.st>>>(
          in.y, in.dy, static_cast<typename Out::storage*>(c.y), c.rows, c.cols, c.p.wpr);
      *status = hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
      return true;
    }
  }
  return false;
}

template <typename In, typename Out, int VW, int... NVs>
int bwd_medium_nv(const Call& c, std::integer_sequence<int, NVs...>) {
  int status = ROWSM_EINVAL;
  (void)(try_bwd_medium<In, Out, VW, NVs + 1>(c, &status) || ...);
  return status;
}

template <typename In, typename Out, int VW, int MODE>
struct BwdMediumLaunch {
  static int run(const Call& c) {
    return bwd_medium_nv<In, Out, VW>(c, std::make_integer_sequence<int, 16>{});
  }
};

template <typename In, typename Out, int VW, int NV>
int launch_bwd_split_nv(const Call& c) {
  const Plan& p = c.p;
  auto kern = bwd_split_kernel<In, Out, VW, NV>;
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(kern),
                                                   p.block, 0) != hipSuccess)
    return ROWSM_EHIP;
  const int64_t slots = split_slots(c, per_cu);
  if (slots < 1) return ROWSM_EINVAL;  // the S blocks of one row cannot be co-resident
  const unsigned grid = (unsigned)(slots * p.split);

  SplitTicket t;
  int r = split_begin(c, (uint64_t)((c.rows + slots - 1) / slots), &t);
  if (r != ROWSM_OK) return r;
  (void)hipGetLastError();
  const BwdPtrs<In> in = bwd_inputs<In>(c);
  kern<<<dim3(grid), dim3(p.block), 0, c.st>>>(in.y, in.dy,
                                               static_cast<typename Out::storage*>(c.y), c.rows,
                                               c.cols, p.split, t.ws, t.tag0);
  const bool launched = hipGetLastError() == hipSuccess;
  r = split_end(&t, c.st, launched);
  return launched ? r : ROWSM_EHIP;
}

template <typename In, typename Out, int VW, int... NVs>
int bwd_split_nv(const Call& c, std::integer_sequence<int, NVs...>) {
  int r = ROWSM_EINVAL;
  (void)((c.p.nv == NVs + 1 && bwd_nv_compiled<In, VW, NVs + 1>()
              ? (r = launch_bwd_split_nv<In, Out, VW,
                                         (bwd_nv_compiled<In, VW, NVs + 1>() ? NVs + 1 : 1)>(c),
                 true)
              : false) ||
         ...);
  return r;
}

template <typename In, typename Out, int VW, int MODE>
struct BwdSplitLaunch {
  static int run(const Call& c) {
    return bwd_split_nv<In, Out, VW>(c, std::make_integer_sequence<int, 16>{});
  }
};

template <typename In, typename Out, int VW, int MODE>
struct BwdLargeLaunch {
  static int run(const Call& c) {
    const BwdPtrs<In> in = bwd_inputs<In>(c);
    auto dxp = static_cast<typename Out::storage*>(c.y);
    const dim3 g((unsigned)c.p.grid), b(c.p.block);
    if (c.p.u == 2)
      bwd_large_kernel<In, Out, VW, 2><<<g, b, 0, c.st>>>(in.y, in.dy, dxp, c.rows, c.cols);
    else if (c.p.u == 4)
      bwd_large_kernel<In, Out, VW, 4><<<g, b, 0, c.st>>>(in.y, in.dy, dxp, c.rows, c.cols);
    else if (c.p.u == 8)
      bwd_large_kernel<In, Out, VW, 8><<<g, b, 0, c.st>>>(in.y, in.dy, dxp, c.rows, c.cols);
    else
      return ROWSM_EINVAL;
    return hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
  }
};

}  // namespace rowsm
