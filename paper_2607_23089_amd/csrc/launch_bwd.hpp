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
  auto kern = bwd_split_kernel<In, Out, VW, NV>;
  const BwdPtrs<In> in = bwd_inputs<In>(c);
  return launch_exchanging(c, kern, c.p.split, [&](unsigned grid, SplitWorkspace ws, uint32_t tag0) {
    kern<<<dim3(grid), dim3(c.p.block), 0, c.st>>>(in.y, in.dy,
                                                  static_cast<typename Out::storage*>(c.y),
                                                  c.rows, c.cols, c.p.split, ws, tag0);
  });
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

// Two-pass backward: one block per row (p.stream == 1, grid p.grid), or
// p.stream blocks per row that exchange their partial dot products.
template <typename In, typename Out, int VW, int U>
int launch_bwd_large_u(const Call& c) {
  auto kern = bwd_large_kernel<In, Out, VW, U>;
  const BwdPtrs<In> in = bwd_inputs<In>(c);
  auto dxp = static_cast<typename Out::storage*>(c.y);
  if (c.p.stream <= 1) {
    (void)hipGetLastError();
    kern<<<dim3((unsigned)c.p.grid), dim3(c.p.block), 0, c.st>>>(in.y, in.dy, dxp, c.rows,
                                                                  c.cols, 1, SplitWorkspace{}, 0);
    return hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
  }
  return launch_exchanging(c, kern, c.p.stream, [&](unsigned grid, SplitWorkspace ws,
                                                    uint32_t tag0) {
    kern<<<dim3(grid), dim3(c.p.block), 0, c.st>>>(in.y, in.dy, dxp, c.rows, c.cols, c.p.stream,
                                                  ws, tag0);
  });
}

template <typename In, typename Out, int VW, int MODE>
struct BwdLargeLaunch {
  static int run(const Call& c) {
    if (c.p.u == 2) return launch_bwd_large_u<In, Out, VW, 2>(c);
    if (c.p.u == 4) return launch_bwd_large_u<In, Out, VW, 4>(c);
    if (c.p.u == 8) return launch_bwd_large_u<In, Out, VW, 8>(c);
    return ROWSM_EINVAL;
  }
};

}  // namespace rowsm
