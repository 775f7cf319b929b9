// Two-pass large-row family launcher, fused instantiations.
#include "large_row.hpp"
#include "launch.hpp"

namespace rowsm {
namespace {

template <typename In, typename Out, int VW, bool FUSED>
struct LargeLaunch {
  static int run(const Call& c) {
    auto xp = static_cast<const typename In::storage*>(c.x);
    auto yp = static_cast<typename Out::storage*>(c.y);
    const dim3 g((unsigned)c.p.grid), b(c.p.block);
    const Fused fz = fused_or_identity(c);
    if (c.p.u == 2)
      large_row_kernel<In, Out, VW, 2, FUSED><<<g, b, 0, c.st>>>(xp, yp, c.rows, c.cols, fz);
    else if (c.p.u == 4)
      large_row_kernel<In, Out, VW, 4, FUSED><<<g, b, 0, c.st>>>(xp, yp, c.rows, c.cols, fz);
    else if (c.p.u == 8)
      large_row_kernel<In, Out, VW, 8, FUSED><<<g, b, 0, c.st>>>(xp, yp, c.rows, c.cols, fz);
    else
      return ROWSM_EINVAL;
    return hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
  }
};

}  // namespace

int launch_large_fused(const Call& c, int in_dt, int out_dt) {
  return dispatch<LargeLaunch, true>(c, in_dt, out_dt);
}

}  // namespace rowsm
