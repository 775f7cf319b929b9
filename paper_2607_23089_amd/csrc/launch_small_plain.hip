// Small-row family launcher, plain instantiations.
#include "launch.hpp"
#include "small_row.hpp"

namespace rowsm {
namespace {

template <typename In, typename Out, int VW, bool FUSED>
struct SmallLaunch {
  static int run(const Call& c) {
    const Plan& p = c.p;
    auto xp = static_cast<const typename In::storage*>(c.x);
    auto yp = static_cast<typename Out::storage*>(c.y);
    const Fused fz = fused_or_identity(c);
#define ROWSM_SMALL_CASE(L, R)                                                        \
    if constexpr (!FUSED || R == 4) {                                                 \
      if (p.lpr == L && p.rpl == R) {                                                 \
        small_row_kernel<In, Out, VW, L, R, FUSED>                                    \
            <<<dim3((unsigned)p.grid), dim3(p.block), 0, c.st>>>(xp, yp, c.rows, c.cols, fz); \
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

}  // namespace

int launch_small_plain(const Call& c, int in_dt, int out_dt) {
  return dispatch<SmallLaunch, false>(c, in_dt, out_dt);
}

}  // namespace rowsm
