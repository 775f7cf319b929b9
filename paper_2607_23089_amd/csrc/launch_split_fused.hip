// Single-read split-row family launcher, fused instantiations.
#include <utility>

#include "launch.hpp"
#include "split_launch.hpp"

namespace rowsm {
namespace {

template <typename In, typename Out, int VW, bool FUSED, int... NVs>
int split_nv(const Call& c, std::integer_sequence<int, NVs...>) {
  int r = ROWSM_EINVAL;
  (void)((c.p.nv == NVs + 1 && (NVs + 1) * VW <= 64
              ? (r = launch_split_nv<In, Out, VW, ((NVs + 1) * VW <= 64 ? NVs + 1 : 1), FUSED>(c),
                 true)
              : false) ||
         ...);
  return r;
}

template <typename In, typename Out, int VW, bool FUSED>
struct SplitLaunch {
  static int run(const Call& c) {
    return split_nv<In, Out, VW, FUSED>(c, std::make_integer_sequence<int, 16>{});
  }
};

}  // namespace

int launch_split_fused(const Call& c, int in_dt, int out_dt) {
  return dispatch<SplitLaunch, true>(c, in_dt, out_dt);
}

}  // namespace rowsm
