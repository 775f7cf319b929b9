// Medium-row family launcher, plain instantiations.
#include <type_traits>
#include <utility>

#include "launch.hpp"
#include "medium_row.hpp"

namespace rowsm {
namespace {

template <typename In, typename Out, int VW, int NV, bool PACKED, bool FUSED>
bool try_medium(const Call& c, int* status) {
  constexpr bool compiled =
      PACKED ? (!FUSED && std::is_same<In, BF16>::value && VW == 8 && NV >= 9 && NV <= 24)
             : (NV * VW <= 64 && NV <= 16);
  if constexpr (compiled) {
    if (c.p.nv == NV && c.p.packed == PACKED) {
      medium_row_kernel<In, Out, VW, NV, PACKED, FUSED>
          <<<dim3((unsigned)c.p.grid), dim3(c.p.block), 0, c.st>>>(
              static_cast<const typename In::storage*>(c.x),
              static_cast<typename Out::storage*>(c.y), c.rows, c.cols, c.p.wpr,
              fused_or_identity(c));
      *status = hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
      return true;
    }
  }
  return false;
}

template <typename In, typename Out, int VW, bool PACKED, bool FUSED, int... NVs>
int medium_nv(const Call& c, std::integer_sequence<int, NVs...>) {
  int status = ROWSM_EINVAL;
  (void)(try_medium<In, Out, VW, NVs + 1, PACKED, FUSED>(c, &status) || ...);
  return status;
}

template <typename In, typename Out, int VW, bool FUSED>
struct MediumLaunch {
  static int run(const Call& c) {
    if (c.p.packed)
      return medium_nv<In, Out, VW, true, FUSED>(c, std::make_integer_sequence<int, 24>{});
    return medium_nv<In, Out, VW, false, FUSED>(c, std::make_integer_sequence<int, 16>{});
  }
};

}  // namespace

int launch_medium_plain(const Call& c, int in_dt, int out_dt) {
  return dispatch<MediumLaunch, false>(c, in_dt, out_dt);
}

}  // namespace rowsm
