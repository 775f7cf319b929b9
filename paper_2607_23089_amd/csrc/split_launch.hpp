// Launch of the single-read split-row kernels: grid sizing from occupancy,
// the exchange workspace (launch_split_common.hip), and the dispatch on the
// compile-time slot count, instantiated once per output form
// (launch_split_<form>.hip).
#pragma once

#include <utility>

#include "launch.hpp"
#include "split_row.hpp"

namespace rowsm {

// Row groups of S blocks in a launch of an exchanging form with occupancy
// per_cu blocks per compute unit and room for max_blocks blocks in its
// exchange workspace, or 0 when the S blocks of one row cannot be resident
// at once.
//   p.grid == 0  one group per row (up to the workspace room, beyond which
//                groups loop over rows): a block exits after its row, so a
//                new block starts loading while the stores of the last one
//                drain.  A block that moves on to another row must first see
//                its stores acknowledged (loads and stores retire through one
//                in-order counter), which measured 3-8% slower on long rows
//                than groups that exit.
//   p.grid < 0   at most -p.grid blocks per compute unit and one full
//                residency of the device: each group loops over rows.
//   S is the launch's blocks per row (p.split, or p.stream for the two-pass
//   form, whose grid is always one group per row).
inline int64_t split_slots(const Call& c, int per_cu, int S, int64_t max_blocks) {
  const Plan& p = c.p;
  if ((int64_t)per_cu * c.cus < S) return 0;
  int64_t slots = c.rows;
  if (p.grid < 0) {
    const int64_t cap = per_cu > -p.grid ? -p.grid : per_cu;
    slots = cap * c.cus / S;
  }
  if (slots > c.rows) slots = c.rows;
  if (slots > max_blocks / S) slots = max_blocks / S;
  return slots;
}

// The exchange workspace of one launch (launch_split_common.hip): a region of
// 32 bytes per block in the device's exchange ring, the give-up counter, the
// wait limit, and ntags consecutive 32-bit tags.  When the stream is being
// captured, exchange_begin() first enqueues a kernel that clears the region
// (a graph replays the tags recorded at capture).
struct Exchange {
  SplitWorkspace ws{};
  uint32_t tag0 = 0;
};
// The ring a launch takes its region from (resolved per launch).
struct ExchangeRing {
  void* ring = nullptr;
  uint32_t* failures = nullptr;
  int64_t max_blocks = 0;  // blocks one launch may take
  bool capturing = false;  // the launch stream is being captured
};
int exchange_ring(const Call& c, ExchangeRing* r);
int exchange_begin(const Call& c, const ExchangeRing& r, int64_t blocks, uint64_t ntags,
                   Exchange* e);

// Launch of a kernel whose S > 1 blocks per row exchange through the
// workspace (the single-read forms, and the two-pass forms with more than
// one block per row): occupancy check, grid, region and tags, then
// go(grid, workspace, tag0) enqueues the kernel itself.  Nothing here waits
// for or orders against any other launch.
template <typename Kern, typename Go>
int launch_exchanging(const Call& c, Kern kern, int S, Go go) {
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(kern),
                                                   c.p.block, 0) != hipSuccess)
    return ROWSM_EHIP;
  ExchangeRing ring;
  int r = exchange_ring(c, &ring);
  if (r != ROWSM_OK) return r;
  const int64_t slots = split_slots(c, per_cu, S, ring.max_blocks);
  if (slots < 1) return ROWSM_EINVAL;  // the S blocks of one row cannot be co-resident
  const unsigned grid = (unsigned)(slots * S);
  Exchange e;
  r = exchange_begin(c, ring, (int64_t)grid, (uint64_t)((c.rows + slots - 1) / slots), &e);
  if (r != ROWSM_OK) return r;
  (void)hipGetLastError();
  go(grid, e.ws, e.tag0);
  return hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
}

template <typename In, typename Out, int VW, int NV, int MODE, bool PIPE>
int launch_split_nv(const Call& c) {
  auto kern = split_row_kernel<In, Out, VW, NV, MODE, PIPE>;
  return launch_exchanging(c, kern, c.p.split, [&](unsigned grid, SplitWorkspace ws, uint32_t tag0) {
    kern<<<dim3(grid), dim3(c.p.block), 0, c.st>>>(
        static_cast<const typename In::storage*>(c.x), static_cast<typename Out::storage*>(c.y),
        c.rows, c.cols, c.p.split, ws, tag0, c.fz);
  });
}

// Values per lane the prefetching form holds at most: the next row's raw
// share comes on top of the current one (more spilled on gfx950): 48, or 44
// for fp32 rows, whose raw share takes a register per value.
template <typename In, typename Out>
constexpr int split_prefetch_max_values() {
  return In::bytes == 4 ? 44 : 48;
}

// Values per lane the planner can choose: 32 for fused rows, 64 otherwise.
template <int MODE>
constexpr int split_max_values() {
  return MODE == kFused ? 32 : 64;
}

template <typename In, typename Out, int VW, int MODE, int... NVs>
int split_nv(const Call& c, std::integer_sequence<int, NVs...>) {
  constexpr int MAXV = split_max_values<MODE>();
  // prefetching: plain and log forms only (the fused form keeps column
  // indices live as well)
  constexpr int PMAXV = MODE == kFused ? 0 : split_prefetch_max_values<In, Out>();
  int r = ROWSM_EINVAL;
  (void)((c.p.nv == NVs + 1 && (NVs + 1) * VW <= MAXV
              ? (r = c.p.prefetch
                         ? ((NVs + 1) * VW <= PMAXV
                                ? launch_split_nv<In, Out, VW,
                                                  ((NVs + 1) * VW <= PMAXV ? NVs + 1 : 1), MODE,
                                                  true>(c)
                                : ROWSM_EINVAL)
                         : launch_split_nv<In, Out, VW, ((NVs + 1) * VW <= MAXV ? NVs + 1 : 1),
                                           MODE, false>(c),
                 true)
              : false) ||
         ...);
  return r;
}

template <typename In, typename Out, int VW, int MODE>
struct SplitLaunch {
  static int run(const Call& c) {
    return split_nv<In, Out, VW, MODE>(c, std::make_integer_sequence<int, 16>{});
  }
};

template <int MODE>
int launch_split(const Call& c, int in_dt, int out_dt) {
  return dispatch<SplitLaunch, MODE>(c, in_dt, out_dt);
}

}  // namespace rowsm
