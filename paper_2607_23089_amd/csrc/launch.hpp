// Launch plans and the per-family launchers.  Each family's kernels are
// instantiated in translation units of their own, one per output form
// (launch_<family>_<form>.hip), so the library builds in parallel; rowsm.hip
// holds the launcher logic and the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rowsm.h"
#include "rowsm_device.hpp"

namespace rowsm {

constexpr int kMaxDevices = 64;
// Blocks one launch of an exchanging form may use in an exchange workspace
// (32 bytes each); larger grids loop their row groups over the rows.
constexpr int kSplitMaxBlocks = 1 << 20;
// Blocks per row of the two-pass LARGE form at most (and at most the compute
// units: all of a row's blocks must be resident at once, and a 1024-thread
// block of it may take a whole compute unit's registers).  Wave 0 of a
// block polls up to 4 peers per lane in its exchange.
constexpr int kStreamMaxSplit = 256;

// The launch the row launcher chose (fields unused by a family stay default).
struct Plan {
  int variant = 0;
  int vw = 1;       // elements per vector
  int nvec = 0;     // vectors per row
  // SMALL
  int lpr = 1, rpl = 4;
  // MEDIUM
  int wpr = 1, vpl = 1, nv = 1;
  bool packed = false;
  // LARGE
  int u = 4;
  int split = 0;    // blocks per row of the single-read form; 0 = two-pass form
  int stream = 1;   // two-pass form: blocks per row (1: one block per row)
  bool prefetch = false;  // single-read form: load the next row during the exchange
  // MEDIUM: a row width that is not a multiple of vw, read in whole vectors
  // aligned to the tensor with element-wise row edges (ragged_row.hpp)
  bool ragged = false;
  // SMALL: short rows of such widths as one flat stream of whole vectors,
  // regrouped into rows through LDS (flat_row.hpp); lpr lanes per row and nv
  // elements per lane in the row phase
  bool flat = false;
  // launch
  int block = 256;
  int64_t grid = 1;  // split form: 0 = one group per row, < 0 = minus the blocks-per-CU cap
};

// One launch request: the plan plus its operands.  mode is the output form
// (kPlain, kFused or kLog); fz holds the scale and mask of kFused and is the
// identity (scale 1, no mask) otherwise.
struct Call {
  Plan p;
  const void* x;
  void* y;
  int64_t rows;
  int cols;
  hipStream_t st;
  int cus;
  int mode = kPlain;
  Fused fz{1.0f, 0, 0};
  const void* dy = nullptr;  // softmax backward: x holds y, dy the gradient, y receives dx
  // Exchanging launches take their workspace from the static `scratch` array
  // (rowsm_forward_noalloc), whatever the device's exchange ring.
  bool noalloc = false;
};

// Calls L<In, Out, VW, MODE>::run(c) for the call's dtype pair and vector
// width (16-byte, 8-byte or single-element input vectors).  Widths whose
// output vector would exceed 16 bytes are never planned (the width rule of
// choose_vw) and are not compiled.  Returns a rowsm_status: ROWSM_EINVAL when
// nothing matches (nothing enqueued).
template <template <typename, typename, int, int> class L, int MODE>
int dispatch(const Call& c, int in_dt, int out_dt) {
  auto io = [&](auto in_tag, auto out_tag) -> int {
    using In = decltype(in_tag);
    using Out = decltype(out_tag);
    constexpr int V16 = 16 / In::bytes, V8 = 8 / In::bytes;
    if (c.p.vw == 1) return L<In, Out, 1, MODE>::run(c);
    if (c.p.vw == V8) {
      if constexpr (V8 * Out::bytes <= 16) return L<In, Out, V8, MODE>::run(c);
    }
    if (c.p.vw == V16) {
      if constexpr (V16 * Out::bytes <= 16) return L<In, Out, V16, MODE>::run(c);
    }
    return ROWSM_EINVAL;
  };
  if (in_dt == ROWSM_F32 && out_dt == ROWSM_F32) return io(F32{}, F32{});
  if (in_dt == ROWSM_F32) return io(F32{}, BF16{});
  if (out_dt == ROWSM_F32) return io(BF16{}, F32{});
  return io(BF16{}, BF16{});
}

// Per-family launchers, defined in launch_<family>.hpp and instantiated for
// each output form in launch_<family>_<form>.hip.
template <int MODE> int launch_small(const Call& c, int in_dt, int out_dt);
template <int MODE> int launch_medium(const Call& c, int in_dt, int out_dt);
template <int MODE> int launch_large(const Call& c, int in_dt, int out_dt);
template <int MODE> int launch_split(const Call& c, int in_dt, int out_dt);
template <int MODE> int launch_ragged(const Call& c, int in_dt, int out_dt);
template <int MODE> int launch_flat(const Call& c, int in_dt, int out_dt);

// Softmax-backward launchers (launch_bwd_<family>.hip).
int launch_bwd_small(const Call& c, int in_dt, int out_dt);
int launch_bwd_medium(const Call& c, int in_dt, int out_dt);
int launch_bwd_split(const Call& c, int in_dt, int out_dt);
int launch_bwd_large(const Call& c, int in_dt, int out_dt);

// MoE group-score launchers (launch_moe_<dtype>.hip).
int launch_moe_f32(const Call& c, int out_dt);
int launch_moe_bf16(const Call& c, int out_dt);

// Exchange workspace diagnostics and test settings (launch_split_common.hip).
int64_t split_wait_failures_current_device();
int64_t split_set_wait_limit(int64_t polls);

}  // namespace rowsm
