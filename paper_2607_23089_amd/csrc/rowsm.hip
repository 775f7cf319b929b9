// Host side of the row-softmax library: argument validation, the template
// dispatch over the kernel families and the C ABI declared in
// include/rowsm.h.  The launcher that picks a family and its
// launch shape for each call is in plan.hip.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstring>

#include "plan.hpp"

namespace rowsm {
namespace {

static_assert(ROWSM_OP_SOFTMAX == kPlain && ROWSM_OP_SCALED_CAUSAL == kFused &&
                  ROWSM_OP_LOG_SOFTMAX == kLog && ROWSM_OP_SOFTMAX_BACKWARD == kBackward,
              "rowsm_op values are the launch modes");
static_assert(ROWSM_OP_MOE_GROUP_TOP2 == kMoe, "rowsm_op values are the launch modes");

// ---- family dispatch ------------------------------------------------------------

template <int MODE>
int launch_mode(const Call& c, int in_dt, int out_dt) {
  switch (c.p.variant) {
    case ROWSM_SMALL:
      if constexpr (MODE == kPlain || MODE == kLog) {
        if (c.p.flat) return launch_flat<MODE>(c, in_dt, out_dt);
      }
      return c.p.flat ? ROWSM_EINVAL : launch_small<MODE>(c, in_dt, out_dt);
    case ROWSM_MEDIUM:
      if constexpr (MODE == kPlain || MODE == kLog) {
        if (c.p.ragged) return launch_ragged<MODE>(c, in_dt, out_dt);
      }
      return c.p.ragged ? ROWSM_EINVAL : launch_medium<MODE>(c, in_dt, out_dt);
    case ROWSM_LARGE:
      return c.p.split > 0 ? launch_split<MODE>(c, in_dt, out_dt)
                           : launch_large<MODE>(c, in_dt, out_dt);
    default: return ROWSM_EINVAL;
  }
}

int launch_backward(const Call& c, int in_dt, int out_dt) {
  switch (c.p.variant) {
    case ROWSM_SMALL:
      return c.p.flat ? launch_flat<kBackward>(c, in_dt, out_dt)
                      : launch_bwd_small(c, in_dt, out_dt);
    case ROWSM_MEDIUM: return launch_bwd_medium(c, in_dt, out_dt);
    case ROWSM_LARGE:
      return c.p.split > 0 ? launch_bwd_split(c, in_dt, out_dt)
                           : launch_bwd_large(c, in_dt, out_dt);
    default: return ROWSM_EINVAL;
  }
}

int launch(const Call& c, int in_dt, int out_dt) {
  switch (c.mode) {
    case kPlain: return launch_mode<kPlain>(c, in_dt, out_dt);
    case kFused: return launch_mode<kFused>(c, in_dt, out_dt);
    case kLog: return launch_mode<kLog>(c, in_dt, out_dt);
    case kBackward: return launch_backward(c, in_dt, out_dt);
    default: return ROWSM_EINVAL;
  }
}

// ---- validation -------------------------------------------------------------

// Host-only argument checks shared by every entry point.  *noop is set when
// the call is valid and has nothing to do.
int validate(const void* x, const void* y, int64_t rows, int64_t cols, int in_dt,
             int out_dt, bool check_ptrs, bool* noop) {
  *noop = false;
  if (!dtype_ok(in_dt) || !dtype_ok(out_dt)) return ROWSM_EDTYPE;
  if (rows < 0 || cols < 0) return ROWSM_EINVAL;
  if (rows == 0 || cols == 0) {
    *noop = true;
    return ROWSM_OK;
  }
  if (cols >= ((int64_t)1 << 30)) return ROWSM_EINVAL;  // row bytes fit 32-bit offsets
  if (rows > ((int64_t)1 << 62) / cols) return ROWSM_EINVAL;
  if (!check_ptrs) return ROWSM_OK;
  if (!x || !y) return ROWSM_EINVAL;
  const uintptr_t xa = (uintptr_t)x, ya = (uintptr_t)y;
  const uint64_t n = (uint64_t)rows * (uint64_t)cols;
  const uint64_t xb = n * (uint64_t)dtype_bytes(in_dt), yb = n * (uint64_t)dtype_bytes(out_dt);
  const bool overlap = xa < ya + yb && ya < xa + xb;
  if (overlap && !(xa == ya && in_dt == out_dt)) return ROWSM_EINVAL;
  return ROWSM_OK;
}

// Backward operands: y and dy (in_dt, read only, may overlap each other) and
// dx (out_dt), which may be y or dy itself when the dtypes match but must not
// overlap either in any other way.
int validate_backward(const void* yp, const void* dyp, const void* dxp, int64_t rows,
                      int64_t cols, int in_dt, int out_dt, bool* noop) {
  int st = validate(yp, dxp, rows, cols, in_dt, out_dt, true, noop);
  if (st != ROWSM_OK || *noop) return st;
  return validate(dyp, dxp, rows, cols, in_dt, out_dt, true, noop);
}

int backward_impl(const void* yp, const void* dyp, void* dxp, int64_t rows, int64_t cols,
                  int in_dt, int out_dt, void* stream, const rowsm_config* cfg) {
  bool noop = false;
  int st = validate_backward(yp, dyp, dxp, rows, cols, in_dt, out_dt, &noop);
  if (st != ROWSM_OK || noop) return st;
  Call c;
  c.cus = cu_count();
  const uintptr_t ia = (uintptr_t)yp | (uintptr_t)dyp;
  const bool inplace = dxp == yp || dxp == dyp;
  st = plan_backward(rows, cols, in_dt, out_dt, ia, (uintptr_t)dxp, cfg, c.cus, inplace, &c.p);
  if (st != ROWSM_OK) return st;
  c.x = yp;
  c.dy = dyp;
  c.y = dxp;
  c.rows = rows;
  c.cols = (int)cols;
  c.st = static_cast<hipStream_t>(stream);
  c.mode = kBackward;
  (void)hipGetLastError();  // do not report an earlier, unrelated error
  return launch(c, in_dt, out_dt);
}

// MoE group-score arguments.  The scores (tokens x experts, in_dt) are read
// only; the group scores (tokens x experts / group, out_dt) must not overlap
// them and must be aligned to their element size.
int validate_moe(const void* sp, const void* op, int64_t tokens, int64_t experts, int64_t group,
                 int in_dt, int out_dt, bool check_ptrs, bool* noop) {
  *noop = false;
  if (!dtype_ok(in_dt) || !dtype_ok(out_dt)) return ROWSM_EDTYPE;
  if (tokens < 0 || experts < 0 || !moe_group_ok(group) || experts % group) return ROWSM_EINVAL;
  if (tokens == 0 || experts == 0) {
    *noop = true;
    return ROWSM_OK;
  }
  if (tokens > ((int64_t)1 << 62) / experts) return ROWSM_EINVAL;
  if (!check_ptrs) return ROWSM_OK;
  if (!sp || !op) return ROWSM_EINVAL;
  const uintptr_t sa = (uintptr_t)sp, oa = (uintptr_t)op;
  if (oa % (uintptr_t)dtype_bytes(out_dt) || sa % (uintptr_t)dtype_bytes(in_dt))
    return ROWSM_EINVAL;
  const uint64_t n = (uint64_t)tokens * (uint64_t)experts;
  const uint64_t sb = n * (uint64_t)dtype_bytes(in_dt);
  const uint64_t ob = n / (uint64_t)group * (uint64_t)dtype_bytes(out_dt);
  if (sa < oa + ob && oa < sa + sb) return ROWSM_EINVAL;
  return ROWSM_OK;
}

int moe_impl(const void* sp, void* op, int64_t tokens, int64_t experts, int64_t group,
             int in_dt, int out_dt, void* stream, const rowsm_config* cfg) {
  bool noop = false;
  int st = validate_moe(sp, op, tokens, experts, group, in_dt, out_dt, true, &noop);
  if (st != ROWSM_OK || noop) return st;
  Call c;
  c.cus = cu_count();
  const int64_t ngroups = tokens * (experts / group);
  st = plan_moe(ngroups, group, in_dt, (uintptr_t)sp, cfg, c.cus, &c.p);
  if (st != ROWSM_OK) return st;
  c.x = sp;
  c.y = op;
  c.rows = ngroups;
  c.cols = (int)group;
  c.st = static_cast<hipStream_t>(stream);
  c.mode = kMoe;
  (void)hipGetLastError();  // do not report an earlier, unrelated error
  return in_dt == ROWSM_F32 ? launch_moe_f32(c, out_dt) : launch_moe_bf16(c, out_dt);
}

int forward_impl(const void* x, void* y, int64_t rows, int64_t cols, int in_dt, int out_dt,
                 void* stream, const rowsm_config* cfg, int mode, Fused fz = {1.0f, 0, 0},
                 bool noalloc = false) {
  bool noop = false;
  int st = validate(x, y, rows, cols, in_dt, out_dt, true, &noop);
  if (st != ROWSM_OK || noop) return st;
  Call c;
  c.cus = cu_count();
  st = plan_for(rows, cols, in_dt, out_dt, (uintptr_t)x, (uintptr_t)y, cfg, c.cus, mode, x == y,
                &c.p);
  if (st != ROWSM_OK) return st;
  c.x = x;
  c.y = y;
  c.rows = rows;
  c.cols = (int)cols;
  c.st = static_cast<hipStream_t>(stream);
  c.mode = mode;
  c.fz = fz;
  c.noalloc = noalloc;
  (void)hipGetLastError();  // do not report an earlier, unrelated error
  return launch(c, in_dt, out_dt);
}

const char* variant_name(int v) {
  switch (v) {
    case ROWSM_SMALL: return "small";
    case ROWSM_MEDIUM: return "medium";
    case ROWSM_LARGE: return "large";
    default: return "?";
  }
}

}  // namespace
}  // namespace rowsm

using namespace rowsm;

extern "C" int rowsm_forward(const void* x, void* y, int64_t rows, int64_t cols, int in_dtype,
                             int out_dtype, void* stream) {
  return forward_impl(x, y, rows, cols, in_dtype, out_dtype, stream, nullptr, kPlain);
}

extern "C" int rowsm_forward_noalloc(const void* x, void* y, int64_t rows, int64_t cols,
                                     int in_dtype, int out_dtype, void* stream) {
  return forward_impl(x, y, rows, cols, in_dtype, out_dtype, stream, nullptr, kPlain,
                      Fused{1.0f, 0, 0}, true);
}

extern "C" int rowsm_forward_variant(const void* x, void* y, int64_t rows, int64_t cols,
                                     int in_dtype, int out_dtype, void* stream, int variant) {
  if (variant < ROWSM_AUTO || variant > ROWSM_LARGE) {
    bool noop = false;
    const int st = validate(x, y, rows, cols, in_dtype, out_dtype, true, &noop);
    return st != ROWSM_OK ? st : ROWSM_EINVAL;
  }
  rowsm_config cfg;
  std::memset(&cfg, 0, sizeof(cfg));
  cfg.variant = variant;
  cfg.packed = -1;
  return forward_impl(x, y, rows, cols, in_dtype, out_dtype, stream, &cfg, kPlain);
}

extern "C" int rowsm_forward_config(const void* x, void* y, int64_t rows, int64_t cols,
                                    int in_dtype, int out_dtype, void* stream,
                                    const rowsm_config* cfg) {
  return forward_impl(x, y, rows, cols, in_dtype, out_dtype, stream, cfg, kPlain);
}

extern "C" int rowsm_forward_scaled_causal(const void* x, void* y, int64_t rows, int64_t cols,
                                           int in_dtype, int out_dtype, float scale,
                                           int64_t causal_period, int64_t causal_offset,
                                           void* stream, const rowsm_config* cfg) {
  if (causal_period < 0) {
    bool noop = false;
    const int st = validate(x, y, rows, cols, in_dtype, out_dtype, true, &noop);
    return st != ROWSM_OK ? st : ROWSM_EINVAL;
  }
  const Fused fz{scale, causal_period, causal_offset};
  return forward_impl(x, y, rows, cols, in_dtype, out_dtype, stream, cfg, kFused, fz);
}

extern "C" int rowsm_log_softmax(const void* x, void* y, int64_t rows, int64_t cols,
                                 int in_dtype, int out_dtype, void* stream,
                                 const rowsm_config* cfg) {
  return forward_impl(x, y, rows, cols, in_dtype, out_dtype, stream, cfg, kLog);
}

extern "C" int rowsm_softmax_backward(const void* y, const void* dy, void* dx, int64_t rows,
                                      int64_t cols, int in_dtype, int out_dtype, void* stream,
                                      const rowsm_config* cfg) {
  return backward_impl(y, dy, dx, rows, cols, in_dtype, out_dtype, stream, cfg);
}

extern "C" int rowsm_moe_group_top2(const void* scores, void* group_scores, int64_t tokens,
                                    int64_t experts, int64_t group_size, int in_dtype,
                                    int out_dtype, void* stream, const rowsm_config* cfg) {
  return moe_impl(scores, group_scores, tokens, experts, group_size, in_dtype, out_dtype,
                  stream, cfg);
}

extern "C" int rowsm_select(int64_t rows, int64_t cols, int in_dtype, int out_dtype) {
  bool noop = false;
  const int st = validate(nullptr, nullptr, rows, cols, in_dtype, out_dtype, false, &noop);
  if (st != ROWSM_OK) return st;
  if (noop) return ROWSM_SMALL;  // nothing is launched; report the smallest family
  Plan p;
  const int r =
      plan_for(rows, cols, in_dtype, out_dtype, 256, 256, nullptr, 256, kPlain, false, &p);
  return r == ROWSM_OK ? p.variant : r;
}

namespace rowsm {
namespace {

// Description of the launch an operation would make (mode: the rowsm_op
// value, which equals the output form and kBackward).
int describe_impl(int mode, int64_t rows, int64_t cols, int in_dt, int out_dt,
                  const rowsm_config* cfg, char* buf, int64_t len) {
  bool noop = false;
  int st = mode == kMoe
               ? validate_moe(nullptr, nullptr, rows, cols, cols, in_dt, out_dt, false, &noop)
               : validate(nullptr, nullptr, rows, cols, in_dt, out_dt, false, &noop);
  if (st == ROWSM_OK && (mode < kPlain || mode > kMoe)) st = ROWSM_EINVAL;
  Plan p;
  if (st == ROWSM_OK && !noop) {
    if (mode == kMoe)
      st = plan_moe(rows, cols, in_dt, 256, cfg, 256, &p);
    else if (mode == kBackward)
      st = plan_backward(rows, cols, in_dt, out_dt, 256, 256, cfg, 256, false, &p);
    else
      st = plan_for(rows, cols, in_dt, out_dt, 256, 256, cfg, 256, mode, false, &p);
  }
  if (buf && len > 0) {
    if (st != ROWSM_OK) {
      std::snprintf(buf, (size_t)len, "error %d", st);
    } else if (noop) {
      std::snprintf(buf, (size_t)len, "empty: no launch");
    } else {
      // The split form's grid: one group of S blocks per row up to the room
      // of the workspace (split_slots()), or a residency sized at launch.
      int64_t grid = p.grid;
      const char* how = "grid assumes 256 CUs";
      const int S = p.split > 0 ? p.split : (p.variant == ROWSM_LARGE ? p.stream : 1);
      if (S > 1 || p.split > 0) {
        const int64_t groups = kSplitMaxBlocks / S;
        grid = p.grid < 0 ? 0 : (rows < groups ? rows : groups) * S;
        how = p.grid < 0 ? "one residency sized from occupancy at launch"
                         : "one group of blocks per row";
      }
      std::snprintf(buf, (size_t)len,
                    "%s vw=%d nvec=%d lpr=%d rpl=%d wpr=%d vpl=%d nv=%d packed=%d u=%d "
                    "split=%d stream=%d prefetch=%d ragged=%d flat=%d block=%d grid=%lld (%s)",
                    variant_name(p.variant), p.vw, p.nvec, p.lpr, p.rpl, p.wpr, p.vpl, p.nv,
                    (int)p.packed, p.u, p.split, p.variant == ROWSM_LARGE && !p.split ? p.stream : 0,
                    (int)p.prefetch, (int)p.ragged, (int)p.flat, p.block, (long long)grid, how);
    }
  }
  return st;
}

}  // namespace
}  // namespace rowsm

extern "C" int rowsm_describe(int64_t rows, int64_t cols, int in_dtype, int out_dtype,
                              int variant, char* buf, int64_t len) {
  if (variant < ROWSM_AUTO || variant > ROWSM_LARGE) {
    if (buf && len > 0) std::snprintf(buf, (size_t)len, "error %d", ROWSM_EINVAL);
    bool noop = false;
    const int st = validate(nullptr, nullptr, rows, cols, in_dtype, out_dtype, false, &noop);
    return st != ROWSM_OK ? st : ROWSM_EINVAL;
  }
  rowsm_config cfg;
  std::memset(&cfg, 0, sizeof(cfg));
  cfg.variant = variant;
  cfg.packed = -1;
  return describe_impl(kPlain, rows, cols, in_dtype, out_dtype, &cfg, buf, len);
}

extern "C" int rowsm_describe_op(int op, int64_t rows, int64_t cols, int in_dtype,
                                 int out_dtype, const rowsm_config* cfg, char* buf,
                                 int64_t len) {
  return describe_impl(op, rows, cols, in_dtype, out_dtype, cfg, buf, len);
}

extern "C" int64_t rowsm_split_wait_failures(void) {
  return split_wait_failures_current_device();
}

extern "C" int64_t rowsm_set_split_wait_limit(int64_t polls) {
  return split_set_wait_limit(polls);
}

extern "C" const char* rowsm_status_string(int status) {
  switch (status) {
    case ROWSM_OK: return "ok";
    case ROWSM_EINVAL: return "invalid argument";
    case ROWSM_EDTYPE: return "unsupported dtype";
    case ROWSM_EHIP: return "HIP launch error";
    default: return "unknown status";
  }
}
