// Streaming conversion copy, y[i] = (Out) x[i]: the measurement aid of
// rowsm_stream_copy (include/rowsm.h).  It moves the bytes a row operation of
// the same dtype pair moves (each input byte read once, each output byte
// written once) in the access pattern that measured fastest on this HBM: one
// vector of at most 16 bytes per thread, each block one contiguous chunk that
// it reads, converts, writes and exits, non-temporal loads and stores.  The
// benchmark times it next to each row kernel as that workload's practical
// ceiling.
#include <hip/hip_runtime.h>

#include "rowsm.h"
#include "rowsm_device.hpp"

namespace rowsm {
namespace {

constexpr int kCopyBlock = 256;

// Block b of the (grid-stride) sequence covers elements [b*CH, b*CH + CH) of
// the n, CH = kCopyBlock * VW; the last chunk may be short, and its partial
// vector is copied element by element.
template <typename In, typename Out, int VW>
__global__ __launch_bounds__(kCopyBlock) void stream_copy_kernel(
    const typename In::storage* x, typename Out::storage* y, int64_t n,
    int64_t nblocks) {
  constexpr int64_t CH = (int64_t)kCopyBlock * VW;
  const int i0 = threadIdx.x * VW;
  // (each block's chunk plays the part of a row for the store policy)
  const bool wl = stores_whole_lines(y, CH * Out::bytes);  // sc1 stores
  for (int64_t b = blockIdx.x; b < nblocks; b += gridDim.x) {
    const int64_t base = b * CH;
    const int cnt = (int)(n - base < CH ? n - base : CH);
    const rsrc_t rx = make_rsrc(x + base, (uint64_t)cnt * In::bytes);
    const rsrc_t ry = make_rsrc(y + base, (uint64_t)cnt * Out::bytes);
    if (i0 + VW <= cnt) {
      InVec<In, VW> v;
      v.load(rx, (uint32_t)i0 * In::bytes, 0);
      float f[VW];
      v.to_float(f);
      store_out<Out, VW>(ry, (uint32_t)i0 * Out::bytes, f, wl);
    } else {
      for (int e = i0; e < cnt; ++e) {
        InVec<In, 1> v;
        v.load(rx, (uint32_t)e * In::bytes, 0);
        float f[1];
        v.to_float(f);
        store_out<Out, 1>(ry, (uint32_t)e * Out::bytes, f, wl);
      }
    }
  }
}

template <typename In, typename Out, int VW>
int launch_copy(const void* x, void* y, int64_t n, hipStream_t st) {
  constexpr int64_t CH = (int64_t)kCopyBlock * VW;
  const int64_t nblocks = (n + CH - 1) / CH;
  const int64_t grid = nblocks < 0x7fffffff ? nblocks : 0x7fffffff;
  (void)hipGetLastError();  // do not report an earlier, unrelated error
  stream_copy_kernel<In, Out, VW><<<dim3((unsigned)grid), dim3(kCopyBlock), 0, st>>>(
      static_cast<const typename In::storage*>(x), static_cast<typename Out::storage*>(y), n,
      nblocks);
  return hipGetLastError() == hipSuccess ? ROWSM_OK : ROWSM_EHIP;
}

// The widest vector of at most 16 bytes on either side that both pointers
// are aligned to, else single elements.
template <typename In, typename Out>
int copy_pair(const void* x, void* y, int64_t n, hipStream_t st) {
  constexpr int VW = 16 / (In::bytes > Out::bytes ? In::bytes : Out::bytes);
  const uintptr_t a = (uintptr_t)x % (VW * In::bytes) | (uintptr_t)y % (VW * Out::bytes);
  return a == 0 ? launch_copy<In, Out, VW>(x, y, n, st) : launch_copy<In, Out, 1>(x, y, n, st);
}

}  // namespace
}  // namespace rowsm

extern "C" int rowsm_stream_copy(const void* x, void* y, int64_t n, int in_dtype, int out_dtype,
                                 void* stream) {
  using namespace rowsm;
  auto ok = [](int dt) { return dt == ROWSM_F32 || dt == ROWSM_BF16; };
  if (!ok(in_dtype) || !ok(out_dtype)) return ROWSM_EDTYPE;
  if (n < 0 || n > ((int64_t)1 << 60)) return ROWSM_EINVAL;
  if (n == 0) return ROWSM_OK;
  if (!x || !y) return ROWSM_EINVAL;
  const int ib = in_dtype == ROWSM_F32 ? 4 : 2, ob = out_dtype == ROWSM_F32 ? 4 : 2;
  const uintptr_t xa = (uintptr_t)x, ya = (uintptr_t)y;
  if (xa % ib || ya % ob) return ROWSM_EINVAL;
  const bool overlap = xa < ya + (uint64_t)n * ob && ya < xa + (uint64_t)n * ib;
  if (overlap && !(xa == ya && in_dtype == out_dtype)) return ROWSM_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (in_dtype == ROWSM_F32)
    return out_dtype == ROWSM_F32 ? copy_pair<F32, F32>(x, y, n, st)
                                  : copy_pair<F32, BF16>(x, y, n, st);
  return out_dtype == ROWSM_F32 ? copy_pair<BF16, F32>(x, y, n, st)
                                : copy_pair<BF16, BF16>(x, y, n, st);
}
