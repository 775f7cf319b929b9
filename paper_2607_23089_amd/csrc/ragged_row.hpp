// Medium-row softmax for rows whose width is not a multiple of the vector
// width VW (16 bytes of the wider dtype): the row is still read and written
// in whole VW-element vectors, on the grid of vectors aligned to the start
// of the tensor, instead of one or two elements per load.
//
// Row r starts h = (r * cols) mod VW elements past a vector boundary, so it
// spans ceil((cols + h) / VW) vectors of that grid.  The descriptors of the
// row are based at that boundary.  Every vector the row touches is read as
// one load, its first and last too: their other elements belong to the
// neighbouring rows (inside the tensor) and are set to -inf once loaded, so
// that every load of a row is in flight at once.  Only a last vector that
// would reach past the end of the tensor (the final row's) is read element
// by element.  Stores write vectors wholly inside the row as one store and
// the row's own elements of the first and last vectors one at a time; rows
// of such widths never start every row on a 128-byte line, so the stores
// are non-temporal without the device-scope bit (kCpolStorePart).
//
// Layout and reductions are the medium kernel's (unpacked form): a row group
// of WPR waves, lane t owns vectors t, t + T, ... of the row's span, NV slots
// (the launcher sizes NV for the longest span, h = VW - 1); softmax and log
// output forms.  Rows past the end hold -inf, load and store nothing.
#pragma once

#include "medium_row.hpp"

namespace rowsm {

template <typename In, typename Out, int VW, int NV, int MODE>
__global__ __launch_bounds__(1024) void ragged_row_kernel(const typename In::storage* x,
                                                          typename Out::storage* y, int64_t rows,
                                                          int cols, int wpr) {
  static_assert(MODE == kPlain || MODE == kLog, "softmax and log forms only");
  static_assert((VW & (VW - 1)) == 0, "power-of-two vectors");
  constexpr bool LOG = MODE == kLog;
  __shared__ float red_m[16];
  __shared__ float red_s[16];

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = wave_id();
  const int rpb = (blockDim.x / kWave) / wpr;
  const int g = wave / wpr;
  const int T = wpr * kWave;
  const int t = (wave - g * wpr) * kWave + lane;
  const float ninf = -__builtin_inff();
  const int64_t total = rows * (int64_t)cols;        // elements of the tensor

  for (int64_t base = (int64_t)blockIdx.x * rpb; base < rows;
       base += (int64_t)gridDim.x * rpb) {
    const int64_t row = base + g;
    const bool row_ok = row < rows;
    const int64_t e0 = (row_ok ? row : 0) * cols;   // first element of the row
    const int h = (int)(e0 & (VW - 1));              // its place in its vector
    const int span = cols + h;                       // elements from the boundary on
    // The row's last vector: its index, owner (lane t1, slot s1) and the
    // number of the row's elements in it (1..VW).
    const int lv = (span - 1) / VW;
    const int s1 = lv / T, t1 = lv - s1 * T;
    const int rem = span - lv * VW;
    // Elements the load descriptor covers: the row's vectors, cut at the end
    // of the tensor (never shorter than span).
    const int64_t room = total - (e0 - h);
    const int lim = (int)((int64_t)(lv + 1) * VW < room ? (int64_t)(lv + 1) * VW : room);
    const rsrc_t rx = make_rsrc(x + (e0 - h), (uint64_t)lim * In::bytes);
    const rsrc_t ry = make_rsrc(y + (e0 - h), (uint64_t)span * Out::bytes);

    float f[NV][VW];
    {
      InVec<In, VW> v[NV];
#pragma unroll
      for (int s = 0; s < NV; ++s) {
        const int first = (s * T + t) * VW;          // the vector's first element
        const bool vec = row_ok && first < span && first + VW <= lim;
        v[s].load_or_neg_inf(vec, rx, (uint32_t)first * In::bytes, 0);
      }
#pragma unroll
      for (int s = 0; s < NV; ++s) v[s].to_float(f[s]);
    }
    // The neighbouring rows' elements of the first and last vectors to -inf;
    // a last vector reaching past the end of the tensor was not loaded and
    // is read element by element.
    if (row_ok && t == 0) {
#pragma unroll
      for (int k = 0; k < VW; ++k)
        if (k < h) f[0][k] = ninf;
    }
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      if (row_ok && s == s1 && t == t1) {
        if ((lv + 1) * VW <= lim) {
#pragma unroll
          for (int k = 0; k < VW; ++k)
            if (k >= rem) f[s][k] = ninf;
        } else {
          const int lo = lv == 0 ? h : 0;
#pragma unroll
          for (int k = 0; k < VW; ++k) {
            InVec<In, 1> u;
            u.load_or_neg_inf(k >= lo && k < rem, rx, (uint32_t)(lv * VW + k) * In::bytes, 0);
            f[s][k] = u.get(0);
          }
        }
      }
    }

    float mx = ninf;
#pragma unroll
    for (int s = 0; s < NV; ++s)
#pragma unroll
      for (int i = 0; i < VW; ++i) mx = fmax_nn(mx, f[s][i]);
    mx = block_row_reduce<MaxOp>(mx, wpr, wave, g, lane, red_m);
    const float nml = -mx * kLog2e;
    float sum = 0.0f;
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      if constexpr (LOG) exp_sum_keep(f[s], mx, &sum);
      else exp_accumulate<false>(f[s], nml, true, &sum);
    }
    sum = block_row_reduce<SumOp>(sum, wpr, wave, g, lane, red_s);
    const float inv = __builtin_amdgcn_rcpf(sum);  // v_rcp_f32, 1 ulp
    const float lns = LOG ? ln_fast(sum) : 0.0f;
#pragma unroll
    for (int s = 0; s < NV; ++s) {
#pragma unroll
      for (int i = 0; i < VW; ++i) f[s][i] = LOG ? (f[s][i] - mx) - lns : f[s][i] * inv;
      const int first = (s * T + t) * VW;
      if (row_ok && first >= h && first + VW <= span)
        store_out<Out, VW>(ry, (uint32_t)first * Out::bytes, f[s], false);
    }
    // The row's own elements of a partial first vector (lane 0, slot 0;
    // when the row has more than one vector) and of a partial last vector.
    if (row_ok && t == 0 && h > 0 && lv > 0) {
#pragma unroll
      for (int k = 0; k < VW; ++k)
        if (k >= h) store_out<Out, 1>(ry, (uint32_t)k * Out::bytes, {f[0][k]}, false);
    }
    if (row_ok && (rem < VW || (lv == 0 && h > 0))) {
      const int lo = lv == 0 ? h : 0;
#pragma unroll
      for (int s = 0; s < NV; ++s) {
        if (s == s1 && t == t1) {
#pragma unroll
          for (int k = 0; k < VW; ++k)
            if (k >= lo && k < rem)
              store_out<Out, 1>(ry, (uint32_t)(lv * VW + k) * Out::bytes, {f[s][k]}, false);
        }
      }
    }
  }
}

}  // namespace rowsm
