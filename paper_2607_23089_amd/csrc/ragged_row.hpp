// Medium-row softmax for rows whose width is not a multiple of the vector
// width VW (16 bytes of the wider dtype): the row is still read and written
// in whole VW-element vectors, on the grid of vectors aligned to the start
// of the tensor, instead of one or two elements per load.
//
// Row r starts h = (r * cols) mod VW elements past a vector boundary, so it
// spans ceil((cols + h) / VW) vectors of that grid.  The descriptors of the
// row are based at that boundary and end at the row's last element; vectors
// wholly inside the row move as one load and one store, and the first and
// last vectors, which share elements with the neighbouring rows, move one
// element at a time (only the row's own elements are read or written).
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

  for (int64_t base = (int64_t)blockIdx.x * rpb; base < rows;
       base += (int64_t)gridDim.x * rpb) {
    const int64_t row = base + g;
    const bool row_ok = row < rows;
    const int64_t e0 = (row_ok ? row : 0) * cols;   // first element of the row
    const int h = (int)(e0 & (VW - 1));              // its place in its vector
    const int span = cols + h;                       // elements from the boundary on
    const rsrc_t rx = make_rsrc(x + (e0 - h), (uint64_t)span * In::bytes);
    const rsrc_t ry = make_rsrc(y + (e0 - h), (uint64_t)span * Out::bytes);

    float f[NV][VW];
    {
      InVec<In, VW> v[NV];
#pragma unroll
      for (int s = 0; s < NV; ++s) {
        const int first = (s * T + t) * VW;          // the vector's first element
        const bool whole = row_ok && first >= h && first + VW <= span;
        v[s].load_or_neg_inf(whole, rx, (uint32_t)first * In::bytes, 0);
      }
#pragma unroll
      for (int s = 0; s < NV; ++s) v[s].to_float(f[s]);
      // The row's first and last vectors, element by element.
#pragma unroll
      for (int s = 0; s < NV; ++s) {
        const int first = (s * T + t) * VW;
        const bool edge = row_ok && first < span && !(first >= h && first + VW <= span);
        if (edge) {
#pragma unroll
          for (int k = 0; k < VW; ++k) {
            const int e = first + k;
            InVec<In, 1> u;
            u.load_or_neg_inf(e >= h && e < span, rx, (uint32_t)e * In::bytes, 0);
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
      if (row_ok && first >= h && first + VW <= span) {
        store_out<Out, VW>(ry, (uint32_t)first * Out::bytes, f[s]);
      } else if (row_ok && first < span) {
#pragma unroll
        for (int k = 0; k < VW; ++k) {
          const int e = first + k;
          if (e >= h && e < span) {
            const float o[1] = {f[s][k]};
            store_out<Out, 1>(ry, (uint32_t)e * Out::bytes, o);
          }
        }
      }
    }
  }
}

}  // namespace rowsm
