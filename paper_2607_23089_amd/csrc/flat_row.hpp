// Short rows of a width that is not a multiple of the 16-byte vector width
// VW: the rows are read and written as one flat stream of whole 16-byte
// vectors on the grid aligned to the start of the tensor, and regrouped into
// rows through LDS.
//
// With narrow vectors such rows move one or two elements per lane and load
// instruction (a 37-element fp32 row, one wave: 148 bytes per instruction);
// here every load and store instruction of a wave moves 64 whole vectors.
//
// A block is one wave.  A tile is G consecutive rows, G the most whose
// elements, from the vector boundary at or before the first, fit S = 4
// vectors per lane (or S = 2: half the registers and LDS).  Per tile:
//   1. each lane loads its S vectors (lane-major, so every instruction reads
//      64 consecutive vectors) and writes them to LDS as fp32; the first and
//      last vectors also hold elements of the neighbouring tiles (inside the
//      tensor), which are loaded and never used; a last vector that would
//      reach past the end of the tensor (the final tile's) is read element
//      by element;
//   2. the rows are taken RPP = 64 / LPR at a time, LPR lanes per row, E
//      elements per lane (element c of a row on lane c mod LPR): max and sum
//      by DPP over the LPR lanes, the output written back over the row in
//      LDS;
//   3. each lane stores its vectors that hold only the tile's elements as
//      one store, and the tile's own elements of its first and last vectors
//      one at a time.
// The arithmetic per row is the small-row kernel's (fp32, exp2 of a fused
// multiply-add, v_rcp_f32 or the log form).  Stores are non-temporal
// without the device-scope bit: rows of such widths never keep every store
// on whole 128-byte lines.
#pragma once

#include "rowsm_device.hpp"

namespace rowsm {

template <typename In, typename Out, int VW, int LPR, int E, int MODE, int S>
__global__ __launch_bounds__(64) void flat_row_kernel(const typename In::storage* x,
                                                      typename Out::storage* y, int64_t rows,
                                                      int cols, int G) {
  static_assert(MODE == kPlain || MODE == kLog, "softmax and log forms only");
  static_assert(LPR >= 1 && LPR <= kWave && (LPR & (LPR - 1)) == 0, "power-of-two row groups");
  static_assert(S == 2 || S == kFlatSlots, "two or four vectors per lane");
  constexpr bool LOG = MODE == kLog;
  constexpr int RPP = kWave / LPR;  // rows per pass
  __shared__ float buf[S * kWave * VW];

  const int lane = threadIdx.x & (kWave - 1);
  const int sub = lane % LPR, grp = lane / LPR;
  const float ninf = -__builtin_inff();
  const int64_t total = rows * (int64_t)cols;
  const int64_t ntiles = (rows + G - 1) / G;

  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t r0 = tile * G;
    const int nr = rows - r0 < G ? (int)(rows - r0) : G;
    const int64_t e0 = r0 * cols;                  // the tile's first element
    const int h = (int)(e0 & (VW - 1));            // its place in its vector
    const int span = nr * cols + h;                // elements from the boundary on
    const int lv = (span - 1) / VW;                // the tile's last vector
    const int64_t room = total - (e0 - h);
    const int lim = (int)((int64_t)(lv + 1) * VW < room ? (int64_t)(lv + 1) * VW : room);
    const rsrc_t rx = make_rsrc(x + (e0 - h), (uint64_t)lim * In::bytes);
    const rsrc_t ry = make_rsrc(y + (e0 - h), (uint64_t)span * Out::bytes);

    {
      InVec<In, VW> v[S];
#pragma unroll
      for (int s = 0; s < S; ++s) {
        const int first = (s * kWave + lane) * VW;
        v[s].load_or_neg_inf(first < span && first + VW <= lim, rx, (uint32_t)first * In::bytes, 0);
      }
#pragma unroll
      for (int s = 0; s < S; ++s) {
        float f[VW];
        v[s].to_float(f);
#pragma unroll
        for (int k = 0; k < VW; ++k) buf[(s * kWave + lane) * VW + k] = f[k];
      }
    }
    if (lim < (lv + 1) * VW) {  // the final tile's last vector, element by element
#pragma unroll
      for (int s = 0; s < S; ++s) {
        if (s * kWave + lane == lv) {
#pragma unroll
          for (int k = 0; k < VW; ++k) {
            const int e = lv * VW + k;
            InVec<In, 1> u;
            u.load_or_neg_inf(e >= h && e < span, rx, (uint32_t)e * In::bytes, 0);
            buf[e] = u.get(0);
          }
        }
      }
    }
    __syncthreads();

    for (int p = 0; p * RPP < nr; ++p) {
      const int g = p * RPP + grp;
      const bool rok = g < nr;
      const int base = h + g * cols;
      float f[E];
#pragma unroll
      for (int i = 0; i < E; ++i) {
        const int c = i * LPR + sub;
        f[i] = rok && c < cols ? buf[base + c] : ninf;
      }
      float m = f[0];
#pragma unroll
      for (int i = 1; i < E; ++i) m = fmax_nn(m, f[i]);
      m = group_reduce<LPR, MaxOp>(m);
      float t = 0.0f;
      if constexpr (LOG) {
        exp_sum_keep(f, m, &t);
      } else {
        const float nml = -m * kLog2e;
#pragma unroll
        for (int i = 0; i < E; ++i) {
          f[i] = exp2_fast(__builtin_fmaf(f[i], kLog2e, nml));
          t += f[i];
        }
      }
      t = group_reduce<LPR, SumOp>(t);
      if constexpr (LOG) {
        const float lns = ln_fast(t);
#pragma unroll
        for (int i = 0; i < E; ++i) f[i] = (f[i] - m) - lns;
      } else {
        const float inv = __builtin_amdgcn_rcpf(t);  // v_rcp_f32, 1 ulp
#pragma unroll
        for (int i = 0; i < E; ++i) f[i] *= inv;
      }
#pragma unroll
      for (int i = 0; i < E; ++i) {
        const int c = i * LPR + sub;
        if (rok && c < cols) buf[base + c] = f[i];
      }
    }
    __syncthreads();

#pragma unroll
    for (int s = 0; s < S; ++s) {
      const int first = (s * kWave + lane) * VW;
      if (first >= h && first + VW <= span) {
        float o[VW];
#pragma unroll
        for (int k = 0; k < VW; ++k) o[k] = buf[first + k];
        store_out<Out, VW>(ry, (uint32_t)first * Out::bytes, o, false);
      } else if (first < span && first + VW > h) {
#pragma unroll
        for (int k = 0; k < VW; ++k) {
          const int e = first + k;
          if (e >= h && e < span) store_out<Out, 1>(ry, (uint32_t)e * Out::bytes, {buf[e]}, false);
        }
      }
    }
    __syncthreads();  // the next tile's loads overwrite buf
  }
}

// Softmax backward of such rows, dx = y (dy - sum(y dy)): the same tiles of
// S vectors per lane (S = 2 keeps the bf16 instantiation at 8 KiB of LDS per
// wave), y and dy each through its own LDS buffer, one dot product per row
// (fp32 fused multiply-adds, then DPP over the LPR lanes), dx written back
// over y.
template <typename In, typename Out, int VW, int LPR, int E, int S>
__global__ __launch_bounds__(64) void bwd_flat_kernel(const typename In::storage* y,
                                                      const typename In::storage* dy,
                                                      typename Out::storage* dx, int64_t rows,
                                                      int cols, int G) {
  static_assert(LPR >= 1 && LPR <= kWave && (LPR & (LPR - 1)) == 0, "power-of-two row groups");
  static_assert(S == 2 || S == kFlatSlots, "two or four vectors per lane");
  constexpr int RPP = kWave / LPR;
  __shared__ float by[S * kWave * VW];
  __shared__ float bd[S * kWave * VW];

  const int lane = threadIdx.x & (kWave - 1);
  const int sub = lane % LPR, grp = lane / LPR;
  const int64_t total = rows * (int64_t)cols;
  const int64_t ntiles = (rows + G - 1) / G;

  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t r0 = tile * G;
    const int nr = rows - r0 < G ? (int)(rows - r0) : G;
    const int64_t e0 = r0 * cols;
    const int h = (int)(e0 & (VW - 1));
    const int span = nr * cols + h;
    const int lv = (span - 1) / VW;
    const int64_t room = total - (e0 - h);
    const int lim = (int)((int64_t)(lv + 1) * VW < room ? (int64_t)(lv + 1) * VW : room);
    const rsrc_t ry = make_rsrc(y + (e0 - h), (uint64_t)lim * In::bytes);
    const rsrc_t rdy = make_rsrc(dy + (e0 - h), (uint64_t)lim * In::bytes);
    const rsrc_t rdx = make_rsrc(dx + (e0 - h), (uint64_t)span * Out::bytes);

    {
      InVec<In, VW> a[S], b[S];
#pragma unroll
      for (int s = 0; s < S; ++s) {
        const int first = (s * kWave + lane) * VW;
        const bool ok = first < span && first + VW <= lim;
        a[s].load_or_neg_inf(ok, ry, (uint32_t)first * In::bytes, 0);
        b[s].load_or_neg_inf(ok, rdy, (uint32_t)first * In::bytes, 0);
      }
#pragma unroll
      for (int s = 0; s < S; ++s) {
        float fa[VW], fb[VW];
        a[s].to_float(fa);
        b[s].to_float(fb);
#pragma unroll
        for (int k = 0; k < VW; ++k) {
          by[(s * kWave + lane) * VW + k] = fa[k];
          bd[(s * kWave + lane) * VW + k] = fb[k];
        }
      }
    }
    if (lim < (lv + 1) * VW) {  // the final tile's last vector, element by element
#pragma unroll
      for (int s = 0; s < S; ++s) {
        if (s * kWave + lane == lv) {
#pragma unroll
          for (int k = 0; k < VW; ++k) {
            const int e = lv * VW + k;
            const bool ok = e >= h && e < span;
            InVec<In, 1> u, v;
            u.load_or_neg_inf(ok, ry, (uint32_t)e * In::bytes, 0);
            v.load_or_neg_inf(ok, rdy, (uint32_t)e * In::bytes, 0);
            by[e] = u.get(0);
            bd[e] = v.get(0);
          }
        }
      }
    }
    __syncthreads();

    for (int p = 0; p * RPP < nr; ++p) {
      const int g = p * RPP + grp;
      const bool rok = g < nr;
      const int base = h + g * cols;
      float a[E], b[E];
#pragma unroll
      for (int i = 0; i < E; ++i) {
        const int c = i * LPR + sub;
        const bool ok = rok && c < cols;
        a[i] = ok ? by[base + c] : 0.0f;
        b[i] = ok ? bd[base + c] : 0.0f;
      }
      float d = 0.0f;
#pragma unroll
      for (int i = 0; i < E; ++i) d = __builtin_fmaf(a[i], b[i], d);
      d = group_reduce<LPR, SumOp>(d);
#pragma unroll
      for (int i = 0; i < E; ++i) {
        const int c = i * LPR + sub;
        if (rok && c < cols) by[base + c] = a[i] * (b[i] - d);
      }
    }
    __syncthreads();

#pragma unroll
    for (int s = 0; s < S; ++s) {
      const int first = (s * kWave + lane) * VW;
      if (first >= h && first + VW <= span) {
        float o[VW];
#pragma unroll
        for (int k = 0; k < VW; ++k) o[k] = by[first + k];
        store_out<Out, VW>(rdx, (uint32_t)first * Out::bytes, o, false);
      } else if (first < span && first + VW > h) {
#pragma unroll
        for (int k = 0; k < VW; ++k) {
          const int e = first + k;
          if (e >= h && e < span) store_out<Out, 1>(rdx, (uint32_t)e * Out::bytes, {by[e]}, false);
        }
      }
    }
    __syncthreads();
  }
}

}  // namespace rowsm
