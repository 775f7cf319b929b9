// Small-row softmax kernel: several rows per 64-lane wavefront.
//
// A row of nvec = cols / VW vectors is held by LPR lanes (LPR the power of two
// >= nvec, at most 32), one vector per lane, so a wave covers 64 / LPR rows
// with each load instruction and the wave's 64 lanes read one contiguous
// stretch of memory when the rows are full.  Each lane repeats this for RPL
// row groups so that RPL independent 16-byte loads per lane are in flight
// before the first reduction.  Max and sum are reduced across the LPR lanes of
// a row with DPP steps only (no LDS, no barrier).  Lanes past the end of a row
// or past the last row load nothing and hold -inf, which leaves the max
// unchanged and contributes exp(-inf) = 0 to the sum.
//
// MODE selects the output form (kPlain, kFused or kLog; see the output forms
// in rowsm_device.hpp).
//
// This is the small-row member of the row-length-specialised family the paper
// names for its running example (small/medium/large row kernels plus a row
// launcher, preamble listing style); the packing, the lane layout and the DPP
// reductions are this library's gfx950 design.
#pragma once

#include "rowsm_device.hpp"

namespace rowsm {

template <typename In, typename Out, int VW, int LPR, int RPL, int MODE>
__global__ __launch_bounds__(256) void small_row_kernel(
    const typename In::storage* x, typename Out::storage* y,
    int64_t rows, int cols, Fused fz) {
  constexpr bool FUSED = MODE == kFused, LOG = MODE == kLog;
  constexpr int RPW = kWave / LPR;     // rows per wave per load instruction
  constexpr int RPT = RPW * RPL;       // rows per wave per task
  const int lane = threadIdx.x & (kWave - 1);
  const bool wl = stores_whole_lines(y, (int64_t)cols * Out::bytes);  // sc1 stores
  const int sub = lane % LPR;          // vector index inside the row
  const int grp = lane / LPR;          // row inside the load group
  const int nvec = cols / VW;
  const bool col_ok = sub < nvec;
  const uint32_t lane_elt = (uint32_t)(grp * cols + sub * VW);  // < 64 * 256
  const uint32_t vin = lane_elt * In::bytes, vout = lane_elt * Out::bytes;
  const uint32_t group_elts = (uint32_t)RPW * (uint32_t)cols;   // elements per load group

  const int waves_per_block = blockDim.x / kWave;
  const int64_t wave = (int64_t)blockIdx.x * waves_per_block + wave_id();
  const int64_t nwaves = (int64_t)gridDim.x * waves_per_block;
  const int64_t ntasks = (rows + RPT - 1) / RPT;

  for (int64_t task = wave; task < ntasks; task += nwaves) {
    const int64_t row0 = task * RPT;
    const int64_t nrows = rows - row0 < RPT ? rows - row0 : RPT;
    const rsrc_t rx = make_rsrc(x + row0 * cols, (uint64_t)(nrows * cols) * In::bytes);
    const rsrc_t ry = make_rsrc(y + row0 * cols, (uint64_t)(nrows * cols) * Out::bytes);

    int lim[RPL];
#pragma unroll
    for (int k = 0; k < RPL; ++k)
      lim[k] = FUSED ? fused_limit(fz, row0 + k * RPW + grp, cols) : cols - 1;

    InVec<In, VW> v[RPL];
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      const bool ok = col_ok && (k * RPW + grp < nrows) && (!FUSED || sub * VW <= lim[k]);
      v[k].load_or_neg_inf(ok, rx, vin, k * group_elts * In::bytes);
    }

    float f[RPL][VW];
    float m[RPL];
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      v[k].to_float(f[k]);
      if constexpr (FUSED) fused_apply(f[k], sub * VW, lim[k], fz.scale);
      float t = f[k][0];
#pragma unroll
      for (int i = 1; i < VW; ++i) t = fmax_nn(t, f[k][i]);
      m[k] = t;
    }
#pragma unroll
    for (int k = 0; k < RPL; ++k) m[k] = group_reduce<LPR, MaxOp>(m[k]);

    float s[RPL];
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      float t = 0.0f;
      if constexpr (LOG) {
        exp_sum_keep(f[k], m[k], &t);
      } else {
        const float nml = -m[k] * kLog2e;
#pragma unroll
        for (int i = 0; i < VW; ++i) {
          f[k][i] = exp2_fast(__builtin_fmaf(f[k][i], kLog2e, nml));
          t += f[k][i];
        }
      }
      s[k] = t;
    }
#pragma unroll
    for (int k = 0; k < RPL; ++k) s[k] = group_reduce<LPR, SumOp>(s[k]);

#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      if constexpr (LOG) {
        const float lns = ln_fast(s[k]);
#pragma unroll
        for (int i = 0; i < VW; ++i) f[k][i] = (f[k][i] - m[k]) - lns;
      } else {
        const float inv = __builtin_amdgcn_rcpf(s[k]);  // v_rcp_f32, 1 ulp
#pragma unroll
        for (int i = 0; i < VW; ++i) f[k][i] *= inv;
      }
      const bool ok = col_ok && (k * RPW + grp < nrows);
      if (ok) store_out<Out, VW>(ry, vout + k * group_elts * Out::bytes, f[k], wl);
    }
  }
}

}  // namespace rowsm
