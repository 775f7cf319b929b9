// Medium-row softmax kernel: one row per group of WPR wavefronts, the whole row
// held in registers, so x is read once and y written once.
//
// A block holds RPB = waves / WPR row groups.  Thread t of a row group
// (t = 64 * wave_in_group + lane, T = 64 * WPR threads) owns the vectors
// t, t + T, ..., t + (NV-1) T of the row, with NV = ceil(nvec / T) fixed at
// compile time so that only the last slot can be partial, and every load
// instruction of a wave reads 64 consecutive vectors.  The row
// maximum and the row sum are reduced inside each wave with DPP and
// permlane swaps, then across the WPR waves through LDS (one barrier each;
// WPR == 1 needs neither LDS nor barriers).
//
// MODE selects the output form (see the output forms in rowsm_device.hpp).
// kFused computes softmax(scale * x + causal mask): columns past the row's
// limit are not loaded and come out as exact zeros.  kLog writes
// (x - m) - ln(sum), which needs x itself and not exp(x - m) at the end.
//
// PACKED == false widens the row to fp32 once and keeps exp(x - m) in
// registers for the normalise step.  PACKED == true keeps the row in its raw
// input form (bf16 pairs take half the registers) and evaluates exp(x - m) a
// second time when normalising; it lets one 1024-thread block hold a longer
// bf16 row in registers.
//
// Blocks loop over rows with a grid stride; the trip count depends only on
// blockIdx, so every wave of a block reaches every barrier.  Rows past the end
// hold -inf, load and store nothing, and take part in the barriers.
//
// This is the medium-row member of the row-length-specialised family the
// paper names for its running example (preamble listing style); the layout and
// reductions are this library's gfx950 design.
#pragma once

#include "rowsm_device.hpp"

namespace rowsm {

// Reduce v over the row group of the calling wave: within the wave, then,
// when the row spans wpr > 1 waves, across them through red[] (one barrier).
// Partial results are combined in wave order, so the result is deterministic.
template <typename Op>
__device__ __forceinline__ float block_row_reduce(float v, int wpr, int wave, int g, int lane,
                                                  float* red) {
  v = group_reduce<kWave, Op>(v);
  if (wpr > 1) {
    if (lane == 0) red[wave] = v;
    __syncthreads();
    v = red[g * wpr];
    for (int w = 1; w < wpr; ++w) v = Op::apply(v, red[g * wpr + w]);
  }
  return v;
}

template <typename In, typename Out, int VW, int NV, bool PACKED, int MODE>
__global__ __launch_bounds__(1024) void medium_row_kernel(
    const typename In::storage* x, typename Out::storage* y,
    int64_t rows, int cols, int wpr, Fused fz) {
  constexpr bool FUSED = MODE == kFused, LOG = MODE == kLog;
  static_assert(!(PACKED && FUSED), "the fused variants keep the row in fp32");
  __shared__ float red_m[16];
  __shared__ float red_s[16];

  const int lane = threadIdx.x & (kWave - 1);
  const bool wl = stores_whole_lines(y, (int64_t)cols * Out::bytes);  // sc1 stores
  const int wave = wave_id();
  const int rpb = (blockDim.x / kWave) / wpr;
  const int g = wave / wpr;
  const int T = wpr * kWave;
  const int t = (wave - g * wpr) * kWave + lane;
  const int nvec = cols / VW;
  const uint32_t vin = (uint32_t)t * (VW * In::bytes);
  const uint32_t vout = (uint32_t)t * (VW * Out::bytes);
  const uint32_t sin = (uint32_t)T * (VW * In::bytes);    // byte stride between slots
  const uint32_t sout = (uint32_t)T * (VW * Out::bytes);
  // Slots 0 .. NV-2 lie wholly inside the row (the launcher picks
  // NV = ceil(nvec / T)); only slot NV-1 needs a per-lane bound.
  const bool last_ok = (NV - 1) * T + t < nvec;

  for (int64_t base = (int64_t)blockIdx.x * rpb; base < rows;
       base += (int64_t)gridDim.x * rpb) {
    const int64_t row = base + g;
    const bool row_ok = row < rows;
    const int64_t rr = row_ok ? row : 0;
    const rsrc_t rx = make_rsrc(x + rr * cols, (uint64_t)cols * In::bytes);
    const rsrc_t ry = make_rsrc(y + rr * cols, (uint64_t)cols * Out::bytes);
    const int lim = FUSED ? fused_limit(fz, rr, cols) : cols - 1;

    if constexpr (PACKED) {
      InVec<In, VW> v[NV];
#pragma unroll
      for (int s = 0; s < NV; ++s) {
        v[s].load_or_neg_inf(row_ok && (s < NV - 1 || last_ok), rx, vin, s * sin);
      }
      float mx = -__builtin_inff();
#pragma unroll
      for (int s = 0; s < NV; ++s)
#pragma unroll
        for (int i = 0; i < VW; ++i) mx = fmax_nn(mx, v[s].get(i));
      mx = block_row_reduce<MaxOp>(mx, wpr, wave, g, lane, red_m);
      const float nml = -mx * kLog2e;
#pragma unroll
      for (int s = 0; s < NV; ++s) v[s].opaque();
      float sum = 0.0f;
#pragma unroll
      for (int s = 0; s < NV; ++s)
#pragma unroll
        for (int i = 0; i < VW; ++i)
          sum += LOG ? exp2_fast((v[s].get(i) - mx) * kLog2e)
                     : exp2_fast(__builtin_fmaf(v[s].get(i), kLog2e, nml));
      sum = block_row_reduce<SumOp>(sum, wpr, wave, g, lane, red_s);
#pragma unroll
      for (int s = 0; s < NV; ++s) v[s].opaque();
      const float inv = __builtin_amdgcn_rcpf(sum);  // v_rcp_f32, 1 ulp
      const float lns = LOG ? ln_fast(sum) : 0.0f;
#pragma unroll
      for (int s = 0; s < NV; ++s) {
        float o[VW];
#pragma unroll
        for (int i = 0; i < VW; ++i)
          o[i] = LOG ? (v[s].get(i) - mx) - lns
                     : exp2_fast(__builtin_fmaf(v[s].get(i), kLog2e, nml)) * inv;
        if (row_ok && (s < NV - 1 || last_ok)) store_out<Out, VW>(ry, vout + s * sout, o, wl);
      }
    } else {
      float f[NV][VW];
      {
        InVec<In, VW> v[NV];
#pragma unroll
        for (int s = 0; s < NV; ++s) {
          v[s].load_or_neg_inf(
              row_ok && (s < NV - 1 || last_ok) && (!FUSED || (s * T + t) * VW <= lim), rx, vin,
              s * sin);
        }
#pragma unroll
        for (int s = 0; s < NV; ++s) {
          v[s].to_float(f[s]);
          if constexpr (FUSED) fused_apply(f[s], (s * T + t) * VW, lim, fz.scale);
        }
      }
      if constexpr (FUSED) {
        // Vectors wholly past the limit are zeros whatever the row's max and
        // sum: store them now, overlapping the loads and the reductions.
        float z[VW];
#pragma unroll
        for (int i = 0; i < VW; ++i) z[i] = 0.0f;
#pragma unroll
        for (int s = 0; s < NV; ++s)
          if (row_ok && (s < NV - 1 || last_ok) && (s * T + t) * VW > lim)
            store_out<Out, VW>(ry, vout + s * sout, z, wl);
      }
      float mx = -__builtin_inff();
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
        else exp_accumulate<FUSED>(f[s], nml, (s * T + t) * VW <= lim, &sum);
      }
      sum = block_row_reduce<SumOp>(sum, wpr, wave, g, lane, red_s);
      const float inv = __builtin_amdgcn_rcpf(sum);  // v_rcp_f32, 1 ulp
      const float lns = LOG ? ln_fast(sum) : 0.0f;
      // A row whose sum is not >= 1 (nothing kept, or a NaN/+inf among the
      // kept values) is all NaN, masked columns included: rewrite those too.
      const bool redo_masked = FUSED && !(sum > 0.5f);
#pragma unroll
      for (int s = 0; s < NV; ++s) {
#pragma unroll
        for (int i = 0; i < VW; ++i) f[s][i] = LOG ? (f[s][i] - mx) - lns : f[s][i] * inv;
        if (row_ok && (s < NV - 1 || last_ok) &&
            (!FUSED || (s * T + t) * VW <= lim || redo_masked))
          store_out<Out, VW>(ry, vout + s * sout, f[s], wl);
      }
    }
  }
}

}  // namespace rowsm
