// Large-row softmax kernel: one block per row, two streaming passes over tiles.
//
// A row too long for the registers of one block is cut into tiles of
// T * U vectors (T threads, U vectors per thread; each load instruction of a
// wave reads 64 consecutive vectors).  Pass 1 keeps a running (max, sum) per
// thread: for each tile it takes the tile maximum M' = max(m, tile max),
// rescales the running sum by exp(m - M') and adds exp(x - M') for the tile's
// entries.  The running sum carries a compensation term (Kahan summation):
// a thread adds one tile sum per tile, up to 2^16 of them on the longest rows,
// and near-equal addends would otherwise round the same way at every step, an
// error that grows with their count.  The per-thread pairs are merged across
// the wave with DPP/permlane steps and across waves through LDS.  Pass 2 reads the row again, last tile
// first so that the most recently fetched tiles are re-read while they are
// most likely still cached, and writes exp(x - m) / sum.
//
// MODE selects the output form (see the output forms in rowsm_device.hpp).
// kFused computes softmax(scale * x + causal mask): columns past the row's
// limit are not loaded and come out as exact zeros.  kLog writes
// (x - m) - ln(sum) in pass 2.
//
// A thread that has seen only -inf so far uses 0 in place of -m*log2e, so a
// fully masked tile adds exp(-inf) = 0 instead of exp(-inf + inf) = NaN; a row
// whose maximum is -inf, +inf or that holds a NaN still ends as all NaN.
//
// This is the large-row member of the row-length-specialised family the paper
// names for its running example (preamble listing style); the tiling and the
// online merge are this library's gfx950 design.
#pragma once

#include "rowsm_device.hpp"

namespace rowsm {

template <typename In, typename Out, int VW, int U, int MODE>
__global__ __launch_bounds__(1024) void large_row_kernel(
    const typename In::storage* __restrict__ x, typename Out::storage* __restrict__ y,
    int64_t rows, int cols, Fused fz) {
  constexpr bool FUSED = MODE == kFused, LOG = MODE == kLog;
  __shared__ float red_m[16];
  __shared__ float red_s[16];

  const int T = blockDim.x;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int nwaves = T / kWave;
  const int nvec = cols / VW;
  const int tile = T * U;
  const int ntiles = (nvec + tile - 1) / tile;
  const float ninf = -__builtin_inff();
  const uint32_t vin = (uint32_t)tid * (VW * In::bytes);
  const uint32_t vout = (uint32_t)tid * (VW * Out::bytes);

  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    const rsrc_t rx = make_rsrc(x + row * cols, (uint64_t)cols * In::bytes);
    const rsrc_t ry = make_rsrc(y + row * cols, (uint64_t)cols * Out::bytes);
    const int lim = FUSED ? fused_limit(fz, row, cols) : cols - 1;

    // Pass 1: running (max, sum); c is the compensation of s (the sum is
    // s - c).
    float m = ninf, s = 0.0f, c = 0.0f;
    for (int tt = 0; tt < ntiles; ++tt) {
      float f[U][VW];
      {
        InVec<In, VW> v[U];
        const bool full = tt < ntiles - 1;  // every tile but the last is whole
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int idx = tt * tile + u * T + tid;
          if ((full || idx < nvec) && (!FUSED || idx * VW <= lim))
            v[u].load(rx, vin, (uint32_t)(tt * tile + u * T) * (VW * In::bytes));
          else
            v[u].set_neg_inf();
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          v[u].to_float(f[u]);
          if constexpr (FUSED) fused_apply(f[u], (tt * tile + u * T + tid) * VW, lim, fz.scale);
        }
      }
      float tm = ninf;
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int i = 0; i < VW; ++i) tm = fmax_nn(tm, f[u][i]);
      const float M = fmax_nn(m, tm);
      const float nml = (M == ninf) ? 0.0f : -M * kLog2e;
      // The tile is summed on its own and then added to the running sum, so
      // a thread's serial chain of additions is one tile plus one per tile.
      float ts = 0.0f;
      if constexpr (LOG) {
        const float ref = exp_ref(M);
#pragma unroll
        for (int u = 0; u < U; ++u) exp_sum_keep(f[u], ref, &ts);
      } else {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
          for (int i = 0; i < VW; ++i)
            ts += exp2_fast(__builtin_fmaf(f[u][i], kLog2e, nml));
      }
      if (M != m) {
        s = rescale(s, m, M);
        c = rescale(c, m, M);
      }
      const float yk = ts - c;
      const float t = s + yk;
      c = (t - s) - yk;
      s = t;
      m = M;
    }

    MaxSum ms = group_merge<kWave>({m, s - c});
    if (lane == 0) {
      red_m[wave] = ms.m;
      red_s[wave] = ms.s;
    }
    __syncthreads();
    ms = {red_m[0], red_s[0]};
    for (int w = 1; w < nwaves; ++w) ms = merge(ms, {red_m[w], red_s[w]});
    __syncthreads();  // every wave has read red_m / red_s before the next row

    const float nml = -ms.m * kLog2e;
    const float inv = __builtin_amdgcn_rcpf(ms.s);  // v_rcp_f32, 1 ulp
    const float lns = LOG ? ln_fast(ms.s) : 0.0f;

    // Pass 2: normalise, last tile first.
    for (int tt = ntiles - 1; tt >= 0; --tt) {
      InVec<In, VW> v[U];
      const bool full = tt < ntiles - 1;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int idx = tt * tile + u * T + tid;
        if ((full || idx < nvec) && (!FUSED || idx * VW <= lim))
          v[u].load(rx, vin, (uint32_t)(tt * tile + u * T) * (VW * In::bytes));
        else
          v[u].set_neg_inf();
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int idx = tt * tile + u * T + tid;
        float o[VW];
        v[u].to_float(o);
        if constexpr (FUSED) fused_apply(o, idx * VW, lim, fz.scale);
#pragma unroll
        for (int i = 0; i < VW; ++i)
          o[i] = LOG ? (o[i] - ms.m) - lns : exp2_fast(__builtin_fmaf(o[i], kLog2e, nml)) * inv;
        if (full || idx < nvec)
          store_out<Out, VW>(ry, vout + (uint32_t)(tt * tile + u * T) * (VW * Out::bytes), o);
      }
    }
  }
}

}  // namespace rowsm
