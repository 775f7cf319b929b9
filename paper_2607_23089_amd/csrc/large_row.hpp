// Large-row softmax kernel, two streaming passes over tiles: the form for
// rows longer than the single-read split form holds in registers (and for
// launches that must keep no state between them).
//
// A row is read by S >= 1 blocks of T threads that act as one group of
// S * T threads: global thread g = c * T + t of block c reads the vectors
// g + j * S * T of the row, U of them per tile (each load instruction of a
// wave reads 64 consecutive vectors).  Pass 1 keeps a running (max, sum) per
// thread: for each tile it takes the tile maximum M' = max(m, tile max),
// rescales the running sum by exp(m - M') and adds exp(x - M') for the tile's
// entries.  The running sum carries a compensation term (Kahan summation): a
// thread adds one tile sum per tile, up to 2^16 of them on the longest rows,
// and near-equal addends would otherwise round the same way at every step, an
// error that grows with their count.  The per-thread pairs are merged across
// the wave with DPP/permlane steps and across waves through LDS.  With S > 1
// the blocks of a row then exchange their pairs once, through the split
// form's tagged words and workspace (split_row.hpp: protocol, tags, forward
// progress), and merge them in block order.  Pass 2 reads the block's share
// again, last tile first so that the most recently fetched tiles are re-read
// while they are most likely still cached, and writes exp(x - M) / sum.
//
// S = 1 is one block per row, for launches of many rows (or a grid capped per
// compute unit, or a capture with no workspace slice left); S > 1 spreads a
// few long rows over the device.
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

#include "split_row.hpp"

namespace rowsm {

template <typename In, typename Out, int VW, int U, int MODE>
__global__ __launch_bounds__(1024) void large_row_kernel(
    const typename In::storage* __restrict__ x, typename Out::storage* __restrict__ y,
    int64_t rows, int cols, int S, SplitWorkspace w, uint32_t tag0, Fused fz) {
  constexpr bool FUSED = MODE == kFused, LOG = MODE == kLog;
  __shared__ float red_m[16];
  __shared__ float red_s[16];
  __shared__ float bcast[2];

  const int T = blockDim.x;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = wave_id();
  const int nwaves = T / kWave;
  const int c = blockIdx.x % S;                 // block of the row group
  const int q = blockIdx.x / S;                 // row group
  const int64_t slots = gridDim.x / S;
  const int RT = S * T;                         // threads of a row
  const int g = c * T + tid;
  const int nvec = cols / VW;
  const int per_thread = (nvec + RT - 1) / RT;  // vector slots of a thread
  const int ntiles = (per_thread + U - 1) / U;
  const float ninf = -__builtin_inff();
  const uint32_t vin = (uint32_t)g * (VW * In::bytes);
  const uint32_t vout = (uint32_t)g * (VW * Out::bytes);
  if (S > 1) tag0 = split_tag0(w, tag0);
  bool gave_up = false;  // per lane of the first wave

  uint32_t k = 0;
  for (int64_t row = q; row < rows; row += slots, ++k) {
    const rsrc_t rx = make_rsrc(x + row * cols, (uint64_t)cols * In::bytes);
    const rsrc_t ry = make_rsrc(y + row * cols, (uint64_t)cols * Out::bytes);
    const int lim = FUSED ? fused_limit(fz, row, cols) : cols - 1;

    // Pass 1: running (max, sum); cs is the compensation of s (the sum is
    // s - cs).
    float m = ninf, s = 0.0f, cs = 0.0f;
    for (int tt = 0; tt < ntiles; ++tt) {
      float f[U][VW];
      {
        InVec<In, VW> v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int j = (tt * U + u) * RT;      // first vector of this slot
          const int idx = j + g;
          if (idx < nvec && (!FUSED || idx * VW <= lim))
            v[u].load(rx, vin, (uint32_t)j * (VW * In::bytes));
          else
            v[u].set_neg_inf();
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          v[u].to_float(f[u]);
          if constexpr (FUSED) fused_apply(f[u], ((tt * U + u) * RT + g) * VW, lim, fz.scale);
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
        cs = rescale(cs, m, M);
      }
      const float yk = ts - cs;
      const float t = s + yk;
      cs = (t - s) - yk;
      s = t;
      m = M;
    }

    MaxSum ms = group_merge<kWave>({m, s - cs});
    if (lane == 0) {
      red_m[wave] = ms.m;
      red_s[wave] = ms.s;
    }
    __syncthreads();
    ms = {red_m[0], red_s[0]};
    for (int i = 1; i < nwaves; ++i) ms = merge(ms, {red_m[i], red_s[i]});

    if (S > 1) {
      // Exchange with the other blocks of the row (first wave only): publish
      // this block's pair, merge all S pairs in block order.
      if (wave == 0) {
        const uint32_t b0 = (uint32_t)q * S;
        const uint64_t tag = (uint64_t)(tag0 + k) << 32;
        const uint32_t slot = k & 1;
        if (lane == 0) {
          __hip_atomic_store(&w.wm[2 * (b0 + c) + slot], tag | __float_as_uint(ms.m),
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(&w.ws[2 * (b0 + c) + slot], tag | __float_as_uint(ms.s),
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        MaxSum p = {ninf, 0.0f};
        for (int b = lane; b < S; b += kWave) p = merge(p, split_poll_pair(w, b0 + b, slot, tag,
                                                                           &gave_up));
        p = group_merge<kWave>(p);  // fixed lane order: deterministic
        if (lane == 0) {
          bcast[0] = p.m;
          bcast[1] = p.s;
        }
      }
      __syncthreads();
      ms = {bcast[0], bcast[1]};
    }

    const float nml = -ms.m * kLog2e;
    const float inv = __builtin_amdgcn_rcpf(ms.s);  // v_rcp_f32, 1 ulp
    const float lns = LOG ? ln_fast(ms.s) : 0.0f;

    // Pass 2: normalise, last tile first.
    for (int tt = ntiles - 1; tt >= 0; --tt) {
      InVec<In, VW> v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = (tt * U + u) * RT;
        const int idx = j + g;
        if (idx < nvec && (!FUSED || idx * VW <= lim))
          v[u].load(rx, vin, (uint32_t)j * (VW * In::bytes));
        else
          v[u].set_neg_inf();
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = (tt * U + u) * RT;
        const int idx = j + g;
        float o[VW];
        v[u].to_float(o);
        if constexpr (FUSED) fused_apply(o, idx * VW, lim, fz.scale);
#pragma unroll
        for (int i = 0; i < VW; ++i)
          o[i] = LOG ? (o[i] - ms.m) - lns : exp2_fast(__builtin_fmaf(o[i], kLog2e, nml)) * inv;
        if (idx < nvec) store_out<Out, VW>(ry, vout + (uint32_t)j * (VW * Out::bytes), o);
      }
    }
    // Every wave has read red_m / red_s and bcast before the next row
    // rewrites them.
    __syncthreads();
  }
}

}  // namespace rowsm
