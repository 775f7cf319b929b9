// Large-row softmax kernel, two streaming passes over tiles: the form for
// rows longer than the single-read split form holds in registers (and for
// launches that must keep no state between them).
//
// A row is read by S >= 1 blocks of T threads that act as one group of
// S * T threads: global thread g = c * T + t of block c reads the vectors
// g + j * S * T of the row, U of them per tile (each load instruction of a
// wave reads 64 consecutive vectors).  Pass 1 keeps a running (reference,
// sum) per thread: for each tile it takes the tile maximum; when that exceeds
// the reference m by more than kRefSlack the reference moves to it (M') and
// the running sum is rescaled by exp(m - M'); then it adds exp(x - m) for the
// tile's entries.  The running sum carries a compensation term (Kahan
// summation): a thread adds one tile sum per tile (1024 of them on the
// longest rows the launcher plans, 2^23 with the narrowest forced shape), and
// near-equal addends would otherwise round the same way at every step, an
// error that grows with their count.  Together the two keep the rounding
// error of the sum independent of the row length.  The per-thread pairs are
// merged across the wave with DPP/permlane steps and across waves through
// LDS (maximum first, then one rescale per partial sum).  With S > 1
// the blocks of a row then exchange their pairs once, through the split
// form's tagged words and workspace (split_row.hpp: protocol, tags, the
// bounded wait), and merge them in block order; a block whose wait for a peer
// gives up runs that peer's pass 1 itself (large_pass1(), the same code), so
// the merged pair does not depend on the wait.  Pass 2 reads the block's share
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

// How far (natural-log units) a tile maximum may exceed the exponent
// reference of pass 1 before the reference moves to it.
constexpr float kRefSlack = 8.0f;

// Pass 1 of the block whose global threads are g = c * T + t: the block's
// (max, sum) pair over its share of the row, merged across the wave and then
// across waves in wave order through red_m / red_s (one barrier).  Called by
// every thread of the block, for its own share and for a peer's.
template <typename In, int VW, int U, int MODE>
__device__ __forceinline__ MaxSum large_pass1(rsrc_t rx, int g, int RT, int nvec, int ntiles, int lim,
                              float scale, float* red_m, float* red_s, int lane, int wave,
                              int nwaves) {
  constexpr bool FUSED = MODE == kFused, LOG = MODE == kLog;
  const float ninf = -__builtin_inff();
  const uint32_t vin = (uint32_t)g * (VW * In::bytes);
  // Running exponent reference m and sum s relative to it; cs is the
  // compensation of s (the sum is s - cs); mx is the running maximum.
  float m = ninf, s = 0.0f, cs = 0.0f, mx = ninf;
  for (int tt = 0; tt < ntiles; ++tt) {
    float f[U][VW];
    {
      InVec<In, VW> v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = (tt * U + u) * RT;      // first vector of this slot
        const int idx = j + g;
        v[u].load_or_neg_inf(idx < nvec && (!FUSED || idx * VW <= lim), rx, vin,
                             (uint32_t)j * (VW * In::bytes));
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        v[u].to_float(f[u]);
        if constexpr (FUSED) fused_apply(f[u], ((tt * U + u) * RT + g) * VW, lim, scale);
      }
    }
    float tm = ninf;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int i = 0; i < VW; ++i) tm = fmax_nn(tm, f[u][i]);
    // The exponent reference m follows the running maximum lazily: it moves
    // only to a tile maximum that exceeds it by more than kRefSlack.  Every
    // term exp(x - m) then stays below e^kRefSlack, and every move scales the
    // sum gathered so far by less than e^-kRefSlack, so the rounding of the
    // rescale factors does not build up with the number of tiles (a reference
    // that followed each rise of the maximum would rescale once per tile on
    // an ascending row).
    const float M = (tm > m + kRefSlack) ? tm : m;
    mx = fmax_nn(mx, tm);
    const float nml = (M == ninf) ? 0.0f : -M * kLog2e;
    // The tile is summed on its own and then added to the running sum, so a
    // thread's serial chain of additions is one tile plus one per tile.
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

  // The thread's pair relative to its maximum (one more rescale), so that
  // every later step sees sums of terms <= 1, as the other forms do.
  MaxSum ms = group_merge<kWave>({mx, rescale(s - cs, m, mx)});
  if (lane == 0) {
    red_m[wave] = ms.m;
    red_s[wave] = ms.s;
  }
  __syncthreads();
  // Across waves: the maximum first, then each wave's sum rescaled once to it
  // and added in wave order.
  float M = red_m[0];
  for (int i = 1; i < nwaves; ++i) M = fmax_nn(M, red_m[i]);
  float s_all = rescale(red_s[0], red_m[0], M);
  for (int i = 1; i < nwaves; ++i) s_all += rescale(red_s[i], red_m[i], M);
  return {M, s_all};
}

template <typename In, typename Out, int VW, int U, int MODE>
__global__ __launch_bounds__(1024) void large_row_kernel(
    const typename In::storage* x, typename Out::storage* y, int64_t rows, int cols, int S,
    SplitWorkspace w, uint32_t tag0, Fused fz) {
  constexpr bool FUSED = MODE == kFused, LOG = MODE == kLog;
  // Wave 0 holds up to kPeersPerLane peers per lane in the exchange.
  constexpr int kPeersPerLane = 4;
  __shared__ float red_m[16];
  __shared__ float red_s[16];
  __shared__ float bcast[2];
  __shared__ uint64_t missing_lanes[kPeersPerLane];
  __shared__ MaxSum peer[kPeersPerLane * kWave];  // the row's pairs, when a wait gave up

  const int T = blockDim.x;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const bool wl = stores_whole_lines(y, (int64_t)cols * Out::bytes);  // sc1 stores
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
  const uint32_t vin = (uint32_t)g * (VW * In::bytes);
  const uint32_t vout = (uint32_t)g * (VW * Out::bytes);
  bool gave_up = false;  // per lane of the first wave

  uint32_t k = 0;
  for (int64_t row = q; row < rows; row += slots, ++k) {
    const rsrc_t rx = make_rsrc(x + row * cols, (uint64_t)cols * In::bytes);
    const rsrc_t ry = make_rsrc(y + row * cols, (uint64_t)cols * Out::bytes);
    const int lim = FUSED ? fused_limit(fz, row, cols) : cols - 1;

    MaxSum ms = large_pass1<In, VW, U, MODE>(rx, g, RT, nvec, ntiles, lim, fz.scale, red_m, red_s,
                                             lane, wave, nwaves);

    if (S > 1) {
      // Exchange with the other blocks of the row: wave 0's lane l holds the
      // pairs of blocks l + 64 j, j < kPeersPerLane; they are merged in block
      // order (per lane over j, then across lanes).  When a wait gave up,
      // wave 0 parks its pairs in LDS (peer[l + 64 j]) and the block
      // recomputes the missing ones.
      auto finish = [&](const MaxSum (&pr)[kPeersPerLane]) {
        // The lane's peers: their maximum, then each sum rescaled once to it
        // and added in block order; then across the lanes.
        MaxSum p = {-__builtin_inff(), 0.0f};
#pragma unroll
        for (int j = 0; j < kPeersPerLane; ++j)
          if (lane + j * kWave < S) p.m = fmax_nn(p.m, pr[j].m);
#pragma unroll
        for (int j = 0; j < kPeersPerLane; ++j)
          if (lane + j * kWave < S) p.s += rescale(pr[j].s, pr[j].m, p.m);
        p = group_merge<kWave>(p);  // fixed lane order: deterministic
        if (lane == 0) {
          bcast[0] = p.m;
          bcast[1] = p.s;
        }
      };
      if (wave == 0) {
        const uint32_t tag = tag0 + k;
        uint64_t* gw = split_group_words(w, q, k & 1, S);
        if (lane == 0) split_publish(gw, S, c, tag, ms.m, ms.s);
        MaxSum pr[kPeersPerLane];
        uint64_t any = 0;
#pragma unroll
        for (int j = 0; j < kPeersPerLane; ++j) {
          const int b = lane + j * kWave;
          bool ok = true;
          pr[j] = {-__builtin_inff(), 0.0f};
          if (b == c) pr[j] = ms;
          else if (b < S) ok = split_poll(w, gw, S, b, tag, &gave_up, &pr[j].m, &pr[j].s);
          const uint64_t miss = lanes_missing(ok);
          if (lane == 0) missing_lanes[j] = miss;
          any |= miss;
        }
        if (any == 0) {
          finish(pr);
        } else {
#pragma unroll
          for (int j = 0; j < kPeersPerLane; ++j) peer[lane + j * kWave] = pr[j];
        }
      }
      __syncthreads();
      uint64_t any = 0;
#pragma unroll
      for (int j = 0; j < kPeersPerLane; ++j) any |= missing_lanes[j];
      if (any != 0) {
#pragma unroll 1
        for (int j = 0; j < kPeersPerLane; ++j) {
          for (uint64_t mm = missing_lanes[j]; mm != 0; mm &= mm - 1) {
            const int l = __builtin_ctzll(mm);
            // red_m / red_s are free again: every wave read them before the
            // barrier above (or before the previous recomputation's).
            __syncthreads();
            const MaxSum r = large_pass1<In, VW, U, MODE>(rx, (l + j * kWave) * T + tid, RT, nvec,
                                                          ntiles, lim, fz.scale, red_m, red_s,
                                                          lane, wave, nwaves);
            if (tid == 0) peer[l + j * kWave] = r;
          }
        }
        __syncthreads();
        if (wave == 0) {
          MaxSum pr[kPeersPerLane];
#pragma unroll
          for (int j = 0; j < kPeersPerLane; ++j) pr[j] = peer[lane + j * kWave];
          finish(pr);
        }
        __syncthreads();
      }
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
        v[u].load_or_neg_inf(idx < nvec && (!FUSED || idx * VW <= lim), rx, vin,
                             (uint32_t)j * (VW * In::bytes));
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
        if (idx < nvec) store_out<Out, VW>(ry, vout + (uint32_t)j * (VW * Out::bytes), o, wl);
      }
    }
    // Every wave has read red_m / red_s, bcast, missing_lanes and peer before
    // the next row rewrites them.
    __syncthreads();
  }
}

}  // namespace rowsm
