// Softmax backward kernels: for every row,
//     dx_j = y_j * (dy_j - d),   d = sum_k y_k * dy_k,
// the product of the softmax Jacobian diag(y) - y y^T with dy, where y is
// the forward output and dy the gradient with respect to it.
//
// The work is one dot product per row and one elementwise pass: two input
// streams (y, dy) and one output stream (dx), HBM bound.  The same
// row-length families as the forward kernels, with the same lane layouts:
//   small   several rows per wave, a row's vectors on LPR lanes, DPP sums;
//   medium  one row per group of WPR waves, the row pair held in registers;
//   split   one row over S co-resident blocks that exchange block partial
//           sums of d (split_row.hpp's protocol, one word per block);
//   large   two streaming passes (dot, then dx) for rows longer than that,
//           over S >= 1 blocks per row.
// The register-resident forms keep y and dy in their raw input form (bf16
// pairs take half the registers) and widen each element where it is used,
// so one read of each input suffices.  The raw words are hidden from the
// optimiser between the dot product and the gradient (InVec::opaque()):
// otherwise it keeps the widened fp32 copies of the first phase alive for the
// second, twice the registers, and the widest bf16 forms spilled.  Lanes past the end of a row hold
// zeros, which add nothing to d.
//
// d is accumulated with fma in fp32: a lane's vectors in slot order, then
// lanes in a fixed DPP tree, waves and blocks in index order, so the result
// is deterministic.  dx may be y or dy itself (same dtype): every element is
// read by the lane that writes it, before the write.
#pragma once

#include "medium_row.hpp"
#include "rowsm_device.hpp"
#include "split_row.hpp"

namespace rowsm {

// d += y . dy over one vector pair.
template <typename In, int VW>
__device__ __forceinline__ float dot_vec(const InVec<In, VW>& a, const InVec<In, VW>& b,
                                         float acc) {
#pragma unroll
  for (int i = 0; i < VW; ++i) acc = __builtin_fmaf(a.get(i), b.get(i), acc);
  return acc;
}

// dx = y * (dy - d) for one vector pair.
template <typename In, int VW>
__device__ __forceinline__ void grad_vec(const InVec<In, VW>& a, const InVec<In, VW>& b, float d,
                                         float (&o)[VW]) {
#pragma unroll
  for (int i = 0; i < VW; ++i) o[i] = a.get(i) * (b.get(i) - d);
}

// ---- small rows ---------------------------------------------------------------

template <typename In, typename Out, int VW, int LPR, int RPL>
__global__ __launch_bounds__(256) void bwd_small_kernel(
    const typename In::storage* y, const typename In::storage* dy,
    typename Out::storage* dx, int64_t rows, int cols) {
  constexpr int RPW = kWave / LPR;     // rows per wave per load instruction
  constexpr int RPT = RPW * RPL;       // rows per wave per task
  const int lane = threadIdx.x & (kWave - 1);
  const bool wl = stores_whole_lines(dx, (int64_t)cols * Out::bytes);  // sc1 stores
  const int sub = lane % LPR;
  const int grp = lane / LPR;
  const int nvec = cols / VW;
  const bool col_ok = sub < nvec;
  const uint32_t lane_elt = (uint32_t)(grp * cols + sub * VW);
  const uint32_t vin = lane_elt * In::bytes, vout = lane_elt * Out::bytes;
  const uint32_t group_elts = (uint32_t)RPW * (uint32_t)cols;

  const int waves_per_block = blockDim.x / kWave;
  const int64_t wave = (int64_t)blockIdx.x * waves_per_block + wave_id();
  const int64_t nwaves = (int64_t)gridDim.x * waves_per_block;
  const int64_t ntasks = (rows + RPT - 1) / RPT;

  for (int64_t task = wave; task < ntasks; task += nwaves) {
    const int64_t row0 = task * RPT;
    const int64_t nrows = rows - row0 < RPT ? rows - row0 : RPT;
    const uint64_t in_bytes = (uint64_t)(nrows * cols) * In::bytes;
    const rsrc_t ry = make_rsrc(y + row0 * cols, in_bytes);
    const rsrc_t rdy = make_rsrc(dy + row0 * cols, in_bytes);
    const rsrc_t rdx = make_rsrc(dx + row0 * cols, (uint64_t)(nrows * cols) * Out::bytes);

    InVec<In, VW> a[RPL], b[RPL];
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      if (col_ok && k * RPW + grp < nrows) {
        a[k].load(ry, vin, k * group_elts * In::bytes);
        b[k].load(rdy, vin, k * group_elts * In::bytes);
      } else {
        a[k].set_zero();
        b[k].set_zero();
      }
    }
    float d[RPL];
#pragma unroll
    for (int k = 0; k < RPL; ++k) d[k] = dot_vec(a[k], b[k], 0.0f);
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      a[k].opaque();
      b[k].opaque();
    }
#pragma unroll
    for (int k = 0; k < RPL; ++k) d[k] = group_reduce<LPR, SumOp>(d[k]);
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      float o[VW];
      grad_vec(a[k], b[k], d[k], o);
      if (col_ok && k * RPW + grp < nrows)
        store_out<Out, VW>(rdx, vout + k * group_elts * Out::bytes, o, wl);
    }
  }
}

// ---- medium rows --------------------------------------------------------------

// Thread t of a row group of WPR waves owns vectors t, t + T, ..., t + (NV-1) T
// (T = 64 WPR; only the last slot can be partial).  One reduction per row:
// its LDS slots alternate between rows, so a wave that runs ahead to the next
// row never overwrites a partial sum a slower wave of its group still reads.
template <typename In, typename Out, int VW, int NV>
__global__ __launch_bounds__(1024) void bwd_medium_kernel(
    const typename In::storage* y, const typename In::storage* dy,
    typename Out::storage* dx, int64_t rows, int cols, int wpr) {
  __shared__ float red[2][16];

  const int lane = threadIdx.x & (kWave - 1);
  const bool wl = stores_whole_lines(dx, (int64_t)cols * Out::bytes);  // sc1 stores
  const int wave = wave_id();
  const int rpb = (blockDim.x / kWave) / wpr;
  const int g = wave / wpr;
  const int T = wpr * kWave;
  const int t = (wave - g * wpr) * kWave + lane;
  const int nvec = cols / VW;
  const uint32_t vin = (uint32_t)t * (VW * In::bytes);
  const uint32_t vout = (uint32_t)t * (VW * Out::bytes);
  const uint32_t sin = (uint32_t)T * (VW * In::bytes);
  const uint32_t sout = (uint32_t)T * (VW * Out::bytes);
  const bool last_ok = (NV - 1) * T + t < nvec;

  int parity = 0;
  for (int64_t base = (int64_t)blockIdx.x * rpb; base < rows;
       base += (int64_t)gridDim.x * rpb, parity ^= 1) {
    const int64_t row = base + g;
    const bool row_ok = row < rows;
    const int64_t rr = row_ok ? row : 0;
    const rsrc_t ry = make_rsrc(y + rr * cols, (uint64_t)cols * In::bytes);
    const rsrc_t rdy = make_rsrc(dy + rr * cols, (uint64_t)cols * In::bytes);
    const rsrc_t rdx = make_rsrc(dx + rr * cols, (uint64_t)cols * Out::bytes);

    InVec<In, VW> a[NV], b[NV];
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      if (row_ok && (s < NV - 1 || last_ok)) {
        a[s].load(ry, vin, s * sin);
        b[s].load(rdy, vin, s * sin);
      } else {
        a[s].set_zero();
        b[s].set_zero();
      }
    }
    float d = 0.0f;
#pragma unroll
    for (int s = 0; s < NV; ++s) d = dot_vec(a[s], b[s], d);
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      a[s].opaque();
      b[s].opaque();
    }
    d = block_row_reduce<SumOp>(d, wpr, wave, g, lane, red[parity]);
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      float o[VW];
      grad_vec(a[s], b[s], d, o);
      if (row_ok && (s < NV - 1 || last_ok)) store_out<Out, VW>(rdx, vout + s * sout, o, wl);
    }
  }
}

// ---- long rows: split over co-resident blocks -----------------------------------
//
// Layout, grid and co-residency as split_row_kernel.  Each block publishes
// its partial d_b through the split form's tagged words (split_row.hpp; both
// words carry d_b) and the first wave polls the S blocks of its row group,
// then sums the partials in block order.  A block whose wait for a peer gives
// up computes that peer's partial itself (bwd_share_dot(), the same steps as
// its own), so the sum does not depend on the wait.  LDS reuse across rows:
// red is rewritten only after a barrier that every wave reaches after reading
// it; bcast, missing_lanes and peer (wave 0) only after the next row's
// reduction barrier, which every wave passes only after reading them.

// Partial dot product of the block whose global threads are gt = c * T + t
// (slots gt + s * RT), reduced over the wave and then over waves in wave
// order through red[] (one barrier): the steps of the kernel's own share,
// for a peer's, one slot at a time.  Called by every thread of the block.
template <typename In, int VW, int NV>
__device__ __forceinline__ float bwd_share_dot(rsrc_t ry, rsrc_t rdy, int gt, int RT, int nvec,
                                               float* red, int lane, int wave, int nwaves) {
  const bool last_ok = (NV - 1) * RT + gt < nvec;
  const uint32_t vin = (uint32_t)gt * (VW * In::bytes);
  const uint32_t sin = (uint32_t)RT * (VW * In::bytes);
  float d = 0.0f;
#pragma unroll 1
  for (int s = 0; s < NV; ++s) {
    InVec<In, VW> a, b;
    if (s < NV - 1 || last_ok) {
      a.load(ry, vin, s * sin);
      b.load(rdy, vin, s * sin);
    } else {
      a.set_zero();
      b.set_zero();
    }
    d = dot_vec(a, b, d);
  }
  return block_sum(d, red, lane, wave, nwaves);
}

template <typename In, typename Out, int VW, int NV>
__global__ __launch_bounds__(1024) void bwd_split_kernel(
    const typename In::storage* y, const typename In::storage* dy, typename Out::storage* dx,
    int64_t rows, int cols, int S, SplitWorkspace w, uint32_t tag0) {
  __shared__ float red[16];
  __shared__ float bcast;
  __shared__ uint64_t missing_lanes;
  __shared__ float peer[kWave];  // the row's partials, when a wait gave up

  const int T = blockDim.x;
  const int lane = threadIdx.x & (kWave - 1);
  const bool wl = stores_whole_lines(dx, (int64_t)cols * Out::bytes);  // sc1 stores
  const int wave = wave_id();
  const int nwaves = T / kWave;
  const int c = blockIdx.x % S;
  const int q = blockIdx.x / S;
  const int64_t slots = gridDim.x / S;
  const int RT = S * T;
  const int gt = c * T + threadIdx.x;
  const int nvec = cols / VW;
  const bool last_ok = (NV - 1) * RT + gt < nvec;
  const uint32_t vin = (uint32_t)gt * (VW * In::bytes);
  const uint32_t vout = (uint32_t)gt * (VW * Out::bytes);
  const uint32_t sin = (uint32_t)RT * (VW * In::bytes);
  const uint32_t sout = (uint32_t)RT * (VW * Out::bytes);

  bool gave_up = false;  // per lane of the first wave
  uint32_t k = 0;
  for (int64_t row = q; row < rows; row += slots, ++k) {
    const rsrc_t ry = make_rsrc(y + row * cols, (uint64_t)cols * In::bytes);
    const rsrc_t rdy = make_rsrc(dy + row * cols, (uint64_t)cols * In::bytes);
    const rsrc_t rdx = make_rsrc(dx + row * cols, (uint64_t)cols * Out::bytes);

    InVec<In, VW> a[NV], b[NV];
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      if (s < NV - 1 || last_ok) {
        a[s].load(ry, vin, s * sin);
        b[s].load(rdy, vin, s * sin);
      } else {
        a[s].set_zero();
        b[s].set_zero();
      }
    }
    // (bwd_share_dot() repeats exactly these steps for a peer's share)
    float d = 0.0f;
#pragma unroll
    for (int s = 0; s < NV; ++s) d = dot_vec(a[s], b[s], d);
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      a[s].opaque();
      b[s].opaque();
    }
    const float db = block_sum(d, red, lane, wave, nwaves);

    // When a wait gave up, wave 0 parks its partials in LDS, the block
    // recomputes the missing ones and then loads its own share again (none
    // of its registers stays live through the recomputation).
    auto finish = [&](float pr) {
      pr = group_reduce<kWave, SumOp>(pr);  // fixed lane order: deterministic
      if (lane == 0) bcast = pr;
    };
    if (wave == 0) {
      const uint32_t tag = tag0 + k;
      uint64_t* gw = split_group_words(w, q, k & 1, S);
      if (lane == 0 && S > 1) split_publish(gw, S, c, tag, db, db);
      float p = 0.0f;
      bool ok = true;
      float unused = 0.0f;
      if (lane == c) p = db;
      else if (lane < S) ok = split_poll(w, gw, S, lane, tag, &gave_up, &unused, &p);
      const uint64_t missing = lanes_missing(ok);
      if (lane == 0) missing_lanes = missing;
      if (missing == 0) finish(p);
      else peer[lane] = p;
    }
    __syncthreads();
    const uint64_t missing = missing_lanes;
    if (missing != 0) {
      for (uint64_t mm = missing; mm != 0; mm &= mm - 1) {
        const int bb = __builtin_ctzll(mm);
        // red is free again: every wave read it before the barrier above
        // (or before the previous recomputation's).
        __syncthreads();
        const float r = bwd_share_dot<In, VW, NV>(ry, rdy, bb * T + threadIdx.x, RT, nvec, red,
                                                  lane, wave, nwaves);
        if (threadIdx.x == 0) peer[bb] = r;
      }
      __syncthreads();
      if (wave == 0) finish(peer[lane]);
      __syncthreads();
#pragma unroll
      for (int s = 0; s < NV; ++s) {
        if (s < NV - 1 || last_ok) {
          a[s].load(ry, vin, s * sin);
          b[s].load(rdy, vin, s * sin);
        } else {
          a[s].set_zero();
          b[s].set_zero();
        }
      }
    }
    d = bcast;
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      float o[VW];
      grad_vec(a[s], b[s], d, o);
      if (s < NV - 1 || last_ok) store_out<Out, VW>(rdx, vout + s * sout, o, wl);
    }
  }
}

// ---- longest rows: two passes ----------------------------------------------------
//
// The two-pass form of the forward (large_row.hpp) for the gradient: S >= 1
// blocks per row with the same layout (global thread g = c * T + t reads the
// vector pairs g + j * S * T, U per tile).  Pass 1 accumulates d over tiles
// (a tile's partial on its own, then added to the running sum with a Kahan
// compensation term: up to 1024 tile partials per thread on the longest
// rows); with S > 1 the blocks exchange their partial d once (as
// bwd_split_kernel, up to 4 peers per lane of wave 0, a peer whose wait gives
// up recomputed with bwd_large_pass1()) and sum them in block order.  Pass 2
// reads the block's share again, last tile first, and writes dx.  An
// infinite running sum drops the compensation, so d keeps IEEE semantics
// (+-inf, or NaN from inf - inf or a NaN term).

// Pass 1 of the block whose global threads are g = c * T + t, reduced over the
// block (wave, then waves in wave order through red[]; one barrier).
template <typename In, int VW, int U>
__device__ __forceinline__ float bwd_large_pass1(rsrc_t ry, rsrc_t rdy, int g, int RT, int nvec, int ntiles,
                                 float* red, int lane, int wave, int nwaves) {
  const uint32_t vin = (uint32_t)g * (VW * In::bytes);
  float d = 0.0f, cd = 0.0f;  // running sum and its compensation
  for (int tt = 0; tt < ntiles; ++tt) {
    InVec<In, VW> a[U], b[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = (tt * U + u) * RT;
      const uint32_t so = (uint32_t)j * (VW * In::bytes);
      if (j + g < nvec) {
        a[u].load(ry, vin, so);
        b[u].load(rdy, vin, so);
      } else {
        a[u].set_zero();
        b[u].set_zero();
      }
    }
    float ts = 0.0f;
#pragma unroll
    for (int u = 0; u < U; ++u) ts = dot_vec(a[u], b[u], ts);
    const float yk = ts - cd;
    const float t = d + yk;
    cd = __builtin_isfinite(t) ? (t - d) - yk : 0.0f;
    d = t;
  }
  d -= cd;
  return block_sum(d, red, lane, wave, nwaves);
}

template <typename In, typename Out, int VW, int U>
__global__ __launch_bounds__(1024) void bwd_large_kernel(
    const typename In::storage* y, const typename In::storage* dy, typename Out::storage* dx,
    int64_t rows, int cols, int S, SplitWorkspace w, uint32_t tag0) {
  constexpr int kPeersPerLane = 4;
  __shared__ float red[16];
  __shared__ float bcast;
  __shared__ uint64_t missing_lanes[kPeersPerLane];
  __shared__ float peer[kPeersPerLane * kWave];  // the row's partials, when a wait gave up

  const int T = blockDim.x;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const bool wl = stores_whole_lines(dx, (int64_t)cols * Out::bytes);  // sc1 stores
  const int wave = wave_id();
  const int nwaves = T / kWave;
  const int c = blockIdx.x % S;
  const int q = blockIdx.x / S;
  const int64_t slots = gridDim.x / S;
  const int RT = S * T;
  const int g = c * T + tid;
  const int nvec = cols / VW;
  const int per_thread = (nvec + RT - 1) / RT;
  const int ntiles = (per_thread + U - 1) / U;
  const uint32_t vin = (uint32_t)g * (VW * In::bytes);
  const uint32_t vout = (uint32_t)g * (VW * Out::bytes);
  bool gave_up = false;  // per lane of the first wave

  uint32_t k = 0;
  for (int64_t row = q; row < rows; row += slots, ++k) {
    const rsrc_t ry = make_rsrc(y + row * cols, (uint64_t)cols * In::bytes);
    const rsrc_t rdy = make_rsrc(dy + row * cols, (uint64_t)cols * In::bytes);
    const rsrc_t rdx = make_rsrc(dx + row * cols, (uint64_t)cols * Out::bytes);

    float d = bwd_large_pass1<In, VW, U>(ry, rdy, g, RT, nvec, ntiles, red, lane, wave, nwaves);

    if (S > 1) {
      // When a wait gave up, wave 0 parks its partials in LDS (peer[l + 64 j])
      // and the block recomputes the missing ones.
      auto finish = [&](const float (&pr)[kPeersPerLane]) {
        float p = 0.0f;
#pragma unroll
        for (int j = 0; j < kPeersPerLane; ++j)
          if (lane + j * kWave < S) p += pr[j];
        p = group_reduce<kWave, SumOp>(p);  // fixed lane order: deterministic
        if (lane == 0) bcast = p;
      };
      if (wave == 0) {
        const uint32_t tag = tag0 + k;
        uint64_t* gw = split_group_words(w, q, k & 1, S);
        if (lane == 0) split_publish(gw, S, c, tag, d, d);
        float pr[kPeersPerLane];
        uint64_t any = 0;
#pragma unroll
        for (int j = 0; j < kPeersPerLane; ++j) {
          const int bb = lane + j * kWave;
          bool ok = true;
          float unused = 0.0f;
          pr[j] = 0.0f;
          if (bb == c) pr[j] = d;
          else if (bb < S) ok = split_poll(w, gw, S, bb, tag, &gave_up, &unused, &pr[j]);
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
            __syncthreads();  // red is free again (read before the last barrier)
            const float r = bwd_large_pass1<In, VW, U>(ry, rdy, (l + j * kWave) * T + tid, RT,
                                                       nvec, ntiles, red, lane, wave, nwaves);
            if (tid == 0) peer[l + j * kWave] = r;
          }
        }
        __syncthreads();
        if (wave == 0) {
          float pr[kPeersPerLane];
#pragma unroll
          for (int j = 0; j < kPeersPerLane; ++j) pr[j] = peer[lane + j * kWave];
          finish(pr);
        }
        __syncthreads();
      }
      d = bcast;
    }

    for (int tt = ntiles - 1; tt >= 0; --tt) {
      InVec<In, VW> a[U], b[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = (tt * U + u) * RT;
        const uint32_t so = (uint32_t)j * (VW * In::bytes);
        if (j + g < nvec) {
          a[u].load(ry, vin, so);
          b[u].load(rdy, vin, so);
        } else {
          a[u].set_zero();
          b[u].set_zero();
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = (tt * U + u) * RT;
        float o[VW];
        grad_vec(a[u], b[u], d, o);
        if (j + g < nvec)
          store_out<Out, VW>(rdx, vout + (uint32_t)j * (VW * Out::bytes), o, wl);
      }
    }
    // Every wave has read red, bcast, missing_lanes and peer before the next
    // row rewrites them.
    __syncthreads();
  }
}

}  // namespace rowsm
