// Split-row softmax kernel: one row spread over S co-resident blocks, each
// holding its share in registers, so x is read once even when a row is far
// larger than one compute unit's registers.
//
// Layout.  The S blocks of a row act as one group of S*T threads (T threads
// per block): global thread g = c*T + t of block c owns the vectors
// g, g + S*T, ..., g + (NV-1) S*T of the row, NV = ceil(nvec / (S*T)) fixed at
// compile time, so only the last slot can be partial and every load
// instruction of a wave reads 64 consecutive vectors.
//
// MODE selects the output form (see the output forms in rowsm_device.hpp).
// kFused computes softmax(scale * x + causal mask): columns past the row's
// limit are not loaded and come out as exact zeros.  kLog keeps x in
// registers and writes (x - M) - ln(S).
//
// Statistics.  Each block reduces its share to a pair (m_b, s_b): m_b the
// block's maximum and s_b = sum exp(x - m_b) over its entries (a block that
// holds only -inf reports (-inf, 0)).  The pairs are exchanged through global
// memory and merged, in block order, with the online identity
//     M = max_b m_b,  S = sum_b s_b * exp(m_b - M),
// and the block writes y = exp(x - m_b) * exp(m_b - M) / S from the values it
// still holds.  One exchange per row.
//
// Exchange protocol (per device workspace, reused across launches).  Each
// block publishes its pair as two self-validating 64-bit words
//     wm[b][k & 1] = (tag << 32) | bits(m_b),   ws[b][k & 1] = (tag << 32) | bits(s_b)
// with relaxed agent-scope atomic stores, where k counts the rows this block
// has processed in this launch and tag = tag0 + k is unique to (launch, k)
// (the host hands out tags; tag 0 never occurs, and fresh memory is zero).
// A peer polls both words with relaxed agent-scope atomic loads until their
// tags match: a 64-bit atomic access is indivisible, so a word with the
// expected tag carries the right value and no ordering between the two
// stores, and no cache write-back or invalidation, is needed.  Two slots per
// block (k & 1) suffice: a block can only rewrite slot k & 1 at row k + 2,
// after every block of the group has published row k + 1, i.e. after all of
// them have read row k's words.
//
// Forward progress.  A block waits only for the other blocks of its own row
// group, never for a later group, and the S blocks of a group fit on the
// device at once (the host checks the occupancy).  Workgroups are dispatched
// in block order on each XCD, so on every XCD the blocks of the lowest row
// group that has not finished are dispatched before any block of a later
// group: if one of them were not yet dispatched, that XCD would hold no block
// of this launch at all and would dispatch it next.  That group therefore
// has all of its blocks resident, completes, and exits, and so on by
// induction, whether the grid is one full residency of the device whose
// groups loop over the rows or one group per row far larger than the device
// (the host's default), and whether or not other work shares the device.
// The wait is bounded regardless: a lane that gives up records the failure
// in the workspace and carries on, so the grid always drains.
#pragma once

#include "rowsm_device.hpp"

namespace rowsm {

// Workspace layout (device memory, zeroed when it is created).
struct SplitWorkspace {
  uint64_t* wm;     // [max_blocks][2]: (tag << 32) | bits(block max)
  uint64_t* ws;     // [max_blocks][2]: (tag << 32) | bits(block sum)
  uint32_t* error;  // [1]: number of waits that gave up
  // Launches recorded under stream capture: the tag base, written by the
  // launch's epoch kernel just before it on every replay (the tag0 argument
  // is then unused); null for eager launches.
  const uint32_t* dtag;
};

// Tag base of a launch: the host's, or a captured launch's from its slice.
__device__ __forceinline__ uint32_t split_tag0(const SplitWorkspace& w, uint32_t tag0) {
  if (w.dtag == nullptr) return tag0;
  return __builtin_amdgcn_readfirstlane(
      __hip_atomic_load(w.dtag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}

// Polls before a wait gives up (about a second at the load latency of an
// agent-scope poll).  A lane that gave up once never waits again in this
// launch, so even a broken exchange lets the whole grid drain quickly.
constexpr uint32_t kSplitSpinLimit = 1u << 20;

// Polls block b's (max, sum) words of the current row (parity slot) until
// both carry the expected tag, and returns the pair.  A lane that gives up
// records it once in the workspace and never waits again in this launch.
__device__ __forceinline__ MaxSum split_poll_pair(const SplitWorkspace& w, uint32_t b,
                                                  uint32_t slot, uint64_t tag, bool* gave_up) {
  const uint32_t i = 2 * b + slot;
  uint64_t vm = 0, vs = 0;
  uint32_t spins = 0;
  while (!*gave_up) {
    vm = __hip_atomic_load(&w.wm[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    vs = __hip_atomic_load(&w.ws[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((vm & ~0xffffffffull) == tag && (vs & ~0xffffffffull) == tag) break;
    __builtin_amdgcn_s_sleep(1);
    if (++spins == kSplitSpinLimit) {
      __hip_atomic_fetch_add(w.error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      *gave_up = true;
    }
  }
  return {__uint_as_float((uint32_t)vm), __uint_as_float((uint32_t)vs)};
}

// The same for a single word per block (the ws words; the softmax backward's
// partial dot products).
__device__ __forceinline__ float split_poll_word(const SplitWorkspace& w, uint32_t b,
                                                 uint32_t slot, uint64_t tag, bool* gave_up) {
  const uint32_t i = 2 * b + slot;
  uint64_t v = 0;
  uint32_t spins = 0;
  while (!*gave_up) {
    v = __hip_atomic_load(&w.ws[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((v & ~0xffffffffull) == tag) break;
    __builtin_amdgcn_s_sleep(1);
    if (++spins == kSplitSpinLimit) {
      __hip_atomic_fetch_add(w.error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      *gave_up = true;
    }
  }
  return __uint_as_float((uint32_t)v);
}

// Loads a block's share of one row (raw), masked as the row's form needs.
template <typename In, int VW, int NV, bool FUSED>
__device__ __forceinline__ void split_load_share(InVec<In, VW> (&v)[NV], rsrc_t rx, uint32_t vin,
                                                 uint32_t sin, int RT, int g, bool last_ok,
                                                 int lim) {
#pragma unroll
  for (int s = 0; s < NV; ++s) {
    if ((s < NV - 1 || last_ok) && (!FUSED || (s * RT + g) * VW <= lim))
      v[s].load(rx, vin, s * sin);
    else
      v[s].set_neg_inf();
  }
}

// PIPE (software pipelining): while a block reduces, exchanges and writes
// row k, the loads of its next row are already in flight, so memory keeps
// streaming through the exchange wait and the write burst (one more raw
// share per lane in registers).
template <typename In, typename Out, int VW, int NV, int MODE, bool PIPE>
__global__ __launch_bounds__(1024) void split_row_kernel(
    const typename In::storage* __restrict__ x, typename Out::storage* __restrict__ y,
    int64_t rows, int cols, int S, SplitWorkspace w, uint32_t tag0, Fused fz) {
  constexpr bool FUSED = MODE == kFused, LOG = MODE == kLog;
  __shared__ float red_m[16];
  __shared__ float red_s[16];
  __shared__ float bcast[3];

  const int T = blockDim.x;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = wave_id();
  const int nwaves = T / kWave;
  const int c = blockIdx.x % S;                 // chunk of the row
  const int q = blockIdx.x / S;                 // row slot
  const int64_t slots = gridDim.x / S;
  const int RT = S * T;
  const int g = c * T + threadIdx.x;
  const int nvec = cols / VW;
  const bool last_ok = (NV - 1) * RT + g < nvec;
  const uint32_t vin = (uint32_t)g * (VW * In::bytes);
  const uint32_t vout = (uint32_t)g * (VW * Out::bytes);
  const uint32_t sin = (uint32_t)RT * (VW * In::bytes);
  const uint32_t sout = (uint32_t)RT * (VW * Out::bytes);
  const float ninf = -__builtin_inff();

  auto row_rsrc = [&](int64_t r) { return make_rsrc(x + r * cols, (uint64_t)cols * In::bytes); };
  auto row_limit = [&](int64_t r) { return FUSED ? fused_limit(fz, r, cols) : cols - 1; };

  tag0 = split_tag0(w, tag0);
  bool gave_up = false;  // per lane of the first wave
  InVec<In, VW> nxt[NV];  // PIPE: the next row's share, in flight
  if constexpr (PIPE) {
    if (q < rows) split_load_share<In, VW, NV, FUSED>(nxt, row_rsrc(q), vin, sin, RT, g, last_ok,
                                                      row_limit(q));
  }
  uint32_t k = 0;
  for (int64_t row = q; row < rows; row += slots, ++k) {
    const rsrc_t ry = make_rsrc(y + row * cols, (uint64_t)cols * Out::bytes);

    const int lim = row_limit(row);
    float f[NV][VW];
    {
      InVec<In, VW> v[NV];
      if constexpr (PIPE) {
#pragma unroll
        for (int s = 0; s < NV; ++s) v[s] = nxt[s];
      } else {
        split_load_share<In, VW, NV, FUSED>(v, row_rsrc(row), vin, sin, RT, g, last_ok, lim);
      }
#pragma unroll
      for (int s = 0; s < NV; ++s) {
        v[s].to_float(f[s]);
        if constexpr (FUSED) fused_apply(f[s], (s * RT + g) * VW, lim, fz.scale);
      }
    }
    if constexpr (PIPE) {
      const int64_t next = row + slots;
      if (next < rows)
        split_load_share<In, VW, NV, FUSED>(nxt, row_rsrc(next), vin, sin, RT, g, last_ok,
                                            row_limit(next));
    }
    if constexpr (FUSED) {
      // Vectors wholly past the limit are zeros whatever the row's max and
      // sum: store them now, overlapping the loads and the exchange.
      float z[VW];
#pragma unroll
      for (int i = 0; i < VW; ++i) z[i] = 0.0f;
#pragma unroll
      for (int s = 0; s < NV; ++s)
        if ((s < NV - 1 || last_ok) && (s * RT + g) * VW > lim)
          store_out<Out, VW>(ry, vout + s * sout, z);
    }

    // Block maximum.
    float mb = ninf;
#pragma unroll
    for (int s = 0; s < NV; ++s)
#pragma unroll
      for (int i = 0; i < VW; ++i) mb = fmax_nn(mb, f[s][i]);
    mb = group_reduce<kWave, MaxOp>(mb);
    if (lane == 0) red_m[wave] = mb;
    __syncthreads();
    mb = red_m[0];
    for (int w = 1; w < nwaves; ++w) mb = fmax_nn(mb, red_m[w]);

    // Block sum relative to the block maximum.
    const float nml = (mb == ninf) ? 0.0f : -mb * kLog2e;
    float sb = 0.0f;
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      if constexpr (LOG) exp_sum_keep(f[s], exp_ref(mb), &sb);
      else exp_accumulate<FUSED>(f[s], nml, (s * RT + g) * VW <= lim, &sb);
    }
    sb = group_reduce<kWave, SumOp>(sb);
    if (lane == 0) red_s[wave] = sb;
    __syncthreads();
    sb = red_s[0];
    for (int w = 1; w < nwaves; ++w) sb += red_s[w];

    // Exchange with the other blocks of the row (first wave only).
    if (wave == 0) {
      const uint32_t b0 = (uint32_t)q * S;
      const uint64_t tag = (uint64_t)(tag0 + k) << 32;
      const uint32_t slot = k & 1;
      if (lane == 0) {
        __hip_atomic_store(&w.wm[2 * (b0 + c) + slot], tag | __float_as_uint(mb),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&w.ws[2 * (b0 + c) + slot], tag | __float_as_uint(sb),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      MaxSum p = {ninf, 0.0f};
      if (lane < S) p = split_poll_pair(w, b0 + lane, slot, tag, &gave_up);
      p = group_merge<kWave>(p);  // fixed lane order: deterministic
      if (lane == 0) {
        // y = exp(x - m_b) * exp(m_b - M) / S
        bcast[0] = exp2_fast((mb - p.m) * kLog2e) * __builtin_amdgcn_rcpf(p.s);
        bcast[1] = (p.s > 0.5f) ? 0.0f : 1.0f;  // row without a normal sum: all NaN
        bcast[2] = p.m;                          // log form: (x - M) - ln(S)
        if (LOG) bcast[0] = ln_fast(p.s);
      }
    }
    __syncthreads();
    const float scale = bcast[0];
    const bool redo_masked = FUSED && bcast[1] != 0.0f;
    const float M = bcast[2];

#pragma unroll
    for (int s = 0; s < NV; ++s) {
#pragma unroll
      for (int i = 0; i < VW; ++i) f[s][i] = LOG ? (f[s][i] - M) - scale : f[s][i] * scale;
      if ((s < NV - 1 || last_ok) && (!FUSED || (s * RT + g) * VW <= lim || redo_masked))
        store_out<Out, VW>(ry, vout + s * sout, f[s]);
    }
    // LDS reuse across rows: red_m is rewritten after this row's last barrier,
    // which every wave passes only after reading red_m (before the second
    // barrier); red_s and bcast are rewritten after the next row's first and
    // second barriers, which every wave reaches only after reading them here.
  }
}

}  // namespace rowsm
