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
// Exchange protocol.  A launch owns a region of an exchange workspace: for
// each row group q and parity p (the parity of the number k of rows the
// group's blocks have processed) a run of 2 S 64-bit words, the S max words
// of the blocks followed by their S sum words.  Block c publishes its pair of
// row k with two relaxed agent-scope atomic stores,
//     max[c] = (T << 32) | bits(m_b),   sum[c] = (T << 32) | bits(s_b),
// where the 32-bit tag T = tag0 + k is never 0 and is unique among the tags
// that may meet in one region: the host hands out tags so that no two
// launches that can leave words in the same region share one (a workspace
// sees fewer than 2^32 tags while anything it holds can still be read, and
// regions that cannot guarantee it are cleared before the launch).  A peer
// polls the sum word, then the max word, until each carries T: a 64-bit
// atomic access is indivisible, so a word carrying T holds the right value,
// and no ordering between the two stores, and no cache write-back or
// invalidation, is needed.  Two parities suffice: a block can only rewrite
// parity k & 1 at row k + 2, after every block of its group has published
// row k + 1, i.e. after all of them have read row k's words.
//
// Results never depend on a peer's timing.  A wait that has polled `limit`
// times gives up (the lane counts it in the workspace's failure counter and
// never waits again in this launch), and the whole block then computes the
// missing block's pair itself from that block's share of x, with the same
// lane layout, the same order of operations and the same reductions, so the
// pair is bit-identical to the one the block would have published and the
// row comes out exactly as it would have.  This reads x again, so only
// launches whose x is not overwritten while they run (no in-place launches;
// the host plans in-place calls without exchanging forms) use it.
//
// Forward progress.  The wait is bounded, so every block finishes whatever
// the device runs besides: a group whose blocks are not all resident (held
// out by other work, or dispatched out of order) costs time, not results.
// In the common case the S blocks of a group are resident together (the host
// checks the occupancy, and workgroups are dispatched in block order on each
// XCD), and waits end within microseconds.
#pragma once

#include "rowsm_device.hpp"

namespace rowsm {

// A launch's part of an exchange workspace (device memory).
struct SplitWorkspace {
  uint64_t* words;  // the launch's region: 4 words per block (2 parities x max, sum)
  uint32_t* error;  // [1]: number of waits that gave up
  uint32_t limit;   // polls a wait makes before it gives up
};

constexpr uint64_t kTagMask = 0xffffffff00000000ull;

// The 2 S words of row group q at parity p.
__device__ __forceinline__ uint64_t* split_group_words(const SplitWorkspace& w, int64_t q,
                                                       uint32_t parity, int S) {
  return w.words + ((uint64_t)q * 2 + parity) * 2 * (uint64_t)S;
}

// Publishes block c's two values (a, b) under tag T.
__device__ __forceinline__ void split_publish(uint64_t* gw, int S, int c, uint32_t T, float a,
                                              float b) {
  const uint64_t tag = (uint64_t)T << 32;
  __hip_atomic_store(&gw[c], tag | __float_as_uint(a), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(&gw[S + c], tag | __float_as_uint(b), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}

// Polls block b's words of tag T; true with (*a, *c) once both carry T,
// false when `limit` polls found them unpublished (or when this lane already
// gave up once in this launch).  A lane that gives up counts it in the
// workspace, once.
__device__ __forceinline__ bool split_poll(const SplitWorkspace& w, const uint64_t* gw, int S,
                                           int b, uint32_t T, bool* gave_up, float* a, float* c) {
  if (*gave_up) return false;
  const uint64_t want = (uint64_t)T << 32;
  bool have_sum = false;
  uint64_t sum = 0;
  for (uint32_t n = 0; n < w.limit; ++n) {
    if (!have_sum) {
      sum = __hip_atomic_load(&gw[S + b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      have_sum = (sum & kTagMask) == want;
    }
    if (have_sum) {
      const uint64_t mx = __hip_atomic_load(&gw[b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if ((mx & kTagMask) == want) {
        *a = __uint_as_float((uint32_t)mx);
        *c = __uint_as_float((uint32_t)sum);
        return true;
      }
    }
    __builtin_amdgcn_s_sleep(2);
  }
  __hip_atomic_fetch_add(w.error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  *gave_up = true;
  return false;
}

// Lanes of wave 0 whose peer's words did not arrive (a 64-bit ballot).
__device__ __forceinline__ uint64_t lanes_missing(bool ok) {
  return __builtin_amdgcn_ballot_w64(!ok);
}

// Loads a block's share of one row (raw), masked as the row's form needs.
template <typename In, int VW, int NV, bool FUSED>
__device__ __forceinline__ void split_load_share(InVec<In, VW> (&v)[NV], rsrc_t rx, uint32_t vin,
                                                 uint32_t sin, int RT, int g, bool last_ok,
                                                 int lim) {
#pragma unroll
  for (int s = 0; s < NV; ++s) {
    v[s].load_or_neg_inf((s < NV - 1 || last_ok) && (!FUSED || (s * RT + g) * VW <= lim), rx,
                         vin, s * sin);
  }
}

// Slot s of global thread g as fp32: loaded, widened and (fused form) scaled
// and masked, exactly as the kernel's own share is.
template <typename In, int VW, int NV, bool FUSED>
__device__ __forceinline__ void split_slot_values(float (&f)[VW], rsrc_t rx, int s, int RT, int g,
                                                  bool last_ok, int lim, float scale) {
  InVec<In, VW> v;
  v.load_or_neg_inf((s < NV - 1 || last_ok) && (!FUSED || (s * RT + g) * VW <= lim), rx,
                    (uint32_t)g * (VW * In::bytes), (uint32_t)(s * RT) * (VW * In::bytes));
  v.to_float(f);
  if constexpr (FUSED) fused_apply(f, (s * RT + g) * VW, lim, scale);
}

// Block-wide maximum and sum of the per-lane values (wave reduction, then the
// waves' results in wave order through red[]; two barriers).  The same code
// reduces a block's own share and a share recomputed for a peer.
__device__ __forceinline__ float block_max(float v, float* red, int lane, int wave, int nwaves) {
  v = group_reduce<kWave, MaxOp>(v);
  if (lane == 0) red[wave] = v;
  __syncthreads();
  v = red[0];
  for (int w = 1; w < nwaves; ++w) v = fmax_nn(v, red[w]);
  return v;
}
__device__ __forceinline__ float block_sum(float v, float* red, int lane, int wave, int nwaves) {
  v = group_reduce<kWave, SumOp>(v);
  if (lane == 0) red[wave] = v;
  __syncthreads();
  v = red[0];
  for (int w = 1; w < nwaves; ++w) v += red[w];
  return v;
}

// Exponent offset of the sum relative to a block maximum mb (0 for a block
// of only -inf, so that exp(-inf - 0) = 0).
__device__ __forceinline__ float split_nml(float mb) {
  return mb == -__builtin_inff() ? 0.0f : -mb * kLog2e;
}

// The (m_b, s_b) pair that block c of the row would publish, computed by the
// calling block from c's share of the row (global threads g = c * T + t): the
// same loads, lane order, reductions and exponentials as the kernel's own
// share, hence the same bits.  x is read twice (maximum, then sum), one slot
// at a time.  Every thread of the block calls it.
template <typename In, int VW, int NV, int MODE>
__device__ __forceinline__ MaxSum split_share_pair(rsrc_t rx, int cols, int g, int RT, int lim,
                                                   float scale, float* red_m, float* red_s,
                                                   int lane, int wave, int nwaves) {
  constexpr bool FUSED = MODE == kFused, LOG = MODE == kLog;
  const int nvec = cols / VW;
  const bool last_ok = (NV - 1) * RT + g < nvec;
  float mb = -__builtin_inff();
#pragma unroll 1
  for (int s = 0; s < NV; ++s) {
    float f[VW];
    split_slot_values<In, VW, NV, FUSED>(f, rx, s, RT, g, last_ok, lim, scale);
#pragma unroll
    for (int i = 0; i < VW; ++i) mb = fmax_nn(mb, f[i]);
  }
  mb = block_max(mb, red_m, lane, wave, nwaves);
  const float nml = split_nml(mb);
  float sb = 0.0f;
#pragma unroll 1
  for (int s = 0; s < NV; ++s) {
    float f[VW];
    split_slot_values<In, VW, NV, FUSED>(f, rx, s, RT, g, last_ok, lim, scale);
    if constexpr (LOG) exp_sum_keep(f, exp_ref(mb), &sb);
    else exp_accumulate<FUSED>(f, nml, (s * RT + g) * VW <= lim, &sb);
  }
  sb = block_sum(sb, red_s, lane, wave, nwaves);
  return {mb, sb};
}

// PIPE (software pipelining): while a block reduces, exchanges and writes
// row k, the loads of its next row are already in flight, so memory keeps
// streaming through the exchange wait and the write burst (one more raw
// share per lane in registers).
template <typename In, typename Out, int VW, int NV, int MODE, bool PIPE>
__global__ __launch_bounds__(1024) void split_row_kernel(
    const typename In::storage* x, typename Out::storage* y, int64_t rows, int cols, int S,
    SplitWorkspace w, uint32_t tag0, Fused fz) {
  constexpr bool FUSED = MODE == kFused, LOG = MODE == kLog;
  __shared__ float red_m[16];
  __shared__ float red_s[16];
  __shared__ float bcast[3];
  __shared__ uint64_t missing_lanes;
  __shared__ MaxSum peer[kWave];  // the row's pairs, when a wait gave up

  const int T = blockDim.x;
  const int lane = threadIdx.x & (kWave - 1);
  const bool wl = stores_whole_lines(y, (int64_t)cols * Out::bytes);  // sc1 stores
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
          store_out<Out, VW>(ry, vout + s * sout, z, wl);
    }

    // Block maximum, then the block sum relative to it (split_share_pair()
    // repeats exactly these steps for a peer's share).
    float mb = ninf;
#pragma unroll
    for (int s = 0; s < NV; ++s)
#pragma unroll
      for (int i = 0; i < VW; ++i) mb = fmax_nn(mb, f[s][i]);
    mb = block_max(mb, red_m, lane, wave, nwaves);
    const float nml = split_nml(mb);
    float sb = 0.0f;
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      if constexpr (LOG) exp_sum_keep(f[s], exp_ref(mb), &sb);
      else exp_accumulate<FUSED>(f[s], nml, (s * RT + g) * VW <= lim, &sb);
    }
    sb = block_sum(sb, red_s, lane, wave, nwaves);

    // Exchange with the other blocks of the row (first wave: lane b holds
    // block b's pair).  When no wait gave up, wave 0 merges right away.
    // Otherwise wave 0 parks the pairs it has in LDS and the block recomputes
    // the missing ones (one slot at a time, next to the share it holds).
    auto finish = [&](MaxSum pr) {
      pr = group_merge<kWave>(pr);  // fixed lane order: deterministic
      if (lane == 0) {
        // y = exp(x - m_b) * exp(m_b - M) / S
        bcast[0] = exp2_fast((mb - pr.m) * kLog2e) * __builtin_amdgcn_rcpf(pr.s);
        bcast[1] = (pr.s > 0.5f) ? 0.0f : 1.0f;  // row without a normal sum: all NaN
        bcast[2] = pr.m;                          // log form: (x - M) - ln(S)
        if (LOG) bcast[0] = ln_fast(pr.s);
      }
    };
    if (wave == 0) {
      const uint32_t tag = tag0 + k;
      uint64_t* gw = split_group_words(w, q, k & 1, S);
      if (lane == 0 && S > 1) split_publish(gw, S, c, tag, mb, sb);
      MaxSum p = {ninf, 0.0f};
      bool ok = true;
      if (lane == c) p = {mb, sb};
      else if (lane < S) ok = split_poll(w, gw, S, lane, tag, &gave_up, &p.m, &p.s);
      const uint64_t missing = lanes_missing(ok);
      if (lane == 0) missing_lanes = missing;
      if (missing == 0) finish(p);
      else peer[lane] = p;
    }
    __syncthreads();
    const uint64_t missing = missing_lanes;
    if (missing != 0) {
      const rsrc_t rx = row_rsrc(row);
      for (uint64_t mm = missing; mm != 0; mm &= mm - 1) {
        const int b = __builtin_ctzll(mm);
        const MaxSum r = split_share_pair<In, VW, NV, MODE>(rx, cols, b * T + threadIdx.x, RT,
                                                            lim, fz.scale, red_m, red_s, lane,
                                                            wave, nwaves);
        if (threadIdx.x == 0) peer[b] = r;
      }
      __syncthreads();
      if (wave == 0) finish(peer[lane]);
      __syncthreads();
    }
    const float scale = bcast[0];
    const bool redo_masked = FUSED && bcast[1] != 0.0f;
    const float M = bcast[2];

#pragma unroll
    for (int s = 0; s < NV; ++s) {
#pragma unroll
      for (int i = 0; i < VW; ++i) f[s][i] = LOG ? (f[s][i] - M) - scale : f[s][i] * scale;
      if ((s < NV - 1 || last_ok) && (!FUSED || (s * RT + g) * VW <= lim || redo_masked))
        store_out<Out, VW>(ry, vout + s * sout, f[s], wl);
    }
    // LDS reuse across rows: red_m and red_s are rewritten only after a
    // barrier that every wave reaches after reading them (the next reduction's
    // barrier, or a recomputation's); bcast, missing_lanes and peer are
    // rewritten by wave 0 after the next row's two reduction barriers, which
    // every wave passes only after reading them here.
  }
}

}  // namespace rowsm
