// MoE group score: for every group of G consecutive expert scores, the sum of
// its two largest values, counted with multiplicity (the paper's running
// example, Motivation section, and the figure of its source rewrite).
//
// The paper rewrites an argmax-and-mask chain into the largest off-diagonal
// pair sum max_{i != j}(v_i + v_j), which it shows equals top1 + top2 with
// ties intact, to get rid of index-producing reductions on its NPU.  On
// gfx950 neither form is needed: the pair (t1, t2) of the two largest values
// seen so far is itself a value-only reduction.  Adding a value v:
//     t1' = max(t1, v),   t2' = max(t2, min(t1, v)),
// and merging two pairs (a1, a2), (b1, b2):
//     (max(a1, b1), max(min(a1, b1), max(a2, b2))),
// which keeps the two largest elements of the union as a multiset (a maximum
// that occurs twice fills both places).  max / min are v_maximum3_f32 /
// v_minimum3_f32, the IEEE maximum and minimum: a NaN anywhere in a group
// makes its score NaN.  Every step is exact, so the result does not depend on
// the reduction order; the sum t1 + t2 is one fp32 addition, then rounded to
// the output type.
//
// Layout (the small-row packing): a group is LPG = G / VW lanes holding one
// VW-element vector each; a wave covers 64 / LPG groups per load instruction
// and RPL such load groups per task, so every lane has RPL independent loads
// in flight before the first reduction.  The pair is reduced across the LPG
// lanes with DPP and permlane steps.  Scores past the last group load nothing
// and hold -inf.  Stores: the task's GPT results are gathered with
// ds_bpermute so that lane q holds the result of the task's group q, and each
// store instruction writes 64 consecutive results (one instruction per task
// when GPT <= 64): whole cache lines instead of one short run per load group.
#pragma once

#include "rowsm_device.hpp"

namespace rowsm {

struct Top2 {
  float t1, t2;
};

__device__ __forceinline__ float ieee_max(float a, float b) {
  return __builtin_elementwise_maximum(a, b);
}
__device__ __forceinline__ float ieee_min(float a, float b) {
  return __builtin_elementwise_minimum(a, b);
}

__device__ __forceinline__ Top2 top2_add(Top2 p, float v) {
  return {ieee_max(p.t1, v), ieee_max(p.t2, ieee_min(p.t1, v))};
}

__device__ __forceinline__ Top2 top2_merge(Top2 a, Top2 b) {
  return {ieee_max(a.t1, b.t1), ieee_max(ieee_min(a.t1, b.t1), ieee_max(a.t2, b.t2))};
}

template <int CTRL>
__device__ __forceinline__ Top2 top2_dpp(Top2 p) {
  return top2_merge(p, {dpp<CTRL>(p.t1), dpp<CTRL>(p.t2)});
}

// All-reduce of the pair over aligned groups of L lanes (L a power of two).
template <int L>
__device__ __forceinline__ Top2 group_top2_reduce(Top2 p) {
  if constexpr (L >= 2) p = top2_dpp<0xB1>(p);   // quad_perm [1,0,3,2]
  if constexpr (L >= 4) p = top2_dpp<0x4E>(p);   // quad_perm [2,3,0,1]
  if constexpr (L >= 8) p = top2_dpp<0x141>(p);  // row_half_mirror
  if constexpr (L >= 16) p = top2_dpp<0x140>(p); // row_mirror
  if constexpr (L >= 32) {
    auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(p.t1), __float_as_uint(p.t1),
                                              false, false);
    auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(p.t2), __float_as_uint(p.t2),
                                              false, false);
    p = top2_merge({__uint_as_float(a[0]), __uint_as_float(b[0])},
                   {__uint_as_float(a[1]), __uint_as_float(b[1])});
  }
  if constexpr (L >= 64) {
    auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(p.t1), __float_as_uint(p.t1),
                                              false, false);
    auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(p.t2), __float_as_uint(p.t2),
                                              false, false);
    p = top2_merge({__uint_as_float(a[0]), __uint_as_float(b[0])},
                   {__uint_as_float(a[1]), __uint_as_float(b[1])});
  }
  return p;
}

template <typename In, typename Out, int VW, int LPG, int RPL>
__global__ __launch_bounds__(256) void group_top2_kernel(
    const typename In::storage* __restrict__ s, typename Out::storage* __restrict__ o,
    int64_t ngroups) {
  constexpr int G = VW * LPG;           // scores per group
  constexpr int GPW = kWave / LPG;      // groups per wave per load instruction
  constexpr int GPT = GPW * RPL;        // groups per wave per task
  const int lane = threadIdx.x & (kWave - 1);
  // (a task's GPT outputs play the part of a row for the store policy)
  const bool wl = stores_whole_lines(o, (int64_t)GPT * Out::bytes);  // sc1 stores
  const int sub = lane % LPG;
  const int grp = lane / LPG;
  const uint32_t vin = (uint32_t)(grp * G + sub * VW) * In::bytes;
  constexpr uint32_t kStepIn = (uint32_t)GPW * G * In::bytes;  // bytes per load group

  const int waves_per_block = blockDim.x / kWave;
  const int64_t wave = (int64_t)blockIdx.x * waves_per_block + wave_id();
  const int64_t nwaves = (int64_t)gridDim.x * waves_per_block;
  const int64_t ntasks = (ngroups + GPT - 1) / GPT;

  for (int64_t task = wave; task < ntasks; task += nwaves) {
    const int64_t g0 = task * GPT;
    const int n = ngroups - g0 < GPT ? (int)(ngroups - g0) : GPT;
    const rsrc_t rs = make_rsrc(s + g0 * G, (uint64_t)n * G * In::bytes);
    const rsrc_t ro = make_rsrc(o + g0, (uint64_t)n * Out::bytes);

    InVec<In, VW> v[RPL];
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      v[k].load_or_neg_inf(k * GPW + grp < n, rs, vin, k * kStepIn);
    }
    Top2 p[RPL];
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      p[k] = {v[k].get(0), -__builtin_inff()};
#pragma unroll
      for (int i = 1; i < VW; ++i) p[k] = top2_add(p[k], v[k].get(i));
    }
#pragma unroll
    for (int k = 0; k < RPL; ++k) p[k] = group_top2_reduce<LPG>(p[k]);
    float r[RPL];
#pragma unroll
    for (int k = 0; k < RPL; ++k) r[k] = p[k].t1 + p[k].t2;
    // Group q of the task is load group q / GPW, held by lanes
    // (q % GPW) * LPG ... + LPG - 1 after the all-reduce.
    constexpr int NSTORE = (GPT + kWave - 1) / kWave;
#pragma unroll
    for (int j = 0; j < NSTORE; ++j) {
      const int q = j * kWave + lane;
      float val;
      if constexpr (LPG == 1) {
        val = r[j];  // GPW == 64: lane q already holds group q of load group j
      } else {
        const int src = (q % GPW) * LPG;
        const int kq = q / GPW;
        val = 0.0f;
#pragma unroll
        for (int k = 0; k < RPL; ++k) {
          const float b = __int_as_float(__builtin_amdgcn_ds_bpermute(src * 4, __float_as_int(r[k])));
          if (kq == k) val = b;
        }
      }
      if (q < n) {
        const float o1[1] = {val};
        store_out<Out, 1>(ro, (uint32_t)q * Out::bytes, o1, wl);
      }
    }
  }
}

}  // namespace rowsm
