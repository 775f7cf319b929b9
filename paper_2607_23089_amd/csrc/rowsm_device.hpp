// Device building blocks shared by the small-, medium- and large-row softmax
// kernels (gfx950, wave64).
//
//  * element types and up-to-16-byte vector I/O through raw buffer
//    descriptors, non-temporal (every byte of x is read once and every byte
//    of y written once, so neither should displace the other in L2 or the
//    memory-side cache);
//  * exact bf16 -> fp32 widening (bits << 16) and round-to-nearest-even
//    fp32 -> bf16 narrowing (v_cvt_pk_bf16_f32);
//  * all-reduce of max and sum over aligned lane groups of 2..64 lanes with
//    DPP quad permutes and mirrors, then v_permlane16/32_swap;
//  * the online (max, sum) merge used when a row is seen in pieces:
//      (m1, s1) + (m2, s2) = (M, s1 * 2^((m1 - M) log2e) + s2 * 2^((m2 - M) log2e)),
//    M = max(m1, m2), where a piece with s == 0 (no finite entry yet)
//    contributes nothing.
//
// Exponentials are taken as exp2(fma(x, log2e, -m*log2e)) on v_exp_f32.  The
// rounding of m*log2e is one constant factor per row, which cancels in the
// normalisation e / sum(e).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rowsm {

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.44269504088896340736f;
constexpr int kWave = 64;
constexpr int kFlatSlots = 4;  // flat short rows: vectors per lane per tile (flat_row.hpp)

// ---- element types --------------------------------------------------------

struct F32 {
  using storage = float;
  static constexpr int bytes = 4;
  static constexpr uint32_t neg_inf_word = 0xff800000u;  // one element
};
struct BF16 {
  using storage = uint16_t;
  static constexpr int bytes = 2;
  static constexpr uint32_t neg_inf_word = 0xff80ff80u;  // two elements
};

template <int BYTES> struct raw_of;
template <> struct raw_of<16> { using type = u32x4; static constexpr int words = 4; };
template <> struct raw_of<8> { using type = u32x2; static constexpr int words = 2; };
template <> struct raw_of<4> { using type = uint32_t; static constexpr int words = 1; };
template <> struct raw_of<2> { using type = uint16_t; static constexpr int words = 0; };

__device__ __forceinline__ float fmax_nn(float a, float b) {
  // maximumNumber: a NaN operand is ignored.  NaN still reaches the row
  // through exp and the sum, so the max needs no NaN rule of its own; this
  // form also avoids the canonicalising moves that fmaxf costs in IEEE mode.
  return __builtin_elementwise_maximumnum(a, b);
}

__device__ __forceinline__ float exp2_fast(float t) {
  return __builtin_amdgcn_exp2f(t);  // v_exp_f32
}

// ---- buffer addressing ----------------------------------------------------------
//
// Every kernel addresses a row (or a group of rows) through a raw buffer
// descriptor whose base is that row's first byte.  An access is then
// descriptor (scalar registers) + one 32-bit per-lane byte offset (one VGPR
// shared by all the accesses of a lane) + a wave-uniform byte offset (scalar),
// instead of a 64-bit address per access.  The descriptor's record count is
// the byte length of the rows it covers, so the hardware range check is a
// second fence behind the kernels' explicit tail masks.

constexpr int32_t kBufDword3 = 0x00020000;  // gfx9-family raw buffer word 3
// Cache policy bits (gfx950: bit 0 sc0, bit 1 nt, bit 4 sc1).  Loads are
// non-temporal (plain loads halved the medium kernel's rate).  Stores are
// non-temporal at device scope (sc1 nt) when every store of the launch covers
// whole 128-byte lines: that wrote a streaming copy 0.5-1.5% faster than nt
// alone and line-aligned rows 1-4% faster (262144 x 64 and 32768 x 4096
// bf16).  Stores that cover part of a line are non-temporal alone: with sc1
// they took up to 1.8x the launch time (12288 x 4004 fp32 rows 79.5 against
// 65.0 us, one-element bf16 vectors 76 against 41 us, the single-lane edge
// stores of ragged rows 57 against 38 us).
constexpr int kCpolLoad = 2;
constexpr int kCpolStore = 18;      // sc1 nt
constexpr int kCpolStorePart = 2;   // nt

// Whether every store of a launch covers whole 128-byte lines: the output
// starts on a line and each row is a whole number of lines, or a power-of-two
// fraction of one (rows then pack lines whole).
__device__ __forceinline__ bool stores_whole_lines(const void* y, int64_t row_bytes) {
  return ((uintptr_t)y & 127) == 0 &&
         ((row_bytes & 127) == 0 || (row_bytes > 0 && row_bytes < 128 && 128 % row_bytes == 0));
}

typedef __amdgpu_buffer_rsrc_t rsrc_t;

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint64_t bytes) {
  const uint32_t n = bytes > 0xffffffffull ? 0xffffffffu : (uint32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n,
                                           kBufDword3);
}

// A buffer offset past the end of every descriptor of up to 2 GiB.
constexpr uint32_t kOutOfRange = 0x80000000u;

template <int BYTES>
__device__ __forceinline__ typename raw_of<BYTES>::type buf_load(rsrc_t r, uint32_t voff,
                                                                  uint32_t soff) {
  if constexpr (BYTES == 16) return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kCpolLoad);
  else if constexpr (BYTES == 8) return __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, kCpolLoad);
  else if constexpr (BYTES == 4) return __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, kCpolLoad);
  else return __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, kCpolLoad);
}

template <int BYTES, int CPOL>
__device__ __forceinline__ void buf_store_cpol(typename raw_of<BYTES>::type v, rsrc_t r,
                                               uint32_t voff, uint32_t soff) {
  if constexpr (BYTES == 16) __builtin_amdgcn_raw_buffer_store_b128(v, r, voff, soff, CPOL);
  else if constexpr (BYTES == 8) __builtin_amdgcn_raw_buffer_store_b64(v, r, voff, soff, CPOL);
  else if constexpr (BYTES == 4) __builtin_amdgcn_raw_buffer_store_b32(v, r, voff, soff, CPOL);
  else __builtin_amdgcn_raw_buffer_store_b16(v, r, voff, soff, CPOL);
}

// sc1: the launch's stores cover whole lines (stores_whole_lines()).
template <int BYTES>
__device__ __forceinline__ void buf_store(typename raw_of<BYTES>::type v, rsrc_t r,
                                          uint32_t voff, uint32_t soff, bool sc1) {
  if (sc1) buf_store_cpol<BYTES, kCpolStore>(v, r, voff, soff);
  else buf_store_cpol<BYTES, kCpolStorePart>(v, r, voff, soff);
}

__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);  // uniform by construction
}

// A vector of VW input elements, held in its raw (packed) form.
template <typename In, int VW>
struct InVec {
  static constexpr int BYTES = VW * In::bytes;
  using R = typename raw_of<BYTES>::type;
  R r;

  __device__ __forceinline__ void load(rsrc_t rs, uint32_t voff, uint32_t soff) {
    r = buf_load<BYTES>(rs, voff, soff);
  }
  // The vector where ok holds, else -inf.  A 2-byte vector (one bf16) is
  // loaded whatever ok says, from an offset past the descriptor's end where
  // ok fails (out of range: the load reads nothing and returns 0), and the
  // result selected afterwards: inside a branch the compiler widens each such
  // value in the branch and waits for every load before issuing the next,
  // one memory round trip per slot.  Where ok fails the caller's offsets may
  // also fall inside the descriptor (readable memory); nothing else is read.
  __device__ __forceinline__ void load_or_neg_inf(bool ok, rsrc_t rs, uint32_t voff,
                                                  uint32_t soff) {
    if constexpr (BYTES == 2) {
      const R t = buf_load<2>(rs, ok ? voff : kOutOfRange, soff);
      r = ok ? t : (R)0xff80u;
    } else {
      if (ok) load(rs, voff, soff);
      else set_neg_inf();
    }
  }
  __device__ __forceinline__ void set_neg_inf() {
    if constexpr (BYTES == 2) {
      r = (uint16_t)0xff80u;
    } else if constexpr (BYTES == 4) {
      r = In::neg_inf_word;
    } else {
      r = In::neg_inf_word;  // splat to every word
    }
  }
  __device__ __forceinline__ void set_zero() {
    if constexpr (BYTES == 2) {
      r = (uint16_t)0;
    } else {
      r = 0u;  // splat to every word
    }
  }
  __device__ __forceinline__ uint32_t word(int w) const {
    if constexpr (BYTES <= 4) {
      return (uint32_t)r;
    } else {
      return r[w];
    }
  }
  // Element i as fp32 (exact).
  __device__ __forceinline__ float get(int i) const {
    if constexpr (In::bytes == 4) {
      return __uint_as_float(word(i));
    } else if constexpr (BYTES == 2) {
      return __uint_as_float((uint32_t)r << 16);
    } else {
      uint32_t w = word(i >> 1);
      return (i & 1) ? __uint_as_float(w & 0xffff0000u) : __uint_as_float(w << 16);
    }
  }
  // Hide the raw words from the optimiser: values widened before this point
  // cannot be reused after it, so a kernel that keeps the row packed widens it
  // again per phase instead of keeping a second, fp32 copy alive.
  __device__ __forceinline__ void opaque() {
    if constexpr (BYTES <= 4) {
      asm volatile("" : "+v"(r));
    } else {
#pragma unroll
      for (int w = 0; w < raw_of<BYTES>::words; ++w) {
        uint32_t t = r[w];
        asm volatile("" : "+v"(t));
        r[w] = t;
      }
    }
  }
  __device__ __forceinline__ void to_float(float (&f)[VW]) const {
#pragma unroll
    for (int i = 0; i < VW; ++i) f[i] = get(i);
  }
};

// Store VW fp32 values as VW Out elements (VW * Out::bytes bytes, naturally
// aligned up to 16 bytes) at byte offset voff of descriptor rs.
//
// Stores carry their whole offset in the VGPR and a constant 0 in soffset.
// With a register soffset the compiler treats the store's data registers as
// free for the next VALU write without a wait state; on gfx950 that lets the
// write overtake the store's read of its data (seen as raw input values in
// the output).  With a constant soffset the compiler inserts the wait states.
template <typename Out, int VW>
__device__ __forceinline__ void store_out(rsrc_t rs, uint32_t voff, const float (&f)[VW],
                                          bool sc1) {
  constexpr uint32_t soff = 0;
  if constexpr (Out::bytes == 4) {
    if constexpr (VW == 1) {
      buf_store<4>(__float_as_uint(f[0]), rs, voff, soff, sc1);
    } else if constexpr (VW == 2) {
      u32x2 v = {__float_as_uint(f[0]), __float_as_uint(f[1])};
      buf_store<8>(v, rs, voff, soff, sc1);
    } else {
#pragma unroll
      for (int c = 0; c < VW; c += 4) {
        u32x4 v = {__float_as_uint(f[c]), __float_as_uint(f[c + 1]),
                   __float_as_uint(f[c + 2]), __float_as_uint(f[c + 3])};
        buf_store<16>(v, rs, voff + 4u * c, soff, sc1);
      }
    }
  } else {
    if constexpr (VW == 1) {
      buf_store<2>(__builtin_bit_cast(uint16_t, (__bf16)f[0]), rs, voff, soff, sc1);
    } else {
      uint32_t w[VW / 2];
#pragma unroll
      for (int i = 0; i < VW / 2; ++i) {
        f32x2 pr = {f[2 * i], f[2 * i + 1]};
        w[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector(pr, bf16x2));
      }
      if constexpr (VW == 2) {
        buf_store<4>(w[0], rs, voff, soff, sc1);
      } else if constexpr (VW == 4) {
        u32x2 v = {w[0], w[1]};
        buf_store<8>(v, rs, voff, soff, sc1);
      } else {
        u32x4 v = {w[0], w[1], w[2], w[3]};
        buf_store<16>(v, rs, voff, soff, sc1);
      }
    }
  }
}

// ---- cross-lane all-reductions -------------------------------------------

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(
      __builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
struct MaxOp {
  __device__ __forceinline__ static float apply(float a, float b) { return fmax_nn(a, b); }
};
struct SumOp {
  __device__ __forceinline__ static float apply(float a, float b) { return a + b; }
};

// All-reduce over aligned groups of G lanes (G a power of two, 1..64): every
// lane of a group ends with the group's result.  After each step the partial
// result is uniform inside the sub-group reduced so far, so a mirror or a
// row swap only has to pair sub-groups, not lanes.
template <int G, typename Op>
__device__ __forceinline__ float group_reduce(float v) {
  if constexpr (G >= 2) v = Op::apply(v, dpp<0xB1>(v));   // quad_perm [1,0,3,2]
  if constexpr (G >= 4) v = Op::apply(v, dpp<0x4E>(v));   // quad_perm [2,3,0,1]
  if constexpr (G >= 8) v = Op::apply(v, dpp<0x141>(v));  // row_half_mirror
  if constexpr (G >= 16) v = Op::apply(v, dpp<0x140>(v)); // row_mirror
  if constexpr (G >= 32) {
    auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v),
                                              false, false);
    v = Op::apply(__uint_as_float(p[0]), __uint_as_float(p[1]));
  }
  if constexpr (G >= 64) {
    auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v),
                                              false, false);
    v = Op::apply(__uint_as_float(p[0]), __uint_as_float(p[1]));
  }
  return v;
}

// ---- output forms of the forward kernels --------------------------------------
//
//   kPlain  y = softmax(x)
//   kFused  y = softmax(scale * x + causal mask)               (see Fused)
//   kLog    y = log softmax(x) = (x - m) - ln(sum_j exp(x_j - m))
//
// In the log form the exponent is taken as (x - m) * log2e, the difference
// first: softmax may round m * log2e once per row because that factor cancels
// in e / sum(e), but in the log form it would not cancel and would add an
// error proportional to |m|.  The logarithm is v_log_f32 (log2) times ln 2.
enum : int { kPlain = 0, kFused = 1, kLog = 2 };

// Tag of the softmax-backward launches in the launcher tables (the backward
// kernels have no output form of their own).
constexpr int kBackward = 3;
// Tag of the MoE group-score launches.
constexpr int kMoe = 4;

constexpr float kLn2 = 0.69314718055994530942f;

__device__ __forceinline__ float ln_fast(float s) {
  return __builtin_amdgcn_logf(s) * kLn2;  // v_log_f32
}

// Reference point for exponents taken relative to a running maximum m: a
// maximum of -inf (only -inf seen) uses 0, so that exp(-inf - 0) = 0 instead
// of exp(-inf + inf) = NaN.
__device__ __forceinline__ float exp_ref(float m) {
  return m == -__builtin_inff() ? 0.0f : m;
}

// Log form: sum of exp(v - m) over one vector, v left unchanged.
template <int VW>
__device__ __forceinline__ void exp_sum_keep(const float (&v)[VW], float m, float* sum) {
#pragma unroll
  for (int i = 0; i < VW; ++i) *sum += exp2_fast((v[i] - m) * kLog2e);
}

// ---- fused scale and causal mask ---------------------------------------------
//
// The fused variants compute softmax(scale * x + mask) with mask(r, c) = -inf
// for c > (r mod period) + offset (period == 0: no mask).  Columns past a
// row's limit are never loaded: they count as -inf, so they add nothing to
// the sum and their outputs are exactly 0.  The product scale * x is formed
// in fp32.

struct Fused {
  float scale;
  int64_t period;
  int64_t offset;
};

// Last kept column of `row` (inclusive), clamped to [-1, cols - 1].
__device__ __forceinline__ int fused_limit(const Fused& f, int64_t row, int cols) {
  if (f.period <= 0) return cols - 1;
  const int64_t lim = row % f.period + f.offset;
  return lim < -1 ? -1 : (lim > cols - 1 ? cols - 1 : (int)lim);
}

// Columns col0 .. col0 + VW - 1 of one vector: scale the kept ones, -inf the
// rest (their loads were skipped or are beyond the limit).
template <int VW>
__device__ __forceinline__ void fused_apply(float (&v)[VW], int col0, int lim, float scale) {
  if (col0 + VW - 1 <= lim) {  // whole vector kept: the common case
#pragma unroll
    for (int i = 0; i < VW; ++i) v[i] *= scale;
  } else {
#pragma unroll
    for (int i = 0; i < VW; ++i) v[i] = (col0 + i <= lim) ? v[i] * scale : -__builtin_inff();
  }
}

// exp(v - m) for the VW values of one vector, added to *sum.  A fused
// vector wholly past the row's limit holds only -inf: its exponentials are
// exactly 0 and are not evaluated.
template <bool FUSED, int VW>
__device__ __forceinline__ void exp_accumulate(float (&v)[VW], float nml, bool live, float* sum) {
  if (!FUSED || live) {
#pragma unroll
    for (int i = 0; i < VW; ++i) {
      v[i] = exp2_fast(__builtin_fmaf(v[i], kLog2e, nml));
      *sum += v[i];
    }
  } else {
#pragma unroll
    for (int i = 0; i < VW; ++i) v[i] = 0.0f;
  }
}

// ---- online (max, sum) ------------------------------------------------------

// Rescale factor of a partial sum taken relative to max m when the reference
// moves to M >= m.  A partial with s == 0 (only -inf seen) contributes 0.
__device__ __forceinline__ float rescale(float s, float m, float M) {
  return s == 0.0f ? 0.0f : s * exp2_fast((m - M) * kLog2e);
}

struct MaxSum {
  float m, s;
};

__device__ __forceinline__ MaxSum merge(MaxSum a, MaxSum b) {
  float M = fmax_nn(a.m, b.m);
  return {M, rescale(a.s, a.m, M) + rescale(b.s, b.m, M)};
}

template <int G>
__device__ __forceinline__ MaxSum group_merge(MaxSum v) {
  // Reduce the max first, then every lane rescales its own sum to the group
  // max and the sums are added: one exp per lane instead of one per step.
  float M = group_reduce<G, MaxOp>(v.m);
  float s = group_reduce<G, SumOp>(rescale(v.s, v.m, M));
  return {M, s};
}

}  // namespace rowsm
