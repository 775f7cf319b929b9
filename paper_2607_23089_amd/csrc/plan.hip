// Launch planning of the row-softmax library: the row-length and row-count
// launcher that picks a kernel family and its launch shape for each
// operation (plan.hpp declares what the dispatch and the C ABI call).
//
// The launcher mirrors the structure the paper names for its running example
// (small-, medium- and large-row kernels selected by a row launcher, preamble
// listing style).  Its thresholds are this library's, stated in plan_for():
//   SMALL   a row is at most 32 vectors (one vector per lane, >= 2 rows per wave)
//   MEDIUM  the row fits the registers of at most 16 waves
//           (<= 64 fp32 values per lane, or <= 24 raw 16-byte bf16 vectors
//           per lane in the packed form)
//   LARGE   anything longer: the row split over S <= 64 co-resident blocks
//           that each hold their share in registers (single read), or, for
//           rows too long even for that, two streaming passes over tiles
//           (several blocks per row for few rows, stream_blocks()).
// Rows of 129-4096 vectors in launches of at least 32 rows per compute unit
// take measured launch shapes (medium or single-read, measured_row_shape()
// and, for the fused form with fp32 output, measured_fused_shape()).
// Row count: a launch of few rows must still fill the device, so fewer than
// cus/4 rows of >= 384 KiB each (at most cus/4 rows for the packed form) take
// the split form rather than one block per row, and the split form gives
// each of fewer than cus rows up to cus/rows blocks (few_rows_split()).
#include <hip/hip_runtime.h>

#include <atomic>

#include "plan.hpp"

namespace rowsm {
namespace {

std::atomic<int> g_cu_count[kMaxDevices];

}  // namespace

// Compute-unit count of the current device (cached per device).  Falls back
// to 256, the MI355X count, when no device can be queried.
int cu_count() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
  int n = g_cu_count[dev].load(std::memory_order_relaxed);
  if (n > 0) return n;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      n <= 0)
    n = 256;
  g_cu_count[dev].store(n, std::memory_order_relaxed);
  return n;
}

int dtype_bytes(int dt) { return dt == ROWSM_F32 ? 4 : 2; }
bool dtype_ok(int dt) { return dt == ROWSM_F32 || dt == ROWSM_BF16; }

namespace {

int next_pow2(int v) {
  int p = 1;
  while (p < v) p <<= 1;
  return p;
}


// Vector widths (elements) with compiled kernels: 16-byte and 8-byte input
// vectors, and single elements for rows that are not 8-byte aligned.
bool vw_supported(int vw, int ib) { return vw == 1 || vw * ib == 16 || vw * ib == 8; }

// Largest supported vector width that divides cols and keeps both the x and
// the y accesses naturally aligned, with at most 16 bytes on either side: a
// lane's output vector then never exceeds one 16-byte store, so each store
// instruction of a wave writes one contiguous stretch of whole cache lines.
int choose_vw(int64_t cols, int ib, int ob, uintptr_t xa, uintptr_t ya) {
  for (int vw = 16 / (ib > ob ? ib : ob); vw > 1; vw >>= 1) {
    if (!vw_supported(vw, ib)) continue;
    const int xal = vw * ib;
    const int yal = vw * ob < 16 ? vw * ob : 16;
    if (cols % vw == 0 && xa % xal == 0 && ya % yal == 0) return vw;
  }
  return 1;
}

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Grid limit of the small, medium and MoE families: one task (row group) per
// wave or block up to 2^30 blocks, the waves striding over any tasks beyond
// that; cfg->blocks_per_cu caps the grid at that many blocks per compute unit.
// Grid-stride loops over a capped grid measured 4-8% slower at 1-4 M rows
// (and slower still in plain store streams): waves that drift apart spread
// the addresses in flight over the whole buffer, while the in-order blocks
// of an uncapped grid keep them in one moving window.  (Medium rows of one
// wave and up to four slots per lane, and small rows of narrow vectors whose
// stores cover parts of lines, are the exception: looping_grid().)
int64_t grid_cap(int bpc, int cus) {
  return bpc ? (int64_t)cus * bpc : ((int64_t)1 << 30);
}

// Vectors per lane of a flat tile (flat_row.hpp): cfg->rows_per_lane when
// given (4, or 2 for bf16 to bf16 rows that fit such a tile), else 2 for
// such rows when two_default, else 4; 0 for a value the form cannot take.
int flat_slots(const rowsm_config* cfg, int ib, int ob, int64_t cols, int vw_full,
               bool two_default) {
  const bool fits2 = ib == 2 && ob == 2 && cols <= 2 * (int64_t)kWave * vw_full - (vw_full - 1);
  const int want = cfg ? cfg->rows_per_lane : 0;
  if (want == 0) return two_default && fits2 ? 2 : kFlatSlots;
  if (want == kFlatSlots || (want == 2 && fits2)) return want;
  return 0;
}

// Lanes per row and elements per lane of a flat plan's row phase: the
// launcher's LPR = the power of two >= cols / 8, within 8..64, and 4 for
// rows of 9-16 columns, or cfg->lanes_per_row when given; E the power of
// two >= cols / LPR, at least 2.  False for a pair launch_flat.hpp does not
// compile.  (Forced row shapes of 1-8 lanes at 9-29 columns, every dtype
// pair, softmax and backward, 64 and 384 MiB: 4 lanes took 0.97x the time
// of 8 on geometric mean at 9-15 columns, 0.86-0.95x at 9 bf16 columns,
// and 0.99x at 21-29; 1 and 2 lanes were fastest only here and there.)
bool flat_row_shape(const rowsm_config* cfg, int64_t cols, int* lpr_out, int* e_out) {
  int lpr = (int)next_pow2((int)cdiv(cols, 8));
  if (lpr < 8) lpr = cols > 8 && cols <= 16 ? 4 : 8;
  if (lpr > kWave) lpr = kWave;
  if (cfg && cfg->lanes_per_row > 0) lpr = cfg->lanes_per_row;
  int e = (int)next_pow2((int)cdiv(cols, lpr));
  if (e < 2) e = 2;
  *lpr_out = lpr;
  *e_out = e;
  switch (lpr) {
    case 4: return e == 4;
    case 8: return e == 2 || e == 4 || e == 8;
    case 16: case 32: return e == 8;
    case 64: return e == 8 || e == 16;
    default: return false;
  }
}

bool medium_unpacked_cap(int vw, int vpl) { return vpl * vw <= 64 && vpl <= 16; }

// Host form of the kernels' stores_whole_lines(): every store of a launch
// covers whole 128-byte lines (the output starts on a line, and a row is a
// whole number of lines or a power-of-two fraction of one).  Such launches
// store with the device-scope bit; the others without it.
bool whole_lines(uintptr_t y, int64_t row_bytes) {
  return (y & 127) == 0 &&
         ((row_bytes & 127) == 0 || (row_bytes > 0 && row_bytes < 128 && 128 % row_bytes == 0));
}

// Launches of short rows whose waves each take few bytes: a grid of about
// one block per `per_block` bytes of traffic, rounded to whole residencies
// (the blocks of `block` threads that fit the compute units at once, 2048
// threads per compute unit), at least one residency and at most the
// uncapped grid (and `max_per_cu` blocks per compute unit when given), each
// block looping over its rows.  Sweeps of one-wave medium rows (33-242
// vectors of one element, half and full width, rows of whole 128-byte lines
// and of parts of lines) and small rows of 11-29 one-element columns, every
// dtype pair, 32 MiB-2 GiB, grids of 4-128 blocks per compute unit, each
// launch alone after a cache-evicting write: the best grid grows with the
// launch (4 blocks per compute unit at 32-64 MiB, 64-128 at 1-2 GiB) and a
// fixed traffic per block tracks it.  Forward one-wave medium rows of one
// to four slots: 32 KiB, 1.4-1.8% above the fastest grid measured on
// geometric mean over four sweeps where the earlier rules (one residency
// of 4 blocks per compute unit for up to 8 input bytes per lane, one-wave
// blocks for same-width rows of one full slot, a block per 8 rows
// otherwise) took 3.4-7.7%.  Forward small rows of narrow vectors whose
// stores cover parts of lines: 16 KiB, at most 128 blocks per compute unit
// (0.9-2.7% against 5.8-17%).  Backward one-wave medium rows of one to four
// slots: 24 KiB of the three streams (1.7-2.3% against 2.3-11%).  A grid of
// 2049 blocks of 512 threads left one block to run alone after two full
// residencies and measured 9% slower than 2048.  (rows / (per_block /
// row_bytes): no product of rows and row bytes is formed.)
int64_t looping_grid(int64_t rows, int64_t row_bytes, int64_t per_block, int64_t dflt,
                       int block, int cus, int max_per_cu = 0) {
  const int64_t rpb = per_block / row_bytes > 1 ? per_block / row_bytes : 1;
  const int64_t unit = (int64_t)cus * (2048 / block > 1 ? 2048 / block : 1);
  int64_t g = (cdiv(rows, rpb) + unit / 2) / unit * unit;
  if (g < unit) g = unit;
  if (max_per_cu > 0 && g > (int64_t)max_per_cu * cus) g = (int64_t)max_per_cu * cus;
  return g < dflt ? g : dflt;
}

// Block size of the small-row and MoE kernels (whose waves work on their own
// rows): 256 threads, or cfg->block when given, at most 256.
int small_block(const rowsm_config* cfg, int* block) {
  *block = 256;
  if (cfg && cfg->block > 0) {
    if (cfg->block > 256) return ROWSM_EINVAL;
    *block = cfg->block;
  }
  return ROWSM_OK;
}

bool pow2_upto(int v, int hi) { return v >= 1 && v <= hi && (v & (v - 1)) == 0; }

// Every override must lie in its documented domain, whichever family or form
// ends up being used.
bool config_in_domain(const rowsm_config* c) {
  if (!c) return true;
  return c->variant >= ROWSM_AUTO && c->variant <= ROWSM_LARGE && c->vw >= 0 &&
         (c->lanes_per_row == 0 || pow2_upto(c->lanes_per_row, 32)) &&
         (c->rows_per_lane == 0 || pow2_upto(c->rows_per_lane, 8)) &&
         (c->waves_per_row == 0 || pow2_upto(c->waves_per_row, 16)) &&
         c->rows_per_block >= 0 && c->rows_per_block <= 16 &&
         c->packed >= -1 && c->packed <= 1 &&
         c->block >= 0 && c->block <= 1024 && c->block % kWave == 0 &&
         (c->tile_vectors == 0 || c->tile_vectors == 2 || c->tile_vectors == 4 ||
          c->tile_vectors == 8) &&
         c->blocks_per_cu >= 0 && c->split_blocks >= -1 && c->split_blocks <= 64 &&
         c->prefetch >= -1 && c->prefetch <= 1;
}

// Row-count rules, from a sweep of 1-128 rows x 4096-262144 columns in every
// dtype pair (cold caches): below ~384 KiB of traffic per row every form sits
// at the launch floor; above it, a block per row on fewer than a quarter of
// the compute units loses up to 17% to the split form (the packed bf16 form
// up to 1.8x, still 1.4x at a quarter), and the split form is fastest with
// about one block per compute unit over the launch.
// The backward moves three streams per element and gains from splitting from
// 512 KiB of traffic per row on.
constexpr int64_t kFewRowsMinBytes = 384 * 1024;
constexpr int64_t kFewRowsMinBytesBackward = 512 * 1024;
bool few_long_rows(int64_t rows, int64_t row_bytes, bool packed, int cus,
                   int64_t min_bytes = kFewRowsMinBytes) {
  return row_bytes >= min_bytes && (packed ? rows <= cus / 4 : rows < cus / 4);
}

// Launch shape of a forward row of 129-4096 full 16-byte vectors in a launch
// of at least 32 rows per compute unit (softmax and log forms): a medium
// group of wpr waves with rpb rows per block (S == 0), or the single-read
// form with S blocks of T threads per row.  From sweeps of 1024-16384
// columns in every dtype pair (8192-262144 rows, launches timed alone after
// a cache-evicting write, two boxes agreeing within 1.5%): the medium form
// is fastest with two to four vectors per lane and one or two rows per
// block, rows of more than about 1280 vectors in the single-read form with
// 512 threads per row; rows that widen (bf16 -> fp32) or narrow
// (fp32 -> bf16) keep the medium form longer.  At the fitted lengths the
// picks are within 3% of the fastest form measured (the previous rule, at
// most 16 fp32 values per lane in 512-thread blocks, up to 24% slower), and
// 1.5% above it on geometric mean at 44 lengths the table was not fitted to
// (the previous rule 5.8%, at most 55%).  The form that wins changes with
// the length in ways no count of slots or bytes per lane predicts (the
// medium and the single-read kernel at the same geometry differ by up to
// 20% either way), hence a table.  Smaller launches keep the previous rule:
// at 8-16 rows per compute unit fewer waves per row measured fastest.
// Widening rows continue to 8192 vectors.  The single-read picks beyond 1280
// vectors were re-measured after the row stores became non-temporal at
// device scope, at 8192, 16384 and 32768 rows of 1536-8192 vectors on three
// boxes (206 launches): the best shape there depends on the row count as
// well (e.g. 2048-vector fp32 rows: one 512-thread block level with two
// 256-thread blocks at 8192 rows, 12% slower at 32768), so each entry is the
// shape with the lowest mean slowdown over the three counts.  The previous
// picks were 1.5% above the fastest shape on geometric mean there (at most
// 13%), these 0.5% (at most 5%); at 60 launches of other lengths and row
// counts (12288 and 24576 rows) 1.6% and 0.6%.
struct RowShape {
  int wpr = 0, rpb = 0, S = 0, T = 0;
};
bool measured_row_shape(int64_t nvec, int ib, int ob, RowShape* r) {
  const bool widen = ob > ib;
  if (nvec <= 128 || nvec > (widen ? 8192 : 4096)) return false;
  struct Row {
    int upto, wpr, rpb, S, T;
  };
  // {longest row (vectors), wpr, rpb, S, T}
  static constexpr Row kSameF32[] = {{256, 2, 1, 0, 0},    {320, 4, 1, 0, 0},
                                     {512, 4, 2, 0, 0},    {640, 4, 1, 0, 0},
                                     {1280, 8, 1, 0, 0},   {1920, 0, 0, 1, 512},
                                     {3584, 0, 0, 2, 256}, {4096, 0, 0, 2, 512}};
  static constexpr Row kSameBf16[] = {{256, 2, 1, 0, 0},    {320, 4, 1, 0, 0},
                                      {512, 4, 2, 0, 0},    {640, 4, 1, 0, 0},
                                      {1280, 8, 1, 0, 0},   {1920, 0, 0, 1, 512},
                                      {3840, 0, 0, 2, 256}, {4096, 0, 0, 4, 256}};
  static constexpr Row kWiden[] = {{256, 2, 1, 0, 0},    {512, 4, 1, 0, 0},
                                   {896, 4, 2, 0, 0},    {1792, 8, 1, 0, 0},
                                   {2432, 0, 0, 1, 512}, {4608, 0, 0, 2, 256},
                                   {8192, 0, 0, 2, 512}};
  static constexpr Row kNarrow[] = {{256, 2, 1, 0, 0},   {768, 4, 1, 0, 0},
                                    {1024, 4, 2, 0, 0},  {1664, 8, 1, 0, 0},
                                    {2816, 0, 0, 1, 512}, {4096, 0, 0, 2, 256}};
  const Row* t = ib == ob ? (ib == 2 ? kSameBf16 : kSameF32) : (widen ? kWiden : kNarrow);
  while (nvec > t->upto) ++t;
  r->wpr = t->wpr;
  r->rpb = t->rpb;
  r->S = t->S;
  r->T = t->T;
  return true;
}

// The same for the fused scale + causal mask form with fp32 output (fp32 or
// bf16 input; the fused form writes every output entry but reads only the
// kept ones, so its traffic leans to writes): the medium form with two to
// five vectors per lane, wave groups growing with the row, and the
// single-read form with 512 threads per row beyond 3072 vectors.  From
// sweeps of 1024-16384-column causal heads (16384-262144 rows, every launch
// timed alone after a cache-evicting write): 0.5% above the fastest form
// measured on geometric mean (at most 3.4%), where the rule of at most 32
// values per lane was 11% above it (at most 22%); 0.7% at lengths held out
// of the fp32 fit (the rule 6%, at most 18%), and 2.2% (at most 9%) at a
// third set of lengths, where the rule was about 4.5% above it (at most
// 13%).  Fused rows with bf16 output
// keep that rule, which was within 3.5% of the fastest form at every length.
bool measured_fused_shape(int64_t nvec, int ib, int ob, RowShape* r) {
  if (ob != 4 || nvec <= 128 || nvec > 4096) return false;
  struct Row {
    int upto, wpr, rpb, S, T;
  };
  static constexpr Row kF32[] = {{256, 2, 1, 0, 0},    {1024, 4, 1, 0, 0},
                                 {2048, 8, 1, 0, 0},   {3072, 16, 1, 0, 0},
                                 {4096, 0, 0, 2, 256}};
  static constexpr Row kWiden[] = {{256, 2, 2, 0, 0},   {512, 2, 1, 0, 0},
                                   {1280, 4, 1, 0, 0},  {2560, 8, 1, 0, 0},
                                   {3072, 16, 1, 0, 0}, {4096, 0, 0, 2, 256}};
  const Row* t = ib == 4 ? kF32 : kWiden;
  while (nvec > t->upto) ++t;
  r->wpr = t->wpr;
  r->rpb = t->rpb;
  r->S = t->S;
  r->T = t->T;
  return true;
}

// The same for the softmax backward (y and dy read, dx written): rows of
// 129-4096 full 16-byte vectors in launches of at least 32 rows per compute
// unit.  The medium form for short rows, the single-read form with one
// block of 256 or 512 threads per row from about 300 vectors (fp32 input,
// or bf16 of one width) and two to four blocks per row from about 1400-2700;
// widening rows (bf16 -> fp32) stay in the medium form throughout.  From
// sweeps of 144-4096 vectors in every dtype pair (56 lengths, two row counts
// each between 8192 and 131072 rows, every launch timed alone after a
// cache-evicting write), each entry the shape with the lowest mean slowdown
// over its lengths, an entry of one length only where it gains several
// percent: 0.4-0.7% above the fastest shape measured on geometric mean per
// dtype pair, where the register-cap rule below was 2.3-4.2% (at most 16%).
// Fitted with each length left out in turn and judged on it: 0.7-1.3% (at
// most 11-13%).  At 21 further lengths used in no fit (149 launches of
// 9216 and 18432 rows): 1.3% above the fastest shape (at most 8.6%), the
// register-cap rule 2.9% (at most 10.1%).
bool measured_backward_shape(int64_t nvec, int ib, int ob, RowShape* r) {
  if (nvec <= 128 || nvec > 4096) return false;
  struct Row {
    int upto, wpr, rpb, S, T;
  };
  // {longest row (vectors), wpr, rpb, S, T}
  static constexpr Row kSameF32[] = {{280, 4, 1, 0, 0},    {432, 0, 0, 1, 256},
                                     {608, 8, 1, 0, 0},    {1312, 0, 0, 1, 512},
                                     {2624, 0, 0, 2, 256}, {4096, 0, 0, 2, 512}};
  static constexpr Row kSameBf16[] = {{168, 2, 1, 0, 0},    {304, 4, 1, 0, 0},
                                      {408, 0, 0, 1, 256},  {736, 8, 1, 0, 0},
                                      {1376, 0, 0, 1, 512}, {1632, 16, 1, 0, 0},
                                      {2112, 0, 0, 2, 256}, {3392, 0, 0, 2, 512},
                                      {4096, 0, 0, 4, 256}};
  static constexpr Row kWiden[] = {{264, 2, 1, 0, 0},  {432, 4, 1, 0, 0},
                                   {608, 4, 2, 0, 0},  {1216, 8, 1, 0, 0},
                                   {2240, 4, 1, 0, 0}, {4096, 16, 1, 0, 0}};
  static constexpr Row kNarrow[] = {{168, 2, 2, 0, 0},    {304, 4, 1, 0, 0},
                                    {432, 0, 0, 1, 256},  {608, 8, 1, 0, 0},
                                    {1120, 0, 0, 1, 512}, {1376, 8, 2, 0, 0},
                                    {2752, 0, 0, 2, 256}, {4096, 0, 0, 2, 512}};
  const bool widen = ob > ib;
  const Row* t = ib == ob ? (ib == 2 ? kSameBf16 : kSameF32) : (widen ? kWiden : kNarrow);
  while (nvec > t->upto) ++t;
  r->wpr = t->wpr;
  r->rpb = t->rpb;
  r->S = t->S;
  r->T = t->T;
  return true;
}

// Blocks per row for a split launch of fewer than cus rows with T-thread
// blocks holding at most nv_cap vectors per thread: about one block per
// compute unit over the launch (the largest power of two with rows * S <=
// cus), at least 8, and at most what gives every thread two vectors (smaller
// blocks measured slower); raised to the power of two that the register cap
// needs.  0 when rows >= cus, or when the result exceeds 64 blocks per row or
// 4 blocks per compute unit over the launch (a register-limited plan with
// fewer, larger blocks then measured faster).
int few_rows_split(int64_t rows, int64_t nvec, int T, int nv_cap, int cus) {
  if (rows >= cus) return 0;
  int sf = 1;
  while (sf < 64 && rows * (sf * 2) <= cus) sf *= 2;
  if (sf < 8) sf = 8;
  while (sf > 1 && (int64_t)sf * T * 2 > nvec) sf >>= 1;
  while ((int64_t)sf * T * nv_cap < nvec) sf *= 2;  // register cap
  if (sf > 64 || rows * sf > 4 * (int64_t)cus) return 0;
  return sf;
}

// Blocks per row of the two-pass LARGE form: 1 for launches of at least
// 2 * cus rows, or with a grid capped per compute unit (bpc); otherwise the
// power of two that gives the launch about two blocks per compute unit, at
// most kStreamMaxSplit and the compute units, and at most what leaves every
// thread U vectors of the row.  One block per row would leave a launch of
// few such rows on a few compute units.
int stream_blocks(int64_t rows, int64_t nvec, int T, int U, int bpc, int cus) {
  if (bpc || rows >= 2 * (int64_t)cus) return 1;
  int S = 1;
  while (S * 2 <= kStreamMaxSplit && S * 2 <= cus && rows * S < 2 * (int64_t)cus) S *= 2;
  while (S > 1 && (int64_t)S * T * U > nvec) S >>= 1;
  return S;
}

}  // namespace

// Forward plan: fills p for the family cfg asks for (AUTO resolves first)
// and the config overrides; returns ROWSM_OK, or ROWSM_EINVAL when the family
// cannot take this shape.  mode is the output form (kPlain, kFused or kLog);
// the log form holds x where softmax holds exp(x - m), so it takes the plain
// plans.
int plan_for(int64_t rows, int64_t cols, int in_dt, int out_dt, uintptr_t xa, uintptr_t ya,
             const rowsm_config* cfg, int cus, int mode, bool inplace, Plan* p) {
  if (!config_in_domain(cfg)) return ROWSM_EINVAL;
  // In place (y == x) no form whose blocks exchange partial results is
  // planned: a block that recomputes a peer's partial reads the peer's share
  // of x, which the peer may already have overwritten.
  if (inplace && cfg && cfg->split_blocks > 0) return ROWSM_EINVAL;
  const bool fused = mode == kFused;
  const int ib = dtype_bytes(in_dt), ob = dtype_bytes(out_dt);
  int vw = choose_vw(cols, ib, ob, xa, ya);
  // Ragged rows (ragged_row.hpp): a width that is not a multiple of the full
  // 16-byte vector width, with both tensors aligned to it, softmax and log
  // forms.  Taken when cfg->vw asks for the full width (with the medium
  // variant or none), and by the launcher for rows that span at least a
  // wave of vectors and fit one block's registers, unless few long rows
  // would leave the device idle; otherwise such rows use narrower vectors.
  const int vw_full = 16 / (ib > ob ? ib : ob);
  const bool ragged_ok = !fused && cols % vw_full != 0 && vw_supported(vw_full, ib) &&
                         xa % (uintptr_t)(vw_full * ib) == 0 &&
                         ya % (uintptr_t)(vw_full * ob < 16 ? vw_full * ob : 16) == 0;
  const int64_t ragged_span = cdiv(cols + vw_full - 1, vw_full);  // longest row span
  // values per lane of the ragged kernels (ragged_cap())
  const int ragged_vals = 40;
  const int64_t ragged_max_span = 16 * (int64_t)kWave * (ragged_vals / vw_full);
  bool ragged = false;
  // Flat short rows (flat_row.hpp): such widths up to what a tile of 4
  // vectors per lane holds in one row, read as one flat stream of whole
  // vectors; taken when cfg asks for the small variant at the full vector
  // width, and by the launcher (below).
  // (at most 1024 columns: 64 lanes of 16 elements in the row phase)
  const int64_t flat_tile_cols = (int64_t)kFlatSlots * kWave * vw_full - (vw_full - 1);
  const int64_t flat_max_cols = flat_tile_cols < 1024 ? flat_tile_cols : 1024;
  bool flat = false;
  if (ragged_ok && cfg && cfg->vw == vw_full && cfg->variant == ROWSM_SMALL) {
    if (cols > flat_max_cols) return ROWSM_EINVAL;
    flat = true;
  } else if (ragged_ok && cfg && cfg->vw == vw_full) {
    if (cfg->variant != ROWSM_AUTO && cfg->variant != ROWSM_MEDIUM) return ROWSM_EINVAL;
    if (ragged_span > ragged_max_span) return ROWSM_EINVAL;
    ragged = true;
  } else if (ragged_ok && (!cfg || (cfg->variant == ROWSM_AUTO && cfg->vw == 0 &&
                                    cfg->waves_per_row == 0 && cfg->rows_per_block == 0 &&
                                    cfg->block == 0 && cfg->split_blocks == 0 &&
                                    cfg->packed != 1))) {
    // (rows whose narrow-vector plan spreads them over several blocks each,
    // too long for one block or few and long, keep it below cus / 4 rows:
    // the ragged form has one block per row.  A sweep of 8-400 rows of
    // 16385-38401 columns in every dtype pair: from 96 rows the ragged form
    // was 0.64-1.06x the split form's time, 0.84x on geometric mean; at 8
    // and 32 rows 1.02-1.40x.)
    const int64_t narrow_nvec = cols / vw;
    const bool narrow_medium =
        narrow_nvec <= 16 * kWave * (64 / vw < 16 ? 64 / vw : 16) &&
        (inplace || !few_long_rows(rows, cols * (ib + ob), false, cus));
    // Spans of 120 vectors up to what 16 waves hold: sweeps of
    // 301-50257-column rows in every dtype pair (96 and 512 MiB launches,
    // each alone after a cache-evicting write) measured the ragged form
    // 0.6-0.9x the narrow-vector time from 256 vectors, and with its edges
    // read as whole vectors 0.85-0.96x at 1001-column rows (126-251
    // vectors); at 88 vectors (701 bf16 columns) up to 7% slower.  (Spans of 8193-10240 fp32-width
    // vectors, 9-10 slots of 16 waves: 0.80-0.94x the split form from 200
    // rows.)
    ragged = ragged_span >= 120 && ragged_span <= ragged_max_span &&
             (inplace || !few_long_rows(rows, cols * (ib + ob), false, cus)) &&
             (narrow_medium || rows >= cus / 4);
  }
  // The launcher takes the flat form for rows of 9-480 columns whose narrow
  // vectors would be of at most 4 bytes (one fp32 or one or two bf16
  // elements).  A sweep of 3-1001-column rows in every dtype pair at 64 and
  // 512 MiB (each launch alone after a cache-evicting write): 1.04-1.37x
  // the time of a plain copy of the same bytes at 13-1001 columns, where
  // the narrow-vector plans took up to 3.9x; against the narrow plans'
  // fastest grid 0.26-0.98x at 13-129 columns (0.35x at 37), level at 257
  // and beyond; slower at 3-7 columns (the small-row kernel packs such rows
  // into its lanes, 1.04-2.0x) and for rows of half-width vectors (60 and
  // 100 bf16 columns, 1.01-1.19x).  At 257-449 columns two more sweeps
  // measured it 0.77-1.04x the narrow plan (0.89x on geometric mean), at
  // 511 level (0.94-1.12x).
  if (!ragged && !flat && ragged_ok && cols > 8 && cols <= 480 &&
      vw * (ib > ob ? ib : ob) <= 4 &&
      (!cfg || (cfg->variant == ROWSM_AUTO && cfg->vw == 0 && cfg->waves_per_row == 0 &&
                cfg->rows_per_block == 0 && cfg->block == 0 && cfg->split_blocks == 0 &&
                cfg->lanes_per_row == 0 && cfg->rows_per_lane == 0 && cfg->packed != 1)))
    flat = true;
  if (flat) {
    // lanes per row and elements per lane of the row phase (launch_flat.hpp)
    int lpr = 0, e = 0;
    if (!flat_row_shape(cfg, cols, &lpr, &e)) return ROWSM_EINVAL;
    // bf16 to bf16 rows of up to 45 columns: tiles of 2 vectors per lane
    // (58-61 VGPRs and 4 KiB of LDS per wave where 4 take 96 and 8 KiB).
    // Forced tiles of both sizes at 64 and 384 MiB, each launch alone after
    // a cache-evicting write: 0.77-0.97x the time of 4 at 9-41 columns
    // (0.88x on geometric mean, softmax and log form alike), 0.92-1.11x at
    // 77-127 and up to 1.3x at 255-479, where a tile holds fewer rows; at
    // 45-63 columns, not fitted, 0.98x at 45 and 0.87-1.12x beyond (1.07-
    // 1.12x at 47-59 columns and 384 MiB).
    const int slots = flat_slots(cfg, ib, ob, cols, vw_full, cols <= 45);
    if (!slots) return ROWSM_EINVAL;
    const int64_t G = ((int64_t)slots * kWave * vw_full - (vw_full - 1)) / cols;
    const int64_t tiles = cdiv(rows, G);
    p->variant = ROWSM_SMALL;
    p->flat = true;
    p->vw = vw_full;
    p->nvec = (int)ragged_span;
    p->lpr = lpr;
    p->nv = e;
    p->vpl = e;
    p->rpl = slots;
    p->block = kWave;
    const int bpc = (cfg && cfg->blocks_per_cu > 0) ? cfg->blocks_per_cu : 0;
    p->grid = tiles < grid_cap(bpc, cus) ? tiles : grid_cap(bpc, cus);
    return ROWSM_OK;
  }
  if (ragged) {
    vw = vw_full;
  } else if (cfg && cfg->vw > 0) {
    const int want = cfg->vw;
    if (want > 16 / (ib > ob ? ib : ob) || (want & (want - 1)) || !vw_supported(want, ib) ||
        cols % want ||
        xa % (want * ib) || ya % (want * ob < 16 ? want * ob : 16))
      return ROWSM_EINVAL;
    vw = want;
  }
  const int nvec = ragged ? (int)ragged_span : (int)(cols / vw);
  p->vw = vw;
  p->nvec = nvec;
  p->ragged = ragged;

  int variant = cfg ? cfg->variant : ROWSM_AUTO;
  if (ragged) variant = ROWSM_MEDIUM;
  const bool auto_variant = (cfg ? cfg->variant : ROWSM_AUTO) == ROWSM_AUTO;
  bool wide_row = false;  // a MEDIUM row redirected to the split form
  RowShape shape;         // measured_row_shape() pick, when it applies
  if (variant == ROWSM_AUTO) {
    if (nvec <= 32) {
      variant = ROWSM_SMALL;
    } else if (nvec <= 16 * kWave * ((fused ? 32 : 64) / vw < 16 ? (fused ? 32 : 64) / vw : 16)) {
      // whole row in the registers of one block, unless few long rows would
      // then leave most of the device idle
      variant = !inplace && few_long_rows(rows, cols * (ib + ob), false, cus) ? ROWSM_LARGE
                                                                             : ROWSM_MEDIUM;
    } else if (!fused && in_dt == ROWSM_BF16 && vw == 8 && nvec <= 16 * kWave * 24) {
      variant = !inplace && few_long_rows(rows, cols * (ib + ob), true, cus) ? ROWSM_LARGE
                                                                            : ROWSM_MEDIUM;
    } else {
      variant = ROWSM_LARGE;
    }
  }
  p->variant = variant;

  const int bpc = (cfg && cfg->blocks_per_cu > 0) ? cfg->blocks_per_cu : 0;
  if (variant == ROWSM_SMALL) {
    if (nvec > 32) return ROWSM_EINVAL;
    p->lpr = next_pow2(nvec);
    if (cfg && cfg->lanes_per_row > 0) {
      const int l = cfg->lanes_per_row;
      if ((l & (l - 1)) || l > 32 || l < p->lpr) return ROWSM_EINVAL;
      p->lpr = l;
    }
    p->rpl = 4;
    if (cfg && cfg->rows_per_lane > 0) {
      const int r = cfg->rows_per_lane;
      if (r != 1 && r != 2 && r != 4 && r != 8) return ROWSM_EINVAL;
      if (fused && r != 4) return ROWSM_EINVAL;  // fused kernels: 4 rows per lane
      p->rpl = r;
    }
    if (small_block(cfg, &p->block) != ROWSM_OK) return ROWSM_EINVAL;
    // Rows that fill their lanes exactly, in launches of at least 40 MiB
    // (softmax and log forms, nothing about the shape forced): for a dtype
    // pair of one width, one-wave blocks with one row group per lane; for a
    // widening or narrowing pair, 128-thread blocks with two row groups per
    // lane.  Sweeps of 16-128-column rows at 24 MiB-2 GiB, each launch alone
    // after a cache-evicting write, on two devices: one-wave blocks were the
    // fastest or within 1% of it at every same-width size from 40 MiB, 3-5%
    // faster than 256-thread blocks of 4 row groups from 256 MiB on; on
    // bf16 <-> fp32 rows they were 5-19% slower than two row groups per lane,
    // which were 2-17% faster than the 256-thread blocks from 40 MiB on.
    // Below 40 MiB, and for rows that leave lanes idle (48 or 96 bf16
    // columns), the 256-thread blocks stay.  (No product of rows and row
    // bytes is formed: rows may be close to 2^62.)
    const int64_t row_bytes = cols * (ib + ob);
    const bool big_launch = rows >= cdiv((int64_t)40 << 20, row_bytes);
    if (auto_variant && !fused && nvec == p->lpr && big_launch &&
        (!cfg || (cfg->lanes_per_row == 0 && cfg->rows_per_lane == 0 && cfg->block == 0))) {
      p->block = ib == ob ? kWave : 2 * kWave;
      p->rpl = ib == ob ? 1 : 2;
    }
    const int64_t rows_per_block = (int64_t)(p->block / kWave) * (kWave / p->lpr) * p->rpl;
    p->grid = cdiv(rows, rows_per_block);
    if (p->grid > grid_cap(bpc, cus)) p->grid = grid_cap(bpc, cus);
    // Narrow-vector rows whose stores cover parts of lines: about 16 KiB of
    // traffic per block (looping_grid()).
    if (auto_variant && !fused && bpc == 0 && vw * (ib > ob ? ib : ob) < 16 &&
        !whole_lines(ya, cols * ob) &&
        (!cfg || (cfg->lanes_per_row == 0 && cfg->rows_per_lane == 0 && cfg->block == 0)))
      p->grid = looping_grid(rows, row_bytes, 16 << 10, p->grid, p->block, cus, 128);
    return ROWSM_OK;
  }
  if (variant == ROWSM_MEDIUM) {
    int wpr = 0, vpl = 0;
    bool packed = false;
    const int want_wpr = (cfg && cfg->waves_per_row > 0) ? cfg->waves_per_row : 0;
    const int want_packed = fused ? 0 : (cfg ? cfg->packed : -1);
    if ((fused || ragged) && cfg && cfg->packed == 1) return ROWSM_EINVAL;
    if (want_wpr && (want_wpr & (want_wpr - 1) || want_wpr > 16)) return ROWSM_EINVAL;
    // Unpacked: the smallest group whose lanes hold <= 16 fp32 values each
    // (<= 32, then <= 64 when the row is longer), unless a group size is
    // forced.  Fewer values per lane and more resident rows measured faster
    // than longer per-lane rows on the 32768 x 4096 workload.
    if (want_packed != 1) {
      // Fused rows keep column indices live as well: at most 32 values, and
      // 32 (fewer waves per row) measured fastest on the causal workload.
      for (int cap_vals : {16, 32, 64}) {
        if (fused && cap_vals != 32) continue;
        for (int w = 1; w <= 16; w <<= 1) {
          if (want_wpr && w != want_wpr) continue;
          const int v = (int)cdiv(nvec, (int64_t)w * kWave);
          if (v * vw <= cap_vals && medium_unpacked_cap(vw, v)) {
            wpr = w;
            vpl = v;
            break;
          }
        }
        if (wpr) break;
      }
    }
    // Ragged rows: the fewest waves whose lanes hold at most 40 values each,
    // or the wave count given if its lanes stay within that.  Over the sweep
    // above: 3.1% above the fastest wave count and rows per block measured
    // on geometric mean, where the 16-value rule took 15% and the
    // narrow-vector plan 20%.
    if (ragged) {
      wpr = 0;
      // (unless a wave count is given: the fewest of 1, 2 or 4 waves whose
      // lanes hold at most 3 vectors, else from 4 waves the fewest within
      // 40 values; over sweeps of 129-2047-column rows in every dtype pair
      // 1.4% above the fastest wave count measured on geometric mean where
      // the fewest waves within 40 values took 3.2%, up to 10% on spans of
      // 376-513 vectors)
      int min_w = 1;
      if (!want_wpr) {
        min_w = 4;
        for (int w = 1; w <= 4; w <<= 1)
          if (cdiv(nvec, (int64_t)w * kWave) <= 3) {
            min_w = w;
            break;
          }
      }
      for (int w = 1; w <= 16; w <<= 1) {
        if (want_wpr && w != want_wpr) continue;
        if (w < min_w) continue;
        const int v = (int)cdiv(nvec, (int64_t)w * kWave);
        if (v * vw <= ragged_vals) {
          wpr = w;
          vpl = v;
          break;
        }
      }
      if (!wpr) return ROWSM_EINVAL;
    }
    if (!wpr && !ragged && want_packed != 0 && in_dt == ROWSM_BF16 && vw == 8) {
      for (int w = 1; w <= 16; w <<= 1) {
        if (want_wpr && w != want_wpr) continue;
        const int v = (int)cdiv(nvec, (int64_t)w * kWave);
        if (v <= 24 && (w == 16 || want_wpr)) {
          wpr = w;
          vpl = v;
          packed = true;
          break;
        }
      }
    }
    if (!wpr) return ROWSM_EINVAL;
    // Slot counts are exact (only the last slot may be partial); packed
    // kernels exist for 9..24 slots.
    if (packed && (vpl < 9 || vpl > 24)) return ROWSM_EINVAL;
    p->wpr = wpr;
    p->vpl = vpl;
    p->packed = packed;
    // Launches of 4-16 rows per compute unit (softmax and log forms, rows of
    // full vectors under 64 KiB of input, nothing about the shape forced):
    // the fewest waves per row, at least what the registers need, that still
    // give the launch about two 512-thread blocks per compute unit, so that
    // each lane keeps more bytes in flight.  From sweeps of 1024-16384
    // columns in every dtype pair: at 1024 and 2048 rows 1.6% above the
    // fastest form measured on geometric mean (at most 9%), where the rule
    // above was 8.9% (at most 54%); at 1536 and 3072 rows, not fitted, 4.8%
    // (at most 24%) against 12% (at most 44%).  At 4096 and 6144 rows the two
    // rules tie on geometric mean and the rule above stays.
    const bool shape_free = !cfg || (cfg->waves_per_row == 0 && cfg->rows_per_block == 0 &&
                                     cfg->packed == -1 && cfg->block == 0 &&
                                     cfg->split_blocks == 0 && cfg->vw == 0);
    // (rows of whole full-width vectors; the ragged form keeps the base rule)
    const bool full_vw = vw * (ib > ob ? ib : ob) == 16 && !ragged;
    if (auto_variant && !fused && shape_free && full_vw && rows >= 4 * (int64_t)cus &&
        rows < 16 * (int64_t)cus && cols * ib < 65536) {
      int target = 1;
      while ((int64_t)target * 2 * rows <= 16 * (int64_t)cus) target <<= 1;
      for (int w = target; w <= 16; w <<= 1) {
        const int v = (int)cdiv(nvec, (int64_t)w * kWave);
        if (v * vw <= 64 && medium_unpacked_cap(vw, v)) {
          p->wpr = w;
          p->vpl = v;
          p->packed = false;
          break;
        }
        // (the packed form up to 8 rows per compute unit: from 9 to 16 it
        // was 5-20% slower than the unpacked rows of more waves, at 8 level
        // or faster; sweeps of 9544-28344 bf16 columns)
        if (in_dt == ROWSM_BF16 && vw == 8 && v >= 9 && v <= 24 && rows <= 8 * (int64_t)cus) {
          p->wpr = w;
          p->vpl = v;
          p->packed = true;
          break;
        }
      }
    }
    // Full launches of rows of 129-4096 full vectors, when nothing about the
    // shape is forced: the measured shapes of measured_row_shape() (fused
    // form: measured_fused_shape()).
    if (auto_variant && shape_free && full_vw && rows >= 32 * (int64_t)cus &&
        (fused ? measured_fused_shape(nvec, ib, ob, &shape)
               : measured_row_shape(nvec, ib, ob, &shape))) {
      // (a single-read pick holds one group of blocks per row only while
      // the rows fit the exchange workspace; beyond, and in place, the
      // medium rule stays)
      if (shape.S > 0 && (inplace || rows * shape.S > kSplitMaxBlocks)) shape = RowShape{};
      if (shape.S > 0) {
        variant = ROWSM_LARGE;
        p->variant = variant;
        p->wpr = 1;
        p->packed = false;
      } else if (shape.wpr > 0) {
        // Lane fill: when the table's wave group leaves too much of its last
        // slot empty (less than 60% of the group's slots hold a vector, 70%
        // for bf16 <-> fp32 rows), the largest smaller group that fills them
        // is taken, in 256-thread blocks.  Rows just past a group boundary
        // (e.g. 260-350 vectors on 4 waves, 136-170 on 2) measured 10-42%
        // slower than the smaller group for bf16 <-> fp32 and up to 15% for
        // one width.  Over 193 full launches of 136-1024-vector rows in every
        // dtype pair (three sweeps, each launch alone after a cache-evicting
        // write) the table's picks were 6.1% above the fastest form on
        // geometric mean and are 2.0% with this rule, no launch more than 2%
        // slower than before; at the 88 lengths of the third sweep, which
        // were not used to set the thresholds, 7.7% and 2.7%.
        const int fill_pct = ib == ob ? 60 : 70;
        auto filled = [&](int w) {
          const int64_t slots = cdiv(nvec, (int64_t)w * kWave) * w * kWave;
          return nvec * 100 >= (int64_t)fill_pct * slots;
        };
        if (!filled(shape.wpr)) {
          for (int w = shape.wpr / 2; w >= 1; w /= 2) {
            const int v = (int)cdiv(nvec, (int64_t)w * kWave);
            if (v * vw > 64 || !medium_unpacked_cap(vw, v)) break;
            if (filled(w)) {
              shape.wpr = w;
              shape.rpb = 4 / w > 1 ? 4 / w : 1;
              break;
            }
          }
        }
        p->wpr = shape.wpr;
        p->vpl = (int)cdiv(nvec, (int64_t)shape.wpr * kWave);
        p->packed = false;
      }
    }
    // Rows under 64 KiB of input that the 16-value rule puts on all 16 waves
    // of a 1024-thread block, in launches that neither the measured shapes
    // (from 32 * cus rows) nor the rule for 4-16 rows per compute unit
    // cover: the fewest waves whose lanes hold at most 48 values (the
    // 16-wave blocks synchronise a compute unit's worth of waves at each
    // reduction).  A sweep of 1-32 rows per compute unit of 1024-40000
    // columns in every dtype pair (each launch alone after a cache-evicting
    // write): 3.1% above the fastest shape measured on geometric mean where
    // the 16-wave rows took 4.8% (at most 33%: 6144 x 8240 bf16 -> fp32),
    // no launch more than 3% slower.
    if (variant == ROWSM_MEDIUM && auto_variant && !fused && shape_free && full_vw &&
        p->wpr == 16 && !p->packed && rows < 32 * (int64_t)cus &&
        !(rows >= 4 * (int64_t)cus && rows < 16 * (int64_t)cus) && cols * ib < 65536) {
      for (int w = 1; w < 16; w <<= 1) {
        const int v = (int)cdiv(nvec, (int64_t)w * kWave);
        if (v * vw <= 48 && medium_unpacked_cap(vw, v)) {
          p->wpr = w;
          p->vpl = v;
          break;
        }
      }
    }
    // A row of at least 64 KiB of input that needs all 16 waves of a
    // 1024-thread block goes to the single-read split form: from 8 * cus
    // rows, or from cus / 4 rows when a lane would hold 64 or more values (or
    // the packed form), with 256-thread blocks and the threads per row of
    // the wide-row plan below (a sweep of 256-8192 rows x 16384-151936
    // columns in every dtype pair: 5-31% faster than the medium form); and,
    // with the register-cap plan, rows of 80 KiB or more at any other row
    // count and shorter ones in launches of fewer than cus / 2 rows.  The
    // 16-wave blocks synchronise a whole compute unit's worth of waves at
    // each reduction and leave at most two blocks per compute unit.  Sweeps
    // of 16-4096 rows of 64-240 KiB in every dtype pair (each launch alone
    // after a cache-evicting write): 2.3% above the fastest shape measured on
    // geometric mean, where the first two conditions alone were 11% (at most
    // 2.07x, few rows); 2.0% at 95 launches of 72-192 KiB rows not used to
    // set the bounds.  Rows of 64-80 KiB in launches of cus / 2 to 8 * cus
    // rows stay in the medium form, up to 18% faster there.
    const bool wide_plan =
        rows >= 8 * (int64_t)cus || ((vpl * vw >= 64 || packed) && rows >= cus / 4);
    if (variant == ROWSM_MEDIUM && auto_variant && !fused && !inplace && !ragged &&
        p->wpr == 16 && cols * ib >= 65536 &&
        (wide_plan || rows < cus / 2 || cols * ib >= 81920)) {
      wide_row = wide_plan;
      variant = ROWSM_LARGE;
      p->variant = variant;
      p->wpr = 1;
      p->packed = false;
    }
  }
  if (variant == ROWSM_MEDIUM) {
    const int wpr = p->wpr;
    p->nv = p->vpl;
    // 512-thread blocks (256 for the fused form, fewer rows per block when a
    // row needs more waves); one block per row group, no grid-stride loop
    // unless capped.
    const int waves_per_block = fused ? 4 : 8;
    int rpb = wpr >= waves_per_block ? 1 : waves_per_block / wpr;
    if (shape.rpb > 0) rpb = shape.rpb;
    // Ragged rows: one row per block.  Over the sweep of 1-32 rows per
    // compute unit: 4.4% above the fastest shape measured on geometric mean
    // where the blocks of 512 threads took 9.1%, none slower.
    if (ragged) rpb = 1;
    if (cfg && cfg->rows_per_block > 0) {
      rpb = cfg->rows_per_block;
      if (rpb * wpr > 16) return ROWSM_EINVAL;
    }
    p->block = rpb * wpr * kWave;
    p->grid = cdiv(rows, rpb);
    if (p->grid > grid_cap(bpc, cus)) p->grid = grid_cap(bpc, cus);
    // One wave per row and one to four slots per lane, softmax and log
    // forms, nothing about the shape or grid given: about 32 KiB of traffic
    // per block, each block looping over its rows (looping_grid()), instead
    // of a block per 8 such short rows.
    if (auto_variant && !fused && !ragged && wpr == 1 && bpc == 0 && p->vpl <= 4 &&
        (!cfg || (cfg->rows_per_block == 0 && cfg->block == 0 && cfg->waves_per_row == 0 &&
                  cfg->vw == 0)))
      p->grid = looping_grid(rows, cols * (ib + ob), 32 << 10, p->grid, p->block, cus);
    return ROWSM_OK;
  }
  if (variant == ROWSM_LARGE) {
    const int want_split = cfg ? cfg->split_blocks : 0;
    if (cfg && cfg->block > 0) {
      const int b = cfg->block;
      if (b % kWave || b > 1024) return ROWSM_EINVAL;
    }
    if (want_split >= 0 && !inplace) {
      // Single-read form: T threads per block, S blocks per row (S <= 64:
      // one wave polls the S peers), at most 64 fp32 values per lane (40
      // for widening rows, bf16 -> f32, which write twice what they read).
      // 512-thread blocks, except 256 where 512 would leave fewer than 8
      // blocks to a row that does not widen (a sweep of 1024-4096 rows x
      // 98304-1048576 columns in every dtype pair, one group per row: 512
      // gains up to 15% on the longest rows; 256 is 8% faster on
      // 1024 x 131072 f32).
      const bool widening = ob > ib;
      const bool forced_block = cfg && cfg->block > 0;
      const int vals = fused ? 32 : (widening ? 40 : 64);
      int nv_cap = vals / vw < 16 ? vals / vw : 16;
      if (nv_cap < 1) nv_cap = 1;
      int T = 512;
      if (forced_block) T = cfg->block;
      else if (!widening && cdiv(nvec, (int64_t)nv_cap * 512) < 8) T = 256;
      int S = want_split > 0 ? want_split : (int)cdiv(nvec, (int64_t)nv_cap * T);
      if (wide_row && want_split == 0 && !forced_block) {
        // Rows redirected from the 16-wave medium form: the power of two of
        // threads per row that gives each lane 64-128 bytes of the input,
        // in 256-thread blocks up to 2048 threads per row and 512-thread
        // blocks beyond, and a power of two of blocks at least as large as
        // the register cap needs (whole slots: 7 blocks of a 65536-wide
        // bf16 -> f32 row measured 10-13% slower than 8).  Fastest or
        // within 3% at 16384-151936 columns and 256-8192 rows.
        int64_t thr = 1;
        while (thr * 128 < cols * ib) thr <<= 1;
        T = thr <= 2048 ? 256 : 512;
        S = thr / T > 1 ? (int)(thr / T) : 1;
        const int64_t s_cap = cdiv(nvec, (int64_t)nv_cap * T);
        while (S < s_cap) S <<= 1;
      }
      if (shape.S > 0) {
        S = shape.S;
        T = shape.T;
      }
      if (S < 1) S = 1;
      // Grid: one group of S blocks per row (0), or with blocks_per_cu
      // given, one residency of at most that many blocks per compute unit
      // whose groups loop over the rows (negative; split_slots()).
      int64_t grid = bpc ? -(int64_t)bpc : 0;
      if (want_split == 0) {
        // Few rows: more, smaller blocks per row so that the launch fills
        // the device (256-thread blocks unless a block size is given; also
        // when the row then has as many threads as in the plan above, which
        // measured up to 9% faster at 16-64 rows of 151936-262144 columns).
        const int Tf = forced_block ? T : 256;
        const int sf = few_rows_split(rows, nvec, Tf, nv_cap, cus);
        if (sf > 0 && (int64_t)sf * Tf >= (int64_t)S * T) {
          S = sf;
          T = Tf;
        }
      }
      const int nv = (int)cdiv(nvec, (int64_t)S * T);
      if (S <= 64 && nv <= nv_cap && nv * vw <= 64) {
        p->split = S;
        p->nv = nv;
        p->vpl = nv;
        p->block = T;
        p->grid = grid;
        p->prefetch = cfg && cfg->prefetch == 1;
        // registers: at most 48 values per lane (44 for fp32 input), plain
        // and log forms only (split_launch.hpp)
        if (p->prefetch && (fused || nv * vw > (ib == 4 ? 44 : 48))) return ROWSM_EINVAL;
        return ROWSM_OK;
      }
      if (want_split > 0) return ROWSM_EINVAL;
    }
    p->split = 0;
    p->u = 4;
    if (cfg && cfg->tile_vectors > 0) {
      const int u = cfg->tile_vectors;
      if (u != 2 && u != 4 && u != 8) return ROWSM_EINVAL;
      p->u = u;
    }
    p->block = (cfg && cfg->block > 0) ? cfg->block : 1024;
    const int64_t cap = (int64_t)cus * (bpc ? bpc : 1);
    p->grid = rows < cap ? rows : cap;
    p->stream = inplace ? 1 : stream_blocks(rows, nvec, p->block, p->u, bpc, cus);
    return ROWSM_OK;
  }
  return ROWSM_EINVAL;
}

// Plan of the softmax backward: y and dy of in_dt (both aligned as ia), dx
// of out_dt at dxa.  The register-resident forms hold y and dy raw; a lane's
// share of each input is at most 128 bytes (and 16 slots).
//   SMALL   a row is at most 32 vectors;
//   MEDIUM  the smallest row group of <= 16 waves whose lanes hold at most 32
//           bytes of each input (then 64, then 128), unless the rows are few
//           and long (the forward's row-count rule, on the backward's bytes);
//   LARGE   the row split over S <= 64 co-resident 512-thread blocks (more,
//           256-thread blocks per row for few rows, as the forward), or two
//           streaming passes for rows longer than that.
int plan_backward(int64_t rows, int64_t cols, int in_dt, int out_dt, uintptr_t ia,
                  uintptr_t dxa, const rowsm_config* cfg, int cus, bool inplace, Plan* p) {
  if (!config_in_domain(cfg)) return ROWSM_EINVAL;
  // In place (dx == y or dx == dy): no exchanging form, as plan_for().
  if (inplace && cfg && cfg->split_blocks > 0) return ROWSM_EINVAL;
  if (cfg && cfg->packed == 1) return ROWSM_EINVAL;  // no packed form: always raw
  const int ib = dtype_bytes(in_dt), ob = dtype_bytes(out_dt);
  int vw = choose_vw(cols, ib, ob, ia, dxa);
  // Flat short rows (flat_row.hpp), as the forward's: a width that is not a
  // multiple of the full 16-byte vector width, y, dy and dx aligned to it;
  // taken when cfg asks for the small variant at the full vector width, and
  // by the launcher for 9-480 columns whose narrow vectors would be of at
  // most 4 bytes, bf16 to bf16 only up to 128 columns.  A sweep of 5-1001
  // columns in every dtype pair at 64 and 384 MiB (each launch alone after
  // a cache-evicting write): 0.85x the narrow-vector plans' time on
  // geometric mean at 9-480 columns with tiles of 4 vectors per lane,
  // 0.40-0.62x at 37-41.  bf16 to bf16 takes tiles of 2 vectors per lane
  // (81 VGPRs and 8 KiB of LDS per wave where 4 took 129 and 16 KiB):
  // 0.35-0.96x at 13-129 columns (41: 198 -> 69 us at 384 MiB), 1.03x on
  // geometric mean at 255-479, where a tile holds 2-3 rows.
  const int vw_full = 16 / (ib > ob ? ib : ob);
  const bool flat_ok = cols % vw_full != 0 && vw_supported(vw_full, ib) &&
                       ia % (uintptr_t)(vw_full * ib) == 0 &&
                       dxa % (uintptr_t)(vw_full * ob < 16 ? vw_full * ob : 16) == 0;
  bool flat = false;
  if (flat_ok && cfg && cfg->vw == vw_full && cfg->variant == ROWSM_SMALL) {
    const int64_t most = (int64_t)kFlatSlots * kWave * vw_full - (vw_full - 1);
    if (cols > (most < 1024 ? most : 1024)) return ROWSM_EINVAL;
    flat = true;
  } else if (flat_ok && cols > 8 && cols <= 480 && vw * (ib > ob ? ib : ob) <= 4 &&
             (ib == 4 || ob == 4 || cols <= 128) &&
             (!cfg || (cfg->variant == ROWSM_AUTO && cfg->vw == 0 && cfg->waves_per_row == 0 &&
                       cfg->rows_per_block == 0 && cfg->block == 0 &&
                       cfg->split_blocks == 0 && cfg->lanes_per_row == 0 &&
                       cfg->rows_per_lane == 0))) {
    flat = true;
  }
  if (flat) {
    int lpr = 0, e = 0;
    if (!flat_row_shape(cfg, cols, &lpr, &e)) return ROWSM_EINVAL;
    // tiles of 4 vectors per lane, 2 for bf16 to bf16 rows that fit them
    const int slots = flat_slots(cfg, ib, ob, cols, vw_full, true);
    if (!slots) return ROWSM_EINVAL;
    const int64_t tiles = cdiv(rows, ((int64_t)slots * kWave * vw_full - (vw_full - 1)) / cols);
    const int bpc = (cfg && cfg->blocks_per_cu > 0) ? cfg->blocks_per_cu : 0;
    p->variant = ROWSM_SMALL;
    p->flat = true;
    p->vw = vw_full;
    p->nvec = (int)cdiv(cols + vw_full - 1, vw_full);
    p->lpr = lpr;
    p->nv = e;
    p->vpl = e;
    p->rpl = slots;
    p->block = kWave;
    p->grid = tiles < grid_cap(bpc, cus) ? tiles : grid_cap(bpc, cus);
    return ROWSM_OK;
  }
  if (cfg && cfg->vw > 0) {
    const int want = cfg->vw;
    if (want > 16 / (ib > ob ? ib : ob) || (want & (want - 1)) || !vw_supported(want, ib) ||
        cols % want || ia % (want * ib) || dxa % (want * ob < 16 ? want * ob : 16))
      return ROWSM_EINVAL;
    vw = want;
  }
  const int nvec = (int)(cols / vw);
  const int vbytes = vw * ib;  // bytes of one input vector
  int nv_cap = 128 / vbytes < 16 ? 128 / vbytes : 16;
  p->vw = vw;
  p->nvec = nvec;

  int variant = cfg ? cfg->variant : ROWSM_AUTO;
  const bool auto_variant = variant == ROWSM_AUTO;
  RowShape shape;  // measured_backward_shape() pick, when it applies
  if (variant == ROWSM_AUTO) {
    if (nvec <= 32)
      variant = ROWSM_SMALL;
    else if (nvec <= 16 * kWave * nv_cap &&
             (inplace ||
              !few_long_rows(rows, cols * (2 * ib + ob), false, cus, kFewRowsMinBytesBackward)))
      variant = ROWSM_MEDIUM;
    else
      variant = ROWSM_LARGE;
  }
  p->variant = variant;
  const int bpc = (cfg && cfg->blocks_per_cu > 0) ? cfg->blocks_per_cu : 0;

  if (variant == ROWSM_SMALL) {
    if (nvec > 32) return ROWSM_EINVAL;
    p->lpr = next_pow2(nvec);
    if (cfg && cfg->lanes_per_row > 0) {
      if (cfg->lanes_per_row < p->lpr) return ROWSM_EINVAL;
      p->lpr = cfg->lanes_per_row;
    }
    p->rpl = (cfg && cfg->rows_per_lane > 0) ? cfg->rows_per_lane : 4;
    if (small_block(cfg, &p->block) != ROWSM_OK) return ROWSM_EINVAL;
    // Rows that fill their lanes exactly, in launches of at least 96 MiB of
    // the three streams (nothing about the shape forced): one-wave blocks
    // with one row group per lane, as the forward's rule for its mid-size
    // launches.  Launches timed alone after a cache-evicting write measured
    // them 1.0-3.4% faster on each of 14 launches of 96-768 MiB (32-256
    // columns, bf16 and fp32) held out from the ones that set the bound, and
    // 2-4% slower on three of four launches of 48 MiB.
    const int64_t bwd_row_bytes = cols * (2 * ib + ob);
    if (auto_variant && nvec == p->lpr && rows >= cdiv((int64_t)96 << 20, bwd_row_bytes) &&
        (!cfg || (cfg->lanes_per_row == 0 && cfg->rows_per_lane == 0 && cfg->block == 0))) {
      p->block = kWave;
      p->rpl = 1;
    }
    const int64_t rows_per_block = (int64_t)(p->block / kWave) * (kWave / p->lpr) * p->rpl;
    p->grid = cdiv(rows, rows_per_block);
    if (p->grid > grid_cap(bpc, cus)) p->grid = grid_cap(bpc, cus);
    return ROWSM_OK;
  }
  if (variant == ROWSM_MEDIUM) {
    const int want_wpr = (cfg && cfg->waves_per_row > 0) ? cfg->waves_per_row : 0;
    int wpr = 0, nv = 0;
    for (int cap_bytes : {32, 64, 128}) {
      for (int w = 1; w <= 16; w <<= 1) {
        if (want_wpr && w != want_wpr) continue;
        const int v = (int)cdiv(nvec, (int64_t)w * kWave);
        if (v * vbytes <= cap_bytes && v <= nv_cap) {
          wpr = w;
          nv = v;
          break;
        }
      }
      if (wpr) break;
    }
    if (!wpr) return ROWSM_EINVAL;
    // Launches of 4-16 rows per compute unit (rows of full vectors under 64
    // KiB of each input, nothing about the shape forced): as the forward,
    // the fewest waves per row that the per-lane cap allows and that keep
    // about two 512-thread blocks per compute unit.  Sweeps of 1024-16384
    // columns in every dtype pair: at 1024 and 2048 rows 3.1% and 2.3% above
    // the fastest form on geometric mean, where the rule above was 7.3% and
    // 3.7%; at 1536 and 3072 rows, not fitted, 3.1% against 5.2%, and level.
    const bool shape_free = !cfg || (cfg->waves_per_row == 0 && cfg->rows_per_block == 0 &&
                                     cfg->block == 0 && cfg->split_blocks == 0 && cfg->vw == 0);
    if (auto_variant && shape_free && vw * (ib > ob ? ib : ob) == 16 &&
        rows >= 4 * (int64_t)cus && rows < 16 * (int64_t)cus && cols * ib < 65536) {
      int target = 1;
      while ((int64_t)target * 2 * rows <= 16 * (int64_t)cus) target <<= 1;
      for (int w = target; w <= 16; w <<= 1) {
        const int v = (int)cdiv(nvec, (int64_t)w * kWave);
        if (v <= nv_cap) {
          wpr = w;
          nv = v;
          break;
        }
      }
    }
    // Full launches of rows of 129-4096 full vectors, when nothing about the
    // shape is forced: the measured shapes of measured_backward_shape() (a
    // single-read pick only out of place and while the rows fit the
    // exchange workspace with one group of blocks per row).
    int table_rpb = 0;
    if (auto_variant && shape_free && vw * (ib > ob ? ib : ob) == 16 &&
        rows >= 32 * (int64_t)cus && measured_backward_shape(nvec, ib, ob, &shape)) {
      if (shape.S > 0 && (inplace || rows * shape.S > kSplitMaxBlocks)) {
        shape = RowShape{};
      } else if (shape.wpr > 0) {
        wpr = shape.wpr;
        nv = (int)cdiv(nvec, (int64_t)wpr * kWave);
        table_rpb = shape.rpb;
      }
    }
    // A row that needs all 16 waves of a 1024-thread block goes to the
    // split form when it holds at least 64 KiB of each input, from 4 * cus
    // rows (measured 4-20% faster there at 16384-65536 columns in every
    // dtype pair, and within 1% of the medium form at 256-512 rows; the
    // forward's reason) and in launches of fewer than cus / 2 rows, where
    // the split form's blocks spread a row over more compute units (16-48
    // rows of 64-96 KiB: 10-43% faster; at cus / 2 rows the medium form is
    // up to 20% ahead).  Sweeps of 16-1536 rows of 64-160 KiB in every dtype
    // pair, each launch alone after a cache-evicting write: 3.7% above the
    // fastest shape measured on geometric mean, where the first bound alone
    // was 10.5%.
    if (shape.S > 0 || (auto_variant && !inplace && wpr == 16 && cols * ib >= 65536 &&
                        (rows >= 4 * (int64_t)cus || rows < cus / 2))) {
      variant = ROWSM_LARGE;
      p->variant = variant;
    } else {
      p->wpr = wpr;
      p->vpl = nv;
      p->nv = nv;
      int rpb = table_rpb ? table_rpb : (wpr >= 8 ? 1 : 8 / wpr);  // 512-thread blocks
      if (cfg && cfg->rows_per_block > 0) {
        rpb = cfg->rows_per_block;
        if (rpb * wpr > 16) return ROWSM_EINVAL;
      }
      p->block = rpb * wpr * kWave;
      p->grid = cdiv(rows, rpb);
      if (p->grid > grid_cap(bpc, cus)) p->grid = grid_cap(bpc, cus);
      // Rows of one wave and one to four slots, nothing about the shape or
      // grid given: about 24 KiB of the three streams per block, each block
      // looping over its rows (looping_grid()).
      if (auto_variant && shape_free && bpc == 0 && wpr == 1 && nv <= 4)
        p->grid = looping_grid(rows, cols * (2 * ib + ob), 24 << 10, p->grid, p->block, cus);
      return ROWSM_OK;
    }
  }
  if (variant == ROWSM_LARGE) {
    const int want_split = cfg ? cfg->split_blocks : 0;
    if (want_split >= 0 && !inplace) {
      // 512-thread blocks (measured 0-4% faster than 256 on long rows of
      // every dtype pair with one group per row); few rows as the forward
      // plan, with 256-thread blocks unless a block size is given.
      const bool forced_block = cfg && cfg->block > 0;
      int T = forced_block ? cfg->block : 512;
      int S = want_split > 0 ? want_split : (int)cdiv(nvec, (int64_t)nv_cap * T);
      if (want_split == 0 && !forced_block && rows >= cus && cols * ib <= 4096 * 128) {
        // Rows of at most 512 KiB per input in launches of at least cus
        // rows: 2048 threads per row, 4096 beyond 128 KiB per input, about
        // 32-64 bytes of each input per lane, in 256- and 512-thread blocks
        // (within 3% of the fastest form at 16384-151936 columns and
        // 256-4096 rows; the register-cap plan above was up to 8% slower);
        // a power of two of blocks at least as large as the cap needs.
        const int64_t thr = cols * ib > 2048 * 64 ? 4096 : 2048;
        T = thr <= 2048 ? 256 : 512;
        S = (int)(thr / T);
        const int64_t s_cap = cdiv(nvec, (int64_t)nv_cap * T);
        while (S < s_cap) S <<= 1;
      }
      if (shape.S > 0) {
        S = shape.S;
        T = shape.T;
      }
      if (S < 1) S = 1;
      if (want_split == 0) {
        // (ties go to the few-rows plan, as in the forward)
        const int Tf = forced_block ? T : 256;
        const int sf = few_rows_split(rows, nvec, Tf, nv_cap, cus);
        if (sf > 0 && (int64_t)sf * Tf >= (int64_t)S * T) {
          S = sf;
          T = Tf;
        }
      }
      const int nv = (int)cdiv(nvec, (int64_t)S * T);
      if (S <= 64 && nv <= nv_cap) {
        p->split = S;
        p->nv = nv;
        p->vpl = nv;
        p->block = T;
        p->grid = bpc ? -(int64_t)bpc : 0;  // as the forward plan
        return ROWSM_OK;
      }
      if (want_split > 0) return ROWSM_EINVAL;
    }
    p->split = 0;
    p->u = (cfg && cfg->tile_vectors > 0) ? cfg->tile_vectors : 4;
    p->block = (cfg && cfg->block > 0) ? cfg->block : 1024;
    const int64_t cap = (int64_t)cus * (bpc ? bpc : 1);
    p->grid = rows < cap ? rows : cap;
    p->stream = inplace ? 1 : stream_blocks(rows, nvec, p->block, p->u, bpc, cus);
    return ROWSM_OK;
  }
  return ROWSM_EINVAL;
}

// Plan of the MoE group score over ngroups groups of g scores (g a power of
// two, 2..64): the widest vector (16 or 8 bytes, else one element) that
// divides g and fits the scores' alignment sa; g / vw lanes per group; 4
// groups per lane (cfg->rows_per_lane overrides); 256-thread blocks, one task
// of 64 / (g / vw) * rpl groups per wave (a grid of up to 2^30 blocks; the
// waves stride over any tasks beyond that).  A grid capped at a few blocks
// per compute unit with the waves striding over tasks measured 14% slower on
// the 1048576 x 256 workload; cfg->blocks_per_cu sets such a cap.
int plan_moe(int64_t ngroups, int64_t g, int in_dt, uintptr_t sa, const rowsm_config* cfg,
             int cus, Plan* p) {
  if (!config_in_domain(cfg)) return ROWSM_EINVAL;
  if (cfg && cfg->variant != ROWSM_AUTO && cfg->variant != ROWSM_SMALL) return ROWSM_EINVAL;
  const int ib = dtype_bytes(in_dt);
  int vw = 1;
  for (int w = 16 / ib; w > 1; w >>= 1)
    if (vw_supported(w, ib) && g % w == 0 && sa % (uintptr_t)(w * ib) == 0) {
      vw = w;
      break;
    }
  if (cfg && cfg->vw > 0) {
    const int w = cfg->vw;
    if (!vw_supported(w, ib) || w * ib > 16 || g % w || sa % (uintptr_t)(w * ib))
      return ROWSM_EINVAL;
    vw = w;
  }
  p->variant = ROWSM_SMALL;
  p->vw = vw;
  p->nvec = (int)(g / vw);
  p->lpr = (int)(g / vw);  // lanes per group
  p->rpl = (cfg && cfg->rows_per_lane > 0) ? cfg->rows_per_lane : 4;
  if (small_block(cfg, &p->block) != ROWSM_OK) return ROWSM_EINVAL;
  const int64_t per_task = (int64_t)(kWave / p->lpr) * p->rpl;
  const int64_t tasks = cdiv(ngroups, per_task);
  const int bpc = (cfg && cfg->blocks_per_cu > 0) ? cfg->blocks_per_cu : 0;
  p->grid = cdiv(tasks, p->block / kWave);
  if (p->grid > grid_cap(bpc, cus)) p->grid = grid_cap(bpc, cus);
  return ROWSM_OK;
}

bool moe_group_ok(int64_t g) { return g >= 2 && g <= kWave && (g & (g - 1)) == 0; }

}  // namespace rowsm
