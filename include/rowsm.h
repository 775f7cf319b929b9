/*
 * rowsm.h -- C ABI of the MI355X (gfx950) row-softmax library.
 *
 * The operation is the numerically stable softmax over the last dimension of a
 * row-major matrix:
 *
 *     y[r, j] = exp(x[r, j] - m_r) / sum_k exp(x[r, k] - m_r),  m_r = max_k x[r, k]
 *
 * The paper names this hot path only through its running-example listing
 * style, which declares a row-length-specialised reduction with small-, medium-
 * and large-row kernels, a row-count launcher and a BLOCK_ROWS tile parameter
 * (preamble listing style for the running example); its benchmark operators
 * are all checked against a PyTorch reference (Evaluation, Experimental
 * Setup), whose softmax over dim -1 is the formula above.  The kernels and the
 * dispatcher behind this header are this library's own gfx950 design.
 *
 * Conventions shared by every entry point
 *   - x and y are DEVICE pointers owned by the caller; the library never frees
 *     or retains them.  Layout: row-major, contiguous, row stride == cols
 *     elements.  x is only read.  y may equal x (in place) when in_dtype ==
 *     out_dtype; any other overlap of the two ranges is rejected.
 *   - dtypes: ROWSM_F32 (IEEE binary32) or ROWSM_BF16 (bfloat16, stored as
 *     its 16-bit pattern).  Every pair {f32, bf16} x {f32, bf16} is supported.
 *     Arithmetic is fp32: bf16 inputs widen exactly, bf16 outputs are rounded
 *     to nearest even.
 *   - stream is a hipStream_t (NULL = the legacy default stream).  The call
 *     only enqueues work on that stream; results are visible once the caller
 *     synchronises it.  No call waits for, or is ordered after, work on any
 *     other stream.  Nothing is allocated per call.  The forms whose blocks
 *     exchange partial results (LARGE with split > 0 in rowsm_describe, or
 *     the two-pass form with several blocks per row) take a region of a
 *     64 MiB exchange ring per device: the library's static device array,
 *     zero when the library's device code is loaded, so the first such call
 *     allocates, clears and waits for nothing either.  After 2^30 rows of
 *     exchanging launches on a device the ring is replaced by a 64 MiB
 *     allocation that the library clears on a private stream of its own and
 *     waits for (outside stream capture only); replaced rings stay allocated
 *     until the process ends.
 *   - Exchanging forms never depend on timing for their results: a block
 *     whose wait for another block's partial result gives up (after about
 *     0.1 s, rowsm_set_split_wait_limit()) computes that partial itself from
 *     the input and the row comes out bit for bit as it would have, so a
 *     launch finishes with the right result whatever else runs on the
 *     device.  rowsm_split_wait_failures() counts such give-ups.  An
 *     in-place call (y == x) is never planned on an exchanging form.
 *   - Errors are reported through the return value only (a rowsm_status);
 *     the library never aborts, prints or throws.  Argument errors are found
 *     on the host before any HIP call.  A failed launch maps to ROWSM_EHIP.
 *   - Special values follow IEEE arithmetic of the formula: a row holding a
 *     NaN or +inf, or only -inf, is all NaN; a -inf entry in a row with a
 *     finite maximum gives exactly +0.
 *   - Limits: rows * cols < 2^62 and cols < 2^30 (every byte offset inside a
 *     row fits 32 bits); larger sizes return ROWSM_EINVAL.
 */
#ifndef ROWSM_H
#define ROWSM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { ROWSM_F32 = 0, ROWSM_BF16 = 1 } rowsm_dtype;

typedef enum {
    ROWSM_OK = 0,
    ROWSM_EINVAL = -1, /* bad size, NULL pointer, bad overlap, bad variant  */
    ROWSM_EDTYPE = -2, /* dtype code outside rowsm_dtype                    */
    ROWSM_EHIP = -3    /* the HIP runtime reported an error for the launch  */
} rowsm_status;

/* Kernel families.  SMALL packs several rows into one 64-lane wavefront;
 * MEDIUM gives each row one workgroup (or one wavefront) and keeps the row in
 * registers; LARGE spreads a row over several workgroups that keep their
 * shares in registers and exchange (max, sum) pairs through the device
 * workspace (single read), or, for rows too long for that,
 * streams the row through tiles twice (online max/sum pass, then normalize),
 * over one block per row for many rows and over up to 256 blocks per row,
 * which exchange their pairs the same way, for few.  Both launch one group
 * of blocks per row; with cfg->blocks_per_cu given, the single-read form
 * launches one residency of the device whose groups loop over the rows, and
 * the two-pass form one block per row.
 *
 * HIP graphs: every entry point may be called on a stream that is being
 * captured, from the first call on, and keeps its plan.  A captured
 * exchanging launch records, before its kernel, a small kernel that clears
 * the launch's region of the exchange ring, so that every replay starts from
 * cleared exchange words (a replay reuses the region and the tags recorded
 * at capture).  Graph executables that contain the same captured launch
 * (e.g. two instantiations of one graph) must not run at the same time.  No
 * entry point records a memset or an allocation into a capture. */
typedef enum {
    ROWSM_AUTO = 0,
    ROWSM_SMALL = 1,
    ROWSM_MEDIUM = 2,
    ROWSM_LARGE = 3
} rowsm_variant;

/* Operations, for rowsm_describe_op. */
typedef enum {
    ROWSM_OP_SOFTMAX = 0,          /* rowsm_forward, rowsm_forward_config      */
    ROWSM_OP_SCALED_CAUSAL = 1,    /* rowsm_forward_scaled_causal              */
    ROWSM_OP_LOG_SOFTMAX = 2,      /* rowsm_log_softmax                        */
    ROWSM_OP_SOFTMAX_BACKWARD = 3, /* rowsm_softmax_backward                   */
    ROWSM_OP_MOE_GROUP_TOP2 = 4    /* rowsm_moe_group_top2: rows = number of
                                      groups, cols = group size               */
} rowsm_op;

/*
 * rowsm_forward: y = softmax(x, dim=-1) for a rows x cols matrix.
 *   x         device pointer, rows*cols elements of in_dtype
 *   y         device pointer, rows*cols elements of out_dtype
 *   rows      >= 0; rows == 0 or cols == 0 is a no-op returning ROWSM_OK
 *   cols      >= 0
 *   in_dtype  rowsm_dtype of x;  out_dtype rowsm_dtype of y
 *   stream    hipStream_t the kernel is enqueued on
 * Returns ROWSM_OK or a negative rowsm_status.  The kernel family is chosen
 * by rowsm_select.
 */
int rowsm_forward(const void *x, void *y, int64_t rows, int64_t cols,
                  int in_dtype, int out_dtype, void *stream);

/*
 * rowsm_select: the kernel family rowsm_forward uses for this shape and dtype
 * pair (the row-count and row-length launcher).  Pure host function, no HIP
 * call.  Returns a rowsm_variant > 0, or a negative rowsm_status for invalid
 * arguments.
 */
int rowsm_select(int64_t rows, int64_t cols, int in_dtype, int out_dtype);

/*
 * rowsm_forward_noalloc: rowsm_forward for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same operation, launcher and kernels, but it
 * never calls hipMalloc, hipFree or any other allocating routine, on any
 * call.  The exchange words of the forms whose blocks share a row live in
 * the library's static device array `scratch` (4 MiB per device, 32 bytes
 * per block, 2^17 blocks), set up on the first call on each device; a launch
 * whose row groups would need more blocks than that loops them over the
 * rows instead, so no shape exceeds it (a launch that still would returns
 * ROWSM_EINVAL without launching).  Each launch of those forms first clears
 * its region of the array with a small kernel on `stream`.  Every call on a
 * device shares the array, which keeps the last call's words: calls that
 * overlap in time on one device may take the same words and slow each other
 * down (a block recomputes what it finds cleared or overwritten), never
 * change each other's results.  Arguments, results and errors as
 * rowsm_forward.
 */
int rowsm_forward_noalloc(const void *x, void *y, int64_t rows, int64_t cols,
                          int in_dtype, int out_dtype, void *stream);

/*
 * rowsm_forward_variant: rowsm_forward with the kernel family forced
 * (ROWSM_AUTO behaves like rowsm_forward).  Used by tests and benchmarks to
 * check every family on every shape it supports.  A family that cannot run
 * this shape (SMALL or MEDIUM with a row too long for registers) returns
 * ROWSM_EINVAL without launching.
 */
int rowsm_forward_variant(const void *x, void *y, int64_t rows, int64_t cols,
                          int in_dtype, int out_dtype, void *stream,
                          int variant);

/*
 * rowsm_config: launch overrides for rowsm_forward_config.  Every field left
 * at 0 (packed: -1) takes the launcher's default for the chosen family.
 */
typedef struct rowsm_config {
    int32_t variant;        /* rowsm_variant; ROWSM_AUTO = launcher's choice      */
    int32_t vw;             /* elements per vector access: power of two that
                               divides cols, <= 16 bytes of input, with x and y
                               aligned to it; or, for a width it does not
                               divide, the full 16-byte width with x and y
                               aligned to 16 bytes: variant SMALL the flat
                               form (rows read as one stream of whole vectors,
                               at most 1024 columns and 4 vectors per lane of
                               a tile; also the backward), AUTO or MEDIUM the
                               ragged form (softmax and log-softmax only)      */
    int32_t lanes_per_row;  /* SMALL: lanes holding one row, power of two <= 32;
                               the flat form: lanes per row of its row phase
                               (4 with 4 elements, 8 with 2-8, 16-32 with 8,
                               64 with 8 or 16 elements per lane)              */
    int32_t rows_per_lane;  /* SMALL: rows each lane handles per pass: 1,2,4,8;
                               the flat form: 16-byte vectors per lane of a
                               tile, 4, or 2 for bf16 to bf16 rows that fit   */
    int32_t waves_per_row;  /* MEDIUM: wavefronts holding one row: 1,2,4,8,16     */
    int32_t rows_per_block; /* MEDIUM: rows per block (rows*waves_per_row <= 16)  */
    int32_t packed;         /* MEDIUM: 1 keep raw bf16 and recompute exp,
                               0 keep fp32 exp values, -1 launcher's choice       */
    int32_t block;          /* LARGE: threads per block, multiple of 64, <= 1024;
                               SMALL and the MoE score: 64, 128 or 256           */
    int32_t tile_vectors;   /* LARGE: vectors per thread per tile: 2, 4, 8        */
    int32_t blocks_per_cu;  /* grid cap = blocks_per_cu * compute units           */
    int32_t split_blocks;   /* LARGE: blocks sharing one row in the single-read
                               form (1..64), 0 launcher's choice, -1 the
                               two-pass streaming form; > 0 in place is
                               ROWSM_EINVAL (no exchanging form in place)         */
    int32_t prefetch;       /* LARGE single-read form: 1 load a block's next row
                               while the current one is exchanged and written
                               (software pipelining; at most 48 values per lane,
                               44 for fp32 input), -1 never, 0 launcher's
                               choice                                             */
} rowsm_config;

/*
 * rowsm_forward_config: rowsm_forward with explicit launch overrides (kernel
 * family, vector width, lane/wave grouping, tile size, grid cap), for tuning
 * sweeps and tests.  cfg == NULL behaves like rowsm_forward.  An override the
 * family cannot honour returns ROWSM_EINVAL without launching.  Results are
 * the same softmax for every accepted configuration.
 */
int rowsm_forward_config(const void *x, void *y, int64_t rows, int64_t cols,
                         int in_dtype, int out_dtype, void *stream,
                         const rowsm_config *cfg);

/*
 * rowsm_forward_scaled_causal: y = softmax(scale * x + mask, dim=-1), the
 * scaled and causally masked attention-score form of the operation:
 *     mask(r, c) = -inf   when causal_period > 0 and
 *                         c > (r mod causal_period) + causal_offset,
 *                  0      otherwise.
 * Row r is query r mod causal_period of its group; causal_offset shifts the
 * diagonal (0: query q sees keys 0..q; cols - causal_period: keys aligned to
 * the end).  causal_period == 0 disables the mask (scale only); < 0 returns
 * ROWSM_EINVAL.  Masked columns are never read and are written as exact
 * zeros; a row whose every column is masked is all NaN, as the plain
 * operation gives for an all -inf row.  scale * x is formed in fp32 (any
 * scale; IEEE semantics for zero, infinite or NaN products).  Other
 * arguments, layout and errors as rowsm_forward; cfg (NULL = launcher's
 * choice) as rowsm_forward_config, except that the packed medium form and
 * rows_per_lane other than 4 are not available here.
 */
int rowsm_forward_scaled_causal(const void *x, void *y, int64_t rows, int64_t cols,
                                int in_dtype, int out_dtype, float scale,
                                int64_t causal_period, int64_t causal_offset,
                                void *stream, const rowsm_config *cfg);

/*
 * rowsm_log_softmax: y = log(softmax(x, dim=-1)), written as
 *     y[r, j] = (x[r, j] - m_r) - ln(sum_k exp(x[r, k] - m_r)),  m_r = max_k x[r, k]
 * (the logarithm of the operation above, never formed as log of a quotient,
 * so entries far below the maximum keep their value instead of underflowing
 * to log(0)).  This is the cross-entropy input form of the operation; it is
 * not part of the paper's operator set and follows the textbook definition.
 * Special values: a row holding NaN or +inf, or only -inf, is all NaN; a -inf
 * entry in a row with a finite maximum gives -inf.  Arguments, layout,
 * dtypes, aliasing, errors and cfg as rowsm_forward_config (NULL cfg = the
 * launcher's choice; every family and form of the plain operation is
 * available).  fp32 accumulation; y in out_dtype.
 */
int rowsm_log_softmax(const void *x, void *y, int64_t rows, int64_t cols, int in_dtype,
                      int out_dtype, void *stream, const rowsm_config *cfg);

/*
 * rowsm_softmax_backward: the gradient of softmax over the last dimension,
 *     dx[r, j] = y[r, j] * (dy[r, j] - sum_k y[r, k] * dy[r, k]),
 * i.e. the softmax Jacobian diag(y_r) - y_r y_r^T applied to dy_r, where y is
 * the forward output and dy the gradient of a loss with respect to y (the
 * textbook derivative of the operation; not part of the paper's operator
 * set).
 *   y, dy     device pointers, rows*cols elements of in_dtype each, row-major
 *             and contiguous (row stride cols); read only; they may overlap
 *             each other (even be the same buffer)
 *   dx        device pointer, rows*cols elements of out_dtype; it may be y or
 *             dy itself when in_dtype == out_dtype (in place), but must not
 *             overlap either in any other way (ROWSM_EINVAL)
 *   stream, rows, cols, dtypes, limits, errors: as rowsm_forward
 *   cfg       NULL = the launcher's choice; otherwise as rowsm_forward_config
 *             with these differences: y and dy are held in their raw form
 *             (packed = 1 is ROWSM_EINVAL), a lane holds at most 128 bytes of
 *             each input, and the single-read LARGE form uses 512-thread
 *             blocks (256 for few rows) unless block is given.
 * The dot product is accumulated in fp32 (fma), in a fixed order: results are
 * deterministic for a given launch shape.  Special values follow IEEE
 * arithmetic in the formula above: a NaN in y or dy makes the dot product,
 * and with it the whole row of dx, NaN; an infinite product makes it +-inf
 * (or NaN), and dx follows from the formula (e.g. -inf where y > 0, NaN where
 * y == 0 or at the infinite entry).  y == 0 with a finite dot product gives
 * an exact zero.  The exchanging LARGE forms share the forward's device
 * workspace and behave as the forward's (see rowsm_split_wait_failures); dx
 * equal to y or dy is never planned on them.
 */
int rowsm_softmax_backward(const void *y, const void *dy, void *dx, int64_t rows, int64_t cols,
                           int in_dtype, int out_dtype, void *stream, const rowsm_config *cfg);

/*
 * rowsm_moe_group_top2: the MoE group score of the paper's running example
 * (Motivation section and the figure of its source rewrite).  The experts
 * scores of each token are cut into consecutive groups of group_size; the
 * score of a group is the sum of its two largest values counted with
 * multiplicity (a maximum that occurs twice counts twice), which the paper
 * shows equals max over i != j of v_i + v_j:
 *     group_scores[t, g] = top1 + top2 of scores[t, g*G .. g*G + G - 1]
 *   scores        device pointer, tokens x experts of in_dtype, row-major and
 *                 contiguous; read only
 *   group_scores  device pointer, tokens x (experts / group_size) of
 *                 out_dtype, aligned to its element size; must not overlap
 *                 scores (ROWSM_EINVAL)
 *   group_size    a power of two from 2 to 64 that divides experts, else
 *                 ROWSM_EINVAL (the paper's operator uses 32)
 *   stream, dtypes, errors: as rowsm_forward; tokens * experts < 2^62
 *   cfg           NULL = the launcher's choice; only variant (AUTO or SMALL),
 *                 vw, rows_per_lane (groups per lane: 1, 2, 4, 8) and
 *                 blocks_per_cu are used
 * The sum is one fp32 addition of the two stored values, rounded to
 * out_dtype (nearest, ties to even, for bf16).  A NaN anywhere in a group
 * makes its score NaN; infinities follow IEEE addition (+inf + -inf = NaN).
 * Results do not depend on the launch shape.
 */
int rowsm_moe_group_top2(const void *scores, void *group_scores, int64_t tokens,
                         int64_t experts, int64_t group_size, int in_dtype, int out_dtype,
                         void *stream, const rowsm_config *cfg);

/*
 * rowsm_describe_op: as rowsm_describe for any operation (op: rowsm_op) and
 * launch overrides cfg (NULL = the launcher's choice).  Returns the status the
 * operation would return for these arguments with valid, 256-byte aligned
 * pointers; ROWSM_EINVAL for an unknown op.
 */
int rowsm_describe_op(int op, int64_t rows, int64_t cols, int in_dtype, int out_dtype,
                      const rowsm_config *cfg, char *buf, int64_t len);

/*
 * rowsm_describe: writes into buf (capacity len, always NUL-terminated when
 * len > 0) a one-line description of the launch rowsm_forward_variant would
 * make: kernel family, template configuration, grid and block sizes.  Pure
 * host function.  Returns the status rowsm_forward_variant would return for
 * these arguments with valid pointers.
 */
int rowsm_describe(int64_t rows, int64_t cols, int in_dtype, int out_dtype,
                   int variant, char *buf, int64_t len);

/*
 * rowsm_split_wait_failures: diagnostics of the exchanging forms on the
 * current device: how many exchange waits have given up since the library's
 * device code was loaded (each one made a block recompute another block's
 * partial result from the input: the results are unaffected, the launch was
 * slower), 0 when no exchanging launch has run, or ROWSM_EHIP.  It first
 * synchronises the device (hipDeviceSynchronize): not to be called while a
 * stream capture is in progress.
 */
int64_t rowsm_split_wait_failures(void);

/*
 * rowsm_set_split_wait_limit: sets how many times an exchange wait polls for
 * another block's partial result before it gives up and recomputes it (for
 * launches made after the call, on every device); polls < 0 restores the
 * default (2^16, about 0.1 s), 0 makes every wait give up at once.  Results
 * are the same for any limit; the setting exists so that tests can drive the
 * recomputation.  Returns the previous limit.  Pure host function.
 */
int64_t rowsm_set_split_wait_limit(int64_t polls);

/*
 * rowsm_stream_copy: y[i] = x[i] converted from in_dtype to out_dtype, for
 * i < n.  Not an operation of the method: a measurement aid.  It moves the
 * bytes a row operation of the same dtype pair moves (every input byte read
 * once, every output byte written once) in the access pattern that streams
 * fastest on this device (one vector of at most 16 bytes per thread, each
 * workgroup one contiguous chunk, non-temporal accesses), and benchmarks time
 * it beside each row kernel as that workload's practical HBM ceiling.
 *   x, y      device pointers to n elements of in_dtype / out_dtype, aligned
 *             to their element size; y may equal x when the dtypes are equal,
 *             any other overlap is rejected
 *   n         >= 0 (n == 0: no launch), at most 2^60
 *   stream    hipStream_t the kernel is enqueued on
 * Conversion: bf16 -> f32 exact; f32 -> bf16 round to nearest even.
 * Returns ROWSM_OK, ROWSM_EDTYPE, ROWSM_EINVAL (checked before any HIP call)
 * or ROWSM_EHIP.
 */
int rowsm_stream_copy(const void *x, void *y, int64_t n, int in_dtype, int out_dtype,
                      void *stream);

/* rowsm_status_string: static, human-readable text for a rowsm_status. */
const char *rowsm_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* ROWSM_H */
