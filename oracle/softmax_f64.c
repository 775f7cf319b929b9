/*
 * Row softmax oracle in fp64 -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
 * build, load or call this file.  The product path (the HIP library) shares no
 * code, header, table or constant with it, and must never fall back to it.
 *
 * What it computes: for every row r of a row-major rows x cols matrix,
 *
 *     m_r    = max_j x[r, j]
 *     e[r,j] = exp(x[r, j] - m_r)
 *     s_r    = sum_j e[r, j]              (sequential, in column order)
 *     y[r,j] = e[r, j] / s_r
 *
 * This is the textbook numerically stable softmax over the last dimension.  The
 * paper never writes the formula: it names a row-length-specialised reduction
 * (small-, medium- and large-row kernels plus a row-count launcher, in the
 * listing style declared in its preamble for the running example), and every
 * benchmark operator it optimises is judged against a PyTorch reference
 * implementation (Evaluation, Experimental Setup).  PyTorch's softmax over
 * dim -1 is exactly the definition above.
 *
 * Special values follow from IEEE arithmetic with no extra case:
 *   - a NaN entry is skipped by the max, but exp(NaN - m) = NaN makes s_r and
 *     then every y[r, :] NaN;
 *   - a +inf entry gives m_r = +inf, inf - inf = NaN, so the row is NaN;
 *   - an all -inf row gives -inf - (-inf) = NaN, so the row is NaN;
 *   - a -inf entry in a row with finite max gives exp(-inf) = +0 exactly.
 *
 * Build flags must keep IEEE semantics: no -ffast-math, -ffp-contract=off.
 * Rows are independent and each is computed serially, so the result is the
 * same for every thread count.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>

/* One row: max, exponentials and their sum, division (definition above). */
static void oracle_row(const double *x, double *y, int64_t cols)
{
    double m = -INFINITY;
    for (int64_t j = 0; j < cols; ++j)
        if (x[j] > m)
            m = x[j];

    /* The max is still -inf for a row of -inf only; subtracting it then
     * yields NaN, the IEEE value of the definition. */
    double s = 0.0;
    for (int64_t j = 0; j < cols; ++j) {
        double e = exp(x[j] - m);
        y[j] = e;
        s += e;
    }
    for (int64_t j = 0; j < cols; ++j)
        y[j] = y[j] / s;
}

/*
 * Log-softmax of one row: y_j = x_j - m - log(sum_k exp(x_k - m)), i.e. the
 * logarithm of the softmax above written without forming the quotient (its
 * tiny entries would underflow).  Same special values: a NaN or +inf entry,
 * or a row of only -inf, gives an all-NaN row; a -inf entry in a row with a
 * finite maximum gives -inf.
 */
static void oracle_row_log(const double *x, double *y, int64_t cols)
{
    double m = -INFINITY;
    for (int64_t j = 0; j < cols; ++j)
        m = fmax(m, x[j]); /* fmax skips a NaN operand, as the comparison above */
    double sum_e = 0.0;
    for (int64_t j = 0; j < cols; ++j)
        sum_e += exp(x[j] - m);
    double lse = m + log(sum_e);
    for (int64_t j = 0; j < cols; ++j)
        y[j] = x[j] - lse;
}

/*
 * Softmax backward of one row: given y = softmax(x) and the gradient dy of a
 * loss with respect to y, dx_j = y_j * (dy_j - sum_k y_k dy_k).  This is the
 * product of the softmax Jacobian (diag(y) - y y^T, symmetric) with dy,
 * written out.
 */
static void oracle_row_backward(const double *yv, const double *dy, double *dx, int64_t cols)
{
    double dot = 0.0;
    for (int64_t k = 0; k < cols; ++k)
        dot += yv[k] * dy[k];
    for (int64_t j = 0; j < cols; ++j)
        dx[j] = yv[j] * (dy[j] - dot);
}

/*
 * Scaled, causally masked rows (attention scores): row r is treated as query
 * q = r mod period, and column c survives when c <= q + offset; the others
 * are -inf.  The row is t_j = scale * x_j for surviving columns, -inf
 * otherwise, and the result is the plain definition above applied to t.
 * period == 0 means no mask.  Written out element by element into a scratch
 * row so that the definition above is applied unchanged.
 */
static void oracle_row_scaled_causal(const double *x, double *y, double *t, int64_t r,
                                     int64_t cols, double scale, int64_t period,
                                     int64_t offset)
{
    for (int64_t j = 0; j < cols; ++j) {
        int masked = period > 0 && j > (r % period) + offset;
        t[j] = masked ? -INFINITY : scale * x[j];
    }
    oracle_row(t, y, cols);
}

enum { ORACLE_SOFTMAX = 0, ORACLE_FUSED = 1, ORACLE_LOG = 2, ORACLE_BACKWARD = 3 };

struct oracle_job {
    const double *x;   /* backward: y */
    double *y;         /* backward: dx */
    int64_t row_begin, row_end, cols;
    int kind;
    double scale;
    int64_t period, offset;
    const double *dy;  /* backward only */
};

static void *oracle_worker(void *arg)
{
    const struct oracle_job *job = (const struct oracle_job *)arg;
    double *t = NULL;
    if (job->kind == ORACLE_FUSED) {
        t = (double *)malloc((size_t)job->cols * sizeof(double));
        if (!t)
            return NULL; /* rows stay unwritten; the wrapper fills NaN first */
    }
    for (int64_t r = job->row_begin; r < job->row_end; ++r) {
        const int64_t o = r * job->cols;
        if (job->kind == ORACLE_FUSED)
            oracle_row_scaled_causal(job->x + o, job->y + o, t, r, job->cols, job->scale,
                                     job->period, job->offset);
        else if (job->kind == ORACLE_LOG)
            oracle_row_log(job->x + o, job->y + o, job->cols);
        else if (job->kind == ORACLE_BACKWARD)
            oracle_row_backward(job->x + o, job->dy + o, job->y + o, job->cols);
        else
            oracle_row(job->x + r * job->cols, job->y + r * job->cols, job->cols);
    }
    free(t);
    return NULL;
}

/* Row-parallel driver shared by both entry points. */
static int oracle_run(struct oracle_job proto, int64_t rows, int threads)
{
    if (threads <= 1 || rows == 1) {
        proto.row_begin = 0;
        proto.row_end = rows;
        oracle_worker(&proto);
        return 0;
    }
    if (threads > rows)
        threads = (int)rows;

    pthread_t *tid = (pthread_t *)calloc((size_t)threads, sizeof(pthread_t));
    struct oracle_job *jobs =
        (struct oracle_job *)calloc((size_t)threads, sizeof(struct oracle_job));
    if (!tid || !jobs) {
        free(tid);
        free(jobs);
        return -2;
    }
    for (int t = 0; t < threads; ++t) {
        jobs[t] = proto;
        jobs[t].row_begin = rows * t / threads;
        jobs[t].row_end = rows * (t + 1) / threads;
    }
    int started = 0;
    while (started < threads &&
           pthread_create(&tid[started], NULL, oracle_worker, &jobs[started]) == 0)
        ++started;
    for (int t = started; t < threads; ++t) /* rows whose thread never started */
        oracle_worker(&jobs[t]);
    for (int t = 0; t < started; ++t)
        pthread_join(tid[t], NULL);
    free(tid);
    free(jobs);
    return 0;
}

/*
 * oracle_softmax_f64: y = softmax(x, dim=-1) for a rows x cols fp64 matrix.
 * x, y: host pointers, row-major, contiguous, rows*cols doubles each, distinct.
 * threads: worker threads (<= 0 means 1); rows are split into contiguous
 * blocks, and rows whose thread cannot be started are done on the caller's
 * thread.  Returns 0 on success, -1 on bad arguments, -2 when the thread
 * bookkeeping cannot be allocated.
 */
int oracle_softmax_f64(const double *x, double *y, int64_t rows, int64_t cols,
                       int threads)
{
    if (rows < 0 || cols < 0)
        return -1;
    if (rows == 0 || cols == 0)
        return 0;
    if (!x || !y)
        return -1;
    struct oracle_job proto = {x, y, 0, 0, cols, ORACLE_SOFTMAX, 1.0, 0, 0, NULL};
    return oracle_run(proto, rows, threads);
}

/*
 * oracle_softmax_scaled_causal_f64: y = softmax(scale * x + mask, dim=-1),
 * mask(r, c) = -inf when period > 0 and c > (r mod period) + offset, else 0
 * (see oracle_row_scaled_causal).  Same arguments and return codes as
 * oracle_softmax_f64, plus scale, period (>= 0) and offset.
 */
int oracle_softmax_scaled_causal_f64(const double *x, double *y, int64_t rows,
                                     int64_t cols, double scale, int64_t period,
                                     int64_t offset, int threads)
{
    if (rows < 0 || cols < 0 || period < 0)
        return -1;
    if (rows == 0 || cols == 0)
        return 0;
    if (!x || !y)
        return -1;
    struct oracle_job proto = {x, y, 0, 0, cols, ORACLE_FUSED, scale, period, offset, NULL};
    return oracle_run(proto, rows, threads);
}

/*
 * oracle_log_softmax_f64: y = log_softmax(x, dim=-1) (oracle_row_log).  Same
 * arguments and return codes as oracle_softmax_f64.
 */
int oracle_log_softmax_f64(const double *x, double *y, int64_t rows, int64_t cols,
                           int threads)
{
    if (rows < 0 || cols < 0)
        return -1;
    if (rows == 0 || cols == 0)
        return 0;
    if (!x || !y)
        return -1;
    struct oracle_job proto = {x, y, 0, 0, cols, ORACLE_LOG, 1.0, 0, 0, NULL};
    return oracle_run(proto, rows, threads);
}

/*
 * oracle_softmax_backward_f64: dx = y * (dy - rowsum(y * dy)) for rows x cols
 * fp64 matrices y, dy, dx (oracle_row_backward).  Return codes as above.
 */
int oracle_softmax_backward_f64(const double *y, const double *dy, double *dx, int64_t rows,
                                int64_t cols, int threads)
{
    if (rows < 0 || cols < 0)
        return -1;
    if (rows == 0 || cols == 0)
        return 0;
    if (!y || !dy || !dx)
        return -1;
    struct oracle_job proto = {y, dx, 0, 0, cols, ORACLE_BACKWARD, 1.0, 0, 0, dy};
    return oracle_run(proto, rows, threads);
}
