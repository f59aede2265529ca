/*
 * bsm_oracle.c -- fp64 CPU oracle for the batched row softmax.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously correct reference that the HIP
 * path is checked against.  Only the tests, the smoke check and the bench's CPU-baseline leg
 * may load it.  It shares no code, header, table or helper with the HIP library, and the HIP
 * library never loads it.
 *
 * What it computes (problem statement, Section 2 of the paper: softmax run on every R x C
 * slice of a tensor that stacks B slices along rows, laid out as (B*R) x C).  Softmax is
 * taken over the C entries of each row of each slice.  For one row x_0 .. x_{C-1}:
 *
 *     m   = max_j x_j
 *     e_j = exp(x_j - m)                (fp64, libm exp)
 *     S   = sum_j e_j                   (left to right)
 *     y_j = e_j / S
 *
 * Subtracting m leaves the mathematical value unchanged and keeps exp in range.
 *
 * Readings where the paper says nothing:
 *   - a row whose entries are all -inf (a fully masked row) gives y = 0 everywhere;
 *   - any NaN in a row makes the whole row NaN; a +inf entry makes the row NaN (inf - inf);
 *   - an empty slice (R == 0 or C == 0) writes nothing.
 *
 * Backward (the gradient pass: Section 1 notes that these batch algorithms run in the forward
 * and in the backward pass).  With y the softmax of a row and dy the gradient of a loss with
 * respect to y, the gradient with respect to the row's input x is the softmax Jacobian
 * diag(y) - y y^T applied to dy:
 *
 *     d    = sum_j dy_j * y_j           (left to right)
 *     dx_j = y_j * (dy_j - d)
 *
 * No special cases: IEEE arithmetic decides (a NaN anywhere in y or dy makes the whole row NaN
 * through d; a fully masked forward row, y = 0, gives dx = 0).
 *
 * Input element types: fp32, bf16 (raw 16-bit patterns, the top half of an fp32), fp64.
 * All three convert to fp64 exactly.  Output is always fp64, at the same element offsets as
 * the input (gaps between slices are never written).
 *
 * Build: gcc -O2 -std=c99 -fPIC -shared -pthread bsm_oracle.c -o libbsm_oracle.so -lm
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORACLE_F32 = 0, ORACLE_BF16 = 1, ORACLE_F64 = 2 };

/* Exact conversion of element i of a typed buffer to fp64. */
static double load_elem(const void* base, int dtype, int64_t i)
{
    if (dtype == ORACLE_F32) {
        return (double)((const float*)base)[i];
    } else if (dtype == ORACLE_BF16) {
        uint32_t bits = ((uint32_t)((const uint16_t*)base)[i]) << 16;
        float f;
        memcpy(&f, &bits, sizeof f);
        return (double)f;
    }
    return ((const double*)base)[i];
}

/* Softmax of one row of n elements starting at element `first` of `in`, written to
 * y[0 .. n). */
static void softmax_row(const void* in, int dtype, int64_t first, int64_t n, double* y)
{
    int64_t j;
    int has_nan = 0;
    double m = -INFINITY;
    double s = 0.0;

    for (j = 0; j < n; ++j) {
        double x = load_elem(in, dtype, first + j);
        if (isnan(x))
            has_nan = 1;
        if (x > m)
            m = x;
    }
    if (has_nan) {
        for (j = 0; j < n; ++j)
            y[j] = NAN;
        return;
    }
    if (m == -INFINITY) { /* every entry masked */
        for (j = 0; j < n; ++j)
            y[j] = 0.0;
        return;
    }
    for (j = 0; j < n; ++j) {
        double e = exp(load_elem(in, dtype, first + j) - m);
        y[j] = e;
        s += e;
    }
    for (j = 0; j < n; ++j)
        y[j] = y[j] / s;
}

/* Softmax backward of one row of n elements: y and dy start at element `first`; dx[0 .. n). */
static void softmax_backward_row(const void* y, const void* dy, int dtype, int64_t first,
                                 int64_t n, double* dx)
{
    int64_t j;
    double d = 0.0;
    for (j = 0; j < n; ++j)
        d += load_elem(dy, dtype, first + j) * load_elem(y, dtype, first + j);
    for (j = 0; j < n; ++j)
        dx[j] = load_elem(y, dtype, first + j) * (load_elem(dy, dtype, first + j) - d);
}

enum { OP_FORWARD = 0, OP_BACKWARD = 1 };

/* Every row of one slice; `in2` is dy for the backward op (then `in` is y). */
static void run_slice(int op, const void* in, const void* in2, int dtype, int64_t offset,
                      int32_t rows, int32_t cols, double* out)
{
    int32_t r;
    for (r = 0; r < rows; ++r) {
        int64_t first = offset + (int64_t)r * cols;
        if (op == OP_FORWARD)
            softmax_row(in, dtype, first, cols, out + first);
        else
            softmax_backward_row(in, in2, dtype, first, cols, out + first);
    }
}

typedef struct {
    int op;
    const void* in;
    const void* in2;
    int dtype;
    const int64_t* offsets;
    const int32_t* rows;
    const int32_t* cols;
    int64_t s_begin, s_end;
    double* out;
} job_t;

static void* run_job(void* arg)
{
    const job_t* jb = (const job_t*)arg;
    int64_t s;
    for (s = jb->s_begin; s < jb->s_end; ++s)
        run_slice(jb->op, jb->in, jb->in2, jb->dtype, jb->offsets[s], jb->rows[s], jb->cols[s],
                  jb->out);
    return NULL;
}

/* Runs `op` over every row of every slice, split over threads by slice. */
static int run_batched(int op, const void* in, const void* in2, int dtype,
                       const int64_t* offsets, const int32_t* rows, const int32_t* cols,
                       int64_t batch, double* out, int nthreads)
{
    int64_t s, total = 0, acc = 0;
    int t, nt;
    job_t* jobs;
    pthread_t* tids;

    if (batch < 0 || (dtype != ORACLE_F32 && dtype != ORACLE_BF16 && dtype != ORACLE_F64))
        return -1;
    if (batch == 0)
        return 0;
    if (!in || !out || !offsets || !rows || !cols || (op == OP_BACKWARD && !in2))
        return -1;
    for (s = 0; s < batch; ++s) {
        if (rows[s] < 0 || cols[s] < 0 || offsets[s] < 0)
            return -1;
        total += (int64_t)rows[s] * cols[s];
    }
    nt = nthreads < 1 ? 1 : nthreads;
    if (nt > batch)
        nt = (int)batch;
    if (nt == 1) {
        job_t jb = {op, in, in2, dtype, offsets, rows, cols, 0, batch, out};
        run_job(&jb);
        return 0;
    }
    jobs = (job_t*)calloc((size_t)nt, sizeof(job_t));
    tids = (pthread_t*)calloc((size_t)nt, sizeof(pthread_t));
    if (!jobs || !tids) {
        free(jobs);
        free(tids);
        return -1;
    }
    /* Thread t takes the slices whose cumulative element count falls in its share. */
    s = 0;
    for (t = 0; t < nt; ++t) {
        int64_t limit = (total * (t + 1)) / nt;
        jobs[t] = (job_t){op, in, in2, dtype, offsets, rows, cols, s, s, out};
        while (s < batch && (acc < limit || t == nt - 1)) {
            acc += (int64_t)rows[s] * cols[s];
            ++s;
        }
        jobs[t].s_end = s;
    }
    for (t = 0; t < nt; ++t)
        if (pthread_create(&tids[t], NULL, run_job, &jobs[t]) != 0)
            run_job(&jobs[t]), tids[t] = 0;
    for (t = 0; t < nt; ++t)
        if (tids[t])
            pthread_join(tids[t], NULL);
    free(jobs);
    free(tids);
    return 0;
}

/*
 * Row softmax of every row of every slice.
 *   in       typed input (dtype 0 = fp32, 1 = bf16 bits, 2 = fp64), indexed by element
 *   offsets  [batch] element offset of slice s (only offsets[0 .. batch-1] are read)
 *   rows     [batch] R_s;  cols [batch] C_s   (row r of slice s starts at offsets[s] + r*C_s)
 *   out      fp64 output, same element indexing as `in`
 *   nthreads >= 1; slices are split into contiguous groups of about equal element count
 * Returns 0, or -1 on a bad argument (nothing written).
 */
int bsm_oracle_softmax(const void* in, int dtype, const int64_t* offsets,
                       const int32_t* rows, const int32_t* cols, int64_t batch,
                       double* out, int nthreads)
{
    return run_batched(OP_FORWARD, in, NULL, dtype, offsets, rows, cols, batch, out, nthreads);
}

/*
 * Softmax backward of every row of every slice: dx from the forward output y and the gradient
 * dy (same dtype, same element indexing), written as fp64 at the same element offsets.
 * Arguments and return value as for bsm_oracle_softmax.
 */
int bsm_oracle_softmax_backward(const void* y, const void* dy, int dtype,
                                const int64_t* offsets, const int32_t* rows,
                                const int32_t* cols, int64_t batch, double* dx, int nthreads)
{
    return run_batched(OP_BACKWARD, y, dy, dtype, offsets, rows, cols, batch, dx, nthreads);
}

/*
 * Softmax of selected rows only (for checks on sampled outputs of very large inputs).
 *   row_first[i]  element offset of sampled row i in `in`;  row_cols[i] its length
 *   out           fp64, rows packed back to back in sample order
 * Returns 0, or -1 on a bad argument.
 */
int bsm_oracle_softmax_rows(const void* in, int dtype, const int64_t* row_first,
                            const int32_t* row_cols, int64_t nrows, double* out)
{
    int64_t i, pos = 0;
    if (nrows < 0 || (dtype != ORACLE_F32 && dtype != ORACLE_BF16 && dtype != ORACLE_F64))
        return -1;
    if (nrows == 0)
        return 0;
    if (!in || !out || !row_first || !row_cols)
        return -1;
    for (i = 0; i < nrows; ++i) {
        if (row_first[i] < 0 || row_cols[i] < 0)
            return -1;
    }
    for (i = 0; i < nrows; ++i) {
        softmax_row(in, dtype, row_first[i], row_cols[i], out + pos);
        pos += row_cols[i];
    }
    return 0;
}

/*
 * Softmax backward of selected rows only: row i has row_cols[i] elements starting at element
 * row_first[i] of y and of dy; dx rows packed back to back in sample order.
 * Returns 0, or -1 on a bad argument.
 */
int bsm_oracle_softmax_backward_rows(const void* y, const void* dy, int dtype,
                                     const int64_t* row_first, const int32_t* row_cols,
                                     int64_t nrows, double* dx)
{
    int64_t i, pos = 0;
    if (nrows < 0 || (dtype != ORACLE_F32 && dtype != ORACLE_BF16 && dtype != ORACLE_F64))
        return -1;
    if (nrows == 0)
        return 0;
    if (!y || !dy || !dx || !row_first || !row_cols)
        return -1;
    for (i = 0; i < nrows; ++i) {
        if (row_first[i] < 0 || row_cols[i] < 0)
            return -1;
    }
    for (i = 0; i < nrows; ++i) {
        softmax_backward_row(y, dy, dtype, row_first[i], row_cols[i], dx + pos);
        pos += row_cols[i];
    }
    return 0;
}
