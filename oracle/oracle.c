/*
 * oracle.c -- plain CPU oracle for the sparse DNN forward pass.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the reference the GPU library is checked
 * against.  Only the test suite, the smoke check and the CPU-baseline leg of
 * the benchmark load it; the library itself never does, and the two share no
 * code.
 *
 * What it computes (Kepner et al., "Enabling Massive Deep Neural Networks with
 * the GraphBLAS", arXiv:1708.02937):
 *   Sec. III, batched inference:  Y_{k+1} = h(W_k Y_k + B_k), B_k = b_k
 *                                 replicated along the batch;
 *   Sec. III, ReLU:               h(y) = max(y, 0).
 * It is written in the transposed orientation Y_{k+1} = h(Y_k W_k + 1 b_k^T):
 * Y is batch x n (one sample per row) and W_k is stored n_in x n_out in CSR,
 * so row i of W_k is the fan-out of input neuron i.  The optional clamp
 * h(y) = min(max(y, 0), ymax) generalises the ReLU (ymax = +inf is the
 * paper's h).  Bias placement has two readings, chosen per call:
 *   bias_mode 0 (default): the bias is added at every position, as the dense
 *     equation states, including positions that receive no product;
 *   bias_mode 1: the bias is added only where Y_k W_k has a structural entry,
 *     the pattern semantics of Fig. 4 (Sec. IV): eWiseMult over max.+ with the
 *     bias matrix keeps only the entries both operands store, and eWiseAdd
 *     with the all-zero matrix leaves 0 elsewhere.  A position is structural
 *     when some stored entry W(i, j) meets a nonzero Y(r, i): activations are
 *     stored as their nonzeros (zeros pruned after every layer), W as its CSR.
 *
 * Arithmetic: the product of two fp32 values is exact in fp64; the products of
 * one output entry are summed in fp64 in ascending order of the sample's
 * nonzero index, the bias is added in fp64, ReLU and clamp are applied in
 * fp64, and the result is rounded once (round to nearest even) to fp32.  That
 * fp32 value is the next layer's input.  Entries equal to zero (-0 included)
 * are not stored (Sec. II, 0-element: it is the additive identity and the
 * multiplicative annihilator, so absent entries contribute nothing).
 *
 * Rows of Y are independent through all layers, so host threads split them.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    const int64_t *row_ptr; /* n + 1 entries */
    const int32_t *col;     /* nnz, ascending within a row, in [0, n) */
    const float *val;       /* nnz */
    const float *bias;      /* n */
} oracle_layer;

typedef struct {
    int64_t n;
    int32_t k0, k1;
    const oracle_layer *layers;
    double ymax;
    int64_t nrows;
    const int64_t *y_row_ptr;
    const int32_t *y_col;
    const float *y_val;
    int64_t *out_count;
    int32_t *out_col;
    float *out_val;
    int64_t *layer_nnz; /* optional: nnz of Y_{k+1} summed over rows, per layer */
    int bias_mode;      /* 0: bias everywhere; 1: bias on the structural pattern only */
    int64_t next_row;   /* shared work counter */
    int status;
} forward_job;

/* One sample through layers [k0, k1).  cur/nxt hold sorted (index, value) lists. */
static void forward_one_row(forward_job *job, int64_t r, double *acc, char *touched, int32_t *cur_col,
                            float *cur_val, int32_t *nxt_col, float *nxt_val, int64_t *layer_cnt)
{
    const int64_t n = job->n;
    int64_t cur_len = 0;
    for (int64_t t = job->y_row_ptr[r]; t < job->y_row_ptr[r + 1]; ++t) {
        cur_col[cur_len] = job->y_col[t];
        cur_val[cur_len] = job->y_val[t];
        ++cur_len;
    }
    for (int32_t k = job->k0; k < job->k1; ++k) {
        const oracle_layer *W = &job->layers[k];
        /* Y_k W_k for this row: acc(j) = sum_i y(i) * W(i, j) */
        for (int64_t j = 0; j < n; ++j) acc[j] = 0.0;
        if (job->bias_mode) memset(touched, 0, (size_t)n);
        for (int64_t t = 0; t < cur_len; ++t) {
            const int32_t i = cur_col[t];
            const double y = (double)cur_val[t];
            for (int64_t e = W->row_ptr[i]; e < W->row_ptr[i + 1]; ++e) {
                acc[W->col[e]] += y * (double)W->val[e];
                if (job->bias_mode && y != 0.0) touched[W->col[e]] = 1;
            }
        }
        /* + b, then h, then round once to fp32; keep only nonzeros */
        int64_t nxt_len = 0;
        for (int64_t j = 0; j < n; ++j) {
            if (job->bias_mode && !touched[j]) continue; /* no structural entry: stays 0 */
            double z = acc[j] + (double)W->bias[j];
            if (z < 0.0) z = 0.0;
            if (z > job->ymax) z = job->ymax;
            const float f = (float)z;
            if (f != 0.0f) {
                nxt_col[nxt_len] = (int32_t)j;
                nxt_val[nxt_len] = f;
                ++nxt_len;
            }
        }
        if (layer_cnt) layer_cnt[k - job->k0] += nxt_len;
        int32_t *tc = cur_col; cur_col = nxt_col; nxt_col = tc;
        float *tv = cur_val; cur_val = nxt_val; nxt_val = tv;
        cur_len = nxt_len;
    }
    job->out_count[r] = cur_len;
    memcpy(job->out_col + r * n, cur_col, (size_t)cur_len * sizeof(int32_t));
    memcpy(job->out_val + r * n, cur_val, (size_t)cur_len * sizeof(float));
}

static void *forward_worker(void *arg)
{
    forward_job *job = (forward_job *)arg;
    const int64_t n = job->n;
    const int32_t nl = job->k1 - job->k0;
    double *acc = (double *)malloc((size_t)n * sizeof(double));
    char *touched = (char *)calloc((size_t)n, 1);
    int32_t *c0 = (int32_t *)malloc((size_t)n * sizeof(int32_t));
    int32_t *c1 = (int32_t *)malloc((size_t)n * sizeof(int32_t));
    float *v0 = (float *)malloc((size_t)n * sizeof(float));
    float *v1 = (float *)malloc((size_t)n * sizeof(float));
    int64_t *cnt = job->layer_nnz ? (int64_t *)calloc((size_t)(nl > 0 ? nl : 1), sizeof(int64_t)) : NULL;
    if (!acc || !touched || !c0 || !c1 || !v0 || !v1 || (job->layer_nnz && !cnt)) {
        __atomic_store_n(&job->status, -2, __ATOMIC_SEQ_CST);
    } else {
        for (;;) {
            const int64_t r = __atomic_fetch_add(&job->next_row, 1, __ATOMIC_SEQ_CST);
            if (r >= job->nrows) break;
            forward_one_row(job, r, acc, touched, c0, v0, c1, v1, cnt);
        }
        if (cnt)
            for (int32_t k = 0; k < nl; ++k) __atomic_fetch_add(&job->layer_nnz[k], cnt[k], __ATOMIC_SEQ_CST);
    }
    free(acc); free(touched); free(c0); free(c1); free(v0); free(v1); free(cnt);
    return NULL;
}

static int check_layer(int64_t n, const oracle_layer *W)
{
    if (!W->row_ptr || !W->bias || (W->row_ptr[n] > 0 && (!W->col || !W->val))) return -1;
    if (W->row_ptr[0] != 0) return -1;
    for (int64_t i = 0; i < n; ++i) {
        if (W->row_ptr[i + 1] < W->row_ptr[i]) return -1;
        for (int64_t e = W->row_ptr[i]; e < W->row_ptr[i + 1]; ++e)
            if (W->col[e] < 0 || W->col[e] >= n) return -1;
    }
    return 0;
}

static int run_threads(void *(*fn)(void *), void *job, int nthreads)
{
    if (nthreads < 1) nthreads = 1;
    pthread_t *tid = (pthread_t *)malloc((size_t)nthreads * sizeof(pthread_t));
    if (!tid) return -2;
    int started = 0;
    for (int t = 0; t < nthreads; ++t)
        if (pthread_create(&tid[t], NULL, fn, job) == 0) ++started;
    if (started == 0) fn(job);
    for (int t = 0; t < started; ++t) pthread_join(tid[t], NULL);
    free(tid);
    return 0;
}

/*
 * Y_{k1} from Y_{k0} for `nrows` samples given as CSR rows (columns ascending).
 * Output row r goes to out_col/out_val[r*n .. r*n + out_count[r]) with ascending
 * columns and no stored zeros.  bias_mode selects the bias reading (see the
 * top of this file).  Returns 0, -1 on invalid input, -2 on allocation failure.
 */
int oracle_forward(int64_t n, int32_t k0, int32_t k1, const oracle_layer *layers, double ymax, int bias_mode,
                   int64_t nrows, const int64_t *y_row_ptr, const int32_t *y_col, const float *y_val,
                   int64_t *out_count, int32_t *out_col, float *out_val, int64_t *layer_nnz, int nthreads)
{
    if (n <= 0 || k0 < 0 || k1 < k0 || nrows < 0 || !y_row_ptr || !out_count || !out_col || !out_val) return -1;
    if (bias_mode != 0 && bias_mode != 1) return -1;
    for (int32_t k = k0; k < k1; ++k)
        if (check_layer(n, &layers[k])) return -1;
    for (int64_t r = 0; r < nrows; ++r) {
        if (y_row_ptr[r + 1] < y_row_ptr[r] || y_row_ptr[r + 1] - y_row_ptr[r] > n) return -1;
        for (int64_t t = y_row_ptr[r]; t < y_row_ptr[r + 1]; ++t)
            if (y_col[t] < 0 || y_col[t] >= n || (t > y_row_ptr[r] && y_col[t] <= y_col[t - 1])) return -1;
    }
    if (layer_nnz)
        for (int32_t k = k0; k < k1; ++k) layer_nnz[k - k0] = 0;
    forward_job job = {n, k0, k1, layers, ymax, nrows, y_row_ptr, y_col, y_val,
                       out_count, out_col, out_val, layer_nnz, bias_mode, 0, 0};
    if (run_threads(forward_worker, &job, nthreads)) return -2;
    return job.status;
}

typedef struct {
    int64_t n;
    const oracle_layer *W;
    int64_t nrows;
    const int64_t *y_row_ptr;
    const int32_t *y_col;
    const float *y_val;
    double *z, *s;
    int64_t next_row;
} preact_job;

static void *preact_worker(void *arg)
{
    preact_job *job = (preact_job *)arg;
    const int64_t n = job->n;
    const oracle_layer *W = job->W;
    for (;;) {
        const int64_t r = __atomic_fetch_add(&job->next_row, 1, __ATOMIC_SEQ_CST);
        if (r >= job->nrows) break;
        double *z = job->z + r * n, *s = job->s + r * n;
        for (int64_t j = 0; j < n; ++j) { z[j] = 0.0; s[j] = 0.0; }
        for (int64_t t = job->y_row_ptr[r]; t < job->y_row_ptr[r + 1]; ++t) {
            const int32_t i = job->y_col[t];
            const double y = (double)job->y_val[t];
            for (int64_t e = W->row_ptr[i]; e < W->row_ptr[i + 1]; ++e) {
                const double p = y * (double)W->val[e];
                z[W->col[e]] += p;
                s[W->col[e]] += fabs(p);
            }
        }
        for (int64_t j = 0; j < n; ++j) {
            z[j] += (double)W->bias[j];
            s[j] += fabs((double)W->bias[j]);
        }
    }
    return NULL;
}

/*
 * Pre-activation of one layer, z = Y W + 1 b^T (fp64), and its condition scale
 * s = |Y| |W| + 1 |b|^T, densely for `nrows` CSR rows (nrows x n each).  Used
 * to decide which output entries sit so close to the ReLU threshold that
 * rounding may legitimately flip them.
 */
int oracle_preact(int64_t n, const oracle_layer *W, int64_t nrows, const int64_t *y_row_ptr,
                  const int32_t *y_col, const float *y_val, double *z, double *s, int nthreads)
{
    if (n <= 0 || !W || nrows < 0 || !y_row_ptr || !z || !s) return -1;
    if (check_layer(n, W)) return -1;
    for (int64_t r = 0; r < nrows; ++r)
        for (int64_t t = y_row_ptr[r]; t < y_row_ptr[r + 1]; ++t)
            if (y_col[t] < 0 || y_col[t] >= n) return -1;
    preact_job job = {n, W, nrows, y_row_ptr, y_col, y_val, z, s, 0};
    if (run_threads(preact_worker, &job, nthreads)) return -2;
    return 0;
}

/*
 * Matrix multiply over a semiring (Sec. II.D: C(i,j) = (+)_k A(i,k) (x) B(k,j)),
 * Z = Y (+).(x) W for `nrows` dense rows of Y (row-major nrows x n) and a CSR
 * W: Z(r, j) = (+) over the stored entries W(i, j) of Y(r, i) (x) W(i, j),
 * starting from the semiring's 0-element, in ascending i, in fp64, rounded
 * once to fp32.  The semirings are those Sec. II names:
 *   0  +.x     on R                   0-element 0
 *   1  max.+   on {-inf} u R          0-element -inf
 *   2  max.min on {-inf} u R          0-element -inf
 *   3  min.max on R u {+inf}          0-element +inf
 *   4  xor.and on {0, 1} (GF(2))      0-element 0; a value counts as 1 when nonzero
 * The bias of W's layer is not used.  Returns 0, or -1 on invalid input.
 */
static double sr_zero(int sr)
{
    switch (sr) {
    case 1: case 2: return -INFINITY;
    case 3: return INFINITY;
    default: return 0.0;
    }
}

static double sr_add(int sr, double a, double b)
{
    switch (sr) {
    case 1: case 2: return a > b ? a : b;
    case 3: return a < b ? a : b;
    case 4: return (double)((a != 0.0) != (b != 0.0));
    default: return a + b;
    }
}

static double sr_mul(int sr, double a, double b)
{
    switch (sr) {
    case 1: return a + b;
    case 2: return a < b ? a : b;
    case 3: return a > b ? a : b;
    case 4: return (double)(a != 0.0 && b != 0.0);
    default: return a * b;
    }
}

int oracle_mxm(int semiring, int64_t n, const oracle_layer *W, int64_t nrows, const float *y, float *z)
{
    if (semiring < 0 || semiring > 4 || n <= 0 || nrows < 0 || !W || (nrows > 0 && (!y || !z))) return -1;
    if (check_layer(n, W)) return -1;
    double *acc = (double *)malloc((size_t)n * sizeof(double));
    if (!acc) return -2;
    for (int64_t r = 0; r < nrows; ++r) {
        for (int64_t j = 0; j < n; ++j) acc[j] = sr_zero(semiring);
        for (int64_t i = 0; i < n; ++i) {
            const double yv = (double)y[r * n + i];
            for (int64_t e = W->row_ptr[i]; e < W->row_ptr[i + 1]; ++e)
                acc[W->col[e]] = sr_add(semiring, acc[W->col[e]], sr_mul(semiring, yv, (double)W->val[e]));
        }
        for (int64_t j = 0; j < n; ++j) z[r * n + j] = (float)acc[j];
    }
    free(acc);
    return 0;
}
