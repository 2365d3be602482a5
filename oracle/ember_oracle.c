/*
 * Ember CPU oracle.  TEST INFRASTRUCTURE ONLY: the tests, the smoke check and
 * the benchmark's CPU-baseline leg call it; the product path never does.  It
 * shares no code, header or constant with the HIP library.
 *
 * What it computes: one iteration of the while-loop of Algorithm 1 ("Ember")
 * of Token Geometry (Section 2, Methods), for a V x D token-interface matrix
 * (embedding table or LM head).  Steps, in the paper's order:
 *
 *   r_t   = beta2 r_{t-1} + (1 - beta2) mean_j g_t^2         (row statistic)
 *   c_t   = beta2 c_{t-1} + (1 - beta2) mean_i g_t^2         (column statistic)
 *   rhat  = r_t / (1 - beta2^t),  chat = c_t / (1 - beta2^t) (bias correction)
 *   s_t   = sqrt( mean(rhat) * mean(chat) )                  (geometric mean)
 *   vtil  = rhat chat^T / s_t                                (never stored; the
 *           paper's "Distributed Ember" paragraph says it is applied as row and
 *           column scalings, here one element at a time)
 *   theta = theta +/- alpha g / (sqrt(vtil) + eps)
 *
 * Arithmetic is float64.  Storage follows the paper: the state r, c is fp32
 * (caption of the model-scaling table: "fp32 optimizer buffers"), so r and c
 * are rounded to fp32 where they are stored; W is rounded to its own storage
 * type (fp32 or bf16, round-to-nearest-even) once per element.
 *
 * Readings of points the paper leaves open (each is also listed in the design
 * notes of the repository):
 *   - sign: Algorithm 1 ascends a reward (theta + ...).  maximize=1 is that
 *     literal form; maximize=0 descends a loss (theta - ...).
 *   - eps is added after the square root, as printed in Algorithm 1.
 *   - s_t == 0 (no nonzero gradient seen yet): vtil is taken as 0.
 *   - beta2 is the fp32 value handed in, widened exactly to float64.
 *   - an element whose update is exactly zero (g == 0 or alpha == 0) keeps its
 *     stored bits.
 *   - sparse rows: the gradient is the dense V x D gradient that is zero on
 *     every row not listed in idx ("dense with zero rows").  Untouched rows
 *     therefore decay r by beta2, keep W unchanged, and the column mean still
 *     divides by V.  Rows of zeros add exact zeros to every float64 sum, so
 *     the loops below skip them without changing a bit.
 *   - idx must hold unique values in [0, V); otherwise the call fails and
 *     modifies nothing.
 *
 * Gradient coalescing (ember_oracle_coalesce, at the end of this file): the
 * per-position embedding gradients of a batch summed into one row per distinct
 * token, the input of the sparse step.
 *
 * LM-head weight gradient (ember_oracle_lmhead_grad, at the end of this file):
 * G = dY^T H, the gradient whose statistics the LM-head step forms inside
 * its matrix product.
 *
 * Row-only Ember (row_only = 1).  Section 2.1 describes a variant that keeps
 * only the V row statistics, bias-corrects them and divides each row's
 * gradient by their square root (the ablation table lists it with state V);
 * no formula is printed.  Reading taken here: the row statistic and bias
 * correction of Algorithm 1 unchanged, vtil_ij = rhat_i (no column factor and
 * no normaliser, since rhat already has the units of g^2), and the same update
 * theta +/- alpha g / (sqrt(vtil) + eps).  c is neither read nor written.
 *
 * Threads (OpenMP): the loops over independent rows (row statistic, update)
 * and over independent column ranges (column statistic, each column still
 * summed over rows in ascending order) may run on several threads; every
 * float64 sum keeps the order written here, so the results are the same bits
 * for any thread count.  The O(V + D) sums of the normaliser stay serial.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_F32 0
#define ORACLE_BF16 1

#define ORACLE_OK 0
#define ORACLE_BAD_ARG -1
#define ORACLE_BAD_INDEX -6

/* bf16 bits -> float64 (exact: bf16 is the top half of an fp32). */
double ember_oracle_bf16_to_f64(uint16_t bits)
{
    uint32_t u = ((uint32_t)bits) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/*
 * float64 -> bf16 with one round-to-nearest-even (no detour through fp32,
 * which would round twice).  bf16 has fp32's exponent range and 8 significant
 * bits, so a finite value |x| >= 2^-126 in binade 2^E is a multiple of
 * 2^(E-7), and below 2^-126 (subnormals) a multiple of 2^-133.
 */
uint16_t ember_oracle_f64_to_bf16(double x)
{
    uint16_t sign = signbit(x) ? 0x8000u : 0u;
    if (isnan(x))
        return (uint16_t)(sign | 0x7FC0u);
    double ax = fabs(x);
    if (isinf(ax))
        return (uint16_t)(sign | 0x7F80u);
    if (ax == 0.0)
        return sign;
    int e2;
    (void)frexp(ax, &e2); /* ax in [2^(e2-1), 2^e2) */
    int E = e2 - 1;
    if (E < -126)
        E = -126;
    double quantum = ldexp(1.0, E - 7);
    double n = rint(ax / quantum); /* exact scaling; rint rounds half to even */
    double v = n * quantum;        /* may be 2^128: overflow to infinity */
    float f = (float)v;            /* exact: v is a bf16 value or overflows */
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return (uint16_t)(sign | (uint16_t)(u >> 16));
}

/* Threads the loops below may use (OpenMP); returns the count now in effect. */
int ember_oracle_set_threads(int n)
{
    if (n > 0)
        omp_set_num_threads(n);
    return omp_get_max_threads();
}

/* Bytes of Ember state for one V x D table: r (V floats) and c (D floats). */
int64_t ember_oracle_state_bytes(int64_t V, int64_t D)
{
    return (int64_t)sizeof(float) * (V + D);
}

static double load_elem(const void* base, int dtype, int64_t off)
{
    if (dtype == ORACLE_F32)
        return (double)((const float*)base)[off];
    return ember_oracle_bf16_to_f64(((const uint16_t*)base)[off]);
}

static void store_elem(void* base, int dtype, int64_t off, double v)
{
    if (dtype == ORACLE_F32)
        ((float*)base)[off] = (float)v;
    else
        ((uint16_t*)base)[off] = ember_oracle_f64_to_bf16(v);
}

/*
 * One Ember step on W (V x D, row stride ldw elements) with gradient G.
 *   idx == NULL : G is dense, V rows of stride ldg.
 *   idx != NULL : G holds n_idx rows (stride ldg); row k is the gradient of
 *                 W's row idx[k]; all other rows of the gradient are zero.
 * r (V floats) and c (D floats) are read and updated in place; t >= 1 is the
 * step being taken.  W is updated in place.
 * w_rows (optional, n_w_rows entries, strictly increasing): when given, only
 * these rows of W are written (a sample for checks at large sizes); the state
 * update is always complete.
 * Returns 0, or a negative code with nothing modified.
 */
int ember_oracle_step(void* W, int w_dtype, int64_t ldw,
                      const void* G, int g_dtype, int64_t ldg,
                      const int64_t* idx, int64_t n_idx,
                      float* r, float* c, int64_t V, int64_t D, int64_t t,
                      float lr, float beta2, float eps, int maximize,
                      const int64_t* w_rows, int64_t n_w_rows, int row_only)
{
    if (V < 1 || D < 1 || ldw < D || ldg < D || t < 1)
        return ORACLE_BAD_ARG;
    if (!W || !r || (!c && !row_only) || (!G && (idx == NULL || n_idx > 0)))
        return ORACLE_BAD_ARG;
    if ((w_dtype != ORACLE_F32 && w_dtype != ORACLE_BF16) ||
        (g_dtype != ORACLE_F32 && g_dtype != ORACLE_BF16))
        return ORACLE_BAD_ARG;
    if (!(beta2 >= 0.0f && beta2 < 1.0f) || !(eps >= 0.0f) || !(lr >= 0.0f))
        return ORACLE_BAD_ARG;
    if (idx != NULL && n_idx < 0)
        return ORACLE_BAD_ARG;
    if (w_rows != NULL) {
        for (int64_t k = 0; k < n_w_rows; ++k)
            if (w_rows[k] < 0 || w_rows[k] >= V || (k > 0 && w_rows[k] <= w_rows[k - 1]))
                return ORACLE_BAD_ARG;
    }

    /* grow[i]: row of G holding gradient row i, or -1 for a zero row. */
    int64_t* grow = (int64_t*)malloc((size_t)V * sizeof(int64_t));
    double* colsum = (double*)calloc((size_t)D, sizeof(double));
    if (!grow || !colsum) {
        free(grow);
        free(colsum);
        return ORACLE_BAD_ARG;
    }
    if (idx == NULL) {
        for (int64_t i = 0; i < V; ++i)
            grow[i] = i;
    } else {
        for (int64_t i = 0; i < V; ++i)
            grow[i] = -1;
        for (int64_t k = 0; k < n_idx; ++k) {
            int64_t i = idx[k];
            if (i < 0 || i >= V || grow[i] != -1) {
                free(grow);
                free(colsum);
                return ORACLE_BAD_INDEX;
            }
            grow[i] = k;
        }
    }

    const double b2 = (double)beta2;
    const double one_minus_b2 = 1.0 - b2;

    /* Row second moment: r_i <- beta2 r_i + (1-beta2) mean_j g_ij^2. */
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < V; ++i) {
        double sumsq = 0.0;
        if (grow[i] >= 0) {
            for (int64_t j = 0; j < D; ++j) {
                double g = load_elem(G, g_dtype, grow[i] * ldg + j);
                sumsq += g * g;
            }
        }
        double mean_j = sumsq / (double)D;
        r[i] = (float)(b2 * (double)r[i] + one_minus_b2 * mean_j);
    }

    /* Column second moment: c_j <- beta2 c_j + (1-beta2) mean_i g_ij^2,
     * summing rows in ascending row order. */
    if (!row_only) {
#pragma omp parallel for schedule(static)
        for (int64_t j0 = 0; j0 < D; j0 += 64) {
            const int64_t j1 = j0 + 64 < D ? j0 + 64 : D;
            for (int64_t i = 0; i < V; ++i) {
                if (grow[i] < 0)
                    continue;
                for (int64_t j = j0; j < j1; ++j) {
                    double g = load_elem(G, g_dtype, grow[i] * ldg + j);
                    colsum[j] += g * g;
                }
            }
        }
        for (int64_t j = 0; j < D; ++j) {
            double mean_i = colsum[j] / (double)V;
            c[j] = (float)(b2 * (double)c[j] + one_minus_b2 * mean_i);
        }
    }

    /* Bias correction, from the fp32-stored state. */
    const double bias = 1.0 - pow(b2, (double)t);

    /* Geometric-mean normaliser s = sqrt(mean(rhat) mean(chat)). */
    double s = 0.0;
    if (!row_only) {
        double sum_rhat = 0.0, sum_chat = 0.0;
        for (int64_t i = 0; i < V; ++i)
            sum_rhat += (double)r[i] / bias;
        for (int64_t j = 0; j < D; ++j)
            sum_chat += (double)c[j] / bias;
        s = sqrt((sum_rhat / (double)V) * (sum_chat / (double)D));
    }

    /* Update with the factored preconditioner vtil_ij = rhat_i chat_j / s. */
    const double alpha = (double)lr;
    const double e = (double)eps;
    const int64_t n_out = (w_rows != NULL) ? n_w_rows : V;
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < n_out; ++k) {
        const int64_t i = (w_rows != NULL) ? w_rows[k] : k;
        if (grow[i] < 0)
            continue; /* zero gradient row: every update is exactly zero */
        const double rhat = (double)r[i] / bias;
        for (int64_t j = 0; j < D; ++j) {
            double g = load_elem(G, g_dtype, grow[i] * ldg + j);
            if (g == 0.0 || alpha == 0.0)
                continue;
            double vtil;
            if (row_only) {
                vtil = rhat;
            } else {
                const double chat = (double)c[j] / bias;
                vtil = (s > 0.0) ? rhat * chat / s : 0.0;
            }
            const double u = alpha * g / (sqrt(vtil) + e);
            const double w = load_elem(W, w_dtype, i * ldw + j);
            store_elem(W, w_dtype, i * ldw + j, maximize ? w + u : w - u);
        }
    }

    free(grow);
    free(colsum);
    return ORACLE_OK;
}

/*
 * Coalescing of per-position embedding gradients into distinct rows.
 *
 * The input-embedding gradient of one position is a one-hot row selector
 * times the back-propagated signal (appendix "Decomposing the Squared
 * Gradient"), so the gradient of row i over a batch is the sum of the signals
 * of the K_i positions holding token i (appendix "The Fisher is Proportional to
 * Inverse Frequency Squared", where the row gradient is that sum).  This
 * produces the (idx, G_rows) pair the sparse step takes:
 *
 *   idx[0..n)   the distinct values of tok[0..P), ascending;
 *   G[k][j]     sum over p = 0, 1, ..., P-1 with tok[p] == idx[k] of U[p][j],
 *               accumulated in float64 in that (ascending position) order and
 *               rounded once to G's storage type.
 *
 * tok[p] must lie in [0, V); otherwise nothing is written and the call
 * returns ORACLE_BAD_INDEX.  *n_out receives n.  P = 0 gives n = 0.
 */
static int cmp_i64(const void* a, const void* b)
{
    int64_t x = *(const int64_t*)a, y = *(const int64_t*)b;
    return (x > y) - (x < y);
}

int ember_oracle_coalesce(const int64_t* tok, int64_t P, const void* U, int u_dtype, int64_t ldu,
                          int64_t V, int64_t D, int64_t* idx, void* G, int g_dtype, int64_t ldg,
                          int64_t* n_out)
{
    if (P < 0 || V < 1 || D < 1 || !n_out || (P > 0 && (!tok || !U || !idx || !G)))
        return ORACLE_BAD_ARG;
    for (int64_t p = 0; p < P; ++p)
        if (tok[p] < 0 || tok[p] >= V)
            return ORACLE_BAD_INDEX;
    /* distinct ids, ascending */
    int64_t* ids = (int64_t*)malloc((size_t)(P > 0 ? P : 1) * sizeof(int64_t));
    if (!ids)
        return ORACLE_BAD_ARG;
    memcpy(ids, tok, (size_t)P * sizeof(int64_t));
    qsort(ids, (size_t)P, sizeof(int64_t), cmp_i64);
    int64_t n = 0;
    for (int64_t p = 0; p < P; ++p)
        if (n == 0 || ids[p] != ids[n - 1])
            ids[n++] = ids[p];
    double* acc = (double*)calloc((size_t)(n > 0 ? n : 1) * (size_t)D, sizeof(double));
    if (!acc) {
        free(ids);
        return ORACLE_BAD_ARG;
    }
    /* the sums, visiting positions in ascending order */
    for (int64_t p = 0; p < P; ++p) {
        const int64_t* hit = (const int64_t*)bsearch(&tok[p], ids, (size_t)n, sizeof(int64_t), cmp_i64);
        int64_t k = hit - ids;
        for (int64_t j = 0; j < D; ++j)
            acc[k * D + j] += load_elem(U, u_dtype, p * ldu + j);
    }
    for (int64_t k = 0; k < n; ++k) {
        idx[k] = ids[k];
        for (int64_t j = 0; j < D; ++j)
            store_elem(G, g_dtype, k * ldg + j, acc[k * D + j]);
    }
    *n_out = n;
    free(acc);
    free(ids);
    return ORACLE_OK;
}

/*
 * LM-head weight gradient.  For an LM head with logits z_m = W h_m and
 * softmax probabilities q_m, the cross-entropy gradient of row i is
 * G_i = sum_m (q_mi - 1[y_m = i]) h_m (appendix "The LM Head Factorizes Like
 * the Embedding Table").  Given dY[m][i] = q_mi - 1[y_m = i] (T x V, bf16
 * bits, row stride ldy) and the hidden states H (T x D, bf16 bits, row stride
 * ldh), this writes G[i][j] = sum over m = 0 .. T-1 of dY[m][i] H[m][j]: the
 * products of two bf16 values are exact in float64, the sum runs in float64
 * in ascending m, and the result is rounded once to g_dtype (nearest-even).
 * T = 0 gives G = 0.  Returns 0, or -1 for a bad argument.
 */
int ember_oracle_lmhead_grad(const uint16_t* dY, int64_t ldy, const uint16_t* H, int64_t ldh, int64_t T,
                             int64_t V, int64_t D, void* G, int g_dtype, int64_t ldg)
{
    if (V < 1 || D < 1 || T < 0 || ldy < V || ldh < D || ldg < D || G == NULL) return -1;
    if (T > 0 && (dY == NULL || H == NULL)) return -1;
    if (g_dtype != ORACLE_F32 && g_dtype != ORACLE_BF16) return -1;
    int failed = 0;
#pragma omp parallel
    {
        double* acc = (double*)malloc((size_t)D * sizeof(double));
        if (acc == NULL) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(static)
        for (int64_t i = 0; i < V; ++i) {
            if (acc == NULL)
                continue;
            for (int64_t j = 0; j < D; ++j) acc[j] = 0.0;
            for (int64_t m = 0; m < T; ++m) {
                const double y = ember_oracle_bf16_to_f64(dY[m * ldy + i]);
                const uint16_t* h = H + m * ldh;
                for (int64_t j = 0; j < D; ++j) acc[j] += y * ember_oracle_bf16_to_f64(h[j]);
            }
            for (int64_t j = 0; j < D; ++j) store_elem(G, g_dtype, i * ldg + j, acc[j]);
        }
        free(acc);
    }
    return failed ? -1 : 0;
}
