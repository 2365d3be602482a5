/*
 * ember.h: C ABI of the Ember token-table optimizer step for AMD MI355X (gfx950).
 *
 * Ember (Token Geometry, Algorithm 1 in Section 2) updates a V x D
 * token-interface matrix W (embedding table or LM head) from its gradient G
 * with O(V + D) state: a row second-moment vector r (V floats) and a column
 * second-moment vector c (D floats).  One step t >= 1 computes
 *
 *   r <- beta2 r + (1 - beta2) mean_j G_ij^2          (row statistic)
 *   c <- beta2 c + (1 - beta2) mean_i G_ij^2          (column statistic)
 *   rhat = r / (1 - beta2^t),  chat = c / (1 - beta2^t)
 *   s = sqrt(mean(rhat) mean(chat))
 *   W_ij <- W_ij -/+ lr G_ij / (sqrt(rhat_i chat_j / s) + eps)
 *
 * The V x D preconditioner rhat chat^T / s is never stored: the update is
 * applied as a row scaling times a column scaling (section "Distributed
 * Ember", paragraph on the preconditioner).  All reductions use a fixed
 * order, with no floating-point atomics, so a given input produces the same
 * bits on every run (same section, on the fused deterministic reduction).
 *
 * Conventions shared by every entry point:
 *  - Memory: every pointer argument except the scalars is DEVICE memory owned
 *    by the caller.  The library never allocates, frees or synchronises,
 *    except ember_get_error (which synchronises the stream it is given).
 *  - Layout: W and G are row-major, row i starting at element i * ld.  Both
 *    base pointers must be 16-byte aligned and ld * element_size must be a
 *    multiple of 16 bytes, so every row starts on a 16-byte boundary.  Only
 *    the first D elements of each row are read or written.  W must not
 *    overlap G, r, c or the workspace.
 *  - dtypes: W and G are EMBER_F32 or EMBER_BF16, independently.  r and c are
 *    always fp32 (the paper keeps optimizer state in fp32).  Arithmetic is
 *    fp32; W is written with round-to-nearest-even; an element whose
 *    gradient is exactly zero keeps its bits.
 *  - Streams: all work is enqueued on `stream` (0 = the null stream) in
 *    order; calls return before the work runs.  One (r, c, workspace) set
 *    must not be used by two streams at once.
 *  - Errors: every argument check below happens on the host before anything
 *    is enqueued; on a negative return nothing was enqueued and no memory was
 *    touched.  EMBER_ERR_HIP means a launch failed after validation.
 *  - Step counter: t is owned by the caller: it starts at 0 and the caller
 *    passes t = 1, 2, ... (Algorithm 1 increments t before each update).
 *  - Sign: maximize = 0 descends a loss (W -= ...); maximize = 1 is the
 *    paper's literal ascent of a reward (W += ...).
 */
#ifndef EMBER_H
#define EMBER_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { EMBER_F32 = 0, EMBER_BF16 = 1 } ember_dtype;

typedef enum {
    EMBER_OK = 0,
    EMBER_ERR_ARG = -1,       /* null pointer, or a scalar out of range */
    EMBER_ERR_SHAPE = -2,     /* V or D < 1 or too large, ld < D, n_idx > V */
    EMBER_ERR_ALIGN = -3,     /* W/G not 16-byte aligned, ld*size not a multiple of 16,
                                 r/c not 4-byte aligned, workspace not 256-byte aligned */
    EMBER_ERR_DTYPE = -4,     /* dtype is not EMBER_F32 or EMBER_BF16 */
    EMBER_ERR_WORKSPACE = -5, /* ws_bytes smaller than ember_workspace_bytes(V, D) */
    EMBER_ERR_INDEX = -6,     /* sparse step: idx holds a value outside [0, V) or a
                                 repeated value, or a device row count is out of
                                 range (reported by ember_get_error) */
    EMBER_ERR_HIP = -7,       /* a HIP runtime call failed */
    EMBER_ERR_DEVICE = -8     /* sparse step (reported by ember_get_error): the blocks of
                                 the one-launch form did not all run at once, so a grid
                                 barrier's bounded wait ran out; W, r and c are then
                                 unspecified.  Not expected on an MI355X that the
                                 calling process has to itself. */
} ember_status;

/* Largest supported V (row indices are kept in 31 bits) and D, and the
 * largest token batch of ember_coalesce_rows. */
#define EMBER_MAX_V ((int64_t)0x7FFFFFFE)
#define EMBER_MAX_D ((int64_t)(1 << 22))
#define EMBER_MAX_TOKENS ((int64_t)(1 << 26))
/* ember_lmhead_step: row strides of dY and H below 2^24 elements (a 64-token
 * slice of either is then addressable with 32-bit offsets), and at most 2^30
 * tokens. */
#define EMBER_LMHEAD_MAX_LD ((int64_t)(1 << 24))
#define EMBER_LMHEAD_MAX_T ((int64_t)(1 << 30))

/*
 * Workspace size for a V x D table, valid for every step (dense, sparse,
 * canonical and row-only).  The workspace holds the per-block partial sums of the fixed-order
 * reductions, a V-entry row-slot table used by the sparse step, and a status
 * word.  It is caller-allocated device memory, 256-byte aligned, and must be
 * initialised once by ember_init_state before its first step.
 * Returns EMBER_OK and sets *bytes, or EMBER_ERR_SHAPE / EMBER_ERR_ARG.
 */
int ember_workspace_bytes(int64_t V, int64_t D, size_t* bytes);

/*
 * Ember state initialisation (Algorithm 1: r_0 = 0 in R^V, c_0 = 0 in R^D,
 * t = 0).  Enqueues zero fills of r (V floats), c (D floats) and the parts
 * of the workspace that must start at zero.  The caller sets t = 0.
 */
int ember_init_state(float* r, float* c, int64_t V, int64_t D,
                     void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * One dense Ember step (Algorithm 1, one pass of its loop body) on W (V x D,
 * row stride ldw, dtype w_dtype) with gradient G (V x D, row stride ldg,
 * dtype g_dtype).  r (V) and c (D) are updated in place, then W.
 * Scalars: t >= 1; lr >= 0 and finite; 0 <= beta2 < 1; eps >= 0 and finite
 * (the paper's defaults: lr = 1e-3, beta2 = 0.999, eps = 1e-8).  beta2 is
 * used as the fp32 value passed.
 */
int ember_step_dense(void* W, int w_dtype, int64_t ldw,
                     const void* G, int g_dtype, int64_t ldg,
                     float* r, float* c, int64_t V, int64_t D, int64_t t,
                     float lr, float beta2, float eps, int maximize,
                     void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * One sparse-row Ember step: the gradient is zero except on the n_idx rows
 * listed in idx (the embedding-table case of Section 2.2, where only the
 * tokens of the batch receive gradient).  G_rows is n_idx x D (row stride
 * ldg, compact: row k is the gradient of W's row idx[k]).  idx is a device
 * array of n_idx int64 values, unique and in [0, V), in any order;
 * n_idx = 0 is allowed (then G_rows and idx may be NULL).
 *
 * The result is the dense step on the gradient that is zero outside idx:
 * every row's r decays by beta2 (touched rows also add their statistic), the
 * column mean still divides by V, s uses all V rows, and W rows outside idx
 * are not touched.
 *
 * Index errors (a value outside [0, V), or a repeated value) are detected on
 * the device: the step then leaves W, r and c unchanged, and the next
 * ember_get_error on this workspace reports EMBER_ERR_INDEX.  The caller
 * should then not advance t.
 */
int ember_step_sparse_rows(void* W, int w_dtype, int64_t ldw,
                           const void* G_rows, int g_dtype, int64_t ldg,
                           const int64_t* idx, int64_t n_idx,
                           float* r, float* c, int64_t V, int64_t D, int64_t t,
                           float lr, float beta2, float eps, int maximize,
                           void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * The sparse step with its row count in device memory, for callers whose
 * count is produced on the device (ember_coalesce_rows writes it): nothing is
 * read back to the host, so coalescing and the step can be enqueued together
 * or captured in one HIP graph.  n_idx_dev points to one int64 in device
 * memory, read when the step runs; max_rows (host) bounds it and sizes the
 * launches; G_rows and idx must hold max_rows rows.  A device count outside
 * [0, max_rows] is reported like an index error (EMBER_ERR_INDEX through
 * ember_get_error; W, r and c untouched).  The step takes the one-launch form
 * of ember_step_sparse_rows whenever the count fits it: decided on the host
 * when max_rows fits, else on the device from the count (the one-launch kernel
 * runs first and, when it has taken the step, the three launches of the other
 * form return at once).  With *n_idx_dev == max_rows, or a count that takes the
 * one-launch form, the result is the same, bit for bit, as
 * ember_step_sparse_rows with n_idx = that count; other counts partition the
 * rows differently and agree within the stated tolerances.  Everything else as
 * for ember_step_sparse_rows.
 */
int ember_step_sparse_rows_devn(void* W, int w_dtype, int64_t ldw,
                                const void* G_rows, int g_dtype, int64_t ldg,
                                const int64_t* idx, const int64_t* n_idx_dev, int64_t max_rows,
                                float* r, float* c, int64_t V, int64_t D, int64_t t,
                                float lr, float beta2, float eps, int maximize,
                                void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * The sparse-row step without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation.  The step is ember_step_sparse_rows's
 * one-launch form (same kernel, same bits as that call with a workspace); its
 * scratch (row marks, barrier flags, per-block partial sums, column factors)
 * is a 16 MiB array inside the library, one per GPU, held until the process
 * ends.  Each call enqueues a small zero fill of that array's first part and
 * of *status, then the step; nothing is allocated.
 *
 * Arguments as for ember_step_sparse_rows (W, G_rows, idx, n_idx, r, c, V, D,
 * t and the scalars), without ws/ws_bytes, plus:
 *   status  device int32 (4-byte aligned, required): set to 0 by the call's
 *           fill, then the step ORs its error bits into it (1: an id outside
 *           [0, V), 2: a repeated id; W, r and c are then unchanged; 8: the
 *           step's blocks did not all run at once, W, r and c unspecified).
 *           Read it after the stream has reached the step.
 * r and c start at zero (Algorithm 1's r_0, c_0) and are the caller's, as is t.
 *
 * Limits (checked on the host before anything is enqueued):
 *   the step's scratch, about 4 V + 1028 D bytes + 23 KiB, at most 16 MiB
 *   (e.g. V up to 3.1 million rows at D = 4096): EMBER_ERR_WORKSPACE otherwise;
 *   the one-launch form must take the step: D a whole number of 16-byte chunks
 *   of G, at most 8 column slabs of 2 KiB (bf16 D <= 8192, fp32 D <= 4096),
 *   n_idx within the rows held on chip (5120 at 4096 bf16 columns), and a
 *   device that keeps 256 blocks of the kernel resident: EMBER_ERR_SHAPE
 *   otherwise.
 * Calls that overlap on one GPU (two streams, or two threads) share the array
 * and race; calls must be ordered.
 */
int ember_step_sparse_rows_static(void* W, int w_dtype, int64_t ldw,
                                  const void* G_rows, int g_dtype, int64_t ldg,
                                  const int64_t* idx, int64_t n_idx,
                                  float* r, float* c, int64_t V, int64_t D, int64_t t,
                                  float lr, float beta2, float eps, int maximize,
                                  int32_t* status, hipStream_t stream);

/*
 * Several Ember steps in one call: the tables of a model (for example the
 * LM head, dense, and the input embedding, sparse rows) each take the step
 * Algorithm 1 defines for them (or the row-only step of Section 2.1), exactly
 * as the single-table entry points would, but the canonical tables share
 * three launches (one statistics pass, one finalize pass, one apply pass over
 * every table) instead of three per table, so the tables share the chip and a
 * small table costs its bytes instead of its launch latency; a sparse table
 * whose rows fit on chip takes its one-launch step (that of
 * ember_step_sparse_rows) ahead of them.  Each table's results are the same bits as its own
 * single-table call (ember_step_dense, ember_step_sparse_rows(_devn), or the
 * row-only entry points declared below).
 *
 * One ember_table_step per table:
 *   W, w_dtype, ldw, G, g_dtype, ldg, r, c, V, D, t, lr, beta2, eps,
 *   maximize, ws, ws_bytes   as for ember_step_dense;
 *   sparse = 0               dense step: G is V x D; idx, n_idx, n_idx_dev unused;
 *   sparse = 1               sparse-row step: G holds n_idx compact rows of the
 *                            rows idx lists, as for ember_step_sparse_rows;
 *                            with n_idx_dev non-NULL the row count is read from
 *                            that device int64 when the step runs and n_idx is
 *                            its maximum, as for ember_step_sparse_rows_devn.
 *   row_only = 1             the row-only step of that table (state r only; c
 *                            may be NULL), as ember_rowonly_step_dense /
 *                            ember_rowonly_step_sparse_rows(_devn) would take
 *                            it: the sparse row-only tables' id checks share one
 *                            launch and the row-only passes one more.
 * Tables may differ in every field (shape, dtypes, scalars, t).  Tables with
 * the same dtypes and the same columns-per-lane plan share launches; others
 * add launches of their own.
 *
 * Errors: each table is checked as its own call would be, and additionally
 * no memory one table writes (workspace, r, c, W) may overlap memory another
 * table reads or writes (those, and G, idx, the device row count), since the
 * tables share launches (EMBER_ERR_ARG); memory the tables only read may be
 * shared.  1 <= n_tables <= EMBER_MAX_TABLES (EMBER_ERR_ARG).  A failed check enqueues nothing for any table.  Index
 * errors of a sparse table leave that table untouched (the others step
 * normally) and are reported by ember_get_error on its workspace.
 */
#define EMBER_MAX_TABLES 8

typedef struct {
    void* W;
    int w_dtype;
    int64_t ldw;
    const void* G;
    int g_dtype;
    int64_t ldg;
    int sparse;
    int row_only;
    const int64_t* idx;
    int64_t n_idx;
    const int64_t* n_idx_dev;
    float* r;
    float* c;
    int64_t V;
    int64_t D;
    int64_t t;
    float lr;
    float beta2;
    float eps;
    int maximize;
    void* ws;
    size_t ws_bytes;
} ember_table_step;

int ember_step_multi(const ember_table_step* tables, int n_tables, hipStream_t stream);

/*
 * Row-only Ember (Section 2.1, the variant the paper analyses most, listed in
 * its ablation table with V floats of state): only the row statistic r is
 * kept, and each row's gradient is divided by the square root of its own
 * bias-corrected statistic:
 *
 *   r <- beta2 r + (1 - beta2) mean_j G_ij^2,   rhat = r / (1 - beta2^t)
 *   W_ij <- W_ij -/+ lr G_ij / (sqrt(rhat_i) + eps)
 *
 * (the canonical step with vtil_ij = rhat_i: no column statistic and no
 * normaliser s).  Each row is then independent of the others, so the step is
 * one pass that reads G and W once and writes W once.  Arguments, layouts,
 * dtypes, streams and error handling are those of the canonical entry points
 * above, without c.  The workspace is sized by ember_workspace_bytes(V, D)
 * and may be shared with nothing else while in use.
 */

/* Row-only state initialisation: zero fills of r (V floats) and of the parts
 * of the workspace that must start at zero.  The caller sets t = 0. */
int ember_rowonly_init_state(float* r, int64_t V, int64_t D,
                             void* ws, size_t ws_bytes, hipStream_t stream);

/* One dense row-only step on W (V x D) with gradient G (V x D); r is updated
 * in place, then W.  Scalar ranges as for ember_step_dense. */
int ember_rowonly_step_dense(void* W, int w_dtype, int64_t ldw,
                             const void* G, int g_dtype, int64_t ldg,
                             float* r, int64_t V, int64_t D, int64_t t,
                             float lr, float beta2, float eps, int maximize,
                             void* ws, size_t ws_bytes, hipStream_t stream);

/* One sparse-row row-only step (G_rows, idx and n_idx as for
 * ember_step_sparse_rows): the dense row-only step on the gradient that is zero
 * outside idx.  Rows outside idx only see r decay by beta2; their W rows are
 * not touched.  Index errors leave W and r unchanged and are reported by
 * ember_get_error. */
int ember_rowonly_step_sparse_rows(void* W, int w_dtype, int64_t ldw,
                                   const void* G_rows, int g_dtype, int64_t ldg,
                                   const int64_t* idx, int64_t n_idx,
                                   float* r, int64_t V, int64_t D, int64_t t,
                                   float lr, float beta2, float eps, int maximize,
                                   void* ws, size_t ws_bytes, hipStream_t stream);

/* The row-only sparse step with its row count in device memory (as for
 * ember_step_sparse_rows_devn). */
int ember_rowonly_step_sparse_rows_devn(void* W, int w_dtype, int64_t ldw,
                                        const void* G_rows, int g_dtype, int64_t ldg,
                                        const int64_t* idx, const int64_t* n_idx_dev, int64_t max_rows,
                                        float* r, int64_t V, int64_t D, int64_t t,
                                        float lr, float beta2, float eps, int maximize,
                                        void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Gradient coalescing: the step before ember_step_sparse_rows.  The gradient
 * of an input embedding for one batch position is the one-hot selector of its
 * token times the back-propagated signal (appendix "Decomposing the Squared
 * Gradient"), so the gradient of row i is the sum of the signals of every
 * position holding token i (appendix "The Fisher is Proportional to Inverse
 * Frequency Squared").  Given n_tok token ids tok (device int64, each in
 * [0, V)) and the per-position signals U (n_tok x D, row stride ldu, dtype
 * u_dtype), this writes
 *
 *   *n_out           n, the number of distinct ids (device int64);
 *   idx[0..n)        the distinct ids, ascending (device int64[n_tok]);
 *   G_rows[k][0..D)  for k < n: the sum of U[p] over the positions p with
 *                    tok[p] == idx[k], accumulated in float64 and rounded once
 *                    (nearest-even) to g_dtype (device, n_tok x D, stride ldg).
 *
 * The sums have a fixed order, so results are reproducible bit for bit: the
 * positions of one id are added in ascending order, within fixed chunks of the
 * id-sorted positions, and chunk partials in chunk order.  idx and G_rows feed
 * ember_step_sparse_rows directly once n is known on the host (read *n_out
 * after synchronising the stream), or feed ember_step_sparse_rows_devn with
 * n_out itself.  Ids outside [0, V) make the call report EMBER_ERR_INDEX
 * through ember_get_error on this workspace and write n = -1 (which a
 * device-count step refuses, leaving its table untouched); idx and G_rows are
 * then unspecified.  n_tok = 0 gives n = 0 (tok, U, idx, G_rows may
 * then be NULL).  Layout and alignment rules of U and G_rows are those of W
 * and G; tok, idx and n_out must be 8-byte aligned.
 *
 * The workspace (device, 256-byte aligned, ember_coalesce_workspace_bytes of
 * at least n_tok tokens) needs no initialisation and may be reused by
 * successive calls on one stream; its size grows with max_tokens (sort
 * buffers) and with D (float64 partial rows of at most 2^25 elements).
 */
int ember_coalesce_workspace_bytes(int64_t max_tokens, int64_t V, int64_t D, size_t* bytes);

int ember_coalesce_rows(const int64_t* tok, int64_t n_tok,
                        const void* U, int u_dtype, int64_t ldu,
                        int64_t V, int64_t D,
                        int64_t* idx, void* G_rows, int g_dtype, int64_t ldg,
                        int64_t* n_out, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * LM-head step with the gradient statistics taken inside the weight-gradient
 * GEMM.  For an LM head with logits z_m = W h_m, the cross-entropy gradient of
 * row i is G_i = sum_m (q_mi - 1[y_m = i]) h_m (appendix "The LM Head
 * Factorizes Like the Embedding Table"): G = dY^T H, with dY (T x V, row
 * stride ldy) the gradient of the logits and H (T x D, row stride ldh) the
 * hidden states, both bf16, token-major as a forward pass produces them.
 *
 * The call computes G with bf16 matrix instructions and fp32 accumulation,
 * rounds it once (nearest-even) to g_dtype and stores it in G (V x D, row
 * stride ldg; the caller keeps it, e.g. for clipping or logging), and takes
 * the dense Ember step on W with that G.  The result is that of
 * ember_step_dense(W, G, ...) on the stored G, up to the summation order of
 * the row and column sums of g^2, which here are formed by the GEMM's
 * epilogue from the stored values (fixed order, bit-reproducible), so the
 * step does not read G a second time for its statistics.
 *
 * T = 0 is allowed (G = 0; dY and H may then be NULL).  W, G, r, c, t, the
 * scalars, the workspace (ember_workspace_bytes(V, D), initialised by
 * ember_init_state) and the error rules are those of ember_step_dense;
 * additionally dY and H follow the layout rules of W and G, ldy and ldh must
 * be below EMBER_LMHEAD_MAX_LD and T at most EMBER_LMHEAD_MAX_T
 * (EMBER_ERR_SHAPE otherwise).  G must not overlap dY, H, W or the state.
 * The row-stride padding of dY and H (columns V..ldy-1 and D..ldh-1) is read
 * but never affects a stored value.
 */
int ember_lmhead_step(void* W, int w_dtype, int64_t ldw,
                      const void* dY, int64_t ldy, const void* H, int64_t ldh, int64_t T,
                      void* G, int g_dtype, int64_t ldg,
                      float* r, float* c, int64_t V, int64_t D, int64_t t,
                      float lr, float beta2, float eps, int maximize,
                      void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Device status of the most recent step enqueued with this workspace.
 * Synchronises `stream`, then sets *device_status to EMBER_OK or
 * EMBER_ERR_INDEX.  Returns EMBER_OK, EMBER_ERR_ARG or EMBER_ERR_HIP.
 */
int ember_get_error(const void* ws, hipStream_t stream, int* device_status);

/* Static description of a status code (never NULL). */
const char* ember_strerror(int status);

/*
 * Kernel timing (diagnostics).  While enabled, each kernel the library
 * launches is bracketed by two HIP events recorded on its stream.
 * ember_profile_collect waits for those events, writes per-kernel totals
 * (name, launch count, summed duration in milliseconds) for up to
 * max_entries kernels, sets *n_entries, and clears the record.
 */
typedef struct {
    const char* name;
    int64_t launches;
    double total_ms;
} ember_kernel_stat;

int ember_profile_enable(int enable);

/*
 * Bound of each grid-barrier wait of the one-launch sparse step
 * (diagnostics, for testing its failure path): `ticks` of the GPU's 100 MHz
 * real-time counter, for the steps enqueued after the call, process-wide;
 * 0 restores the default (1e8 ticks, about one second).  A wait that runs
 * out ends the launch normally and sets the timeout bit that
 * ember_get_error reports as EMBER_ERR_DEVICE (the state is then unspecified
 * until ember_init_state).  Returns EMBER_ERR_ARG for ticks < 0, else
 * EMBER_OK.
 */
int ember_set_barrier_wait_ticks(int64_t ticks);

/*
 * Streaming probe (diagnostics): reference rates of plain streaming kernels
 * over the same bytes as the passes above (not ceilings: the passes keep more
 * rows in flight per wavefront, and the apply pass finds part of G in the
 * last-level cache, so it runs faster than mode 2).  Enqueues one grid-stride
 * kernel with 16-byte non-temporal accesses over `bytes` bytes of each operand:
 *   mode 0: reads a (dst receives at most 4 bytes, in practice none);
 *   mode 1: dst <- a (copy);
 *   mode 2: dst <- a + b in 32-bit integer lanes (two reads, one write, as
 *           the apply pass reads G and W and writes W).
 * dst, a (and b for mode 2) are device pointers, 16-byte aligned, each
 * covering `bytes`, which must be a multiple of 16; dst must not overlap a
 * or b.  Returns EMBER_ERR_ARG (mode or null pointer), EMBER_ERR_SHAPE,
 * EMBER_ERR_ALIGN, EMBER_ERR_HIP or EMBER_OK.
 */
int ember_stream_probe(int mode, void* dst, const void* a, const void* b, size_t bytes, hipStream_t stream);
int ember_profile_collect(ember_kernel_stat* out, int max_entries, int* n_entries);

#ifdef __cplusplus
}
#endif

#endif /* EMBER_H */
