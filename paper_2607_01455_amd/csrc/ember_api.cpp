// Host side of the Ember C ABI (include/ember.h): argument validation, scalar
// preparation in float64, workspace layout and the launch sequence of one step.
// Every check runs before anything is enqueued.

#include "ember.h"

#include <atomic>
#include <cmath>
#include <mutex>
#include <string>
#include <vector>

#include "ember_launch.h"

namespace {

using ember::StepArgs;
using ember::WsLayout;

bool dtype_ok(int d) { return d == EMBER_F32 || d == EMBER_BF16; }
size_t dtype_size(int d) { return d == EMBER_F32 ? 4 : 2; }

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int check_shape(int64_t V, int64_t D) {
    if (V < 1 || D < 1 || V > EMBER_MAX_V || D > EMBER_MAX_D) return EMBER_ERR_SHAPE;
    return EMBER_OK;
}

int check_matrix(const void* p, int dtype, int64_t ld, int64_t D, bool may_be_null) {
    if (!dtype_ok(dtype)) return EMBER_ERR_DTYPE;
    if (ld < D) return EMBER_ERR_SHAPE;
    if (p == nullptr) return may_be_null ? EMBER_OK : EMBER_ERR_ARG;
    if (!aligned(p, 16) || ((ld * (int64_t)dtype_size(dtype)) % 16) != 0) return EMBER_ERR_ALIGN;
    return EMBER_OK;
}

int check_scalars(int64_t t, float lr, float beta2, float eps) {
    if (t < 1) return EMBER_ERR_ARG;
    if (!(beta2 >= 0.0f && beta2 < 1.0f)) return EMBER_ERR_ARG;
    if (!(lr >= 0.0f) || !std::isfinite(lr)) return EMBER_ERR_ARG;
    if (!(eps >= 0.0f) || !std::isfinite(eps)) return EMBER_ERR_ARG;
    return EMBER_OK;
}

int check_state(const float* r, const float* c, const void* ws, size_t ws_bytes, int64_t V, int64_t D) {
    if (r == nullptr || c == nullptr || ws == nullptr) return EMBER_ERR_ARG;
    if (!aligned(r, 4) || !aligned(c, 4) || !aligned(ws, 256)) return EMBER_ERR_ALIGN;
    if (ws_bytes < ember::ws_layout(V, D).total) return EMBER_ERR_WORKSPACE;
    return EMBER_OK;
}

// ---------------------------------------------------------------------------
// optional kernel timing
// ---------------------------------------------------------------------------

struct Record {
    const char* name;
    hipEvent_t start;
    hipEvent_t stop;
};

std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<Record> g_records;
std::vector<hipEvent_t> g_free_events;

hipEvent_t take_event() {
    if (!g_free_events.empty()) {
        hipEvent_t e = g_free_events.back();
        g_free_events.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

template <typename F>
hipError_t timed(const char* name, hipStream_t s, F&& launch) {
    if (!g_prof_on) return launch();
    std::lock_guard<std::mutex> lock(g_prof_mu);
    Record rec{name, take_event(), take_event()};
    if (rec.start) (void)hipEventRecord(rec.start, s);
    hipError_t err = launch();
    if (rec.stop) (void)hipEventRecord(rec.stop, s);
    if (rec.start && rec.stop) g_records.push_back(rec);
    return err;
}

// ---------------------------------------------------------------------------
// one step
// ---------------------------------------------------------------------------

void set_scalars(StepArgs& a, float lr, float beta2, float eps, int64_t t, int maximize);

int run_step(StepArgs& a, float lr, float beta2, float eps, int64_t t, int maximize, hipStream_t s) {
    set_scalars(a, lr, beta2, eps, t, maximize);
    // A sparse step whose rows fit on chip runs as one launch.
    if (ember::onchip_fits(a)) {
        const hipError_t e = timed("ember_sparse_onchip", s, [&] {
            return ember::launch_sparse_onchip(a, ember::onchip_space(a), s);
        });
        return e == hipSuccess ? EMBER_OK : EMBER_ERR_HIP;
    }
    // A device-count step whose maximum does not fit may still hold few enough
    // rows: the one-launch kernel reads the count and takes the step when it
    // fits (marking that in the workspace), and the three launches below then
    // return at once; otherwise they take it.
    hipError_t e = hipSuccess;
    if (a.n_dev != nullptr && ember::onchip_shape_fits(a)) {
        a.taken = reinterpret_cast<int*>(a.ws + ember::ws_layout(a.V, a.D).taken);
        e = timed("ember_sparse_onchip", s, [&] { return ember::launch_sparse_onchip(a, ember::onchip_space(a), s); });
    }
    if (e == hipSuccess) e = timed("ember_stats", s, [&] { return ember::launch_stats(a, s); });
    if (e == hipSuccess) e = timed("ember_finalize", s, [&] { return ember::launch_finalize(a, s); });
    // lr == 0 leaves every weight bit unchanged, so the dense step skips the
    // apply pass; the sparse apply pass also clears the index-error flag for the
    // next step, so it always runs (and returns before the row loop when lr == 0).
    if (e == hipSuccess && (lr > 0.0f || a.sparse))
        e = timed("ember_apply", s, [&] { return ember::launch_apply(a, s); });
    return e == hipSuccess ? EMBER_OK : EMBER_ERR_HIP;
}

// Bound of a grid-barrier wait of the one-launch sparse step (real-time counter
// ticks); 0: the default.  Set by ember_set_barrier_wait_ticks.
std::atomic<int64_t> g_barrier_wait_ticks{0};

void set_scalars(StepArgs& a, float lr, float beta2, float eps, int64_t t, int maximize) {
    const double b2 = (double)beta2;
    a.beta2 = beta2;
    a.one_minus_beta2 = (float)(1.0 - b2);
    a.inv_bias = 1.0 / (1.0 - std::pow(b2, (double)t));
    const double alpha_s = maximize ? (double)lr : -(double)lr;
    a.inv_alpha = lr > 0.0f ? 1.0 / alpha_s : 0.0;
    a.eps_over_alpha = lr > 0.0f ? (float)((double)eps / alpha_s) : 0.0f;
    const int64_t w = g_barrier_wait_ticks.load(std::memory_order_relaxed);
    a.spin_ticks = w > 0 ? w : ember::kOnchipSpinTicks;
}

// LM-head step: the weight-gradient GEMM writes G and the statistics
// partials, then the finalize and apply passes of the dense step run on them.
int run_lmhead_step(StepArgs& a, const ember::LmheadArgs& x, float lr, float beta2, float eps, int64_t t,
                    int maximize, hipStream_t s) {
    set_scalars(a, lr, beta2, eps, t, maximize);
    const ember::LmheadPlan pl = ember::lmhead_plan(a.V, a.D);
    a.fin_nb = pl.MT;
    a.fin_nslab = pl.NT;
    hipError_t e = timed("ember_lmhead_grad", s, [&] { return ember::launch_lmhead_grad(x, s); });
    if (e == hipSuccess) e = timed("ember_finalize", s, [&] { return ember::launch_finalize(a, s); });
    if (e == hipSuccess && lr > 0.0f) e = timed("ember_apply", s, [&] { return ember::launch_apply(a, s); });
    return e == hipSuccess ? EMBER_OK : EMBER_ERR_HIP;
}

int run_rowonly_step(StepArgs& a, float lr, float beta2, float eps, int64_t t, int maximize, hipStream_t s) {
    set_scalars(a, lr, beta2, eps, t, maximize);
    hipError_t e = hipSuccess;
    if (a.sparse) e = timed("ember_rowonly_validate", s, [&] { return ember::launch_rowonly_validate(a, s); });
    if (e == hipSuccess) e = timed("ember_rowonly", s, [&] { return ember::launch_rowonly(a, s); });
    return e == hipSuccess ? EMBER_OK : EMBER_ERR_HIP;
}

// Arguments of the sparse steps whose row count is in device memory.
int check_devn(const void* W, int w_dtype, int64_t ldw, const void* G_rows, int g_dtype, int64_t ldg,
               const int64_t* idx, const int64_t* n_dev, int64_t max_rows, int64_t V, int64_t D) {
    int st = check_shape(V, D);
    if (st == EMBER_OK && (max_rows < 0 || max_rows > V)) st = EMBER_ERR_SHAPE;
    if (st == EMBER_OK) st = check_matrix(W, w_dtype, ldw, D, false);
    if (st == EMBER_OK) st = check_matrix(G_rows, g_dtype, ldg, D, max_rows == 0);
    if (st == EMBER_OK && ((max_rows > 0 && idx == nullptr) || n_dev == nullptr)) st = EMBER_ERR_ARG;
    if (st == EMBER_OK && ((idx != nullptr && !aligned(idx, 8)) || !aligned(n_dev, 8))) st = EMBER_ERR_ALIGN;
    return st;
}

int check_rowonly_state(const float* r, const void* ws, size_t ws_bytes, int64_t V, int64_t D) {
    if (r == nullptr || ws == nullptr) return EMBER_ERR_ARG;
    if (!aligned(r, 4) || !aligned(ws, 256)) return EMBER_ERR_ALIGN;
    if (ws_bytes < ember::ws_layout(V, D).total) return EMBER_ERR_WORKSPACE;
    return EMBER_OK;
}

// Byte range [lo, hi) of device memory an argument covers.
struct Span {
    uintptr_t lo, hi;
};
bool overlap(Span a, Span b) { return a.lo < b.hi && b.lo < a.hi; }
Span span_of(const void* p, size_t bytes) {
    const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
    return Span{lo, lo + bytes};
}

// Checks one table of ember_step_multi as its own call would check it.
int check_table(const ember_table_step& x) {
    int st = check_shape(x.V, x.D);
    if (st != EMBER_OK) return st;
    if (x.sparse != 0 && x.sparse != 1) return EMBER_ERR_ARG;
    if (!x.sparse) {
        st = check_matrix(x.W, x.w_dtype, x.ldw, x.D, false);
        if (st == EMBER_OK) st = check_matrix(x.G, x.g_dtype, x.ldg, x.D, false);
    } else if (x.n_idx_dev != nullptr) {
        st = check_devn(x.W, x.w_dtype, x.ldw, x.G, x.g_dtype, x.ldg, x.idx, x.n_idx_dev, x.n_idx, x.V, x.D);
    } else {
        if (x.n_idx < 0 || x.n_idx > x.V) st = EMBER_ERR_SHAPE;
        if (st == EMBER_OK) st = check_matrix(x.W, x.w_dtype, x.ldw, x.D, false);
        if (st == EMBER_OK) st = check_matrix(x.G, x.g_dtype, x.ldg, x.D, x.n_idx == 0);
        if (st == EMBER_OK && x.n_idx > 0 && x.idx == nullptr) st = EMBER_ERR_ARG;
        if (st == EMBER_OK && x.idx != nullptr && !aligned(x.idx, 8)) st = EMBER_ERR_ALIGN;
    }
    if (st == EMBER_OK && x.row_only != 0 && x.row_only != 1) st = EMBER_ERR_ARG;
    if (st == EMBER_OK)
        st = x.row_only ? check_rowonly_state(x.r, x.ws, x.ws_bytes, x.V, x.D)
                        : check_state(x.r, x.c, x.ws, x.ws_bytes, x.V, x.D);
    if (st == EMBER_OK) st = check_scalars(x.t, x.lr, x.beta2, x.eps);
    return st;
}

// Bytes of a rows x D matrix with leading dimension ld (0 rows: none).
size_t matrix_bytes(int64_t rows, int64_t ld, int64_t D, int dtype) {
    return rows > 0 ? ((size_t)(rows - 1) * (size_t)ld + (size_t)D) * dtype_size(dtype) : 0;
}

// The memory one table writes: workspace, r, c and W ...
constexpr int kWriteSpans = 4;
void table_write_spans(const ember_table_step& x, Span out[kWriteSpans]) {
    out[0] = span_of(x.ws, ember::ws_layout(x.V, x.D).total);
    out[1] = span_of(x.r, (size_t)x.V * 4);
    out[2] = x.row_only ? span_of(nullptr, 0) : span_of(x.c, (size_t)x.D * 4);
    out[3] = span_of(x.W, matrix_bytes(x.V, x.ldw, x.D, x.w_dtype));
}

// ... and the memory it only reads: G (V rows, or the n_idx rows of a sparse
// step), the id list and the device row count.
constexpr int kReadSpans = 3;
void table_read_spans(const ember_table_step& x, Span out[kReadSpans]) {
    const int64_t rows = x.sparse ? x.n_idx : x.V;
    out[0] = span_of(x.G, matrix_bytes(rows, x.ldg, x.D, x.g_dtype));
    out[1] = x.sparse ? span_of(x.idx, (size_t)(x.n_idx > 0 ? x.n_idx : 0) * 8) : span_of(nullptr, 0);
    out[2] = x.sparse && x.n_idx_dev != nullptr ? span_of(x.n_idx_dev, 8) : span_of(nullptr, 0);
}

// Whether a span table i writes overlaps any span of table j.
bool writes_overlap(const ember_table_step& i, const ember_table_step& j) {
    Span wi[kWriteSpans], wj[kWriteSpans], rj[kReadSpans];
    table_write_spans(i, wi);
    table_write_spans(j, wj);
    table_read_spans(j, rj);
    for (const Span& a : wi) {
        for (const Span& b : wj)
            if (overlap(a, b)) return true;
        for (const Span& b : rj)
            if (overlap(a, b)) return true;
    }
    return false;
}

// Launches of one phase: tables in `order`, grouped by kernel key in order of
// first appearance, one launcher call per group.
template <typename Key, typename Launch>
hipError_t run_phase(const std::vector<const StepArgs*>& order, Key key, Launch launch, hipStream_t s) {
    std::vector<int> keys;
    for (const StepArgs* a : order) {
        const int k = key(*a);
        bool seen = false;
        for (int q : keys) seen = seen || q == k;
        if (!seen) keys.push_back(k);
    }
    for (int k : keys) {
        std::vector<const StepArgs*> group;
        for (const StepArgs* a : order)
            if (key(*a) == k) group.push_back(a);
        const hipError_t e = launch(group.data(), (int)group.size(), s);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

} // namespace

extern "C" {

int ember_workspace_bytes(int64_t V, int64_t D, size_t* bytes) {
    if (bytes == nullptr) return EMBER_ERR_ARG;
    int st = check_shape(V, D);
    if (st != EMBER_OK) return st;
    *bytes = ember::ws_layout(V, D).total;
    return EMBER_OK;
}

int ember_init_state(float* r, float* c, int64_t V, int64_t D, void* ws, size_t ws_bytes, hipStream_t stream) {
    int st = check_shape(V, D);
    if (st != EMBER_OK) return st;
    st = check_state(r, c, ws, ws_bytes, V, D);
    if (st != EMBER_OK) return st;
    const WsLayout L = ember::ws_layout(V, D);
    hipError_t e = ember::launch_zero(r, (size_t)V * 4, stream);
    if (e == hipSuccess) e = ember::launch_zero(c, (size_t)D * 4, stream);
    if (e == hipSuccess) e = ember::launch_zero(ws, L.zero_end, stream);
    return e == hipSuccess ? EMBER_OK : EMBER_ERR_HIP;
}

int ember_step_dense(void* W, int w_dtype, int64_t ldw, const void* G, int g_dtype, int64_t ldg,
                     float* r, float* c, int64_t V, int64_t D, int64_t t,
                     float lr, float beta2, float eps, int maximize,
                     void* ws, size_t ws_bytes, hipStream_t stream) {
    int st = check_shape(V, D);
    if (st == EMBER_OK) st = check_matrix(W, w_dtype, ldw, D, false);
    if (st == EMBER_OK) st = check_matrix(G, g_dtype, ldg, D, false);
    if (st == EMBER_OK) st = check_state(r, c, ws, ws_bytes, V, D);
    if (st == EMBER_OK) st = check_scalars(t, lr, beta2, eps);
    if (st != EMBER_OK) return st;
    StepArgs a{};
    a.sparse = false;
    a.W = W;
    a.w_dtype = w_dtype;
    a.ldw = ldw;
    a.G = G;
    a.g_dtype = g_dtype;
    a.ldg = ldg;
    a.idx = nullptr;
    a.rows = V;
    a.r = r;
    a.c = c;
    a.V = V;
    a.D = D;
    a.ws = static_cast<char*>(ws);
    return run_step(a, lr, beta2, eps, t, maximize, stream);
}

int ember_lmhead_step(void* W, int w_dtype, int64_t ldw,
                      const void* dY, int64_t ldy, const void* H, int64_t ldh, int64_t T,
                      void* G, int g_dtype, int64_t ldg,
                      float* r, float* c, int64_t V, int64_t D, int64_t t,
                      float lr, float beta2, float eps, int maximize,
                      void* ws, size_t ws_bytes, hipStream_t stream) {
    int st = check_shape(V, D);
    if (st == EMBER_OK && (T < 0 || T > EMBER_LMHEAD_MAX_T)) st = EMBER_ERR_SHAPE;
    if (st == EMBER_OK && (ldy >= EMBER_LMHEAD_MAX_LD || ldh >= EMBER_LMHEAD_MAX_LD)) st = EMBER_ERR_SHAPE;
    if (st == EMBER_OK) st = check_matrix(W, w_dtype, ldw, D, false);
    if (st == EMBER_OK) st = check_matrix(G, g_dtype, ldg, D, false);
    if (st == EMBER_OK) st = check_matrix(dY, EMBER_BF16, ldy, V, T == 0);
    if (st == EMBER_OK) st = check_matrix(H, EMBER_BF16, ldh, D, T == 0);
    if (st == EMBER_OK) st = check_state(r, c, ws, ws_bytes, V, D);
    if (st == EMBER_OK) st = check_scalars(t, lr, beta2, eps);
    if (st != EMBER_OK) return st;
    const WsLayout L = ember::ws_layout(V, D);
    ember::LmheadArgs x{};
    x.dY = dY;
    x.ldy = ldy;
    x.H = H;
    x.ldh = ldh;
    x.T = T;
    x.V = V;
    x.D = D;
    x.G = G;
    x.g_dtype = g_dtype;
    x.ldg = ldg;
    x.rowpart = reinterpret_cast<float*>(static_cast<char*>(ws) + L.rowpart);
    x.P = reinterpret_cast<float*>(static_cast<char*>(ws) + L.p);
    StepArgs a{};
    a.sparse = false;
    a.W = W;
    a.w_dtype = w_dtype;
    a.ldw = ldw;
    a.G = G;
    a.g_dtype = g_dtype;
    a.ldg = ldg;
    a.idx = nullptr;
    a.rows = V;
    a.r = r;
    a.c = c;
    a.V = V;
    a.D = D;
    a.ws = static_cast<char*>(ws);
    return run_lmhead_step(a, x, lr, beta2, eps, t, maximize, stream);
}

int ember_step_sparse_rows(void* W, int w_dtype, int64_t ldw, const void* G_rows, int g_dtype, int64_t ldg,
                           const int64_t* idx, int64_t n_idx,
                           float* r, float* c, int64_t V, int64_t D, int64_t t,
                           float lr, float beta2, float eps, int maximize,
                           void* ws, size_t ws_bytes, hipStream_t stream) {
    int st = check_shape(V, D);
    if (st == EMBER_OK && (n_idx < 0 || n_idx > V)) st = EMBER_ERR_SHAPE;
    if (st == EMBER_OK) st = check_matrix(W, w_dtype, ldw, D, false);
    if (st == EMBER_OK) st = check_matrix(G_rows, g_dtype, ldg, D, n_idx == 0);
    if (st == EMBER_OK && n_idx > 0 && idx == nullptr) st = EMBER_ERR_ARG;
    if (st == EMBER_OK && idx != nullptr && !aligned(idx, 8)) st = EMBER_ERR_ALIGN;
    if (st == EMBER_OK) st = check_state(r, c, ws, ws_bytes, V, D);
    if (st == EMBER_OK) st = check_scalars(t, lr, beta2, eps);
    if (st != EMBER_OK) return st;
    StepArgs a{};
    a.sparse = true;
    a.W = W;
    a.w_dtype = w_dtype;
    a.ldw = ldw;
    a.G = G_rows;
    a.g_dtype = g_dtype;
    a.ldg = ldg;
    a.idx = idx;
    a.rows = n_idx;
    a.r = r;
    a.c = c;
    a.V = V;
    a.D = D;
    a.ws = static_cast<char*>(ws);
    return run_step(a, lr, beta2, eps, t, maximize, stream);
}

int ember_step_multi(const ember_table_step* tables, int n_tables, hipStream_t stream) {
    if (tables == nullptr || n_tables < 1 || n_tables > EMBER_MAX_TABLES) return EMBER_ERR_ARG;
    for (int i = 0; i < n_tables; ++i) {
        const int st = check_table(tables[i]);
        if (st != EMBER_OK) return st;
    }
    // no table may write memory another table reads or writes (the tables
    // share launches, so such a pair would race); read-only spans may be shared
    for (int i = 0; i < n_tables; ++i)
        for (int j = 0; j < n_tables; ++j)
            if (i != j && writes_overlap(tables[i], tables[j])) return EMBER_ERR_ARG;
    std::vector<StepArgs> args((size_t)n_tables);
    for (int i = 0; i < n_tables; ++i) {
        const ember_table_step& x = tables[i];
        StepArgs& a = args[(size_t)i];
        a = StepArgs{};
        a.sparse = x.sparse != 0;
        a.W = x.W;
        a.w_dtype = x.w_dtype;
        a.ldw = x.ldw;
        a.G = x.G;
        a.g_dtype = x.g_dtype;
        a.ldg = x.ldg;
        a.idx = a.sparse ? x.idx : nullptr;
        a.n_dev = a.sparse ? x.n_idx_dev : nullptr;
        a.rows = a.sparse ? x.n_idx : x.V;
        a.r = x.r;
        a.c = x.row_only ? nullptr : x.c;
        a.V = x.V;
        a.D = x.D;
        a.ws = static_cast<char*>(x.ws);
        set_scalars(a, x.lr, x.beta2, x.eps, x.t, x.maximize);
    }
    std::vector<bool> row_only((size_t)n_tables);
    for (int i = 0; i < n_tables; ++i) row_only[(size_t)i] = tables[i].row_only != 0;
    // Canonical sparse tables whose rows fit on chip take the one-launch step
    // (the same kernel as their own call), before the shared launches: its
    // ~116 MB of traffic would otherwise pass through the last-level cache
    // between the dense tables' statistics and apply passes.
    // The other canonical tables share a statistics, a finalize and an apply
    // launch.  Statistics blocks: dense tables first (a sparse table's few
    // blocks first would delay a whole round of the long dense blocks), then
    // the sparse ones; the apply pass keeps that order, so the dense rows that
    // the statistics pass read last (left in the last-level cache, read first
    // by the apply pass going from high rows to low) come first.  A dense
    // table with lr = 0 keeps every weight and has no apply blocks; a sparse
    // one still clears its index-error flag there.
    // Row-only tables: the sparse ones' id checks, then one fused pass.
    std::vector<const StepArgs*> onchip, stats_order, apply_order, ro_sparse, ro_all;
    for (size_t i = 0; i < args.size(); ++i)
        if (!row_only[i] && ember::onchip_fits(args[i])) onchip.push_back(&args[i]);
    auto shared = [&](size_t i) {
        if (row_only[i]) return false;
        for (const StepArgs* o : onchip)
            if (o == &args[i]) return false;
        return true;
    };
    for (size_t i = 0; i < args.size(); ++i)
        if (shared(i) && !args[i].sparse) stats_order.push_back(&args[i]);
    for (size_t i = 0; i < args.size(); ++i)
        if (shared(i) && args[i].sparse) stats_order.push_back(&args[i]);
    for (const StepArgs* a : stats_order)
        if (a->sparse || a->inv_alpha != 0.0) apply_order.push_back(a);
    for (size_t i = 0; i < args.size(); ++i) {
        if (!row_only[i]) continue;
        // a sparse table with no rows and a host count has no ids to check
        if (args[i].sparse && (args[i].rows > 0 || args[i].n_dev != nullptr)) ro_sparse.push_back(&args[i]);
        ro_all.push_back(&args[i]);
    }
    hipError_t e = hipSuccess;
    for (const StepArgs* a : onchip) {
        if (e == hipSuccess)
            e = timed("ember_sparse_onchip", stream, [&] {
                return ember::launch_sparse_onchip(*a, ember::onchip_space(*a), stream);
            });
    }
    if (e == hipSuccess && !ro_sparse.empty())
        e = timed("ember_rowonly_validate_multi", stream, [&] {
            return run_phase(ro_sparse, [](const StepArgs&) { return 0; }, ember::launch_rowonly_validate_multi,
                             stream);
        });
    if (e == hipSuccess && !stats_order.empty())
        e = timed("ember_stats_multi", stream, [&] {
            return run_phase(stats_order, ember::stats_key, ember::launch_stats_multi, stream);
        });
    if (e == hipSuccess && !stats_order.empty())
        e = timed("ember_finalize_multi", stream, [&] {
            return run_phase(stats_order, [](const StepArgs&) { return 0; }, ember::launch_finalize_multi, stream);
        });
    if (e == hipSuccess && !apply_order.empty())
        e = timed("ember_apply_multi", stream, [&] {
            return run_phase(apply_order, ember::apply_key, ember::launch_apply_multi, stream);
        });
    if (e == hipSuccess && !ro_all.empty())
        e = timed("ember_rowonly_multi", stream, [&] {
            return run_phase(ro_all, ember::rowonly_key, ember::launch_rowonly_multi, stream);
        });
    return e == hipSuccess ? EMBER_OK : EMBER_ERR_HIP;
}

int ember_step_sparse_rows_static(void* W, int w_dtype, int64_t ldw, const void* G_rows, int g_dtype, int64_t ldg,
                                  const int64_t* idx, int64_t n_idx, float* r, float* c, int64_t V, int64_t D,
                                  int64_t t, float lr, float beta2, float eps, int maximize, int32_t* status,
                                  hipStream_t stream) {
    int st = check_shape(V, D);
    if (st == EMBER_OK && (n_idx < 0 || n_idx > V)) st = EMBER_ERR_SHAPE;
    if (st == EMBER_OK) st = check_matrix(W, w_dtype, ldw, D, false);
    if (st == EMBER_OK) st = check_matrix(G_rows, g_dtype, ldg, D, n_idx == 0);
    if (st == EMBER_OK && ((n_idx > 0 && idx == nullptr) || r == nullptr || c == nullptr || status == nullptr))
        st = EMBER_ERR_ARG;
    if (st == EMBER_OK && ((idx != nullptr && !aligned(idx, 8)) || !aligned(r, 4) || !aligned(c, 4) ||
                           !aligned(status, 4)))
        st = EMBER_ERR_ALIGN;
    if (st == EMBER_OK) st = check_scalars(t, lr, beta2, eps);
    ember::OnchipSpace sp{};
    if (st == EMBER_OK && ember::static_layout(V, D, &sp) > ember::kStaticScratchBytes) st = EMBER_ERR_WORKSPACE;
    if (st != EMBER_OK) return st;
    StepArgs a{};
    a.sparse = true;
    a.W = W;
    a.w_dtype = w_dtype;
    a.ldw = ldw;
    a.G = G_rows;
    a.g_dtype = g_dtype;
    a.ldg = ldg;
    a.idx = idx;
    a.rows = n_idx;
    a.r = r;
    a.c = c;
    a.V = V;
    a.D = D;
    set_scalars(a, lr, beta2, eps, t, maximize);
    if (!ember::onchip_fits(a)) return EMBER_ERR_SHAPE;
    if (ember::static_scratch(&sp.base) != hipSuccess) return EMBER_ERR_HIP;
    sp.status_ptr = status;
    hipError_t e = ember::launch_static_prep(sp.base, sp.zero_end, status, stream);
    if (e == hipSuccess)
        e = timed("ember_sparse_onchip", stream, [&] { return ember::launch_sparse_onchip(a, sp, stream); });
    return e == hipSuccess ? EMBER_OK : EMBER_ERR_HIP;
}

int ember_rowonly_init_state(float* r, int64_t V, int64_t D, void* ws, size_t ws_bytes, hipStream_t stream) {
    int st = check_shape(V, D);
    if (st != EMBER_OK) return st;
    st = check_rowonly_state(r, ws, ws_bytes, V, D);
    if (st != EMBER_OK) return st;
    const WsLayout L = ember::ws_layout(V, D);
    hipError_t e = ember::launch_zero(r, (size_t)V * 4, stream);
    if (e == hipSuccess) e = ember::launch_zero(ws, L.zero_end, stream);
    return e == hipSuccess ? EMBER_OK : EMBER_ERR_HIP;
}

int ember_rowonly_step_dense(void* W, int w_dtype, int64_t ldw, const void* G, int g_dtype, int64_t ldg,
                             float* r, int64_t V, int64_t D, int64_t t,
                             float lr, float beta2, float eps, int maximize,
                             void* ws, size_t ws_bytes, hipStream_t stream) {
    int st = check_shape(V, D);
    if (st == EMBER_OK) st = check_matrix(W, w_dtype, ldw, D, false);
    if (st == EMBER_OK) st = check_matrix(G, g_dtype, ldg, D, false);
    if (st == EMBER_OK) st = check_rowonly_state(r, ws, ws_bytes, V, D);
    if (st == EMBER_OK) st = check_scalars(t, lr, beta2, eps);
    if (st != EMBER_OK) return st;
    StepArgs a{};
    a.sparse = false;
    a.W = W;
    a.w_dtype = w_dtype;
    a.ldw = ldw;
    a.G = G;
    a.g_dtype = g_dtype;
    a.ldg = ldg;
    a.idx = nullptr;
    a.rows = V;
    a.r = r;
    a.c = nullptr;
    a.V = V;
    a.D = D;
    a.ws = static_cast<char*>(ws);
    return run_rowonly_step(a, lr, beta2, eps, t, maximize, stream);
}

int ember_rowonly_step_sparse_rows(void* W, int w_dtype, int64_t ldw, const void* G_rows, int g_dtype, int64_t ldg,
                                   const int64_t* idx, int64_t n_idx,
                                   float* r, int64_t V, int64_t D, int64_t t,
                                   float lr, float beta2, float eps, int maximize,
                                   void* ws, size_t ws_bytes, hipStream_t stream) {
    int st = check_shape(V, D);
    if (st == EMBER_OK && (n_idx < 0 || n_idx > V)) st = EMBER_ERR_SHAPE;
    if (st == EMBER_OK) st = check_matrix(W, w_dtype, ldw, D, false);
    if (st == EMBER_OK) st = check_matrix(G_rows, g_dtype, ldg, D, n_idx == 0);
    if (st == EMBER_OK && n_idx > 0 && idx == nullptr) st = EMBER_ERR_ARG;
    if (st == EMBER_OK && idx != nullptr && !aligned(idx, 8)) st = EMBER_ERR_ALIGN;
    if (st == EMBER_OK) st = check_rowonly_state(r, ws, ws_bytes, V, D);
    if (st == EMBER_OK) st = check_scalars(t, lr, beta2, eps);
    if (st != EMBER_OK) return st;
    StepArgs a{};
    a.sparse = true;
    a.W = W;
    a.w_dtype = w_dtype;
    a.ldw = ldw;
    a.G = G_rows;
    a.g_dtype = g_dtype;
    a.ldg = ldg;
    a.idx = idx;
    a.rows = n_idx;
    a.r = r;
    a.c = nullptr;
    a.V = V;
    a.D = D;
    a.ws = static_cast<char*>(ws);
    return run_rowonly_step(a, lr, beta2, eps, t, maximize, stream);
}

int ember_step_sparse_rows_devn(void* W, int w_dtype, int64_t ldw, const void* G_rows, int g_dtype, int64_t ldg,
                                const int64_t* idx, const int64_t* n_idx_dev, int64_t max_rows,
                                float* r, float* c, int64_t V, int64_t D, int64_t t,
                                float lr, float beta2, float eps, int maximize,
                                void* ws, size_t ws_bytes, hipStream_t stream) {
    int st = check_devn(W, w_dtype, ldw, G_rows, g_dtype, ldg, idx, n_idx_dev, max_rows, V, D);
    if (st == EMBER_OK) st = check_state(r, c, ws, ws_bytes, V, D);
    if (st == EMBER_OK) st = check_scalars(t, lr, beta2, eps);
    if (st != EMBER_OK) return st;
    StepArgs a{};
    a.sparse = true;
    a.W = W;
    a.w_dtype = w_dtype;
    a.ldw = ldw;
    a.G = G_rows;
    a.g_dtype = g_dtype;
    a.ldg = ldg;
    a.idx = idx;
    a.n_dev = n_idx_dev;
    a.rows = max_rows;
    a.r = r;
    a.c = c;
    a.V = V;
    a.D = D;
    a.ws = static_cast<char*>(ws);
    return run_step(a, lr, beta2, eps, t, maximize, stream);
}

int ember_rowonly_step_sparse_rows_devn(void* W, int w_dtype, int64_t ldw, const void* G_rows, int g_dtype,
                                        int64_t ldg, const int64_t* idx, const int64_t* n_idx_dev,
                                        int64_t max_rows, float* r, int64_t V, int64_t D, int64_t t,
                                        float lr, float beta2, float eps, int maximize,
                                        void* ws, size_t ws_bytes, hipStream_t stream) {
    int st = check_devn(W, w_dtype, ldw, G_rows, g_dtype, ldg, idx, n_idx_dev, max_rows, V, D);
    if (st == EMBER_OK) st = check_rowonly_state(r, ws, ws_bytes, V, D);
    if (st == EMBER_OK) st = check_scalars(t, lr, beta2, eps);
    if (st != EMBER_OK) return st;
    StepArgs a{};
    a.sparse = true;
    a.W = W;
    a.w_dtype = w_dtype;
    a.ldw = ldw;
    a.G = G_rows;
    a.g_dtype = g_dtype;
    a.ldg = ldg;
    a.idx = idx;
    a.n_dev = n_idx_dev;
    a.rows = max_rows;
    a.r = r;
    a.c = nullptr;
    a.V = V;
    a.D = D;
    a.ws = static_cast<char*>(ws);
    return run_rowonly_step(a, lr, beta2, eps, t, maximize, stream);
}

int ember_coalesce_workspace_bytes(int64_t max_tokens, int64_t V, int64_t D, size_t* bytes) {
    if (bytes == nullptr) return EMBER_ERR_ARG;
    int st = check_shape(V, D);
    if (st != EMBER_OK) return st;
    if (max_tokens < 0 || max_tokens > EMBER_MAX_TOKENS) return EMBER_ERR_SHAPE;
    *bytes = ember::coal_plan(max_tokens, V, D).total;
    return EMBER_OK;
}

int ember_coalesce_rows(const int64_t* tok, int64_t n_tok, const void* U, int u_dtype, int64_t ldu,
                        int64_t V, int64_t D, int64_t* idx, void* G_rows, int g_dtype, int64_t ldg,
                        int64_t* n_out, void* ws, size_t ws_bytes, hipStream_t stream) {
    int st = check_shape(V, D);
    if (st == EMBER_OK && (n_tok < 0 || n_tok > EMBER_MAX_TOKENS)) st = EMBER_ERR_SHAPE;
    if (st == EMBER_OK) st = check_matrix(U, u_dtype, ldu, D, n_tok == 0);
    if (st == EMBER_OK) st = check_matrix(G_rows, g_dtype, ldg, D, n_tok == 0);
    if (st == EMBER_OK && n_tok > 0 && (tok == nullptr || idx == nullptr)) st = EMBER_ERR_ARG;
    if (st == EMBER_OK && n_out == nullptr) st = EMBER_ERR_ARG;
    if (st == EMBER_OK && ws == nullptr) st = EMBER_ERR_ARG;
    if (st == EMBER_OK && ((tok != nullptr && !aligned(tok, 8)) || (idx != nullptr && !aligned(idx, 8)) ||
                           !aligned(n_out, 8) || !aligned(ws, 256)))
        st = EMBER_ERR_ALIGN;
    if (st == EMBER_OK && ws_bytes < ember::coal_plan(n_tok, V, D).total) st = EMBER_ERR_WORKSPACE;
    if (st != EMBER_OK) return st;
    ember::CoalArgs a;
    a.tok = tok;
    a.P = n_tok;
    a.U = U;
    a.u_dtype = u_dtype;
    a.ldu = ldu;
    a.V = V;
    a.D = D;
    a.idx = idx;
    a.G = G_rows;
    a.g_dtype = g_dtype;
    a.ldg = ldg;
    a.n_out = n_out;
    a.ws = static_cast<char*>(ws);
    hipError_t e = timed("ember_coalesce", stream, [&] { return ember::launch_coalesce(a, stream); });
    return e == hipSuccess ? EMBER_OK : EMBER_ERR_HIP;
}

int ember_get_error(const void* ws, hipStream_t stream, int* device_status) {
    if (ws == nullptr || device_status == nullptr) return EMBER_ERR_ARG;
    if (!aligned(ws, 256)) return EMBER_ERR_ALIGN;
    if (hipStreamSynchronize(stream) != hipSuccess) return EMBER_ERR_HIP;
    int flag = 0;
    const char* base = static_cast<const char*>(ws);
    if (hipMemcpy(&flag, base + ember::ws_layout(1, 1).status, sizeof flag, hipMemcpyDeviceToHost) != hipSuccess)
        return EMBER_ERR_HIP;
    *device_status = (flag & ember::kFlagTimeout) ? EMBER_ERR_DEVICE : flag != 0 ? EMBER_ERR_INDEX : EMBER_OK;
    return EMBER_OK;
}

const char* ember_strerror(int status) {
    switch (status) {
    case EMBER_OK: return "success";
    case EMBER_ERR_ARG: return "invalid argument (null pointer or scalar out of range)";
    case EMBER_ERR_SHAPE: return "invalid shape (V, D, leading dimension or index count)";
    case EMBER_ERR_ALIGN: return "misaligned pointer or leading dimension";
    case EMBER_ERR_DTYPE: return "unsupported dtype (expected EMBER_F32 or EMBER_BF16)";
    case EMBER_ERR_WORKSPACE: return "workspace too small";
    case EMBER_ERR_INDEX: return "row index out of range or repeated";
    case EMBER_ERR_HIP: return "HIP runtime error";
    case EMBER_ERR_DEVICE: return "device-side failure: the blocks of the one-launch sparse step were not all resident";
    default: return "unknown status";
    }
}

int ember_stream_probe(int mode, void* dst, const void* a, const void* b, size_t bytes, hipStream_t stream) {
    if (mode < 0 || mode > 2 || dst == nullptr || a == nullptr || (mode == 2 && b == nullptr))
        return EMBER_ERR_ARG;
    if (bytes % 16 != 0) return EMBER_ERR_SHAPE;
    if (!aligned(dst, 16) || !aligned(a, 16) || (b != nullptr && !aligned(b, 16))) return EMBER_ERR_ALIGN;
    const hipError_t e = timed("ember_stream_probe", stream,
                               [&] { return ember::launch_stream_probe(mode, dst, a, b, bytes, stream); });
    return e == hipSuccess ? EMBER_OK : EMBER_ERR_HIP;
}

int ember_set_barrier_wait_ticks(int64_t ticks) {
    if (ticks < 0) return EMBER_ERR_ARG;
    g_barrier_wait_ticks.store(ticks, std::memory_order_relaxed);
    return EMBER_OK;
}

int ember_profile_enable(int enable) {
    std::lock_guard<std::mutex> lock(g_prof_mu);
    g_prof_on = enable != 0;
    return EMBER_OK;
}

int ember_profile_collect(ember_kernel_stat* out, int max_entries, int* n_entries) {
    if (n_entries == nullptr || (out == nullptr && max_entries > 0)) return EMBER_ERR_ARG;
    std::lock_guard<std::mutex> lock(g_prof_mu);
    std::vector<ember_kernel_stat> stats;
    int rc = EMBER_OK;
    for (const Record& rec : g_records) {
        float ms = 0.0f;
        if (hipEventSynchronize(rec.stop) != hipSuccess || hipEventElapsedTime(&ms, rec.start, rec.stop) != hipSuccess)
            rc = EMBER_ERR_HIP;
        size_t k = 0;
        while (k < stats.size() && std::string(stats[k].name) != rec.name) ++k;
        if (k == stats.size()) stats.push_back(ember_kernel_stat{rec.name, 0, 0.0});
        stats[k].launches += 1;
        stats[k].total_ms += ms;
        g_free_events.push_back(rec.start);
        g_free_events.push_back(rec.stop);
    }
    g_records.clear();
    int n = 0;
    for (const ember_kernel_stat& st : stats) {
        if (n < max_entries) out[n] = st;
        ++n;
    }
    *n_entries = n < max_entries ? n : max_entries;
    return rc;
}

} // extern "C"
