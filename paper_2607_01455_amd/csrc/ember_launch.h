// Internal interface between the host API (ember_api.cpp) and the HIP kernels
// (ember_kernels.hip).  Not installed; the public ABI is include/ember.h.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "ember.h"

namespace ember {

constexpr int kWave = 64;           // CDNA wavefront width
constexpr int kBlock = 256;         // threads per block: 4 waves
constexpr int kWaves = kBlock / kWave;

// Tuning constants of the kernels (measured choices; compile-time).
constexpr int kSlabChunks = 128;    // 16-byte chunks of a row per block (2 KiB)
constexpr int kStatsRows = 4;       // rows in flight per wave, statistics pass
constexpr int kApplyRows = 2;       // rows in flight per wave, apply pass
constexpr int kApplyBatches = 1;    // row batches per wave, apply pass
constexpr int kStatsKeepMB = 224;   // the statistics pass loads G non-temporally except its last
                                    // kStatsKeepMB of rows, which stay cached for the apply pass
constexpr bool kApplyNT = true;     // apply pass: non-temporal gradient loads and weight stores
constexpr bool kApplyWNT = true;    // apply pass: non-temporal weight loads
constexpr int kSparseRowsPerBlock = 32;   // minimum gradient rows per block, sparse step
constexpr int kSparseApplyBatches = 1;    // row batches per wave, apply pass of the sparse step
constexpr bool kRowOnlyNT = true;   // row-only kernels: non-temporal G/W loads and W stores
constexpr int kMaxBlocks = 384;     // row blocks of the statistics pass
constexpr int kRowsPerBlockMin = 8; // fewer rows than this per block: fewer blocks
constexpr int kVRowsPerThread = 1; // rows per thread in the r pass of finalize
constexpr int kFinCols = 64;        // columns per column block of finalize (16, 32 or 64)
constexpr int kDecayRows = 1024;    // rows per decay block of the row-only sparse step
constexpr int kTicketGroups = 16;   // first-level completion counters of the row-only sparse step ...
constexpr int kTicketStride = 64;   // ... this many words (256 bytes) apart
constexpr int64_t kMaxGridBlocks = (int64_t)1 << 20;  // launched blocks per kernel at most
int64_t capped_blocks(int64_t blocks);

// LM-head gradient GEMM tiles (ember_lmhead.hip): kLmheadTile x kLmheadTile
// tiles of G, kLmheadK tokens per step.
constexpr int kLmheadTile = 256;
constexpr int kLmheadK = 64;        // tokens per step

// Status bits written by the sparse statistics pass.
constexpr int kFlagRange = 1;
constexpr int kFlagDuplicate = 2;
constexpr int kFlagCount = 4;       // a device-side row count outside [0, max rows]
constexpr int kFlagTimeout = 8;     // the one-launch sparse step: a grid barrier's bounded wait ran
                                    // out (kept in the status word until ember_init_state)

// Column tiling of one launch for a given gradient dtype (16-byte chunks).
struct ColPlan {
    int epc;          // elements per 16-byte chunk of G: 4 (fp32) or 8 (bf16)
    int total_chunks; // ceil(D / epc)
    int nslab;        // column slabs: blocks per row block of the streaming kernels
    int slab_chunks;  // chunks per slab (last slab may hold fewer)
    int m;            // chunks per lane per slab: 1 or 2 (kSlabChunks / 64)
};

// Row blocking of the statistics pass for `rows` gradient rows of a table
// whose rows are cut into `nslab` column slabs.  The block count depends only
// on the row count, the slab count and the step kind, so results do not
// depend on the device.  At most kMaxBlocks row blocks, or more for narrow
// tables so that the launch still has about kStatsMinBlocks blocks (a
// 151936 x 896 fp32 table with two slabs: 1024 blocks instead of 768, which
// left a quarter of the chip's block slots empty; 113 -> 100 us).  The sparse
// step uses fewer, fuller blocks: its few thousand rows would otherwise
// produce more column partials than gradient.
constexpr int64_t kStatsMinBlocks = 1024;
inline int row_blocks(int64_t rows, int nslab, bool sparse = false) {
    const int64_t per = sparse ? kSparseRowsPerBlock : kRowsPerBlockMin;
    int64_t nb = (rows + per - 1) / per;
    int64_t cap = kStatsMinBlocks / (nslab > 0 ? nslab : 1);
    if (cap < kMaxBlocks) cap = kMaxBlocks;
    if (nb < 1) nb = 1;
    if (nb > cap) nb = cap;
    return (int)nb;
}
// Largest slab count over both gradient dtypes (fp32 has more chunks per row).
inline int nslab_for(int64_t D) {
    const int64_t chunks = (D + 3) / 4;
    return (int)((chunks + kSlabChunks - 1) / kSlabChunks);
}
// Row blocks of the apply pass (any count gives the same bits).  The sparse
// step has few rows, so its blocks are smaller to spread them over the chip.
inline int apply_blocks(int64_t rows, bool sparse = false) {
    const int64_t per = (int64_t)kWaves * kApplyRows * (sparse ? kSparseApplyBatches : kApplyBatches);
    int64_t nb = (rows + per - 1) / per;
    return (int)(nb < 1 ? 1 : nb);
}

ColPlan col_plan(int64_t D, int g_dtype);

// Workspace regions (byte offsets from the workspace base, 256-byte aligned).
struct WsLayout {
    size_t flag;    // int32: index-error bits set by the sparse statistics pass
    size_t status;  // int32: status of the last step (read by ember_get_error)
    size_t ticket;  // int32: blocks of the finalize pass that have finished
    size_t scale;   // float: sqrt(1 / (bias s)) / alpha_s of the last step
    size_t epoch;   // uint32: one-launch sparse steps taken (numbers their grid barriers)
    size_t oflag;   // int32[2]: error bits of the one-launch sparse steps, by epoch parity
    size_t taken;   // int32: 1 when the one-launch kernel took the current device-count step
    size_t arrive;  // uint32[kOnchipBlocks * kArriveStride]: last barrier number of each block
    size_t tgroups; // int32[kTicketGroups * kTicketStride]: first-level completion counters of the
                    // row-only sparse step
    size_t slot;    // int32[V]: 1 + position in idx of a touched row, else 0
    size_t zero_end;// [0, zero_end) must be zero before the first step
    size_t qa;      // float[D rounded up to 8]: column factors sqrt(c_j)
    size_t rowpart; // float[max(nslab, NT)][V]: per-slab (or per-column-tile) row sums of g^2
    size_t rsum;    // float[ceil(V / 1024)]: per-block sums of the new r
    size_t csum;    // float[ceil(D / kFinCols)]: per-block sums of the new c
    size_t p;       // float[max(row_blocks(V, nslab) over both dtypes, MT, kOnchipBlocks)][D]:
                    // per-block (or per-row-tile) column sums of g^2
    size_t parts;   // double[3][kOnchipBlocks]: per-block sums of the one-launch sparse step
    size_t cnew;    // float[D]: the new c of the one-launch sparse step until its stores
    size_t total;
};
WsLayout ws_layout(int64_t V, int64_t D);

struct StepArgs {
    void* W;
    int w_dtype;
    int64_t ldw;
    const void* G;
    int g_dtype;
    int64_t ldg;
    bool sparse;        // sparse-row step: G holds `rows` rows mapped through idx
    const int64_t* idx;    // sparse steps: device array of `rows` row indices
    const int64_t* n_dev;  // sparse steps: row count in device memory (rows is then its maximum), or null
    int* taken;         // device-count steps whose maximum is too large for the one-launch form: written
                        // by that launch (1: it took the step, the three launches then return at once),
                        // or null
    int64_t rows;       // V (dense) or n_idx (sparse)
    float* r;
    float* c;
    int64_t V;
    int64_t D;
    float beta2;
    float one_minus_beta2;
    double inv_bias;    // 1 / (1 - beta2^t)
    double inv_alpha;   // 1 / (+lr or -lr); 0 when lr == 0 (no apply launch)
    float eps_over_alpha;
    char* ws;
    int fin_nb;         // finalize: partial rows of P and row slabs of rowpart, when
    int fin_nslab;      // they come from the LM-head gradient GEMM (0: the statistics pass's)
    int64_t spin_ticks; // one-launch sparse step: bound of a grid-barrier wait (real-time
                        // counter ticks, 100 MHz)
};

// The sparse-row step in one launch (ember_kernels.hip): kOnchipBlocks blocks
// of kOnchipThreads threads, one per compute unit, all resident at once; each
// block holds its share of the gradient rows and of the weight rows they
// update in registers from the statistics to the update, and two grid
// barriers separate the statistics, the state update and the weight update.
constexpr int kOnchipBlocks = 256;
constexpr int kOnchipThreads = 512;
constexpr int kArriveStride = 16;  // words between two blocks' barrier flags (64 bytes)
constexpr int64_t kOnchipSpinTicks = 100000000;   // ~1 s: a barrier wait that long means lost residency
// True when the step's rows fit the launch (dtypes, slabs and row count) and
// the current device keeps every block of it resident.
bool onchip_fits(const StepArgs& a);
// The same without the row count: the launch could take the step for a count
// small enough (a device-count step decides on the device).
bool onchip_shape_fits(const StepArgs& a);
// Byte offsets (from base) of the regions the one-launch step uses.
struct OnchipSpace {
    char* base;
    size_t flag, flag_odd, status, epoch, arrive, slot, zero_end, qa, p, parts, cnew;
    int* status_ptr;    // if set, the status word (else base + status)
};
OnchipSpace onchip_space(const StepArgs& a);       // in the caller's workspace
hipError_t launch_sparse_onchip(const StepArgs& a, const OnchipSpace& sp, hipStream_t s);

// The one-launch step without a workspace (ember_step_sparse_rows_static): its
// regions sit in a kStaticScratchBytes array inside the library, one per
// device.  static_layout gives the offsets and the bytes a (V, D) step needs;
// static_scratch the array's device address on the current device;
// launch_static_prep zeroes [0, zero_bytes) of it and the caller's status word.
constexpr size_t kStaticScratchBytes = (size_t)16 << 20;
size_t static_layout(int64_t V, int64_t D, OnchipSpace* sp);
hipError_t static_scratch(char** out);
hipError_t launch_static_prep(char* base, size_t zero_bytes, int* status, hipStream_t s);

// Each launcher enqueues one kernel on `s` and returns hipGetLastError().
hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);
hipError_t launch_stats(const StepArgs& a, hipStream_t s);
hipError_t launch_finalize(const StepArgs& a, hipStream_t s);
hipError_t launch_apply(const StepArgs& a, hipStream_t s);

// Streaming probe (ember_probe.hip): mode 0 read, 1 copy, 2 dst = a + b.
hipError_t launch_stream_probe(int mode, void* dst, const void* a, const void* b, size_t bytes, hipStream_t s);

// Several tables per launch (ember_step_multi).  Tables whose keys are equal
// use the same kernel instance and may share a launch; each launcher takes
// tables of one key, in the order their blocks are to be numbered.
constexpr int kMaxTables = EMBER_MAX_TABLES;
int stats_key(const StepArgs& a);
int apply_key(const StepArgs& a);
hipError_t launch_stats_multi(const StepArgs* const* t, int n, hipStream_t s);
hipError_t launch_finalize_multi(const StepArgs* const* t, int n, hipStream_t s);
hipError_t launch_apply_multi(const StepArgs* const* t, int n, hipStream_t s);
// Row-only tables: id validation of the sparse ones (one launch), then the
// fused pass; rowonly_key is -1 for tables whose rows are too long for the
// one-wave kernel (each of those gets a launch of its own).
int rowonly_key(const StepArgs& a);
hipError_t launch_rowonly_validate_multi(const StepArgs* const* t, int n, hipStream_t s);
hipError_t launch_rowonly_multi(const StepArgs* const* t, int n, hipStream_t s);

// LM-head weight gradient G = dY^T H with the statistics partials in the
// epilogue (ember_lmhead.hip): rowpart[NT][V] and P[MT][D] in the workspace.
struct LmheadPlan {
    int MT;   // row tiles: ceil(V / kLmheadTile)
    int NT;   // column tiles: ceil(D / kLmheadTile)
};
LmheadPlan lmhead_plan(int64_t V, int64_t D);
struct LmheadArgs {
    const void* dY;    // [T][ldy] bf16
    int64_t ldy;
    const void* H;     // [T][ldh] bf16
    int64_t ldh;
    int64_t T;
    int64_t V;
    int64_t D;
    void* G;           // [V][ldg]
    int g_dtype;
    int64_t ldg;
    float* rowpart;
    float* P;
};
hipError_t launch_lmhead_grad(const LmheadArgs& a, hipStream_t s);

// Row-only Ember (one fused pass over the rows; the sparse step first
// validates idx and marks the touched rows).
hipError_t launch_rowonly_validate(const StepArgs& a, hipStream_t s);
hipError_t launch_rowonly(const StepArgs& a, hipStream_t s);

// Gradient coalescing (ember_coalesce.hip): token ids and per-position rows
// -> distinct ids and summed rows.
struct CoalArgs {
    const int64_t* tok;
    int64_t P;
    const void* U;
    int u_dtype;
    int64_t ldu;
    int64_t V;
    int64_t D;
    int64_t* idx;
    void* G;
    int g_dtype;
    int64_t ldg;
    int64_t* n_out;
    char* ws;
};

struct CoalPlan {
    int ntiles;        // sort tiles
    int passes;        // radix passes
    int digit_bits;
    int64_t L;         // chunk length of the sums
    int nchunks;
    int nslabs;
    size_t keys_a, vals_a, keys_b, vals_b, hist, offs, tile_bad, tilecnt, tileoff, uid, seg_start;
    size_t part_a, part_b, fix_list, fix_count;
    size_t total;      // workspace bytes
};
CoalPlan coal_plan(int64_t P, int64_t V, int64_t D);
hipError_t launch_coalesce(const CoalArgs& a, hipStream_t s);

} // namespace ember
