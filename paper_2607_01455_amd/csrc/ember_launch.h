// Internal interface between the host API (ember_api.cpp) and the HIP kernels
// (ember_kernels.hip).  Not installed; the public ABI is include/ember.h.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

namespace ember {

constexpr int kWave = 64;           // CDNA wavefront width
constexpr int kBlock = 256;         // threads per block: 4 waves
constexpr int kMaxBlocks = 1024;    // row blocks of the statistics pass
constexpr int kRowsPerBlockMin = 8; // fewer rows than this per block: fewer blocks
constexpr int kGroup = 16;          // partial rows summed per first-level column group
constexpr int kVRowsPerThread = 4;  // rows per thread in the r pass
constexpr int kVRowsPerBlock = kBlock * kVRowsPerThread;
constexpr int kMaxAcc = 64;         // fp32 column accumulators per lane (one slab)
constexpr int kSlabCols = 4096;     // columns per slab for both dtypes (64 lanes x 64 acc)

// Status bits written by the sparse statistics pass.
constexpr int kFlagRange = 1;
constexpr int kFlagDuplicate = 2;

// Column tiling of one launch for a given gradient dtype (16-byte chunks).
struct ColPlan {
    int epc;          // elements per 16-byte chunk of G: 4 (fp32) or 8 (bf16)
    int total_chunks; // ceil(D / epc)
    int nslab;        // grid.y of the streaming kernels
    int slab_chunks;  // chunks per slab (last slab may hold fewer)
    int m;            // chunks per lane per slab, a power of two in 1..16
};

// Row blocking of the statistics pass for `rows` gradient rows.  The block
// count depends only on the row count, so results do not depend on the device.
inline int row_blocks(int64_t rows) {
    int64_t nb = (rows + kRowsPerBlockMin - 1) / kRowsPerBlockMin;
    if (nb < 1) nb = 1;
    if (nb > kMaxBlocks) nb = kMaxBlocks;
    return (int)nb;
}
inline int col_groups(int nb) { return (nb + kGroup - 1) / kGroup; }
inline int nslab_for(int64_t D) { return (int)((D + kSlabCols - 1) / kSlabCols); }

ColPlan col_plan(int64_t D, int g_dtype);

// Workspace regions (byte offsets from the workspace base, 256-byte aligned).
struct WsLayout {
    size_t flag;    // int32: index-error bits set by the sparse statistics pass
    size_t status;  // int32: status of the last step (read by ember_get_error)
    size_t slot;    // int32[V]: 1 + position in idx of a touched row, else 0
    size_t zero_end;// [0, zero_end) must be zero before the first step
    size_t rowpart; // float[nslab][V]: per-slab row sums of g^2
    size_t rsum;    // float[ceil(V / kVRowsPerBlock)]: per-block sums of the new r
    size_t csum;    // float[ceil(D / kBlock)]: per-block sums of the new c
    size_t p;       // float[row_blocks(V)][D]: per-block column sums of g^2
    size_t p2;      // float[col_groups(row_blocks(V))][D]
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
    const int64_t* idx; // device array of `rows` row indices (sparse only)
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
};

// Each launcher enqueues one kernel on `s` and returns hipGetLastError().
hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);
hipError_t launch_stats(const StepArgs& a, hipStream_t s);
hipError_t launch_finalize_rows(const StepArgs& a, hipStream_t s);
hipError_t launch_finalize_cols(const StepArgs& a, hipStream_t s);
hipError_t launch_apply(const StepArgs& a, hipStream_t s);

} // namespace ember
