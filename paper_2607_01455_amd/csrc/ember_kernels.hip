// HIP kernels of the Ember step for gfx950 (MI355X).
//
// One step (Token Geometry, Algorithm 1) is four launches on one stream:
//   ember_stats        reads G once: per-row sums of g^2 (wave reduction) and
//                      per-block column sums of g^2 (per-lane registers, then
//                      a fixed-order LDS combine of the block's 4 waves).
//                      The sparse form also validates idx and marks touched rows.
//   ember_finalize_rows  first level of the column reduction (groups of 16
//                      block partials) and the r update over all V rows.
//   ember_finalize_cols  second level of the column reduction and the c update.
//   ember_apply        reads G and W, writes W: the update with the factored
//                      preconditioner applied as a row factor times a column
//                      factor (never stored).
// Every reduction runs in an order fixed by (V, D, n), with no floating-point
// atomics, so results are bitwise reproducible.
//
// Mapping of the two streaming kernels: one wavefront per gradient row, each
// lane owning 16-byte chunks lane, lane + 64, ... of a column slab (<= 4096
// columns), so every load and store is a coalesced 1 KiB wave access.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ember_launch.h"

namespace ember {
namespace {

// ---------------------------------------------------------------------------
// element access
// ---------------------------------------------------------------------------

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

typedef float float2_v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));

// Round-to-nearest-even of two floats to bf16 (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    float2_v f = {lo, hi};
    bf16x2_v b = __builtin_convertvector(f, bf16x2_v);
    return __builtin_bit_cast(uint32_t, b);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float x) {
    return (uint16_t)(pack_bf16x2(x, 0.0f) & 0xFFFFu);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
    static __device__ __forceinline__ float load(const float* p) { return *p; }
    static __device__ __forceinline__ void store(float* p, float v) { *p = v; }
};
template <> struct Elem<uint16_t> {
    static __device__ __forceinline__ float load(const uint16_t* p) { return bf16_to_f32(*p); }
    static __device__ __forceinline__ void store(uint16_t* p, float v) { *p = f32_to_bf16(v); }
};

template <typename T, int N>
__device__ __forceinline__ void decode(const uint32_t* u, float (&x)[N]) {
    if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int e = 0; e < N; ++e) x[e] = __uint_as_float(u[e]);
    } else {
#pragma unroll
        for (int e = 0; e < N / 2; ++e) {
            x[2 * e] = bf16_lo(u[e]);
            x[2 * e + 1] = bf16_hi(u[e]);
        }
    }
}

template <typename T, int N>
__device__ __forceinline__ void encode(const float (&x)[N], uint32_t* u) {
    if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int e = 0; e < N; ++e) u[e] = __float_as_uint(x[e]);
    } else {
#pragma unroll
        for (int e = 0; e < N / 2; ++e) u[e] = pack_bf16x2(x[2 * e], x[2 * e + 1]);
    }
}

// Vector load/store of N elements at p (16-byte aligned, or 8 for 8-byte chunks).
template <typename T, int N>
__device__ __forceinline__ void vload(const T* p, float (&x)[N]) {
    constexpr int kWords = N * (int)sizeof(T) / 4;
    uint32_t u[kWords];
    if constexpr (kWords == 2) {
        uint2 v = *reinterpret_cast<const uint2*>(p);
        u[0] = v.x; u[1] = v.y;
    } else {
#pragma unroll
        for (int q = 0; q < kWords / 4; ++q) {
            uint4 v = reinterpret_cast<const uint4*>(p)[q];
            u[4 * q] = v.x; u[4 * q + 1] = v.y; u[4 * q + 2] = v.z; u[4 * q + 3] = v.w;
        }
    }
    decode<T, N>(u, x);
}

template <typename T, int N>
__device__ __forceinline__ void vstore(T* p, const float (&x)[N]) {
    constexpr int kWords = N * (int)sizeof(T) / 4;
    uint32_t u[kWords];
    encode<T, N>(x, u);
    if constexpr (kWords == 2) {
        *reinterpret_cast<uint2*>(p) = make_uint2(u[0], u[1]);
    } else {
#pragma unroll
        for (int q = 0; q < kWords / 4; ++q)
            reinterpret_cast<uint4*>(p)[q] = make_uint4(u[4 * q], u[4 * q + 1], u[4 * q + 2], u[4 * q + 3]);
    }
}

// Chunk `col .. col+N` of a row: vector access when it lies inside [0, D),
// element access for the partial last chunk, zeros when `valid` is false.
template <typename T, int N>
__device__ __forceinline__ void load_chunk(const T* row, int64_t col, bool valid, int64_t D, float (&x)[N]) {
    if (valid && col + N <= D) {
        vload<T, N>(row + col, x);
    } else {
#pragma unroll
        for (int e = 0; e < N; ++e) x[e] = (valid && col + e < D) ? Elem<T>::load(row + col + e) : 0.0f;
    }
}

template <typename T, int N>
__device__ __forceinline__ void store_chunk(T* row, int64_t col, int64_t D, const float (&x)[N]) {
    if (col + N <= D) {
        vstore<T, N>(row + col, x);
    } else {
#pragma unroll
        for (int e = 0; e < N; ++e)
            if (col + e < D) Elem<T>::store(row + col + e, x[e]);
    }
}

// ---------------------------------------------------------------------------
// fixed-order reductions
// ---------------------------------------------------------------------------

// Butterfly sum over the 64 lanes.  x + y == y + x in IEEE arithmetic, so every
// lane ends with the same bits and the order is fixed.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

// Sum of one float per thread of the block: waves first, then wave 0..3 in order.
__device__ __forceinline__ float block_sum(float v, float* lds4) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    v = wave_sum(v);
    if (lane == 0) lds4[wave] = v;
    __syncthreads();
    return ((lds4[0] + lds4[1]) + lds4[2]) + lds4[3];
}

__device__ __forceinline__ void row_range(int64_t rows, int nb, int b, int64_t& r0, int64_t& r1) {
    r0 = rows * b / nb;
    r1 = rows * (b + 1) / nb;
}

// ---------------------------------------------------------------------------
// statistics pass: row sums and per-block column sums of g^2
// ---------------------------------------------------------------------------

struct StatsParams {
    const void* G;
    int64_t ldg;
    int64_t rows;
    int64_t D;
    int total_chunks;
    int slab_chunks;
    int nb;
    float* rowpart;      // [nslab][rows]
    float* P;            // [nb][D]
    const int64_t* idx;  // sparse only
    int64_t V;
    int* slot;
    int* flag;
};

template <typename GT, int M, bool kSparse>
__global__ __launch_bounds__(kBlock) void ember_stats(StatsParams a) {
    constexpr int EPC = 16 / (int)sizeof(GT);
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int slab = blockIdx.y;
    int64_t r0, r1;
    row_range(a.rows, a.nb, blockIdx.x, r0, r1);
    const int cbeg = slab * a.slab_chunks;
    const int cend = min(cbeg + a.slab_chunks, a.total_chunks);
    const GT* G = static_cast<const GT*>(a.G);

    float acc[M][EPC];
#pragma unroll
    for (int m = 0; m < M; ++m)
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[m][e] = 0.0f;

    for (int64_t row = r0 + wave; row < r1; row += kBlock / kWave) {
        const GT* grow = G + row * a.ldg;
        float x[M][EPC];
#pragma unroll
        for (int m = 0; m < M; ++m) {
            const int ch = cbeg + lane + kWave * m;
            load_chunk<GT, EPC>(grow, (int64_t)ch * EPC, ch < cend, a.D, x[m]);
        }
        float rs0 = 0.0f, rs1 = 0.0f;
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                acc[m][e] = fmaf(x[m][e], x[m][e], acc[m][e]);
                if (e & 1) rs1 = fmaf(x[m][e], x[m][e], rs1);
                else rs0 = fmaf(x[m][e], x[m][e], rs0);
            }
        const float rs = wave_sum(rs0 + rs1);
        if (lane == 0) {
            a.rowpart[(int64_t)slab * a.rows + row] = rs;
            if (kSparse && slab == 0) {
                const int64_t i = a.idx[row];
                if (i < 0 || i >= a.V) {
                    atomicOr(a.flag, kFlagRange);
                } else if (atomicCAS(&a.slot[i], 0, (int)(row + 1)) != 0) {
                    atomicOr(a.flag, kFlagDuplicate);
                }
            }
        }
    }

    // Combine the 4 waves' column sums in a fixed order, one chunk column at a time.
    __shared__ float lds[kBlock / kWave][kWave * EPC];
    float* P = a.P + (int64_t)blockIdx.x * a.D;
#pragma unroll
    for (int m = 0; m < M; ++m) {
#pragma unroll
        for (int e = 0; e < EPC; ++e) lds[wave][lane * EPC + e] = acc[m][e];
        __syncthreads();
        for (int x = threadIdx.x; x < kWave * EPC; x += kBlock) {
            const int ch = cbeg + kWave * m + x / EPC;
            const int64_t col = (int64_t)(cbeg + kWave * m) * EPC + x;
            if (ch < cend && col < a.D)
                P[col] = ((lds[0][x] + lds[1][x]) + lds[2][x]) + lds[3][x];
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// finalize, rows: column partials level 1, and r over all V rows
// ---------------------------------------------------------------------------

struct FinRowsParams {
    const float* P;
    float* P2;
    int nb;
    int ng;
    int64_t D;
    int ncolblocks;
    const float* rowpart;
    int nslab;
    int64_t rows;
    int64_t V;
    float* r;
    int* slot;
    const int* flag;
    float beta2;
    float one_minus_beta2;
    float* rsum;
};

template <bool kSparse>
__global__ __launch_bounds__(kBlock) void ember_finalize_rows(FinRowsParams a) {
    __shared__ float lds4[kBlock / kWave];
    if ((int)blockIdx.x < a.ncolblocks) {
        const int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
        if (t >= (int64_t)a.ng * a.D) return;
        const int g = (int)(t / a.D);
        const int64_t j = t - (int64_t)g * a.D;
        const int b0 = g * kGroup;
        const int b1 = min(b0 + kGroup, a.nb);
        float s = 0.0f;
        for (int b = b0; b < b1; ++b) s += a.P[(int64_t)b * a.D + j];
        a.P2[(int64_t)g * a.D + j] = s;
        return;
    }
    const int vb = blockIdx.x - a.ncolblocks;
    const int err = kSparse ? *a.flag : 0;
    const double invD = 1.0 / (double)a.D;
    float part = 0.0f;
#pragma unroll
    for (int q = 0; q < kVRowsPerThread; ++q) {
        const int64_t i = (int64_t)vb * kVRowsPerBlock + q * kBlock + threadIdx.x;
        if (i >= a.V) continue;
        int64_t k = i;
        bool touched = true;
        if (kSparse) {
            const int sl = a.slot[i];
            touched = sl != 0;
            k = (int64_t)sl - 1;
            if (sl != 0) a.slot[i] = 0;
        }
        if (err) continue;
        float rn;
        if (touched) {
            float sum = 0.0f;
            for (int sb = 0; sb < a.nslab; ++sb) sum += a.rowpart[(int64_t)sb * a.rows + k];
            const float mean = (float)((double)sum * invD);
            rn = fmaf(a.beta2, a.r[i], a.one_minus_beta2 * mean);
        } else {
            rn = a.beta2 * a.r[i];
        }
        a.r[i] = rn;
        part += rn;
    }
    const float tot = block_sum(part, lds4);
    if (threadIdx.x == 0) a.rsum[vb] = tot;
}

// ---------------------------------------------------------------------------
// finalize, columns: column partials level 2 and c
// ---------------------------------------------------------------------------

struct FinColsParams {
    const float* P2;
    int ng;
    int64_t D;
    int64_t V;
    float* c;
    const int* flag;   // nullptr: dense step
    int* status;
    float beta2;
    float one_minus_beta2;
    float* csum;
};

__global__ __launch_bounds__(kBlock) void ember_finalize_cols(FinColsParams a) {
    __shared__ float lds4[kBlock / kWave];
    const int64_t j = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int err = a.flag ? *a.flag : 0;
    const double invV = 1.0 / (double)a.V;
    float cn = 0.0f;
    if (j < a.D) {
        float s = 0.0f;
        for (int g = 0; g < a.ng; ++g) s += a.P2[(int64_t)g * a.D + j];
        if (!err) {
            const float mean = (float)((double)s * invV);
            cn = fmaf(a.beta2, a.c[j], a.one_minus_beta2 * mean);
            a.c[j] = cn;
        }
    }
    const float tot = block_sum(cn, lds4);
    if (threadIdx.x == 0) {
        a.csum[blockIdx.x] = tot;
        if (blockIdx.x == 0) *a.status = err;
    }
}

// ---------------------------------------------------------------------------
// apply: W += g * alpha_s / (a_i q_j + eps), a_i = sqrt(rhat_i), q_j = sqrt(chat_j / s)
// ---------------------------------------------------------------------------

struct ApplyParams {
    void* W;
    int64_t ldw;
    const void* G;
    int64_t ldg;
    int64_t rows;
    int64_t D;
    int total_chunks;
    int slab_chunks;
    int nb;
    const int64_t* idx;   // sparse only
    const float* r;
    const float* c;
    const float* rsum;
    int nrsum;
    const float* csum;
    int ncsum;
    int64_t V;
    double inv_bias;
    double inv_alpha;     // 1 / alpha_s, alpha_s = -lr (descent) or +lr (ascent)
    float eps_over_alpha; // eps / alpha_s
    const int* status;    // sparse only: skip when the statistics pass flagged idx
    int* flag;            // sparse only: cleared for the next step
};

template <typename GT, typename WT, int M, bool kSparse>
__global__ __launch_bounds__(kBlock) void ember_apply(ApplyParams a) {
    constexpr int EPC = 16 / (int)sizeof(GT);
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    if (kSparse) {
        if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *a.flag = 0;
        if (*a.status != 0) return;
    }
    if (a.inv_alpha == 0.0) return;   // lr == 0: every weight keeps its bits

    // Normaliser s = sqrt(mean(rhat) mean(chat)) from the per-block sums, in a
    // fixed order (identical in every wave of every block).
    double sr = 0.0, sc = 0.0;
    for (int k = lane; k < a.nrsum; k += kWave) sr += (double)a.rsum[k];
    for (int k = lane; k < a.ncsum; k += kWave) sc += (double)a.csum[k];
    sr = wave_sum(sr);
    sc = wave_sum(sc);
    const double mean_rhat = sr / (double)a.V * a.inv_bias;
    const double mean_chat = sc / (double)a.D * a.inv_bias;
    const double s = sqrt(mean_rhat * mean_chat);

    const int slab = blockIdx.y;
    const int cbeg = slab * a.slab_chunks;
    const int cend = min(cbeg + a.slab_chunks, a.total_chunks);

    // Column factors of this lane's columns, pre-divided by alpha_s.
    const double kq = s > 0.0 ? a.inv_bias / s : 0.0;
    float qa[M][EPC];
#pragma unroll
    for (int m = 0; m < M; ++m) {
        const int ch = cbeg + lane + kWave * m;
#pragma unroll
        for (int e = 0; e < EPC; ++e) {
            const int64_t col = (int64_t)ch * EPC + e;
            float q = 0.0f;
            if (ch < cend && col < a.D && s > 0.0)
                q = (float)(sqrt((double)a.c[col] * kq) * a.inv_alpha);
            qa[m][e] = q;
        }
    }
    const float epsa = a.eps_over_alpha;
    const float ibias = (float)a.inv_bias;

    // Row blocks in reverse order: the rows the statistics pass read last are
    // the likeliest still to sit in the last-level cache.
    int64_t r0, r1;
    row_range(a.rows, a.nb, a.nb - 1 - (int)blockIdx.x, r0, r1);
    const GT* G = static_cast<const GT*>(a.G);
    WT* W = static_cast<WT*>(a.W);

    for (int64_t row = r0 + wave; row < r1; row += kBlock / kWave) {
        const int64_t wrow = kSparse ? a.idx[row] : row;
        const float ai = sqrtf(a.r[wrow] * ibias);
        const GT* grow = G + row * a.ldg;
        WT* wr = W + wrow * a.ldw;
        float g[M][EPC], w[M][EPC];
#pragma unroll
        for (int m = 0; m < M; ++m) {
            const int ch = cbeg + lane + kWave * m;
            load_chunk<GT, EPC>(grow, (int64_t)ch * EPC, ch < cend, a.D, g[m]);
            load_chunk<WT, EPC>(wr, (int64_t)ch * EPC, ch < cend, a.D, w[m]);
        }
#pragma unroll
        for (int m = 0; m < M; ++m) {
            const int ch = cbeg + lane + kWave * m;
            float o[EPC];
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                const float d = fmaf(ai, qa[m][e], epsa);
                const float upd = fmaf(g[m][e], __builtin_amdgcn_rcpf(d), w[m][e]);
                o[e] = (g[m][e] == 0.0f) ? w[m][e] : upd;
            }
            if (ch < cend) store_chunk<WT, EPC>(wr, (int64_t)ch * EPC, a.D, o);
        }
    }
}

// ---------------------------------------------------------------------------
// zero fill (used instead of a memset node so the step stays capturable)
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void ember_zero(uint32_t* p, int64_t words) {
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < words; i += (int64_t)gridDim.x * kBlock)
        p[i] = 0u;
}

// ---------------------------------------------------------------------------
// dispatch on (G dtype, W dtype, chunks per lane)
// ---------------------------------------------------------------------------

template <typename GT, bool kSparse>
hipError_t stats_dispatch(const StatsParams& p, int m, dim3 grid, hipStream_t s) {
    switch (m) {
    case 1: ember_stats<GT, 1, kSparse><<<grid, kBlock, 0, s>>>(p); break;
    case 2: ember_stats<GT, 2, kSparse><<<grid, kBlock, 0, s>>>(p); break;
    case 4: ember_stats<GT, 4, kSparse><<<grid, kBlock, 0, s>>>(p); break;
    case 8: ember_stats<GT, 8, kSparse><<<grid, kBlock, 0, s>>>(p); break;
    case 16:
        if constexpr (sizeof(GT) == 4) { ember_stats<GT, 16, kSparse><<<grid, kBlock, 0, s>>>(p); break; }
        return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <typename GT, typename WT, bool kSparse>
hipError_t apply_dispatch(const ApplyParams& p, int m, dim3 grid, hipStream_t s) {
    switch (m) {
    case 1: ember_apply<GT, WT, 1, kSparse><<<grid, kBlock, 0, s>>>(p); break;
    case 2: ember_apply<GT, WT, 2, kSparse><<<grid, kBlock, 0, s>>>(p); break;
    case 4: ember_apply<GT, WT, 4, kSparse><<<grid, kBlock, 0, s>>>(p); break;
    case 8: ember_apply<GT, WT, 8, kSparse><<<grid, kBlock, 0, s>>>(p); break;
    case 16:
        if constexpr (sizeof(GT) == 4) { ember_apply<GT, WT, 16, kSparse><<<grid, kBlock, 0, s>>>(p); break; }
        return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <typename GT, bool kSparse>
hipError_t apply_dispatch_w(const ApplyParams& p, int w_dtype, int m, dim3 grid, hipStream_t s) {
    if (w_dtype == 0) return apply_dispatch<GT, float, kSparse>(p, m, grid, s);
    return apply_dispatch<GT, uint16_t, kSparse>(p, m, grid, s);
}

} // namespace

ColPlan col_plan(int64_t D, int g_dtype) {
    ColPlan cp;
    cp.epc = g_dtype == 0 ? 4 : 8;
    cp.total_chunks = (int)((D + cp.epc - 1) / cp.epc);
    const int max_m = kMaxAcc / cp.epc;               // 16 (fp32) or 8 (bf16)
    cp.nslab = (cp.total_chunks + kWave * max_m - 1) / (kWave * max_m);
    cp.slab_chunks = (cp.total_chunks + cp.nslab - 1) / cp.nslab;
    const int need = (cp.slab_chunks + kWave - 1) / kWave;
    cp.m = 1;
    while (cp.m < need) cp.m *= 2;
    return cp;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

WsLayout ws_layout(int64_t V, int64_t D) {
    WsLayout L;
    const int nb = row_blocks(V);
    size_t off = 0;
    L.flag = off;
    L.status = off + 4;
    off = align256(8);
    L.slot = off;
    off = align256(off + (size_t)V * 4);
    L.zero_end = off;
    L.rowpart = off;
    off = align256(off + (size_t)nslab_for(D) * (size_t)V * 4);
    L.rsum = off;
    off = align256(off + (size_t)((V + kVRowsPerBlock - 1) / kVRowsPerBlock) * 4);
    L.csum = off;
    off = align256(off + (size_t)((D + kBlock - 1) / kBlock) * 4);
    L.p = off;
    off = align256(off + (size_t)nb * (size_t)D * 4);
    L.p2 = off;
    off = align256(off + (size_t)col_groups(nb) * (size_t)D * 4);
    L.total = off;
    return L;
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s) {
    const int64_t words = (int64_t)(bytes / 4);
    if (words == 0) return hipSuccess;
    int64_t blocks = (words + kBlock - 1) / kBlock;
    if (blocks > 4096) blocks = 4096;
    ember_zero<<<dim3((unsigned)blocks), kBlock, 0, s>>>(static_cast<uint32_t*>(p), words);
    return hipGetLastError();
}

hipError_t launch_stats(const StepArgs& a, hipStream_t s) {
    const WsLayout L = ws_layout(a.V, a.D);
    const ColPlan cp = col_plan(a.D, a.g_dtype);
    StatsParams p;
    p.G = a.G;
    p.ldg = a.ldg;
    p.rows = a.rows;
    p.D = a.D;
    p.total_chunks = cp.total_chunks;
    p.slab_chunks = cp.slab_chunks;
    p.nb = row_blocks(a.rows);
    p.rowpart = reinterpret_cast<float*>(a.ws + L.rowpart);
    p.P = reinterpret_cast<float*>(a.ws + L.p);
    p.idx = a.idx;
    p.V = a.V;
    p.slot = reinterpret_cast<int*>(a.ws + L.slot);
    p.flag = reinterpret_cast<int*>(a.ws + L.flag);
    const dim3 grid((unsigned)p.nb, (unsigned)cp.nslab);
    const bool sparse = a.sparse;
    if (a.g_dtype == 0)
        return sparse ? stats_dispatch<float, true>(p, cp.m, grid, s) : stats_dispatch<float, false>(p, cp.m, grid, s);
    return sparse ? stats_dispatch<uint16_t, true>(p, cp.m, grid, s) : stats_dispatch<uint16_t, false>(p, cp.m, grid, s);
}

hipError_t launch_finalize_rows(const StepArgs& a, hipStream_t s) {
    const WsLayout L = ws_layout(a.V, a.D);
    FinRowsParams p;
    p.P = reinterpret_cast<const float*>(a.ws + L.p);
    p.P2 = reinterpret_cast<float*>(a.ws + L.p2);
    p.nb = row_blocks(a.rows);
    p.ng = col_groups(p.nb);
    p.D = a.D;
    p.ncolblocks = (int)(((int64_t)p.ng * a.D + kBlock - 1) / kBlock);
    p.rowpart = reinterpret_cast<const float*>(a.ws + L.rowpart);
    p.nslab = col_plan(a.D, a.g_dtype).nslab;
    p.rows = a.rows;
    p.V = a.V;
    p.r = a.r;
    p.slot = reinterpret_cast<int*>(a.ws + L.slot);
    p.flag = reinterpret_cast<const int*>(a.ws + L.flag);
    p.beta2 = a.beta2;
    p.one_minus_beta2 = a.one_minus_beta2;
    p.rsum = reinterpret_cast<float*>(a.ws + L.rsum);
    const int nvb = (int)((a.V + kVRowsPerBlock - 1) / kVRowsPerBlock);
    const dim3 grid((unsigned)(p.ncolblocks + nvb));
    if (a.sparse)
        ember_finalize_rows<true><<<grid, kBlock, 0, s>>>(p);
    else
        ember_finalize_rows<false><<<grid, kBlock, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_finalize_cols(const StepArgs& a, hipStream_t s) {
    const WsLayout L = ws_layout(a.V, a.D);
    FinColsParams p;
    p.P2 = reinterpret_cast<const float*>(a.ws + L.p2);
    p.ng = col_groups(row_blocks(a.rows));
    p.D = a.D;
    p.V = a.V;
    p.c = a.c;
    p.flag = a.sparse ? reinterpret_cast<const int*>(a.ws + L.flag) : nullptr;
    p.status = reinterpret_cast<int*>(a.ws + L.status);
    p.beta2 = a.beta2;
    p.one_minus_beta2 = a.one_minus_beta2;
    p.csum = reinterpret_cast<float*>(a.ws + L.csum);
    const dim3 grid((unsigned)((a.D + kBlock - 1) / kBlock));
    ember_finalize_cols<<<grid, kBlock, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_apply(const StepArgs& a, hipStream_t s) {
    const WsLayout L = ws_layout(a.V, a.D);
    const ColPlan cp = col_plan(a.D, a.g_dtype);
    ApplyParams p;
    p.W = a.W;
    p.ldw = a.ldw;
    p.G = a.G;
    p.ldg = a.ldg;
    p.rows = a.rows;
    p.D = a.D;
    p.total_chunks = cp.total_chunks;
    p.slab_chunks = cp.slab_chunks;
    p.nb = row_blocks(a.rows);
    p.idx = a.idx;
    p.r = a.r;
    p.c = a.c;
    p.rsum = reinterpret_cast<const float*>(a.ws + L.rsum);
    p.nrsum = (int)((a.V + kVRowsPerBlock - 1) / kVRowsPerBlock);
    p.csum = reinterpret_cast<const float*>(a.ws + L.csum);
    p.ncsum = (int)((a.D + kBlock - 1) / kBlock);
    p.V = a.V;
    p.inv_bias = a.inv_bias;
    p.inv_alpha = a.inv_alpha;
    p.eps_over_alpha = a.eps_over_alpha;
    p.status = reinterpret_cast<const int*>(a.ws + L.status);
    p.flag = reinterpret_cast<int*>(a.ws + L.flag);
    const dim3 grid((unsigned)p.nb, (unsigned)cp.nslab);
    const bool sparse = a.sparse;
    if (a.g_dtype == 0)
        return sparse ? apply_dispatch_w<float, true>(p, a.w_dtype, cp.m, grid, s)
                      : apply_dispatch_w<float, false>(p, a.w_dtype, cp.m, grid, s);
    return sparse ? apply_dispatch_w<uint16_t, true>(p, a.w_dtype, cp.m, grid, s)
                  : apply_dispatch_w<uint16_t, false>(p, a.w_dtype, cp.m, grid, s);
}

} // namespace ember
