// HIP kernels of the Ember step for gfx950 (MI355X).
//
// One dense step (Token Geometry, Algorithm 1) is three launches on one
// stream (a sparse step whose rows fit on chip is one launch, ember_sparse_onchip,
// further down; larger sparse batches take the same three):
//   ember_stats          reads G once: per-row sums of g^2 and per-block
//                        column sums of g^2 (per-lane registers, then a
//                        fixed-order LDS combine of the block's 4 waves).  The
//                        sparse form also validates idx and marks touched rows.
//   ember_finalize       the column reduction of the block partials and the c
//                        update, and the r update over all V rows.
//   ember_apply          reads G and W, writes W: the update with the factored
//                        preconditioner applied as a row factor times a column
//                        factor (never stored).
// Every reduction runs in an order fixed by (V, D, n), with no floating-point
// atomics, so results are bitwise reproducible.
//
// Tiling of the two streaming kernels: a row is cut into column slabs of
// kSlabChunks 16-byte chunks (2 KiB); one block covers one slab of a range of
// rows, one wavefront streams one row's slab at a time (lane l owns chunks l
// and l + 64), and each wave keeps several rows in flight.  Blocks are
// numbered slab-fastest, so neighbouring blocks read neighbouring slabs of the
// same rows.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>

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

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <bool NT, typename V>
__device__ __forceinline__ V ld(const V* p) {
    if constexpr (NT) return __builtin_nontemporal_load(p);
    else return *p;
}
template <bool NT, typename V>
__device__ __forceinline__ void st(V* p, V v) {
    if constexpr (NT) __builtin_nontemporal_store(v, p);
    else *p = v;
}

// Words of a chunk of N elements of T (N * sizeof(T) is 8, 16 or 32 bytes).
template <typename T, int N> struct Raw { uint32_t u[N * sizeof(T) / 4]; };

// Makes the compiler treat the words as rewritten (no instruction is emitted),
// so values decoded from them before this point are not kept alive to be
// reused after it: a decode is two ALU operations, a register held per
// element across a reduction costs occupancy.
template <typename T, int N>
__device__ __forceinline__ void launder(Raw<T, N>& r) {
#pragma unroll
    for (int q = 0; q < N * (int)sizeof(T) / 4; ++q) asm volatile("" : "+v"(r.u[q]));
}

template <typename T>
__device__ __forceinline__ uint32_t elem_bits(const T* p) {
    if constexpr (sizeof(T) == 4) return __float_as_uint(*p);
    else return (uint32_t)*p;
}

// Raw words of the chunk `col .. col+N` of a row: one vector access when it
// lies inside [0, D), element access for the partial last chunk, zero words
// (zero values) when `valid` is false.  Decoding is left to the point of use so
// that bf16 data occupies half the registers while loads are in flight.
template <typename T, int N, bool NT>
__device__ __forceinline__ void load_raw(const T* row, int64_t col, bool valid, int64_t D, Raw<T, N>& r) {
    constexpr int kWords = N * (int)sizeof(T) / 4;
    if (valid && col + N <= D) {
        if constexpr (kWords == 2) {
            const u32x2 v = ld<NT>(reinterpret_cast<const u32x2*>(row + col));
            r.u[0] = v.x; r.u[1] = v.y;
        } else {
#pragma unroll
            for (int q = 0; q < kWords / 4; ++q) {
                const u32x4 v = ld<NT>(reinterpret_cast<const u32x4*>(row + col) + q);
                r.u[4 * q] = v.x; r.u[4 * q + 1] = v.y; r.u[4 * q + 2] = v.z; r.u[4 * q + 3] = v.w;
            }
        }
    } else {
#pragma unroll
        for (int q = 0; q < kWords; ++q) r.u[q] = 0u;
#pragma unroll
        for (int e = 0; e < N; ++e) {
            if (valid && col + e < D) {
                const uint32_t b = elem_bits(row + col + e);
                if constexpr (sizeof(T) == 4) r.u[e] = b;
                else r.u[e / 2] |= b << (16 * (e & 1));
            }
        }
    }
}

// Raw buffer access to one row (base and byte length in a buffer resource).
// The hardware checks every access against the length: loads past it return
// zero and stores past it are dropped, so the row tail and absent rows (length
// 0) need no branch.  Lengths here are multiples of 16 bytes, so a chunk is
// wholly inside or wholly outside.
constexpr int kBufferWord3 = 0x00020000;  // raw 32-bit data format, gfx9 family
constexpr int kCachePolicy = kRowOnlyNT ? 2 : 0;  // 2: non-temporal

__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_buffer(const void* row, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(row), 0, bytes, kBufferWord3);
}

template <typename T, int N>
__device__ __forceinline__ void buf_load(__amdgpu_buffer_rsrc_t rs, int byte_off, Raw<T, N>& r) {
    constexpr int kWords = N * (int)sizeof(T) / 4;
    if constexpr (kWords == 2) {
        const u32x2 v = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rs, byte_off, 0, kCachePolicy));
        r.u[0] = v.x; r.u[1] = v.y;
    } else {
#pragma unroll
        for (int q = 0; q < kWords / 4; ++q) {
            const u32x4 v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, byte_off + 16 * q, 0, kCachePolicy));
            r.u[4 * q] = v.x; r.u[4 * q + 1] = v.y; r.u[4 * q + 2] = v.z; r.u[4 * q + 3] = v.w;
        }
    }
}

template <typename T, int N>
__device__ __forceinline__ void buf_store(__amdgpu_buffer_rsrc_t rs, int byte_off, const float (&x)[N]) {
    constexpr int kWords = N * (int)sizeof(T) / 4;
    uint32_t u[kWords];
    encode<T, N>(x, u);
    if constexpr (kWords == 2) {
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b64(rs, 0, 0, 0)), u32x2{u[0], u[1]}),
                                              rs, byte_off, 0, kCachePolicy);
    } else {
#pragma unroll
        for (int q = 0; q < kWords / 4; ++q)
            __builtin_amdgcn_raw_buffer_store_b128(
                __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(rs, 0, 0, 0)),
                                   u32x4{u[4 * q], u[4 * q + 1], u[4 * q + 2], u[4 * q + 3]}),
                rs, byte_off + 16 * q, 0, kCachePolicy);
    }
}

template <typename T, int N>
__device__ __forceinline__ void decode(const Raw<T, N>& r, float (&x)[N]) { decode<T, N>(r.u, x); }

// N fp32 values from a buffer padded to a multiple of 8 floats; zeros past D.
template <int N>
__device__ __forceinline__ void load_chunk_f32(const float* p, int64_t col, bool valid, int64_t D, float (&x)[N]) {
#pragma unroll
    for (int e = 0; e < N; ++e) x[e] = 0.0f;
    if (!valid) return;
#pragma unroll
    for (int q = 0; q < N / 4; ++q) {
        const float4 v = reinterpret_cast<const float4*>(p + col)[q];
        x[4 * q] = v.x; x[4 * q + 1] = v.y; x[4 * q + 2] = v.z; x[4 * q + 3] = v.w;
    }
#pragma unroll
    for (int e = 0; e < N; ++e)
        if (col + e >= D) x[e] = 0.0f;
}

template <typename T, int N, bool NT>
__device__ __forceinline__ void vstore(T* p, const float (&x)[N]) {
    constexpr int kWords = N * (int)sizeof(T) / 4;
    uint32_t u[kWords];
    encode<T, N>(x, u);
    if constexpr (kWords == 2) {
        st<NT>(reinterpret_cast<u32x2*>(p), u32x2{u[0], u[1]});
    } else {
#pragma unroll
        for (int q = 0; q < kWords / 4; ++q)
            st<NT>(reinterpret_cast<u32x4*>(p) + q, u32x4{u[4 * q], u[4 * q + 1], u[4 * q + 2], u[4 * q + 3]});
    }
}

template <typename T, int N, bool NT>
__device__ __forceinline__ void store_chunk(T* row, int64_t col, int64_t D, const float (&x)[N]) {
    if (col + N <= D) {
        vstore<T, N, NT>(row + col, x);
    } else {
#pragma unroll
        for (int e = 0; e < N; ++e)
            if (col + e < D) Elem<T>::store(row + col + e, x[e]);
    }
}

// Stores and loads at agent scope: coherent across the XCDs' L2 caches without
// an L2 write-back, for the few values one block hands to another inside a
// launch.
__device__ __forceinline__ void st_agent(float* p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_agent(const float* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Completion ticket of a block: every wave waits until its own stores have
// completed, then one thread counts the block.  Returns true (in every thread)
// for the block that completes the count of `total`.  The ticket orders work;
// no value is accumulated through it.
__device__ __forceinline__ bool block_ticket(int* ticket, int total, int* lds_flag) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
        const int t = __hip_atomic_fetch_add(ticket, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *lds_flag = t == total - 1;
    }
    __syncthreads();
    return *lds_flag != 0;
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
    int nslab;
    int nb;
    int64_t cached_from; // gradient rows >= this one are loaded through the caches
    float* rowpart;      // [nslab][rows]
    float* P;            // [nb][D]
    const int64_t* idx;  // sparse only
    const int64_t* n_dev; // sparse only: device row count, or null
    int64_t V;
    int* slot;
    int* flag;
    const int* taken;     // set: the one-launch kernel may have taken this step (then return)
};

// Sums N values per lane over the 64 lanes, N rows at once (reduce-scatter
// butterfly): at distance X each lane keeps half of its rows and adds the
// partner's copy of them, until one row is left; plain butterfly steps then
// finish it.  On return lane l holds the total of row l >> (6 - log2 N).  Each
// partial sum is formed by one lane (or by two lanes as a + b and b + a, which
// are equal), so the order of every sum is fixed.
template <int N, int X>
__device__ __forceinline__ float rows_sum_step(const float (&v)[N], int lane) {
    if constexpr (N == 1) {
        float t = v[0];
#pragma unroll
        for (int off = X; off >= 1; off >>= 1) t += __shfl_xor(t, off, kWave);
        return t;
    } else {
        constexpr int H = N / 2;
        const bool hi = (lane & X) != 0;
        float nv[H];
#pragma unroll
        for (int j = 0; j < H; ++j) {
            const float keep = hi ? v[H + j] : v[j];
            const float send = hi ? v[j] : v[H + j];
            nv[j] = keep + __shfl_xor(send, X, kWave);
        }
        return rows_sum_step<H, X / 2>(nv, lane);
    }
}
template <int R>
__device__ __forceinline__ float rows_sum(const float (&v)[R], int lane) {
    static_assert(R == 1 || R == 2 || R == 4 || R == 8 || R == 16, "rows per batch");
    return rows_sum_step<R, kWave / 2>(v, lane);
}

// Row count of a sparse step: the host's, or the one in device memory (then
// a.rows is its maximum, which sizes the grids and the row-sum stride).  An
// out-of-range device count gives no rows and sets `bad`.
__device__ __forceinline__ int64_t active_rows(const int64_t* n_dev, int64_t rows_max, bool& bad) {
    bad = false;
    if (n_dev == nullptr) return rows_max;
    const int64_t n = *n_dev;
    bad = n < 0 || n > rows_max;
    return bad ? 0 : n;
}

// Rows of row block b: a contiguous range, fixed by (rows, nb).
struct RowSet {
    int64_t first, stride, count;
};
__device__ __forceinline__ RowSet stats_rows(int64_t rows, int nb, int b) {
    RowSet rs;
    int64_t r0, r1;
    row_range(rows, nb, b, r0, r1);
    rs.first = r0;
    rs.stride = 1;
    rs.count = r1 - r0;
    return rs;
}

// The apply pass walks rows from high to low, so the rows this pass reads
// last are the first it reads again: rows >= cached_from are loaded through
// the caches (and can be served from the last-level cache later), the others
// with non-temporal loads.
// kWide (more than kWideRowsPerWave rows per wavefront, i.e. very tall
// tables): the per-lane column sums are kept in fp32 over kWideRowsPerWave
// rows at a time and gathered in float64, so their error does not grow with
// the row count.
constexpr int64_t kWideRowsPerWave = 1024;

// More than kWideRowsPerWave rows per wavefront: the kWide instance.
static bool stats_wide(const StatsParams& p) {
    return (p.rows + (int64_t)p.nb * kWaves - 1) / ((int64_t)p.nb * kWaves) > kWideRowsPerWave;
}

// Block `blk` of the statistics pass of one table; `lds` is the block's
// [kWaves][kWave * EPC] staging area for the column-sum combine.
template <typename GT, int M, int R, bool kSparseArg, bool kWide, bool kRuntime = false>
__device__ __forceinline__ void stats_block(const StatsParams& a, unsigned blk, float (*lds)[kWave * 16 / sizeof(GT)],
                                           bool sparse_rt = false) {
    const bool kSparse = kRuntime ? sparse_rt : kSparseArg;
    constexpr int EPC = 16 / (int)sizeof(GT);
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int slab = (int)(blk % (unsigned)a.nslab);
    const int b = (int)(blk / (unsigned)a.nslab);
    bool bad_count = false;
    const int64_t nrows = kSparse ? active_rows(a.n_dev, a.rows, bad_count) : a.rows;
    if (kSparse && bad_count && blk == 0 && threadIdx.x == 0) atomicOr(a.flag, kFlagCount);
    const RowSet rset = stats_rows(nrows, a.nb, b);
    const int cbeg = slab * a.slab_chunks;
    const int cend = min(cbeg + a.slab_chunks, a.total_chunks);
    const GT* G = static_cast<const GT*>(a.G);

    float acc[M][EPC];
    double wide[kWide ? M : 1][kWide ? EPC : 1];
#pragma unroll
    for (int m = 0; m < M; ++m)
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[m][e] = 0.0f;
    if constexpr (kWide) {
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
            for (int e = 0; e < EPC; ++e) wide[m][e] = 0.0;
    }
    auto gather = [&]() {
        if constexpr (kWide) {
#pragma unroll
            for (int m = 0; m < M; ++m)
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    wide[m][e] += (double)acc[m][e];
                    acc[m][e] = 0.0f;
                }
        }
    };

    // this wave's rows: the block's rows wave, wave + 4, wave + 8, ...
    const int64_t span = rset.count - wave;
    const int64_t nk = span > 0 ? (span + kWaves - 1) / kWaves : 0;
    auto row_of = [&](int64_t k) { return rset.first + rset.stride * (wave + kWaves * k); };
    Raw<GT, EPC> raw[R][M];
    auto load_batch = [&](int64_t k0) {
        // one load policy per batch (uniform across the wave)
        const bool cached = row_of(k0) >= a.cached_from;
#pragma unroll
        for (int j = 0; j < R; ++j) {
            const bool rv = k0 + j < nk;
            const GT* grow = G + row_of(k0 + j) * a.ldg;
#pragma unroll
            for (int m = 0; m < M; ++m) {
                const int ch = cbeg + lane + kWave * m;
                if (cached)
                    load_raw<GT, EPC, false>(grow, (int64_t)ch * EPC, rv && ch < cend, a.D, raw[j][m]);
                else
                    load_raw<GT, EPC, true>(grow, (int64_t)ch * EPC, rv && ch < cend, a.D, raw[j][m]);
            }
        }
    };
    if (nk > 0) load_batch(0);
    for (int64_t k0 = 0; k0 < nk; k0 += R) {
        float rs[R];
#pragma unroll
        for (int j = 0; j < R; ++j) {
            float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
            for (int m = 0; m < M; ++m) {
                float x[EPC];
                decode(raw[j][m], x);
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    acc[m][e] = fmaf(x[e], x[e], acc[m][e]);
                    if (e & 1) s1 = fmaf(x[e], x[e], s1);
                    else s0 = fmaf(x[e], x[e], s0);
                }
            }
            rs[j] = s0 + s1;
        }
        // the registers of this batch are free: start the next batch's loads
        // before the cross-lane reduction
        if (k0 + R < nk) load_batch(k0 + R);
        const float tot = rows_sum<R>(rs, lane);
        constexpr int kLanesPerRow = kWave / R;
        const int j = lane / kLanesPerRow;
        if ((lane & (kLanesPerRow - 1)) == 0 && k0 + j < nk) {
            const int64_t row = row_of(k0 + j);
            a.rowpart[(int64_t)slab * a.rows + row] = tot;
            if (kSparse && slab == 0) {
                const int64_t i = a.idx[row];
                if (i < 0 || i >= a.V) {
                    atomicOr(a.flag, kFlagRange);
                } else if (atomicCAS(&a.slot[i], 0, (int)(row + 1)) != 0) {
                    atomicOr(a.flag, kFlagDuplicate);
                }
            }
        }
        if (kWide && (k0 / R + 1) % (kWideRowsPerWave / R) == 0) gather();
    }
    if constexpr (kWide) {
        gather();
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
            for (int e = 0; e < EPC; ++e) acc[m][e] = (float)wide[m][e];
    }

    // Combine the 4 waves' column sums in a fixed order, one chunk column at a time.
    float* P = a.P + (int64_t)b * a.D;
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

template <typename GT, int M, int R, bool kSparse, bool kWide>
__global__ __launch_bounds__(kBlock) void ember_stats(StatsParams a) {
    __shared__ float lds[kWaves][kWave * 16 / sizeof(GT)];
    if (a.taken != nullptr && *a.taken != 0) return;
    stats_block<GT, M, R, kSparse, kWide>(a, blockIdx.x, lds);
}

// Several tables in one launch: table k owns blocks [first[k], first[k+1]).
// Each table's blocks do exactly what its own launch would, so the results
// are the same bits; one launch lets the tables share the chip instead of
// each paying its own ramp and tail.
template <typename P>
struct MultiParams {
    int ntab;
    unsigned first[kMaxTables + 1];
    int sparse[kMaxTables];
    P p[kMaxTables];
};

__device__ __forceinline__ int multi_table(const unsigned* first, int ntab) {
    int k = 0;
#pragma unroll
    for (int j = 1; j < kMaxTables; ++j) k += (j < ntab && blockIdx.x >= first[j]) ? 1 : 0;
    return k;
}

// At least the occupancy of the single-table kernel (three waves per SIMD for
// two chunks per lane).  The table's parameters are copied out of the
// argument array first (uniform values, loaded once).
template <typename GT, int M, int R, bool kWide>
__global__ __launch_bounds__(kBlock, (M == 2 && !kWide) ? 3 : 1) void ember_stats_multi(MultiParams<StatsParams> g) {
    __shared__ float lds[kWaves][kWave * 16 / sizeof(GT)];
    const int k = multi_table(g.first, g.ntab);
    const unsigned blk = blockIdx.x - g.first[k];
    const StatsParams p = g.p[k];
    stats_block<GT, M, R, false, kWide, true>(p, blk, lds, g.sparse[k] != 0);
}

// ---------------------------------------------------------------------------
// finalize: column sums -> c, row sums -> r (one launch, fixed orders)
// ---------------------------------------------------------------------------

constexpr int kFinThreads = 1024;                  // 16 waves
constexpr int kFinWaves = kFinThreads / kWave;
constexpr int kFinRowsPerBlock = kFinThreads * kVRowsPerThread;
constexpr int kFinGroups = kFinThreads / kFinCols;  // row groups of a column block
static_assert(kFinCols == 16 || kFinCols == 32 || kFinCols == 64, "a column block's columns lie in one wave");

struct FinParams {
    const float* P;        // [nb][D] per-block column sums of g^2
    int nb;
    int64_t D;
    int ncolblocks;        // ceil(D / kFinCols)
    const float* rowpart;  // [nslab][rows]
    int nslab;
    int64_t rows;
    int64_t V;
    float* r;
    float* c;
    int* slot;             // sparse only
    const int* flag;       // sparse only
    int* status;
    float beta2;
    float one_minus_beta2;
    float* rsum;           // [ceil(V / kFinRowsPerBlock)]
    float* csum;           // [ncolblocks]
    int* ticket;           // finished blocks; the last one derives the step scale
    float* qa;             // [D rounded up to 8] column factors sqrt(c_j)
    float* scale;          // sqrt(1 / (bias s)) / alpha_s
    double inv_bias;
    double inv_alpha;
    const int* taken;      // set: the one-launch kernel may have taken this step (then return)
};

// Run by the last block of the finalize pass, once every r, c and partial sum
// of this step is stored: s = sqrt(mean(rhat) mean(chat)) from the per-block
// sums in a fixed order, and the step scale sqrt(1 / (bias s)) / alpha_s.  The
// preconditioner's root sqrt(rhat_i chat_j / s) / alpha_s is applied as
// [sqrt(r_i / bias) * scale] * sqrt(c_j): a row factor times the column factor
// the column blocks stored, which needs no pass over the columns here.  Every
// thread of the block takes part: thread t adds entries t, t + 1024, ... in
// float64, then the waves' sums are added in wave order.
__device__ void step_scale(const FinParams& a, int nrsum, double (*lds2)[kFinWaves]) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    double sr = 0.0, sc = 0.0;
    for (int k = threadIdx.x; k < nrsum; k += kFinThreads) sr += (double)ld_agent(a.rsum + k);
    for (int k = threadIdx.x; k < a.ncolblocks; k += kFinThreads) sc += (double)ld_agent(a.csum + k);
    sr = wave_sum(sr);
    sc = wave_sum(sc);
    if (lane == 0) {
        lds2[0][wave] = sr;
        lds2[1][wave] = sc;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        sr = 0.0;
        sc = 0.0;
        for (int w = 0; w < kFinWaves; ++w) {
            sr += lds2[0][w];
            sc += lds2[1][w];
        }
        const double mean_rhat = sr / (double)a.V * a.inv_bias;
        const double mean_chat = sc / (double)a.D * a.inv_bias;
        const double s = sqrt(mean_rhat * mean_chat);
        *a.scale = s > 0.0 ? (float)(sqrt(a.inv_bias / s) * a.inv_alpha) : 0.0f;
    }
}

// Sum of one float per thread of a 1024-thread block: waves, then waves 0..15 in order.
__device__ __forceinline__ float block_sum_1024(float v, float* lds16) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    v = wave_sum(v);
    if (lane == 0) lds16[wave] = v;
    __syncthreads();
    float t = 0.0f;
#pragma unroll
    for (int w = 0; w < kFinWaves; ++w) t += lds16[w];
    return t;
}

template <bool kSparse>
__device__ __forceinline__ void finalize_body(const FinParams& a, int blk, int err, float (*part)[kFinCols],
                                              float* lds16);

// Shared memory of a finalize block.
struct FinLds {
    float part[kFinGroups][kFinCols];
    float lds16[kFinWaves];
    double lds2[2][kFinWaves];
    int last;
};

// Block `blk` of the `nblocks` finalize blocks of one table.
template <bool kSparse>
__device__ __forceinline__ void finalize_block(const FinParams& a, int blk, int nblocks, FinLds& sh) {
    const int err = kSparse ? *a.flag : 0;
    if (blk == 0 && threadIdx.x == 0) *a.status = err | (*a.status & kFlagTimeout);
    finalize_body<kSparse>(a, blk, err, sh.part, sh.lds16);

    // The block that finishes last derives the step scale from the per-block
    // sums (written with agent-scope stores).
    if (!block_ticket(a.ticket, nblocks, &sh.last)) return;
    const int nrsum = (int)((a.V + kFinRowsPerBlock - 1) / kFinRowsPerBlock);
    if (!err) step_scale(a, nrsum, sh.lds2);
    if (threadIdx.x == 0) *a.ticket = 0;
}

template <bool kSparse>
__global__ __launch_bounds__(kFinThreads) void ember_finalize(FinParams a) {
    __shared__ FinLds sh;
    if (a.taken != nullptr && *a.taken != 0) return;
    finalize_block<kSparse>(a, (int)blockIdx.x, (int)gridDim.x, sh);
}

__global__ __launch_bounds__(kFinThreads) void ember_finalize_multi(MultiParams<FinParams> g) {
    __shared__ FinLds sh;
    const int k = multi_table(g.first, g.ntab);
    const int blk = (int)(blockIdx.x - g.first[k]);
    const int nblocks = (int)(g.first[k + 1] - g.first[k]);
    if (g.sparse[k]) finalize_block<true>(g.p[k], blk, nblocks, sh);
    else finalize_block<false>(g.p[k], blk, nblocks, sh);
}

template <bool kSparse>
__device__ __forceinline__ void finalize_body(const FinParams& a, int blk, int err, float (*part)[kFinCols],
                                              float* lds16) {
    const int lane = threadIdx.x & (kWave - 1);
    if (blk < a.ncolblocks) {
        // kFinCols columns: thread (g, x) sums partial rows g, g + kFinGroups, ...
        // of column x in ascending order, then the first kFinCols threads add
        // the kFinGroups group sums in group order.
        const int x = threadIdx.x % kFinCols;
        const int g = threadIdx.x / kFinCols;
        const int64_t j = (int64_t)blk * kFinCols + x;
        const bool jv = j < a.D;
        float s = 0.0f;
        if (jv) {
#pragma unroll 8
            for (int b = g; b < a.nb; b += kFinGroups) s += a.P[(int64_t)b * a.D + j];
        }
        part[g][x] = s;
        __syncthreads();
        if (threadIdx.x < kWave) {
            float cn = 0.0f;
            if (lane < kFinCols) {
                float colsum = 0.0f;
                for (int w = 0; w < kFinGroups; ++w) colsum += part[w][lane];
                if (jv && !err) {
                    const float mean = (float)((double)colsum / (double)a.V);
                    cn = fmaf(a.beta2, a.c[j], a.one_minus_beta2 * mean);
                    st_agent(a.c + j, cn);
                    a.qa[j] = sqrtf(cn);
                }
            }
            cn = wave_sum(cn);
            if (lane == 0) st_agent(a.csum + blk, cn);
        }
        return;
    }

    const int vb = blk - a.ncolblocks;
    const double invD = 1.0 / (double)a.D;
    float psum = 0.0f;
#pragma unroll
    for (int q = 0; q < kVRowsPerThread; ++q) {
        const int64_t i = (int64_t)vb * kFinRowsPerBlock + q * kFinThreads + threadIdx.x;
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
            double sum = 0.0;
            for (int sb = 0; sb < a.nslab; ++sb) sum += (double)a.rowpart[(int64_t)sb * a.rows + k];
            const float mean = (float)(sum * invD);
            rn = fmaf(a.beta2, a.r[i], a.one_minus_beta2 * mean);
        } else {
            rn = a.beta2 * a.r[i];
        }
        a.r[i] = rn;
        psum += rn;
    }
    const float tot = block_sum_1024(psum, lds16);
    if (threadIdx.x == 0) st_agent(a.rsum + vb, tot);
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
    int nslab;
    int nb;
    const int64_t* idx;   // sparse only
    const int64_t* n_dev; // sparse only: device row count, or null
    const float* r;
    const float* qa;      // [D rounded up to 8] column factors sqrt(c_j)
    const float* scale;   // sqrt(1 / (bias s)) / alpha_s
    double inv_bias;
    double inv_alpha;     // 1 / alpha_s, alpha_s = -lr (descent) or +lr (ascent)
    float eps_over_alpha; // eps / alpha_s
    const int* status;    // sparse only: skip when the statistics pass flagged idx
    int* flag;            // sparse only: cleared for the next step
    const int* taken;     // set: the one-launch kernel may have taken this step (then return)
};

// Block `blk` of the `nblk` apply blocks of one table.
template <typename GT, typename WT, int M, int R, bool kSparseArg, bool kRuntime = false>
__device__ __forceinline__ void apply_block(const ApplyParams& a, unsigned blk, unsigned nblk, bool sparse_rt = false) {
    const bool kSparse = kRuntime ? sparse_rt : kSparseArg;
    constexpr int EPC = 16 / (int)sizeof(GT);
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    if (kSparse) {
        if (blk == 0 && threadIdx.x == 0) *a.flag = 0;
        if ((*a.status & ~kFlagTimeout) != 0) return;
    }
    if (a.inv_alpha == 0.0) return;   // lr == 0: every weight keeps its bits
    bool bad_count = false;
    const int64_t nrows = kSparse ? active_rows(a.n_dev, a.rows, bad_count) : a.rows;

    // (row block, slab) pairs, slab-fastest; the grid is capped, so a block may
    // take several pairs
    const int64_t nvb = (int64_t)a.nb * a.nslab;
    for (int64_t vb = blk; vb < nvb; vb += nblk) {
        const int slab = (int)(vb % a.nslab);
        // Row blocks in reverse order: the rows the statistics pass read last are
        // the likeliest still to sit in the last-level cache.
        const int b = a.nb - 1 - (int)(vb / a.nslab);
        const int cbeg = slab * a.slab_chunks;
        const int cend = min(cbeg + a.slab_chunks, a.total_chunks);

        // Column factors sqrt(c_j) of this lane's columns, stored by the finalize
        // pass; the row factor carries sqrt(1 / bias) and the step scale.
        float qa[M][EPC];
#pragma unroll
        for (int m = 0; m < M; ++m) {
            const int ch = cbeg + lane + kWave * m;
            load_chunk_f32<EPC>(a.qa, (int64_t)ch * EPC, ch < cend, a.D, qa[m]);
        }
        const float epsa = a.eps_over_alpha;
        const float ibias = (float)a.inv_bias;
        const float scale = *a.scale;

        int64_t r0, r1;
        row_range(nrows, a.nb, b, r0, r1);
        const GT* G = static_cast<const GT*>(a.G);
        WT* W = static_cast<WT*>(a.W);

        const int64_t span = r1 - r0 - wave;
        const int64_t nk = span > 0 ? (span + kWaves - 1) / kWaves : 0;
        for (int64_t k0 = 0; k0 < nk; k0 += R) {
            Raw<GT, EPC> graw[R][M];
            Raw<WT, EPC> wraw[R][M];
            float ai[R];
            WT* wr[R];
#pragma unroll
            for (int j = 0; j < R; ++j) {
                const bool rv = k0 + j < nk;
                const int64_t row = rv ? r0 + wave + kWaves * (k0 + j) : r0;
                const int64_t wrow = kSparse ? a.idx[row] : row;
                ai[j] = sqrtf(a.r[wrow] * ibias) * scale;
                const GT* grow = G + row * a.ldg;
                wr[j] = W + wrow * a.ldw;
#pragma unroll
                for (int m = 0; m < M; ++m) {
                    const int ch = cbeg + lane + kWave * m;
                    load_raw<GT, EPC, kApplyNT>(grow, (int64_t)ch * EPC, rv && ch < cend, a.D, graw[j][m]);
                    load_raw<WT, EPC, kApplyWNT>(wr[j], (int64_t)ch * EPC, rv && ch < cend, a.D, wraw[j][m]);
                }
            }
#pragma unroll
            for (int j = 0; j < R; ++j) {
                if (k0 + j >= nk) break;
#pragma unroll
                for (int m = 0; m < M; ++m) {
                    const int ch = cbeg + lane + kWave * m;
                    float g[EPC], w[EPC], o[EPC];
                    decode(graw[j][m], g);
                    decode(wraw[j][m], w);
#pragma unroll
                    for (int e = 0; e < EPC; ++e) {
                        const float d = fmaf(ai[j], qa[m][e], epsa);
                        const float upd = fmaf(g[e], __builtin_amdgcn_rcpf(d), w[e]);
                        o[e] = (g[e] == 0.0f) ? w[e] : upd;
                    }
                    if (ch < cend) store_chunk<WT, EPC, kApplyNT>(wr[j], (int64_t)ch * EPC, a.D, o);
                }
            }
        }
    }
}

template <typename GT, typename WT, int M, int R, bool kSparse>
__global__ __launch_bounds__(kBlock) void ember_apply(ApplyParams a) {
    if (a.taken != nullptr && *a.taken != 0) return;
    apply_block<GT, WT, M, R, kSparse>(a, blockIdx.x, gridDim.x);
}

template <typename GT, typename WT, int M, int R>
__global__ __launch_bounds__(kBlock) void ember_apply_multi(MultiParams<ApplyParams> g) {
    const int k = multi_table(g.first, g.ntab);
    const unsigned blk = blockIdx.x - g.first[k];
    const unsigned nblk = g.first[k + 1] - g.first[k];
    const ApplyParams p = g.p[k];
    apply_block<GT, WT, M, R, false, true>(p, blk, nblk, g.sparse[k] != 0);
}

// ---------------------------------------------------------------------------
// row-only Ember (Section 2.1): vtil_ij = rhat_i, so the whole step is one pass
// over the rows, W += g / (sqrt(rhat_i) / alpha_s + eps / alpha_s)
// ---------------------------------------------------------------------------

constexpr int kRowOnlyRows = 2;                          // rows in flight per block
constexpr int kRowOnlyMaxWaves = 8;                      // waves per block
constexpr int kRowOnlyRowsPerBlock = 16;                 // rows per block
constexpr int kRowOnlyWaveRows = 2;                      // rows in flight per wave (one-wave rows)
// The single-table sparse step of the one-wave kernel: one row per wave and
// one row per wave of a block, so the few thousand rows of a batch are all in
// flight at once (about half the registers, more waves per SIMD) instead of
// taking two rounds of two rows per wave.
constexpr int kRowOnlySparseRowsPerBlock = 4;
constexpr int kRowOnlySparseWaveRows = 1;
constexpr int kRowOnlyWaveChunks = 16 * kWave;           // longest row held by one wave, in chunks

struct RowOnlyParams {
    void* W;
    int64_t ldw;
    const void* G;
    int64_t ldg;
    int64_t rows;          // V (dense) or n (sparse)
    int64_t D;
    int total_chunks;
    int slab_chunks;
    int nslab;
    int64_t nb;            // row blocks
    int64_t nvb;           // row blocks + decay blocks (sparse)
    int rows_per_block;    // gradient rows per row block
    int* tgroups;          // sparse only: first-level completion counters
    const int64_t* idx;    // sparse only
    const int64_t* n_dev;  // sparse only: device row count, or null
    float* r;
    int64_t V;
    float beta2;
    float one_minus_beta2;
    float inv_bias;
    float inv_alpha;       // 1 / alpha_s; 0 when lr == 0 (no weight is written)
    float eps_over_alpha;
    int* slot;             // sparse only
    int* flag;             // sparse only: index-error bits, cleared by the last block
    int* ticket;           // sparse only
    int* status;
};

// The rows of one block, kRowOnlyRows at a time.  Resident: the block has
// ceil(nslab / S) waves and wave w holds slabs w*S .. w*S+S-1 of the rows in
// registers from the row sum to the update, so G is read once.  Otherwise
// (rows too long to hold) wave w takes slabs w, w + nw, ... and reads them
// once for the row sum and again, with W, for the update.
template <typename GT, typename WT, int M, int S, bool kSparse, bool kResident>
__device__ __forceinline__ void rowonly_rows(const RowOnlyParams& a, int64_t nrows, int64_t vb,
                                             float (*part)[kRowOnlyRows], float* rn_lds) {
    constexpr int EPC = 16 / (int)sizeof(GT);
    constexpr int R = kRowOnlyRows;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int nw = blockDim.x / kWave;
    const bool update = a.inv_alpha != 0.0f;

    const int64_t r0 = vb * a.rows_per_block;
    const int64_t r1 = min(r0 + a.rows_per_block, nrows);
    const GT* G = static_cast<const GT*>(a.G);
    WT* W = static_cast<WT*>(a.W);
    const double invD = 1.0 / (double)a.D;

    for (int64_t k0 = r0; k0 < r1; k0 += R) {
        const GT* gr[R];
        WT* wr[R];
        int64_t wrow[R];
        bool rv[R];
#pragma unroll
        for (int j = 0; j < R; ++j) {
            rv[j] = k0 + j < r1;
            const int64_t row = rv[j] ? k0 + j : r0;
            wrow[j] = kSparse ? a.idx[row] : row;
            gr[j] = G + row * a.ldg;
            wr[j] = W + wrow[j] * a.ldw;
        }
        float s0[R], s1[R];
#pragma unroll
        for (int j = 0; j < R; ++j) s0[j] = s1[j] = 0.0f;
        auto accumulate = [&](const Raw<GT, EPC>& raw, int j) {
            float x[EPC];
            decode(raw, x);
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                if (e & 1) s1[j] = fmaf(x[e], x[e], s1[j]);
                else s0[j] = fmaf(x[e], x[e], s0[j]);
            }
        };
        auto apply = [&](const Raw<GT, EPC>& graw, const Raw<WT, EPC>& wraw, float rc, WT* wrow_ptr, int ch) {
            float g[EPC], w[EPC], o[EPC];
            decode(graw, g);
            decode(wraw, w);
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                const float upd = fmaf(g[e], rc, w[e]);
                o[e] = (g[e] == 0.0f) ? w[e] : upd;
            }
            store_chunk<WT, EPC, kRowOnlyNT>(wrow_ptr, (int64_t)ch * EPC, a.D, o);
        };

        Raw<GT, EPC> graw[R][S][M];
        Raw<WT, EPC> wraw[R][S][M];
        if constexpr (kResident) {
#pragma unroll
            for (int j = 0; j < R; ++j)
#pragma unroll
                for (int q = 0; q < S; ++q) {
                    const int slab = wave * S + q;
                    const int cbeg = slab * a.slab_chunks;
                    const int cend = min(cbeg + a.slab_chunks, a.total_chunks);
#pragma unroll
                    for (int m = 0; m < M; ++m) {
                        const int ch = cbeg + lane + kWave * m;
                        const bool v = rv[j] && slab < a.nslab && ch < cend;
                        load_raw<GT, EPC, kRowOnlyNT>(gr[j], (int64_t)ch * EPC, v, a.D, graw[j][q][m]);
                        load_raw<WT, EPC, kRowOnlyNT>(wr[j], (int64_t)ch * EPC, v && update, a.D,
                                                            wraw[j][q][m]);
                    }
                }
#pragma unroll
            for (int j = 0; j < R; ++j)
#pragma unroll
                for (int q = 0; q < S; ++q)
#pragma unroll
                    for (int m = 0; m < M; ++m) accumulate(graw[j][q][m], j);
        } else {
            // long rows: each slab's fp32 sum is gathered in float64
            double wsum[R];
#pragma unroll
            for (int j = 0; j < R; ++j) wsum[j] = 0.0;
            for (int slab = wave; slab < a.nslab; slab += nw) {
                const int cbeg = slab * a.slab_chunks;
                const int cend = min(cbeg + a.slab_chunks, a.total_chunks);
#pragma unroll
                for (int j = 0; j < R; ++j)
#pragma unroll
                    for (int m = 0; m < M; ++m) {
                        const int ch = cbeg + lane + kWave * m;
                        load_raw<GT, EPC, false>(gr[j], (int64_t)ch * EPC, rv[j] && ch < cend, a.D, graw[j][0][m]);
                    }
#pragma unroll
                for (int j = 0; j < R; ++j) {
#pragma unroll
                    for (int m = 0; m < M; ++m) accumulate(graw[j][0][m], j);
                    wsum[j] += (double)s0[j] + (double)s1[j];
                    s0[j] = s1[j] = 0.0f;
                }
            }
#pragma unroll
            for (int j = 0; j < R; ++j) s0[j] = (float)wsum[j];
        }

        // Row sums of g^2: this wave's part, then the waves in order.
        float rs[R];
#pragma unroll
        for (int j = 0; j < R; ++j) rs[j] = s0[j] + s1[j];
        const float tot = rows_sum<R>(rs, lane);
        if ((lane & (kWave / R - 1)) == 0) part[wave][lane / (kWave / R)] = tot;
        __syncthreads();
        if (threadIdx.x < R && rv[threadIdx.x]) {
            const int j = threadIdx.x;
            float sum = 0.0f;
            for (int w = 0; w < nw; ++w) sum += part[w][j];
            const float mean = (float)((double)sum * invD);
            const float rnew = fmaf(a.beta2, a.r[wrow[j]], a.one_minus_beta2 * mean);
            a.r[wrow[j]] = rnew;
            rn_lds[j] = rnew;
        }
        __syncthreads();
        if (update) {
            float rc[R];
#pragma unroll
            for (int j = 0; j < R; ++j)
                rc[j] = __builtin_amdgcn_rcpf(fmaf(sqrtf(rn_lds[j] * a.inv_bias), a.inv_alpha, a.eps_over_alpha));
            if constexpr (kResident) {
#pragma unroll
                for (int j = 0; j < R; ++j) {
                    if (!rv[j]) break;
#pragma unroll
                    for (int q = 0; q < S; ++q) {
                        const int slab = wave * S + q;
                        const int cbeg = slab * a.slab_chunks;
                        const int cend = min(cbeg + a.slab_chunks, a.total_chunks);
#pragma unroll
                        for (int m = 0; m < M; ++m) {
                            const int ch = cbeg + lane + kWave * m;
                            if (slab < a.nslab && ch < cend) apply(graw[j][q][m], wraw[j][q][m], rc[j], wr[j], ch);
                        }
                    }
                }
            } else {
                for (int slab = wave; slab < a.nslab; slab += nw) {
                    const int cbeg = slab * a.slab_chunks;
                    const int cend = min(cbeg + a.slab_chunks, a.total_chunks);
#pragma unroll
                    for (int j = 0; j < R; ++j)
#pragma unroll
                        for (int m = 0; m < M; ++m) {
                            const int ch = cbeg + lane + kWave * m;
                            const bool v = rv[j] && ch < cend;
                            load_raw<GT, EPC, true>(gr[j], (int64_t)ch * EPC, v, a.D, graw[j][0][m]);
                            load_raw<WT, EPC, true>(wr[j], (int64_t)ch * EPC, v, a.D, wraw[j][0][m]);
                        }
#pragma unroll
                    for (int j = 0; j < R; ++j) {
                        if (!rv[j]) break;
#pragma unroll
                        for (int m = 0; m < M; ++m) {
                            const int ch = cbeg + lane + kWave * m;
                            if (ch < cend) apply(graw[j][0][m], wraw[j][0][m], rc[j], wr[j], ch);
                        }
                    }
                }
            }
        }
        __syncthreads();  // part and rn_lds are reused by the next rows
    }
}

// Rows up to 1024 chunks (bf16 D <= 8192, fp32 D <= 4096): one wave per row.
// Lane l holds chunks l, l + 64, ..., l + 64 (C - 1) of G and W in registers,
// the row sum is a butterfly over the wave, and no barrier is needed.  Each
// wave takes kRowOnlyWaveRows adjacent rows at a time; the waves of a block
// interleave over the block's rows.
template <typename GT, typename WT, int C, bool kSparse, bool kExact, bool kRuntime = false>
__device__ __forceinline__ void rowonly_wave_rows(const RowOnlyParams& a, int64_t nrows, int64_t vb,
                                                  bool sparse_rt = false) {
    constexpr int EPC = 16 / (int)sizeof(GT);
    constexpr int R = (kSparse && !kRuntime) ? kRowOnlySparseWaveRows : kRowOnlyWaveRows;
    constexpr int kWBytes = EPC * (int)sizeof(WT);   // bytes of W per chunk
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const bool update = a.inv_alpha != 0.0f;
    const int64_t r0 = vb * a.rows_per_block;
    const int64_t r1 = min(r0 + a.rows_per_block, nrows);
    const GT* G = static_cast<const GT*>(a.G);
    WT* W = static_cast<WT*>(a.W);
    const double invD = 1.0 / (double)a.D;
    const int gbytes = (int)a.D * (int)sizeof(GT);
    const int wbytes = (int)a.D * (int)sizeof(WT);

    for (int64_t k0 = r0 + (int64_t)wave * R; k0 < r1; k0 += (int64_t)kWaves * R) {
        const GT* gr[R];
        WT* wr[R];
        int64_t wrow[R];
        bool rv[R];
        float rold[R];
        Raw<GT, EPC> graw[R][C];
        Raw<WT, EPC> wraw[R][C];
        __amdgpu_buffer_rsrc_t gb[R], wb[R];
#pragma unroll
        for (int j = 0; j < R; ++j) {
            rv[j] = k0 + j < r1;
            const int64_t row = rv[j] ? k0 + j : r0;
            wrow[j] = (kRuntime ? sparse_rt : kSparse) ? a.idx[row] : row;
            gr[j] = G + row * a.ldg;
            wr[j] = W + wrow[j] * a.ldw;
            rold[j] = a.r[wrow[j]];
            gb[j] = row_buffer(gr[j], rv[j] ? gbytes : 0);
            wb[j] = row_buffer(wr[j], rv[j] && update ? wbytes : 0);
        }
        // G first: the row sums wait only for these loads, W arrives meanwhile.
#pragma unroll
        for (int j = 0; j < R; ++j)
#pragma unroll
            for (int c = 0; c < C; ++c) {
                const int ch = lane + kWave * c;
                if constexpr (kExact) buf_load<GT, EPC>(gb[j], ch * 16, graw[j][c]);
                else load_raw<GT, EPC, kRowOnlyNT>(gr[j], (int64_t)ch * EPC, rv[j] && ch < a.total_chunks,
                                                         a.D, graw[j][c]);
            }
#pragma unroll
        for (int j = 0; j < R; ++j)
#pragma unroll
            for (int c = 0; c < C; ++c) {
                const int ch = lane + kWave * c;
                if constexpr (kExact) buf_load<WT, EPC>(wb[j], ch * kWBytes, wraw[j][c]);
                else load_raw<WT, EPC, kRowOnlyNT>(wr[j], (int64_t)ch * EPC,
                                                         rv[j] && ch < a.total_chunks && update, a.D, wraw[j][c]);
            }
        // Keep every load of the rows issued before the first wait.
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < R; ++j) {
            float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
            for (int c = 0; c < C; ++c) {
                float x[EPC];
                decode(graw[j][c], x);
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    if (e & 1) s1 = fmaf(x[e], x[e], s1);
                    else s0 = fmaf(x[e], x[e], s0);
                }
            }
            const float sum = wave_sum(s0 + s1);
            const float mean = (float)((double)sum * invD);
            const float rnew = fmaf(a.beta2, rold[j], a.one_minus_beta2 * mean);
#pragma unroll
            for (int c = 0; c < C; ++c) launder(graw[j][c]);
            if (!rv[j]) continue;
            if (lane == 0) a.r[wrow[j]] = rnew;
            if (!update) continue;
            const float rc = __builtin_amdgcn_rcpf(fmaf(sqrtf(rnew * a.inv_bias), a.inv_alpha, a.eps_over_alpha));
#pragma unroll
            for (int c = 0; c < C; ++c) {
                const int ch = lane + kWave * c;
                if (!kExact && ch >= a.total_chunks) continue;
                float g[EPC], w[EPC], o[EPC];
                decode(graw[j][c], g);
                decode(wraw[j][c], w);
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    const float upd = fmaf(g[e], rc, w[e]);
                    o[e] = (g[e] == 0.0f) ? w[e] : upd;
                }
                if constexpr (kExact) buf_store<WT, EPC>(wb[j], ch * kWBytes, o);
                else store_chunk<WT, EPC, kRowOnlyNT>(wr[j], (int64_t)ch * EPC, a.D, o);
            }
        }
    }
}

// Blocks nb.. of the sparse row-only step: beta2 r on every row outside idx,
// and the row marks cleared (r is left alone when idx was rejected).
__device__ __forceinline__ void rowonly_decay(const RowOnlyParams& a, int err, int64_t db) {
    const int64_t i0 = db * kDecayRows;
    for (int64_t i = i0 + threadIdx.x; i < i0 + kDecayRows && i < a.V; i += blockDim.x) {
        const int sl = a.slot[i];
        if (sl != 0) a.slot[i] = 0;
        else if (!err) a.r[i] = a.beta2 * a.r[i];
    }
}

// Every block of the sparse step has read the error bits before it counts
// itself; the last one clears them for the next step.
// The count has two levels, so the blocks' atomics do not all queue on one
// address: block b counts itself in group b % kTicketGroups (counters
// kTicketStride words apart), and the last block of each group counts the
// group at the top counter (the ticket word).  Each last block resets the
// counter it completed.
__device__ __forceinline__ void rowonly_clear_flag(const RowOnlyParams& a, int blk, int nblocks) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x != 0) return;
    const int g = blk % kTicketGroups;
    const int members = (nblocks - g + kTicketGroups - 1) / kTicketGroups;
    const int groups = nblocks < kTicketGroups ? nblocks : kTicketGroups;
    int* gc = a.tgroups + g * kTicketStride;
    if (__hip_atomic_fetch_add(gc, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != members - 1) return;
    *gc = 0;
    if (__hip_atomic_fetch_add(a.ticket, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != groups - 1) return;
    *a.ticket = 0;
    *a.flag = 0;
}

// Dense: blocks [0, nb) over the V rows.  Sparse: the same over the n gradient
// rows (mapped through idx), then the decay blocks.  kExact: D is a multiple
// of the chunk width, so no chunk is partial.
// Block `blk` of the `nblk` blocks of one table (kRuntime: dense or sparse is
// the uniform flag sparse_rt, one body for both kinds in a multi-table launch).
template <typename GT, typename WT, int C, bool kSparseArg, bool kExact, bool kRuntime = false>
__device__ __forceinline__ void rowonly_wave_block(const RowOnlyParams& a, unsigned blk, unsigned nblk,
                                                   bool sparse_rt = false) {
    const bool kSparse = kRuntime ? sparse_rt : kSparseArg;
    if (!kSparse) {
        if (blk == 0 && threadIdx.x == 0) *a.status &= kFlagTimeout;
        for (int64_t vb = blk; vb < a.nb; vb += nblk)
            rowonly_wave_rows<GT, WT, C, false, kExact, kRuntime>(a, a.rows, vb, false);
        return;
    }
    const int err = *a.flag;
    if (blk == 0 && threadIdx.x == 0) *a.status = err | (*a.status & kFlagTimeout);
    bool bad_count = false;
    const int64_t nrows = active_rows(a.n_dev, a.rows, bad_count);
    for (int64_t vb = blk; vb < a.nvb; vb += nblk) {
        if (vb >= a.nb) rowonly_decay(a, err, vb - a.nb);
        else if (!err) rowonly_wave_rows<GT, WT, C, true, kExact, kRuntime>(a, nrows, vb, true);
    }
    rowonly_clear_flag(a, (int)blk, (int)nblk);
}

template <typename GT, typename WT, int C, bool kSparse, bool kExact>
__global__ __launch_bounds__(kBlock) void ember_rowonly_wave(RowOnlyParams a) {
    rowonly_wave_block<GT, WT, C, kSparse, kExact>(a, blockIdx.x, gridDim.x);
}

template <typename GT, typename WT, int C, bool kExact>
__global__ __launch_bounds__(kBlock) void ember_rowonly_wave_multi(MultiParams<RowOnlyParams> g) {
    const int k = multi_table(g.first, g.ntab);
    const RowOnlyParams p = g.p[k];
    rowonly_wave_block<GT, WT, C, false, kExact, true>(p, blockIdx.x - g.first[k], g.first[k + 1] - g.first[k],
                                                       g.sparse[k] != 0);
}

// Longer rows: a block of waves per row (see rowonly_rows).
template <typename GT, typename WT, int M, int S, bool kSparse, bool kResident>
__global__ __launch_bounds__(kRowOnlyMaxWaves * kWave) void ember_rowonly(RowOnlyParams a) {
    __shared__ float part[kRowOnlyMaxWaves][kRowOnlyRows];
    __shared__ float rn_lds[kRowOnlyRows];
    if (!kSparse) {
        if (blockIdx.x == 0 && threadIdx.x == 0) *a.status &= kFlagTimeout;
        for (int64_t vb = blockIdx.x; vb < a.nb; vb += gridDim.x)
            rowonly_rows<GT, WT, M, S, false, kResident>(a, a.rows, vb, part, rn_lds);
        return;
    }
    const int err = *a.flag;
    if (blockIdx.x == 0 && threadIdx.x == 0) *a.status = err | (*a.status & kFlagTimeout);
    bool bad_count = false;
    const int64_t nrows = active_rows(a.n_dev, a.rows, bad_count);
    for (int64_t vb = blockIdx.x; vb < a.nvb; vb += gridDim.x) {
        if (vb >= a.nb) rowonly_decay(a, err, vb - a.nb);
        else if (!err) rowonly_rows<GT, WT, M, S, true, kResident>(a, nrows, vb, part, rn_lds);
    }
    rowonly_clear_flag(a, (int)blockIdx.x, (int)gridDim.x);
}

// Sparse row-only step, first launch: validates idx and marks the touched rows
// (slot = 1 + position in idx).  Error bits are ORed into the flag, which the
// fused launch reads and clears.
struct ValidateParams {
    const int64_t* idx;
    int64_t n_max;
    const int64_t* n_dev;
    int64_t V;
    int* slot;
    int* flag;
};

// Block `blk` of the row-only sparse step's id validation of one table.
__device__ __forceinline__ void rowonly_validate_block(const ValidateParams& a, unsigned blk) {
    const int64_t* idx = a.idx;
    const int64_t V = a.V;
    int* slot = a.slot;
    int* flag = a.flag;
    bool bad_count = false;
    const int64_t n = active_rows(a.n_dev, a.n_max, bad_count);
    if (bad_count && blk == 0 && threadIdx.x == 0) atomicOr(flag, kFlagCount);
    const int64_t k = (int64_t)blk * kBlock + threadIdx.x;
    if (k >= n) return;
    const int64_t i = idx[k];
    int bits = 0;
    if (i < 0 || i >= V) bits = kFlagRange;
    else if (atomicCAS(&slot[i], 0, (int)(k + 1)) != 0) bits = kFlagDuplicate;
    if (bits) atomicOr(flag, bits);
}

__global__ __launch_bounds__(kBlock) void ember_rowonly_validate(const int64_t* idx, int64_t n_max,
                                                                const int64_t* n_dev, int64_t V, int* slot,
                                                                int* flag) {
    rowonly_validate_block(ValidateParams{idx, n_max, n_dev, V, slot, flag}, blockIdx.x);
}

__global__ __launch_bounds__(kBlock) void ember_rowonly_validate_multi(MultiParams<ValidateParams> g) {
    const int k = multi_table(g.first, g.ntab);
    rowonly_validate_block(g.p[k], blockIdx.x - g.first[k]);
}

// ---------------------------------------------------------------------------
// sparse-row step in one launch: the rows stay on chip
// ---------------------------------------------------------------------------
//
// A sparse step touches few rows (an embedding batch of 16384 tokens has
// ~4700 distinct ids: 38 MB of bf16 gradient at D = 4096), far less than the
// register files of the chip's 256 compute units (512 KB each).  One block
// per compute unit loads its share of the gradient rows, and of the weight
// rows they update, into registers once; two grid barriers separate
//   1. the slab sums of g^2 of each row (-> mean g^2 per row), the block's
//      column sums of g^2, and the id checks (slot marks);
//   2. the column reduction with the c update and the column factors, and r
//      of every row (decay, or update from the row's mean), with per-block
//      sums of the new r and c;
//   3. s and the step scale from the per-block sums, then the update of the
//      weight rows held since phase 1.
// G is read once (the three-launch path reads it twice), and no launch ramp
// or tail separates the phases.  Wave w of a block takes column slab
// w % nslab of the block's rows r0 + w / nslab + Q u (u < U, Q = 8 / nslab).
// Values one block hands to another inside the launch are stored and loaded
// at agent scope (coherent across the XCDs' L2 caches); the grid barriers'
// waits are bounded and report kFlagTimeout when they run out.

constexpr int kOnchipWaves = kOnchipThreads / kWave;   // 8: two per SIMD
constexpr int kAgentScopeLoad = 16;                     // sc1: buffer loads at agent scope
constexpr int kColGroups = kOnchipThreads / 16;         // phase 2: 16 columns x 32 partial groups

struct OnchipParams {
    void* W;
    int64_t ldw;
    const void* G;
    int64_t ldg;
    const int64_t* idx;
    const int64_t* n_dev;   // device row count, or null
    int64_t rows;           // row count (host), or the maximum of the device count
    int64_t V;
    int64_t D;
    int total_chunks;
    int slab_chunks;
    int nslab;              // at most kOnchipWaves
    int q_lanes;            // kOnchipWaves / nslab: waves per slab
    float* r;
    float* c;
    float beta2;
    float one_minus_beta2;
    double inv_bias;
    double inv_alpha;       // 0 when lr == 0 (no weight is read or written)
    float eps_over_alpha;
    int* slot;              // [V]: marks of the rows of idx (0 between steps)
    int* flag;              // error bits of the launches with an even epoch
    int* flag_odd;          // error bits of the launches with an odd epoch (words of
                            // their own: the other sparse paths keep theirs at zero)
    int* status;            // error bits of the last step (ember_get_error)
    unsigned* epoch;        // launches of this step so far (numbers the barriers)
    unsigned* arrive;       // [kOnchipBlocks * kArriveStride]: each block's last barrier number
    float* P;               // [kOnchipBlocks][D]: per-block column sums of g^2
    double* parts;          // [3][kOnchipBlocks]: per-block sums of the new r (untouched,
                            // touched rows) and of the new c
    float* qa;              // [D rounded up to 8]: column factors sqrt(c_j)
    float* cnew;            // [D]: the new c, stored in phase 3
    int64_t spin_ticks;     // bound of a barrier wait in real-time counter ticks
    int* taken;             // device-count steps beyond the launch's row capacity: 1 when this
                            // launch takes the step (the count fits), else 0 and nothing is done;
                            // null when the host already knows the rows fit
};

__device__ __forceinline__ int ld_agent_i(const int* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned ld_agent_u(const unsigned* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double ld_agent_d(const double* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent_u(unsigned* p, unsigned v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent_d(double* p, double v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Grid barrier number `gen` of the one-launch step: every wave waits until
// its own memory operations have completed, one thread publishes the block's
// arrival in its own flag (no shared counter: 256 atomics on one address
// serialize), and 256 threads poll one flag each until every block has
// arrived, with a bounded wait on the real-time counter.  Flag values only
// grow (two barriers per launch, numbered from the step's epoch), so no flag
// is ever reset.  Returns false when a wait ran out, and records that in the
// step's error bits and in the status word (where it stays until
// ember_init_state: the state is then unspecified).
__device__ bool grid_barrier(unsigned* arrive, unsigned gen, int64_t spin_ticks, int* flag, int* status,
                             int* lds_ok) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
        st_agent_u(arrive + (size_t)blockIdx.x * kArriveStride, gen);
        *lds_ok = 1;
    }
    __syncthreads();
    if (threadIdx.x < kOnchipBlocks) {
        const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
        while ((int)(ld_agent_u(arrive + (size_t)threadIdx.x * kArriveStride) - gen) < 0) {
            if ((int64_t)(__builtin_amdgcn_s_memrealtime() - t0) > spin_ticks) {
                *lds_ok = 0;
                atomicOr(flag, kFlagTimeout);
                atomicOr(status, kFlagTimeout);
                break;
            }
        }
    }
    __syncthreads();
    return *lds_ok != 0;
}

// Gradient and weight rows held per wave (u < U): a unit takes two chunks of
// G and two of W per lane (4 registers per 16-byte chunk, 8 for the 32 bytes
// of fp32 W next to a bf16 chunk of G); U keeps them within ~160 of the 256
// registers a wave has at two waves per SIMD.
template <typename GT, typename WT>
constexpr int onchip_units() {
    constexpr int words = 2 * (4 + (16 / (int)sizeof(GT)) * (int)sizeof(WT) / 4);
    return 160 / words < 10 ? 160 / words : 10;
}

// Sum of one double per thread of the block: waves, then waves in order.
__device__ __forceinline__ double onchip_block_sum(double v, double* lds8) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    v = wave_sum(v);
    if (lane == 0) lds8[wave] = v;
    __syncthreads();
    double t = 0.0;
#pragma unroll
    for (int w = 0; w < kOnchipWaves; ++w) t += lds8[w];
    __syncthreads();
    return t;
}

template <typename GT, typename WT, int M, int U>
__global__ __launch_bounds__(kOnchipThreads, 1) void ember_sparse_onchip(OnchipParams a) {
    constexpr int EPC = 16 / (int)sizeof(GT);
    constexpr int NB = kOnchipBlocks;
    constexpr int kRowsMax = kOnchipWaves * U;        // rows of a block at most
    __shared__ float cl[kOnchipWaves][kWave * EPC];   // the waves' column sums, one chunk column
    __shared__ float rsl2[kRowsMax];                  // slab sums of g^2 of the block's rows
    __shared__ int64_t id_lds[kRowsMax];              // ids of the block's rows (-1: out of range)
    __shared__ float ro_lds[kRowsMax];                // r of those rows before the step
    __shared__ float rn_lds[kRowsMax];                // r of those rows after the step
    __shared__ float part[kColGroups][16];            // column reduction
    __shared__ double dsum[kOnchipWaves];
    __shared__ int sh_ok, sh_err;
    __shared__ float sh_scale;

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int b = blockIdx.x;
    const int64_t V = a.V, D = a.D;
    // ---- phase 1: load the rows, row and column sums of g^2, row marks ----
    bool bad_count = false;
    const int64_t n = active_rows(a.n_dev, a.rows, bad_count);
    if (a.taken != nullptr) {
        // the count decides (the same in every block): more rows per block than
        // the waves hold and the three-launch form takes the step instead
        const bool fits = (n + NB - 1) / NB <= (int64_t)a.q_lanes * U;
        if (b == 0 && threadIdx.x == 0) *a.taken = fits ? 1 : 0;
        if (!fits) return;
    }
    int64_t r0, r1;
    row_range(n, NB, b, r0, r1);
    const int nloc = (int)(r1 - r0);
    const int Q = a.q_lanes;
    const int slab = wave % a.nslab;
    const int q = wave / a.nslab;
    const bool on = q < Q;
    const int cbeg = slab * a.slab_chunks;
    const int cend = min(cbeg + a.slab_chunks, a.total_chunks);
    const bool write_w = a.inv_alpha != 0.0;
    const GT* G = static_cast<const GT*>(a.G);
    WT* W = static_cast<WT*>(a.W);

    // Rows go through raw buffer resources (base = the row, length = its bytes,
    // 0 for an absent row): loads past the length return zero and stores past
    // it are dropped.  Lanes whose chunk lies outside the wave's slab get an
    // offset past every length.  Weight rows are only addressed through ids
    // inside [0, V), and nothing is stored before the step's error bits are
    // final (phase 3).
    constexpr int kWChunkBytes = EPC * (int)sizeof(WT);
    constexpr int kOutside = 1 << 30;   // past the length of every row on this path
    int goff[M], woff[M];
#pragma unroll
    for (int m = 0; m < M; ++m) {
        const int ch = cbeg + lane + kWave * m;
        goff[m] = (on && ch < cend) ? ch * 16 : kOutside;
        woff[m] = (on && ch < cend) ? ch * kWChunkBytes : kOutside;
    }
    const int gbytes = (int)D * (int)sizeof(GT);
    const int wbytes = (int)D * (int)sizeof(WT);
    // lane u holds the id of unit u: one load for all units, issued first
    const int64_t lrow = r0 + q + (int64_t)Q * lane;
    const bool lrv = on && lane < U && lrow < r1;
    const int64_t lid = lrv ? a.idx[lrow] : -1;
    const bool lin = lrv && lid >= 0 && lid < V;
    bool rv[U], wv[U];
    __amdgpu_buffer_rsrc_t wb[U];
    Raw<GT, EPC> graw[U][M];
    Raw<WT, EPC> wraw[U][M];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t row = r0 + q + (int64_t)Q * u;
        rv[u] = on && row < r1;
        const __amdgpu_buffer_rsrc_t gb = row_buffer(G + (rv[u] ? row : 0) * a.ldg, rv[u] ? gbytes : 0);
#pragma unroll
        for (int m = 0; m < M; ++m) buf_load<GT, EPC>(gb, goff[m], graw[u][m]);
    }
    // Every wave reads the epoch itself, once its gradient loads are in flight
    // (no wait and no block barrier in front of them).  The error bits
    // alternate between two words by launch, so block 0 can clear the next
    // launch's word while this launch still reads its own.
    const unsigned epoch = __builtin_amdgcn_readfirstlane(*a.epoch);
    int* flag = (epoch & 1u) ? a.flag_odd : a.flag;
    // Row marks (lane u of each slab-0 wave, unit u's row): a count per id,
    // read in phase 2 (0: untouched, 1: touched, more: a repeated id), so no
    // result has to come back here; and r of the row, loaded before the weight
    // rows so that waiting for it waits for the gradient rows only.
    float rold = 0.0f;
    if (slab == 0 && lrv) {
        if (!lin) {
            atomicOr(flag, kFlagRange);
        } else {
            __hip_atomic_fetch_add(a.slot + lid, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            rold = a.r[lid];
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t i = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(lid >> 32), u) << 32) |
                                    (uint32_t)__builtin_amdgcn_readlane((int)lid, u));
        wv[u] = rv[u] && i >= 0 && i < V;
        wb[u] = row_buffer(W + (wv[u] ? i : 0) * a.ldw, wv[u] && write_w ? wbytes : 0);
#pragma unroll
        for (int m = 0; m < M; ++m) buf_load<WT, EPC>(wb[u], woff[m], wraw[u][m]);
    }
    // every load is issued before the first wait, and no decode moves above them
    __builtin_amdgcn_sched_barrier(0);
    if (bad_count && b == 0 && threadIdx.x == 0) atomicOr(flag, kFlagCount);

    float acc[M][EPC];
#pragma unroll
    for (int m = 0; m < M; ++m)
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[m][e] = 0.0f;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
        for (int m = 0; m < M; ++m) {
            float x[EPC];
            decode(graw[u][m], x);
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                acc[m][e] = fmaf(x[e], x[e], acc[m][e]);
                if (e & 1) s1 = fmaf(x[e], x[e], s1);
                else s0 = fmaf(x[e], x[e], s0);
            }
        }
        const float ss = wave_sum(s0 + s1);
        if (lane == 0 && rv[u]) rsl2[(q + Q * u) * a.nslab + slab] = ss;
        // The column sums are complete for this unit here (the compiler would
        // otherwise defer the additions and keep every decoded value live), and
        // phase 3 decodes the raw words again.
#pragma unroll
        for (int m = 0; m < M; ++m) {
#pragma unroll
            for (int e = 0; e < EPC; ++e) asm volatile("" : "+v"(acc[m][e]));
            launder(graw[u][m]);
        }
        __builtin_amdgcn_sched_barrier(0);
    }

    // column sums of the block: the Q waves of each slab in order -> P[b]
    const __amdgpu_buffer_rsrc_t prs_w = __builtin_amdgcn_make_buffer_rsrc(a.P + (int64_t)b * D, 0, (int)(D * 4),
                                                                           kBufferWord3);
#pragma unroll
    for (int m = 0; m < M; ++m) {
#pragma unroll
        for (int e = 0; e < EPC; ++e) cl[wave][lane * EPC + e] = acc[m][e];
        __syncthreads();
        // four consecutive columns per thread, one 16-byte agent-scope store
        for (int x4 = threadIdx.x; x4 < a.nslab * kWave * EPC / 4; x4 += kOnchipThreads) {
            const int x = 4 * x4;
            const int s = x / (kWave * EPC);
            const int off = x - s * (kWave * EPC);
            const int ch = s * a.slab_chunks + kWave * m + off / EPC;
            const int send = min((s + 1) * a.slab_chunks, a.total_chunks);
            if (ch < send) {
                float4 v = *reinterpret_cast<const float4*>(&cl[s][off]);
                for (int qq = 1; qq < Q; ++qq) {
                    const float4 w = *reinterpret_cast<const float4*>(&cl[qq * a.nslab + s][off]);
                    v.x += w.x;
                    v.y += w.y;
                    v.z += w.z;
                    v.w += w.w;
                }
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), prs_w,
                                                       (ch * EPC + off % EPC) * 4, 0, kAgentScopeLoad);
            }
        }
        __syncthreads();
    }
    if (slab == 0 && lrv) {
        const int t = q + Q * lane;
        id_lds[t] = lin ? lid : -1;
        ro_lds[t] = rold;
    }
    __syncthreads();
    // the block's rows: mean g^2 from the slab sums (slab order, float64),
    // the new r, and the sum of the new r in row order
    double tsum = 0.0;
    {
        const double invD = 1.0 / (double)D;
        float rn = 0.0f;
        if (threadIdx.x < nloc) {
            double sum = 0.0;
            for (int sb = 0; sb < a.nslab; ++sb) sum += (double)rsl2[threadIdx.x * a.nslab + sb];
            const float mean = (float)(sum * invD);
            rn = fmaf(a.beta2, ro_lds[threadIdx.x], a.one_minus_beta2 * mean);
            rn_lds[threadIdx.x] = rn;
        }
        tsum = onchip_block_sum((double)rn, dsum);
    }

    const unsigned gen = 2u * epoch + 1u;
    const bool ok1 = grid_barrier(a.arrive, gen, a.spin_ticks, flag, a.status, &sh_ok);

    // ---- phase 2: c and the column factors; r of every row (kept until phase 3) ----
    // Block b owns columns [c0, c1) and rows [v0, v1).  Each round takes 16
    // columns (thread (g, x) adds partials g, g + 32, ... of column c0 + x,
    // then 16 threads add the 32 group sums in group order) and 512 rows (one
    // per thread: untouched rows decay, a count above one is a repeated id,
    // marks are cleared); all loads of a round are issued before the first is
    // used.  The new c and r are stored in phase 3, once the error bits are
    // final.
    const int64_t c0 = D * b / NB, c1 = D * (b + 1) / NB;
    const int64_t v0 = V * b / NB, v1 = V * (b + 1) / NB;
    // at least one round; the new values of the first round stay in registers
    const int64_t rounds = max((int64_t)1, max((c1 - c0 + 15) / 16, (v1 - v0 + kOnchipThreads - 1) / kOnchipThreads));
    float rn0 = 0.0f;
    bool rn0_set = false;
    double csum = 0.0, usum = 0.0;
    int dup = 0;
    {
        const int x = threadIdx.x % 16, g = threadIdx.x / 16;
        const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(a.P, 0, (int)(NB * D * 4), kBufferWord3);
        const int prow = kColGroups * (int)D * 4;
        for (int64_t k = 0; k < rounds; ++k) {
            const int64_t j = c0 + 16 * k + x;
            const bool jv = j < c1;
            const int vo = jv ? (g * (int)D + (int)j) * 4 : kOutside;
            uint32_t pv[NB / kColGroups];
#pragma unroll
            for (int q2 = 0; q2 < NB / kColGroups; ++q2)
                pv[q2] = __builtin_amdgcn_raw_buffer_load_b32(prs, vo, q2 * prow, kAgentScopeLoad);
            const float cold = (jv && g == 0) ? a.c[j] : 0.0f;
            const int64_t i = v0 + k * kOnchipThreads + threadIdx.x;
            const bool iv = i < v1;
            const int cnt = iv ? ld_agent_i(a.slot + i) : 0;
            const float ri = iv ? a.r[i] : 0.0f;
            float sp = 0.0f;
#pragma unroll
            for (int q2 = 0; q2 < NB / kColGroups; ++q2) sp += __uint_as_float(pv[q2]);
            part[g][x] = sp;
            __syncthreads();
            if (threadIdx.x < 16 && jv) {
                float colsum = 0.0f;
                for (int w = 0; w < kColGroups; ++w) colsum += part[w][x];
                const float mean = (float)((double)colsum / (double)V);
                const float cn = fmaf(a.beta2, cold, a.one_minus_beta2 * mean);
                st_agent(a.qa + j, sqrtf(cn));
                a.cnew[j] = cn;
                csum += (double)cn;
            }
            if (iv) {
                dup |= cnt > 1;
                if (cnt == 0) usum += (double)(a.beta2 * ri);
                // the first round's rows: the mark is cleared and the new r kept
                // here; later rounds read their marks again in phase 3
                if (k == 0) {
                    if (cnt != 0) {
                        a.slot[i] = 0;
                    } else {
                        rn0 = a.beta2 * ri;
                        rn0_set = true;
                    }
                }
            }
            __syncthreads();   // part is reused by the next round
        }
    }
    if (dup) atomicOr(flag, kFlagDuplicate);
    usum = onchip_block_sum(usum, dsum);
    if (threadIdx.x < kWave) csum = wave_sum(csum);
    if (threadIdx.x == 0) {
        st_agent_d(a.parts + b, usum);
        st_agent_d(a.parts + NB + b, tsum);
        st_agent_d(a.parts + 2 * NB + b, csum);
        // the next launch's error bits start from zero
        if (b == 0) *((epoch & 1u) ? a.flag : a.flag_odd) = 0;
    }

    const bool ok2 = grid_barrier(a.arrive, gen + 1u, a.spin_ticks, flag, a.status, &sh_ok);

    // ---- phase 3: error bits, s, then every store of the step ----
    // wave 0: the error bits and the per-block sums, then s and the step scale
    // in a fixed order (every block alike); every wave: its column factors
    const __amdgpu_buffer_rsrc_t qrs = __builtin_amdgcn_make_buffer_rsrc(a.qa, 0, (int)((D + 7) / 8 * 8 * 4),
                                                                         kBufferWord3);
    u32x4 qraw[M][EPC / 4];
#pragma unroll
    for (int m = 0; m < M; ++m) {
        const int ch = cbeg + lane + kWave * m;
        const int qoff = (on && ch < cend && write_w) ? ch * EPC * 4 : kOutside;
#pragma unroll
        for (int k = 0; k < EPC / 4; ++k)
            qraw[m][k] = __builtin_bit_cast(u32x4,
                                            __builtin_amdgcn_raw_buffer_load_b128(qrs, qoff + 16 * k, 0, kAgentScopeLoad));
    }
    if (threadIdx.x < kWave) {
        const int fl = ld_agent_i(flag);
        double pu[NB / kWave], pt[NB / kWave], pc[NB / kWave];
#pragma unroll
        for (int k = 0; k < NB / kWave; ++k) {
            const int bb = lane * (NB / kWave) + k;
            pu[k] = ld_agent_d(a.parts + bb);
            pt[k] = ld_agent_d(a.parts + NB + bb);
            pc[k] = ld_agent_d(a.parts + 2 * NB + bb);
        }
        double sr = 0.0, sc = 0.0;
#pragma unroll
        for (int k = 0; k < NB / kWave; ++k) {
            sr += pu[k] + pt[k];
            sc += pc[k];
        }
        sr = wave_sum(sr);
        sc = wave_sum(sc);
        if (threadIdx.x == 0) {
            const int err = fl | (ok1 && ok2 ? 0 : kFlagTimeout);
            sh_err = err;
            const double mean_rhat = sr / (double)V * a.inv_bias;
            const double mean_chat = sc / (double)D * a.inv_bias;
            const double s = sqrt(mean_rhat * mean_chat);
            sh_scale = s > 0.0 ? (float)(sqrt(a.inv_bias / s) * a.inv_alpha) : 0.0f;
            // block 0 records the step's error bits (keeping a timeout bit) and
            // numbers the next launch's barriers
            if (b == 0) {
                atomicAnd(a.status, kFlagTimeout);
                atomicOr(a.status, err);
                *a.epoch = epoch + 1u;
            }
        }
    }
    __syncthreads();
    const int err = sh_err;
    // rows beyond the first round: marks read again, cleared, r decayed
    for (int64_t k = 1; k < rounds; ++k) {
        const int64_t i = v0 + k * kOnchipThreads + threadIdx.x;
        if (i >= v1) continue;
        if (ld_agent_i(a.slot + i) != 0) a.slot[i] = 0;
        else if (!err) a.r[i] = a.beta2 * a.r[i];
    }
    if (err) return;
    // the state: this block's columns and rows
    for (int64_t j = c0 + threadIdx.x; j < c1; j += kOnchipThreads) a.c[j] = a.cnew[j];
    if (rn0_set) a.r[v0 + threadIdx.x] = rn0;
    if (threadIdx.x < nloc && id_lds[threadIdx.x] >= 0) a.r[id_lds[threadIdx.x]] = rn_lds[threadIdx.x];
    if (!write_w) return;
    // the weight rows held since phase 1
    const float scale = sh_scale;
    const float epsa = a.eps_over_alpha;
    const float ibias = (float)a.inv_bias;
    float qv[M][EPC];
#pragma unroll
    for (int m = 0; m < M; ++m)
#pragma unroll
        for (int k = 0; k < EPC / 4; ++k) {
            qv[m][4 * k] = __uint_as_float(qraw[m][k].x);
            qv[m][4 * k + 1] = __uint_as_float(qraw[m][k].y);
            qv[m][4 * k + 2] = __uint_as_float(qraw[m][k].z);
            qv[m][4 * k + 3] = __uint_as_float(qraw[m][k].w);
        }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        if (!wv[u]) continue;
        const float ai = sqrtf(rn_lds[q + Q * u] * ibias) * scale;
#pragma unroll
        for (int m = 0; m < M; ++m) {
            // the words are decoded here and nowhere earlier
            launder(graw[u][m]);
            launder(wraw[u][m]);
            float gx[EPC], wx[EPC], o[EPC];
            decode(graw[u][m], gx);
            decode(wraw[u][m], wx);
#pragma unroll
            for (int e = 0; e < EPC; ++e) {
                const float d = fmaf(ai, qv[m][e], epsa);
                const float upd = fmaf(gx[e], __builtin_amdgcn_rcpf(d), wx[e]);
                o[e] = (gx[e] == 0.0f) ? wx[e] : upd;
            }
            buf_store<WT, EPC>(wb[u], woff[m], o);
        }
        __builtin_amdgcn_sched_barrier(0);   // one unit's decoded values at a time
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
    const bool wide = stats_wide(p);
    if (m == 1 && !wide) ember_stats<GT, 1, kStatsRows, kSparse, false><<<grid, kBlock, 0, s>>>(p);
    else if (m == 2 && !wide) ember_stats<GT, 2, kStatsRows, kSparse, false><<<grid, kBlock, 0, s>>>(p);
    else if (m == 1) ember_stats<GT, 1, kStatsRows, kSparse, true><<<grid, kBlock, 0, s>>>(p);
    else if (m == 2) ember_stats<GT, 2, kStatsRows, kSparse, true><<<grid, kBlock, 0, s>>>(p);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

template <typename GT, typename WT, bool kSparse>
hipError_t apply_dispatch(const ApplyParams& p, int m, dim3 grid, hipStream_t s) {
    if (m == 1) ember_apply<GT, WT, 1, kApplyRows, kSparse><<<grid, kBlock, 0, s>>>(p);
    else if (m == 2) ember_apply<GT, WT, 2, kApplyRows, kSparse><<<grid, kBlock, 0, s>>>(p);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

template <typename GT, bool kSparse>
hipError_t apply_dispatch_w(const ApplyParams& p, int w_dtype, int m, dim3 grid, hipStream_t s) {
    if (w_dtype == 0) return apply_dispatch<GT, float, kSparse>(p, m, grid, s);
    return apply_dispatch<GT, uint16_t, kSparse>(p, m, grid, s);
}

// Launch shapes of the row-only kernel: (chunks per lane, slabs per wave,
// resident).  Rows of up to 8 slabs take one slab per wave, up to 16 two.
template <typename GT, typename WT, bool kSparse>
hipError_t rowonly_dispatch(const RowOnlyParams& p, int m, int spw, bool resident, dim3 grid, int threads,
                            hipStream_t s) {
    if (!resident) ember_rowonly<GT, WT, 2, 1, kSparse, false><<<grid, threads, 0, s>>>(p);
    else if (m == 1 && spw == 1) ember_rowonly<GT, WT, 1, 1, kSparse, true><<<grid, threads, 0, s>>>(p);
    else if (m == 2 && spw == 1) ember_rowonly<GT, WT, 2, 1, kSparse, true><<<grid, threads, 0, s>>>(p);
    else if (m == 2 && spw == 2) ember_rowonly<GT, WT, 2, 2, kSparse, true><<<grid, threads, 0, s>>>(p);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

template <typename GT, typename WT, bool kSparse, bool kExact>
hipError_t rowonly_wave_dispatch_c(const RowOnlyParams& p, int c, dim3 grid, hipStream_t s) {
    switch (c) {
    case 1: ember_rowonly_wave<GT, WT, 1, kSparse, kExact><<<grid, kBlock, 0, s>>>(p); break;
    case 2: ember_rowonly_wave<GT, WT, 2, kSparse, kExact><<<grid, kBlock, 0, s>>>(p); break;
    case 4: ember_rowonly_wave<GT, WT, 4, kSparse, kExact><<<grid, kBlock, 0, s>>>(p); break;
    case 8: ember_rowonly_wave<GT, WT, 8, kSparse, kExact><<<grid, kBlock, 0, s>>>(p); break;
    case 16: ember_rowonly_wave<GT, WT, 16, kSparse, kExact><<<grid, kBlock, 0, s>>>(p); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <typename GT, typename WT, bool kSparse>
hipError_t rowonly_wave_dispatch(const RowOnlyParams& p, int c, dim3 grid, hipStream_t s) {
    constexpr int EPC = 16 / (int)sizeof(GT);
    return p.D % EPC == 0 ? rowonly_wave_dispatch_c<GT, WT, kSparse, true>(p, c, grid, s)
                          : rowonly_wave_dispatch_c<GT, WT, kSparse, false>(p, c, grid, s);
}

template <bool kSparse>
hipError_t rowonly_wave_dispatch_t(const RowOnlyParams& p, int g_dtype, int w_dtype, int c, dim3 grid,
                                   hipStream_t s) {
    if (g_dtype == 0)
        return w_dtype == 0 ? rowonly_wave_dispatch<float, float, kSparse>(p, c, grid, s)
                            : rowonly_wave_dispatch<float, uint16_t, kSparse>(p, c, grid, s);
    return w_dtype == 0 ? rowonly_wave_dispatch<uint16_t, float, kSparse>(p, c, grid, s)
                        : rowonly_wave_dispatch<uint16_t, uint16_t, kSparse>(p, c, grid, s);
}

template <bool kSparse>
hipError_t rowonly_dispatch_t(const RowOnlyParams& p, int g_dtype, int w_dtype, int m, int spw, bool resident,
                              dim3 grid, int threads, hipStream_t s) {
    if (g_dtype == 0)
        return w_dtype == 0 ? rowonly_dispatch<float, float, kSparse>(p, m, spw, resident, grid, threads, s)
                            : rowonly_dispatch<float, uint16_t, kSparse>(p, m, spw, resident, grid, threads, s);
    return w_dtype == 0 ? rowonly_dispatch<uint16_t, float, kSparse>(p, m, spw, resident, grid, threads, s)
                        : rowonly_dispatch<uint16_t, uint16_t, kSparse>(p, m, spw, resident, grid, threads, s);
}

} // namespace

// A launch's work-item count is 32 bits wide in the dispatch packet, so grids
// stay far below 2^32 threads: kernels whose natural block count can exceed
// kMaxGridBlocks loop over their virtual blocks.
int64_t capped_blocks(int64_t blocks) { return blocks < kMaxGridBlocks ? blocks : kMaxGridBlocks; }

ColPlan col_plan(int64_t D, int g_dtype) {
    static_assert(kSlabChunks == 64 || kSlabChunks == 128, "one or two chunks per lane");
    ColPlan cp;
    cp.epc = g_dtype == 0 ? 4 : 8;
    cp.total_chunks = (int)((D + cp.epc - 1) / cp.epc);
    cp.nslab = (cp.total_chunks + kSlabChunks - 1) / kSlabChunks;
    cp.slab_chunks = (cp.total_chunks + cp.nslab - 1) / cp.nslab;
    cp.m = cp.slab_chunks > kWave ? 2 : 1;
    return cp;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

WsLayout ws_layout(int64_t V, int64_t D) {
    WsLayout L;
    // the LM-head gradient GEMM writes its partials into the same regions
    const LmheadPlan lp = lmhead_plan(V, D);
    // the narrower plan (bf16: half the slabs of fp32) allows the most row blocks
    int nb = row_blocks(V, col_plan(D, 1).nslab);
    if (row_blocks(V, col_plan(D, 0).nslab) > nb) nb = row_blocks(V, col_plan(D, 0).nslab);
    if (lp.MT > nb) nb = lp.MT;
    if (kOnchipBlocks > nb) nb = kOnchipBlocks;
    const int nslab = nslab_for(D) > lp.NT ? nslab_for(D) : lp.NT;
    size_t off = 0;
    L.flag = off;
    L.status = off + 4;
    L.ticket = off + 8;
    L.scale = off + 12;
    L.epoch = off + 16;
    L.oflag = off + 20;
    L.taken = off + 28;
    off = align256(32);
    L.arrive = off;
    off = align256(off + (size_t)kOnchipBlocks * kArriveStride * 4);
    L.tgroups = off;
    off = align256(off + (size_t)kTicketGroups * kTicketStride * 4);
    L.slot = off;
    off = align256(off + (size_t)V * 4);
    L.zero_end = off;
    L.qa = off;
    off = align256(off + (size_t)((D + 7) / 8 * 8) * 4);
    L.rowpart = off;
    off = align256(off + (size_t)nslab * (size_t)V * 4);
    L.rsum = off;
    off = align256(off + (size_t)((V + kFinRowsPerBlock - 1) / kFinRowsPerBlock) * 4);
    L.csum = off;
    off = align256(off + (size_t)((D + kFinCols - 1) / kFinCols) * 4);
    L.p = off;
    off = align256(off + (size_t)nb * (size_t)D * 4);
    L.parts = off;
    off = align256(off + (size_t)3 * kOnchipBlocks * 8);
    L.cnew = off;
    off = align256(off + (size_t)D * 4);
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

static StatsParams stats_params(const StepArgs& a) {
    const WsLayout L = ws_layout(a.V, a.D);
    const ColPlan cp = col_plan(a.D, a.g_dtype);
    StatsParams p;
    p.G = a.G;
    p.ldg = a.ldg;
    p.rows = a.rows;
    p.D = a.D;
    p.total_chunks = cp.total_chunks;
    p.slab_chunks = cp.slab_chunks;
    p.nslab = cp.nslab;
    p.nb = a.fin_nb > 0 ? a.fin_nb : row_blocks(a.rows, col_plan(a.D, a.g_dtype).nslab, a.sparse);
    {
        const double row_bytes = (double)a.D * (a.g_dtype == 0 ? 4 : 2);
        const int64_t keep = (int64_t)((double)kStatsKeepMB * 1048576.0 / row_bytes);
        p.cached_from = keep >= a.rows ? 0 : a.rows - keep;
    }
    p.rowpart = reinterpret_cast<float*>(a.ws + L.rowpart);
    p.P = reinterpret_cast<float*>(a.ws + L.p);
    p.idx = a.idx;
    p.n_dev = a.n_dev;
    p.V = a.V;
    p.slot = reinterpret_cast<int*>(a.ws + L.slot);
    p.flag = reinterpret_cast<int*>(a.ws + L.flag);
    p.taken = a.taken;
    return p;
}

hipError_t launch_stats(const StepArgs& a, hipStream_t s) {
    const StatsParams p = stats_params(a);
    const ColPlan cp = col_plan(a.D, a.g_dtype);
    // at most 384 row blocks x D / 512 slabs: far below the 2^32-thread limit
    const dim3 grid((unsigned)((int64_t)p.nb * cp.nslab));
    const bool sparse = a.sparse;
    if (a.g_dtype == 0)
        return sparse ? stats_dispatch<float, true>(p, cp.m, grid, s) : stats_dispatch<float, false>(p, cp.m, grid, s);
    return sparse ? stats_dispatch<uint16_t, true>(p, cp.m, grid, s) : stats_dispatch<uint16_t, false>(p, cp.m, grid, s);
}

static FinParams finalize_params(const StepArgs& a) {
    const WsLayout L = ws_layout(a.V, a.D);
    FinParams p;
    p.P = reinterpret_cast<const float*>(a.ws + L.p);
    p.nb = a.fin_nb > 0 ? a.fin_nb : row_blocks(a.rows, col_plan(a.D, a.g_dtype).nslab, a.sparse);
    p.D = a.D;
    p.ncolblocks = (int)((a.D + kFinCols - 1) / kFinCols);
    p.rowpart = reinterpret_cast<const float*>(a.ws + L.rowpart);
    p.nslab = a.fin_nslab > 0 ? a.fin_nslab : col_plan(a.D, a.g_dtype).nslab;
    p.rows = a.rows;
    p.V = a.V;
    p.r = a.r;
    p.c = a.c;
    p.slot = reinterpret_cast<int*>(a.ws + L.slot);
    p.flag = reinterpret_cast<int*>(a.ws + L.flag);
    p.ticket = reinterpret_cast<int*>(a.ws + L.ticket);
    p.status = reinterpret_cast<int*>(a.ws + L.status);
    p.beta2 = a.beta2;
    p.one_minus_beta2 = a.one_minus_beta2;
    p.rsum = reinterpret_cast<float*>(a.ws + L.rsum);
    p.csum = reinterpret_cast<float*>(a.ws + L.csum);
    p.ticket = reinterpret_cast<int*>(a.ws + L.ticket);
    p.qa = reinterpret_cast<float*>(a.ws + L.qa);
    p.scale = reinterpret_cast<float*>(a.ws + L.scale);
    p.inv_bias = a.inv_bias;
    p.inv_alpha = a.inv_alpha;
    p.taken = a.taken;
    return p;
}

static int64_t finalize_blocks(const StepArgs& a) {
    return (a.D + kFinCols - 1) / kFinCols + (a.V + kFinRowsPerBlock - 1) / kFinRowsPerBlock;
}

hipError_t launch_finalize(const StepArgs& a, hipStream_t s) {
    const FinParams p = finalize_params(a);
    const dim3 grid((unsigned)finalize_blocks(a));
    if (a.sparse)
        ember_finalize<true><<<grid, kFinThreads, 0, s>>>(p);
    else
        ember_finalize<false><<<grid, kFinThreads, 0, s>>>(p);
    return hipGetLastError();
}

static ApplyParams apply_params(const StepArgs& a) {
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
    p.nslab = cp.nslab;
    p.nb = apply_blocks(a.rows, a.sparse);
    p.idx = a.idx;
    p.n_dev = a.n_dev;
    p.r = a.r;
    p.qa = reinterpret_cast<const float*>(a.ws + L.qa);
    p.scale = reinterpret_cast<const float*>(a.ws + L.scale);
    p.inv_bias = a.inv_bias;
    p.inv_alpha = a.inv_alpha;
    p.eps_over_alpha = a.eps_over_alpha;
    p.status = reinterpret_cast<const int*>(a.ws + L.status);
    p.flag = reinterpret_cast<int*>(a.ws + L.flag);
    p.taken = a.taken;
    return p;
}

hipError_t launch_apply(const StepArgs& a, hipStream_t s) {
    const ApplyParams p = apply_params(a);
    const ColPlan cp = col_plan(a.D, a.g_dtype);
    const dim3 grid((unsigned)capped_blocks((int64_t)p.nb * cp.nslab));
    const bool sparse = a.sparse;
    if (a.g_dtype == 0)
        return sparse ? apply_dispatch_w<float, true>(p, a.w_dtype, cp.m, grid, s)
                      : apply_dispatch_w<float, false>(p, a.w_dtype, cp.m, grid, s);
    return sparse ? apply_dispatch_w<uint16_t, true>(p, a.w_dtype, cp.m, grid, s)
                  : apply_dispatch_w<uint16_t, false>(p, a.w_dtype, cp.m, grid, s);
}

// ---------------------------------------------------------------------------
// sparse-row step in one launch
// ---------------------------------------------------------------------------

namespace {

template <typename GT, typename WT>
const void* onchip_kernel_m(int m) {
    if (m == 1) return reinterpret_cast<const void*>(&ember_sparse_onchip<GT, WT, 1, onchip_units<GT, WT>()>);
    return reinterpret_cast<const void*>(&ember_sparse_onchip<GT, WT, 2, onchip_units<GT, WT>()>);
}

const void* onchip_kernel(int g_dtype, int w_dtype, int m) {
    if (g_dtype == 0) return w_dtype == 0 ? onchip_kernel_m<float, float>(m) : onchip_kernel_m<float, uint16_t>(m);
    return w_dtype == 0 ? onchip_kernel_m<uint16_t, float>(m) : onchip_kernel_m<uint16_t, uint16_t>(m);
}

int onchip_units_for(int g_dtype, int w_dtype) {
    if (g_dtype == 0) return w_dtype == 0 ? onchip_units<float, float>() : onchip_units<float, uint16_t>();
    return w_dtype == 0 ? onchip_units<uint16_t, float>() : onchip_units<uint16_t, uint16_t>();
}

// Whether every block of the launch can be resident at once on the current
// device: kOnchipBlocks blocks against compute units x blocks per unit of
// this kernel instance (checked once per device and instance).
bool onchip_resident(int g_dtype, int w_dtype, int m) {
    constexpr int kMaxDevices = 64;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return false;
    const int key = (g_dtype * 2 + w_dtype) * 2 + (m - 1);
    static std::mutex mu;
    static signed char known[kMaxDevices][8];
    std::lock_guard<std::mutex> lock(mu);
    signed char& k = known[dev][key];
    if (k == 0) {
        int cus = 0, per_cu = 0;
        const bool ok =
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, onchip_kernel(g_dtype, w_dtype, m),
                                                         kOnchipThreads, 0) == hipSuccess &&
            (int64_t)cus * per_cu >= kOnchipBlocks;
        k = ok ? 1 : -1;
    }
    return k > 0;
}

} // namespace

bool onchip_shape_fits(const StepArgs& a) {
    if (!a.sparse || a.c == nullptr) return false;
    const ColPlan cp = col_plan(a.D, a.g_dtype);
    // whole 16-byte chunks only (rows are read through buffer resources)
    if (cp.nslab > kOnchipWaves || a.D % cp.epc != 0) return false;
    return onchip_resident(a.g_dtype, a.w_dtype, cp.m);
}

bool onchip_fits(const StepArgs& a) {
    if (!onchip_shape_fits(a)) return false;
    const ColPlan cp = col_plan(a.D, a.g_dtype);
    const int64_t per_block = (a.rows + kOnchipBlocks - 1) / kOnchipBlocks;
    return per_block <= (int64_t)(kOnchipWaves / cp.nslab) * onchip_units_for(a.g_dtype, a.w_dtype);
}

OnchipSpace onchip_space(const StepArgs& a) {
    const WsLayout L = ws_layout(a.V, a.D);
    OnchipSpace sp;
    sp.base = a.ws;
    sp.flag = L.oflag;
    sp.flag_odd = L.oflag + 4;
    sp.status = L.status;
    sp.epoch = L.epoch;
    sp.arrive = L.arrive;
    sp.slot = L.slot;
    sp.qa = L.qa;
    sp.cnew = L.cnew;
    sp.p = L.p;
    sp.parts = L.parts;
    sp.status_ptr = nullptr;
    return sp;
}

hipError_t launch_sparse_onchip(const StepArgs& a, const OnchipSpace& sp, hipStream_t s) {
    const ColPlan cp = col_plan(a.D, a.g_dtype);
    OnchipParams p;
    p.W = a.W;
    p.ldw = a.ldw;
    p.G = a.G;
    p.ldg = a.ldg;
    p.idx = a.idx;
    p.n_dev = a.n_dev;
    p.rows = a.rows;
    p.V = a.V;
    p.D = a.D;
    p.total_chunks = cp.total_chunks;
    p.slab_chunks = cp.slab_chunks;
    p.nslab = cp.nslab;
    p.q_lanes = kOnchipWaves / cp.nslab;
    p.r = a.r;
    p.c = a.c;
    p.beta2 = a.beta2;
    p.one_minus_beta2 = a.one_minus_beta2;
    p.inv_bias = a.inv_bias;
    p.inv_alpha = a.inv_alpha;
    p.eps_over_alpha = a.eps_over_alpha;
    p.slot = reinterpret_cast<int*>(sp.base + sp.slot);
    p.flag = reinterpret_cast<int*>(sp.base + sp.flag);
    p.flag_odd = reinterpret_cast<int*>(sp.base + sp.flag_odd);
    p.status = sp.status_ptr ? sp.status_ptr : reinterpret_cast<int*>(sp.base + sp.status);
    p.epoch = reinterpret_cast<unsigned*>(sp.base + sp.epoch);
    p.arrive = reinterpret_cast<unsigned*>(sp.base + sp.arrive);
    p.P = reinterpret_cast<float*>(sp.base + sp.p);
    p.parts = reinterpret_cast<double*>(sp.base + sp.parts);
    p.qa = reinterpret_cast<float*>(sp.base + sp.qa);
    p.cnew = reinterpret_cast<float*>(sp.base + sp.cnew);
    p.spin_ticks = a.spin_ticks;
    p.taken = a.taken;
    // A plain launch: the residency check above (blocks per compute unit x
    // compute units >= kOnchipBlocks) is what the grid barriers rely on, and
    // their bounded waits turn a violation into EMBER_ERR_DEVICE instead of a
    // hang.  (hipLaunchCooperativeKernel measured ~17 us slower per step here.)
    void* args[] = {&p};
    return hipLaunchKernel(onchip_kernel(a.g_dtype, a.w_dtype, cp.m), dim3(kOnchipBlocks), dim3(kOnchipThreads), args,
                           0, s);
}

// ---------------------------------------------------------------------------
// the one-launch sparse step with its scratch inside the library
// ---------------------------------------------------------------------------

namespace {

// Scratch of ember_step_sparse_rows_static.  In host code this name is a
// host-side stand-in, not a device address: kernels and fills only ever get
// the address hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

// Zero fill of the scratch's first `words` words and the caller's status.
__global__ __launch_bounds__(kBlock) void ember_static_prep(uint32_t* p, int64_t words, int* status) {
    if (blockIdx.x == 0 && threadIdx.x == 0) *status = 0;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < words; i += (int64_t)gridDim.x * kBlock)
        p[i] = 0u;
}

} // namespace

size_t static_layout(int64_t V, int64_t D, OnchipSpace* sp) {
    size_t off = 0;
    sp->status = 4;
    sp->epoch = 16;
    sp->flag = 20;
    sp->flag_odd = 24;
    off = align256(28);
    sp->arrive = off;
    off = align256(off + (size_t)kOnchipBlocks * kArriveStride * 4);
    sp->slot = off;
    off = align256(off + (size_t)V * 4);
    sp->zero_end = off;
    sp->qa = off;
    off = align256(off + (size_t)((D + 7) / 8 * 8) * 4);
    sp->p = off;
    off = align256(off + (size_t)kOnchipBlocks * (size_t)D * 4);
    sp->parts = off;
    off = align256(off + (size_t)3 * kOnchipBlocks * 8);
    sp->cnew = off;
    off = align256(off + (size_t)D * 4);
    return off;
}

hipError_t static_scratch(char** out) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static char* addr[kMaxDevices];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (addr[dev] == nullptr) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = static_cast<char*>(ptr);
    }
    *out = addr[dev];
    return hipSuccess;
}

hipError_t launch_static_prep(char* base, size_t zero_bytes, int* status, hipStream_t s) {
    const int64_t words = (int64_t)(zero_bytes / 4);
    int64_t blocks = (words + kBlock - 1) / kBlock;
    if (blocks < 1) blocks = 1;
    if (blocks > 1024) blocks = 1024;
    ember_static_prep<<<dim3((unsigned)blocks), kBlock, 0, s>>>(reinterpret_cast<uint32_t*>(base), words, status);
    return hipGetLastError();
}

hipError_t launch_rowonly_validate(const StepArgs& a, hipStream_t s) {
    const WsLayout L = ws_layout(a.V, a.D);
    if (a.rows == 0 && a.n_dev == nullptr) return hipSuccess;
    const unsigned nblk = (unsigned)(a.rows > 0 ? (a.rows + kBlock - 1) / kBlock : 1);
    ember_rowonly_validate<<<nblk, kBlock, 0, s>>>(a.idx, a.rows, a.n_dev, a.V, reinterpret_cast<int*>(a.ws + L.slot),
                                                   reinterpret_cast<int*>(a.ws + L.flag));
    return hipGetLastError();
}

static RowOnlyParams rowonly_params(const StepArgs& a) {
    const WsLayout L = ws_layout(a.V, a.D);
    const ColPlan cp = col_plan(a.D, a.g_dtype);
    RowOnlyParams p;
    p.W = a.W;
    p.ldw = a.ldw;
    p.G = a.G;
    p.ldg = a.ldg;
    p.rows = a.rows;
    p.D = a.D;
    p.total_chunks = cp.total_chunks;
    p.slab_chunks = cp.slab_chunks;
    p.nslab = cp.nslab;
    p.rows_per_block = kRowOnlyRowsPerBlock;
    p.nb = (a.rows + kRowOnlyRowsPerBlock - 1) / kRowOnlyRowsPerBlock;
    p.idx = a.idx;
    p.n_dev = a.n_dev;
    p.r = a.r;
    p.V = a.V;
    p.beta2 = a.beta2;
    p.one_minus_beta2 = a.one_minus_beta2;
    p.inv_bias = (float)a.inv_bias;
    p.inv_alpha = (float)a.inv_alpha;
    p.eps_over_alpha = a.eps_over_alpha;
    p.slot = reinterpret_cast<int*>(a.ws + L.slot);
    p.flag = reinterpret_cast<int*>(a.ws + L.flag);
    p.ticket = reinterpret_cast<int*>(a.ws + L.ticket);
    p.tgroups = reinterpret_cast<int*>(a.ws + L.tgroups);
    p.status = reinterpret_cast<int*>(a.ws + L.status);
    const int64_t ndecay = a.sparse ? (a.V + kDecayRows - 1) / kDecayRows : 0;
    p.nvb = p.nb + ndecay;
    return p;
}

// Chunks per lane of the one-wave-per-row kernel, or 0 for rows too long for it.
static int rowonly_wave_chunks(const StepArgs& a) {
    const ColPlan cp = col_plan(a.D, a.g_dtype);
    if (cp.total_chunks > kRowOnlyWaveChunks) return 0;
    int c = 1;
    while (c * kWave < cp.total_chunks) c *= 2;
    return c;
}

hipError_t launch_rowonly(const StepArgs& a, hipStream_t s) {
    const ColPlan cp = col_plan(a.D, a.g_dtype);
    const bool resident = cp.nslab <= 2 * kRowOnlyMaxWaves;
    const int spw = cp.nslab <= kRowOnlyMaxWaves ? 1 : 2;
    const int waves = resident ? (cp.nslab + spw - 1) / spw : kRowOnlyMaxWaves;
    if ((spw == 2 || !resident) && cp.m != 2) return hipErrorInvalidValue;
    RowOnlyParams p = rowonly_params(a);
    const int c = rowonly_wave_chunks(a);
    if (c > 0 && a.sparse) {
        p.rows_per_block = kRowOnlySparseRowsPerBlock;
        p.nb = (a.rows + p.rows_per_block - 1) / p.rows_per_block;
        p.nvb = p.nb + (a.V + kDecayRows - 1) / kDecayRows;
    }
    if (p.nvb == 0) return hipSuccess;
    const dim3 grid((unsigned)capped_blocks(p.nvb));
    if (c > 0)
        return a.sparse ? rowonly_wave_dispatch_t<true>(p, a.g_dtype, a.w_dtype, c, grid, s)
                        : rowonly_wave_dispatch_t<false>(p, a.g_dtype, a.w_dtype, c, grid, s);
    if (a.sparse)
        return rowonly_dispatch_t<true>(p, a.g_dtype, a.w_dtype, cp.m, spw, resident, grid, waves * kWave, s);
    return rowonly_dispatch_t<false>(p, a.g_dtype, a.w_dtype, cp.m, spw, resident, grid, waves * kWave, s);
}

// ---------------------------------------------------------------------------
// several tables per launch
// ---------------------------------------------------------------------------

// Threads of one multi-table launch at most (the dispatch packet counts work
// items in 32 bits); the tables past it go to the next launch.
constexpr int64_t kMultiMaxThreads = (int64_t)1 << 31;

namespace {

template <typename GT>
hipError_t stats_multi_dispatch(const MultiParams<StatsParams>& g, int m, bool wide, dim3 grid, hipStream_t s) {
    if (m == 1 && !wide) ember_stats_multi<GT, 1, kStatsRows, false><<<grid, kBlock, 0, s>>>(g);
    else if (m == 2 && !wide) ember_stats_multi<GT, 2, kStatsRows, false><<<grid, kBlock, 0, s>>>(g);
    else if (m == 1) ember_stats_multi<GT, 1, kStatsRows, true><<<grid, kBlock, 0, s>>>(g);
    else if (m == 2) ember_stats_multi<GT, 2, kStatsRows, true><<<grid, kBlock, 0, s>>>(g);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

template <typename GT, typename WT>
hipError_t apply_multi_dispatch(const MultiParams<ApplyParams>& g, int m, dim3 grid, hipStream_t s) {
    if (m == 1) ember_apply_multi<GT, WT, 1, kApplyRows><<<grid, kBlock, 0, s>>>(g);
    else if (m == 2) ember_apply_multi<GT, WT, 2, kApplyRows><<<grid, kBlock, 0, s>>>(g);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

// Packs tables t[0..n) in order into as few launches as the table and thread
// limits allow; build(a) gives a table's parameters, blocks(a) its block count.
template <typename P, typename Build, typename Blocks, typename Launch>
hipError_t launch_groups(const StepArgs* const* t, int n, int threads, Build build, Blocks blocks, Launch launch) {
    int k = 0;
    while (k < n) {
        MultiParams<P> g{};
        int64_t total = 0;
        while (k < n && g.ntab < kMaxTables) {
            const int64_t nb = blocks(*t[k]);
            if (g.ntab > 0 && (total + nb) * threads > kMultiMaxThreads) break;
            g.first[g.ntab] = (unsigned)total;
            g.sparse[g.ntab] = t[k]->sparse ? 1 : 0;
            g.p[g.ntab] = build(*t[k]);
            total += nb;
            ++g.ntab;
            ++k;
        }
        for (int j = g.ntab; j <= kMaxTables; ++j) g.first[j] = (unsigned)total;
        const hipError_t e = launch(g, dim3((unsigned)total));
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

} // namespace

int stats_key(const StepArgs& a) {
    return a.g_dtype * 4 + (col_plan(a.D, a.g_dtype).m - 1) * 2 + (stats_wide(stats_params(a)) ? 1 : 0);
}

int apply_key(const StepArgs& a) {
    return a.g_dtype * 4 + a.w_dtype * 2 + (col_plan(a.D, a.g_dtype).m - 1);
}

hipError_t launch_stats_multi(const StepArgs* const* t, int n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const StepArgs& a0 = *t[0];
    const int m = col_plan(a0.D, a0.g_dtype).m;
    const bool wide = stats_wide(stats_params(a0));
    return launch_groups<StatsParams>(
        t, n, kBlock, stats_params,
        [](const StepArgs& a) {
            const StatsParams p = stats_params(a);
            return (int64_t)p.nb * p.nslab;
        },
        [&](const MultiParams<StatsParams>& g, dim3 grid) {
            return a0.g_dtype == 0 ? stats_multi_dispatch<float>(g, m, wide, grid, s)
                                   : stats_multi_dispatch<uint16_t>(g, m, wide, grid, s);
        });
}

hipError_t launch_finalize_multi(const StepArgs* const* t, int n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    return launch_groups<FinParams>(
        t, n, kFinThreads, finalize_params, finalize_blocks,
        [&](const MultiParams<FinParams>& g, dim3 grid) {
            ember_finalize_multi<<<grid, kFinThreads, 0, s>>>(g);
            return hipGetLastError();
        });
}

hipError_t launch_apply_multi(const StepArgs* const* t, int n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const StepArgs& a0 = *t[0];
    const int m = col_plan(a0.D, a0.g_dtype).m;
    return launch_groups<ApplyParams>(
        t, n, kBlock, apply_params,
        [](const StepArgs& a) {
            const ApplyParams p = apply_params(a);
            return capped_blocks((int64_t)p.nb * p.nslab);
        },
        [&](const MultiParams<ApplyParams>& g, dim3 grid) {
            if (a0.g_dtype == 0)
                return a0.w_dtype == 0 ? apply_multi_dispatch<float, float>(g, m, grid, s)
                                       : apply_multi_dispatch<float, uint16_t>(g, m, grid, s);
            return a0.w_dtype == 0 ? apply_multi_dispatch<uint16_t, float>(g, m, grid, s)
                                   : apply_multi_dispatch<uint16_t, uint16_t>(g, m, grid, s);
        });
}


// Row-only tables of ember_step_multi.

namespace {

template <typename GT, typename WT, bool kExact>
hipError_t rowonly_wave_multi_c(const MultiParams<RowOnlyParams>& g, int c, dim3 grid, hipStream_t s) {
    switch (c) {
    case 1: ember_rowonly_wave_multi<GT, WT, 1, kExact><<<grid, kBlock, 0, s>>>(g); break;
    case 2: ember_rowonly_wave_multi<GT, WT, 2, kExact><<<grid, kBlock, 0, s>>>(g); break;
    case 4: ember_rowonly_wave_multi<GT, WT, 4, kExact><<<grid, kBlock, 0, s>>>(g); break;
    case 8: ember_rowonly_wave_multi<GT, WT, 8, kExact><<<grid, kBlock, 0, s>>>(g); break;
    case 16: ember_rowonly_wave_multi<GT, WT, 16, kExact><<<grid, kBlock, 0, s>>>(g); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <typename GT, typename WT>
hipError_t rowonly_wave_multi_x(const MultiParams<RowOnlyParams>& g, int c, bool exact, dim3 grid, hipStream_t s) {
    return exact ? rowonly_wave_multi_c<GT, WT, true>(g, c, grid, s) : rowonly_wave_multi_c<GT, WT, false>(g, c, grid, s);
}

bool rowonly_exact(const StepArgs& a) { return a.D % col_plan(a.D, a.g_dtype).epc == 0; }

} // namespace

int rowonly_key(const StepArgs& a) {
    const int c = rowonly_wave_chunks(a);
    if (c == 0) return -1;   // rows too long for the one-wave kernel: a launch of its own
    int lc = 0;
    while ((1 << lc) < c) ++lc;
    return ((a.g_dtype * 2 + a.w_dtype) * 8 + lc) * 2 + (rowonly_exact(a) ? 1 : 0);
}

hipError_t launch_rowonly_multi(const StepArgs* const* t, int n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const StepArgs& a0 = *t[0];
    const int c = rowonly_wave_chunks(a0);
    if (c == 0) {
        for (int k = 0; k < n; ++k) {
            const hipError_t e = launch_rowonly(*t[k], s);
            if (e != hipSuccess) return e;
        }
        return hipSuccess;
    }
    const bool exact = rowonly_exact(a0);
    return launch_groups<RowOnlyParams>(
        t, n, kBlock, rowonly_params,
        [](const StepArgs& a) { return capped_blocks(rowonly_params(a).nvb); },
        [&](const MultiParams<RowOnlyParams>& g, dim3 grid) {
            if (a0.g_dtype == 0)
                return a0.w_dtype == 0 ? rowonly_wave_multi_x<float, float>(g, c, exact, grid, s)
                                       : rowonly_wave_multi_x<float, uint16_t>(g, c, exact, grid, s);
            return a0.w_dtype == 0 ? rowonly_wave_multi_x<uint16_t, float>(g, c, exact, grid, s)
                                   : rowonly_wave_multi_x<uint16_t, uint16_t>(g, c, exact, grid, s);
        });
}

hipError_t launch_rowonly_validate_multi(const StepArgs* const* t, int n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    return launch_groups<ValidateParams>(
        t, n, kBlock,
        [](const StepArgs& a) {
            const WsLayout L = ws_layout(a.V, a.D);
            return ValidateParams{a.idx, a.rows, a.n_dev, a.V, reinterpret_cast<int*>(a.ws + L.slot),
                                  reinterpret_cast<int*>(a.ws + L.flag)};
        },
        [](const StepArgs& a) { return (int64_t)(a.rows > 0 ? (a.rows + kBlock - 1) / kBlock : 1); },
        [&](const MultiParams<ValidateParams>& g, dim3 grid) {
            ember_rowonly_validate_multi<<<grid, kBlock, 0, s>>>(g);
            return hipGetLastError();
        });
}

} // namespace ember
