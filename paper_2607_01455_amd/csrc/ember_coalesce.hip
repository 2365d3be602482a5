// Coalescing of per-position token gradients into the (idx, G_rows) input of the
// sparse Ember step, on the GPU.
//
// The input-embedding gradient of one batch position is a one-hot row selector
// times the back-propagated signal (appendix "Decomposing the Squared
// Gradient"); the gradient of row i is the sum of the signals of the positions
// holding token i (appendix "The Fisher is Proportional to Inverse Frequency
// Squared").  Given token ids tok[P] and per-position rows U[P][D]:
//
//   idx[0..n)  the distinct ids, ascending;
//   G[k][j]    the sum of U[p][j] over the positions p with tok[p] == idx[k],
//              in float64, rounded once to G's type.
//
// Pipeline (all integer work is exact and order-independent; every floating
// point sum has a fixed order):
//   1. stable LSD radix sort of (id, position) pairs by id, 1-4 passes of up
//      to 10 bits (digit histograms per tile, offsets, stable scatter ranked with
//      wavefront ballots), so the positions of one id stay ascending;
//   2. head flags of the sorted ids -> distinct ids, segment starts, and the
//      segment number of every sorted entry;
//   3. the sums: the sorted entries are cut into chunks of about L positions
//      (boundaries at multiples of L, moved back to a segment head unless the
//      segment is longer than L); a wavefront sums one chunk for 256 columns
//      in float64, position by position, and writes every segment that lies
//      inside the chunk; the pieces of the segments longer than L go to
//      float64 partial rows; the chunks where such segments end are listed
//      with the chunk each began in, and a last launch adds each one's pieces
//      in chunk order.
// A segment of at most L positions is therefore summed exactly in ascending
// position order; a longer one is summed in that order within each piece of L
// positions and then piece by piece.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ember_launch.h"

namespace ember {
namespace {

constexpr int kCoalThreads = 256;                    // 4 wavefronts
constexpr int kCoalWaves = kCoalThreads / kWave;
constexpr int kCoalItems = 4;                        // keys per thread per tile
constexpr int kTile = kCoalThreads * kCoalItems;     // keys per tile
constexpr int kMaxDigitBits = 10;
constexpr int kMaxBins = 1 << kMaxDigitBits;         // digits of up to 10 bits
constexpr int kInBlockOffsetTiles = 64;              // up to this many tiles the
                                                     // scatter derives its own offsets
constexpr int kRunRows = 16;                         // rows a wavefront holds at once
constexpr int kMinChunkBatches = 3;                  // a chunk is at least this many batches
                                                     // (fewer, longer chunks: at 16384 tokens and
                                                     // D = 4096 every wavefront of the sums is then
                                                     // resident at once, six per SIMD)
constexpr int kMaxChunks = 4096;                     // bound on the chunks ...
constexpr int64_t kMaxPartialElems = (int64_t)1 << 25; // ... and on chunks x D
constexpr int kColsPerLane = 4;                      // columns per lane (4 or 8)
constexpr int kSlabCols = kWave * kColsPerLane;      // columns per wavefront

struct SortPass {
    const int64_t* tok;       // first pass: token ids (clamped into [0, V); tiles flag bad ones)
    const uint32_t* keys_in;  // later passes
    const uint32_t* vals_in;
    uint32_t* keys_out;
    uint32_t* vals_out;
    int64_t P;
    int64_t V;
    int shift;
    int bits;
    int ntiles;
    uint32_t* hist;           // [bins][ntiles] digit counts per tile
    const uint32_t* offs;     // [bins][ntiles] exclusive offsets, or null (derived in the block)
    uint32_t* tile_bad;       // first pass: 1 where the tile holds an id outside [0, V)
};

__device__ __forceinline__ uint32_t key_of(const SortPass& a, int64_t i, int& bad) {
    if (a.tok == nullptr) return a.keys_in[i];
    const int64_t id = a.tok[i];
    if (id < 0) { bad = 1; return 0u; }
    if (id >= a.V) { bad = 1; return (uint32_t)(a.V - 1); }
    return (uint32_t)id;
}

// Digit histogram of one tile.  The first pass also records whether the tile
// holds an invalid id (a plain store per tile: no flag to reset).
__global__ __launch_bounds__(kCoalThreads) void coal_hist(SortPass a) {
    __shared__ uint32_t h[kMaxBins];
    __shared__ int any_bad;
    const int bins = 1 << a.bits;
    for (int b = threadIdx.x; b < bins; b += kCoalThreads) h[b] = 0;
    if (threadIdx.x == 0) any_bad = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kTile;
    int bad = 0;
    // every item's key is loaded before the first is counted
    uint32_t key[kCoalItems];
#pragma unroll
    for (int j = 0; j < kCoalItems; ++j) {
        const int64_t i = base + (int64_t)j * kCoalThreads + threadIdx.x;
        key[j] = i < a.P ? key_of(a, i, bad) : 0u;
    }
#pragma unroll
    for (int j = 0; j < kCoalItems; ++j) {
        const int64_t i = base + (int64_t)j * kCoalThreads + threadIdx.x;
        if (i < a.P) atomicAdd(&h[(key[j] >> a.shift) & (uint32_t)(bins - 1)], 1u);
    }
    if (bad) any_bad = 1;
    __syncthreads();
    for (int b = threadIdx.x; b < bins; b += kCoalThreads)
        a.hist[(int64_t)b * a.ntiles + blockIdx.x] = h[b];
    if (a.tok != nullptr && threadIdx.x == 0) a.tile_bad[blockIdx.x] = (uint32_t)any_bad;
}

// Exclusive prefix sums of n counts with one block (integer: exact).
__global__ __launch_bounds__(1024) void coal_scan(const uint32_t* in, uint32_t* out, int64_t n) {
    __shared__ uint32_t part[1024];
    const int t = threadIdx.x;
    const int64_t per = (n + 1023) / 1024;
    const int64_t b0 = min(n, (int64_t)t * per);
    const int64_t b1 = min(n, b0 + per);
    uint32_t s = 0;
    for (int64_t i = b0; i < b1; ++i) s += in[i];
    part[t] = s;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
        const uint32_t v = t >= off ? part[t - off] : 0u;
        __syncthreads();
        part[t] += v;
        __syncthreads();
    }
    uint32_t run = part[t] - s;
    for (int64_t i = b0; i < b1; ++i) {
        const uint32_t x = in[i];
        out[i] = run;
        run += x;
    }
}

// Exclusive scan of one value per thread over the block (256 threads): an
// inclusive scan inside each wavefront with lane shuffles, then the totals of
// the lower wavefronts from LDS (two block barriers in all).  lds holds at
// least kCoalWaves words.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* lds, uint32_t* total) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    uint32_t x = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const uint32_t y = __shfl_up(x, off, kWave);
        if (lane >= off) x += y;
    }
    if (lane == kWave - 1) lds[wave] = x;
    __syncthreads();
    uint32_t before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kCoalWaves; ++w) {
        const uint32_t c = lds[w];
        before += w < wave ? c : 0u;
        all += c;
    }
    *total = all;
    __syncthreads();
    return before + x - v;
}

// Stable scatter of one tile by the current digit.  Tile keys are taken in
// position order (item j of thread t is key base + j * 256 + t), in groups of
// 64 keys (group j * kCoalWaves + w: item j of wavefront w).  A key's rank
// among equal digits is the number of equal digits in lower lanes of its group
// (from one ballot per digit bit) plus the count of that digit in earlier
// groups: every group's digit counts are written first, then one prefix pass
// per digit over the groups, so the whole ranking takes two block barriers.
constexpr int kGroups = kCoalItems * kCoalWaves;   // groups of 64 keys in a tile

__global__ __launch_bounds__(kCoalThreads) void coal_scatter(SortPass a) {
    __shared__ uint32_t off[kMaxBins];
    // [group][digit]: the group's count of the digit, then the count in the
    // earlier groups of the tile (< kTile, so 16 bits)
    __shared__ uint16_t cnt[kGroups * kMaxBins];
    __shared__ uint32_t scan_lds[kCoalWaves];
    const int bins = 1 << a.bits;
    const int tile = blockIdx.x;
    const int t = threadIdx.x;
    const int lane = t & (kWave - 1);
    const int wave = t / kWave;

    // the tile's keys and values, loaded before the offsets are worked out
    const int64_t base = (int64_t)tile * kTile;
    uint32_t key[kCoalItems], val[kCoalItems];
#pragma unroll
    for (int j = 0; j < kCoalItems; ++j) {
        const int64_t i = base + (int64_t)j * kCoalThreads + t;
        int bad = 0;
        key[j] = 0;
        val[j] = 0;
        if (i < a.P) {
            key[j] = key_of(a, i, bad);
            val[j] = a.tok != nullptr ? (uint32_t)i : a.vals_in[i];
        }
    }

    if (a.offs != nullptr) {
        for (int b = t; b < bins; b += kCoalThreads) off[b] = a.offs[(int64_t)b * a.ntiles + tile];
    } else {
        // offset of digit b in this tile = keys of smaller digits in every tile
        // + keys of digit b in earlier tiles; thread t owns digits
        // [t * per, (t + 1) * per)
        const int per = bins > kCoalThreads ? bins / kCoalThreads : 1;
        uint32_t tot[kMaxBins / kCoalThreads], before[kMaxBins / kCoalThreads];
        uint32_t mine = 0;
        for (int q = 0; q < per; ++q) {
            const int b = t * per + q;
            tot[q] = 0;
            before[q] = 0;
            if (b < bins) {
#pragma unroll 16
                for (int k = 0; k < a.ntiles; ++k) {
                    const uint32_t c = a.hist[(int64_t)b * a.ntiles + k];
                    tot[q] += c;
                    if (k < tile) before[q] += c;
                }
            }
            mine += tot[q];
        }
        uint32_t all;
        uint32_t excl = block_excl_scan(mine, scan_lds, &all);
        for (int q = 0; q < per; ++q) {
            const int b = t * per + q;
            if (b < bins) off[b] = excl + before[q];
            excl += tot[q];
        }
    }
    {
        // clear the counts, two 16-bit entries per word
        uint32_t* c32 = reinterpret_cast<uint32_t*>(cnt);
        for (int x = t; x < kGroups * bins / 2; x += kCoalThreads) c32[x] = 0u;
    }
    __syncthreads();

    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (kWave - lane));
    uint32_t rank[kCoalItems], dig[kCoalItems];
#pragma unroll
    for (int j = 0; j < kCoalItems; ++j) {
        const int64_t i = base + (int64_t)j * kCoalThreads + t;
        const bool valid = i < a.P;
        const uint32_t d = (key[j] >> a.shift) & (uint32_t)(bins - 1);
        uint64_t peers = __ballot(valid);
        for (int b = 0; b < a.bits; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t m = __ballot(bit);
            peers &= bit ? m : ~m;
        }
        rank[j] = (uint32_t)__popcll(peers & below);
        dig[j] = d;
        if (valid && rank[j] == 0) cnt[(j * kCoalWaves + wave) * bins + d] = (uint16_t)__popcll(peers);
    }
    __syncthreads();
    // per digit: counts of the earlier groups, in position order
    for (int b = t; b < bins; b += kCoalThreads) {
        uint32_t r = 0;
#pragma unroll
        for (int g = 0; g < kGroups; ++g) {
            const uint32_t c = cnt[g * bins + b];
            cnt[g * bins + b] = (uint16_t)r;
            r += c;
        }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kCoalItems; ++j) {
        const int64_t i = base + (int64_t)j * kCoalThreads + t;
        if (i < a.P) {
            const uint32_t dst = off[dig[j]] + cnt[(j * kCoalWaves + wave) * bins + dig[j]] + rank[j];
            a.keys_out[dst] = key[j];
            a.vals_out[dst] = val[j];
        }
    }
}

// ---------------------------------------------------------------------------
// distinct ids and segments of the sorted keys
// ---------------------------------------------------------------------------

struct HeadParams {
    const uint32_t* K;        // sorted ids
    int64_t P;
    int ntiles;
    uint32_t* tilecnt;        // heads per tile
    const uint32_t* tileoff;  // exclusive offsets, or null (derived in the block)
    uint32_t* uid;            // [P] segment number of every sorted entry
    uint32_t* seg_start;      // [n + 1]
    int64_t* idx;             // [n] the distinct ids
    int64_t* n_out;
    uint32_t* fix_count;      // cleared here for the sums
    const uint32_t* tile_bad; // index errors found by the first sort pass
    int* status;
};

// Head flags of a thread's kCoalItems sorted entries k0, k0 + 1, ...: the
// entries and the one before them are loaded before any is compared.
__device__ __forceinline__ uint32_t head_bits(const uint32_t* K, int64_t k0, int64_t P) {
    uint32_t v[kCoalItems + 1];
#pragma unroll
    for (int e = 0; e <= kCoalItems; ++e) {
        const int64_t k = k0 - 1 + e;
        v[e] = (k >= 0 && k < P) ? K[k] : 0u;
    }
    uint32_t bits = 0;
#pragma unroll
    for (int e = 0; e < kCoalItems; ++e) {
        const int64_t k = k0 + e;
        if (k < P && (k == 0 || v[e + 1] != v[e])) bits |= 1u << e;
    }
    return bits;
}

// Tiles here are kTile consecutive sorted entries, kCoalItems per thread.
// This launch also clears the count of chunks listed for the fixup.
__global__ __launch_bounds__(kCoalThreads) void coal_heads_count(HeadParams a) {
    __shared__ uint32_t lds[kCoalThreads];
    if (blockIdx.x == 0 && threadIdx.x == 0) *a.fix_count = 0;
    const int64_t k0 = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kCoalItems;
    const uint32_t c = (uint32_t)__popc(head_bits(a.K, k0, a.P));
    uint32_t total;
    (void)block_excl_scan(c, lds, &total);
    if (threadIdx.x == 0) a.tilecnt[blockIdx.x] = total;
}

__global__ __launch_bounds__(kCoalThreads) void coal_heads_write(HeadParams a) {
    __shared__ uint32_t lds[kCoalThreads];
    __shared__ uint32_t tile_base;
    const int64_t k0 = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kCoalItems;
    const uint32_t hb = head_bits(a.K, k0, a.P);
    if (a.tileoff != nullptr) {
        if (threadIdx.x == 0) tile_base = a.tileoff[blockIdx.x];
    } else {
        uint32_t s = 0;
        for (int k = threadIdx.x; k < (int)blockIdx.x; k += kCoalThreads) s += a.tilecnt[k];
        uint32_t total;
        (void)block_excl_scan(s, lds, &total);
        if (threadIdx.x == 0) tile_base = total;
    }
    __syncthreads();
    uint32_t total;
    const uint32_t excl = block_excl_scan((uint32_t)__popc(hb), lds, &total);
    uint32_t u = tile_base + excl;   // segment number of the next head
#pragma unroll
    for (int e = 0; e < kCoalItems; ++e) {
        const int64_t k = k0 + e;
        if (k < a.P) {
            if ((hb >> e) & 1u) {
                a.idx[u] = (int64_t)a.K[k];
                a.seg_start[u] = (uint32_t)k;
                ++u;
            }
            a.uid[k] = u - 1;
        }
    }
    if (blockIdx.x == a.ntiles - 1) {
        // index errors (marked per tile by the first sort pass) -> status, n = -1
        uint32_t bad = 0;
        for (int k = threadIdx.x; k < a.ntiles; k += kCoalThreads) bad |= a.tile_bad[k];
        uint32_t nbad;
        (void)block_excl_scan(bad, lds, &nbad);
        if (threadIdx.x == 0) {
            const uint32_t n = tile_base + total;
            a.seg_start[n] = (uint32_t)a.P;
            *a.n_out = nbad ? -1 : (int64_t)n;   // -1: a device-count step refuses it
            *a.status = nbad ? 1 : 0;
        }
    }
}

// ---------------------------------------------------------------------------
// the sums
// ---------------------------------------------------------------------------

struct SumParams {
    const uint32_t* K;
    const uint32_t* pos;      // sorted positions
    const uint32_t* uid;
    const uint32_t* seg_start;
    const void* U;
    int64_t ldu;
    void* G;
    int64_t ldg;
    int64_t P;
    int64_t D;
    int64_t L;                // chunk length (a multiple of kRunRows)
    int nchunks;
    int nslabs;
    double* partA;            // [nchunks][D]: the first segment of a chunk, begun in an earlier chunk
    double* partB;            // [nchunks][D]: the last segment, continued in a later chunk
    uint32_t* fix_list;       // [4 per entry]: chunk where a segment that began in an earlier chunk
                              // ends, the chunk it began in, its segment number
    uint32_t* fix_count;      // entries of fix_list (cleared by the heads launch)
};

// One lane's kColsPerLane columns of a row: its words, widened to float64.
template <typename T> struct Cols {
    static constexpr int kWords = kColsPerLane * (int)sizeof(T) / 4;
    using raw = uint32_t __attribute__((ext_vector_type(kWords)));
    static __device__ __forceinline__ void widen(const raw& r, double (&x)[kColsPerLane]) {
#pragma unroll
        for (int w = 0; w < kWords; ++w) {
            if constexpr (sizeof(T) == 4) {
                x[w] = (double)__uint_as_float(r[w]);
            } else {
                x[2 * w] = (double)__uint_as_float(r[w] << 16);
                x[2 * w + 1] = (double)__uint_as_float(r[w] & 0xFFFF0000u);
            }
        }
    }
};

// float64 -> bf16, one round-to-nearest-even.  Rounding to fp32 (nearest-even)
// and then to bf16 (nearest-even) gives the correctly rounded result except
// where the fp32 value is a bf16 midpoint that x itself is not: fp32's grid
// refines bf16's and holds every bf16 midpoint, so the first rounding never
// crosses a midpoint, it can only land on one.  In that case (low 16 bits of
// the fp32 value 0x8000, fp32 inexact) the side of the midpoint x lies on
// decides; only then are float64 comparisons needed.
__device__ __forceinline__ uint16_t f64_to_bf16(double x) {
    const float f = (float)x;
    const uint32_t b0 = __float_as_uint(f);
    uint32_t r = (b0 + 0x7FFFu + ((b0 >> 16) & 1u)) >> 16;
    if ((b0 & 0xFFFFu) == 0x8000u) {
        const double fd = (double)f;
        if (fd != x) r = (b0 >> 16) + (fabs(x) > fabs(fd) ? 1u : 0u);
    }
    if (f != f) r = (b0 >> 16) | 0x0040u;   // NaN stays NaN (quiet)
    return (uint16_t)r;
}

// fp32 bits of one input value as a float64 sum of that value alone gives them
// back: 0 + (-0) = +0, and a NaN comes back quiet.
__device__ __forceinline__ uint32_t one_row_f32(uint32_t w) {
    if ((w & 0x7FFFFFFFu) > 0x7F800000u) return w | 0x00400000u;
    return w == 0x80000000u ? 0u : w;
}

// fp32 bits -> bf16, nearest-even (a NaN stays a quiet NaN)
__device__ __forceinline__ uint32_t f32_bits_to_bf16(uint32_t w) {
    if ((w & 0x7FFFFFFFu) > 0x7F800000u) return (w >> 16) | 0x0040u;
    return (w + 0x7FFFu + ((w >> 16) & 1u)) >> 16;
}

template <typename GT>
__device__ __forceinline__ void store_cols(void* G, int64_t ldg, uint32_t u, int64_t col, int64_t D,
                                           const double (&x)[kColsPerLane]) {
    GT* row = static_cast<GT*>(G) + (int64_t)u * ldg;
#pragma unroll
    for (int e = 0; e < kColsPerLane; ++e) {
        if (col + e < D) {
            if constexpr (sizeof(GT) == 4) row[col + e] = (float)x[e];
            else row[col + e] = f64_to_bf16(x[e]);
        }
    }
}

template <typename UT>
__device__ __forceinline__ void load_cols(const UT* row, int64_t col, int64_t D, bool valid,
                                          typename Cols<UT>::raw& r) {
    using raw = typename Cols<UT>::raw;
    r = raw{};
    if (!valid) return;
    if (col + kColsPerLane <= D) {
        r = *reinterpret_cast<const raw*>(row + col);
    } else {
        UT tmp[kColsPerLane] = {};
        for (int e = 0; e < kColsPerLane; ++e)
            if (col + e < D) tmp[e] = row[col + e];
        r = *reinterpret_cast<const raw*>(tmp);
    }
}

// Stores of one lane's 4 columns through a buffer resource whose length is the
// row's D columns: the hardware drops the stores of lanes past the end (D is a
// multiple of 4 where these are used), so no lane-divergent branch is needed.
constexpr int kBufferWord3 = 0x00020000;  // raw 32-bit data format, gfx9 family

__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(void* row, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(row, 0, (int)bytes, kBufferWord3);
}

// One lane's columns of row u of G, already in G's format (kWords words).
template <typename GT>
__device__ __forceinline__ void buf_store_words(void* G, int64_t ldg, uint32_t u, int col, int64_t D,
                                                const uint32_t (&w)[Cols<GT>::kWords]) {
    GT* row = static_cast<GT*>(G) + (int64_t)u * ldg;
    const __amdgpu_buffer_rsrc_t rs = row_rsrc(row, D * (int64_t)sizeof(GT));
    using v4 = decltype(__builtin_amdgcn_raw_buffer_load_b128(rs, 0, 0, 0));
    using v2 = decltype(__builtin_amdgcn_raw_buffer_load_b64(rs, 0, 0, 0));
    constexpr int kW = Cols<GT>::kWords;
    const int byte0 = col * (int)sizeof(GT);
    if constexpr (kW % 4 == 0) {
#pragma unroll
        for (int g = 0; g < kW; g += 4)
            __builtin_amdgcn_raw_buffer_store_b128(v4{w[g], w[g + 1], w[g + 2], w[g + 3]}, rs, byte0 + 4 * g, 0, 0);
    } else {
        static_assert(kW == 2, "4 bf16 columns per lane");
        __builtin_amdgcn_raw_buffer_store_b64(v2{w[0], w[1]}, rs, byte0, 0, 0);
    }
}

// A finished float64 sum, rounded once to G's type.
template <typename GT>
__device__ __forceinline__ void buf_store_cols(void* G, int64_t ldg, uint32_t u, int col, int64_t D,
                                               const double (&x)[kColsPerLane]) {
    uint32_t w[Cols<GT>::kWords];
#pragma unroll
    for (int e = 0; e < Cols<GT>::kWords; ++e) {
        if constexpr (sizeof(GT) == 4) w[e] = __float_as_uint((float)x[e]);
        else w[e] = (uint32_t)f64_to_bf16(x[2 * e]) | ((uint32_t)f64_to_bf16(x[2 * e + 1]) << 16);
    }
    buf_store_words<GT>(G, ldg, u, col, D, w);
}

// A segment of one row: its sum is that row's value, which G's type holds
// exactly when the types agree (else one rounding, fp32 -> bf16), so the
// value is converted without float64 arithmetic; -0 and NaN come out as the
// float64 sum gives them.
template <typename UT, typename GT>
__device__ __forceinline__ void buf_store_one_row(void* G, int64_t ldg, uint32_t u, int col, int64_t D,
                                                  const typename Cols<UT>::raw& r) {
    uint32_t f[kColsPerLane];   // fp32 bits per column
#pragma unroll
    for (int e = 0; e < kColsPerLane; ++e) {
        if constexpr (sizeof(UT) == 4) f[e] = one_row_f32(r[e]);
        else f[e] = one_row_f32((e & 1) ? (r[e / 2] & 0xFFFF0000u) : (r[e / 2] << 16));
    }
    uint32_t w[Cols<GT>::kWords];
#pragma unroll
    for (int e = 0; e < Cols<GT>::kWords; ++e) {
        if constexpr (sizeof(GT) == 4) w[e] = f[e];
        else w[e] = f32_bits_to_bf16(f[2 * e]) | (f32_bits_to_bf16(f[2 * e + 1]) << 16);
    }
    buf_store_words<GT>(G, ldg, u, col, D, w);
}

__device__ __forceinline__ void store_partial(double* row, int64_t col, int64_t D, const double (&x)[kColsPerLane]) {
#pragma unroll
    for (int e = 0; e < kColsPerLane; ++e)
        if (col + e < D) row[col + e] = x[e];
}

// Start of chunk c: the position c * L, moved back to the head of its segment
// when that segment is not longer than L.  Only segments longer than L are then
// cut by chunk boundaries (always at multiples of L); a chunk holds between 1
// and 2L - 1 positions.
// Also returns the segment number at c * L and that segment's start.
__device__ __forceinline__ int64_t chunk_start(const SumParams& a, int64_t c, uint32_t& u, int64_t& s) {
    const int64_t x = c * a.L;
    u = 0;
    s = 0;
    if (x >= a.P) return a.P;
    u = a.uid[x];
    s = a.seg_start[u];
    const int64_t e = a.seg_start[u + 1];
    return e - s > a.L ? x : s;
}

// One wavefront per (chunk, 256-column slab); slabs of a chunk are adjacent,
// and chunks go to wavefronts in reverse order: the last chunks hold the rare
// ids (a segment per row or two, so the most stores and roundings per row)
// and start first, while the long segments of the frequent ids, which only
// stream rows, fill the slots that free up.
// kExact (D a multiple of 4): the wavefront loads kRunRows rows at a time into
// registers (lanes past D read column 0 and store nothing), then walks them in
// order; a row that starts a segment resets the sum, a row that ends one
// stores it.  Segment boundaries depend only on the sorted ids, so every branch
// is uniform across the wavefront.  Otherwise one row at a time.
template <typename UT, typename GT, bool kExact>
__global__ __launch_bounds__(kCoalThreads) void coal_segsum(SumParams a) {
    using raw = typename Cols<UT>::raw;
    const int lane = threadIdx.x & (kWave - 1);
    const int item = blockIdx.x * kCoalWaves + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int ci = item / a.nslabs;
    if (ci >= a.nchunks) return;
    const int slab = item - ci * a.nslabs;
    const int c = a.nchunks - 1 - ci;
    const int64_t col = (int64_t)slab * kSlabCols + (int64_t)lane * kColsPerLane;
    const bool col_ok = col < a.D;
    uint32_t seg0, seg1;
    int64_t start0, start1;
    const int64_t k0 = chunk_start(a, c, seg0, start0);
    const int64_t k1 = chunk_start(a, (int64_t)c + 1, seg1, start1);
    const UT* U = static_cast<const UT*>(a.U);
    const bool began_before = k0 > 0 && a.K[k0] == a.K[k0 - 1];
    const bool ends_after = k1 < a.P && a.K[k1] == a.K[k1 - 1];

    double acc[kColsPerLane] = {};
    int64_t run0 = k0;
    // the chunk's first segment began earlier and ends here: list the chunk
    // for the launch that adds the pieces (once, from the first slab)
    bool ends_crossing = false;
    if constexpr (kExact) {
        const int64_t colc = col_ok ? col : 0;
        // ids, positions and segment numbers of a batch, one per lane (lane nr
        // holds the id after the batch, if any); read back per row with lane
        // reads instead of a memory round trip per row.  The next batch's are
        // loaded behind the current batch's rows.
        auto batch_meta = [&](int64_t s0, uint32_t& kv, uint32_t& pv, uint32_t& uv) {
            const int nr = (int)min((int64_t)kRunRows, k1 - s0);
            const int64_t kl = s0 + min(lane, nr);
            const bool in = s0 < k1;
            kv = in && lane <= nr && kl < a.P ? a.K[kl] : 0xFFFFFFFFu;
            pv = in && lane < nr ? a.pos[kl] : 0u;
            uv = in && lane < nr ? a.uid[kl] : 0u;
        };
        uint32_t kv, pv, uv;
        batch_meta(k0, kv, pv, uv);
        uint32_t kprev = 0;   // id of the row before the batch (read only past the chunk's first row)
        for (int64_t s0 = k0; s0 < k1; s0 += kRunRows) {
            const int nr = (int)min((int64_t)kRunRows, k1 - s0);
            raw rows[kRunRows];
#pragma unroll
            for (int r = 0; r < kRunRows; ++r) {
                const uint32_t p = (uint32_t)__builtin_amdgcn_readlane((int)pv, r < nr ? r : 0);
                rows[r] = *reinterpret_cast<const raw*>(U + (int64_t)p * a.ldu + colc);
            }
            uint32_t kn, pn, un;
            batch_meta(s0 + kRunRows, kn, pn, un);
#pragma unroll
            for (int r = 0; r < kRunRows; ++r) {
                const int64_t k = s0 + r;
                if (r < nr) {
                    const uint32_t kr = (uint32_t)__builtin_amdgcn_readlane((int)kv, r);
                    if (k > run0 && (r == 0 ? kprev != kr
                                            : (uint32_t)__builtin_amdgcn_readlane((int)kv, r - 1) != kr)) {
                        run0 = k;
#pragma unroll
                        for (int e = 0; e < kColsPerLane; ++e) acc[e] = 0.0;
                    }
                    double x[kColsPerLane];
                    Cols<UT>::widen(rows[r], x);
#pragma unroll
                    for (int e = 0; e < kColsPerLane; ++e) acc[e] += x[e];
                    const bool chunk_end = k + 1 == k1;
                    if (chunk_end || (uint32_t)__builtin_amdgcn_readlane((int)kv, r + 1) != kr) {
                        const bool first = run0 == k0 && began_before;
                        const uint32_t u = (uint32_t)__builtin_amdgcn_readlane((int)uv, r);
                        if (first || (chunk_end && ends_after)) {
                            store_partial((first ? a.partA : a.partB) + (int64_t)c * a.D, col, a.D, acc);
                            ends_crossing |= first && !(chunk_end && ends_after);
                        } else if (run0 == k) {
                            buf_store_one_row<UT, GT>(a.G, a.ldg, u, (int)col, a.D, rows[r]);
                        } else {
                            buf_store_cols<GT>(a.G, a.ldg, u, (int)col, a.D, acc);
                        }
                    }
                }
            }
            kprev = (uint32_t)__builtin_amdgcn_readlane((int)kv, kRunRows - 1);
            kv = kn;
            pv = pn;
            uv = un;
        }
    } else {
        for (int64_t k = k0; k < k1; ++k) {
            if (k > run0 && a.K[k] != a.K[k - 1]) {
                run0 = k;
                for (int e = 0; e < kColsPerLane; ++e) acc[e] = 0.0;
            }
            raw r;
            load_cols<UT>(U + (int64_t)a.pos[k] * a.ldu, col, a.D, col_ok, r);
            double x[kColsPerLane];
            Cols<UT>::widen(r, x);
            for (int e = 0; e < kColsPerLane; ++e) acc[e] += x[e];
            const bool chunk_end = k + 1 == k1;
            if (chunk_end || a.K[k + 1] != a.K[k]) {
                const bool first = run0 == k0 && began_before;
                if (first || (chunk_end && ends_after)) {
                    store_partial((first ? a.partA : a.partB) + (int64_t)c * a.D, col, a.D, acc);
                    ends_crossing |= first && !(chunk_end && ends_after);
                } else if (col_ok) {
                    store_cols<GT>(a.G, a.ldg, a.uid[k], col, a.D, acc);
                }
            }
        }
    }
    // (a chunk that begins inside a segment begins at c L, so seg0 and start0
    // are that segment's number and start)
    if (ends_crossing && slab == 0 && lane == 0) {
        const uint32_t e = atomicAdd(a.fix_count, 1u);
        *reinterpret_cast<uint4*>(a.fix_list + 4 * (int64_t)e) =
            make_uint4((uint32_t)c, (uint32_t)(start0 / a.L), seg0, 0u);
    }
}

// Segments that cross chunk boundaries: for each listed chunk (where such a
// segment ends), add the segment's pieces in chunk order: the start chunk's
// last-segment partial, then the first-segment partials of the later chunks.
// One column per lane, 64 columns per wavefront, kFixBatch partial rows loaded
// at a time; the grid walks the (listed chunk, column slab) items.  The
// list order varies from run to run; each item's result does not.
constexpr int kFixBatch = 64;
constexpr int kFixBlocks = 1024;

template <typename GT>
__global__ __launch_bounds__(kCoalThreads) void coal_fixup(SumParams a) {
    const int lane = threadIdx.x & (kWave - 1);
    const int nslabs = (int)((a.D + kWave - 1) / kWave);
    const int64_t items = (int64_t)(*a.fix_count) * nslabs;
    const int64_t wave0 = (int64_t)blockIdx.x * kCoalWaves + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    for (int64_t item = wave0; item < items; item += (int64_t)gridDim.x * kCoalWaves) {
        const uint4 f = *reinterpret_cast<const uint4*>(a.fix_list + 4 * (item / nslabs));
        const int c = (int)f.x;
        const int c0 = (int)f.y;
        const uint32_t u = f.z;
        const int slab = (int)(item % nslabs);
        const int64_t col = (int64_t)slab * kWave + lane;
        const bool ok = col < a.D;
        const int64_t colc = ok ? col : 0;
        double acc = a.partB[(int64_t)c0 * a.D + colc];
        for (int cc = c0 + 1; cc <= c; cc += kFixBatch) {
            double x[kFixBatch];
#pragma unroll
            for (int q = 0; q < kFixBatch; ++q) {
                const int ccq = cc + q <= c ? cc + q : c;
                x[q] = a.partA[(int64_t)ccq * a.D + colc];
            }
#pragma unroll
            for (int q = 0; q < kFixBatch; ++q)
                if (cc + q <= c) acc += x[q];
        }
        if (ok) {
            GT* row = static_cast<GT*>(a.G) + (int64_t)u * a.ldg;
            if constexpr (sizeof(GT) == 4) row[col] = (float)acc;
            else row[col] = f64_to_bf16(acc);
        }
    }
}

// P == 0: no rows, no error.
__global__ void coal_empty(int* status, int64_t* n_out) {
    *status = 0;
    *n_out = 0;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int bits_for(int64_t V) {
    int b = 0;
    while (b < 31 && ((int64_t)1 << b) < V) ++b;
    return b < 1 ? 1 : b;
}

} // namespace

CoalPlan coal_plan(int64_t P, int64_t V, int64_t D) {
    CoalPlan c;
    c.ntiles = (int)((P + kTile - 1) / kTile);
    const int bits = bits_for(V);
    c.passes = (bits + kMaxDigitBits - 1) / kMaxDigitBits;
    c.digit_bits = (bits + c.passes - 1) / c.passes;
    int64_t maxc = kMaxPartialElems / (D > 0 ? D : 1);
    maxc = maxc < 1 ? 1 : (maxc > kMaxChunks ? kMaxChunks : maxc);
    int64_t m = (P + (int64_t)kRunRows * maxc - 1) / ((int64_t)kRunRows * maxc);
    if (m < kMinChunkBatches) m = kMinChunkBatches;
    c.L = (int64_t)kRunRows * m;
    c.nchunks = (int)((P + c.L - 1) / c.L);
    c.nslabs = (int)((D + kSlabCols - 1) / kSlabCols);
    size_t off = 256;   // status words, shared layout with the step workspace
    const size_t nt = (size_t)(c.ntiles > 0 ? c.ntiles : 1);
    const size_t np = (size_t)(P > 0 ? P : 1);
    c.keys_a = off; off = align256(off + np * 4);
    c.vals_a = off; off = align256(off + np * 4);
    c.keys_b = off; off = align256(off + np * 4);
    c.vals_b = off; off = align256(off + np * 4);
    c.hist = off; off = align256(off + (size_t)kMaxBins * nt * 4);
    c.offs = off; off = align256(off + (size_t)kMaxBins * nt * 4);
    c.tile_bad = off; off = align256(off + nt * 4);
    c.tilecnt = off; off = align256(off + nt * 4);
    c.tileoff = off; off = align256(off + nt * 4);
    c.uid = off; off = align256(off + np * 4);
    c.seg_start = off; off = align256(off + (np + 1) * 4);
    const size_t nc = (size_t)(c.nchunks > 0 ? c.nchunks : 1);
    c.part_a = off; off = align256(off + nc * (size_t)D * 8);
    c.part_b = off; off = align256(off + nc * (size_t)D * 8);
    c.fix_list = off; off = align256(off + nc * 16);
    c.fix_count = off; off = align256(off + 4);
    c.total = off;
    return c;
}

hipError_t launch_coalesce(const CoalArgs& a, hipStream_t s) {
    const CoalPlan c = coal_plan(a.P, a.V, a.D);
    char* ws = a.ws;
    int* status = reinterpret_cast<int*>(ws + 4);
    if (a.P == 0) {
        coal_empty<<<1, 1, 0, s>>>(status, a.n_out);
        return hipGetLastError();
    }
    uint32_t* ka = reinterpret_cast<uint32_t*>(ws + c.keys_a);
    uint32_t* va = reinterpret_cast<uint32_t*>(ws + c.vals_a);
    uint32_t* kb = reinterpret_cast<uint32_t*>(ws + c.keys_b);
    uint32_t* vb = reinterpret_cast<uint32_t*>(ws + c.vals_b);
    uint32_t* hist = reinterpret_cast<uint32_t*>(ws + c.hist);
    uint32_t* offs = reinterpret_cast<uint32_t*>(ws + c.offs);
    uint32_t* tile_bad = reinterpret_cast<uint32_t*>(ws + c.tile_bad);
    const bool in_block = c.ntiles <= kInBlockOffsetTiles;

    // 1. sort
    const uint32_t* kin = nullptr;
    const uint32_t* vin = nullptr;
    for (int q = 0; q < c.passes; ++q) {
        SortPass p;
        p.tok = q == 0 ? a.tok : nullptr;
        p.keys_in = kin;
        p.vals_in = vin;
        p.keys_out = (q & 1) ? kb : ka;
        p.vals_out = (q & 1) ? vb : va;
        p.P = a.P;
        p.V = a.V;
        p.shift = q * c.digit_bits;
        p.bits = c.digit_bits;
        p.ntiles = c.ntiles;
        p.hist = hist;
        p.offs = in_block ? nullptr : offs;
        p.tile_bad = tile_bad;
        coal_hist<<<c.ntiles, kCoalThreads, 0, s>>>(p);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        if (!in_block) {
            coal_scan<<<1, 1024, 0, s>>>(hist, offs, (int64_t)c.ntiles << p.bits);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        coal_scatter<<<c.ntiles, kCoalThreads, 0, s>>>(p);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        kin = p.keys_out;
        vin = p.vals_out;
    }

    // 2. distinct ids and segments
    HeadParams h;
    h.K = kin;
    h.P = a.P;
    h.ntiles = c.ntiles;
    h.tilecnt = reinterpret_cast<uint32_t*>(ws + c.tilecnt);
    h.tileoff = in_block ? nullptr : reinterpret_cast<uint32_t*>(ws + c.tileoff);
    h.uid = reinterpret_cast<uint32_t*>(ws + c.uid);
    h.seg_start = reinterpret_cast<uint32_t*>(ws + c.seg_start);
    h.idx = a.idx;
    h.n_out = a.n_out;
    h.fix_count = reinterpret_cast<uint32_t*>(ws + c.fix_count);
    h.tile_bad = tile_bad;
    h.status = status;
    coal_heads_count<<<c.ntiles, kCoalThreads, 0, s>>>(h);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (!in_block) {
        coal_scan<<<1, 1024, 0, s>>>(h.tilecnt, reinterpret_cast<uint32_t*>(ws + c.tileoff), c.ntiles);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    coal_heads_write<<<c.ntiles, kCoalThreads, 0, s>>>(h);
    e = hipGetLastError();
    if (e != hipSuccess) return e;

    // 3. sums
    SumParams m;
    m.K = kin;
    m.pos = vin;
    m.uid = h.uid;
    m.seg_start = h.seg_start;
    m.U = a.U;
    m.ldu = a.ldu;
    m.G = a.G;
    m.ldg = a.ldg;
    m.P = a.P;
    m.D = a.D;
    m.L = c.L;
    m.nchunks = c.nchunks;
    m.nslabs = c.nslabs;
    m.partA = reinterpret_cast<double*>(ws + c.part_a);
    m.partB = reinterpret_cast<double*>(ws + c.part_b);
    m.fix_list = reinterpret_cast<uint32_t*>(ws + c.fix_list);
    m.fix_count = h.fix_count;
    const int64_t items = (int64_t)c.nchunks * c.nslabs;
    const unsigned grid = (unsigned)((items + kCoalWaves - 1) / kCoalWaves);
    const bool exact = a.D % kColsPerLane == 0;
    if (a.u_dtype == 0) {
        if (a.g_dtype == 0) {
            if (exact) coal_segsum<float, float, true><<<grid, kCoalThreads, 0, s>>>(m);
            else coal_segsum<float, float, false><<<grid, kCoalThreads, 0, s>>>(m);
        } else {
            if (exact) coal_segsum<float, uint16_t, true><<<grid, kCoalThreads, 0, s>>>(m);
            else coal_segsum<float, uint16_t, false><<<grid, kCoalThreads, 0, s>>>(m);
        }
    } else {
        if (a.g_dtype == 0) {
            if (exact) coal_segsum<uint16_t, float, true><<<grid, kCoalThreads, 0, s>>>(m);
            else coal_segsum<uint16_t, float, false><<<grid, kCoalThreads, 0, s>>>(m);
        } else {
            if (exact) coal_segsum<uint16_t, uint16_t, true><<<grid, kCoalThreads, 0, s>>>(m);
            else coal_segsum<uint16_t, uint16_t, false><<<grid, kCoalThreads, 0, s>>>(m);
        }
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    // one (listed chunk, 64-column slab) item per wavefront in the worst case
    const int64_t fix_items = (int64_t)c.nchunks * ((a.D + kWave - 1) / kWave);
    // (a grid-stride loop: the listed chunks are few, and a block that finds no
    // item costs a launch slot)
    const unsigned fix_blocks = (unsigned)min((fix_items + kCoalWaves - 1) / kCoalWaves, (int64_t)kFixBlocks);
    if (a.g_dtype == 0) coal_fixup<float><<<fix_blocks, kCoalThreads, 0, s>>>(m);
    else coal_fixup<uint16_t><<<fix_blocks, kCoalThreads, 0, s>>>(m);
    return hipGetLastError();
}

} // namespace ember
