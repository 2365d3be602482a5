// LM-head weight gradient with the Ember statistics in its epilogue (gfx950).
//
// For an LM head z_m = W h_m the cross-entropy gradient of row i is
// G_i = sum_m (q_mi - 1[y_m = i]) h_m (appendix, "The LM Head Factorizes Like
// the Embedding Table"), i.e. G = dY^T H with dY[T][V] the logits gradient and
// H[T][D] the hidden states.  This kernel forms G with bf16 MFMA (fp32
// accumulation), rounds it once to its storage dtype, stores it, and, from the
// stored values, writes the two partial reductions the Ember step starts from
// (Algorithm 1, the row and column means of g^2):
//   rowpart[tn][i] = sum of g_ij^2 over the tile's columns j,
//   P[tm][j]       = sum of g_ij^2 over the tile's rows i,
// in fixed orders.  The finalize pass of the step reduces both arrays exactly
// as it reduces the statistics pass's partials, so the step's first read of G
// is gone.
//
// Tiling: one block computes a 256 x 256 tile of G (256 rows of the
// vocabulary, 256 hidden columns) with 8 wavefronts, two per SIMD, so one
// wave's MFMAs run while the other waits on LDS or a barrier; wave w owns the
// 64 x 128 part (w % 4, w / 4) as 2 x 4 MFMA 32x32x16 tiles (a 4-wave form
// with 128 x 128 parts is a compile-time option).  The contraction runs over
// the tokens in steps of 64.  Both operands are stored token-major, so each
// step's 64 x 256 slices go from global memory straight into LDS as they are
// (16-byte buffer loads with an LDS destination) and are turned into the MFMA
// operand layout (8 consecutive tokens per lane) by the LDS transpose read
// ds_read_b64_tr_b16.  A ring of LDS stages keeps the loads of the next
// step(s) in flight while a step is multiplied, and the operand reads of
// each 16-token sub-step run in the shadow of the previous sub-step's MFMAs.
// Tiles are numbered so that the blocks one XCD runs at a time share a few
// row tiles and a window of column tiles (its L2 holds their slices).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "ember_launch.h"

namespace ember {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kGemmWaves = 8;                   // wavefronts per block
constexpr int kThreads = kGemmWaves * kWave;
constexpr int kWavesN = 2;                      // wave grid over the tile: kWavesM x 2
constexpr int kWavesM = kGemmWaves / kWavesN;
constexpr int kBM = kLmheadTile;        // rows of G per block (vocabulary)
constexpr int kBN = kLmheadTile;        // columns of G per block (hidden)
constexpr int kBK = kLmheadK;           // tokens per step
constexpr int kStages = 2;                      // LDS stages (steps in flight)
constexpr int kGroupM = 2;                      // row tiles per group of the tile order
constexpr int kRowBytes = kBM * 2;              // one token's 256 bf16 of one operand
constexpr int kOperandBytes = kBK * kRowBytes;  // one operand's slice of a step
constexpr int kStageBytes = 2 * kOperandBytes;  // dY slice, then H slice
constexpr int kRowsPerLoad = kWave * 16 / kRowBytes;            // rows one wave-wide load fills (2)
constexpr int kLoadsPerWave = kBK / kRowsPerLoad / kGemmWaves;  // per operand and step
constexpr int kWaveRows = kBM / kWavesM;        // rows of one wave's part of the tile (64)
constexpr int kWaveCols = kBN / kWavesN;        // its columns (128)
constexpr int kMT = kWaveRows / 32;             // 32 x 32 MFMA tiles per wave: kMT x kNT
constexpr int kNT = kWaveCols / 32;
constexpr int kXcds = 8;
constexpr int kBufferWord3 = 0x00020000;  // raw 32-bit data format, gfx9 family

static_assert(kBM == kBN, "both operand slices share one LDS layout");
static_assert(kBM == 256 && kBK % 16 == 0, "wave tiling assumes 256 x 256 tiles");
static_assert(kGemmWaves == 8, "8 wavefronts per block");
static_assert(kStages >= 2 && kLoadsPerWave * kRowsPerLoad * kGemmWaves == kBK, "load split");
static_assert(kStages * kStageBytes <= 160 * 1024, "LDS of one CU");
static_assert((kStages - 2) * 2 * kLoadsPerWave < 64, "vmcnt range");
static_assert(kStages == 2, "a ring of two stages");

struct Params {
    const uint16_t* dY;   // [T][ldy] bf16
    int64_t ldy;
    const uint16_t* H;    // [T][ldh] bf16
    int64_t ldh;
    int64_t T;
    int64_t V;
    int64_t D;
    void* G;              // [V][ldg], float or bf16
    int64_t ldg;
    float* rowpart;       // [NT][V]
    float* P;             // [MT][D]
    int MT;
    int NT;
    int64_t tile0;        // this launch's tiles: [tile0, tile1) of the MT * NT
    int64_t tile1;
    int64_t per_xcd;      // tiles per XCD: ceil((tile1 - tile0) / 8)
    int group_m;          // row tiles per group of the tile order
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, int64_t bytes) {
    const int n = bytes > 0x7FFFFFF0 ? 0x7FFFFFF0 : (int)bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, n, kBufferWord3);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float x) {
    const uint32_t u = __float_as_uint(x);
    const uint32_t rne = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
    return (x != x) ? ((u >> 16) | 0x0040u) : rne;
}

// Logical tile -> (row tile, column tile): groups of group_m row tiles, row
// tile fastest inside a group, so a run of consecutive tiles covers group_m
// row tiles and a window of column tiles.
__device__ __forceinline__ void tile_of(const Params& a, int64_t l, int& tm, int& tn) {
    const int64_t per_group = (int64_t)a.group_m * a.NT;
    const int64_t g = l / per_group;
    const int first = (int)(g * a.group_m);
    const int gm = min(a.MT - first, a.group_m);
    const int64_t q = l - g * per_group;
    tm = first + (int)(q % gm);
    tn = (int)(q / gm);
}

// Epilogue of one tile.  Each wavefront takes its kWaveRows x 128 part in
// strips of kStripRows rows: the strip's values are rounded to the G dtype
// (the statistics are taken from the rounded values, as the step would read
// them) and written to a wave-private LDS strip in the MFMA layout; the column
// sums are accumulated on the way.  The strip is then read back row by row,
// stored to G with 16-byte stores, and its row sums are formed by the lanes
// that share a row.  Last, the waves that share rows (or columns) add their
// partials in a fixed order through LDS.
template <typename GT>
constexpr int kStripRows = sizeof(GT) == 4 ? 16 : 32;
template <typename GT>
constexpr int kStripPitch = 128 * (int)sizeof(GT) + 16;    // bytes per strip row (padded)
template <typename GT>
constexpr int kStripBytes = kStripRows<GT> * kStripPitch<GT>;
constexpr int kRedBytes = (kWavesN + kWavesM) * kLmheadTile * 4;   // row and column partials

template <typename GT>
__device__ __forceinline__ void epilogue(const Params& a, int tm, int tn, f32x16 (&acc)[kMT][kNT], uint8_t* strip,
                                         uint8_t* red) {
    constexpr int kEs = (int)sizeof(GT);
    constexpr int kRows = kStripRows<GT>;
    constexpr int kPitch = kStripPitch<GT>;
    constexpr int kChunksPerRow = 128 * kEs / 16;          // 16-byte chunks per strip row
    constexpr int kLanesPerRow = kChunksPerRow < kWave ? kChunksPerRow : kWave;
    constexpr int kRowsPerPass = kWave / kLanesPerRow;
    constexpr int kEpc = 16 / kEs;                          // elements per chunk
    constexpr int kRegsPerStrip = kRows / 2;                // MFMA registers i of one strip
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int wm = wave % kWavesM, wn = wave / kWavesM;
    const int64_t m0 = (int64_t)tm * kBM + wm * kWaveRows;
    const int64_t n0 = (int64_t)tn * kBN + wn * kWaveCols;
    const int half = lane >> 5, col = lane & 31;
    float* rows_lds = reinterpret_cast<float*>(red);   // [kWavesN][256 rows]
    float* cols_lds = rows_lds + kWavesN * kBM;         // [kWavesM][256 columns]

    float cs[kNT];
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) cs[nt] = 0.0f;
    // read-back mapping: lane -> row pass offset lane / kLanesPerRow, chunk lane % kLanesPerRow
    const int rb_row = lane / kLanesPerRow, rb_chunk = lane % kLanesPerRow;

    __syncthreads();   // every wave is done with the operand stages
#pragma unroll
    for (int mt = 0; mt < kMT; ++mt) {
#pragma unroll
        for (int sp = 0; sp < 32 / kRows; ++sp) {
            // rows sp * kRows .. of the 32-row MFMA tile: registers i with
            // 8 (i / 4) + 4 half + i % 4 in that range, i.e. i in [sp kRows / 2, ...)
            const int64_t mstrip = m0 + mt * 32 + sp * kRows;
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt) {
                const bool nv = n0 + nt * 32 + col < a.D;
#pragma unroll
                for (int ii = 0; ii < kRegsPerStrip; ++ii) {
                    const int i = sp * kRegsPerStrip + ii;
                    const int r = 8 * (i >> 2) + 4 * half + (i & 3) - sp * kRows;
                    const bool v = nv && mstrip + r < a.V;
                    float g;
                    uint8_t* e = strip + r * kPitch + (nt * 32 + col) * kEs;
                    if constexpr (kEs == 2) {
                        const uint32_t h = f32_to_bf16_bits(acc[mt][nt][i]);
                        *reinterpret_cast<uint16_t*>(e) = (uint16_t)h;
                        g = bf16_bits_to_f32(h);
                    } else {
                        g = acc[mt][nt][i];
                        *reinterpret_cast<float*>(e) = g;
                    }
                    cs[nt] += v ? g * g : 0.0f;
                }
            }
            __syncthreads();
            // read back, store, row sums
#pragma unroll
            for (int pass = 0; pass < kRows / kRowsPerPass; ++pass) {
                const int r = pass * kRowsPerPass + rb_row;
                const int64_t m = mstrip + r;
                const int64_t n = n0 + rb_chunk * kEpc;
                const u32x4 w = *reinterpret_cast<const u32x4*>(strip + r * kPitch + rb_chunk * 16);
                float rsum = 0.0f;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if constexpr (kEs == 2) {
                        const float lo = bf16_bits_to_f32(w[q] & 0xFFFFu), hi = bf16_bits_to_f32(w[q] >> 16);
                        rsum += n + 2 * q < a.D ? lo * lo : 0.0f;
                        rsum += n + 2 * q + 1 < a.D ? hi * hi : 0.0f;
                    } else {
                        const float x = __uint_as_float(w[q]);
                        rsum += n + q < a.D ? x * x : 0.0f;
                    }
                }
                if (m < a.V) {
                    char* grow = static_cast<char*>(a.G) + (m * a.ldg + n) * kEs;
                    if (n + kEpc <= a.D) {
                        *reinterpret_cast<u32x4*>(grow) = w;
                    } else {
                        for (int e = 0; e < kEpc && n + e < a.D; ++e) {
                            if constexpr (kEs == 2)
                                reinterpret_cast<uint16_t*>(grow)[e] = (uint16_t)(w[e >> 1] >> (16 * (e & 1)));
                            else
                                reinterpret_cast<uint32_t*>(grow)[e] = w[e];
                        }
                    }
                }
#pragma unroll
                for (int x = 1; x < kLanesPerRow; x <<= 1) rsum += __shfl_xor(rsum, x);
                if (rb_chunk == 0) rows_lds[wn * kBM + wm * kWaveRows + mt * 32 + sp * kRows + r] = rsum;
            }
            __syncthreads();   // the strip is rewritten next
        }
    }
    // columns: rows of the low lane half, then of the high half
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
        const float other = __shfl_xor(cs[nt], 32);
        const float c2 = half == 0 ? cs[nt] + other : other + cs[nt];
        if (half == 0) cols_lds[wm * kBN + wn * kWaveCols + nt * 32 + col] = c2;
    }
    __syncthreads();
    const int x = threadIdx.x;
    if (x < kBM) {
        const int64_t m = (int64_t)tm * kBM + x;
        if (m < a.V) a.rowpart[(int64_t)tn * a.V + m] = rows_lds[x] + rows_lds[kBM + x];
        const int64_t n = (int64_t)tn * kBN + x;
        float c = cols_lds[x];
#pragma unroll
        for (int q = 1; q < kWavesM; ++q) c += cols_lds[q * kBN + x];
        if (n < a.D) a.P[(int64_t)tm * a.D + n] = c;
    }
}

// 16 bytes per lane from a buffer into LDS at lds_base + 16 lane (lanes
// outside the buffer's range write zeros).  Issued as inline assembly so that
// the compiler does not treat every later LDS read as dependent on it (it
// would wait for all such loads before any LDS read); completion is awaited
// explicitly with wait_vmcnt and a barrier before a stage is read.  M0 holds
// the LDS base (wave-uniform) for the load and is restored afterwards; one
// wait state separates its write from the load.
__device__ __forceinline__ void load_to_lds(__amdgpu_buffer_rsrc_t rs, const void* lds_base, int voffset) {
    const uint32_t base = __builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)lds_base);
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
                 "buffer_load_dwordx4 %2, %3, 0 offen lds\n\ts_mov_b32 m0, %0"
                 : "=&s"(saved)
                 : "s"(base), "v"(voffset), "s"(rs)
                 : "memory");
}

// Wait until at most N vector-memory loads of this wave are outstanding
// (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt and lgkmcnt at their
// "no wait" maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <typename GT>
__global__ __launch_bounds__(kThreads) void ember_lmhead_grad(Params a) {
    // kStages ring of (dY slice, H slice) of kBK tokens each, one LDS array
    // per stage, addressed statically (the step loop is unrolled by the ring
    // size; with the compiler's load builtin this also lets it tell the stage
    // being loaded from the stage being read).  Each slice
    // row (one token, 256 columns, 512 bytes) is stored unpadded, its 16-byte
    // chunks XOR-permuted by the row: chunk c of token row k sits at position
    // c ^ (4 (k % 4)).  The transpose reads of a quarter-wave then cover all
    // LDS banks once (no conflicts), and every wave-wide load still fills two
    // whole rows, as the LDS-direct load requires (lane l -> base + 16 l).
    __shared__ __attribute__((aligned(1024))) uint8_t lds0[kStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t lds1[kStageBytes];
    auto stage = [&](auto sc) -> uint8_t* {
        constexpr int k = decltype(sc)::value;
        if constexpr (k == 0) return lds0;
        else return lds1;
    };
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int wm = wave % kWavesM, wn = wave / kWavesM;

    // one tile per block (a loop over tiles would keep per-lane epilogue
    // values live across the contraction); blocks of one XCD take consecutive
    // tiles of this launch's range
    const int64_t l = a.tile0 + (int64_t)(blockIdx.x % kXcds) * a.per_xcd + blockIdx.x / kXcds;
    if (l >= a.tile1) return;
    const int64_t nk = (a.T + kBK - 1) / kBK;
    int tm, tn;
    tile_of(a, l, tm, tn);
    const int64_t v0 = (int64_t)tm * kBM;
    const int64_t d0 = (int64_t)tn * kBN;

    // loads: wave w fills slice row pairs w, w + kGemmWaves, ...; lane l writes row
    // 2 j + l / 32 at chunk position l % 32, i.e. global chunk (l % 32) ^ 4 (row % 4)
    int off_y[kLoadsPerWave], off_h[kLoadsPerWave];
#pragma unroll
    for (int i = 0; i < kLoadsPerWave; ++i) {
        const int row = kRowsPerLoad * (wave + kGemmWaves * i) + lane / 32;
        const int chunk = (lane & 31) ^ (4 * (row & 3));
        off_y[i] = (int)((row * a.ldy + chunk * 8) * 2);
        off_h[i] = (int)((row * a.ldh + chunk * 8) * 2);
    }
    auto issue = [&](int64_t kt, uint8_t* st) {
        // past the last step the resources cover no bytes: the loads write
        // zeros into a stage that is not read again
        const bool in = kt < nk;
        const int64_t k0 = in ? kt * kBK : 0;
        const __amdgpu_buffer_rsrc_t ra = rsrc(a.dY + k0 * a.ldy + v0, in ? ((a.T - k0) * a.ldy - v0) * 2 : 0);
        const __amdgpu_buffer_rsrc_t rb = rsrc(a.H + k0 * a.ldh + d0, in ? ((a.T - k0) * a.ldh - d0) * 2 : 0);
#pragma unroll
        for (int i = 0; i < kLoadsPerWave; ++i) {
            uint8_t* dst = st + (wave + kGemmWaves * i) * (kRowsPerLoad * kRowBytes);
            load_to_lds(ra, dst, off_y[i]);
            load_to_lds(rb, dst + kOperandBytes, off_h[i]);
        }
    };

    // transpose reads: lane l reads token row 8 (l / 32) + (l % 16) / 4 (+ 4),
    // columns 16 ((l / 16) % 2) + 4 (l % 4) + 32 t of its wave's part; with
    // the chunk permutation the byte offset of tile t within a row is
    // 16 (chunk ^ 4 (row % 4)) + 8 (l % 2), and row % 4 = (l % 16) / 4 here
    const int tr_row = 8 * (lane >> 5) + ((lane & 15) >> 2);
    const int cpart = 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1);
    int tr_a[kMT], tr_b[kNT];
#pragma unroll
    for (int t = 0; t < kMT; ++t) {
        const int chunk = wm * (kWaveRows / 8) + t * 4 + cpart;
        tr_a[t] = tr_row * kRowBytes + (chunk ^ (4 * (tr_row & 3))) * 16 + 8 * (lane & 1);
    }
#pragma unroll
    for (int t = 0; t < kNT; ++t) {
        const int chunk = wn * (kWaveCols / 8) + t * 4 + cpart;
        tr_b[t] = tr_row * kRowBytes + (chunk ^ (4 * (tr_row & 3))) * 16 + 8 * (lane & 1) + kOperandBytes;
    }
    auto rd = [&](const uint8_t* p) {
        return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
    };
    auto frags = [&](const uint8_t* st, int kk, bf16x8 (&af)[kMT], bf16x8 (&bfr)[kNT]) {
#pragma unroll
        for (int t = 0; t < kMT; ++t) {
            const uint8_t* pa = st + tr_a[t] + kk * 16 * kRowBytes;
            af[t] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(rd(pa), rd(pa + 4 * kRowBytes),
                                                                      0, 1, 2, 3, 4, 5, 6, 7));
        }
#pragma unroll
        for (int t = 0; t < kNT; ++t) {
            const uint8_t* pb = st + tr_b[t] + kk * 16 * kRowBytes;
            bfr[t] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(rd(pb), rd(pb + 4 * kRowBytes),
                                                                       0, 1, 2, 3, 4, 5, 6, 7));
        }
    };

    f32x16 acc[kMT][kNT];
#pragma unroll
    for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[mt][nt][i] = 0.0f;

    // step kt (stage kt % kStages): this wave's loads of step kt are done
    // once at most the later steps' are outstanding; the barrier makes every
    // wave's visible and frees the stage of step kt - 1, which then takes the
    // loads of step kt + kStages - 1
    auto step = [&](int64_t kt, auto sc) {
        constexpr int k = decltype(sc)::value;
        wait_vmcnt<(kStages - 2) * 2 * kLoadsPerWave>();
        __syncthreads();
        // the first sub-step's operand reads go out first, the loads of step
        // kt + kStages - 1 behind them (the loads' inline assembly is a
        // compiler memory barrier, so this order holds): the read latency
        // overlaps the load issue, and the loads still have the whole step
        const uint8_t* st = stage(sc);
        bf16x8 af[2][kMT], bfr[2][kNT];
        frags(st, 0, af[0], bfr[0]);
        issue(kt + kStages - 1, stage(std::integral_constant<int, (k + kStages - 1) % kStages>{}));
        // scheduling fences between sub-steps: the MFMAs of sub-step kk use
        // operands read in an earlier region, and the reads of sub-step kk + 1
        // fill their shadow (without the fences the scheduler fetches every
        // operand just before its MFMA and waits for it)
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kk = 0; kk < kBK / 16; ++kk) {
            const int cur = kk & 1;
            if (kk + 1 < kBK / 16) frags(st, kk + 1, af[cur ^ 1], bfr[cur ^ 1]);
#pragma unroll
            for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
                for (int nt = 0; nt < kNT; ++nt)
                    acc[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][mt], bfr[cur][nt], acc[mt][nt],
                                                                          0, 0, 0);
            // each MFMA followed by its share of the next sub-step's transpose reads
            if (kk + 1 < kBK / 16) {
                constexpr int kM = kMT * kNT, kR = 2 * (kMT + kNT);
                constexpr int kRpm = (kR + kM - 1) / kM;   // reads after each MFMA
#pragma unroll
                for (int i = 0; i < kM; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
#pragma unroll
                    for (int q = 0; q < kRpm; ++q)
                        if (i * kRpm + q < kR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // step 0 before the loop; step 1 is issued by step 0
    issue(0, lds0);
    // whole rounds of kStages steps (one loop exit keeps the accumulators in
    // place); the up to kStages - 1 steps past the last one multiply the zeros
    // their loads wrote, which adds exact zeros
    for (int64_t kt = 0; kt < nk; kt += kStages) {
        step(kt, std::integral_constant<int, 0>{});
        step(kt + 1, std::integral_constant<int, 1>{});
    }
    wait_vmcnt<0>();   // the zero-filling loads past the end, before the LDS is reused
    // epilogue scratch: wave w's strip in stage array w % kStages (after the
    // strips of the lower waves there), the block's partial sums after the
    // strips in lds1
    constexpr int kStrip = kStripBytes<GT>;
    constexpr int kStripsPerArray = (kGemmWaves + kStages - 1) / kStages;
    static_assert(kStripsPerArray * kStrip + kRedBytes <= kStageBytes, "epilogue scratch fits the stages");
    const int sarr = wave % kStages;
    uint8_t* const sbase = sarr == 0 ? lds0 : lds1;
    uint8_t* const strip = sbase + (wave / kStages) * kStrip;
    uint8_t* const red = lds1 + kStripsPerArray * kStrip;
    epilogue<GT>(a, tm, tn, acc, strip, red);
}

} // namespace

LmheadPlan lmhead_plan(int64_t V, int64_t D) {
    LmheadPlan p;
    p.MT = (int)((V + kLmheadTile - 1) / kLmheadTile);
    p.NT = (int)((D + kLmheadTile - 1) / kLmheadTile);
    return p;
}

hipError_t launch_lmhead_grad(const LmheadArgs& x, hipStream_t s) {
    const LmheadPlan pl = lmhead_plan(x.V, x.D);
    Params p;
    p.dY = static_cast<const uint16_t*>(x.dY);
    p.ldy = x.ldy;
    p.H = static_cast<const uint16_t*>(x.H);
    p.ldh = x.ldh;
    p.T = x.T;
    p.V = x.V;
    p.D = x.D;
    p.G = x.G;
    p.ldg = x.ldg;
    p.rowpart = x.rowpart;
    p.P = x.P;
    p.MT = pl.MT;
    p.NT = pl.NT;
    p.group_m = kGroupM;
    const int64_t total = (int64_t)pl.MT * pl.NT;
    const int64_t per_launch = kMaxGridBlocks;   // a multiple of kXcds
    for (int64_t t0 = 0; t0 < total; t0 += per_launch) {
        p.tile0 = t0;
        p.tile1 = t0 + per_launch < total ? t0 + per_launch : total;
        p.per_xcd = (p.tile1 - t0 + kXcds - 1) / kXcds;
        const dim3 grid((unsigned)(p.per_xcd * kXcds));
        if (x.g_dtype == 0)
            ember_lmhead_grad<float><<<grid, kThreads, 0, s>>>(p);
        else
            ember_lmhead_grad<uint16_t><<<grid, kThreads, 0, s>>>(p);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipGetLastError();
}

} // namespace ember
