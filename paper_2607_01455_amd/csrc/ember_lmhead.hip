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
// Tiling: one block of 4 wavefronts computes a 256 x 256 tile of G (256 rows of
// the vocabulary, 256 hidden columns); wavefront w owns the 128 x 128 quarter
// (w % 2, w / 2) as 4 x 4 MFMA 32x32x16 tiles.  The contraction runs over the
// tokens in steps of 64.  Both operands are stored token-major (the token index
// is the outer one), so each step's 64 x 256 slices are copied to LDS as they
// are (16-byte loads and stores) and turned into the MFMA operand layout (8
// consecutive tokens per lane) by the LDS transpose read ds_read_b64_tr_b16.
// Two LDS stages: the loads of step k + 2 are in flight while step k is
// multiplied.  Tiles are numbered so that the blocks one XCD runs at a time
// share a few row tiles and a window of column tiles (its L2 holds them).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ember_launch.h"

namespace ember {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kThreads = 256;
constexpr int kBM = kLmheadTile;        // rows of G per block (vocabulary)
constexpr int kBN = kLmheadTile;        // columns of G per block (hidden)
constexpr int kBK = kLmheadK;           // tokens per step
constexpr int kPad = EMBER_LMHEAD_PAD;  // bf16 elements after each LDS row
constexpr int kPitch = kBM + kPad;      // LDS row pitch (elements), both operands
constexpr int kOperandElems = kBK * kPitch;
constexpr int kLoads = kBK * kBM / 8 / kThreads;  // 16-byte loads per thread per operand
constexpr int kXcds = 8;
constexpr int kBufferWord3 = 0x00020000;  // raw 32-bit data format, gfx9 family

static_assert(kBM == kBN, "both operand slices share one LDS layout");
static_assert(kBM == 256 && kBK % 16 == 0, "wave tiling assumes 256 x 256 tiles");

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

// Epilogue of one tile.  Each wavefront takes its 128 x 128 quarter in four
// strips of 32 rows: the strip's values are rounded to the G dtype (the
// statistics are taken from the rounded values, as the step would read them)
// and written to a wave-private LDS strip in the MFMA layout; the column sums
// are accumulated on the way.  The strip is then read back row by row, stored
// to G with 16-byte stores, and its row sums are formed by the lanes that
// share a row.  Last, the two waves that share rows (or columns) add their
// partials in a fixed order through LDS.
template <typename GT>
__device__ __forceinline__ void epilogue(const Params& a, int tm, int tn, f32x16 (&acc)[4][4], uint8_t* smem) {
    constexpr int kEs = (int)sizeof(GT);
    constexpr int kStripPitch = 128 * kEs + 16;            // bytes per strip row (padded)
    constexpr int kChunksPerRow = 128 * kEs / 16;          // 16-byte chunks per strip row
    constexpr int kLanesPerRow = kChunksPerRow < kWave ? kChunksPerRow : kWave;
    constexpr int kRowsPerPass = kWave / kLanesPerRow;
    constexpr int kEpc = 16 / kEs;                          // elements per chunk
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int wm = wave & 1, wn = wave >> 1;
    const int64_t m0 = (int64_t)tm * kBM + wm * 128;
    const int64_t n0 = (int64_t)tn * kBN + wn * 128;
    const int half = lane >> 5, col = lane & 31;
    uint8_t* strip = smem + wave * (32 * kStripPitch);
    float* rows_lds = reinterpret_cast<float*>(smem + 4 * 32 * kStripPitch);   // [2 column halves][256 rows]
    float* cols_lds = rows_lds + 2 * kBM;                                        // [2 row halves][256 columns]

    float cs[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) cs[nt] = 0.0f;
    // read-back mapping: lane -> row pass offset lane / kLanesPerRow, chunk lane % kLanesPerRow
    const int rb_row = lane / kLanesPerRow, rb_chunk = lane % kLanesPerRow;

    __syncthreads();   // every wave is done with the operand stages
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
        const int64_t mstrip = m0 + mt * 32;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            const bool nv = n0 + nt * 32 + col < a.D;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int r = 8 * (i >> 2) + 4 * half + (i & 3);
                const bool v = nv && mstrip + r < a.V;
                float g;
                uint8_t* e = strip + r * kStripPitch + (nt * 32 + col) * kEs;
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
        for (int pass = 0; pass < 32 / kRowsPerPass; ++pass) {
            const int r = pass * kRowsPerPass + rb_row;
            const int64_t m = mstrip + r;
            const int64_t n = n0 + rb_chunk * kEpc;
            const u32x4 w = *reinterpret_cast<const u32x4*>(strip + r * kStripPitch + rb_chunk * 16);
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
            if (rb_chunk == 0) rows_lds[wn * kBM + wm * 128 + mt * 32 + r] = rsum;
        }
        __syncthreads();   // the strip is rewritten by the next mt
    }
    // columns: rows of the low lane half, then of the high half
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
        const float other = __shfl_xor(cs[nt], 32);
        const float c2 = half == 0 ? cs[nt] + other : other + cs[nt];
        if (half == 0) cols_lds[wm * kBN + wn * 128 + nt * 32 + col] = c2;
    }
    __syncthreads();
    const int x = threadIdx.x;
    const int64_t m = (int64_t)tm * kBM + x;
    if (m < a.V) a.rowpart[(int64_t)tn * a.V + m] = rows_lds[x] + rows_lds[kBM + x];
    const int64_t n = (int64_t)tn * kBN + x;
    if (n < a.D) a.P[(int64_t)tm * a.D + n] = cols_lds[x] + cols_lds[kBN + x];
    __syncthreads();   // the next tile's first stage overwrites the LDS
}

template <typename GT>
__global__ __launch_bounds__(kThreads) void ember_lmhead_grad(Params a) {
    __shared__ __attribute__((aligned(16))) uint16_t lds[2][2][kOperandElems];   // [stage][operand]
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int wm = wave & 1, wn = wave >> 1;

    // copy slice: thread -> rows tid / 32 + 8 q, 16-byte column chunk tid % 32
    const int ld_row = tid >> 5, ld_chunk = tid & 31;
    // transpose-read base (elements) of this lane within a stage: token
    // 8 (lane / 32) + (lane % 16) / 4, column 16 ((lane / 16) % 2) + 4 (lane % 4)
    const int tr_base = (8 * (lane >> 5) + ((lane & 15) >> 2)) * kPitch + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    const int a_base = tr_base + wm * 128;
    const int b_base = tr_base + wn * 128;

    // one tile per block (a loop over tiles would keep per-lane epilogue
    // values live across the contraction); blocks of one XCD take consecutive
    // tiles of this launch's range
    const int64_t l = a.tile0 + (int64_t)(blockIdx.x % kXcds) * a.per_xcd + blockIdx.x / kXcds;
    if (l >= a.tile1) return;
    const int64_t nk = (a.T + kBK - 1) / kBK;
    {
        int tm, tn;
        tile_of(a, l, tm, tn);
        const int64_t v0 = (int64_t)tm * kBM;
        const int64_t d0 = (int64_t)tn * kBN;

        u32x4 sa[kLoads], sb[kLoads];
        auto gload = [&](int64_t kt) {
            const int64_t k0 = kt * kBK;
            const uint16_t* pa = a.dY + k0 * a.ldy + v0;
            const uint16_t* pb = a.H + k0 * a.ldh + d0;
            const __amdgpu_buffer_rsrc_t ra = rsrc(pa, ((a.T - k0) * a.ldy - v0) * 2);
            const __amdgpu_buffer_rsrc_t rb = rsrc(pb, ((a.T - k0) * a.ldh - d0) * 2);
#pragma unroll
            for (int q = 0; q < kLoads; ++q) {
                const int row = ld_row + 8 * q;
                sa[q] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                            ra, (int)((row * a.ldy + ld_chunk * 8) * 2), 0, 0));
                sb[q] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                            rb, (int)((row * a.ldh + ld_chunk * 8) * 2), 0, 0));
            }
        };
        auto lstore = [&](int stage) {
#pragma unroll
            for (int q = 0; q < kLoads; ++q) {
                const int off = (ld_row + 8 * q) * kPitch + ld_chunk * 8;
                *reinterpret_cast<u32x4*>(&lds[stage][0][off]) = sa[q];
                *reinterpret_cast<u32x4*>(&lds[stage][1][off]) = sb[q];
            }
        };

        f32x16 acc[4][4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int nt = 0; nt < 4; ++nt)
#pragma unroll
                for (int i = 0; i < 16; ++i) acc[mt][nt][i] = 0.0f;

        if (nk > 0) {
            gload(0);
            lstore(0);
        }
        if (nk > 1) gload(1);
        __syncthreads();
        for (int64_t kt = 0; kt < nk; ++kt) {
            const int st = (int)(kt & 1);
            const uint16_t* As = lds[st][0];
            const uint16_t* Bs = lds[st][1];
#pragma unroll
            for (int kk = 0; kk < kBK / 16; ++kk) {
                bf16x8 af[4], bfr[4];
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const int oa = a_base + kk * 16 * kPitch + t * 32;
                    const int ob = b_base + kk * 16 * kPitch + t * 32;
                    const i16x4 a_lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(As + oa));
                    const i16x4 a_hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(As + oa + 4 * kPitch));
                    const i16x4 b_lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(Bs + ob));
                    const i16x4 b_hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(Bs + ob + 4 * kPitch));
                    af[t] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(a_lo, a_hi, 0, 1, 2, 3, 4, 5, 6, 7));
                    bfr[t] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(b_lo, b_hi, 0, 1, 2, 3, 4, 5, 6, 7));
                }
#pragma unroll
                for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt)
                        acc[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mt], bfr[nt], acc[mt][nt], 0, 0, 0);
            }
            if (kt + 1 < nk) {
                lstore(st ^ 1);
                if (kt + 2 < nk) gload(kt + 2);
            }
            __syncthreads();
        }
        epilogue<GT>(a, tm, tn, acc, reinterpret_cast<uint8_t*>(&lds[0][0][0]));
    }
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
    p.group_m = EMBER_LMHEAD_GROUP_M;
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
