// Batched (several tokens per weight set) activation-sparse dReLU FFN for
// gfx950, on the matrix cores (v_mfma_f32_16x16x32_bf16), bf16 weights.
//
// With a batch, a weight row is needed when ANY token needs it: W_up rows
// for the union over tokens of the open gates, W_down_t rows for the union
// of the non-zero Combined activations (Eq. drelu of Turbo Sparse, arXiv
// 2406.05955; zero activations contribute nothing, section 6.2).  Each such
// row is read once for the whole batch and contracted with all tokens at
// once; tokens for which the row is inactive get exact zeros (their gate or
// up is not positive, so their Combined value is 0).
//
// A group is one weight set and the tokens routed to it: the FFN has one
// group, the MoE layer one per expert (tokens listed on the device by
// bx_dispatch, ascending).  Kernels:
//   bx_dispatch  routing table -> per-group token lists and slots
//   bx_prep      x of each group's tokens split into bf16 high and low parts
//                (x = hi + lo to 16 significant bits, so the bf16 products
//                keep fp32-level accuracy)
//   bx_gate_up   per 32-neuron tile (4 waves, each a quarter of the hidden
//                dimension): gate MFMA for all tokens, union of open gates,
//                up MFMA over the union rows only, Combined, union of
//                non-zero Combined (the tile's active rows and their values)
//   bx_down      per (tile chunk, 256-column slice): active W_down_t rows
//                staged through LDS in transposed order (the neuron index is
//                the contraction axis but the slow axis of the row-major
//                matrix), MFMA with Combined as the other operand
//   bx_reduce    sums the chunk partials in a fixed order, applies routing
//                weights; deterministic
//   bx_stats     optional activity report from the per-tile bit masks
// With `dense` set every row joins both unions: the dense comparator, which
// reads all three matrices once for the whole batch.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "ts_batch.h"
#include "ts_device.h"
#include "ts_plan.h"
#include "ts_runtime.h"
#include "turbosparse.h"

namespace ts {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x4 mfma_bf16(const u32x4 a, const u32x4 b, const f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
}

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t bf16_bits(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ void split_hi_lo(float x, uint32_t &hi, uint32_t &lo) {
    hi = bf16_bits(x);
    lo = bf16_bits(x - __uint_as_float(hi << 16));
}

struct BxArgs {
    const float *x;          // [tokens][H] (already offset to the pass's first token)
    const void *wg, *wu, *wd;
    size_t expert_stride;    // elements per expert matrix (0: one weight set)
    int B, H, I, G, K, bpad, nt, hpad, ntiles, nslices, nchunks, tpc;
    const int32_t *topk;     // [B][K] routed experts, or null (FFN)
    const float *topw;       // [B][K] routing weights, or null
    int32_t *gcount;         // [G]
    int32_t *gtok;           // [G][bpad] token of each slot, -1 past the count
    int32_t *tslot;          // [B][K][2] (group, slot) of each routed token
    uint16_t *xhl;           // [G][2][bpad][hpad]
    int32_t *cnt;            // [G][ntiles][2] |union G|, |union A|
    int32_t *aseg;           // [G][ntiles][32] union-active rows (global index)
    float *hseg;             // [G][ntiles][32][bpad] Combined per token
    uint32_t *gmask;         // [G][ntiles][bpad] open-gate rows of the tile per token
    uint32_t *amask;         // [G][ntiles][bpad] active rows of the tile per token
    float *partial;          // [G][bpad][nchunks][H]
    float *out;              // [tokens][H]
    int want_masks;
    int dense;               // 1: every row is taken (the dense comparator)
};

// ---------------------------------------------------------------------------
// Routing table -> groups.  One wave; (token, rank) pairs are taken in
// token-major order, so each expert's token list comes out ascending.
__global__ __launch_bounds__(64) void bx_dispatch(BxArgs a) {
    __shared__ int s_base[kMaxExperts];
    const int lane = threadIdx.x;
    if (!a.topk) {
        for (int s = lane; s < a.bpad; s += 64) a.gtok[s] = s < a.B ? s : -1;
        for (int t = lane; t < a.B; t += 64) {
            a.tslot[t * 2] = 0;
            a.tslot[t * 2 + 1] = t;
        }
        if (lane == 0) a.gcount[0] = a.B;
        return;
    }
    for (int e = lane; e < a.G; e += 64) s_base[e] = 0;
    for (int i = lane; i < a.G * a.bpad; i += 64) a.gtok[i] = -1;
    __syncthreads();
    const int np = a.B * a.K;
    for (int p0 = 0; p0 < np; p0 += 64) {
        const int p = p0 + lane;
        const int e = p < np ? a.topk[p] : -1;
        for (int ex = 0; ex < a.G; ++ex) {
            const uint64_t m = __ballot(e == ex);
            if (m == 0) continue;
            const int base = s_base[ex];
            if (e == ex) {
                const int rank = base + lane_prefix(m, lane);
                a.gtok[ex * a.bpad + rank] = p / a.K;
                a.tslot[p * 2] = ex;
                a.tslot[p * 2 + 1] = rank;
            }
            __syncthreads();  // one wave: orders the read of s_base before the update
            if (lane == 0) s_base[ex] = base + __popcll(m);
            __syncthreads();
        }
    }
    for (int e = lane; e < a.G; e += 64) a.gcount[e] = s_base[e];
}

// x rows of each group's slots, split into bf16 high / low parts, zero past
// the token count and past H (to hpad).  One block per (group, slot).
__global__ __launch_bounds__(256) void bx_prep(BxArgs a) {
    const int g = blockIdx.x / a.bpad;
    const int s = blockIdx.x % a.bpad;
    const int t = a.gtok[g * a.bpad + s];
    uint16_t *hi = a.xhl + ((size_t)(g * 2) * a.bpad + s) * a.hpad;
    uint16_t *lo = a.xhl + ((size_t)(g * 2 + 1) * a.bpad + s) * a.hpad;
    for (int k = threadIdx.x; k < a.hpad; k += 256) {
        const float v = (t >= 0 && k < a.H) ? a.x[(size_t)t * a.H + k] : 0.f;
        uint32_t h, l;
        split_hi_lo(v, h, l);
        hi[k] = (uint16_t)h;
        lo[k] = (uint16_t)l;
    }
}

// ---------------------------------------------------------------------------
// K loop of the gate / up contraction for MT 16-row m-tiles (rows given per
// lane) and NT 16-token n-tiles, over 64-wide K blocks [kb0, kb1).  A K block
// reads 128 contiguous bytes of each row: lane (lm, lq) takes 16 bytes at
// 8*lq and at 32 + 8*lq, the x fragments use the same K positions, so each
// MFMA pairs matching K indices.  Weight chunks past H re-read the row's last
// chunk; x is zero there.
template <int MT, int NT>
__device__ __forceinline__ void bx_kloop(const uint16_t *const (&rows)[MT], int H, const uint16_t *__restrict__ xh,
                                         const uint16_t *__restrict__ xl, int hpad, int kb0, int kb1, int lm, int lq,
                                         f32x4 (&acc)[MT][NT]) {
    constexpr int U = NT <= 2 ? 2 : 1;  // K blocks per batch of loads
    for (int kb = kb0; kb < kb1; kb += U) {
        u32x4 w[U][MT][2], bh[U][NT][2], bl[U][NT][2];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kk = (kb + u < kb1 ? kb + u : kb) * 64;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int k = kk + 32 * h + 8 * lq;
                const int kw = k < H ? k : H - 8;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) w[u][mt][h] = ld_stream(rows[mt] + kw);
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) {
                    const size_t xo = (size_t)(16 * nt + lm) * hpad + k;
                    bh[u][nt][h] = ld_cached(xh + xo);
                    bl[u][nt][h] = ld_cached(xl + xo);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (kb + u < kb1) {
#pragma unroll
                for (int h = 0; h < 2; ++h)
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                        for (int nt = 0; nt < NT; ++nt) {
                            acc[mt][nt] = mfma_bf16(w[u][mt][h], bh[u][nt][h], acc[mt][nt]);
                            acc[mt][nt] = mfma_bf16(w[u][mt][h], bl[u][nt][h], acc[mt][nt]);
                        }
            }
        }
    }
}

// Sum the four waves' K-quarter accumulators (fixed order); every wave gets
// the totals for its own lane positions.
template <int NT>
__device__ __forceinline__ void bx_combine(f32x4 (&acc)[2][NT], f32x4 (*s_red)[2][NT][64], int wave, int lane) {
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) s_red[wave][mt][nt][lane] = acc[mt][nt];
    __syncthreads();
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
            acc[mt][nt] = (s_red[0][mt][nt][lane] + s_red[1][mt][nt][lane]) +
                          (s_red[2][mt][nt][lane] + s_red[3][mt][nt][lane]);
    __syncthreads();
}

// Bit j (j < 32) set where row j of the tile has pred true for some token:
// lane (lm, lq), register i, m-tile mt holds row 16*mt + 4*lq + i.
template <int NT>
__device__ __forceinline__ uint32_t bx_any_rows(const bool (&pred)[2][NT][4]) {
    uint32_t bits = 0;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            uint64_t m = 0;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) m |= __ballot(pred[mt][nt][i]);
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if ((m >> (16 * q)) & 0xFFFFull) bits |= 1u << (16 * mt + 4 * q + i);
        }
    return bits;
}

// Per token (lane lm of n-tile nt) the 32-bit mask of rows with pred true,
// rows mapped through rowbit (tile-local row of union index j).
template <int NT>
__device__ __forceinline__ void bx_token_masks(const bool (&pred)[2][NT][4], const int (&rowbit)[2][4], int lq,
                                               uint32_t (&tm)[NT]) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        uint32_t m = 0;
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (pred[mt][nt][i]) m |= 1u << rowbit[mt][i];
        m |= (uint32_t)__shfl_xor((int)m, 16, 64);
        m |= (uint32_t)__shfl_xor((int)m, 32, 64);
        tm[nt] = m;
    }
    (void)lq;
}

__device__ __forceinline__ int nth_set_bit(uint32_t m, int n) {
    for (int b = 0; b < 32; ++b) {
        if ((m >> b) & 1u) {
            if (n == 0) return b;
            --n;
        }
    }
    return 0;
}

template <int NT>
__global__ __launch_bounds__(256) void bx_gate_up(BxArgs a) {
    __shared__ f32x4 s_red[4][2][NT][64];
    __shared__ float s_g[kBxRows][NT * 16];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lm = lane & 15, lq = lane >> 4;
    const int g = blockIdx.x / a.ntiles;
    const int tile = blockIdx.x % a.ntiles;
    const size_t tix = (size_t)g * a.ntiles + tile;
    const int ng = a.gcount[g];
    if (ng == 0) {
        if (tid == 0) {
            a.cnt[tix * 2] = 0;
            a.cnt[tix * 2 + 1] = 0;
        }
        if (a.want_masks)
            for (int s = tid; s < a.bpad; s += 256) {
                a.gmask[tix * a.bpad + s] = 0;
                a.amask[tix * a.bpad + s] = 0;
            }
        return;
    }
    const int r0 = tile * kBxRows;
    const uint16_t *wg = reinterpret_cast<const uint16_t *>(a.wg) + (size_t)g * a.expert_stride;
    const uint16_t *wu = reinterpret_cast<const uint16_t *>(a.wu) + (size_t)g * a.expert_stride;
    const uint16_t *xh = a.xhl + (size_t)(g * 2) * a.bpad * a.hpad;
    const uint16_t *xl = a.xhl + (size_t)(g * 2 + 1) * a.bpad * a.hpad;
    const int nkb = a.hpad / 64;
    const int kb0 = wave * nkb / 4, kb1 = (wave + 1) * nkb / 4;

    // ---- gate: 32 rows x all tokens --------------------------------------
    f32x4 acc[2][NT];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    {
        const uint16_t *rows[2];
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) rows[mt] = wg + (size_t)min(r0 + 16 * mt + lm, a.I - 1) * a.H;
        bx_kloop<2, NT>(rows, a.H, xh, xl, a.hpad, kb0, kb1, lm, lq, acc);
    }
    bx_combine<NT>(acc, s_red, wave, lane);

    bool open[2][NT][4];
    int rowbit[2][4];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = 16 * mt + 4 * lq + i;
            rowbit[mt][i] = r;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                open[mt][nt][i] = r0 + r < a.I && (a.dense || acc[mt][nt][i] > 0.f);
                if (wave == 0) s_g[r][16 * nt + lm] = acc[mt][nt][i];
            }
        }
    const uint32_t umask = bx_any_rows<NT>(open);
    const int nu = __popc(umask);
    if (a.want_masks) {
        uint32_t tm[NT];
        bx_token_masks<NT>(open, rowbit, lq, tm);
        if (wave == 0 && lq == 0)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) a.gmask[tix * a.bpad + 16 * nt + lm] = tm[nt];
    }
    __syncthreads();  // s_g complete

    // ---- up: the union rows, gathered ------------------------------------
    f32x4 uacc[2][NT];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) uacc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    int urow[2];  // tile-local row of union index 16*mt + lm (lanes past nu repeat the first)
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
        const int j = 16 * mt + lm;
        urow[mt] = nth_set_bit(umask, j < nu ? j : 0);
    }
    if (nu > 16) {
        const uint16_t *rows[2] = {wu + (size_t)(r0 + urow[0]) * a.H, wu + (size_t)(r0 + urow[1]) * a.H};
        bx_kloop<2, NT>(rows, a.H, xh, xl, a.hpad, kb0, kb1, lm, lq, uacc);
    } else if (nu > 0) {
        const uint16_t *rows[1] = {wu + (size_t)(r0 + urow[0]) * a.H};
        f32x4 u1[1][NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) u1[0][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        bx_kloop<1, NT>(rows, a.H, xh, xl, a.hpad, kb0, kb1, lm, lq, u1);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) uacc[0][nt] = u1[0][nt];
    }
    bx_combine<NT>(uacc, s_red, wave, lane);

    // ---- Combined for union index j = 16*mt + 4*lq + i, token 16*nt + lm ----
    bool act[2][NT][4];
    float hv[2][NT][4];
    int ubit[2][4];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int j = 16 * mt + 4 * lq + i;
            const int r = nth_set_bit(umask, j < nu ? j : 0);
            ubit[mt][i] = r;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const float gv = s_g[r][16 * nt + lm];
                const float uv = uacc[mt][nt][i];
                const bool on = j < nu && gv > 0.f && uv > 0.f;
                act[mt][nt][i] = on || (a.dense && j < nu);
                hv[mt][nt][i] = on ? gv * uv : 0.f;
            }
        }
    const uint32_t amask_u = bx_any_rows<NT>(act);  // over union indices
    const int na = __popc(amask_u);
    if (a.want_masks) {
        uint32_t tm[NT];
        bx_token_masks<NT>(act, ubit, lq, tm);
        if (wave == 0 && lq == 0)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) a.amask[tix * a.bpad + 16 * nt + lm] = tm[nt];
    }
    if (wave == 0) {
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int j = 16 * mt + 4 * lq + i;
                if ((amask_u >> j) & 1u) {
                    const int rank = __popc(amask_u & ((1u << j) - 1u));
                    float *hrow = a.hseg + (tix * kBxRows + rank) * a.bpad;
#pragma unroll
                    for (int nt = 0; nt < NT; ++nt) hrow[16 * nt + lm] = hv[mt][nt][i];
                    if (lm == 0) a.aseg[tix * kBxRows + rank] = r0 + ubit[mt][i];
                }
            }
        if (lane == 0) {
            a.cnt[tix * 2] = nu;
            a.cnt[tix * 2 + 1] = na;
        }
    }
}

// ---------------------------------------------------------------------------
// Down: workgroup (group, chunk of tiles, 256-column slice), 4 waves.  The
// chunk's active rows are processed in K blocks of 32 rows: each block's
// W_down_t[row][slice] (16 KB) and Combined[row][tokens] are loaded with
// coalesced 16-byte loads, written to LDS transposed (column-major W,
// token-major Combined split into bf16 high / low parts), and contracted:
// wave w owns columns 64w..64w+63 (4 n-tiles), all token m-tiles.  The next
// block's loads are in flight while the current block is contracted.

constexpr int kBxPadRows = kBxBlockRows + 8;  // LDS row stride in the transposed tiles

template <int NT>
__global__ __launch_bounds__(256) void bx_down(BxArgs a) {
    constexpr int TOK = NT * 16;
    constexpr int HQ = (kBxBlockRows * TOK / 4 + 255) / 256;  // Combined float4 per thread per block
    __shared__ int s_row[kDownMaxRows];
    __shared__ int s_hidx[kDownMaxRows];
    __shared__ int s_cnt[kDownMaxTiles + 1];
    __shared__ uint16_t sW[2][kBxSliceCols][kBxPadRows];
    __shared__ uint16_t sH[2][2][TOK][kBxPadRows];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lm = lane & 15, lq = lane >> 4;
    const int slice = blockIdx.x % a.nslices;
    const int chunk = (blockIdx.x / a.nslices) % a.nchunks;
    const int g = blockIdx.x / (a.nslices * a.nchunks);
    const int ng = a.gcount[g];
    if (ng == 0) return;
    const int H = a.H;
    const int t0 = chunk * a.tpc;
    const int ntc = min(a.tpc, a.ntiles - t0);
    const size_t tbase = (size_t)g * a.ntiles + t0;

    // 1. rows of the chunk (ascending tiles, ascending within a tile)
    for (int t = tid; t < ntc; t += 256) s_cnt[t] = a.cnt[(tbase + t) * 2 + 1];
    __syncthreads();
    if (tid == 0) {
        int off = 0;
        for (int t = 0; t < ntc; ++t) {
            const int c = s_cnt[t];
            s_cnt[t] = off;
            off += c;
        }
        s_cnt[ntc] = off;
    }
    __syncthreads();
    for (int e = tid; e < ntc * kBxRows; e += 256) {
        const int t = e / kBxRows, q = e % kBxRows;
        if (q < s_cnt[t + 1] - s_cnt[t]) {
            s_row[s_cnt[t] + q] = a.aseg[(tbase + t) * kBxRows + q];
            s_hidx[s_cnt[t] + q] = (int)((tbase + t) * kBxRows + q);
        }
    }
    __syncthreads();
    const int nrows = s_cnt[ntc];
    const int nblk = (nrows + kBxBlockRows - 1) / kBxBlockRows;

    const uint16_t *wd = reinterpret_cast<const uint16_t *>(a.wd) + (size_t)g * a.expert_stride;
    const int col0 = slice * kBxSliceCols;

    // per-thread share of a block: 4 W chunks (row = item / 32, 8 columns at
    // 8 * (item % 32)) and HQ Combined float4 (row = q / (TOK/4), tokens 4x)
    u32x4 wv[4];
    f32x4 hq[HQ];
    auto load_block = [&](int blk) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int item = tid + 256 * j;
            const int r = blk * kBxBlockRows + item / 32;
            const int row = s_row[r < nrows ? r : 0];
            int c = col0 + 8 * (item % 32);
            c = c < H ? c : H - 8;
            wv[j] = ld_stream(wd + (size_t)row * H + c);
        }
#pragma unroll
        for (int j = 0; j < HQ; ++j) {
            const int q = tid + 256 * j;
            const int rl = q / (TOK / 4);
            const int r = blk * kBxBlockRows + rl;
            const bool ok = rl < kBxBlockRows && r < nrows;
            const f32x4 v = *reinterpret_cast<const f32x4 *>(a.hseg + (size_t)s_hidx[ok ? r : 0] * a.bpad +
                                                             4 * (q % (TOK / 4)));
            hq[j] = ok ? v : f32x4{0.f, 0.f, 0.f, 0.f};
        }
    };
    auto store_block = [&](int buf) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int item = tid + 256 * j;
            const int rl = item / 32, cb = 8 * (item % 32);
            const uint32_t w4[4] = {wv[j].x, wv[j].y, wv[j].z, wv[j].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                sW[buf][cb + 2 * e][rl] = (uint16_t)(w4[e] & 0xFFFFu);
                sW[buf][cb + 2 * e + 1][rl] = (uint16_t)(w4[e] >> 16);
            }
        }
#pragma unroll
        for (int j = 0; j < HQ; ++j) {
            const int q = tid + 256 * j;
            const int rl = q / (TOK / 4);
            if (rl < kBxBlockRows) {
                const int tk = 4 * (q % (TOK / 4));
                const float v4[4] = {hq[j].x, hq[j].y, hq[j].z, hq[j].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    uint32_t hi, lo;
                    split_hi_lo(v4[e], hi, lo);
                    sH[buf][0][tk + e][rl] = (uint16_t)hi;
                    sH[buf][1][tk + e][rl] = (uint16_t)lo;
                }
            }
        }
    };

    f32x4 acc[NT][4];
#pragma unroll
    for (int mt = 0; mt < NT; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[mt][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    if (nblk > 0) {
        load_block(0);
        store_block(0);
    }
    __syncthreads();
    for (int blk = 0; blk < nblk; ++blk) {
        const int buf = blk & 1;
        if (blk + 1 < nblk) load_block(blk + 1);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = 64 * wave + 16 * j + lm;
            const u32x4 bw = *reinterpret_cast<const u32x4 *>(&sW[buf][col][8 * lq]);
#pragma unroll
            for (int mt = 0; mt < NT; ++mt) {
                const u32x4 ah = *reinterpret_cast<const u32x4 *>(&sH[buf][0][16 * mt + lm][8 * lq]);
                const u32x4 al = *reinterpret_cast<const u32x4 *>(&sH[buf][1][16 * mt + lm][8 * lq]);
                acc[mt][j] = mfma_bf16(ah, bw, acc[mt][j]);
                acc[mt][j] = mfma_bf16(al, bw, acc[mt][j]);
            }
        }
        if (blk + 1 < nblk) store_block(buf ^ 1);
        __syncthreads();
    }

    // D[m = token 16*mt + 4*lq + i][n = column 64*wave + 16*j + lm]
#pragma unroll
    for (int mt = 0; mt < NT; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = col0 + 64 * wave + 16 * j + lm;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int tok = 16 * mt + 4 * lq + i;
                if (tok < ng && col < H)
                    a.partial[(((size_t)g * a.bpad + tok) * a.nchunks + chunk) * H + col] = acc[mt][j][i];
            }
        }
}

// out[t][:] = sum over routed ranks k (ascending) of w[t][k] times the sum
// over chunks (ascending within each thread's share) of the partial row of
// (group, slot) = tslot[t][k].  Block: 16 columns x 64 shares, fixed LDS tree.
__global__ __launch_bounds__(256) void bx_reduce(BxArgs a) {
    __shared__ f32x4 red[64][4];
    const int t = blockIdx.y;
    const int q = threadIdx.x & 3;
    const int grp = threadIdx.x >> 2;
    const int c4 = blockIdx.x * 4 + q;
    const int nq = a.H / 4;
    const int total = a.K * a.nchunks;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int p = grp; p < total; p += 64) {
        const int k = p / a.nchunks, c = p % a.nchunks;
        const int g = a.tslot[(t * a.K + k) * 2], s = a.tslot[(t * a.K + k) * 2 + 1];
        const float w = a.topw ? a.topw[t * a.K + k] : 1.f;
        const f32x4 v = ld_f32x4_masked(a.partial + (((size_t)g * a.bpad + s) * a.nchunks + c) * a.H, c4, nq);
        acc.x = fmaf(w, v.x, acc.x);
        acc.y = fmaf(w, v.y, acc.y);
        acc.z = fmaf(w, v.z, acc.z);
        acc.w = fmaf(w, v.w, acc.w);
    }
    red[grp][q] = acc;
    __syncthreads();
    for (int st = 32; st >= 1; st >>= 1) {
        if (grp < st) red[grp][q] += red[grp + st][q];
        __syncthreads();
    }
    if (grp == 0 && c4 < nq) *reinterpret_cast<f32x4 *>(a.out + (size_t)t * a.H + c4 * 4) = red[0][q];
}

// Activity report from the per-tile masks: one block per (token, rank).
__global__ __launch_bounds__(256) void bx_stats(BxArgs a, int32_t *n_gate, int32_t *n_active, int32_t *gate_idx,
                                                int32_t *active_idx, int inter, int out_base) {
    __shared__ int s_sc[2][256];
    const int p = blockIdx.x;  // t * K + k
    const int g = a.tslot[p * 2], s = a.tslot[p * 2 + 1];
    const int tid = threadIdx.x;
    const size_t o = (size_t)(out_base + p);
    int cg = 0, ca = 0;
    for (int base = 0; base < a.ntiles; base += 256) {
        const int tile = base + tid;
        const size_t ti = (size_t)g * a.ntiles + tile;
        const uint32_t gm = tile < a.ntiles ? a.gmask[ti * a.bpad + s] : 0u;
        const uint32_t am = tile < a.ntiles ? a.amask[ti * a.bpad + s] : 0u;
        const int ng = __popc(gm), na = __popc(am);
        s_sc[0][tid] = ng;
        s_sc[1][tid] = na;
        __syncthreads();
        for (int off = 1; off < 256; off <<= 1) {
            const int vg = tid >= off ? s_sc[0][tid - off] : 0;
            const int va = tid >= off ? s_sc[1][tid - off] : 0;
            __syncthreads();
            s_sc[0][tid] += vg;
            s_sc[1][tid] += va;
            __syncthreads();
        }
        int og = cg + s_sc[0][tid] - ng, oa = ca + s_sc[1][tid] - na;
        for (int b = 0; b < 32; ++b) {
            if ((gm >> b) & 1u) {
                if (gate_idx) gate_idx[o * inter + og] = tile * kBxRows + b;
                ++og;
            }
            if ((am >> b) & 1u) {
                if (active_idx) active_idx[o * inter + oa] = tile * kBxRows + b;
                ++oa;
            }
        }
        cg += s_sc[0][255];
        ca += s_sc[1][255];
        __syncthreads();
    }
    if (tid == 0) {
        if (n_gate) n_gate[o] = cg;
        if (n_active) n_active[o] = ca;
    }
}

__global__ __launch_bounds__(256) void bx_union(BxArgs a, int32_t *n_union) {
    __shared__ int s[2][256];
    int u = 0, v = 0;
    for (int i = threadIdx.x; i < a.G * a.ntiles; i += 256) {
        u += a.cnt[(size_t)i * 2];
        v += a.cnt[(size_t)i * 2 + 1];
    }
    s[0][threadIdx.x] = u;
    s[1][threadIdx.x] = v;
    __syncthreads();
    for (int st = 128; st >= 1; st >>= 1) {
        if ((int)threadIdx.x < st) {
            s[0][threadIdx.x] += s[0][threadIdx.x + st];
            s[1][threadIdx.x] += s[1][threadIdx.x + st];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        n_union[0] = s[0][0];
        n_union[1] = s[1][0];
    }
}

// ---------------------------------------------------------------------------

namespace {

template <typename T>
T *ws_at(void *ws, size_t off) {
    return reinterpret_cast<T *>(static_cast<char *>(ws) + off);
}

template <int NT>
void launch_nt(const BatchPlan &p, const BxArgs &a, hipStream_t st) {
    launch("batch_gate_up", bx_gate_up<NT>, dim3((unsigned)(p.groups * p.ntiles)), dim3(256), st, a);
    launch("batch_down", bx_down<NT>, dim3((unsigned)(p.groups * p.nchunks * p.nslices)), dim3(256), st, a);
}

}  // namespace

// One pass of the batched path for up to kBxMaxTokens tokens.  x and out are
// offset to the pass's first token; topk / topw (MoE) are [batch][K] for the
// pass's tokens.  Stats arrays are indexed from stats_base.
ts_status run_batch(const float *x, const void *wg, const void *wu, const void *wd, size_t expert_stride,
                    const int32_t *topk, const float *topw, const BatchPlan &p, float *out,
                    const ts_ffn_stats *stats, int stats_base, void *ws, hipStream_t st, bool dense) {
    BxArgs a;
    a.dense = dense ? 1 : 0;
    a.x = x;
    a.wg = wg;
    a.wu = wu;
    a.wd = wd;
    a.expert_stride = expert_stride;
    a.B = p.batch;
    a.H = p.hidden;
    a.I = p.inter;
    a.G = p.groups;
    a.K = p.top_k;
    a.bpad = p.bpad;
    a.nt = p.nt;
    a.hpad = p.hpad;
    a.ntiles = p.ntiles;
    a.nslices = p.nslices;
    a.nchunks = p.nchunks;
    a.tpc = p.tpc;
    a.topk = topk;
    a.topw = topw;
    a.gcount = ws_at<int32_t>(ws, p.off_gcount);
    a.gtok = ws_at<int32_t>(ws, p.off_gtok);
    a.tslot = ws_at<int32_t>(ws, p.off_tslot);
    a.xhl = ws_at<uint16_t>(ws, p.off_xhl);
    a.cnt = ws_at<int32_t>(ws, p.off_cnt);
    a.aseg = ws_at<int32_t>(ws, p.off_aseg);
    a.hseg = ws_at<float>(ws, p.off_hseg);
    a.gmask = ws_at<uint32_t>(ws, p.off_gmask);
    a.amask = ws_at<uint32_t>(ws, p.off_amask);
    a.partial = ws_at<float>(ws, p.off_partial);
    a.out = out;
    const bool want_lists = stats && (stats->n_gate || stats->n_active || stats->gate_idx || stats->active_idx);
    a.want_masks = want_lists ? 1 : 0;

    launch("batch_dispatch", bx_dispatch, dim3(1), dim3(64), st, a);
    launch("batch_prep", bx_prep, dim3((unsigned)(p.groups * p.bpad)), dim3(256), st, a);
    switch (p.nt) {
    case 1: launch_nt<1>(p, a, st); break;
    case 2: launch_nt<2>(p, a, st); break;
    default: launch_nt<4>(p, a, st); break;
    }
    launch("batch_reduce", bx_reduce, dim3((unsigned)((p.hidden / 4 + 3) / 4), (unsigned)p.batch), dim3(256), st, a);
    ts_status s = check_launch("batch path");
    if (s != TS_OK) return s;
    if (want_lists) {
        launch("batch_stats", bx_stats, dim3((unsigned)(p.batch * p.top_k)), dim3(256), st, a, stats->n_gate,
               stats->n_active, stats->gate_idx, stats->active_idx, p.inter, stats_base);
        s = check_launch("batch_stats");
        if (s != TS_OK) return s;
    }
    if (stats && stats->n_union) {
        launch("batch_stats", bx_union, dim3(1), dim3(256), st, a, stats->n_union);
        s = check_launch("batch_union");
        if (s != TS_OK) return s;
    }
    return TS_OK;
}

}  // namespace ts
