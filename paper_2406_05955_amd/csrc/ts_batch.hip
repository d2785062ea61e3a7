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
// bx_prep, ascending).  x and Combined enter the matrix cores as two bf16
// parts (v = hi + lo to 16 significant bits), so the products keep fp32-level
// accuracy; with at most 8 token slots both parts share one 16-column MFMA
// tile (columns 0-7 high, 8-15 low) and are added at the end.  Kernels:
//   bx_prep      routing table -> per-group token lists (MoE), and x of each
//                group's tokens split into bf16 high and low parts (the
//                batched FFN; in the MoE layer the router writes every
//                token's split once, and bx_gate_up lists its group's tokens
//                and gathers their columns itself)
//   bx_gate_up   per 32-neuron tile, 4 waves each a quarter of the hidden
//                dimension with its own pipelined loads (no barrier inside
//                the K loop): gate for all tokens, union of open gates, up
//                over the union rows only (gathered), Combined, the tile's
//                active rows as 32 slots and their Combined values as MFMA
//                operand fragments
//   bx_down      per (tile chunk, 128-column slice): 4 waves split the
//                chunk's non-empty tiles; each wave stages a tile's active
//                W_down_t rows in its own LDS region (row-major, XOR-swizzled
//                16-byte chunks) and reads them back column-wise as the MFMA
//                operand (the neuron index is the contraction axis but the
//                slow axis of the row-major matrix); the 4 waves' sums are
//                added in a fixed order at the end
//   bx_reduce    sums the chunk partials in a fixed order, applies routing
//                weights; deterministic
//   bx_stats     optional activity report from the per-tile bit masks
// With `dense` set every row joins both unions: the dense comparator, which
// reads all three matrices once for the whole batch.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "ts_batch.h"
#include "ts_device.h"
#include "ts_plan.h"
#include "ts_runtime.h"
#include "turbosparse.h"

namespace ts {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x4 mfma_bf16(const u32x4 a, const u32x4 b, const f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
}

// Shape constants per token-slot count TOK (8, 16, 32, 64).
template <int TOK>
struct Bx {
    static constexpr bool PACK = TOK == 8;          // high and low parts share one 16-column tile
    static constexpr int NT = PACK ? 1 : TOK / 16;  // 16-token accumulator tiles
    static constexpr int NX = PACK ? 1 : 2 * NT;    // operand fragments per 32-wide k-step (x or Combined)
    // k-steps per batch of gate / up loads (default; measured: 2 at 8 token
    // slots, 4 at 16, 2 past that, where deeper rings spill)
    static constexpr int KS = PACK ? 2 : (NX <= 2 ? 4 : 2);
    static constexpr int D = 2;                     // gate / up batches in flight per wave (default)
    static constexpr int DD = 2;                    // down blocks in flight per wave (default)
};

struct BxArgs {
    const float *x;          // [tokens][H] (already offset to the pass's first token)
    const void *wg, *wu, *wd;
    size_t expert_stride;    // elements per expert matrix (0: one weight set)
    int B, H, I, G, K, bpad, hpad, ntiles, nslices, nchunks, tpc;
    int vpe;                 // groups per weight set: group g uses weight set g / vpe
    const int32_t *topk;     // [B][K] routed experts, or null (FFN)
    const float *topw;       // [B][K] routing weights, or null
    int32_t *gcount;         // [G]
    int32_t *tslot;          // [B][K][2] (group, slot) of each routed token
    uint16_t *xhl;           // x fragments [G][hpad / 32][NX][64 lanes][8] bf16 (MFMA operand order)
    int32_t *cnt;            // [G][ntiles][2] |union G|, |union A|
    uint8_t *arow;           // [G][ntiles][32] row within the tile of each active slot (slot 0's past |union A|)
    uint16_t *hfrag;         // [G][ntiles][32 slots][2][bpad] Combined per active slot, bf16 high / low
    uint32_t *gmask;         // [G][ntiles][bpad] open-gate rows of the tile per token
    uint32_t *amask;         // [G][ntiles][bpad] active rows of the tile per token
    float *partial;          // [G][bpad][nchunks][H]
    float *out;              // [tokens][H]
    int want_masks;
    int dense;               // 1: every row is taken (the dense comparator)
    const uint16_t *xtok;    // or null: every token's x as bf16 high / low parts, token-major (the MoE
                             // router's split: per token xchunks chunks of 8 values, 32 bytes each)
    int xchunks;
};

// x operand source of the gate / up K loop: the per-group fragments built by
// bx_prep (frag), or (GATHER) this lane's columns gathered from the
// token-major split, off[f] = the byte offset of fragment f's column at
// k-step 0 (past the resource for an empty slot: zeros).
template <int NX>
struct BxX {
    const u32x4 *frag;
    __amdgpu_buffer_rsrc_t rs;
    uint32_t off[NX];
};

// The gate / up kernels' x source for group g: lane (lm, lq) of fragment f
// holds column lm = (part, slot) as bx_prep lays it out; gathered from the
// token-major split when the router wrote one (a.xtok), each column at
// 16 bytes of its token's 32-byte chunk 4 ks + lq (high part first).
template <int TOK, bool GATHER>
__device__ __forceinline__ BxX<Bx<TOK>::NX> bx_xsource(const BxArgs &a, int g, int lane, const int *s_tok) {
    using S = Bx<TOK>;
    constexpr int NX = S::NX;
    const int lm = lane & 15, lq = lane >> 4;
    BxX<NX> xs;
    xs.frag = reinterpret_cast<const u32x4 *>(a.xhl) + (size_t)g * (a.hpad / 32) * NX * 64;
    if constexpr (GATHER) {
        const uint32_t rowb = (uint32_t)a.xchunks * 32u;
        xs.rs = make_rsrc(a.xtok, (uint32_t)a.B * rowb);
#pragma unroll
        for (int f = 0; f < NX; ++f) {
            const int hl = S::PACK ? (lm >> 3) : (f & 1);
            const int slot = S::PACK ? (lm & 7) : 16 * (f >> 1) + lm;
            const int tk = s_tok[slot];
            xs.off[f] = tk >= 0 ? (uint32_t)tk * rowb + 32u * (uint32_t)lq + 16u * (uint32_t)hl : kOutOfRange;
        }
    } else {
        xs.rs = make_rsrc(a.xhl, 0u);
#pragma unroll
        for (int f = 0; f < NX; ++f) xs.off[f] = kOutOfRange;
    }
    return xs;
}

// Group g's token list (MoE): the tokens routed to expert g / vpe, entries
// [r0, r0 + TOK) of that expert's ascending list, by one wave scanning the
// (token, rank) pairs in token-major order; s_tok[slot] = token, -1 past the
// count.  With `tables`, also the group's token count and the (group, slot)
// of each of its routed pairs (for the reduce and the report).  Returns the
// count (on every lane).
template <int TOK>
__device__ __forceinline__ int bx_list_group(const BxArgs &a, int g, int lane, int *s_tok, bool tables) {
    const int np = a.B * a.K;
    const int e = g / a.vpe, r0 = (g - e * a.vpe) * TOK;
    int base = 0;
    for (int p0 = 0; p0 < np; p0 += 64) {
        const int p = p0 + lane;
        const bool mine = p < np && a.topk[p] == e;
        const uint64_t m = __ballot(mine);
        const int rank = base + lane_prefix(m, lane) - r0;  // rank within this group
        if (mine && rank >= 0 && rank < TOK) {
            s_tok[rank] = p / a.K;
            if (tables) {
                a.tslot[p * 2] = g;
                a.tslot[p * 2 + 1] = rank;
            }
        }
        base += __popcll(m);
    }
    const int n = min(max(base - r0, 0), TOK);
    for (int sl = n + lane; sl < TOK; sl += 64) s_tok[sl] = -1;
    if (tables && lane == 0) a.gcount[g] = n;
    return n;
}

// ---------------------------------------------------------------------------
// x of each group's token slots as MFMA operand fragments: for k-step ks (32
// wide) and fragment f, lane (lm, lq) holds the 8 values at k = 32 ks + 8 lq
// of column lm, column = (high or low part, token slot); fragments are 1 KB
// contiguous, so a wave loads one with a single fully coalesced instruction.
// Zero past the token count and past H (to hpad).  One thread per (group,
// k-step, fragment, lane); a block's 256 threads belong to one group (hpad /
// 32 k-steps per group is a multiple of 32).  Without a routing table (the
// FFN) the slots are the tokens themselves.  With one (the MoE layer), one
// wave of each block lists its group's tokens: the (token, rank) pairs are
// scanned in token-major order, so each expert's list comes out ascending.
// The group's first block also writes the group tables (token count, and
// the (group, slot) of each routed pair for the reduce and the report).
template <int TOK>
__global__ __launch_bounds__(256) void bx_prep(BxArgs a) {
    using S = Bx<TOK>;
    constexpr int NX = S::NX;
    __shared__ int s_tok[TOK];
    const int nks = a.hpad / 32;
    const int g = (blockIdx.x * 4) / (NX * nks);
    const bool first = blockIdx.x * 4 == g * NX * nks;
    if (a.topk) {
        if (threadIdx.x < 64) bx_list_group<TOK>(a, g, threadIdx.x, s_tok, first);
        __syncthreads();
    } else if (blockIdx.x == 0) {
        for (int t = threadIdx.x; t < a.B; t += 256) {
            a.tslot[t * 2] = 0;
            a.tslot[t * 2 + 1] = t;
        }
        if (threadIdx.x == 0) a.gcount[0] = a.B;
    }
    const int idx = blockIdx.x * 256 + threadIdx.x;
    if (idx >= a.G * nks * NX * 64) return;
    const int lane = idx & 63, lm = lane & 15, lq = lane >> 4;
    const int f = (idx >> 6) % NX;
    const int ks = (idx >> 6) / NX % nks;
    const int hl = S::PACK ? (lm >> 3) : (f & 1);
    const int slot = S::PACK ? (lm & 7) : 16 * (f >> 1) + lm;
    const int t = a.topk ? s_tok[slot] : (slot < a.B ? slot : -1);
    const int k0 = ks * 32 + 8 * lq;
    float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (t >= 0 && k0 < a.H) {  // H is a multiple of 8, so all 8 are in range
        const f32x4 *src = reinterpret_cast<const f32x4 *>(a.x + (size_t)t * a.H + k0);
        const f32x4 p = src[0], q = src[1];
        v[0] = p.x; v[1] = p.y; v[2] = p.z; v[3] = p.w;
        v[4] = q.x; v[5] = q.y; v[6] = q.z; v[7] = q.w;
    }
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        uint32_t h0, l0, h1, l1;
        split_hi_lo(v[2 * e], h0, l0);
        split_hi_lo(v[2 * e + 1], h1, l1);
        o[e] = hl ? (l0 | (l1 << 16)) : (h0 | (h1 << 16));
    }
    reinterpret_cast<u32x4 *>(a.xhl)[idx] = u32x4{o[0], o[1], o[2], o[3]};
}

// ---------------------------------------------------------------------------
// K loop of the gate / up contraction of one wave: MT 16-row m-tiles against
// the NX x fragments, over nbat batches of KS k-steps (32 wide) starting at
// k-step ks0.  A batch spans CPR = 4 KS 16-byte chunks of each of the 16 MT
// rows and is loaded RPI = 16 / KS rows per instruction (CPR lanes per row,
// so every instruction reads whole 128-byte lines: 256 or 128 contiguous
// bytes per row); wrow[j] is this lane's row for instruction j.  The chunks
// go to the wave's own LDS region, chunk c of row r at position
// swz(r, c), and come back as MFMA operands (lane (lm, lq) of k-step s:
// row 16 mt + lm, chunk 4 s + lq); the swizzle spreads both the writes and
// the 16 rows of a read over all banks.  x fragments are loaded directly
// (1 KB contiguous each).  The loads of the next D - 1 batches are in
// flight while a batch is contracted.  Chunks past H re-read the row's last
// chunk; x is zero there.
template <int KS>
__device__ __forceinline__ int bx_swz(int r, int c) {
    return KS == 4 ? (c ^ (r & 15)) : (c ^ ((r >> 1) & 7));
}

template <int TOK, int MT, int KS, int D, bool GATHER = false>
__device__ __forceinline__ void bx_kloop(const char *wbase, const uint32_t (&roff)[MT * KS], int H,
                                         const BxX<Bx<TOK>::NX> &xs, int ks0, int nbat, int lane, u32x4 *sw,
                                         f32x4 (&acc)[MT][Bx<TOK>::NT]) {
    using S = Bx<TOK>;
    constexpr int NX = S::NX, CPR = 4 * KS, RPI = 16 / KS, NI = MT * KS;
    // each wave's k-steps (hpad / 128, hpad a multiple of kBxKQuant) come in
    // batches of KS; the ring below needs their count to be a multiple of D
    static_assert((kBxKQuant / 128 / KS) % D == 0, "k-step batches per wave must be a multiple of D");
    const int lm = lane & 15, lq = lane >> 4;
    const int lc = lane % CPR, lr = lane / CPR;
    u32x4 w[D][NI], xv[D][NX][KS];
    // weights: uniform base + 32-bit per-lane byte offset (row * H * 2 + k * 2)
    auto issue = [&](int d, int b) {
        const int kb = (ks0 + b * KS) * 32;
        const int k = kb + 8 * lc;
        const uint32_t kw = 2u * (uint32_t)(k < H ? k : H - 8);
#pragma unroll
        for (int j = 0; j < NI; ++j) w[d][j] = ld_stream(wbase + (roff[j] + kw));
        if constexpr (GATHER) {
            // 128 bytes per token and k-step: the lane's 16 (its k-range, its part)
#pragma unroll
            for (int s = 0; s < KS; ++s)
#pragma unroll
                for (int f = 0; f < NX; ++f)
                    xv[d][f][s] = __builtin_amdgcn_raw_buffer_load_b128(
                        xs.rs, xs.off[f] + (uint32_t)(ks0 + b * KS + s) * 128u, 0, 0);
        } else {
            const u32x4 *xb = xs.frag + (size_t)(ks0 + b * KS) * NX * 64;
#pragma unroll
            for (int s = 0; s < KS; ++s)
#pragma unroll
                for (int f = 0; f < NX; ++f) xv[d][f][s] = ld_cached(xb + (s * NX + f) * 64 + lane);
        }
    };
    auto mma = [&](int d) {
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int r = RPI * j + lr;
            sw[r * CPR + bx_swz<KS>(r, lc)] = w[d][j];
        }
        __builtin_amdgcn_wave_barrier();
        u32x4 av[MT][KS];
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const int r = 16 * mt + lm;
                av[mt][s] = sw[r * CPR + bx_swz<KS>(r, 4 * s + lq)];
            }
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
            for (int f = 0; f < NX; ++f)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    f32x4 &c = acc[mt][S::PACK ? 0 : f >> 1];
                    c = mfma_bf16(av[mt][s], xv[d][f][s], c);
                }
        __builtin_amdgcn_wave_barrier();
    };
    // nbat is a positive multiple of D (hpad is a multiple of 4 waves x 32 x
    // KS x D).  The steady loop has no branch and the ring registers need no
    // copies, so the waits before each batch's MFMAs leave the later batches
    // in flight; the scheduling barriers keep each batch's loads together
    // and in ring order.
#pragma unroll
    for (int d = 0; d < D; ++d) {
        issue(d, d);
        __builtin_amdgcn_sched_barrier(0);
    }
    for (int it = 0; it + D < nbat; it += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            mma(d);
            __builtin_amdgcn_sched_barrier(0);
            issue(d, it + D + d);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
#pragma unroll
    for (int d = 0; d < D; ++d) mma(d);
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

// With packed fragments, column lm holds the high-part sum of token lm & 7
// (lm < 8) or its low-part sum (lm >= 8): add the partner column, so both
// lanes of a pair end with the same total.
template <int TOK>
__device__ __forceinline__ void bx_pair_sum(f32x4 (&acc)[2][Bx<TOK>::NT]) {
    if (!Bx<TOK>::PACK) return;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[mt][0][i] += dpp_f32<0x128>(acc[mt][0][i]);  // row_ror:8
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
__device__ __forceinline__ void bx_token_masks(const bool (&pred)[2][NT][4], const int (&rowbit)[2][4],
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
}

// Position of the n-th (from 0) set bit of m, by halving with population
// counts; n < popcount(m) (otherwise some position in 0..31).
__device__ __forceinline__ int nth_set_bit(uint32_t m, int n) {
    int pos = 0;
#pragma unroll
    for (int w = 16; w >= 1; w >>= 1) {
        const int c = __popc(m & ((1u << w) - 1u));
        if (n >= c) {
            n -= c;
            m >>= w;
            pos += w;
        }
    }
    return pos;
}

template <int TOK, int KS, int D, bool GATHER = false>
__global__ __launch_bounds__(256, TOK >= 64 ? 1 : 2) void bx_gate_up(BxArgs a) {
    using S = Bx<TOK>;
    constexpr int NT = S::NT, NX = S::NX;
    constexpr int CPR = 4 * KS, RPI = 16 / KS;
    __shared__ f32x4 s_red[4][2][NT][64];
    __shared__ float s_g[kBxRows][TOK];
    __shared__ __attribute__((aligned(16))) uint16_t s_h[kBxRows][2 * TOK];
    __shared__ u32x4 s_stage[4][kBxRows * CPR];  // per-wave weight staging
    __shared__ int s_tok[GATHER ? TOK : 1];
    __shared__ int s_ng;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lm = lane & 15, lq = lane >> 4;
    const int g = bx_group_at(blockIdx.x / a.ntiles, a.G, a.vpe);
    const int tile = blockIdx.x % a.ntiles;
    const size_t tix = (size_t)g * a.ntiles + tile;
    int ng;
    if constexpr (GATHER) {
        // the group's tokens from the routing table; its first tile's
        // workgroup writes the group tables
        if (wave == 0) {
            const int n = bx_list_group<TOK>(a, g, lane, s_tok, tile == 0);
            if (lane == 0) s_ng = n;
        }
        __syncthreads();
        ng = s_ng;
    } else {
        ng = a.gcount[g];
    }
    if (ng == 0) {
        if (tid == 0) {
            a.cnt[tix * 2] = 0;
            a.cnt[tix * 2 + 1] = 0;
        }
        if (a.want_masks)
            for (int s = tid; s < TOK; s += 256) {
                a.gmask[tix * TOK + s] = 0;
                a.amask[tix * TOK + s] = 0;
            }
        return;
    }
    for (int e = tid; e < 2 * TOK * kBxRows / 8; e += 256)
        reinterpret_cast<u32x4 *>(&s_h[0][0])[e] = u32x4{0u, 0u, 0u, 0u};

    const int r0 = tile * kBxRows;
    const uint16_t *wg = reinterpret_cast<const uint16_t *>(a.wg) + (size_t)(g / a.vpe) * a.expert_stride;
    const uint16_t *wu = reinterpret_cast<const uint16_t *>(a.wu) + (size_t)(g / a.vpe) * a.expert_stride;
    const int nks = a.hpad / 32;
    const BxX<NX> xs = bx_xsource<TOK, GATHER>(a, g, lane, s_tok);
    const int kpw = nks / 4;  // k-steps per wave
    const int ks0 = wave * kpw, nbat = kpw / KS;
    u32x4 *sw = s_stage[wave];
    const int lr = lane / CPR;  // row of this lane within an instruction's RPI rows
    // token of this lane's accumulator column, and whether the lane reports it
    const bool tok_lane = !S::PACK || lm < 8;

    // ---- gate: 32 rows x all tokens --------------------------------------
    f32x4 acc[2][NT];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    {
        uint32_t roff[2 * KS];
#pragma unroll
        for (int j = 0; j < 2 * KS; ++j) roff[j] = 2u * (uint32_t)min(r0 + RPI * j + lr, a.I - 1) * (uint32_t)a.H;
        bx_kloop<TOK, 2, KS, D, GATHER>(reinterpret_cast<const char *>(wg), roff, a.H, xs, ks0, nbat, lane, sw, acc);
    }
    bx_combine<NT>(acc, s_red, wave, lane);
    bx_pair_sum<TOK>(acc);

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
                if (wave == 0 && tok_lane) s_g[r][S::PACK ? lm : 16 * nt + lm] = acc[mt][nt][i];
            }
        }
    const uint32_t umask = bx_any_rows<NT>(open);
    const int nu = __popc(umask);
    if (a.want_masks) {
        uint32_t tm[NT];
        bx_token_masks<NT>(open, rowbit, tm);
        if (wave == 0 && lq == 0 && tok_lane)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) a.gmask[tix * TOK + (S::PACK ? lm : 16 * nt + lm)] = tm[nt];
    }
    __syncthreads();  // s_g complete

    // ---- up: the union rows, gathered ------------------------------------
    f32x4 uacc[2][NT];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) uacc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (nu > 16) {
        uint32_t roff[2 * KS];
#pragma unroll
        for (int j = 0; j < 2 * KS; ++j) {
            const int u = RPI * j + lr;
            roff[j] = 2u * (uint32_t)(r0 + nth_set_bit(umask, u < nu ? u : 0)) * (uint32_t)a.H;
        }
        bx_kloop<TOK, 2, KS, D, GATHER>(reinterpret_cast<const char *>(wu), roff, a.H, xs, ks0, nbat, lane, sw, uacc);
    } else if (nu > 0) {
        uint32_t roff[KS];
#pragma unroll
        for (int j = 0; j < KS; ++j) {
            const int u = RPI * j + lr;
            roff[j] = 2u * (uint32_t)(r0 + nth_set_bit(umask, u < nu ? u : 0)) * (uint32_t)a.H;
        }
        f32x4 u1[1][NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) u1[0][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        bx_kloop<TOK, 1, KS, D, GATHER>(reinterpret_cast<const char *>(wu), roff, a.H, xs, ks0, nbat, lane, sw, u1);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) uacc[0][nt] = u1[0][nt];
    }
    bx_combine<NT>(uacc, s_red, wave, lane);
    bx_pair_sum<TOK>(uacc);

    // ---- Combined for union index j = 16*mt + 4*lq + i -------------------
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
                const float gv = s_g[r][S::PACK ? (lm & 7) : 16 * nt + lm];
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
        bx_token_masks<NT>(act, ubit, tm);
        if (wave == 0 && lq == 0 && tok_lane)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) a.amask[tix * TOK + (S::PACK ? lm : 16 * nt + lm)] = tm[nt];
    }
    // active union index j -> slot (its rank); Combined into the fragment block
    if (wave == 0 && tok_lane) {
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int j = 16 * mt + 4 * lq + i;
                if ((amask_u >> j) & 1u) {
                    const int slot = __popc(amask_u & ((1u << j) - 1u));
#pragma unroll
                    for (int nt = 0; nt < NT; ++nt) {
                        const int t = S::PACK ? lm : 16 * nt + lm;
                        uint32_t hi, lo;
                        split_hi_lo(hv[mt][nt][i], hi, lo);
                        s_h[slot][t] = (uint16_t)hi;
                        s_h[slot][TOK + t] = (uint16_t)lo;
                    }
                }
            }
    }
    __syncthreads();  // s_h complete
    u32x4 *hdst = reinterpret_cast<u32x4 *>(a.hfrag + tix * (2 * TOK * kBxRows));
    for (int e = tid; e < 2 * TOK * kBxRows / 8; e += 256) hdst[e] = reinterpret_cast<const u32x4 *>(&s_h[0][0])[e];
    if (wave == 0) {
        if (lane < kBxRows) {  // an empty tile lists row 0 (always < I), never used
            const int j = nth_set_bit(amask_u, lane < na ? lane : 0);
            a.arow[tix * kBxRows + lane] = na > 0 ? (uint8_t)nth_set_bit(umask, j) : (uint8_t)0;
        }
        if (lane == 0) {
            a.cnt[tix * 2] = nu;
            a.cnt[tix * 2 + 1] = na;
        }
    }
}

// ---------------------------------------------------------------------------
// Gate + up over two 32-row tiles per workgroup (16 or more token slots).
// The x fragments of a group are the largest stream the gate / up kernel
// reads besides the weights: every workgroup reads all of them, once for the
// gate and once for the up pass, so their L2 traffic is (workgroups) x (x
// size) x 2.  At 32 token slots that is twice the weight bytes, and measured
// as the kernel's limit (without the x loads the same kernel streams 5.8
// against 3.6 TB/s).  Workgroups of 64 rows halve that traffic.  The K loop,
// its load shapes and the accumulation order are bx_gate_up's with four
// m-tiles instead of two, so every gate and up value is the same bits; the
// outputs are written per 32-row tile in bx_gate_up's layout (bx_down, the
// report and the union count read them unchanged).

__device__ __forceinline__ int nth_set_bit64(uint64_t m, int n) {
    const uint32_t lo = (uint32_t)m;
    const int c = __popc(lo);
    return n < c ? nth_set_bit(lo, n) : 32 + nth_set_bit((uint32_t)(m >> 32), n - c);
}

// bx_combine for MT m-tiles, two at a time through the same LDS buffer.
template <int MT, int NT>
__device__ __forceinline__ void bx_combine_mt(f32x4 (&acc)[MT][NT], f32x4 (*s_red)[2][NT][64], int wave, int lane) {
#pragma unroll
    for (int m0 = 0; m0 < MT; m0 += 2) {
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                if (m0 + mt < MT) s_red[wave][mt][nt][lane] = acc[m0 + mt][nt];
        __syncthreads();
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                if (m0 + mt < MT)
                    acc[m0 + mt][nt] = (s_red[0][mt][nt][lane] + s_red[1][mt][nt][lane]) +
                                       (s_red[2][mt][nt][lane] + s_red[3][mt][nt][lane]);
        __syncthreads();
    }
}

// Bit j (j < 64) set where row j has pred true for some token (layout as
// bx_any_rows, four m-tiles).
template <int NT>
__device__ __forceinline__ uint64_t bx_any_rows64(const bool (&pred)[4][NT][4]) {
    uint64_t bits = 0;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            uint64_t m = 0;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) m |= __ballot(pred[mt][nt][i]);
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if ((m >> (16 * q)) & 0xFFFFull) bits |= 1ull << (16 * mt + 4 * q + i);
        }
    return bits;
}

// Per token (lane lm of n-tile nt) the 64-bit mask of rows with pred true,
// rows mapped through rowbit (0..63).
template <int NT>
__device__ __forceinline__ void bx_token_masks64(const bool (&pred)[4][NT][4], const int (&rowbit)[4][4],
                                                 uint64_t (&tm)[NT]) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        uint64_t m = 0;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (pred[mt][nt][i]) m |= 1ull << rowbit[mt][i];
        uint32_t lo = (uint32_t)m, hi = (uint32_t)(m >> 32);
        lo |= (uint32_t)__shfl_xor((int)lo, 16, 64);
        hi |= (uint32_t)__shfl_xor((int)hi, 16, 64);
        lo |= (uint32_t)__shfl_xor((int)lo, 32, 64);
        hi |= (uint32_t)__shfl_xor((int)hi, 32, 64);
        tm[nt] = (uint64_t)lo | ((uint64_t)hi << 32);
    }
}

template <int TOK, int KS, int D, bool GATHER = false>
__global__ __launch_bounds__(256, TOK >= 64 ? 1 : 2) void bx_gate_up64(BxArgs a) {
    using S = Bx<TOK>;
    static_assert(!S::PACK, "the 64-row kernel serves 16 or more token slots");
    constexpr int NT = S::NT;
    constexpr int CPR = 4 * KS, RPI = 16 / KS;
    constexpr int RW = 2 * kBxRows;  // rows per workgroup
    __shared__ f32x4 s_red[4][2][NT][64];
    __shared__ float s_g[RW][TOK];
    __shared__ __attribute__((aligned(16))) uint16_t s_h[2][kBxRows][2 * TOK];
    __shared__ u32x4 s_stage[4][RW * CPR];  // per-wave weight staging
    __shared__ int s_tok[GATHER ? TOK : 1];
    __shared__ int s_ng;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lm = lane & 15, lq = lane >> 4;
    const int ntiles2 = (a.ntiles + 1) / 2;
    const int g = bx_group_at(blockIdx.x / ntiles2, a.G, a.vpe);
    const int t2 = blockIdx.x % ntiles2;
    const int tile0 = 2 * t2;
    const int nsub = min(2, a.ntiles - tile0);  // 32-row tiles this workgroup writes
    const size_t tix0 = (size_t)g * a.ntiles + tile0;
    int ng;
    if constexpr (GATHER) {
        // the group's tokens from the routing table; its first workgroup
        // writes the group tables
        if (wave == 0) {
            const int n = bx_list_group<TOK>(a, g, lane, s_tok, t2 == 0);
            if (lane == 0) s_ng = n;
        }
        __syncthreads();
        ng = s_ng;
    } else {
        ng = a.gcount[g];
    }
    if (ng == 0) {
        if (tid < 2 * nsub) a.cnt[tix0 * 2 + tid] = 0;
        if (a.want_masks)
            for (int s = tid; s < nsub * TOK; s += 256) {
                a.gmask[tix0 * TOK + s] = 0;
                a.amask[tix0 * TOK + s] = 0;
            }
        return;
    }
    for (int e = tid; e < 2 * 2 * TOK * kBxRows / 8; e += 256)
        reinterpret_cast<u32x4 *>(&s_h[0][0][0])[e] = u32x4{0u, 0u, 0u, 0u};

    const int r0 = tile0 * kBxRows;
    const uint16_t *wg = reinterpret_cast<const uint16_t *>(a.wg) + (size_t)(g / a.vpe) * a.expert_stride;
    const uint16_t *wu = reinterpret_cast<const uint16_t *>(a.wu) + (size_t)(g / a.vpe) * a.expert_stride;
    const int nks = a.hpad / 32;
    const BxX<S::NX> xs = bx_xsource<TOK, GATHER>(a, g, lane, s_tok);
    const int kpw = nks / 4;  // k-steps per wave
    const int ks0 = wave * kpw, nbat = kpw / KS;
    u32x4 *sw = s_stage[wave];
    const int lr = lane / CPR;

    // ---- gate: 64 rows x all tokens --------------------------------------
    f32x4 acc[4][NT];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    {
        uint32_t roff[4 * KS];
#pragma unroll
        for (int j = 0; j < 4 * KS; ++j) roff[j] = 2u * (uint32_t)min(r0 + RPI * j + lr, a.I - 1) * (uint32_t)a.H;
        bx_kloop<TOK, 4, KS, D, GATHER>(reinterpret_cast<const char *>(wg), roff, a.H, xs, ks0, nbat, lane, sw, acc);
    }
    bx_combine_mt<4, NT>(acc, s_red, wave, lane);

    bool open[4][NT][4];
    int rowbit[4][4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
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
    const uint64_t umask = bx_any_rows64<NT>(open);
    const int nu = __popcll(umask);
    if (a.want_masks) {
        uint64_t tm[NT];
        bx_token_masks64<NT>(open, rowbit, tm);
        if (wave == 0 && lq == 0)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                for (int h = 0; h < nsub; ++h)
                    a.gmask[(tix0 + h) * TOK + 16 * nt + lm] = (uint32_t)(tm[nt] >> (32 * h));
    }
    __syncthreads();  // s_g complete

    // ---- up: the union rows, gathered (as many m-tiles as they need) -----
    f32x4 uacc[4][NT];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) uacc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    auto up_pass = [&](auto mtc) {
        constexpr int MU = decltype(mtc)::value;
        uint32_t roff[MU * KS];
#pragma unroll
        for (int j = 0; j < MU * KS; ++j) {
            const int u = RPI * j + lr;
            roff[j] = 2u * (uint32_t)(r0 + nth_set_bit64(umask, u < nu ? u : 0)) * (uint32_t)a.H;
        }
        f32x4 ua[MU][NT];
#pragma unroll
        for (int mt = 0; mt < MU; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) ua[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        bx_kloop<TOK, MU, KS, D, GATHER>(reinterpret_cast<const char *>(wu), roff, a.H, xs, ks0, nbat, lane, sw, ua);
#pragma unroll
        for (int mt = 0; mt < MU; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) uacc[mt][nt] = ua[mt][nt];
    };
    if (nu > 48) up_pass(std::integral_constant<int, 4>{});
    else if (nu > 32) up_pass(std::integral_constant<int, 3>{});
    else if (nu > 16) up_pass(std::integral_constant<int, 2>{});
    else if (nu > 0) up_pass(std::integral_constant<int, 1>{});
    bx_combine_mt<4, NT>(uacc, s_red, wave, lane);

    // ---- Combined for union index j = 16*mt + 4*lq + i -------------------
    bool act[4][NT][4];
    float hv[4][NT][4];
    int ubit[4][4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int j = 16 * mt + 4 * lq + i;
            const int r = nth_set_bit64(umask, j < nu ? j : 0);
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
    const uint64_t amask_u = bx_any_rows64<NT>(act);  // over union indices
    // union indices below nu0 are rows of the first 32-row tile
    const int nu0 = __popc((uint32_t)umask);
    const uint64_t below0 = nu0 >= 64 ? ~0ull : ((1ull << nu0) - 1ull);
    const uint64_t am[2] = {amask_u & below0, amask_u & ~below0};
    if (a.want_masks) {
        uint64_t tm[NT];
        bx_token_masks64<NT>(act, ubit, tm);
        if (wave == 0 && lq == 0)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                for (int h = 0; h < nsub; ++h)
                    a.amask[(tix0 + h) * TOK + 16 * nt + lm] = (uint32_t)(tm[nt] >> (32 * h));
    }
    // active union index j of tile h -> slot (its rank within the tile)
    if (wave == 0) {
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int j = 16 * mt + 4 * lq + i;
                if ((amask_u >> j) & 1ull) {
                    const int h = j < nu0 ? 0 : 1;
                    const int slot = __popcll(am[h] & ((1ull << j) - 1ull));
#pragma unroll
                    for (int nt = 0; nt < NT; ++nt) {
                        const int t = 16 * nt + lm;
                        uint32_t hi, lo;
                        split_hi_lo(hv[mt][nt][i], hi, lo);
                        s_h[h][slot][t] = (uint16_t)hi;
                        s_h[h][slot][TOK + t] = (uint16_t)lo;
                    }
                }
            }
    }
    __syncthreads();  // s_h complete
    for (int h = 0; h < nsub; ++h) {
        u32x4 *hdst = reinterpret_cast<u32x4 *>(a.hfrag + (tix0 + h) * (2 * TOK * kBxRows));
        for (int e = tid; e < 2 * TOK * kBxRows / 8; e += 256)
            hdst[e] = reinterpret_cast<const u32x4 *>(&s_h[h][0][0])[e];
    }
    if (wave == 0) {
        for (int h = 0; h < nsub; ++h) {
            const int na = __popcll(am[h]);
            if (lane < kBxRows) {  // an empty tile lists row 0 (always < I), never used
                const int j = nth_set_bit64(am[h], lane < na ? lane : 0);
                a.arow[(tix0 + h) * kBxRows + lane] =
                    na > 0 ? (uint8_t)(nth_set_bit64(umask, j) - kBxRows * h) : (uint8_t)0;
            }
            if (lane == 0) {
                a.cnt[(tix0 + h) * 2] = __popc((uint32_t)(umask >> (32 * h)));
                a.cnt[(tix0 + h) * 2 + 1] = na;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Down: workgroup (group, chunk of tiles, 128-column slice), 4 waves.  The
// chunk's active rows, tile after tile in ascending order, are listed once
// in LDS (4 bytes each: the tile within the chunk, the slot of its Combined
// record, the row within the tile; up to bx_down_tiles(TOK) tiles) and cut
// into K blocks of 32; wave w takes blocks w, w + 4, ...  A block's W_down_t rows x the
// slice's 128 columns (8 KB) are loaded as 8 coalesced 16-byte loads per
// lane (lane (lq, lm): slot 8 lq + q, columns 8 lm .. 8 lm + 7) and written
// to the wave's own LDS region row-major, the 16-byte chunk c of slot s at
// position c ^ (2 ((s >> 3) & 3)).  The MFMA operand of n-tile nc (columns
// 16 nc + lm) takes slots 8 lq .. 8 lq + 7 of one column: eight 2-byte LDS
// reads whose 16 lanes of each lq hit 8 banks of their own (the swizzle
// moves the four lq groups apart), so neither the writes nor the reads
// conflict.  The block's Combined values (slot-major records written by
// bx_gate_up) are transposed through a small LDS tile into the other
// operand (token rows, 8 consecutive slots per lane).  Slots past the last
// row load zeros (out-of-range buffer offset) with zero Combined.  Loads of the next DD - 1
// blocks are in flight while a block is contracted; the four waves' sums
// are added in a fixed order at the end.
constexpr uint32_t kPadRow = 0xFFFFFFFFu;  // row-list padding of bx_down

template <int TOK, int DD>
__global__ __launch_bounds__(256, TOK <= 16 ? 2 : 1) void bx_down(BxArgs a) {
    using S = Bx<TOK>;
    constexpr int NT = S::NT, NX = S::NX;
    constexpr int REG = 512 * NT;  // 16-byte units per wave: 8 KB staging, or its 8 x NT accumulators
    constexpr int BG = 2;          // n-tiles whose operands are read from LDS together
    constexpr int AP = 40;         // bf16 per row of the Combined tile (80 bytes: 16-row reads do not conflict)
    constexpr int HC = TOK / 8;    // 16-byte Combined chunks per lane (token half of one slot)
    constexpr int MAXT = bx_down_tiles(TOK);  // tiles per chunk at most
    constexpr int MAXR = MAXT * kBxRows;       // list entries at most
    constexpr int WPT = MAXR / 4 / 256;        // row-byte words (4 rows each) per thread
    static_assert(MAXT <= 512 && MAXR % 1024 == 0, "two tiles per thread in the count scan; whole words per thread");
    __shared__ u32x4 s_lds[4 * REG];
    // listed rows: (tile within the chunk) << 10 | slot << 5 | row within the tile, or kPadRow
    __shared__ __attribute__((aligned(16))) uint32_t s_ent[MAXR];
    __shared__ int s_pre[MAXT + 1];
    __shared__ int s_wsum[4];
    // the Combined tile: past the staging 8 KB of the wave's region when it has room (NT >= 2)
    constexpr bool AIN = NT >= 2;
    __shared__ __attribute__((aligned(16))) uint16_t s_a_own[AIN ? 1 : 4][2 * TOK][AP];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lm = lane & 15, lq = lane >> 4;
    // Work item (group, chunk, slice).  The dispatcher hands workgroup b to
    // XCD b % 8; when the (group, chunk) pairs come in multiples of 8, each
    // pair goes to one XCD with all of its slices, so the pair's Combined
    // fragments and row lists are fetched into one XCD's L2 only (spread
    // over all eight they were fetched eight times: 13% of the kernel's HBM
    // reads at batch 32).  In round j XCD q takes pair 8 j + (q - j) mod 8,
    // so that work that repeats with period 8 (groups of 8 chunks) still
    // reaches every XCD.  Pairs are numbered group by group in the order of
    // bx_group_at (the nearly always empty further groups last).  Any
    // dispatch order gives the same results.
    int slice, pair;
    const int npairs = a.G * a.nchunks;
    if (npairs % 8 == 0) {
        const int q = blockIdx.x % 8, r = blockIdx.x / 8;
        const int j = r / a.nslices;
        slice = r % a.nslices;
        pair = 8 * j + ((q - j) & 7);
    } else {
        slice = blockIdx.x % a.nslices;
        pair = blockIdx.x / a.nslices;
    }
    const int chunk = pair % a.nchunks;
    const int g = bx_group_at(pair / a.nchunks, a.G, a.vpe);
    const int ng = a.gcount[g];
    if (ng == 0) return;
    const int H = a.H;
    const int t0 = chunk * a.tpc;
    const int ntc = min(a.tpc, a.ntiles - t0);
    const size_t tbase = (size_t)g * a.ntiles + t0;

    // ---- the chunk's row list: the tiles' counts and row bytes are read in
    // one round trip (bx_gate_up writes all 32 row bytes of a tile, 8 words)
    uint32_t rbw[WPT];
    const uint32_t *arow32 = reinterpret_cast<const uint32_t *>(a.arow) + tbase * (kBxRows / 4);
#pragma unroll
    for (int u = 0; u < WPT; ++u) {
        const int w = tid + 256 * u;
        rbw[u] = w < ntc * (kBxRows / 4) ? arow32[w] : 0u;
    }
    // exclusive prefix of the active counts: thread i holds tiles 2i, 2i + 1
    const int ta = 2 * tid;
    const int na_a = ta < ntc ? a.cnt[(tbase + ta) * 2 + 1] : 0;
    const int na_b = ta + 1 < ntc ? a.cnt[(tbase + ta + 1) * 2 + 1] : 0;
    {
        const int v = na_a + na_b;
        int inc = v;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int t = __shfl_up(inc, o, 64);
            if (lane >= o) inc += t;
        }
        if (lane == 63) s_wsum[wave] = inc;
        __syncthreads();
        int before = 0;
#pragma unroll
        for (int w = 0; w < 4; ++w) before += w < wave ? s_wsum[w] : 0;
        const int ex = before + inc - v;
        if (ta < ntc) s_pre[ta] = ex;
        if (ta + 1 < ntc) s_pre[ta + 1] = ex + na_a;
        if (tid == 255) s_pre[ntc] = ex + v;
    }
    __syncthreads();
    const int total = s_pre[ntc];
    const int nblk = (total + kBxRows - 1) / kBxRows;
    // listed rows; the block padding past `total` loads at an out-of-range
    // offset (zeros, no traffic) and has zero Combined
#pragma unroll
    for (int u = 0; u < WPT; ++u) {
        const int w = tid + 256 * u;
        if (w < ntc * (kBxRows / 4)) {
            const int t = w / (kBxRows / 4), s4 = 4 * (w % (kBxRows / 4));
            const int base = s_pre[t], na = s_pre[t + 1] - base;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (s4 + j < na)
                    s_ent[base + s4 + j] =
                        ((uint32_t)t << 10) | ((uint32_t)(s4 + j) << 5) | ((rbw[u] >> (8 * j)) & 31u);
        }
    }
    for (int e = total + tid; e < nblk * kBxRows; e += 256) s_ent[e] = kPadRow;
    __syncthreads();

    const uint16_t *wde = reinterpret_cast<const uint16_t *>(a.wd) + (size_t)(g / a.vpe) * a.expert_stride;
    const __amdgpu_buffer_rsrc_t rwd = make_rsrc(wde, (uint32_t)a.I * (uint32_t)H * 2u);
    const int col0 = slice * kBxSliceCols;
    const uint32_t cw = 2u * (uint32_t)min(col0 + 8 * lm, H - 8);
    const uint32_t H2 = 2u * (uint32_t)H;
    u32x4 *sw = s_lds + wave * REG;
    const uint16_t *sw16 = reinterpret_cast<const uint16_t *>(sw);
    uint16_t(*s_a)[AP] = AIN ? reinterpret_cast<uint16_t(*)[AP]>(sw + 512) : s_a_own[AIN ? 0 : wave];
    const int hj = lane & 31, hh = lane >> 5;  // Combined staging: slot, token half (high / low part)

    f32x4 acc[8][NT];
#pragma unroll
    for (int nc = 0; nc < 8; ++nc)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[nc][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nbw = nblk > wave ? (nblk - wave + 3) / 4 : 0;  // this wave's blocks
    if (nbw > 0) {
        u32x4 wv[DD][8], hq[DD][HC];
        bool hok[DD];
        int kk = 0;  // blocks issued so far; past the last, block `wave` is re-read and never used
        auto issue = [&](int d) {
            const int bb = kk < nbw ? wave + 4 * kk : wave;
            ++kk;
            const u32x4 ra = *reinterpret_cast<const u32x4 *>(&s_ent[bb * kBxRows + 8 * lq]);
            const u32x4 rb = *reinterpret_cast<const u32x4 *>(&s_ent[bb * kBxRows + 8 * lq + 4]);
            const uint32_t rr[8] = {ra.x, ra.y, ra.z, ra.w, rb.x, rb.y, rb.z, rb.w};
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const uint32_t row = (uint32_t)(t0 + (int)(rr[q] >> 10)) * kBxRows + (rr[q] & 31u);
                wv[d][q] = ld_buf_stream(rwd, rr[q] == kPadRow ? kOutOfRange : row * H2 + cw);
            }
            const uint32_t he = s_ent[bb * kBxRows + hj];
            hok[d] = he != kPadRow;
            const size_t hx = hok[d] ? (tbase + (he >> 10)) * kBxRows + ((he >> 5) & 31u) : 0;
            const uint16_t *hs = a.hfrag + hx * (2 * TOK) + hh * TOK;
#pragma unroll
            for (int c = 0; c < HC; ++c) hq[d][c] = ld_cached(hs + 8 * c);
        };
        auto mma = [&](int d) {
#pragma unroll
            for (int q = 0; q < 8; ++q) sw[(8 * lq + q) * 16 + (lm ^ (2 * lq))] = wv[d][q];
#pragma unroll
            for (int c = 0; c < HC; ++c) {
                const uint32_t w4[4] = {hq[d][c].x, hq[d][c].y, hq[d][c].z, hq[d][c].w};
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint16_t v = (uint16_t)(e & 1 ? w4[e >> 1] >> 16 : w4[e >> 1] & 0xFFFFu);
                    s_a[hh * TOK + 8 * c + e][hj] = hok[d] ? v : (uint16_t)0;
                }
            }
            __builtin_amdgcn_wave_barrier();
            u32x4 af[NX];
#pragma unroll
            for (int f = 0; f < NX; ++f) {
                const int ar = S::PACK ? lm : (f & 1) * TOK + 16 * (f >> 1) + lm;
                af[f] = *reinterpret_cast<const u32x4 *>(&s_a[ar][8 * lq]);
            }
#pragma unroll
            for (int n2 = 0; n2 < 8; n2 += BG) {
                u16x8 bfr[BG];
#pragma unroll
                for (int u = 0; u < BG; ++u) {
                    const int pos = (2 * (n2 + u) + (lm >> 3)) ^ (2 * lq);
                    const uint16_t *src = sw16 + (8 * lq) * kBxSliceCols + 8 * pos + (lm & 7);
#pragma unroll
                    for (int j = 0; j < 8; ++j) bfr[u][j] = src[j * kBxSliceCols];
                }
#pragma unroll
                for (int u = 0; u < BG; ++u) {
                    const u32x4 b = __builtin_bit_cast(u32x4, bfr[u]);
#pragma unroll
                    for (int f = 0; f < NX; ++f) {
                        f32x4 &c = acc[n2 + u][S::PACK ? 0 : f >> 1];
                        c = mfma_bf16(af[f], b, c);
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            __builtin_amdgcn_wave_barrier();
        };

        // steady loop without branches (every issue is a real block), then
        // the last (fewer than 2 DD) blocks
#pragma unroll
        for (int d = 0; d < DD; ++d) issue(d);
        int b = 0;
        for (; b + 2 * DD <= nbw; b += DD) {
#pragma unroll
            for (int d = 0; d < DD; ++d) {
                mma(d);
                issue(d);
            }
        }
#pragma unroll
        for (int d = 0; d < DD; ++d) {
            if (b + d < nbw) {
                mma(d);
                if (b + d + DD < nbw) issue(d);
            }
        }
#pragma unroll
        for (int d = 0; d < DD; ++d)
            if (b + DD + d < nbw) mma(d);
    }

    // the four waves' sums, added in a fixed order; wave w finishes n-tiles 2w, 2w + 1
    f32x4 *sa = reinterpret_cast<f32x4 *>(sw);
#pragma unroll
    for (int nc = 0; nc < 8; ++nc)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) sa[(nc * NT + nt) * 64 + lane] = acc[nc][nt];
    __syncthreads();
    const f32x4 *s0 = reinterpret_cast<const f32x4 *>(s_lds);
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
        const int nc = 2 * wave + k2;
        const int col = col0 + 16 * nc + lm;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const int e = (nc * NT + nt) * 64 + lane;
            f32x4 v = (s0[e] + s0[REG + e]) + (s0[2 * REG + e] + s0[3 * REG + e]);
            if (S::PACK) {
#pragma unroll
                for (int i = 0; i < 4; ++i) v[i] += __shfl_xor(v[i], 32, 64);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int tok = 16 * nt + 4 * lq + i;
                const bool ok = (S::PACK ? lq < 2 : true) && tok < ng && col < H;
                if (ok) a.partial[(((size_t)g * TOK + tok) * a.nchunks + chunk) * H + col] = v[i];
            }
        }
    }
}

// out[t][:] = sum over routed ranks k (ascending) of w[t][k] times the sum
// over chunks of the partial row of (group, slot) = tslot[t][k].  Block:
// 256 columns (64 float4, one per lane) x 4 share groups (one per wave); a
// thread adds shares grp, grp + 4, ... (share k * nchunks + c) in order, and
// the four groups' sums are combined in a fixed order through LDS.  One
// block per (256 columns, token): the shares are few (top_k x chunks), so a
// wide block keeps the grid small.
__global__ __launch_bounds__(256) void bx_reduce(BxArgs a) {
    __shared__ f32x4 red[4][64];
    const int t = blockIdx.y;
    const int q = threadIdx.x & 63;
    const int grp = threadIdx.x >> 6;
    const int c4 = blockIdx.x * 64 + q;
    const int nq = a.H / 4;
    const int total = a.K * a.nchunks;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int p = grp; p < total; p += 4) {
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
    if (grp == 0 && c4 < nq)
        *reinterpret_cast<f32x4 *>(a.out + (size_t)t * a.H + c4 * 4) = (red[0][q] + red[1][q]) + (red[2][q] + red[3][q]);
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

// gate+up load shape: k-steps per batch x batches in flight ("bx_gate" knob,
// 0 = the default for the token count)
template <int TOK>
void launch_gate_up(const BatchPlan &p, const BxArgs &a, hipStream_t st) {
    const dim3 grid((unsigned)(p.groups * p.ntiles));
    if constexpr (TOK >= 16) {
        // 16 or more token slots: two 32-row tiles per workgroup (half the x
        // traffic); knobs 1-3 keep one tile per workgroup
        if (tuned("bx_gate") == 0) {
            const dim3 grid2((unsigned)(p.groups * ((p.ntiles + 1) / 2)));
            // 2 k-steps per load batch (4 at 16 slots spills registers with four m-tiles)
            if (a.xtok) launch("batch_gate_up", bx_gate_up64<TOK, 2, 2, true>, grid2, dim3(256), st, a);
            else launch("batch_gate_up", bx_gate_up64<TOK, 2, 2>, grid2, dim3(256), st, a);
            return;
        }
    }
    if (a.xtok) {  // x gathered from the router's token-major split
        if constexpr (TOK <= 16) {
            if (tuned("bx_gate") == 2) {
                launch("batch_gate_up", bx_gate_up<TOK, 2, 4, true>, grid, dim3(256), st, a);
                return;
            }
        }
        if (TOK == 8 || tuned("bx_gate") == 1)
            launch("batch_gate_up", bx_gate_up<TOK, 2, 2, true>, grid, dim3(256), st, a);
        else
            launch("batch_gate_up", bx_gate_up<TOK, Bx<TOK>::KS, Bx<TOK>::D, true>, grid, dim3(256), st, a);
        return;
    }
    if constexpr (TOK <= 16) {  // deeper shapes spill registers at 32 tokens and run slower
        switch (tuned("bx_gate")) {
        case 1: launch("batch_gate_up", bx_gate_up<TOK, 2, 2>, grid, dim3(256), st, a); return;
        case 2: launch("batch_gate_up", bx_gate_up<TOK, 2, 4>, grid, dim3(256), st, a); return;
        default: break;
        }
    }
    launch("batch_gate_up", bx_gate_up<TOK, Bx<TOK>::KS, Bx<TOK>::D>, grid, dim3(256), st, a);
}

template <int TOK>
void launch_tok(const BatchPlan &p, const BxArgs &a, hipStream_t st) {
    if (!a.xtok) {
        const int nthreads = p.groups * (p.hpad / 32) * Bx<TOK>::NX * 64;
        launch("batch_prep", bx_prep<TOK>, dim3((unsigned)((nthreads + 255) / 256)), dim3(256), st, a);
    }
    launch_gate_up<TOK>(p, a, st);
    const dim3 grid((unsigned)(p.groups * p.nchunks * p.nslices));
    if constexpr (TOK <= 32) {
        if (tuned("bx_down") == 1) {
            launch("batch_down", bx_down<TOK, 3>, grid, dim3(256), st, a);
            return;
        }
    }
    launch("batch_down", bx_down<TOK, Bx<TOK>::DD>, grid, dim3(256), st, a);
}

}  // namespace

// One pass of the batched path for up to kBxMaxTokens tokens.  x and out are
// offset to the pass's first token; topk / topw (MoE) are [batch][K] for the
// pass's tokens.  Stats arrays are indexed from stats_base.
ts_status run_batch(const float *x, const void *wg, const void *wu, const void *wd, size_t expert_stride,
                    const int32_t *topk, const float *topw, const BatchPlan &p, float *out,
                    const ts_ffn_stats *stats, int stats_base, void *ws, hipStream_t st, bool dense, bool xtok) {
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
    a.vpe = p.vpe;
    a.K = p.top_k;
    a.bpad = p.bpad;
    a.hpad = p.hpad;
    a.ntiles = p.ntiles;
    a.nslices = p.nslices;
    a.nchunks = p.nchunks;
    a.tpc = p.tpc;
    a.topk = topk;
    a.topw = topw;
    a.gcount = ws_at<int32_t>(ws, p.off_gcount);
    a.tslot = ws_at<int32_t>(ws, p.off_tslot);
    a.xhl = ws_at<uint16_t>(ws, p.off_xhl);
    a.cnt = ws_at<int32_t>(ws, p.off_cnt);
    a.arow = ws_at<uint8_t>(ws, p.off_arow);
    a.hfrag = ws_at<uint16_t>(ws, p.off_hfrag);
    a.gmask = ws_at<uint32_t>(ws, p.off_gmask);
    a.amask = ws_at<uint32_t>(ws, p.off_amask);
    a.partial = ws_at<float>(ws, p.off_partial);
    a.out = out;
    // the router's split exists only with a routing table
    a.xtok = (xtok && topk) ? ws_at<uint16_t>(ws, p.off_xhl) : nullptr;
    a.xchunks = p.hpad / 8;
    const bool want_lists = stats && (stats->n_gate || stats->n_active || stats->gate_idx || stats->active_idx);
    a.want_masks = want_lists ? 1 : 0;

    switch (p.tok) {
    case 8: launch_tok<8>(p, a, st); break;
    case 16: launch_tok<16>(p, a, st); break;
    case 32: launch_tok<32>(p, a, st); break;
    default: launch_tok<64>(p, a, st); break;
    }
    launch("batch_reduce", bx_reduce, dim3((unsigned)((p.hidden / 4 + 63) / 64), (unsigned)p.batch), dim3(256), st, a);
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
