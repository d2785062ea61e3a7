// Single-token ("slot") kernels of the activation-sparse dReLU FFN for gfx950
// and the ts_ffn_* / ts_moe_* entry points.
//
// One slot is one token evaluated against one weight set (the FFN's, or the
// routed expert's in the MoE layer).  Eq. (drelu) of Turbo Sparse (arXiv
// 2406.05955): Combined = max(0, x W_gate) * max(0, x W_up), out = Combined
// W_down.  Skipping the zero Combined terms (section 6.2) leaves the output
// unchanged, so only the W_up rows of open gates and the W_down rows of
// non-zero Combined activations are read.
//
// Three kernel sequences serve a call (all end in ffn_reduce, which sums
// fp32 partial rows in a fixed order: deterministic, no atomics):
//
// pipe   (ffn_pipe, the default): as fused below, but each wave streams its
//        gate rows two deep and issues an open row's W_up loads at once, so
//        the up traffic travels with the gate stream (described at the
//        kernel).
//
// fused  (ffn_fused, 8 waves per workgroup, one tile of neurons each)
//   gate   every lane holds its share of x in registers; each wave dots whole
//          W_gate rows (16-byte streaming loads, RIF rows in flight); the
//          gates meet in LDS, one wave ballots `gate > 0` and prefix-counts
//          the ballot into the tile's ascending open-gate list G;
//   up     the waves dot the W_up rows of G; a second ballot compacts the
//          neurons with up > 0 into A with Combined = gate * up;
//   down   the 512 threads split the hidden dimension (16 bytes each) and run
//          an axpy over the W_down_t rows of A in ascending order into the
//          tile's partial output row.
//   The dense comparator is this kernel with every neuron taken.
//   In pipe and fused the tiles interleave (tile t of T holds t, t + T, ...)
//   where the matrices allow it, so the grid streams one narrow band of
//   each matrix at a time.
//
// split  (ffn_gate_up with 4-wave workgroups, then ffn_down)
//   gate and up as above, the tile's A segment and Combined values go to the
//   workspace; ffn_down gives each (chunk of tiles, 64-chunk column slice) a
//   workgroup that lists the chunk's active rows in LDS and accumulates
//   their W_down_t slices into a partial row per chunk.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <mutex>

#include "ts_batch.h"
#include "ts_device.h"
#include "ts_plan.h"
#include "ts_runtime.h"
#include "turbosparse.h"

namespace ts {

// W_down_t rows whose loads are in flight together in the down phases: 16
// covers the active rows of nearly every 56- or 64-neuron tile at 90%
// sparsity in one round trip (with 8, ~9% of 56-neuron tiles needed a
// second one, and the slowest tile sets the kernel's end: 0.2 us per layer)
constexpr int kDownUnroll = 16;
// ffn_given builds a buffer resource per row; its short chunks (often 4
// entries at high sparsity) measured faster with 8
constexpr int kGivenDownUnroll = 8;

// Lane `lane` keeps chunks lane, lane + 64, ... of x (fp32) in registers.
template <typename WT, int NC>
__device__ __forceinline__ void load_x(const float *__restrict__ x, int lane, int nch,
                                       float (&xr)[NC][WTraits<WT>::CE]) {
    constexpr int CE = WTraits<WT>::CE;
    constexpr int Q = CE / 4;  // float4 per chunk
    f32x4 v[NC][Q];
#pragma unroll
    for (int k = 0; k < NC; ++k)
#pragma unroll
        for (int q = 0; q < Q; ++q) v[k][q] = ld_f32x4_masked(x, (lane + 64 * k) * Q + q, nch * Q);
#pragma unroll
    for (int k = 0; k < NC; ++k)
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            xr[k][4 * q] = v[k][q].x;
            xr[k][4 * q + 1] = v[k][q].y;
            xr[k][4 * q + 2] = v[k][q].z;
            xr[k][4 * q + 3] = v[k][q].w;
        }
}

// Dot products of R weight rows with the x chunks held in registers.  All
// R * NC loads are issued before any arithmetic; rows with valid[k] false
// (and chunks past the row end) read a clamped address and count as zero.
// Streaming loads, or (CACHED) the default cache policy for rows that many
// workgroups read.  Returns wave-uniform sums.
template <typename WT, int NC, int R, bool CACHED = false>
__device__ __forceinline__ void dot_rows(const WT *const (&rows)[R], const bool (&valid)[R],
                                         const float (&xr)[NC][WTraits<WT>::CE], int lane, int nch,
                                         float (&out)[R]) {
    constexpr int CE = WTraits<WT>::CE;
    u32x4 v[R][NC];
#pragma unroll
    for (int k = 0; k < R; ++k)
#pragma unroll
        for (int c0 = 0; c0 < NC; ++c0) {
            if constexpr (CACHED) v[k][c0] = ld_cached_masked(rows[k], lane + 64 * c0, nch, 16, valid[k]);
            else v[k][c0] = ld_stream_masked(rows[k], lane + 64 * c0, nch, 16, valid[k]);
        }
#pragma unroll
    for (int k = 0; k < R; ++k) {
        float d = 0.f;
#pragma unroll
        for (int c0 = 0; c0 < NC; ++c0) {
            float f[CE];
            unpack<WT>(v[k][c0], f);
#pragma unroll
            for (int e = 0; e < CE; ++e) d = fmaf(f[e], xr[c0][e], d);
        }
        out[k] = wave_sum(d);
    }
}

struct SlotArgs {
    const float *x;          // [tokens][H]
    const void *wg;          // [experts][I][H] (one expert for the FFN)
    const void *wu;
    const void *wd;
    const int32_t *route;    // [slots] expert of each slot, or null (FFN)
    size_t expert_stride;    // elements per expert matrix
    int H, I, tile, ntiles, slots_per_tok;
    int32_t *cnt;            // [slots][ntiles][2] = |G|, |A| of the tile
    int32_t *gseg;           // [slots][ntiles][tile] tile's G, ascending (if want_seg)
    int32_t *aseg;           // [slots][ntiles][tile] tile's A, ascending (if want_seg)
    float *partial;          // [slots][ntiles][H]
    float *hseg;             // [slots][ntiles][tile] Combined values of aseg (pipelined kernel, emit mode)
    int want_seg;
    // In-kernel routing (pipelined kernel, route == null): router weights
    // [E][H]; the tile-0 workgroup of each slot records its expert and
    // renormalised weight in ridx / rw ([tokens][K]).
    const void *wr;
    int E, K;
    int32_t *ridx;
    float *rw;
    // Activation: 0 = dReLU (Eq. drelu), 1 = gate-only ReLU with threshold
    // `tau` (Combined = max(0, gate - tau) * up: ReGLU at tau = 0).
    int act;
    float tau;
    // Neurons of a tile: rstride <= 1, tile t holds [t * tile, t * tile + tile);
    // rstride = ntiles (interleaved), tile t holds t, t + ntiles, t + 2 ntiles,
    // ..., so that at any moment the grid reads one narrow band of each
    // matrix.  The segments hold neuron ids either way.
    int rstride;
};

// The open-gate threshold and the Combined activation of a neuron whose
// gate passed it, for either activation.
__device__ __forceinline__ float gate_threshold(int act, float tau) { return act ? tau : 0.f; }
__device__ __forceinline__ bool combined_nonzero(int act, float u) { return act ? u != 0.f : u > 0.f; }
__device__ __forceinline__ float combined_value(int act, float tau, float g, float u) {
    return act ? (g - tau) * u : g * u;
}

// The router's decision for one token (section 6.2: top-k gating over the
// softmax of the router logits), by one wave: softmax over the E (<= 64)
// logits, the top K (strictly larger wins, so the lower index wins exact
// ties) and their weights renormalised over the K.  Lane e holds expert e;
// every reduction is a register butterfly whose result is the same on all
// lanes (max and arg-max are exact; the softmax sum is taken from lane 0),
// and nothing is indexed at run time, so no private memory is used.  Lane
// k < K ends with the expert of rank k in *idx and its weight in *w.
__device__ inline void route_wave(const float *logit, int E, int K, int lane, int *idx, float *w) {
    const bool in = lane < E;
    const float l = in ? logit[lane] : -INFINITY;
    float m = l;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    float p = in ? expf(l - m) : 0.f;
    float z = p;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) z += __shfl_xor(z, o, 64);
    z = __shfl(z, 0, 64);
    p *= 1.f / z;
    bool taken = false;
    float ps = 0.f, mine = 0.f;
    int mi = -1;
#pragma unroll
    for (int k = 0; k < kMaxTopK; ++k) {
        if (k < K) {
            float v = (in && !taken) ? p : -1.f;  // probabilities are >= 0
            int bi = lane;
#pragma unroll
            for (int o = 32; o >= 1; o >>= 1) {
                const float ov = __shfl_xor(v, o, 64);
                const int oi = __shfl_xor(bi, o, 64);
                if (ov > v || (ov == v && oi < bi)) {
                    v = ov;
                    bi = oi;
                }
            }
            if (lane == bi) taken = true;
            ps += v;
            if (lane == k) {
                mi = bi;
                mine = v;
            }
        }
    }
    *idx = mi;
    *w = mine / ps;
}

template <typename WT, int NC, bool DENSE, int RIF>
__global__ __launch_bounds__(kThreads) void ffn_fused(SlotArgs a) {
    constexpr int CE = WTraits<WT>::CE;
    constexpr int NCD = (NC * 64 + kThreads - 1) / kThreads;

    __shared__ float s_g[kMaxTile];
    __shared__ float s_h[kMaxTile];
    __shared__ int s_on[kMaxTile];
    __shared__ int s_gl[kMaxTile];
    __shared__ int s_al[kMaxTile];
    __shared__ float s_av[kMaxTile];
    __shared__ int s_n[2];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int tile = blockIdx.x % a.ntiles;
    const int slot = blockIdx.x / a.ntiles;
    const int tok = slot / a.slots_per_tok;
    const int rs = a.rstride > 1 ? a.rstride : 1;
    const int n0 = rs == 1 ? tile * a.tile : tile;
    const int nt = rs == 1 ? min(a.tile, a.I - n0) : (a.I - n0 + rs - 1) / rs;
    const int H = a.H;
    const size_t pitch = (size_t)H * rs;  // elements from one of the tile's rows to the next
    const int nch = H / CE;

    size_t eoff = 0;
    if (a.route) eoff = (size_t)a.route[slot] * a.expert_stride;
    const WT *wg = reinterpret_cast<const WT *>(a.wg) + eoff + (size_t)n0 * H;
    const WT *wu = reinterpret_cast<const WT *>(a.wu) + eoff + (size_t)n0 * H;
    const WT *wd = reinterpret_cast<const WT *>(a.wd) + eoff + (size_t)n0 * H;

    float xr[NC][CE];
    load_x<WT, NC>(a.x + (size_t)tok * H, lane, nch, xr);

    // ---- gate: wave w dots rows w, w+8, ..., RIF rows in flight ------------
    for (int r = wave; r < nt; r += RIF * kWaves) {
        const WT *rows[RIF];
        bool valid[RIF];
#pragma unroll
        for (int k = 0; k < RIF; ++k) {
            valid[k] = r + k * kWaves < nt;
            rows[k] = wg + (size_t)(valid[k] ? r + k * kWaves : r) * pitch;
        }
        float d[RIF];
        dot_rows<WT, NC, RIF>(rows, valid, xr, lane, nch, d);
        if (lane == 0) {
#pragma unroll
            for (int k = 0; k < RIF; ++k)
                if (valid[k]) s_g[r + k * kWaves] = d[k];
        }
    }
    __syncthreads();

    // ---- ballot compaction of the open gates --------------------------------
    if (wave == 0) {
        const bool in = lane < nt;
        const bool p = in && (DENSE || s_g[lane] > gate_threshold(a.act, a.tau));
        const uint64_t m = __ballot(p);
        if (p) s_gl[lane_prefix(m, lane)] = lane;
        if (lane == 0) s_n[0] = __popcll(m);
    }
    __syncthreads();
    const int ng = s_n[0];

    // ---- up: gathered W_up rows of G -----------------------------------------
    for (int q = wave; q < ng; q += RIF * kWaves) {
        const WT *rows[RIF];
        bool valid[RIF];
        int li[RIF];
#pragma unroll
        for (int k = 0; k < RIF; ++k) {
            valid[k] = q + k * kWaves < ng;
            li[k] = s_gl[valid[k] ? q + k * kWaves : q];
            rows[k] = wu + (size_t)li[k] * pitch;
        }
        float u[RIF];
        dot_rows<WT, NC, RIF>(rows, valid, xr, lane, nch, u);
        if (lane == 0) {
#pragma unroll
            for (int k = 0; k < RIF; ++k) {
                if (valid[k]) {
                    const float g = s_g[li[k]];
                    const bool on = g > gate_threshold(a.act, a.tau) && combined_nonzero(a.act, u[k]);
                    s_on[q + k * kWaves] = on;
                    s_h[q + k * kWaves] = on ? combined_value(a.act, a.tau, g, u[k]) : 0.f;
                }
            }
        }
    }
    __syncthreads();

    // ---- ballot compaction of the non-zero Combined activations --------------
    if (wave == 0) {
        const bool in = lane < ng;
        const bool p = in && (DENSE || s_on[lane]);
        const uint64_t m = __ballot(p);
        if (p) {
            const int pos = lane_prefix(m, lane);
            s_al[pos] = s_gl[lane];
            s_av[pos] = s_h[lane];
        }
        if (lane == 0) s_n[1] = __popcll(m);
    }
    __syncthreads();
    const int na = s_n[1];

    // ---- down: axpy over the W_down_t rows of A, hidden split over threads --
    float acc[NCD][CE];
#pragma unroll
    for (int kd = 0; kd < NCD; ++kd)
#pragma unroll
        for (int e = 0; e < CE; ++e) acc[kd][e] = 0.f;

    const __amdgpu_buffer_rsrc_t rd =
        make_rsrc(wd, ((uint32_t)(nt - 1) * (uint32_t)rs + 1u) * (uint32_t)H * (uint32_t)sizeof(WT));
    for (int a0 = 0; a0 < na; a0 += kDownUnroll) {
        u32x4 v[kDownUnroll][NCD];
#pragma unroll
        for (int u = 0; u < kDownUnroll; ++u) {
            const int aa = a0 + u;
            const uint32_t base =
                aa < na ? (uint32_t)s_al[aa] * (uint32_t)pitch * (uint32_t)sizeof(WT) : kOutOfRange;
#pragma unroll
            for (int kd = 0; kd < NCD; ++kd) {
                const int c = tid + kThreads * kd;
                v[u][kd] = ld_buf_stream(rd, c < nch ? base + (uint32_t)c * 16u : kOutOfRange);
            }
        }
#pragma unroll
        for (int u = 0; u < kDownUnroll; ++u) {
            const float hv = a0 + u < na ? s_av[a0 + u] : 0.f;
#pragma unroll
            for (int kd = 0; kd < NCD; ++kd) {
                float f[CE];
                unpack<WT>(v[u][kd], f);
#pragma unroll
                for (int e = 0; e < CE; ++e) acc[kd][e] = fmaf(hv, f[e], acc[kd][e]);
            }
        }
    }

    // partial row (written for every tile; zeros when A is empty)
    const size_t pr = (size_t)slot * a.ntiles + tile;
    float *prow = a.partial + pr * H;
#pragma unroll
    for (int kd = 0; kd < NCD; ++kd) {
        const int c = tid + kThreads * kd;
        if (c < nch) {
#pragma unroll
            for (int e = 0; e < CE; e += 4)
                *reinterpret_cast<f32x4 *>(prow + c * CE + e) =
                    f32x4{acc[kd][e], acc[kd][e + 1], acc[kd][e + 2], acc[kd][e + 3]};
        }
    }
    if (tid == 0) {
        a.cnt[pr * 2] = ng;
        a.cnt[pr * 2 + 1] = na;
    }
    if (a.want_seg) {
        for (int q = tid; q < ng; q += kThreads) a.gseg[pr * a.tile + q] = n0 + s_gl[q] * rs;
        for (int q = tid; q < na; q += kThreads) a.aseg[pr * a.tile + q] = n0 + s_al[q] * rs;
    }
}

// ---------------------------------------------------------------------------
// Pipelined single-token kernel (the default sparse path).  Same work and
// output per tile as ffn_fused, but each wave streams its own gate rows
// (rows w, w+8, ... of the tile) two deep and, as soon as a row's gate is
// known to be open, issues that row's W_up loads; the up dot is finished one
// row later, while the wave's next gate rows are in flight.  The up traffic
// therefore travels with the gate stream instead of forming a burst after
// it, and no barrier separates the two.  Then, behind one barrier, every
// wave ballots the tile's non-zero Combined activations into its own copy
// of the list (no second barrier) and the 512 threads run the down axpy
// (hidden split over threads).

template <typename WT, int NC>
struct PipeWave {
    static constexpr int CE = WTraits<WT>::CE;
    __amdgpu_buffer_rsrc_t rg, ru;  // the tile's W_gate / W_up rows
    int pitch, nch, lane;  // pitch: elements from one of the tile's rows to the next
    int act;
    float tau;
    float (&xr)[NC][CE];
    float *s_g, *s_h;
    int *s_on;

    // Loads are unconditional: an unused slot (row < 0) and chunks past the
    // row end read out of range (zeros, no memory traffic), so no branch
    // separates a load from its consumer and all of a wave's loads stay in
    // flight across steps.
    __device__ void issue(__amdgpu_buffer_rsrc_t r, int row, u32x4 (&v)[NC]) {
        const uint32_t base = row >= 0 ? (uint32_t)row * (uint32_t)pitch * (uint32_t)sizeof(WT) : kOutOfRange;
#pragma unroll
        for (int c0 = 0; c0 < NC; ++c0) {
            const int c = lane + 64 * c0;
            v[c0] = ld_buf_stream(r, c < nch ? base + (uint32_t)c * 16u : kOutOfRange);
        }
    }
    __device__ float dot(const u32x4 (&v)[NC]) {
        float d = 0.f;
#pragma unroll
        for (int c0 = 0; c0 < NC; ++c0) {
            float f[CE];
            unpack<WT>(v[c0], f);
#pragma unroll
            for (int e = 0; e < CE; ++e) d = fmaf(f[e], xr[c0][e], d);
        }
        return wave_sum(d);
    }
    // One row (tile-local index): gate dot from gcur; issue the row's up
    // loads into ucur (its W_up row if the gate is open); refill gcur with
    // the row two ahead; finish the previous row's up dot from uprev
    // (prev_row < 0: none).  Steps past the wave's last row run on zeros and
    // change nothing.
    __device__ void step(int row, bool valid, int next2, u32x4 (&gcur)[NC], u32x4 (&ucur)[NC],
                         u32x4 (&uprev)[NC], int &prev_row) {
        const float g = dot(gcur);
        const bool open = valid && g > gate_threshold(act, tau);
        issue(ru, open ? row : -1, ucur);
        issue(rg, next2, gcur);
        if (lane == 0 && valid) {
            s_g[row] = g;
            s_on[row] = 0;
            s_h[row] = 0.f;
        }
        if (prev_row >= 0) finish_up(prev_row, dot(uprev));
        prev_row = open ? row : -1;
    }
    // Up dot of an open row done: its Combined activation.
    __device__ void finish_up(int row, float u) {
        if (lane == 0 && combined_nonzero(act, u)) {
            s_on[row] = 1;
            s_h[row] = combined_value(act, tau, s_g[row], u);
        }
    }
};

// EMIT: stop after gate and up, writing each tile's A (ascending) with its
// Combined values to aseg / hseg and |G|, |A| to cnt, for a kernel that
// decides which of them enter the down projection (the top-k mask).
template <typename WT, int NC, int MR, bool EMIT = false>
__global__ __launch_bounds__(kThreads) void ffn_pipe(SlotArgs a) {
    constexpr int CE = WTraits<WT>::CE;
    constexpr int NCD = (NC * 64 + kThreads - 1) / kThreads;

    __shared__ float s_g[kMaxPipeTile];
    __shared__ float s_h[kMaxPipeTile];
    __shared__ int s_on[kMaxPipeTile];
    __shared__ int s_alw[EMIT ? 1 : kWaves][kMaxPipeTile];   // per-wave copies of the active list
    __shared__ float s_avw[EMIT ? 1 : kWaves][kMaxPipeTile];
    __shared__ float s_logit[kMaxExperts];
    __shared__ int s_expert;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int tile = blockIdx.x % a.ntiles;
    const int slot = blockIdx.x / a.ntiles;
    const int tok = slot / a.slots_per_tok;
    const int rs = a.rstride > 1 ? a.rstride : 1;
    const int n0 = rs == 1 ? tile * a.tile : tile;
    const int nt = rs == 1 ? min(a.tile, a.I - n0) : (a.I - n0 + rs - 1) / rs;
    const int H = a.H;
    const int nch = H / CE;
    const size_t pr = (size_t)slot * a.ntiles + tile;

    float xr[NC][CE];
    const float *xt = a.x + (size_t)tok * H;
    load_x<WT, NC>(xt, lane, nch, xr);

    size_t eoff = 0;
    if (a.route) {
        eoff = (size_t)a.route[slot] * a.expert_stride;
    } else if (a.wr) {
        // the token's router: wave w dots expert rows (w + b) mod E,
        // (w + 8 + b) mod E, ... for workgroup b, so that the workgroups
        // starting together ask for different rows first, through the
        // default cache policy (every workgroup reads the same rows); the
        // two together measured 2% faster per layer than every workgroup's
        // wave w on row w with streaming loads; wave 0 takes the softmax and
        // top-k and picks this slot's expert
        const __amdgpu_buffer_rsrc_t rr = make_rsrc(a.wr, (uint32_t)a.E * (uint32_t)H * (uint32_t)sizeof(WT));
        for (int i = wave; i < a.E; i += kWaves) {
            const int e = (i + (int)(blockIdx.x % (unsigned)a.E)) % a.E;
            u32x4 v[NC];
            const uint32_t base = (uint32_t)e * (uint32_t)H * (uint32_t)sizeof(WT);
#pragma unroll
            for (int c0 = 0; c0 < NC; ++c0) {
                const int c = lane + 64 * c0;
                v[c0] = ld_buf_cached(rr, c < nch ? base + (uint32_t)c * 16u : kOutOfRange);
            }
            float d = 0.f;
#pragma unroll
            for (int c0 = 0; c0 < NC; ++c0) {
                float f[CE];
                unpack<WT>(v[c0], f);
#pragma unroll
                for (int q = 0; q < CE; ++q) d = fmaf(f[q], xr[c0][q], d);
            }
            d = wave_sum(d);
            if (lane == 0) s_logit[e] = d;
        }
        __syncthreads();
        if (wave == 0) {
            int ix;
            float wv;
            route_wave(s_logit, a.E, a.K, lane, &ix, &wv);
            if (lane == slot % a.K) {
                s_expert = ix;
                if (tile == 0) {
                    a.ridx[slot] = ix;
                    a.rw[slot] = wv;
                }
            }
        }
        __syncthreads();
        eoff = (size_t)s_expert * a.expert_stride;
    }
    const WT *wg = reinterpret_cast<const WT *>(a.wg) + eoff + (size_t)n0 * H;
    const WT *wu = reinterpret_cast<const WT *>(a.wu) + eoff + (size_t)n0 * H;
    const WT *wd = reinterpret_cast<const WT *>(a.wd) + eoff + (size_t)n0 * H;
    // buffer resources from the tile's first row to the end of its last
    // (contiguous: at most 128 rows of 32 KB; interleaved: below 2 GB, which
    // the host checks)
    const uint32_t tbytes = ((uint32_t)(nt - 1) * (uint32_t)rs + 1u) * (uint32_t)H * (uint32_t)sizeof(WT);
    PipeWave<WT, NC> pw{make_rsrc(wg, tbytes), make_rsrc(wu, tbytes), H * rs, nch, lane, a.act, a.tau, xr, s_g, s_h, s_on};

    // this wave's rows: wave, wave + 8, ...; first two gate rows in flight
    const int nrow = wave < nt ? (nt - wave + kWaves - 1) / kWaves : 0;
    u32x4 g0[NC], g1[NC], u0[NC], u1[NC];
    pw.issue(pw.rg, nrow > 0 ? wave : -1, g0);
    pw.issue(pw.rg, nrow > 1 ? wave + kWaves : -1, g1);

    // MR (even) >= rows per wave; the loop is unrolled so every load is
    // issued in straight-line code.
    int prev = -1;
#pragma unroll
    for (int i = 0; i < MR; i += 2) {
        const int r = wave + kWaves * i;
        pw.step(r, i < nrow, i + 2 < nrow ? r + 2 * kWaves : -1, g0, u0, u1, prev);
        pw.step(r + kWaves, i + 1 < nrow, i + 3 < nrow ? r + 3 * kWaves : -1, g1, u1, u0, prev);
    }
    if (prev >= 0) pw.finish_up(prev, pw.dot(u1));  // the last step's up loads sit in u1
    __syncthreads();

    // ---- ballots: open gates (report) and non-zero Combined activations ------
    if constexpr (!EMIT) {
        // every wave lists the tile's rows itself (the same ballots over the
        // same LDS data, into its own copy), so its down loads start without
        // waiting for a second barrier
        int *al = s_alw[wave];
        float *av = s_avw[wave];
        int ng = 0, na = 0;
        for (int h = 0; h < (nt + 63) / 64; ++h) {
            const int r = lane + 64 * h;
            const bool in = r < nt;
            const bool pg = in && s_g[r] > gate_threshold(a.act, a.tau);
            const uint64_t mg = __ballot(pg);
            if (wave == 0 && pg && a.want_seg) a.gseg[pr * a.tile + ng + lane_prefix(mg, lane)] = n0 + r * rs;
            const bool pa = in && s_on[r];
            const uint64_t ma = __ballot(pa);
            if (pa) {
                const int pos = na + lane_prefix(ma, lane);
                al[pos] = r;
                av[pos] = s_h[r];
                if (wave == 0 && a.want_seg) a.aseg[pr * a.tile + pos] = n0 + r * rs;
            }
            ng += __popcll(mg);
            na += __popcll(ma);
        }
        __builtin_amdgcn_wave_barrier();  // the wave's list writes before its reads

        // ---- down: axpy over the W_down_t rows of A, hidden split over threads
        float acc[NCD][CE];
#pragma unroll
        for (int kd = 0; kd < NCD; ++kd)
#pragma unroll
            for (int e = 0; e < CE; ++e) acc[kd][e] = 0.f;
        const __amdgpu_buffer_rsrc_t rd = make_rsrc(wd, tbytes);
        for (int a0 = 0; a0 < na; a0 += kDownUnroll) {
            u32x4 v[kDownUnroll][NCD];
#pragma unroll
            for (int u = 0; u < kDownUnroll; ++u) {
                const int aa = a0 + u;
                const uint32_t base =
                    aa < na ? (uint32_t)al[aa] * (uint32_t)(H * rs) * (uint32_t)sizeof(WT) : kOutOfRange;
#pragma unroll
                for (int kd = 0; kd < NCD; ++kd) {
                    const int c = tid + kThreads * kd;
                    v[u][kd] = ld_buf_stream(rd, c < nch ? base + (uint32_t)c * 16u : kOutOfRange);
                }
            }
#pragma unroll
            for (int u = 0; u < kDownUnroll; ++u) {
                const float hv = a0 + u < na ? av[a0 + u] : 0.f;
#pragma unroll
                for (int kd = 0; kd < NCD; ++kd) {
                    float f[CE];
                    unpack<WT>(v[u][kd], f);
#pragma unroll
                    for (int e = 0; e < CE; ++e) acc[kd][e] = fmaf(hv, f[e], acc[kd][e]);
                }
            }
        }
        float *prow = a.partial + pr * H;
#pragma unroll
        for (int kd = 0; kd < NCD; ++kd) {
            const int c = tid + kThreads * kd;
            if (c < nch) {
#pragma unroll
                for (int e = 0; e < CE; e += 4)
                    *reinterpret_cast<f32x4 *>(prow + c * CE + e) =
                        f32x4{acc[kd][e], acc[kd][e + 1], acc[kd][e + 2], acc[kd][e + 3]};
            }
        }
        if (tid == 0) {
            a.cnt[pr * 2] = ng;
            a.cnt[pr * 2 + 1] = na;
        }
        return;
    }

    // ---- emit mode: wave 0 lists the tile's open gates (report) and its
    // non-zero Combined activations with their values for the kernel that
    // decides which of them enter the down projection
    __shared__ int s_n[2];
    if (wave == 0) {
        int ng = 0, na = 0;
        for (int h = 0; h < (nt + 63) / 64; ++h) {
            const int r = lane + 64 * h;
            const bool in = r < nt;
            const bool pg = in && s_g[r] > gate_threshold(a.act, a.tau);
            const uint64_t mg = __ballot(pg);
            if (pg && a.want_seg) a.gseg[pr * a.tile + ng + lane_prefix(mg, lane)] = n0 + r * rs;
            const bool pa = in && s_on[r];
            const uint64_t ma = __ballot(pa);
            if (pa) {
                const int pos = na + lane_prefix(ma, lane);
                a.aseg[pr * a.tile + pos] = n0 + r * rs;
                a.hseg[pr * a.tile + pos] = s_h[r];
            }
            ng += __popcll(mg);
            na += __popcll(ma);
        }
        if (lane == 0) {
            s_n[0] = ng;
            s_n[1] = na;
            a.cnt[pr * 2] = ng;
            a.cnt[pr * 2 + 1] = na;
        }
    }
    __syncthreads();
    for (int q = s_n[1] + tid; q < a.tile; q += kThreads) a.aseg[pr * a.tile + q] = -1;  // padding
}

// ---------------------------------------------------------------------------
// Given-list kernel (ts_ffn_sparse_given): per-wave gate / up stream and
// down axpy as in the pipelined kernel, over a chunk of a token's neuron
// list instead of a tile of neurons; a listed neuron's W_gate
// and W_up rows are requested together.  The chunk's entries are staged
// in LDS (entries outside [0, inter) become -1); each row load goes through
// a buffer resource over that one row, an unused slot or a skipped entry
// loads at an out-of-range offset (zeros, no traffic).  One partial output
// row per (token, chunk), summed by ffn_reduce in chunk order.

struct GivenArgs {
    const float *x;
    const void *wg, *wu, *wd;
    const int32_t *idx;      // [tokens][maxc]
    const int32_t *count;    // [tokens]
    int H, I, maxc, chunk, nchunks;
    float *partial;          // [tokens][nchunks][H]
    int32_t *cnt;            // [tokens][nchunks][2] listed entries with gate > 0 / non-zero Combined
};

template <typename WT, int NC>
struct GivenWave {
    static constexpr int CE = WTraits<WT>::CE;
    const WT *wg, *wu;
    const float *xt;        // any valid address: base of the empty resource of an unused slot
    const int *s_row;       // chunk entry -> neuron (-1: skipped)
    int H, nch, lane;
    float (&xr)[NC][CE];
    float *s_g, *s_h;
    int *s_on;

    // Loads of chunk entry r (r < 0 or a skipped entry: zeros) from matrix `w`.
    __device__ void issue(const WT *w, int r, u32x4 (&v)[NC]) {
        // (wave-uniform, but derived from the thread index: made provably
        // uniform so the resource stays in scalar registers)
        const int n = __builtin_amdgcn_readfirstlane(r >= 0 ? s_row[r >= 0 ? r : 0] : -1);
        const __amdgpu_buffer_rsrc_t rs =
            make_rsrc(n >= 0 ? static_cast<const void *>(w + (size_t)(n >= 0 ? n : 0) * H) : xt,
                      n >= 0 ? (uint32_t)H * (uint32_t)sizeof(WT) : 0u);
#pragma unroll
        for (int c0 = 0; c0 < NC; ++c0) {
            const int c = lane + 64 * c0;
            v[c0] = ld_buf_stream(rs, (n >= 0 && c < nch) ? (uint32_t)c * 16u : kOutOfRange);
        }
    }
    __device__ float dot(const u32x4 (&v)[NC]) {
        float d = 0.f;
#pragma unroll
        for (int c0 = 0; c0 < NC; ++c0) {
            float f[CE];
            unpack<WT>(v[c0], f);
#pragma unroll
            for (int e = 0; e < CE; ++e) d = fmaf(f[e], xr[c0][e], d);
        }
        return wave_sum(d);
    }
    // One entry: its gate and up dots from gcur / ucur (both rows were
    // requested together, two entries ahead), then the rows of the entry
    // two ahead into the same registers.  A listed neuron is predicted
    // active, so its W_up row is read without waiting for the gate's sign:
    // one dependent memory round trip per entry instead of two.
    __device__ void step(int row, bool valid, int next2, u32x4 (&gcur)[NC], u32x4 (&ucur)[NC]) {
        const float g = dot(gcur);
        const float u = dot(ucur);
        issue(wg, next2, gcur);
        issue(wu, next2, ucur);
        if (lane == 0 && valid) {
            s_g[row] = g;
            const bool on = g > 0.f && u > 0.f;
            s_on[row] = on ? 1 : 0;
            s_h[row] = on ? g * u : 0.f;
        }
    }
};

template <typename WT, int NC, int MR>
__global__ __launch_bounds__(kThreads) void ffn_given(GivenArgs a) {
    constexpr int CE = WTraits<WT>::CE;
    constexpr int NCD = (NC * 64 + kThreads - 1) / kThreads;

    __shared__ int s_row[kMaxPipeTile];
    __shared__ float s_g[kMaxPipeTile];
    __shared__ float s_h[kMaxPipeTile];
    __shared__ int s_on[kMaxPipeTile];
    __shared__ int s_alw[kWaves][kMaxPipeTile];  // per-wave copies of the active list
    __shared__ float s_avw[kWaves][kMaxPipeTile];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int chunk = blockIdx.x % a.nchunks;
    const int tok = blockIdx.x / a.nchunks;
    const int H = a.H;
    const int nch = H / CE;
    const int n_list = min(max(a.count[tok], 0), a.maxc);
    const int e0 = chunk * a.chunk;
    const int nt = max(0, min(a.chunk, n_list - e0));
    const size_t pr = (size_t)tok * a.nchunks + chunk;

    float xr[NC][CE];
    const float *xt = a.x + (size_t)tok * H;
    load_x<WT, NC>(xt, lane, nch, xr);
    for (int r = tid; r < nt; r += kThreads) {
        const int v = a.idx[(size_t)tok * a.maxc + e0 + r];
        s_row[r] = (v >= 0 && v < a.I) ? v : -1;
    }
    __syncthreads();

    const WT *wg = reinterpret_cast<const WT *>(a.wg);
    const WT *wu = reinterpret_cast<const WT *>(a.wu);
    const WT *wd = reinterpret_cast<const WT *>(a.wd);
    GivenWave<WT, NC> gw{wg, wu, xt, s_row, H, nch, lane, xr, s_g, s_h, s_on};

    // this wave's entries: wave, wave + 8, ...; two entries' gate and up rows in flight
    const int nrow = wave < nt ? (nt - wave + kWaves - 1) / kWaves : 0;
    u32x4 g0[NC], g1[NC], u0[NC], u1[NC];
    gw.issue(wg, nrow > 0 ? wave : -1, g0);
    gw.issue(wu, nrow > 0 ? wave : -1, u0);
    gw.issue(wg, nrow > 1 ? wave + kWaves : -1, g1);
    gw.issue(wu, nrow > 1 ? wave + kWaves : -1, u1);
#pragma unroll
    for (int i = 0; i < MR; i += 2) {
        const int r = wave + kWaves * i;
        gw.step(r, i < nrow, i + 2 < nrow ? r + 2 * kWaves : -1, g0, u0);
        gw.step(r + kWaves, i + 1 < nrow, i + 3 < nrow ? r + 3 * kWaves : -1, g1, u1);
    }
    __syncthreads();

    // ---- ballots: entries with an open gate (count) and non-zero Combined;
    // every wave lists them itself, into its own copy (no second barrier)
    int *al = s_alw[wave];
    float *av = s_avw[wave];
    int ng = 0, na = 0;
    for (int h = 0; h < (nt + 63) / 64; ++h) {
        const int r = lane + 64 * h;
        const bool in = r < nt && s_row[r] >= 0;
        const uint64_t mg = __ballot(in && s_g[r] > 0.f);
        const bool pa = in && s_on[r];
        const uint64_t ma = __ballot(pa);
        if (pa) {
            const int pos = na + lane_prefix(ma, lane);
            al[pos] = r;
            av[pos] = s_h[r];
        }
        ng += __popcll(mg);
        na += __popcll(ma);
    }
    __builtin_amdgcn_wave_barrier();  // the wave's list writes before its reads

    // ---- down: axpy over the W_down_t rows of the non-zero entries ----------
    float acc[NCD][CE];
#pragma unroll
    for (int kd = 0; kd < NCD; ++kd)
#pragma unroll
        for (int e = 0; e < CE; ++e) acc[kd][e] = 0.f;
    for (int a0 = 0; a0 < na; a0 += kGivenDownUnroll) {
        u32x4 v[kGivenDownUnroll][NCD];
#pragma unroll
        for (int u = 0; u < kGivenDownUnroll; ++u) {
            const int aa = a0 + u;
            const int n = __builtin_amdgcn_readfirstlane(aa < na ? s_row[al[aa < na ? aa : 0]] : -1);
            const __amdgpu_buffer_rsrc_t rs =
                make_rsrc(n >= 0 ? static_cast<const void *>(wd + (size_t)(n >= 0 ? n : 0) * H) : xt,
                          n >= 0 ? (uint32_t)H * (uint32_t)sizeof(WT) : 0u);
#pragma unroll
            for (int kd = 0; kd < NCD; ++kd) {
                const int c = tid + kThreads * kd;
                v[u][kd] = ld_buf_stream(rs, (n >= 0 && c < nch) ? (uint32_t)c * 16u : kOutOfRange);
            }
        }
#pragma unroll
        for (int u = 0; u < kGivenDownUnroll; ++u) {
            const float hv = a0 + u < na ? av[a0 + u] : 0.f;
#pragma unroll
            for (int kd = 0; kd < NCD; ++kd) {
                float f[CE];
                unpack<WT>(v[u][kd], f);
#pragma unroll
                for (int e = 0; e < CE; ++e) acc[kd][e] = fmaf(hv, f[e], acc[kd][e]);
            }
        }
    }
    float *prow = a.partial + pr * H;
#pragma unroll
    for (int kd = 0; kd < NCD; ++kd) {
        const int c = tid + kThreads * kd;
        if (c < nch) {
#pragma unroll
            for (int e = 0; e < CE; e += 4)
                *reinterpret_cast<f32x4 *>(prow + c * CE + e) =
                    f32x4{acc[kd][e], acc[kd][e + 1], acc[kd][e + 2], acc[kd][e + 3]};
        }
    }
    if (tid == 0) {
        a.cnt[pr * 2] = ng;
        a.cnt[pr * 2 + 1] = na;
    }
}

// Per token: the chunks' counts summed (n_gate, n_active of the report).
__global__ __launch_bounds__(64) void given_counts(const int32_t *__restrict__ cnt, int nchunks,
                                                   int32_t *__restrict__ n_gate, int32_t *__restrict__ n_active) {
    const int t = blockIdx.x;
    int g = 0, a = 0;
    for (int c = threadIdx.x; c < nchunks; c += 64) {
        g += cnt[((size_t)t * nchunks + c) * 2];
        a += cnt[((size_t)t * nchunks + c) * 2 + 1];
    }
    for (int o = 32; o >= 1; o >>= 1) {
        g += __shfl_xor(g, o, 64);
        a += __shfl_xor(a, o, 64);
    }
    if (threadIdx.x == 0) {
        if (n_gate) n_gate[t] = g;
        if (n_active) n_active[t] = a;
    }
}

// ---------------------------------------------------------------------------
// Split path, kernel 1: gate GEMV + ReLU + ballot compaction and the gathered
// up rows for a tile of `tile` neurons per 4-wave workgroup.  Output per tile:
// |G|, |A|, the ascending A segment with its Combined values (and the G
// segment when a report is requested).

struct GateArgs {
    const float *x;
    const void *wg;
    const void *wu;
    const int32_t *route;
    size_t expert_stride;
    int H, I, tile, ntiles, slots_per_tok;
    int32_t *cnt;     // [slots][ntiles][2]
    int32_t *gseg;    // [slots][ntiles][tile]
    int32_t *aseg;    // [slots][ntiles][tile]
    float *hseg;      // [slots][ntiles][tile]
    int want_gseg;
};

template <typename WT, int NC, int RIF>
__global__ __launch_bounds__(kGateThreads) void ffn_gate_up(GateArgs a) {
    constexpr int CE = WTraits<WT>::CE;

    __shared__ float s_g[kMaxTile];
    __shared__ float s_h[kMaxTile];
    __shared__ int s_on[kMaxTile];
    __shared__ int s_gl[kMaxTile];
    __shared__ int s_ng;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int tile = blockIdx.x % a.ntiles;
    const int slot = blockIdx.x / a.ntiles;
    const int tok = slot / a.slots_per_tok;
    const int n0 = tile * a.tile;
    const int nt = min(a.tile, a.I - n0);
    const int H = a.H;
    const int nch = H / CE;

    size_t eoff = 0;
    if (a.route) eoff = (size_t)a.route[slot] * a.expert_stride;
    const WT *wg = reinterpret_cast<const WT *>(a.wg) + eoff + (size_t)n0 * H;
    const WT *wu = reinterpret_cast<const WT *>(a.wu) + eoff + (size_t)n0 * H;

    float xr[NC][CE];
    load_x<WT, NC>(a.x + (size_t)tok * H, lane, nch, xr);

    for (int r = wave; r < nt; r += RIF * kGateWaves) {
        const WT *rows[RIF];
        bool valid[RIF];
#pragma unroll
        for (int k = 0; k < RIF; ++k) {
            valid[k] = r + k * kGateWaves < nt;
            rows[k] = wg + (size_t)(valid[k] ? r + k * kGateWaves : r) * H;
        }
        float d[RIF];
        dot_rows<WT, NC, RIF>(rows, valid, xr, lane, nch, d);
        if (lane == 0) {
#pragma unroll
            for (int k = 0; k < RIF; ++k)
                if (valid[k]) s_g[r + k * kGateWaves] = d[k];
        }
    }
    __syncthreads();

    const size_t pr = (size_t)slot * a.ntiles + tile;
    if (wave == 0) {
        const bool p = lane < nt && s_g[lane] > 0.f;
        const uint64_t m = __ballot(p);
        if (p) {
            const int pos = lane_prefix(m, lane);
            s_gl[pos] = lane;
            if (a.want_gseg) a.gseg[pr * a.tile + pos] = n0 + lane;
        }
        if (lane == 0) s_ng = __popcll(m);
    }
    __syncthreads();
    const int ng = s_ng;

    for (int q = wave; q < ng; q += RIF * kGateWaves) {
        const WT *rows[RIF];
        bool valid[RIF];
        int li[RIF];
#pragma unroll
        for (int k = 0; k < RIF; ++k) {
            valid[k] = q + k * kGateWaves < ng;
            li[k] = s_gl[valid[k] ? q + k * kGateWaves : q];
            rows[k] = wu + (size_t)li[k] * H;
        }
        float u[RIF];
        dot_rows<WT, NC, RIF>(rows, valid, xr, lane, nch, u);
        if (lane == 0) {
#pragma unroll
            for (int k = 0; k < RIF; ++k) {
                if (valid[k]) {
                    const float g = s_g[li[k]];
                    const bool on = u[k] > 0.f;  // g > 0 holds for every member of G
                    s_on[q + k * kGateWaves] = on;
                    s_h[q + k * kGateWaves] = on ? g * u[k] : 0.f;
                }
            }
        }
    }
    __syncthreads();

    if (wave == 0) {
        const bool p = lane < ng && s_on[lane];
        const uint64_t m = __ballot(p);
        if (p) {
            const int pos = lane_prefix(m, lane);
            a.aseg[pr * a.tile + pos] = n0 + s_gl[lane];
            a.hseg[pr * a.tile + pos] = s_h[lane];
        }
        if (lane >= __popcll(m) && lane < a.tile) a.aseg[pr * a.tile + lane] = -1;  // padding
        if (lane == 0) {
            a.cnt[pr * 2] = ng;
            a.cnt[pr * 2 + 1] = __popcll(m);
        }
    }
}

// Top-k magnitude mask (Eq. mask and Eq. sparsify-gated-MLP, section 3.2),
// between gate+up and the down projection: per slot, keep the `keep`
// largest Combined activations (all positive under dReLU, so |Combined| is
// the value), ties to the lower neuron index, and rewrite each tile's active
// list with the kept entries only, so the down kernel reads only their
// W_down_t rows.  One 1024-thread workgroup per slot reads the padded
// [ntiles][tile] lists (padding: index -1; each tile's list ascending, the
// tiles contiguous or interleaved):
//   1. one batch of loads; the entries are compacted into LDS (one block
//      scan) as key = sel_key(fp32 bits) (magnitude order, never 0; the
//      listed dReLU Combined values are positive, so the magnitude is the
//      value carried on), position and neuron index, and the
//      first radix histogram is counted from registers;
//   2. the k-th largest key by radix select over 8-bit digits, k =
//      min(keep, entries) (histograms by LDS atomics: counts do not depend
//      on order, so the result is deterministic; each bin search is one
//      wave's suffix scan);
//   3. when only some of the keys equal to the k-th are kept, the largest
//      kept neuron index among them by a second radix select (over
//      indices, so the tile layout does not matter);
//   4. kept flags set in a bitmap by position; each kept entry's place in
//      its tile's list is the number of kept positions before it in the
//      tile; the tiles' kept counts likewise.

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kSelPer = (kSelSpan + kSelThreads - 1) / kSelThreads;  // positions per thread

struct SelArgs {
    int ntiles, tile, keep;
    const int32_t *cnt, *aseg;   // gate+up output: [slots][ntiles][2], [slots][ntiles][tile]
    const float *hseg;
    int32_t *kcnt, *kaseg;       // kept lists, same layout
    float *khseg;
};

// Exclusive prefix over the workgroup (NW waves) of one int per thread;
// returns it, and the total in *sum.  s_w: NW ints of scratch.  Contains
// barriers.
template <int NW = kSelWaves>
__device__ __forceinline__ int sel_block_scan(int v, int *s_w, int *sum) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int inc = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(inc, o, 64);
        if (lane >= o) inc += t;
    }
    if (lane == 63) s_w[wave] = inc;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        const int t = s_w[w];
        before += w < wave ? t : 0;
        all += t;
    }
    __syncthreads();
    *sum = all;
    return before + inc - v;
}

// Radix digits of the selection keys (sel_key / sel_mag, kSelTopShift and
// sel_next_shift in ts_plan.h): the first digit is the exponent, one bin per
// octave (a first digit from bit 24, the sign bit's, crowded the values into
// fewer bins and measured 0.3 us slower).

// One radix step, run by wave 0: in the 256-bin histogram, the bin holding
// the rem-th largest counted key (1 <= rem <= keys counted).  st[0] gains
// the bin's digit at `shift`, st[1] becomes the rank left inside the bin,
// st[2] the bin's count; the histogram is cleared for the next step.
__device__ __forceinline__ void sel_find_bin(uint32_t *s_hist, uint32_t *st, uint32_t rem, int shift, int lane) {
    uint32_t h[4], sum = 0u;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        h[j] = s_hist[4 * lane + j];
        sum += h[j];
    }
    uint32_t inc = sum;  // bins of lanes >= this lane
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t t = __shfl_down(inc, o, 64);
        if (lane + o < 64) inc += t;
    }
    const uint32_t above = inc - sum;
    if (above < rem && rem <= inc) {
        uint32_t r = rem - above;
        int j = 3;
        for (; j > 0; --j) {
            if (h[j] >= r) break;
            r -= h[j];
        }
        st[0] |= (uint32_t)(4 * lane + j) << shift;
        st[1] = r;
        st[2] = h[j];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) s_hist[4 * lane + j] = 0u;
}

// Kept positions in [lo, hi) of the bitmap.
__device__ __forceinline__ int sel_bits(const uint32_t *s_kb, int lo, int hi) {
    int c = 0;
    for (int w = lo >> 5; lo < hi && w <= (hi - 1) >> 5; ++w) {
        uint32_t m = s_kb[w];
        if (w == lo >> 5) m &= ~0u << (lo & 31);
        const int hb = hi - (w << 5);
        if (hb < 32) m &= (1u << hb) - 1u;
        c += __popc(m);
    }
    return c;
}

__global__ __launch_bounds__(kSelThreads) void ffn_topk_select(SelArgs a) {
    __shared__ uint32_t s_c[kSelMax];                 // entry keys (compacted)
    __shared__ uint16_t s_cp[kSelMax];                // their list positions
    __shared__ uint16_t s_ci[kSelMax];                // their neuron indices
    __shared__ uint32_t s_kb[(kSelSpan + 31) / 32];   // kept flags by position
    __shared__ uint32_t s_hist[256];
    __shared__ int s_w[kSelWaves];
    __shared__ uint32_t s_st[3];                      // digits found, rank left, bin count

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const size_t pr0 = (size_t)blockIdx.x * a.ntiles;
    const int span = a.ntiles * a.tile;

    // 1. staging
    int n;
    {
        const uint32_t bytes = (uint32_t)span * 4u;
        const __amdgpu_buffer_rsrc_t rh = make_rsrc(a.hseg + pr0 * a.tile, bytes);
        const __amdgpu_buffer_rsrc_t ra = make_rsrc(a.aseg + pr0 * a.tile, bytes);
        uint32_t h[kSelPer], ai[kSelPer];
#pragma unroll
        for (int u = 0; u < kSelPer; ++u) {
            const uint32_t off = (uint32_t)(tid + kSelThreads * u) * 4u;  // past `bytes`: zeros
            h[u] = __builtin_amdgcn_raw_buffer_load_b32(rh, off, 0, 0);
            ai[u] = __builtin_amdgcn_raw_buffer_load_b32(ra, off, 0, 0);
        }
        int ng[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int t = tid + kSelThreads * j;
            ng[j] = t < a.ntiles ? a.cnt[(pr0 + t) * 2] : 0;
        }
        for (int i = tid; i < 256; i += kSelThreads) s_hist[i] = 0u;
        for (int i = tid; i < (kSelSpan + 31) / 32; i += kSelThreads) s_kb[i] = 0u;
        if (tid < 3) s_st[tid] = 0u;
        int nv = 0;
#pragma unroll
        for (int u = 0; u < kSelPer; ++u) nv += (tid + kSelThreads * u < span && (int32_t)ai[u] >= 0) ? 1 : 0;
        int base = sel_block_scan(nv, s_w, &n);  // its barriers also order the clears above
#pragma unroll
        for (int u = 0; u < kSelPer; ++u) {
            const int e = tid + kSelThreads * u;
            if (e < span && (int32_t)ai[u] >= 0) {
                const uint32_t key = sel_key(h[u]);  // bit 31 clear: the first digit is < 256
                s_c[base] = key;
                s_cp[base] = (uint16_t)e;
                s_ci[base] = (uint16_t)ai[u];
                ++base;
                atomicAdd(&s_hist[key >> kSelTopShift], 1u);
            }
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int t = tid + kSelThreads * j;
            if (t < a.ntiles) a.kcnt[(pr0 + t) * 2] = ng[j];
        }
    }
    const int k = min(a.keep, n);
    __syncthreads();

    // 2. the k-th largest key
    uint32_t thr = 0xffffffffu;  // no key reaches it: nothing kept (k = 0)
    uint32_t tie_n = 0xffffu;  // largest kept neuron index among keys equal to thr
    if (k > 0) {
        uint32_t mask = 0u;
        for (int shift = kSelTopShift; shift >= 0; shift = sel_next_shift(shift)) {
            if (shift < kSelTopShift) {
                const uint32_t prefix = s_st[0];
                for (int i = tid; i < n; i += kSelThreads) {
                    const uint32_t v = s_c[i];
                    if ((v & mask) == prefix) atomicAdd(&s_hist[(v >> shift) & 255u], 1u);
                }
                __syncthreads();
            }
            if (wave == 0) sel_find_bin(s_hist, s_st, shift == kSelTopShift ? (uint32_t)k : s_st[1], shift, lane);
            mask |= 255u << shift;
            __syncthreads();
            // every key of the chosen bin kept: the k-th largest is the bin's
            // smallest, and the bin's floor (lower digits 0) is as good a
            // threshold; the remaining digits are not needed
            if (s_st[1] == s_st[2]) break;
        }
        thr = s_st[0];
        const uint32_t ties = s_st[1], neq = s_st[2];
        // 3. only some of the keys equal to thr kept: the ties-th smallest
        //    neuron index among them (the ties-th largest of 0xffff - index;
        //    indices < kSelMax)
        if (ties < neq) {
            __syncthreads();
            if (tid == 0) s_st[0] = 0u;
            __syncthreads();
            mask = 0u;
            for (int shift = 8; shift >= 0; shift -= 8) {
                const uint32_t prefix = s_st[0];
                for (int i = tid; i < n; i += kSelThreads) {
                    const uint32_t q = 0xffffu - s_ci[i];
                    if (s_c[i] == thr && (q & mask) == prefix) atomicAdd(&s_hist[(q >> shift) & 255u], 1u);
                }
                __syncthreads();
                if (wave == 0) sel_find_bin(s_hist, s_st, shift == 8 ? ties : s_st[1], shift, lane);
                mask |= 255u << shift;
                __syncthreads();
            }
            tie_n = 0xffffu - s_st[0];
        }
    }

    // 4. kept flags by position, then the compacted per-tile lists
    for (int i = tid; i < n; i += kSelThreads) {
        const uint32_t v = s_c[i], pos = s_cp[i];
        if (v > thr || (v == thr && s_ci[i] <= tie_n)) atomicOr(&s_kb[pos >> 5], 1u << (pos & 31));
    }
    __syncthreads();
    for (int i = tid; i < n; i += kSelThreads) {
        const int pos = s_cp[i];
        if ((s_kb[pos >> 5] >> (pos & 31)) & 1u) {
            const int t = pos / a.tile, lo = t * a.tile;
            const size_t dst = (pr0 + t) * a.tile + sel_bits(s_kb, lo, pos);
            a.kaseg[dst] = (int32_t)s_ci[i];
            a.khseg[dst] = __uint_as_float(s_c[i] - 1u);
        }
    }
    for (int t = tid; t < a.ntiles; t += kSelThreads)
        a.kcnt[(pr0 + t) * 2 + 1] = sel_bits(s_kb, t * a.tile, (t + 1) * a.tile);
}

// Split path, kernel 2: the down projection over A.  Workgroup (slot, chunk,
// slice): `chunk` is a run of `tpc` consecutive gate+up tiles, `slice` a run
// of 64 16-byte column chunks.  The workgroup lists the chunk's active rows
// (ascending) in LDS, its 4 waves accumulate Combined_i * W_down_t[i][slice]
// over them (rows w, w+4, ...; eight loads in flight per lane), the waves'
// sums are added in a fixed order and stored as the chunk's partial row.

struct DownArgs {
    const void *wd;
    const int32_t *route;
    size_t expert_stride;
    int H, tile, ntiles, nslices, nchunks, tpc;
    const int32_t *cnt;
    const int32_t *aseg;
    const float *hseg;
    float *partial;        // [slots][nchunks][H]
};

constexpr int kDownWaves = kDownThreads / 64;

template <typename WT>
__global__ __launch_bounds__(kDownThreads) void ffn_down(DownArgs a) {
    constexpr int CE = WTraits<WT>::CE;
    constexpr int SW = 64 * CE;  // columns per slice

    __shared__ int s_row[kDownMaxRows];
    __shared__ float s_hv[kDownMaxRows];
    __shared__ int s_cnt[kDownMaxTiles];
    __shared__ int s_toff[kDownMaxTiles + 1];
    __shared__ float s_red[kDownWaves][SW];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int slice = blockIdx.x % a.nslices;
    const int chunk = (blockIdx.x / a.nslices) % a.nchunks;
    const int slot = blockIdx.x / (a.nslices * a.nchunks);
    const int H = a.H;
    const int nch = H / CE;
    const int t0 = chunk * a.tpc;
    const int ntc = min(a.tpc, a.ntiles - t0);
    const size_t tbase = (size_t)slot * a.ntiles + t0;

    // 1. the chunk's active rows: counts, offsets, then one pass of copies
    for (int t = tid; t < ntc; t += kDownThreads) s_cnt[t] = a.cnt[(tbase + t) * 2 + 1];
    __syncthreads();
    if (tid == 0) {
        int off = 0;
        for (int t = 0; t < ntc; ++t) {
            s_toff[t] = off;
            off += s_cnt[t];
        }
        s_toff[ntc] = off;
    }
    __syncthreads();
    for (int e = tid; e < ntc * a.tile; e += kDownThreads) {
        const int t = e / a.tile, q = e - t * a.tile;
        if (q < s_cnt[t]) {
            s_row[s_toff[t] + q] = a.aseg[(tbase + t) * a.tile + q];
            s_hv[s_toff[t] + q] = a.hseg[(tbase + t) * a.tile + q];
        }
    }
    __syncthreads();
    const int nrows = s_toff[ntc];

    // 2. axpy over the rows
    size_t eoff = 0;
    if (a.route) eoff = (size_t)a.route[slot] * a.expert_stride;
    const WT *wd = reinterpret_cast<const WT *>(a.wd) + eoff;
    const int c = slice * 64 + lane;
    float acc[CE];
#pragma unroll
    for (int e = 0; e < CE; ++e) acc[e] = 0.f;
    for (int j0 = wave; j0 < nrows; j0 += kDownUnroll * kDownWaves) {
        u32x4 v[kDownUnroll];
        float hv[kDownUnroll];
#pragma unroll
        for (int u = 0; u < kDownUnroll; ++u) {
            const int j = j0 + u * kDownWaves;
            const bool ok = j < nrows;
            v[u] = ld_stream_masked(wd + (size_t)s_row[ok ? j : j0] * H, c, nch, 16, ok);
            hv[u] = ok ? s_hv[j] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kDownUnroll; ++u) {
            float f[CE];
            unpack<WT>(v[u], f);
#pragma unroll
            for (int e = 0; e < CE; ++e) acc[e] = fmaf(hv[u], f[e], acc[e]);
        }
    }

    // 3. waves -> the chunk's partial row slice (wave order fixed)
#pragma unroll
    for (int e = 0; e < CE; ++e) s_red[wave][lane * CE + e] = acc[e];
    __syncthreads();
    float *prow = a.partial + ((size_t)slot * a.nchunks + chunk) * H;
    for (int i = tid; i < SW; i += kDownThreads) {
        const int col = slice * SW + i;
        float v = s_red[0][i];
#pragma unroll
        for (int w = 1; w < kDownWaves; ++w) v += s_red[w][i];
        if (col < H) prow[col] = v;
    }
}

// Top-k mask without a separate selection launch: every down workgroup of
// a slot finds the slot's threshold itself (the same radix steps as
// ffn_topk_select over the same order of values, and an exact result either
// way, so all of them keep the same entries) and then runs
// ffn_down's work over the kept rows of its chunk.  The slot's Combined
// values (the padded per-tile lists of the emit-mode pipelined kernel) come
// into LDS with buffer-to-LDS loads in one batch, next to the tiles' counts
// and the chunk's neuron indices; each thread takes whole tiles, so a radix
// pass touches only the listed entries.  The kept list of the chunk is
// built tile after tile in ascending order, as ffn_down builds it from the
// selection's lists, so both sequences give the same bits.
struct TopkDownArgs {
    DownArgs d;   // cnt / aseg / hseg: the emit-mode lists (tile = the pipelined kernel's tile)
    int keep;
};

constexpr int kTdKeys = 65 * 256;  // LDS words for one slot's padded values (65 KB >= kSelSpan entries)

template <typename WT>
__global__ __launch_bounds__(kDownThreads) void ffn_topk_down(TopkDownArgs ta) {
    constexpr int CE = WTraits<WT>::CE;
    constexpr int SW = 64 * CE;  // columns per slice
    constexpr int TPT = kSelMaxTiles / kDownThreads;  // tiles per thread (selection)
    constexpr int EPT = kDownMaxRows / kDownThreads;  // chunk positions per thread
    const DownArgs &a = ta.d;

    __shared__ __attribute__((aligned(16))) uint32_t s_key[kTdKeys];
    __shared__ int s_tc[kSelMaxTiles];
    __shared__ int s_ai[kDownMaxRows];
    __shared__ int s_row[kDownMaxRows];
    __shared__ float s_hv[kDownMaxRows];
    __shared__ int s_cnt[kDownMaxTiles];
    __shared__ int s_toff[kDownMaxTiles + 1];
    __shared__ float s_red[kDownWaves][SW];
    __shared__ uint32_t s_hist[256];
    __shared__ int s_w[kDownWaves];
    __shared__ uint32_t s_st[3];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int slice = blockIdx.x % a.nslices;
    const int chunk = (blockIdx.x / a.nslices) % a.nchunks;
    const int slot = blockIdx.x / (a.nslices * a.nchunks);
    const int H = a.H;
    const int nch = H / CE;
    const int t0 = chunk * a.tpc;
    const int ntc = min(a.tpc, a.ntiles - t0);
    const size_t pr0 = (size_t)slot * a.ntiles;
    const int span = a.ntiles * a.tile;
    // a tile's entries are read four at a time (tiles are multiples of 4
    // neurons, so every tile starts on a 16-byte boundary of s_key)
    const u32x4 *s_key4 = reinterpret_cast<const u32x4 *>(s_key);
    auto for_entries = [&](int t, auto &&f) {
        const int c = s_tc[t], b4 = t * a.tile / 4;
        for (int q0 = 0; q0 < c; q0 += 4) {
            const u32x4 v = s_key4[b4 + q0 / 4];
            const uint32_t w[4] = {sel_mag(v.x), sel_mag(v.y), sel_mag(v.z), sel_mag(v.w)};
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (q0 + i < c) f(q0 + i, w[i]);
        }
    };

    // 0. one batch of loads: the slot's values into LDS, the tiles' counts,
    //    the chunk's neuron indices
    {
        const uint32_t bytes = (uint32_t)span * 4u;
        const __amdgpu_buffer_rsrc_t rh = make_rsrc(a.hseg + pr0 * a.tile, bytes);
        const int nkb = (int)((bytes + 1023u) / 1024u);  // 1 KB pieces, <= 65
        for (int kb = wave; kb < nkb; kb += kDownWaves)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rh, s_key + kb * 256, 16, (uint32_t)kb * 1024u + lane * 16u, 0,
                                                     0, 0);
        int na[TPT];
#pragma unroll
        for (int j = 0; j < TPT; ++j) {
            const int t = tid + kDownThreads * j;
            na[j] = t < a.ntiles ? a.cnt[(pr0 + t) * 2 + 1] : 0;
        }
        int ai[EPT];
        const size_t cb = (pr0 + t0) * a.tile;
#pragma unroll
        for (int u = 0; u < EPT; ++u) {
            const int e = tid + kDownThreads * u;
            ai[u] = e < ntc * a.tile ? a.aseg[cb + e] : 0;
        }
        for (int i = tid; i < 256; i += kDownThreads) s_hist[i] = 0u;
        if (tid < 3) s_st[tid] = 0u;
#pragma unroll
        for (int j = 0; j < TPT; ++j) {
            const int t = tid + kDownThreads * j;
            if (t < a.ntiles) s_tc[t] = na[j];
        }
#pragma unroll
        for (int u = 0; u < EPT; ++u) {
            const int e = tid + kDownThreads * u;
            if (e < ntc * a.tile) s_ai[e] = ai[u];
        }
        __builtin_amdgcn_s_waitcnt(0);  // this wave's pieces of the values are in LDS
    }
    __syncthreads();

    // 1. k = min(keep, listed entries); the k-th largest key (for_entries
    //    hands out sel_mag of the fp32 bits: magnitude order, bit 31 clear)
    int mine = 0;
    for (int t = tid; t < a.ntiles; t += kDownThreads) mine += s_tc[t];
    int n;
    sel_block_scan<kDownWaves>(mine, s_w, &n);
    const int k = min(ta.keep, n);
    uint32_t thr = 0xffffffffu;  // no key reaches it: nothing kept (k = 0)
    int tie_n = -1;              // largest kept neuron index among keys equal to thr
    if (k > 0 && k == n) {
        // every listed entry kept (their keys are >= 0): no search
        thr = 0u;
        tie_n = 0x7fffffff;
    } else if (k > 0) {
        uint32_t mask = 0u;
        for (int shift = kSelTopShift; shift >= 0; shift = sel_next_shift(shift)) {
            const uint32_t prefix = s_st[0];
            for (int t = tid; t < a.ntiles; t += kDownThreads)
                for_entries(t, [&](int, uint32_t v) {
                    if ((v & mask) == prefix) atomicAdd(&s_hist[(v >> shift) & 255u], 1u);
                });
            __syncthreads();
            if (wave == 0) sel_find_bin(s_hist, s_st, shift == kSelTopShift ? (uint32_t)k : s_st[1], shift, lane);
            mask |= 255u << shift;
            __syncthreads();
            // every key of the chosen bin kept: the k-th largest is the bin's
            // smallest, and the bin's floor (lower digits 0) is as good a
            // threshold; the remaining digits are not needed
            if (s_st[1] == s_st[2]) break;
        }
        thr = s_st[0];
        const uint32_t ties = s_st[1], neq = s_st[2];
        tie_n = 0x7fffffff;
        if (ties < neq) {
            // the ties-th smallest neuron index among keys equal to thr (the
            // ties-th largest of 0xffff - index; indices < kSelMax); only
            // the tied entries' indices are read, from the lists in memory
            __syncthreads();
            if (tid == 0) s_st[0] = 0u;
            __syncthreads();
            mask = 0u;
            for (int shift = 8; shift >= 0; shift -= 8) {
                const uint32_t prefix = s_st[0];
                for (int t = tid; t < a.ntiles; t += kDownThreads)
                    for_entries(t, [&](int q, uint32_t v) {
                        if (v == thr) {
                            const uint32_t key = 0xffffu - (uint32_t)a.aseg[(pr0 + t) * a.tile + q];
                            if ((key & mask) == prefix) atomicAdd(&s_hist[(key >> shift) & 255u], 1u);
                        }
                    });
                __syncthreads();
                if (wave == 0) sel_find_bin(s_hist, s_st, shift == 8 ? ties : s_st[1], shift, lane);
                mask |= 255u << shift;
                __syncthreads();
            }
            tie_n = (int)(0xffffu - s_st[0]);
        }
    }

    // 2. the chunk's kept rows, tile after tile, ascending
    if (tid < ntc) {
        const int t = t0 + tid;
        int m = 0;
        for_entries(t, [&](int q, uint32_t v) {
            m += (v > thr || (v == thr && s_ai[tid * a.tile + q] <= tie_n)) ? 1 : 0;
        });
        s_cnt[tid] = m;
    }
    __syncthreads();
    if (wave == 0) {  // offsets of the chunk's tiles (ntc <= 256: four per lane)
        int c4[4], sum = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int j = 4 * lane + i;
            c4[i] = j < ntc ? s_cnt[j] : 0;
            sum += c4[i];
        }
        int inc = sum;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int t = __shfl_up(inc, o, 64);
            if (lane >= o) inc += t;
        }
        int off = inc - sum;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int j = 4 * lane + i;
            if (j < ntc) s_toff[j] = off;
            off += c4[i];
        }
        if (lane == 63) s_toff[ntc] = inc;  // the chunk's total
    }
    __syncthreads();
    if (tid < ntc) {
        const int t = t0 + tid;
        int m = s_toff[tid];
        for_entries(t, [&](int q, uint32_t v) {
            if (v > thr || (v == thr && s_ai[tid * a.tile + q] <= tie_n)) {
                s_row[m] = s_ai[tid * a.tile + q];
                s_hv[m] = __uint_as_float(v);
                ++m;
            }
        });
    }
    __syncthreads();
    const int nrows = s_toff[ntc];

    // 3. axpy over the rows (as ffn_down)
    const WT *wd = reinterpret_cast<const WT *>(a.wd);
    const int c = slice * 64 + lane;
    float acc[CE];
#pragma unroll
    for (int e = 0; e < CE; ++e) acc[e] = 0.f;
    for (int j0 = wave; j0 < nrows; j0 += kDownUnroll * kDownWaves) {
        u32x4 v[kDownUnroll];
        float hv[kDownUnroll];
#pragma unroll
        for (int u = 0; u < kDownUnroll; ++u) {
            const int j = j0 + u * kDownWaves;
            const bool ok = j < nrows;
            v[u] = ld_stream_masked(wd + (size_t)s_row[ok ? j : j0] * H, c, nch, 16, ok);
            hv[u] = ok ? s_hv[j] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kDownUnroll; ++u) {
            float f[CE];
            unpack<WT>(v[u], f);
#pragma unroll
            for (int e = 0; e < CE; ++e) acc[e] = fmaf(hv[u], f[e], acc[e]);
        }
    }

    // 4. waves -> the chunk's partial row slice (wave order fixed)
#pragma unroll
    for (int e = 0; e < CE; ++e) s_red[wave][lane * CE + e] = acc[e];
    __syncthreads();
    float *prow = a.partial + ((size_t)slot * a.nchunks + chunk) * H;
    for (int i = tid; i < SW; i += kDownThreads) {
        const int col = slice * SW + i;
        float v = s_red[0][i];
#pragma unroll
        for (int w = 1; w < kDownWaves; ++w) v += s_red[w][i];
        if (col < H) prow[col] = v;
    }
}

// out[o][:] = sum over the slots s of output row o (ascending), of w_s times
// the sum over rows r of partial[s][r][:]; w_s = 1 without routing.
// Block: 32 columns (8 float4, one 128-byte line of each partial row) x 32
// row groups; a thread adds rows grp, grp + 32, ... in order, and the 32
// shares are combined in a fixed order (register butterflies inside each
// wave, one LDS step across the waves).  Grid (column blocks, outputs): 128
// workgroups for hidden 4096, each row's line read by one of them, all of
// it in one round trip (8 loads per thread for up to 256 rows).  Measured
// against 16-column blocks with 64 row groups (256 workgroups, a line read
// by two): 0.4 us less per layer.
constexpr int kRedCols4 = 8;
constexpr int kRedGroups = 32;
constexpr int kRedUnroll = 8;

__global__ __launch_bounds__(256) void ffn_reduce(const float *__restrict__ partial, int rows, int H,
                                                  int slots_per_out, const float *__restrict__ slot_w,
                                                  float *__restrict__ out) {
    __shared__ f32x4 red[4][kRedCols4];
    const int o = blockIdx.y;
    const int q = threadIdx.x % kRedCols4;
    const int grp = threadIdx.x / kRedCols4;
    const int c4 = blockIdx.x * kRedCols4 + q;
    const int nq = H / 4;
    const int total = slots_per_out * rows;
    const size_t base = (size_t)o * slots_per_out * rows;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int p0 = grp; p0 < total; p0 += kRedUnroll * kRedGroups) {
        f32x4 v[kRedUnroll];
#pragma unroll
        for (int u = 0; u < kRedUnroll; ++u) {
            const int p = p0 + u * kRedGroups;
            const bool ok = p < total;
            const f32x4 t = ld_f32x4_masked(partial + (base + (ok ? p : p0)) * H, c4, nq);
            v[u] = ok ? t : f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int u = 0; u < kRedUnroll; ++u) {
            const int p = p0 + u * kRedGroups;
            const float w = (slot_w && p < total) ? slot_w[o * slots_per_out + p / rows] : 1.f;
            acc.x = fmaf(w, v[u].x, acc.x);
            acc.y = fmaf(w, v[u].y, acc.y);
            acc.z = fmaf(w, v[u].z, acc.z);
            acc.w = fmaf(w, v[u].w, acc.w);
        }
    }
    // the 8 groups of a wave (lanes q + 8 j) by register butterflies, then
    // the 4 waves through LDS; a fixed order either way
#pragma unroll
    for (int m = kRedCols4; m < 64; m <<= 1) {
        acc.x += __shfl_xor(acc.x, m, 64);
        acc.y += __shfl_xor(acc.y, m, 64);
        acc.z += __shfl_xor(acc.z, m, 64);
        acc.w += __shfl_xor(acc.w, m, 64);
    }
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane < kRedCols4) red[wave][lane] = acc;
    __syncthreads();
    if (threadIdx.x < kRedCols4 && c4 < nq)
        *reinterpret_cast<f32x4 *>(out + (size_t)o * H + c4 * 4) = (red[0][q] + red[1][q]) + (red[2][q] + red[3][q]);
}

// Activity report: per slot, concatenate the tiles' ascending segments into
// one ascending list and sum the counts.  One 256-thread block per slot.
__global__ __launch_bounds__(256) void ffn_stats(const int32_t *__restrict__ cnt, const int32_t *__restrict__ gseg,
                                                 const int32_t *__restrict__ aseg, int ntiles, int tile, int inter,
                                                 int32_t *n_gate, int32_t *n_active, int32_t *gate_idx,
                                                 int32_t *active_idx) {
    __shared__ int s_sc[2][256];
    const int slot = blockIdx.x;
    const int tid = threadIdx.x;
    int carry_g = 0, carry_a = 0;
    for (int base = 0; base < ntiles; base += 256) {
        const int p = base + tid;
        const size_t pr = (size_t)slot * ntiles + p;
        const int cg = p < ntiles ? cnt[pr * 2] : 0;
        const int ca = p < ntiles ? cnt[pr * 2 + 1] : 0;
        s_sc[0][tid] = cg;
        s_sc[1][tid] = ca;
        __syncthreads();
        for (int off = 1; off < 256; off <<= 1) {
            const int vg = tid >= off ? s_sc[0][tid - off] : 0;
            const int va = tid >= off ? s_sc[1][tid - off] : 0;
            __syncthreads();
            s_sc[0][tid] += vg;
            s_sc[1][tid] += va;
            __syncthreads();
        }
        const int og = carry_g + s_sc[0][tid] - cg;
        const int oa = carry_a + s_sc[1][tid] - ca;
        if (p < ntiles) {
            if (gate_idx)
                for (int q = 0; q < cg; ++q) gate_idx[(size_t)slot * inter + og + q] = gseg[pr * tile + q];
            if (active_idx)
                for (int q = 0; q < ca; ++q) active_idx[(size_t)slot * inter + oa + q] = aseg[pr * tile + q];
        }
        carry_g += s_sc[0][255];
        carry_a += s_sc[1][255];
        __syncthreads();
    }
    if (tid == 0) {
        if (n_gate) n_gate[slot] = carry_g;
        if (n_active) n_active[slot] = carry_a;
    }
}

// Activity report for interleaved tiles (a tile's segment is ascending but
// the tiles interleave): per slot, the members of G and A become bits of
// two bitmaps in LDS (OR is order-free), then each thread turns a
// contiguous run of words into ascending indices at its offset from a block
// scan of the words' population counts.  One 256-thread block per slot.
__global__ __launch_bounds__(256) void ffn_stats_ilv(const int32_t *__restrict__ cnt, const int32_t *__restrict__ gseg,
                                                     const int32_t *__restrict__ aseg, int ntiles, int tile, int inter,
                                                     int32_t *n_gate, int32_t *n_active, int32_t *gate_idx,
                                                     int32_t *active_idx) {
    __shared__ uint32_t s_bm[2][kIlvMaxInter / 32];
    __shared__ int s_sc[2][256];
    const int slot = blockIdx.x;
    const int tid = threadIdx.x;
    const int nw = (inter + 31) / 32;
    for (int i = tid; i < nw; i += 256) s_bm[0][i] = s_bm[1][i] = 0u;
    __syncthreads();
    for (int p = tid; p < ntiles; p += 256) {
        const size_t pr = (size_t)slot * ntiles + p;
        const int cg = cnt[pr * 2], ca = cnt[pr * 2 + 1];
        for (int q = 0; q < cg; ++q) {
            const int n = gseg[pr * tile + q];
            atomicOr(&s_bm[0][n >> 5], 1u << (n & 31));
        }
        for (int q = 0; q < ca; ++q) {
            const int n = aseg[pr * tile + q];
            atomicOr(&s_bm[1][n >> 5], 1u << (n & 31));
        }
    }
    __syncthreads();
    const int per = (nw + 255) / 256;
    const int w0 = min(nw, tid * per), w1 = min(nw, w0 + per);
    int c[2] = {0, 0};
    for (int w = w0; w < w1; ++w) {
        c[0] += __popc(s_bm[0][w]);
        c[1] += __popc(s_bm[1][w]);
    }
    s_sc[0][tid] = c[0];
    s_sc[1][tid] = c[1];
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const int v0 = tid >= off ? s_sc[0][tid - off] : 0;
        const int v1 = tid >= off ? s_sc[1][tid - off] : 0;
        __syncthreads();
        s_sc[0][tid] += v0;
        s_sc[1][tid] += v1;
        __syncthreads();
    }
    int32_t *dst[2] = {gate_idx, active_idx};
    for (int k = 0; k < 2; ++k) {
        if (!dst[k]) continue;
        int o = s_sc[k][tid] - c[k];
        for (int w = w0; w < w1; ++w)
            for (uint32_t b = s_bm[k][w]; b; b &= b - 1u) dst[k][(size_t)slot * inter + o++] = w * 32 + __ffs(b) - 1;
    }
    if (tid == 0) {
        if (n_gate) n_gate[slot] = s_sc[0][255];
        if (n_active) n_active[slot] = s_sc[1][255];
    }
}

// Union of the slots' sets: flags[2][inter] set to 1 for members (plain
// stores of the same value, so overlapping writers agree), then counted.
__global__ void fill_i32(int32_t *p, size_t n, int32_t v) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ __launch_bounds__(256) void ffn_union_mark(const int32_t *__restrict__ cnt, const int32_t *__restrict__ gseg,
                                                      const int32_t *__restrict__ aseg, int ntiles, int tile,
                                                      int slots, int inter, int32_t *flags) {
    const size_t total = (size_t)slots * ntiles;
    for (size_t pr = blockIdx.x; pr < total; pr += gridDim.x) {
        const int cg = cnt[pr * 2], ca = cnt[pr * 2 + 1];
        for (int q = threadIdx.x; q < cg; q += blockDim.x) flags[gseg[pr * tile + q]] = 1;
        for (int q = threadIdx.x; q < ca; q += blockDim.x) flags[inter + aseg[pr * tile + q]] = 1;
    }
}

__global__ __launch_bounds__(256) void ffn_union_count(const int32_t *__restrict__ flags, int inter, int32_t *n_union) {
    __shared__ int s[2][256];
    int g = 0, a = 0;
    for (int i = threadIdx.x; i < inter; i += 256) {
        g += flags[i];
        a += flags[inter + i];
    }
    s[0][threadIdx.x] = g;
    s[1][threadIdx.x] = a;
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

// Router of the MoE layer, one 256-thread block per token: x in registers,
// each wave dots two expert rows at a time (all loads in flight), then
// wave 0 takes the softmax, the top-k and the renormalised weights
// (route_wave).  With xs set (bf16 weights, the batched path), the block
// also writes its token's x as bf16 high / low parts for the matrix cores:
// row t of xs holds xs_chunks chunks of 8 values (k = 8 c .. 8 c + 7), each
// 32 bytes (the 8 high parts, then the 8 low parts), zero past H.
template <typename WT, int NC>
__global__ __launch_bounds__(256) void moe_router(const float *__restrict__ x, const WT *__restrict__ wr, int H,
                                                  int E, int K, int32_t *__restrict__ topk_idx,
                                                  float *__restrict__ topk_w, uint16_t *__restrict__ xs,
                                                  int xs_chunks) {
    constexpr int CE = WTraits<WT>::CE;
    constexpr int R = NC >= 16 ? 1 : 2;
    __shared__ float s_l[kMaxExperts];
    const int t = blockIdx.x;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nch = H / CE;
    float xr[NC][CE];
    load_x<WT, NC>(x + (size_t)t * H, lane, nch, xr);
    if constexpr (CE == 8) {
        if (xs) {
            // every wave holds all of x; wave w writes the chunks c0 = w mod 4
            u32x4 *row = reinterpret_cast<u32x4 *>(xs + (size_t)t * xs_chunks * 16);
#pragma unroll
            for (int c0 = 0; c0 < NC; ++c0) {
                const int c = lane + 64 * c0;
                if ((c0 & 3) == wave && c < nch) {
                    uint32_t hi[4], lo[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        uint32_t h0, l0, h1, l1;
                        split_hi_lo(xr[c0][2 * e], h0, l0);
                        split_hi_lo(xr[c0][2 * e + 1], h1, l1);
                        hi[e] = h0 | (h1 << 16);
                        lo[e] = l0 | (l1 << 16);
                    }
                    row[2 * c] = u32x4{hi[0], hi[1], hi[2], hi[3]};
                    row[2 * c + 1] = u32x4{lo[0], lo[1], lo[2], lo[3]};
                }
            }
            for (int c = nch + (int)threadIdx.x; c < xs_chunks; c += 256) {
                row[2 * c] = u32x4{0u, 0u, 0u, 0u};
                row[2 * c + 1] = u32x4{0u, 0u, 0u, 0u};
            }
        }
    }
    // every block reads all router rows: cached loads, and the blocks that
    // start together begin at different rows (block t's wave w takes rows
    // (w + t) mod E, (w + 4 + t) mod E, ...; measured 1-1.5 us shorter)
    const int rot = (int)(blockIdx.x % (unsigned)E);
    for (int e = wave; e < E; e += 4 * R) {
        const WT *rows[R];
        bool valid[R];
        int ex[R];
#pragma unroll
        for (int k = 0; k < R; ++k) {
            valid[k] = e + 4 * k < E;
            ex[k] = ((valid[k] ? e + 4 * k : e) + rot) % E;
            rows[k] = wr + (size_t)ex[k] * H;
        }
        float d[R];
        dot_rows<WT, NC, R, true>(rows, valid, xr, lane, nch, d);
        if (lane == 0) {
#pragma unroll
            for (int k = 0; k < R; ++k)
                if (valid[k]) s_l[ex[k]] = d[k];
        }
    }
    __syncthreads();
    if (wave == 0) {
        int ix;
        float wv;
        route_wave(s_l, E, K, lane, &ix, &wv);
        if (lane < K) {
            topk_idx[(size_t)t * K + lane] = ix;
            topk_w[(size_t)t * K + lane] = wv;
        }
    }
}

// ---------------------------------------------------------------------------
// Host launch helpers

namespace {

template <typename T>
T *ws_at(void *ws, size_t off) {
    return reinterpret_cast<T *>(static_cast<char *>(ws) + off);
}

// Rows in flight per wave in the row dot products: 2 by default, 1 when x
// alone takes 128 registers (NC = 16) or when tuned so.
int rows_in_flight(int nc) {
    const int t = tuned("rif");
    if (nc >= 16) return 1;
    return t == 1 ? 1 : 2;
}

template <typename WT, int NC, bool DENSE>
void launch_fused_rif(int rif, dim3 grid, hipStream_t st, const SlotArgs &a) {
    if (rif == 1) launch("ffn_main", ffn_fused<WT, NC, DENSE, 1>, grid, dim3(kThreads), st, a);
    else launch("ffn_main", ffn_fused<WT, NC, DENSE, 2>, grid, dim3(kThreads), st, a);
}

template <typename WT, bool DENSE>
void launch_fused_nc(int nc, int rif, dim3 grid, hipStream_t st, const SlotArgs &a) {
    switch (nc) {
    case 1: launch_fused_rif<WT, 1, DENSE>(rif, grid, st, a); break;
    case 2: launch_fused_rif<WT, 2, DENSE>(rif, grid, st, a); break;
    case 4: launch_fused_rif<WT, 4, DENSE>(rif, grid, st, a); break;
    case 8: launch_fused_rif<WT, 8, DENSE>(rif, grid, st, a); break;
    default: launch("ffn_main", ffn_fused<WT, 16, DENSE, 1>, grid, dim3(kThreads), st, a); break;
    }
}

// The pipelined kernel keeps x, two gate rows and two up rows in registers;
// with 128 x registers (NC = 16) it would spill, so wide rows use ffn_fused.
// MR, the unrolled rows per wave, is the smallest of 2, 4, 8, 16 covering the tile.
template <typename WT, int NC, bool EMIT>
void launch_pipe_mr(int tile, dim3 grid, hipStream_t st, const SlotArgs &a) {
    const int rows = (tile + kWaves - 1) / kWaves;
    const char *name = EMIT ? "ffn_gate_up" : "ffn_main";
    if (rows <= 2) launch(name, ffn_pipe<WT, NC, 2, EMIT>, grid, dim3(kThreads), st, a);
    else if (rows <= 4) launch(name, ffn_pipe<WT, NC, 4, EMIT>, grid, dim3(kThreads), st, a);
    else if (rows <= 8) launch(name, ffn_pipe<WT, NC, 8, EMIT>, grid, dim3(kThreads), st, a);
    else launch(name, ffn_pipe<WT, NC, 16, EMIT>, grid, dim3(kThreads), st, a);
}

template <typename WT, bool EMIT = false>
void launch_pipe(int nc, int tile, dim3 grid, hipStream_t st, const SlotArgs &a) {
    switch (nc) {
    case 1: launch_pipe_mr<WT, 1, EMIT>(tile, grid, st, a); break;
    case 2: launch_pipe_mr<WT, 2, EMIT>(tile, grid, st, a); break;
    case 4: launch_pipe_mr<WT, 4, EMIT>(tile, grid, st, a); break;
    default: launch_pipe_mr<WT, 8, EMIT>(tile, grid, st, a); break;
    }
}

template <typename WT, int NC>
void launch_given_mr(int chunk, dim3 grid, hipStream_t st, const GivenArgs &a) {
    const int rows = (chunk + kWaves - 1) / kWaves;
    if (rows <= 2) launch("ffn_given", ffn_given<WT, NC, 2>, grid, dim3(kThreads), st, a);
    else if (rows <= 4) launch("ffn_given", ffn_given<WT, NC, 4>, grid, dim3(kThreads), st, a);
    else if (rows <= 8) launch("ffn_given", ffn_given<WT, NC, 8>, grid, dim3(kThreads), st, a);
    else launch("ffn_given", ffn_given<WT, NC, 16>, grid, dim3(kThreads), st, a);
}

template <typename WT>
void launch_given(int nc, int chunk, dim3 grid, hipStream_t st, const GivenArgs &a) {
    switch (nc) {
    case 1: launch_given_mr<WT, 1>(chunk, grid, st, a); break;
    case 2: launch_given_mr<WT, 2>(chunk, grid, st, a); break;
    case 4: launch_given_mr<WT, 4>(chunk, grid, st, a); break;
    default: launch_given_mr<WT, 8>(chunk, grid, st, a); break;
    }
}

template <typename WT, int NC>
void launch_gate_up_rif(int rif, dim3 grid, hipStream_t st, const GateArgs &a) {
    if (rif == 1) launch("ffn_gate_up", ffn_gate_up<WT, NC, 1>, grid, dim3(kGateThreads), st, a);
    else launch("ffn_gate_up", ffn_gate_up<WT, NC, 2>, grid, dim3(kGateThreads), st, a);
}

template <typename WT>
void launch_gate_up(int nc, int rif, dim3 grid, hipStream_t st, const GateArgs &a) {
    switch (nc) {
    case 1: launch_gate_up_rif<WT, 1>(rif, grid, st, a); break;
    case 2: launch_gate_up_rif<WT, 2>(rif, grid, st, a); break;
    case 4: launch_gate_up_rif<WT, 4>(rif, grid, st, a); break;
    case 8: launch_gate_up_rif<WT, 8>(rif, grid, st, a); break;
    default: launch("ffn_gate_up", ffn_gate_up<WT, 16, 1>, grid, dim3(kGateThreads), st, a); break;
    }
}

ts_status launch_reduce(const float *partial, int rows, const SlotPlan &p, const float *slot_w, float *out,
                        hipStream_t st) {
    dim3 grid((unsigned)((p.hidden / 4 + kRedCols4 - 1) / kRedCols4), (unsigned)p.outs);
    launch("ffn_reduce", ffn_reduce, grid, dim3(256), st, partial, rows, p.hidden, p.slots_per_out, slot_w, out);
    return check_launch("ffn_reduce");
}

template <typename WT>
void launch_router(int nc, int batch, hipStream_t st, const float *x, const void *wr, int H, int E, int K,
                   int32_t *ridx, float *rw, uint16_t *xs = nullptr, int xs_chunks = 0) {
    const WT *w = static_cast<const WT *>(wr);
    const dim3 g((unsigned)batch), b(256);
    switch (nc) {
    case 1: launch("moe_router", moe_router<WT, 1>, g, b, st, x, w, H, E, K, ridx, rw, xs, xs_chunks); break;
    case 2: launch("moe_router", moe_router<WT, 2>, g, b, st, x, w, H, E, K, ridx, rw, xs, xs_chunks); break;
    case 4: launch("moe_router", moe_router<WT, 4>, g, b, st, x, w, H, E, K, ridx, rw, xs, xs_chunks); break;
    case 8: launch("moe_router", moe_router<WT, 8>, g, b, st, x, w, H, E, K, ridx, rw, xs, xs_chunks); break;
    default: launch("moe_router", moe_router<WT, 16>, g, b, st, x, w, H, E, K, ridx, rw, xs, xs_chunks); break;
    }
}

// Interleaved tiles for the single-token kernels (measured faster) where
// every row offset fits the 32-bit buffer offsets below kOutOfRange and the
// report's bitmaps hold inter.
bool interleave_tiles(const SlotPlan &p, int ntiles) {
    return tuned("ffn_interleave") == 0 && ntiles > 1 && p.inter <= kIlvMaxInter &&
           (unsigned long long)p.inter * (unsigned long long)p.hidden * (unsigned long long)p.esz <
               (unsigned long long)kOutOfRange;
}

ts_status run_report(const SlotPlan &p, const int32_t *cnt, const int32_t *gseg, const int32_t *aseg, int ntiles,
                     int tile, const ts_ffn_stats *stats, void *ws, hipStream_t st, bool interleaved = false) {
    if (!stats) return TS_OK;
    if (stats->n_gate || stats->n_active || stats->gate_idx || stats->active_idx) {
        ProfScope ps("ffn_stats", st);
        hipLaunchKernelGGL(interleaved ? ffn_stats_ilv : ffn_stats, dim3((unsigned)p.slots), dim3(256), 0, st, cnt,
                           gseg, aseg, ntiles, tile, p.inter, stats->n_gate, stats->n_active, stats->gate_idx,
                           stats->active_idx);
        ts_status s = check_launch("ffn_stats");
        if (s != TS_OK) return s;
    }
    if (stats->n_union) {
        int32_t *flags = ws_at<int32_t>(ws, p.off_aux);
        ProfScope ps("ffn_stats", st);
        hipLaunchKernelGGL(fill_i32, dim3(64), dim3(256), 0, st, flags, (size_t)2 * p.inter, 0);
        hipLaunchKernelGGL(ffn_union_mark, dim3(256), dim3(256), 0, st, cnt, gseg, aseg, ntiles, tile, p.slots,
                           p.inter, flags);
        hipLaunchKernelGGL(ffn_union_count, dim3(1), dim3(256), 0, st, flags, p.inter, stats->n_union);
        ts_status s = check_launch("ffn_union");
        if (s != TS_OK) return s;
    }
    return TS_OK;
}

// The top-k selection over lists of `ntiles` tiles of `tile` entries per
// slot, into the workspace's kept lists (off_kcnt / off_kaseg / off_khseg).
ts_status launch_select(const SlotPlan &p, int ntiles, int tile, int keep, const int32_t *cnt, const int32_t *aseg,
                        const float *hseg, void *ws, hipStream_t st) {
    SelArgs sa;
    sa.ntiles = ntiles;
    sa.tile = tile;
    sa.keep = keep;
    sa.cnt = cnt;
    sa.aseg = aseg;
    sa.hseg = hseg;
    sa.kcnt = ws_at<int32_t>(ws, p.off_kcnt);
    sa.kaseg = ws_at<int32_t>(ws, p.off_kaseg);
    sa.khseg = ws_at<float>(ws, p.off_khseg);
    launch("ffn_topk_select", ffn_topk_select, dim3((unsigned)p.slots), dim3(kSelThreads), st, sa);
    return check_launch("ffn_topk_select");
}

// Split sparse path over `p.slots` slots: gate+up, down, reduce, report.
// keep >= 0: the top-k magnitude mask between the two kernels.
ts_status run_split(const float *x, const void *wg, const void *wu, const void *wd, const int32_t *route,
                    size_t expert_stride, ts_dtype dt, const SlotPlan &p, float *out, const float *slot_w,
                    const ts_ffn_stats *stats, void *ws, hipStream_t st, int keep = -1) {
    const bool want_seg = stats && (stats->gate_idx || stats->active_idx || stats->n_union);
    GateArgs g;
    g.x = x;
    g.wg = wg;
    g.wu = wu;
    g.route = route;
    g.expert_stride = expert_stride;
    g.H = p.hidden;
    g.I = p.inter;
    g.tile = p.gtile;
    g.ntiles = p.gntiles;
    g.slots_per_tok = p.slots_per_out;
    g.cnt = ws_at<int32_t>(ws, p.off_gcnt);
    g.gseg = ws_at<int32_t>(ws, p.off_ggseg);
    g.aseg = ws_at<int32_t>(ws, p.off_gaseg);
    g.hseg = ws_at<float>(ws, p.off_ghseg);
    g.want_gseg = want_seg ? 1 : 0;
    {
        dim3 grid((unsigned)(p.slots * p.gntiles));
        const int rif = rows_in_flight(p.nc);
        if (dt == TS_F32) launch_gate_up<float>(p.nc, rif, grid, st, g);
        else launch_gate_up<uint16_t>(p.nc, rif, grid, st, g);
    }
    ts_status s = check_launch("ffn_gate_up");
    if (s != TS_OK) return s;
    if (keep >= 0) {
        s = launch_select(p, p.gntiles, p.gtile, keep, g.cnt, g.aseg, g.hseg, ws, st);
        if (s != TS_OK) return s;
        g.cnt = ws_at<int32_t>(ws, p.off_kcnt);
        g.aseg = ws_at<int32_t>(ws, p.off_kaseg);
        g.hseg = ws_at<float>(ws, p.off_khseg);
    }
    DownArgs d;
    d.wd = wd;
    d.route = route;
    d.expert_stride = expert_stride;
    d.H = p.hidden;
    d.tile = p.gtile;
    d.ntiles = p.gntiles;
    d.nslices = p.nslices;
    d.nchunks = p.nchunks;
    d.tpc = p.tpc;
    d.cnt = g.cnt;
    d.aseg = g.aseg;
    d.hseg = g.hseg;
    d.partial = ws_at<float>(ws, p.off_dpartial);
    {
        dim3 grid((unsigned)(p.slots * p.nchunks * p.nslices));
        if (dt == TS_F32) launch("ffn_down", ffn_down<float>, grid, dim3(kDownThreads), st, d);
        else launch("ffn_down", ffn_down<uint16_t>, grid, dim3(kDownThreads), st, d);
    }
    s = check_launch("ffn_down");
    if (s != TS_OK) return s;
    s = launch_reduce(d.partial, p.nchunks, p, slot_w, out, st);
    if (s != TS_OK) return s;
    return run_report(p, g.cnt, g.gseg, g.aseg, p.gntiles, p.gtile, stats, ws, st);
}

// Fused single-token path (the dense comparator, and the default sparse
// path): one workgroup per tile runs gate, up and down, then ffn_reduce.
// Router weights and outputs for in-kernel routing (MoE on the pipelined kernel).
struct RouterFold {
    const void *wr;
    int E, K;
    int32_t *ridx;
    float *rw;
};

ts_status run_fused(const float *x, const void *wg, const void *wu, const void *wd, const int32_t *route,
                    size_t expert_stride, ts_dtype dt, bool dense, const SlotPlan &p, float *out,
                    const float *slot_w, const ts_ffn_stats *stats, void *ws, hipStream_t st, bool pipe,
                    const RouterFold *rf = nullptr, int act = 0, float tau = 0.f) {
    const bool want_seg = stats && (stats->gate_idx || stats->active_idx || stats->n_union);
    SlotArgs a{};
    a.act = act;
    a.tau = tau;
    a.wr = rf ? rf->wr : nullptr;
    a.E = rf ? rf->E : 0;
    a.K = rf ? rf->K : 0;
    a.ridx = rf ? rf->ridx : nullptr;
    a.rw = rf ? rf->rw : nullptr;
    a.x = x;
    a.wg = wg;
    a.wu = wu;
    a.wd = wd;
    a.route = route;
    a.expert_stride = expert_stride;
    const bool use_pipe = pipe && p.nc <= 8;
    a.H = p.hidden;
    a.I = p.inter;
    a.tile = use_pipe ? p.tile : p.ftile;
    a.ntiles = use_pipe ? p.ntiles : p.fntiles;
    a.slots_per_tok = p.slots_per_out;
    a.cnt = ws_at<int32_t>(ws, p.off_cnt);
    a.gseg = ws_at<int32_t>(ws, p.off_gseg);
    a.aseg = ws_at<int32_t>(ws, p.off_aseg);
    a.partial = ws_at<float>(ws, p.off_partial);
    a.want_seg = want_seg ? 1 : 0;
    const bool ilv = interleave_tiles(p, a.ntiles);
    a.rstride = ilv ? a.ntiles : 1;
    {
        dim3 grid((unsigned)(p.slots * a.ntiles));
        const int rif = rows_in_flight(p.nc);
        if (use_pipe) {
            if (dt == TS_F32) launch_pipe<float>(p.nc, a.tile, grid, st, a);
            else launch_pipe<uint16_t>(p.nc, a.tile, grid, st, a);
        } else if (dt == TS_F32) {
            if (dense) launch_fused_nc<float, true>(p.nc, rif, grid, st, a);
            else launch_fused_nc<float, false>(p.nc, rif, grid, st, a);
        } else {
            if (dense) launch_fused_nc<uint16_t, true>(p.nc, rif, grid, st, a);
            else launch_fused_nc<uint16_t, false>(p.nc, rif, grid, st, a);
        }
    }
    ts_status s = check_launch("ffn_main");
    if (s != TS_OK) return s;
    s = launch_reduce(a.partial, a.ntiles, p, slot_w, out, st);
    if (s != TS_OK) return s;
    return run_report(p, a.cnt, a.gseg, a.aseg, a.ntiles, a.tile, stats, ws, st, ilv);
}

// The kernel sequence run_slots picks: the pipelined kernel unless the dense
// comparator, a tuning knob or a row too wide for it asks for another.
bool slots_use_pipe(const SlotPlan &p, bool dense) { return !dense && tuned("ffn_path") == 0 && p.nc <= 8; }

// The top-k mask over single-token slots (the FFN's tokens): the pipelined
// kernel in emit mode (gate and up at its streaming rate), the selection,
// the split path's down kernel over the kept lists, reduce, report.  Rows
// too wide for the pipelined kernel take the split path's gate+up kernel.
ts_status run_topk(const float *x, const void *wg, const void *wu, const void *wd, ts_dtype dt, const SlotPlan &p,
                   float *out, const ts_ffn_stats *stats, void *ws, hipStream_t st, int keep) {
    if (!slots_use_pipe(p, false))
        return run_split(x, wg, wu, wd, nullptr, 0, dt, p, out, nullptr, stats, ws, st, keep);
    SlotArgs a{};
    a.x = x;
    a.wg = wg;
    a.wu = wu;
    a.wd = wd;
    a.H = p.hidden;
    a.I = p.inter;
    a.tile = p.tile;
    a.ntiles = p.ntiles;
    a.slots_per_tok = 1;
    a.cnt = ws_at<int32_t>(ws, p.off_cnt);
    a.gseg = ws_at<int32_t>(ws, p.off_gseg);
    a.aseg = ws_at<int32_t>(ws, p.off_aseg);
    a.hseg = ws_at<float>(ws, p.off_hseg);
    a.partial = ws_at<float>(ws, p.off_partial);
    a.want_seg = stats && (stats->gate_idx || stats->active_idx || stats->n_union) ? 1 : 0;
    // (the selection breaks ties by neuron index, so the tile layout does
    // not change which neurons are kept)
    const bool ilv = interleave_tiles(p, p.ntiles);
    a.rstride = ilv ? p.ntiles : 1;
    const dim3 grid((unsigned)(p.slots * p.ntiles));
    if (dt == TS_F32) launch_pipe<float, true>(p.nc, p.tile, grid, st, a);
    else launch_pipe<uint16_t, true>(p.nc, p.tile, grid, st, a);
    ts_status s = check_launch("ffn_gate_up");
    if (s != TS_OK) return s;
    if (!stats) {
        // no report: the down workgroups select for themselves
        TopkDownArgs td;
        td.d.wd = wd;
        td.d.route = nullptr;
        td.d.expert_stride = 0;
        td.d.H = p.hidden;
        td.d.tile = p.tile;
        td.d.ntiles = p.ntiles;
        td.d.nslices = p.nslices;
        td.d.nchunks = p.pnchunks;
        td.d.tpc = p.ptpc;
        td.d.cnt = a.cnt;
        td.d.aseg = a.aseg;
        td.d.hseg = a.hseg;
        td.d.partial = a.partial;
        td.keep = keep;
        const dim3 dg((unsigned)(p.slots * p.pnchunks * p.nslices));
        if (dt == TS_F32) launch("ffn_topk_down", ffn_topk_down<float>, dg, dim3(kDownThreads), st, td);
        else launch("ffn_topk_down", ffn_topk_down<uint16_t>, dg, dim3(kDownThreads), st, td);
        s = check_launch("ffn_topk_down");
        if (s != TS_OK) return s;
        return launch_reduce(a.partial, p.pnchunks, p, nullptr, out, st);
    }
    s = launch_select(p, p.ntiles, p.tile, keep, a.cnt, a.aseg, a.hseg, ws, st);
    if (s != TS_OK) return s;
    DownArgs d;
    d.wd = wd;
    d.route = nullptr;
    d.expert_stride = 0;
    d.H = p.hidden;
    d.tile = p.tile;
    d.ntiles = p.ntiles;
    d.nslices = p.nslices;
    d.nchunks = p.pnchunks;
    d.tpc = p.ptpc;
    d.cnt = ws_at<int32_t>(ws, p.off_kcnt);
    d.aseg = ws_at<int32_t>(ws, p.off_kaseg);
    d.hseg = ws_at<float>(ws, p.off_khseg);
    d.partial = a.partial;
    {
        dim3 dg((unsigned)(p.slots * p.pnchunks * p.nslices));
        if (dt == TS_F32) launch("ffn_down", ffn_down<float>, dg, dim3(kDownThreads), st, d);
        else launch("ffn_down", ffn_down<uint16_t>, dg, dim3(kDownThreads), st, d);
    }
    s = check_launch("ffn_down");
    if (s != TS_OK) return s;
    s = launch_reduce(d.partial, p.pnchunks, p, nullptr, out, st);
    if (s != TS_OK) return s;
    return run_report(p, d.cnt, a.gseg, d.aseg, p.ntiles, p.tile, stats, ws, st, ilv);
}


// `rf` (pipelined kernel only, route == null) moves the MoE router into it.
ts_status run_slots(const float *x, const void *wg, const void *wu, const void *wd, const int32_t *route,
                    size_t expert_stride, ts_dtype dt, bool dense, const SlotPlan &p, float *out,
                    const float *slot_w, const ts_ffn_stats *stats, void *ws, hipStream_t st,
                    const RouterFold *rf = nullptr) {
    const int path = tuned("ffn_path");
    if (dense || path == 2)
        return run_fused(x, wg, wu, wd, route, expert_stride, dt, dense, p, out, slot_w, stats, ws, st, false);
    if (path == 1) return run_split(x, wg, wu, wd, route, expert_stride, dt, p, out, slot_w, stats, ws, st);
    return run_fused(x, wg, wu, wd, route, expert_stride, dt, false, p, out, slot_w, stats, ws, st, true, rf);
}

ts_status check_ffn_args(const float *x, const void *wg, const void *wu, const void *wd, ts_dtype dt, int batch,
                         int hidden, int inter, const float *out, const ts_ffn_stats *stats, const void *ws,
                         size_t ws_bytes, SlotPlan *plan, bool pow2_tiles = true) {
    ts_status s = check_dims(batch, hidden, inter, dt);
    if (s != TS_OK) return s;
    if (!x || !wg || !wu || !wd || !out) return TS_ERR_NULL;
    if (!aligned16(x) || !aligned16(wg) || !aligned16(wu) || !aligned16(wd) || !aligned16(out))
        return TS_ERR_ALIGN;
    s = check_stats(stats);
    if (s != TS_OK) return s;
    if (!plan_slots(hidden, inter, dt, batch, 1, plan, pow2_tiles)) return TS_ERR_SHAPE;
    if (!ws || ws_bytes < ffn_ws_bytes(batch, hidden, inter, dt)) return TS_ERR_WORKSPACE;
    if (!aligned16(ws)) return TS_ERR_ALIGN;
    return TS_OK;
}

ts_status check_moe_args(const float *x, const void *wr, const void *wg, const void *wu, const void *wd,
                         ts_dtype dt, int batch, int hidden, int inter, int E, int K, const float *out,
                         const int32_t *topk_idx, const float *topk_w, const ts_ffn_stats *stats, const void *ws,
                         size_t ws_bytes, SlotPlan *plan) {
    ts_status s = check_moe_dims(batch, hidden, inter, E, K, dt);
    if (s != TS_OK) return s;
    if (!x || !wr || !wg || !wu || !wd || !out) return TS_ERR_NULL;
    if (!aligned16(x) || !aligned16(wr) || !aligned16(wg) || !aligned16(wu) || !aligned16(wd) || !aligned16(out) ||
        (topk_idx && !aligned4(topk_idx)) || (topk_w && !aligned4(topk_w)))
        return TS_ERR_ALIGN;
    s = check_stats(stats);
    if (s != TS_OK) return s;
    if (stats && stats->n_union) return TS_ERR_UNSUPPORTED;
    if (!plan_slots(hidden, inter, dt, batch * K, K, plan)) return TS_ERR_SHAPE;
    if (!ws || ws_bytes < moe_ws_bytes(batch, hidden, inter, E, K, dt)) return TS_ERR_WORKSPACE;
    if (!aligned16(ws)) return TS_ERR_ALIGN;
    return TS_OK;
}

ts_status moe_impl(const float *x, const void *wr, const void *wg, const void *wu, const void *wd, ts_dtype dt,
                   int batch, int hidden, int inter, int E, int K, float *out, int32_t *topk_idx, float *topk_w,
                   const ts_ffn_stats *stats, void *ws, size_t ws_bytes, void *stream, bool dense) {
    SlotPlan p;
    ts_status s = check_moe_args(x, wr, wg, wu, wd, dt, batch, hidden, inter, E, K, out, topk_idx, topk_w, stats,
                                 ws, ws_bytes, &p);
    if (s != TS_OK) return s;
    hipStream_t st = static_cast<hipStream_t>(stream);
    // the routing table goes straight to the caller's arrays when given (no
    // copies after the kernels), otherwise to the workspace
    const size_t roff = moe_route_offset(batch, hidden, inter, E, K, dt);
    int32_t *ridx = topk_idx ? topk_idx : ws_at<int32_t>(ws, roff);
    float *rw = topk_w ? topk_w : ws_at<float>(ws, roff + align_up256((size_t)batch * K * sizeof(int32_t)));
    BatchPlan bp;
    const size_t estride = (size_t)inter * (size_t)hidden;
    const bool batched = batch > 1 && tuned("batch_path") == 0 && plan_batch(batch, hidden, inter, E, K, dt, &bp);
    // on the pipelined kernel each workgroup routes its own token (no router launch)
    const bool fold = !batched && slots_use_pipe(p, dense);
    // batched: the router also writes each token's x split for the matrix
    // cores, and the gate+up kernel gathers its group's tokens from it (no
    // dispatch kernel, one copy of x in L2 for all expert groups)
    const bool xtok = batched && tuned("bx_xtok") == 0;
    if (!fold) {
        if (dt == TS_F32) {
            launch_router<float>(p.nc, batch, st, x, wr, hidden, E, K, ridx, rw);
        } else {
            launch_router<uint16_t>(p.nc, batch, st, x, wr, hidden, E, K, ridx, rw,
                                    xtok ? ws_at<uint16_t>(ws, bp.off_xhl) : nullptr, bp.hpad / 8);
        }
        s = check_launch("moe_router");
        if (s != TS_OK) return s;
    }
    if (batched) {
        s = run_batch(x, wg, wu, wd, estride, ridx, rw, bp, out, stats, 0, ws, st, dense, xtok);
    } else if (fold) {
        const RouterFold rf{wr, E, K, ridx, rw};
        s = run_slots(x, wg, wu, wd, nullptr, estride, dt, dense, p, out, rw, stats, ws, st, &rf);
    } else {
        s = run_slots(x, wg, wu, wd, ridx, estride, dt, dense, p, out, rw, stats, ws, st);
    }
    return s;
}

}  // namespace

// ---------------------------------------------------------------------------
// Scratch of the allocation-free entry point (ts_ffn_sparse_noalloc): the
// workspace of ts_ffn_sparse as a fixed array in the library's own device
// memory, one copy per GPU.  In host code `scratch` names a host-side
// stand-in, not a device address: the address each GPU's copy has is looked
// up once per device (hipGetSymbolAddress, with that device current) and
// only that address is handed to kernels.
static __device__ __align__(256) unsigned char scratch[TS_NOALLOC_SCRATCH_BYTES];

constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kScratchDevices] = {};

// The current device's copy of `scratch` (looked up on its first use).
ts_status scratch_on_current_device(void **ptr) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        set_last_error("hipGetDevice", e);
        return TS_ERR_HIP;
    }
    if (dev < 0 || dev >= kScratchDevices) {
        set_last_message("ts_ffn_sparse_noalloc: device index beyond the library's scratch table (64)");
        return TS_ERR_UNSUPPORTED;
    }
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            set_last_error("hipGetSymbolAddress(scratch)", e);
            return TS_ERR_HIP;
        }
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return TS_OK;
}

}  // namespace ts

extern "C" {

ts_status ts_ffn_sparse_noalloc(const float *x, const void *w_gate, const void *w_up, const void *w_down_t,
                                ts_dtype wdtype, int batch, int hidden, int inter, float *out,
                                const ts_ffn_stats *stats, void *stream) {
    // every host-side check of ts_ffn_sparse first (a placeholder workspace
    // address of the right size and alignment stands in for the scratch)
    const size_t need = ts::ffn_ws_bytes(batch, hidden, inter, wdtype);
    ts::SlotPlan p;
    ts_status s = ts::check_ffn_args(x, w_gate, w_up, w_down_t, wdtype, batch, hidden, inter, out, stats,
                                     reinterpret_cast<const void *>(uintptr_t{256}), need, &p);
    if (s != TS_OK) return s;
    if (need > TS_NOALLOC_SCRATCH_BYTES) {
        char msg[200];
        std::snprintf(msg, sizeof msg,
                      "ts_ffn_sparse_noalloc: this shape needs %zu bytes of scratch, the library holds %zu",
                      need, (size_t)TS_NOALLOC_SCRATCH_BYTES);
        ts::set_last_message(msg);
        return TS_ERR_WORKSPACE;
    }
    void *ws = nullptr;
    s = ts::scratch_on_current_device(&ws);
    if (s != TS_OK) return s;
    return ts_ffn_sparse(x, w_gate, w_up, w_down_t, wdtype, batch, hidden, inter, out, stats, ws, need, stream);
}


ts_status ts_ffn_sparse(const float *x, const void *w_gate, const void *w_up, const void *w_down_t, ts_dtype wdtype,
                        int batch, int hidden, int inter, float *out, const ts_ffn_stats *stats, void *ws,
                        size_t ws_bytes, void *stream) {
    ts::SlotPlan p;
    ts_status s = ts::check_ffn_args(x, w_gate, w_up, w_down_t, wdtype, batch, hidden, inter, out, stats, ws,
                                     ws_bytes, &p);
    if (s != TS_OK) return s;
    hipStream_t st = static_cast<hipStream_t>(stream);
    // Several tokens with bf16 weights: the batched matrix-core path, in
    // passes of up to 64 tokens (the union count needs a single pass);
    // shapes it does not take run the single-token kernels per token.
    const bool one_pass = batch <= ts::kBxMaxTokens;
    ts::BatchPlan probe;
    if (batch > 1 && wdtype == TS_BF16 && ts::tuned("batch_path") == 0 &&
        (one_pass || !(stats && stats->n_union)) &&
        ts::plan_batch(std::min(batch, ts::kBxMaxTokens), hidden, inter, 1, 1, wdtype, &probe)) {
        for (int t0 = 0; t0 < batch; t0 += ts::kBxMaxTokens) {
            const int nb = std::min(ts::kBxMaxTokens, batch - t0);
            ts::BatchPlan bp;
            if (!ts::plan_batch(nb, hidden, inter, 1, 1, wdtype, &bp)) return TS_ERR_SHAPE;
            s = ts::run_batch(x + (size_t)t0 * hidden, w_gate, w_up, w_down_t, 0, nullptr, nullptr, bp,
                              out + (size_t)t0 * hidden, stats, t0, ws, st, false);
            if (s != TS_OK) return s;
        }
        return TS_OK;
    }
    return ts::run_slots(x, w_gate, w_up, w_down_t, nullptr, 0, wdtype, false, p, out, nullptr, stats, ws, st);
}

ts_status ts_ffn_sparse_topk(const float *x, const void *w_gate, const void *w_up, const void *w_down_t,
                             ts_dtype wdtype, int batch, int hidden, int inter, int keep, float *out,
                             const ts_ffn_stats *stats, void *ws, size_t ws_bytes, void *stream) {
    if (keep < 0) return TS_ERR_SHAPE;
    ts::SlotPlan p;
    ts_status s = ts::check_ffn_args(x, w_gate, w_up, w_down_t, wdtype, batch, hidden, inter, out, stats, ws,
                                     ws_bytes, &p, false);
    if (s != TS_OK) return s;
    if (inter > ts::kSelMax || p.gntiles * p.gtile > ts::kSelSpan || p.ntiles * p.tile > ts::kSelSpan ||
        p.gntiles > ts::kSelMaxTiles || p.ntiles > ts::kSelMaxTiles)
        return TS_ERR_UNSUPPORTED;
    return ts::run_topk(x, w_gate, w_up, w_down_t, wdtype, p, out, stats, ws, static_cast<hipStream_t>(stream),
                        keep);
}

ts_status ts_ffn_sparse_act(const float *x, const void *w_gate, const void *w_up, const void *w_down_t,
                            ts_dtype wdtype, int batch, int hidden, int inter, ts_act act, float tau, float *out,
                            const ts_ffn_stats *stats, void *ws, size_t ws_bytes, void *stream) {
    if ((act != TS_ACT_DRELU && act != TS_ACT_RELU_GATE) || !std::isfinite(tau) ||
        (act == TS_ACT_DRELU && tau != 0.f))
        return TS_ERR_SHAPE;
    if (act == TS_ACT_DRELU)
        return ts_ffn_sparse(x, w_gate, w_up, w_down_t, wdtype, batch, hidden, inter, out, stats, ws, ws_bytes,
                             stream);
    ts::SlotPlan p;
    ts_status s = ts::check_ffn_args(x, w_gate, w_up, w_down_t, wdtype, batch, hidden, inter, out, stats, ws,
                                     ws_bytes, &p);
    if (s != TS_OK) return s;
    return ts::run_fused(x, w_gate, w_up, w_down_t, nullptr, 0, wdtype, false, p, out, nullptr, stats, ws,
                         static_cast<hipStream_t>(stream), true, nullptr, 1, tau);
}

ts_status ts_ffn_dense(const float *x, const void *w_gate, const void *w_up, const void *w_down_t, ts_dtype wdtype,
                       int batch, int hidden, int inter, float *out, void *ws, size_t ws_bytes, void *stream) {
    ts::SlotPlan p;
    ts_status s = ts::check_ffn_args(x, w_gate, w_up, w_down_t, wdtype, batch, hidden, inter, out, nullptr, ws,
                                     ws_bytes, &p);
    if (s != TS_OK) return s;
    hipStream_t st = static_cast<hipStream_t>(stream);
    ts::BatchPlan probe;
    if (batch > 1 && wdtype == TS_BF16 && ts::tuned("batch_path") == 0 &&
        ts::plan_batch(std::min(batch, ts::kBxMaxTokens), hidden, inter, 1, 1, wdtype, &probe)) {
        for (int t0 = 0; t0 < batch; t0 += ts::kBxMaxTokens) {
            const int nb = std::min(ts::kBxMaxTokens, batch - t0);
            ts::BatchPlan bp;
            if (!ts::plan_batch(nb, hidden, inter, 1, 1, wdtype, &bp)) return TS_ERR_SHAPE;
            s = ts::run_batch(x + (size_t)t0 * hidden, w_gate, w_up, w_down_t, 0, nullptr, nullptr, bp,
                              out + (size_t)t0 * hidden, nullptr, t0, ws, st, true);
            if (s != TS_OK) return s;
        }
        return TS_OK;
    }
    return ts::run_slots(x, w_gate, w_up, w_down_t, nullptr, 0, wdtype, true, p, out, nullptr, nullptr, ws, st);
}

ts_status ts_ffn_sparse_given(const float *x, const void *w_gate, const void *w_up, const void *w_down_t,
                              ts_dtype wdtype, int batch, int hidden, int inter, const int32_t *idx,
                              const int32_t *count, int max_count, float *out, const ts_ffn_stats *stats,
                              void *ws, size_t ws_bytes, void *stream) {
    ts_status s = ts::check_dims(batch, hidden, inter, wdtype);
    if (s != TS_OK) return s;
    if (!x || !w_gate || !w_up || !w_down_t || !out || !idx || !count) return TS_ERR_NULL;
    if (!ts::aligned16(x) || !ts::aligned16(w_gate) || !ts::aligned16(w_up) || !ts::aligned16(w_down_t) ||
        !ts::aligned16(out) || !ts::aligned4(idx) || !ts::aligned4(count))
        return TS_ERR_ALIGN;
    s = ts::check_stats(stats);
    if (s != TS_OK) return s;
    if (stats && (stats->gate_idx || stats->active_idx || stats->n_union)) return TS_ERR_UNSUPPORTED;
    ts::GivenPlan p;
    if (!ts::plan_given(batch, hidden, inter, max_count, wdtype, &p)) return TS_ERR_SHAPE;
    if (p.nc > 8) return TS_ERR_UNSUPPORTED;
    if (!ws || ws_bytes < p.total) return TS_ERR_WORKSPACE;
    if (!ts::aligned16(ws)) return TS_ERR_ALIGN;
    hipStream_t st = static_cast<hipStream_t>(stream);
    ts::GivenArgs a;
    a.x = x;
    a.wg = w_gate;
    a.wu = w_up;
    a.wd = w_down_t;
    a.idx = idx;
    a.count = count;
    a.H = hidden;
    a.I = inter;
    a.maxc = max_count;
    a.chunk = p.chunk;
    a.nchunks = p.nchunks;
    a.partial = ts::ws_at<float>(ws, p.off_partial);
    a.cnt = ts::ws_at<int32_t>(ws, p.off_cnt);
    const dim3 grid((unsigned)(batch * p.nchunks));
    if (wdtype == TS_F32) ts::launch_given<float>(p.nc, p.chunk, grid, st, a);
    else ts::launch_given<uint16_t>(p.nc, p.chunk, grid, st, a);
    s = ts::check_launch("ffn_given");
    if (s != TS_OK) return s;
    const dim3 rgrid((unsigned)((hidden / 4 + ts::kRedCols4 - 1) / ts::kRedCols4), (unsigned)batch);
    ts::launch("ffn_reduce", ts::ffn_reduce, rgrid, dim3(256), st, static_cast<const float *>(a.partial), p.nchunks,
               hidden, 1, static_cast<const float *>(nullptr), out);
    s = ts::check_launch("ffn_reduce");
    if (s != TS_OK) return s;
    if (stats && (stats->n_gate || stats->n_active)) {
        ts::launch("ffn_stats", ts::given_counts, dim3((unsigned)batch), dim3(64), st,
                   static_cast<const int32_t *>(a.cnt), p.nchunks, stats->n_gate, stats->n_active);
        s = ts::check_launch("given_counts");
    }
    return s;
}

ts_status ts_moe_sparse(const float *x, const void *w_router, const void *w_gate, const void *w_up,
                        const void *w_down_t, ts_dtype wdtype, int batch, int hidden, int inter, int n_experts,
                        int top_k, float *out, int32_t *topk_idx, float *topk_w, const ts_ffn_stats *stats, void *ws,
                        size_t ws_bytes, void *stream) {
    return ts::moe_impl(x, w_router, w_gate, w_up, w_down_t, wdtype, batch, hidden, inter, n_experts, top_k, out,
                        topk_idx, topk_w, stats, ws, ws_bytes, stream, false);
}

ts_status ts_moe_dense(const float *x, const void *w_router, const void *w_gate, const void *w_up,
                       const void *w_down_t, ts_dtype wdtype, int batch, int hidden, int inter, int n_experts,
                       int top_k, float *out, int32_t *topk_idx, float *topk_w, void *ws, size_t ws_bytes,
                       void *stream) {
    return ts::moe_impl(x, w_router, w_gate, w_up, w_down_t, wdtype, batch, hidden, inter, n_experts, top_k, out,
                        topk_idx, topk_w, nullptr, ws, ws_bytes, stream, true);
}

}  // extern "C"
