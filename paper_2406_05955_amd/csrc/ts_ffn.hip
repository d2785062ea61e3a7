// Single-token ("slot") kernels of the activation-sparse dReLU FFN for gfx950
// and the ts_ffn_* / ts_moe_* entry points.
//
// One slot is one token evaluated against one weight set (the FFN's, or the
// routed expert's in the MoE layer).  For each slot the work is split into
// tiles of `tile` consecutive neurons, one 512-thread workgroup (8 wave64s)
// per tile, and each workgroup runs the whole dReLU FFN for its neurons:
//
//   gate   every lane holds its share of x in registers; each wave dots whole
//          W_gate rows (16-byte streaming loads, two rows in flight) and the
//          results meet in LDS; one wave ballots `gate > 0` and prefix-counts
//          the ballot into the tile's ascending open-gate list G.
//   up     the waves dot the W_up rows of G only, Combined = gate * up where
//          up > 0; a second ballot compacts the non-zero ones into A.
//   down   the 512 threads split the hidden dimension (16 bytes each) and run
//          an axpy over the W_down_t rows of A in ascending order; the tile's
//          partial output row goes to the workspace (skipped when A is empty).
//
// A second kernel sums the partial rows of every tile in a fixed order
// (deterministic, no atomics), applying the routing weights in the MoE form.
//
// Eq. (drelu) of Turbo Sparse (arXiv 2406.05955): Combined = max(0, x W_gate)
// * max(0, x W_up); skipping the zero Combined terms (section 6.2) leaves
// the output unchanged.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "ts_device.h"
#include "ts_plan.h"
#include "ts_runtime.h"
#include "turbosparse.h"

namespace ts {

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
    int want_seg;
};

constexpr int kDownUnroll = 8;

// Dot products of R weight rows (those with valid[k]) with the x chunks held
// in registers; all R rows' loads are issued before any arithmetic.  Every
// lane returns the full sums.
template <typename WT, int NC, int R>
__device__ __forceinline__ void dot_rows(const WT *const (&rows)[R], const bool (&valid)[R],
                                         const float (&xr)[NC][WTraits<WT>::CE], int lane, int nch,
                                         float (&out)[R]) {
    constexpr int CE = WTraits<WT>::CE;
    u32x4 v[R][NC];
#pragma unroll
    for (int k = 0; k < R; ++k)
#pragma unroll
        for (int c0 = 0; c0 < NC; ++c0) {
            const int c = lane + 64 * c0;
            v[k][c0] = (valid[k] && c < nch) ? ld_stream(rows[k] + c * CE) : u32x4{0u, 0u, 0u, 0u};
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

template <typename WT, int NC, bool DENSE>
__global__ __launch_bounds__(kThreads) void ffn_slot_main(SlotArgs a) {
    constexpr int CE = WTraits<WT>::CE;
    constexpr int NCD = (NC * 64 + kThreads - 1) / kThreads;
    constexpr int RIF = NC >= 16 ? 1 : 2;  // weight rows in flight per wave

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
    const int n0 = tile * a.tile;
    const int nt = min(a.tile, a.I - n0);
    const int H = a.H;
    const int nch = H / CE;

    size_t eoff = 0;
    if (a.route) eoff = (size_t)a.route[slot] * a.expert_stride;
    const WT *wg = reinterpret_cast<const WT *>(a.wg) + eoff + (size_t)n0 * H;
    const WT *wu = reinterpret_cast<const WT *>(a.wu) + eoff + (size_t)n0 * H;
    const WT *wd = reinterpret_cast<const WT *>(a.wd) + eoff + (size_t)n0 * H;
    const float *x = a.x + (size_t)tok * H;

    // x in registers: lane owns chunks lane, lane + 64, ... of every row.
    float xr[NC][CE];
#pragma unroll
    for (int k = 0; k < NC; ++k) {
        const int c = lane + 64 * k;
#pragma unroll
        for (int e = 0; e < CE; e += 4) {
            f32x4 v = {0.f, 0.f, 0.f, 0.f};
            if (c < nch) v = *reinterpret_cast<const f32x4 *>(x + c * CE + e);
            xr[k][e] = v.x;
            xr[k][e + 1] = v.y;
            xr[k][e + 2] = v.z;
            xr[k][e + 3] = v.w;
        }
    }

    // ---- gate: wave w dots rows w, w+8, ..., RIF rows in flight ------------
    for (int r = wave; r < nt; r += RIF * kWaves) {
        const WT *rows[RIF];
        bool valid[RIF];
#pragma unroll
        for (int k = 0; k < RIF; ++k) {
            valid[k] = r + k * kWaves < nt;
            rows[k] = wg + (size_t)(valid[k] ? r + k * kWaves : r) * H;
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
        const bool p = in && (DENSE || s_g[lane] > 0.f);
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
            rows[k] = wu + (size_t)li[k] * H;
        }
        float u[RIF];
        dot_rows<WT, NC, RIF>(rows, valid, xr, lane, nch, u);
        if (lane == 0) {
#pragma unroll
            for (int k = 0; k < RIF; ++k) {
                if (valid[k]) {
                    const float g = s_g[li[k]];
                    const bool on = g > 0.f && u[k] > 0.f;
                    s_on[q + k * kWaves] = on;
                    s_h[q + k * kWaves] = on ? g * u[k] : 0.f;
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

    for (int a0 = 0; a0 < na; a0 += kDownUnroll) {
        u32x4 v[kDownUnroll][NCD];
#pragma unroll
        for (int u = 0; u < kDownUnroll; ++u) {
            const int aa = a0 + u;
            const WT *row = wd + (size_t)(aa < na ? s_al[aa] : 0) * H;
#pragma unroll
            for (int kd = 0; kd < NCD; ++kd) {
                const int c = tid + kThreads * kd;
                v[u][kd] = (aa < na && c < nch) ? ld_stream(row + c * CE) : u32x4{0u, 0u, 0u, 0u};
            }
        }
#pragma unroll
        for (int u = 0; u < kDownUnroll; ++u) {
            const int aa = a0 + u;
            if (aa < na) {
                const float hv = s_av[aa];
#pragma unroll
                for (int kd = 0; kd < NCD; ++kd) {
                    float f[CE];
                    unpack<WT>(v[u][kd], f);
#pragma unroll
                    for (int e = 0; e < CE; ++e) acc[kd][e] = fmaf(hv, f[e], acc[kd][e]);
                }
            }
        }
    }

    const size_t pr = (size_t)slot * a.ntiles + tile;
    if (na > 0) {
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
    }
    if (tid == 0) {
        a.cnt[pr * 2] = ng;
        a.cnt[pr * 2 + 1] = na;
    }
    if (a.want_seg) {
        for (int q = tid; q < ng; q += kThreads) a.gseg[pr * a.tile + q] = n0 + s_gl[q];
        for (int q = tid; q < na; q += kThreads) a.aseg[pr * a.tile + q] = n0 + s_al[q];
    }
}

// out[o][:] = sum over the slots s of output row o, and over tiles p in
// ascending order, of w_s * partial[s][p][:] (w_s = 1 without routing).
// Block: 32 columns (8 float4) x 32 row groups; grid (column blocks, outs).
constexpr int kRedCols4 = 8;
constexpr int kRedGroups = 32;

__global__ __launch_bounds__(256) void ffn_reduce(const float *__restrict__ partial, const int32_t *__restrict__ cnt,
                                                  int ntiles, int H, int slots_per_out,
                                                  const float *__restrict__ slot_w, float *__restrict__ out) {
    __shared__ f32x4 red[kRedGroups][kRedCols4];
    const int o = blockIdx.y;
    const int q = threadIdx.x % kRedCols4;
    const int grp = threadIdx.x / kRedCols4;
    const int c4 = blockIdx.x * kRedCols4 + q;
    const int nq = H / 4;
    const int nrows = slots_per_out * ntiles;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    if (c4 < nq) {
        for (int r0 = grp; r0 < nrows; r0 += 4 * kRedGroups) {
            int act[4];
            size_t prs[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int r = r0 + u * kRedGroups;
                const size_t s = (size_t)o * slots_per_out + (r / ntiles);
                prs[u] = s * ntiles + (r % ntiles);
                act[u] = r < nrows ? cnt[prs[u] * 2 + 1] : 0;
            }
            f32x4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                v[u] = act[u] > 0 ? *reinterpret_cast<const f32x4 *>(partial + prs[u] * H + c4 * 4)
                                  : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (act[u] > 0) {
                    const float w = slot_w ? slot_w[prs[u] / ntiles] : 1.f;
                    acc.x = fmaf(w, v[u].x, acc.x);
                    acc.y = fmaf(w, v[u].y, acc.y);
                    acc.z = fmaf(w, v[u].z, acc.z);
                    acc.w = fmaf(w, v[u].w, acc.w);
                }
            }
        }
    }
    red[grp][q] = acc;
    __syncthreads();
    for (int st = kRedGroups / 2; st >= 1; st >>= 1) {
        if (grp < st) red[grp][q] += red[grp + st][q];
        __syncthreads();
    }
    if (grp == 0 && c4 < nq) *reinterpret_cast<f32x4 *>(out + (size_t)o * H + c4 * 4) = red[0][q];
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

// Router of the MoE layer, one 256-thread block per token: logits = W_r x
// (one wave per expert row), then softmax, top-k (strictly larger wins, so
// the lower index wins exact ties) and renormalisation by thread 0.
template <typename WT>
__global__ __launch_bounds__(256) void moe_router(const float *__restrict__ x, const WT *__restrict__ wr, int H,
                                                  int E, int K, int32_t *__restrict__ topk_idx,
                                                  float *__restrict__ topk_w) {
    constexpr int CE = WTraits<WT>::CE;
    __shared__ float s_l[kMaxExperts];
    const int t = blockIdx.x;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const float *xt = x + (size_t)t * H;
    const int nch = H / CE;
    for (int e = wave; e < E; e += 4) {
        const WT *row = wr + (size_t)e * H;
        float d = 0.f;
        for (int c = lane; c < nch; c += 64) {
            float f[CE];
            unpack<WT>(ld_cached(row + c * CE), f);
#pragma unroll
            for (int q = 0; q < CE; ++q) d = fmaf(f[q], xt[c * CE + q], d);
        }
        d = wave_sum(d);
        if (lane == 0) s_l[e] = d;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        float m = s_l[0];
        for (int e = 1; e < E; ++e) m = fmaxf(m, s_l[e]);
        float p[kMaxExperts];
        float z = 0.f;
        for (int e = 0; e < E; ++e) {
            p[e] = expf(s_l[e] - m);
            z += p[e];
        }
        const float inv = 1.f / z;
        for (int e = 0; e < E; ++e) p[e] *= inv;
        uint64_t taken = 0;
        int idx[kMaxTopK];
        float ps = 0.f;
        for (int k = 0; k < K; ++k) {
            int best = -1;
            for (int e = 0; e < E; ++e)
                if (!((taken >> e) & 1ull) && (best < 0 || p[e] > p[best])) best = e;
            taken |= 1ull << best;
            idx[k] = best;
            ps += p[best];
        }
        for (int k = 0; k < K; ++k) {
            topk_idx[(size_t)t * K + k] = idx[k];
            topk_w[(size_t)t * K + k] = p[idx[k]] / ps;
        }
    }
}

// ---------------------------------------------------------------------------
// Host launch helpers

namespace {

template <typename WT, bool DENSE>
void launch_main_nc(int nc, dim3 grid, hipStream_t st, const SlotArgs &a) {
    switch (nc) {
    case 1: hipLaunchKernelGGL((ffn_slot_main<WT, 1, DENSE>), grid, dim3(kThreads), 0, st, a); break;
    case 2: hipLaunchKernelGGL((ffn_slot_main<WT, 2, DENSE>), grid, dim3(kThreads), 0, st, a); break;
    case 4: hipLaunchKernelGGL((ffn_slot_main<WT, 4, DENSE>), grid, dim3(kThreads), 0, st, a); break;
    case 8: hipLaunchKernelGGL((ffn_slot_main<WT, 8, DENSE>), grid, dim3(kThreads), 0, st, a); break;
    default: hipLaunchKernelGGL((ffn_slot_main<WT, 16, DENSE>), grid, dim3(kThreads), 0, st, a); break;
    }
}

void launch_main(ts_dtype dt, bool dense, const SlotPlan &p, hipStream_t st, const SlotArgs &a) {
    dim3 grid((unsigned)(p.slots * p.ntiles));
    if (dt == TS_F32) {
        if (dense) launch_main_nc<float, true>(p.nc, grid, st, a);
        else launch_main_nc<float, false>(p.nc, grid, st, a);
    } else {
        if (dense) launch_main_nc<uint16_t, true>(p.nc, grid, st, a);
        else launch_main_nc<uint16_t, false>(p.nc, grid, st, a);
    }
}

template <typename T>
T *ws_at(void *ws, size_t off) {
    return reinterpret_cast<T *>(static_cast<char *>(ws) + off);
}

// The single-token path over `p.slots` slots: main, reduce, optional report.
ts_status run_slots(const float *x, const void *wg, const void *wu, const void *wd, const int32_t *route,
                    size_t expert_stride, ts_dtype dt, bool dense, const SlotPlan &p, float *out,
                    const float *slot_w, const ts_ffn_stats *stats, void *ws, hipStream_t st) {
    const bool want_seg = stats && (stats->gate_idx || stats->active_idx || stats->n_union);
    SlotArgs a;
    a.x = x;
    a.wg = wg;
    a.wu = wu;
    a.wd = wd;
    a.route = route;
    a.expert_stride = expert_stride;
    a.H = p.hidden;
    a.I = p.inter;
    a.tile = p.tile;
    a.ntiles = p.ntiles;
    a.slots_per_tok = p.slots_per_out;
    a.cnt = ws_at<int32_t>(ws, p.off_cnt);
    a.gseg = ws_at<int32_t>(ws, p.off_gseg);
    a.aseg = ws_at<int32_t>(ws, p.off_aseg);
    a.partial = ws_at<float>(ws, p.off_partial);
    a.want_seg = want_seg ? 1 : 0;
    {
        ProfScope ps("ffn_main", st);
        launch_main(dt, dense, p, st, a);
    }
    ts_status s = check_launch("ffn_main");
    if (s != TS_OK) return s;
    {
        ProfScope ps("ffn_reduce", st);
        dim3 grid((unsigned)((p.hidden / 4 + kRedCols4 - 1) / kRedCols4), (unsigned)p.outs);
        hipLaunchKernelGGL(ffn_reduce, grid, dim3(256), 0, st, a.partial, a.cnt, p.ntiles, p.hidden,
                           p.slots_per_out, slot_w, out);
    }
    s = check_launch("ffn_reduce");
    if (s != TS_OK) return s;
    if (stats && (stats->n_gate || stats->n_active || stats->gate_idx || stats->active_idx)) {
        ProfScope ps("ffn_stats", st);
        hipLaunchKernelGGL(ffn_stats, dim3((unsigned)p.slots), dim3(256), 0, st, a.cnt, a.gseg, a.aseg, p.ntiles,
                           p.tile, p.inter, stats->n_gate, stats->n_active, stats->gate_idx, stats->active_idx);
        s = check_launch("ffn_stats");
        if (s != TS_OK) return s;
    }
    if (stats && stats->n_union) {
        int32_t *flags = ws_at<int32_t>(ws, p.off_aux);
        ProfScope ps("ffn_stats", st);
        hipLaunchKernelGGL(fill_i32, dim3(64), dim3(256), 0, st, flags, (size_t)2 * p.inter, 0);
        hipLaunchKernelGGL(ffn_union_mark, dim3(256), dim3(256), 0, st, a.cnt, a.gseg, a.aseg, p.ntiles, p.tile,
                           p.slots, p.inter, flags);
        hipLaunchKernelGGL(ffn_union_count, dim3(1), dim3(256), 0, st, flags, p.inter, stats->n_union);
        s = check_launch("ffn_union");
        if (s != TS_OK) return s;
    }
    return TS_OK;
}

ts_status check_ffn_args(const float *x, const void *wg, const void *wu, const void *wd, ts_dtype dt, int batch,
                         int hidden, int inter, const float *out, const ts_ffn_stats *stats, const void *ws,
                         size_t ws_bytes, SlotPlan *plan) {
    ts_status s = check_dims(batch, hidden, inter, dt);
    if (s != TS_OK) return s;
    if (!x || !wg || !wu || !wd || !out) return TS_ERR_NULL;
    if (!aligned16(x) || !aligned16(wg) || !aligned16(wu) || !aligned16(wd) || !aligned16(out))
        return TS_ERR_ALIGN;
    s = check_stats(stats);
    if (s != TS_OK) return s;
    if (!plan_slots(hidden, inter, dt, batch, 1, plan)) return TS_ERR_SHAPE;
    if (!ws || ws_bytes < plan->total) return TS_ERR_WORKSPACE;
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
        (topk_idx && !aligned16(topk_idx)) || (topk_w && !aligned16(topk_w)))
        return TS_ERR_ALIGN;
    s = check_stats(stats);
    if (s != TS_OK) return s;
    if (stats && stats->n_union) return TS_ERR_UNSUPPORTED;
    if (!plan_slots(hidden, inter, dt, batch * K, K, plan)) return TS_ERR_SHAPE;
    if (!ws || ws_bytes < plan->total) return TS_ERR_WORKSPACE;
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
    int32_t *ridx = ws_at<int32_t>(ws, p.off_route_idx);
    float *rw = ws_at<float>(ws, p.off_route_w);
    {
        ProfScope ps("moe_router", st);
        if (dt == TS_F32)
            hipLaunchKernelGGL(moe_router<float>, dim3((unsigned)batch), dim3(256), 0, st, x,
                               static_cast<const float *>(wr), hidden, E, K, ridx, rw);
        else
            hipLaunchKernelGGL(moe_router<uint16_t>, dim3((unsigned)batch), dim3(256), 0, st, x,
                               static_cast<const uint16_t *>(wr), hidden, E, K, ridx, rw);
    }
    s = check_launch("moe_router");
    if (s != TS_OK) return s;
    s = run_slots(x, wg, wu, wd, ridx, (size_t)inter * (size_t)hidden, dt, dense, p, out, rw, stats, ws, st);
    if (s != TS_OK) return s;
    if (topk_idx) {
        if (hipMemcpyAsync(topk_idx, ridx, (size_t)batch * K * sizeof(int32_t), hipMemcpyDeviceToDevice, st) !=
            hipSuccess)
            return check_launch("topk_idx copy");
    }
    if (topk_w) {
        if (hipMemcpyAsync(topk_w, rw, (size_t)batch * K * sizeof(float), hipMemcpyDeviceToDevice, st) != hipSuccess)
            return check_launch("topk_w copy");
    }
    return TS_OK;
}

}  // namespace
}  // namespace ts

extern "C" {

ts_status ts_ffn_sparse(const float *x, const void *w_gate, const void *w_up, const void *w_down_t, ts_dtype wdtype,
                        int batch, int hidden, int inter, float *out, const ts_ffn_stats *stats, void *ws,
                        size_t ws_bytes, void *stream) {
    ts::SlotPlan p;
    ts_status s = ts::check_ffn_args(x, w_gate, w_up, w_down_t, wdtype, batch, hidden, inter, out, stats, ws,
                                     ws_bytes, &p);
    if (s != TS_OK) return s;
    return ts::run_slots(x, w_gate, w_up, w_down_t, nullptr, 0, wdtype, false, p, out, nullptr, stats, ws,
                         static_cast<hipStream_t>(stream));
}

ts_status ts_ffn_dense(const float *x, const void *w_gate, const void *w_up, const void *w_down_t, ts_dtype wdtype,
                       int batch, int hidden, int inter, float *out, void *ws, size_t ws_bytes, void *stream) {
    ts::SlotPlan p;
    ts_status s = ts::check_ffn_args(x, w_gate, w_up, w_down_t, wdtype, batch, hidden, inter, out, nullptr, ws,
                                     ws_bytes, &p);
    if (s != TS_OK) return s;
    return ts::run_slots(x, w_gate, w_up, w_down_t, nullptr, 0, wdtype, true, p, out, nullptr, nullptr, ws,
                         static_cast<hipStream_t>(stream));
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
