// Host-side planning and validation (no HIP headers; see ts_plan.h).
#include "ts_plan.h"

#include <algorithm>
#include <atomic>
#include <cstring>

namespace ts {

namespace {
std::atomic<int> g_tile{0};
std::atomic<int> g_gate_tile{0};
std::atomic<int> g_down_chunks{0};
std::atomic<int> g_path{0};
std::atomic<int> g_rif{0};
std::atomic<int> g_batch{0};
std::atomic<int> g_bx_gate{0};
std::atomic<int> g_bx_down{0};
std::atomic<int> g_bx_vgroup{0};
std::atomic<int> g_interleave{0};
std::atomic<int> g_bx_xtok{0};

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }
int esize(ts_dtype dt) { return dt == TS_F32 ? 4 : 2; }
}  // namespace

int tuned_tile() { return g_tile.load(); }

size_t align_up256(size_t v) { return align256(v); }

int tuned(const char *key) {
    if (std::strcmp(key, "ffn_tile") == 0) return g_tile.load();
    if (std::strcmp(key, "gate_tile") == 0) return g_gate_tile.load();
    if (std::strcmp(key, "down_chunks") == 0) return g_down_chunks.load();
    if (std::strcmp(key, "ffn_path") == 0) return g_path.load();
    if (std::strcmp(key, "rif") == 0) return g_rif.load();
    if (std::strcmp(key, "batch_path") == 0) return g_batch.load();
    if (std::strcmp(key, "bx_gate") == 0) return g_bx_gate.load();
    if (std::strcmp(key, "bx_down") == 0) return g_bx_down.load();
    if (std::strcmp(key, "bx_vgroup") == 0) return g_bx_vgroup.load();
    if (std::strcmp(key, "ffn_interleave") == 0) return g_interleave.load();
    if (std::strcmp(key, "bx_xtok") == 0) return g_bx_xtok.load();
    return 0;
}

// Neurons per workgroup for the single-token kernels: enough workgroups for
// one per compute unit over all slots (256 on MI355X), a multiple of 8 rows,
// at most `cap` (64 fused, 128 pipelined).  The ffn_tile knob overrides.
int choose_tile(int inter, int slots, int cap) {
    int t = tuned_tile();
    if (t > 0) return std::min(t, cap);
    long long per = ((long long)inter * slots + kTargetTiles - 1) / kTargetTiles;
    per = (per + 7) / 8 * 8;
    return (int)std::min<long long>(cap, std::max<long long>(8, per));
}

// The single-token kernels unroll each wave's rows (pipelined: a power of
// two of them, in pairs): rows per wave rounded up to a power of two leave
// no idle step, and measured faster (56 -> 64 neurons at inter 14336, 224
// workgroups: the dense comparator 3% less time, the sparse kernel 0.5-2.3%
// across 50-99% sparsity) as long as the grid keeps 7/8 of its target size.
int choose_pow2_tile(int inter, int slots, int cap) {
    const int t = choose_tile(inter, slots, cap);
    if (tuned_tile() > 0) return t;
    int r2 = 1;
    while (r2 * kWaves < t) r2 <<= 1;
    const int t2 = std::min(cap, r2 * kWaves);
    const long long wgs = (long long)slots * ((inter + t2 - 1) / t2);
    return wgs * 8 >= 7LL * kTargetTiles ? t2 : t;
}

ts_status check_dims(int batch, int hidden, int inter, ts_dtype dt) {
    if (dt != TS_F32 && dt != TS_BF16) return TS_ERR_DTYPE;
    if (batch < 1 || batch > kMaxBatch || inter < 1 || hidden < 8) return TS_ERR_SHAPE;
    if (dt == TS_BF16 && (hidden % 8 != 0 || hidden > 8192)) return TS_ERR_SHAPE;
    if (dt == TS_F32 && (hidden % 4 != 0 || hidden > 4096)) return TS_ERR_SHAPE;
    // every [inter][hidden] matrix must be indexable with 64-bit offsets and
    // the per-slot neuron count must fit a 32-bit index
    if ((long long)inter * (long long)hidden > (1LL << 40)) return TS_ERR_SHAPE;
    return TS_OK;
}

ts_status check_moe_dims(int batch, int hidden, int inter, int n_experts, int top_k, ts_dtype dt) {
    ts_status s = check_dims(batch, hidden, inter, dt);
    if (s != TS_OK) return s;
    if (n_experts < 1 || n_experts > kMaxExperts) return TS_ERR_SHAPE;
    if (top_k < 1 || top_k > n_experts || top_k > kMaxTopK) return TS_ERR_SHAPE;
    return TS_OK;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

ts_status check_stats(const ts_ffn_stats *s) {
    if (!s) return TS_OK;
    const void *ps[] = {s->n_gate, s->n_active, s->gate_idx, s->active_idx, s->n_union};
    for (const void *p : ps)
        if (p && !aligned4(p)) return TS_ERR_ALIGN;
    return TS_OK;
}

bool plan_slots(int hidden, int inter, ts_dtype dt, int slots, int slots_per_out, SlotPlan *p, bool pow2_tiles) {
    if (check_dims(1, hidden, inter, dt) != TS_OK || slots < 1 || slots_per_out < 1 ||
        slots % slots_per_out != 0)
        return false;
    SlotPlan q;
    q.hidden = hidden;
    q.inter = inter;
    q.esz = esize(dt);
    q.ce = 16 / q.esz;
    q.nch = hidden / q.ce;
    int need = (q.nch + 63) / 64;
    q.nc = 1;
    while (q.nc < need) q.nc <<= 1;
    q.tile = pow2_tiles ? choose_pow2_tile(inter, slots, kMaxPipeTile) : choose_tile(inter, slots, kMaxPipeTile);
    q.ntiles = (inter + q.tile - 1) / q.tile;
    q.ftile = pow2_tiles ? choose_pow2_tile(inter, slots, kMaxTile) : choose_tile(inter, slots, kMaxTile);
    q.fntiles = (inter + q.ftile - 1) / q.ftile;
    q.slots = slots;
    q.slots_per_out = slots_per_out;
    q.outs = slots / slots_per_out;
    // regions sized for whichever kernel runs (the fused one has more tiles)
    const size_t nst = (size_t)slots * (size_t)std::max(q.ntiles, q.fntiles);
    const size_t nseg = (size_t)slots * std::max((size_t)q.ntiles * q.tile, (size_t)q.fntiles * q.ftile);
    size_t off = 0;
    q.off_cnt = off;
    off = align256(off + nst * 2 * sizeof(int32_t));
    q.off_gseg = off;
    off = align256(off + nseg * sizeof(int32_t));
    q.off_aseg = off;
    off = align256(off + nseg * sizeof(int32_t));
    q.off_hseg = off;
    off = align256(off + nseg * sizeof(float));
    q.off_partial = off;
    off = align256(off + nst * (size_t)hidden * sizeof(float));
    q.off_route_idx = off;
    off = align256(off + (size_t)slots * sizeof(int32_t));
    q.off_route_w = off;
    off = align256(off + (size_t)slots * sizeof(float));
    q.off_aux = off;  // union flags of the activity report: [2][inter]
    off = align256(off + (size_t)2 * (size_t)inter * sizeof(int32_t));

    // Split path.  Gate+up tiles: about three 4-wave workgroups per compute
    // unit over all slots, a multiple of 4 rows (one share per wave).
    int gt = g_gate_tile.load();
    if (gt <= 0) {
        long long per = ((long long)inter * slots + kGateTargetBlocks - 1) / kGateTargetBlocks;
        per = (per + 3) / 4 * 4;
        gt = (int)std::min<long long>(kMaxTile, std::max<long long>(8, per));
    }
    q.gtile = gt;
    q.gntiles = (inter + gt - 1) / gt;
    // Down: 64 chunks of 16 bytes per slice; chunks of tiles sized so that a
    // chunk's rows fit the LDS list and there are ~256 workgroups in all.
    q.nslices = (q.nch + 63) / 64;
    // tpc * gt <= kDownMaxRows and tpc <= kDownMaxTiles bound the LDS lists.
    int want = g_down_chunks.load();
    if (want <= 0) want = std::max(1, kDownTargetBlocks / std::max(1, q.nslices * slots));
    int nchunks = std::max(1, std::min(want, q.gntiles));
    int tpc = (q.gntiles + nchunks - 1) / nchunks;
    tpc = std::min(tpc, std::min(kDownMaxTiles, kDownMaxRows / gt));
    q.tpc = std::max(1, tpc);
    q.nchunks = (q.gntiles + q.tpc - 1) / q.tpc;
    {
        // the same decomposition over the pipelined kernel's tiles (its
        // partial rows go to off_partial, which holds one per tile)
        int pn = std::max(1, std::min(want, q.ntiles));
        int ptpc = (q.ntiles + pn - 1) / pn;
        ptpc = std::min(ptpc, std::min(kDownMaxTiles, kDownMaxRows / q.tile));
        q.ptpc = std::max(1, ptpc);
        q.pnchunks = (q.ntiles + q.ptpc - 1) / q.ptpc;
    }
    size_t gst = (size_t)slots * (size_t)q.gntiles;
    q.off_gcnt = off;
    off = align256(off + gst * 2 * sizeof(int32_t));
    q.off_ggseg = off;
    off = align256(off + gst * (size_t)gt * sizeof(int32_t));
    q.off_gaseg = off;
    off = align256(off + gst * (size_t)gt * sizeof(int32_t));
    q.off_ghseg = off;
    off = align256(off + gst * (size_t)gt * sizeof(float));
    q.off_dpartial = off;
    off = align256(off + (size_t)slots * q.nchunks * (size_t)hidden * sizeof(float));
    const size_t kst = std::max(gst, (size_t)slots * (size_t)q.ntiles);
    const size_t kseg = std::max(gst * (size_t)gt, (size_t)slots * (size_t)q.ntiles * q.tile);
    q.off_kcnt = off;
    off = align256(off + kst * 2 * sizeof(int32_t));
    q.off_kaseg = off;
    off = align256(off + kseg * sizeof(int32_t));
    q.off_khseg = off;
    off = align256(off + kseg * sizeof(float));
    q.total = off;
    *p = q;
    return true;
}

bool plan_batch(int batch, int hidden, int inter, int experts, int top_k, ts_dtype dt, BatchPlan *p) {
    if (check_dims(batch, hidden, inter, dt) != TS_OK || dt != TS_BF16 || experts < 1 || top_k < 1) return false;
    if (batch > kBxMaxTokens) return false;
    // the gate / up kernel addresses rows with 32-bit byte offsets into one matrix
    if ((unsigned long long)inter * (unsigned long long)hidden * 2ull >= (1ull << 32)) return false;
    BatchPlan q;
    q.batch = batch;
    q.hidden = hidden;
    q.inter = inter;
    q.top_k = top_k;
    q.experts = experts;
    // token slots per group (the kernels are built for 8, 16, 32 and 64):
    // the batch for one weight set; for several, twice an expert's expected
    // load batch * top_k / experts (the "bx_vgroup" knob 1: the batch)
    int slots = batch;
    if (experts > 1 && g_bx_vgroup.load() == 0)
        slots = std::min(batch, 2 * ((batch * top_k + experts - 1) / experts));
    q.tok = slots <= 8 ? 8 : (slots <= 16 ? 16 : (slots <= 32 ? 32 : 64));
    q.vpe = (batch + q.tok - 1) / q.tok;  // an expert holds each token at most once
    q.groups = experts * q.vpe;
    const int groups = q.groups;
    q.bpad = q.tok;
    q.hpad = (hidden + kBxKQuant - 1) / kBxKQuant * kBxKQuant;
    q.ntiles = (inter + kBxRows - 1) / kBxRows;
    q.nslices = (hidden + kBxSliceCols - 1) / kBxSliceCols;
    // down: about one workgroup per compute unit (measured: two rounds of
    // workgroups, or two per unit, run slower than one with longer lists)
    int want = g_down_chunks.load();
    if (want <= 0) want = std::max(1, 256 / (q.nslices * groups));
    q.nchunks = std::max(1, std::min(want, q.ntiles));
    q.tpc = std::min((q.ntiles + q.nchunks - 1) / q.nchunks, bx_down_tiles(q.tok));
    q.nchunks = (q.ntiles + q.tpc - 1) / q.tpc;
    const size_t G = (size_t)groups, T = (size_t)q.ntiles;
    size_t off = 0;
    q.off_gcount = off;  // tokens per group
    off = align256(off + G * sizeof(int32_t));
    q.off_tslot = off;   // (group, slot) of each (token, routed rank)
    off = align256(off + (size_t)batch * top_k * 2 * sizeof(int32_t));
    q.off_xhl = off;     // x split into bf16 high and low parts: [G][2][tok][hpad]
    off = align256(off + G * 2 * q.tok * q.hpad * sizeof(uint16_t));
    q.off_cnt = off;     // per tile: |union G|, |union A|
    off = align256(off + G * T * 2 * sizeof(int32_t));
    q.off_arow = off;    // per tile: row (within the tile) of each of its 32 active slots, bytes
    off = align256(off + G * T * kBxRows);
    q.off_hfrag = off;   // per tile: Combined as bf16 high / low, [2][tok][32 slots]
    off = align256(off + G * T * 2 * q.tok * kBxRows * sizeof(uint16_t));
    q.off_gmask = off;   // per tile and token: open-gate rows (bit mask)
    off = align256(off + G * T * q.tok * sizeof(uint32_t));
    q.off_amask = off;   // per tile and token: active rows (bit mask)
    off = align256(off + G * T * q.tok * sizeof(uint32_t));
    q.off_partial = off; // down partials: [G][tok][nchunks][hidden]
    off = align256(off + G * q.tok * (size_t)q.nchunks * hidden * sizeof(float));
    q.off_union = off;
    off = align256(off + 4 * sizeof(int32_t));
    q.total = off;
    *p = q;
    return true;
}

// Chunk of list entries per workgroup: enough workgroups for one per compute
// unit over the whole batch (one 8-wave workgroup fills a compute unit), a
// multiple of 4 up to 8 entries and of 8 above, at most 128; the ffn_tile
// knob overrides.
bool plan_given(int batch, int hidden, int inter, int max_count, ts_dtype dt, GivenPlan *p) {
    if (check_dims(batch, hidden, inter, dt) != TS_OK || max_count < 1 || max_count > kMaxGivenList) return false;
    GivenPlan q;
    q.batch = batch;
    q.hidden = hidden;
    q.inter = inter;
    q.maxc = max_count;
    q.nch = hidden / (16 / esize(dt));
    const int need = (q.nch + 63) / 64;
    q.nc = 1;
    while (q.nc < need) q.nc <<= 1;
    int t = tuned_tile();
    if (t <= 0) {
        long long per = ((long long)max_count * batch + kTargetTiles - 1) / kTargetTiles;
        // past one entry per wave, whole entries per wave (a multiple of 8:
        // 16 against 12 at the 90% workload measured 3.5% faster)
        per = per > kWaves ? (per + kWaves - 1) / kWaves * kWaves : (per + 3) / 4 * 4;
        t = (int)std::max(4LL, std::min((long long)kMaxPipeTile, per));
    }
    q.chunk = std::min(t, kMaxPipeTile);
    q.nchunks = (max_count + q.chunk - 1) / q.chunk;
    const size_t rows = (size_t)batch * q.nchunks;
    size_t off = 0;
    q.off_partial = off;  // [batch][nchunks][hidden] partial output rows
    off = align256(off + rows * (size_t)hidden * sizeof(float));
    q.off_cnt = off;      // [batch][nchunks][2] listed entries with gate > 0 / non-zero Combined
    off = align256(off + rows * 2 * sizeof(int32_t));
    q.total = off;
    *p = q;
    return true;
}

size_t given_ws_bytes(int batch, int hidden, int inter, int max_count, ts_dtype dt) {
    GivenPlan g;
    return plan_given(batch, hidden, inter, max_count, dt, &g) ? g.total : 0;
}

// Both the single-token and the batched plans must fit (the entry points
// pick a path at call time, and the tuning knobs can move the choice).
size_t ffn_ws_bytes(int batch, int hidden, int inter, ts_dtype dt) {
    if (check_dims(batch, hidden, inter, dt) != TS_OK) return 0;
    SlotPlan sp, tp;
    if (!plan_slots(hidden, inter, dt, batch, 1, &sp) || !plan_slots(hidden, inter, dt, batch, 1, &tp, false))
        return 0;
    size_t n = std::max(sp.total, tp.total);  // (tp: the top-k mask's plan)
    BatchPlan bp;
    if (batch > 1 && plan_batch(std::min(batch, kBxMaxTokens), hidden, inter, 1, 1, dt, &bp))
        n = std::max(n, bp.total);
    return n;
}

size_t moe_route_offset(int batch, int hidden, int inter, int n_experts, int top_k, ts_dtype dt) {
    SlotPlan sp;
    if (!plan_slots(hidden, inter, dt, batch * top_k, top_k, &sp)) return 0;
    size_t n = sp.total;
    BatchPlan bp;
    if (batch > 1 && plan_batch(batch, hidden, inter, n_experts, top_k, dt, &bp)) n = std::max(n, bp.total);
    return align256(n);
}

size_t moe_ws_bytes(int batch, int hidden, int inter, int n_experts, int top_k, ts_dtype dt) {
    if (check_moe_dims(batch, hidden, inter, n_experts, top_k, dt) != TS_OK) return 0;
    // the router's outputs (expert ids, then weights) live past both plans
    return moe_route_offset(batch, hidden, inter, n_experts, top_k, dt) +
           2 * align256((size_t)batch * top_k * sizeof(int32_t));
}

}  // namespace ts

extern "C" {

const char *ts_status_str(ts_status s) {
    switch (s) {
    case TS_OK: return "TS_OK";
    case TS_ERR_NULL: return "TS_ERR_NULL: a required pointer is NULL";
    case TS_ERR_SHAPE: return "TS_ERR_SHAPE: size argument out of range";
    case TS_ERR_DTYPE: return "TS_ERR_DTYPE: unknown weight dtype";
    case TS_ERR_ALIGN: return "TS_ERR_ALIGN: pointer not aligned";
    case TS_ERR_WORKSPACE: return "TS_ERR_WORKSPACE: workspace missing or too small";
    case TS_ERR_HIP: return "TS_ERR_HIP: HIP runtime failure";
    case TS_ERR_UNSUPPORTED: return "TS_ERR_UNSUPPORTED: request not served by the library";
    }
    return "unknown ts_status";
}

size_t ts_ffn_workspace_bytes(int batch, int hidden, int inter, ts_dtype wdtype) {
    return ts::ffn_ws_bytes(batch, hidden, inter, wdtype);
}

size_t ts_ffn_given_workspace_bytes(int batch, int hidden, int inter, int max_count, ts_dtype wdtype) {
    return ts::given_ws_bytes(batch, hidden, inter, max_count, wdtype);
}

size_t ts_moe_workspace_bytes(int batch, int hidden, int inter, int n_experts, int top_k, ts_dtype wdtype) {
    return ts::moe_ws_bytes(batch, hidden, inter, n_experts, top_k, wdtype);
}

ts_status ts_tune_set(const char *key, int value) {
    if (!key) return TS_ERR_NULL;
    if (std::strcmp(key, "ffn_tile") == 0) {
        if (value != 0 && (value < 4 || value > ts::kMaxPipeTile || value % 4 != 0)) return TS_ERR_SHAPE;
        ts::g_tile.store(value);
        return TS_OK;
    }
    if (std::strcmp(key, "gate_tile") == 0) {
        if (value != 0 && (value < 4 || value > ts::kMaxTile || value % 4 != 0)) return TS_ERR_SHAPE;
        ts::g_gate_tile.store(value);
        return TS_OK;
    }
    if (std::strcmp(key, "down_chunks") == 0) {
        if (value < 0 || value > 4096) return TS_ERR_SHAPE;
        ts::g_down_chunks.store(value);
        return TS_OK;
    }
    if (std::strcmp(key, "ffn_path") == 0) {
        if (value < 0 || value > 2) return TS_ERR_SHAPE;
        ts::g_path.store(value);
        return TS_OK;
    }
    if (std::strcmp(key, "rif") == 0) {
        if (value < 0 || value > 2) return TS_ERR_SHAPE;
        ts::g_rif.store(value);
        return TS_OK;
    }
    if (std::strcmp(key, "batch_path") == 0) {
        if (value < 0 || value > 1) return TS_ERR_SHAPE;
        ts::g_batch.store(value);
        return TS_OK;
    }
    if (std::strcmp(key, "bx_gate") == 0) {
        if (value < 0 || value > 3) return TS_ERR_SHAPE;
        ts::g_bx_gate.store(value);
        return TS_OK;
    }
    if (std::strcmp(key, "bx_down") == 0) {
        if (value < 0 || value > 1) return TS_ERR_SHAPE;
        ts::g_bx_down.store(value);
        return TS_OK;
    }
    if (std::strcmp(key, "bx_vgroup") == 0) {
        if (value < 0 || value > 1) return TS_ERR_SHAPE;
        ts::g_bx_vgroup.store(value);
        return TS_OK;
    }
    if (std::strcmp(key, "ffn_interleave") == 0) {
        if (value < 0 || value > 1) return TS_ERR_SHAPE;
        ts::g_interleave.store(value);
        return TS_OK;
    }
    if (std::strcmp(key, "bx_xtok") == 0) {
        if (value < 0 || value > 1) return TS_ERR_SHAPE;
        ts::g_bx_xtok.store(value);
        return TS_OK;
    }
    return TS_ERR_SHAPE;
}

const char *ts_version(void) { return "turbosparse-gfx950 0.1"; }

}  // extern "C"
