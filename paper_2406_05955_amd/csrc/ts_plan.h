// Host-side planning and argument validation for the turbosparse C ABI.
// This unit includes no HIP header: it decides launch shapes and workspace
// layout and rejects bad arguments before anything touches a device.
#pragma once

#include <cstddef>
#include <cstdint>

#include "turbosparse.h"

namespace ts {

constexpr int kMaxBatch = 256;
constexpr int kMaxExperts = 64;
constexpr int kMaxTopK = 8;
constexpr int kWaves = 8;                 // waves per workgroup of the single-token kernel
constexpr int kThreads = kWaves * 64;     // 512 threads
constexpr int kMaxTile = 64;              // neurons per workgroup of the fused / gate+up kernels (one ballot)
constexpr int kMaxPipeTile = 128;         // neurons per workgroup of the pipelined kernel (two ballots)
constexpr int kTargetTiles = 256;         // one workgroup per compute unit on MI355X
constexpr int kGateWaves = 4;             // waves per workgroup of the gate+up kernel
constexpr int kGateThreads = kGateWaves * 64;
constexpr int kGateTargetBlocks = 768;    // three 4-wave workgroups per compute unit
constexpr int kDownThreads = 256;         // 4 waves per down workgroup
constexpr int kDownMaxRows = 1024;        // active rows one down workgroup can list in LDS
constexpr int kDownTargetBlocks = 256;
constexpr int kDownMaxTiles = 256;        // gate+up tiles one down workgroup can list
constexpr int kSelMax = 16384;            // Combined values the top-k selection holds in LDS (inter limit)
constexpr int kSelMaxTiles = 2048;        // gate+up tiles per slot the selection lists (inter / 8)
constexpr int kSelSpan = kSelMax + 128;   // padded list positions per slot it holds (last tile's padding)
constexpr int kIlvMaxInter = 131072;     // interleaved tiles: the activity report's LDS bitmaps hold this many neurons

// Selection keys of the top-k magnitude mask (Eq. mask: the largest
// |Combined| are kept).  A key is the fp32 bit pattern of the magnitude:
// the sign bit cleared and NaN patterns clamped to +inf, so bit 31 is always
// 0 and unsigned key order is magnitude order.  The selection kernel adds
// one (sel_key) so that no listed entry has key 0.  Radix digits are 8 bits
// from bit 23 up (the exponent first), then bits 22..15, 14..7 and 7..0;
// the last digit repeats bit 7, which the prefix already fixes.  The
// functions are constexpr so the kernels and the host-side checks share one
// definition.
constexpr uint32_t sel_mag(uint32_t bits) {
    return (bits & 0x7fffffffu) > 0x7f800000u ? 0x7f800000u : (bits & 0x7fffffffu);
}
constexpr uint32_t sel_key(uint32_t bits) { return sel_mag(bits) + 1u; }
constexpr int kSelTopShift = 23;
constexpr int sel_next_shift(int shift) { return shift >= 8 ? shift - 8 : (shift > 0 ? 0 : -1); }

// Workspace layout and launch shape shared by the single-token path (one
// "slot" = one (token, expert) pair processed against one weight set).
struct SlotPlan {
    int hidden = 0, inter = 0, esz = 0;
    int ce = 0;        // weight elements per 16-byte chunk
    int nch = 0;       // 16-byte chunks per weight row
    int nc = 0;        // chunks per lane in the row dot products (power of two)
    int tile = 0;      // neurons per workgroup of the pipelined kernel
    int ntiles = 0;    // its workgroups per slot
    int ftile = 0;     // neurons per workgroup of the fused kernel
    int fntiles = 0;   // its workgroups per slot
    int slots = 0;     // number of slots
    int outs = 0;      // output rows (slots / slots_per_out)
    int slots_per_out = 1;
    // split sparse path: gate+up kernel tiles and down kernel decomposition
    int gtile = 0;     // neurons per gate+up workgroup
    int gntiles = 0;   // gate+up workgroups per slot
    int nslices = 0;   // column slices of the down kernel (64 chunks of 16 bytes each)
    int nchunks = 0;   // groups of gate+up tiles per slot in the down kernel
    int tpc = 0;       // gate+up tiles per chunk
    int pnchunks = 0;  // the down kernel over the pipelined kernel's tiles (top-k mask): chunks per slot
    int ptpc = 0;      // and pipelined tiles per chunk
    // byte offsets into the workspace
    size_t off_cnt = 0, off_gseg = 0, off_aseg = 0, off_partial = 0;
    size_t off_route_idx = 0, off_route_w = 0, off_aux = 0;
    size_t off_gcnt = 0, off_ggseg = 0, off_gaseg = 0, off_ghseg = 0, off_dpartial = 0;
    size_t off_hseg = 0;  // Combined values of aseg (pipelined kernel's emit mode)
    // the top-k mask's kept lists (either kernel's tile layout)
    size_t off_kcnt = 0, off_kaseg = 0, off_khseg = 0;
    size_t total = 0;
};

// Batched path (bf16 weights, several tokens per weight set): every weight
// row is read once per pass for up to kBxMaxTokens tokens, the contractions
// run on the matrix cores.  A "group" is one weight set with its tokens: the
// FFN has one group holding the batch, the MoE layer one group per expert
// holding the tokens routed to it.
constexpr int kBxMaxTokens = 64;  // tokens per group and pass
constexpr int kBxRows = 32;       // neurons per gate+up workgroup tile (and per down K block)
constexpr int kBxSliceCols = 128; // output columns per down wave
// gate+up tiles per down workgroup at most: its row list (4 bytes per
// entry, room for every row of every tile) lives in LDS next to the
// staging.  At 32 token slots a compute unit holds one workgroup whatever
// the list, so a workgroup takes up to 224 tiles (half a 14336-neuron
// expert: two rounds of workgroups instead of fourteen, MoE batch 64 down
// 112 -> 86 us; whole experts, one round, 89 us: the experts drawing the
// most tokens set that round's length; 160 or 128 tiles 92-93 us); at 8
// and 16, 64 tiles (shorter workgroups, three or two per unit, measured
// faster than 96- or 224-tile ones at 85% in-expert sparsity); at 64 the
// staging leaves room for 64.
constexpr int bx_down_tiles(int tok) { return tok == 32 ? 224 : 64; }

// Group at grid position gi of the batched gate / up and down grids: every
// weight set's first group before any further one.  An expert's further
// groups take the tokens past its first `tok` and are nearly always empty;
// their workgroups, which only find that out and exit, then come at the end
// of the grid instead of between the working ones (MoE batch 16: 223
// against 227 us per layer).  A bijection on [0, G) for G = weight sets x
// vpe, which plan_batch guarantees.
constexpr int bx_group_at(int gi, int G, int vpe) { return (gi % (G / vpe)) * vpe + gi / (G / vpe); }
constexpr int kBxKQuant = 1024;   // the hidden dimension is padded to this (4 waves x 2 batches x 128)

// A "group" is one weight set with up to `tok` of its tokens.  The FFN has
// one group holding the batch.  In the MoE layer each expert's token list
// (known only on the device) is cut into `vpe` groups of `tok` consecutive
// entries, with tok about twice the expected load of an expert: an expert
// that draws more tokens than that takes a second group (its weights are
// read once more), and a group that draws none exits at once.
struct BatchPlan {
    int batch = 0, hidden = 0, inter = 0, groups = 1, top_k = 1;
    int experts = 1;     // weight sets
    int vpe = 1;         // groups per weight set (groups = experts * vpe)
    int tok = 0;         // token slots per group: 8 (high / low x parts share one MFMA tile), 16, 32 or 64
    int bpad = 0;        // = tok
    int hpad = 0;        // hidden rounded up to kBxKQuant (gate / up K range, zero x past hidden)
    int ntiles = 0;      // 32-neuron tiles per group
    int nslices = 0;     // 128-column slices of the down kernel
    int nchunks = 0;     // tile chunks per group in the down kernel
    int tpc = 0;         // tiles per chunk (<= bx_down_tiles(tok))
    size_t off_gcount = 0, off_tslot = 0, off_xhl = 0, off_cnt = 0, off_arow = 0, off_hfrag = 0;
    size_t off_gmask = 0, off_amask = 0, off_partial = 0, off_union = 0;
    size_t total = 0;
};

// Given-list path (ts_ffn_sparse_given): each token's list is cut into
// chunks of `chunk` entries, one pipelined workgroup per (token, chunk).
constexpr int kMaxGivenList = 1 << 24;  // entries per token list
struct GivenPlan {
    int batch = 0, hidden = 0, inter = 0, maxc = 0;
    int nch = 0, nc = 0;     // 16-byte chunks per row, per lane (power of two)
    int chunk = 0, nchunks = 0;
    size_t off_partial = 0, off_cnt = 0, total = 0;
};
bool plan_given(int batch, int hidden, int inter, int max_count, ts_dtype dt, GivenPlan *p);
size_t given_ws_bytes(int batch, int hidden, int inter, int max_count, ts_dtype dt);

int tuned_tile();
int choose_tile(int inter, int slots, int cap);
int choose_pow2_tile(int inter, int slots, int cap);
int tuned(const char *key);
// pow2_tiles: the pipelined / fused kernels' tiles per choose_pow2_tile (the
// default); false: per choose_tile (the top-k mask's sequence, measured
// faster with the finer tiles)
bool plan_slots(int hidden, int inter, ts_dtype dt, int slots, int slots_per_out, SlotPlan *p,
                bool pow2_tiles = true);
bool plan_batch(int batch, int hidden, int inter, int groups, int top_k, ts_dtype dt, BatchPlan *p);

ts_status check_dims(int batch, int hidden, int inter, ts_dtype dt);
ts_status check_moe_dims(int batch, int hidden, int inter, int n_experts, int top_k, ts_dtype dt);
bool aligned16(const void *p);
bool aligned4(const void *p);
ts_status check_stats(const ts_ffn_stats *s);

size_t ffn_ws_bytes(int batch, int hidden, int inter, ts_dtype dt);
size_t moe_ws_bytes(int batch, int hidden, int inter, int n_experts, int top_k, ts_dtype dt);
size_t moe_route_offset(int batch, int hidden, int inter, int n_experts, int top_k, ts_dtype dt);
size_t align_up256(size_t v);

}  // namespace ts
