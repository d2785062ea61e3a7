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
constexpr int kMaxTile = 64;              // neurons per workgroup: one wave ballot covers the tile
constexpr int kTargetTiles = 256;         // one workgroup per compute unit on MI355X

// Workspace layout and launch shape shared by the single-token path (one
// "slot" = one (token, expert) pair processed against one weight set).
struct SlotPlan {
    int hidden = 0, inter = 0, esz = 0;
    int ce = 0;        // weight elements per 16-byte chunk
    int nch = 0;       // 16-byte chunks per weight row
    int nc = 0;        // chunks per lane in the row dot products (power of two)
    int tile = 0;      // neurons per workgroup
    int ntiles = 0;    // workgroups per slot
    int slots = 0;     // number of slots
    int outs = 0;      // output rows (slots / slots_per_out)
    int slots_per_out = 1;
    // byte offsets into the workspace
    size_t off_cnt = 0, off_gseg = 0, off_aseg = 0, off_partial = 0;
    size_t off_route_idx = 0, off_route_w = 0, off_aux = 0;
    size_t total = 0;
};

// Batched (batch > 1) FFN path: row unions and matrix-core contraction.
struct BatchPlan {
    int batch = 0, hidden = 0, inter = 0, esz = 0;
    int bpad = 0;            // batch rounded up to the MFMA tile (16 or 32)
    int gate_rows = 0;       // neurons per gate workgroup
    int gate_blocks = 0;
    int up_rows = 0;         // union rows per up workgroup
    int down_split = 0;      // split of the union list in the down contraction
    int down_cols = 0;       // output columns per down workgroup
    size_t off_mask = 0, off_g = 0, off_cnt = 0, off_list = 0, off_h = 0, off_partial = 0, off_misc = 0;
    size_t total = 0;
};

int tuned_tile();
int choose_tile(int inter);
bool plan_slots(int hidden, int inter, ts_dtype dt, int slots, int slots_per_out, SlotPlan *p);
bool plan_batch(int batch, int hidden, int inter, ts_dtype dt, BatchPlan *p);

ts_status check_dims(int batch, int hidden, int inter, ts_dtype dt);
ts_status check_moe_dims(int batch, int hidden, int inter, int n_experts, int top_k, ts_dtype dt);
bool aligned16(const void *p);
bool aligned4(const void *p);
ts_status check_stats(const ts_ffn_stats *s);

size_t ffn_ws_bytes(int batch, int hidden, int inter, ts_dtype dt);
size_t moe_ws_bytes(int batch, int hidden, int inter, int n_experts, int top_k, ts_dtype dt);

}  // namespace ts
