// Host-only check of the launch planner's invariants over a grid of shapes.
// Built with g++ (sanitizers on) by tests/test_plan_cpu.py; prints "ok" or
// the first violated invariant.
#include <algorithm>
#include <cstdio>
#include <vector>

#include "ts_plan.h"

using namespace ts;

static int fail(const char *what, int B, int H, int I, int S) {
    std::printf("FAIL %s B=%d H=%d I=%d slots=%d\n", what, B, H, I, S);
    return 1;
}

int main() {
    // the tile rule: about one workgroup per compute unit, rows per wave a
    // power of two while the grid keeps 7/8 of its size
    if (choose_pow2_tile(14336, 1, kMaxPipeTile) != 64) return fail("pow2 tile 14336", 0, 0, 14336, 1);
    if (choose_pow2_tile(14336, 2, kMaxPipeTile) != 128) return fail("pow2 tile 14336 x2", 0, 0, 14336, 2);
    if (choose_pow2_tile(9000, 1, kMaxPipeTile) != 40) return fail("pow2 tile 9000", 0, 0, 9000, 1);
    if (choose_pow2_tile(14336, 1, kMaxTile) != 64) return fail("pow2 fused tile 14336", 0, 0, 14336, 1);
    if (choose_tile(14336, 1, kMaxPipeTile) != 56) return fail("tile 14336", 0, 0, 14336, 1);
    for (int I = 1; I <= 40000; I += 37)
        for (int S : {1, 2, 3, 16}) {
            const int t = choose_pow2_tile(I, S, kMaxPipeTile), b = choose_tile(I, S, kMaxPipeTile);
            if (t % 8 || t < b || t > kMaxPipeTile) return fail("pow2 tile bounds", 0, 0, I, S);
            if (t != b && (long long)S * ((I + t - 1) / t) * 8 < 7LL * kTargetTiles) return fail("pow2 tile grid", 0, 0, I, S);
        }
    const int Hs[] = {8, 16, 40, 200, 512, 1000, 2048, 4096, 6144, 8192};
    const int Is[] = {1, 3, 7, 8, 9, 63, 64, 65, 130, 777, 1792, 3001, 14336, 28672, 100000};
    const int Ss[] = {1, 2, 3, 8, 16, 32, 64, 256, 512, 2048};
    const int tiles[] = {0, 4, 8, 12, 20, 64};
    const int ftiles[] = {0, 8, 56, 100, 128};
    const int chunks[] = {0, 1, 7, 32, 4096};
    const ts_dtype dts[] = {TS_F32, TS_BF16};
    for (ts_dtype dt : dts)
        for (int H : Hs)
            for (int I : Is)
                for (int S : Ss)
                    for (int gt : tiles)
                        for (int ch : chunks) {
                            const int ft = ftiles[(gt + ch) % 5];
                            if (ts_tune_set("ffn_tile", ft) != TS_OK) return fail("tune ffn_tile", 0, H, I, S);
                            if (ts_tune_set("gate_tile", gt) != TS_OK) return fail("tune gate_tile", 0, H, I, S);
                            if (ts_tune_set("down_chunks", ch) != TS_OK) return fail("tune down_chunks", 0, H, I, S);
                            SlotPlan p;
                            bool ok = plan_slots(H, I, dt, S, 1, &p);
                            bool valid = check_dims(1, H, I, dt) == TS_OK;
                            if (ok != valid) return fail("plan/validation disagree", 1, H, I, S);
                            if (!ok) continue;
                            if (p.gtile < 4 || p.gtile > kMaxTile || p.gtile % 4) return fail("gtile", 1, H, I, S);
                            if ((long long)p.gntiles * p.gtile < I || (long long)(p.gntiles - 1) * p.gtile >= I)
                                return fail("gntiles", 1, H, I, S);
                            if (p.tpc < 1 || p.tpc > kDownMaxTiles || p.tpc * p.gtile > kDownMaxRows)
                                return fail("tpc bounds", 1, H, I, S);
                            if ((long long)p.nchunks * p.tpc < p.gntiles || (long long)(p.nchunks - 1) * p.tpc >= p.gntiles)
                                return fail("nchunks cover", 1, H, I, S);
                            if (p.nslices * 64 < p.nch || (p.nslices - 1) * 64 >= p.nch) return fail("nslices", 1, H, I, S);
                            if (p.nc * 64 < p.nch || p.nc > 16) return fail("nc", 1, H, I, S);
                            if (p.tile < 8 || p.tile > kMaxPipeTile) return fail("tile", 1, H, I, S);
                            if ((long long)p.ntiles * p.tile < I) return fail("ntiles", 1, H, I, S);
                            if (p.ftile < 8 || p.ftile > kMaxTile) return fail("ftile", 1, H, I, S);
                            if ((long long)p.fntiles * p.ftile < I) return fail("fntiles", 1, H, I, S);
                            if (p.off_gseg - p.off_cnt < (size_t)S * std::max(p.ntiles, p.fntiles) * 8)
                                return fail("cnt size", 1, H, I, S);
                            if (p.off_aseg - p.off_gseg <
                                (size_t)S * std::max((size_t)p.ntiles * p.tile, (size_t)p.fntiles * p.ftile) * 4)
                                return fail("seg size", 1, H, I, S);
                            if (p.off_route_idx - p.off_partial <
                                (size_t)S * std::max(p.ntiles, p.fntiles) * (size_t)H * 4)
                                return fail("partial size", 1, H, I, S);
                            // workspace regions ordered, aligned and inside total
                            size_t offs[] = {p.off_cnt, p.off_gseg, p.off_aseg, p.off_partial, p.off_route_idx,
                                             p.off_route_w, p.off_aux, p.off_gcnt, p.off_ggseg, p.off_gaseg,
                                             p.off_ghseg, p.off_dpartial, p.off_kcnt, p.total};
                            for (int k = 1; k < 14; ++k)
                                if (offs[k] < offs[k - 1] || offs[k] % 256) return fail("ws layout", 1, H, I, S);
                            size_t need_dp = (size_t)S * p.nchunks * H * 4;
                            if (p.off_kcnt - p.off_dpartial < need_dp) return fail("dpartial size", 1, H, I, S);
                            if (p.off_gaseg - p.off_ggseg < (size_t)S * p.gntiles * p.gtile * 4)
                                return fail("gseg size", 1, H, I, S);
                        }
    ts_tune_set("gate_tile", 0);
    ts_tune_set("down_chunks", 0);
    ts_tune_set("ffn_tile", 0);

    // the batched (matrix-core) plan: token slots per group, groups per
    // weight set, the down kernel's chunks within its row list, and the
    // workspace regions the kernels index (the x region also holds the
    // router's token-major x split: batch x hpad x 4 bytes)
    const int Bs[] = {2, 3, 8, 9, 16, 17, 32, 33, 48, 64};
    const int Es[] = {1, 2, 3, 8, 64};
    for (int vg : {0, 1})
        for (int dc : {0, 7, 14})
            for (int B : Bs)
                for (int E : Es)
                    for (int K : {1, 2, 8})
                        for (int H : {8, 200, 1032, 4096, 8192})
                            for (int I : {1, 33, 700, 14336, 14368}) {
                                if (K > E) continue;
                                ts_tune_set("bx_vgroup", vg);
                                ts_tune_set("down_chunks", dc);
                                BatchPlan p;
                                if (!plan_batch(B, H, I, E, K, TS_BF16, &p)) return fail("batch plan refused", B, H, I, E);
                                if (plan_batch(B, H, I, E, K, TS_F32, &p)) return fail("batch plan fp32", B, H, I, E);
                                plan_batch(B, H, I, E, K, TS_BF16, &p);
                                const int want = (E > 1 && vg == 0) ? std::min(B, 2 * ((B * K + E - 1) / E)) : B;
                                if (p.tok != 8 && p.tok != 16 && p.tok != 32 && p.tok != 64) return fail("tok", B, H, I, E);
                                if (p.tok < want || (p.tok > 8 && p.tok / 2 >= want)) return fail("tok size", B, H, I, E);
                                if ((long long)p.vpe * p.tok < B || p.groups != E * p.vpe) return fail("groups", B, H, I, E);
                                {
                                    // the kernels' grid order of the groups: a permutation, first groups first
                                    std::vector<char> seen((size_t)p.groups, 0);
                                    for (int gi = 0; gi < p.groups; ++gi) {
                                        const int g = bx_group_at(gi, p.groups, p.vpe);
                                        if (g < 0 || g >= p.groups || seen[(size_t)g]) return fail("group order", B, H, I, E);
                                        seen[(size_t)g] = 1;
                                        if ((gi < E) != (g % p.vpe == 0)) return fail("group order first", B, H, I, E);
                                    }
                                }
                                if (p.hpad < H || p.hpad % kBxKQuant) return fail("hpad", B, H, I, E);
                                if (p.ntiles != (I + kBxRows - 1) / kBxRows) return fail("ntiles", B, H, I, E);
                                if (p.nslices != (H + kBxSliceCols - 1) / kBxSliceCols) return fail("nslices", B, H, I, E);
                                if (p.tpc < 1 || p.tpc > bx_down_tiles(p.tok)) return fail("down chunk", B, H, I, E);
                                if ((long long)p.nchunks * p.tpc < p.ntiles || (long long)(p.nchunks - 1) * p.tpc >= p.ntiles)
                                    return fail("down chunks cover", B, H, I, E);
                                const size_t G = (size_t)p.groups, T = (size_t)p.ntiles;
                                const size_t offs[] = {p.off_gcount, p.off_tslot, p.off_xhl, p.off_cnt, p.off_arow,
                                                       p.off_hfrag, p.off_gmask, p.off_amask, p.off_partial,
                                                       p.off_union, p.total};
                                for (size_t k = 0; k + 1 < sizeof(offs) / sizeof(offs[0]); ++k)
                                    if (offs[k] % 256 || offs[k + 1] < offs[k]) return fail("batch offsets", B, H, I, E);
                                if (p.off_tslot - p.off_gcount < G * 4) return fail("gcount size", B, H, I, E);
                                if (p.off_xhl - p.off_tslot < (size_t)B * K * 8) return fail("tslot size", B, H, I, E);
                                const size_t xfrag = G * 2 * p.tok * p.hpad * 2, xtok = (size_t)B * p.hpad * 4;
                                if (p.off_cnt - p.off_xhl < std::max(xfrag, xtok)) return fail("x region", B, H, I, E);
                                if (p.off_arow - p.off_cnt < G * T * 8) return fail("cnt size", B, H, I, E);
                                if (p.off_hfrag - p.off_arow < G * T * kBxRows) return fail("arow size", B, H, I, E);
                                if (p.off_gmask - p.off_hfrag < G * T * 2 * p.tok * kBxRows * 2) return fail("hfrag size", B, H, I, E);
                                if (p.off_partial - p.off_amask < G * T * p.tok * 4) return fail("amask size", B, H, I, E);
                                if (p.off_union - p.off_partial < G * p.tok * (size_t)p.nchunks * H * 4)
                                    return fail("partial size", B, H, I, E);
                            }
    ts_tune_set("bx_vgroup", 0);
    ts_tune_set("down_chunks", 0);
    BatchPlan q;
    if (plan_batch(65, 4096, 14336, 8, 2, TS_BF16, &q)) return fail("batch above 64", 65, 4096, 14336, 8);
    std::printf("ok\n");
    return 0;
}
