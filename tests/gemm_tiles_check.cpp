// Host-side check of the tiled GEMM's launch geometry and block -> tile map.
//
// Test infrastructure: this program compiles the library's gemm.hip for the
// host only and calls its own functions (plan_for_role, tile_geometry,
// tile_job) for the projections of every workload shape and a set of edge
// shapes, then checks that
//   - tile_corner maps the linear tile indices one to one onto the tiles;
//   - every output tile is produced exactly once: by one block over all of
//     its K tiles, or by `splits` blocks whose K ranges partition them;
//   - the LoRA K tiles of an output group go only to an active group, to the
//     last split, with that group's activation columns;
//   - every partial tile sits where its reduce kernel reads it (uniform split:
//     ws + split M N, row stride N; ragged tail: ws + (split tail_tiles + tail
//     index) BM BN, row stride BN) and inside the workspace, and no two blocks
//     write the same partial tile.
// Prints one line per failure (at most 20) and a summary; exit status 1 on
// any failure.
#include "gemm_plan.h"

#include <cstdio>
#include <map>
#include <set>
#include <utility>
#include <vector>

namespace {

struct Case {
    char name[96];
    int role, M, N, K1, K2, group;
    uint32_t mask;
    int64_t x2_stride;
    size_t ws_bytes;
};

int failures = 0;
long blocks_checked = 0;
std::map<std::string, int> plans;

#define CHECK(cond, ...)                                   \
    do {                                                   \
        if (!(cond)) {                                     \
            if (failures < 20) {                           \
                std::printf("FAIL %s: ", c.name);          \
                std::printf(__VA_ARGS__);                  \
                std::printf("\n");                         \
            }                                              \
            ++failures;                                    \
            return;                                        \
        }                                                  \
    } while (0)

template <int BM, int BN>
void check_plan(const Case& c, const pb::GemmParams& p, const pb::GemmWorkspace& wsp, const pb::TilePlan& tp) {
    using namespace pb;
    const TileGeometry g = tile_geometry<BM, BN>(p, wsp, tp.splits, tp.ragged_tail);
    const SplitArgs& sa = g.sa;
    const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN, tiles = tiles_m * tiles_n;
    const int nk1 = p.K1 / BK;
    const float* ws = (const float*)wsp.ws;
    char key[64];
    std::snprintf(key, sizeof key, "%dx%d split %d%s", BM, BN, sa.splits, sa.full_tiles > 0 ? " ragged" : "");
    ++plans[key];

    // linear tile index <-> corner
    std::map<std::pair<int, int>, int> lin;
    for (int t = 0; t < tiles; ++t) {
        int m0, n0;
        tile_corner<BM, BN>(p, t, m0, n0);
        CHECK(m0 >= 0 && m0 < p.M && m0 % BM == 0 && n0 >= 0 && n0 < p.N && n0 % BN == 0,
              "tile %d at (%d, %d)", t, m0, n0);
        CHECK(lin.emplace(std::make_pair(m0, n0), t).second, "tiles share the corner (%d, %d)", m0, n0);
    }
    CHECK(sa.splits >= 1 && g.grid >= tiles, "grid %d for %d tiles, %d splits", g.grid, tiles, sa.splits);
    if (sa.splits > 1 && sa.full_tiles == 0)
        CHECK((double)sa.splits * p.M * p.N * 4 <= (double)wsp.bytes, "%d partials overflow the workspace", sa.splits);
    if (sa.full_tiles > 0)
        CHECK(sa.full_tiles + sa.tail_tiles == tiles &&
                  (double)sa.splits * sa.tail_tiles * BM * BN * 4 <= (double)wsp.bytes,
              "ragged split: %d whole + %d tail tiles of %d, %d splits", sa.full_tiles, sa.tail_tiles, tiles,
              sa.splits);

    std::vector<int> whole(tiles, 0), parts(tiles, 0);
    std::vector<std::vector<unsigned char>> kc(tiles);
    std::set<std::pair<int, int>> part_seen;
    for (int bid = 0; bid < g.grid; ++bid) {
        const TileJob j = tile_job<BM, BN>(p, sa, bid, g.grid);
        ++blocks_checked;
        const auto it = lin.find(std::make_pair(j.m0, j.n0));
        CHECK(it != lin.end(), "block %d at (%d, %d), not a tile corner", bid, j.m0, j.n0);
        const int t = it->second;
        const int grp = j.n0 / p.group;
        const bool active = p.K2 > 0 && ((p.k2_mask >> grp) & 1u);
        const int nkt = nk1 + (active ? p.K2 / BK : 0);
        CHECK(j.nk1 == nk1, "block %d: %d base K tiles, expected %d", bid, j.nk1, nk1);
        CHECK(j.nk >= 1 && j.t_begin >= 0 && j.t_begin + j.nk <= nkt, "block %d: K range [%d, %d) of %d", bid,
              j.t_begin, j.t_begin + j.nk, nkt);
        if (active)
            CHECK(j.X2 == (const void*)((const char*)p.X2 + (int64_t)grp * p.x2_group_stride * 2),
                  "block %d: LoRA activations of group %d", bid, grp);
        if (j.t_begin + j.nk > nk1)
            CHECK(!j.partial || j.split == sa.splits - 1, "block %d: LoRA K tiles in split %d of %d", bid, j.split,
                  sa.splits);
        if (!j.partial) {
            CHECK(j.t_begin == 0 && j.nk == nkt, "block %d: whole tile with K range [%d, %d) of %d", bid,
                  j.t_begin, j.t_begin + j.nk, nkt);
            CHECK(sa.splits == 1 || (sa.full_tiles > 0 && t < sa.full_tiles), "block %d: tile %d whole in a split launch",
                  bid, t);
            ++whole[t];
            continue;
        }
        CHECK(sa.splits > 1 && j.split >= 0 && j.split < sa.splits, "block %d: split %d of %d", bid, j.split,
              sa.splits);
        CHECK(part_seen.emplace(t, j.split).second, "tile %d split %d written twice", t, j.split);
        if (sa.full_tiles > 0) {
            CHECK(t >= sa.full_tiles, "block %d: whole-round tile %d split", bid, t);
            const int64_t at = ((int64_t)j.split * sa.tail_tiles + (t - sa.full_tiles)) * BM * BN;
            CHECK(j.pbase == ws + at && j.ldp == BN && j.om == j.m0 && j.on == j.n0,
                  "block %d: tail partial at %ld (row stride %d), reduce reads %ld", bid, (long)(j.pbase - ws), j.ldp,
                  (long)at);
        } else {
            const int64_t at = (int64_t)j.split * p.M * p.N;
            CHECK(j.pbase == ws + at && j.ldp == p.N && j.om == 0 && j.on == 0,
                  "block %d: partial at %ld (row stride %d), reduce reads %ld", bid, (long)(j.pbase - ws), j.ldp,
                  (long)at);
        }
        ++parts[t];
        if (kc[t].empty()) kc[t].assign(nkt, 0);
        for (int k = j.t_begin; k < j.t_begin + j.nk; ++k) ++kc[t][k];
    }
    for (int t = 0; t < tiles; ++t) {
        CHECK(whole[t] + (parts[t] > 0) == 1 && whole[t] <= 1, "tile %d: %d whole blocks, %d partial blocks", t,
              whole[t], parts[t]);
        if (parts[t] == 0) continue;
        CHECK(parts[t] == sa.splits, "tile %d: %d partial blocks for %d splits", t, parts[t], sa.splits);
        for (size_t k = 0; k < kc[t].size(); ++k)
            CHECK(kc[t][k] == 1, "tile %d: K tile %zu covered %d times", t, k, kc[t][k]);
    }
}

void run(const Case& c) {
    pb::GemmParams p{};
    p.M = c.M;
    p.N = c.N;
    p.K1 = c.K1;
    p.ldx = p.ldw = c.K1;
    if (c.K2 > 0) {
        p.X2 = (const void*)0x100000;  // only compared, never read
        p.K2 = c.K2;
        p.group = c.group;
        p.k2_mask = c.mask;
        p.x2_group_stride = c.x2_stride;
    } else {
        p.group = c.N;
    }
    static char ln_dummy;
    if (c.role == 1 || c.role == 3) p.ln_out = &ln_dummy;  // the planner prices the LayerNorm that follows
    const pb::GemmWorkspace wsp{(void*)0x40000000, c.ws_bytes};
    const pb::TilePlan tp = pb::plan_for_role(c.role, p, wsp);
    if (tp.tile == 256) check_plan<256, 256>(c, p, wsp, tp);
    else if (tp.tile == 128) check_plan<128, 128>(c, p, wsp, tp);
    else check_plan<64, 64>(c, p, wsp, tp);
}

}  // namespace

int main() {
    struct Model { const char* name; int d, F, tokens; };
    // the workloads' shapes (tokens = batch x prompt) and the tiny test model
    const Model models[] = {{"tiny", 256, 1024, 32},       {"opt-1.3b", 2048, 8192, 512},
                            {"opt-6.7b", 4096, 16384, 4096}, {"opt-13b", 5120, 20480, 2048},
                            {"opt-66b", 9216, 36864, 4096}};
    // other prompt lengths, ragged ones included (at most 8 rows go to the GEMV)
    const int extra_tokens[] = {9, 100, 513, 1000, 1100, 2000};
    long cases = 0;
    for (const Model& mo : models) {
        std::vector<int> toks{mo.tokens};
        for (int t : extra_tokens) toks.push_back(t);
        for (int M : toks) {
            // workspace as the model sizes it: 4 fp32 [tokens, d] partials, 64 MiB .. 1 GiB
            const size_t want = (size_t)4 * M * mo.d * 4;
            const size_t ws = std::min<size_t>(std::max<size_t>(want, 64u << 20), 1u << 30);
            for (int kw : {0, 64, 128}) {
                const int d = mo.d;
                std::vector<Case> cs;
                auto add = [&](const char* what, int role, int N, int K1, int K2, int group, uint32_t mask,
                               int64_t xs) {
                    Case c{};
                    std::snprintf(c.name, sizeof c.name, "%s M=%d kw=%d %s", mo.name, M, kw, what);
                    c.role = role; c.M = M; c.N = N; c.K1 = K1; c.K2 = K2; c.group = group; c.mask = mask;
                    c.x2_stride = xs; c.ws_bytes = ws;
                    cs.push_back(c);
                };
                if (kw == 0) {
                    add("qkv", 0, 3 * d, d, 0, 0, 0, 0);
                    add("o", 1, d, d, 0, 0, 0, 0);
                    add("fc1", 2, mo.F, d, 0, 0, 0, 0);
                    add("fc2", 3, d, mo.F, 0, 0, 0, 0);
                } else {
                    add("qkv, LoRA q,v", 0, 3 * d, d, kw, d, 5u, kw);
                    add("qkv, LoRA q,k,v", 0, 3 * d, d, kw, d, 7u, kw);
                    add("qkv, LoRA k", 0, 3 * d, d, kw, d, 2u, kw);
                    add("q only (cached keys and values), LoRA q", 0, d, d, kw, d, 1u, kw);
                    add("o, LoRA o", 1, d, d, kw, d, 1u, 0);
                    add("shrink q,k,v", 4, 3 * kw, d, 0, 0, 0, 0);
                    add("shrink o", 4, kw, d, 0, 0, 0, 0);
                }
                for (const Case& c : cs) {
                    run(c);
                    ++cases;
                }
            }
        }
    }
    std::printf("%ld cases, %ld blocks checked, %d failures; plans:", cases, blocks_checked, failures);
    for (const auto& kv : plans) std::printf(" [%s] %d", kv.first.c_str(), kv.second);
    std::printf("\n");
    return failures ? 1 : 0;
}
