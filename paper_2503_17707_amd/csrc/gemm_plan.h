// Launch planning of the tiled GEMM (host) and the block -> tile map shared by
// the kernels and the host (host and device): which tile shape and K split a
// launch uses, its grid and split arguments, and which output tile and K range
// each block computes.  Kept apart from the kernels so that a host-only build
// (the CPU test of this map) can use the very same functions.
#pragma once

#include <algorithm>

#include "kernels.h"

namespace pb {

namespace {

#ifndef PB_GEMM_SPLIT_TARGET
#define PB_GEMM_SPLIT_TARGET 256  // blocks a split launch aims for
#endif
#ifndef PB_GEMM_MIN_KT
#define PB_GEMM_MIN_KT 8  // fewest K tiles a split-K block gets
#endif
#ifndef PB_GEMM_RAGGED
#define PB_GEMM_RAGGED 1  // split only the tail tiles of a ragged last round
#endif

constexpr int BK = 64;      // K tile
constexpr int GROUP_M = 8;  // tile-rows per group of the tile walk

struct SplitArgs {
    int splits;     // number of K splits (1 = none)
    int kt_split;   // K tiles per split (the LoRA tiles go to the last split)
    float* ws;      // [splits][M][N] fp32 partials when splits > 1
    // ragged-round split (full_tiles > 0): tiles [0, full_tiles) run whole
    // through the epilogue, only the tail tiles [full_tiles, full_tiles +
    // tail_tiles) are split `splits` ways, their partials packed as
    // [split][tail tile][BM][BN]; full_tiles and tail_tiles * splits are
    // multiples of 8
    int full_tiles, tail_tiles;
};

// Which output tile and K range a block works on: the hardware deals
// consecutive blocks round-robin to the 8 XCDs, so the block id is remapped to
// give each XCD a contiguous run; runs are split-major, and tiles are walked in
// groups of GROUP_M tile-rows so that blocks sharing an XCD's L2 share rows of
// X and of W.  Split s takes base K tiles [s kt, (s+1) kt), the last split
// also the LoRA K tiles of its output group (if that group is active).
struct TileJob {
    int m0, n0, split, nk1, t_begin, nk;
    bool partial;    // writes an fp32 partial tile (split along K) instead of the epilogue
    float* pbase;    // ... at pbase + (m - om) * ldp + (n - on)
    int ldp, om, on;
    const void* X2;  // LoRA activations of the tile's output group
};

// Output tile index -> its corner: tiles are walked in groups of GROUP_M
// tile-rows (blocks that share an XCD's L2 share rows of X and of W).
template <int BM, int BN>
__host__ __device__ __forceinline__ void tile_corner(const GemmParams& p, int tile, int& m0, int& n0) {
    const int tiles_m = (p.M + BM - 1) / BM;
    const int tiles_n = (p.N + BN - 1) / BN;
    const int per_group = GROUP_M * tiles_n;
    const int first_m = (tile / per_group) * GROUP_M;
    const int gsize = tiles_m - first_m < GROUP_M ? tiles_m - first_m : GROUP_M;
    m0 = (first_m + (tile % per_group) % gsize) * BM;
    n0 = ((tile % per_group) / gsize) * BN;
}

// (host-callable: block bid of a grid of nblk blocks)
template <int BM, int BN>
__host__ __device__ __forceinline__ TileJob tile_job(const GemmParams& p, const SplitArgs& sa, int bid, int nblk) {
    const int tiles_m = (p.M + BM - 1) / BM;
    const int tiles_n = (p.N + BN - 1) / BN;
    const int tiles = tiles_m * tiles_n;
    int tile, split;
    bool partial;
    if (sa.full_tiles > 0) {
        // the whole tiles first, then the split tail tiles, each part dealt
        // XCD-contiguously on its own so that the tail round spreads over all
        // eight XCDs
        if (bid < sa.full_tiles) {
            tile = (sa.full_tiles & 7) ? bid : (bid & 7) * (sa.full_tiles >> 3) + (bid >> 3);
            split = 0;
            partial = false;
        } else {
            const int r = bid - sa.full_tiles, nt = nblk - sa.full_tiles;
            const int rr = (nt & 7) ? r : (r & 7) * (nt >> 3) + (r >> 3);
            tile = sa.full_tiles + rr % sa.tail_tiles;
            split = rr / sa.tail_tiles;
            partial = true;
        }
    } else {
        if ((nblk & 7) == 0) bid = (bid & 7) * (nblk >> 3) + (bid >> 3);
        tile = bid % tiles;
        split = bid / tiles;
        partial = sa.splits > 1;
    }
    TileJob j;
    tile_corner<BM, BN>(p, tile, j.m0, j.n0);
    j.split = split;
    j.partial = partial;
    if (sa.full_tiles > 0) {
        j.pbase = sa.ws + ((int64_t)split * sa.tail_tiles + (tile - sa.full_tiles)) * (BM * BN);
        j.ldp = BN;
        j.om = j.m0;
        j.on = j.n0;
    } else {
        j.pbase = sa.ws + (int64_t)split * p.M * p.N;
        j.ldp = p.N;
        j.om = j.on = 0;
    }
    j.nk1 = p.K1 / BK;
    int nk2 = 0;
    j.X2 = p.X2;
    if (p.K2 > 0) {
        const int g = j.n0 / p.group;
        if ((p.k2_mask >> g) & 1u) {
            nk2 = p.K2 / BK;
            j.X2 = (const char*)p.X2 + (int64_t)g * p.x2_group_stride * 2;
        }
    }
    if (!partial) {
        j.t_begin = 0;
        j.nk = j.nk1 + nk2;
    } else {
        j.t_begin = split * sa.kt_split;
        const int t_end = (split == sa.splits - 1) ? j.nk1 + nk2
                          : (j.nk1 < j.t_begin + sa.kt_split ? j.nk1 : j.t_begin + sa.kt_split);
        j.nk = t_end - j.t_begin;
    }
    return j;
}

// K split into `splits` ranges: splits 0..S-2 take kt_split base tiles each,
// the last one the rest (and the LoRA tiles); S = ceil(nk1 / kt_split) leaves
// no split empty.
SplitArgs make_split(const GemmParams& p, const GemmWorkspace& wsp, int splits) {
    const int nk1 = p.K1 / BK;
    SplitArgs sa;
    sa.kt_split = (nk1 + splits - 1) / splits;
    sa.splits = (nk1 + sa.kt_split - 1) / sa.kt_split;
    sa.ws = (float*)wsp.ws;
    sa.full_tiles = sa.tail_tiles = 0;
    return sa;
}

// Grid and split arguments of a tile launch (host side): a uniform K split
// into `splits` ranges, or with ragged_tail > 0 the whole tiles first and the
// last `ragged_tail` tiles split (falling back to whole tiles only when the
// split does not come out as planned).
struct TileGeometry {
    SplitArgs sa;
    int grid;
};

template <int BM, int BN>
TileGeometry tile_geometry(const GemmParams& p, const GemmWorkspace& wsp, int splits, int ragged_tail) {
    const int tiles = ((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN);
    TileGeometry g;
    g.sa = make_split(p, wsp, splits);
    if (ragged_tail > 0) {
        if (g.sa.splits >= 2 && (tiles - ragged_tail) % 8 == 0 && (ragged_tail * g.sa.splits) % 8 == 0) {
            g.sa.full_tiles = tiles - ragged_tail;
            g.sa.tail_tiles = ragged_tail;
            g.grid = g.sa.full_tiles + ragged_tail * g.sa.splits;
            return g;
        }
        g.sa = make_split(p, wsp, 1);
    }
    g.grid = tiles * g.sa.splits;
    return g;
}

// Tile shape and K split of a launch, from a cost model: a block's time is
// its MFMA work at the rate one CU reaches with that tile (measured: 256 x 256
// ~4.5 TFLOP/s, 128 x 128 ~2.6), blocks run in rounds of 256 (one per CU), and
// a split adds its fp32 partials (written, then read by the reduce) at
// ~4 TB/s.  Splits keep >= PB_GEMM_MIN_KT K tiles each and fit the workspace.
struct TilePlan {
    int tile;    // 256, 128 or 64
    int splits;
    int ragged_tail;  // > 0: whole tiles, then this many tail tiles split `splits` ways
};

TilePlan plan_tiles(const GemmParams& p, const GemmWorkspace& wsp) {
    const int nk1 = p.K1 / BK;
    const double out_bytes = (double)p.M * p.N * 4;
    // the LayerNorm that follows o or fc2 rides on a uniform split's reduce;
    // otherwise it is a pass of its own over the fp32 rows (read) and dt rows (write)
    const double ln_pass = p.ln_out ? (double)p.M * p.N * 6 / 4e12 : 0.0;
    TilePlan best{64, 1, 0};
    double best_t = 1e30;
    auto consider = [&](int t, double rate) {
        if (p.N % t) return;
        const long tiles = (long)((p.M + t - 1) / t) * (p.N / t);
        const double t_tile = 2.0 * t * t * p.K1 / rate;
        for (int s = 1; s <= 8; ++s) {
            if (s > 1 && (nk1 / s < PB_GEMM_MIN_KT || !wsp.ws || out_bytes * s > (double)wsp.bytes)) break;
            const long rounds = (tiles * s + 255) / 256;
            const double tt = rounds * (t_tile / s) + (s > 1 ? 2.0 * out_bytes * s / 4e12 : ln_pass);
            if (tt < best_t * 0.98) {  // prefer the simpler plan on near ties
                best_t = tt;
                best = {t, s, 0};
            }
        }
        // ragged last round: whole rounds unsplit, the tail tiles split to fill one round
        const long tail = tiles % 256, full = tiles - tail;
        if (PB_GEMM_RAGGED && full > 0 && tail > 0 && wsp.ws) {
            const int s = (int)std::min<long>(8, 256 / tail);
            const double pbytes = (double)tail * t * t * 4 * s;
            if (s >= 2 && nk1 / s >= PB_GEMM_MIN_KT && full % 8 == 0 && (tail * s) % 8 == 0 &&
                pbytes <= (double)wsp.bytes) {
                const double tt = (full / 256) * t_tile + t_tile / s + 2.0 * pbytes / 4e12 + ln_pass;
                if (tt < best_t * 0.98) {
                    best_t = tt;
                    best = {t, s, (int)tail};
                }
            }
        }
    };
    consider(256, 4.5e12);
    consider(128, 2.6e12);
    if (best_t >= 1e30) {  // N not a multiple of 128: 64 x 64 tiles, split when few
        const long tiles = (long)((p.M + 63) / 64) * (p.N / 64);
        int s = 1;
        if (tiles < 256 && wsp.ws) {
            s = std::min<long>((PB_GEMM_SPLIT_TARGET + tiles - 1) / tiles, std::max(1, nk1 / PB_GEMM_MIN_KT));
            while (s > 1 && out_bytes * s > (double)wsp.bytes) --s;
        }
        best = {64, std::max(1, s), 0};
    }
    return best;
}

// Tile plan of a launch by role: the projections by the cost model above,
// the LoRA shrink (role 4) always 64 x 64, split along K when few.
TilePlan plan_for_role(int role, const GemmParams& p, const GemmWorkspace& wsp) {
    if (role != 4) return plan_tiles(p, wsp);
    const long tiles = (long)((p.M + 63) / 64) * (p.N / 64);
    int sp = 1;
    if (tiles < 256 && wsp.ws) {
        sp = std::min<long>((PB_GEMM_SPLIT_TARGET + tiles - 1) / tiles, std::max(1, p.K1 / BK / PB_GEMM_MIN_KT));
        while (sp > 1 && (double)p.M * p.N * 4 * sp > (double)wsp.bytes) --sp;
    }
    return {64, std::max(1, sp), 0};
}

}  // namespace

}  // namespace pb
