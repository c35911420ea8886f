// causal.hpp -- workgroup numbering over the causal recursion (Alg. 5
// unrolled): level l has 2^l segments whose future halves hold
// half_l = N >> (l + 1) sorted queries (and whose past halves hold as many
// sorted keys); the leaves are the N / n_leaf runs of n_leaf tokens.
// Segment and leaf lengths need not be multiples of the 64-row tile: each
// segment (leaf) gets ceil(length / 64) tiles, the last one ragged, so a
// tile never straddles two segments (leaves).
#pragma once
#include <hip/hip_runtime.h>

namespace elsaa {

constexpr int kMaxLevels = 26;
constexpr int kRowTile = 64;

struct LevelTiles {
    int first[kMaxLevels + 1];   // first tile of level l; first[Lv] = tiles of all levels
    int per_leaf;                // tiles per leaf
    int leaves;                  // N / n_leaf
    int leaf_tiles() const { return per_leaf * leaves; }
};

inline LevelTiles level_tiles(int N, int Lv, int n_leaf)
{
    LevelTiles t = {};
    int acc = 0;
    for (int l = 0; l < Lv; ++l) {
        t.first[l] = acc;
        const int half = N >> (l + 1);
        acc += (1 << l) * ((half + kRowTile - 1) / kRowTile);
    }
    t.first[Lv] = acc;
    t.per_leaf = (n_leaf + kRowTile - 1) / kRowTile;
    t.leaves = N / n_leaf;
    return t;
}

// tile -> (level, half length, segment, first sorted position of the tile)
__device__ __forceinline__ void level_tile(const LevelTiles& lt, int Lv, int N, int tile, int& level,
                                           int& half, int& seg, int& p0)
{
    level = 0;
    while (level + 1 < Lv && tile >= lt.first[level + 1]) ++level;
    const int t = tile - lt.first[level];
    half = N >> (level + 1);
    const int tps = (half + kRowTile - 1) / kRowTile;
    seg = t / tps;
    p0 = (t - seg * tps) * kRowTile;
}

// tile -> (first token of its leaf, first token of the tile, end of the leaf)
__device__ __forceinline__ void leaf_tile(const LevelTiles& lt, int n_leaf, int tile, int& lbeg, int& t0,
                                          int& lend)
{
    const int leaf = tile / lt.per_leaf;
    lbeg = leaf * n_leaf;
    t0 = lbeg + (tile - leaf * lt.per_leaf) * kRowTile;
    lend = lbeg + n_leaf;
}

// This workgroup's (tile, h, b) in a grid of (tiles, H, B), renumbered so
// that consecutive tiles run on the same XCD: the chip deals workgroups to
// its 8 XCDs round-robin by linear id, and each XCD has its own L2, so
// neighbouring tiles that read the same rows (the tiles of one causal leaf,
// the query tiles of one sorted block) share them through one L2.  Linear
// ids 8 q + x (q < total / 8) become tile x * (total / 8) + q; a remainder
// of fewer than 8 keeps its own numbering.
__device__ __forceinline__ void xcd_tile(int& tile, int& h, int& b)
{
    const int nx = gridDim.x, ny = gridDim.y;
    const int total = nx * ny * gridDim.z;
    const int lin = blockIdx.x + nx * (blockIdx.y + ny * blockIdx.z);
    const int per = total >> 3;
    const int t = lin < 8 * per ? (lin & 7) * per + (lin >> 3) : lin;
    tile = t % nx;
    const int rest = t / nx;
    h = rest % ny;
    b = rest / ny;
}

}  // namespace elsaa
