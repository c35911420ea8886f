// causal.hpp -- geometry of the causal recursion (Alg. 5 unrolled) and the
// workgroup numbering over it.
//
// A segment of the recursion is a list of L_l entries at depth l: a range
// of real tokens [a, a + r) followed by L_l - r zero tokens.  A segment
// longer than n0 is split (Alg. 5): an odd list is padded with one zero
// token, then its first m = ceil(L_l / 2) entries form the past half and the
// other m the future half, so L_{l+1} = m for every segment of the next
// depth, and
//   past child   = real [a, a + m), no zero tokens;
//   future child = real [a + m, a + r), the rest zero tokens.
// Zero tokens therefore only ever trail a future half, and the depth Lv is
// the same for every segment (the smallest with L_Lv <= n0).  Level l's
// SortLSH calls are the 2^l (future half, past half) pairs of depth-l
// segments; its sorted lists take m_l = L_{l+1} entries each, stored segment
// after segment, level after level (per (b,h): off[l] .. off[l] + 2^l m_l);
// a zero token's entry in a query list is -1.  Without any padding
// (N = n0' 2^Lv) this is L_l = N >> l and off[l] = l N / 2.
//
// Tiles: level l has 2^l segments x ceil(m_l / 64) tiles, each leaf
// ceil(L_Lv / 64) tiles; a tile never straddles two segments (leaves), and
// the last tile of each is ragged (masked).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace elsaa {

constexpr int kMaxLevels = 26;
constexpr int kRowTile = 64;

struct LevelTiles {
    int Lv;                      // levels (0 non-causal or a single leaf)
    int len[kMaxLevels + 1];     // list length L_l of a depth-l segment (len[0] = N)
    int64_t off[kMaxLevels + 1]; // first entry of level l's lists within one (b,h); off[Lv] = all levels
    int first[kMaxLevels + 1];   // first tile of level l; first[Lv] = tiles of all levels
    int per_leaf;                // tiles per leaf
    int leaves;                  // 2^Lv
    int padded;                  // some segment carries zero tokens
    int leaf_tiles() const { return per_leaf * leaves; }
};

// Geometry of the recursion for N tokens and base length n0; returns false
// when some past half would have to hold a zero token (its real tokens fewer
// than half the list), which the kernels do not implement, or when the depth
// exceeds kMaxLevels.
inline bool level_tiles(int N, int n0, LevelTiles& t)
{
    t = LevelTiles{};
    int L = N, lv = 0, pads = 0;                 // pads: the most zero tokens of any depth-lv segment
    t.len[0] = N;
    int64_t off = 0;
    int acc = 0;
    while (L > n0) {
        if (lv >= kMaxLevels) return false;
        const int m = (L + 1) / 2;
        if (pads > L - m) return false;          // the past half would reach a zero token
        t.off[lv] = off;
        t.first[lv] = acc;
        off += (int64_t)m << lv;
        acc += (1 << lv) * ((m + kRowTile - 1) / kRowTile);
        pads += L & 1;                           // the all-future path collects every pad
        L = m;
        ++lv;
        t.len[lv] = L;
        if (pads) t.padded = 1;
    }
    t.Lv = lv;
    t.off[lv] = off;
    t.first[lv] = acc;
    t.per_leaf = (L + kRowTile - 1) / kRowTile;
    t.leaves = 1 << lv;
    return true;
}

// Real token range [a, a + r) of segment s at depth l.
__device__ __forceinline__ void seg_range(const LevelTiles& lt, int l, int s, int& a, int& r)
{
    a = 0;
    r = lt.len[0];
    for (int j = 0; j < l; ++j) {
        const int m = lt.len[j + 1];
        if ((s >> (l - 1 - j)) & 1) {
            a += m;
            r = r > m ? r - m : 0;
        } else {
            r = m;
        }
    }
}

// Entry of token t in the level-l lists of one (b,h): the entry of the same
// rank within its segment's future half (future = true) or past half.
__device__ __forceinline__ int64_t level_entry(const LevelTiles& lt, int l, int t, bool future)
{
    int a = 0, s = 0;
    for (int j = 0; j < l; ++j) {
        const int m = lt.len[j + 1];
        const int f = t >= a + m;
        s = 2 * s + f;
        if (f) a += m;
    }
    const int m = lt.len[l + 1];
    return lt.off[l] + (int64_t)s * m + (t - a - (future ? m : 0));
}

// Per-level rows (the causal levels' partial results, one row per list
// entry) of segment seg at level l: token t of that segment has its row at
// base + t, i.e. the entry of the same rank within the segment's future half
// (future = true) or past half, after the (b,h)s before it.  Every token of a
// sorted block, a level tile or a leaf lies in one segment per level, so
// callers form the base once from uniform values (scalar work) and add the
// token.
__device__ __forceinline__ int64_t seg_slot_base(const LevelTiles& lt, size_t bh, int l, int seg, bool future)
{
    int a, r;
    seg_range(lt, l, seg, a, r);
    const int m = lt.len[l + 1];
    return (int64_t)(bh * (size_t)lt.off[lt.Lv] + (size_t)lt.off[l]) + (int64_t)seg * m - a - (future ? m : 0);
}

// Levels whose partials leaf s adds: bit l set when the leaf lies in the
// future half (future = true) or in the past half of its level-l segment.
__device__ __forceinline__ unsigned leaf_levels(const LevelTiles& lt, int leaf, bool future)
{
    unsigned mask = 0;
    for (int l = 0; l < lt.Lv; ++l)
        if ((((leaf >> (lt.Lv - 1 - l)) & 1) != 0) == future) mask |= 1u << l;
    return mask;
}

// tile -> (level, half length m_l, segment, first list position of the tile)
__device__ __forceinline__ void level_tile(const LevelTiles& lt, int tile, int& level, int& half, int& seg, int& p0)
{
    level = 0;
    while (level + 1 < lt.Lv && tile >= lt.first[level + 1]) ++level;
    const int t = tile - lt.first[level];
    half = lt.len[level + 1];
    const int tps = (half + kRowTile - 1) / kRowTile;
    seg = t / tps;
    p0 = (t - seg * tps) * kRowTile;
}

// tile -> (leaf, first token of its leaf, first token of the tile, end of
// the leaf's real tokens); tiles past the real tokens have t0 >= lend.
__device__ __forceinline__ void leaf_tile(const LevelTiles& lt, int tile, int& leaf, int& lbeg, int& t0, int& lend)
{
    leaf = tile / lt.per_leaf;
    int r;
    seg_range(lt, lt.Lv, leaf, lbeg, r);
    t0 = lbeg + (tile - leaf * lt.per_leaf) * kRowTile;
    lend = lbeg + r;
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
