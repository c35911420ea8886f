// sparse_bwd.hip -- backward of the sortLSH sparse branch.
//
// With the selection fixed, the sparse branch is exact softmax attention
// restricted to each query's support S(i), normalised by d_s + eps.  Its
// gradient (no formula in the paper; the exact derivative of the forward):
//   P_ij  = exp(z_ij - log(d_s,i + eps)),  z_ij = tau <Q_i, K_j>
//   dO_s  = g_s m dO            (row scale sc_s = g_s m)
//   dz_ij = P_ij (<dO_s,i, V_j> - Delta_i)
//   dQ_i += tau sum_j dz_ij K_j;  dK_j += tau sum_i dz_ij Q_i;  dV_j += sum_i P_ij dO_s,i
// where Delta_i = <dO_s,i, O_s,i> - dm_i m_i (1 - m_i)(d_s,i + eps)/d_s,i also
// carries the gradient through the denominator-aware multiplier m.
//
// Two passes, no atomics: a query-centric pass (dQ; one workgroup per 64
// queries, keys streamed through LDS) and a key-centric pass (dK, dV; one
// workgroup per 64 keys, queries streamed through LDS).  Both have the three
// modes of the forward (non-causal blocks, causal levels, causal leaf).  The
// level passes write per-level partials by natural token index in the
// storage dtype (each level's contribution rounded once; the sum over levels
// is float32); the leaf passes add the partials of every level and the
// low-rank gradient and store the final dQ, dK, dV in the storage dtype.
#include "common.hpp"
#include "internal.hpp"
#include "causal.hpp"
#include "tile.hpp"

namespace elsaa {

namespace {

constexpr int kT = 64;
constexpr int kThreads = 256;
static_assert(kT == kRowTile, "causal tiles are numbered in 64-row tiles");

enum Mode { kBlocks = 0, kLevels = 1, kLeaf = 2 };

struct BArgs {
    const void* Q;
    const void* K;
    const void* V;
    const void* dO;
    const int32_t* perm_q;
    const int32_t* perm_k;
    const float* rs;          // row scalars, see internal.hpp
    const void* du_q;         // low-rank gradients of the Q / K projections, storage dtype [BHN][wk]
    const void* du_k;
    const void* wt_hi;        // W' = W_hi' + W_lo' per head, storage dtype [H][D][wk]
    const void* wt_lo;
    const void* dv_lr;        // storage dtype [BHN][D] low-rank dV
    void* part_dq;            // [BH][Lv][N/2][D] per-level partials, storage dtype
    void* part_dk;
    void* part_dv;
    void* dQ;
    void* dK;
    void* dV;
    int H, N, k, Lv, wk;
    LevelTiles lt;            // causal recursion geometry and tile numbering
    int nbr;                  // neighbouring sorted blocks on each side
    int nbx, nblk;            // whole-block kernel: blocks per head, blocks in all
    size_t BHN;
    float tau, tau2;
};


// The low-rank part of dQ (dK) of one token for the 16-row slice dt of d:
// (du W')^T, rows d = 16 dt + 4 g + i, the token in the lane's column (du_row
// = its du row, wth / wtl = the head's W' parts).  The same matrix-core
// products, in the same order, as the low-rank pass would use to form it.
template <class T>
__device__ __forceinline__ f32x4 lowrank_tile(const typename T::store_t* du_row, const typename T::store_t* wth,
                                              const typename T::store_t* wtl, int wk, int g, int col, int dt)
{
    f32x4 acc = {0, 0, 0, 0};
    for (int kp = 0; kp < wk; kp += 32) {
        const typename T::frag_t df = T::ld8(du_row + kp + 8 * g);
        const size_t o = (size_t)(16 * dt + col) * wk + kp + 8 * g;
        acc = T::mma(T::ld8(wth + o), df, acc);
        if (T::kSplit) acc = T::mma(T::ld8(wtl + o), df, acc);
    }
    return acc;
}

// W' = W_hi' + W_lo' of one head staged in LDS for the low-rank parts of the
// epilogues: each part [D][wk + 8] (the pad spreads a slice's 16 rows over
// the banks).  Loaded into registers with the first tile's rows and written
// to LDS before that tile's barrier, so the epilogue reads it without a
// global round trip and every wave of the workgroup shares one copy.
template <class T, int D>
struct WtStage {
    using S = typename T::store_t;
    static constexpr int kMaxWk = 64;
    static constexpr int EPC = 16 / T::bytes;                  // elements per 16-byte piece
    static constexpr int PARTS = T::kSplit ? 2 : 1;
    __host__ __device__ static constexpr size_t bytes(int wk) { return (size_t)PARTS * D * (wk + 8) * T::bytes; }
    // global -> LDS directly (gfx950 global_load_lds_dwordx4: one wave
    // instruction writes 64 consecutive 16-byte pieces of LDS, piece l from
    // lane l; no registers hold the data).  The LDS bytes are cut into
    // 16-byte pieces q = ((part * D + row) * CR + c); the pad piece of a row
    // fetches the row's first piece again and is never read.  Issued before
    // any other load of the workgroup, so the wait for the first tile's rows
    // (the memory counter retires loads in order) also covers it.
    __device__ __forceinline__ static void issue(const S* wth, const S* wtl, int wk, S* lds)
    {
        typedef __attribute__((address_space(3))) void lds_void_t;
        const int CR = (wk + 8) * T::bytes / 16, CD = wk * T::bytes / 16;
        const int pieces = PARTS * D * CR, per_part = D * CR;
        const int w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6), lane = threadIdx.x & 63;
        for (int j = w; 64 * j < pieces; j += kThreads / 64) {
            const int q = 64 * j + lane;
            if (q < pieces) {
                const int part = q >= per_part, rem = q - part * per_part;
                const int row = rem / CR, c = rem - row * CR;
                const S* src = (part ? wtl : wth) + (size_t)row * wk + (c < CD ? c : 0) * EPC;
                __builtin_amdgcn_global_load_lds(src, (lds_void_t*)(lds + (size_t)64 * j * EPC), 16, 0, 0);
            }
        }
    }
};

// lowrank_tile with W' from the LDS copy (wt = WtStage layout) and the
// token's du fragments already in registers (du_f[j]: elements 32 j + 8 g ..).
template <class T, int D>
__device__ __forceinline__ f32x4 lowrank_lds(const typename T::frag_t (&du_f)[2], const typename T::store_t* wt,
                                             int wk, int g, int col, int dt)
{
    const int wkp = wk + 8;
    f32x4 acc = {0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 2; ++j)
        if (32 * j < wk) {
            const typename T::store_t* p = wt + (16 * dt + col) * wkp + 32 * j + 8 * g;
            acc = T::mma(T::ld8(p), du_f[j], acc);
            if (T::kSplit) acc = T::mma(T::ld8(p + D * wkp), du_f[j], acc);
        }
    return acc;
}

// du fragments of one token row (wk <= 64 values, zero k-steps past wk).
template <class T>
__device__ __forceinline__ void du_frags(const typename T::store_t* du_row, int wk, int g,
                                         typename T::frag_t (&f)[2])
{
#pragma unroll
    for (int j = 0; j < 2; ++j)
        if (32 * j < wk) f[j] = T::ld8(du_row + 32 * j + 8 * g);
}

// ------------------------------------------------------------------------
// dQ: query-centric.  One workgroup per 64 queries (16 per wave, one per
// lane column); key tiles of 64 rows stream through LDS (tile.hpp) with the
// next tile's rows loaded into registers meanwhile.  Per tile: S^T = K Q^T
// and dP^T = V dO^T (key rows from LDS, this lane's query in registers),
// dS^T in registers, dQ^T += K^T dS^T with K^T from the transposed LDS read.
// ------------------------------------------------------------------------
// LDS bytes of the query-centric pass (K and V tiles, W' for the epilogue).
template <class T, int D, int MODE>
__host__ __device__ constexpr size_t dq_lds_bytes(int wk)
{
    return 2 * (size_t)tile::Tile<T, D, kThreads>::elems(kT) * T::bytes +
           (MODE == kLevels ? 0 : WtStage<T, D>::bytes(wk));
}

template <class T, int D, int MODE>
__device__ __forceinline__ void sparse_dq_body(const BArgs& a, int tile, int h, int b, char* smem)
{
    using S = typename T::store_t;
    using F = typename T::frag_t;
    constexpr int KS = D / 32, DT = D / 16;
    using TD = tile::Tile<T, D, kThreads>;
    constexpr int PT = TD::PER_THREAD;
    S* const sk = (S*)smem;
    S* const sv = sk + TD::elems(kT);
    S* const swt = sv + TD::elems(kT);          // W' (leaf, blocks)
    const size_t bh = (size_t)b * a.H + h;
    const int N = a.N;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int g = lane >> 4, qq = lane & 15;
    const S* Q = (const S*)a.Q + bh * N * D;
    const S* K = (const S*)a.K + bh * N * D;
    const S* V = (const S*)a.V + bh * N * D;
    const S* dO = (const S*)a.dO + bh * N * D;

    int level = 0, half = N, qpos, qtok, kbeg, kend, bq = 1;
    int qrow0 = 0, nq = 0;                       // blocks, leaf: first query position of the tile, its queries
    int64_t slot0 = 0;                           // levels: partial row of token t at slot0 + t
    const int32_t* klist = nullptr;
    if (MODE == kBlocks) {
        bq = min(a.k, N);
        const int p0 = tile * kT;
        qrow0 = p0;
        nq = min(kT, N - p0);
        qpos = p0 + 16 * w + qq;
        qtok = qpos < N ? a.perm_q[bh * N + qpos] : -1;
        const int plast = min(p0 + kT, N) - 1;
        kbeg = max(0, (p0 / bq - a.nbr) * bq);
        kend = min(N, (plast / bq + 1 + a.nbr) * bq);
        klist = a.perm_k + bh * N;
    } else if (MODE == kLevels) {
        int seg, p0;
        level_tile(a.lt, tile, level, half, seg, p0);
        bq = min(a.k, half);
        qpos = p0 + 16 * w + qq;
        const size_t lbase = bh * (size_t)a.lt.off[a.Lv] + (size_t)a.lt.off[level] + (size_t)seg * half;
        qtok = qpos < half ? a.perm_q[lbase + qpos] : -1;      // -1 also for a zero token
        slot0 = seg_slot_base(a.lt, bh, level, seg, true);
        kbeg = max(0, (p0 / bq - a.nbr) * bq);
        kend = min(half, ((min(p0 + kT, half) - 1) / bq + 1 + a.nbr) * bq);
        klist = a.perm_k + lbase;
    } else {
        int q0, lend, leaf;
        leaf_tile(a.lt, tile, leaf, kbeg, q0, lend);
        qtok = q0 + 16 * w + qq;
        qpos = qtok;
        if (qtok >= lend) qtok = -1;
        kend = q0 < lend ? min(q0 + kT, lend) : kbeg;    // a tile past the leaf's real tokens has no work
        qrow0 = q0;
        nq = max(0, min(kT, lend - q0));
    }
    const int blk_lo = (MODE == kLeaf) ? 0 : max(0, (qpos / bq - a.nbr) * bq);
    const int blk_hi = (MODE == kLeaf) ? 0 : min((MODE == kBlocks ? N : half), (qpos / bq + 1 + a.nbr) * bq);

    // key rows of the tile at k0 that this thread stages: positions past the
    // scanned range repeat its last key (a real row: key lists hold no zero
    // tokens), whose scores the mask drops, so the loads need no per-row
    // branch
    auto tokens = [&](int k0, int (&tok)[PT]) {
#pragma unroll
        for (int j = 0; j < PT; ++j) {
            const int p = min(k0 + TD::row_of(j), kend - 1);
            tok[j] = (MODE == kLeaf) ? p : klist[p];
        }
    };
    const int ntiles = (kend - kbeg + kT - 1) / kT;
    int tok[PT];
    uint4 rk[PT], rv[PT];
    if (MODE != kLevels) {
        const size_t wh = (bh % a.H) * D * a.wk;
        WtStage<T, D>::issue((const S*)a.wt_hi + wh, (const S*)a.wt_lo + wh, a.wk, swt);
    }
    if (ntiles > 0) {
        tokens(kbeg, tok);
        TD::load_all(K, tok, rk);
        TD::load_all(V, tok, rv);
    }
    if (ntiles > 1) tokens(kbeg + kT, tok);

    float lse2 = 0.f, delta = 0.f, scs = 0.f;
    F qf[KS], df[KS];
    {
        float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        const F zf = T::pack(z);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) { qf[ks] = zf; df[ks] = zf; }
    }
    if (qtok >= 0) {
        const size_t row = bh * N + qtok;
        lse2 = a.rs[row];
        delta = a.rs[a.BHN + row];
        scs = a.rs[2 * a.BHN + row];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            qf[ks] = T::ld8(Q + (size_t)qtok * D + 32 * ks + 8 * g);
            df[ks] = T::ld8(dO + (size_t)qtok * D + 32 * ks + 8 * g);
        }
    }
    f32x4 acc[DT];   // dQ^T: rows d = 16 dt + 4 g + i, column = this lane's query
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[dt] = f32x4{0, 0, 0, 0};

    if (MODE != kLevels && ntiles == 0) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
    }
    for (int t = 0; t < ntiles; ++t) {
        const int k0 = kbeg + t * kT;
        if (t > 0) __syncthreads();
        TD::store(sk, rk);
        TD::store(sv, rv);
        if (MODE != kLevels && t == 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // W' in LDS
        __syncthreads();
        if (t + 1 < ntiles) {
            TD::load_all(K, tok, rk);
            TD::load_all(V, tok, rv);
            if (t + 2 < ntiles) tokens(k0 + 2 * kT, tok);
        }
        // a key tile every lane sees whole skips the mask (one wave vote)
        const bool full = __all(qtok >= 0 && k0 + kT <= kend &&
                                (MODE == kLeaf ? k0 + kT - 1 <= qtok : (k0 >= blk_lo && k0 + kT <= blk_hi)));
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            float v8[8];
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                const int s = 2 * kk + h2;
                f32x4 st = {0, 0, 0, 0}, dp = {0, 0, 0, 0};
                const int kr = krow_of(s, qq);
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    st = T::mma(TD::row8(sk, kr, 32 * ks + 8 * g), qf[ks], st);
                    dp = T::mma(TD::row8(sv, kr, 32 * ks + 8 * g), df[ks], dp);
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float P = fast_exp2(fmaf(st[i], a.tau2, -lse2));
                    if (!full) {
                        const int p = k0 + key_of(s, g, i);
                        bool ok = p < kend && qtok >= 0;
                        if (MODE == kLeaf) ok = ok && p <= qtok;
                        else ok = ok && p >= blk_lo && p < blk_hi;
                        P = ok ? P : 0.f;
                    }
                    v8[4 * h2 + i] = P * fmaf(scs, dp[i], -delta);
                }
            }
            const F bf = T::pack(v8);
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) acc[dt] = T::mma(TD::col8(sk, 32 * kk, 16 * dt), bf, acc[dt]);
        }
    }
    if (MODE == kLevels) {
        // partial rows through LDS as rows, stored as 16-byte pieces of whole
        // rows (16 or 8 lanes a row)
        constexpr int RS = D + 4;
        static_assert(64 * RS * 4 + 64 * 4 <= dq_lds_bytes<T, D, MODE>(WtStage<T, D>::kMaxWk), "rows fit in LDS");
        float* const eo = (float*)smem;
        int* const eq = (int*)(eo + 64 * RS);     // query of each row (-1 = none)
        __syncthreads();                          // every wave is done with the tiles
        const int r0 = 16 * w + qq;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) *(f32x4*)&eo[r0 * RS + 16 * dt + 4 * g] = acc[dt] * a.tau;
        if (g == 0) eq[r0] = qtok;
        __syncthreads();
        constexpr int PPR = D / 8, RPP = kThreads / PPR, NPASS = 64 / RPP;
        const int c8 = 8 * ((int)threadIdx.x % PPR);
#pragma unroll
        for (int ps = 0; ps < NPASS; ++ps) {
            const int r = ps * RPP + (int)threadIdx.x / PPR;
            const int q = eq[r];
            if (q < 0) continue;
            float x[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] = eo[r * RS + c8 + e];
            store8<T>((S*)a.part_dq + (size_t)(slot0 + q) * D + c8, x);
        }
        return;
    }
    // dQ = this pass + the low-rank part (W' from LDS) + (leaf) the partials
    // of the levels where the query was a future query, added in that order.
    // The low-rank part is a product across the wave's lanes, so every lane
    // takes part (a lane without a query uses row 0 and discards the
    // result).  The rest runs on whole rows: the float32 sums go to LDS (the
    // tile and W' space is free now) as rows [query][d], and each thread
    // then adds 8 consecutive elements of the partial rows (two levels at a
    // time) and stores them, so a row moves as 16-byte pieces.
    const size_t row = bh * N + max(qtok, 0);
    F duf[2];
    du_frags<T>((const S*)a.du_q + row * a.wk, a.wk, g, duf);
    f32x4 tot[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) tot[dt] = acc[dt] * a.tau + lowrank_lds<T, D>(duf, swt, a.wk, g, qq, dt);
    constexpr int RS = D + 4;                     // LDS row stride (floats)
    static_assert(MODE == kLevels || 64 * RS * 4 <= dq_lds_bytes<T, D, MODE>(WtStage<T, D>::kMaxWk),
                  "row sums fit in the pass's LDS");
    float* const eq = (float*)smem;
    __syncthreads();                              // every wave is done with the tiles and W'
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) *(f32x4*)&eq[(16 * w + qq) * RS + 16 * dt + 4 * g] = tot[dt];
    __syncthreads();
    if (nq <= 0) return;
    constexpr int PPR = D / 8, RPP = kThreads / PPR, NPASS = 64 / RPP;
    const int c8 = 8 * ((int)threadIdx.x % PPR);
    // rows past the tile's queries read the first query's rows (loads
    // without a branch) and store nothing
    const int tok0 = MODE == kLeaf ? qrow0 : a.perm_q[bh * N + qrow0];
    int tokr[NPASS], tokl[NPASS];
    float s8[NPASS][8];
#pragma unroll
    for (int ps = 0; ps < NPASS; ++ps) {
        const int r = ps * RPP + (int)threadIdx.x / PPR;
        tokr[ps] = r < nq ? (MODE == kLeaf ? qrow0 + r : a.perm_q[bh * N + qrow0 + r]) : -1;
        tokl[ps] = tokr[ps] >= 0 ? tokr[ps] : tok0;
#pragma unroll
        for (int e = 0; e < 8; ++e) s8[ps][e] = eq[r * RS + c8 + e];
    }
    const int leaf = tile / a.lt.per_leaf;
    unsigned lmask = MODE == kLeaf ? leaf_levels(a.lt, leaf, true) : 0u;
    while (lmask) {
        int64_t base[2];
        bool use[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            use[j] = lmask != 0;
            base[j] = 0;
            if (use[j]) {
                const int l = __builtin_ctz(lmask);
                lmask &= lmask - 1;
                base[j] = seg_slot_base(a.lt, bh, l, leaf >> (a.Lv - l), true);
            }
        }
#pragma unroll
        for (int j = 0; j < 2; ++j)
            if (use[j])
#pragma unroll
                for (int ps = 0; ps < NPASS; ++ps) {
                    add8<T>((const S*)a.part_dq + (size_t)(base[j] + tokl[ps]) * D + c8, s8[ps]);
                }
    }
#pragma unroll
    for (int ps = 0; ps < NPASS; ++ps)
        if (tokr[ps] >= 0) store8<T>((S*)a.dQ + (bh * N + tokr[ps]) * D + c8, s8[ps]);
}

// ------------------------------------------------------------------------
// dK, dV: key-centric.  One workgroup per 64 keys (16 per wave, one per lane
// column, K and V rows in registers); query tiles of 64 rows stream through
// LDS with the next tile's rows and row scalars loaded meanwhile.  Per tile:
// S = Q K^T and dP = dO V^T (query rows from LDS), then dV^T += dO^T P and
// dK^T += Q^T dS with the transposed operands read from the query tiles.
// ------------------------------------------------------------------------
// LDS bytes of the key-centric pass (Q and dO tiles, the tile's row
// scalars, W' for the epilogue).
template <class T, int D, int MODE>
__host__ __device__ constexpr size_t dkv_lds_bytes(int wk)
{
    return 2 * (size_t)tile::Tile<T, D, kThreads>::elems(kT) * T::bytes + 4 * kT * 4 +
           (MODE == kLevels ? 0 : WtStage<T, D>::bytes(wk));
}

template <class T, int D, int MODE>
__device__ __forceinline__ void sparse_dkv_body(const BArgs& a, int tile, int h, int b, char* smem)
{
    using S = typename T::store_t;
    using F = typename T::frag_t;
    constexpr int KS = D / 32, DT = D / 16;
    using TD = tile::Tile<T, D, kThreads>;
    constexpr int PT = TD::PER_THREAD;
    S* const sq = (S*)smem;
    S* const so = sq + TD::elems(kT);
    static_assert(TD::elems(kT) * T::bytes % 16 == 0, "row scalars 16-byte aligned");
    float* const s_l2 = (float*)(so + TD::elems(kT));
    float* const s_de = s_l2 + kT;
    float* const s_sc = s_de + kT;
    int* const s_ok = (int*)(s_sc + kT);
    S* const swt = (S*)(s_ok + kT);              // W' (leaf, blocks)
    const size_t bh = (size_t)b * a.H + h;
    const int N = a.N;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int g = lane >> 4, col = lane & 15;
    const S* Q = (const S*)a.Q + bh * N * D;
    const S* K = (const S*)a.K + bh * N * D;
    const S* V = (const S*)a.V + bh * N * D;
    const S* dO = (const S*)a.dO + bh * N * D;

    int level = 0, half = N, kpos, ktok, qbeg, qend, bq = 1, j0 = 0;
    int64_t slot0 = 0;                           // levels: partial row of token t at slot0 + t
    const int32_t* qlist = nullptr;
    const int32_t* klist = nullptr;
    if (MODE == kBlocks) {
        bq = min(a.k, N);
        const int p0 = tile * kT;
        kpos = p0 + 16 * w + col;
        klist = a.perm_k + bh * N;
        ktok = kpos < N ? klist[kpos] : -1;
        const int plast = min(p0 + kT, N) - 1;
        qbeg = max(0, (p0 / bq - a.nbr) * bq);
        qend = min(N, (plast / bq + 1 + a.nbr) * bq);
        qlist = a.perm_q + bh * N;
        j0 = p0;
    } else if (MODE == kLevels) {
        int seg, p0;
        level_tile(a.lt, tile, level, half, seg, p0);
        bq = min(a.k, half);
        kpos = p0 + 16 * w + col;
        const size_t lbase = bh * (size_t)a.lt.off[a.Lv] + (size_t)a.lt.off[level] + (size_t)seg * half;
        klist = a.perm_k + lbase;
        ktok = kpos < half ? klist[kpos] : -1;
        slot0 = seg_slot_base(a.lt, bh, level, seg, false);
        qbeg = max(0, (p0 / bq - a.nbr) * bq);
        qend = min(half, ((min(p0 + kT, half) - 1) / bq + 1 + a.nbr) * bq);
        qlist = a.perm_q + lbase;
        j0 = p0;
    } else {
        int lbeg, lend, leaf;
        leaf_tile(a.lt, tile, leaf, lbeg, j0, lend);
        ktok = j0 + 16 * w + col;
        kpos = ktok;
        if (ktok >= lend) ktok = -1;
        qbeg = j0;
        qend = max(lend, j0);                            // a tile past the leaf's real tokens has no work
    }
    const int blk_lo = (MODE == kLeaf) ? 0 : max(0, (kpos / bq - a.nbr) * bq);
    const int blk_hi = (MODE == kLeaf) ? 0 : min((MODE == kBlocks ? N : half), (kpos / bq + 1 + a.nbr) * bq);

    // query rows of the tile at q0 that this thread stages, and the scalars
    // of query q0 + threadIdx.x (threads < 64).  Staged rows past the
    // scanned range repeat its last entry and a zero token's entry (-1)
    // reads row 0: real rows whose scores the mask drops (the scalars mark
    // them), so the loads need no per-row branch.
    auto tokens = [&](int q0, int (&tok)[PT], int& qt) {
#pragma unroll
        for (int j = 0; j < PT; ++j) {
            const int p = min(q0 + TD::row_of(j), qend - 1);
            tok[j] = (MODE == kLeaf) ? p : max(qlist[p], 0);
        }
        qt = -1;
        if (threadIdx.x < kT) {
            const int p = q0 + threadIdx.x;
            qt = p < qend ? ((MODE == kLeaf) ? p : qlist[p]) : -1;
        }
    };
    float l2 = 0.f, de = 0.f, sc = 0.f;
    auto scalars = [&](int qt) {
        l2 = de = sc = 0.f;
        if (qt >= 0) {
            const size_t row = bh * N + qt;
            l2 = a.rs[row];
            de = a.rs[a.BHN + row];
            sc = a.rs[2 * a.BHN + row];
        }
    };
    const int ntiles = (qend - qbeg + kT - 1) / kT;
    int tok[PT], qt_cur, qt_next = -1;
    uint4 rq[PT], ro[PT];
    if (MODE != kLevels) {
        const size_t wh = (bh % a.H) * D * a.wk;
        WtStage<T, D>::issue((const S*)a.wt_hi + wh, (const S*)a.wt_lo + wh, a.wk, swt);
    }
    qt_cur = -1;
    if (ntiles > 0) {
        tokens(qbeg, tok, qt_cur);
        TD::load_all(Q, tok, rq);
        TD::load_all(dO, tok, ro);
    }
    scalars(qt_cur);
    if (ntiles > 1) tokens(qbeg + kT, tok, qt_next);

    F kf[KS], vf[KS];
    {
        float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        const F zf = T::pack(z);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) { kf[ks] = zf; vf[ks] = zf; }
    }
    if (ktok >= 0) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            kf[ks] = T::ld8(K + (size_t)ktok * D + 32 * ks + 8 * g);
            vf[ks] = T::ld8(V + (size_t)ktok * D + 32 * ks + 8 * g);
        }
    }
    f32x4 akT[DT], avT[DT];   // rows d = 16 dt + 4 g + i, column = this lane's key
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) { akT[dt] = f32x4{0, 0, 0, 0}; avT[dt] = f32x4{0, 0, 0, 0}; }

    if (MODE != kLevels && ntiles == 0) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
    }
    for (int t = 0; t < ntiles; ++t) {
        const int q0 = qbeg + t * kT;
        if (t > 0) __syncthreads();
        TD::store(sq, rq);
        TD::store(so, ro);
        if (threadIdx.x < kT) {
            s_l2[threadIdx.x] = l2;
            s_de[threadIdx.x] = de;
            s_sc[threadIdx.x] = sc;
            s_ok[threadIdx.x] = qt_cur >= 0;
        }
        if (MODE != kLevels && t == 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // W' in LDS
        __syncthreads();
        if (t + 1 < ntiles) {
            TD::load_all(Q, tok, rq);
            TD::load_all(dO, tok, ro);
            scalars(qt_next);
            qt_cur = qt_next;
            if (t + 2 < ntiles) tokens(q0 + 2 * kT, tok, qt_next);
        }
        // a query tile every lane's key sees whole skips the mask (one wave
        // vote; the query lists of a padded recursion may hold zero tokens)
        const bool full = __all(ktok >= 0 && q0 + kT <= qend && !(MODE == kLevels && a.lt.padded) &&
                                (MODE == kLeaf ? q0 >= ktok : (q0 >= blk_lo && q0 + kT <= blk_hi)));
        F pf[2], zf[2];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            float p8[8], z8[8];
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                const int s = 2 * kk + h2;
                f32x4 st = {0, 0, 0, 0}, dp = {0, 0, 0, 0};
                const int qr = krow_of(s, col);
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    st = T::mma(TD::row8(sq, qr, 32 * ks + 8 * g), kf[ks], st);
                    dp = T::mma(TD::row8(so, qr, 32 * ks + 8 * g), vf[ks], dp);
                }
                // this lane's four queries are consecutive: one 16-byte read per scalar
                const int q4 = key_of(s, g, 0);
                const f32x4 l2v = *(const f32x4*)&s_l2[q4], scv = *(const f32x4*)&s_sc[q4],
                            dev = *(const f32x4*)&s_de[q4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float P = fast_exp2(fmaf(st[i], a.tau2, -l2v[i]));
                    if (!full) {
                        const int p = q0 + q4 + i;
                        bool ok = ktok >= 0 && s_ok[q4 + i];
                        if (MODE == kLeaf) ok = ok && p >= ktok;
                        else ok = ok && p >= blk_lo && p < blk_hi;
                        P = ok ? P : 0.f;
                    }
                    p8[4 * h2 + i] = P * scv[i];
                    z8[4 * h2 + i] = P * fmaf(scv[i], dp[i], -dev[i]);
                }
            }
            pf[kk] = T::pack(p8);
            zf[kk] = T::pack(z8);
        }
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                avT[dt] = T::mma(TD::col8(so, 32 * kk, 16 * dt), pf[kk], avT[dt]);
                akT[dt] = T::mma(TD::col8(sq, 32 * kk, 16 * dt), zf[kk], akT[dt]);
            }
    }

    if (MODE == kLevels) {
        // partial rows through LDS as rows, stored as 16-byte pieces of whole
        // rows (16 or 8 lanes a row)
        constexpr int RS = D + 4;
        static_assert(2 * 64 * RS * 4 + 64 * 4 <= dkv_lds_bytes<T, D, MODE>(WtStage<T, D>::kMaxWk) ||
                      64 * RS * 4 + 64 * 4 <= dkv_lds_bytes<T, D, MODE>(WtStage<T, D>::kMaxWk), "rows fit in LDS");
        float* const eo = (float*)smem;
        int* const ek = (int*)(eo + 64 * RS);     // key of each row (-1 = none)
        const int r0 = 16 * w + col;
        constexpr int PPR = D / 8, RPP = kThreads / PPR, NPASS = 64 / RPP;
        const int c8 = 8 * ((int)threadIdx.x % PPR);
        // dK, then dV through the same rows
#pragma unroll
        for (int part = 0; part < 2; ++part) {
            __syncthreads();                      // the tiles (or the previous part's rows) are done with
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
                *(f32x4*)&eo[r0 * RS + 16 * dt + 4 * g] = part == 0 ? akT[dt] * a.tau : avT[dt];
            if (g == 0) ek[r0] = ktok;
            __syncthreads();
            S* dst = (S*)(part == 0 ? a.part_dk : a.part_dv);
#pragma unroll
            for (int ps = 0; ps < NPASS; ++ps) {
                const int r = ps * RPP + (int)threadIdx.x / PPR;
                const int k = ek[r];
                if (k < 0) continue;
                float x[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] = eo[r * RS + c8 + e];
                store8<T>(dst + (size_t)(slot0 + k) * D + c8, x);
            }
        }
        return;
    }
    // dK, dV = this pass + the low-rank parts + (leaf) the partials of the
    // levels where the key was a past key, added in that order.  The du and
    // low-rank dV rows are requested together, before the low-rank product
    // (W' from LDS); the partial rows follow two (dK, dV) pairs at a time so
    // their loads are in flight together.  The low-rank dK part is a product
    // across the wave's lanes, so every lane takes part (a lane without a
    // key uses row 0).
    const size_t row = bh * N + max(ktok, 0);
    F duf[2];
    du_frags<T>((const S*)a.du_k + row * a.wk, a.wk, g, duf);
    f32x4 tk[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) tk[dt] = akT[dt] * a.tau + lowrank_lds<T, D>(duf, swt, a.wk, g, col, dt);

    // The rest runs on whole rows: the two float32 sums go to LDS (the tile,
    // scalar and W' space is free now) as rows [key][d], and each thread
    // then takes 8 consecutive elements of a row, so the low-rank dV rows,
    // the partial rows and the results move as 16-byte pieces with 16 (d_h
    // 128) or 8 lanes covering a row, instead of 8-byte pieces of 16 rows
    // per instruction.
    constexpr int RS = D + 4;                     // LDS row stride (floats)
    static_assert(MODE == kLevels || 2 * 64 * RS * 4 <= dkv_lds_bytes<T, D, MODE>(WtStage<T, D>::kMaxWk),
                  "row sums fit in the pass's LDS");
    float* const ek = (float*)smem;               // dK rows
    float* const ev = ek + 64 * RS;               // dV rows
    __syncthreads();                              // every wave is done with the tiles and W'
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
        const int r = 16 * w + col, c = 16 * dt + 4 * g;
        *(f32x4*)&ek[r * RS + c] = tk[dt];
        *(f32x4*)&ev[r * RS + c] = avT[dt];
    }
    __syncthreads();
    constexpr int PPR = D / 8, RPP = kThreads / PPR, NPASS = 64 / RPP;
    const int piece = threadIdx.x % PPR, c8 = 8 * piece;
    // rows past the keys of the list (or leaf) read the tile's first key's
    // rows (loads without a branch) and store nothing
    const int nrow = MODE == kLeaf ? qend - j0 : min(64, N - j0);
    if (nrow <= 0) return;
    const int tok0 = MODE == kLeaf ? j0 : klist[j0];
    int tokr[NPASS], tokl[NPASS];
    float sk8[NPASS][8], sv8[NPASS][8];
#pragma unroll
    for (int ps = 0; ps < NPASS; ++ps) {
        const int r = ps * RPP + (int)threadIdx.x / PPR;
        tokr[ps] = r < nrow ? (MODE == kLeaf ? j0 + r : klist[j0 + r]) : -1;
        tokl[ps] = tokr[ps] >= 0 ? tokr[ps] : tok0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            sk8[ps][e] = ek[r * RS + c8 + e];
            sv8[ps][e] = ev[r * RS + c8 + e];
        }
    }
#pragma unroll
    for (int ps = 0; ps < NPASS; ++ps) add8<T>((const S*)a.dv_lr + (bh * N + tokl[ps]) * D + c8, sv8[ps]);
    const int leaf = tile / a.lt.per_leaf;
    unsigned lmask = MODE == kLeaf ? leaf_levels(a.lt, leaf, false) : 0u;
    while (lmask) {
        // two levels at a time, for every row of the thread
        int64_t base[2];
        bool use[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            use[j] = lmask != 0;
            base[j] = 0;
            if (use[j]) {
                const int l = __builtin_ctz(lmask);
                lmask &= lmask - 1;
                base[j] = seg_slot_base(a.lt, bh, l, leaf >> (a.Lv - l), false);
            }
        }
#pragma unroll
        for (int j = 0; j < 2; ++j)
            if (use[j])
#pragma unroll
                for (int ps = 0; ps < NPASS; ++ps) {
                    const size_t slot = (size_t)(base[j] + tokl[ps]);
                    add8<T>((const S*)a.part_dk + slot * D + c8, sk8[ps]);
                    add8<T>((const S*)a.part_dv + slot * D + c8, sv8[ps]);
                }
    }
#pragma unroll
    for (int ps = 0; ps < NPASS; ++ps)
        if (tokr[ps] >= 0) {
            const size_t o = (bh * N + tokr[ps]) * D + c8;
            store8<T>((S*)a.dK + o, sk8[ps]);
            store8<T>((S*)a.dV + o, sv8[ps]);
        }
}

// float32 storage at d_h 128 holds twice the operand registers: one wave
// per SIMD, so the accumulation registers can take what does not fit
template <class T, int D>
constexpr int two_pass_waves() { return T::bytes == 4 && D == 128 ? 1 : 2; }

// LDS of the two passes: the tiles plus, outside the levels, W' sized for
// the largest wk (64).
template <class T, int D, int MODE>
constexpr size_t dq_lds() { return dq_lds_bytes<T, D, MODE>(WtStage<T, D>::kMaxWk); }
template <class T, int D, int MODE>
constexpr size_t dkv_lds() { return dkv_lds_bytes<T, D, MODE>(WtStage<T, D>::kMaxWk); }

template <class T, int D, int MODE>
__global__ __launch_bounds__(kThreads, (two_pass_waves<T, D>())) void sparse_dq_kernel(BArgs a)
{
    __shared__ __attribute__((aligned(16))) char smem[dq_lds<T, D, MODE>()];
    int tile, h, b;
    xcd_tile(tile, h, b);
    sparse_dq_body<T, D, MODE>(a, tile, h, b, smem);
}

template <class T, int D, int MODE>
__global__ __launch_bounds__(kThreads, (two_pass_waves<T, D>())) void sparse_dkv_kernel(BArgs a)
{
    __shared__ __attribute__((aligned(16))) char smem[dkv_lds<T, D, MODE>()];
    int tile, h, b;
    xcd_tile(tile, h, b);
    sparse_dkv_body<T, D, MODE>(a, tile, h, b, smem);
}

// Both leaf passes in one launch: the workgroups of a leaf (its query tiles
// for dQ, then its key tiles for dK, dV) are consecutive, so they run on one
// XCD at about the same time and the leaf's Q, K, V, dO rows, read by both
// passes, come from that XCD's L2 the second time.
template <class T, int D>
__global__ __launch_bounds__(kThreads, (two_pass_waves<T, D>())) void sparse_leaf_bwd_kernel(BArgs a)
{
    int t2, h, b;
    xcd_tile(t2, h, b);
    const int per = a.lt.per_leaf, leaf = t2 / (2 * per), r = t2 - leaf * 2 * per;
    // the two passes share one LDS region (a workgroup runs one of them)
    constexpr size_t q = dq_lds<T, D, kLeaf>(), kv = dkv_lds<T, D, kLeaf>();
    __shared__ __attribute__((aligned(16))) char smem[q > kv ? q : kv];
    if (r < per) sparse_dq_body<T, D, kLeaf>(a, leaf * per + r, h, b, smem);
    else sparse_dkv_body<T, D, kLeaf>(a, leaf * per + r - per, h, b, smem);
}

// ------------------------------------------------------------------------
// Whole sorted blocks at once (b = BQ in {64, 128}): each block is BQ sorted
// queries and the BQ sorted keys they see (Alg. 4 blocks; the per-level
// SortLSH calls of Alg. 5).  BQ / 16 waves each own 16 keys (their V rows in
// registers, dK^T and dV^T accumulators); the block's queries stream through
// LDS in tiles of 64 with the next tile's rows loaded into registers
// meanwhile.  Per tile: S = Q K^T and dP = dO V^T (query rows from LDS), P
// and dS in registers, dV^T += dO^T P and dK^T += Q^T dS with the transposed
// operands read from the query tiles, then dS^T goes to LDS and the tile's
// complete dQ^T = K^T dS^T is formed from the block's K tile.  Every input
// row is read once per block and dQ, dK, dV are each written once: partials
// by natural token index (levels) or the final sums with the low-rank parts
// in the storage dtype (non-causal blocks).
//
// The grid holds as many workgroups as the device runs at once and each
// walks the blocks id, id + gridDim.x, ...  The next block's loads overlap
// the current block's last tile: its index lists at the start of the tile,
// its V rows (into the V registers) and K rows once dP is formed, and its
// first Q / dO tile at the end; the current block's dK, dV are stored once
// the next block's rows are in LDS.  At the levels every row load reads a
// real row (a short block's missing rows repeat its last entry and are
// masked), so loads there carry no per-row branch and the compiler can wait
// for exactly the loads it needs (its memory counter retires in order).
// ------------------------------------------------------------------------
//
// Blocks of QB = 256 (the levels only) are two consecutive work items of one
// workgroup, one per 128-key half: each streams all 256 queries of the block
// (the second time from the compute unit's caches), so dK and dV of the
// half's keys are complete.  The first half's dQ tiles wait in LDS (bf16,
// each thread keeps the values it will add itself) and the second half adds
// them before storing the block's dQ partials, so each level entry still has
// one dQ partial row.
//
// waves per SIMD: three for 64-key blocks at d_h 64, two otherwise (a
// 128-key block is 8 waves, two per SIMD)
template <int D, int BQ>
constexpr int block_waves() { return BQ == 64 && D == 64 ? 3 : 2; }

template <class T, int D, int BQ, int MODE, int QB = BQ, bool FULL = MODE == kLevels>
__global__ __launch_bounds__(BQ * 4, (block_waves<D, BQ>())) void sparse_bwd_block_kernel(BArgs a)
{
    using S = typename T::store_t;
    using F = typename T::frag_t;
    constexpr int NW = BQ / 16, NT = 64 * NW;
    constexpr int KS = D / 32, DT = D / 16, NQT = QB / 64, NKT = BQ / 64;
    constexpr int HALVES = QB / BQ;                       // work items per block
    static_assert(HALVES == 1 || (HALVES == 2 && MODE == kLevels), "key halves: levels only");
    constexpr int PER_WQ = DT * 4 / NW;                   // dQ output tiles per wave and query tile
    // the first key half's dQ tiles, thread by thread (bf16, 4 values per tile)
    __shared__ __attribute__((aligned(16))) S sdq[HALVES == 2 ? NQT * PER_WQ * NT * 4 : 1];
    using TD = tile::Tile<T, D, NT>;        // Q, dO, K tiles (rows of D)
    using TS = tile::Tile<T, 64, NT>;       // dS^T tile (BQ rows of 64 queries)
    constexpr int PT = TD::PER_THREAD;
    // every block holds QB valid queries and BQ valid keys (the levels, unless
    // a level's half length is not a multiple of QB: then its last block is short)
    constexpr bool kFull = FULL;
    static_assert(!FULL || MODE == kLevels, "full blocks: levels only");
    // levels: rows past a short block's entries are loaded from its last
    // entry (a real row, masked out), so the row loads carry no branch
    constexpr bool kClamp = MODE == kLevels;
    static_assert(TS::elems(BQ) <= 2 * TD::elems(64), "dS^T fits in the query tiles");
    __shared__ __attribute__((aligned(16))) S sk[TD::elems(BQ)];
    __shared__ __attribute__((aligned(16))) S sqo[2 * TD::elems(64)];   // Q tile, dO tile; later dS^T
    __shared__ __attribute__((aligned(16))) float s_l2[64], s_de[64], s_sc[64];
    __shared__ __attribute__((aligned(16))) int s_qt[64];
    S* const sq = sqo;
    S* const so = sqo + TD::elems(64);
    S* const sds = sqo;

    const int N = a.N;
    const int w = threadIdx.x >> 6;
    // lane coordinates from a fresh copy of the thread index at every block
    // (lane-dependent LDS addresses are formed where used instead of held in
    // registers across the block loop)
    int tx, g, col, kloc;                                // kloc: this lane's key within a block
    auto lanes = [&]() {
        tx = threadIdx.x;
        asm volatile("" : "+v"(tx));
        g = (tx & 63) >> 4;
        col = tx & 15;
        kloc = 16 * w + col;
    };
    lanes();

    // ---- block id -> head and the sorted positions [p0, p0 + nv) of its lists
    struct Blk {
        size_t bh;
        int nv, nvk;                                 // valid queries, valid keys of the item
        int half;                                    // key half of a 256-key block (0 otherwise)
        int64_t qslot, kslot;                        // levels: partial rows of token t at qslot + t (as a
                                                     // query) and kslot + t (as a key)
        const int32_t* ql;
        const int32_t* kl;
    };
    auto block_of = [&](int id) {
        Blk k;
        // key halves: items 2 m and 2 m + 1 are the halves of block m
        const int item = HALVES == 1 ? id : id >> 1;
        k.half = HALVES == 1 ? 0 : id & 1;
        const int x = item % a.nbx;
        k.bh = (size_t)(item / a.nbx);                   // b * H + h
        if (MODE == kLevels && !FULL) {
            // level lists of any even length: ceil(h / QB) blocks per list of
            // h entries, the last one short (no zero tokens: unpadded levels)
            int level = 0, first = 0;
            for (;;) {
                const int cnt = ((a.lt.len[level + 1] + QB - 1) / QB) << level;
                if (x < first + cnt || level + 1 >= a.Lv) break;
                first += cnt;
                ++level;
            }
            const int h = a.lt.len[level + 1], nbs = (h + QB - 1) / QB;
            const int j = x - first, seg = j / nbs, p0 = (j - seg * nbs) * QB;
            const size_t base = k.bh * (size_t)a.lt.off[a.Lv] + (size_t)a.lt.off[level] + (size_t)seg * h + p0;
            k.nv = min(QB, h - p0);
            k.nvk = max(0, min(BQ, k.nv - k.half * BQ));
            k.ql = a.perm_q + base;
            k.kl = a.perm_k + base + (k.nvk > 0 ? k.half * BQ : 0);   // (no keys: rows of half 0, masked)
            k.qslot = seg_slot_base(a.lt, k.bh, level, seg, true);
            k.kslot = seg_slot_base(a.lt, k.bh, level, seg, false);
        } else if (MODE == kLevels) {
            // (whole-block levels are never padded: N / 2 entries per level)
            const int per_level = (N / 2) / QB;
            const int level = x / per_level;
            const int t = x - level * per_level;
            const size_t base = k.bh * (size_t)a.lt.off[a.Lv] + (size_t)a.lt.off[level] + (size_t)t * QB;
            k.ql = a.perm_q + base;
            k.kl = a.perm_k + base + k.half * BQ;
            k.nv = QB;
            k.nvk = BQ;
            // a block never straddles a segment (the half length is a multiple of QB)
            const int seg = t * QB / a.lt.len[level + 1];
            k.qslot = seg_slot_base(a.lt, k.bh, level, seg, true);
            k.kslot = seg_slot_base(a.lt, k.bh, level, seg, false);
        } else {
            const int p0 = x * BQ;
            k.qslot = k.kslot = 0;
            k.ql = a.perm_q + k.bh * N + p0;
            k.kl = a.perm_k + k.bh * N + p0;
            k.nv = min(BQ, N - p0);
            k.nvk = k.nv;
        }
        return k;
    };
    // index lists of a block: K tile rows, this lane's key, every query tile
    struct Idx {
        int ktk[NKT][PT];
        int ktok;
        int qtk[NQT][PT];
        int qt1[NQT];                                    // query 64 qt + (tx % 64) (scalars, dQ rows)
    };
    // the key lists of a block, and the query list entries of its tile t
    // (a block's later query tiles are indexed while its first is consumed,
    // so their entries are not held in registers across the block change)
    auto indices_k = [&](const Blk& k, Idx& ix) {
#pragma unroll
        for (int t = 0; t < NKT; ++t)
#pragma unroll
            for (int j = 0; j < PT; ++j) {
                const int r = 64 * t + TD::row_of(j, tx);
                if constexpr (kFull) ix.ktk[t][j] = k.kl[(uint32_t)r];
                else if constexpr (kClamp) ix.ktk[t][j] = k.kl[(uint32_t)min(r, max(k.nvk, 1) - 1)];
                else ix.ktk[t][j] = r < k.nvk ? k.kl[(uint32_t)r] : -1;
            }
        ix.ktok = (kFull || kloc < k.nvk) ? k.kl[(uint32_t)kloc] : -1;
    };
    auto indices_q = [&](const Blk& k, Idx& ix, int t) {
#pragma unroll
        for (int j = 0; j < PT; ++j) {
            const int r = 64 * t + TD::row_of(j, tx);
            if constexpr (kFull) ix.qtk[t][j] = k.ql[(uint32_t)r];
            else if constexpr (kClamp) ix.qtk[t][j] = k.ql[(uint32_t)min(r, k.nv - 1)];
            else ix.qtk[t][j] = r < k.nv ? k.ql[(uint32_t)r] : -1;
        }
        const int r = 64 * t + (tx & 63);
        ix.qt1[t] = (kFull || r < k.nv) ? k.ql[(uint32_t)r] : -1;
    };
    auto kload = [&](size_t bh, const Idx& ix, uint4 (&rk)[NKT][PT]) {
        const S* K = (const S*)a.K + bh * N * D;
#pragma unroll
        for (int t = 0; t < NKT; ++t) {
            if constexpr (kFull || kClamp) TD::load_all(K, ix.ktk[t], rk[t], tx);
            else TD::load(K, ix.ktk[t], rk[t], tx);
        }
    };
    auto vload = [&](size_t bh, int ktok, F (&vf)[KS]) {
        const S* V = (const S*)a.V + bh * N * D;
        if (kFull || ktok >= 0) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) vf[ks] = T::ld8(V + (size_t)ktok * D + 32 * ks + 8 * g);
        } else {
            float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) vf[ks] = T::pack(z);
        }
    };
    uint4 rq[PT], ro[PT];
    float l2 = 0.f, de = 0.f, sc = 0.f;
    // rows and row scalars of query tile qt (every thread reads the scalars
    // of query 64 qt + tx % 64; threads < 64 publish them)
    auto qload = [&](size_t bh, const Idx& ix, int qt) {
        const S* Q = (const S*)a.Q + bh * N * D;
        const S* dO = (const S*)a.dO + bh * N * D;
        if constexpr (kFull || kClamp) {
            TD::load_all(Q, ix.qtk[qt], rq, tx);
            TD::load_all(dO, ix.qtk[qt], ro, tx);
        } else {
            TD::load(Q, ix.qtk[qt], rq, tx);
            TD::load(dO, ix.qtk[qt], ro, tx);
        }
        const float* rs = a.rs + bh * N;
        const uint32_t t = (uint32_t)max(ix.qt1[qt], 0);
        l2 = rs[t];
        de = (rs + a.BHN)[t];
        sc = (rs + 2 * a.BHN)[t];
    };

    // dK, dV of a lane's key: rows d = 16 dt + 4 g + i of the accumulators
    f32x4 akT[DT], avT[DT];
    auto store_dkv = [&](size_t bh, int64_t kslot, int ktok) {
        if (MODE == kLevels) {
            if (!(kFull || ktok >= 0)) return;
            const size_t slot = (size_t)(kslot + ktok);
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const int d0 = 16 * dt + 4 * g;
                store4<T>((S*)a.part_dk + slot * D + d0, akT[dt] * a.tau);
                store4<T>((S*)a.part_dv + slot * D + d0, avT[dt]);
            }
        } else {
            // the low-rank dK part is a product across the wave's lanes: every
            // lane takes part (a lane without a key uses row 0), then stores
            // (one 16-row slice at a time, so only one slice of it is live)
            const size_t wh = (bh % a.H) * D * a.wk;
            const S* du = (const S*)a.du_k + (bh * N + max(ktok, 0)) * a.wk;
            const size_t row = bh * N + max(ktok, 0);
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const f32x4 lr = lowrank_tile<T>(du, (const S*)a.wt_hi + wh, (const S*)a.wt_lo + wh, a.wk, g, col, dt);
                if (ktok >= 0) {
                    const int d0 = 16 * dt + 4 * g;
                    store4<T>((S*)a.dK + row * D + d0, akT[dt] * a.tau + lr);
                    store4<T>((S*)a.dV + row * D + d0, avT[dt] + load4<T>((const S*)a.dv_lr + row * D + d0));
                }
            }
        }
    };

    // items of this workgroup: id, id + gridDim.x, ... (key halves: the two
    // halves of blocks blockIdx.x, blockIdx.x + gridDim.x, ... in turn)
    int id = HALVES == 1 ? (int)blockIdx.x : 2 * (int)blockIdx.x;
    Blk blk = block_of(id);
    Idx ix;
    indices_k(blk, ix);
    indices_q(blk, ix, 0);
    uint4 rk[NKT][PT];
    F vf[KS];
    kload(blk.bh, ix, rk);
    vload(blk.bh, ix.ktok, vf);
    qload(blk.bh, ix, 0);
    // a block's dK, dV leave once the next block's rows are in LDS (so no
    // wait for those rows also waits for the stores): the previous block
    size_t prev_bh = 0;
    int64_t prev_kslot = 0;
    int prev_ktok = -1;
    bool first = true;
    for (;;) {
        lanes();
        const size_t bh = blk.bh;
        const int64_t qslot = blk.qslot, kslot = blk.kslot;
        const int half = blk.half;
        const int ktok = ix.ktok;
        if (!first) __syncthreads();                     // the previous block's dQ phase is done with LDS
#pragma unroll
        for (int t = 0; t < NKT; ++t) TD::store(sk, rk[t], 64 * t, tx);
        // (this lane's K row is read from the block's K tile when needed)

        const int nid = HALVES == 1 ? id + (int)gridDim.x : ((id & 1) ? id - 1 + 2 * (int)gridDim.x : id + 1);
        const bool has_next = nid < a.nblk;
        Blk nblk = blk;
        Idx nix;

#pragma unroll
        for (int qt = 0; qt < NQT; ++qt) {
            const bool last = qt + 1 == NQT;
            if (qt > 0) __syncthreads();                 // previous dS^T / dQ phase done
            TD::store(sq, rq, 0, tx);
            TD::store(so, ro, 0, tx);
            if (threadIdx.x < 64) {
                // (a short block's missing query: an infinite log denominator, P = 0)
                s_l2[tx] = (kFull || ix.qt1[qt] >= 0) ? l2 : (kClamp ? INFINITY : 0.f);
                s_de[tx] = de;
                s_sc[tx] = sc;
                s_qt[tx] = ix.qt1[qt];
            }
            __syncthreads();
            if (qt == 0) {                               // the previous block's dK, dV leave now
                if (!first) store_dkv(prev_bh, prev_kslot, prev_ktok);
                first = false;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) { akT[dt] = f32x4{0, 0, 0, 0}; avT[dt] = f32x4{0, 0, 0, 0}; }
            }
            if (!last) {
                indices_q(blk, ix, qt + 1);
                qload(bh, ix, qt + 1);                   // next tile in flight
            } else if (has_next) {
                nblk = block_of(nid);                    // the next block's index lists
                indices_k(nblk, nix);
                indices_q(nblk, nix, 0);
            }

            // S and dP for the 64 queries x this wave's 16 keys (rows: queries);
            // P sc and dS packed at once as the 32-query k-step operands
            F pf[2], zf[2];
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                float p8[8], z8[8];
#pragma unroll
                for (int h2 = 0; h2 < 2; ++h2) {
                    const int s = 2 * kk + h2;
                    f32x4 st = {0, 0, 0, 0}, dp = {0, 0, 0, 0};
                    const int qr = krow_of(s, col);
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) {
                        st = T::mma(TD::row8(sq, qr, 32 * ks + 8 * g), TD::row8(sk, kloc, 32 * ks + 8 * g), st);
                        dp = T::mma(TD::row8(so, qr, 32 * ks + 8 * g), vf[ks], dp);
                    }
                    // this lane's four queries are consecutive: 16-byte scalar reads
                    const int q4 = key_of(s, g, 0);
                    const f32x4 l2v = *(const f32x4*)&s_l2[q4], scv = *(const f32x4*)&s_sc[q4],
                                dev = *(const f32x4*)&s_de[q4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const bool ok = kFull || (kClamp ? ktok >= 0 : (ktok >= 0 && s_qt[q4 + i] >= 0));
                        const float P = ok ? fast_exp2(fmaf(st[i], a.tau2, -l2v[i])) : 0.f;
                        p8[4 * h2 + i] = P * scv[i];
                        z8[4 * h2 + i] = P * fmaf(scv[i], dp[i], -dev[i]);
                    }
                }
                pf[kk] = T::pack(p8);
                zf[kk] = T::pack(z8);
            }
            if (last && has_next) {                      // V and K rows of the next block
                vload(nblk.bh, nix.ktok, vf);
                kload(nblk.bh, nix, rk);
            }
            // dV^T += dO^T (P sc), dK^T += Q^T dS over two 32-query k-steps
#pragma unroll
            for (int kk = 0; kk < 2; ++kk)
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) {
                    avT[dt] = T::mma(TD::col8(so, 32 * kk, 16 * dt, tx), pf[kk], avT[dt]);
                    akT[dt] = T::mma(TD::col8(sq, 32 * kk, 16 * dt, tx), zf[kk], akT[dt]);
                }
            if (last && has_next) qload(nblk.bh, nix, 0);  // the next block's first Q / dO tile, under the dQ phase
            __syncthreads();                             // query tiles no longer read
            // dS^T [key][query] into the query-tile space: slots 8g + j of k-step kk
            // hold queries 32 kk + 8 g + j, eight consecutive queries per write
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                const int q0 = 32 * kk + 8 * g;
                S* dst = &sds[TS::row(kloc) + q0];
                if constexpr (T::bytes == 2) {
                    *(F*)dst = zf[kk];
                } else {
#pragma unroll
                    for (int j = 0; j < 8; ++j) dst[j] = zf[kk][j];
                }
            }
            __syncthreads();
            // dQ^T = K^T dS^T for this tile: DT x 4 output tiles spread over the
            // waves, each wave's tiles sharing one 16-row slice dt of K^T when it
            // has four or more
            constexpr int TILES = DT * 4, PER_W = TILES / NW;
            static_assert(TILES % NW == 0 && (PER_W % 4 == 0 || 4 % PER_W == 0), "dQ tiles per wave");
            f32x4 dq[PER_W];
#pragma unroll
            for (int u = 0; u < PER_W; ++u) dq[u] = f32x4{0, 0, 0, 0};
#pragma unroll
            for (int kb = 0; kb < BQ; kb += 32) {
                F kt_frag = TD::col8(sk, kb, 16 * ((w * PER_W) / 4), tx);
#pragma unroll
                for (int u = 0; u < PER_W; ++u) {
                    const int tix = w * PER_W + u, dt = tix / 4, qtile = tix % 4;
                    if (u > 0 && qtile == 0) kt_frag = TD::col8(sk, kb, 16 * dt, tx);
                    dq[u] = T::mma(kt_frag, TS::col8(sds, kb, 16 * qtile, tx), dq[u]);
                }
            }
#pragma unroll
            for (int u = 0; u < PER_W; ++u) {
                const int tix = w * PER_W + u, dt = tix / 4, qtile = tix % 4;
                const int qtok = s_qt[16 * qtile + col];
                const int d0 = 16 * dt + 4 * g;
                if (MODE == kLevels) {
                    if (!kFull && qtok < 0) continue;
                    f32x4 v = dq[u] * a.tau;
                    if constexpr (HALVES == 2) {
                        S* keep = sdq + (((qt * PER_WQ + u) * NT) + tx) * 4;
                        if (half == 0) {                 // first key half: kept for the second
                            store4<T>(keep, v);
                            continue;
                        }
                        v += load4<T>(keep);
                    }
                    S* out = (S*)a.part_dq + (size_t)(qslot + qtok) * D + d0;
                    store4<T>(out, v);
                } else {
                    // the low-rank part is a product across the wave's lanes:
                    // every lane takes part (a lane without a query uses row 0)
                    const size_t wh = (bh % a.H) * D * a.wk;
                    const f32x4 lr = lowrank_tile<T>((const S*)a.du_q + (bh * N + max(qtok, 0)) * a.wk,
                                                     (const S*)a.wt_hi + wh, (const S*)a.wt_lo + wh, a.wk, g, col, dt);
                    if (qtok < 0) continue;
                    const size_t row = bh * N + qtok;
                    store4<T>((S*)a.dQ + row * D + d0, dq[u] * a.tau + lr);
                }
            }
        }

        prev_bh = bh;
        prev_kslot = kslot;
        prev_ktok = ktok;
        if (!has_next) break;
        id = nid;
        blk = nblk;
        ix = nix;
    }
    store_dkv(prev_bh, prev_kslot, prev_ktok);
}

// Whole-block launch: as many workgroups as the device runs at once (cached
// per instantiation and device), each walking its share of the blocks.
template <class T, int D, int BQ, int MODE, int QB = BQ, bool FULL = MODE == kLevels>
void launch_blocks(const char* name, BArgs a, int nbx, int BH, hipStream_t st)
{
    static int resident[64] = {0};
    auto kern = sparse_bwd_block_kernel<T, D, BQ, MODE, QB, FULL>;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
    int& res = resident[dev & 63];
    if (res == 0) {
        int cus = 0, per = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            cus = 256;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kern, BQ * 4, 0) != hipSuccess || per <= 0) per = 1;
        res = cus * per;
    }
    a.nbx = nbx;
    a.nblk = nbx * BH * (QB / BQ);                       // work items (key halves of QB = 256)
    const int blocks = nbx * BH;                         // a workgroup starts at a block's first item
    const int grid = blocks < res ? blocks : res;
    ELSAA_LAUNCH(name, kern, dim3(grid), dim3(BQ * 4), 0, st, a);
}

// causal b = 256 levels run as two 128-key halves per block (bf16, no
// neighbouring blocks, no padded level)
bool block_halves(const Shape& s)
{
    return s.causal && s.bf16 && s.Lv > 0 && s.k == 256 && s.neighbors == 0 && !s.lt.padded;
}

template <class T, int D>
hipError_t launch_t(const Shape& s, const BArgs& a, hipStream_t st, int parts)
{
    hipError_t e;
    // whole-block kernel: b in {64, 128}, blocks never straddle a segment;
    // b = 128 only where its registers fit without spilling (bf16 storage;
    // non-causal blocks, which also form the low-rank parts, only at d_h 64);
    // causal b = 256 (block_halves) as two 128-key halves per block
    const int bq = s.k;
    const bool fits128 = T::bytes == 2 && (s.causal || D == 64);
    const bool whole = (bq == 64 || (bq == 128 && fits128)) && s.neighbors == 0 &&
                       (s.causal ? (!s.lt.padded && s.n_leaf % bq == 0) : true);
    if (!s.causal) {
        if (whole) {
            if (!(parts & kSparseFinalQ)) return hipSuccess;
            const int nbx = (s.N + bq - 1) / bq;
            if (bq == 64) launch_blocks<T, D, 64, kBlocks>("sparse_bwd_blocks", a, nbx, s.B * s.H, st);
            else if constexpr (T::bytes == 2 && D == 64)
                launch_blocks<T, D, 128, kBlocks>("sparse_bwd_blocks", a, nbx, s.B * s.H, st);
            return hipGetLastError();
        }
        dim3 grid((s.N + kT - 1) / kT, s.H, s.B);
        if (parts & kSparseFinalQ) {
            ELSAA_LAUNCH("sparse_dq_blocks", (sparse_dq_kernel<T, D, kBlocks>), grid, dim3(kThreads), 0, st, a);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        if (parts & kSparseFinalKV) {
            ELSAA_LAUNCH("sparse_dkv_blocks", (sparse_dkv_kernel<T, D, kBlocks>), grid, dim3(kThreads), 0, st, a);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        return hipSuccess;
    }
    if (s.Lv > 0 && (parts & kSparseLevels)) {
        if (whole) {
            const int nbx = s.Lv * (s.N / 2) / bq;
            if (bq == 64) launch_blocks<T, D, 64, kLevels>("sparse_bwd_levels", a, nbx, s.B * s.H, st);
            else if constexpr (T::bytes == 2) launch_blocks<T, D, 128, kLevels>("sparse_bwd_levels", a, nbx, s.B * s.H, st);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        } else if (block_halves(s)) {
            // 256-key blocks as two 128-key halves in turn; a level whose
            // half length is not a multiple of 256 ends its lists with a short block
            if (s.n_leaf % 256 == 0) {
                const int nbx = s.Lv * (s.N / 2) / 256;
                if constexpr (T::bytes == 2)
                    launch_blocks<T, D, 128, kLevels, 256>("sparse_bwd_levels", a, nbx, s.B * s.H, st);
            } else {
                int nbx = 0;
                for (int l = 0; l < s.Lv; ++l) nbx += ((s.lt.len[l + 1] + 255) / 256) << l;
                if constexpr (T::bytes == 2)
                    launch_blocks<T, D, 128, kLevels, 256, false>("sparse_bwd_levels", a, nbx, s.B * s.H, st);
            }
            if ((e = hipGetLastError()) != hipSuccess) return e;
        } else {
            dim3 grid(a.lt.first[s.Lv], s.H, s.B);
            ELSAA_LAUNCH("sparse_dq_levels", (sparse_dq_kernel<T, D, kLevels>), grid, dim3(kThreads), 0, st, a);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            ELSAA_LAUNCH("sparse_dkv_levels", (sparse_dkv_kernel<T, D, kLevels>), grid, dim3(kThreads), 0, st, a);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
    }
    if ((parts & kSparseFinal) == kSparseFinal) {
        dim3 grid(2 * a.lt.leaf_tiles(), s.H, s.B);
        ELSAA_LAUNCH("sparse_leaf_bwd", (sparse_leaf_bwd_kernel<T, D>), grid, dim3(kThreads), 0, st, a);
        return hipGetLastError();
    }
    dim3 grid(a.lt.leaf_tiles(), s.H, s.B);
    if (parts & kSparseFinalQ) {
        ELSAA_LAUNCH("sparse_dq_leaf", (sparse_dq_kernel<T, D, kLeaf>), grid, dim3(kThreads), 0, st, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (parts & kSparseFinalKV) {
        ELSAA_LAUNCH("sparse_dkv_leaf", (sparse_dkv_kernel<T, D, kLeaf>), grid, dim3(kThreads), 0, st, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace

hipError_t launch_sparse_bwd(const Shape& s, const void* Q, const void* K, const void* V,
                             const void* dO, const int32_t* perm_q, const int32_t* perm_k,
                             const float* rs, const void* du_q, const void* du_k, const void* wt_hi,
                             const void* wt_lo, const void* dv_lr, void* part_dq, void* part_dk, void* part_dv,
                             void* dQ, void* dK, void* dV, hipStream_t st, int parts)
{
    BArgs a;
    a.Q = Q; a.K = K; a.V = V; a.dO = dO;
    a.perm_q = perm_q; a.perm_k = perm_k; a.rs = rs;
    a.du_q = du_q; a.du_k = du_k; a.wt_hi = wt_hi; a.wt_lo = wt_lo; a.dv_lr = dv_lr;
    a.wk = race_wk(s);
    a.part_dq = part_dq; a.part_dk = part_dk; a.part_dv = part_dv;
    a.dQ = dQ; a.dK = dK; a.dV = dV;
    a.H = s.H; a.N = s.N; a.k = s.k; a.Lv = s.Lv;
    a.lt = s.lt;
    a.nbr = s.neighbors;
    a.BHN = (size_t)s.B * s.H * s.N;
    a.tau = s.tau; a.tau2 = s.tau * kLog2e;
    if (s.bf16) return s.D == 64 ? launch_t<BF16, 64>(s, a, st, parts) : launch_t<BF16, 128>(s, a, st, parts);
    return s.D == 64 ? launch_t<F32, 64>(s, a, st, parts) : launch_t<F32, 128>(s, a, st, parts);
}

}  // namespace elsaa
