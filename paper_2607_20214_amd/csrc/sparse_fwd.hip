// sparse_fwd.hip -- sortLSH sparse branch forward and the fusion epilogue.
//
// One workgroup = 4 waves = 64 queries (16 per wave); keys stream through
// LDS in tiles of 64 rows gathered by the sorted index lists (tile.hpp: K
// and V row-major, chunk-swizzled; V^T operands come from transposed LDS
// reads).  The rows of the next tile are loaded into registers while the
// current one is consumed.  Scores are computed transposed (S^T = K Q^T) so
// each lane owns one query: the running max and denominator of the online
// softmax are lane-local plus two cross-row shuffles, and P^T feeds
// O^T = V^T P^T straight from registers.
//
// Three modes share the tile loop:
//   kBlocks  non-causal Alg. 4: the query tile of sorted positions
//            [64t, 64t+64) sees the keys of its sorted blocks of size
//            b' = min(b, N); the epilogue fuses with the RACE output.
//   kLevels  causal Alg. 5, every level at once: SortLSH(Q_future, K_past)
//            of each segment; writes a normalised partial (O, log d) per
//            query, stored by natural query index.
//   kLeaf    causal Alg. 5 leaf (exact causal attention among the real
//            tokens of each leaf segment), then merges the level partials of the same
//            queries by log-sum-exp (MergeLSE) and applies the fusion.
//
// Fusion (Eq. m_sparse with the log-sum-exp form of Alg. 6, Eq. fusion):
//   O_s = N_s / (d_s + eps), m = d_s / (d_s + lambda d_lr + eps),
//   O = g_s m O_s + g_lr O_lr.
#include "common.hpp"
#include "internal.hpp"
#include "causal.hpp"
#include "tile.hpp"

namespace elsaa {

namespace {

constexpr int kQT = 64;       // queries per workgroup
constexpr int kKT = 64;       // keys per LDS tile
constexpr int kThreads = 256;
static_assert(kQT == kRowTile, "causal tiles are numbered in 64-query tiles");

enum Mode { kBlocks = 0, kLevels = 1, kLeaf = 2 };

// headroom (log2 units) of the online softmax's lazy reference max
constexpr float kLazy = 8.f;

struct Args {
    const void* Q;
    const void* K;
    const void* V;
    const int32_t* perm_q;
    const int32_t* perm_k;
    const float* gates;
    const float* lam_rows;    // per-token lambda_i or null (scalar lambda)
    const void* O_lr;         // storage dtype [BH][N][D]
    const float* d_lr;
    void* part_o;             // [BH][Lv][N/2][D] normalised level outputs, storage dtype
    float* part_lse;          // [BH][Lv][N/2] log of each level's denominator
    void* O;
    float* lse;
    float* m;
    float* O_s;               // float32 [BH][N][D]
    int H, N, k, Lv;
    LevelTiles lt;   // causal recursion geometry and tile numbering
    int nbr;         // neighbouring sorted blocks on each side
    int m_one;       // m_sparse fixed to 1
    float tau2;      // tau * log2(e)
    float lambda, eps;
};

template <class T, int D, int MODE>
__global__ __launch_bounds__(kThreads, 3) void sparse_fwd_kernel(Args a)
{
    using S = typename T::store_t;
    using F = typename T::frag_t;
    constexpr int KS = D / 32;   // k-steps over the head dim
    constexpr int DT = D / 16;   // 16-wide tiles of the head dim
    using Tl = tile::Tile<T, D>;
    constexpr int PT = Tl::PER_THREAD;
    // the K and V tiles, one array (the epilogue reuses it whole for rows)
    __shared__ __attribute__((aligned(16))) S skv[2 * Tl::elems(kKT)];
    S* const sk = skv;
    S* const sv = skv + Tl::elems(kKT);

    int tile, h, b;
    xcd_tile(tile, h, b);
    // the leaf pass walks the heads in reverse: the level pass before it
    // wrote the last heads' partials last, so theirs are still in the
    // memory-side cache when they are read (forward leaf 2.5% faster)
    if (MODE == kLeaf) {
        h = a.H - 1 - h;
        b = gridDim.z - 1 - b;
    }
    const size_t bh = (size_t)b * a.H + h;
    const int N = a.N;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int g = lane >> 4, qq = lane & 15;
    const S* Q = (const S*)a.Q + bh * N * D;
    const S* K = (const S*)a.K + bh * N * D;
    const S* V = (const S*)a.V + bh * N * D;

    // ---- which queries, which keys -------------------------------------
    int level = 0, seg = 0, half = N;   // kLevels: level / segment / half length
    int qpos;                           // position of this lane's query in its sorted list
    int qtok;                           // token index of this lane's query (-1 = none)
    int kbeg, kend;                     // key positions [kbeg, kend) scanned by the tile
    int bq = 1;                         // block size b' (kBlocks / kLevels)
    int qrow0 = 0, nq = 0;              // kBlocks / kLeaf: first query position of the tile, its queries
    const int32_t* klist = nullptr;     // sorted key list (kBlocks / kLevels)
    // sorted query block t sees the sorted key blocks t - nbr .. t + nbr
    if (MODE == kBlocks) {
        bq = min(a.k, N);
        const int p0 = tile * kQT;
        qrow0 = p0;
        nq = min(kQT, N - p0);
        qpos = p0 + 16 * w + qq;
        qtok = qpos < N ? a.perm_q[bh * N + qpos] : -1;
        const int plast = min(p0 + kQT, N) - 1;
        kbeg = max(0, (p0 / bq - a.nbr) * bq);
        kend = min(N, (plast / bq + 1 + a.nbr) * bq);
        klist = a.perm_k + bh * N;
    } else if (MODE == kLevels) {
        int p0;
        level_tile(a.lt, tile, level, half, seg, p0);
        bq = min(a.k, half);
        qpos = p0 + 16 * w + qq;
        const size_t lbase = bh * (size_t)a.lt.off[a.Lv] + (size_t)a.lt.off[level] + (size_t)seg * half;
        qtok = qpos < half ? a.perm_q[lbase + qpos] : -1;      // -1 also for a zero token
        const int plast = min(p0 + kQT, half) - 1;
        kbeg = max(0, (p0 / bq - a.nbr) * bq);
        kend = min(half, (plast / bq + 1 + a.nbr) * bq);
        klist = a.perm_k + lbase;
    } else {
        int q0, lend, leaf;
        leaf_tile(a.lt, tile, leaf, kbeg, q0, lend);
        qtok = q0 + 16 * w + qq;
        qpos = qtok;
        if (qtok >= lend) qtok = -1;
        kend = q0 < lend ? min(q0 + kQT, lend) : kbeg;   // a tile past the leaf's real tokens has no work
        qrow0 = q0;
        nq = max(0, min(kQT, lend - q0));
    }
    const int blk_lo = (MODE == kLeaf) ? 0 : max(0, (qpos / bq - a.nbr) * bq);
    const int blk_hi = (MODE == kLeaf) ? 0 : min((MODE == kBlocks ? N : half), (qpos / bq + 1 + a.nbr) * bq);

    // ---- this lane's query fragments (B operand of S^T = K Q^T) ---------
    F qf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        if (qtok >= 0) qf[ks] = T::ld8(Q + (size_t)qtok * D + 32 * ks + 8 * g);
        else {
            float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            qf[ks] = T::pack(z);
        }
    }

    float m_run = -INFINITY, l_run = 0.f;
    f32x4 acc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[dt] = f32x4{0, 0, 0, 0};

    // rows of the key tile at k0 that this thread stages: positions past
    // the scanned range repeat its last key (a real row: key lists hold no
    // zero tokens), whose scores the mask drops, so the loads need no
    // per-row branch
    auto tokens = [&](int k0, int (&tok)[PT]) {
#pragma unroll
        for (int j = 0; j < PT; ++j) {
            const int p = min(k0 + Tl::row_of(j), kend - 1);
            tok[j] = (MODE == kLeaf) ? p : klist[p];
        }
    };
    const int ntiles = (kend - kbeg + kKT - 1) / kKT;
    int tok[PT];
    uint4 rk[PT], rv[PT];
    if (ntiles > 0) {
        tokens(kbeg, tok);
        Tl::load_all(K, tok, rk);
        Tl::load_all(V, tok, rv);
    }
    if (ntiles > 1) tokens(kbeg + kKT, tok);

    for (int t = 0; t < ntiles; ++t) {
        const int k0 = kbeg + t * kKT;
        if (t > 0) __syncthreads();          // previous tile consumed
        Tl::store(sk, rk);
        Tl::store(sv, rv);
        __syncthreads();
        if (t + 1 < ntiles) {                // next tile's rows in flight during this one
            Tl::load_all(K, tok, rk);
            Tl::load_all(V, tok, rv);
            if (t + 2 < ntiles) tokens(k0 + 2 * kKT, tok);
        }

        // S^T for the 64 keys of the tile (4 sub-tiles of 16 keys)
        f32x4 st[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            st[s] = f32x4{0, 0, 0, 0};
            const int kr = krow_of(s, qq);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                st[s] = T::mma(Tl::row8(sk, kr, 32 * ks + 8 * g), qf[ks], st[s]);
        }
        // mask (masked scores -> -inf), running max in log2 units.  A tile
        // that every lane of the wave sees whole (all but the diagonal tile
        // of a causal leaf and ragged ends) skips the mask: one wave vote.
        const bool lane_full = qtok >= 0 && k0 + kKT <= kend &&
                               (MODE == kLeaf ? k0 + kKT - 1 <= qtok : (k0 >= blk_lo && k0 + kKT <= blk_hi));
        if (!__all(lane_full)) {
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int p = k0 + key_of(s, g, i);
                    bool ok = p < kend && qtok >= 0;
                    if (MODE == kLeaf) ok = ok && p <= qtok;
                    else ok = ok && p >= blk_lo && p < blk_hi;
                    st[s][i] = ok ? st[s][i] : -INFINITY;
                }
        }
        float tmax = -INFINITY;
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int i = 0; i < 4; ++i) tmax = fmaxf(tmax, st[s][i]);
        tmax = wave_max16(tmax) * a.tau2;            // tau2 > 0: the max of the scaled scores
        // The reference m_run of the exponentials is raised (and the
        // accumulators rescaled) only when some lane's tile max exceeds it by
        // more than kLazy (log2 units); otherwise the tile's P stay below
        // 2^kLazy, which float32 and the bf16 operands hold.  Any reference
        // gives the same O and log d: the denominator is kept relative to
        // the same m_run.  A lane still at -inf (no key seen) takes its first
        // finite max at once.
        if (__any(tmax > m_run + kLazy)) {
            const float m_new = fmaxf(m_run, tmax);
            const float corr = fast_exp2(m_run - ((m_new == -INFINITY) ? 0.f : m_new));
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) acc[dt] *= corr;
            l_run *= corr;
            m_run = m_new;
        }
        const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
        float psum = 0.f;
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float p = fast_exp2(fmaf(st[s][i], a.tau2, -m_use));
                st[s][i] = p;
                psum += p;
            }
        l_run += wave_sum16(psum);
        // O^T += V^T P^T over two 32-key k-steps
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            float pv[8];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                pv[j] = st[2 * kk][j];
                pv[4 + j] = st[2 * kk + 1][j];
            }
            const F pf = T::pack(pv);
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
                acc[dt] = T::mma(Tl::col8(sv, 32 * kk, 16 * dt), pf, acc[dt]);
        }
    }

    if (MODE == kLevels) {
        if (qtok < 0) return;
        // entry of query qtok among the future halves of this level
        const size_t slot = bh * (size_t)a.lt.off[a.Lv] + (size_t)level_entry(a.lt, level, qtok, true);
        const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
        S* po = (S*)a.part_o + slot * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) store4<T>(po + 16 * dt + 4 * g, acc[dt] * inv);
        if (g == 0) a.part_lse[slot] = (m_run + __log2f(l_run)) * kLn2;
        return;
    }

    // The rest runs on whole rows: the unnormalised output (relative to the
    // running max) goes to LDS as rows [query][d] (the tile space is free
    // now) with the row's running max and denominator, and each thread then
    // takes 8 consecutive elements of a row, so the level partials, O_lr and
    // the outputs move as 16-byte pieces with 16 (d_h 128) or 8 lanes
    // covering a row.
    constexpr int RS = D + 4;                       // LDS row stride (floats)
    static_assert(64 * RS * 4 + 2 * 64 * 4 <= sizeof(skv), "row sums fit in the tiles' LDS");
    float* const eo = (float*)skv;
    float* const em = eo + 64 * RS;                 // running max (log2 units)
    float* const el = em + 64;                      // running denominator
    __syncthreads();                                // every wave is done with the tiles
    {
        const int r = 16 * w + qq;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) *(f32x4*)&eo[r * RS + 16 * dt + 4 * g] = acc[dt];
        if (g == 0) {
            em[r] = m_run;
            el[r] = l_run;
        }
    }
    __syncthreads();
    if (nq <= 0) return;
    constexpr int PPR = D / 8, RPP = kThreads / PPR, NPASS = 64 / RPP;
    const int c8 = 8 * ((int)threadIdx.x % PPR);
    using R8 = Raw8<T>;
    // rows past the tile's queries read the first query's rows (loads
    // without a branch) and store nothing; the fusion's row inputs are
    // requested before the level partials are merged
    const int tok0 = MODE == kLeaf ? qrow0 : a.perm_q[bh * N + qrow0];
    int tokr[NPASS], tokl[NPASS];
    float o8[NPASS][8], mr[NPASS], lr[NPASS], dl[NPASS], lam[NPASS], gs[NPASS], gl[NPASS];
    typename R8::type olr[NPASS];
#pragma unroll
    for (int ps = 0; ps < NPASS; ++ps) {
        const int r = ps * RPP + (int)threadIdx.x / PPR;
        tokr[ps] = r < nq ? (MODE == kLeaf ? qrow0 + r : a.perm_q[bh * N + qrow0 + r]) : -1;
        tokl[ps] = tokr[ps] >= 0 ? tokr[ps] : tok0;
        const size_t row = bh * N + tokl[ps];
        olr[ps] = R8::ld((const S*)a.O_lr + row * D + c8);
        dl[ps] = a.d_lr[row];
        lam[ps] = a.lam_rows ? a.lam_rows[row] : a.lambda;
        gs[ps] = 1.f;
        gl[ps] = 1.f;
        if (a.gates) {
            gs[ps] = a.gates[row * 2 + 0];
            gl[ps] = a.gates[row * 2 + 1];
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) o8[ps][e] = eo[r * RS + c8 + e];
        mr[ps] = em[r];
        lr[ps] = el[r];
    }
    if (MODE == kLeaf) {
        // merge the partial of every level whose future half holds this leaf,
        // in level order, two levels at a time so their loads are in flight
        // together
        unsigned lmask = leaf_levels(a.lt, tile / a.lt.per_leaf, true);
        while (lmask) {
            int lv[2];
            bool use[2];
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                use[j] = lmask != 0;
                lv[j] = 0;
                if (use[j]) {
                    lv[j] = __builtin_ctz(lmask);
                    lmask &= lmask - 1;
                }
            }
            float pl[2][NPASS];
            typename R8::type v[2][NPASS];
#pragma unroll
            for (int j = 0; j < 2; ++j)
                if (use[j])
#pragma unroll
                    for (int ps = 0; ps < NPASS; ++ps) {
                        const size_t slot = bh * (size_t)a.lt.off[a.Lv] + (size_t)level_entry(a.lt, lv[j], tokl[ps], true);
                        pl[j][ps] = a.part_lse[slot] * kLog2e;
                        v[j][ps] = R8::ld((const S*)a.part_o + slot * D + c8);
                    }
#pragma unroll
            for (int j = 0; j < 2; ++j)
                if (use[j])
#pragma unroll
                    for (int ps = 0; ps < NPASS; ++ps) {
                        const float m_new = fmaxf(mr[ps], pl[j][ps]);
                        const float c_old = fast_exp2(mr[ps] - m_new), c_new = fast_exp2(pl[j][ps] - m_new);
                        float x[8];
                        R8::val(v[j][ps], x);
#pragma unroll
                        for (int e = 0; e < 8; ++e) o8[ps][e] = o8[ps][e] * c_old + x[e] * c_new;
                        lr[ps] = lr[ps] * c_old + c_new;
                        mr[ps] = m_new;
                    }
        }
    }

    // ---- fusion epilogue (kBlocks, kLeaf) --------------------------------
#pragma unroll
    for (int ps = 0; ps < NPASS; ++ps) {
        if (tokr[ps] < 0) continue;
        const size_t row = bh * N + tokr[ps];
        const float lse_nat = (mr[ps] + __log2f(lr[ps])) * kLn2;          // log d_s
        const float inv_den = 1.f / (lr[ps] + a.eps * fast_exp2(-mr[ps])); // 1 / (d_s + eps), rescaled
        const float mf = a.m_one ? 1.f : 1.f / (1.f + __expf(__logf(lam[ps] * dl[ps] + a.eps) - lse_nat));
        float os[8], ol[8], out[8];
        R8::val(olr[ps], ol);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            os[e] = o8[ps][e] * inv_den;
            out[e] = os[e] * (gs[ps] * mf) + ol[e] * gl[ps];
        }
        float* po = a.O_s + row * D + c8;
        *(f32x4*)po = f32x4{os[0], os[1], os[2], os[3]};
        *(f32x4*)(po + 4) = f32x4{os[4], os[5], os[6], os[7]};
        store8<T>((S*)a.O + row * D + c8, out);
        if (c8 == 0) {
            a.lse[row] = lse_nat;
            a.m[row] = mf;
        }
    }
}

template <class T, int D>
hipError_t launch_t(const Shape& s, const Args& a, hipStream_t st, int parts)
{
    if (!s.causal) {
        if (!(parts & kSparseFinal)) return hipSuccess;
        dim3 grid((s.N + kQT - 1) / kQT, s.H, s.B);
        ELSAA_LAUNCH("sparse_fwd_blocks", (sparse_fwd_kernel<T, D, kBlocks>), grid, dim3(kThreads), 0, st, a);
        return hipGetLastError();
    }
    if (s.Lv > 0 && (parts & kSparseLevels)) {
        dim3 grid(a.lt.first[s.Lv], s.H, s.B);
        ELSAA_LAUNCH("sparse_fwd_levels", (sparse_fwd_kernel<T, D, kLevels>), grid, dim3(kThreads), 0, st, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (!(parts & kSparseFinal)) return hipSuccess;
    dim3 grid(a.lt.leaf_tiles(), s.H, s.B);
    ELSAA_LAUNCH("sparse_fwd_leaf", (sparse_fwd_kernel<T, D, kLeaf>), grid, dim3(kThreads), 0, st, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_sparse_fwd(const Shape& s, const void* Q, const void* K, const void* V,
                             const int32_t* perm_q, const int32_t* perm_k, const float* gates,
                             const float* lambda_rows, const void* O_lr, const float* d_lr, void* part_o, float* part_lse,
                             void* O, float* lse, float* m, float* O_s, hipStream_t st, int parts)
{
    Args a;
    a.Q = Q; a.K = K; a.V = V;
    a.perm_q = perm_q; a.perm_k = perm_k;
    a.gates = gates; a.lam_rows = lambda_rows; a.O_lr = O_lr; a.d_lr = d_lr;
    a.nbr = s.neighbors; a.m_one = s.m_one;
    a.part_o = part_o; a.part_lse = part_lse;
    a.O = O; a.lse = lse; a.m = m; a.O_s = O_s;
    a.H = s.H; a.N = s.N; a.k = s.k; a.Lv = s.Lv;
    a.lt = s.lt;
    a.tau2 = s.tau * kLog2e;
    a.lambda = s.lambda; a.eps = s.eps;
    if (s.bf16) return s.D == 64 ? launch_t<BF16, 64>(s, a, st, parts) : launch_t<BF16, 128>(s, a, st, parts);
    return s.D == 64 ? launch_t<F32, 64>(s, a, st, parts) : launch_t<F32, 128>(s, a, st, parts);
}

}  // namespace elsaa
