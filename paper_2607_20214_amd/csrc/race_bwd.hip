// race_bwd.hip -- backward of the RACE low-rank branch (Alg. 2 / Alg. 3 differentiated).
//
// With dNum_i = g_lr dO_i / (Den_i + eps) and dDen_i (row scalars of the
// backward preprocess), and V~_j = [V_j, 1], dN~_i = [dNum_i, dDen_i]:
//   dphi(q_i) = (1/L) sum_{j <= i} <dN~_i, V~_j> phi(k_j)          (kernel LB1, forward time)
//   dphi(k_j) = (1/L) sum_{i >= j} <dN~_i, V~_j> phi(q_i)          (kernel LB2, reverse time)
//   dV_j      = (1/L) sum_{i >= j} <phi(q_i), phi(k_j)> dNum_i      (kernel LB3, reverse time)
// (non-causal: all i, j).  Each is a linear-attention pass over 64-token
// chunks with a running state: LB1 reads S = sum phi(k) V', A = sum phi(k)
// (the forward's segment prefix states); LB2 and LB3 read the suffix states
// dS = (1/L) sum phi(q) dNum', dA = (1/L) sum phi(q) dDen.  LB1 and LB2
// contract their state over d, so each wave owns a quarter of the features;
// LB3 contracts over the features, so each wave owns a quarter of d.
// dphi is chained through phi = prod sigmoid(2 beta v t), t = tanh(W x) to
// du, the gradient of the projections u = W x.  LB1 and LB2 store du (storage
// dtype, [BH][N][wk], wk = 4L padded to 32) and the sparse backward forms
// dQ (dK) += du W on MFMA where it adds its own part, so only wk values per
// row cross HBM instead of d float32 ones; this pass provides W' = W_hi' +
// W_lo' ([H][D][wk], bf16 parts of float32 accuracy).  The running states
// enter the MFMAs split the same way: their products cancel against the dDen
// terms.  LB3 writes dV in the storage dtype [BH][N][D]; the sparse backward
// adds it to its float32 dV before the final rounding.
#include "internal.hpp"
#include "race_common.hpp"

namespace elsaa {

using namespace race;

namespace {

struct LbArgs {
    const float* Uq;        // projections of Q rows [BH][N][RP/4]
    const float* Uk;        // projections of K rows
    const void* V;
    const void* dO;
    const float* rs;        // row scalars (sc_lr at 3*BHN, dDen at 4*BHN)
    const float* states;    // LB1: forward prefix states; LB2/LB3: backward suffix states
    void* out;              // LB1 / LB2: du rows [BH][N][wk]; LB3: dV rows [BH][N][D] (storage dtype)
    int H, N, L, seg_len, nseg, causal;
    size_t BHN;
    float two_beta, beta, inv_L;
};

template <class T, int D, int RP>
struct Lb1Smem {
    using S = typename T::store_t;
    S vt[D][kC + kPad];            // V chunk transposed
    S dn[kC][D + kPad];            // dO chunk, rows (dNum_i = sc_lr,i dO_i: the products apply sc_lr)
    S pk[kC][RP + kPad];           // Phi_K chunk, rows (Phi_K^T operands: transposed LDS reads)
    S gg[kC][kC + kPad];           // G[i][j] = <dNum_i, V_j> + dDen_i, j <= i
    float ts[kC][RP / 4];          // tanh(W q) of the chunk's queries
    S du[kC][w_kdim<RP>() + kPad];
    float dden[kC];
    float sc[kC];                  // sc_lr of the chunk's queries
};

template <class T, int D, int RP>
struct Lb2Smem {
    using S = typename T::store_t;
    S vr[kC][D + kPad];            // V chunk, rows
    S dnt[D][kC + kPad];           // dNum / L chunk, transposed
    S pqt[RP][kC + kPad];          // Phi_Q transposed
    S ggt[kC][kC + kPad];          // G'[j][i] / L, i >= j
    float ts[kC][RP / 4];          // tanh(W k) of the chunk's keys
    S du[kC][w_kdim<RP>() + kPad];
    float dden[kC];
    float a_state[RP];             // dA = (1/L) sum phi(q) dDen of the queries after the chunk
};

template <class T, int D, int RP>
struct Lb3Smem {
    using S = typename T::store_t;
    S dnt[D][kC + kPad];           // dNum / L chunk, transposed
    S pk[kC][RP + kPad];           // Phi_K rows
    S pq[kC][RP + kPad];           // Phi_Q rows (Phi_Q^T operands: transposed LDS reads)
    S mt[kC][kC + kPad];           // M'[j][i] = <phi(k_j), phi(q_i)>, i >= j
};

template <class T, int D, int RP>
constexpr bool bwd_fits()
{
    return sizeof(Lb1Smem<T, D, RP / table_split<RP>()>) <= kMaxLds &&
           sizeof(Lb2Smem<T, D, RP / table_split<RP>()>) <= kMaxLds &&
           sizeof(Lb3Smem<T, D, RP>) <= kMaxLds;
}

// du rows [t0, t0 + 64) of the chunk (LDS, storage dtype) -> rows of out
// [N][WK], 16 bytes per thread and store.
template <class T, int RPW, int RP>
__device__ __forceinline__ void store_du(const typename T::store_t (*du)[w_kdim<RPW>() + kPad],
                                         typename T::store_t* out, int t0, int N)
{
    // a workgroup holding all the features writes whole (padded) rows,
    // one holding some of the tables their RPW / 4 columns
    constexpr int WK = w_kdim<RP>(), COLS = RPW == RP ? WK : RPW / 4;
    constexpr int PER = 16 / T::bytes, CH = COLS / PER;
    static_assert(COLS % PER == 0, "du row of whole 16-byte pieces");
    for (int it = threadIdx.x; it < kC * CH; it += kThreads) {
        const int r = it / CH, c = it % CH;
        if (t0 + r < N) stg16(out + (size_t)(t0 + r) * WK + c * PER, *(const uint4*)&du[r][c * PER]);
    }
}

// W' = W_hi' + W_lo' of every head, [H][D][WK] (rows 4l + b, zero past 4L).
template <class T>
__global__ __launch_bounds__(256) void race_wt_kernel(const float* W, typename T::store_t* hi,
                                                      typename T::store_t* lo, int L, int D, int WK)
{
    const int h = blockIdx.y;
    const int it = blockIdx.x * 256 + threadIdx.x;
    if (it >= D * WK) return;
    const int d = it / WK, p = it % WK;
    const float w = p < 4 * L ? W[((size_t)h * 4 * L + p) * D + d] : 0.f;
    const typename T::store_t vh = T::store(w);
    hi[((size_t)h * D + d) * WK + p] = vh;
    lo[((size_t)h * D + d) * WK + p] = T::store(T::kSplit ? w - T::load(vh) : 0.f);
}

// ---------------------------------------------------------------- LB1: dQ
template <class T, int D, int RP>
__global__ __launch_bounds__(kThreads, 2) void race_dq_kernel(LbArgs a)
{
    using St = typename T::store_t;
    using F = typename T::frag_t;
    constexpr int SPLIT = table_split<RP>(), RPW = RP / SPLIT;   // features of this workgroup
    constexpr int DT = D / 16, KS = D / 32, FT = RPW / 16, NFT = (FT + 3) / 4;
    __shared__ Lb1Smem<T, D, RPW> sm;
    const int seg = blockIdx.x / SPLIT, part = blockIdx.x % SPLIT, h = blockIdx.y, b = blockIdx.z;
    const int F0 = part * RPW, L = a.L - F0 / 16;                  // first feature; tables from here on
    const size_t bh = (size_t)b * a.H + h;
    const float* Uq = a.Uq + bh * a.N * (RP / 4) + F0 / 4;
    const float* Uk = a.Uk + bh * a.N * (RP / 4) + F0 / 4;
    const St* V = (const St*)a.V + bh * a.N * D;
    const St* dO = (const St*)a.dO + bh * a.N * D;
    const float* sclr = a.rs + 3 * a.BHN + bh * a.N;
    const float* dden = a.rs + 4 * a.BHN + bh * a.N;
    St* du_out = (St*)a.out + bh * a.N * w_kdim<RP>() + F0 / 4;
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int g = lane >> 4, col = lane & 15;

    for (int it = threadIdx.x; it < kC * (w_kdim<RPW>() + kPad); it += kThreads)
        (&sm.du[0][0])[it] = T::store(0.f);
    // state S'[d][f] for the wave's features f = 16 (w + 4j) + col, and
    // A[f] of the same feature tiles (lane (g, col) register i: feature
    // 16 (w + 4j) + 4 g + i, every column alike; token_sums keeps it so)
    f32x4 St_[NFT][DT], Aacc[NFT];
    const float* st_in = a.states + (bh * a.nseg + seg) * (size_t)(RP * D + RP);
#pragma unroll
    for (int j = 0; j < NFT; ++j) {
        const int ft = w + 4 * j;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                St_[j][dt][i] = ft < FT ? st_in[(size_t)(F0 + 16 * ft + col) * D + 16 * dt + 4 * g + i] : 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) Aacc[j][i] = ft < FT ? st_in[RP * D + F0 + 16 * ft + 4 * g + i] : 0.f;
    }

    const int t_beg = seg * a.seg_len, t_end = min(a.N, t_beg + a.seg_len);
    URegs<RPW> uq, uk;                    // projections of the chunk, loaded one chunk ahead
    uq.load(Uq, t_beg, a.N, RP / 4);
    if (a.causal) uk.load(Uk, t_beg, a.N, RP / 4);
    for (int t0 = t_beg; t0 < t_end; t0 += kC) {
        __syncthreads();
        // every global load of the chunk is issued first; the features (vector
        // work) run while they are in flight, then the rows go to LDS
        StageR<T, D> sdn;
        sdn.load(dO, t0, a.N, nullptr);
        StageT<T, D> svt;
        if (a.causal) svt.load(V, t0, a.N, nullptr, 1.f);
        const bool in = threadIdx.x < kC && t0 + (int)threadIdx.x < a.N;
        const float ddv = in ? dden[t0 + threadIdx.x] : 0.f, scv = in ? sclr[t0 + threadIdx.x] : 0.f;
        features_from<T, RPW>(uq, t0, a.N, L, a.two_beta, nullptr, nullptr, sm.ts);
        if (a.causal) features_from<T, RPW>(uk, t0, a.N, L, a.two_beta, sm.pk, nullptr, nullptr);
        sdn.store(sm.dn, false);
        if (a.causal) svt.store(sm.vt, false);
        if (threadIdx.x < kC) {
            sm.dden[threadIdx.x] = ddv;
            sm.sc[threadIdx.x] = scv;
        }
        __syncthreads();
        {
            // next chunk's projections (the last chunk reloads its own, so
            // the loads are unconditional)
            const int tn = t0 + kC < t_end ? t0 + kC : t0;
            uq.load(Uq, tn, a.N, RP / 4);
            if (a.causal) uk.load(Uk, tn, a.N, RP / 4);
        }
        if (a.causal) {
            // G rows [16w, 16w + 16): sc_lr,i <dO_i, V_j> + dDen_i for j <= i,
            // formed transposed (lane (g, col): keys 16 kt + 4 g + i of query
            // 16 w + col) so each lane stores four entries of its row at once
            const int qi = 16 * w + col;
            const float scq = sm.sc[qi], ddq = sm.dden[qi];
            for (int kt = 0; kt < 4; ++kt) {
                f32x4 acc = {0, 0, 0, 0};
                if (kt <= w) {
                    // V rows of keys 16 kt .. 16 kt + 15 from the transposed chunk tile
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks)
                        acc = T::mma(col8_t<T, kC + kPad>(sm.vt, 32 * ks, 16 * kt),
                                     T::ld8(&sm.dn[16 * w + col][32 * ks + 8 * g]), acc);
                }
                f32x4 v;
#pragma unroll
                for (int i = 0; i < 4; ++i) v[i] = 16 * kt + 4 * g + i <= qi ? acc[i] * scq + ddq : 0.f;
                store4<T>(&sm.gg[qi][16 * kt + 4 * g], v);
            }
        }
        __syncthreads();
        // dphi(q)' tiles [features of table ft] x [16 queries]: sc_lr S dO + A dDen + intra
        // (the state's hi / lo bf16 split is made once per chunk and k-step)
#pragma unroll
        for (int j = 0; j < NFT; ++j) {
            const int ft = w + 4 * j;
            if (ft >= FT) break;
            f32x4 acc[4];
#pragma unroll
            for (int qt = 0; qt < 4; ++qt) acc[qt] = f32x4{0, 0, 0, 0};
#pragma unroll
            for (int ds = 0; ds < KS; ++ds) {
                float sv[8];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    sv[i] = St_[j][2 * ds][i];
                    sv[4 + i] = St_[j][2 * ds + 1][i];
                }
                F shi, slo;
                T::split(sv, shi, slo);
#pragma unroll
                for (int qt = 0; qt < 4; ++qt) {
                    const F bf = T::ld44(&sm.dn[16 * qt + col][32 * ds + 4 * g],
                                         &sm.dn[16 * qt + col][32 * ds + 16 + 4 * g]);
                    acc[qt] = T::mma(shi, bf, acc[qt]);
                    if (T::kSplit) acc[qt] = T::mma(slo, bf, acc[qt]);
                }
            }
            for (int qt = 0; qt < 4; ++qt) {
                const float ddq = sm.dden[16 * qt + col], scq = sm.sc[16 * qt + col];
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[qt][i] = acc[qt][i] * scq + Aacc[j][i] * ddq;
                if (a.causal) {
#pragma unroll
                    for (int kk = 0; kk < 2; ++kk)
                        acc[qt] = T::mma(phi_t8<T, RPW>(sm.pk, 32 * kk, 16 * ft),
                                         T::ld8(&sm.gg[16 * qt + col][32 * kk + 8 * g]), acc[qt]);
                }
                acc[qt] *= a.inv_L;
                chain_rule_t<T, RPW>(acc[qt], qt, ft, L, a.beta, sm.ts, sm.du);
            }
        }
        __syncthreads();
        store_du<T, RPW, RP>(sm.du, du_out, t0, a.N);
        if (a.causal) {
            // S' += V' Phi_K (chunk), A += Phi_K' 1 (one Phi_K^T fragment each)
#pragma unroll
            for (int j = 0; j < NFT; ++j) {
                const int ft = w + 4 * j;
                if (ft >= FT) break;
#pragma unroll
                for (int kk = 0; kk < 2; ++kk) {
                    const F bf = phi_t8<T, RPW>(sm.pk, 32 * kk, 16 * ft);
#pragma unroll
                    for (int dt = 0; dt < DT; ++dt)
                        St_[j][dt] = T::mma(T::ld8(&sm.vt[16 * dt + col][32 * kk + 8 * g]), bf, St_[j][dt]);
                    Aacc[j] = token_sums<T>(bf, Aacc[j]);
                }
            }
        }
    }
}

// ---------------------------------------------------------------- LB2: dK
template <class T, int D, int RP>
__global__ __launch_bounds__(kThreads, 2) void race_dk_kernel(LbArgs a)
{
    using St = typename T::store_t;
    using F = typename T::frag_t;
    constexpr int SPLIT = table_split<RP>(), RPW = RP / SPLIT;   // features of this workgroup
    constexpr int DT = D / 16, KS = D / 32, FT = RPW / 16, NFT = (FT + 3) / 4;
    __shared__ Lb2Smem<T, D, RPW> sm;
    const int seg = blockIdx.x / SPLIT, part = blockIdx.x % SPLIT, h = blockIdx.y, b = blockIdx.z;
    const int F0 = part * RPW, L = a.L - F0 / 16;                  // first feature; tables from here on
    const size_t bh = (size_t)b * a.H + h;
    const float* Uq = a.Uq + bh * a.N * (RP / 4) + F0 / 4;
    const float* Uk = a.Uk + bh * a.N * (RP / 4) + F0 / 4;
    const St* V = (const St*)a.V + bh * a.N * D;
    const St* dO = (const St*)a.dO + bh * a.N * D;
    const float* sclr = a.rs + 3 * a.BHN + bh * a.N;
    const float* dden = a.rs + 4 * a.BHN + bh * a.N;
    St* du_out = (St*)a.out + bh * a.N * w_kdim<RP>() + F0 / 4;
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int g = lane >> 4, col = lane & 15;

    for (int it = threadIdx.x; it < kC * (w_kdim<RPW>() + kPad); it += kThreads)
        (&sm.du[0][0])[it] = T::store(0.f);
    f32x4 St_[NFT][DT];
    const float* st_in = a.states + (bh * a.nseg + seg) * (size_t)(RP * D + RP);
    for (int f = threadIdx.x; f < RPW; f += kThreads) sm.a_state[f] = st_in[RP * D + F0 + f];
#pragma unroll
    for (int j = 0; j < NFT; ++j) {
        const int ft = w + 4 * j;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                St_[j][dt][i] = ft < FT ? st_in[(size_t)(F0 + 16 * ft + col) * D + 16 * dt + 4 * g + i] : 0.f;
    }

    const int t_beg = seg * a.seg_len, t_end = min(a.N, t_beg + a.seg_len);
    const int nch = (t_end - t_beg + kC - 1) / kC;
    URegs<RPW> uq, uk;                    // projections of the chunk, loaded one chunk ahead
    uk.load(Uk, t_beg + (nch - 1) * kC, a.N, RP / 4);
    if (a.causal) uq.load(Uq, t_beg + (nch - 1) * kC, a.N, RP / 4);
    for (int c = nch - 1; c >= 0; --c) {
        const int t0 = t_beg + c * kC;
        __syncthreads();
        // loads first, features under them, then the LDS stores
        StageR<T, D> svr;
        svr.load(V, t0, a.N, nullptr);
        StageT<T, D> sdn;
        if (a.causal) sdn.load(dO, t0, a.N, sclr, a.inv_L);
        const bool in = threadIdx.x < kC && t0 + (int)threadIdx.x < a.N;
        const float ddv = in ? dden[t0 + threadIdx.x] : 0.f;
        features_from<T, RPW>(uk, t0, a.N, L, a.two_beta, nullptr, nullptr, sm.ts);
        if (a.causal) features_from<T, RPW>(uq, t0, a.N, L, a.two_beta, nullptr, sm.pqt, nullptr);
        svr.store(sm.vr, false);
        if (a.causal) sdn.store(sm.dnt, true);
        if (threadIdx.x < kC) sm.dden[threadIdx.x] = ddv;
        __syncthreads();
        {
            // previous chunk's projections (unconditional: chunk 0 reloads its own)
            const int tn = c > 0 ? t0 - kC : t0;
            uk.load(Uk, tn, a.N, RP / 4);
            if (a.causal) uq.load(Uq, tn, a.N, RP / 4);
        }
        if (a.causal) {
            // G' rows j in [16w, 16w + 16): (<V_j, dNum_i> + dDen_i) / L for
            // i >= j, formed transposed (lane (g, col): queries 16 it + 4 g + i
            // of key 16 w + col) so each lane stores four entries of its row at once
            const int kj = 16 * w + col;
            for (int it = 0; it < 4; ++it) {
                f32x4 acc = {0, 0, 0, 0};
                if (it >= w) {
                    // dNum / L rows of queries 16 it .. 16 it + 15 from the transposed chunk tile
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks)
                        acc = T::mma(col8_t<T, kC + kPad>(sm.dnt, 32 * ks, 16 * it),
                                     T::ld8(&sm.vr[16 * w + col][32 * ks + 8 * g]), acc);
                }
                const f32x4 dd = *(const f32x4*)&sm.dden[16 * it + 4 * g];
                f32x4 v;
#pragma unroll
                for (int i = 0; i < 4; ++i) v[i] = 16 * it + 4 * g + i >= kj ? acc[i] + dd[i] * a.inv_L : 0.f;
                store4<T>(&sm.ggt[kj][16 * it + 4 * g], v);
            }
        }
        __syncthreads();
        // dphi(k)' tiles [features of table ft] x [16 keys]: dS V + dA + intra
        // (the state's hi / lo bf16 split is made once per chunk and k-step)
#pragma unroll
        for (int j = 0; j < NFT; ++j) {
            const int ft = w + 4 * j;
            if (ft >= FT) break;
            f32x4 acc[4];
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) acc[kt] = f32x4{0, 0, 0, 0};
#pragma unroll
            for (int ds = 0; ds < KS; ++ds) {
                float sv[8];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    sv[i] = St_[j][2 * ds][i];
                    sv[4 + i] = St_[j][2 * ds + 1][i];
                }
                F shi, slo;
                T::split(sv, shi, slo);
#pragma unroll
                for (int kt = 0; kt < 4; ++kt) {
                    const F bf = T::ld44(&sm.vr[16 * kt + col][32 * ds + 4 * g],
                                         &sm.vr[16 * kt + col][32 * ds + 16 + 4 * g]);
                    acc[kt] = T::mma(shi, bf, acc[kt]);
                    if (T::kSplit) acc[kt] = T::mma(slo, bf, acc[kt]);
                }
            }
            for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[kt][i] += sm.a_state[16 * ft + 4 * g + i];
                if (a.causal) {
#pragma unroll
                    for (int kk = 0; kk < 2; ++kk)
                        acc[kt] = T::mma(T::ld8(&sm.pqt[16 * ft + col][32 * kk + 8 * g]),
                                         T::ld8(&sm.ggt[16 * kt + col][32 * kk + 8 * g]), acc[kt]);
                }
                chain_rule_t<T, RPW>(acc[kt], kt, ft, L, a.beta, sm.ts, sm.du);
            }
        }
        __syncthreads();
        store_du<T, RPW, RP>(sm.du, du_out, t0, a.N);
        if (a.causal) {
            // dS' += (dNum / L)' Phi_Q (chunk), dA += (1/L) Phi_Q' dDen
#pragma unroll
            for (int j = 0; j < NFT; ++j) {
                const int ft = w + 4 * j;
                if (ft >= FT) break;
#pragma unroll
                for (int kk = 0; kk < 2; ++kk) {
                    const F bf = T::ld8(&sm.pqt[16 * ft + col][32 * kk + 8 * g]);
#pragma unroll
                    for (int dt = 0; dt < DT; ++dt)
                        St_[j][dt] = T::mma(T::ld8(&sm.dnt[16 * dt + col][32 * kk + 8 * g]), bf, St_[j][dt]);
                }
            }
            add_chunk_sums<T, RPW>(sm.pqt, sm.dden, a.inv_L, sm.a_state);
        }
    }
}

// ---------------------------------------------------------------- LB3: dV
template <class T, int D, int RP>
__global__ __launch_bounds__(kThreads, 2) void race_dv_kernel(LbArgs a)
{
    using St = typename T::store_t;
    using F = typename T::frag_t;
    constexpr int DW = D / 64, FS = RP / 32;
    __shared__ Lb3Smem<T, D, RP> sm;
    const int seg = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const size_t bh = (size_t)b * a.H + h;
    const float* Uq = a.Uq + bh * a.N * (RP / 4);
    const float* Uk = a.Uk + bh * a.N * (RP / 4);
    const St* dO = (const St*)a.dO + bh * a.N * D;
    const float* sclr = a.rs + 3 * a.BHN + bh * a.N;
    St* out = (St*)a.out + bh * a.N * D;
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int g = lane >> 4, col = lane & 15;

    const float* st_in = a.states + (bh * a.nseg + seg) * (size_t)(RP * D + RP);
    f32x4 S[RP / 16][DW];
#pragma unroll
    for (int ft = 0; ft < RP / 16; ++ft)
#pragma unroll
        for (int j = 0; j < DW; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                S[ft][j][i] = st_in[(size_t)(16 * ft + 4 * g + i) * D + 16 * (w * DW + j) + col];

    const int t_beg = seg * a.seg_len, t_end = min(a.N, t_beg + a.seg_len);
    const int nch = (t_end - t_beg + kC - 1) / kC;
    URegs<RP> uq, uk;                    // projections of the chunk, loaded one chunk ahead
    uk.load(Uk, t_beg + (nch - 1) * kC, a.N, RP / 4);
    if (a.causal) uq.load(Uq, t_beg + (nch - 1) * kC, a.N, RP / 4);
    for (int c = nch - 1; c >= 0; --c) {
        const int t0 = t_beg + c * kC;
        __syncthreads();
        // loads first, features under them, then the LDS stores
        StageT<T, D> sdn;
        if (a.causal) sdn.load(dO, t0, a.N, sclr, a.inv_L);
        features_from<T, RP>(uk, t0, a.N, a.L, a.two_beta, sm.pk, nullptr, nullptr);
        if (a.causal) {
            features_from<T, RP>(uq, t0, a.N, a.L, a.two_beta, sm.pq, nullptr, nullptr);
            sdn.store(sm.dnt, true);
        }
        __syncthreads();
        {
            // previous chunk's projections (unconditional: chunk 0 reloads its own)
            const int tn = c > 0 ? t0 - kC : t0;
            uk.load(Uk, tn, a.N, RP / 4);
            if (a.causal) uq.load(Uq, tn, a.N, RP / 4);
        }
        if (a.causal) {
            // M' rows j in [16w, 16w + 16): <phi(k_j), phi(q_i)> for i >= j,
            // formed transposed (lane (g, col): queries 16 it + 4 g + i of key
            // 16 w + col) so each lane stores four entries of its row at once
            const int kj = 16 * w + col;
            for (int it = 0; it < 4; ++it) {
                f32x4 acc = {0, 0, 0, 0};
                if (it >= w) {
#pragma unroll
                    for (int fs = 0; fs < FS; ++fs)
                        acc = T::mma(T::ld8(&sm.pq[16 * it + col][32 * fs + 8 * g]),
                                     T::ld8(&sm.pk[16 * w + col][32 * fs + 8 * g]), acc);
                }
                f32x4 v;
#pragma unroll
                for (int i = 0; i < 4; ++i) v[i] = 16 * it + 4 * g + i >= kj ? acc[i] : 0.f;
                store4<T>(&sm.mt[kj][16 * it + 4 * g], v);
            }
        }
        __syncthreads();
        f32x4 accs[4][DW];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
            for (int j = 0; j < DW; ++j) accs[kt][j] = f32x4{0, 0, 0, 0};
#pragma unroll
        for (int fs = 0; fs < FS; ++fs) {
            F shi[DW], slo[DW];
#pragma unroll
            for (int j = 0; j < DW; ++j) {
                float sv[8];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    sv[i] = S[2 * fs][j][i];
                    sv[4 + i] = S[2 * fs + 1][j][i];
                }
                T::split(sv, shi[j], slo[j]);
            }
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) {
                const F bf = T::ld44(&sm.pk[16 * kt + col][32 * fs + 4 * g], &sm.pk[16 * kt + col][32 * fs + 16 + 4 * g]);
#pragma unroll
                for (int j = 0; j < DW; ++j) {
                    accs[kt][j] = T::mma(shi[j], bf, accs[kt][j]);
                    if (T::kSplit) accs[kt][j] = T::mma(slo[j], bf, accs[kt][j]);
                }
            }
        }
        // dV^T: lane (g, col) holds d = 16 (w DW + j) + 4 g + i of key 16 kt + col
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
            f32x4 (&acc)[DW] = accs[kt];
            if (a.causal) {
#pragma unroll
                for (int kk = 0; kk < 2; ++kk) {
                    const F bf = T::ld8(&sm.mt[16 * kt + col][32 * kk + 8 * g]);
#pragma unroll
                    for (int j = 0; j < DW; ++j)
                        acc[j] = T::mma(T::ld8(&sm.dnt[16 * (w * DW + j) + col][32 * kk + 8 * g]), bf, acc[j]);
                }
            }
            const int tok = t0 + 16 * kt + col;
            if (tok < a.N)
#pragma unroll
                for (int j = 0; j < DW; ++j) store4<T>(out + (size_t)tok * D + 16 * (w * DW + j) + 4 * g, acc[j]);
        }
        if (a.causal) {
            // dS += Phi_Q' (dNum / L) (chunk)
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                F bv[DW];
#pragma unroll
                for (int j = 0; j < DW; ++j) bv[j] = T::ld8(&sm.dnt[16 * (w * DW + j) + col][32 * kk + 8 * g]);
#pragma unroll
                for (int ft = 0; ft < RP / 16; ++ft) {
                    const F af = phi_t8<T, RP>(sm.pq, 32 * kk, 16 * ft);
#pragma unroll
                    for (int j = 0; j < DW; ++j) S[ft][j] = T::mma(af, bv[j], S[ft][j]);
                }
            }
        }
    }
}

template <class T, int D, int RP>
struct BwdFn {
    static hipError_t run(const Shape& s, const LbArgs& a1, const LbArgs& a2, const LbArgs& a3, hipStream_t st)
    {
        if constexpr (!bwd_fits<T, D, RP>()) {
            return hipErrorInvalidConfiguration;
        } else {
            dim3 grid(s.nseg, s.H, s.B), grid_t(s.nseg * table_split<RP>(), s.H, s.B);
            ELSAA_LAUNCH("race_dq", (race_dq_kernel<T, D, RP>), grid_t, dim3(kThreads), 0, st, a1);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
            ELSAA_LAUNCH("race_dk", (race_dk_kernel<T, D, RP>), grid_t, dim3(kThreads), 0, st, a2);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            ELSAA_LAUNCH("race_dv", (race_dv_kernel<T, D, RP>), grid, dim3(kThreads), 0, st, a3);
            return hipGetLastError();
        }
    }
};

template <class T, int D, int RP>
struct BwdFitsFn {
    static hipError_t run(const Shape&) { return bwd_fits<T, D, RP>() ? hipSuccess : hipErrorInvalidConfiguration; }
};

template <template <class, int, int> class Fn, class... A>
hipError_t dispatch(const Shape& s, A&&... args)
{
    const int rp = race_padded_features(s.r);
#define ELSAA_RP(T_, D_)                                                        \
    switch (rp) {                                                               \
        case 32: return Fn<T_, D_, 32>::run(s, args...);                        \
        case 64: return Fn<T_, D_, 64>::run(s, args...);                        \
        case 128: return Fn<T_, D_, 128>::run(s, args...);                      \
        default: return Fn<T_, D_, 256>::run(s, args...);                       \
    }
    if (s.bf16) {
        if (s.D == 64) { ELSAA_RP(BF16, 64) }
        ELSAA_RP(BF16, 128)
    }
    if (s.D == 64) { ELSAA_RP(F32, 64) }
    ELSAA_RP(F32, 128)
#undef ELSAA_RP
}

}  // namespace

bool race_bwd_fits(const Shape& s) { return dispatch<BwdFitsFn>(s) == hipSuccess; }

size_t race_wt_bytes(const Shape& s)
{
    const int rp = race_padded_features(s.r);
    const size_t wk = rp / 4 < 32 ? 32 : rp / 4;
    return (size_t)s.H * s.D * wk * (s.bf16 ? 2 : 4);
}

int race_wk(const Shape& s)
{
    const int rp = race_padded_features(s.r);
    return rp / 4 < 32 ? 32 : rp / 4;
}

hipError_t launch_race_bwd(const Shape& s, const float* Uq, const float* Uk, const void* V,
                           const void* dO, const float* W_race, const float* rs,
                           const float* states_f, float* states_b, void* wt_hi, void* wt_lo,
                           void* du_q, void* du_k, void* dv_lr, hipStream_t st)
{
    {
        const int rp = race_padded_features(s.r);
        const int wk = rp / 4 < 32 ? 32 : rp / 4;
        dim3 grid((s.D * wk + 255) / 256, s.H);
        if (s.bf16)
            ELSAA_LAUNCH("race_wt", race_wt_kernel<BF16>, grid, dim3(256), 0, st, W_race,
                         (uint16_t*)wt_hi, (uint16_t*)wt_lo, s.L, s.D, wk);
        else
            ELSAA_LAUNCH("race_wt", race_wt_kernel<F32>, grid, dim3(256), 0, st, W_race, (float*)wt_hi,
                         (float*)wt_lo, s.L, s.D, wk);
        hipError_t e0 = hipGetLastError();
        if (e0 != hipSuccess) return e0;
    }
    const size_t BHN = (size_t)s.B * s.H * s.N;
    // backward suffix states of phi(q) dNum' / L and phi(q) dDen / L (the
    // forward prefix states of phi(k) V' and phi(k) come from the forward)
    hipError_t e = launch_race_states(s, Uq, dO, rs + 3 * BHN, rs + 4 * BHN, 1.f / (float)s.L, states_b,
                                      s.causal ? 2 : 0, st);
    if (e != hipSuccess) return e;
    LbArgs a;
    a.Uq = Uq; a.Uk = Uk; a.V = V; a.dO = dO; a.rs = rs;
    a.H = s.H; a.N = s.N; a.L = s.L; a.seg_len = s.seg_len; a.nseg = s.nseg; a.causal = s.causal;
    a.BHN = BHN;
    a.two_beta = 2.f * s.beta; a.beta = s.beta; a.inv_L = 1.f / (float)s.L;
    LbArgs a1 = a, a2 = a, a3 = a;
    a1.states = states_f; a1.out = du_q;
    a2.states = states_b; a2.out = du_k;
    a3.states = states_b; a3.out = dv_lr;
    return dispatch<BwdFn>(s, a1, a2, a3, st);
}

}  // namespace elsaa
