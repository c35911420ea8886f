// race_common.hpp -- device helpers of the RACE low-rank kernels (forward and backward).
//
// Features (Alg. 2): for table l, u = W_l x (4 projections), t = tanh(u), and
// for bucket c of the hypercube {+-1}^4 (bit b of c set <-> v_cb = +1)
//   phi_c = exp(beta t.v_c) / sum_c' exp(beta t.v_c') = prod_b sigmoid(2 beta v_cb t_b).
// The projection kernel forms u = W x once per row and stores t = tanh(u)
// in float32 (every pass uses u only through t); chunks are 64 tokens; each
// workgroup is 4 waves,
// wave w handles tokens 16w .. 16w+15 of a chunk when computing features.
#pragma once
#include "common.hpp"

namespace elsaa {
namespace race {

constexpr int kC = 64;
constexpr int kThreads = 256;
constexpr int kPad = 8;
constexpr size_t kMaxLds = 160 * 1024;

// sigmoid(x) and sigmoid(-x) from one hardware exp and reciprocal: with
// e = exp(-|x|) in (0, 1], sigmoid(|x|) = 1 / (1 + e) and
// sigmoid(-|x|) = e / (1 + e), each within a few ulp and without overflow.
__device__ __forceinline__ void sigmoid_pair(float x, float& sp, float& sn)
{
    const float e = __expf(-fabsf(x));
    const float big = __builtin_amdgcn_rcpf(1.f + e), small = e * big;
    sp = x >= 0.f ? big : small;
    sn = x >= 0.f ? small : big;
}

// tanh(u) = 1 - 2 / (1 + e^{2u}), absolute error about 1e-7 (the features use
// t only through sigmoid(2 beta t) and the chain rule through 1 - t^2)
__device__ __forceinline__ float tanh_abs(float u)
{
    return 1.f - 2.f * __builtin_amdgcn_rcpf(1.f + __expf(2.f * u));
}

// 8-slot operand fragment from a tile stored transposed, xt[k][n] (row
// stride LD elements): lane (i = lane % 16, g = lane / 16) receives column
// c0 + i at rows kb + 8 g + j, j = 0..7 (16-bit: two transposed LDS reads).
template <class T, int LD>
__device__ __forceinline__ typename T::frag_t col8_t(const typename T::store_t (*xt)[LD], int kb, int c0)
{
    const int lane = threadIdx.x & 63, g = lane >> 4, i = lane & 15;
    const int r = kb + 8 * g;
    if constexpr (T::bytes == 2) {
        const bf16x4 lo = lds_read_tr4((const uint16_t*)&xt[r + (i >> 2)][c0 + 4 * (i & 3)]);
        const bf16x4 hi = lds_read_tr4((const uint16_t*)&xt[r + 4 + (i >> 2)][c0 + 4 * (i & 3)]);
        return typename T::frag_t{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    } else {
        typename T::frag_t f;
#pragma unroll
        for (int j = 0; j < 8; ++j) f[j] = xt[r + j][c0 + i];
        return f;
    }
}

// Phi^T operand fragment from a row-major feature tile ph[token][feature]:
// lane (i, g) receives feature f0 + i at tokens kb + 8 g + j (transposed LDS
// reads, so no transposed copy of the tile is kept).
template <class T, int RP>
__device__ __forceinline__ typename T::frag_t phi_t8(const typename T::store_t (*ph)[RP + kPad], int kb, int f0)
{
    return col8_t<T, RP + kPad>(ph, kb, f0);
}

// Sums over 32 of the chunk's tokens on the matrix cores: Phi^T x 1 (every
// entry of the B operand 1), so every lane of the product tile holds the
// sums of its rows' features: lane (g, col) register i += sum over tokens
// kb .. kb + 31 of phi_{f0 + 4g + i} (phit from phi_t8 at feature f0).
template <class T>
__device__ __forceinline__ f32x4 token_sums(typename T::frag_t phit, f32x4 acc)
{
    float one[8] = {1.f, 1.f, 1.f, 1.f, 1.f, 1.f, 1.f, 1.f};
    return T::mma(phit, T::pack(one), acc);
}

// a_state[f] += scale * sum over the chunk's tokens k of xt[f][k] (* wk[k] when
// wk is not null), xt a transposed feature tile [RP][kC + kPad]; all threads,
// 256 / RP per feature (16-byte LDS reads, then a lane reduction).
template <class T, int RP>
__device__ __forceinline__ void add_chunk_sums(const typename T::store_t (*xt)[kC + kPad], const float* wk,
                                               float scale, float* a_state)
{
    constexpr int TPF = RP >= kThreads ? 1 : kThreads / RP;   // threads per feature
    constexpr int PER = kC / TPF;                               // tokens per thread
    static_assert(PER % 8 == 0, "chunk split");
    for (int f0 = 0; f0 < RP; f0 += kThreads / TPF) {
        const int f = f0 + (int)threadIdx.x / TPF, part = threadIdx.x % TPF;
        float s = 0.f;
#pragma unroll
        for (int k8 = 0; k8 < PER; k8 += 8) {
            const int k = part * PER + k8;
            const auto v = T::ld8(&xt[f][k]);
#pragma unroll
            for (int j = 0; j < 8; ++j) s += wk ? (float)v[j] * wk[k + j] : (float)v[j];
        }
#pragma unroll
        for (int m = 1; m < TPF; m <<= 1) s += __shfl_xor(s, m);
        if (part == 0) a_state[f] += s * scale;
    }
}

// projection count padded to whole 32-wide k-steps (backward du x W)
template <int RP> constexpr int w_kdim() { return RP / 4 < 32 ? 32 : RP / 4; }

// Workgroups per sequence segment in the passes whose feature tables are
// independent (the state sums and the dQ / dK chain rules): each holds
// RP / split consecutive features (whole tables), reads the same chunk rows
// and writes its own state rows or du columns.  256 features split in two,
// so a workgroup's registers and LDS are those of the 128-feature passes.
template <int RP> constexpr int table_split() { return RP == 256 ? 2 : 1; }

// Rows [t0, t0 + 64) of X (zero past N), each multiplied by scale[row] * mul
// when scale != nullptr (by mul otherwise), into a transposed tile
// xt[d][token].  load() issues every global load of the thread into
// registers and store() writes them to LDS, so a caller can load the next
// chunk while the current one is consumed; stage_t does both at once.
template <class T, int D>
struct StageT {
    using S = typename T::store_t;
    static constexpr int PER = 16 / T::bytes;
    static constexpr int CH = D / PER;
    static constexpr int ITEMS = (kC / 2) * CH, PT = ITEMS / kThreads;
    static_assert(ITEMS % kThreads == 0, "staging split");
    uint4 va[PT], vb[PT];
    float sa[PT], sb[PT];   // row scales as loaded (mul is applied in store())
    float mul_;
    int t0_, n_;
    // Rows past N are loaded clamped to row N - 1 and zeroed in store(), so
    // the loads carry no per-lane branches and later waits count exactly.
    __device__ __forceinline__ void load(const S* X, int t0, int N, const float* scale, float mul)
    {
        t0_ = t0;
        n_ = N;
        mul_ = mul;
#pragma unroll
        for (int j = 0; j < PT; ++j) {
            const int it = threadIdx.x + j * kThreads;
            const int p = it & (kC / 2 - 1), c = it / (kC / 2);
            const int r0 = min(t0 + 2 * p, N - 1), r1 = min(t0 + 2 * p + 1, N - 1);
            va[j] = ldg16(X + (size_t)r0 * D + c * PER);
            vb[j] = ldg16(X + (size_t)r1 * D + c * PER);
            sa[j] = scale ? scale[r0] : 1.f;
            sb[j] = scale ? scale[r1] : 1.f;
        }
    }
    // the two rows of an item are adjacent in the transposed tile: one
    // store per element pair
    __device__ __forceinline__ void store(S (*xt)[kC + kPad], bool scaled) const
    {
#pragma unroll
        for (int j = 0; j < PT; ++j) {
            const int it = threadIdx.x + j * kThreads;
            const int p = it & (kC / 2 - 1), c = it / (kC / 2);
            const bool in0 = t0_ + 2 * p < n_, in1 = t0_ + 2 * p + 1 < n_;
            const S* ea = (const S*)&va[j];
            const S* eb = (const S*)&vb[j];
#pragma unroll
            for (int e = 0; e < PER; ++e) {
                S x0 = in0 ? ea[e] : T::store(0.f), x1 = in1 ? eb[e] : T::store(0.f);
                if (scaled) {
                    x0 = T::store(T::load(x0) * (sa[j] * mul_));
                    x1 = T::store(T::load(x1) * (sb[j] * mul_));
                }
                S* dst = &xt[c * PER + e][2 * p];
                if constexpr (T::bytes == 2)
                    *(uint32_t*)dst = (uint32_t)x0 | ((uint32_t)x1 << 16);
                else
                    *(float2*)dst = make_float2(x0, x1);
            }
        }
    }
};

template <class T, int D>
__device__ void stage_t(typename T::store_t (*xt)[kC + kPad], const typename T::store_t* X,
                        int t0, int N, const float* scale = nullptr, float mul = 1.f)
{
    StageT<T, D> st;
    st.load(X, t0, N, scale, mul);
    st.store(xt, scale || mul != 1.f);
}

// Rows [t0, t0 + 64) of X (zero past N), optionally scaled per row, row-major;
// load() / store() as in StageT, stage_r does both.
template <class T, int D>
struct StageR {
    using S = typename T::store_t;
    static constexpr int PER = 16 / T::bytes;
    static constexpr int CH = D / PER;
    static constexpr int ITEMS = kC * CH, PT = ITEMS / kThreads;
    static_assert(ITEMS % kThreads == 0, "staging split");
    uint4 v[PT];
    float sc[PT];
    int t0_, n_;
    // rows past N: loaded clamped, zeroed in store() (see StageT)
    __device__ __forceinline__ void load(const S* X, int t0, int N, const float* scale)
    {
        t0_ = t0;
        n_ = N;
#pragma unroll
        for (int j = 0; j < PT; ++j) {
            const int it = threadIdx.x + j * kThreads;
            const int row = it % kC, c = it / kC;
            const int r = min(t0 + row, N - 1);
            v[j] = ldg16(X + (size_t)r * D + c * PER);
            sc[j] = scale ? scale[r] : 0.f;
        }
    }
    __device__ __forceinline__ void store(S (*x)[D + kPad], bool scaled)
    {
#pragma unroll
        for (int j = 0; j < PT; ++j) {
            const int it = threadIdx.x + j * kThreads;
            const int row = it % kC, c = it / kC;
            if (t0_ + row >= n_) v[j] = make_uint4(0, 0, 0, 0);
            if (scaled) {
                S* e = (S*)&v[j];
#pragma unroll
                for (int q = 0; q < PER; ++q) e[q] = T::store(T::load(e[q]) * sc[j]);
            }
            *(uint4*)&x[row][c * PER] = v[j];
        }
    }
};

template <class T, int D>
__device__ void stage_r(typename T::store_t (*x)[D + kPad], const typename T::store_t* X, int t0,
                        int N, const float* scale = nullptr)
{
    StageR<T, D> st;
    st.load(X, t0, N, scale);
    st.store(x, scale != nullptr);
}

// Projections t = tanh(u) of the tables this lane handles for chunk tokens
// [t0 + 16w, t0 + 16w + 16) (table tb = g + 4 m of token 16w + col), loaded
// ahead of features_from so that the next chunk's loads overlap this one.
template <int RP>
struct URegs {
    static constexpr int NU = (RP / 16 + 3) / 4;
    f32x4 u[NU];
    // Rows past N and tables past RP / 16 load clamped in-range values
    // (features_from zeroes those rows' features and skips those tables), so
    // the loads carry no per-lane branches.
    // stride: floats per projection row (RP / 4 unless this workgroup holds
    // only some of the row's tables, U then pointing at its first table)
    __device__ __forceinline__ void load(const float* U, int t0, int N, int stride = RP / 4)
    {
        const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
        const int g = lane >> 4, col = lane & 15;
        const int tok = min(t0 + 16 * wv + col, N - 1);
#pragma unroll
        for (int m = 0; m < NU; ++m) {
            const int tb = min(g + 4 * m, RP / 16 - 1);
            u[m] = *(const f32x4*)(U + (size_t)tok * stride + 4 * tb);
        }
    }
};

// Features of chunk tokens [t0 + 16w, t0 + 16w + 16) for every table, from
// the projections t = tanh(u) in ur (URegs::load of the same chunk).
// Writes phi (as T) row-major into ph[token][feature] and/or transposed into
// pht[feature][token], and t into ts[token][4 * table + bit].
template <class T, int RP>
__device__ void features_from(const URegs<RP>& ur, int t0, int N, int L, float two_beta,
                              typename T::store_t (*ph)[RP + kPad], typename T::store_t (*pht)[kC + kPad],
                              float (*ts)[RP / 4])
{
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int g = lane >> 4, col = lane & 15;
    const int tl = 16 * wv + col;
    const int tok = t0 + tl;
#pragma unroll
    for (int m = 0; m < URegs<RP>::NU; ++m) {   // this lane: table tb of token tl
        const int tb = g + 4 * m;
        if (tb >= RP / 16) break;
        const f32x4 t = ur.u[m];                 // t = tanh(W x), formed by the projection pass
        const bool live = tb < L && tok < N;
        float sp[4], sn[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) sigmoid_pair(two_beta * t[i], sp[i], sn[i]);
        if (ts) *(f32x4*)&ts[tl][4 * tb] = f32x4{t[0], t[1], t[2], t[3]};
        float phi[16];
#pragma unroll
        for (int c = 0; c < 16; ++c) {
            const float v = ((c & 1) ? sp[0] : sn[0]) * ((c & 2) ? sp[1] : sn[1]) *
                            ((c & 4) ? sp[2] : sn[2]) * ((c & 8) ? sp[3] : sn[3]);
            phi[c] = live ? v : 0.f;
        }
        if (ph) {
            using F = typename T::frag_t;
            *(F*)&ph[tl][16 * tb] = T::pack(phi);
            *(F*)&ph[tl][16 * tb + 8] = T::pack(phi + 8);
        }
        if (pht) {
#pragma unroll
            for (int c = 0; c < 16; ++c) pht[16 * tb + c][tl] = T::store(phi[c]);
        }
    }
}

// features_from with the projections loaded on the spot.
template <class T, int RP>
__device__ void features(const float* U, int t0, int N, int L, float two_beta,
                         typename T::store_t (*ph)[RP + kPad], typename T::store_t (*pht)[kC + kPad],
                         float (*ts)[RP / 4])
{
    URegs<RP> ur;
    ur.load(U, t0, N);
    features_from<T, RP>(ur, t0, N, L, two_beta, ph, pht, ts);
}

// Chain rule from a transposed feature-gradient tile to the projection
// gradients du.  dphi: accumulator tile of the 16 features of table tb x 16
// rows (lane (g, col) register i holds feature c = 4g + i of row
// 16*qt + col).  With phi_c = prod_b sigmoid(2 beta v_cb t_b), t = tanh(u):
//   dt_b = beta * sum_c dphi_c phi_c (v_cb - tanh(beta t_b)),  du_b = dt_b (1 - t_b^2)
// (tanh(beta t_b) = sigmoid(2 beta t_b) - sigmoid(-2 beta t_b) is the mean of
// v_cb under phi).  Sums over c: 4 registers, then the 4 lane groups.  Lane
// group g writes du[row][4 tb + g] (zero for padded tables).
template <class T, int RP>
__device__ __forceinline__ void chain_rule_t(f32x4 dphi, int qt, int tb, int L, float beta,
                                             const float (*ts)[RP / 4],
                                             typename T::store_t (*du)[w_kdim<RP>() + kPad])
{
    const int lane = threadIdx.x & 63;
    const int g = lane >> 4, col = lane & 15;
    const int row = 16 * qt + col;
    // lane group g evaluates bit g's sigmoid pair; the groups then share them
    const float tg = ts[row][4 * tb + g];
    float spg, sng, sp[4], sn[4];
    sigmoid_pair(2.f * beta * tg, spg, sng);
    gather16x4(spg, sp);
    gather16x4(sng, sn);
    // features c = 4g + i: bits 0, 1 from i, bits 2, 3 from g
    const float hi = ((g & 1) ? sp[2] : sn[2]) * ((g & 2) ? sp[3] : sn[3]);
    float p0 = 0.f, p1 = 0.f, p2 = 0.f;       // sums over i of x, x v_c0, x v_c1
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float phi = ((i & 1) ? sp[0] : sn[0]) * ((i & 2) ? sp[1] : sn[1]) * hi;
        const float x = dphi[i] * phi;
        p0 += x;
        p1 += (i & 1) ? x : -x;
        p2 += (i & 2) ? x : -x;
    }
    // over the lane groups: g & 1 (lane bit 4) is feature bit 2, g >> 1 (lane
    // bit 5) feature bit 3; each exchange gives both the sum and the
    // difference of the two groups
    const LanePair a0 = xpair16(p0), a1 = xpair16(p1), a2 = xpair16(p2);
    const LanePair b0 = xpair32(a0.lo + a0.hi), bd = xpair32(a0.hi - a0.lo);
    const LanePair b1 = xpair32(a1.lo + a1.hi), b2 = xpair32(a2.lo + a2.hi);
    const float s0 = b0.lo + b0.hi;            // sum over c of x_c
    // sums over c of x_c v_cb for b = 0..3
    const float sb[4] = {b1.lo + b1.hi, b2.lo + b2.hi, bd.lo + bd.hi, b0.hi - b0.lo};
    const float sbg = g == 0 ? sb[0] : g == 1 ? sb[1] : g == 2 ? sb[2] : sb[3];
    const float v = beta * (sbg - (spg - sng) * s0) * (1.f - tg * tg);
    du[row][4 * tb + g] = T::store(tb < L ? v : 0.f);
}

}  // namespace race
}  // namespace elsaa
