// token_rules.hip -- token-wise rules of the fusion, forward and backward:
//   * the gate network (Sec. 3.3, Alg. 1; a two-layer MLP with SiLU and two
//     independent sigmoid outputs in the experimental setup):
//         (g_sparse, g_lr) = sigmoid(W2 SiLU(W1 q_i + b1) + b2);
//   * the query-dependent coefficient of the ELSAA configuration appendix:
//         lambda_i = max(lambda_min, c + sigmoid(w^T q_i + b)),
//     with q_i detached from this path.
// Every head has its own parameters; q_i is the head's query row.
//
// Both rules read each query row once.  The first layer runs on the matrix
// cores with q as the A operand; w is appended to W1 as row G (rows
// G+1 .. G+15 are zero), so w^T q comes out of the same products.  Weights
// keep float32 accuracy as bf16 hi + lo pairs for bf16 storage and are exact
// for float32 storage.  A workgroup of NW waves walks the RT = 32 NW row
// tiles of one (b, h) row chunk, each wave owning 32 rows of a tile, with the
// next tile's rows prefetched into registers.  The two 16-row products of a
// wave are fed in the krow_of row order, so lane group g ends up holding rows
// 8g .. 8g+7 of its hidden column: the layout the backward needs to use the
// hidden-layer gradient as a 32-row k-step operand.
//
// Backward: dz2 = dg g (1 - g), da = W2^T dz2, dz1 = da SiLU'(z1); the lambda
// path contributes t = dlambda [c + s >= lambda_min] s (1 - s) as row G.
// dz1^T is staged in LDS; dW1 (with dw as row G) = dz1^T q is contracted over
// the tile's rows on the matrix cores, each wave owning a column slice, and
// dq += W1^T dz1 over the G hidden units for the wave's own rows.  Parameter
// gradients are summed per workgroup into a partial buffer and reduced over
// the workgroups in a fixed order (deterministic).
#include "common.hpp"
#include "internal.hpp"
#include "tile.hpp"

#include <type_traits>

namespace elsaa {
namespace {

struct TrArgs {
    const void* Q;
    const float *W1, *b1, *W2, *b2;     // gate network of every head
    const float *lw, *lb, *lc;          // lambda rule of every head
    float lam_min;
    float* gates;                       // forward outputs [BHN][2], [BHN]
    float* lam;
    const float* dg;                    // backward inputs [BHN][2], [BHN]
    const float* dlam;
    void* dQ;                           // accumulated in place (may be null)
    float* part;                        // per-workgroup partial sums
    int H, N, nchunk, chunk_rows;
};

__device__ __forceinline__ float sigm(float x) { return 1.f / (1.f + __expf(-x)); }

template <class T, int D, int G, bool LAM>
struct TokenRules {
    static constexpr int NW = T::bytes == 2 ? 4 : 2;
    static constexpr int NT = 64 * NW;
    static constexpr int RT = 32 * NW;               // rows per tile
    static constexpr int GX = G + (LAM ? 16 : 0);    // first-layer columns
    static constexpr int NB = GX / 16;
    static constexpr int NG = G / 16;                // gate hidden column blocks
    static constexpr int CBW = D / 16 / NW;          // dW1 column blocks per wave
    static constexpr int HALVES = RT / 64;           // 64-row staging passes per tile
    static constexpr bool SPLIT = T::bytes == 2;     // W1 as bf16 hi + lo
    static constexpr bool DQ_EARLY = G <= 64 && T::bytes == 2;   // dQ rows fetched before the products
    using S = typename T::store_t;
    using F = typename T::frag_t;
    using TQ = tile::Tile<T, D, NT>;                 // rows of D elements (q, W1)
    using TZ = tile::Tile<T, RT, NT>;                // rows of RT elements (dz1^T)
    static_assert(CBW >= 1 && GX >= 16, "shape");

    struct Smem {
        S qt[TQ::elems(RT)];
        S whi[TQ::elems(GX)];
        S wlo[SPLIT ? TQ::elems(GX) : 1];
        float b1[G > 0 ? G : 1];
        float w2[G > 0 ? 2 * G : 1];
    };
    struct SmemB {
        Smem m;
        S zt[TZ::elems(GX)];                         // dz1^T, rows = hidden units
    };

    // ---- staging -------------------------------------------------------
    __device__ static void load_rows(const S* X, int row0, int N, uint4 (&r)[HALVES][TQ::PER_THREAD])
    {
#pragma unroll
        for (int hf = 0; hf < HALVES; ++hf) {
            int tok[TQ::PER_THREAD];
#pragma unroll
            for (int j = 0; j < TQ::PER_THREAD; ++j) {
                const int row = row0 + 64 * hf + TQ::row_of(j);
                tok[j] = row < N ? row : -1;
            }
            TQ::load(X, tok, r[hf]);
        }
    }
    __device__ static void store_rows(S* qt, const uint4 (&r)[HALVES][TQ::PER_THREAD])
    {
#pragma unroll
        for (int hf = 0; hf < HALVES; ++hf) TQ::store(qt, r[hf], 64 * hf);
    }

    // W1 of head h (w as row G) into LDS, split into hi / lo for bf16; b1, W2.
    __device__ static void stage_params(const TrArgs& a, int h, Smem& sm)
    {
        constexpr int Q4 = D / 4;
        for (int c = threadIdx.x; c < GX * Q4; c += NT) {
            const int n = c / Q4, e = (c % Q4) * 4;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (n < G) v = *(const float4*)(a.W1 + ((size_t)h * G + n) * D + e);
            else if (LAM && n == G) v = *(const float4*)(a.lw + (size_t)h * D + e);
            if constexpr (SPLIT) {
                const float f[4] = {v.x, v.y, v.z, v.w};
                uint32_t hi[4], lo[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const uint16_t hb = f32_to_bf16(f[j]);
                    hi[j] = hb;
                    lo[j] = f32_to_bf16(f[j] - bf16_to_f32(hb));
                }
                *(uint2*)&sm.whi[TQ::row(n) + e] = make_uint2(hi[0] | (hi[1] << 16), hi[2] | (hi[3] << 16));
                *(uint2*)&sm.wlo[TQ::row(n) + e] = make_uint2(lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16));
            } else {
                *(float4*)&sm.whi[TQ::row(n) + e] = v;
            }
        }
        if constexpr (G > 0) {
            for (int n = threadIdx.x; n < G; n += NT) {
                sm.b1[n] = a.b1[(size_t)h * G + n];
                sm.w2[n] = a.W2[((size_t)h * 2 + 0) * G + n];
                sm.w2[G + n] = a.W2[((size_t)h * 2 + 1) * G + n];
            }
        }
    }

    // ---- first layer ---------------------------------------------------
    // acc[s][cb] register i of lane group g: z1 (without b1) of tile row
    // wr0 + 8g + 4s + i, column 16 cb + lane % 16.
    __device__ static void first_layer(const Smem& sm, int wr0, f32x4 (&acc)[2][NB])
    {
        const int lane = threadIdx.x & 63, g = lane >> 4, rho = lane & 15;
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
            for (int cb = 0; cb < NB; ++cb) acc[s][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
        const int r0 = wr0 + krow_of(0, rho), r1 = wr0 + krow_of(1, rho);
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) {
            const F a0 = TQ::row8(sm.qt, r0, 32 * ks + 8 * g);
            const F a1 = TQ::row8(sm.qt, r1, 32 * ks + 8 * g);
#pragma unroll
            for (int cb = 0; cb < NB; ++cb) {
                const F bh = TQ::row8(sm.whi, 16 * cb + rho, 32 * ks + 8 * g);
                acc[0][cb] = T::mma(a0, bh, acc[0][cb]);
                acc[1][cb] = T::mma(a1, bh, acc[1][cb]);
                if constexpr (SPLIT) {
                    const F bl = TQ::row8(sm.wlo, 16 * cb + rho, 32 * ks + 8 * g);
                    acc[0][cb] = T::mma(a0, bl, acc[0][cb]);
                    acc[1][cb] = T::mma(a1, bl, acc[1][cb]);
                }
            }
        }
    }

    // Second-layer logits of the 8 rows of the lane group (all 16 lanes of
    // the group get them): z2[o][s][i] for row 8g + 4s + i.
    __device__ static void second_layer(const Smem& sm, const f32x4 (&acc)[2][NB], float b20, float b21,
                                        float (&z2)[2][2][4])
    {
        const int rho = threadIdx.x & 15;
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
            for (int i = 0; i < 4; ++i) z2[0][s][i] = z2[1][s][i] = 0.f;
#pragma unroll
        for (int cb = 0; cb < NG; ++cb) {
            const int n = 16 * cb + rho;
            const float bb = sm.b1[n], w0 = sm.w2[n], w1 = sm.w2[G + n];
#pragma unroll
            for (int s = 0; s < 2; ++s)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float z = acc[s][cb][i] + bb;
                    const float av = z * sigm(z);
                    z2[0][s][i] += w0 * av;
                    z2[1][s][i] += w1 * av;
                }
        }
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                z2[0][s][i] = row_sum16(z2[0][s][i]) + b20;
                z2[1][s][i] = row_sum16(z2[1][s][i]) + b21;
            }
    }

    // value of row 8g + rho (rho < 8) from the group-wide registers
    __device__ static float pick(const float (&v)[2][4], int rho)
    {
        float r = 0.f;
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
            for (int i = 0; i < 4; ++i) r = (4 * s + i == rho) ? v[s][i] : r;
        return r;
    }

    // chunk of rows of this workgroup
    __device__ static void chunk(const TrArgs& a, int& bh, int& h, int& rbeg, int& rend)
    {
        bh = blockIdx.x / a.nchunk;
        h = bh % a.H;
        rbeg = (blockIdx.x % a.nchunk) * a.chunk_rows;
        rend = min(a.N, rbeg + a.chunk_rows);
    }

    // ---- forward -------------------------------------------------------
    __device__ static void fwd(const TrArgs& a, Smem& sm)
    {
        int bh, h, rbeg, rend;
        chunk(a, bh, h, rbeg, rend);
        const int N = a.N;
        const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, rho = lane & 15;
        const int wr0 = 32 * w;
        const S* X = (const S*)a.Q + (size_t)bh * N * D;
        float b20 = 0.f, b21 = 0.f, lb = 0.f, lc = 0.f;
        if constexpr (G > 0) { b20 = a.b2[2 * h]; b21 = a.b2[2 * h + 1]; }
        if constexpr (LAM) { lb = a.lb[h]; lc = a.lc[h]; }

        uint4 rg[HALVES][TQ::PER_THREAD];
        load_rows(X, rbeg, N, rg);
        stage_params(a, h, sm);
        for (int row0 = rbeg; row0 < rend; row0 += RT) {
            store_rows(sm.qt, rg);
            if (row0 + RT < rend) load_rows(X, row0 + RT, N, rg);
            __syncthreads();
            f32x4 acc[2][NB];
            first_layer(sm, wr0, acc);
            const int row = row0 + wr0 + 8 * g + rho;     // row written by lanes rho < 8
            const bool wr = rho < 8 && row < rend;
            if constexpr (G > 0) {
                float z2[2][2][4];
                second_layer(sm, acc, b20, b21, z2);
                const float v0 = pick(z2[0], rho), v1 = pick(z2[1], rho);
                if (wr) *(float2*)&a.gates[((size_t)bh * N + row) * 2] = make_float2(sigm(v0), sigm(v1));
            }
            if constexpr (LAM) {
                float zl[2][4];
#pragma unroll
                for (int s = 0; s < 2; ++s)
#pragma unroll
                    for (int i = 0; i < 4; ++i) zl[s][i] = __shfl(acc[s][NG][i], lane & 48);
                const float z = pick(zl, rho) + lb;
                if (wr) a.lam[(size_t)bh * N + row] = fmaxf(a.lam_min, lc + sigm(z));
            }
            __syncthreads();
        }
    }

    // ---- backward ------------------------------------------------------
    __device__ static void bwd(const TrArgs& a, SmemB& sb)
    {
        Smem& sm = sb.m;
        int bh, h, rbeg, rend;
        chunk(a, bh, h, rbeg, rend);
        const int N = a.N;
        const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, rho = lane & 15;
        const int wr0 = 32 * w;
        const S* X = (const S*)a.Q + (size_t)bh * N * D;
        float b20 = 0.f, b21 = 0.f, lb = 0.f, lc = 0.f;
        if constexpr (G > 0) { b20 = a.b2[2 * h]; b21 = a.b2[2 * h + 1]; }
        if constexpr (LAM) { lb = a.lb[h]; lc = a.lc[h]; }

        // per-lane running sums
        f32x4 accW[NB][CBW];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int j = 0; j < CBW; ++j) accW[nb][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        float sb1[NG > 0 ? NG : 1], sw20[NG > 0 ? NG : 1], sw21[NG > 0 ? NG : 1];
#pragma unroll
        for (int cb = 0; cb < (NG > 0 ? NG : 1); ++cb) sb1[cb] = sw20[cb] = sw21[cb] = 0.f;
        float sb20 = 0.f, sb21 = 0.f, slb = 0.f, slc = 0.f;

        uint4 rg[HALVES][TQ::PER_THREAD];
        load_rows(X, rbeg, N, rg);
        stage_params(a, h, sm);
        for (int row0 = rbeg; row0 < rend; row0 += RT) {
            store_rows(sm.qt, rg);
            if (row0 + RT < rend) load_rows(X, row0 + RT, N, rg);
            __syncthreads();
            // the row gradients and the dQ rows this wave adds to, loaded
            // before the products so that their latency is hidden
            const size_t rb = (size_t)bh * N + row0 + wr0 + 8 * g;   // row of (s, i): rb + 4s + i
            const int rleft = rend - (row0 + wr0 + 8 * g);           // rows of the group before rend
            float2 dgv[2][4];
            float dlv[2][4];
#pragma unroll
            for (int s = 0; s < 2; ++s)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const bool ok = 4 * s + i < rleft;
                    dgv[s][i] = (G > 0 && ok) ? *(const float2*)&a.dg[(rb + 4 * s + i) * 2] : make_float2(0.f, 0.f);
                    dlv[s][i] = (LAM && ok && rho == 0) ? a.dlam[rb + 4 * s + i] : 0.f;
                }
            DqRegs dqv;
            if constexpr (G > 0 && DQ_EARLY)
                if (a.dQ) dq_load((const S*)a.dQ + (size_t)bh * N * D, row0, wr0, rend, dqv);
            {
                f32x4 acc[2][NB];
                first_layer(sm, wr0, acc);
                if constexpr (G > 0) {
                    float z2[2][2][4], dz0[2][4], dz1[2][4];
                    second_layer(sm, acc, b20, b21, z2);
#pragma unroll
                    for (int s = 0; s < 2; ++s)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float2 d = dgv[s][i];
                            const float g0 = sigm(z2[0][s][i]), g1 = sigm(z2[1][s][i]);
                            dz0[s][i] = d.x * g0 * (1.f - g0);
                            dz1[s][i] = d.y * g1 * (1.f - g1);
                            if (rho == 0) { sb20 += dz0[s][i]; sb21 += dz1[s][i]; }
                        }
#pragma unroll
                    for (int cb = 0; cb < NG; ++cb) {
                        const int n = 16 * cb + rho;
                        const float bb = sm.b1[n], w0 = sm.w2[n], w1 = sm.w2[G + n];
                        float dzv[2][4];
#pragma unroll
                        for (int s = 0; s < 2; ++s)
#pragma unroll
                            for (int i = 0; i < 4; ++i) {
                                const float z = acc[s][cb][i] + bb;
                                const float sg = sigm(z);
                                const float av = z * sg;
                                sw20[cb] += dz0[s][i] * av;
                                sw21[cb] += dz1[s][i] * av;
                                const float da = w0 * dz0[s][i] + w1 * dz1[s][i];
                                const float d = da * sg * (1.f + z * (1.f - sg));
                                sb1[cb] += d;
                                dzv[s][i] = d;
                            }
                        put4(sb.zt, n, wr0 + 8 * g, dzv);
                    }
                }
                if constexpr (LAM) {
                    float tv[2][4];
#pragma unroll
                    for (int s = 0; s < 2; ++s)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            tv[s][i] = 0.f;
                            if (rho == 0) {
                                const float dl = dlv[s][i];
                                const float sl = sigm(acc[s][NG][i] + lb);
                                const float e = (lc + sl >= a.lam_min) ? dl : 0.f;
                                const float t = e * sl * (1.f - sl);
                                slb += t;
                                slc += e;
                                tv[s][i] = t;
                            }
                        }
                    put4(sb.zt, G + rho, wr0 + 8 * g, tv);
                }
            }
            __syncthreads();
            // dW1 (and dw as row G) += dz1^T q over the tile's rows
#pragma unroll
            for (int kr = 0; kr < RT / 32; ++kr) {
                F bq[CBW];
#pragma unroll
                for (int j = 0; j < CBW; ++j) bq[j] = TQ::col8(sm.qt, 32 * kr, 16 * (w * CBW + j));
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    const F az = TZ::row8(sb.zt, 16 * nb + rho, 32 * kr + 8 * g);
#pragma unroll
                    for (int j = 0; j < CBW; ++j) accW[nb][j] = T::mma(az, bq[j], accW[nb][j]);
                }
            }
            // dq += W1^T dz1 for the wave's own rows (q^T layout: lane holds 4
            // consecutive columns of one row)
            if constexpr (G > 0) {
                if (a.dQ) {
                    S* dQ = (S*)a.dQ + (size_t)bh * N * D;
                    if constexpr (DQ_EARLY) {
#pragma unroll
                        for (int cbk = 0; cbk < D / 16; ++cbk) dq_block(sb, dQ, cbk, row0, wr0, rend, dqv);
                    } else {
#pragma unroll 1
                        for (int cbk = 0; cbk < D / 16; ++cbk) dq_block(sb, dQ, cbk, row0, wr0, rend, dqv);
                    }
                }
            }
            __syncthreads();
        }

        // ---- per-workgroup partial sums --------------------------------
        constexpr TrLayout lay{G, D, LAM ? 1 : 0};
        float* P = a.part + (size_t)blockIdx.x * lay.stride();
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int j = 0; j < CBW; ++j) {
                const int c = 16 * (w * CBW + j) + rho;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int n = 16 * nb + 4 * g + i;
                    if (n < G) P[lay.w1() + n * D + c] = accW[nb][j][i];
                    else if (LAM && n == G) P[lay.lw() + c] = accW[nb][j][i];
                }
            }
        // vectors and scalars: sum the four lane groups, then the waves in order
        constexpr int NV = 3 * G + 4;
        float* red = (float*)sm.qt;                    // NW x NV floats (the q tile is free now)
#pragma unroll
        for (int cb = 0; cb < NG; ++cb) {
            const float v0 = wave_sum16(sb1[cb]), v1 = wave_sum16(sw20[cb]), v2 = wave_sum16(sw21[cb]);
            if (g == 0) {
                red[w * NV + 16 * cb + rho] = v0;
                red[w * NV + G + 16 * cb + rho] = v1;
                red[w * NV + 2 * G + 16 * cb + rho] = v2;
            }
        }
        {
            const float v0 = wave_sum16(sb20), v1 = wave_sum16(sb21), v2 = wave_sum16(slb), v3 = wave_sum16(slc);
            if (lane == 0) {
                red[w * NV + 3 * G + 0] = v0;
                red[w * NV + 3 * G + 1] = v1;
                red[w * NV + 3 * G + 2] = v2;
                red[w * NV + 3 * G + 3] = v3;
            }
        }
        __syncthreads();
        for (int e = threadIdx.x; e < NV; e += NT) {
            float s = 0.f;
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) s += red[ww * NV + e];
            if (e < G) P[lay.b1() + e] = s;
            else if (e < 3 * G) P[lay.w2() + e - G] = s;
            else if (e < 3 * G + 2) { if (G > 0) P[lay.b2() + e - 3 * G] = s; }
            else if (LAM && e == 3 * G + 2) P[lay.lb()] = s;
            else if (LAM && e == 3 * G + 3) P[lay.lc()] = s;
        }
    }

    // 4 values of rows c0 + 4s + i (i = 0..3) into row n of dz1^T
    __device__ static void put4(S* zt, int n, int c0, const float (&v)[2][4])
    {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            S* p = &zt[TZ::row(n) + c0 + 4 * s];
            if constexpr (T::bytes == 2) {
                const uint32_t lo = f32_to_bf16(v[s][0]) | ((uint32_t)f32_to_bf16(v[s][1]) << 16);
                const uint32_t hi = f32_to_bf16(v[s][2]) | ((uint32_t)f32_to_bf16(v[s][3]) << 16);
                *(uint2*)p = make_uint2(lo, hi);
            } else {
                *(float4*)p = make_float4(v[s][0], v[s][1], v[s][2], v[s][3]);
            }
        }
    }

    // the wave's dQ values in the q^T accumulator layout: [cbk][r] holds
    // columns 16 cbk + 4g .. +3 of row row0 + wr0 + 16 r + lane % 16
    using DqPiece = typename std::conditional<T::bytes == 2, uint2, float4>::type;
    struct DqRegs {
        DqPiece v[D / 16][2];
    };
    // dq += W1^T dz1 for columns 16 cbk .. +15 of the wave's own rows (q^T
    // layout: the lane holds 4 consecutive columns of one row)
    __device__ static void dq_block(const SmemB& sb, S* dQ, int cbk, int row0, int wr0, int rend, const DqRegs& dqv)
    {
        const int lane = threadIdx.x & 63, g = lane >> 4, rho = lane & 15;
        DqPiece old[2];
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int row = row0 + wr0 + 16 * r + rho;
            if constexpr (DQ_EARLY) old[r] = dqv.v[cbk][r];
            else old[r] = row < rend ? *(const DqPiece*)(dQ + (size_t)row * D + 16 * cbk + 4 * g) : DqPiece{};
        }
        f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
        for (int kn = 0; kn < G / 32; ++kn) {
            const F ah = TQ::col8(sb.m.whi, 32 * kn, 16 * cbk);
            const F al = SPLIT ? TQ::col8(sb.m.wlo, 32 * kn, 16 * cbk) : ah;
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                const F bz = TZ::col8(sb.zt, 32 * kn, wr0 + 16 * r);
                acc[r] = T::mma(ah, bz, acc[r]);
                if constexpr (SPLIT) acc[r] = T::mma(al, bz, acc[r]);
            }
        }
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int row = row0 + wr0 + 16 * r + rho;
            if (row < rend) dq_store(dQ + (size_t)row * D + 16 * cbk + 4 * g, old[r], acc[r]);
        }
    }

    __device__ static void dq_load(const S* dQ, int row0, int wr0, int rend, DqRegs& q)
    {
        const int lane = threadIdx.x & 63, g = lane >> 4, rho = lane & 15;
#pragma unroll
        for (int cbk = 0; cbk < D / 16; ++cbk)
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                const int row = row0 + wr0 + 16 * r + rho;
                q.v[cbk][r] = row < rend ? *(const DqPiece*)(dQ + (size_t)row * D + 16 * cbk + 4 * g) : DqPiece{};
            }
    }
    // p[0..3] = old + v (storage precision)
    __device__ static void dq_store(S* p, DqPiece o, f32x4 v)
    {
        if constexpr (T::bytes == 2) {
            const float x0 = bf16_to_f32(o.x & 0xffff) + v[0], x1 = bf16_to_f32(o.x >> 16) + v[1];
            const float x2 = bf16_to_f32(o.y & 0xffff) + v[2], x3 = bf16_to_f32(o.y >> 16) + v[3];
            *(uint2*)p = make_uint2(f32_to_bf16(x0) | ((uint32_t)f32_to_bf16(x1) << 16),
                                    f32_to_bf16(x2) | ((uint32_t)f32_to_bf16(x3) << 16));
        } else {
            *(float4*)p = make_float4(o.x + v[0], o.y + v[1], o.z + v[2], o.w + v[3]);
        }
    }
};

template <class T, int D, int G, bool LAM>
__global__ __launch_bounds__(T::bytes == 2 ? 256 : 128, 1) void token_rules_fwd_kernel(TrArgs a)
{
    __shared__ __attribute__((aligned(16))) typename TokenRules<T, D, G, LAM>::Smem sm;
    TokenRules<T, D, G, LAM>::fwd(a, sm);
}

template <class T, int D, int G, bool LAM>
__global__ __launch_bounds__(T::bytes == 2 ? 256 : 128, 1) void token_rules_bwd_kernel(TrArgs a)
{
    __shared__ __attribute__((aligned(16))) typename TokenRules<T, D, G, LAM>::SmemB sm;
    TokenRules<T, D, G, LAM>::bwd(a, sm);
}

// out[h][e] = sum over (b, chunk) of the partials of head h, in order
struct TrRedArgs {
    const float* part;
    float *dW1, *db1, *dW2, *db2, *dlw, *dlb, *dlc;
    TrLayout lay;
    int B, H, nchunk;
};

__global__ __launch_bounds__(256) void token_rules_reduce_kernel(TrRedArgs r)
{
    const int h = blockIdx.y, e = blockIdx.x * 256 + threadIdx.x;
    const TrLayout& L = r.lay;
    if (e >= L.total()) return;
    float s = 0.f;
    for (int b = 0; b < r.B; ++b) {
        const float* p = r.part + ((size_t)(b * r.H + h) * r.nchunk) * L.stride() + e;
        for (int c = 0; c < r.nchunk; ++c) s += p[(size_t)c * L.stride()];
    }
    const int G = L.G, D = L.D;
    if (e < L.lw()) { if (r.dW1) r.dW1[(size_t)h * G * D + e] = s; }
    else if (e < L.b1()) { if (r.dlw) r.dlw[(size_t)h * D + e - L.lw()] = s; }
    else if (e < L.w2()) { if (r.db1) r.db1[(size_t)h * G + e - L.b1()] = s; }
    else if (e < L.b2()) { if (r.dW2) r.dW2[(size_t)h * 2 * G + e - L.w2()] = s; }
    else if (e < L.lb()) { if (r.db2) r.db2[(size_t)h * 2 + e - L.b2()] = s; }
    else if (e < L.lc()) { if (r.dlb) r.dlb[h] = s; }
    else { if (r.dlc) r.dlc[h] = s; }
}

// rows per workgroup chunk: about `target` workgroups, whole tiles
void plan_chunks(const Shape& s, int rt, int target, int& nchunk, int& chunk_rows)
{
    const int64_t bh = (int64_t)s.B * s.H;
    int64_t want = (target + bh - 1) / bh;
    const int64_t tiles = (s.N + rt - 1) / rt;
    if (want > tiles) want = tiles;
    if (want < 1) want = 1;
    const int64_t per = (tiles + want - 1) / want;
    chunk_rows = (int)(per * rt);
    nchunk = (int)((s.N + chunk_rows - 1) / chunk_rows);
}

constexpr int kFwdTarget = 512, kBwdTarget = 256;

int rt_of(const Shape& s) { return s.bf16 ? 128 : 64; }

template <class T, int D, int G, bool LAM>
hipError_t launch_fwd_t(const Shape& s, TrArgs a, hipStream_t st)
{
    using C = TokenRules<T, D, G, LAM>;
    plan_chunks(s, C::RT, kFwdTarget, a.nchunk, a.chunk_rows);
    a.H = s.H; a.N = s.N;
    ELSAA_LAUNCH("token_rules_fwd", (token_rules_fwd_kernel<T, D, G, LAM>),
                 dim3(s.B * s.H * a.nchunk), dim3(C::NT), 0, st, a);
    return hipGetLastError();
}

template <class T, int D, int G, bool LAM>
hipError_t launch_bwd_t(const Shape& s, TrArgs a, const TrGrads& gr, hipStream_t st)
{
    using C = TokenRules<T, D, G, LAM>;
    plan_chunks(s, C::RT, kBwdTarget, a.nchunk, a.chunk_rows);
    a.H = s.H; a.N = s.N;
    ELSAA_LAUNCH("token_rules_bwd", (token_rules_bwd_kernel<T, D, G, LAM>),
                 dim3(s.B * s.H * a.nchunk), dim3(C::NT), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    TrRedArgs r;
    r.part = a.part;
    r.dW1 = gr.dW1; r.db1 = gr.db1; r.dW2 = gr.dW2; r.db2 = gr.db2;
    r.dlw = gr.dlw; r.dlb = gr.dlb; r.dlc = gr.dlc;
    r.lay = TrLayout{G, D, LAM ? 1 : 0};
    r.B = s.B; r.H = s.H; r.nchunk = a.nchunk;
    ELSAA_LAUNCH("token_rules_reduce", token_rules_reduce_kernel,
                 dim3((r.lay.total() + 255) / 256, s.H), dim3(256), 0, st, r);
    return hipGetLastError();
}

template <class T, int D>
hipError_t dispatch(const Shape& s, int G, bool lam, bool bwd, const TrArgs& a, const TrGrads& gr,
                    hipStream_t st)
{
#define ELSAA_TR_CASE(GG, LL)                                                          \
    if (G == GG && lam == LL)                                                          \
        return bwd ? launch_bwd_t<T, D, GG, LL>(s, a, gr, st) : launch_fwd_t<T, D, GG, LL>(s, a, st);
    ELSAA_TR_CASE(0, true)
    ELSAA_TR_CASE(64, false)
    ELSAA_TR_CASE(64, true)
    ELSAA_TR_CASE(128, false)
    ELSAA_TR_CASE(128, true)
#undef ELSAA_TR_CASE
    return hipErrorInvalidValue;
}

hipError_t dispatch_all(const Shape& s, int G, bool lam, bool bwd, const TrArgs& a, const TrGrads& gr,
                        hipStream_t st)
{
    if (s.bf16) return s.D == 64 ? dispatch<BF16, 64>(s, G, lam, bwd, a, gr, st)
                                 : dispatch<BF16, 128>(s, G, lam, bwd, a, gr, st);
    return s.D == 64 ? dispatch<F32, 64>(s, G, lam, bwd, a, gr, st) : dispatch<F32, 128>(s, G, lam, bwd, a, gr, st);
}

}  // namespace

size_t token_rules_workspace_bytes(const Shape& s, int G, bool lam)
{
    int nchunk, rows;
    plan_chunks(s, rt_of(s), kBwdTarget, nchunk, rows);
    const TrLayout L{G, s.D, lam ? 1 : 0};
    return (size_t)s.B * s.H * nchunk * L.stride() * sizeof(float);
}

hipError_t launch_token_rules_fwd(const Shape& s, const TrParams& p, const void* Q, float* gates,
                                  float* lambda_rows, hipStream_t st)
{
    TrArgs a = {};
    a.Q = Q;
    a.W1 = p.W1; a.b1 = p.b1; a.W2 = p.W2; a.b2 = p.b2;
    a.lw = p.lw; a.lb = p.lb; a.lc = p.lc; a.lam_min = p.lam_min;
    a.gates = gates; a.lam = lambda_rows;
    return dispatch_all(s, p.G, p.lam != 0, false, a, TrGrads{}, st);
}

hipError_t launch_token_rules_bwd(const Shape& s, const TrParams& p, const void* Q, const float* dgates,
                                  const float* dlambda, void* dQ, const TrGrads& gr, float* part,
                                  hipStream_t st)
{
    TrArgs a = {};
    a.Q = Q;
    a.W1 = p.W1; a.b1 = p.b1; a.W2 = p.W2; a.b2 = p.b2;
    a.lw = p.lw; a.lb = p.lb; a.lc = p.lc; a.lam_min = p.lam_min;
    a.dg = dgates; a.dlam = dlambda; a.dQ = dQ; a.part = part;
    return dispatch_all(s, p.G, p.lam != 0, true, a, gr, st);
}

}  // namespace elsaa
