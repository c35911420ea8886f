// race_fwd.hip -- RACE low-rank branch forward (Alg. 2; causal chunked form Alg. 3),
// and the segment-state kernels the backward reuses.
//
// Num = (1/L) sum_l Phi_Q^l B^l, Den = (1/L) sum_l Phi_Q^l A^l with
// A^l = Phi_K^l' 1, B^l = Phi_K^l' V; the causal form restricts both sums to
// keys j <= i.  O_lr = Num / (Den + eps), d_lr = Den.
//
// Features come from t = tanh(W x), stored by the projection kernel.
// The sequence of each (b,h) is cut into segments of whole 64-token chunks:
//   state  one workgroup per segment: S = sum_j phi(x_j) v_j' (r x d) and
//          A = sum_j a_j phi(x_j) over the segment (forward: x = k, v = V,
//          a = 1; the backward reuses it with x = q, v = dNum, a = dDen);
//   scan   per (b,h): exclusive prefix (causal forward), exclusive suffix
//          (causal backward) or the total in every segment (non-causal);
//   out    one workgroup per segment: starting from its prefix state, each
//          chunk computes Num = (1/L) Phi_Q S + tril(Phi_Q Phi_K'/L) V (the
//          masked part only when causal), then adds the chunk to S.
// Each of the 4 waves owns d/4 columns of S, held as float32 matrix-core
// accumulators for the whole segment; the intra-chunk kernel matrix and every
// contraction run on MFMA (bf16 or float32 operands, float32 accumulation).
#include "internal.hpp"
#include "race_common.hpp"

namespace elsaa {

using namespace race;

namespace {

template <class T, int D, int RP>
struct StateSmem {
    using S = typename T::store_t;
    S vt[D][kC + kPad];
    S pht[RP][kC + kPad];
    float aw[kC];
    float a_state[RP];
};

template <class T, int D, int RP>
struct OutSmem {
    using S = typename T::store_t;
    S vt[D][kC + kPad];           // V chunk, transposed
    S phq[kC][RP + kPad];         // Phi_Q chunk
    S phk[kC][RP + kPad];         // Phi_K chunk (its transpose is read with transposed LDS reads)
    S mm[kC][kC + kPad];          // tril(Phi_Q Phi_K') / L
    float a_state[RP];
    float den_a[kC];
    float den_b[kC];
};

struct StateArgs {
    const float* U;       // projections of the feature rows [BH][N][RP/4]
    const void* Val;      // value rows [BH][N][D]
    const float* vscale;  // per-row value scale [BH][N] or null
    const float* aw;      // per-row weight of A [BH][N] or null (1)
    float* states;        // [BH][nseg][RP*D + RP]
    int H, N, L, seg_len, nseg;
    float two_beta, mul;
};

template <class T, int D, int RP>
__global__ __launch_bounds__(kThreads) void race_state_kernel(StateArgs a)
{
    using St = typename T::store_t;
    constexpr int DW = D / 64;
    constexpr int SPLIT = table_split<RP>(), RPW = RP / SPLIT;   // features of this workgroup
    __shared__ StateSmem<T, D, RPW> sm;
    const int seg = blockIdx.x / SPLIT, part = blockIdx.x % SPLIT, h = blockIdx.y, b = blockIdx.z;
    const int F0 = part * RPW, L = a.L - F0 / 16;                  // first feature; tables from here on
    const size_t bh = (size_t)b * a.H + h;
    const float* U = a.U + bh * a.N * (RP / 4) + F0 / 4;
    const St* Vl = (const St*)a.Val + bh * a.N * D;
    const float* vs = a.vscale ? a.vscale + bh * a.N : nullptr;
    const float* aw = a.aw ? a.aw + bh * a.N : nullptr;
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int g = lane >> 4, col = lane & 15;

    for (int f = threadIdx.x; f < RPW; f += kThreads) sm.a_state[f] = 0.f;
    f32x4 S[RPW / 16][DW];
#pragma unroll
    for (int ft = 0; ft < RPW / 16; ++ft)
#pragma unroll
        for (int j = 0; j < DW; ++j) S[ft][j] = f32x4{0, 0, 0, 0};

    const int t_beg = seg * a.seg_len, t_end = min(a.N, t_beg + a.seg_len);
    // projections, value rows and A weights of the chunk, loaded one chunk ahead
    URegs<RPW> ur;
    StageT<T, D> vr;
    float awv = 0.f;
    auto load_chunk = [&](int c0) {
        ur.load(U, c0, a.N, RP / 4);
        vr.load(Vl, c0, a.N, vs, 1.f);
        const int r = min(c0 + (int)threadIdx.x, a.N - 1);
        awv = aw ? aw[r] : 1.f;   // masked to the chunk's rows where stored
    };
    load_chunk(t_beg);
    for (int t0 = t_beg; t0 < t_end; t0 += kC) {
        __syncthreads();
        vr.store(sm.vt, vs != nullptr);
        if (threadIdx.x < kC) sm.aw[threadIdx.x] = t0 + (int)threadIdx.x < a.N ? awv : 0.f;
        features_from<T, RPW>(ur, t0, a.N, L, a.two_beta, nullptr, sm.pht, nullptr);
        __syncthreads();
        load_chunk(t0 + kC < t_end ? t0 + kC : t0);   // the last chunk reloads its own (unconditional loads)
        // S[f][cols of wave] += Phi'[f][rows] V[rows][cols]
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            typename T::frag_t bv[DW];
#pragma unroll
            for (int j = 0; j < DW; ++j) bv[j] = T::ld8(&sm.vt[16 * (w * DW + j) + col][32 * kk + 8 * g]);
#pragma unroll
            for (int ft = 0; ft < RPW / 16; ++ft) {
                const auto af = T::ld8(&sm.pht[16 * ft + col][32 * kk + 8 * g]);
#pragma unroll
                for (int j = 0; j < DW; ++j) S[ft][j] = T::mma(af, bv[j], S[ft][j]);
            }
        }
        for (int f = threadIdx.x; f < RPW; f += kThreads) {
            float s = 0.f;
            for (int k = 0; k < kC; ++k) s += T::load(sm.pht[f][k]) * sm.aw[k];
            sm.a_state[f] += s;
        }
    }
    __syncthreads();
    float* out = a.states + (bh * a.nseg + seg) * (size_t)(RP * D + RP);
#pragma unroll
    for (int ft = 0; ft < RPW / 16; ++ft)
#pragma unroll
        for (int j = 0; j < DW; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                out[(size_t)(F0 + 16 * ft + 4 * g + i) * D + 16 * (w * DW + j) + col] = S[ft][j][i] * a.mul;
    for (int f = threadIdx.x; f < RPW; f += kThreads) out[RP * D + F0 + f] = sm.a_state[f] * a.mul;
}

// mode 0: total in every segment; 1: exclusive prefix; 2: exclusive suffix.
// Each thread owns one element of the state and walks the segments in
// batches of kBatch independent loads.
__global__ __launch_bounds__(256) void race_scan_kernel(float* states, int nseg, int per, int mode)
{
    constexpr int kBatch = 16;
    const size_t bh = blockIdx.y;
    const int e = blockIdx.x * 256 + threadIdx.x;
    if (e >= per) return;
    float* base = states + bh * (size_t)nseg * per + e;
    float run = 0.f;
    for (int s0 = 0; s0 < nseg; s0 += kBatch) {
        float v[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            const int s = mode == 2 ? nseg - 1 - (s0 + j) : s0 + j;
            v[j] = (s0 + j < nseg) ? base[(size_t)s * per] : 0.f;
        }
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            if (s0 + j >= nseg) break;
            const int s = mode == 2 ? nseg - 1 - (s0 + j) : s0 + j;
            if (mode != 0) base[(size_t)s * per] = run;
            run += v[j];
        }
    }
    if (mode == 0)
        for (int s = 0; s < nseg; ++s) base[(size_t)s * per] = run;
}

struct OutArgs {
    const float* Uq;      // projections of Q rows [BH][N][RP/4]
    const float* Uk;      // projections of K rows
    const void* V;
    const float* states;
    void* O_lr;           // storage dtype [BH][N][D]
    float* d_lr;
    int H, N, L, seg_len, nseg, causal;
    float two_beta, inv_L, eps;
};

template <class T, int D, int RP>
__global__ __launch_bounds__(kThreads, 2) void race_out_kernel(OutArgs a)
{
    using St = typename T::store_t;
    using F = typename T::frag_t;
    constexpr int DW = D / 64;
    constexpr int FS = RP / 32;
    __shared__ OutSmem<T, D, RP> sm;
    const int seg = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const size_t bh = (size_t)b * a.H + h;
    const float* Uq = a.Uq + bh * a.N * (RP / 4);
    const float* Uk = a.Uk + bh * a.N * (RP / 4);
    const St* V = (const St*)a.V + bh * a.N * D;
    St* Olr = (St*)a.O_lr + bh * a.N * D;
    float* dlr = a.d_lr + bh * a.N;
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);   // wave-uniform, as in race_state
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
    for (int f = threadIdx.x; f < RP; f += kThreads) sm.a_state[f] = st_in[RP * D + f];
    // A runs on the matrix cores (causal): wave w keeps the feature tiles
    // ft = w, w + 4, ... in accumulator tiles (every column holds the sums;
    // column 0 starts from the segment's prefix state and is published to
    // a_state after each chunk)
    constexpr int FT = RP / 16, NFA = (FT + 3) / 4;
    f32x4 Aacc[NFA];
#pragma unroll
    for (int j = 0; j < NFA; ++j) {
        const int ft = w + 4 * j;
#pragma unroll
        for (int i = 0; i < 4; ++i) Aacc[j][i] = ft < FT && col == 0 ? st_in[RP * D + 16 * ft + 4 * g + i] : 0.f;
    }

    const int t_beg = seg * a.seg_len, t_end = min(a.N, t_beg + a.seg_len);
    URegs<RP> uq, uk;                    // projections and V rows of the chunk, loaded one chunk ahead
    StageT<T, D> vr;
    uq.load(Uq, t_beg, a.N);
    if (a.causal) uk.load(Uk, t_beg, a.N);
    vr.load(V, t_beg, a.N, nullptr, 1.f);
    for (int t0 = t_beg; t0 < t_end; t0 += kC) {
        __syncthreads();
        vr.store(sm.vt, false);
        features_from<T, RP>(uq, t0, a.N, a.L, a.two_beta, sm.phq, nullptr, nullptr);
        if (a.causal) features_from<T, RP>(uk, t0, a.N, a.L, a.two_beta, sm.phk, nullptr, nullptr);
        __syncthreads();
        {
            // next chunk's rows (the last chunk reloads its own: unconditional loads)
            const int tn = t0 + kC < t_end ? t0 + kC : t0;
            uq.load(Uq, tn, a.N);
            if (a.causal) uk.load(Uk, tn, a.N);
            vr.load(V, tn, a.N, nullptr, 1.f);
        }
        // Den, inter part: (1/L) Phi_Q . A   (4 threads per query)
        {
            const int q = threadIdx.x >> 2, part = threadIdx.x & 3;
            float s = 0.f;
#pragma unroll
            for (int f0 = part * (RP / 4); f0 < (part + 1) * (RP / 4); f0 += 8) {
                const auto ph = T::ld8(&sm.phq[q][f0]);
                const f32x4 a0 = *(const f32x4*)&sm.a_state[f0], a1 = *(const f32x4*)&sm.a_state[f0 + 4];
#pragma unroll
                for (int j = 0; j < 4; ++j) s += (float)ph[j] * a0[j] + (float)ph[4 + j] * a1[j];
            }
            s += __shfl_xor(s, 1);
            s += __shfl_xor(s, 2);
            if (part == 0) sm.den_a[q] = s * a.inv_L;
        }
        // intra-chunk kernel matrix rows [16w, 16w + 16) (causal), formed
        // transposed: lane (g, col) holds keys 16 kt + 4 g + i of query
        // 16 w + col, so a row's four entries leave in one store and its sum
        // is in-lane plus one exchange over the lane groups
        if (a.causal) {
            const int qi = 16 * w + col;
            float rs = 0.f;
            for (int kt = 0; kt < 4; ++kt) {
                f32x4 mt = {0, 0, 0, 0};
                if (kt <= w) {
#pragma unroll
                    for (int fs = 0; fs < FS; ++fs)
                        mt = T::mma(T::ld8(&sm.phk[16 * kt + col][32 * fs + 8 * g]),
                                    T::ld8(&sm.phq[16 * w + col][32 * fs + 8 * g]), mt);
                }
                f32x4 v;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int kj = 16 * kt + 4 * g + i;
                    v[i] = (kj <= qi) ? mt[i] * a.inv_L : 0.f;
                    rs += v[i];
                }
                store4<T>(&sm.mm[qi][16 * kt + 4 * g], v);
            }
            rs = wave_sum16(rs);
            if (g == 0) sm.den_b[qi] = rs;
        }
        __syncthreads();
        // Num^T for the wave's d columns, all 64 queries (lane (g, col) holds
        // d = 16 (w DW + j) + 4 g + i of query 16 qt + col): inter-chunk part
        // with S rounded to the storage dtype once per chunk (the forward
        // sums positive features against it, no cancellation), then the
        // masked intra-chunk part
        f32x4 num[4][DW];
#pragma unroll
        for (int qt = 0; qt < 4; ++qt)
#pragma unroll
            for (int j = 0; j < DW; ++j) num[qt][j] = f32x4{0, 0, 0, 0};
#pragma unroll
        for (int fs = 0; fs < FS; ++fs) {
            F sf[DW];
#pragma unroll
            for (int j = 0; j < DW; ++j) {
                float sv[8];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    sv[i] = S[2 * fs][j][i];
                    sv[4 + i] = S[2 * fs + 1][j][i];
                }
                sf[j] = T::pack(sv);
            }
#pragma unroll
            for (int qt = 0; qt < 4; ++qt) {
                const F af = T::ld44(&sm.phq[16 * qt + col][32 * fs + 4 * g],
                                     &sm.phq[16 * qt + col][32 * fs + 16 + 4 * g]);
#pragma unroll
                for (int j = 0; j < DW; ++j) num[qt][j] = T::mma(sf[j], af, num[qt][j]);
            }
        }
#pragma unroll
        for (int qt = 0; qt < 4; ++qt) {
#pragma unroll
            for (int j = 0; j < DW; ++j) num[qt][j] *= a.inv_L;
            if (a.causal) {
#pragma unroll
                for (int kk = 0; kk < 2; ++kk) {
                    const F bf = T::ld8(&sm.mm[16 * qt + col][32 * kk + 8 * g]);
#pragma unroll
                    for (int j = 0; j < DW; ++j)
                        num[qt][j] = T::mma(T::ld8(&sm.vt[16 * (w * DW + j) + col][32 * kk + 8 * g]), bf, num[qt][j]);
                }
            }
            const int ql = 16 * qt + col;
            const int tok = t0 + ql;
            if (tok < a.N) {
                const float den = sm.den_a[ql] + (a.causal ? sm.den_b[ql] : 0.f);
                const float inv = 1.f / (den + a.eps);
#pragma unroll
                for (int j = 0; j < DW; ++j)
                    store4<T>(Olr + (size_t)tok * D + 16 * (w * DW + j) + 4 * g, num[qt][j] * inv);
            }
        }
        if (threadIdx.x < kC && t0 + threadIdx.x < a.N)
            dlr[t0 + threadIdx.x] = sm.den_a[threadIdx.x] + (a.causal ? sm.den_b[threadIdx.x] : 0.f);
        if (a.causal) {
            // S += Phi_K' V (chunk), A += Phi_K' 1
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                F bv[DW];
#pragma unroll
                for (int j = 0; j < DW; ++j) bv[j] = T::ld8(&sm.vt[16 * (w * DW + j) + col][32 * kk + 8 * g]);
#pragma unroll
                for (int ft = 0; ft < FT; ++ft) {
                    const F af = phi_t8<T, RP>(sm.phk, 32 * kk, 16 * ft);
#pragma unroll
                    for (int j = 0; j < DW; ++j) S[ft][j] = T::mma(af, bv[j], S[ft][j]);
                    if (ft % 4 == w) Aacc[ft / 4] = token_sums<T>(af, Aacc[ft / 4]);
                }
            }
            // the den of the next chunk reads a_state after its first barrier
#pragma unroll
            for (int j = 0; j < NFA; ++j) {
                const int ft = w + 4 * j;
                if (ft < FT && col == 0)
#pragma unroll
                    for (int i = 0; i < 4; ++i) sm.a_state[16 * ft + 4 * g + i] = Aacc[j][i];
            }
        }
    }
}

template <class T, int D, int RP>
constexpr bool fits()
{
    return sizeof(StateSmem<T, D, RP / table_split<RP>()>) <= kMaxLds && sizeof(OutSmem<T, D, RP>) <= kMaxLds;
}

template <class T, int D, int RP>
hipError_t launch_states_t(const Shape& s, const StateArgs& a, int scan_mode, hipStream_t st)
{
    if constexpr (!fits<T, D, RP>()) {
        return hipErrorInvalidConfiguration;
    } else {
        dim3 grid(s.nseg * table_split<RP>(), s.H, s.B);
        // the forward sums key rows, the backward (vscale set) query rows
        const bool bwd = a.vscale != nullptr;
        ELSAA_LAUNCH(bwd ? "race_state_bwd" : "race_state_fwd", (race_state_kernel<T, D, RP>), grid, dim3(kThreads),
                     0, st, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int per = RP * D + RP;
        ELSAA_LAUNCH(bwd ? "race_scan_bwd" : "race_scan_fwd", race_scan_kernel, dim3((per + 255) / 256, s.B * s.H), dim3(256), 0, st,
                           a.states, s.nseg, per, scan_mode);
        return hipGetLastError();
    }
}

template <class T, int D, int RP>
hipError_t launch_out_t(const Shape& s, const OutArgs& a, hipStream_t st)
{
    if constexpr (!fits<T, D, RP>()) {
        return hipErrorInvalidConfiguration;
    } else {
        dim3 grid(s.nseg, s.H, s.B);
        ELSAA_LAUNCH("race_out", (race_out_kernel<T, D, RP>), grid, dim3(kThreads), 0, st, a);
        return hipGetLastError();
    }
}

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

template <class T, int D, int RP>
struct StatesFn {
    static hipError_t run(const Shape& s, const StateArgs& a, int mode, hipStream_t st)
    {
        return launch_states_t<T, D, RP>(s, a, mode, st);
    }
};

template <class T, int D, int RP>
struct OutFn {
    static hipError_t run(const Shape& s, const OutArgs& a, hipStream_t st) { return launch_out_t<T, D, RP>(s, a, st); }
};

template <class T, int D, int RP>
struct FitsFn {
    static hipError_t run(const Shape&) { return fits<T, D, RP>() ? hipSuccess : hipErrorInvalidConfiguration; }
};

}  // namespace

// Padded feature count of the GPU path: r rounded up to 32, 64, 128 or 256.
int race_padded_features(int r) { return r <= 32 ? 32 : r <= 64 ? 64 : r <= 128 ? 128 : 256; }

size_t race_state_floats(const Shape& s)
{
    const int rp = race_padded_features(s.r);
    return (size_t)s.B * s.H * s.nseg * ((size_t)rp * s.D + rp);
}

bool race_fwd_fits(const Shape& s) { return dispatch<FitsFn>(s) == hipSuccess; }

int race_proj_stride(const Shape& s) { return race_padded_features(s.r) / 4; }

hipError_t launch_race_states(const Shape& s, const float* U, const void* Val, const float* vscale,
                              const float* aw, float mul, float* states, int scan_mode, hipStream_t st)
{
    StateArgs a;
    a.U = U; a.Val = Val; a.vscale = vscale; a.aw = aw; a.states = states;
    a.H = s.H; a.N = s.N; a.L = s.L; a.seg_len = s.seg_len; a.nseg = s.nseg;
    a.two_beta = 2.f * s.beta; a.mul = mul;
    return dispatch<StatesFn>(s, a, scan_mode, st);
}

hipError_t launch_race_fwd(const Shape& s, const float* Uq, const float* Uk, const void* V,
                           float* states, void* O_lr, float* d_lr, hipStream_t st)
{
    hipError_t e = launch_race_states(s, Uk, V, nullptr, nullptr, 1.f, states, s.causal ? 1 : 0, st);
    if (e != hipSuccess) return e;
    OutArgs a;
    a.Uq = Uq; a.Uk = Uk; a.V = V; a.states = states;
    a.O_lr = O_lr; a.d_lr = d_lr;
    a.H = s.H; a.N = s.N; a.L = s.L; a.seg_len = s.seg_len; a.nseg = s.nseg; a.causal = s.causal;
    a.two_beta = 2.f * s.beta; a.inv_L = 1.f / (float)s.L; a.eps = s.eps;
    return dispatch<OutFn>(s, a, st);
}

}  // namespace elsaa
