// race_fwd.hip -- RACE low-rank branch forward (Alg. 2; causal chunked form Alg. 3).
//
// Features (Alg. 2): for table l, u = W_l x (race_bits = 4 projections),
// t = tanh(u), and for bucket c of the 2^4-vertex hypercube
//   phi_c = exp(beta t.v_c) / sum_c' exp(beta t.v_c') = prod_b sigmoid(2 beta v_cb t_b)
// (the softmax over {+-1}^4 factorises per bit).  Num = (1/L) sum_l Phi_Q^l B^l,
// Den = (1/L) sum_l Phi_Q^l A^l with A^l = Phi_K^l' 1, B^l = Phi_K^l' V; the
// causal form restricts both sums to keys j <= i.  O_lr = Num / (Den + eps),
// d_lr = Den.
//
// The sequence of each (b,h) is cut into segments of whole 64-token chunks:
//   phase A  one workgroup per segment: the segment's state
//            S = sum_j phi(k_j) v_j' (r x d) and A = sum_j phi(k_j);
//   phase B  per (b,h): exclusive prefix of the segment states (causal), or
//            the total written to every segment (non-causal);
//   phase C  one workgroup per segment: starting from its prefix state, each
//            chunk computes Num = (1/L) Phi_Q S + tril(Phi_Q Phi_K'/L) V
//            (the masked part only when causal), then adds the chunk to S.
// Within a workgroup each of the 4 waves owns d/4 columns of S, kept as
// matrix-core accumulators (float32) for the whole segment.  Projections,
// the intra-chunk kernel matrix and all contractions run on MFMA with
// bf16 (or float32) operands and float32 accumulation.
#include "common.hpp"
#include "internal.hpp"

namespace elsaa {

namespace {

constexpr int kC = 64;          // chunk length (tokens)
constexpr int kThreads = 256;
constexpr int kPad = 8;
constexpr size_t kMaxLds = 160 * 1024;

// projection rows held in LDS: 4 per table, padded to whole 16-row MFMA tiles
template <int RP>
constexpr int w_rows() { return RP / 4 < 16 ? 16 : RP / 4; }

template <class T, int D, int RP>
struct RaceSmem {
    using S = typename T::store_t;
    S w[w_rows<RP>()][D + kPad];    // projection rows (4 per table), padded tables are zero
    S vt[D][kC + kPad];             // V chunk, transposed
    S phq[kC][RP + kPad];           // Phi_Q chunk (row-major)
    S phk[kC][RP + kPad];           // Phi_K chunk (row-major)
    S phkt[RP][kC + kPad];          // Phi_K chunk, transposed
    S mm[kC][kC + kPad];            // intra-chunk kernel matrix (masked, / L)
    float a_state[RP];
    float den_a[kC];
    float den_b[kC];
};

struct RArgs {
    const void* Q;
    const void* K;
    const void* V;
    const float* W;     // [H][L][4][D]
    float* states;      // [B*H][nseg][RP*D + RP]
    void* O_lr;
    float* d_lr;
    int H, N, L, seg_len, nseg, causal;
    float two_beta, inv_L, eps;
};

template <class T, int D, int RP>
__device__ void load_w(RaceSmem<T, D, RP>& sm, const float* W, int L)
{
    // rows 4*l + b for l < L, zero for padded tables
    for (int it = threadIdx.x; it < w_rows<RP>() * D; it += kThreads) {
        const int row = it / D, c = it % D;
        const float v = (row < 4 * L) ? W[(size_t)row * D + c] : 0.f;
        sm.w[row][c] = T::store(v);
    }
}

template <class T, int D, int RP>
__device__ void load_vt(RaceSmem<T, D, RP>& sm, const typename T::store_t* V, int t0, int N)
{
    using S = typename T::store_t;
    constexpr int PER = 16 / T::bytes;
    constexpr int CH = D / PER;
    for (int it = threadIdx.x; it < (kC / 2) * CH; it += kThreads) {
        const int p = it & (kC / 2 - 1), c = it / (kC / 2);
        const int r0 = t0 + 2 * p, r1 = r0 + 1;
        uint4 a = make_uint4(0, 0, 0, 0), b = make_uint4(0, 0, 0, 0);
        if (r0 < N) a = ldg16(V + (size_t)r0 * D + c * PER);
        if (r1 < N) b = ldg16(V + (size_t)r1 * D + c * PER);
        const S* ea = (const S*)&a;
        const S* eb = (const S*)&b;
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            S* dst = &sm.vt[c * PER + j][2 * p];
            dst[0] = ea[j];
            dst[1] = eb[j];
        }
    }
}

// Features of the 16 tokens [t0 + 16w, t0 + 16w + 16) of X for every table.
// Writes Phi row-major (and transposed when kt) into LDS.
template <class T, int D, int RP>
__device__ void features(RaceSmem<T, D, RP>& sm, const typename T::store_t* X, int t0, int N,
                         int L, float two_beta, typename T::store_t (*ph)[RP + kPad],
                         typename T::store_t (*pht)[kC + kPad])
{
    using F = typename T::frag_t;
    constexpr int KS = D / 32;
    constexpr int PT = w_rows<RP>() / 16;   // projection row tiles of 16 rows = 4 tables
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int g = lane >> 4, col = lane & 15;
    const int tl = 16 * w + col;        // token within the chunk
    const int tok = t0 + tl;
    F xf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        if (tok < N) xf[ks] = T::ld8(X + (size_t)tok * D + 32 * ks + 8 * g);
        else {
            float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            xf[ks] = T::pack(z);
        }
    }
#pragma unroll
    for (int pt = 0; pt < PT; ++pt) {
        f32x4 u = {0, 0, 0, 0};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) u = T::mma(T::ld8(&sm.w[16 * pt + col][32 * ks + 8 * g]), xf[ks], u);
        // lane holds the 4 projections of table 4*pt + g for token tl
        const int tb = 4 * pt + g;
        float sp[4], sn[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float t = tanhf(u[i]);
            sp[i] = 1.f / (1.f + __expf(-two_beta * t));
            sn[i] = 1.f / (1.f + __expf(two_beta * t));
        }
        const bool live = tb < L && tok < N;
        float phi[16];
#pragma unroll
        for (int c = 0; c < 16; ++c) {
            float v = ((c & 1) ? sp[0] : sn[0]) * ((c & 2) ? sp[1] : sn[1]) *
                      ((c & 4) ? sp[2] : sn[2]) * ((c & 8) ? sp[3] : sn[3]);
            phi[c] = live ? v : 0.f;
        }
        if (tb < RP / 16) {
#pragma unroll
            for (int c = 0; c < 16; ++c) ph[tl][16 * tb + c] = T::store(phi[c]);
            if (pht) {
#pragma unroll
                for (int c = 0; c < 16; ++c) pht[16 * tb + c][tl] = T::store(phi[c]);
            }
        }
    }
}

// S[f][cols of wave] += Phi_K'[f][keys] V[keys][cols]; A[f] += sum_k Phi_K[k][f]
template <class T, int D, int RP>
__device__ __forceinline__ void update_state(RaceSmem<T, D, RP>& sm, f32x4 (&S)[RP / 16][D / 64])
{
    constexpr int DW = D / 64;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int g = lane >> 4, col = lane & 15;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
        typename T::frag_t bv[DW];
#pragma unroll
        for (int j = 0; j < DW; ++j) bv[j] = T::ld8(&sm.vt[16 * (w * DW + j) + col][32 * kk + 8 * g]);
#pragma unroll
        for (int ft = 0; ft < RP / 16; ++ft) {
            const auto af = T::ld8(&sm.phkt[16 * ft + col][32 * kk + 8 * g]);
#pragma unroll
            for (int j = 0; j < DW; ++j) S[ft][j] = T::mma(af, bv[j], S[ft][j]);
        }
    }
    for (int f = threadIdx.x; f < RP; f += kThreads) {
        float s = 0.f;
        for (int k = 0; k < kC; ++k) s += T::load(sm.phkt[f][k]);
        sm.a_state[f] += s;
    }
}

template <class T, int D, int RP>
__global__ __launch_bounds__(kThreads) void race_state_kernel(RArgs a)
{
    using St = typename T::store_t;
    constexpr int DW = D / 64;
    __shared__ RaceSmem<T, D, RP> sm;
    const int seg = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const size_t bh = (size_t)b * a.H + h;
    const St* K = (const St*)a.K + bh * a.N * D;
    const St* V = (const St*)a.V + bh * a.N * D;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int g = lane >> 4, col = lane & 15;

    load_w<T, D, RP>(sm, a.W + (size_t)h * a.L * 4 * D, a.L);
    for (int f = threadIdx.x; f < RP; f += kThreads) sm.a_state[f] = 0.f;
    f32x4 S[RP / 16][DW];
#pragma unroll
    for (int ft = 0; ft < RP / 16; ++ft)
#pragma unroll
        for (int j = 0; j < DW; ++j) S[ft][j] = f32x4{0, 0, 0, 0};

    const int t_beg = seg * a.seg_len, t_end = min(a.N, t_beg + a.seg_len);
    for (int t0 = t_beg; t0 < t_end; t0 += kC) {
        __syncthreads();
        load_vt<T, D, RP>(sm, V, t0, a.N);
        features<T, D, RP>(sm, K, t0, a.N, a.L, a.two_beta, sm.phk, sm.phkt);
        __syncthreads();
        update_state<T, D, RP>(sm, S);
    }
    __syncthreads();
    float* out = a.states + (bh * a.nseg + seg) * (size_t)(RP * D + RP);
#pragma unroll
    for (int ft = 0; ft < RP / 16; ++ft)
#pragma unroll
        for (int j = 0; j < DW; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                out[(size_t)(16 * ft + 4 * g + i) * D + 16 * (w * DW + j) + col] = S[ft][j][i];
    for (int f = threadIdx.x; f < RP; f += kThreads) out[RP * D + f] = sm.a_state[f];
}

// Exclusive prefix over segments (causal) or the total in every segment.
__global__ __launch_bounds__(256) void race_scan_kernel(float* states, int nseg, int per, int causal)
{
    const size_t bh = blockIdx.y;
    const int e = blockIdx.x * 256 + threadIdx.x;
    if (e >= per) return;
    float* base = states + bh * (size_t)nseg * per + e;
    float run = 0.f;
    for (int s = 0; s < nseg; ++s) {
        const float v = base[(size_t)s * per];
        if (causal) base[(size_t)s * per] = run;
        run += v;
    }
    if (!causal)
        for (int s = 0; s < nseg; ++s) base[(size_t)s * per] = run;
}

template <class T, int D, int RP>
__global__ __launch_bounds__(kThreads) void race_out_kernel(RArgs a)
{
    using St = typename T::store_t;
    using F = typename T::frag_t;
    constexpr int DW = D / 64;
    constexpr int FS = RP / 32;   // 32-feature k-steps
    __shared__ RaceSmem<T, D, RP> sm;
    const int seg = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const size_t bh = (size_t)b * a.H + h;
    const St* Q = (const St*)a.Q + bh * a.N * D;
    const St* K = (const St*)a.K + bh * a.N * D;
    const St* V = (const St*)a.V + bh * a.N * D;
    St* Olr = (St*)a.O_lr + bh * a.N * D;
    float* dlr = a.d_lr + bh * a.N;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int g = lane >> 4, col = lane & 15;

    load_w<T, D, RP>(sm, a.W + (size_t)h * a.L * 4 * D, a.L);
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

    const int t_beg = seg * a.seg_len, t_end = min(a.N, t_beg + a.seg_len);
    for (int t0 = t_beg; t0 < t_end; t0 += kC) {
        __syncthreads();
        load_vt<T, D, RP>(sm, V, t0, a.N);
        features<T, D, RP>(sm, Q, t0, a.N, a.L, a.two_beta, sm.phq, nullptr);
        if (a.causal) features<T, D, RP>(sm, K, t0, a.N, a.L, a.two_beta, sm.phk, sm.phkt);
        __syncthreads();
        // Den, inter part: (1/L) Phi_Q . A   (4 threads per query)
        {
            const int q = threadIdx.x >> 2, part = threadIdx.x & 3;
            float s = 0.f;
            for (int f = part * (RP / 4); f < (part + 1) * (RP / 4); ++f)
                s += T::load(sm.phq[q][f]) * sm.a_state[f];
            s += __shfl_xor(s, 1);
            s += __shfl_xor(s, 2);
            if (part == 0) sm.den_a[q] = s * a.inv_L;
        }
        // intra-chunk kernel matrix rows [16w, 16w + 16) (causal)
        if (a.causal) {
            float rs[4] = {0, 0, 0, 0};
            for (int kt = 0; kt < 4; ++kt) {
                f32x4 mt = {0, 0, 0, 0};
                if (kt <= w) {
#pragma unroll
                    for (int fs = 0; fs < FS; ++fs)
                        mt = T::mma(T::ld8(&sm.phq[16 * w + col][32 * fs + 8 * g]),
                                    T::ld8(&sm.phk[16 * kt + col][32 * fs + 8 * g]), mt);
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int qi = 16 * w + 4 * g + i, kj = 16 * kt + col;
                    const float v = (kj <= qi) ? mt[i] * a.inv_L : 0.f;
                    rs[i] += v;
                    sm.mm[qi][kj] = T::store(v);
                }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float s = row_sum16(rs[i]);
                if (col == 0) sm.den_b[16 * w + 4 * g + i] = s;
            }
        }
        __syncthreads();
        // Num for the wave's d columns, all 64 queries
#pragma unroll
        for (int qt = 0; qt < 4; ++qt) {
            f32x4 num[DW];
#pragma unroll
            for (int j = 0; j < DW; ++j) num[j] = f32x4{0, 0, 0, 0};
#pragma unroll
            for (int fs = 0; fs < FS; ++fs) {
                const F af = T::ld44(&sm.phq[16 * qt + col][32 * fs + 4 * g],
                                     &sm.phq[16 * qt + col][32 * fs + 16 + 4 * g]);
#pragma unroll
                for (int j = 0; j < DW; ++j) {
                    float sv[8];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        sv[i] = S[2 * fs][j][i];
                        sv[4 + i] = S[2 * fs + 1][j][i];
                    }
                    num[j] = T::mma(af, T::pack(sv), num[j]);
                }
            }
#pragma unroll
            for (int j = 0; j < DW; ++j) num[j] *= a.inv_L;
            if (a.causal) {
#pragma unroll
                for (int kk = 0; kk < 2; ++kk) {
                    const F af = T::ld8(&sm.mm[16 * qt + col][32 * kk + 8 * g]);
#pragma unroll
                    for (int j = 0; j < DW; ++j)
                        num[j] = T::mma(af, T::ld8(&sm.vt[16 * (w * DW + j) + col][32 * kk + 8 * g]), num[j]);
                }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int ql = 16 * qt + 4 * g + i;
                const int tok = t0 + ql;
                if (tok >= a.N) continue;
                const float den = sm.den_a[ql] + (a.causal ? sm.den_b[ql] : 0.f);
                const float inv = 1.f / (den + a.eps);
#pragma unroll
                for (int j = 0; j < DW; ++j) Olr[(size_t)tok * D + 16 * (w * DW + j) + col] = T::store(num[j][i] * inv);
            }
        }
        if (threadIdx.x < kC && t0 + threadIdx.x < a.N)
            dlr[t0 + threadIdx.x] = sm.den_a[threadIdx.x] + (a.causal ? sm.den_b[threadIdx.x] : 0.f);
        if (a.causal) update_state<T, D, RP>(sm, S);
    }
}

template <class T, int D, int RP>
hipError_t launch_t(const Shape& s, const RArgs& a, hipStream_t st)
{
    if constexpr (sizeof(RaceSmem<T, D, RP>) > kMaxLds) {
        return hipErrorInvalidConfiguration;   // rejected earlier by the host validation
    } else {
    dim3 grid(s.nseg, s.H, s.B);
    hipLaunchKernelGGL((race_state_kernel<T, D, RP>), grid, dim3(kThreads), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int per = RP * D + RP;
    hipLaunchKernelGGL(race_scan_kernel, dim3((per + 255) / 256, s.B * s.H), dim3(256), 0, st,
                       a.states, s.nseg, per, s.causal);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((race_out_kernel<T, D, RP>), grid, dim3(kThreads), 0, st, a);
    return hipGetLastError();
    }
}

template <class T, int D>
hipError_t launch_d(const Shape& s, const RArgs& a, hipStream_t st)
{
    switch (s.Lp * 16) {
        case 32: return launch_t<T, D, 32>(s, a, st);
        case 64: return launch_t<T, D, 64>(s, a, st);
        case 128: return launch_t<T, D, 128>(s, a, st);
        default: return launch_t<T, D, 256>(s, a, st);
    }
}

}  // namespace

// Padded feature count of the GPU path: r rounded up to 32, 64, 128 or 256.
int race_padded_features(int r)
{
    return r <= 32 ? 32 : r <= 64 ? 64 : r <= 128 ? 128 : 256;
}

bool race_fits(int bf16, int D, int r)
{
    const int rp = race_padded_features(r);
    const size_t es = bf16 ? 2 : 4;
    const size_t wr = rp / 4 < 16 ? 16 : rp / 4;
    const size_t bytes = es * (wr * (D + kPad) + (size_t)D * (kC + kPad) + 2 * (size_t)kC * (rp + kPad) +
                               (size_t)rp * (kC + kPad) + (size_t)kC * (kC + kPad)) +
                         4 * ((size_t)rp + 2 * kC);
    return bytes <= kMaxLds;
}

size_t race_state_floats(const Shape& s)
{
    const int rp = race_padded_features(s.r);
    return (size_t)s.B * s.H * s.nseg * ((size_t)rp * s.D + rp);
}

hipError_t launch_race_fwd(const Shape& s, const void* Q, const void* K, const void* V,
                           const float* W_race, float* states, void* O_lr, float* d_lr,
                           hipStream_t st)
{
    RArgs a;
    a.Q = Q; a.K = K; a.V = V; a.W = W_race;
    a.states = states; a.O_lr = O_lr; a.d_lr = d_lr;
    a.H = s.H; a.N = s.N; a.L = s.L; a.seg_len = s.seg_len; a.nseg = s.nseg; a.causal = s.causal;
    a.two_beta = 2.f * s.beta; a.inv_L = 1.f / (float)s.L; a.eps = s.eps;
    if (s.bf16) return s.D == 64 ? launch_d<BF16, 64>(s, a, st) : launch_d<BF16, 128>(s, a, st);
    return s.D == 64 ? launch_d<F32, 64>(s, a, st) : launch_d<F32, 128>(s, a, st);
}

}  // namespace elsaa
