// select.hip -- sortLSH selection (sign hash, per-segment stable sort) and
// the RACE projections of the same rows.
//
// Hash (Alg. 4, step "Hash"): bit t of row x is set iff the float32 fused
// multiply-add chain over e = 0..d-1 of W_sort[h][t][e] * x[e] is > 0; the key
// is the rank of the bit code in the reflected Gray sequence so neighbouring
// buckets differ in one bit (sorted Hamming LSH, Sec. 3).  The same pass over
// Q or K also computes the RACE projections u = W_race x (Alg. 2), so each
// input row is read once for both branches' hashing.
// Sort (Alg. 4, step "Sort"; one call per half-segment of each level of
// Alg. 5): ascending by (key, token index), i.e. a stable counting sort over
// at most 2^sort_bits buckets, one workgroup per sorted list.
#include "common.hpp"
#include "internal.hpp"

namespace elsaa {

constexpr int kProjRows = 64;
constexpr int kProjThreads = 256;
constexpr int kProjPad = 8;

// Per 64-row tile of X (Q or K of one (b,h)): the sortLSH bucket key of every
// row and, when W_race is given, the RACE projections u = W_race x of every
// row in float32 accuracy: W = W_hi + W_lo split into two bf16 parts for the
// bf16 MFMA path (the residual is below 2^-16 relative), plain float32 MFMA
// for float32 storage.  u is stored [BH][N][UP] (UP = padded projections).
template <class T, int D, int WR>
struct ProjSmem {
    typename T::store_t x[kProjRows][D + kProjPad];
    typename T::store_t whi[WR][D + kProjPad];
    typename T::store_t wlo[T::bytes == 2 ? WR : 1][D + kProjPad];   // (no low part for float32)
    float ws[8][D];
    uint32_t code[kProjRows];
};

template <class T, int D, int WR>
__global__ __launch_bounds__(kProjThreads) void proj_kernel(const typename T::store_t* __restrict__ X,
                                                            const float* __restrict__ Wsort,
                                                            const float* __restrict__ Wrace,
                                                            uint8_t* __restrict__ keys,
                                                            float* __restrict__ U, int H, int N,
                                                            int bits, int L, int UP)
{
    using S = typename T::store_t;
    using F = typename T::frag_t;
    constexpr int PER = 16 / T::bytes;
    constexpr int CH = D / PER;
    constexpr int KS = D / 32;
    __shared__ ProjSmem<T, D, WR> sm;
    const int h = blockIdx.y, b = blockIdx.z;
    const int row0 = blockIdx.x * kProjRows;
    const int rows = min(kProjRows, N - row0);
    const size_t bh = (size_t)b * H + h;
    const S* Xt = X + (bh * N + row0) * D;
    for (int e = threadIdx.x; e < bits * D; e += kProjThreads) sm.ws[e / D][e % D] = Wsort[(size_t)h * bits * D + e];
    for (int it = threadIdx.x; it < kProjRows * CH; it += kProjThreads) {
        const int r = it / CH, c = it % CH;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (r < rows) v = ldg16(Xt + (size_t)r * D + c * PER);
        *(uint4*)&sm.x[r][c * PER] = v;
    }
    if (threadIdx.x < kProjRows) sm.code[threadIdx.x] = 0;
    if (Wrace) {
        for (int it = threadIdx.x; it < WR * D; it += kProjThreads) {
            const int row = it / D, c = it % D;
            const float w = row < 4 * L ? Wrace[((size_t)h * L * 4 + row) * D + c] : 0.f;
            const S hi = T::store(w);
            sm.whi[row][c] = hi;
            if (T::bytes == 2) sm.wlo[row][c] = T::store(w - T::load(hi));
        }
    }
    __syncthreads();
    // hash: thread (row, bit group) runs the float32 fma chains of its bits
    // over the row, read from LDS in 16-byte pieces
    {
        const int r = threadIdx.x & (kProjRows - 1);
        uint32_t c = 0;
        for (int bit = threadIdx.x / kProjRows; bit < bits; bit += kProjThreads / kProjRows) {
            float p = 0.0f;
#pragma unroll 4
            for (int e0 = 0; e0 < D; e0 += PER) {
                const uint4 v = *(const uint4*)&sm.x[r][e0];
                const S* xs = (const S*)&v;
#pragma unroll
                for (int j = 0; j < PER; ++j) p = __builtin_fmaf(sm.ws[bit][e0 + j], T::load(xs[j]), p);
            }
            if (p > 0.0f) c |= 1u << bit;
        }
        if (c) atomicOr(&sm.code[r], c);
    }
    __syncthreads();
    if (threadIdx.x < rows) {
        const uint32_t code = sm.code[threadIdx.x];
        uint32_t rank = code;
        for (uint32_t sft = code >> 1; sft; sft >>= 1) rank ^= sft;
        keys[bh * N + row0 + threadIdx.x] = (uint8_t)rank;
    }
    if (!Wrace) return;
    // u[token][p] for the wave's 16 tokens: A = W rows, B = X rows
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int g = lane >> 4, col = lane & 15;
    const int tl = 16 * w + col;
    F xf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) xf[ks] = T::ld8(&sm.x[tl][32 * ks + 8 * g]);
#pragma unroll
    for (int pt = 0; pt < WR / 16; ++pt) {
        f32x4 acc = {0, 0, 0, 0};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            acc = T::mma(T::ld8(&sm.whi[16 * pt + col][32 * ks + 8 * g]), xf[ks], acc);
            if (T::bytes == 2) acc = T::mma(T::ld8(&sm.wlo[16 * pt + col][32 * ks + 8 * g]), xf[ks], acc);
        }
        const int p0 = 16 * pt + 4 * g;
        if (tl < rows && p0 < UP) *(f32x4*)(U + (bh * N + row0 + tl) * UP + p0) = acc;
    }
}

template <class T, int D>
hipError_t launch_proj_t(const Shape& s, const void* X, const float* W_sort, const float* W_race,
                         uint8_t* keys, float* U, hipStream_t st)
{
    dim3 grid((s.N + kProjRows - 1) / kProjRows, s.H, s.B);
    const int UP = race_proj_stride(s);
    const int wr = UP < 16 ? 16 : UP;
#define ELSAA_PROJ(WR_)                                                                          \
    ELSAA_LAUNCH("project", (proj_kernel<T, D, WR_>), grid, dim3(kProjThreads), 0, st,                 \
                       (const typename T::store_t*)X, W_sort, W_race, keys, U, s.H, s.N,          \
                       s.sort_bits, s.L, UP)
    if (wr == 16) ELSAA_PROJ(16);
    else if (wr == 32) ELSAA_PROJ(32);
    else ELSAA_PROJ(64);
#undef ELSAA_PROJ
    return hipGetLastError();
}

hipError_t launch_project(const Shape& s, const void* X, const float* W_sort, const float* W_race,
                          uint8_t* keys, float* U, hipStream_t st)
{
    if (s.bf16) return s.D == 64 ? launch_proj_t<BF16, 64>(s, X, W_sort, W_race, keys, U, st)
                                 : launch_proj_t<BF16, 128>(s, X, W_sort, W_race, keys, U, st);
    return s.D == 64 ? launch_proj_t<F32, 64>(s, X, W_sort, W_race, keys, U, st)
                     : launch_proj_t<F32, 128>(s, X, W_sort, W_race, keys, U, st);
}

// --------------------------------------------------------------------------
// Stable counting sort, one workgroup per list.
// Lists of one (b,h):
//   non-causal: task 0 = all queries, task 1 = all keys;
//   causal: level l has 2^l segments of length n = N >> l; task (l, s, q/k)
//           sorts the future half [a + n/2, a + n) of the query keys or the
//           past half [a, a + n/2) of the key keys, a = s * n.
// --------------------------------------------------------------------------

constexpr int kSortThreads = 256;
constexpr int kSortWaves = kSortThreads / kWave;

__global__ __launch_bounds__(kSortThreads) void sort_kernel(const uint8_t* __restrict__ keyq,
                                                            const uint8_t* __restrict__ keyk,
                                                            int32_t* __restrict__ perm_q,
                                                            int32_t* __restrict__ perm_k, int H,
                                                            int N, int causal, int Lv, int bits)
{
    __shared__ int hist[256];
    __shared__ int base[256];
    __shared__ int cnt[kSortWaves][256];
    const int h = blockIdx.y, b = blockIdx.z;
    const int task = blockIdx.x;
    const int nb = 1 << bits;
    const size_t bh = (size_t)b * H + h;

    int start, len, is_k;
    size_t out_off;
    if (!causal) {
        is_k = task;
        start = 0;
        len = N;
        out_off = bh * N;
    } else {
        // level l owns tasks [2^(l+1) - 2, 2^(l+2) - 2)
        int l = 31 - __clz(task + 2) - 1;
        int t2 = task - ((1 << (l + 1)) - 2);
        int seg = t2 >> 1;
        is_k = t2 & 1;
        int n = N >> l, half = n >> 1;
        int a = seg * n;
        start = is_k ? a : a + half;
        len = half;
        // causal lists: [b,h][Lv][N/2]; level l, segment seg starts at seg * half
        out_off = (bh * Lv + l) * (size_t)(N / 2) + (size_t)seg * half;
    }
    const uint8_t* key = (is_k ? keyk : keyq) + bh * N + start;
    int32_t* out = (is_k ? perm_k : perm_q) + out_off;

    for (int i = threadIdx.x; i < nb; i += kSortThreads) hist[i] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < len; i += kSortThreads) atomicAdd(&hist[key[i]], 1);
    __syncthreads();
    if (threadIdx.x == 0) {
        int acc = 0;
        for (int i = 0; i < nb; ++i) { base[i] = acc; acc += hist[i]; }
    }
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
    for (int c0 = 0; c0 < len; c0 += kSortThreads) {
        for (int i = threadIdx.x; i < kSortWaves * nb; i += kSortThreads) cnt[i / nb][i % nb] = 0;
        __syncthreads();
        const int i = c0 + threadIdx.x;
        const bool valid = i < len;
        const int kk = valid ? key[i] : 0;
        // lanes of this wave holding the same key
        uint64_t same = __ballot(valid);
        for (int bit = 0; bit < bits; ++bit) {
            uint64_t ones = __ballot(valid && ((kk >> bit) & 1));
            same &= ((kk >> bit) & 1) ? ones : ~ones;
        }
        const int rank_in_wave = __popcll(same & lt);
        if (valid && rank_in_wave == 0) cnt[wave][kk] = __popcll(same);
        __syncthreads();
        if (valid) {
            int pos = base[kk] + rank_in_wave;
            for (int w = 0; w < wave; ++w) pos += cnt[w][kk];
            out[pos] = start + i;
        }
        __syncthreads();
        for (int k2 = threadIdx.x; k2 < nb; k2 += kSortThreads) {
            int add = 0;
            for (int w = 0; w < kSortWaves; ++w) add += cnt[w][k2];
            base[k2] += add;
        }
        __syncthreads();
    }
}

hipError_t launch_sort(const Shape& s, const uint8_t* keyq, const uint8_t* keyk, int32_t* perm_q,
                       int32_t* perm_k, hipStream_t st)
{
    const int tasks = s.causal ? (1 << (s.Lv + 1)) - 2 : 2;
    if (tasks <= 0) return hipSuccess;
    dim3 grid(tasks, s.H, s.B);
    ELSAA_LAUNCH("sort", sort_kernel, grid, dim3(kSortThreads), 0, st, keyq, keyk, perm_q, perm_k,
                       s.H, s.N, s.causal, s.Lv, s.sort_bits);
    return hipGetLastError();
}

}  // namespace elsaa
