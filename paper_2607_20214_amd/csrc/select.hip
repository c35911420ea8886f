// select.hip -- sortLSH selection: sign hash and per-segment stable sort.
//
// Hash (Alg. 4, step "Hash"): bit t of row x is set iff the float32 fused
// multiply-add chain over e = 0..d-1 of W_sort[h][t][e] * x[e] is > 0; the key
// is the rank of the bit code in the reflected Gray sequence so neighbouring
// buckets differ in one bit (sorted Hamming LSH, Sec. 3).
// Sort (Alg. 4, step "Sort"; one call per half-segment of each level of
// Alg. 5): ascending by (key, token index), i.e. a stable counting sort over
// at most 2^sort_bits buckets, one workgroup per sorted list.
#include "common.hpp"
#include "internal.hpp"

namespace elsaa {

constexpr int kHashRows = 64;

template <class T>
__global__ __launch_bounds__(kHashRows) void hash_kernel(const typename T::store_t* __restrict__ X,
                                                         const float* __restrict__ W,
                                                         uint8_t* __restrict__ keys, int H, int N,
                                                         int D, int bits)
{
    __shared__ float w_s[8 * 128];
    __shared__ float x_s[kHashRows * 129];
    const int h = blockIdx.y, b = blockIdx.z;
    const int row0 = blockIdx.x * kHashRows;
    const int rows = min(kHashRows, N - row0);
    const size_t rowbase = ((size_t)b * H + h) * N + row0;
    for (int e = threadIdx.x; e < bits * D; e += kHashRows) w_s[e] = W[(size_t)h * bits * D + e];
    // the tile's rows are contiguous in memory: read it in 16-byte pieces
    constexpr int per16 = 16 / T::bytes;
    const int nchunk = rows * D / per16;
    const uint4* src = (const uint4*)(X + rowbase * D);
    for (int c = threadIdx.x; c < nchunk; c += kHashRows) {
        uint4 v = src[c];
        const typename T::store_t* e = (const typename T::store_t*)&v;
        const int flat = c * per16;
        const int r = flat / D, col = flat % D;
#pragma unroll
        for (int j = 0; j < per16; ++j) x_s[r * (D + 1) + col + j] = T::load(e[j]);
    }
    __syncthreads();
    const int t = threadIdx.x;
    if (t >= rows) return;
    uint32_t code = 0;
    for (int bit = 0; bit < bits; ++bit) {
        float p = 0.0f;
        const float* w = w_s + bit * D;
        const float* x = x_s + t * (D + 1);
        for (int e = 0; e < D; ++e) p = __builtin_fmaf(w[e], x[e], p);
        if (p > 0.0f) code |= 1u << bit;
    }
    uint32_t rank = code;
    for (uint32_t s = code >> 1; s; s >>= 1) rank ^= s;
    keys[rowbase + t] = (uint8_t)rank;
}

hipError_t launch_hash(const Shape& s, const void* X, const float* W_sort, uint8_t* keys,
                       hipStream_t st)
{
    dim3 grid((s.N + kHashRows - 1) / kHashRows, s.H, s.B);
    if (s.bf16)
        hipLaunchKernelGGL(hash_kernel<BF16>, grid, dim3(kHashRows), 0, st,
                           (const uint16_t*)X, W_sort, keys, s.H, s.N, s.D, s.sort_bits);
    else
        hipLaunchKernelGGL(hash_kernel<F32>, grid, dim3(kHashRows), 0, st, (const float*)X,
                           W_sort, keys, s.H, s.N, s.D, s.sort_bits);
    return hipGetLastError();
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
    hipLaunchKernelGGL(sort_kernel, grid, dim3(kSortThreads), 0, st, keyq, keyk, perm_q, perm_k,
                       s.H, s.N, s.causal, s.Lv, s.sort_bits);
    return hipGetLastError();
}

}  // namespace elsaa
