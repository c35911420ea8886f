// select.hip -- sortLSH selection (sign hash, per-segment stable sort) and
// the RACE projections of the same rows.
//
// Hash (Alg. 4, step "Hash"): bit t of row x is set iff the float32 fused
// multiply-add chain over e = 0..d-1 of W_sort[h][t][e] * x[e] is > 0; the key
// is the rank of the bit code in the reflected Gray sequence so neighbouring
// buckets differ in one bit (sorted Hamming LSH, Sec. 3).  The same pass over
// Q or K also computes the RACE projections u = W_race x (Alg. 2) and stores
// t = tanh(u), so each input row is read once for both branches' hashing.
// Sort (Alg. 4, step "Sort"; one call per half-segment of each level of
// Alg. 5): ascending by (key, token index), i.e. a stable counting sort over
// at most 2^sort_bits buckets, one workgroup per sorted list.
#include "common.hpp"
#include "internal.hpp"
#include "causal.hpp"
#include "race_common.hpp"

namespace elsaa {

constexpr int kProjRows = 64;
constexpr int kProjThreads = 256;
constexpr int kProjWaves = kProjThreads / kWave;
constexpr int kProjPad = 8;
constexpr int kProjTarget = 1024;      // workgroups per launch (about four per CU)

// A workgroup walks a chunk of 64-row tiles of X (Q or K of one (b,h)); for
// every row it writes the sortLSH bucket key and, when W_race is given, the
// RACE projections u = W_race x in float32 accuracy: W = W_hi + W_lo split
// into two bf16 parts for the bf16 MFMA path (the residual is below 2^-16
// relative), plain float32 MFMA for float32 storage.  t = tanh(u) is stored
// [BH][N][UP] (UP = padded projections).  W is staged once per workgroup;
// the next tile's rows are loaded into registers while the current one is
// hashed and projected.
template <class T, int D, int WR>
struct ProjSmem {
    typename T::store_t x[kProjRows][D + kProjPad];
    typename T::store_t whi[WR][D + kProjPad];
    typename T::store_t wlo[T::bytes == 2 ? WR : 1][D + kProjPad];   // (no low part for float32)
    uint32_t code[kProjRows];
};

// One launch covers Q and K: grid.z runs over 2B, the second half being K.
struct ProjIO {
    const void* X[2];     // Q rows, K rows
    uint8_t* keys[2];
    float* U[2];          // RACE projections (ignored when Wrace is null)
};

template <class T, int D, int WR>
__global__ __launch_bounds__(kProjThreads) void proj_kernel(ProjIO io, const float* __restrict__ Wsort,
                                                            const float* __restrict__ Wrace, int B, int H, int N,
                                                            int bits, int L, int UP, int chunk_rows)
{
    using S = typename T::store_t;
    using F = typename T::frag_t;
    constexpr int PER = 16 / T::bytes;           // elements per 16-byte piece
    constexpr int CH = D / PER;                  // pieces per row
    constexpr int KS = D / 32;
    constexpr int PT = kProjRows * CH / kProjThreads;   // pieces staged per thread
    __shared__ ProjSmem<T, D, WR> sm;
    const int h = blockIdx.y, which = blockIdx.z >= B, b = blockIdx.z - (which ? B : 0);
    const size_t bh = (size_t)b * H + h;
    const int rbeg = blockIdx.x * chunk_rows;
    const int rend = min(N, rbeg + chunk_rows);
    const S* Xh = (const S*)io.X[which] + bh * N * D;
    uint8_t* __restrict__ keys = io.keys[which];
    float* __restrict__ U = io.U[which];
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

    // rows [row0, row0 + 64) -> registers (zero past rend)
    uint4 rx[PT];
    auto load = [&](int row0) {
#pragma unroll
        for (int j = 0; j < PT; ++j) {
            const int it = threadIdx.x + kProjThreads * j;
            const int r = it / CH, c = it % CH;
            rx[j] = row0 + r < rend ? ldg16(Xh + (size_t)(row0 + r) * D + c * PER) : make_uint4(0, 0, 0, 0);
        }
    };
    load(rbeg);
    if (Wrace) {
        // W staged up to eight loads per thread at a time (one round trip each)
        constexpr int PW = (WR * D) / kProjThreads < 8 ? (WR * D) / kProjThreads : 8;
        static_assert(PW >= 1 && (WR * D) % (PW * kProjThreads) == 0, "W staging split");
        for (int it0 = 0; it0 < WR * D; it0 += PW * kProjThreads) {
            float wv[PW];
#pragma unroll
            for (int j = 0; j < PW; ++j) {
                const int it = it0 + j * kProjThreads + threadIdx.x;
                const int row = it / D, c = it % D;
                wv[j] = row < 4 * L ? Wrace[((size_t)h * L * 4 + row) * D + c] : 0.f;
            }
#pragma unroll
            for (int j = 0; j < PW; ++j) {
                const int it = it0 + j * kProjThreads + threadIdx.x;
                const int row = it / D, c = it % D;
                const S hi = T::store(wv[j]);
                sm.whi[row][c] = hi;
                if (T::bytes == 2) sm.wlo[row][c] = T::store(wv[j] - T::load(hi));
            }
        }
    }
    const float* ws_h = Wsort + (size_t)h * bits * D;
    static_assert(2 * kProjWaves >= 8, "two hash bits per wave cover sort_bits <= 8");
    for (int row0 = rbeg; row0 < rend; row0 += kProjRows) {
        __syncthreads();                          // previous tile consumed
#pragma unroll
        for (int j = 0; j < PT; ++j) {
            const int it = threadIdx.x + kProjThreads * j;
            *(uint4*)&sm.x[it / CH][(it % CH) * PER] = rx[j];
        }
        if (threadIdx.x < kProjRows) sm.code[threadIdx.x] = 0;
        __syncthreads();
        if (row0 + kProjRows < rend) load(row0 + kProjRows);
        const int rows = min(kProjRows, rend - row0);

        // hash: lane = row; wave w runs the float32 fma chains of bits w and
        // w + 4 (sort_bits <= 8) side by side over the same row reads, so a
        // second bit adds little to the chain latency; W_sort rows are
        // wave-uniform.  Each chain keeps the order e = 0 .. d-1.
        if (w < bits) {
            const int b1 = w + kProjWaves < bits ? w + kProjWaves : w;
            const float* w0 = ws_h + (size_t)w * D;
            const float* w1 = ws_h + (size_t)b1 * D;
            float p0 = 0.0f, p1 = 0.0f;
#pragma unroll
            for (int e0 = 0; e0 < D; e0 += PER) {
                const uint4 v = *(const uint4*)&sm.x[lane][e0];
                const S* xs = (const S*)&v;
#pragma unroll
                for (int j = 0; j < PER; ++j) {
                    const float xv = T::load(xs[j]);
                    p0 = __builtin_fmaf(w0[e0 + j], xv, p0);
                    p1 = __builtin_fmaf(w1[e0 + j], xv, p1);
                }
            }
            const uint32_t c = (p0 > 0.0f ? 1u << w : 0u) | (p1 > 0.0f ? 1u << b1 : 0u);
            if (c) atomicOr(&sm.code[lane], c);
        }
        // u[token][p] for the wave's 16 tokens: A = W rows, B = X rows
        if (Wrace) {
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
                if (tl < rows && p0 < UP) {
                    // the RACE passes use u only through t = tanh(u): store t
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc[i] = race::tanh_abs(acc[i]);
                    *(f32x4*)(U + (bh * N + row0 + tl) * UP + p0) = acc;
                }
            }
        }
        __syncthreads();
        if (threadIdx.x < rows) {
            const uint32_t code = sm.code[threadIdx.x];
            uint32_t rank = code;
            for (uint32_t sft = code >> 1; sft; sft >>= 1) rank ^= sft;
            keys[bh * N + row0 + threadIdx.x] = (uint8_t)rank;
        }
    }
}

template <class T, int D>
hipError_t launch_proj_t(const Shape& s, const ProjIO& io, const float* W_sort, const float* W_race, hipStream_t st)
{
    // about kProjTarget workgroups for both tensors together
    const int64_t tiles = (s.N + kProjRows - 1) / kProjRows;
    const int64_t lists = 2 * (int64_t)s.B * s.H;
    int64_t want = (kProjTarget + lists - 1) / lists;
    if (want > tiles) want = tiles;
    const int64_t per = (tiles + want - 1) / want;
    const int chunk_rows = (int)(per * kProjRows);
    dim3 grid((s.N + chunk_rows - 1) / chunk_rows, s.H, 2 * s.B);
    const int UP = race_proj_stride(s);
    const int wr = UP < 16 ? 16 : UP;
#define ELSAA_PROJ(WR_)                                                                          \
    ELSAA_LAUNCH("project", (proj_kernel<T, D, WR_>), grid, dim3(kProjThreads), 0, st, io, W_sort, W_race, \
                 s.B, s.H, s.N, s.sort_bits, s.L, UP, chunk_rows)
    if (wr == 16) ELSAA_PROJ(16);
    else if (wr == 32) ELSAA_PROJ(32);
    else ELSAA_PROJ(64);
#undef ELSAA_PROJ
    return hipGetLastError();
}

hipError_t launch_project(const Shape& s, const void* Q, const void* K, const float* W_sort,
                          const float* W_race, uint8_t* keyq, uint8_t* keyk, float* Uq, float* Uk,
                          hipStream_t st)
{
    ProjIO io;
    io.X[0] = Q;
    io.X[1] = K;
    io.keys[0] = keyq;
    io.keys[1] = keyk;
    io.U[0] = Uq;
    io.U[1] = Uk;
    if (s.bf16) return s.D == 64 ? launch_proj_t<BF16, 64>(s, io, W_sort, W_race, st)
                                 : launch_proj_t<BF16, 128>(s, io, W_sort, W_race, st);
    return s.D == 64 ? launch_proj_t<F32, 64>(s, io, W_sort, W_race, st)
                     : launch_proj_t<F32, 128>(s, io, W_sort, W_race, st);
}

// --------------------------------------------------------------------------
// Stable counting sort, one workgroup per list.
// Lists of one (b,h):
//   non-causal: task 0 = all queries, task 1 = all keys;
//   causal: level l has 2^l segments (causal.hpp); task (l, s, q/k) sorts
//           the future half of segment s by the query keys or its past half
//           by the key keys, m_l entries each.  A future half's trailing
//           zero tokens (Alg. 5's padding of odd lists) take the key of the
//           zero vector, 0 (no sign bit is set), and sort after every real
//           token of that key; their entries are -1.
// --------------------------------------------------------------------------

constexpr int kSortThreads = 256;
constexpr int kSortWaves = kSortThreads / kWave;
constexpr int kKeyCache = 16384;       // keys of a list staged in LDS (longer lists read the rest from HBM)

// One workgroup per list.  The list is cut into one contiguous quarter per
// wave.  A histogram of every quarter gives each wave, for every bucket, the
// output position of its first element of that bucket (all smaller buckets,
// then the same bucket in earlier quarters); each wave then ranks its
// quarter 64 keys at a time (lanes of equal key found by ballots over the
// key bits) with no further synchronisation, so equal keys keep their index
// order within the whole list.
__global__ __launch_bounds__(kSortThreads) void sort_kernel(const uint8_t* __restrict__ keyq,
                                                            const uint8_t* __restrict__ keyk,
                                                            int32_t* __restrict__ perm_q,
                                                            int32_t* __restrict__ perm_k, int H,
                                                            int N, int causal, LevelTiles lt, int bits)
{
    __shared__ int hist[kSortWaves][256];   // per quarter; then its running output positions
    __shared__ uint8_t kc[kKeyCache];
    const int h = blockIdx.y, b = blockIdx.z;
    const int task = blockIdx.x;
    const int nb = 1 << bits;
    const size_t bh = (size_t)b * H + h;

    int start, len, nreal, is_k;             // list entries [0, len): tokens start + i for i < nreal
    size_t out_off;
    if (!causal) {
        is_k = task;
        start = 0;
        len = nreal = N;
        out_off = bh * N;
    } else {
        // level l owns tasks [2^(l+1) - 2, 2^(l+2) - 2)
        const int l = 31 - __clz(task + 2) - 1;
        const int t2 = task - ((1 << (l + 1)) - 2);
        const int seg = t2 >> 1;
        is_k = t2 & 1;
        int a, r;
        seg_range(lt, l, seg, a, r);
        const int half = lt.len[l + 1];
        start = is_k ? a : a + half;
        len = half;
        nreal = is_k ? half : (r > half ? r - half : 0);
        out_off = bh * (size_t)lt.off[lt.Lv] + (size_t)lt.off[l] + (size_t)seg * half;
    }
    const uint8_t* key = (is_k ? keyk : keyq) + bh * N + start;
    int32_t* out = (is_k ? perm_k : perm_q) + out_off;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
    const int quarter = (len + kSortWaves - 1) / kSortWaves;
    const int qbeg = min(len, wave * quarter), qend = min(len, qbeg + quarter);

    for (int i = threadIdx.x; i < kSortWaves * 256; i += kSortThreads) (&hist[0][0])[i] = 0;
    __syncthreads();
    // the quarter's histogram; the first kKeyCache keys of the list are staged
    // in LDS on the way, eight loads per lane in flight at a time
    for (int i0 = qbeg; i0 < qend; i0 += 8 * kWave) {
        uint8_t v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int i = i0 + j * kWave + lane;
            v[j] = i < qend && i < nreal ? key[i] : 0;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int i = i0 + j * kWave + lane;
            if (i < qend) {
                if (i < kKeyCache) kc[i] = v[j];
                atomicAdd(&hist[wave][v[j]], 1);
            }
        }
    }
    __syncthreads();
    // first output position of bucket c in quarter w: all keys < c, then key c
    // in quarters before w (one wave scans the buckets, 64 at a time)
    if (wave == 0) {
        int carry = 0;
        for (int c0 = 0; c0 < nb; c0 += kWave) {
            const int c = c0 + lane;
            int cnt[kSortWaves], tot = 0;
#pragma unroll
            for (int w = 0; w < kSortWaves; ++w) {
                cnt[w] = c < nb ? hist[w][c] : 0;
                tot += cnt[w];
            }
            int incl = tot;                                  // inclusive scan over the lanes
#pragma unroll
            for (int d = 1; d < kWave; d <<= 1) {
                const int y = __shfl_up(incl, d);
                if (lane >= d) incl += y;
            }
            int pos = carry + incl - tot;
            if (c < nb)
#pragma unroll
                for (int w = 0; w < kSortWaves; ++w) {
                    hist[w][c] = pos;
                    pos += cnt[w];
                }
            carry += __shfl(incl, kWave - 1);
        }
    }
    __syncthreads();
    // rank the quarter, 64 keys per step; hist[wave][c] is the next output
    // position of bucket c in this quarter
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
    for (int i0 = qbeg; i0 < qend; i0 += kWave) {
        const int i = i0 + lane;
        const bool valid = i < qend;
        const int kk = valid && i < nreal ? (i < kKeyCache ? kc[i] : key[i]) : 0;
        uint64_t same = __ballot(valid);
        for (int bit = 0; bit < bits; ++bit) {
            const uint64_t ones = __ballot(valid && ((kk >> bit) & 1));
            same &= ((kk >> bit) & 1) ? ones : ~ones;
        }
        const int rank = __popcll(same & below);
        const int pos = valid ? hist[wave][kk] + rank : 0;
        __builtin_amdgcn_wave_barrier();                     // every lane has read before the leaders advance
        if (valid) out[pos] = i < nreal ? start + i : -1;
        if (valid && rank == 0) hist[wave][kk] += __popcll(same);
    }
}

hipError_t launch_sort(const Shape& s, const uint8_t* keyq, const uint8_t* keyk, int32_t* perm_q,
                       int32_t* perm_k, hipStream_t st)
{
    const int tasks = s.causal ? (1 << (s.Lv + 1)) - 2 : 2;
    if (tasks <= 0) return hipSuccess;
    dim3 grid(tasks, s.H, s.B);
    ELSAA_LAUNCH("sort", sort_kernel, grid, dim3(kSortThreads), 0, st, keyq, keyk, perm_q, perm_k,
                       s.H, s.N, s.causal, s.lt, s.sort_bits);
    return hipGetLastError();
}

}  // namespace elsaa
