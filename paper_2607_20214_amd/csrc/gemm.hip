// gemm.hip -- bfloat16 matrix-core GEMM for the dense projections around the
// attention operator (Alg. 1 / Alg. 6: Q, K, V = X W_{Q,K,V}; O_head W_O).
//
// Workgroup tile 128 x 128 x 64, four waves in a 2 x 2 grid, each wave a
// 64 x 64 block of 4 x 4 accumulators of v_mfma_f32_16x16x32_bf16.  The
// kernel computes C^T tiles (the B operand feeds the MFMA's first input) so
// that every lane ends with four consecutive columns of one C row, which
// makes the stores 8- or 16-byte vectors.
//
// Operands are staged through LDS in the orientation in which they are
// stored: a tile whose contraction dimension is contiguous is read with
// 16-byte LDS loads; a tile stored the other way round ([K][M] for A^T,
// [K][N] for B) is read with the gfx950 transposed LDS load, so no operand
// is ever transposed in memory.  Global loads of the next K-tile are issued
// into registers before the MFMAs of the current one (two LDS buffers, one
// barrier per K-tile).
//
// Long-K products with few output tiles (the weight gradients) split K over
// workgroups; float32 partials go to the workspace and a second kernel sums
// them in split order.  Workgroup ids are remapped so that each of the
// eight XCDs (own L2) works on a contiguous group of tiles.
#include <algorithm>
#include <cstring>

#include "common.hpp"
#include "elsaa.h"
#include "internal.hpp"

namespace elsaa {

namespace {

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int kThreads = 256;
constexpr int kLdD = BK + 8;      // row stride of a tile stored [rows][k]
constexpr int kLdT = BM + 16;     // row stride of a tile stored [k][rows]
constexpr int kTileElems = 128 * kLdD;
static_assert(128 * kLdD == 64 * kLdT, "both tile orientations use the same LDS size");
constexpr int kGroupM = 8;        // M tiles per launch-order group

// One stored matrix: plain row-major (heads == 0) or head-major.
struct Mat {
    void* p;
    int64_t ld;
    int heads, seq, dh_shift;
};

__device__ __forceinline__ int64_t mat_offset(const Mat& m, int r, int c)
{
    if (m.heads == 0) return (int64_t)r * m.ld + c;
    const int b = r / m.seq, n = r - b * m.seq;
    const int h = c >> m.dh_shift, e = c & ((1 << m.dh_shift) - 1);
    return ((((int64_t)b * m.heads + h) * m.seq + n) << m.dh_shift) + e;
}

struct GArgs {
    Mat A, B, C;
    int M, N, K;
    int tiles_m, tiles_n, splits, kper;
    float* part;   // [splits][M][N] float32 when splits > 1
};

// Tile coordinates of this workgroup: XCD-contiguous id, then groups of
// kGroupM M-tiles swept along N.
__device__ __forceinline__ void tile_of(const GArgs& a, int& sp, int& tm, int& tn)
{
    const int total = a.tiles_m * a.tiles_n * a.splits;
    int id = blockIdx.x;
    const int full = total & ~7;
    if (id < full) id = (id & 7) * (full >> 3) + (id >> 3);
    const int per = a.tiles_m * a.tiles_n;
    sp = id / per;
    const int t = id - sp * per;
    const int group = t / (kGroupM * a.tiles_n);
    const int m0 = group * kGroupM;
    const int gm = min(kGroupM, a.tiles_m - m0);
    const int r = t - group * kGroupM * a.tiles_n;
    tm = m0 + r % gm;
    tn = r / gm;
}

// Global -> register staging of one K-tile of a stored operand.  KMAJOR:
// the operand is stored [k][x] (x = m or n contiguous); else [x][k].
template <bool KMAJOR>
__device__ __forceinline__ void load_tile(const Mat& m, int x0, int xlim, int k0, int klim, uint4 (&r)[4])
{
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const int id = threadIdx.x + kThreads * c;
        int row, col;
        bool ok;
        if (KMAJOR) {
            row = k0 + (id >> 4);
            col = x0 + (id & 15) * 8;
            ok = row < klim && col < xlim;
        } else {
            row = x0 + (id >> 3);
            col = k0 + (id & 7) * 8;
            ok = row < xlim && col < klim;
        }
        r[c] = ok ? ldg16((const uint16_t*)m.p + mat_offset(m, row, col)) : make_uint4(0, 0, 0, 0);
    }
}

template <bool KMAJOR>
__device__ __forceinline__ void store_tile(uint16_t* s, const uint4 (&r)[4])
{
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const int id = threadIdx.x + kThreads * c;
        if (KMAJOR) *(uint4*)&s[(id >> 4) * kLdT + (id & 15) * 8] = r[c];
        else *(uint4*)&s[(id >> 3) * kLdD + (id & 7) * 8] = r[c];
    }
}

// Operand fragment of rows x0 .. x0+15 for k-step ks (32 values of k).
template <bool KMAJOR>
__device__ __forceinline__ bf16x8 frag(const uint16_t* s, int x0, int ks)
{
    const int lane = threadIdx.x & 63, g = lane >> 4, i = lane & 15;
    if (KMAJOR) {
        const uint16_t* p = &s[(32 * ks + 8 * g + (i >> 2)) * kLdT + x0 + 4 * (i & 3)];
        const bf16x4 lo = lds_read_tr4(p), hi = lds_read_tr4(p + 4 * kLdT);
        return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    }
    return *(const bf16x8*)&s[(x0 + i) * kLdD + 32 * ks + 8 * g];
}

template <bool TA, bool BKN, bool OUT_BF16>
__global__ __launch_bounds__(kThreads, 2) void gemm_kernel(GArgs a)
{
    __shared__ __attribute__((aligned(16))) uint16_t sa[2][kTileElems];
    __shared__ __attribute__((aligned(16))) uint16_t sb[2][kTileElems];
    int sp, tm, tn;
    tile_of(a, sp, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    const int kb = sp * a.kper, ke = min(a.K, kb + a.kper);
    const int nkt = (ke - kb + BK - 1) / BK;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int wm = w & 1, wn = w >> 1;
    const int g = lane >> 4, col = lane & 15;

    f32x4 acc[4][4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[j][i] = f32x4{0, 0, 0, 0};

    uint4 ra[4], rb[4];
    load_tile<TA>(a.A, m0, a.M, kb, ke, ra);
    load_tile<BKN>(a.B, n0, a.N, kb, ke, rb);
    store_tile<TA>(sa[0], ra);
    store_tile<BKN>(sb[0], rb);
    __syncthreads();

    for (int t = 0; t < nkt; ++t) {
        const bool more = t + 1 < nkt;
        if (more) {
            load_tile<TA>(a.A, m0, a.M, kb + (t + 1) * BK, ke, ra);
            load_tile<BKN>(a.B, n0, a.N, kb + (t + 1) * BK, ke, rb);
        }
        const uint16_t* A_ = sa[t & 1];
        const uint16_t* B_ = sb[t & 1];
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
            bf16x8 xf[4], yf[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) xf[j] = frag<BKN>(B_, 64 * wn + 16 * j, ks);
#pragma unroll
            for (int i = 0; i < 4; ++i) yf[i] = frag<TA>(A_, 64 * wm + 16 * i, ks);
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xf[j], yf[i], acc[j][i], 0, 0, 0);
        }
        if (more) {
            store_tile<TA>(sa[(t + 1) & 1], ra);
            store_tile<BKN>(sb[(t + 1) & 1], rb);
        }
        __syncthreads();
    }

    // lane holds C[m0 + 64 wm + 16 i + col][n0 + 64 wn + 16 j + 4 g + (0..3)]
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = m0 + 64 * wm + 16 * i + col;
        if (m >= a.M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int n = n0 + 64 * wn + 16 * j + 4 * g;
            if (n >= a.N) continue;
            const f32x4 v = acc[j][i];
            if (a.splits > 1) {
                *(f32x4*)(a.part + ((size_t)sp * a.M + m) * a.N + n) = v;
            } else if (OUT_BF16) {
                const uint32_t lo = f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
                const uint32_t hi = f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16);
                *(uint2*)((uint16_t*)a.C.p + mat_offset(a.C, m, n)) = make_uint2(lo, hi);
            } else {
                *(f32x4*)((float*)a.C.p + mat_offset(a.C, m, n)) = v;
            }
        }
    }
}

// C = sum over splits of the partials, in split order.
template <bool OUT_BF16>
__global__ __launch_bounds__(256) void gemm_reduce_kernel(const float* part, Mat C, int M, int N, int splits)
{
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // one 4-column chunk
    const int n4 = N / 4;
    if (q >= (int64_t)M * n4) return;
    const int m = (int)(q / n4), n = (int)(q - (int64_t)m * n4) * 4;
    const size_t plane = (size_t)M * N;
    f32x4 v = *(const f32x4*)(part + (size_t)m * N + n);
    for (int s = 1; s < splits; ++s) v += *(const f32x4*)(part + s * plane + (size_t)m * N + n);
    if (OUT_BF16) {
        const uint32_t lo = f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
        const uint32_t hi = f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16);
        *(uint2*)((uint16_t*)C.p + mat_offset(C, m, n)) = make_uint2(lo, hi);
    } else {
        *(f32x4*)((float*)C.p + mat_offset(C, m, n)) = v;
    }
}

struct Plan {
    int tiles_m, tiles_n, splits, kper;
    size_t ws_bytes;
};

Plan plan_of(const elsaa_gemm_desc* d)
{
    Plan p;
    p.tiles_m = (d->M + BM - 1) / BM;
    p.tiles_n = (d->N + BN - 1) / BN;
    const int tiles = p.tiles_m * p.tiles_n;
    const int ktiles = (d->K + BK - 1) / BK;
    int splits = 1;
    // fewer than two workgroups per compute unit and a long K: split K,
    // keeping at least 8 K-tiles per split
    if (tiles < 512 && ktiles >= 16) splits = std::min((512 + tiles - 1) / tiles, ktiles / 8);
    const int per = (ktiles + splits - 1) / splits;
    p.kper = per * BK;
    p.splits = (d->K + p.kper - 1) / p.kper;
    p.ws_bytes = p.splits > 1 ? (size_t)p.splits * d->M * d->N * sizeof(float) : 0;
    return p;
}

int log2_exact(int v)
{
    int s = 0;
    while ((1 << s) < v) ++s;
    return (1 << s) == v ? s : -1;
}

int check_mat(const char* name, const void* ptr, int rows, int cols, int64_t ld, int heads, int seq, Mat* out)
{
    if (!ptr) return api_fail(ELSAA_ERR_INVALID_ARG, "%s is NULL", name);
    if (((uintptr_t)ptr & 15) != 0) return api_fail(ELSAA_ERR_INVALID_ARG, "%s must be 16-byte aligned", name);
    out->p = const_cast<void*>(ptr);
    out->ld = ld;
    out->heads = heads;
    out->seq = seq;
    out->dh_shift = 0;
    if (heads < 0) return api_fail(ELSAA_ERR_INVALID_ARG, "%s: heads must be >= 0 (got %d)", name, heads);
    if (heads == 0) {
        if (ld < cols || ld % 8 != 0)
            return api_fail(ELSAA_ERR_INVALID_ARG, "%s: ld must be >= %d and a multiple of 8 (got %lld)", name, cols,
                            (long long)ld);
        return ELSAA_OK;
    }
    if (cols % heads != 0)
        return api_fail(ELSAA_ERR_INVALID_ARG, "%s: %d columns do not split into %d heads", name, cols, heads);
    const int dh = cols / heads, sh = log2_exact(dh);
    if (sh < 3)
        return api_fail(ELSAA_ERR_UNSUPPORTED, "%s: head width %d must be a power of two >= 8", name, dh);
    if (seq < 1 || rows % seq != 0)
        return api_fail(ELSAA_ERR_INVALID_ARG, "%s: %d rows are not a whole number of sequences of %d", name, rows, seq);
    out->dh_shift = sh;
    return ELSAA_OK;
}

int validate(const elsaa_gemm_desc* d)
{
    if (!d) return api_fail(ELSAA_ERR_INVALID_ARG, "desc is NULL");
    if (d->M < 1 || d->N < 1 || d->K < 1)
        return api_fail(ELSAA_ERR_INVALID_ARG, "M, N, K must be >= 1 (got %d, %d, %d)", d->M, d->N, d->K);
    if (d->M % 8 || d->N % 8 || d->K % 8)
        return api_fail(ELSAA_ERR_UNSUPPORTED, "M, N, K must be multiples of 8 (got %d, %d, %d)", d->M, d->N, d->K);
    if ((d->trans_a != 0 && d->trans_a != 1) || (d->trans_b != 0 && d->trans_b != 1))
        return api_fail(ELSAA_ERR_INVALID_ARG, "trans_a and trans_b must be 0 or 1");
    if (d->c_dtype != ELSAA_F32 && d->c_dtype != ELSAA_BF16)
        return api_fail(ELSAA_ERR_INVALID_ARG, "unknown c_dtype %d", d->c_dtype);
    return ELSAA_OK;
}

}  // namespace

}  // namespace elsaa

using namespace elsaa;

extern "C" {

int elsaa_gemm_workspace_bytes(const elsaa_gemm_desc* desc, size_t* bytes)
{
    int st = validate(desc);
    if (st != ELSAA_OK) return st;
    if (!bytes) return api_fail(ELSAA_ERR_INVALID_ARG, "bytes is NULL");
    *bytes = plan_of(desc).ws_bytes;
    return ELSAA_OK;
}

int elsaa_gemm(const elsaa_gemm_desc* d, const void* A, const void* B, void* C, void* workspace,
               size_t workspace_bytes, hipStream_t stream)
{
    int st = validate(d);
    if (st != ELSAA_OK) return st;
    GArgs a;
    std::memset(&a, 0, sizeof a);
    const int ar = d->trans_a ? d->K : d->M, ac = d->trans_a ? d->M : d->K;
    const int br = d->trans_b ? d->N : d->K, bc = d->trans_b ? d->K : d->N;
    if ((st = check_mat("A", A, ar, ac, d->lda, d->a_heads, d->seq, &a.A)) != ELSAA_OK) return st;
    if ((st = check_mat("B", B, br, bc, d->ldb, d->b_heads, d->seq, &a.B)) != ELSAA_OK) return st;
    if ((st = check_mat("C", C, d->M, d->N, d->ldc, d->c_heads, d->seq, &a.C)) != ELSAA_OK) return st;
    const Plan p = plan_of(d);
    if (p.ws_bytes > 0) {
        if (!workspace) return api_fail(ELSAA_ERR_INVALID_ARG, "workspace is NULL (%zu bytes needed)", p.ws_bytes);
        if (workspace_bytes < p.ws_bytes)
            return api_fail(ELSAA_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", workspace_bytes, p.ws_bytes);
        if (((uintptr_t)workspace & 15) != 0) return api_fail(ELSAA_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
    }
    a.M = d->M; a.N = d->N; a.K = d->K;
    a.tiles_m = p.tiles_m; a.tiles_n = p.tiles_n; a.splits = p.splits; a.kper = p.kper;
    a.part = (float*)workspace;

    const dim3 grid(p.tiles_m * p.tiles_n * p.splits), block(kThreads);
    const bool bkn = d->trans_b == 0, out_bf16 = d->c_dtype == ELSAA_BF16;
#define ELSAA_GEMM_CASE(TA, BKN, OB)                                                                 \
    if (d->trans_a == TA && bkn == BKN && out_bf16 == OB)                                             \
        ELSAA_LAUNCH("gemm", (gemm_kernel<TA, BKN, OB>), grid, block, 0, stream, a);
    ELSAA_GEMM_CASE(0, 0, 0) ELSAA_GEMM_CASE(0, 0, 1) ELSAA_GEMM_CASE(0, 1, 0) ELSAA_GEMM_CASE(0, 1, 1)
    ELSAA_GEMM_CASE(1, 0, 0) ELSAA_GEMM_CASE(1, 0, 1) ELSAA_GEMM_CASE(1, 1, 0) ELSAA_GEMM_CASE(1, 1, 1)
#undef ELSAA_GEMM_CASE
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return api_hip_fail(e, "gemm launch");
    if (p.splits > 1) {
        const int64_t chunks = (int64_t)d->M * (d->N / 4);
        const dim3 rgrid((unsigned)((chunks + 255) / 256));
        if (out_bf16) ELSAA_LAUNCH("gemm_reduce", gemm_reduce_kernel<true>, rgrid, dim3(256), 0, stream, a.part, a.C, a.M, a.N, a.splits);
        else ELSAA_LAUNCH("gemm_reduce", gemm_reduce_kernel<false>, rgrid, dim3(256), 0, stream, a.part, a.C, a.M, a.N, a.splits);
        e = hipGetLastError();
        if (e != hipSuccess) return api_hip_fail(e, "gemm reduce launch");
    }
    return ELSAA_OK;
}

}  // extern "C"
