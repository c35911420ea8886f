// gemm.hip -- bfloat16 matrix-core GEMM for the dense projections around the
// attention operator (Alg. 1 / Alg. 6: Q, K, V = X W_{Q,K,V}; O_head W_O).
//
// Two kernels.  Products whose M and N are multiples of 256 and K of 64 run
// gemm_big_kernel (256 x 256 tiles, one workgroup per compute unit, 128 x 128
// per wave with the accumulators in the accumulation registers; see the
// large-tile section).  Every other shape runs gemm_kernel: workgroup tile
// 128 x 128 x 64, four waves in a 2 x 2 grid, each wave a 64 x 64 block of
// 4 x 4 accumulators of v_mfma_f32_16x16x32_bf16.  Both compute C^T tiles
// (the B operand feeds the MFMA's first input) so that every lane ends with
// four consecutive columns of one C row, which makes the stores 8- or
// 16-byte vectors.
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

// ---------------------------------------------------------------- large tiles
// Workgroup tile 256 x 256 x 64 for products whose M and N are multiples of
// 256 and K of 64: four waves in a 2 x 2 grid, each a 128 x 128 block of
// 8 x 8 accumulators (256 float32 per lane, held in the accumulation
// registers; one workgroup per compute unit).  Per 32-wide k-step a wave
// reads 16 operand fragments for 64 matrix-core operations, half the LDS
// traffic per operation of the 64 x 64 wave block, and one K-tile keeps the
// matrix cores busy long enough to cover the next tile's global loads.
namespace big {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kLdD = BK + 8;       // [rows][k] row stride
constexpr int kLdT = BM + 16;      // [k][rows] row stride
constexpr int kTile = BM * kLdD;   // elements of one operand tile (either orientation)
static_assert(BK * kLdT <= kTile, "tile orientations fit one buffer");
static_assert(BK == 64, "two 32-wide k-steps per K-tile");
constexpr int kChunks = BM * BK / 8 / kThreads;   // 16-byte chunks per thread per operand tile
static_assert(kChunks == 8, "one chunk of each operand per group of eight operations");

// Element offset of (row r, column c) split into a row part and a column
// part.  Within an aligned block of rows that does not cross a sequence
// (head-major operands have seq % 256 == 0 on this path), the row part is
// affine in r with stride row_stride(); blk0 is the block's first row.
__device__ __forceinline__ int64_t row_part(const Mat& m, int r, int blk0)
{
    if (m.heads == 0) return (int64_t)r * m.ld;
    const int b = blk0 / m.seq;
    return ((int64_t)r + (int64_t)b * (m.heads - 1) * m.seq) << m.dh_shift;
}
__device__ __forceinline__ int64_t row_stride(const Mat& m) { return m.heads == 0 ? m.ld : ((int64_t)1 << m.dh_shift); }
__device__ __forceinline__ int64_t col_part(const Mat& m, int c)
{
    if (m.heads == 0) return c;
    return (((int64_t)(c >> m.dh_shift) * m.seq) << m.dh_shift) + (c & ((1 << m.dh_shift) - 1));
}

// Global -> registers: K-tile [k0, k0 + 64) of the operand rows [x0, x0 + 256).
// KMAJOR: stored [k][x], thread tx loads k-rows k0 + tx / 32 + 8 c at columns
// x0 + 8 (tx % 32); else stored [x][k], rows x0 + tx / 8 + 32 c at k0 + 8 (tx % 8).
// Each address is a per-thread offset fixed for the whole tile plus a
// workgroup-uniform offset of the K-tile: the rows of a K-tile (KMAJOR) or of
// the tile (else) lie in one sequence, and 64 consecutive k of a [x][k]
// operand in one head (head widths >= 64 on this path).
template <bool KMAJOR>
struct Stream {
    const uint16_t* p;
    int64_t rs;      // element stride between rows of one sequence
    int64_t toff;    // this thread's fixed element offset
    __device__ __forceinline__ void init(const Mat& m, int x0)
    {
        const int tx = threadIdx.x;
        p = (const uint16_t*)m.p;
        rs = row_stride(m);
        if (KMAJOR) toff = (int64_t)(tx >> 5) * rs + col_part(m, x0 + (tx & 31) * 8);
        else toff = row_part(m, x0 + (tx >> 3), x0) + (tx & 7) * 8;
    }
    // first element of K-tile k0 for chunk 0 (uniform part only)
    __device__ __forceinline__ const uint16_t* tile(const Mat& m, int k0) const
    {
        return p + (KMAJOR ? row_part(m, k0, k0) : col_part(m, k0));
    }
    __device__ __forceinline__ uint4 chunk(const uint16_t* q, int c) const
    {
        return ldg16(q + (KMAJOR ? 8 : 32) * c * rs + toff);
    }
    __device__ __forceinline__ void load(const Mat& m, int k0, uint4 (&r)[kChunks]) const
    {
        const uint16_t* q = tile(m, k0);
#pragma unroll
        for (int c = 0; c < kChunks; ++c) r[c] = chunk(q, c);
    }
};

template <bool KMAJOR>
__device__ __forceinline__ void store1(uint16_t* s, uint4 v, int c)
{
    const int tx = threadIdx.x;
    if (KMAJOR) *(uint4*)&s[((tx >> 5) + 8 * c) * kLdT + (tx & 31) * 8] = v;
    else *(uint4*)&s[((tx >> 3) + 32 * c) * kLdD + (tx & 7) * 8] = v;
}
template <bool KMAJOR>
__device__ __forceinline__ void store(uint16_t* s, const uint4 (&r)[kChunks])
{
#pragma unroll
    for (int c = 0; c < kChunks; ++c) store1<KMAJOR>(s, r[c], c);
}

// Operand fragment of rows x0 .. x0+15 for k-step ks.
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

// acc += a x b with acc tied to accumulation registers: the 64 accumulators
// fill all 256 of them, and with the builtin the register allocator moves
// some through vector registers on every iteration.  The compiler does not
// see this as a matrix-core instruction: the statements keep program order
// (an accumulator is reused only after the 63 others), and reads of acc
// after the last one are separated by the wait states in mfma_drain.
__device__ __forceinline__ void mfma_acc(f32x4& acc, bf16x8 a, bf16x8 b)
{
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
__device__ __forceinline__ void mfma_drain()
{
    asm volatile("s_nop 15\n\ts_nop 15\n\ts_nop 15\n\ts_nop 15" ::: "memory");
}

template <bool TA, bool BKN, bool OUT_BF16>
__global__ __launch_bounds__(kThreads, 1) void gemm_big_kernel(GArgs a)
{
    __shared__ __attribute__((aligned(16))) uint16_t lds[4][kTile];
    uint16_t(*sa)[kTile] = lds;
    uint16_t(*sb)[kTile] = lds + 2;
    int sp, tm, tn;
    tile_of(a, sp, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    const int kb = sp * a.kper, ke = min(a.K, kb + a.kper);
    const int nkt = (ke - kb) / BK;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int wm = w & 1, wn = w >> 1;
    const int g = lane >> 4, col = lane & 15;

    f32x4 acc[8][8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[j][i] = f32x4{0, 0, 0, 0};

    Stream<TA> gA;
    Stream<BKN> gB;
    gA.init(a.A, m0);
    gB.init(a.B, n0);
    // Pipeline: LDS buffer t & 1 holds K-tile t, the registers K-tile t + 1.
    // The first half of an iteration runs k-step 0 of tile t (fragments
    // already read) in eight groups of eight operations; before group i it
    // reads fragment pair i of k-step 1, stores chunk i of both operands of
    // tile t + 1 to the other buffer and reloads those registers with chunk
    // i of tile t + 2.  After the one barrier, the second half runs k-step 1
    // the same way, reading k-step 0 of tile t + 1.  Spreading the loads and
    // stores keeps the in-order wave from stalling on a burst of memory
    // instructions while the matrix cores idle, and each load has a whole
    // iteration to arrive.  Tile indices past the end are clamped to the
    // last tile (the redundant loads and stores are never read), so the
    // groups carry no branches.
    uint4 ra[kChunks], rb[kChunks];
    gA.load(a.A, kb, ra);
    gB.load(a.B, kb, rb);
    store<TA>(sa[0], ra);
    store<BKN>(sb[0], rb);
    {
        // same issue order as the loop's loads (A and B chunks alternating),
        // so the stores' waits count exactly across the loop entry
        const uint16_t* qa = gA.tile(a.A, kb + min(1, nkt - 1) * BK);
        const uint16_t* qb = gB.tile(a.B, kb + min(1, nkt - 1) * BK);
#pragma unroll
        for (int i = 0; i < kChunks; ++i) {
            ra[i] = gA.chunk(qa, i);
            rb[i] = gB.chunk(qb, i);
        }
    }
    __syncthreads();
    bf16x8 x0[8], y0[8], x1[8], y1[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        x0[j] = frag<BKN>(sb[0], 128 * wn + 16 * j, 0);
        y0[j] = frag<TA>(sa[0], 128 * wm + 16 * j, 0);
    }

    for (int t = 0; t < nkt; ++t) {
        const uint16_t* A_ = sa[t & 1];
        const uint16_t* B_ = sb[t & 1];
        uint16_t* An = sa[(t + 1) & 1];
        uint16_t* Bn = sb[(t + 1) & 1];
        const int k2 = kb + min(t + 2, nkt - 1) * BK;
        const uint16_t* qa = gA.tile(a.A, k2);
        const uint16_t* qb = gB.tile(a.B, k2);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            x1[i] = frag<BKN>(B_, 128 * wn + 16 * i, 1);
            y1[i] = frag<TA>(A_, 128 * wm + 16 * i, 1);
            store1<TA>(An, ra[i], i);
            store1<BKN>(Bn, rb[i], i);
            ra[i] = gA.chunk(qa, i);
            rb[i] = gB.chunk(qb, i);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int j = 0; j < 8; ++j) mfma_acc(acc[j][i], x0[j], y0[i]);
            __builtin_amdgcn_sched_barrier(0);
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            x0[i] = frag<BKN>(Bn, 128 * wn + 16 * i, 0);
            y0[i] = frag<TA>(An, 128 * wm + 16 * i, 0);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int j = 0; j < 8; ++j) mfma_acc(acc[j][i], x1[j], y1[i]);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    __syncthreads();
    mfma_drain();

    if (OUT_BF16 && a.splits == 1) {
        // bf16 output: the float32 accumulators pass through LDS (each wave
        // its own 64 x 128 block per half, row stride 132) and leave as
        // 16-byte pieces of C rows.  Accumulators are only ever stored, never
        // operated on, so they stay in the accumulation registers.
        constexpr int kLdC = 132;
        float* cs = (float*)&lds[0][0] + w * 64 * kLdC;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 8; ++j) *(f32x4*)&cs[(16 * i + col) * kLdC + 16 * j + 4 * g] = acc[j][4 * hh + i];
            __syncthreads();
#pragma unroll 4
            for (int it = 0; it < 16; ++it) {
                const int r = 4 * it + (lane >> 4), c8 = (lane & 15) * 8;
                const f32x4 x = *(const f32x4*)&cs[r * kLdC + c8];
                const f32x4 y = *(const f32x4*)&cs[r * kLdC + c8 + 4];
                uint4 o;
                o.x = f32_to_bf16(x[0]) | ((uint32_t)f32_to_bf16(x[1]) << 16);
                o.y = f32_to_bf16(x[2]) | ((uint32_t)f32_to_bf16(x[3]) << 16);
                o.z = f32_to_bf16(y[0]) | ((uint32_t)f32_to_bf16(y[1]) << 16);
                o.w = f32_to_bf16(y[2]) | ((uint32_t)f32_to_bf16(y[3]) << 16);
                const int m = m0 + 128 * wm + 64 * hh + r, n = n0 + 128 * wn + c8;
                stg16((uint16_t*)a.C.p + row_part(a.C, m, m0) + col_part(a.C, n), o);
            }
            __syncthreads();
        }
        return;
    }
    // float32 output or split partials: lane holds
    // C[m0 + 128 wm + 16 i + col][n0 + 128 wn + 16 j + 4 g + (0..3)]
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int m = m0 + 128 * wm + 16 * i + col;
        const int64_t ro = a.splits > 1 ? ((int64_t)sp * a.M + m) * a.N : row_part(a.C, m, m0);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int n = n0 + 128 * wn + 16 * j + 4 * g;
            if (a.splits > 1) *(f32x4*)(a.part + ro + n) = acc[j][i];
            else *(f32x4*)((float*)a.C.p + ro + col_part(a.C, n)) = acc[j][i];
        }
    }
}

}  // namespace big

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
    bool big;                 // 256 x 256 tiles (gemm_big_kernel)
    int tiles_m, tiles_n, splits, kper;
    size_t ws_bytes;
};

// The large-tile kernel takes whole tiles only, head-major operands whose
// sequences hold whole 256-row blocks (so no tile or K-tile crosses one) and
// head-major A / B with heads at least 64 wide.
bool big_fits(const elsaa_gemm_desc* d)
{
    if (d->M % big::BM || d->N % big::BN || d->K % big::BK) return false;
    const bool hm = d->a_heads > 0 || d->b_heads > 0 || d->c_heads > 0;
    if (hm && (d->seq <= 0 || d->seq % 256 != 0)) return false;
    const int a_cols = d->trans_a ? d->M : d->K, b_cols = d->trans_b ? d->K : d->N;
    if (d->a_heads > 0 && a_cols / d->a_heads < 64) return false;
    if (d->b_heads > 0 && b_cols / d->b_heads < 64) return false;
    return true;
}

Plan plan_of(const elsaa_gemm_desc* d)
{
    Plan p;
    p.big = big_fits(d);
    const int bm = p.big ? big::BM : BM, bn = p.big ? big::BN : BN, bk = p.big ? big::BK : BK;
    // workgroups resident per compute unit (256 compute units)
    const int fill = p.big ? 256 : 512;
    p.tiles_m = (d->M + bm - 1) / bm;
    p.tiles_n = (d->N + bn - 1) / bn;
    const int tiles = p.tiles_m * p.tiles_n;
    const int ktiles = (d->K + bk - 1) / bk;
    int splits = 1;
    // fewer tiles than resident workgroups and a long K: split K into as
    // many parts as fit in one round of resident workgroups, keeping at
    // least 8 K-tiles per split
    if (tiles < fill && ktiles >= 16) splits = std::max(1, std::min(fill / tiles, ktiles / 8));
    const int per = (ktiles + splits - 1) / splits;
    p.kper = per * bk;
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
    if (d->trans_a == TA && bkn == BKN && out_bf16 == OB) {                                           \
        if (p.big) ELSAA_LAUNCH("gemm", (big::gemm_big_kernel<TA, BKN, OB>), grid, block, 0, stream, a); \
        else ELSAA_LAUNCH("gemm", (gemm_kernel<TA, BKN, OB>), grid, block, 0, stream, a);              \
    }
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
