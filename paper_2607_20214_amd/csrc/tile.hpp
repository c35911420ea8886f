// tile.hpp -- LDS tiles of gathered rows for the sparse-branch kernels.
//
// A tile holds up to 64 rows of D elements, row-major with no padding.  The
// 16-byte chunks of each row are permuted by an XOR swizzle of the row index
// so that the three access patterns of the kernels hit distinct LDS banks:
//   * 16-byte operand reads of 16 rows (consecutive rows, or the interleaved
//     row order of key_of / krow_of), one chunk per lane;
//   * transposed operand reads (ds_read_b64_tr_b16): 4 consecutive rows by
//     32 contiguous bytes per 16-lane group;
//   * 16-byte stores of whole rows by consecutive lanes.
// Rows are staged global -> registers -> LDS by all threads of the
// workgroup; the global loads of the next tile are issued before the
// current tile is consumed.
#pragma once
#include "common.hpp"

namespace elsaa {
namespace tile {

constexpr int kRows = 64;

// Chunk permutation of row r for rows of CPR chunks (CPR >= 8).
template <int CPR>
__device__ __forceinline__ int swz(int r)
{
    const int b24 = ((r >> 2) ^ (r >> 4)) & 1;
    if (CPR >= 16) return b24 | ((r & 1) << 1) | ((r & 2) << 1) | (r & 8);
    return b24 | ((r & 2)) | ((r >> 1) & 4);
}

// Tiles of 64 rows of D elements staged by NT threads.
template <class T, int D, int NT = 256>
struct Tile {
    using S = typename T::store_t;
    using F = typename T::frag_t;
    static constexpr int EPC = 16 / T::bytes;         // elements per 16-byte chunk
    static constexpr int CPR = D / EPC;               // chunks per row
    static constexpr int PER_THREAD = kRows * CPR / NT;   // chunks staged per thread
    static_assert(CPR >= 8 && PER_THREAD >= 1, "tile shape");

    // element offset of chunk c of row r
    __device__ static __forceinline__ int off(int r, int c) { return r * D + ((c ^ swz<CPR>(r)) * EPC); }

    // row of the j-th chunk this thread stages (and the chunk index)
    __device__ static __forceinline__ int row_of(int j) { return (threadIdx.x + NT * j) / CPR; }
    __device__ static __forceinline__ int chunk_of(int j) { return (threadIdx.x + NT * j) % CPR; }

    // global -> registers: rows tok[j] (token index, -1 = none) of X
    __device__ static __forceinline__ void load(const S* X, const int (&tok)[PER_THREAD], uint4 (&r)[PER_THREAD])
    {
#pragma unroll
        for (int j = 0; j < PER_THREAD; ++j)
            r[j] = tok[j] >= 0 ? ldg16(X + (size_t)tok[j] * D + chunk_of(j) * EPC) : make_uint4(0, 0, 0, 0);
    }
    // registers -> LDS (rows row0 .. row0 + 63 of the tile)
    __device__ static __forceinline__ void store(S* t, const uint4 (&r)[PER_THREAD], int row0 = 0)
    {
#pragma unroll
        for (int j = 0; j < PER_THREAD; ++j) *(uint4*)&t[off(row0 + row_of(j), chunk_of(j))] = r[j];
    }

    // 8-slot operand fragment: elements [e0, e0 + 8) of row r (e0 % 8 == 0)
    __device__ static __forceinline__ F row8(const S* t, int r, int e0)
    {
        if (T::bytes == 2) return T::ld8(&t[off(r, e0 / EPC)]);
        return T::ld44(&t[off(r, e0 / EPC)], &t[off(r, e0 / EPC + 1)]);
    }

    // 8-slot operand fragment of the transposed tile: lane (i = lane % 16,
    // g = lane / 16) receives column c0 + i at rows kb + 8g + j, j = 0..7
    // (c0 % 16 == 0).
    __device__ static __forceinline__ F col8(const S* t, int kb, int c0)
    {
        const int lane = threadIdx.x & 63, g = lane >> 4, i = lane & 15;
        const int r = kb + 8 * g;
        if constexpr (T::bytes == 2) {
            // 16-bit: two transposed reads of 4 rows each
            const int e = c0 + 4 * (i & 3);
            const S* p0 = &t[off(r + (i >> 2), e / EPC) + (e % EPC)];
            const S* p1 = &t[off(r + 4 + (i >> 2), e / EPC) + (e % EPC)];
            const bf16x4 lo = lds_read_tr4((const uint16_t*)p0), hi = lds_read_tr4((const uint16_t*)p1);
            return F{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        } else {
            const int e = c0 + i;
            F f;
#pragma unroll
            for (int j = 0; j < 8; ++j) f[j] = t[off(r + j, e / EPC) + (e % EPC)];
            return f;
        }
    }
};

}  // namespace tile
}  // namespace elsaa
