// tile.hpp -- LDS tiles of gathered rows for the sparse-branch kernels.
//
// A tile holds rows of D elements, row-major with a pad of 8 elements per
// row.  Row r of the tile is placed in LDS row slot slot_of(r), a fixed
// permutation of the row index's low five bits, chosen so that the three
// access patterns of the kernels hit distinct LDS banks:
//   * 16-byte operand reads of 16 rows (consecutive rows, or the interleaved
//     row order of key_of / krow_of), one chunk per lane;
//   * transposed operand reads (ds_read_b64_tr_b16): 4 consecutive rows by
//     32 contiguous bytes per 16-lane group;
//   * 16-byte stores of whole rows by consecutive lanes.
// Within a row, elements stay in order, so every operand address is one row
// base per lane plus compile-time offsets.  Rows are staged
// global -> registers -> LDS by all threads of the workgroup; the global
// loads of the next tile are issued before the current tile is consumed.
#pragma once
#include "common.hpp"

namespace elsaa {
namespace tile {

constexpr int kRows = 64;
constexpr int kPad = 8;

// LDS row slot of tile row r: low five bits (b0..b4) -> (b2^b4, b0, b1, b3, b4).
__device__ __forceinline__ int slot_of(int r)
{
    const int lo = (((r >> 2) ^ (r >> 4)) & 1) | ((r & 3) << 1) | (r & 24);
    return (r & ~31) | lo;
}

// Tiles of 64 rows of D elements staged by NT threads.
template <class T, int D, int NT = 256>
struct Tile {
    using S = typename T::store_t;
    using F = typename T::frag_t;
    static constexpr int EPC = 16 / T::bytes;         // elements per 16-byte chunk
    static constexpr int CPR = D / EPC;               // chunks per row
    static constexpr int LD = D + kPad;               // LDS row stride (elements)
    static constexpr int PER_THREAD = kRows * CPR / NT;   // chunks staged per thread
    static_assert(CPR >= 8 && PER_THREAD >= 1, "tile shape");

    // elements of an LDS tile of `rows` rows
    static constexpr int elems(int rows) { return rows * LD; }
    // element offset of row r
    __device__ static __forceinline__ int row(int r) { return slot_of(r) * LD; }
    // element offset of chunk c of row r
    __device__ static __forceinline__ int off(int r, int c) { return row(r) + c * EPC; }

    // Row of the j-th chunk thread tx stages (and the chunk index).  The
    // helpers take the thread index as an argument (default threadIdx.x):
    // a kernel that loops over work items passes a copy the compiler cannot
    // hoist, so lane addresses are formed where used, not kept in registers.
    __device__ static __forceinline__ int row_of(int j, int tx = threadIdx.x) { return (tx + NT * j) / CPR; }
    __device__ static __forceinline__ int chunk_of(int j, int tx = threadIdx.x) { return (tx + NT * j) % CPR; }

    // global -> registers: rows tok[j] (token index, -1 = none) of X.  The
    // byte offset from X fits 32 bits (rows of one head), so each address is
    // the uniform base plus one 32-bit register per lane.
    __device__ static __forceinline__ void load(const S* X, const int (&tok)[PER_THREAD], uint4 (&r)[PER_THREAD],
                                                int tx = threadIdx.x)
    {
#pragma unroll
        for (int j = 0; j < PER_THREAD; ++j) {
            const uint32_t off = (uint32_t)tok[j] * (uint32_t)(D * sizeof(S)) + (uint32_t)chunk_of(j, tx) * 16u;
            r[j] = tok[j] >= 0 ? ldg16((const char*)X + off) : make_uint4(0, 0, 0, 0);
        }
    }
    // the same when every tok[j] is a valid row (no per-row branch)
    __device__ static __forceinline__ void load_all(const S* X, const int (&tok)[PER_THREAD],
                                                    uint4 (&r)[PER_THREAD], int tx = threadIdx.x)
    {
#pragma unroll
        for (int j = 0; j < PER_THREAD; ++j) {
            const uint32_t off = (uint32_t)tok[j] * (uint32_t)(D * sizeof(S)) + (uint32_t)chunk_of(j, tx) * 16u;
            r[j] = ldg16((const char*)X + off);
        }
    }
    // registers -> LDS (rows row0 .. row0 + 63 of the tile)
    __device__ static __forceinline__ void store(S* t, const uint4 (&r)[PER_THREAD], int row0 = 0,
                                                 int tx = threadIdx.x)
    {
#pragma unroll
        for (int j = 0; j < PER_THREAD; ++j) *(uint4*)&t[off(row0 + row_of(j, tx), chunk_of(j, tx))] = r[j];
    }

    // 8-slot operand fragment: elements [e0, e0 + 8) of row r (e0 % 8 == 0)
    __device__ static __forceinline__ F row8(const S* t, int r, int e0)
    {
        const S* p = &t[row(r) + e0];
        if (T::bytes == 2) return T::ld8(p);
        return T::ld44(p, p + 4);
    }

    // 8-slot operand fragment of the transposed tile: lane (i = lane % 16,
    // g = lane / 16) receives column c0 + i at rows kb + 8g + j, j = 0..7
    // (c0 % 16 == 0).
    __device__ static __forceinline__ F col8(const S* t, int kb, int c0, int tx = threadIdx.x)
    {
        const int lane = tx & 63, g = lane >> 4, i = lane & 15;
        const int r = kb + 8 * g;
        if constexpr (T::bytes == 2) {
            // 16-bit: two transposed reads of 4 rows each
            const int e = c0 + 4 * (i & 3);
            const S* p0 = &t[row(r + (i >> 2)) + e];
            const S* p1 = &t[row(r + 4 + (i >> 2)) + e];
            const bf16x4 lo = lds_read_tr4((const uint16_t*)p0), hi = lds_read_tr4((const uint16_t*)p1);
            return F{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        } else {
            F f;
#pragma unroll
            for (int j = 0; j < 8; ++j) f[j] = t[row(r + j) + c0 + i];
            return f;
        }
    }
};

}  // namespace tile
}  // namespace elsaa
