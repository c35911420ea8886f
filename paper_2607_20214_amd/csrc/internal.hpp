// internal.hpp -- launchers shared between the library's own source files.
// Not part of the public C ABI (include/elsaa.h).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace elsaa {

// Validated shape information of one operator call.
struct Shape {
    int B, H, N, D;       // D = head dim (64 or 128)
    int k;                // sortLSH block size
    int r, L, Lp;         // RACE features, tables, tables padded to a multiple of 4
    int sort_bits;
    int Lv;               // causal recursion levels (0 non-causal)
    int n_leaf;           // causal leaf length N / 2^Lv
    int causal;
    int bf16;             // storage dtype: 1 bf16, 0 float32
    float beta, lambda, eps, tau;
    int seg_len, nseg;    // RACE sequence segments (multiple of the 64-token chunk)
    int64_t P() const { return causal ? (int64_t)Lv * (N / 2) : (int64_t)N; }  // perm length per (b,h)
};

// selection: hash keys then per-segment stable counting sort
hipError_t launch_hash(const Shape& s, const void* X, const float* W_sort, uint8_t* keys,
                       hipStream_t st);
hipError_t launch_sort(const Shape& s, const uint8_t* keyq, const uint8_t* keyk, int32_t* perm_q,
                       int32_t* perm_k, hipStream_t st);

// RACE low-rank branch forward: segment states, scan, readout
hipError_t launch_race_fwd(const Shape& s, const void* Q, const void* K, const void* V,
                           const float* W_race, float* states, void* O_lr, float* d_lr,
                           hipStream_t st);

// sortLSH sparse branch forward + fusion epilogue
hipError_t launch_sparse_fwd(const Shape& s, const void* Q, const void* K, const void* V,
                             const int32_t* perm_q, const int32_t* perm_k, const float* gates,
                             const void* O_lr, const float* d_lr, float* part_o, float* part_lse,
                             void* O, float* lse, float* m, void* O_s, hipStream_t st);

}  // namespace elsaa
