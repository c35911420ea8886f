// internal.hpp -- launchers shared between the library's own source files.
// Not part of the public C ABI (include/elsaa.h).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "causal.hpp"

namespace elsaa {

// Validated shape information of one operator call.
struct Shape {
    int B, H, N, D;       // D = head dim (64 or 128)
    int k;                // sortLSH block size
    int r, L, Lp;         // RACE features, tables, tables padded to a multiple of 4
    int sort_bits;
    int Lv;               // causal recursion levels (0 non-causal)
    int n_leaf;           // causal leaf list length (real tokens plus zero tokens)
    LevelTiles lt;        // causal recursion geometry (causal.hpp)
    int causal;
    int bf16;             // storage dtype: 1 bf16, 0 float32
    float beta, lambda, eps, tau;
    int seg_len, nseg;    // RACE sequence segments (multiple of the 64-token chunk)
    int neighbors;        // r neighbouring sorted blocks on each side
    int m_one;            // m_sparse fixed to 1
    int64_t P() const { return causal ? lt.off[Lv] : (int64_t)N; }  // perm length per (b,h)
};

// Record an error message for elsaa_last_error() and return `code`.
int api_fail(int code, const char* fmt, ...);
int api_hip_fail(hipError_t e, const char* what);

// Opt-in per-kernel event timing (elsaa_profile_enable): construct around a
// launch; records an event pair on the stream when profiling is on.
class ProfScope {
public:
    ProfScope(const char* name, hipStream_t st);
    ~ProfScope();
    ProfScope(const ProfScope&) = delete;
    ProfScope& operator=(const ProfScope&) = delete;

private:
    hipStream_t stream_;
    bool active_;
};

// hipLaunchKernelGGL with profiling: ELSAA_LAUNCH("name", kernel, grid, block, lds, stream, args...)
#define ELSAA_LAUNCH(name, kernel, grid, block, lds, stream, ...)                 \
    do {                                                                           \
        ::elsaa::ProfScope prof_scope_(name, stream);                              \
        hipLaunchKernelGGL(kernel, grid, block, lds, stream, __VA_ARGS__);         \
    } while (0)

// selection: hash keys (and the RACE projections U = W_race x when W_race
// is not null, [BH][N][race_proj_stride]) then per-segment stable counting sort
// (Q and K in one launch)
hipError_t launch_project(const Shape& s, const void* Q, const void* K, const float* W_sort,
                          const float* W_race, uint8_t* keyq, uint8_t* keyk, float* Uq, float* Uk,
                          hipStream_t st);
hipError_t launch_sort(const Shape& s, const uint8_t* keyq, const uint8_t* keyk, int32_t* perm_q,
                       int32_t* perm_k, hipStream_t st);

// RACE low-rank branch
int race_padded_features(int r);            // r rounded up to 32, 64, 128 or 256
int race_proj_stride(const Shape& s);        // floats per row of U (padded 4 * tables)
size_t race_state_floats(const Shape& s);    // floats of one set of segment states
bool race_fwd_fits(const Shape& s);          // kernels' LDS fits for this dtype / d / r
bool race_bwd_fits(const Shape& s);
// segment states S = mul * sum phi(u) (scale * val)', A = mul * sum aw phi(u);
// scan_mode 0: total in every segment, 1: exclusive prefix, 2: exclusive suffix
hipError_t launch_race_states(const Shape& s, const float* U, const void* Val, const float* vscale,
                              const float* aw, float mul, float* states, int scan_mode, hipStream_t st);
hipError_t launch_race_fwd(const Shape& s, const float* Uq, const float* Uk, const void* V,
                           float* states, void* O_lr, float* d_lr, hipStream_t st);
size_t race_wt_bytes(const Shape& s);       // one of the W' hi / lo buffers
int race_wk(const Shape& s);                // columns of W' and of a du row (4 L padded to 32)
// states_f: the forward's segment prefix states (elsaa_fwd keeps them in saved);
// du_q, du_k: gradients of the RACE projections of the Q / K rows, storage
// dtype [BH][N][race_wk]; dv_lr: storage dtype [BH][N][D]; wt_hi / wt_lo receive W'
hipError_t launch_race_bwd(const Shape& s, const float* Uq, const float* Uk, const void* V,
                           const void* dO, const float* W_race, const float* rs,
                           const float* states_f, float* states_b, void* wt_hi, void* wt_lo,
                           void* du_q, void* du_k, void* dv_lr, hipStream_t st);

// which kernels of a sparse-branch pass to launch: the causal levels (they
// need only the selection), the rest (leaf or sorted blocks, which also need
// the low-rank branch), or both.  The backward's rest can be split into its
// dQ kernel and its dK, dV kernel (the whole-block kernel counts as dQ).
enum SparsePart {
    kSparseLevels = 1,
    kSparseFinalQ = 2,
    kSparseFinalKV = 4,
    kSparseFinal = kSparseFinalQ | kSparseFinalKV,
    kSparseAll = kSparseLevels | kSparseFinal
};

// sortLSH sparse branch forward + fusion epilogue; the causal level partials
// part_o ([BH][Lv][N/2][D]) are kept in the storage dtype
hipError_t launch_sparse_fwd(const Shape& s, const void* Q, const void* K, const void* V,
                             const int32_t* perm_q, const int32_t* perm_k, const float* gates,
                             const float* lambda_rows,
                             const void* O_lr, const float* d_lr, void* part_o, float* part_lse,
                             void* O, float* lse, float* m, float* O_s, hipStream_t st,
                             int parts = kSparseAll);

// backward: per-row scalars rs[5][BHN] (log2(d_s+eps), Delta, sc_s, sc_lr, dDen)
hipError_t launch_bwd_rows(const Shape& s, const void* dO, const float* Os, const void* Olr,
                           const float* m, const float* lse, const float* dlr, const float* gates,
                           const float* lambda_rows, float* rs, float* dgates, float* dlambda,
                           hipStream_t st);
// sparse backward; adds the low-rank parts (du W' for dQ and dK, the dV rows)
// and writes dQ, dK, dV; the causal level partials part_dq / part_dk / part_dv
// ([BH][Lv][N/2][D]) are kept in the storage dtype
hipError_t launch_sparse_bwd(const Shape& s, const void* Q, const void* K, const void* V,
                             const void* dO, const int32_t* perm_q, const int32_t* perm_k,
                             const float* rs, const void* du_q, const void* du_k, const void* wt_hi,
                             const void* wt_lo, const void* dv_lr, void* part_dq, void* part_dk, void* part_dv,
                             void* dQ, void* dK, void* dV, hipStream_t st, int parts = kSparseAll);

// token-wise rules: gate network and query-dependent lambda (token_rules.hip)
struct TrParams {
    int G;                              // gate hidden width: 0, 64 or 128
    int lam;                            // 1: lambda rule on
    const float *W1, *b1, *W2, *b2;     // [H][G][D], [H][G], [H][2][G], [H][2]
    const float *lw, *lb, *lc;          // [H][D], [H], [H]
    float lam_min;
};
struct TrGrads {
    float *dW1, *db1, *dW2, *db2, *dlw, *dlb, *dlc;   // any may be null
};
// float offsets of one workgroup's partial sums of the parameter gradients
struct TrLayout {
    int G, D, lam;
    __host__ __device__ constexpr int w1() const { return 0; }
    __host__ __device__ constexpr int lw() const { return G * D; }
    __host__ __device__ constexpr int b1() const { return lw() + (lam ? D : 0); }
    __host__ __device__ constexpr int w2() const { return b1() + G; }
    __host__ __device__ constexpr int b2() const { return w2() + 2 * G; }
    __host__ __device__ constexpr int lb() const { return b2() + (G ? 2 : 0); }
    __host__ __device__ constexpr int lc() const { return lb() + (lam ? 1 : 0); }
    __host__ __device__ constexpr int total() const { return lc() + (lam ? 1 : 0); }
    __host__ __device__ constexpr int stride() const { return (total() + 63) & ~63; }
};
size_t token_rules_workspace_bytes(const Shape& s, int G, bool lam);
hipError_t launch_token_rules_fwd(const Shape& s, const TrParams& p, const void* Q, float* gates,
                                  float* lambda_rows, hipStream_t st);
// dQ (may be null) is accumulated in place; part: token_rules_workspace_bytes
hipError_t launch_token_rules_bwd(const Shape& s, const TrParams& p, const void* Q, const float* dgates,
                                  const float* dlambda, void* dQ, const TrGrads& gr, float* part,
                                  hipStream_t st);

}  // namespace elsaa
