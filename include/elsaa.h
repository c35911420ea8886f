/*
 * elsaa.h -- C ABI of the ELSAA attention operator on AMD Instinct MI355X (gfx950).
 *
 * ELSAA ("Efficient Low-Rank and Sparse Approximation of Attention")
 * replaces dense softmax attention of one head by two branches and a fusion:
 *   - a sparse branch (sortLSH, Alg. 4; causal divide-and-conquer, Alg. 5):
 *     queries and keys are hashed with a sign hash, sorted by bucket, cut
 *     into equal blocks of b keys, and each query takes exact exp-weighted
 *     sums over its block: O_s = N_s / (d_s + eps), d_s = sum of e^{z};
 *   - a low-rank branch (RACE, Alg. 2; causal chunked form, Alg. 3): soft
 *     hypercube-hash features phi(x) of L tables with 2^gamma buckets give
 *     O_lr = Num / (Den + eps) and the denominator proxy d_lr = Den;
 *   - the denominator-aware fusion (Eq. m_sparse, Eq. elsaa_fusion_output,
 *     log-sum-exp form of Alg. 6):
 *        m = d_s / (d_s + lambda d_lr + eps),
 *        O = g_s * m * O_s + g_lr * O_lr.
 * The backward returns dQ, dK, dV (and optionally the gate gradients) with
 * the selection held fixed; the paper does not write a backward, it is the
 * exact gradient of the forward above.
 *
 * Tensor layout: Q, K, V, O, dO, dQ, dK, dV are [B, H, N, d_h] contiguous
 * row-major in the storage dtype (float32 or bfloat16); all accumulation is
 * float32.  Per-row outputs (lse, d_lr) are float32 [B, H, N].  The hash
 * projections are float32: W_sort [H, sort_bits, d_h] and
 * W_race [H, L, race_bits, d_h] with L = r / 2^race_bits, shared across the
 * batch.  gates is float32 [B, H, N, 2] = (g_sparse, g_lr) or NULL (all 1).
 *
 * Memory: every pointer except cfg is a device pointer owned by the caller.
 * The library never allocates or frees device memory and never synchronises
 * the caller's stream: it enqueues kernels and returns; results are valid
 * once the given stream has completed.  `saved` (elsaa_saved_bytes) is
 * written by elsaa_fwd and read by elsaa_bwd; `workspace`
 * (elsaa_workspace_bytes) is scratch for one call and may be reused by the
 * next call on the same stream.  Calls that share a workspace on different
 * streams race.
 *
 * Library-owned HIP objects: on its first call on a device, elsaa_fwd
 * creates one non-blocking stream of default priority and two events on
 * that device and keeps them until the process ends.  Each elsaa_fwd call
 * records an event on the given stream, runs the sort of the selection on
 * that second stream while the given stream runs the low-rank branch, and
 * makes the given stream wait for the second stream before the sparse
 * kernels (also when a launch in between failed), so the call behaves as if
 * everything ran on the given stream.  Concurrent elsaa_fwd calls on one
 * device share the second stream, so their sorts run one after another.
 *
 * Graph capture: elsaa_fwd and elsaa_bwd enqueue only kernels and event
 * record / wait pairs, so both can be captured into a HIP graph on the given
 * stream (the second stream joins the capture through the fork event) and
 * replayed; make one uncaptured call on the device first, which creates the
 * second stream and caches launch geometry.
 *
 * Errors: every entry point validates all arguments on the host before any
 * launch, so a rejected call writes nothing and leaves the stream untouched.
 * It returns a negative elsaa_status; elsaa_last_error() gives a message
 * (thread-local, valid until the next call on the same thread).
 */
#ifndef ELSAA_H
#define ELSAA_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    ELSAA_OK = 0,
    ELSAA_ERR_INVALID_ARG = -1,   /* null pointer, out-of-range value */
    ELSAA_ERR_UNSUPPORTED = -2,   /* valid for the method, not implemented on the GPU path */
    ELSAA_ERR_WORKSPACE = -3,     /* saved / workspace buffer smaller than required */
    ELSAA_ERR_HIP = -4            /* a HIP launch or runtime call failed */
} elsaa_status;

typedef enum { ELSAA_F32 = 0, ELSAA_BF16 = 1 } elsaa_dtype;

typedef struct {
    int32_t B, H, N, d_h;   /* batch, heads, sequence length, head dim (64 or 128);         */
                            /* GPU path: N <= 2^26 and N * d_h * element bytes < 2^32        */
    int32_t k;              /* sortLSH block size b: keys per sorted block, 1 <= k           */
    int32_t r;              /* RACE features L * 2^race_bits (the low-rank rank)             */
    int32_t race_bits;      /* gamma, hash bits per RACE table (GPU path: 4)                 */
    int32_t sort_bits;      /* gamma_sort, sign-hash bits of the sortLSH selector (1..8)      */
    int32_t n0;             /* causal base length N_0 of Alg. 5; <= 0 selects 2k             */
    int32_t causal;         /* 0: Alg. 1 / 2 / 4;  1: Alg. 6 / 3 / 5                          */
    int32_t dtype;          /* elsaa_dtype of Q,K,V,O,dO,dQ,dK,dV                             */
    float beta;             /* RACE temperature beta > 0 (Alg. 2)                            */
    float lambda;           /* fusion coefficient lambda >= 0 (Eq. m_sparse)                 */
    float eps;              /* numerical floor eps > 0                                       */
    float scale;            /* score scale tau; <= 0 selects 1/sqrt(d_h)                     */
    int32_t neighbors;      /* r >= 0: each sorted query block also sees the r neighbouring  */
                            /* sorted key blocks on each side (Sec. 6; 0 = the main setting)  */
    int32_t m_one;          /* 1: m_sparse = 1, the Sort_Lsh_RACE ablation (Sec. 7); 0: ELSAA */
} elsaa_config;

/* Number of causal recursion levels Lv (0 for non-causal).  Alg. 5 splits
 * every list longer than n0 into halves, padding an odd list with one zero
 * token first, so the lists at depth l all have L_l entries with L_0 = N,
 * L_{l+1} = ceil(L_l / 2), and Lv is the smallest depth with L_Lv <= n0.
 * Returns a negative status where a past half would have to hold a zero
 * token (fewer real tokens than half its list; never for n0 >= 2 * Lv). */
int elsaa_num_levels(const elsaa_config* cfg);

/* Entries of perm_q / perm_k per (b, h): N non-causal; causal the sum over
 * levels l < Lv of 2^l * L_{l+1} (= Lv * N / 2 when no list is padded). */
int64_t elsaa_perm_length(const elsaa_config* cfg);

/* Bytes of the `saved` buffer elsaa_fwd fills and elsaa_bwd reads, and of
 * the per-call scratch `workspace` (pass 0: elsaa_fwd / elsaa_select,
 * pass 1: elsaa_bwd).  Validates cfg. */
int elsaa_saved_bytes(const elsaa_config* cfg, size_t* bytes);
int elsaa_workspace_bytes(const elsaa_config* cfg, int pass, size_t* bytes);

/* Byte offsets inside `saved` (each 256-byte aligned):
 *   perm_q, perm_k  int32 sorted index lists (layout as elsaa_select);
 *   m               float32 [B,H,N] denominator-aware multiplier;
 *   o_sparse        float32 [B,H,N,d_h] sparse-branch output O_s (float32:
 *                   the backward's <dO, O_s> cancels against <dO, V_j> of
 *                   the dominant keys when attention is peaked);
 *   o_lowrank       storage dtype [B,H,N,d_h] low-rank output O_lr (its
 *                   weights are diffuse, so <dO, O_lr> has no such
 *                   cancellation);
 *   u_q, u_k        float32 [B,H,N,P] tanh of the RACE projections, t = tanh(W_race x),
 *                   of the Q and K rows (P = 4 L rounded up to 8, 16, 32 or 64;
 *                   padded tables 0);
 *   race_states     float32 RACE segment states phi(k) V' and phi(k) of the key
 *                   rows before each sequence segment (causal; the totals when
 *                   non-causal), [B*H][segments][r_p * d_h + r_p] with r_p = r
 *                   rounded up to 32, 64, 128 or 256; the segment length is an
 *                   internal choice, so only the library reads this region. */
typedef struct {
    size_t perm_q, perm_k, m, o_sparse, o_lowrank, u_q, u_k, race_states, total;
} elsaa_saved_layout;
int elsaa_get_saved_layout(const elsaa_config* cfg, elsaa_saved_layout* out);

/* Selection (Alg. 4 steps Hash / Sort / Partition; per level of Alg. 5).
 * Hash: bit t of a row x is set iff the float32 fused multiply-add chain
 * p = fma(W_sort[h][t][e], x[e], p) over e = 0..d_h-1 is > 0; the bucket key
 * is the position of that bit code in the reflected Gray sequence, so
 * neighbouring buckets differ in one bit ("sorted Hamming LSH", Sec. 3).
 * Sort: ascending by (key, token index), ties to the lower index.
 * Output (int32 token indices within one (b,h)):
 *   non-causal: perm_q, perm_k [B,H,N]; sorted block t = positions
 *               [t*k, (t+1)*k) and query block t sees key block t;
 *   causal:     perm_q, perm_k [B,H,P] (P = elsaa_perm_length); level l
 *               holds its 2^l segments in order, each giving its future
 *               half's queries (perm_q) and its past half's keys (perm_k)
 *               sorted, L_{l+1} entries each (elsaa_num_levels); a segment
 *               spans the real tokens [a, a + r) of its list, the rest of the
 *               list being Alg. 5's zero tokens, which trail future halves
 *               only: they take the bucket of the zero vector (key 0), sort
 *               after the real tokens of that bucket, and appear in perm_q
 *               as -1.  Without padding this is [B,H,Lv,N/2]. */
int elsaa_select(const elsaa_config* cfg, const void* Q, const void* K, const float* W_sort,
                 int32_t* perm_q, int32_t* perm_k, void* workspace, size_t workspace_bytes,
                 hipStream_t stream);

/* The selection above for callers that cannot allocate: code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation.  Same
 * arguments and results as elsaa_select (perm_q, perm_k are the caller's),
 * without `workspace`: the hash keys (2 * B*H*N bytes, each half 256-byte
 * aligned) go to a fixed 32 MiB device array inside the library, which every
 * device the library runs on holds until the process ends.  Rejects
 * B*H*N above 16777088 tokens with ELSAA_ERR_WORKSPACE before any launch.
 * Calls no allocating routine (the device address of the array is looked up
 * once per device, on the first call with that device current).  All calls
 * on one device share the array: calls that overlap on one device (other
 * streams, other threads) race; calls on one stream are ordered. */
int elsaa_select_noalloc(const elsaa_config* cfg, const void* Q, const void* K, const float* W_sort,
                         int32_t* perm_q, int32_t* perm_k, hipStream_t stream);

/* Forward (Alg. 1 / Alg. 6 without the projections).  gates is [B,H,N,2]
 * float32 (g_sparse, g_lr) or NULL (all 1); lambda_rows is the per-token
 * coefficient lambda_i of Eq. m_sparse, [B,H,N] float32 >= 0, or NULL (the
 * scalar cfg->lambda for every token).  Writes
 *   O        [B,H,N,d_h] storage dtype, fused output;
 *   lse      [B,H,N] float32, log d_sparse (log of the sparse denominator);
 *   d_lr     [B,H,N] float32, RACE denominator proxy Den;
 *   saved    selection, m, O_s, O_lr, the RACE projections and states for
 *            the backward (elsaa_saved_layout). */
int elsaa_fwd(const elsaa_config* cfg, const void* Q, const void* K, const void* V,
              const float* W_sort, const float* W_race, const float* gates, const float* lambda_rows,
              void* O, float* lse, float* d_lr, void* saved, size_t saved_bytes,
              void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Backward.  dO is the upstream gradient of O; gates, lambda_rows, lse, d_lr
 * and saved are what elsaa_fwd was given / wrote for the same inputs.
 * Writes dQ, dK, dV [B,H,N,d_h] (storage dtype) and, when not NULL,
 * dgates [B,H,N,2] float32 (d/dg_sparse, d/dg_lr) and dlambda [B,H,N]
 * float32 (d/dlambda_i; the gradient of a scalar lambda is their sum, that
 * of lambda = exp(l) is lambda times it; zero when m_one).  W_sort is not
 * read (the selection comes from saved) and may be NULL. */
int elsaa_bwd(const elsaa_config* cfg, const void* Q, const void* K, const void* V,
              const float* W_sort, const float* W_race, const float* gates, const float* lambda_rows,
              const void* dO, const float* lse, const float* d_lr, const void* saved, size_t saved_bytes,
              void* dQ, void* dK, void* dV, float* dgates, float* dlambda,
              void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Token-wise rules that feed the fusion: the gate network and the
 * query-dependent lambda.
 *   gates (Sec. 3.3, Alg. 1; the two-layer SiLU MLP with two independent,
 *   unnormalised sigmoid outputs of the experimental setup):
 *       (g_sparse, g_lr)_i = sigmoid(W2 SiLU(W1 q_i + b1) + b2)
 *   lambda (the query-dependent coefficient of the ELSAA configuration
 *   appendix, q_i detached from this path):
 *       lambda_i = max(lambda_min, c + sigmoid(w . q_i + b))
 * q_i is row i of the head's Q; every head has its own parameters.  The
 * caller keeps c >= 0 (it is used as given); lambda_min is 1e-6 in the paper.
 * Layouts (float32, contiguous, W1 and w 16-byte aligned):
 *   W1 [H, G, d_h], b1 [H, G], W2 [H, 2, G] (row 0 -> g_sparse), b2 [H, 2];
 *   w [H, d_h], b [H], c [H].
 * gate_hidden G is 0 (no gate network), 64 or 128 (the paper's text and
 * vision widths); lambda_rule is 0 or 1; at least one must be on.  Pointers
 * of a rule that is off are not read. */
typedef struct {
    int32_t gate_hidden;
    const float* W1;
    const float* b1;
    const float* W2;
    const float* b2;
    int32_t lambda_rule;
    const float* lam_w;
    const float* lam_b;
    const float* lam_c;
    float lambda_min;
} elsaa_token_rules;

/* Forward of the rules: writes gates [B,H,N,2] (when gate_hidden > 0) and
 * lambda_rows [B,H,N] (when lambda_rule), both float32, ready to pass to
 * elsaa_fwd / elsaa_bwd.  Q is the operator's Q (cfg->dtype storage). */
int elsaa_token_rules_fwd(const elsaa_config* cfg, const elsaa_token_rules* rules, const void* Q,
                          float* gates, float* lambda_rows, hipStream_t stream);

/* Bytes of the workspace elsaa_token_rules_bwd needs (per-workgroup partial
 * sums of the parameter gradients). */
int elsaa_token_rules_workspace_bytes(const elsaa_config* cfg, const elsaa_token_rules* rules,
                                      size_t* bytes);

/* Backward of the rules, given dgates and dlambda (what elsaa_bwd wrote):
 *   dQ      accumulated IN PLACE: dQ += d/dQ of sum(dgates * gates), the
 *           gate network's contribution (the lambda path is detached);
 *           NULL skips it;
 *   dW1, db1, dW2, db2, dlam_w, dlam_b, dlam_c: parameter gradients with the
 *           shapes of the parameters, summed over B and N (overwritten);
 *           any may be NULL.
 * dgates is read when gate_hidden > 0, dlambda when lambda_rule.  The sums
 * are taken in a fixed order (deterministic). */
int elsaa_token_rules_bwd(const elsaa_config* cfg, const elsaa_token_rules* rules, const void* Q,
                          const float* dgates, const float* dlambda, void* dQ,
                          float* dW1, float* db1, float* dW2, float* db2,
                          float* dlam_w, float* dlam_b, float* dlam_c,
                          void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Dense projections of the attention block (Alg. 1 and Alg. 6: Q = X W_Q,
 * K = X W_K, V = X W_V before the operator, O_head W_O after it; the paper
 * keeps these matrices dense, Sec. 1 and the parameter-overhead appendix).
 *
 * elsaa_gemm computes C = op(A) op(B) with op(A) [M,K], op(B) [K,N],
 * C [M,N], bfloat16 operands and float32 accumulation; C is bfloat16 or
 * float32 (c_dtype).  op(X) = X, or X^T when trans_x = 1, of the STORED
 * matrix X: A is stored [M,K] (trans_a = 0) or [K,M] (trans_a = 1), B is
 * stored [K,N] (trans_b = 0) or [N,K] (trans_b = 1).
 *
 * Each stored matrix (and C) is in one of two layouts, chosen per operand:
 *   plain       row-major with row stride ld (elements), ld >= its columns;
 *   head-major  (x_heads = Hx > 0) the stored matrix of R rows and Hx * dh
 *               columns is kept as [R / seq][Hx][seq][dh] contiguous: row
 *               r = b * seq + n, column c = h * dh + e lives at
 *               ((b * Hx + h) * seq + n) * dh + e.  This is the [B,H,N,d_h]
 *               layout of Q, K, V, O and their gradients, so the projections
 *               read and write attention tensors without a reshape copy.
 *               dh = columns / Hx must be a multiple of 8 and R a multiple
 *               of seq; ld is ignored.
 * Requirements: M, N, K >= 1 and multiples of 8, plain ld multiples of 8,
 * pointers 16-byte aligned, A / B / C not overlapping.  A and B are never
 * written.  When the output has few tiles and K is long, the K range is
 * split over workgroups whose float32 partial products go to `workspace`
 * (elsaa_gemm_workspace_bytes; 0 when no split is used) and are summed in a
 * fixed order, so results are deterministic run to run. */
typedef struct {
    int32_t M, N, K;
    int32_t trans_a, trans_b;
    int64_t lda, ldb, ldc;
    int32_t a_heads, b_heads, c_heads;   /* 0 = plain, Hx > 0 = head-major */
    int32_t seq;                         /* rows per sequence of head-major operands */
    int32_t c_dtype;                     /* elsaa_dtype of C */
} elsaa_gemm_desc;

int elsaa_gemm_workspace_bytes(const elsaa_gemm_desc* desc, size_t* bytes);
int elsaa_gemm(const elsaa_gemm_desc* desc, const void* A, const void* B, void* C,
               void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Opt-in kernel timing.  While enabled, every kernel launch of the library
 * is bracketed by two HIP events recorded on its stream (one extra event pair
 * per launch, no synchronisation); elsaa_profile_count / elsaa_profile_get
 * wait for the recorded launches and report, per kernel name, the summed
 * event time in milliseconds and the number of launches.  Enabling clears
 * the previous totals.  Process-wide; disabled by default. */
int elsaa_profile_enable(int on);
int elsaa_profile_count(void);
int elsaa_profile_get(int index, char* name, size_t name_len, double* total_ms, int64_t* launches);

const char* elsaa_status_string(int status);
const char* elsaa_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* ELSAA_H */
