/*
 * elsaa_oracle.c -- plain, slow CPU reference of the ELSAA attention operator.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may load or call this library.  The GPU
 * library never links, loads or calls it, and it shares no code with it.
 *
 * Everything is per attention head: Q, K, V are [N, d] row-major float
 * arrays (bf16 inputs are passed as the float32 holding the same value) and
 * all arithmetic is double precision, except the sortLSH sign hash, which
 * the paper leaves unspecified and which is fixed here as a float32 fused
 * multiply-add chain so that the selected indices are defined exactly.
 *
 * What each part follows (paper: "ELSAA: Efficient Low-Rank and Sparse
 * Approximation of Attention"):
 *   ora_hash            sortLSH hash H(.) of Alg. 4 (step "Hash"), sorted
 *                       Hamming LSH of Sec. 3 with the bit-vector ranked in
 *                       reflected-Gray order so adjacent buckets differ in
 *                       one bit.
 *   ora_select          Alg. 4 steps "Sort" and "Partition" (non-causal) and
 *                       the per-level SortLSH(Q_future, K_past) calls of
 *                       Alg. 5, in the layout the GPU library writes.
 *   ora_support         the key support S(i) of every query: one sorted
 *                       block (Alg. 4) or the causal divide-and-conquer of
 *                       Alg. 5 (leaf of exact causal attention, zero-token
 *                       padding of odd lengths, one future-past SortLSH call
 *                       per level), built by running that recursion.
 *   ora_features        RACE soft-hash features phi of Alg. 2 (softmax over
 *                       the hypercube vertices of beta*tanh(W x)).
 *   ora_forward         sparse sums of Alg. 4 over S(i) (exp-weighted value
 *                       sum and denominator, O_s = N_s/(d_s+eps)); RACE
 *                       numerator/denominator of Alg. 2 (non-causal) and of
 *                       Alg. 3 (causal: keys j <= i), O_lr = Num/(Den+eps);
 *                       denominator-aware multiplier of Eq. (m_sparse) in the
 *                       log-sum-exp form of Alg. 6; fused output of
 *                       Eq. (elsaa_fusion_output).
 *   ora_backward        exact gradient of ora_forward with respect to Q, K,
 *                       V (and the gate values and the per-token lambda_i)
 *                       with the selection, W_sort and W_race held fixed;
 *                       the paper gives no backward.
 * Variants the paper names: r neighbouring sorted blocks on each side of a
 * query's own block (Sec. 6 cost discussion, "Neighbor blocks" of the
 * hyper-parameter table; 0 in the main setting), a per-token coefficient
 * lambda_i (Eq. m_sparse with query-dependent lambda) and the Sort_Lsh_RACE
 * ablation that fixes m_sparse = 1 (Sec. 7).
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int32_t N, d;
    int32_t k;          /* sortLSH block size b */
    int32_t r;          /* RACE features L * 2^race_bits */
    int32_t race_bits;  /* gamma */
    int32_t sort_bits;  /* gamma_sort */
    int32_t n0;         /* causal base length N_0 */
    int32_t causal;
    double beta, lambda, eps, scale;  /* scale <= 0 -> 1/sqrt(d) */
    int32_t neighbors;  /* r neighbouring sorted blocks on each side (0 = own block only) */
    int32_t m_one;      /* 1: m_sparse = 1 (the Sort_Lsh_RACE ablation) */
} ora_cfg;

enum { ORA_OK = 0, ORA_EINVAL = -1, ORA_ENOMEM = -2 };

static double tau_of(const ora_cfg* c) { return c->scale > 0 ? c->scale : 1.0 / sqrt((double)c->d); }

static int cfg_ok(const ora_cfg* c)
{
    if (!c || c->N < 1 || c->d < 1 || c->k < 1 || c->race_bits < 1 || c->race_bits > 12 ||
        c->sort_bits < 1 || c->sort_bits > 8 || c->n0 < 1)
        return 0;
    if (c->r < (1 << c->race_bits) || c->r % (1 << c->race_bits)) return 0;
    if (!(c->eps > 0) || !(c->lambda >= 0) || !(c->beta > 0)) return 0;
    if (c->neighbors < 0 || (c->m_one != 0 && c->m_one != 1)) return 0;
    return 1;
}

/* ------------------------------------------------------------------------ */
/* Hash (Alg. 4, step "Hash")                                                */
/* ------------------------------------------------------------------------ */

/* Sign bits of W x for one row, each projection a float32 fmaf chain over
 * the coordinates in index order; bit t is set iff the projection is > 0. */
static uint32_t sign_code(int d, const float* x, int bits, const float* W)
{
    uint32_t code = 0;
    for (int t = 0; t < bits; ++t) {
        float p = 0.0f;
        for (int e = 0; e < d; ++e) p = fmaf(W[(size_t)t * d + e], x[e], p);
        if (p > 0.0f) code |= 1u << t;
    }
    return code;
}

/* Position of a code in the reflected Gray sequence (inverse Gray map). */
static uint32_t gray_rank(uint32_t code)
{
    uint32_t r = code;
    for (uint32_t s = code >> 1; s; s >>= 1) r ^= s;
    return r;
}

int ora_hash(int n, int d, const float* X, int bits, const float* W, uint8_t* key)
{
    if (n < 0 || d < 1 || bits < 1 || bits > 8 || !X || !W || !key) return ORA_EINVAL;
    for (int i = 0; i < n; ++i) key[i] = (uint8_t)gray_rank(sign_code(d, X + (size_t)i * d, bits, W));
    return ORA_OK;
}

/* ------------------------------------------------------------------------ */
/* Sort (Alg. 4, step "Sort"): ascending by (hash key, position)            */
/* ------------------------------------------------------------------------ */

typedef struct { uint32_t key; int32_t pos; } kp_t;

static int kp_cmp(const void* a, const void* b)
{
    const kp_t* x = (const kp_t*)a;
    const kp_t* y = (const kp_t*)b;
    if (x->key != y->key) return x->key < y->key ? -1 : 1;
    return (x->pos > y->pos) - (x->pos < y->pos);
}

/* order[p] = list position of the p-th element when sorted by (key, position). */
static void sort_positions(int n, const uint32_t* keys, int32_t* order, kp_t* tmp)
{
    for (int i = 0; i < n; ++i) { tmp[i].key = keys[i]; tmp[i].pos = i; }
    qsort(tmp, (size_t)n, sizeof(kp_t), kp_cmp);
    for (int i = 0; i < n; ++i) order[i] = tmp[i].pos;
}

/* Number of levels of the Alg. 5 recursion: every list longer than n0 is
 * padded to even length with one zero token (Alg. 5) and halved, so all
 * lists of depth l have L_l entries (L_0 = N, L_{l+1} = ceil(L_l / 2)) and
 * Lv is the smallest depth with L_Lv <= n0.  Zero tokens only trail future
 * halves; -1 if some past half would have to hold one (its list has fewer
 * real tokens than half its length), a case the sorted-list layout below
 * does not describe. */
int ora_num_levels(const ora_cfg* c)
{
    if (!cfg_ok(c)) return -1;
    if (!c->causal) return 0;
    int lv = 0;
    int64_t n = c->N, pads = 0;   /* pads: most zero tokens of a depth-lv list (all-future path) */
    while (n > c->n0) {
        const int64_t m = (n + 1) / 2;
        if (pads > n - m) return -1;
        pads += n & 1;
        n = m;
        ++lv;
    }
    return lv;
}

/* Entries per (b,h) of the causal sorted lists: level l has 2^l lists of
 * L_{l+1} entries. */
int64_t ora_perm_length(const ora_cfg* c)
{
    const int lv = ora_num_levels(c);
    if (lv < 0) return -1;
    if (!c->causal) return c->N;
    int64_t n = c->N, total = 0;
    for (int l = 0; l < lv; ++l) {
        n = (n + 1) / 2;
        total += n << l;
    }
    return total;
}

/* Sorted index lists in the layout the GPU library writes:
 *   non-causal: perm_q[N], perm_k[N] = token indices in sorted order;
 *   causal:     per level l, its 2^l segments in order, each contributing
 *               its future half's queries (perm_q) and its past half's keys
 *               (perm_k) sorted, L_{l+1} entries each.  A segment's list is
 *               a run of real tokens [a, a + r) followed by zero tokens; the
 *               zero tokens of a future half take the hash key of the zero
 *               vector, sort by (key, list position) with the real tokens,
 *               and are written as -1. */
int ora_select(const ora_cfg* c, const float* Q, const float* K, const float* Wsort,
               int32_t* perm_q, int32_t* perm_k)
{
    if (!cfg_ok(c) || !Q || !K || !Wsort || !perm_q || !perm_k) return ORA_EINVAL;
    const int N = c->N, d = c->d;
    uint8_t* kq = (uint8_t*)malloc((size_t)N);
    uint8_t* kk = (uint8_t*)malloc((size_t)N);
    uint32_t* kb = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)N);
    int32_t* ord = (int32_t*)malloc(sizeof(int32_t) * (size_t)N);
    kp_t* tmp = (kp_t*)malloc(sizeof(kp_t) * (size_t)N);
    int64_t* sa = NULL;        /* real range [sa, sa + sr) of each segment of the current depth */
    int64_t* sr = NULL;
    int rc = ORA_OK;
    if (!kq || !kk || !kb || !ord || !tmp) { rc = ORA_ENOMEM; goto done; }
    ora_hash(N, d, Q, c->sort_bits, Wsort, kq);
    ora_hash(N, d, K, c->sort_bits, Wsort, kk);
    if (!c->causal) {
        for (int i = 0; i < N; ++i) kb[i] = kq[i];
        sort_positions(N, kb, perm_q, tmp);
        for (int i = 0; i < N; ++i) kb[i] = kk[i];
        sort_positions(N, kb, perm_k, tmp);
    } else {
        const int lv = ora_num_levels(c);
        if (lv < 0) { rc = ORA_EINVAL; goto done; }
        float* zero = (float*)calloc((size_t)d, sizeof(float));
        uint8_t zk = 0;
        if (!zero) { rc = ORA_ENOMEM; goto done; }
        ora_hash(1, d, zero, c->sort_bits, Wsort, &zk);
        free(zero);
        sa = (int64_t*)malloc(sizeof(int64_t) << (lv > 0 ? lv : 1));
        sr = (int64_t*)malloc(sizeof(int64_t) << (lv > 0 ? lv : 1));
        if (!sa || !sr) { rc = ORA_ENOMEM; goto done; }
        sa[0] = 0;
        sr[0] = N;
        int64_t len = N, out = 0;
        for (int l = 0; l < lv; ++l) {
            const int64_t m = (len + 1) / 2;      /* halves after the zero-token padding of an odd list */
            for (int64_t s = 0; s < ((int64_t)1 << l); ++s) {
                const int64_t a = sa[s], r = sr[s];
                const int64_t rf = r > m ? r - m : 0;  /* real tokens of the future half */
                int32_t* oq = perm_q + out + s * m;
                int32_t* ok = perm_k + out + s * m;
                for (int64_t p = 0; p < m; ++p) kb[p] = p < rf ? kq[a + m + p] : zk;
                sort_positions((int)m, kb, ord, tmp);
                for (int64_t p = 0; p < m; ++p) oq[p] = ord[p] < rf ? (int32_t)(a + m + ord[p]) : -1;
                for (int64_t p = 0; p < m; ++p) kb[p] = kk[a + p];
                sort_positions((int)m, kb, ord, tmp);
                for (int64_t p = 0; p < m; ++p) ok[p] = (int32_t)(a + ord[p]);
            }
            /* the next depth: past child (a, m), future child (a + m, rf), in segment order */
            for (int64_t s = ((int64_t)1 << l) - 1; s >= 0; --s) {
                const int64_t a = sa[s], r = sr[s];
                sa[2 * s] = a;
                sr[2 * s] = m;
                sa[2 * s + 1] = a + m;
                sr[2 * s + 1] = r > m ? r - m : 0;
            }
            out += m << l;
            len = m;
        }
    }
done:
    free(kq); free(kk); free(kb); free(ord); free(tmp); free(sa); free(sr);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Support S(i): Alg. 4 blocks, or the Alg. 5 recursion                      */
/* ------------------------------------------------------------------------ */

#define PAD_TOKEN (-1)

typedef struct {
    const ora_cfg* c;
    const uint8_t* kq;   /* hash keys of the real queries */
    const uint8_t* kk;   /* hash keys of the real keys */
    uint32_t pad_key;    /* hash key of the zero token used for padding */
    int64_t* count;      /* per-query support size (pass 1) */
    int64_t* cursor;     /* per-query write cursor (pass 2) */
    int32_t* cols;       /* CSR columns (pass 2) */
    int fill;            /* 0 = count, 1 = fill */
    int failed;
} sup_ctx;

static void emit(sup_ctx* x, int32_t qi, int32_t kj)
{
    if (qi < 0 || kj < 0) return;   /* padding tokens are dropped on return */
    if (x->fill) x->cols[x->cursor[qi]++] = kj;
    else x->count[qi]++;
}

/* SortLSH(Qs, Ks; b) on token lists (Alg. 4): sort both lists by
 * (hash key, list position), cut into consecutive blocks of
 * b' = min(b, n) (the last block may be shorter), and let the t-th query
 * block see the t-th key block and its r neighbouring key blocks on each
 * side (r = neighbors, clipped to the list). */
static void sortlsh_lists(sup_ctx* x, const int32_t* qtok, int nq, const int32_t* ktok, int nk)
{
    int n = nq > nk ? nq : nk;
    uint32_t* keys = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)n);
    int32_t* oq = (int32_t*)malloc(sizeof(int32_t) * (size_t)nq);
    int32_t* ok = (int32_t*)malloc(sizeof(int32_t) * (size_t)nk);
    kp_t* tmp = (kp_t*)malloc(sizeof(kp_t) * (size_t)n);
    if (!keys || !oq || !ok || !tmp) { x->failed = 1; goto done; }
    for (int p = 0; p < nq; ++p) keys[p] = qtok[p] < 0 ? x->pad_key : x->kq[qtok[p]];
    sort_positions(nq, keys, oq, tmp);
    for (int p = 0; p < nk; ++p) keys[p] = ktok[p] < 0 ? x->pad_key : x->kk[ktok[p]];
    sort_positions(nk, keys, ok, tmp);
    {
        const int bq = x->c->k < nq ? x->c->k : nq;
        const int r = x->c->neighbors;
        for (int p = 0; p < nq; ++p) {
            const int t = p / bq;
            const int k0 = t - r > 0 ? (t - r) * bq : 0;
            const int k1 = (t + r + 1) * bq < nk ? (t + r + 1) * bq : nk;
            for (int q = k0; q < k1; ++q) emit(x, qtok[oq[p]], ktok[ok[q]]);
        }
    }
done:
    free(keys); free(oq); free(ok); free(tmp);
}

/* CausalSparse of Alg. 5 on a token list (real indices ascending, padding
 * tokens only at the end). */
static void causal_rec(sup_ctx* x, const int32_t* tok, int n)
{
    if (x->failed) return;
    if (n <= x->c->n0) {
        /* exact causal attention: every query sees itself and all earlier keys */
        for (int p = 0; p < n; ++p)
            for (int q = 0; q <= p; ++q) emit(x, tok[p], tok[q]);
        return;
    }
    const int np = n + (n & 1);
    int32_t* t2 = (int32_t*)malloc(sizeof(int32_t) * (size_t)np);
    if (!t2) { x->failed = 1; return; }
    memcpy(t2, tok, sizeof(int32_t) * (size_t)n);
    if (np > n) t2[n] = PAD_TOKEN;
    const int m = np / 2;
    causal_rec(x, t2, m);              /* past-past */
    causal_rec(x, t2 + m, m);          /* future-future */
    sortlsh_lists(x, t2 + m, m, t2, m);/* future-past */
    free(t2);
}

static int cmp_i32(const void* a, const void* b)
{
    int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
    return (x > y) - (x < y);
}

static int build_support(sup_ctx* x, int N, int64_t* rowptr, int32_t* cols)
{
    int32_t* tok = (int32_t*)malloc(sizeof(int32_t) * (size_t)N);
    if (!tok) return ORA_ENOMEM;
    for (int i = 0; i < N; ++i) tok[i] = i;
    for (int pass = 0; pass < 2; ++pass) {
        x->fill = pass;
        if (pass == 1) {
            rowptr[0] = 0;
            for (int i = 0; i < N; ++i) rowptr[i + 1] = rowptr[i] + x->count[i];
            if (!cols) break;
            x->cols = cols;
            for (int i = 0; i < N; ++i) x->cursor[i] = rowptr[i];
        }
        if (x->c->causal) causal_rec(x, tok, N);
        else sortlsh_lists(x, tok, N, tok, N);
        if (x->failed) { free(tok); return ORA_ENOMEM; }
    }
    free(tok);
    if (cols)
        for (int i = 0; i < N; ++i)
            qsort(cols + rowptr[i], (size_t)(rowptr[i + 1] - rowptr[i]), sizeof(int32_t), cmp_i32);
    return ORA_OK;
}

static int make_ctx(const ora_cfg* c, const float* Q, const float* K, const float* Wsort,
                    sup_ctx* x, uint8_t** kq, uint8_t** kk)
{
    const int N = c->N, d = c->d;
    memset(x, 0, sizeof(*x));
    x->c = c;
    *kq = (uint8_t*)malloc((size_t)N);
    *kk = (uint8_t*)malloc((size_t)N);
    x->count = (int64_t*)calloc((size_t)N, sizeof(int64_t));
    x->cursor = (int64_t*)calloc((size_t)N, sizeof(int64_t));
    float* zero = (float*)calloc((size_t)d, sizeof(float));
    if (!*kq || !*kk || !x->count || !x->cursor || !zero) { free(zero); return ORA_ENOMEM; }
    ora_hash(N, d, Q, c->sort_bits, Wsort, *kq);
    ora_hash(N, d, K, c->sort_bits, Wsort, *kk);
    uint8_t zk;
    ora_hash(1, d, zero, c->sort_bits, Wsort, &zk);
    x->pad_key = zk;
    free(zero);
    x->kq = *kq;
    x->kk = *kk;
    return ORA_OK;
}

static void free_ctx(sup_ctx* x, uint8_t* kq, uint8_t* kk)
{
    free(x->count); free(x->cursor); free(kq); free(kk);
}

/* Size of the support CSR: returns the total number of (query, key) pairs,
 * or a negative error code. */
int64_t ora_support_size(const ora_cfg* c, const float* Q, const float* K, const float* Wsort)
{
    if (!cfg_ok(c) || !Q || !K || !Wsort) return ORA_EINVAL;
    sup_ctx x; uint8_t *kq = NULL, *kk = NULL;
    int rc = make_ctx(c, Q, K, Wsort, &x, &kq, &kk);
    int64_t total = rc;
    if (rc == ORA_OK) {
        int64_t* rp = (int64_t*)malloc(sizeof(int64_t) * ((size_t)c->N + 1));
        if (!rp) total = ORA_ENOMEM;
        else {
            rc = build_support(&x, c->N, rp, NULL);
            total = rc == ORA_OK ? rp[c->N] : rc;
            free(rp);
        }
    }
    free_ctx(&x, kq, kk);
    return total;
}

/* Support CSR: rowptr[N+1]; cols[rowptr[N]] with each row's keys ascending. */
int ora_support(const ora_cfg* c, const float* Q, const float* K, const float* Wsort,
                int64_t* rowptr, int32_t* cols)
{
    if (!cfg_ok(c) || !Q || !K || !Wsort || !rowptr || !cols) return ORA_EINVAL;
    sup_ctx x; uint8_t *kq = NULL, *kk = NULL;
    int rc = make_ctx(c, Q, K, Wsort, &x, &kq, &kk);
    if (rc == ORA_OK) rc = build_support(&x, c->N, rowptr, cols);
    free_ctx(&x, kq, kk);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* RACE features (Alg. 2)                                                    */
/* ------------------------------------------------------------------------ */

/* phi[n][r]: for table l and vertex c (bit b of c set -> v_{c,b} = +1, else
 * -1), phi[l*2^g + c] = exp(beta * tanh(W_l x) . v_c) / sum over c'. */
int ora_features(int n, int d, const float* X, int L, int g, double beta, const float* Wrace,
                 double* phi)
{
    if (n < 0 || d < 1 || L < 1 || g < 1 || g > 12 || !X || !Wrace || !phi) return ORA_EINVAL;
    const int R = 1 << g;
    #pragma omp parallel
    {
        double* t = (double*)malloc(sizeof(double) * (size_t)g);
        double* e = (double*)malloc(sizeof(double) * (size_t)R);
        #pragma omp for schedule(static)
        for (int i = 0; i < n; ++i) {
            const float* x = X + (size_t)i * d;
            for (int l = 0; l < L; ++l) {
                for (int b = 0; b < g; ++b) {
                    const float* w = Wrace + ((size_t)l * g + b) * d;
                    double u = 0;
                    for (int q = 0; q < d; ++q) u += (double)w[q] * (double)x[q];
                    t[b] = tanh(u);
                }
                double mx = -INFINITY;
                for (int cc = 0; cc < R; ++cc) {
                    double s = 0;
                    for (int b = 0; b < g; ++b) s += ((cc >> b) & 1) ? t[b] : -t[b];
                    e[cc] = beta * s;
                    if (e[cc] > mx) mx = e[cc];
                }
                double den = 0;
                for (int cc = 0; cc < R; ++cc) { e[cc] = exp(e[cc] - mx); den += e[cc]; }
                double* out = phi + (size_t)i * L * R + (size_t)l * R;
                for (int cc = 0; cc < R; ++cc) out[cc] = e[cc] / den;
            }
        }
        free(t); free(e);
    }
    return ORA_OK;
}

/* ------------------------------------------------------------------------ */
/* Forward                                                                   */
/* ------------------------------------------------------------------------ */

typedef struct {
    /* per row, all N rows */
    double *Os, *lse, *Olr, *Den, *m, *logD;
} fwd_state;

static double dot(int d, const float* a, const float* b)
{
    double s = 0;
    for (int e = 0; e < d; ++e) s += (double)a[e] * (double)b[e];
    return s;
}

/* Sparse sums of Alg. 4 over the support of query i (max-shifted). */
static void sparse_row(const ora_cfg* c, const float* Q, const float* K, const float* V,
                       const int64_t* rp, const int32_t* cols, int i, double* Os, double* lse)
{
    const int d = c->d;
    const double tau = tau_of(c);
    const float* q = Q + (size_t)i * d;
    double mx = -INFINITY;
    for (int64_t p = rp[i]; p < rp[i + 1]; ++p) {
        double z = tau * dot(d, q, K + (size_t)cols[p] * d);
        if (z > mx) mx = z;
    }
    double s = 0;
    for (int e = 0; e < d; ++e) Os[e] = 0;
    for (int64_t p = rp[i]; p < rp[i + 1]; ++p) {
        const float* kv = K + (size_t)cols[p] * d;
        const float* vv = V + (size_t)cols[p] * d;
        double w = exp(tau * dot(d, q, kv) - mx);
        s += w;
        for (int e = 0; e < d; ++e) Os[e] += w * vv[e];
    }
    /* d_s = e^mx * s ; O_s = N_s / (d_s + eps) */
    double den = s + c->eps * exp(-mx);
    for (int e = 0; e < d; ++e) Os[e] /= den;
    *lse = mx + log(s);
}

/* RACE readout (Alg. 2 / Alg. 3) for all rows: Num_i, Den_i averaged over
 * the L tables; causal rows see keys j <= i. */
static int race_rows(const ora_cfg* c, const double* phq, const double* phk, const float* V,
                     double* Num, double* Den)
{
    const int N = c->N, d = c->d, r = c->r;
    const int L = r >> c->race_bits;
    double* A = (double*)calloc((size_t)r, sizeof(double));
    double* Bm = (double*)calloc((size_t)r * d, sizeof(double));
    if (!A || !Bm) { free(A); free(Bm); return ORA_ENOMEM; }
    if (!c->causal) {
        for (int j = 0; j < N; ++j)
            for (int f = 0; f < r; ++f) {
                const double ph = phk[(size_t)j * r + f];
                A[f] += ph;
                for (int e = 0; e < d; ++e) Bm[(size_t)f * d + e] += ph * V[(size_t)j * d + e];
            }
    }
    for (int i = 0; i < N; ++i) {
        if (c->causal) {
            /* running prefix state, key i included */
            for (int f = 0; f < r; ++f) {
                const double ph = phk[(size_t)i * r + f];
                A[f] += ph;
                for (int e = 0; e < d; ++e) Bm[(size_t)f * d + e] += ph * V[(size_t)i * d + e];
            }
        }
        double den = 0;
        double* nu = Num + (size_t)i * d;
        for (int e = 0; e < d; ++e) nu[e] = 0;
        for (int f = 0; f < r; ++f) {
            const double ph = phq[(size_t)i * r + f];
            den += ph * A[f];
            for (int e = 0; e < d; ++e) nu[e] += ph * Bm[(size_t)f * d + e];
        }
        for (int e = 0; e < d; ++e) nu[e] /= L;
        Den[i] = den / L;
    }
    free(A); free(Bm);
    return ORA_OK;
}

static double gate_of(const float* gates, int i, int which)
{
    return gates ? (double)gates[(size_t)i * 2 + which] : 1.0;
}

/* Full forward for one head into fwd_state (all rows; row_mask limits the
 * sparse sums to the marked rows when not NULL). */
static double lambda_of(const ora_cfg* c, const float* lam_rows, int i)
{
    return lam_rows ? (double)lam_rows[i] : c->lambda;
}

static int forward_all(const ora_cfg* c, const float* Q, const float* K, const float* V,
                       const float* Wsort, const float* Wrace, const float* lam_rows,
                       const uint8_t* row_mask, fwd_state* st, int64_t** rp_out, int32_t** cols_out)
{
    const int N = c->N, d = c->d, r = c->r;
    const int L = r >> c->race_bits;
    int rc;
    int64_t total = ora_support_size(c, Q, K, Wsort);
    if (total < 0) return (int)total;
    int64_t* rp = (int64_t*)malloc(sizeof(int64_t) * ((size_t)N + 1));
    int32_t* cols = (int32_t*)malloc(sizeof(int32_t) * (size_t)(total > 0 ? total : 1));
    double* phq = (double*)malloc(sizeof(double) * (size_t)N * r);
    double* phk = (double*)malloc(sizeof(double) * (size_t)N * r);
    if (!rp || !cols || !phq || !phk) { rc = ORA_ENOMEM; goto fail; }
    rc = ora_support(c, Q, K, Wsort, rp, cols);
    if (rc) goto fail;
    #pragma omp parallel for schedule(dynamic, 16)
    for (int i = 0; i < N; ++i) {
        if (row_mask && !row_mask[i]) continue;
        sparse_row(c, Q, K, V, rp, cols, i, st->Os + (size_t)i * d, st->lse + i);
    }
    ora_features(N, d, Q, L, c->race_bits, c->beta, Wrace, phq);
    ora_features(N, d, K, L, c->race_bits, c->beta, Wrace, phk);
    rc = race_rows(c, phq, phk, V, st->Olr, st->Den);
    if (rc) goto fail;
    for (int i = 0; i < N; ++i) {
        const double den = st->Den[i] + c->eps;
        for (int e = 0; e < d; ++e) st->Olr[(size_t)i * d + e] /= den;
    }
    /* log D = logsumexp(log d_s, log lambda_i + log d_lr, log eps); m = d_s / D
     * (m = 1 in the Sort_Lsh_RACE ablation) */
    for (int i = 0; i < N; ++i) {
        if (row_mask && !row_mask[i]) continue;
        const double lam = lambda_of(c, lam_rows, i);
        double t[3];
        int nt = 0;
        t[nt++] = st->lse[i];
        if (lam > 0 && st->Den[i] > 0) t[nt++] = log(lam) + log(st->Den[i]);
        t[nt++] = log(c->eps);
        double mx = t[0];
        for (int a = 1; a < nt; ++a) if (t[a] > mx) mx = t[a];
        double s = 0;
        for (int a = 0; a < nt; ++a) s += exp(t[a] - mx);
        st->logD[i] = mx + log(s);
        st->m[i] = c->m_one ? 1.0 : exp(st->lse[i] - st->logD[i]);
    }
    free(phq); free(phk);
    *rp_out = rp;
    *cols_out = cols;
    return ORA_OK;
fail:
    free(rp); free(cols); free(phq); free(phk);
    return rc;
}

static int alloc_state(fwd_state* st, int N, int d)
{
    st->Os = (double*)calloc((size_t)N * d, sizeof(double));
    st->Olr = (double*)calloc((size_t)N * d, sizeof(double));
    st->lse = (double*)calloc((size_t)N, sizeof(double));
    st->Den = (double*)calloc((size_t)N, sizeof(double));
    st->m = (double*)calloc((size_t)N, sizeof(double));
    st->logD = (double*)calloc((size_t)N, sizeof(double));
    return (st->Os && st->Olr && st->lse && st->Den && st->m && st->logD) ? ORA_OK : ORA_ENOMEM;
}

static void free_state(fwd_state* st)
{
    free(st->Os); free(st->Olr); free(st->lse); free(st->Den); free(st->m); free(st->logD);
}

/* Forward of one head.  Outputs (any may be NULL):
 *   O[N][d]   fused output g_s*m*O_s + g_lr*O_lr (Eq. elsaa_fusion_output)
 *   lse[N]    log d_sparse
 *   dlr[N]    d_lr = Den
 *   m[N]      denominator-aware multiplier
 *   Os[N][d], Olr[N][d]  branch outputs
 * lam_rows (optional): per-token lambda_i [N] (NULL: the scalar c->lambda).
 * row_mask (optional): only marked rows of O, lse, m, Os are computed
 * (Olr and dlr are always computed for every row). */
int ora_forward(const ora_cfg* c, const float* Q, const float* K, const float* V,
                const float* Wsort, const float* Wrace, const float* gates, const float* lam_rows,
                const uint8_t* row_mask, double* O, double* lse, double* dlr, double* m,
                double* Os, double* Olr)
{
    if (!cfg_ok(c) || !Q || !K || !V || !Wsort || !Wrace) return ORA_EINVAL;
    const int N = c->N, d = c->d;
    fwd_state st;
    int rc = alloc_state(&st, N, d);
    int64_t* rp = NULL;
    int32_t* cols = NULL;
    if (rc == ORA_OK) rc = forward_all(c, Q, K, V, Wsort, Wrace, lam_rows, row_mask, &st, &rp, &cols);
    if (rc == ORA_OK) {
        for (int i = 0; i < N; ++i) {
            const int on = !row_mask || row_mask[i];
            const double gs = gate_of(gates, i, 0), gl = gate_of(gates, i, 1);
            for (int e = 0; e < d; ++e) {
                const size_t ix = (size_t)i * d + e;
                if (O && on) O[ix] = gs * st.m[i] * st.Os[ix] + gl * st.Olr[ix];
                if (Os && on) Os[ix] = st.Os[ix];
                if (Olr) Olr[ix] = st.Olr[ix];
            }
            if (lse && on) lse[i] = st.lse[i];
            if (m && on) m[i] = st.m[i];
            if (dlr) dlr[i] = st.Den[i];
        }
    }
    free(rp); free(cols);
    free_state(&st);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Backward                                                                  */
/* ------------------------------------------------------------------------ */

/* Chain a feature gradient dphi[r] of row x back to dx[d] (accumulated):
 * phi_c = softmax_c(beta t.v_c), t = tanh(W_l x). */
static void feature_vjp(const ora_cfg* c, const float* x, const float* Wrace, const double* dphi,
                        double* dx, double* tb, double* ph)
{
    const int d = c->d, g = c->race_bits, R = 1 << g, L = c->r >> g;
    for (int l = 0; l < L; ++l) {
        for (int b = 0; b < g; ++b) {
            const float* w = Wrace + ((size_t)l * g + b) * d;
            double u = 0;
            for (int q = 0; q < d; ++q) u += (double)w[q] * (double)x[q];
            tb[b] = tanh(u);
        }
        double mx = -INFINITY;
        for (int cc = 0; cc < R; ++cc) {
            double s = 0;
            for (int b = 0; b < g; ++b) s += ((cc >> b) & 1) ? tb[b] : -tb[b];
            ph[cc] = c->beta * s;
            if (ph[cc] > mx) mx = ph[cc];
        }
        double den = 0;
        for (int cc = 0; cc < R; ++cc) { ph[cc] = exp(ph[cc] - mx); den += ph[cc]; }
        for (int cc = 0; cc < R; ++cc) ph[cc] /= den;
        const double* dp = dphi + (size_t)l * R;
        for (int b = 0; b < g; ++b) {
            /* d phi_c / d t_b = beta * phi_c * (v_cb - sum_c' phi_c' v_c'b) */
            double mean = 0;
            for (int cc = 0; cc < R; ++cc) mean += ph[cc] * (((cc >> b) & 1) ? 1.0 : -1.0);
            double dt = 0;
            for (int cc = 0; cc < R; ++cc)
                dt += dp[cc] * c->beta * ph[cc] * ((((cc >> b) & 1) ? 1.0 : -1.0) - mean);
            const double du = dt * (1.0 - tb[b] * tb[b]);
            const float* w = Wrace + ((size_t)l * g + b) * d;
            for (int q = 0; q < d; ++q) dx[q] += du * (double)w[q];
        }
    }
}

/* Backward of one head.  dO[N][d] is the upstream gradient of O.
 * Outputs dQ, dK, dV [N][d] (required), dgates [N][2] (optional:
 * d/dg_sparse, d/dg_lr) and dlambda [N] (optional: d/dlambda_i; the
 * gradient of a scalar lambda is their sum).  q_mask / k_mask (optional) restrict the sparse
 * part of dQ (rows) and of dK, dV (keys) to the marked indices; the
 * low-rank part is always computed for every row, so unmarked rows hold
 * only that part. */
int ora_backward(const ora_cfg* c, const float* Q, const float* K, const float* V,
                 const float* Wsort, const float* Wrace, const float* gates, const float* lam_rows,
                 const float* dO, const uint8_t* q_mask, const uint8_t* k_mask,
                 double* dQ, double* dK, double* dV, double* dgates, double* dlambda)
{
    if (!cfg_ok(c) || !Q || !K || !V || !Wsort || !Wrace || !dO || !dQ || !dK || !dV)
        return ORA_EINVAL;
    const int N = c->N, d = c->d, r = c->r, g = c->race_bits, R = 1 << g;
    const int L = r >> g;
    const double tau = tau_of(c), eps = c->eps;
    fwd_state st;
    int64_t *rp = NULL, *tp = NULL;
    int32_t *cols = NULL, *tcols = NULL;
    double *dOs = NULL, *Delta = NULL, *lse1 = NULL, *dNum = NULL, *dDen = NULL;
    double *phq = NULL, *phk = NULL, *dphq = NULL, *dphk = NULL;
    double *A = NULL, *Bm = NULL;
    int rc = alloc_state(&st, N, d);
    if (rc == ORA_OK) rc = forward_all(c, Q, K, V, Wsort, Wrace, lam_rows, NULL, &st, &rp, &cols);
    if (rc) goto out;
    memset(dQ, 0, sizeof(double) * (size_t)N * d);
    memset(dK, 0, sizeof(double) * (size_t)N * d);
    memset(dV, 0, sizeof(double) * (size_t)N * d);
    dOs = (double*)malloc(sizeof(double) * (size_t)N * d);
    dNum = (double*)malloc(sizeof(double) * (size_t)N * d);
    Delta = (double*)malloc(sizeof(double) * (size_t)N);
    lse1 = (double*)malloc(sizeof(double) * (size_t)N);
    dDen = (double*)malloc(sizeof(double) * (size_t)N);
    if (!dOs || !dNum || !Delta || !lse1 || !dDen) { rc = ORA_ENOMEM; goto out; }

    /* Row quantities: u = dO_i,
     *   dO_s = g_s m u;   dm = g_s <O_s, u>;   dO_lr = g_lr u
     *   Delta = <dO_s, O_s> - dm m (1-m) (d_s+eps)/d_s        (dm/dlog d_s = m(1-m))
     *   dNum = dO_lr / (Den+eps)
     *   dDen = -<dO_lr, O_lr>/(Den+eps) - dm m lambda / D      (dm/dDen = -m lambda/D)
     *   dlambda = -dm m Den / D                                 (dm/dlambda = -m Den/D)
     * With m fixed to 1 (Sort_Lsh_RACE) every dm term vanishes. */
    for (int i = 0; i < N; ++i) {
        const double gs = gate_of(gates, i, 0), gl = gate_of(gates, i, 1);
        const double mi = st.m[i];
        double uos = 0, uol = 0;
        for (int e = 0; e < d; ++e) {
            const double ue = dO[(size_t)i * d + e];
            uos += ue * st.Os[(size_t)i * d + e];
            uol += ue * st.Olr[(size_t)i * d + e];
        }
        const double dm = c->m_one ? 0.0 : gs * uos;
        const double lam = lambda_of(c, lam_rows, i);
        const double rel = eps * exp(-st.lse[i]);   /* eps / d_s */
        for (int e = 0; e < d; ++e) {
            const double ue = dO[(size_t)i * d + e];
            dOs[(size_t)i * d + e] = gs * mi * ue;
            dNum[(size_t)i * d + e] = gl * ue / (st.Den[i] + eps);
        }
        Delta[i] = gs * mi * uos - dm * mi * (1.0 - mi) * (1.0 + rel);
        lse1[i] = st.lse[i] + log1p(rel);   /* P_ij = exp(z_ij - log(d_s + eps)) */
        dDen[i] = -gl * uol / (st.Den[i] + eps) - dm * mi * lam / exp(st.logD[i]);
        if (dgates) {
            dgates[(size_t)i * 2 + 0] = mi * uos;
            dgates[(size_t)i * 2 + 1] = uol;
        }
        if (dlambda) dlambda[i] = -dm * mi * st.Den[i] / exp(st.logD[i]);
    }

    /* Sparse part: for j in S(i), P_ij = e^{z_ij}/(d_s+eps),
     *   dz_ij = P_ij (<dO_s,i, V_j> - Delta_i)
     *   dQ_i += tau dz_ij K_j;  dK_j += tau dz_ij Q_i;  dV_j += P_ij dO_s,i */
    #pragma omp parallel for schedule(dynamic, 16)
    for (int i = 0; i < N; ++i) {
        if (q_mask && !q_mask[i]) continue;
        const float* q = Q + (size_t)i * d;
        for (int64_t p = rp[i]; p < rp[i + 1]; ++p) {
            const int j = cols[p];
            const double P = exp(tau * dot(d, q, K + (size_t)j * d) - lse1[i]);
            double dv = 0;
            for (int e = 0; e < d; ++e) dv += dOs[(size_t)i * d + e] * V[(size_t)j * d + e];
            const double dz = P * (dv - Delta[i]);
            for (int e = 0; e < d; ++e) dQ[(size_t)i * d + e] += tau * dz * K[(size_t)j * d + e];
        }
    }
    {
        /* transpose of the support: for each key, the queries that see it */
        const int64_t total = rp[N];
        tp = (int64_t*)calloc((size_t)N + 1, sizeof(int64_t));
        tcols = (int32_t*)malloc(sizeof(int32_t) * (size_t)(total > 0 ? total : 1));
        int64_t* cur = (int64_t*)malloc(sizeof(int64_t) * (size_t)N);
        if (!tp || !tcols || !cur) { free(cur); rc = ORA_ENOMEM; goto out; }
        for (int64_t p = 0; p < total; ++p) tp[cols[p] + 1]++;
        for (int j = 0; j < N; ++j) tp[j + 1] += tp[j];
        for (int j = 0; j < N; ++j) cur[j] = tp[j];
        for (int i = 0; i < N; ++i)
            for (int64_t p = rp[i]; p < rp[i + 1]; ++p) tcols[cur[cols[p]]++] = i;
        free(cur);
    }
    #pragma omp parallel for schedule(dynamic, 16)
    for (int j = 0; j < N; ++j) {
        if (k_mask && !k_mask[j]) continue;
        const float* kv = K + (size_t)j * d;
        const float* vv = V + (size_t)j * d;
        for (int64_t p = tp[j]; p < tp[j + 1]; ++p) {
            const int i = tcols[p];
            const double P = exp(tau * dot(d, Q + (size_t)i * d, kv) - lse1[i]);
            double dv = 0;
            for (int e = 0; e < d; ++e) dv += dOs[(size_t)i * d + e] * vv[e];
            const double dz = P * (dv - Delta[i]);
            for (int e = 0; e < d; ++e) {
                dK[(size_t)j * d + e] += tau * dz * Q[(size_t)i * d + e];
                dV[(size_t)j * d + e] += P * dOs[(size_t)i * d + e];
            }
        }
    }

    /* Low-rank part (Alg. 2 / Alg. 3 differentiated):
     *   dphi(q_i) = (1/L) (B dNum_i + A dDen_i)      with the state seen by row i
     *   dB = (1/L) sum_i phi(q_i) dNum_i^T, dA = (1/L) sum_i phi(q_i) dDen_i
     *        over the rows that see key j (all rows, or i >= j when causal)
     *   dV_j += dB^T phi(k_j);  dphi(k_j) = dB V_j + dA */
    phq = (double*)malloc(sizeof(double) * (size_t)N * r);
    phk = (double*)malloc(sizeof(double) * (size_t)N * r);
    dphq = (double*)calloc((size_t)N * r, sizeof(double));
    dphk = (double*)calloc((size_t)N * r, sizeof(double));
    A = (double*)calloc((size_t)r, sizeof(double));
    Bm = (double*)calloc((size_t)r * d, sizeof(double));
    if (!phq || !phk || !dphq || !dphk || !A || !Bm) { rc = ORA_ENOMEM; goto out; }
    ora_features(N, d, Q, L, g, c->beta, Wrace, phq);
    ora_features(N, d, K, L, g, c->beta, Wrace, phk);
    if (!c->causal)
        for (int j = 0; j < N; ++j)
            for (int f = 0; f < r; ++f) {
                A[f] += phk[(size_t)j * r + f];
                for (int e = 0; e < d; ++e) Bm[(size_t)f * d + e] += phk[(size_t)j * r + f] * V[(size_t)j * d + e];
            }
    for (int i = 0; i < N; ++i) {
        if (c->causal)
            for (int f = 0; f < r; ++f) {
                A[f] += phk[(size_t)i * r + f];
                for (int e = 0; e < d; ++e) Bm[(size_t)f * d + e] += phk[(size_t)i * r + f] * V[(size_t)i * d + e];
            }
        for (int f = 0; f < r; ++f) {
            double s = A[f] * dDen[i];
            for (int e = 0; e < d; ++e) s += Bm[(size_t)f * d + e] * dNum[(size_t)i * d + e];
            dphq[(size_t)i * r + f] = s / L;
        }
    }
    memset(A, 0, sizeof(double) * (size_t)r);
    memset(Bm, 0, sizeof(double) * (size_t)r * d);
    if (!c->causal)
        for (int i = 0; i < N; ++i)
            for (int f = 0; f < r; ++f) {
                A[f] += phq[(size_t)i * r + f] * dDen[i] / L;
                for (int e = 0; e < d; ++e) Bm[(size_t)f * d + e] += phq[(size_t)i * r + f] * dNum[(size_t)i * d + e] / L;
            }
    for (int j = N - 1; j >= 0; --j) {
        if (c->causal)
            for (int f = 0; f < r; ++f) {
                A[f] += phq[(size_t)j * r + f] * dDen[j] / L;
                for (int e = 0; e < d; ++e) Bm[(size_t)f * d + e] += phq[(size_t)j * r + f] * dNum[(size_t)j * d + e] / L;
            }
        for (int f = 0; f < r; ++f) {
            const double ph = phk[(size_t)j * r + f];
            double s = A[f];
            for (int e = 0; e < d; ++e) {
                s += Bm[(size_t)f * d + e] * V[(size_t)j * d + e];
                dV[(size_t)j * d + e] += ph * Bm[(size_t)f * d + e];
            }
            dphk[(size_t)j * r + f] = s;
        }
    }
    #pragma omp parallel
    {
        double* tb = (double*)malloc(sizeof(double) * (size_t)g);
        double* ph = (double*)malloc(sizeof(double) * (size_t)R);
        #pragma omp for schedule(static)
        for (int i = 0; i < N; ++i) {
            feature_vjp(c, Q + (size_t)i * d, Wrace, dphq + (size_t)i * r, dQ + (size_t)i * d, tb, ph);
            feature_vjp(c, K + (size_t)i * d, Wrace, dphk + (size_t)i * r, dK + (size_t)i * d, tb, ph);
        }
        free(tb); free(ph);
    }
out:
    free_state(&st);
    free(rp); free(cols); free(tp); free(tcols);
    free(dOs); free(Delta); free(lse1); free(dNum); free(dDen);
    free(phq); free(phk); free(dphq); free(dphk); free(A); free(Bm);
    return rc;
}

/* Threads of the OpenMP loops above, for timing runs: n > 0 sets the count
 * used by later calls; returns the count now in effect.  No arithmetic. */
int ora_threads(int n)
{
    if (n > 0) omp_set_num_threads(n);
    return omp_get_max_threads();
}
