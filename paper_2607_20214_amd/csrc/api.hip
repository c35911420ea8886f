// api.hip -- host side of the C ABI (include/elsaa.h): argument validation,
// buffer layouts and the launch sequence of each entry point.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "elsaa.h"
#include "causal.hpp"
#include "fork_join.hpp"
#include "internal.hpp"

using namespace elsaa;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_fail(hipError_t e, const char* what)
{
    return fail(ELSAA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace

int elsaa::api_fail(int code, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int elsaa::api_hip_fail(hipError_t e, const char* what) { return hip_fail(e, what); }

namespace {

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int validate(const elsaa_config* c, Shape* s)
{
    if (!c) return fail(ELSAA_ERR_INVALID_ARG, "cfg is NULL");
    if (c->B < 1 || c->H < 1 || c->N < 1)
        return fail(ELSAA_ERR_INVALID_ARG, "B, H, N must be >= 1 (got %d, %d, %d)", c->B, c->H, c->N);
    if (c->d_h < 1) return fail(ELSAA_ERR_INVALID_ARG, "d_h must be >= 1 (got %d)", c->d_h);
    if (c->k < 1) return fail(ELSAA_ERR_INVALID_ARG, "k (sortLSH block size) must be >= 1 (got %d)", c->k);
    if (c->race_bits < 1 || c->race_bits > 12)
        return fail(ELSAA_ERR_INVALID_ARG, "race_bits must be in [1, 12] (got %d)", c->race_bits);
    if (c->r < (1 << c->race_bits) || c->r % (1 << c->race_bits))
        return fail(ELSAA_ERR_INVALID_ARG, "r must be a positive multiple of 2^race_bits (got r=%d)", c->r);
    if (c->sort_bits < 1 || c->sort_bits > 8)
        return fail(ELSAA_ERR_INVALID_ARG, "sort_bits must be in [1, 8] (got %d)", c->sort_bits);
    if (c->causal != 0 && c->causal != 1) return fail(ELSAA_ERR_INVALID_ARG, "causal must be 0 or 1");
    if (c->dtype != ELSAA_F32 && c->dtype != ELSAA_BF16) return fail(ELSAA_ERR_INVALID_ARG, "unknown dtype %d", c->dtype);
    if (!(c->beta > 0) || !std::isfinite(c->beta)) return fail(ELSAA_ERR_INVALID_ARG, "beta must be finite and > 0");
    if (!(c->lambda >= 0) || !std::isfinite(c->lambda)) return fail(ELSAA_ERR_INVALID_ARG, "lambda must be finite and >= 0");
    if (!(c->eps > 0) || !std::isfinite(c->eps)) return fail(ELSAA_ERR_INVALID_ARG, "eps must be finite and > 0");
    if (!std::isfinite(c->scale)) return fail(ELSAA_ERR_INVALID_ARG, "scale must be finite");
    if (c->neighbors < 0) return fail(ELSAA_ERR_INVALID_ARG, "neighbors must be >= 0 (got %d)", c->neighbors);
    if (c->m_one != 0 && c->m_one != 1) return fail(ELSAA_ERR_INVALID_ARG, "m_one must be 0 or 1");
    // GPU path limits
    if (c->d_h != 64 && c->d_h != 128) return fail(ELSAA_ERR_UNSUPPORTED, "d_h must be 64 or 128 (got %d)", c->d_h);
    if (c->race_bits != 4) return fail(ELSAA_ERR_UNSUPPORTED, "the GPU path implements race_bits = 4 only (got %d)", c->race_bits);
    if (c->r > 256) return fail(ELSAA_ERR_UNSUPPORTED, "r must be <= 256 (got %d)", c->r);
    if ((int64_t)c->N > (1 << 26)) return fail(ELSAA_ERR_UNSUPPORTED, "N must be <= 2^26");
    const int bf16 = c->dtype == ELSAA_BF16;
    // the sparse kernels address a head's rows with 32-bit byte offsets
    if ((int64_t)c->N * c->d_h * (bf16 ? 2 : 4) >= ((int64_t)1 << 32))
        return fail(ELSAA_ERR_UNSUPPORTED, "N * d_h * element bytes must be < 2^32 (one head's rows)");
    const int n0 = c->n0 > 0 ? c->n0 : 2 * c->k;
    int lv = 0, n_leaf = c->N;
    s->lt = LevelTiles{};
    if (c->causal) {
        // the recursion of Alg. 5 with its zero-token padding of odd lists
        if (!level_tiles(c->N, n0, s->lt))
            return fail(ELSAA_ERR_UNSUPPORTED,
                        "causal N = %d with n0 = %d: more than %d levels, or a past half that would hold "
                        "a zero token",
                        c->N, n0, kMaxLevels);
        lv = s->lt.Lv;
        n_leaf = s->lt.len[lv];
    }
    s->B = c->B; s->H = c->H; s->N = c->N; s->D = c->d_h;
    s->k = c->k;
    s->r = c->r; s->L = c->r >> c->race_bits;
    s->Lp = race_padded_features(c->r) / 16;
    s->sort_bits = c->sort_bits;
    s->Lv = lv; s->n_leaf = n_leaf;
    s->causal = c->causal; s->bf16 = bf16;
    s->beta = c->beta; s->lambda = c->lambda; s->eps = c->eps;
    s->tau = c->scale > 0 ? c->scale : 1.0f / std::sqrt((float)c->d_h);
    s->neighbors = c->neighbors;
    s->m_one = c->m_one;
    // RACE segments: enough workgroups to fill the chip, whole 64-token chunks
    const int64_t chunks = (c->N + 63) / 64;
    const int64_t bh = (int64_t)c->B * c->H;
    int64_t nseg = (512 + bh - 1) / bh;     // about two segment workgroups per compute unit
    if (nseg > chunks) nseg = chunks;
    if (nseg < 1) nseg = 1;
    const int64_t per = (chunks + nseg - 1) / nseg;
    s->seg_len = (int)(per * 64);
    s->nseg = (int)((c->N + s->seg_len - 1) / s->seg_len);
    if (!race_fwd_fits(*s) || !race_bwd_fits(*s))
        return fail(ELSAA_ERR_UNSUPPORTED, "r = %d with d_h = %d in %s exceeds the RACE kernels' LDS", c->r,
                    c->d_h, bf16 ? "bf16" : "float32");
    return ELSAA_OK;
}

struct SavedLayout {
    size_t perm_q, perm_k, m, o_s, o_lr, u_q, u_k, race_states, total;
};

SavedLayout saved_layout(const Shape& s)
{
    SavedLayout L;
    const size_t bh = (size_t)s.B * s.H;
    size_t off = 0;
    L.perm_q = off; off = align256(off + bh * s.P() * 4);
    L.perm_k = off; off = align256(off + bh * s.P() * 4);
    L.m = off; off = align256(off + bh * s.N * 4);
    L.o_s = off; off = align256(off + bh * s.N * s.D * 4);   // float32: Delta = <dO, O_s> cancels against dP
                                                              // of the dominant keys when attention is peaked
    L.o_lr = off; off = align256(off + bh * s.N * s.D * (s.bf16 ? 2 : 4));   // storage dtype (diffuse weights)
    L.u_q = off; off = align256(off + bh * s.N * race_proj_stride(s) * 4);
    L.u_k = off; off = align256(off + bh * s.N * race_proj_stride(s) * 4);
    L.race_states = off; off = align256(off + race_state_floats(s) * 4);   // RACE segment prefix states
    L.total = off;
    return L;
}

struct FwdWorkspace {
    size_t keyq, keyk, part_o, part_lse, total;
};

FwdWorkspace fwd_workspace(const Shape& s)
{
    FwdWorkspace W;
    const size_t bh = (size_t)s.B * s.H;
    size_t off = 0;
    W.keyq = off; off = align256(off + bh * s.N);
    W.keyk = off; off = align256(off + bh * s.N);
    const size_t npart = s.causal ? bh * (size_t)s.P() : 0;   // one entry per level list entry
    W.part_o = off; off = align256(off + npart * s.D * (s.bf16 ? 2 : 4));   // storage dtype
    W.part_lse = off; off = align256(off + npart * 4);
    W.total = off;
    return W;
}

struct BwdWorkspace {
    size_t rs, states_b, wt_hi, wt_lo, du_q, du_k, dv_lr, part_dq, part_dk, part_dv, total;
};

BwdWorkspace bwd_workspace(const Shape& s)
{
    BwdWorkspace W;
    const size_t bh = (size_t)s.B * s.H;
    const size_t bhn = bh * s.N;
    const size_t npart = s.causal ? bh * (size_t)s.P() : 0;
    size_t off = 0;
    W.rs = off; off = align256(off + 5 * bhn * 4);
    W.states_b = off; off = align256(off + race_state_floats(s) * 4);
    W.wt_hi = off; off = align256(off + race_wt_bytes(s));
    W.wt_lo = off; off = align256(off + race_wt_bytes(s));
    W.du_q = off; off = align256(off + bhn * race_wk(s) * (s.bf16 ? 2 : 4));
    W.du_k = off; off = align256(off + bhn * race_wk(s) * (s.bf16 ? 2 : 4));
    W.dv_lr = off; off = align256(off + bhn * s.D * (s.bf16 ? 2 : 4));   // storage dtype
    W.part_dq = off; off = align256(off + npart * s.D * (s.bf16 ? 2 : 4));   // storage dtype
    W.part_dk = off; off = align256(off + npart * s.D * (s.bf16 ? 2 : 4));
    W.part_dv = off; off = align256(off + npart * s.D * (s.bf16 ? 2 : 4));
    W.total = off;
    return W;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

template <class P>
P* at(void* base, size_t off) { return (P*)((char*)base + off); }

// A second stream per device for work that shares no buffer with what the
// caller's stream runs meanwhile (the forward's sort beside the low-rank
// branch).  Fork: an event on the caller's stream that
// the side stream waits for; join: the reverse.  Host-side enqueueing of a
// fork / join pair holds a per-device lock, so that concurrent calls cannot
// interleave their event records.  Default priority, created on first use
// and kept until the process ends; without it both parts run on the
// caller's stream.
struct Side {
    std::mutex mu;
    bool init = false;
    bool ok = false;
    hipStream_t stream = nullptr;
    hipEvent_t fork = nullptr, join = nullptr;
};
constexpr int kMaxDevices = 64;
Side g_side[kMaxDevices];

Side* side_stream()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    Side& sd = g_side[dev];
    std::lock_guard<std::mutex> lk(sd.mu);
    if (!sd.init) {
        sd.init = true;
        sd.ok = hipStreamCreateWithFlags(&sd.stream, hipStreamNonBlocking) == hipSuccess &&
                hipEventCreateWithFlags(&sd.fork, hipEventDisableTiming) == hipSuccess &&
                hipEventCreateWithFlags(&sd.join, hipEventDisableTiming) == hipSuccess;
    }
    return sd.ok ? &sd : nullptr;
}

hipError_t record_event(hipEvent_t e, hipStream_t s) { return hipEventRecord(e, s); }
hipError_t clear_error() { return hipGetLastError(); }
const StreamOps kHipStreamOps = {record_event, hipStreamWaitEvent, hipStreamSynchronize, clear_error};

// first(side) on the device's side stream beside second(main) (fork_join.hpp);
// without a side stream both run on `main` in order.
template <class A, class B>
hipError_t fork_join(hipStream_t main, A first, B second)
{
    Side* sd = side_stream();
    if (!sd) {
        hipError_t e = first(main);
        return e != hipSuccess ? e : second(main);
    }
    std::lock_guard<std::mutex> lk(sd->mu);
    return elsaa::fork_join(kHipStreamOps, main, sd->stream, sd->fork, sd->join, first, second);
}

// Fixed device scratch of the entry point that allocates nothing
// (elsaa_select_noalloc): the hash keys of the Q and K rows.  In host code
// `scratch` names a host-side stand-in, not the device array, so only the
// per-device address from hipGetSymbolAddress is ever handed to a kernel.
constexpr size_t kNoallocScratchBytes = (size_t)32 << 20;
__device__ __attribute__((aligned(256))) uint8_t scratch[kNoallocScratchBytes];

struct ScratchAddr {
    std::once_flag once;
    void* ptr = nullptr;
    hipError_t err = hipSuccess;
};
ScratchAddr g_scratch[kMaxDevices];

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
hipError_t scratch_address(void** out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    ScratchAddr& sa = g_scratch[dev];
    std::call_once(sa.once, [&sa]() {
        void* p = nullptr;
        sa.err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (sa.err == hipSuccess) sa.ptr = p;
    });
    if (sa.err != hipSuccess) return sa.err;
    if (!sa.ptr) return hipErrorInvalidSymbol;
    *out = sa.ptr;
    return hipSuccess;
}

int check_rules(const elsaa_token_rules* r, TrParams* p)
{
    if (!r) return fail(ELSAA_ERR_INVALID_ARG, "rules is NULL");
    if (r->gate_hidden != 0 && r->gate_hidden != 64 && r->gate_hidden != 128)
        return fail(ELSAA_ERR_UNSUPPORTED, "gate_hidden must be 0, 64 or 128 (got %d)", r->gate_hidden);
    if (r->lambda_rule != 0 && r->lambda_rule != 1) return fail(ELSAA_ERR_INVALID_ARG, "lambda_rule must be 0 or 1");
    if (r->gate_hidden == 0 && r->lambda_rule == 0) return fail(ELSAA_ERR_INVALID_ARG, "no rule is on");
    if (r->gate_hidden && (!r->W1 || !r->b1 || !r->W2 || !r->b2))
        return fail(ELSAA_ERR_INVALID_ARG, "gate network parameters must not be NULL");
    if (r->lambda_rule && (!r->lam_w || !r->lam_b || !r->lam_c))
        return fail(ELSAA_ERR_INVALID_ARG, "lambda rule parameters must not be NULL");
    if ((r->gate_hidden && !aligned16(r->W1)) || (r->lambda_rule && !aligned16(r->lam_w)))
        return fail(ELSAA_ERR_INVALID_ARG, "W1 and lam_w must be 16-byte aligned");
    if (r->lambda_rule && (!(r->lambda_min >= 0) || !std::isfinite(r->lambda_min)))
        return fail(ELSAA_ERR_INVALID_ARG, "lambda_min must be finite and >= 0");
    p->G = r->gate_hidden;
    p->lam = r->lambda_rule;
    p->W1 = r->W1; p->b1 = r->b1; p->W2 = r->W2; p->b2 = r->b2;
    p->lw = r->lam_w; p->lb = r->lam_b; p->lc = r->lam_c;
    p->lam_min = r->lambda_min;
    return ELSAA_OK;
}

}  // namespace

extern "C" {

int elsaa_num_levels(const elsaa_config* cfg)
{
    Shape s;
    int rc = validate(cfg, &s);
    if (rc) return rc;
    return s.Lv;
}

int64_t elsaa_perm_length(const elsaa_config* cfg)
{
    Shape s;
    int rc = validate(cfg, &s);
    if (rc) return rc;
    return s.P();
}

int elsaa_saved_bytes(const elsaa_config* cfg, size_t* bytes)
{
    Shape s;
    int rc = validate(cfg, &s);
    if (rc) return rc;
    if (!bytes) return fail(ELSAA_ERR_INVALID_ARG, "bytes is NULL");
    *bytes = saved_layout(s).total;
    return ELSAA_OK;
}

int elsaa_workspace_bytes(const elsaa_config* cfg, int pass, size_t* bytes)
{
    Shape s;
    int rc = validate(cfg, &s);
    if (rc) return rc;
    if (!bytes) return fail(ELSAA_ERR_INVALID_ARG, "bytes is NULL");
    if (pass == 0) *bytes = fwd_workspace(s).total;
    else if (pass == 1) *bytes = bwd_workspace(s).total;
    else return fail(ELSAA_ERR_INVALID_ARG, "pass must be 0 (forward) or 1 (backward)");
    return ELSAA_OK;
}

int elsaa_get_saved_layout(const elsaa_config* cfg, elsaa_saved_layout* out)
{
    Shape s;
    int rc = validate(cfg, &s);
    if (rc) return rc;
    if (!out) return fail(ELSAA_ERR_INVALID_ARG, "out is NULL");
    SavedLayout L = saved_layout(s);
    out->perm_q = L.perm_q;
    out->perm_k = L.perm_k;
    out->m = L.m;
    out->o_sparse = L.o_s;
    out->o_lowrank = L.o_lr;
    out->u_q = L.u_q;
    out->u_k = L.u_k;
    out->race_states = L.race_states;
    out->total = L.total;
    return ELSAA_OK;
}

int elsaa_select(const elsaa_config* cfg, const void* Q, const void* K, const float* W_sort,
                 int32_t* perm_q, int32_t* perm_k, void* workspace, size_t workspace_bytes,
                 hipStream_t stream)
{
    Shape s;
    int rc = validate(cfg, &s);
    if (rc) return rc;
    if (!Q || !K || !W_sort || !perm_q || !perm_k || !workspace)
        return fail(ELSAA_ERR_INVALID_ARG, "a required pointer is NULL");
    if (!aligned16(Q) || !aligned16(K) || !aligned16(workspace))
        return fail(ELSAA_ERR_INVALID_ARG, "Q, K and workspace must be 16-byte aligned");
    FwdWorkspace W = fwd_workspace(s);
    if (workspace_bytes < W.keyk + (size_t)s.B * s.H * s.N)
        return fail(ELSAA_ERR_WORKSPACE, "workspace too small");
    uint8_t* kq = at<uint8_t>(workspace, W.keyq);
    uint8_t* kk = at<uint8_t>(workspace, W.keyk);
    hipError_t e;
    if ((e = launch_project(s, Q, K, W_sort, nullptr, kq, kk, nullptr, nullptr, stream)) != hipSuccess)
        return hip_fail(e, "hash");
    if ((e = launch_sort(s, kq, kk, perm_q, perm_k, stream)) != hipSuccess) return hip_fail(e, "sort");
    return ELSAA_OK;
}

int elsaa_select_noalloc(const elsaa_config* cfg, const void* Q, const void* K, const float* W_sort,
                         int32_t* perm_q, int32_t* perm_k, hipStream_t stream)
{
    Shape s;
    int rc = validate(cfg, &s);
    if (rc) return rc;
    if (!Q || !K || !W_sort || !perm_q || !perm_k) return fail(ELSAA_ERR_INVALID_ARG, "a required pointer is NULL");
    if (!aligned16(Q) || !aligned16(K)) return fail(ELSAA_ERR_INVALID_ARG, "Q and K must be 16-byte aligned");
    const size_t bhn = (size_t)s.B * s.H * s.N;
    const size_t keyk = align256(bhn);
    if (keyk + bhn > kNoallocScratchBytes)
        return fail(ELSAA_ERR_WORKSPACE, "B*H*N = %zu tokens need %zu bytes of scratch; the fixed scratch holds %zu",
                    bhn, keyk + bhn, kNoallocScratchBytes);
    void* base = nullptr;
    hipError_t e;
    if ((e = scratch_address(&base)) != hipSuccess) return hip_fail(e, "scratch address");
    uint8_t* kq = (uint8_t*)base;
    uint8_t* kk = (uint8_t*)base + keyk;
    // every key the sort reads is written by the hash pass first: nothing to clear
    if ((e = launch_project(s, Q, K, W_sort, nullptr, kq, kk, nullptr, nullptr, stream)) != hipSuccess)
        return hip_fail(e, "hash");
    if ((e = launch_sort(s, kq, kk, perm_q, perm_k, stream)) != hipSuccess) return hip_fail(e, "sort");
    return ELSAA_OK;
}

int elsaa_fwd(const elsaa_config* cfg, const void* Q, const void* K, const void* V,
              const float* W_sort, const float* W_race, const float* gates, const float* lambda_rows,
              void* O, float* lse, float* d_lr, void* saved, size_t saved_bytes,
              void* workspace, size_t workspace_bytes, hipStream_t stream)
{
    Shape s;
    int rc = validate(cfg, &s);
    if (rc) return rc;
    if (!Q || !K || !V || !W_sort || !W_race || !O || !lse || !d_lr || !saved || !workspace)
        return fail(ELSAA_ERR_INVALID_ARG, "a required pointer is NULL");
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O) || !aligned16(saved) ||
        !aligned16(workspace))
        return fail(ELSAA_ERR_INVALID_ARG, "Q, K, V, O, saved and workspace must be 16-byte aligned");
    SavedLayout SL = saved_layout(s);
    FwdWorkspace W = fwd_workspace(s);
    if (saved_bytes < SL.total)
        return fail(ELSAA_ERR_WORKSPACE, "saved buffer too small (%zu < %zu bytes)", saved_bytes, SL.total);
    if (workspace_bytes < W.total)
        return fail(ELSAA_ERR_WORKSPACE, "workspace too small (%zu < %zu bytes)", workspace_bytes, W.total);
    uint8_t* kq = at<uint8_t>(workspace, W.keyq);
    uint8_t* kk = at<uint8_t>(workspace, W.keyk);
    int32_t* pq = at<int32_t>(saved, SL.perm_q);
    int32_t* pk = at<int32_t>(saved, SL.perm_k);
    float* m = at<float>(saved, SL.m);
    float* o_s = at<float>(saved, SL.o_s);
    void* o_lr = at<char>(saved, SL.o_lr);
    float* uq = at<float>(saved, SL.u_q);
    float* uk = at<float>(saved, SL.u_k);
    hipError_t e;
    if ((e = launch_project(s, Q, K, W_sort, W_race, kq, kk, uq, uk, stream)) != hipSuccess)
        return hip_fail(e, "project");
    void* part_o = at<char>(workspace, W.part_o);
    float* part_lse = at<float>(workspace, W.part_lse);
    // the sort on the side stream beside the low-rank branch (its kernels and
    // the level kernel's cannot share a compute unit, so the levels run after
    // it rather than competing for the device), then the causal levels, then
    // the leaf (or sorted blocks) with the fusion epilogue
    e = fork_join(
        stream, [&](hipStream_t st) { return launch_sort(s, kq, kk, pq, pk, st); },
        [&](hipStream_t st) { return launch_race_fwd(s, uq, uk, V, at<float>(saved, SL.race_states), o_lr, d_lr, st); });
    if (e == hipSuccess)
        e = launch_sparse_fwd(s, Q, K, V, pq, pk, gates, lambda_rows, o_lr, d_lr, part_o, part_lse, O, lse, m, o_s,
                              stream, kSparseLevels);
    if (e != hipSuccess) return hip_fail(e, "selection / levels / race forward");
    if ((e = launch_sparse_fwd(s, Q, K, V, pq, pk, gates, lambda_rows, o_lr, d_lr, part_o, part_lse, O, lse, m,
                               o_s, stream, kSparseFinal)) != hipSuccess)
        return hip_fail(e, "sparse forward");
    return ELSAA_OK;
}

int elsaa_bwd(const elsaa_config* cfg, const void* Q, const void* K, const void* V,
              const float* W_sort, const float* W_race, const float* gates, const float* lambda_rows,
              const void* dO, const float* lse, const float* d_lr, const void* saved, size_t saved_bytes,
              void* dQ, void* dK, void* dV, float* dgates, float* dlambda,
              void* workspace, size_t workspace_bytes, hipStream_t stream)
{
    Shape s;
    int rc = validate(cfg, &s);
    if (rc) return rc;
    (void)W_sort;   // the selection is read from saved
    if (!Q || !K || !V || !W_race || !dO || !lse || !d_lr || !saved || !dQ || !dK || !dV || !workspace)
        return fail(ELSAA_ERR_INVALID_ARG, "a required pointer is NULL");
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(dO) || !aligned16(saved) ||
        !aligned16(dQ) || !aligned16(dK) || !aligned16(dV) || !aligned16(workspace))
        return fail(ELSAA_ERR_INVALID_ARG, "Q, K, V, dO, dQ, dK, dV, saved and workspace must be 16-byte aligned");
    SavedLayout SL = saved_layout(s);
    BwdWorkspace W = bwd_workspace(s);
    if (saved_bytes < SL.total)
        return fail(ELSAA_ERR_WORKSPACE, "saved buffer too small (%zu < %zu bytes)", saved_bytes, SL.total);
    if (workspace_bytes < W.total)
        return fail(ELSAA_ERR_WORKSPACE, "workspace too small (%zu < %zu bytes)", workspace_bytes, W.total);
    void* sv = const_cast<void*>(saved);
    const int32_t* pq = at<int32_t>(sv, SL.perm_q);
    const int32_t* pk = at<int32_t>(sv, SL.perm_k);
    const float* m = at<float>(sv, SL.m);
    const float* o_s = at<float>(sv, SL.o_s);
    const void* o_lr = at<char>(sv, SL.o_lr);
    const float* uq = at<float>(sv, SL.u_q);
    const float* uk = at<float>(sv, SL.u_k);
    float* rs = at<float>(workspace, W.rs);
    void* du_q = at<char>(workspace, W.du_q);
    void* du_k = at<char>(workspace, W.du_k);
    void* wt_hi = at<char>(workspace, W.wt_hi);
    void* wt_lo = at<char>(workspace, W.wt_lo);
    void* dv_lr = at<uint8_t>(workspace, W.dv_lr);
    hipError_t e;
    if ((e = launch_bwd_rows(s, dO, o_s, o_lr, m, lse, d_lr, gates, lambda_rows, rs, dgates, dlambda, stream)) !=
        hipSuccess)
        return hip_fail(e, "backward row scalars");
    void* part_dq = at<char>(workspace, W.part_dq);
    void* part_dk = at<char>(workspace, W.part_dk);
    void* part_dv = at<char>(workspace, W.part_dv);
    // the causal levels' backward, then the low-rank backward, then the leaf
    // (or sorted blocks), which add the level partials and low-rank
    // gradients (one kernel at a time: each kernel's time is its own)
    auto levels = [&](hipStream_t st) {
        return launch_sparse_bwd(s, Q, K, V, dO, pq, pk, rs, du_q, du_k, wt_hi, wt_lo, dv_lr, part_dq, part_dk,
                                 part_dv, dQ, dK, dV, st, kSparseLevels);
    };
    auto race = [&](hipStream_t st) {
        return launch_race_bwd(s, uq, uk, V, dO, W_race, rs, at<float>(sv, SL.race_states),
                               at<float>(workspace, W.states_b), wt_hi, wt_lo, du_q, du_k, dv_lr, st);
    };
    if ((e = levels(stream)) != hipSuccess) return hip_fail(e, "sparse levels backward");
    if ((e = race(stream)) != hipSuccess) return hip_fail(e, "race backward");
    if ((e = launch_sparse_bwd(s, Q, K, V, dO, pq, pk, rs, du_q, du_k, wt_hi, wt_lo, dv_lr, part_dq, part_dk,
                               part_dv, dQ, dK, dV, stream, kSparseFinal)) != hipSuccess)
        return hip_fail(e, "sparse backward");
    return ELSAA_OK;
}

int elsaa_token_rules_fwd(const elsaa_config* cfg, const elsaa_token_rules* rules, const void* Q,
                          float* gates, float* lambda_rows, hipStream_t stream)
{
    Shape s;
    int rc = validate(cfg, &s);
    if (rc) return rc;
    TrParams p;
    if ((rc = check_rules(rules, &p))) return rc;
    if (!Q) return fail(ELSAA_ERR_INVALID_ARG, "Q is NULL");
    if (!aligned16(Q)) return fail(ELSAA_ERR_INVALID_ARG, "Q must be 16-byte aligned");
    if (p.G && !gates) return fail(ELSAA_ERR_INVALID_ARG, "gates is NULL");
    if (p.lam && !lambda_rows) return fail(ELSAA_ERR_INVALID_ARG, "lambda_rows is NULL");
    if (p.G && ((uintptr_t)gates & 7)) return fail(ELSAA_ERR_INVALID_ARG, "gates must be 8-byte aligned");
    hipError_t e = launch_token_rules_fwd(s, p, Q, p.G ? gates : nullptr, p.lam ? lambda_rows : nullptr, stream);
    if (e != hipSuccess) return hip_fail(e, "token rules forward");
    return ELSAA_OK;
}

int elsaa_token_rules_workspace_bytes(const elsaa_config* cfg, const elsaa_token_rules* rules, size_t* bytes)
{
    Shape s;
    int rc = validate(cfg, &s);
    if (rc) return rc;
    TrParams p;
    if ((rc = check_rules(rules, &p))) return rc;
    if (!bytes) return fail(ELSAA_ERR_INVALID_ARG, "bytes is NULL");
    *bytes = token_rules_workspace_bytes(s, p.G, p.lam != 0);
    return ELSAA_OK;
}

int elsaa_token_rules_bwd(const elsaa_config* cfg, const elsaa_token_rules* rules, const void* Q,
                          const float* dgates, const float* dlambda, void* dQ,
                          float* dW1, float* db1, float* dW2, float* db2,
                          float* dlam_w, float* dlam_b, float* dlam_c,
                          void* workspace, size_t workspace_bytes, hipStream_t stream)
{
    Shape s;
    int rc = validate(cfg, &s);
    if (rc) return rc;
    TrParams p;
    if ((rc = check_rules(rules, &p))) return rc;
    if (!Q || !workspace) return fail(ELSAA_ERR_INVALID_ARG, "Q and workspace must not be NULL");
    if (!aligned16(Q) || !aligned16(workspace) || (dQ && !aligned16(dQ)))
        return fail(ELSAA_ERR_INVALID_ARG, "Q, dQ and workspace must be 16-byte aligned");
    if (p.G && !dgates) return fail(ELSAA_ERR_INVALID_ARG, "dgates is NULL");
    if (p.G && ((uintptr_t)dgates & 7)) return fail(ELSAA_ERR_INVALID_ARG, "dgates must be 8-byte aligned");
    if (p.lam && !dlambda) return fail(ELSAA_ERR_INVALID_ARG, "dlambda is NULL");
    if (workspace_bytes < token_rules_workspace_bytes(s, p.G, p.lam != 0))
        return fail(ELSAA_ERR_WORKSPACE, "workspace too small (elsaa_token_rules_workspace_bytes)");
    TrGrads g = {dW1, db1, dW2, db2, dlam_w, dlam_b, dlam_c};
    if (!p.G) g.dW1 = g.db1 = g.dW2 = g.db2 = nullptr;
    if (!p.lam) g.dlw = g.dlb = g.dlc = nullptr;
    hipError_t e = launch_token_rules_bwd(s, p, Q, p.G ? dgates : nullptr, p.lam ? dlambda : nullptr,
                                          p.G ? dQ : nullptr, g, (float*)workspace, stream);
    if (e != hipSuccess) return hip_fail(e, "token rules backward");
    return ELSAA_OK;
}

const char* elsaa_status_string(int status)
{
    switch (status) {
        case ELSAA_OK: return "ok";
        case ELSAA_ERR_INVALID_ARG: return "invalid argument";
        case ELSAA_ERR_UNSUPPORTED: return "unsupported on the GPU path";
        case ELSAA_ERR_WORKSPACE: return "buffer too small";
        case ELSAA_ERR_HIP: return "HIP error";
        default: return "unknown status";
    }
}

const char* elsaa_last_error(void) { return g_err.c_str(); }

}  // extern "C"
