// bwd_rows.hip -- per-row scalars of the backward.
//
// For u = dO_i, with O = g_s m O_s + g_lr O_lr, m = d_s / D, D = d_s + lambda Den + eps,
// O_s = N_s / (d_s + eps), O_lr = Num / (Den + eps):
//   dm    = g_s <O_s, u>                      (dm / d log d_s = m (1 - m))
//   sc_s  = g_s m                             (dO_s = sc_s u)
//   Delta = sc_s <u, O_s> - dm m (1 - m)(d_s + eps) / d_s
//   sc_lr = g_lr / (Den + eps)                (dNum = sc_lr u)
//   dDen  = -g_lr <u, O_lr> / (Den + eps) - dm m lambda / D
//   dg_s  = m <O_s, u>,  dg_lr = <O_lr, u>,  dlambda = -dm m Den / D
// (lambda per token when given; with m fixed to 1 every dm term is zero).
// Stored as rs[f][BHN] with f = 0: log2(d_s + eps), 1: Delta, 2: sc_s,
// 3: sc_lr, 4: dDen.  16 lanes per row; O_s float32, O_lr in the storage dtype.
#include "common.hpp"
#include "internal.hpp"

namespace elsaa {

namespace {

template <class T, int D>
__global__ __launch_bounds__(256) void bwd_rows_kernel(const typename T::store_t* __restrict__ dO,
                                                       const float* __restrict__ Os,
                                                       const typename T::store_t* __restrict__ Olr,
                                                       const float* __restrict__ m,
                                                       const float* __restrict__ lse,
                                                       const float* __restrict__ dlr,
                                                       const float* __restrict__ gates,
                                                       const float* __restrict__ lam_rows,
                                                       float* __restrict__ rs, float* __restrict__ dg,
                                                       float* __restrict__ dlam, size_t BHN, float lambda,
                                                       float eps, int m_one)
{
    constexpr int PL = D / 16;   // elements per lane
    const size_t row = (size_t)blockIdx.x * 16 + threadIdx.x / 16;
    const int sub = threadIdx.x & 15;
    if (row >= BHN) return;   // whole 16-lane groups leave together
    float uos = 0.f, uol = 0.f;
    const size_t base = row * D + sub * PL;
#pragma unroll
    for (int e = 0; e < PL; e += 4) {
        const f32x4 u = load4<T>(dO + base + e), xs = *(const f32x4*)(Os + base + e), xl = load4<T>(Olr + base + e);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            uos += u[i] * xs[i];
            uol += u[i] * xl[i];
        }
    }
    uos = row_sum16(uos);
    uol = row_sum16(uol);
    if (sub != 0) return;
    const float gs = gates ? gates[row * 2] : 1.f;
    const float gl = gates ? gates[row * 2 + 1] : 1.f;
    const float mi = m[row], ls = lse[row], den = dlr[row];
    const float rel = eps * __expf(fminf(-ls, 80.f));   // eps / d_s
    const float dm = m_one ? 0.f : gs * uos;
    const float lam = lam_rows ? lam_rows[row] : lambda;
    const float scs = gs * mi;
    const float delta = scs * uos - dm * mi * (1.f - mi) * (1.f + rel);
    const float inv_den = 1.f / (den + eps);
    const float Dtot = __expf(fminf(ls, 80.f)) + lam * den + eps;
    const float dden = -gl * uol * inv_den - dm * mi * lam / Dtot;
    rs[row] = (ls + log1pf(rel)) * kLog2e;
    rs[BHN + row] = delta;
    rs[2 * BHN + row] = scs;
    rs[3 * BHN + row] = gl * inv_den;
    rs[4 * BHN + row] = dden;
    if (dg) {
        dg[row * 2] = mi * uos;
        dg[row * 2 + 1] = uol;
    }
    if (dlam) dlam[row] = -dm * mi * den / Dtot;
}

}  // namespace

hipError_t launch_bwd_rows(const Shape& s, const void* dO, const float* Os, const void* Olr,
                           const float* m, const float* lse, const float* dlr, const float* gates,
                           const float* lambda_rows, float* rs, float* dgates, float* dlambda,
                           hipStream_t st)
{
    const size_t BHN = (size_t)s.B * s.H * s.N;
    dim3 grid((unsigned)((BHN + 15) / 16));
#define ELSAA_ROWS(T_, D_)                                                                       \
    ELSAA_LAUNCH("bwd_rows", (bwd_rows_kernel<T_, D_>), grid, dim3(256), 0, st,                          \
                       (const T_::store_t*)dO, Os, (const T_::store_t*)Olr, m, \
                       lse, dlr, gates, lambda_rows, rs, dgates, dlambda, BHN, s.lambda, s.eps, s.m_one)
    if (s.bf16) {
        if (s.D == 64) ELSAA_ROWS(BF16, 64);
        else ELSAA_ROWS(BF16, 128);
    } else {
        if (s.D == 64) ELSAA_ROWS(F32, 64);
        else ELSAA_ROWS(F32, 128);
    }
#undef ELSAA_ROWS
    return hipGetLastError();
}

}  // namespace elsaa
