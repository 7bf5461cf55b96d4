// TVB: integer per-layer budgets of each sequence (Sec. 3.2 Eq. (5), Sec. 3.3 Eq. (6)).
//
// Layer l's share of the sequence budget is m_l / sum_l' m_l', with m_l the summed
// text->vision attention.  The paper states the share as a fraction; the integer
// counts that retention (Eq. (10)) compares with N_t come from: a per-layer
// floor (forced tokens) given first; the rest water-filled in proportion to
// the shares with a cap of N per layer; largest-remainder rounding with ties to
// the lower layer.  One thread per sequence runs the whole computation in
// float64 with no contraction, in a fixed order, so the result is a pure
// function of the float32 masses.  L is small (tens of layers): this is a
// latency-bound kernel by construction.
#pragma clang fp contract(off)

#include "tgvkv_device.h"
#include "tgvkv_shape.h"

namespace tgvkv {
namespace {

constexpr int kMaxLayers = 512;

__global__ __launch_bounds__(64) void budget_kernel(Shape s, const float* __restrict__ tv_mass, long long total,
                                                    int reserve, int n_forced, int32_t* __restrict__ budgets,
                                                    int64_t* __restrict__ idx_off, int64_t* __restrict__ seg_off) {
    __shared__ double f[kMaxLayers];
    __shared__ double x[kMaxLayers];
    __shared__ long long bcount[kMaxLayers];
    __shared__ unsigned char active[kMaxLayers];
    __shared__ unsigned char taken[kMaxLayers];
    if (threadIdx.x != 0) return;
    const int b = blockIdx.x;
    const int L = s.L;
    const long long N = s.N;

    long long F = n_forced;
    if (total / L < F) F = total / L;
    if (N < F) F = N;
    const long long cap = N - F;
    const long long R = total - (long long)L * F;

    double S = 0.0;
    for (int l = 0; l < L; ++l) {
        const float mv = tv_mass[(size_t)b * L + l];
        const double m = (isfinite(mv) && mv > 0.f) ? (double)mv : 0.0;
        x[l] = m;  // masses, temporarily
        S += m;
    }
    for (int l = 0; l < L; ++l) f[l] = S > 0.0 ? x[l] / S : 1.0 / (double)L;

    for (int l = 0; l < L; ++l) active[l] = 1;
    int n_active = L;
    double remaining = (double)R;
    const double capd = (double)cap;
    while (n_active > 0) {
        double Fa = 0.0;
        for (int l = 0; l < L; ++l)
            if (active[l]) Fa += f[l];
        for (int l = 0; l < L; ++l)
            if (active[l]) x[l] = Fa > 0.0 ? (remaining * f[l]) / Fa : remaining / (double)n_active;
        bool any = false;
        for (int l = 0; l < L; ++l) {
            taken[l] = active[l] && x[l] > capd;
            any = any || taken[l];
        }
        if (!any) break;
        for (int l = 0; l < L; ++l) {
            if (taken[l]) {
                x[l] = capd;
                active[l] = 0;
                remaining -= capd;
                --n_active;
            }
        }
    }

    long long sum = 0;
    for (int l = 0; l < L; ++l) {
        const double fl = floor(x[l]);
        long long base = (long long)fl;
        if (base > cap) base = cap;
        bcount[l] = F + base;
        x[l] = x[l] - fl;  // fractional part
        taken[l] = 0;
        sum += bcount[l];
    }
    long long r = total - sum;
    // +1 to the r layers with the largest fractional parts (ties: lower layer), below the cap
    while (r > 0) {
        int best = -1;
        for (int l = 0; l < L; ++l) {
            if (taken[l] || bcount[l] >= N) continue;
            if (best < 0 || x[l] > x[best]) best = l;
        }
        if (best < 0) break;  // cannot happen when total <= L*N
        taken[best] = 1;
        ++bcount[best];
        --r;
    }

    const long long g = s.ngroups;
    long long io = (long long)b * total * g;
    long long so = (long long)b * (total + (long long)L * reserve);
    for (int l = 0; l < L; ++l) {
        const size_t bl = (size_t)b * L + l;
        budgets[bl] = (int32_t)bcount[l];
        idx_off[bl] = io;
        seg_off[bl] = so;
        io += g * bcount[l];
        so += bcount[l] + reserve;
    }
    if (b == s.B - 1) {
        idx_off[(size_t)s.B * L] = (long long)s.B * total * g;
        seg_off[(size_t)s.B * L] = (long long)s.B * (total + (long long)L * reserve);
    }
}

}  // namespace

hipError_t launch_budget(const Shape& s, const float* tv_mass, int64_t total, int32_t reserve, int32_t n_forced,
                         int32_t* budgets, int64_t* idx_off, int64_t* seg_off, hipStream_t st) {
    if (s.B == 0) return hipSuccess;
    hipLaunchKernelGGL(budget_kernel, dim3(s.B), dim3(64), 0, st, s, tv_mass, (long long)total, reserve, n_forced,
                       budgets, idx_off, seg_off);
    return hipGetLastError();
}

}  // namespace tgvkv
