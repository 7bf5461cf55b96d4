// TVB: integer per-layer budgets of each sequence (Sec. 3.2 Eq. (5), Sec. 3.3 Eq. (6)).
//
// Layer l's share of the sequence budget is m_l / sum_l' m_l', with m_l the summed
// text->vision attention.  The paper states the share as a fraction; the integer
// counts that retention (Eq. (10)) compares with N_t come from: a per-layer
// floor (forced tokens) given first; the rest water-filled in proportion to
// the shares with a cap of N per layer; largest-remainder rounding with ties to
// the lower layer.  Vision-only eviction (App. B.3) shares out a vision budget the
// same way with the cap n_vis, and each layer then also keeps its N_t text tokens.
//
// One workgroup per sequence, layers spread over the threads.  Every float64
// sum runs on one thread in layer order and no operation is contracted, so the
// budgets are a pure function of the float32 masses (element-wise steps are
// order-free).  The largest-remainder step ranks each eligible layer by
// (fraction desc, layer asc) with an all-pairs count, which gives the same set
// as sorting.  The same count by (budget desc, layer asc) gives decode's
// dispatch order: rank-major over the batch, so every sequence's longest
// segments are started first (longest-processing-time-first scheduling).
#pragma clang fp contract(off)

#include "tgvkv_device.h"
#include "tgvkv_shape.h"

namespace tgvkv {
namespace {

constexpr int kMaxLayers = 512;
constexpr int kThreads = 256;

// For every layer l, the number of layers j that precede it in a strict order (prec(j, l)).
// The L x L comparisons are spread over the workgroup: each layer's j range in nch chunks,
// whose counts part[] holds until they are added in chunk order (integers, so exact).
// emit(l, count) runs on thread l % kThreads.  Every thread must call it (a barrier inside).
template <class Prec, class Emit>
__device__ void rank_layers(int L, int* part, Prec prec, Emit emit) {
    const int tid = threadIdx.x;
    const int nch = L <= kThreads / 2 ? kThreads / max(L, 1) : 1;
    const int per = (L + nch - 1) / nch;
    for (int t = tid; t < nch * L; t += kThreads) {
        const int l = t % L, c = t / L;
        const int j1 = min(L, (c + 1) * per);
        int n = 0;
        for (int j = c * per; j < j1; ++j) n += prec(j, l);
        if (nch == 1) emit(l, n);
        else part[t] = n;  // t < nch * L <= kThreads
    }
    if (nch > 1) {
        __syncthreads();
        for (int l = tid; l < L; l += kThreads) {
            int n = 0;
            for (int c = 0; c < nch; ++c) n += part[c * L + l];
            emit(l, n);
        }
    }
}

__global__ __launch_bounds__(kThreads) void budget_kernel(Shape s, const float* __restrict__ tv_mass, long long total,
                                                          int cap_tokens, int add, int reserve, int n_forced,
                                                          int32_t* __restrict__ budgets,
                                                          int64_t* __restrict__ idx_off,
                                                          int64_t* __restrict__ seg_off,
                                                          int32_t* __restrict__ unit_order) {
    __shared__ double f[kMaxLayers];
    __shared__ double x[kMaxLayers];
    __shared__ long long bcount[kMaxLayers];
    __shared__ unsigned char active[kMaxLayers];
    __shared__ double sh_sum;
    const int tid = threadIdx.x;
    const int b = blockIdx.x;
    const int L = s.L;
    const long long N = cap_tokens;  // per-layer cap of the shared-out count

    long long F = n_forced;
    if (total / L < F) F = total / L;
    if (N < F) F = N;
    const long long cap = N - F;
    const long long R = total - (long long)L * F;
    const double capd = (double)cap;

    for (int l = tid; l < L; l += kThreads) {
        const float mv = tv_mass[(size_t)b * L + l];
        double m = (isfinite(mv) && mv > 0.f) ? (double)mv : 0.0;
        // the variants of Table 1(a): uniform, or the text->text mass N_t - m
        if (s.budget_rule == 1) m = 1.0;
        else if (s.budget_rule == 2) m = fmax((double)s.Nt - m, 0.0);
        x[l] = m;  // masses, for now
        active[l] = 1;
    }
    __syncthreads();
    if (tid == 0) {
        double S = 0.0;
#pragma unroll 8
        for (int l = 0; l < L; ++l) S += x[l];
        sh_sum = S;
    }
    __syncthreads();
    const double S = sh_sum;
    for (int l = tid; l < L; l += kThreads) f[l] = S > 0.0 ? x[l] / S : 1.0 / (double)L;
    __syncthreads();

    // water-fill: capped layers are fixed and the remainder is re-shared
    double remaining = (double)R;
    int n_active = L;
    __shared__ int sh_over;
    while (n_active > 0) {
        if (tid == 0) {
            // a capped layer's share is 0 (set when it is capped): adding +0.0 leaves the bits
            // of the sum as they are (it starts at +0.0 and every share is >= 0), and with no
            // test per layer the loads of a group of layers issue together
            double Fa = 0.0;
#pragma unroll 8
            for (int l = 0; l < L; ++l) Fa += f[l];
            sh_sum = Fa;
            sh_over = 0;
        }
        __syncthreads();
        const double Fa = sh_sum;
        int over = 0;
        for (int l = tid; l < L; l += kThreads) {
            if (active[l]) {
                x[l] = Fa > 0.0 ? (remaining * f[l]) / Fa : remaining / (double)n_active;
                over += x[l] > capd;
            }
        }
        // a thread holds up to kMaxLayers / kThreads layers: the count is a sum, not a vote
        if (over) atomicAdd(&sh_over, over);
        __syncthreads();
        const int n_over = sh_over;
        if (n_over == 0) break;
        for (int l = tid; l < L; l += kThreads) {
            if (active[l] && x[l] > capd) {
                x[l] = capd;
                active[l] = 0;
                f[l] = 0.0;
            }
        }
        // remaining and cap are integers below 2^53: the subtraction is exact in any order
        remaining -= capd * (double)n_over;
        n_active -= n_over;
        __syncthreads();
    }

    // x becomes the fractional part of each layer still below the cap, -1 for the others
    // (fractions lie in [0, 1), so -1 ranks below every eligible layer and ties none)
    long long part = 0;
    for (int l = tid; l < L; l += kThreads) {
        const double fl = floor(x[l]);
        long long base = (long long)fl;
        if (base > cap) base = cap;
        bcount[l] = F + base;
        x[l] = F + base < N ? x[l] - fl : -1.0;
        part += base;
    }
    // the floors' sum (integers, exact in any order): per wave by shuffles, then the wave sums
    __shared__ long long wpart[kThreads / 64];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) part += shfl_xor(part, o);
    if ((tid & 63) == 0) wpart[tid >> 6] = part;
    __syncthreads();
    long long base_sum = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) base_sum += wpart[w];
    const long long r = total - ((long long)L * F + base_sum);

    // +1 to the r eligible layers ranked first by (fraction desc, layer asc); every rank is
    // taken before any count changes
    __shared__ int cnt[kMaxLayers];
    __shared__ int rank_part[kThreads];
    rank_layers(
        L, rank_part, [&](int j, int l) { return (x[j] > x[l]) || (x[j] == x[l] && j < l) ? 1 : 0; },
        [&](int l, int rank) { cnt[l] = (int)bcount[l] + (x[l] >= 0.0 && rank < r ? 1 : 0); });
    __syncthreads();

    if (unit_order != nullptr) {
        rank_layers(
            L, rank_part, [&](int j, int l) { return (cnt[j] > cnt[l]) || (cnt[j] == cnt[l] && j < l) ? 1 : 0; },
            [&](int l, int rank) { unit_order[(size_t)rank * s.B + b] = b * L + l; });
    }

    // budgets and the two offset tables: prefix sums of the per-layer counts (integers, so
    // the order of the additions does not matter), 64 layers at a time by wave 0
    if (tid < 64) {
        const long long g = s.ngroups;
        const long long kept = total + (long long)L * add;  // tokens each sequence keeps
        const long long io0 = (long long)b * kept * g;
        const long long so0 = (long long)b * (kept + (long long)L * reserve);
        long long carry = 0;
        for (int c0 = 0; c0 < L; c0 += 64) {
            const int l = c0 + tid;
            const int v = l < L ? add + cnt[l] : 0;  // tokens layer l keeps (< 2^24)
            int incl = v;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const int y = __shfl_up(incl, o, 64);
                if (tid >= o) incl += y;
            }
            if (l < L) {
                const size_t bl = (size_t)b * L + l;
                const long long before = carry + (incl - v);
                budgets[bl] = v;
                idx_off[bl] = io0 + g * before;
                seg_off[bl] = so0 + before + (long long)l * reserve;
            }
            carry += __shfl(incl, 63, 64);
        }
        if (b == s.B - 1 && tid == 0) {
            idx_off[(size_t)s.B * L] = (long long)s.B * kept * g;
            seg_off[(size_t)s.B * L] = (long long)s.B * (kept + (long long)L * reserve);
        }
    }
}

}  // namespace

hipError_t launch_budget(const Shape& s, const float* tv_mass, int64_t total, int32_t cap_tokens, int32_t add,
                         int32_t reserve, int32_t n_floor, int32_t* budgets, int64_t* idx_off, int64_t* seg_off,
                         int32_t* unit_order, hipStream_t st) {
    if (s.B == 0) return hipSuccess;
    hipLaunchKernelGGL(budget_kernel, dim3(s.B), dim3(kThreads), 0, st, s, tv_mass, (long long)total, cap_tokens,
                       add, reserve, n_floor, budgets, idx_off, seg_off, unit_order);
    return hipGetLastError();
}

}  // namespace tgvkv
