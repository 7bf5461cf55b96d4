// TPR: text-prioritised retention (Sec. 3.3, Eq. (10)).
//
// One workgroup per (sequence, layer, group).  The retained set is forced
// positions first (first n_sink, last n_recent), then either the top text tokens
// by s^T (the budget does not cover the remaining text) or all text and the top
// vision tokens by s^V.  The top-k is an exact radix select on order-preserving
// 32-bit keys (4 passes of 8 bits with an LDS histogram; the digit holding the
// k-th key is found by a wave-wide scan of the histogram), which yields the k-th
// largest key and how many of its ties to take; ties go to the lower position.
// The retained positions are then emitted already in ascending order, with no sort:
// each wave takes a contiguous run of 64-position groups, wave ballots count and rank
// the ties and the kept positions, and the waves' counts, added across one barrier, give
// each run the rank of its first tie and the output slot of its first kept position.
// The workgroup has 1024 threads: the work is a few latency-bound rounds per
// (sequence, layer, group), and there are few such units.  Without TPR (an ablation of Table 5)
// all non-forced positions compete on one scale: text by s^T, vision by s^V times
// a factor (N_t under TWR, whose weights sum to 1).  Candidate keys are read from global
// memory once and kept in LDS when the row fits (N <= kLdsKeys).
#include "tgvkv_device.h"
#include "tgvkv_shape.h"

namespace tgvkv {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kLdsKeys = 12288;  // 48 KB of LDS keys per workgroup
enum { MODE_FORCED = 0, MODE_TEXT = 1, MODE_VIS = 2, MODE_JOINT = 3 };
constexpr uint32_t kNotCand = 0u;  // keys of real candidates have the top bit or are >= 1

struct RowCtx {
    int N, Ns, Nv, Nt, fs, fr;  // forced = [0, fs) U [fr, N)
    int mode;
    float vscale;               // factor on s^V in the joint ranking
    const float* sv;            // s_vis row (n_vis)
    const float* st;            // s_txt row (N_t)
    __device__ bool forced(int p) const { return p < fs || p >= fr; }
    __device__ bool is_vis(int p) const { return p >= Ns && p < Ns + Nv; }
    __device__ bool cand(int p) const {
        if (mode == MODE_FORCED) return forced(p);
        if (forced(p)) return false;
        if (mode == MODE_JOINT) return true;
        return mode == MODE_VIS ? is_vis(p) : !is_vis(p);
    }
    // key of a candidate (only called when cand(p)); never kNotCand for finite scores.  The
    // forced positions all get one key, so the ties-to-lower-position rule takes the first ones.
    __device__ uint32_t key(int p) const {
        if (mode == MODE_FORCED) return 1u;
        if (mode == MODE_VIS) return ordered_key(sv[p - Ns]);
        if (mode == MODE_JOINT && is_vis(p)) return ordered_key(sv[p - Ns] * vscale);
        return ordered_key(st[p < Ns ? p : p - Nv]);
    }
    // kept without competing (forced in the text/vision modes, all text in the vision mode)
    __device__ bool kept_outright(int p) const {
        if (mode == MODE_FORCED) return false;
        if (forced(p)) return true;
        return mode == MODE_VIS && !is_vis(p);
    }
};

// Wave 0 finds the digit d (scanning 255 down to 0) where the running count of
// larger digits first reaches kr; writes d and kr minus the count above d.
__device__ void find_digit(const int* hist, int kr, uint32_t* sel) {
    const int lane = threadIdx.x & 63;
    // lane j owns digits 255-4j .. 252-4j
    int c[4];
    int tot = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        c[i] = hist[255 - 4 * lane - i];
        tot += c[i];
    }
    int incl = tot;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o, 64);
        if (lane >= o) incl += y;
    }
    const int excl = incl - tot;
    const unsigned long long hit = __ballot(incl >= kr);
    const int first = hit ? __ffsll((long long)hit) - 1 : 63;
    if (lane == first) {
        int above = excl, d = 252 - 4 * lane;
        for (int i = 0; i < 4; ++i) {
            if (above + c[i] >= kr) {
                d = 255 - 4 * lane - i;
                break;
            }
            above += c[i];
        }
        sel[0] = (uint32_t)d;
        sel[1] = (uint32_t)(kr - above);
    }
}

template <bool LDS_KEYS>
__global__ __launch_bounds__(kThreads) void select_kernel(Shape s, const float* __restrict__ s_vis,
                                                          const float* __restrict__ s_txt,
                                                          const int32_t* __restrict__ budgets,
                                                          const int64_t* __restrict__ idx_off,
                                                          int32_t* __restrict__ idx) {
    __shared__ int hist[256];
    __shared__ int wtot[kWaves][2];
    __shared__ uint32_t sel[2];
    __shared__ uint32_t keys[LDS_KEYS ? kLdsKeys : 1];
    const int tid = threadIdx.x;
    const int gi = blockIdx.x % s.ngroups;
    const int bl = blockIdx.x / s.ngroups;
    const int bgt = budgets[bl];
    int32_t* out = idx + idx_off[bl] + (int64_t)gi * bgt;

    RowCtx c;
    c.N = s.N;
    c.Ns = s.Ns;
    c.Nv = s.Nv;
    c.Nt = s.Nt;
    c.fs = min(s.n_sink, s.N);
    c.fr = max(s.N - s.n_recent, c.fs);
    c.vscale = s.vision_rank == 0 ? (float)s.Nt : 1.f;
    c.sv = s_vis + ((size_t)bl * s.ngroups + gi) * s.Nv;
    c.st = s_txt + ((size_t)bl * s.ngroups + gi) * s.Nt;

    // forced positions, and text positions that are not forced: [fs, min(Ns, fr)) and
    // [max(Ns + Nv, fs), fr), from the layout alone
    const int nf = c.fs + (s.N - c.fr);
    const int ntf = max(0, min(s.Ns, c.fr) - c.fs) + max(0, c.fr - max(s.Ns + s.Nv, c.fs));

    int k;
    if (bgt <= nf) { c.mode = MODE_FORCED; k = bgt; }
    else if (s.joint_rank) { c.mode = MODE_JOINT; k = bgt - nf; }
    else if (bgt - nf <= ntf) { c.mode = MODE_TEXT; k = bgt - nf; }
    else { c.mode = MODE_VIS; k = bgt - nf - ntf; }
    const int nc = c.mode == MODE_FORCED ? nf
                 : c.mode == MODE_JOINT  ? s.N - nf
                 : c.mode == MODE_TEXT   ? ntf
                                         : s.N - nf - ntf;

    // key lookup: from LDS when the row fits (kNotCand marks non-candidates), else re-read
    auto key_at = [&](int p) -> uint32_t { return LDS_KEYS ? keys[p] : (c.cand(p) ? c.key(p) : kNotCand); };
    if (LDS_KEYS) {
        for (int p = tid; p < s.N; p += kThreads) keys[p] = c.cand(p) ? c.key(p) : kNotCand;
        __syncthreads();
    }

    uint32_t thr;
    int take_ties;
    if (k <= 0) { thr = 0xFFFFFFFFu; take_ties = 0; }
    else if (k >= nc) { thr = 0u; take_ties = nc; }
    else {
        uint32_t prefix = 0u, mask = 0u;
        int kr = k;
        for (int shift = 24; shift >= 0; shift -= 8) {
            if (tid < 256) hist[tid] = 0;
            __syncthreads();
            for (int p = tid; p < s.N; p += kThreads) {
                const uint32_t key = key_at(p);
                if (key != kNotCand && (key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1);
            }
            __syncthreads();
            if (tid < 64) find_digit(hist, kr, sel);
            __syncthreads();
            prefix |= sel[0] << shift;
            mask |= 0xFFu << shift;
            kr = (int)sel[1];
        }
        thr = prefix;
        take_ties = kr;
    }

    // ordered emission.  A tie is kept while its rank among the ties (in position order) is
    // below take_ties, so the kept ties before a position are min(take_ties, ties before it).
    // Each wave owns a contiguous run of 64-position groups.  It counts its ties and its other
    // kept positions (ballots only); one barrier, and every wave adds the counts of the waves
    // before it; then it walks its groups again, ranking each group's ties and kept positions
    // by ballots, and writes the kept positions in order.
    const int lane = tid & 63, wave = tid >> 6;
    const unsigned long long below = (1ull << lane) - 1ull;
    const int ngrp = (s.N + 63) >> 6;
    const int gpw = (ngrp + kWaves - 1) / kWaves;
    const int g0 = min(wave * gpw, ngrp), g1 = min(g0 + gpw, ngrp);
    auto classify = [&](int p, bool& tie) {  // kept outright or above the threshold; tie
        tie = false;
        if (p >= s.N) return false;
        const uint32_t key = key_at(p);
        const bool outright = c.kept_outright(p);
        const bool cand = !outright && key != kNotCand && c.cand(p);
        tie = cand && key == thr;
        return outright || (cand && key > thr);
    };
    int nt = 0, nk = 0;  // uniform over the wave
    for (int gq = g0; gq < g1; ++gq) {
        bool tie;
        const bool other = classify(gq * 64 + lane, tie);
        nt += __popcll(__ballot(tie));
        nk += __popcll(__ballot(other));
    }
    if (lane == 0) {
        wtot[wave][0] = nt;
        wtot[wave][1] = nk;
    }
    __syncthreads();
    int tb = 0, ob = 0;  // ties and other kept positions before this wave's run
    for (int w = 0; w < wave; ++w) {
        tb += wtot[w][0];
        ob += wtot[w][1];
    }
    for (int gq = g0; gq < g1; ++gq) {
        const int p = gq * 64 + lane;
        bool tie;
        const bool other = classify(p, tie);
        const unsigned long long tm = __ballot(tie);
        const bool keep = other || (tie && tb + __popcll(tm & below) < take_ties);
        const unsigned long long km = __ballot(keep);
        const int pos = ob + min(take_ties, tb) + __popcll(km & below);
        if (keep && pos < bgt) out[pos] = p;
        tb += __popcll(tm);
        ob += __popcll(__ballot(other));
    }
}

}  // namespace

hipError_t launch_select(const Shape& s, const float* s_vis, const float* s_txt, const int32_t* budgets,
                         const int64_t* idx_off, int32_t* idx, hipStream_t st) {
    const long long nblk = (long long)s.B * s.L * s.ngroups;
    if (nblk == 0) return hipSuccess;
    if (s.N <= kLdsKeys)
        hipLaunchKernelGGL(select_kernel<true>, dim3((unsigned)nblk), dim3(kThreads), 0, st, s, s_vis, s_txt, budgets,
                           idx_off, idx);
    else
        hipLaunchKernelGGL(select_kernel<false>, dim3((unsigned)nblk), dim3(kThreads), 0, st, s, s_vis, s_txt,
                           budgets, idx_off, idx);
    return hipGetLastError();
}

}  // namespace tgvkv
