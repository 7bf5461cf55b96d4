// TPR: text-prioritised retention (Sec. 3.3, Eq. (10)).
//
// One workgroup per (sequence, layer, group).  The retained set is forced
// positions first (first n_sink, last n_recent), then either the top text tokens
// by s^T (budget does not cover the remaining text) or all text and the top
// vision tokens by s^V.  The top-k is an exact radix select on order-preserving
// 32-bit keys (4 passes of 8 bits with an LDS histogram), which yields the k-th
// largest key and how many of its ties to take; ties go to the lower position.
// A single ordered scan over all N positions then emits the retained positions
// already in ascending order, with no sort.
#include "tgvkv_device.h"
#include "tgvkv_shape.h"

namespace tgvkv {
namespace {

constexpr int kThreads = 256;
enum { MODE_FORCED = 0, MODE_TEXT = 1, MODE_VIS = 2 };

struct RowCtx {
    int N, Ns, Nv, Nt, fs, fr;  // forced = [0, fs) U [fr, N)
    int mode;
    const float* sv;            // s_vis row (n_vis)
    const float* st;            // s_txt row (N_t)
    __device__ bool forced(int p) const { return p < fs || p >= fr; }
    __device__ bool is_vis(int p) const { return p >= Ns && p < Ns + Nv; }
    // candidate of the top-k in this mode, and its key
    __device__ bool cand(int p, uint32_t& key) const {
        if (mode == MODE_FORCED) {
            key = 0u;
            return forced(p);
        }
        if (forced(p)) return false;
        if (mode == MODE_VIS) {
            if (!is_vis(p)) return false;
            key = ordered_key(sv[p - Ns]);
            return true;
        }
        if (is_vis(p)) return false;
        key = ordered_key(st[p < Ns ? p : p - Nv]);
        return true;
    }
    // kept without competing (forced in the text/vision modes, all text in the vision mode)
    __device__ bool kept_outright(int p) const {
        if (mode == MODE_FORCED) return false;
        if (forced(p)) return true;
        return mode == MODE_VIS && !is_vis(p);
    }
};

// Exclusive scan of one int per thread across the block; returns the prefix, total in *tot.
__device__ int block_exclusive_scan(int v, int* tot, int* sh) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    if (lane == 63) sh[wave] = x;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) {
        const int t = sh[w];
        if (w < wave) before += t;
        all += t;
    }
    __syncthreads();
    *tot = all;
    return before + x - v;
}

__global__ __launch_bounds__(kThreads) void select_kernel(Shape s, const float* __restrict__ s_vis,
                                                          const float* __restrict__ s_txt,
                                                          const int32_t* __restrict__ budgets,
                                                          const int64_t* __restrict__ idx_off,
                                                          int32_t* __restrict__ idx) {
    __shared__ int hist[256];
    __shared__ int sh[8];
    __shared__ uint32_t sel[2];  // threshold key, remaining count
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
    c.sv = s_vis + ((size_t)bl * s.ngroups + gi) * s.Nv;
    c.st = s_txt + ((size_t)bl * s.ngroups + gi) * s.Nt;

    // counts: forced, text not forced
    int nf = 0, ntf = 0;
    for (int p = tid; p < s.N; p += kThreads) {
        if (c.forced(p)) ++nf;
        else if (!c.is_vis(p)) ++ntf;
    }
    int tot;
    block_exclusive_scan(nf, &tot, sh);
    nf = tot;
    block_exclusive_scan(ntf, &tot, sh);
    ntf = tot;

    int k;
    if (bgt <= nf) { c.mode = MODE_FORCED; k = bgt; }
    else if (bgt - nf <= ntf) { c.mode = MODE_TEXT; k = bgt - nf; }
    else { c.mode = MODE_VIS; k = bgt - nf - ntf; }

    // candidate count
    int nc = 0;
    for (int p = tid; p < s.N; p += kThreads) {
        uint32_t key;
        if (c.cand(p, key)) ++nc;
    }
    block_exclusive_scan(nc, &tot, sh);
    nc = tot;

    uint32_t thr;
    int take_ties;
    if (k <= 0) { thr = 0xFFFFFFFFu; take_ties = 0; }
    else if (k >= nc) { thr = 0u; take_ties = nc; }
    else {
        uint32_t prefix = 0u, mask = 0u;
        int kr = k;
        for (int shift = 24; shift >= 0; shift -= 8) {
            hist[tid] = 0;
            __syncthreads();
            for (int p = tid; p < s.N; p += kThreads) {
                uint32_t key;
                if (c.cand(p, key) && (key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1);
            }
            __syncthreads();
            if (tid == 0) {
                int above = 0, d = 255;
                for (; d > 0; --d) {
                    if (above + hist[d] >= kr) break;
                    above += hist[d];
                }
                sel[0] = (uint32_t)d;
                sel[1] = (uint32_t)(kr - above);
            }
            __syncthreads();
            prefix |= sel[0] << shift;
            mask |= 0xFFu << shift;
            kr = (int)sel[1];
            __syncthreads();
        }
        thr = prefix;
        take_ties = kr;
    }

    // ordered emission: thread t owns positions [t*chunk, (t+1)*chunk)
    const int chunk = (s.N + kThreads - 1) / kThreads;
    const int p0 = min(tid * chunk, s.N), p1 = min(p0 + chunk, s.N);
    int nties = 0;
    for (int p = p0; p < p1; ++p) {
        uint32_t key;
        if (c.cand(p, key) && key == thr) ++nties;
    }
    int tie_rank = block_exclusive_scan(nties, &tot, sh);
    int nkeep = 0;
    {
        int tr = tie_rank;
        for (int p = p0; p < p1; ++p) {
            uint32_t key;
            bool keep = c.kept_outright(p);
            if (!keep && c.cand(p, key)) {
                if (key > thr) keep = true;
                else if (key == thr) keep = (tr++ < take_ties);
            }
            nkeep += keep;
        }
    }
    int pos = block_exclusive_scan(nkeep, &tot, sh);
    {
        int tr = tie_rank;
        for (int p = p0; p < p1; ++p) {
            uint32_t key;
            bool keep = c.kept_outright(p);
            if (!keep && c.cand(p, key)) {
                if (key > thr) keep = true;
                else if (key == thr) keep = (tr++ < take_ties);
            }
            if (keep && pos < bgt) out[pos++] = p;
        }
    }
}

}  // namespace

hipError_t launch_select(const Shape& s, const float* s_vis, const float* s_txt, const int32_t* budgets,
                         const int64_t* idx_off, int32_t* idx, hipStream_t st) {
    const long long nblk = (long long)s.B * s.L * s.ngroups;
    if (nblk == 0) return hipSuccess;
    hipLaunchKernelGGL(select_kernel, dim3((unsigned)nblk), dim3(kThreads), 0, st, s, s_vis, s_txt, budgets,
                       idx_off, idx);
    return hipGetLastError();
}

}  // namespace tgvkv
