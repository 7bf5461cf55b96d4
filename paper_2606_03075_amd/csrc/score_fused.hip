// TWR / TVB scoring as one persistent kernel (gfx950).
//
// Both sweeps over K of a (sequence, layer) must finish the first before the
// second starts (the second needs every row's normaliser and the text weights,
// which depend on all heads of the layer), so run one after the other over the
// whole batch they re-read all of K from HBM.  Here the work is cut into items
// that workgroups take in ticket order:
//   A item (unit u, key split p): statistics sweep of u's question rows over one
//     contiguous key range -> partial (max, sum, vision sum) per row;
//   B item (unit u, vision split p): text-weighted column sums of u's question
//     rows over one range of vision keys.
// Tickets give layer bl's A items `lag` layers before its B items, so when a B
// item re-reads its keys the layer was streamed a few layers earlier: the
// re-read hits the last-level (MALL) cache instead of HBM.
//
// Completion is resolved by counters in the workspace, "last arriver does the
// next step": the last A item of a unit merges the partial statistics (split
// order, deterministic) and runs the text x text pass of the unit; the last
// unit of a layer computes the layer's s^T, w~ and text->vision mass and raises
// the layer's ready flag; B items wait for it; with one retained set per layer
// the last B item of a layer sums the KV heads' partials into s^V.
//
// Progress: a B item waits only for A items of its own layer, which hold
// earlier tickets, were handed to running workgroups and never wait; so every
// wait ends.  The wait is still bounded: past the limit the item is dropped and
// an error word is set in the workspace, so the kernel always drains.
// Cross-workgroup data: writers store, barrier, then one thread fences at agent
// scope and increments the counter; readers see the counter, fence, barrier,
// then load.
#include <algorithm>

#include "score_core.h"

namespace tgvkv {
namespace {

using namespace core;

constexpr int kMaxQRows = 24 * 16;          // question rows of a unit in the fused path
constexpr int kSpinLimit = 1 << 18;         // bounded wait for a layer's ready flag (~0.1 s)

__device__ __forceinline__ void decode_ticket(const FusedPlan& fp, long long t, bool& isA, int& bl, int& idx) {
    const long long P = fp.lag, nA = fp.nA, nB = fp.nB, nbl = fp.nbl;
    if (t < P * nA) {
        isA = true;
        bl = (int)(t / nA);
        idx = (int)(t % nA);
        return;
    }
    long long t1 = t - P * nA;
    const long long mid = (nbl - P) * (nA + nB);
    if (t1 < mid) {
        const long long j = t1 / (nA + nB), r = t1 % (nA + nB);
        if (r < nB) {
            isA = false;
            bl = (int)j;
            idx = (int)r;
        } else {
            isA = true;
            bl = (int)(j + P);
            idx = (int)(r - nB);
        }
        return;
    }
    t1 -= mid;
    isA = false;
    bl = (int)((nbl - P) + t1 / nB);
    idx = (int)(t1 % nB);
}

template <int D, int NSLOT, int KS>
__global__ __launch_bounds__(kThreads) void score_fused_kernel(
    Shape s, FusedPlan fp, const uint16_t* __restrict__ q_text, const uint16_t* __restrict__ k,
    float* __restrict__ lse, float* __restrict__ s_txt, float* __restrict__ w_txt, float* __restrict__ tv_mass,
    float* __restrict__ s_vis, float* __restrict__ part_stats, float* __restrict__ ws_colsum,
    float* __restrict__ ws_vmh, float* __restrict__ ws_part, int* __restrict__ sync) {
    constexpr int RSETS = 4 / KS;
    __shared__ __attribute__((aligned(16))) char tiles[2][Geo<D>::TILE_BYTES];
    __shared__ float red[2][RSETS][kTile];
    __shared__ float obuf[kOutTiles * kTile];
    __shared__ float fin_red[kThreads];
    __shared__ float vm_s[kMaxQRows];
    __shared__ int sh_ticket, sh_flag;
    extern __shared__ float lse2s[];  // [G][N_t], base-2 units

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int rs = wave % RSETS, kp = wave / RSETS;
    const int QB = (s.Nq + 15) >> 4;
    const int NB = s.G * QB;
    const int NBR = NB * 16;
    const int U = s.B * s.L * s.Hkv;
    const int nbl = s.B * s.L;
    int* ticket = sync;
    int* err = sync + 1;
    int* cntA = sync + 2;
    int* cntL = cntA + U;
    int* cntB = cntL + nbl;
    int* ready = cntB + nbl;

    // Every loop decision below is made on a wave-uniform (scalar) value, read
    // once from LDS after a barrier, and the loop has a single back edge through
    // the ticket fetch: barriers then sit in uniform control flow only.
    for (;;) {
        if (tid == 0) sh_ticket = atomicAdd(ticket, 1);
        __syncthreads();
        const int t = __builtin_amdgcn_readfirstlane(sh_ticket);
        __syncthreads();
        if ((long long)t >= fp.total) break;
        bool isA;
        int bl, idx;
        decode_ticket(fp, t, isA, bl, idx);
        bl = __builtin_amdgcn_readfirstlane(bl);
        idx = __builtin_amdgcn_readfirstlane(idx);

        if (isA) {
            const int kvh = idx / fp.sa, sp = idx % fp.sa;
            const int u = bl * s.Hkv + kvh;
            {
                bf16x8 qf[NSLOT][Geo<D>::KSTEPS];
                int qrow[NSLOT];
                load_qrows<D, NSLOT, KS>(s, q_text, bl, kvh, 0, qf, qrow);
                float m[NSLOT], lsum[NSLOT], vsum[NSLOT];
                const uint16_t* kbase = k + (size_t)u * s.N * D;
                const int kb = sp * fp.cs, ke = min(s.N, kb + fp.cs);
                stats_sweep<D, NSLOT, KS>(s, kbase, kb, ke, qf, qrow, tiles, m, lsum, vsum);
                if (kp == 0 && lane < 16) {
#pragma unroll
                    for (int sl = 0; sl < NSLOT; ++sl) {
                        const int rb = rs + sl * RSETS;
                        if (rb < NB) {
                            float* p = part_stats + (((size_t)u * fp.sa + sp) * NBR + rb * 16 + lane) * 3;
                            p[0] = m[sl];
                            p[1] = lsum[sl];
                            p[2] = vsum[sl];
                        }
                    }
                }
            }
            __syncthreads();
            if (tid == 0) {
                __threadfence();
                const int last = atomicAdd(&cntA[u], 1) == fp.sa - 1;
                if (last) __threadfence();
                sh_flag = last;
            }
            __syncthreads();
            const int unit_last = __builtin_amdgcn_readfirstlane(sh_flag);
            if (unit_last) {
                // last split of the unit: final normalisers and vision mass of its question rows
                const size_t head0 = (size_t)bl * s.H + kvh * s.G;
                for (int r = tid; r < NBR; r += kThreads) {
                    const int rb = r >> 4, g = rb / QB, qi = (rb % QB) * 16 + (r & 15);
                    if (qi < s.Nq) {
                        float M = kNegInf, Ls = 0.f, Vs = 0.f;
                        for (int p2 = 0; p2 < fp.sa; ++p2) {
                            const float* p = part_stats + (((size_t)u * fp.sa + p2) * NBR + r) * 3;
                            merge_stats(M, Ls, Vs, p[0], p[1], p[2]);
                        }
                        const float L2 = M + log2f(Ls);
                        lse[(head0 + g) * s.Nt + s.Ns + qi] = L2 * kLn2;
                        lse2s[g * s.Nt + s.Ns + qi] = L2;
                        vm_s[r] = Vs / Ls;
                    }
                }
                __syncthreads();
                if (tid < s.G) {
                    float a = 0.f;
                    for (int qi = 0; qi < s.Nq; ++qi) a += vm_s[tid * QB * 16 + qi];
                    ws_vmh[head0 + tid] = a;
                }
                text_pass<D>(s, bl, kvh, q_text, k, lse, lse2s, ws_colsum);
                if (tid == 0) {
                    __threadfence();
                    const int last = atomicAdd(&cntL[bl], 1) == s.Hkv - 1;
                    if (last) __threadfence();
                    sh_flag = last;
                }
                __syncthreads();
                const int layer_last = __builtin_amdgcn_readfirstlane(sh_flag);
                if (layer_last) {
                    // last unit of the layer: head means, weights, text->vision mass; release the layer
                    for (int gi = 0; gi < s.ngroups; ++gi)
                        finalize_group(s, bl, gi, ws_colsum, ws_vmh, s_txt, w_txt, tv_mass, fin_red);
                    if (tid == 0) {
                        __threadfence();
                        __hip_atomic_store(&ready[bl], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
                    }
                }
            }
        } else {
            const int kvh = idx / fp.sb, sp = idx % fp.sb;
            const int u = bl * s.Hkv + kvh;
            if (tid == 0) {
                int ok = 1;
                int spins = 0;
                while (__hip_atomic_load(&ready[bl], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) == 0) {
                    __builtin_amdgcn_s_sleep(8);
                    if (++spins > kSpinLimit) {
                        ok = 0;
                        atomicExch(err, 1);
                        break;
                    }
                }
                if (ok) __threadfence();
                sh_flag = ok;
            }
            __syncthreads();
            const int ready_ok = __builtin_amdgcn_readfirstlane(sh_flag);
            if (ready_ok) {
                {
                    bf16x8 qf[NSLOT][Geo<D>::KSTEPS];
                    int qrow[NSLOT];
                    load_qrows<D, NSLOT, KS>(s, q_text, bl, kvh, 0, qf, qrow);
                    float lse2[NSLOT][4], coef[NSLOT][4];
                    load_row_coefs<NSLOT, KS>(s, bl, kvh, 0, lse, w_txt, lse2, coef);
                    const uint16_t* kvis = k + ((size_t)u * s.N + s.Ns) * D;
                    const int vb = sp * fp.cv, ve = min(s.Nv, vb + fp.cv);
                    float* out = s.head_mode == 0 ? ws_part + (size_t)u * s.Nv : s_vis + (size_t)u * s.Nv;
                    float rsum_unused[NSLOT][4];
                    vision_sweep<D, NSLOT, KS>(s, kvis, vb, ve, qf, lse2, coef, 0, NB, tiles, red, obuf, kOutTiles, out,
                                               rsum_unused);
                }
                if (s.head_mode == 0) {
                    if (tid == 0) {
                        __threadfence();
                        const int last = atomicAdd(&cntB[bl], 1) == s.Hkv * fp.sb - 1;
                        if (last) __threadfence();
                        sh_flag = last;
                    }
                    __syncthreads();
                    const int vis_last = __builtin_amdgcn_readfirstlane(sh_flag);
                    if (vis_last) {
                        // last vision item of the layer: sum the KV heads' partials, in head order
                        for (int j = tid; j < s.Nv; j += kThreads) {
                            float a = 0.f;
                            for (int kv = 0; kv < s.Hkv; ++kv) a += ws_part[((size_t)bl * s.Hkv + kv) * s.Nv + j];
                            s_vis[(size_t)bl * s.Nv + j] = a;
                        }
                    }
                }
            }
        }
        __syncthreads();
    }
}

__global__ void zero_words_kernel(int* __restrict__ p, long long n) {
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x)
        p[i] = 0;
}

template <int D, int NSLOT, int KS>
hipError_t launch_fused_t(const Shape& s, FusedPlan fp, const FusedPtrs& p, hipStream_t st) {
    auto kern = score_fused_kernel<D, NSLOT, KS>;
    const size_t lds = sizeof(float) * (size_t)s.G * s.Nt;
    int per_cu = 0, cus = 0, dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kThreads, lds);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    long long grid = (long long)std::max(per_cu, 1) * std::max(cus, 1);
    if (grid > fp.total) grid = fp.total;
    // lookahead: a layer's B items come after about one grid's worth of A items
    const long long per_layer = (long long)fp.nA + fp.nB;
    long long lag = fp.nB > 0 ? (grid + per_layer - 1) / per_layer + 1 : fp.nbl;
    if (fp.lag > 0) lag = fp.lag;
    fp.lag = (int)std::min<long long>(std::max<long long>(lag, 1), fp.nbl);
    const long long nwords = fused_sync_words(s);
    hipLaunchKernelGGL(zero_words_kernel, dim3((unsigned)std::min<long long>((nwords + 255) / 256, 1024)), dim3(256),
                       0, st, p.sync, nwords);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), lds, st, s, fp, p.q_text, p.k, p.lse, p.s_txt,
                       p.w_txt, p.tv_mass, p.s_vis, p.part_stats, p.ws_colsum, p.ws_vmh, p.ws_part, p.sync);
    return hipGetLastError();
}

}  // namespace

long long fused_sync_words(const Shape& s) {
    const long long U = (long long)s.B * s.L * s.Hkv, nbl = (long long)s.B * s.L;
    return 2 + U + 3 * nbl;
}

bool fused_eligible(const Shape& s, const RowPlan& rp) {
    return s.Nq > 0 && rp.rowgroups == 1 && s.G * ((s.Nq + 15) / 16) * 16 <= kMaxQRows;
}

FusedPlan plan_fused(const Shape& s, bool with_vision) {
    FusedPlan fp;
    // about 160 KB of K per statistics item (640 keys at head_dim 128)
    const long long target_keys = 81920 / s.D;
    fp.sa = (int)std::max<long long>(1, std::min<long long>(16, (s.N + target_keys - 1) / target_keys));
    fp.cs = ((s.N + fp.sa - 1) / fp.sa + kTile - 1) / kTile * kTile;
    fp.sa = (s.N + fp.cs - 1) / fp.cs;
    if (with_vision && s.Nv > 0) {
        fp.sb = (int)std::max<long long>(1, std::min<long long>(16, (s.Nv + target_keys - 1) / target_keys));
        fp.cv = ((s.Nv + fp.sb - 1) / fp.sb + kTile - 1) / kTile * kTile;
        fp.sb = (s.Nv + fp.cv - 1) / fp.cv;
    } else {
        fp.sb = 0;
        fp.cv = 0;
    }
    fp.nbl = s.B * s.L;
    fp.nA = s.Hkv * fp.sa;
    fp.nB = s.Hkv * fp.sb;
    fp.total = (long long)fp.nbl * (fp.nA + fp.nB);
    fp.lag = 0;  // chosen at launch from the persistent grid size
    return fp;
}

hipError_t launch_score_fused(const Shape& s, const RowPlan& rp, const FusedPlan& fp, const FusedPtrs& p,
                              hipStream_t st) {
    if (fp.total == 0) return hipSuccess;
    if (s.D == 128) {
        if (rp.ks == 4) return launch_fused_t<128, 1, 4>(s, fp, p, st);
        if (rp.ks == 2 && rp.nslot == 1) return launch_fused_t<128, 1, 2>(s, fp, p, st);
        if (rp.ks == 2) return launch_fused_t<128, 2, 2>(s, fp, p, st);
        if (rp.nslot == 1) return launch_fused_t<128, 1, 1>(s, fp, p, st);
        if (rp.nslot == 2) return launch_fused_t<128, 2, 1>(s, fp, p, st);
        if (rp.nslot == 4) return launch_fused_t<128, 4, 1>(s, fp, p, st);
        return launch_fused_t<128, 6, 1>(s, fp, p, st);
    }
    if (rp.ks == 4) return launch_fused_t<64, 1, 4>(s, fp, p, st);
    if (rp.ks == 2 && rp.nslot == 1) return launch_fused_t<64, 1, 2>(s, fp, p, st);
    if (rp.ks == 2) return launch_fused_t<64, 2, 2>(s, fp, p, st);
    if (rp.nslot == 1) return launch_fused_t<64, 1, 1>(s, fp, p, st);
    if (rp.nslot == 2) return launch_fused_t<64, 2, 1>(s, fp, p, st);
    if (rp.nslot == 4) return launch_fused_t<64, 4, 1>(s, fp, p, st);
    return launch_fused_t<64, 6, 1>(s, fp, p, st);
}

}  // namespace tgvkv
