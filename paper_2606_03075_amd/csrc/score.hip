// TWR / TVB scoring, one kernel per phase (gfx950).
//
// The method reads only the rows of the causal softmax A = softmax(tau Q K^T + M)
// (Sec. 3.1, Eq. (2)) whose queries are text tokens.  Those rows are recomputed
// here from the cached keys, because a fused prefill attention kernel does not
// return probabilities.  Two sweeps over K are unavoidable: the text-weighted
// vision scores (Eq. (8)) need each row's final normaliser and the weights w~
// (Eq. (7)), which depend on every head of the layer.
//
//   score_stats   sweep 1: question rows x all visible keys -> row log-sum-exp
//                 and vision mass, online (one K read);
//   score_stats_text  sweep 1 followed by the unit's text pass in the same
//                 workgroup, when one workgroup holds all of a unit's question rows;
//   score_text    text rows x text keys: system-row normalisers, then the
//                 text->text probabilities' column sums per head (Eq. (9));
//   score_fin     head means -> s^T, w, w~ (Eq. (7), (9)) and the layer's
//                 text->vision mass (Eq. (5)-(6));
//   score_vision  sweep 2: question rows x vision keys, p = exp(z - lse),
//                 column sums weighted by w~ (Eq. (8));
//   score_vis_reduce  deterministic sum of the per-(KV head, row group) partials;
//   score_mass    layer TV mass from per-row vision masses, when the caller gives
//                 the rows' normalisers (from its prefill) and sweep 1 is skipped:
//                 the vision sweep then also yields each row's vision mass, so K
//                 is read once.
//
// These kernels serve phase-by-phase calls (and the vision pass restricted to
// layers whose budget reaches past the text).
#include <algorithm>
#include <map>
#include <mutex>
#include <tuple>
#include <type_traits>

#include "score_core.h"

namespace tgvkv {
namespace {

using namespace core;

template <int D, int NSLOT, int KS>
__global__ __launch_bounds__(kThreads) void score_stats_kernel(Shape s, int rowgroups,
                                                               const uint16_t* __restrict__ q_text,
                                                               const uint16_t* __restrict__ k,
                                                               float* __restrict__ lse,
                                                               float* __restrict__ ws_vm) {
    constexpr int RSETS = 4 / KS;
    __shared__ __attribute__((aligned(16))) char tiles[2][Geo<D>::TILE_BYTES];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int rs = wave % RSETS, kp = wave / RSETS;
    int bid = blockIdx.x;
    const int rg = bid % rowgroups;
    bid /= rowgroups;
    const int kvh = bid % s.Hkv;
    const int bl = bid / s.Hkv;
    const int QB = (s.Nq + 15) >> 4;
    const int NB = s.G * QB;
    const int rb0 = rg * RSETS * NSLOT;

    bf16x8 qf[NSLOT][Geo<D>::KSTEPS];
    int qrow[NSLOT];
    load_qrows<D, NSLOT, KS>(s, q_text, bl, kvh, rb0, qf, qrow);
    float m[NSLOT], lsum[NSLOT], vsum[NSLOT];
    const uint16_t* kbase = k + ((size_t)bl * s.Hkv + kvh) * (size_t)s.N * D;
    stats_sweep<D, NSLOT, KS>(s, kbase, 0, s.N, qf, qrow, tiles, m, lsum, vsum);
    if (kp == 0 && lane < 16) {
#pragma unroll
        for (int sl = 0; sl < NSLOT; ++sl) {
            const int rb = slot_block<RSETS>(rb0, rs, sl);
            const int qi = qrow[sl];
            if (rb < NB && qi < s.Nq) {
                const size_t head = (size_t)bl * s.H + kvh * s.G + rb / QB;
                lse[head * s.Nt + s.Ns + qi] = (m[sl] + log2f(lsum[sl])) * kLn2;
                ws_vm[head * s.Nq + qi] = vsum[sl] / lsum[sl];
            }
        }
    }
}

// Sweep 1 and the text pass of one unit in one workgroup, for shapes where one
// workgroup holds all question rows of a (sequence, layer, KV head): the text
// pass is latency-bound, so running it as each unit's sweep ends hides it behind
// the other workgroups' key streams, and the question rows' normalisers go to
// the text pass through LDS.  The row statistics are bit-identical to
// score_stats'; the text pass stages the unit's text keys in the freed tiles
// when they fit (a different summation order of the same column sums).
// Row plans whose statistics+text kernel has text mode 2 (text_pass_qregs): with four row
// slots per wave the sweep sets the kernel's register count, and the pass fits beside it;
// with fewer slots it would cost occupancy, with six it would spill.
template <int NSLOT, int KS>
constexpr bool kQregsText = NSLOT == 4 && KS == 1;

// With four row slots the kernel is held to 168 registers, 3 waves per SIMD: it then spills
// 96 bytes a lane, all outside the sweep's tile loops (at its phase changes and in the text
// pass), and at the 13B stress shape it took 6.84 ms against 7.21-7.25 ms at 2 waves per SIMD.
template <int D, int NSLOT, int KS>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(NSLOT == 4 ? 3 : 1))) void
score_stats_text_kernel(Shape s, const uint16_t* __restrict__ q_text, const uint16_t* __restrict__ k,
                        float* __restrict__ lse, float* __restrict__ ws_vm, float* __restrict__ ws_colsum,
                        float* __restrict__ ws_vmh, int text_mode) {
    constexpr int RSETS = 4 / KS;
    __shared__ __attribute__((aligned(16))) char tiles[2][Geo<D>::TILE_BYTES];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int rs = wave % RSETS, kp = wave / RSETS;
    const int kvh = blockIdx.x % s.Hkv;
    const int bl = blockIdx.x / s.Hkv;
    const int QB = (s.Nq + 15) >> 4;
    const int NB = s.G * QB;
    const size_t head0 = (size_t)bl * s.H + kvh * s.G;

    bf16x8 qf[NSLOT][Geo<D>::KSTEPS];
    int qrow[NSLOT];
    load_qrows<D, NSLOT, KS>(s, q_text, bl, kvh, 0, qf, qrow);
    float m[NSLOT], lsum[NSLOT], vsum[NSLOT];
    const uint16_t* kbase = k + ((size_t)bl * s.Hkv + kvh) * (size_t)s.N * D;
    stats_sweep<D, NSLOT, KS>(s, kbase, 0, s.N, qf, qrow, tiles, m, lsum, vsum);

    // [G][N_t] normalisers (base 2), then [G][N_q] vision masses: in the dynamic LDS area
    // (text mode 2, whose text pass streams keys through the tiles), else in the freed tiles
    extern __shared__ float tarea[];
    float* lse2s = text_mode == 2 ? tarea : reinterpret_cast<float*>(&tiles[0][0]);
    float* vms = lse2s + (size_t)s.G * s.Nt;
    if (kp == 0 && lane < 16) {
#pragma unroll
        for (int sl = 0; sl < NSLOT; ++sl) {
            const int rb = slot_block<RSETS>(0, rs, sl);
            const int qi = qrow[sl];
            if (rb < NB && qi < s.Nq) {
                const int g = rb / QB;
                const float ln = (m[sl] + log2f(lsum[sl])) * kLn2;
                const float vm = vsum[sl] / lsum[sl];
                lse[(head0 + g) * s.Nt + s.Ns + qi] = ln;
                ws_vm[(head0 + g) * s.Nq + qi] = vm;
                lse2s[g * s.Nt + s.Ns + qi] = ln * kLog2e;
                vms[g * s.Nq + qi] = vm;
            }
        }
    }
    __syncthreads();
    // per query head: the sum of its question rows' vision masses (one wave per head)
    for (int g = tid >> 6; g < s.G; g += kThreads / 64) {
        float a = 0.f;
        for (int qi = tid & 63; qi < s.Nq; qi += 64) a += vms[g * s.Nq + qi];
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) a += shfl_xor(a, off);
        if ((tid & 63) == 0) ws_vmh[head0 + g] = a;
    }
    if constexpr (kQregsText<NSLOT, KS>) {
        if (text_mode == 2) {
            // the question rows' fragments are still in registers: only text keys are loaded
            text_pass_qregs<D, NSLOT, KS>(s, bl, kvh, q_text, k, lse, qf, lse2s, vms + (size_t)s.G * s.Nq, tiles,
                                          ws_colsum);
            return;
        }
    }
    if (text_mode == 1) {
        // the unit's text keys go into the freed tiles after the normalisers and masses
        const size_t off = ((size_t)s.G * (s.Nt + s.Nq) * sizeof(float) + 15) & ~(size_t)15;
        text_pass_lds<D>(s, bl, kvh, q_text, k, lse, lse2s, &tiles[0][0] + off,
                         2LL * Geo<D>::TILE_BYTES - (long long)off, ws_colsum);
    } else {
        text_pass<D>(s, bl, kvh, q_text, k, lse, lse2s, ws_colsum);
    }
}

template <int D>
__global__ __launch_bounds__(kThreads) void score_text_kernel(Shape s, const uint16_t* __restrict__ q_text,
                                                              const uint16_t* __restrict__ k,
                                                              float* __restrict__ lse,
                                                              const float* __restrict__ ws_vm,
                                                              float* __restrict__ ws_colsum,
                                                              float* __restrict__ ws_vmh, int lse_given,
                                                              long long kl_bytes) {
    // [G][N_t] row normalisers, base-2 units; with kl_bytes > 0, then the staged text pass's
    // LDS (text_pass_lds), 16-byte aligned
    extern __shared__ float lse2s[];
    const int tid = threadIdx.x;
    const int kvh = blockIdx.x % s.Hkv;
    const int bl = blockIdx.x / s.Hkv;
    const size_t head0 = (size_t)bl * s.H + kvh * s.G;
    if (lse_given) {
        // every text row's normaliser comes from the caller (a prefill kernel's row log-sum-exp)
        for (int x = tid; x < s.G * s.Nt; x += kThreads) lse2s[x] = lse[head0 * s.Nt + x] * kLog2e;
        if (kl_bytes > 0) {
            __syncthreads();
            char* kl = reinterpret_cast<char*>(lse2s) + ((size_t)s.G * s.Nt * sizeof(float) + 15) / 16 * 16;
            text_pass_lds<D>(s, bl, kvh, q_text, k, lse, lse2s, kl, kl_bytes, ws_colsum, true);
            return;
        }
    } else {
        for (int x = tid; x < s.G * s.Nq; x += kThreads) {
            const int g = x / s.Nq, qi = x % s.Nq;
            lse2s[g * s.Nt + s.Ns + qi] = lse[(head0 + g) * s.Nt + s.Ns + qi] * kLog2e;
        }
        if (tid < s.G) {
            float a = 0.f;
            for (int qi = 0; qi < s.Nq; ++qi) a += ws_vm[(head0 + tid) * s.Nq + qi];
            ws_vmh[head0 + tid] = a;
        }
    }
    __syncthreads();
    text_pass<D>(s, bl, kvh, q_text, k, lse, lse2s, ws_colsum, lse_given != 0);
}

// One wave per (unit, query head, 16-key block) of the text->text column sums, when
// every text row's normaliser is given.
template <int D>
__global__ __launch_bounds__(64) void score_text_cols_kernel(Shape s, const uint16_t* __restrict__ q_text,
                                                             const uint16_t* __restrict__ k,
                                                             const float* __restrict__ lse,
                                                             float* __restrict__ ws_colsum) {
    const int TB = (s.Nt + 15) >> 4;
    long long item = blockIdx.x;
    const int kb = (int)(item % TB);
    item /= TB;
    const int g = (int)(item % s.G);
    item /= s.G;
    const int kvh = (int)(item % s.Hkv);
    const int bl = (int)(item / s.Hkv);
    text_cols_item<D>(s, bl, kvh, g, kb, q_text, k, lse, ws_colsum);
}

__global__ __launch_bounds__(kThreads) void score_fin_kernel(Shape s, const float* __restrict__ ws_colsum,
                                                             const float* __restrict__ ws_vmh,
                                                             float* __restrict__ s_txt,
                                                             float* __restrict__ w_txt,
                                                             float* __restrict__ tv_mass, int with_mass) {
    __shared__ float red[kThreads];
    finalize_group(s, (int)(blockIdx.x / s.ngroups), (int)(blockIdx.x % s.ngroups), ws_colsum, ws_vmh, s_txt, w_txt,
                   tv_mass, red, with_mass != 0);
}

// Layer TV mass (Eq. (5)-(6)) from per-row vision masses, in the same order as the
// two-sweep path: per head over question rows, then the mean over heads.
// ws_vm holds one row-mass partial per share of the vision keys ([vsplit][B*L*H][N_q]); a
// row's shares are added first, in share order.
__global__ __launch_bounds__(kThreads) void score_mass_kernel(Shape s, const float* __restrict__ ws_vm,
                                                              float* __restrict__ ws_vmh,
                                                              float* __restrict__ tv_mass, int vsplit) {
    const int bl = blockIdx.x;
    const size_t share = (size_t)s.B * s.L * s.H * s.Nq;
    for (int h = threadIdx.x; h < s.H; h += kThreads) {
        float a = 0.f;
        if (s.Nv > 0) {  // with no vision keys the vision sweep does not run and every mass is 0
            const float* vm = ws_vm + ((size_t)bl * s.H + h) * s.Nq;
            for (int qi = 0; qi < s.Nq; ++qi) {
                float r = vm[qi];
                for (int sp = 1; sp < vsplit; ++sp) r += vm[sp * share + qi];
                a += r;
            }
        }
        ws_vmh[(size_t)bl * s.H + h] = a;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        float a = 0.f;
        if (s.Nt > 0)
            for (int h = 0; h < s.H; ++h) a += ws_vmh[(size_t)bl * s.H + h];
        tv_mass[bl] = a / (float)s.H;
    }
}

// How the vision sweep's workgroups are dealt out: each (unit, row group) has vsplit shares
// of its vision keys; workgroup b < nfull takes share b whole, and the shares after those are
// each cut into `pieces` workgroups.  The cut shares are the last ones dispatched: they would
// otherwise run as a partial last round whose few workgroups, one or two key tiles in flight
// each, cannot keep HBM busy (at llavanext 4096 units over 768 resident workgroups leave 256
// for a sixth round).
struct VisionDeal {
    int vsplit;
    long long nfull;
    int pieces;
};

template <int D, int NSLOT, int KS, bool MASS>
__global__ __launch_bounds__(kThreads) void score_vision_kernel(Shape s, int rowgroups,
                                                                const uint16_t* __restrict__ q_text,
                                                                const uint16_t* __restrict__ k,
                                                                const float* __restrict__ lse,
                                                                const float* __restrict__ w_txt,
                                                                const int32_t* __restrict__ budgets,
                                                                int vis_threshold,
                                                                float* __restrict__ ws_part,
                                                                float* __restrict__ ws_vm, int out_tiles,
                                                                VisionDeal deal) {
    constexpr int RSETS = 4 / KS;
    __shared__ __attribute__((aligned(16))) char tiles[2][Geo<D>::TILE_BYTES];
    __shared__ float red[2][RSETS][kTile];
    extern __shared__ float obuf[];  // out_tiles * kTile scores
    const int vsplit = deal.vsplit;
    long long sh = blockIdx.x;  // this workgroup's share of the vision keys, and its piece of it
    int piece = 0, npieces = 1;
    if (sh >= deal.nfull) {
        const long long j = sh - deal.nfull;
        sh = deal.nfull + j / deal.pieces;
        piece = (int)(j % deal.pieces);
        npieces = deal.pieces;
    }
    const int sp = (int)(sh % vsplit);
    int bid = (int)(sh / vsplit);
    const int rg = bid % rowgroups;
    bid /= rowgroups;
    const int kvh = bid % s.Hkv;
    const int bl = bid / s.Hkv;
    const int QB = (s.Nq + 15) >> 4;
    const int NB = s.G * QB;
    const int rb0 = rg * RSETS * NSLOT;

    // a layer whose budget leaves no room for vision tokens needs no scores: its workgroups
    // leave before loading anything (at the 13B stress shape with i.i.d. text queries every
    // layer is such a layer, and loading the rows first cost 0.27 ms of a launch that computes
    // nothing)
    if (budgets != nullptr && budgets[bl] <= vis_threshold) return;
    bf16x8 qf[NSLOT][Geo<D>::KSTEPS];
    int qrow[NSLOT];
    load_qrows<D, NSLOT, KS, false>(s, q_text, bl, kvh, rb0, qf, qrow);
    float lse2[NSLOT][4], coef[NSLOT][4];
    load_row_coefs<NSLOT, KS, false>(s, bl, kvh, rb0, lse, w_txt, lse2, coef);
    settle_qrows<D, NSLOT>(qf);
#pragma unroll
    for (int sl = 0; sl < NSLOT; ++sl)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            settle(lse2[sl][j]);
            settle(coef[sl][j]);
        }
    const uint16_t* kvis = k + (((size_t)bl * s.Hkv + kvh) * (size_t)s.N + s.Ns) * D;
    float* out = ws_part + (((size_t)bl * s.Hkv + kvh) * rowgroups + rg) * (size_t)s.Nv;
    float rsum[NSLOT][4];
    // every key's score is a sum over this workgroup's rows only, so the keys split freely
    const int ntv = (s.Nv + kTile - 1) / kTile;
    const int per_t = (ntv + vsplit - 1) / vsplit;
    const int t0 = min(sp * per_t, ntv), t1 = min(t0 + per_t, ntv);
    const int per_p = (t1 - t0 + npieces - 1) / npieces;
    const int p0 = min(t0 + piece * per_p, t1), p1 = min(p0 + per_p, t1);
    const int vbeg = min(p0 * kTile, s.Nv), vend = min(p1 * kTile, s.Nv);
    vision_sweep<D, NSLOT, KS, MASS>(s, kvis, vbeg, vend, qf, lse2, coef, rb0, NB, tiles, red, obuf, out_tiles, out,
                                     rsum);
    if (MASS) {
        // each row's vision mass: the sum of its probabilities over all vision keys
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        const int rs = wave % RSETS, kp = wave / RSETS;
        if (kp == 0 && (lane & 15) == 0) {
#pragma unroll
            for (int sl = 0; sl < NSLOT; ++sl) {
                const int rb = slot_block<RSETS>(rb0, rs, sl);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int qj = (rb % QB) * 16 + (lane >> 4) * 4 + j;
                    if (rb < NB && qj < s.Nq)
                        ws_vm[((size_t)sp * s.B * s.L * s.H + (size_t)bl * s.H + kvh * s.G + rb / QB) * s.Nq + qj] =
                            rsum[sl][j];
                }
            }
        }
    }
}

__global__ __launch_bounds__(kThreads) void score_vis_reduce_kernel(Shape s, int rowgroups,
                                                                    const float* __restrict__ ws_part,
                                                                    const int32_t* __restrict__ budgets,
                                                                    int vis_threshold,
                                                                    float* __restrict__ s_vis) {
    const int j = blockIdx.x * kThreads + threadIdx.x;
    const int gi = blockIdx.y % s.ngroups;
    const int bl = blockIdx.y / s.ngroups;
    if (j >= s.Nv) return;
    if (budgets != nullptr && budgets[bl] <= vis_threshold) return;
    const int kv0 = s.head_mode == 0 ? 0 : gi;
    const int kvn = s.head_mode == 0 ? s.Hkv : 1;
    // the partials of (KV head, row group) pairs are consecutive rows of n_vis: eight in flight
    const float* src = ws_part + ((size_t)bl * s.Hkv + kv0) * rowgroups * (size_t)s.Nv + j;
    const int n = kvn * rowgroups;
    float a[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    int i = 0;
    for (; i + 8 <= n; i += 8) {
#pragma unroll
        for (int u = 0; u < 8; ++u) a[u] += src[(size_t)(i + u) * s.Nv];
    }
    for (; i < n; ++i) a[0] += src[(size_t)i * s.Nv];
    s_vis[((size_t)bl * s.ngroups + gi) * s.Nv + j] = ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]));
}

#define TGVKV_ROWPLAN_DISPATCH(KERNEL, D, rp, ...)                                                \
    do {                                                                                          \
        if (rp.ks == 4) hipLaunchKernelGGL((KERNEL<D, 1, 4>), __VA_ARGS__);                       \
        else if (rp.ks == 2 && rp.nslot == 1) hipLaunchKernelGGL((KERNEL<D, 1, 2>), __VA_ARGS__); \
        else if (rp.ks == 2) hipLaunchKernelGGL((KERNEL<D, 2, 2>), __VA_ARGS__);                  \
        else if (rp.nslot == 1) hipLaunchKernelGGL((KERNEL<D, 1, 1>), __VA_ARGS__);               \
        else if (rp.nslot == 2) hipLaunchKernelGGL((KERNEL<D, 2, 1>), __VA_ARGS__);               \
        else if (rp.nslot == 4) hipLaunchKernelGGL((KERNEL<D, 4, 1>), __VA_ARGS__);               \
        else hipLaunchKernelGGL((KERNEL<D, 6, 1>), __VA_ARGS__);                                  \
    } while (0)

#define TGVKV_ROWPLAN_DISPATCH_M(KERNEL, D, M, rp, ...)                                                   \
    do {                                                                                                  \
        if (rp.ks == 4) hipLaunchKernelGGL((KERNEL<D, 1, 4, M>), __VA_ARGS__);                            \
        else if (rp.ks == 2 && rp.nslot == 1) hipLaunchKernelGGL((KERNEL<D, 1, 2, M>), __VA_ARGS__);      \
        else if (rp.ks == 2) hipLaunchKernelGGL((KERNEL<D, 2, 2, M>), __VA_ARGS__);                       \
        else if (rp.nslot == 1) hipLaunchKernelGGL((KERNEL<D, 1, 1, M>), __VA_ARGS__);                    \
        else if (rp.nslot == 2) hipLaunchKernelGGL((KERNEL<D, 2, 1, M>), __VA_ARGS__);                    \
        else if (rp.nslot == 4) hipLaunchKernelGGL((KERNEL<D, 4, 1, M>), __VA_ARGS__);                    \
        else hipLaunchKernelGGL((KERNEL<D, 6, 1, M>), __VA_ARGS__);                                       \
    } while (0)

template <int N>
using IC = std::integral_constant<int, N>;

// Calls f(IC<D>, IC<NSLOT>, IC<KS>, IC<MASS>) for the score_vision_kernel variant that
// launch_score_vision runs for row plan rp (NB row blocks per unit).
template <typename F>
void with_vision_variant(int d, bool mass, const RowPlan& rp, int NB, F&& f) {
    auto plan = [&](auto dd, auto m) {
        if (!decltype(m)::value && rp.nslot == 1 && rp.ks == 1) {
            if (NB == 3) f(dd, IC<2>{}, IC<2>{}, m);
            else if constexpr (!decltype(m)::value) f(dd, IC<4>{}, IC<4>{}, m);
        } else if (rp.ks == 4) f(dd, IC<1>{}, IC<4>{}, m);
        else if (rp.ks == 2 && rp.nslot == 1) f(dd, IC<1>{}, IC<2>{}, m);
        else if (rp.ks == 2) f(dd, IC<2>{}, IC<2>{}, m);
        else if (rp.nslot == 1) f(dd, IC<1>{}, IC<1>{}, m);
        else if (rp.nslot == 2) f(dd, IC<2>{}, IC<1>{}, m);
        else if (rp.nslot == 4) f(dd, IC<4>{}, IC<1>{}, m);
        else f(dd, IC<6>{}, IC<1>{}, m);
    };
    auto with_d = [&](auto m) {
        if (d == 128) plan(IC<128>{}, m);
        else plan(IC<64>{}, m);
    };
    if (mass) with_d(IC<1>{});
    else with_d(IC<0>{});
}

// Workgroups of `kernel` that the current device holds at once (its occupancy per CU times
// the CU count), asked of the runtime once per device and kernel; 0 if it cannot tell.
int resident_workgroups(const void* kernel, size_t dyn_lds) {
    static std::mutex mu;
    static std::map<std::tuple<int, const void*, size_t>, int> known;
    int dev = 0;
    if (kernel == nullptr || hipGetDevice(&dev) != hipSuccess) return 0;
    const auto key = std::make_tuple(dev, kernel, dyn_lds);
    std::lock_guard<std::mutex> lock(mu);
    const auto it = known.find(key);
    if (it != known.end()) return it->second;
    int cus = 0, per_cu = 0, n = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kThreads, dyn_lds) == hipSuccess)
        n = cus * per_cu;
    else
        (void)hipGetLastError();
    known[key] = n;
    return n;
}

}  // namespace

RowPlan plan_question_rows(const Shape& s) {
    const int QB = (s.Nq + 15) / 16;
    const int NB = s.G * QB;
    RowPlan rp;
    if (NB <= 1) { rp.nslot = 1; rp.ks = 4; }
    else if (NB == 2) { rp.nslot = 1; rp.ks = 2; }
    else if (NB == 3) { rp.nslot = 1; rp.ks = 1; }  // the vision sweep runs these as (2, 2)
    else if (NB <= 4) { rp.nslot = 1; rp.ks = 1; }
    else if (NB <= 8) { rp.nslot = 2; rp.ks = 1; }
    else if (NB <= 16) { rp.nslot = 4; rp.ks = 1; }
    else { rp.nslot = 6; rp.ks = 1; }
    const int per_group = (4 / rp.ks) * rp.nslot;
    rp.rowgroups = NB > 0 ? (NB + per_group - 1) / per_group : 0;
    return rp;
}

hipError_t launch_score_stats(const Shape& s, const RowPlan& rp, const uint16_t* q_text, const uint16_t* k,
                              float* lse, float* ws_vm, hipStream_t st) {
    const long long nblk = (long long)s.B * s.L * s.Hkv * rp.rowgroups;
    if (nblk == 0) return hipSuccess;
    dim3 grid((unsigned)nblk), block(kThreads);
    if (s.D == 128)
        TGVKV_ROWPLAN_DISPATCH(score_stats_kernel, 128, rp, grid, block, 0, st, s, rp.rowgroups, q_text, k, lse, ws_vm);
    else
        TGVKV_ROWPLAN_DISPATCH(score_stats_kernel, 64, rp, grid, block, 0, st, s, rp.rowgroups, q_text, k, lse, ws_vm);
    return hipGetLastError();
}

bool stats_text_eligible(const Shape& s, const RowPlan& rp) {
    if (rp.rowgroups != 1 || s.Nt == 0) return false;
    const long long floats = (long long)s.G * (s.Nt + s.Nq);
    const long long tile_bytes = 2LL * kTile * (2 * s.D + 16);
    return floats * 4 <= tile_bytes;
}

hipError_t launch_score_stats_text(const Shape& s, const RowPlan& rp, const uint16_t* q_text, const uint16_t* k,
                                   float* lse, float* ws_vm, float* ws_colsum, float* ws_vmh, hipStream_t st) {
    const long long nblk = (long long)s.B * s.L * s.Hkv;
    if (nblk == 0) return hipSuccess;
    dim3 grid((unsigned)nblk), block(kThreads);
    // Text mode 2 (the question rows' fragments reused from the sweep, the system keys staged
    // in the tiles, the question keys streamed through them) needs the normalisers, masses and
    // column partials in a dynamic LDS area that leaves the kernel's occupancy as it is.
    // Otherwise mode 1 stages the unit's text keys (in chunks of key blocks, if need be) in
    // the freed key tiles, after the normalisers and masses, when its partials and the system
    // keys' blocks fit there; else mode 0 reads them from memory.
    const long long tile_bytes = 2LL * kTile * (2 * s.D + 16);
    const long long area = text_area_floats(s.G, s.Nt, s.Nq) * (long long)sizeof(float);
    const int occupancy = rp.nslot == 1 ? 4 : rp.nslot == 2 ? 3 : rp.nslot == 4 ? 3 : 2;
    const bool qregs = rp.nslot == 4 && rp.ks == 1 && s.Ns <= 2 * kTile && area <= 163840 / occupancy - tile_bytes;
    const long long head = ((long long)s.G * (s.Nt + s.Nq) * 4 + 15) / 16 * 16;
    const size_t dyn = qregs ? (size_t)area : 0;
    if (s.D == 128) {
        const int mode = qregs ? 2 : text_lds_fits<128>(s.G, s.Ns, s.Nt, tile_bytes - head) ? 1 : 0;
        TGVKV_ROWPLAN_DISPATCH(score_stats_text_kernel, 128, rp, grid, block, dyn, st, s, q_text, k, lse, ws_vm,
                               ws_colsum, ws_vmh, mode);
    } else {
        const int mode = qregs ? 2 : text_lds_fits<64>(s.G, s.Ns, s.Nt, tile_bytes - head) ? 1 : 0;
        TGVKV_ROWPLAN_DISPATCH(score_stats_text_kernel, 64, rp, grid, block, dyn, st, s, q_text, k, lse, ws_vm,
                               ws_colsum, ws_vmh, mode);
    }
    return hipGetLastError();
}

hipError_t launch_score_text(const Shape& s, const uint16_t* q_text, const uint16_t* k, float* lse,
                             const float* ws_vm, float* ws_colsum, float* ws_vmh, bool lse_given, hipStream_t st) {
    const long long nblk = (long long)s.B * s.L * s.Hkv;
    if (nblk == 0 || s.Nt == 0) return hipSuccess;
    if (lse_given) {
        // the unit's text keys staged in LDS by one workgroup per unit (text_pass_lds; in
        // chunks of key blocks when they do not all fit beside the normalisers within 64 KB):
        // against one wave per (unit, head, 16-key block) walking the row blocks from global
        // memory, at llavanext 80 -> 20 us
        const int TB = (s.Nt + 15) / 16;
        const long long head = ((long long)s.G * s.Nt * 4 + 15) / 16 * 16;
        const long long kl = std::min<long long>(
            (s.D == 128 ? text_part_bytes<128>(s.G, s.Nt) : text_part_bytes<64>(s.G, s.Nt)) +
                16LL * TB * (2 * s.D + 16),
            65536 - head);
        const bool fits = s.D == 128 ? text_lds_fits<128>(s.G, 0, s.Nt, kl) : text_lds_fits<64>(s.G, 0, s.Nt, kl);
        if (s.Nt > 0 && kl > 0 && fits) {
            const size_t lds = (size_t)(head + kl);
            if (s.D == 128)
                hipLaunchKernelGGL(score_text_kernel<128>, dim3((unsigned)nblk), dim3(kThreads), lds, st, s, q_text,
                                   k, lse, ws_vm, ws_colsum, ws_vmh, 1, kl);
            else
                hipLaunchKernelGGL(score_text_kernel<64>, dim3((unsigned)nblk), dim3(kThreads), lds, st, s, q_text,
                                   k, lse, ws_vm, ws_colsum, ws_vmh, 1, kl);
            return hipGetLastError();
        }
        const long long items = nblk * s.G * ((s.Nt + 15) / 16);
        if (s.D == 128)
            hipLaunchKernelGGL(score_text_cols_kernel<128>, dim3((unsigned)items), dim3(64), 0, st, s, q_text, k, lse,
                               ws_colsum);
        else
            hipLaunchKernelGGL(score_text_cols_kernel<64>, dim3((unsigned)items), dim3(64), 0, st, s, q_text, k, lse,
                               ws_colsum);
        return hipGetLastError();
    }
    dim3 grid((unsigned)nblk), block(kThreads);
    const size_t lds = sizeof(float) * (size_t)s.G * s.Nt;
    if (s.D == 128)
        hipLaunchKernelGGL(score_text_kernel<128>, grid, block, lds, st, s, q_text, k, lse, ws_vm, ws_colsum, ws_vmh,
                           (int)lse_given, 0LL);
    else
        hipLaunchKernelGGL(score_text_kernel<64>, grid, block, lds, st, s, q_text, k, lse, ws_vm, ws_colsum, ws_vmh,
                           (int)lse_given, 0LL);
    return hipGetLastError();
}

hipError_t launch_score_fin(const Shape& s, const float* ws_colsum, const float* ws_vmh, float* s_txt,
                            float* w_txt, float* tv_mass, bool with_mass, hipStream_t st) {
    const long long nblk = (long long)s.B * s.L * s.ngroups;
    if (nblk == 0) return hipSuccess;
    hipLaunchKernelGGL(score_fin_kernel, dim3((unsigned)nblk), dim3(kThreads), 0, st, s, ws_colsum, ws_vmh,
                       s_txt, w_txt, tv_mass, (int)with_mass);
    return hipGetLastError();
}

int vision_splits(const Shape& s, const RowPlan& rp) {
    // With few (unit, row group) workgroups the vision keys are split over several: at the
    // Qwen2-VL shape (896 units, 2 workgroups per CU) two splits balance the last round
    // (805 -> 740 us); at 4096 units a split only adds prologues.  The mass-collecting variant
    // writes one row-mass partial per share, which score_mass adds.
    const long long units = (long long)s.B * s.L * s.Hkv * rp.rowgroups;
    return units <= 0 ? 1 : (int)std::min<long long>(std::max<long long>(2048 / units, 1), 4);
}

hipError_t launch_score_vision(const Shape& s, const RowPlan& rp, const uint16_t* q_text, const uint16_t* k,
                               const float* lse, const float* w_txt, const int32_t* budgets,
                               int32_t vis_threshold, float* ws_part, float* ws_vm, hipStream_t st) {
    const bool mass = ws_vm != nullptr;
    const long long units = (long long)s.B * s.L * s.Hkv * rp.rowgroups;
    const int vsplit = vision_splits(s, rp);
    const long long nsh = units * vsplit;
    if (nsh == 0 || s.Nv == 0) return hipSuccess;
    // a unit's scores are kept in LDS and written once at the end when they fit (no global
    // store among the key loads); otherwise in bursts of kOutTiles tiles
    const int ntiles = ((s.Nv + kTile - 1) / kTile + vsplit - 1) / vsplit;
    const int out_tiles = (!mass && ntiles * kTile * (int)sizeof(float) <= kWholeOutBytes) ? ntiles : kOutTiles;
    const size_t obytes = (size_t)out_tiles * kTile * sizeof(float);
    // the kernel variant this plan runs, and how many of its workgroups the GPU holds at once
    const int NB = s.G * ((s.Nq + 15) / 16);
    const void* fn = nullptr;
    with_vision_variant(s.D, mass, rp, NB, [&](auto d, auto ns, auto kss, auto m) {
        fn = (const void*)&score_vision_kernel<decltype(d)::value, decltype(ns)::value, decltype(kss)::value,
                                               decltype(m)::value != 0>;
    });
    // the shares that would make a partial last round are cut into pieces that fill it (each
    // piece at least 4 key tiles); the mass-collecting sweep keeps one row-mass partial per share
    VisionDeal deal{vsplit, nsh, 1};
    const int slots = mass ? 0 : resident_workgroups(fn, obytes);
    if (slots > 0 && nsh % slots != 0) {
        const long long r = nsh % slots;
        const int most = std::max(ntiles / 4, 1);
        const int pieces = (int)std::min<long long>((slots + r - 1) / r, most);
        if (pieces > 1) deal = VisionDeal{vsplit, nsh - r, pieces};
    }
    const long long nblk = deal.nfull + (nsh - deal.nfull) * deal.pieces;
    dim3 grid((unsigned)nblk), block(kThreads);
    if (mass) {
        if (s.D == 128) TGVKV_ROWPLAN_DISPATCH_M(score_vision_kernel, 128, true, rp, grid, block, obytes, st, s, rp.rowgroups, q_text, k, lse, w_txt, budgets, vis_threshold, ws_part, ws_vm, out_tiles, deal);
        else TGVKV_ROWPLAN_DISPATCH_M(score_vision_kernel, 64, true, rp, grid, block, obytes, st, s, rp.rowgroups, q_text, k, lse, w_txt, budgets, vis_threshold, ws_part, ws_vm, out_tiles, deal);
    } else if (rp.nslot == 1 && rp.ks == 1 && (s.G * ((s.Nq + 15) / 16)) == 3) {
        // three 16-row blocks per unit: two slots over half of each key tile (same row groups);
        // at the LLaVA-1.5 shape 43 us against 46-48 us for the four-slot shape below
        const RowPlan r2{2, 2, rp.rowgroups};
        if (s.D == 128)
            TGVKV_ROWPLAN_DISPATCH_M(score_vision_kernel, 128, false, r2, grid, block, obytes, st, s, rp.rowgroups, q_text, k, lse, w_txt, budgets, vis_threshold, ws_part, ws_vm, out_tiles, deal);
        else
            TGVKV_ROWPLAN_DISPATCH_M(score_vision_kernel, 64, false, r2, grid, block, obytes, st, s, rp.rowgroups, q_text, k, lse, w_txt, budgets, vis_threshold, ws_part, ws_vm, out_tiles, deal);
    } else if (rp.nslot == 1 && rp.ks == 1) {
        // four 16-row blocks per unit: the vision sweep runs faster with every wave holding all
        // four blocks over a quarter of each key tile (same row groups, so the same partials)
        if (s.D == 128)
            hipLaunchKernelGGL((score_vision_kernel<128, 4, 4, false>), grid, block, obytes, st, s, rp.rowgroups,
                               q_text, k, lse, w_txt, budgets, vis_threshold, ws_part, ws_vm, out_tiles, deal);
        else
            hipLaunchKernelGGL((score_vision_kernel<64, 4, 4, false>), grid, block, obytes, st, s, rp.rowgroups,
                               q_text, k, lse, w_txt, budgets, vis_threshold, ws_part, ws_vm, out_tiles, deal);
    } else {
        if (s.D == 128) TGVKV_ROWPLAN_DISPATCH_M(score_vision_kernel, 128, false, rp, grid, block, obytes, st, s, rp.rowgroups, q_text, k, lse, w_txt, budgets, vis_threshold, ws_part, ws_vm, out_tiles, deal);
        else TGVKV_ROWPLAN_DISPATCH_M(score_vision_kernel, 64, false, rp, grid, block, obytes, st, s, rp.rowgroups, q_text, k, lse, w_txt, budgets, vis_threshold, ws_part, ws_vm, out_tiles, deal);
    }
    return hipGetLastError();
}

hipError_t launch_score_mass(const Shape& s, const RowPlan& rp, const float* ws_vm, float* ws_vmh, float* tv_mass,
                             hipStream_t st) {
    const long long nblk = (long long)s.B * s.L;
    if (nblk == 0) return hipSuccess;
    hipLaunchKernelGGL(score_mass_kernel, dim3((unsigned)nblk), dim3(kThreads), 0, st, s, ws_vm, ws_vmh, tv_mass,
                       vision_splits(s, rp));
    return hipGetLastError();
}

hipError_t launch_score_vis_reduce(const Shape& s, const RowPlan& rp, const float* ws_part, const int32_t* budgets,
                                   int32_t vis_threshold, float* s_vis, hipStream_t st) {
    const long long ny = (long long)s.B * s.L * s.ngroups;
    if (ny == 0 || s.Nv == 0) return hipSuccess;
    // With no question rows there are no partials (rowgroups == 0) and every score is zero.
    dim3 grid((s.Nv + kThreads - 1) / kThreads, (unsigned)ny);
    hipLaunchKernelGGL(score_vis_reduce_kernel, grid, dim3(kThreads), 0, st, s, rp.rowgroups, ws_part, budgets,
                       vis_threshold, s_vis);
    return hipGetLastError();
}

}  // namespace tgvkv
