// TWR / TVB scoring kernels (gfx950).
//
// The method reads only the rows of the causal softmax A = softmax(tau Q K^T + M)
// (Sec. 3.1, Eq. (2)) whose queries are text tokens.  Those rows are recomputed
// here from the cached keys, because a fused prefill attention kernel does not
// return probabilities.  Two sweeps over K are unavoidable: the text-weighted
// vision scores (Eq. (8)) need each row's final normaliser and the weights w~
// (Eq. (7)), which depend on every head of the layer.
//
//   score_stats   sweep 1 (the hot loop): question rows x all visible keys ->
//                 row log-sum-exp and vision mass, online (one K read);
//   score_text    text rows x text keys: system-row normalisers, then the
//                 text->text probabilities' column sums per head (Eq. (9));
//   score_fin     head means -> s^T, w, w~ (Eq. (7), (9)) and the layer's
//                 text->vision mass (Eq. (5)-(6));
//   score_vision  sweep 2: question rows x vision keys, p = exp(z - lse),
//                 column sums weighted by w~ (Eq. (8));
//   score_vis_reduce  deterministic sum of the per-(KV head, row group) partials.
//
// MFMA layout: v_mfma_f32_16x16x32_bf16.  A 16-key block of K sits in LDS
// (rows padded by 16 bytes so the 16 lanes reading one column chunk hit
// distinct banks); the question rows of one 16-row block stay in registers for
// the whole sweep.  Sweep 1 computes C[key][row] (keys on the M side) so that
// each lane owns one row and keeps its own running max / sum with no
// cross-lane traffic in the loop; sweep 2 computes C[row][key] so that each
// lane owns one key and sums its column in registers.
#include "tgvkv_device.h"
#include "tgvkv_shape.h"

namespace tgvkv {
namespace {

constexpr int kThreads = 256;
constexpr int kTile = 64;  // keys per LDS tile

template <int D>
struct Geo {
    static constexpr int KSTEPS = D / 32;                  // MFMA k-steps over the head dim
    static constexpr int CPR = D / 8;                      // 16-byte chunks per key row
    static constexpr int ROWB = D * 2 + 16;                // padded LDS row, bytes
    static constexpr int TILE_BYTES = kTile * ROWB;
    static constexpr int LOADS = kTile * CPR / kThreads;   // 16-byte loads per thread per tile
};

template <int D>
__device__ __forceinline__ void load_tile_regs(u32x4 (&r)[Geo<D>::LOADS], const uint16_t* kbase,
                                               int key0, int key_last, int tid) {
#pragma unroll
    for (int it = 0; it < Geo<D>::LOADS; ++it) {
        const int c = it * kThreads + tid;
        const int row = c / Geo<D>::CPR, cc = c % Geo<D>::CPR;
        const int key = min(key0 + row, key_last);
        r[it] = load16(kbase + (size_t)key * D + cc * 8);
    }
}

template <int D>
__device__ __forceinline__ void store_tile_lds(char* buf, const u32x4 (&r)[Geo<D>::LOADS], int tid) {
#pragma unroll
    for (int it = 0; it < Geo<D>::LOADS; ++it) {
        const int c = it * kThreads + tid;
        const int row = c / Geo<D>::CPR, cc = c % Geo<D>::CPR;
        store16(buf + row * Geo<D>::ROWB + cc * 16, r[it]);
    }
}

__device__ __forceinline__ bf16x8 zero_frag() {
    u32x4 z = {0u, 0u, 0u, 0u};
    return as_bf16x8(z);
}

// ---------------------------------------------------------------------------------- sweep 1
template <int D, int NSLOT, int KS>
__global__ __launch_bounds__(kThreads) void score_stats_kernel(Shape s, int rowgroups,
                                                               const uint16_t* __restrict__ q_text,
                                                               const uint16_t* __restrict__ k,
                                                               float* __restrict__ lse,
                                                               float* __restrict__ ws_vm) {
    using GG = Geo<D>;
    constexpr int RSETS = 4 / KS;   // row sets (waves sharing a key part)
    constexpr int KBW = 4 / KS;     // 16-key blocks per wave per tile
    __shared__ __attribute__((aligned(16))) char tiles[2][GG::TILE_BYTES];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int rs = wave % RSETS, kp = wave / RSETS;
    int bid = blockIdx.x;
    const int rg = bid % rowgroups;
    bid /= rowgroups;
    const int kvh = bid % s.Hkv;
    const int bl = bid / s.Hkv;

    const int QB = (s.Nq + 15) >> 4;
    const int NB = s.G * QB;
    const int rb0 = rg * RSETS * NSLOT;

    bf16x8 qf[NSLOT][GG::KSTEPS];
    float m[NSLOT], lsum[NSLOT], vsum[NSLOT];
    int qrow[NSLOT];
#pragma unroll
    for (int sl = 0; sl < NSLOT; ++sl) {
        const int rb = rb0 + rs + sl * RSETS;
        const int g = rb / QB;
        const int qi = (rb % QB) * 16 + (lane & 15);
        qrow[sl] = qi;
        m[sl] = kNegInf;
        lsum[sl] = 0.f;
        vsum[sl] = 0.f;
        const bool valid = rb < NB && qi < s.Nq;
        const uint16_t* qp = q_text + (((size_t)bl * s.H + kvh * s.G + (valid ? g : 0)) * s.Nt + s.Ns +
                                       (valid ? qi : 0)) * D + (lane >> 4) * 8;
#pragma unroll
        for (int ks = 0; ks < GG::KSTEPS; ++ks) qf[sl][ks] = valid ? as_bf16x8(load16(qp + ks * 32)) : zero_frag();
    }

    const uint16_t* kbase = k + ((size_t)bl * s.Hkv + kvh) * (size_t)s.N * D;
    const int ntiles = (s.N + kTile - 1) / kTile;
    const int vis0 = s.Ns, vis1 = s.Ns + s.Nv;

    u32x4 pre[GG::LOADS];
    load_tile_regs<D>(pre, kbase, 0, s.N - 1, tid);
    store_tile_lds<D>(tiles[0], pre, tid);
    __syncthreads();

    for (int t = 0; t < ntiles; ++t) {
        const char* buf = tiles[t & 1];
        if (t + 1 < ntiles) load_tile_regs<D>(pre, kbase, (t + 1) * kTile, s.N - 1, tid);
        const int key0 = t * kTile;
        const bool pure_vis = key0 >= vis0 && key0 + kTile <= vis1;
#pragma unroll
        for (int kbi = 0; kbi < KBW; ++kbi) {
            const int kb = kp + kbi * KS;
            bf16x8 kf[GG::KSTEPS];
            const char* src = buf + (kb * 16 + (lane & 15)) * GG::ROWB + (lane >> 4) * 16;
#pragma unroll
            for (int ks = 0; ks < GG::KSTEPS; ++ks) kf[ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(src + ks * 64));
            const int kfirst = key0 + kb * 16 + (lane >> 4) * 4;  // key of accumulator element 0
#pragma unroll
            for (int sl = 0; sl < NSLOT; ++sl) {
                if (rb0 + rs + sl * RSETS >= NB) continue;
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < GG::KSTEPS; ++ks) acc = mfma16x16x32(kf[ks], qf[sl][ks], acc);
                if (pure_vis) {
                    const float z0 = acc[0] * s.scale2, z1 = acc[1] * s.scale2;
                    const float z2 = acc[2] * s.scale2, z3 = acc[3] * s.scale2;
                    const float mx = fmaxf(fmaxf(z0, z1), fmaxf(z2, z3));
                    if (mx > m[sl]) {
                        const float sc = fast_exp2(m[sl] - mx);
                        lsum[sl] *= sc;
                        vsum[sl] *= sc;
                        m[sl] = mx;
                    }
                    const float e = (fast_exp2(z0 - m[sl]) + fast_exp2(z1 - m[sl])) +
                                    (fast_exp2(z2 - m[sl]) + fast_exp2(z3 - m[sl]));
                    lsum[sl] += e;
                    vsum[sl] += e;
                } else {
                    float z[4];
                    bool ok[4], isv[4];
                    float mx = kNegInf;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int key = kfirst + j;
                        ok[j] = key < s.N && (key < vis1 || key - vis1 <= qrow[sl]);
                        isv[j] = key >= vis0 && key < vis1;
                        z[j] = ok[j] ? acc[j] * s.scale2 : kNegInf;
                        mx = fmaxf(mx, z[j]);
                    }
                    if (mx > m[sl]) {
                        const float sc = fast_exp2(m[sl] - mx);
                        lsum[sl] *= sc;
                        vsum[sl] *= sc;
                        m[sl] = mx;
                    }
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        if (ok[j]) {
                            const float e = fast_exp2(z[j] - m[sl]);
                            lsum[sl] += e;
                            if (isv[j]) vsum[sl] += e;
                        }
                    }
                }
            }
        }
        if (t + 1 < ntiles) store_tile_lds<D>(tiles[(t + 1) & 1], pre, tid);
        __syncthreads();
    }

    // The four lane quarters of a wave saw different keys of the same rows.
#pragma unroll
    for (int sl = 0; sl < NSLOT; ++sl) {
#pragma unroll
        for (int off = 16; off < 64; off <<= 1) {
            const float m2 = shfl_xor(m[sl], off), l2 = shfl_xor(lsum[sl], off), v2 = shfl_xor(vsum[sl], off);
            merge_stats(m[sl], lsum[sl], vsum[sl], m2, l2, v2);
        }
    }
    if (KS > 1) {
        // waves of other key parts hand their partials to the key-part-0 wave of their row set
        float* red = reinterpret_cast<float*>(tiles[0]);  // [wave][NSLOT][16][3]
        if (kp > 0 && lane < 16) {
#pragma unroll
            for (int sl = 0; sl < NSLOT; ++sl) {
                float* r = red + ((wave * NSLOT + sl) * 16 + lane) * 3;
                r[0] = m[sl];
                r[1] = lsum[sl];
                r[2] = vsum[sl];
            }
        }
        __syncthreads();
        if (kp == 0 && lane < 16) {
            for (int p = 1; p < KS; ++p) {
                const int w2 = p * RSETS + rs;
#pragma unroll
                for (int sl = 0; sl < NSLOT; ++sl) {
                    const float* r = red + ((w2 * NSLOT + sl) * 16 + lane) * 3;
                    merge_stats(m[sl], lsum[sl], vsum[sl], r[0], r[1], r[2]);
                }
            }
        }
    }
    if (kp == 0 && lane < 16) {
#pragma unroll
        for (int sl = 0; sl < NSLOT; ++sl) {
            const int rb = rb0 + rs + sl * RSETS;
            const int qi = qrow[sl];
            if (rb < NB && qi < s.Nq) {
                const size_t head = (size_t)bl * s.H + kvh * s.G + rb / QB;
                lse[head * s.Nt + s.Ns + qi] = (m[sl] + log2f(lsum[sl])) * kLn2;
                ws_vm[head * s.Nq + qi] = vsum[sl] / lsum[sl];
            }
        }
    }
}

// ---------------------------------------------------------------------------------- text x text
template <int D>
__global__ __launch_bounds__(kThreads) void score_text_kernel(Shape s, const uint16_t* __restrict__ q_text,
                                                              const uint16_t* __restrict__ k,
                                                              float* __restrict__ lse,
                                                              const float* __restrict__ ws_vm,
                                                              float* __restrict__ ws_colsum,
                                                              float* __restrict__ ws_vmh) {
    using GG = Geo<D>;
    extern __shared__ float lse2s[];  // [G][N_t] row normalisers, base-2 units
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int kvh = blockIdx.x % s.Hkv;
    const int bl = blockIdx.x / s.Hkv;
    const size_t head0 = (size_t)bl * s.H + kvh * s.G;
    const uint16_t* kbase = k + ((size_t)bl * s.Hkv + kvh) * (size_t)s.N * D;
    const int koff = (lane >> 4) * 8;

    for (int x = tid; x < s.G * s.Nq; x += kThreads) {
        const int g = x / s.Nq, qi = x % s.Nq;
        lse2s[g * s.Nt + s.Ns + qi] = lse[(head0 + g) * s.Nt + s.Ns + qi] * kLog2e;
    }
    if (tid < s.G) {
        float a = 0.f;
        for (int qi = 0; qi < s.Nq; ++qi) a += ws_vm[(head0 + tid) * s.Nq + qi];
        ws_vmh[head0 + tid] = a;
    }

    // System rows see only system keys (causal): their normalisers come from this small block.
    const int SB = (s.Ns + 15) >> 4;
    for (int item = wave; item < s.G * SB; item += 4) {
        const int g = item / SB, rb = item % SB;
        const int i = rb * 16 + (lane & 15);
        const bool rv = i < s.Ns;
        bf16x8 qf[GG::KSTEPS];
        const uint16_t* qp = q_text + ((head0 + g) * s.Nt + (rv ? i : 0)) * D + koff;
#pragma unroll
        for (int ks = 0; ks < GG::KSTEPS; ++ks) qf[ks] = rv ? as_bf16x8(load16(qp + ks * 32)) : zero_frag();
        float m = kNegInf, l = 0.f, dummy = 0.f;
        for (int kb = 0; kb <= rb; ++kb) {
            const int jc = min(kb * 16 + (lane & 15), s.Ns - 1);
            bf16x8 kf[GG::KSTEPS];
#pragma unroll
            for (int ks = 0; ks < GG::KSTEPS; ++ks) kf[ks] = as_bf16x8(load16(kbase + (size_t)jc * D + koff + ks * 32));
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < GG::KSTEPS; ++ks) acc = mfma16x16x32(kf[ks], qf[ks], acc);
            float z[4];
            float mx = kNegInf;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int key = kb * 16 + (lane >> 4) * 4 + j;
                z[j] = (key <= i && key < s.Ns) ? acc[j] * s.scale2 : kNegInf;
                mx = fmaxf(mx, z[j]);
            }
            if (mx > m) {
                l *= fast_exp2(m - mx);
                m = mx;
            }
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (z[j] != kNegInf) l += fast_exp2(z[j] - m);
        }
#pragma unroll
        for (int off = 16; off < 64; off <<= 1) {
            const float m2 = shfl_xor(m, off), l2 = shfl_xor(l, off), d2 = shfl_xor(dummy, off);
            merge_stats(m, l, dummy, m2, l2, d2);
        }
        if (lane < 16 && rv) {
            const float L2 = m + log2f(l);
            lse2s[g * s.Nt + i] = L2;
            lse[(head0 + g) * s.Nt + i] = L2 * kLn2;
        }
    }
    __syncthreads();

    // Column sums of the text->text probabilities, per head: s^T before the head mean.
    const int TB = (s.Nt + 15) >> 4;
    for (int item = wave; item < s.G * TB; item += 4) {
        const int g = item / TB, kb = item % TB;
        const int j = kb * 16 + (lane & 15);
        const int jc = min(j, s.Nt - 1);
        const int pos = jc < s.Ns ? jc : jc + s.Nv;
        bf16x8 kf[GG::KSTEPS];
#pragma unroll
        for (int ks = 0; ks < GG::KSTEPS; ++ks) kf[ks] = as_bf16x8(load16(kbase + (size_t)pos * D + koff + ks * 32));
        float col = 0.f;
        for (int rb = kb; rb < TB; ++rb) {
            const int i = rb * 16 + (lane & 15);
            const bool rv = i < s.Nt;
            bf16x8 qf[GG::KSTEPS];
            const uint16_t* qp = q_text + ((head0 + g) * s.Nt + (rv ? i : 0)) * D + koff;
#pragma unroll
            for (int ks = 0; ks < GG::KSTEPS; ++ks) qf[ks] = rv ? as_bf16x8(load16(qp + ks * 32)) : zero_frag();
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < GG::KSTEPS; ++ks) acc = mfma16x16x32(qf[ks], kf[ks], acc);
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const int ii = rb * 16 + (lane >> 4) * 4 + jj;
                if (ii < s.Nt && j <= ii) col += fast_exp2(acc[jj] * s.scale2 - lse2s[g * s.Nt + ii]);
            }
        }
        col += shfl_xor(col, 16);
        col += shfl_xor(col, 32);
        if (lane < 16 && j < s.Nt) ws_colsum[(head0 + g) * s.Nt + j] = col;
    }
}

// ---------------------------------------------------------------------------------- finalize
__global__ __launch_bounds__(kThreads) void score_fin_kernel(Shape s, const float* __restrict__ ws_colsum,
                                                             const float* __restrict__ ws_vmh,
                                                             float* __restrict__ s_txt,
                                                             float* __restrict__ w_txt,
                                                             float* __restrict__ tv_mass) {
    __shared__ float red[kThreads];
    const int tid = threadIdx.x;
    const int gi = blockIdx.x % s.ngroups;
    const int bl = blockIdx.x / s.ngroups;
    const int h0 = s.head_mode == 0 ? 0 : gi * s.G;
    const int hn = s.head_mode == 0 ? s.H : s.G;
    const float inv = 1.0f / (float)hn;
    const float* cs = ws_colsum + ((size_t)bl * s.H + h0) * s.Nt;
    const size_t obase = ((size_t)bl * s.ngroups + gi) * s.Nt;

    float part = 0.f;
    for (int j = tid; j < s.Nt; j += kThreads) {
        float a = 0.f;
        for (int h = 0; h < hn; ++h) a += cs[(size_t)h * s.Nt + j];
        const float st = a * inv;
        s_txt[obase + j] = st;
        part += st / (float)(s.Nt - j);
    }
    red[tid] = part;
    __syncthreads();
    for (int o = kThreads / 2; o > 0; o >>= 1) {
        if (tid < o) red[tid] += red[tid + o];
        __syncthreads();
    }
    const float W = red[0];
    for (int j = tid; j < s.Nt; j += kThreads) {
        const float w = s_txt[obase + j] / (float)(s.Nt - j);
        w_txt[obase + j] = W > 0.f ? w / W : 0.f;
    }
    if (gi == 0 && tid == 0) {
        float a = 0.f;
        if (s.Nt > 0)
            for (int h = 0; h < s.H; ++h) a += ws_vmh[(size_t)bl * s.H + h];
        tv_mass[bl] = a / (float)s.H;
    }
}

// ---------------------------------------------------------------------------------- sweep 2
template <int D, int NSLOT, int KS>
__global__ __launch_bounds__(kThreads) void score_vision_kernel(Shape s, int rowgroups,
                                                                const uint16_t* __restrict__ q_text,
                                                                const uint16_t* __restrict__ k,
                                                                const float* __restrict__ lse,
                                                                const float* __restrict__ w_txt,
                                                                const int32_t* __restrict__ budgets,
                                                                int vis_threshold,
                                                                float* __restrict__ ws_part) {
    using GG = Geo<D>;
    constexpr int RSETS = 4 / KS;
    constexpr int KBW = 4 / KS;
    __shared__ __attribute__((aligned(16))) char tiles[2][GG::TILE_BYTES];
    __shared__ float red[2][RSETS][kTile];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int rs = wave % RSETS, kp = wave / RSETS;
    int bid = blockIdx.x;
    const int rg = bid % rowgroups;
    bid /= rowgroups;
    const int kvh = bid % s.Hkv;
    const int bl = bid / s.Hkv;
    if (budgets != nullptr && budgets[bl] <= vis_threshold) return;

    const int QB = (s.Nq + 15) >> 4;
    const int NB = s.G * QB;
    const int rb0 = rg * RSETS * NSLOT;
    const float inv_heads = s.head_mode == 0 ? 1.0f / (float)s.H : 1.0f / (float)s.G;

    bf16x8 qf[NSLOT][GG::KSTEPS];
    float lse2[NSLOT][4], coef[NSLOT][4];
#pragma unroll
    for (int sl = 0; sl < NSLOT; ++sl) {
        const int rb = rb0 + rs + sl * RSETS;
        const int g = rb / QB;
        const int qi = (rb % QB) * 16 + (lane & 15);
        const bool valid = rb < NB && qi < s.Nq;
        const uint16_t* qp = q_text + (((size_t)bl * s.H + kvh * s.G + (valid ? g : 0)) * s.Nt + s.Ns +
                                       (valid ? qi : 0)) * D + (lane >> 4) * 8;
#pragma unroll
        for (int ks = 0; ks < GG::KSTEPS; ++ks) qf[sl][ks] = valid ? as_bf16x8(load16(qp + ks * 32)) : zero_frag();
        // accumulator rows of this lane: 4*(lane/16) + j of the block
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int qj = (rb % QB) * 16 + (lane >> 4) * 4 + j;
            const bool vj = rb < NB && qj < s.Nq;
            lse2[sl][j] = 0.f;
            coef[sl][j] = 0.f;
            if (vj) {
                const size_t head = (size_t)bl * s.H + kvh * s.G + g;
                lse2[sl][j] = lse[head * s.Nt + s.Ns + qj] * kLog2e;
                const size_t wrow = s.head_mode == 0 ? (size_t)bl * s.Nt : ((size_t)bl * s.Hkv + kvh) * s.Nt;
                coef[sl][j] = w_txt[wrow + s.Ns + qj] * inv_heads;
            }
        }
    }

    const uint16_t* kbase = k + (((size_t)bl * s.Hkv + kvh) * (size_t)s.N + s.Ns) * D;
    const int ntiles = (s.Nv + kTile - 1) / kTile;
    float* out = ws_part + (((size_t)bl * s.Hkv + kvh) * rowgroups + rg) * (size_t)s.Nv;

    u32x4 pre[GG::LOADS];
    load_tile_regs<D>(pre, kbase, 0, s.Nv - 1, tid);
    store_tile_lds<D>(tiles[0], pre, tid);
    __syncthreads();

    for (int t = 0; t < ntiles; ++t) {
        const char* buf = tiles[t & 1];
        if (t + 1 < ntiles) load_tile_regs<D>(pre, kbase, (t + 1) * kTile, s.Nv - 1, tid);
#pragma unroll
        for (int kbi = 0; kbi < KBW; ++kbi) {
            const int kb = kp + kbi * KS;
            bf16x8 kf[GG::KSTEPS];
            const char* src = buf + (kb * 16 + (lane & 15)) * GG::ROWB + (lane >> 4) * 16;
#pragma unroll
            for (int ks = 0; ks < GG::KSTEPS; ++ks) kf[ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(src + ks * 64));
            float col = 0.f;
#pragma unroll
            for (int sl = 0; sl < NSLOT; ++sl) {
                if (rb0 + rs + sl * RSETS >= NB) continue;
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < GG::KSTEPS; ++ks) acc = mfma16x16x32(qf[sl][ks], kf[ks], acc);
#pragma unroll
                for (int j = 0; j < 4; ++j) col += coef[sl][j] * fast_exp2(acc[j] * s.scale2 - lse2[sl][j]);
            }
            col += shfl_xor(col, 16);
            col += shfl_xor(col, 32);
            if (lane < 16) red[t & 1][rs][kb * 16 + lane] = col;
        }
        if (t + 1 < ntiles) store_tile_lds<D>(tiles[(t + 1) & 1], pre, tid);
        __syncthreads();
        if (tid < kTile) {
            const int key = t * kTile + tid;
            if (key < s.Nv) {
                float a = 0.f;
#pragma unroll
                for (int r = 0; r < RSETS; ++r) a += red[t & 1][r][tid];
                out[key] = a;
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
    float a = 0.f;
    for (int kv = kv0; kv < kv0 + kvn; ++kv)
        for (int rg = 0; rg < rowgroups; ++rg)
            a += ws_part[(((size_t)bl * s.Hkv + kv) * rowgroups + rg) * (size_t)s.Nv + j];
    s_vis[((size_t)bl * s.ngroups + gi) * s.Nv + j] = a;
}

// ---------------------------------------------------------------------------------- dispatch
#define TGVKV_ROWPLAN_DISPATCH(KERNEL, D, rp, ...)                                              \
    do {                                                                                        \
        if (rp.ks == 4) hipLaunchKernelGGL((KERNEL<D, 1, 4>), __VA_ARGS__);                     \
        else if (rp.ks == 2 && rp.nslot == 1) hipLaunchKernelGGL((KERNEL<D, 1, 2>), __VA_ARGS__); \
        else if (rp.ks == 2) hipLaunchKernelGGL((KERNEL<D, 2, 2>), __VA_ARGS__);                \
        else if (rp.nslot == 1) hipLaunchKernelGGL((KERNEL<D, 1, 1>), __VA_ARGS__);             \
        else if (rp.nslot == 2) hipLaunchKernelGGL((KERNEL<D, 2, 1>), __VA_ARGS__);             \
        else if (rp.nslot == 4) hipLaunchKernelGGL((KERNEL<D, 4, 1>), __VA_ARGS__);             \
        else hipLaunchKernelGGL((KERNEL<D, 6, 1>), __VA_ARGS__);                                \
    } while (0)

}  // namespace

RowPlan plan_question_rows(const Shape& s) {
    const int QB = (s.Nq + 15) / 16;
    const int NB = s.G * QB;
    RowPlan rp;
    if (NB <= 1) { rp.nslot = 1; rp.ks = 4; }
    else if (NB == 2) { rp.nslot = 1; rp.ks = 2; }
    else if (NB == 3) { rp.nslot = 2; rp.ks = 2; }
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

hipError_t launch_score_text(const Shape& s, const uint16_t* q_text, const uint16_t* k, float* lse,
                             const float* ws_vm, float* ws_colsum, float* ws_vmh, hipStream_t st) {
    const long long nblk = (long long)s.B * s.L * s.Hkv;
    if (nblk == 0 || s.Nt == 0) return hipSuccess;
    dim3 grid((unsigned)nblk), block(kThreads);
    const size_t lds = sizeof(float) * (size_t)s.G * s.Nt;
    if (s.D == 128)
        hipLaunchKernelGGL(score_text_kernel<128>, grid, block, lds, st, s, q_text, k, lse, ws_vm, ws_colsum, ws_vmh);
    else
        hipLaunchKernelGGL(score_text_kernel<64>, grid, block, lds, st, s, q_text, k, lse, ws_vm, ws_colsum, ws_vmh);
    return hipGetLastError();
}

hipError_t launch_score_fin(const Shape& s, const float* ws_colsum, const float* ws_vmh, float* s_txt,
                            float* w_txt, float* tv_mass, hipStream_t st) {
    const long long nblk = (long long)s.B * s.L * s.ngroups;
    if (nblk == 0) return hipSuccess;
    hipLaunchKernelGGL(score_fin_kernel, dim3((unsigned)nblk), dim3(kThreads), 0, st, s, ws_colsum, ws_vmh,
                       s_txt, w_txt, tv_mass);
    return hipGetLastError();
}

hipError_t launch_score_vision(const Shape& s, const RowPlan& rp, const uint16_t* q_text, const uint16_t* k,
                               const float* lse, const float* w_txt, const int32_t* budgets,
                               int32_t vis_threshold, float* ws_part, hipStream_t st) {
    const long long nblk = (long long)s.B * s.L * s.Hkv * rp.rowgroups;
    if (nblk == 0 || s.Nv == 0) return hipSuccess;
    dim3 grid((unsigned)nblk), block(kThreads);
    if (s.D == 128)
        TGVKV_ROWPLAN_DISPATCH(score_vision_kernel, 128, rp, grid, block, 0, st, s, rp.rowgroups, q_text, k, lse,
                               w_txt, budgets, vis_threshold, ws_part);
    else
        TGVKV_ROWPLAN_DISPATCH(score_vision_kernel, 64, rp, grid, block, 0, st, s, rp.rowgroups, q_text, k, lse,
                               w_txt, budgets, vis_threshold, ws_part);
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
