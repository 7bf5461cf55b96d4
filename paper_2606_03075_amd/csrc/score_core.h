// Device building blocks of the TWR / TVB scoring passes (kernels in score.hip).
//
// A "unit" is one (sequence b, layer l, KV head) slice: bl = b * L + l.  Its
// question rows (query heads sharing the KV head x question tokens) are cut into
// 16-row blocks, QB = ceil(N_q / 16) per head; block rb covers head rb / QB and
// question indices (rb % QB) * 16 .. + 15.  The 4 waves of a workgroup split the
// blocks into RSETS row sets of up to NSLOT blocks each (slot_block) and, when there
// are few blocks, each 64-key tile into KS key parts (RSETS * KS = 4).
//
// MFMA layout: v_mfma_f32_16x16x32_bf16.  A 64-key tile of K sits in LDS with
// rows padded by 16 bytes (the 16 lanes reading one 16-byte column chunk of 16
// consecutive keys then hit distinct banks); the question rows stay in
// registers for the whole sweep.  The statistics sweep computes C[key][row]
// (keys on the M side) so that each lane owns one row and keeps its running
// max / sum with no cross-lane traffic in the loop; the vision sweep computes
// C[row][key] so that each lane owns one key and sums its column in registers.
#pragma once

#include "tgvkv_device.h"
#include "tgvkv_shape.h"

#include <type_traits>

namespace tgvkv {
namespace core {

constexpr int kThreads = 256;
constexpr int kTile = 64;  // keys per LDS tile
constexpr int kOutTiles = 8;  // vision-score tiles buffered in LDS per burst of global writes
constexpr int kWholeOutBytes = 16384;  // up to this many bytes of a unit's scores are written once, at the end

template <int D>
struct Geo {
    static constexpr int KSTEPS = D / 32;                  // MFMA k-steps over the head dim
    static constexpr int CPR = D / 8;                      // 16-byte chunks per key row
    static constexpr int ROWB = D * 2 + 16;                // padded LDS row, bytes
    static constexpr int TILE_BYTES = kTile * ROWB;
    static constexpr int LOADS = kTile * CPR / kThreads;   // 16-byte loads per thread per tile
};

template <int D>
__device__ __forceinline__ void load_tile_regs(u32x4 (&r)[Geo<D>::LOADS], const uint16_t* kbase, int key0,
                                               int key_last, int tid) {
#pragma unroll
    for (int it = 0; it < Geo<D>::LOADS; ++it) {
        const int c = it * kThreads + tid;
        const int row = c / Geo<D>::CPR, cc = c % Geo<D>::CPR;
        const int key = min(key0 + row, key_last);
        r[it] = load16_stream(kbase + (size_t)key * D + cc * 8);
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

// The tile pipeline with its tiles split into phases (see tile_pipeline below for
// the pipeline itself).
template <int D, int DEPTH, typename Edge, typename Mid, typename Post>
__device__ __forceinline__ void tile_pipeline_phased(const uint16_t* kbase, int kbeg, int kend,
                                                     char (*tiles)[Geo<D>::TILE_BYTES], int mid_beg, int mid_end,
                                                     Edge&& edge, Mid&& mid, Post&& post) {
    static_assert(DEPTH == 1 || DEPTH == 2, "tile pipeline depth");
    const int tid = threadIdx.x;
    const int ntiles = (kend - kbeg + kTile - 1) / kTile;
    // tiles [mid_beg, mid_end) run `mid`, the others `edge`; each phase is its own loop, so the
    // compiler lays out and allocates the middle loop without the edge tiles' code in it
    if (DEPTH == 1) {
        u32x4 pre[Geo<D>::LOADS];
        if (ntiles > 0) {
            load_tile_regs<D>(pre, kbase, kbeg, kend - 1, tid);
            store_tile_lds<D>(tiles[0], pre, tid);
        }
        __syncthreads();
        auto step = [&](int t, auto& compute) {
            const int key0 = kbeg + t * kTile;
            if (t + 1 < ntiles) load_tile_regs<D>(pre, kbase, key0 + kTile, kend - 1, tid);
            compute(tiles[t & 1], key0, t);
            if (t + 1 < ntiles) store_tile_lds<D>(tiles[(t + 1) & 1], pre, tid);
            __syncthreads();
            post(key0, t);
        };
        int t = 0;
        for (; t < min(mid_beg, ntiles); ++t) step(t, edge);
        for (; t < min(mid_end, ntiles); ++t) step(t, mid);
        for (; t < ntiles; ++t) step(t, edge);
        return;
    }
    // Loads past the last tile are issued anyway (their key index is clamped to
    // the last key, so they re-read one cached row): with a fixed number of loads
    // per step the compiler's wait before each LDS store counts only that tile's
    // loads instead of draining the one fetched behind it.
    if (ntiles <= 0) {
        __syncthreads();
        return;
    }
    u32x4 ra[Geo<D>::LOADS], rb[Geo<D>::LOADS];
    load_tile_regs<D>(ra, kbase, kbeg, kend - 1, tid);
    store_tile_lds<D>(tiles[0], ra, tid);
    load_tile_regs<D>(rb, kbase, kbeg + kTile, kend - 1, tid);
    load_tile_regs<D>(ra, kbase, kbeg + 2 * kTile, kend - 1, tid);
    __syncthreads();
    // An odd tile count runs one more half-step without compute or post (its load
    // and store touch only clamped rows and the free buffer), so the loop has no
    // exit in the middle; with one, the compiler's wait counting loses track of
    // the loads in flight at the loop head and drains them all.  Two tiles per
    // step: the phase boundaries are taken at even tiles (a pure tile run as an
    // edge tile gives the same result).
    auto step2 = [&](int t, auto& compute) {
        // tile t in tiles[0], tile t+1 in rb, tile t+2 in ra; tiles[1] is free
        const int key0 = kbeg + t * kTile;
        compute(tiles[0], key0, t);
        store_tile_lds<D>(tiles[1], rb, tid);
        load_tile_regs<D>(rb, kbase, key0 + 3 * kTile, kend - 1, tid);
        __syncthreads();
        post(key0, t);
        // tile t+1 in tiles[1], tile t+2 in ra, tile t+3 in rb; tiles[0] is free
        const bool more = t + 1 < ntiles;
        if (more) compute(tiles[1], key0 + kTile, t + 1);
        store_tile_lds<D>(tiles[0], ra, tid);
        load_tile_regs<D>(ra, kbase, key0 + 4 * kTile, kend - 1, tid);
        __syncthreads();
        if (more) post(key0 + kTile, t + 1);
    };
    const int m0 = min((mid_beg + 1) & ~1, ntiles), m1 = max(min(mid_end & ~1, ntiles), m0);
    int t = 0;
    for (; t < m0; t += 2) step2(t, edge);
    for (; t < m1; t += 2) step2(t, mid);
    for (; t < ntiles; t += 2) step2(t, edge);
}

// Streams the 64-key tiles of keys [kbeg, kend) through the two LDS buffers.
// With DEPTH 2 two tiles are in flight per workgroup: while tile t is consumed
// from LDS, tile t+1 waits in registers and tile t+2 is being fetched (costs
// one more tile of registers); with DEPTH 1 only tile t+1 is fetched meanwhile.
// compute(buf, key0, t) runs on tile t; post(key0, t) runs after the barrier
// that ends tile t.  Returns right after the last post (no barrier after it).
// Every barrier is reached by all threads (the tile count is uniform).
template <int D, int DEPTH, typename Compute, typename Post>
__device__ __forceinline__ void tile_pipeline(const uint16_t* kbase, int kbeg, int kend,
                                              char (*tiles)[Geo<D>::TILE_BYTES], Compute&& compute, Post&& post) {
    tile_pipeline_phased<D, DEPTH>(kbase, kbeg, kend, tiles, 0, 0, compute, compute, post);
}

// Tiles in flight per workgroup for a row plan: two while the question rows
// leave room in registers.
template <int NSLOT>
struct PipeDepth {
    static constexpr int value = NSLOT <= 2 ? 2 : 1;
};

// Row block held by slot sl of row set rs, in the row group starting at block rb0.  The sets
// take the blocks in a snake order (0 1 2 3, then 7 6 5 4, 8 9 10 11, ...), so that with several
// slots per wave every wave holds rows from early and late in the question: the causally masked
// question-key work of the statistics sweep's last tiles and of the text pass is then nearly the
// same for every wave (in the plain order the last wave's rows see the most keys, and the
// per-tile barrier waits for it).  At the 13B stress shape: 6.75 against 6.79-6.82 ms.
template <int RSETS>
__device__ __forceinline__ int slot_block(int rb0, int rs, int sl) {
    return rb0 + sl * RSETS + ((sl & 1) ? RSETS - 1 - rs : rs);
}

__device__ __forceinline__ bf16x8 zero_frag() {
    u32x4 z = {0u, 0u, 0u, 0u};
    return as_bf16x8(z);
}

template <int D>
__device__ __forceinline__ void load_kfrag(bf16x8 (&kf)[Geo<D>::KSTEPS], const char* buf, int kb, int lane) {
    const char* src = buf + (kb * 16 + (lane & 15)) * Geo<D>::ROWB + (lane >> 4) * 16;
#pragma unroll
    for (int ks = 0; ks < Geo<D>::KSTEPS; ++ks) kf[ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(src + ks * 64));
}

template <int D, int NSLOT>
__device__ __forceinline__ void settle_qrows(const bf16x8 (&qf)[NSLOT][Geo<D>::KSTEPS]) {
#pragma unroll
    for (int sl = 0; sl < NSLOT; ++sl)
#pragma unroll
        for (int ks = 0; ks < Geo<D>::KSTEPS; ++ks) settle(qf[sl][ks]);
}

// Question-row fragments of the row set of this wave (lane: row lane & 15 of each block).
template <int D, int NSLOT, int KS, bool SETTLE = true>
__device__ __forceinline__ void load_qrows(const Shape& s, const uint16_t* q_text, int bl, int kvh, int rb0,
                                           bf16x8 (&qf)[NSLOT][Geo<D>::KSTEPS], int (&qrow)[NSLOT]) {
    constexpr int RSETS = 4 / KS;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int rs = wave % RSETS;
    const int QB = (s.Nq + 15) >> 4;
    const int NB = s.G * QB;
#pragma unroll
    for (int sl = 0; sl < NSLOT; ++sl) {
        const int rb = slot_block<RSETS>(rb0, rs, sl);
        const int g = rb / QB;
        const int qi = (rb % QB) * 16 + (lane & 15);
        qrow[sl] = qi;
        const bool valid = rb < NB && qi < s.Nq;
        const uint16_t* qp = q_text + (((size_t)bl * s.H + kvh * s.G + (valid ? g : 0)) * s.Nt + s.Ns +
                                       (valid ? qi : 0)) * D + (lane >> 4) * 8;
#pragma unroll
        for (int ks = 0; ks < Geo<D>::KSTEPS; ++ks)
            qf[sl][ks] = valid ? as_bf16x8(load16(qp + ks * 32)) : zero_frag();
    }
    if (SETTLE) settle_qrows<D, NSLOT>(qf);
}

// Statistics sweep over keys [kbeg, kend) of one unit (kbeg a multiple of kTile):
// per question row a reference max m (base-2 units, within 8 of the row's largest
// logit), the sum of exp2(z - m) over visible keys and the same sum over vision
// keys, so that m + log2(sum) is the row's normaliser.  On return the key-part-0
// waves hold, in lanes 0..15, the merged statistics of their rows; the workgroup
// is synced.
template <int D, int NSLOT, int KS>
__device__ void stats_sweep(const Shape& s, const uint16_t* kbase, int kbeg, int kend,
                            const bf16x8 (&qf)[NSLOT][Geo<D>::KSTEPS], const int (&qrow)[NSLOT],
                            char (*tiles)[Geo<D>::TILE_BYTES], float (&m)[NSLOT], float (&lsum)[NSLOT],
                            float (&vsum)[NSLOT]) {
    using GG = Geo<D>;
    constexpr int RSETS = 4 / KS;
    constexpr int KBW = 4 / KS;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int rs = wave % RSETS, kp = wave / RSETS;
    const int vis0 = s.Ns, vis1 = s.Ns + s.Nv;
    float tsum[NSLOT];
#pragma unroll
    for (int sl = 0; sl < NSLOT; ++sl) {
        m[sl] = kNegInf;
        tsum[sl] = 0.f;
        vsum[sl] = 0.f;
    }
    // One tile's statistics; PURE: every key of the tile is a vision key (visible to every
    // question row).  Every row slot is computed, also past the last row block (zero query
    // fragments, never written): with no per-slot branch the compiler interleaves one slot's
    // softmax steps with the next slot's MFMAs.  The lane keeps a reference max m per row and
    // rescales its sums only when needed (one uniform branch per key block, rarely taken), so
    // the sums hold terms up to about 2^kSlack, far from overflow, and m + log2(sum) is the
    // same normaliser.  An all-vision block exponentiates against the current reference
    // first and rescales when the 4 terms of a lane sum past 2^kSlack (an overflow to inf,
    // the first block's case, included): it needs no max of its own.  A masked block tests
    // its largest visible logit against m + kSlack.  The text and vision terms go to
    // separate sums (tsum, vsum), so an all-vision block adds once.
    constexpr float kSlack = 8.f;
    constexpr float kSlackSum = 256.f;  // 2^kSlack
    auto tile = [&](const char* buf, int key0, auto pure_tag) {
        constexpr bool PURE = decltype(pure_tag)::value;
        // sum of a slot's 4 all-vision terms against its reference max
        auto pure_terms = [&](const f32x4& zz, float mref) {
            const float nm = -mref;
            return (fast_exp2(__builtin_fmaf(zz[0], s.scale2, nm)) + fast_exp2(__builtin_fmaf(zz[1], s.scale2, nm))) +
                   (fast_exp2(__builtin_fmaf(zz[2], s.scale2, nm)) + fast_exp2(__builtin_fmaf(zz[3], s.scale2, nm)));
        };
#pragma unroll
        for (int kbi = 0; kbi < KBW; ++kbi) {
            const int kb = kp + kbi * KS;
            bf16x8 kf[GG::KSTEPS];
            load_kfrag<D>(kf, buf, kb, lane);
            const int kfirst = key0 + kb * 16 + (lane >> 4) * 4;  // key of accumulator element 0
            f32x4 z[NSLOT];
            float mx[NSLOT];  // PURE: the slot's term sum; masked: its largest visible logit
            bool grow = false;
#pragma unroll
            for (int sl = 0; sl < NSLOT; ++sl) {
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                // With 6 slots (2 waves per SIMD) a wave issuing its MFMAs goes first, the other
                // wave's softmax fills in: 763-780 against 819-821 us per launch at the
                // Qwen2-VL shape; at 4 slots it changed nothing, and the vision sweep lost.
                if (NSLOT >= 6 && KS == 1) __builtin_amdgcn_s_setprio(1);
#pragma unroll
                for (int ks = 0; ks < GG::KSTEPS; ++ks) acc = mfma16x16x32(kf[ks], qf[sl][ks], acc);
                if (NSLOT >= 6 && KS == 1) __builtin_amdgcn_s_setprio(0);
                if (PURE) {
                    z[sl] = acc;  // logits in MFMA units; scaled inside the exponent
                    mx[sl] = pure_terms(acc, m[sl]);
                    grow |= !(mx[sl] <= kSlackSum);
                } else {
                    // a question row sees every key below vis1 and the question keys up to its own
                    const int lim = min(kend - 1, vis1 + qrow[sl]);
                    mx[sl] = kNegInf;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        z[sl][j] = kfirst + j <= lim ? acc[j] * s.scale2 : kNegInf;
                        mx[sl] = fmaxf(mx[sl], z[sl][j]);
                    }
                    grow |= mx[sl] > m[sl] + kSlack;
                }
            }
            if (__builtin_amdgcn_ballot_w64(grow) != 0) {
#pragma unroll
                for (int sl = 0; sl < NSLOT; ++sl) {
                    const float bmax = PURE ? fmaxf(fmaxf(z[sl][0], z[sl][1]), fmaxf(z[sl][2], z[sl][3])) * s.scale2
                                            : mx[sl];
                    const float mn = fmaxf(m[sl], bmax);
                    if (mn != kNegInf) {
                        const float sc = fast_exp2(m[sl] - mn);
                        tsum[sl] *= sc;
                        vsum[sl] *= sc;
                        m[sl] = mn;
                    }
                    if (PURE) mx[sl] = pure_terms(z[sl], m[sl]);  // the terms against the new reference
                }
            }
#pragma unroll
            for (int sl = 0; sl < NSLOT; ++sl) {
                if (PURE) {
                    vsum[sl] += mx[sl];
                } else {
                    const float mu = m[sl] == kNegInf ? 0.f : m[sl];  // a row with no visible key yet
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int key = kfirst + j;
                        const float e = fast_exp2(z[sl][j] - mu);  // 0 for a masked key
                        const bool isv = (key >= vis0) & (key < vis1);
                        vsum[sl] += isv ? e : 0.f;
                        tsum[sl] += isv ? 0.f : e;
                    }
                }
            }
        }
    };
    // tiles [t0, t1) lie wholly inside the vision keys (and below kend): they skip the masks
    const int t0 = vis0 > kbeg ? (vis0 - kbeg + kTile - 1) / kTile : 0;
    const int t1 = max((min(vis1, kend) - kbeg) / kTile, t0);
    tile_pipeline_phased<D, PipeDepth<NSLOT>::value>(
        kbase, kbeg, kend, tiles, t0, t1,
        [&](const char* buf, int key0, int) { tile(buf, key0, std::false_type{}); },
        [&](const char* buf, int key0, int) { tile(buf, key0, std::true_type{}); },
        [](int, int) {});
#pragma unroll
    for (int sl = 0; sl < NSLOT; ++sl) lsum[sl] = tsum[sl] + vsum[sl];
    // the four lane quarters of a wave saw different keys of the same rows
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
        __syncthreads();
    }
}

// Per-lane row coefficients of the vision sweep: the accumulator rows of a lane
// are 4*(lane/16) + j of each block; lse2 in base-2 units, coef = w~_i / heads.
template <int NSLOT, int KS, bool SETTLE = true>
__device__ __forceinline__ void load_row_coefs(const Shape& s, int bl, int kvh, int rb0, const float* lse,
                                               const float* w_txt, float (&lse2)[NSLOT][4],
                                               float (&coef)[NSLOT][4]) {
    constexpr int RSETS = 4 / KS;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int rs = wave % RSETS;
    const int QB = (s.Nq + 15) >> 4;
    const int NB = s.G * QB;
    const float inv_heads = s.head_mode == 0 ? 1.0f / (float)s.H : 1.0f / (float)s.G;
    const size_t wrow = s.head_mode == 0 ? (size_t)bl * s.Nt : ((size_t)bl * s.Hkv + kvh) * s.Nt;
    // every load is issued (invalid rows read row 0 of the unit) so that they are all
    // in flight together; invalid rows then get zero coefficients
    float lv[NSLOT][4], wv[NSLOT][4];
    bool ok[NSLOT][4];
#pragma unroll
    for (int sl = 0; sl < NSLOT; ++sl) {
        const int rb = slot_block<RSETS>(rb0, rs, sl);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int qj = (rb % QB) * 16 + (lane >> 4) * 4 + j;
            ok[sl][j] = rb < NB && qj < s.Nq;
            const int g = ok[sl][j] ? rb / QB : 0;
            const int qc = ok[sl][j] ? qj : 0;
            const size_t head = (size_t)bl * s.H + kvh * s.G + g;
            lv[sl][j] = lse[head * s.Nt + s.Ns + qc];
            wv[sl][j] = w_txt[wrow + s.Ns + qc];
        }
    }
#pragma unroll
    for (int sl = 0; sl < NSLOT; ++sl)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            lse2[sl][j] = ok[sl][j] ? lv[sl][j] * kLog2e : 0.f;
            coef[sl][j] = ok[sl][j] ? wv[sl][j] * inv_heads : 0.f;
        }
    if (SETTLE) {
#pragma unroll
        for (int sl = 0; sl < NSLOT; ++sl)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                settle(lse2[sl][j]);
                settle(coef[sl][j]);
            }
    }
}

// Vision sweep over vision keys [vbeg, vend) (vbeg a multiple of kTile; kvis
// points at the first vision key of the unit): out[j] = sum over this
// workgroup's rows of coef * exp(z - lse), for every key j of the range.
// obuf: out_tiles * kTile floats of LDS; scores are written in bursts of
// out_tiles tiles (all of them at the end when out_tiles covers the range).  With MASS the sweep also sums each
// row's probabilities over the range (its vision mass when the range is all
// vision keys): on return rsum[sl][j] of the key-part-0 waves holds the sum of
// accumulator row 4*(lane/16) + j of slot sl, in every lane of the 16.
template <int D, int NSLOT, int KS, bool MASS = false>
__device__ void vision_sweep(const Shape& s, const uint16_t* kvis, int vbeg, int vend,
                             const bf16x8 (&qf)[NSLOT][Geo<D>::KSTEPS], const float (&lse2)[NSLOT][4],
                             const float (&coef)[NSLOT][4], int rb0, int NB, char (*tiles)[Geo<D>::TILE_BYTES],
                             float (*red)[4 / KS][kTile], float* obuf, int out_tiles, float* out,
                             float (&rsum)[NSLOT][4]) {
    using GG = Geo<D>;
    constexpr int RSETS = 4 / KS;
    constexpr int KBW = 4 / KS;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int rs = wave % RSETS, kp = wave / RSETS;
    const int ntiles = (vend - vbeg + kTile - 1) / kTile;
    if (MASS) {
#pragma unroll
        for (int sl = 0; sl < NSLOT; ++sl)
#pragma unroll
            for (int j = 0; j < 4; ++j) rsum[sl][j] = 0.f;
    }
    // Without row masses a row's coefficient goes into its exponent: coef * 2^(x - lse2) =
    // 2^(x - c2), c2 = lse2 - log2(coef) (+inf for a zero coefficient, so rows past N_q add 0).
    // One per-row constant instead of two: at the Qwen2-VL shape's six slots the sweep's
    // compute runs about 4 % faster (probe of the key-block code).
    float c2[NSLOT][4];
#pragma unroll
    for (int sl = 0; sl < NSLOT; ++sl)
#pragma unroll
        for (int j = 0; j < 4; ++j) c2[sl][j] = MASS ? 0.f : lse2[sl][j] - fast_log2(coef[sl][j]);
    tile_pipeline<D, PipeDepth<NSLOT>::value>(
        kvis, vbeg, vend, tiles,
        [&](const char* buf, int key0, int t) {
#pragma unroll
            for (int kbi = 0; kbi < KBW; ++kbi) {
                const int kb = kp + kbi * KS;
                bf16x8 kf[GG::KSTEPS];
                load_kfrag<D>(kf, buf, kb, lane);
                const int kcol = key0 + kb * 16 + (lane & 15);  // this lane's key (accumulator column)
                // the last tile repeats the last key past vend (clamped loads): not a key, weight 0
                // in the row sums (one multiply-add per probability, no per-element branch)
                const float inr = kcol < vend ? 1.f : 0.f;
                float col = 0.f;
#pragma unroll
                for (int sl = 0; sl < NSLOT; ++sl) {
                    if (slot_block<RSETS>(rb0, rs, sl) >= NB) continue;
                    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int ks = 0; ks < GG::KSTEPS; ++ks) acc = mfma16x16x32(qf[sl][ks], kf[ks], acc);
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        if (MASS) {
                            const float p = fast_exp2(acc[j] * s.scale2 - lse2[sl][j]);
                            col += coef[sl][j] * p;
                            rsum[sl][j] = __builtin_fmaf(p, inr, rsum[sl][j]);
                        } else {
                            col += fast_exp2(acc[j] * s.scale2 - c2[sl][j]);
                        }
                    }
                }
                col = sum_xor32(sum_xor16(col));
                if (lane < 16) red[t & 1][rs][kb * 16 + lane] = col;
            }
        },
        [&](int, int t) {
            // Each of the first 64 threads parks its key's score in its own LDS slot and
            // writes out_tiles of them at once, then waits for the writes: a global store
            // pending among the tile loads would make the compiler drain every load in
            // flight at each tile, not once per out_tiles tiles.
            if (tid < kTile) {
                float a = 0.f;
#pragma unroll
                for (int r = 0; r < RSETS; ++r) a += red[t & 1][r][tid];
                const int slot = t % out_tiles;
                obuf[slot * kTile + tid] = a;
                if (slot == out_tiles - 1 || t == ntiles - 1) {
                    for (int i = 0; i <= slot; ++i) {
                        const int key = vbeg + (t - slot + i) * kTile + tid;
                        if (key < vend) out[key] = obuf[i * kTile + tid];
                    }
                    wait_vmem_all();
                }
            }
        });
    __syncthreads();
    if (MASS) {
        // a row's keys are spread over the 16 lanes of its quarter, then over the key parts
#pragma unroll
        for (int sl = 0; sl < NSLOT; ++sl)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                rsum[sl][j] = group_sum<16>(rsum[sl][j]);
        if (KS > 1) {
            float* buf = reinterpret_cast<float*>(tiles[0]);  // [wave][NSLOT][16]
            if (kp > 0 && (lane & 15) == 0) {
#pragma unroll
                for (int sl = 0; sl < NSLOT; ++sl)
#pragma unroll
                    for (int j = 0; j < 4; ++j) buf[(wave * NSLOT + sl) * 16 + (lane >> 4) * 4 + j] = rsum[sl][j];
            }
            __syncthreads();
            if (kp == 0) {
                for (int p2 = 1; p2 < KS; ++p2) {
                    const int w2 = p2 * RSETS + rs;
#pragma unroll
                    for (int sl = 0; sl < NSLOT; ++sl)
#pragma unroll
                        for (int j = 0; j < 4; ++j) rsum[sl][j] += buf[(w2 * NSLOT + sl) * 16 + (lane >> 4) * 4 + j];
                }
            }
            __syncthreads();
        }
    }
}

// Text x text pass of one unit.  lse2s [G][N_t] (LDS, base-2 units) must hold the
// question rows' normalisers.  Computes the system rows' normalisers (system
// rows see only system keys, causally) into lse2s and lse, then the column sums
// of the text->text probabilities per query head into ws_colsum [.., N_t].
// The work is small and latency-bound: each wave walks its items with the next
// block's 16-byte fragments fetched while the current block is used (two
// register sets, loads clamped into the unit so that every one is issued).
// With lse_given every text row's normaliser is already in lse2s (taken from the
// caller), the system rows are not recomputed and lse is not written.
template <int D>
__device__ void text_pass(const Shape& s, int bl, int kvh, const uint16_t* __restrict__ q_text,
                          const uint16_t* __restrict__ k, float* __restrict__ lse, float* lse2s,
                          float* __restrict__ ws_colsum, bool lse_given = false) {
    using GG = Geo<D>;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const size_t head0 = (size_t)bl * s.H + kvh * s.G;
    const uint16_t* kbase = k + ((size_t)bl * s.Hkv + kvh) * (size_t)s.N * D;
    const int koff = (lane >> 4) * 8;
    auto load_frag = [&](bf16x8 (&f)[GG::KSTEPS], const uint16_t* row) {
#pragma unroll
        for (int ks = 0; ks < GG::KSTEPS; ++ks) f[ks] = as_bf16x8(load16(row + koff + ks * 32));
    };

    // system rows x system keys: row normalisers (C[key][row]: a lane owns row i)
    const int SB = lse_given ? 0 : (s.Ns + 15) >> 4;
    for (int item = wave; item < s.G * SB; item += 4) {
        const int g = item / SB, rb = item % SB;
        const int i = rb * 16 + (lane & 15);
        const bool rv = i < s.Ns;
        bf16x8 qf[GG::KSTEPS], ka[GG::KSTEPS], kb2[GG::KSTEPS];
        load_frag(qf, q_text + ((head0 + g) * s.Nt + min(i, s.Ns - 1)) * D);
        auto krow = [&](int kb) { return kbase + (size_t)min(kb * 16 + (lane & 15), s.Ns - 1) * D; };
        load_frag(ka, krow(0));
        float m = kNegInf, l = 0.f, dummy = 0.f;
        auto step = [&](const bf16x8 (&kf)[GG::KSTEPS], int kb) {
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
        };
        // key blocks 0..rb; a block past rb is masked out by key <= i
        for (int kb = 0; kb <= rb; kb += 2) {
            load_frag(kb2, krow(kb + 1));
            step(ka, kb);
            load_frag(ka, krow(kb + 2));
            step(kb2, kb + 1);
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

    // all text rows x text keys: column sums (C[row][key]: a lane owns key j)
    const int TB = (s.Nt + 15) >> 4;
    for (int item = wave; item < s.G * TB; item += 4) {
        const int g = item / TB, kb = item % TB;
        const int j = kb * 16 + (lane & 15);
        const int jc = min(j, s.Nt - 1);
        const int pos = jc < s.Ns ? jc : jc + s.Nv;
        auto qrow = [&](int rb) { return q_text + ((head0 + g) * s.Nt + min(rb * 16 + (lane & 15), s.Nt - 1)) * D; };
        bf16x8 kf[GG::KSTEPS], qa[GG::KSTEPS], qb[GG::KSTEPS];
        load_frag(kf, kbase + (size_t)pos * D);
        load_frag(qa, qrow(kb));
        float col = 0.f;
        auto step = [&](const bf16x8 (&qf)[GG::KSTEPS], int rb) {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < GG::KSTEPS; ++ks) acc = mfma16x16x32(qf[ks], kf[ks], acc);
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const int ii = rb * 16 + (lane >> 4) * 4 + jj;
                if (ii < s.Nt && j <= ii) col += fast_exp2(acc[jj] * s.scale2 - lse2s[g * s.Nt + ii]);
            }
        };
        // row blocks kb..TB-1; a block past the last is masked out by ii < N_t
        for (int rb = kb; rb < TB; rb += 2) {
            load_frag(qb, qrow(rb + 1));
            step(qa, rb);
            load_frag(qa, qrow(rb + 2));
            step(qb, rb + 1);
        }
        col = sum_xor32(sum_xor16(col));
        if (lane < 16 && j < s.Nt) ws_colsum[(head0 + g) * s.Nt + j] = col;
    }
    __syncthreads();
}

// LDS layout of text_pass_lds in kl_bytes of 16-byte aligned LDS: the per-wave column
// partials [4][G][TK] (TK = N_t rounded up to 16 rows), then as many 16-row blocks of
// text keys as fit.  text_chunk_blocks gives that count; the pass needs at least the
// system keys' blocks and one block (else it is not used).
template <int D>
__host__ __device__ constexpr long long text_part_bytes(int G, int Nt) {
    return ((4LL * G * ((Nt + 15) / 16) * 16 * (long long)sizeof(float)) + 15) / 16 * 16;
}
template <int D>
__host__ __device__ constexpr int text_chunk_blocks(int G, int Nt, long long kl_bytes) {
    return (int)((kl_bytes - text_part_bytes<D>(G, Nt)) / (16LL * Geo<D>::ROWB));
}
template <int D>
__host__ __device__ constexpr bool text_lds_fits(int G, int Ns, int Nt, long long kl_bytes) {
    return kl_bytes > text_part_bytes<D>(G, Nt) &&
           text_chunk_blocks<D>(G, Nt, kl_bytes) >= ((Ns + 15) / 16 > 1 ? (Ns + 15) / 16 : 1);
}

// The text pass of text_pass with the unit's text keys staged in LDS (one round of
// loads by the whole workgroup per chunk of key blocks).  Each wave owns 16-row blocks
// of text rows: it fetches a block's query fragments from global memory (the next
// item's while the current one is used) and reads every key block it needs from LDS,
// so the pass costs a few load latencies per chunk instead of one per (row block, key
// block).  When the text keys do not all fit, they are staged in chunks of key blocks
// and each row block is revisited for every chunk up to its own keys (the causal mask
// keeps row block rb to key blocks <= rb).  The system keys are in the first chunk.
// Column sums: per (row block, key block) the 16 rows' probabilities are summed across
// the lane groups and added to the wave's own LDS partial for those keys; the four
// waves' partials are then added in wave order.  lse2s holds [G][N_t] base-2
// normalisers (the question rows' on entry; every row's with lse_given, and then the
// system rows' are not computed and lse is not written); kl points at kl_bytes of 16-byte
// aligned LDS with text_lds_fits<D>(G, N_s, N_t, kl_bytes).
template <int D>
__device__ void text_pass_lds(const Shape& s, int bl, int kvh, const uint16_t* __restrict__ q_text,
                              const uint16_t* __restrict__ k, float* __restrict__ lse, float* lse2s, char* kl,
                              long long kl_bytes, float* __restrict__ ws_colsum, bool lse_given = false) {
    using GG = Geo<D>;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const size_t head0 = (size_t)bl * s.H + kvh * s.G;
    const uint16_t* kbase = k + ((size_t)bl * s.Hkv + kvh) * (size_t)s.N * D;
    const int TB = (s.Nt + 15) >> 4;
    const int TK = TB * 16;                                       // key rows (the last block padded)
    float* part = reinterpret_cast<float*>(kl);                   // [4 waves][G][TK]
    char* kst = kl + text_part_bytes<D>(s.G, s.Nt);               // staged key blocks
    const int KC = min(text_chunk_blocks<D>(s.G, s.Nt, kl_bytes), TB);
    const int SB = lse_given ? 0 : (s.Ns + 15) >> 4;              // system-row blocks to normalise

    const int koff = (lane >> 4) * 8;
    auto load_q = [&](bf16x8 (&f)[GG::KSTEPS], int g, int row) {
        const uint16_t* src = q_text + ((head0 + g) * s.Nt + row) * D + koff;
#pragma unroll
        for (int ks = 0; ks < GG::KSTEPS; ++ks) f[ks] = as_bf16x8(load16(src + ks * 32));
    };
    auto sys_item_q = [&](bf16x8 (&f)[GG::KSTEPS], int item) {
        const int it = min(item, s.G * SB - 1);
        load_q(f, it / SB, min((it % SB) * 16 + (lane & 15), s.Ns - 1));
    };
    // column items of a chunk starting at key block c0: row blocks rb >= c0 of every head
    auto col_item_q = [&](bf16x8 (&f)[GG::KSTEPS], int item, int c0) {
        const int nrb = TB - c0;
        const int it = min(item, s.G * nrb - 1);
        load_q(f, it / nrb, min((c0 + it % nrb) * 16 + (lane & 15), s.Nt - 1));
    };

    // one round of loads: key blocks [c0, c1) (text order: system keys, then question keys),
    // with this wave's first items' query fragments; then the keys go to LDS
    constexpr int kStage = 8;  // 16-byte key loads per thread per round
    bf16x8 qs[GG::KSTEPS], qa[GG::KSTEPS], qb[GG::KSTEPS];
    auto stage = [&](int c0, int c1) {
        const int nch = (c1 - c0) * 16 * GG::CPR;
        for (int x0 = 0; x0 < nch; x0 += kStage * kThreads) {
            u32x4 r[kStage];
#pragma unroll
            for (int i = 0; i < kStage; ++i) {
                const int c = min(x0 + i * kThreads + tid, nch - 1);
                const int t = min(c0 * 16 + c / GG::CPR, s.Nt - 1);
                const int pos = t < s.Ns ? t : t + s.Nv;
                r[i] = load16(kbase + (size_t)pos * D + (c % GG::CPR) * 8);
            }
            if (x0 == 0) {
                if (c0 == 0 && SB > 0) sys_item_q(qs, wave);
                col_item_q(qa, wave, c0);
            }
#pragma unroll
            for (int i = 0; i < kStage; ++i) {
                const int c = x0 + i * kThreads + tid;
                if (c < nch) store16(kst + (c / GG::CPR) * GG::ROWB + (c % GG::CPR) * 16, r[i]);
            }
        }
    };
    stage(0, KC);
    for (int x = tid; x < 4 * s.G * TK; x += kThreads) part[x] = 0.f;
    __syncthreads();

    // system rows x system keys (all in the first chunk): row normalisers (C[key][row]: a
    // lane owns row i)
    for (int item = wave; item < s.G * SB; item += 4) {
        const int g = item / SB, rb = item % SB;
        const int i = rb * 16 + (lane & 15);
        if (item != wave) sys_item_q(qs, item);
        float m = kNegInf, l = 0.f;
        for (int kb = 0; kb <= rb; ++kb) {
            bf16x8 kf[GG::KSTEPS];
            load_kfrag<D>(kf, kst, kb, lane);
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < GG::KSTEPS; ++ks) acc = mfma16x16x32(kf[ks], qs[ks], acc);
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
        float dummy = 0.f;
#pragma unroll
        for (int off = 16; off < 64; off <<= 1) {
            const float m2 = shfl_xor(m, off), l2 = shfl_xor(l, off), d2 = shfl_xor(dummy, off);
            merge_stats(m, l, dummy, m2, l2, d2);
        }
        if (lane < 16 && i < s.Ns) {
            const float L2 = m + log2f(l);
            lse2s[g * s.Nt + i] = L2;
            lse[(head0 + g) * s.Nt + i] = L2 * kLn2;
        }
    }
    __syncthreads();

    // all text rows x text keys (C[row][key]: a lane owns key j, rows 4*(lane/16) + jj), one
    // chunk of key blocks [c0, c1) at a time
    for (int c0 = 0; c0 < TB; c0 += KC) {
        const int c1 = min(c0 + KC, TB);
        if (c0 > 0) {
            stage(c0, c1);
            __syncthreads();
        }
        const int nrb = TB - c0;
        const int items = s.G * nrb;
        auto consume = [&](const bf16x8 (&qf)[GG::KSTEPS], int item) {
            const int g = item / nrb, rb = c0 + item % nrb;
            float* wpart = part + ((size_t)wave * s.G + g) * TK;
            float l2[4];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj)
                l2[jj] = lse2s[g * s.Nt + min(rb * 16 + (lane >> 4) * 4 + jj, s.Nt - 1)];
            const int kend = min(rb, c1 - 1);
            for (int kb = c0; kb <= kend; ++kb) {
                bf16x8 kf[GG::KSTEPS];
                load_kfrag<D>(kf, kst, kb - c0, lane);
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < GG::KSTEPS; ++ks) acc = mfma16x16x32(qf[ks], kf[ks], acc);
                const int j = kb * 16 + (lane & 15);
                float col = 0.f;
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const int ii = rb * 16 + (lane >> 4) * 4 + jj;
                    if (ii < s.Nt && j <= ii) col += fast_exp2(acc[jj] * s.scale2 - l2[jj]);
                }
                col = sum_xor32(sum_xor16(col));
                if (lane < 16) wpart[j] += col;
            }
        };
        // this wave's items are wave, wave + 4, ...: two register sets, the next item's
        // fragments fetched while the current one is used (qa already holds the first)
        const int steps = (items + 3) / 4;
        int item = wave;
        for (int st = 0; st < steps; st += 2) {
            const int nx = item + 4;
            col_item_q(qb, nx, c0);
            if (item < items) consume(qa, item);
            const int nx2 = item + 8;
            col_item_q(qa, nx2, c0);
            if (nx < items) consume(qb, nx);
            item = nx2;
        }
        __syncthreads();  // the chunk's keys are done with before the next is staged
    }
    for (int x = tid; x < s.G * s.Nt; x += kThreads) {
        const int g = x / s.Nt, j = x % s.Nt;
        float a = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) a += part[((size_t)w * s.G + g) * TK + j];
        ws_colsum[(head0 + g) * s.Nt + j] = a;
    }
    __syncthreads();
}

// LDS of text_pass_qregs outside the key tiles, in floats: [G][N_t] normalisers (base 2),
// [G][N_q] vision masses, then the per-wave column partials [4][G][TK] (TK = N_t rounded up
// to 16 rows).
__host__ __device__ constexpr long long text_area_floats(int G, int Nt, int Nq) {
    return (long long)G * Nt + (long long)G * Nq + 4LL * G * ((Nt + 15) / 16) * 16;
}

// The text pass of a unit whose question rows are held in registers by the statistics
// sweep (qf, the sweep's row plan; rb0 = 0).  The question rows' text->text probabilities
// are recomputed from those fragments: against the system keys, staged once in the key
// tiles, and against the question keys, streamed through the tile pipeline, so that the
// pass loads no question-row fragment and only the text keys.  The system rows (which see
// only system keys) load their fragments: first their normalisers, then their column
// sums.  Column sums go to per-wave LDS partials, which are then added in wave order.
// lse2s [G][N_t] holds the question rows' normalisers (base 2) on entry; part is
// 4*G*TK floats of LDS; the two key tiles must hold the system keys (N_s <= 2 * kTile).
template <int D, int NSLOT, int KS>
__device__ void text_pass_qregs(const Shape& s, int bl, int kvh, const uint16_t* __restrict__ q_text,
                                const uint16_t* __restrict__ k, float* __restrict__ lse,
                                const bf16x8 (&qf)[NSLOT][Geo<D>::KSTEPS], float* lse2s, float* part,
                                char (*tiles)[Geo<D>::TILE_BYTES], float* __restrict__ ws_colsum) {
    using GG = Geo<D>;
    constexpr int RSETS = 4 / KS;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int rs = wave % RSETS, kp = wave / RSETS;
    const size_t head0 = (size_t)bl * s.H + kvh * s.G;
    const uint16_t* kbase = k + ((size_t)bl * s.Hkv + kvh) * (size_t)s.N * D;
    const int QB = (s.Nq + 15) >> 4;
    const int NB = s.G * QB;
    const int TK = ((s.Nt + 15) >> 4) * 16;
    const int SB = (s.Ns + 15) >> 4;
    const int koff = (lane >> 4) * 8;
    char* sysk = &tiles[0][0];  // the system keys' 16-row blocks, ROWB bytes a row

    // per slot: its head, its first question row, and the normalisers of this lane's
    // accumulator rows 4*(lane/16) + j in C[row][key] (+inf for rows past N_q: p = 0)
    int gsl[NSLOT], q0s[NSLOT];
    bool sok[NSLOT];
    float l2r[NSLOT][4];
#pragma unroll
    for (int sl = 0; sl < NSLOT; ++sl) {
        const int rb = slot_block<RSETS>(0, rs, sl);
        sok[sl] = rb < NB;
        gsl[sl] = sok[sl] ? rb / QB : sl > 0 ? gsl[sl - 1] : 0;
        q0s[sl] = (rb % QB) * 16;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int qi = q0s[sl] + (lane >> 4) * 4 + j;
            l2r[sl][j] = (sok[sl] && qi < s.Nq) ? lse2s[gsl[sl] * s.Nt + s.Ns + qi] : __builtin_inff();
        }
    }
    // adds a 16-key block's column sums (lane: key lane % 16, 4 rows each) of head g to this
    // wave's partial at text index t0 + lane % 16, for the block's first kn keys
    auto flush = [&](float col, int g, int t0, int kn) {
        col = sum_xor32(sum_xor16(col));
        if (lane < min(kn, 16)) part[((size_t)wave * s.G + g) * TK + t0 + lane] += col;
    };
    // question rows x one 16-key block kf of text keys, of which the first kn are keys; c0:
    // the block's first question-key index (causal: keys of later question tokens are masked),
    // kSysBlock for system keys (visible to every question row); t0: the block's text index.
    // Every slot is computed, with no per-slot branch (a slot past the last row block has
    // normalisers +inf, so p = 0; keys past a row are masked by a select): per tile the loop
    // then runs like the sweep's, where skipping the causally hidden blocks of a wave's slots
    // (branches between a slot's MFMAs and its exponentials, and spills at the 168-register
    // cap) had taken 29 of the pass's 39 us at the 13B stress shape.  The column sums of the
    // slots of one query head go to one flush; a wave whose slots span two heads flushes at
    // the change (wave-uniform).
    constexpr int kSysBlock = -(1 << 30);
    auto qrow_block = [&](const bf16x8 (&kf)[GG::KSTEPS], int c0, int t0, int kn) {
        float colacc = 0.f;
        int gcur = gsl[0];
#pragma unroll
        for (int sl = 0; sl < NSLOT; ++sl) {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < GG::KSTEPS; ++ks) acc = mfma16x16x32(qf[sl][ks], kf[ks], acc);
            const int lim = q0s[sl] + (lane >> 4) * 4 - c0 - (lane & 15);  // key visible to row j iff lim + j >= 0
            float col = 0.f;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float p = fast_exp2(acc[j] * s.scale2 - l2r[sl][j]);
                col += lim + j >= 0 ? p : 0.f;
            }
            if (sl > 0 && gsl[sl] != gcur) {
                flush(colacc, gcur, t0, kn);
                colacc = 0.f;
                gcur = gsl[sl];
            }
            colacc += col;
        }
        flush(colacc, gcur, t0, kn);
    };

    // 1. the system keys into the tiles (every load of a round issued before its stores);
    //    the partials zeroed
    {
        constexpr int kStage = 8;
        const int nch = SB * 16 * GG::CPR;
        for (int x0 = 0; x0 < nch; x0 += kStage * kThreads) {
            u32x4 r[kStage];
#pragma unroll
            for (int i = 0; i < kStage; ++i) {
                const int c = min(x0 + i * kThreads + tid, nch - 1);
                r[i] = load16(kbase + (size_t)min(c / GG::CPR, s.Ns - 1) * D + (c % GG::CPR) * 8);
            }
#pragma unroll
            for (int i = 0; i < kStage; ++i) {
                const int c = x0 + i * kThreads + tid;
                if (c < nch) store16(sysk + (c / GG::CPR) * GG::ROWB + (c % GG::CPR) * 16, r[i]);
            }
        }
        for (int x = tid; x < 4 * s.G * TK; x += kThreads) part[x] = 0.f;
    }
    __syncthreads();

    // 2. system rows x system keys: the system rows' normalisers (C[key][row]: a lane owns row i)
    auto load_q = [&](bf16x8 (&f)[GG::KSTEPS], int g, int row) {
        const uint16_t* src = q_text + ((head0 + g) * s.Nt + row) * D + koff;
#pragma unroll
        for (int ks = 0; ks < GG::KSTEPS; ++ks) f[ks] = as_bf16x8(load16(src + ks * 32));
    };
    for (int item = wave; item < s.G * SB; item += 4) {
        const int g = item / SB, rb = item % SB;
        const int i = rb * 16 + (lane & 15);
        bf16x8 qs[GG::KSTEPS];
        load_q(qs, g, min(i, s.Ns - 1));
        float m = kNegInf, l = 0.f;
        for (int kb = 0; kb <= rb; ++kb) {
            bf16x8 kf[GG::KSTEPS];
            load_kfrag<D>(kf, sysk, kb, lane);
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < GG::KSTEPS; ++ks) acc = mfma16x16x32(kf[ks], qs[ks], acc);
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
        float dummy = 0.f;
#pragma unroll
        for (int off = 16; off < 64; off <<= 1) {
            const float m2 = shfl_xor(m, off), l2 = shfl_xor(l, off), d2 = shfl_xor(dummy, off);
            merge_stats(m, l, dummy, m2, l2, d2);
        }
        if (lane < 16 && i < s.Ns) {
            const float L2 = m + log2f(l);
            lse2s[g * s.Nt + i] = L2;
            lse[(head0 + g) * s.Nt + i] = L2 * kLn2;
        }
    }
    __syncthreads();

    // 3. column sums over the system keys: system rows (C[row][key]: a lane owns key j), then
    //    question rows from their registers (key blocks dealt over the key parts)
    for (int item = wave; item < s.G * SB; item += 4) {
        const int g = item / SB, rb = item % SB;
        bf16x8 qs[GG::KSTEPS];
        load_q(qs, g, min(rb * 16 + (lane & 15), s.Ns - 1));
        float l2[4];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) l2[jj] = lse2s[g * s.Nt + min(rb * 16 + (lane >> 4) * 4 + jj, s.Ns - 1)];
        for (int kb = 0; kb <= rb; ++kb) {
            bf16x8 kf[GG::KSTEPS];
            load_kfrag<D>(kf, sysk, kb, lane);
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < GG::KSTEPS; ++ks) acc = mfma16x16x32(qs[ks], kf[ks], acc);
            const int j = kb * 16 + (lane & 15);
            float col = 0.f;
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const int ii = rb * 16 + (lane >> 4) * 4 + jj;
                if (ii < s.Ns && j <= ii) col += fast_exp2(acc[jj] * s.scale2 - l2[jj]);
            }
            flush(col, g, kb * 16, s.Ns - kb * 16);
        }
    }
    for (int kb = kp; kb < SB; kb += KS) {
        bf16x8 kf[GG::KSTEPS];
        load_kfrag<D>(kf, sysk, kb, lane);
        qrow_block(kf, kSysBlock, kb * 16, s.Ns - kb * 16);
    }
    __syncthreads();  // the tiles are free for the question keys

    // 4. question rows x question keys, through the tile pipeline (one tile in flight: the
    //    pass is compute-paced here, and a second register tile would spill)
    const int qbeg = s.Ns + s.Nv;
    tile_pipeline<D, 1>(
        kbase, qbeg, s.N, tiles,
        [&](const char* buf, int key0, int) {
#pragma unroll
            for (int kb = 0; kb < kTile / 16; ++kb) {
                if (kb % KS != kp) continue;
                const int c0 = key0 - qbeg + kb * 16;
                if (c0 >= s.Nq) continue;  // the last tile's clamped keys
                bf16x8 kf[GG::KSTEPS];
                load_kfrag<D>(kf, buf, kb, lane);
                qrow_block(kf, c0, s.Ns + c0, s.Nq - c0);
            }
        },
        [](int, int) {});
    __syncthreads();

    // 5. the four waves' partials, in wave order
    for (int x = tid; x < s.G * s.Nt; x += kThreads) {
        const int g = x / s.Nt, j = x % s.Nt;
        float a = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) a += part[((size_t)w * s.G + g) * TK + j];
        ws_colsum[(head0 + g) * s.Nt + j] = a;
    }
}

// Column sums of the text->text probabilities for one 16-key block kb of query
// head g of a unit, by one wave, with every text row's normaliser given (natural
// log, lse [.., N_t] of the head): the items of a unit are independent, so each
// is its own wave and their latencies overlap.  C[row][key]: a lane owns key
// j = 16*kb + lane%16; the row fragments and the rows' normalisers of the next
// 16-row block are fetched while the current block is used.
template <int D>
__device__ void text_cols_item(const Shape& s, int bl, int kvh, int g, int kb, const uint16_t* __restrict__ q_text,
                               const uint16_t* __restrict__ k, const float* __restrict__ lse,
                               float* __restrict__ ws_colsum) {
    using GG = Geo<D>;
    const int lane = threadIdx.x & 63;
    const size_t head = (size_t)bl * s.H + kvh * s.G + g;
    const uint16_t* kbase = k + ((size_t)bl * s.Hkv + kvh) * (size_t)s.N * D;
    const int koff = (lane >> 4) * 8;
    const int TB = (s.Nt + 15) >> 4;
    const int j = kb * 16 + (lane & 15);
    const int jc = min(j, s.Nt - 1);
    const int pos = jc < s.Ns ? jc : jc + s.Nv;
    auto load_frag = [&](bf16x8 (&f)[GG::KSTEPS], const uint16_t* row) {
#pragma unroll
        for (int ks = 0; ks < GG::KSTEPS; ++ks) f[ks] = as_bf16x8(load16(row + koff + ks * 32));
    };
    auto qrow = [&](int rb) { return q_text + (head * s.Nt + min(rb * 16 + (lane & 15), s.Nt - 1)) * D; };
    // the normalisers of this lane's accumulator rows 16*rb + 4*(lane/16) + jj (clamped into the head)
    auto load_lse = [&](float (&l2)[4], int rb) {
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) l2[jj] = lse[head * s.Nt + min(rb * 16 + (lane >> 4) * 4 + jj, s.Nt - 1)];
    };
    bf16x8 kf[GG::KSTEPS], qa[GG::KSTEPS], qb[GG::KSTEPS];
    float la[4], lb[4];
    load_frag(kf, kbase + (size_t)pos * D);
    load_frag(qa, qrow(kb));
    load_lse(la, kb);
    float col = 0.f;
    auto step = [&](const bf16x8 (&qf)[GG::KSTEPS], const float (&l2)[4], int rb) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < GG::KSTEPS; ++ks) acc = mfma16x16x32(qf[ks], kf[ks], acc);
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int ii = rb * 16 + (lane >> 4) * 4 + jj;
            if (ii < s.Nt && j <= ii) col += fast_exp2(acc[jj] * s.scale2 - l2[jj] * kLog2e);
        }
    };
    // row blocks kb..TB-1; a block past the last is masked out by ii < N_t
    for (int rb = kb; rb < TB; rb += 2) {
        load_frag(qb, qrow(rb + 1));
        load_lse(lb, rb + 1);
        step(qa, la, rb);
        load_frag(qa, qrow(rb + 2));
        load_lse(la, rb + 2);
        step(qb, lb, rb + 1);
    }
    col = sum_xor32(sum_xor16(col));
    if (lane < 16 && j < s.Nt) ws_colsum[head * s.Nt + j] = col;
}

// Head means of one (sequence, layer, group): s^T (Eq. (9)), w and w~ (Eq. (7)),
// and for group 0 the layer's text->vision mass (Eq. (5)-(6)).  red: 256 floats of LDS.
__device__ inline void finalize_group(const Shape& s, int bl, int gi, const float* ws_colsum, const float* ws_vmh,
                                      float* s_txt, float* w_txt, float* tv_mass, float* red, bool with_mass = true) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h0 = s.head_mode == 0 ? 0 : gi * s.G;
    const int hn = s.head_mode == 0 ? s.H : s.G;
    const float inv = 1.0f / (float)hn;
    const float* cs = ws_colsum + ((size_t)bl * s.H + h0) * s.Nt;
    const size_t obase = ((size_t)bl * s.ngroups + gi) * s.Nt;
    // s^T[j]: the head mean of the column sums, eight heads' loads in flight per thread
    auto column = [&](int j) {
        float a[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        int h = 0;
        for (; h + 8 <= hn; h += 8) {
#pragma unroll
            for (int u = 0; u < 8; ++u) a[u] += cs[(size_t)(h + u) * s.Nt + j];
        }
        for (; h < hn; ++h) a[0] += cs[(size_t)h * s.Nt + j];
        return (((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]))) * inv;
    };
    constexpr int kCols = 4;  // columns per thread kept in registers
    float wv[kCols];
    const bool cached = s.Nt <= kCols * kThreads;
    float part = 0.f;
    if (cached) {
#pragma unroll
        for (int c = 0; c < kCols; ++c) {
            const int j = tid + c * kThreads;
            wv[c] = 0.f;
            if (j < s.Nt) {
                const float st = column(j);
                s_txt[obase + j] = st;
                wv[c] = st / (float)(s.Nt - j);
                part += wv[c];
            }
        }
    } else {
        for (int j = tid; j < s.Nt; j += kThreads) {
            const float st = column(j);
            s_txt[obase + j] = st;
            part += st / (float)(s.Nt - j);
        }
    }
    // W = sum_j w_j: within each wave, then over the waves in order
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) part += shfl_xor(part, off);
    if (lane == 0) red[wave] = part;
    __syncthreads();
    float W = 0.f;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) W += red[w];
    // the plain attention sum (Table 5) weighs every text row 1
    auto weight = [&](float w) { return s.vision_rank == 1 ? 1.f : (W > 0.f ? w / W : 0.f); };
    if (cached) {
#pragma unroll
        for (int c = 0; c < kCols; ++c) {
            const int j = tid + c * kThreads;
            if (j < s.Nt) w_txt[obase + j] = weight(wv[c]);
        }
    } else {
        __syncthreads();  // every s_txt store of the workgroup precedes the reads below
        for (int j = tid; j < s.Nt; j += kThreads) w_txt[obase + j] = weight(s_txt[obase + j] / (float)(s.Nt - j));
    }
    if (with_mass && gi == 0 && wave == 0) {
        // the layer's TV mass: the mean over all query heads of their vision masses
        float a = 0.f;
        if (s.Nt > 0)
            for (int h = lane; h < s.H; h += 64) a += ws_vmh[(size_t)bl * s.H + h];
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) a += shfl_xor(a, off);
        if (lane == 0) tv_mass[bl] = a / (float)s.H;
    }
    __syncthreads();
}

}  // namespace core
}  // namespace tgvkv
