/*
 * tgvkv.h -- C ABI of libtgvkv, the MI355X (gfx950) implementation of the
 * post-prefill KV eviction pass of TGV-KV ("Text-Grounded KV Eviction for
 * Vision-Language Models") and of single-query decode attention over the
 * pruned, per-layer ragged cache it produces.
 *
 * The pass runs once after prefill (Sec. 3.3):
 *   tgvkv_score   Text-Weighted Ranking scores and per-layer text->vision mass
 *                 (Eq. (2), (6)-(9));
 *   tgvkv_budget  Text-Vision Budgeting: integer per-layer budgets (Eq. (5)-(6));
 *   tgvkv_select  Text-Prioritised Retention: retained positions (Eq. (10));
 *   tgvkv_compact gather of the retained K/V rows into a ragged cache;
 * then every decode step appends one key/value and attends (Eq. (3)-(4)):
 *   tgvkv_decode_attn.
 * The same cache can instead live in fixed-size pages of a shared pool, for
 * serving with continuous batching: tgvkv_page_plan, tgvkv_page_table,
 * tgvkv_compact_paged, tgvkv_decode_attn_paged.
 *
 * Conventions shared by every call
 *  - Token layout of each sequence: n_sys system-text tokens, then n_vis vision
 *    tokens, then n_qst question-text tokens; N = n_sys + n_vis + n_qst.  The
 *    text set T (Eq. (10)) is positions [0, n_sys) U [n_sys + n_vis, N), in
 *    "text order" (system rows first); the vision set V is [n_sys, n_sys + n_vis).
 *  - All tensors are row-major, contiguous, device memory owned by the caller,
 *    16-byte aligned.  bf16 tensors are passed as raw 16-bit patterns.
 *  - Every call validates its arguments on the host before any HIP call; an
 *    invalid call returns a negative status and launches nothing.  Kernels are
 *    enqueued asynchronously on `stream`; the library never allocates, frees or
 *    synchronises, and keeps no pointer after a call returns.  A launch failure
 *    returns TGVKV_E_HIP.  Calls are thread-safe (no global mutable state), except
 *    that tgvkv_decode_attn_noalloc calls share one buffer per GPU (see there).
 *  - Query head h reads KV head h / (heads_q / heads_kv).
 *  - "groups" g: 1 when opts.head_mode == 0 (one retained set per sequence and
 *    layer, from attention averaged over all query heads), heads_kv when
 *    head_mode == 1 (one retained set per KV head, from the mean over the query
 *    heads sharing it).
 */
#ifndef TGVKV_H
#define TGVKV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TGVKV_ABI_VERSION 8

typedef enum tgvkv_status {
    TGVKV_OK = 0,
    TGVKV_E_INVAL = -1,        /* null pointer, negative size, inconsistent shape or option   */
    TGVKV_E_UNSUPPORTED = -2,  /* valid, but outside what these kernels implement (head_dim,
                                  sizes beyond the documented limits)                          */
    TGVKV_E_WORKSPACE = -3,    /* workspace missing or smaller than tgvkv_workspace_size()    */
    TGVKV_E_CAPACITY = -4,     /* budget above L*N, or decode step outside the reserve        */
    TGVKV_E_HIP = -5           /* a kernel launch failed                                      */
} tgvkv_status;

/* Shape of one batch of prefills.  head_dim must be 64 or 128.  Limits
 * (TGVKV_E_UNSUPPORTED beyond them): layers <= 512, N <= 2^24,
 * heads_q / heads_kv <= 16, and the text rows one KV head scores,
 * (heads_q / heads_kv) * (n_sys + n_qst), at most 16384.  heads_q must be a
 * multiple of heads_kv; every count is >= 0 and N >= 1 (TGVKV_E_INVAL). */
typedef struct tgvkv_problem {
    int32_t batch;
    int32_t layers;
    int32_t heads_q;
    int32_t heads_kv;
    int32_t head_dim;
    int32_t n_sys;
    int32_t n_vis;
    int32_t n_qst;
} tgvkv_problem;

/* Options.  Passing NULL selects the defaults (all 0: the paper's TGV-KV). */
typedef struct tgvkv_opts {
    float   sm_scale;    /* logit scale; <= 0 selects 1/sqrt(head_dim)                       */
    int32_t head_mode;   /* 0: per-layer retained set (paper); 1: per-KV-head retained sets  */
    int32_t n_sink;      /* first n_sink positions are always kept (App. A.2 keeps 4)         */
    int32_t n_recent;    /* last n_recent positions are always kept (App. A.2 keeps 1)        */
    int32_t vision_only; /* 0: evict among all tokens (TPR, Eq. (10)); 1: vision-only eviction
                            of App. B.3: every layer keeps all text, and the budget given to
                            tgvkv_budget counts vision tokens only (see there)                */
    /* The paper's variants (Table 1(a), Table 5), for ablations:                            */
    int32_t budget_rule; /* layer budgets in proportion to 0: the text->vision mass (TVB);
                            1: nothing (uniform); 2: the text->text mass, N_t - tv_mass      */
    int32_t vision_rank; /* vision importance 0: TWR, Eq. (8); 1: the plain text-row attention
                            sum s_vis[j] = sum_i Abar[i, n_sys + j] (w_txt is then all ones) */
    int32_t joint_rank;  /* 0: TPR, Eq. (10); 1: no TPR: forced tokens, then all others ranked
                            together, text by s_txt and vision by s_vis (times N_t under TWR,
                            whose weights sum to 1).  Not with vision_only.                  */
} tgvkv_opts;

/* Score phases (bit mask for tgvkv_score). */
enum {
    TGVKV_SCORE_STATS  = 1,  /* question-row softmax statistics over all visible keys        */
    TGVKV_SCORE_TEXT   = 2,  /* text scores s^T, weights w~, per-layer text->vision mass      */
    TGVKV_SCORE_VISION = 4,  /* text-weighted vision scores s^V                               */
    TGVKV_SCORE_ALL    = 7,
    TGVKV_SCORE_LSE_IN = 16  /* with exactly TEXT|VISION: lse is an input holding every text
                                row's normaliser, as a prefill attention kernel returns it;
                                the statistics sweep is skipped, the vision sweep also gives
                                each row's vision mass (so tv_mass), and K is read once.
                                Needs budgets_or_null == NULL (every layer gets s^V).        */
};

/* Which call a workspace is sized for. */
enum { TGVKV_CALL_SCORE = 0, TGVKV_CALL_DECODE = 1 };

/*
 * tgvkv_score -- TWR scores and TVB masses of every (sequence, layer).
 *
 * Rows of the causal softmax A = softmax(tau Q K^T + M) of Eq. (2) whose queries
 * are text tokens, tau = sm_scale.  Let Abar be A averaged over the query heads
 * of a group.  Then, per group:
 *   s_txt[j] = sum_{i >= j} Abar[i, pi(j)]                       (Eq. (9))
 *   w_j      = s_txt[j] / (N_t - j),  w_txt = w / sum(w)         (Eq. (7))
 *   s_vis[j] = sum_i w_txt[i] Abar[i, n_sys + j]                  (Eq. (8))
 * and per layer (always the mean over all query heads)
 *   tv_mass  = sum_{i in T, j in V} Abar[i, j]                    (Eq. (5)-(6)).
 *
 * q_text  bf16 [B][L][heads_q][N_t][head_dim]   text-row queries, text order
 * k       bf16 [B][L][heads_kv][N][head_dim]    cached keys (after any positional encoding)
 * lse     f32  [B][L][heads_q][N_t]  out (in with TGVKV_SCORE_LSE_IN): natural log-sum-exp of each
 *                                   text row's scaled logits over its visible keys
 * s_txt   f32  [B][L][g][N_t]        out
 * w_txt   f32  [B][L][g][N_t]        out (normalised weights; all 0 if sum(w) == 0)
 * tv_mass f32  [B][L]                out
 * s_vis   f32  [B][L][g][n_vis]      out
 * budgets_or_null  int32 [B][L]: if given, the VISION phase skips every layer
 *                  whose budget leaves no room for vision tokens (budget <=
 *                  |forced U T|, or <= |forced| with opts.joint_rank: the
 *                  vision threshold of tgvkv_sizes); s_vis of skipped layers is
 *                  left untouched.
 * phases  any non-empty OR of STATS, TEXT, VISION; or exactly TEXT|VISION|LSE_IN
 *         (see TGVKV_SCORE_LSE_IN).
 *         Phases must run in the order STATS, TEXT, VISION, with the same
 *         workspace and outputs; a later phase reads what the earlier ones left
 *         there.  Pointers of phases not requested may be NULL (lse is needed by
 *         all three, w_txt by VISION).
 * workspace / workspace_bytes  >= tgvkv_workspace_size(p, o, TGVKV_CALL_SCORE).
 */
tgvkv_status tgvkv_score(const tgvkv_problem* problem, const tgvkv_opts* opts, int32_t phases,
                         const void* q_text, const void* k,
                         float* lse, float* s_txt, float* w_txt, float* tv_mass, float* s_vis,
                         const int32_t* budgets_or_null,
                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * tgvkv_budget -- TVB: integer budgets b_l of every layer of every sequence.
 *
 * Eq. (5)-(6) give layer l the share m_l / sum_l' m_l' of the sequence budget.
 * Counts: a floor F = min(|forced|, total/L, N) per layer first; the rest
 * R = total - L*F water-filled in proportion to the shares with each layer
 * capped at N - F (uniform shares if all masses are 0; non-finite or negative
 * masses count as 0); then largest-remainder rounding with ties to the lower
 * layer.  float64 throughout.  sum_l b_l == total for every sequence.
 *
 * With opts.vision_only (App. B.3: all text kept, the retention ratio counts
 * vision tokens) every layer keeps its N_t text tokens and its F_v forced vision
 * positions; total_budget is the vision budget V_tot (e.g. round(rho * n_vis * L))
 * over the other vision tokens, shared out the same way with N replaced by
 * n_vis - F_v and no floor; layer l keeps b_l = N_t + F_v + v_l tokens, so
 * sum_l b_l == L*(N_t + F_v) + V_tot.
 *
 * tv_mass        f32   [B][L]     per-layer masses (from tgvkv_score)
 * total_budget   per-sequence budget B_tot (e.g. round(rho * N * L)), 0 <= B_tot <= L*N;
 *                with vision_only V_tot, 0 <= V_tot <= L*(n_vis - F_v)
 * decode_reserve token slots reserved after each layer's retained tokens for decode (>= 0)
 * budgets        int32 [B][L]     out
 * idx_offsets    int64 [B*L + 1]  out: start of each (b, l) block of tgvkv_select's output,
 *                                 block size g * b_l; idx_offsets[B*L] = B * K * g, where
 *                                 K = B_tot (K = L*(N_t + F_v) + V_tot with vision_only) is the
 *                                 number of tokens each sequence keeps
 * seg_offsets    int64 [B*L + 1]  out: start of each (b, l) cache segment, in units of
 *                                 heads_kv * head_dim elements; segment size b_l + reserve;
 *                                 seg_offsets[B*L] = B * (K + L * reserve)
 * unit_order_or_null int32 [B*L]  optional out: decode's dispatch order, longest segments
 *                                 first.  With r_b(l) the rank of layer l in sequence b by
 *                                 (b_l desc, l asc): unit_order[r_b(l) * B + b] = b*L + l.
 *                                 A permutation of [0, B*L); pass it to tgvkv_compact and
 *                                 tgvkv_decode_attn.
 */
tgvkv_status tgvkv_budget(const tgvkv_problem* problem, const tgvkv_opts* opts,
                          const float* tv_mass, int64_t total_budget, int32_t decode_reserve,
                          int32_t* budgets, int64_t* idx_offsets, int64_t* seg_offsets,
                          int32_t* unit_order_or_null, hipStream_t stream);

/*
 * tgvkv_select -- TPR: retained positions of every (sequence, layer, group), Eq. (10).
 *
 * Forced positions (first n_sink, last n_recent) first; then, if b_l minus the
 * forced count is at most the remaining text count, the top text tokens by
 * s_txt, else all text and the top vision tokens by s_vis.  With no forced
 * tokens this is exactly Eq. (10).  Ties go to the lower position; -0.0 equals
 * +0.0; scores must not be NaN.  Positions are written in ascending order:
 * idx[idx_offsets[b*L + l] + gi * b_l + n], n < b_l.
 *
 * s_vis  f32 [B][L][g][n_vis]; s_txt f32 [B][L][g][N_t]; budgets, idx_offsets from tgvkv_budget.
 * idx    int32 out, idx_offsets[B*L] entries.
 */
tgvkv_status tgvkv_select(const tgvkv_problem* problem, const tgvkv_opts* opts,
                          const float* s_vis, const float* s_txt, const int32_t* budgets,
                          const int64_t* idx_offsets, int32_t* idx, hipStream_t stream);

/*
 * tgvkv_compact -- gather the retained K/V rows into the ragged per-layer cache.
 *
 * The cache of Sec. 3.1 (K, V per layer) keeps only the retained tokens, in
 * ascending position: for every (b, l), KV head h and n < b_l,
 *   kc[(seg_offsets[b*L+l] * heads_kv + h * cap + n) * head_dim + :] = k[b][l][h][I[n]][:]
 * with cap = b_l + decode_reserve and I the (group of h's) retained set.  Same for v.
 * Bit-exact copy.  Slots b_l .. cap-1 are left for tgvkv_decode_attn.
 * total_budget / decode_reserve: the values given to tgvkv_budget (they size the
 * launch on the host: B * K rows per KV head are moved, K as in tgvkv_budget).
 * kc, vc  bf16, seg_offsets[B*L] * heads_kv * head_dim elements each.
 * unit_order_or_null  int32 [B*L], optional: dispatch order of the (sequence, layer) units,
 *         e.g. tgvkv_budget's longest-first order; as for tgvkv_decode_attn, the result does
 *         not depend on it, and it must be a permutation of [0, B*L).
 */
tgvkv_status tgvkv_compact(const tgvkv_problem* problem, const tgvkv_opts* opts,
                           const void* k, const void* v, const int32_t* idx,
                           const int32_t* budgets, const int64_t* idx_offsets,
                           const int64_t* seg_offsets, int64_t total_budget, int32_t decode_reserve,
                           void* kc, void* vc, const int32_t* unit_order_or_null, hipStream_t stream);

/*
 * tgvkv_decode_attn -- one decode step over the pruned cache, Eq. (3)-(4).
 *
 * For every (b, l): writes k_new / v_new at slot b_l + step of each KV head's
 * segment, then for each query head h computes
 *   out[b][l][h] = softmax_n(tau q[b][l][h] . Kc[n]) Vc[n],  n < b_l + step + 1.
 * Steps must run in order 0, 1, ... on the same cache; 0 <= step < decode_reserve.
 * Arithmetic: logits and sums in fp32.  Up to 2 query heads per KV head the products
 * are fp32 on the vector units; from 3 on they run on the matrix cores, with the
 * probabilities entering P V as a high and a low bf16 part (about 16 significant
 * bits), so results differ from the vector path in the last bits only.
 *
 * q      bf16 [B][L][heads_q][head_dim];  k_new, v_new bf16 [B][L][heads_kv][head_dim]
 * out    f32  [B][L][heads_q][head_dim]
 * workspace >= tgvkv_workspace_size(p, o, TGVKV_CALL_DECODE) (may be 0 bytes).
 * unit_order_or_null  int32 [B*L], optional: the order in which (sequence, layer) units
 *        are dispatched, e.g. tgvkv_budget's longest-first order.  Results do not depend
 *        on it (each unit's arithmetic is the same); it only shortens the tail of a
 *        launch whose segments differ in length.  It must be a permutation of [0, B*L):
 *        entries are clamped into that range, and a unit the order misses is not computed.
 */
tgvkv_status tgvkv_decode_attn(const tgvkv_problem* problem, const tgvkv_opts* opts,
                               void* kc, void* vc, const int32_t* budgets,
                               const int64_t* seg_offsets, int32_t decode_reserve, int32_t step,
                               const void* q, const void* k_new, const void* v_new, float* out,
                               void* workspace, size_t workspace_bytes, const int32_t* unit_order_or_null,
                               hipStream_t stream);

/*
 * tgvkv_decode_attn_noalloc -- tgvkv_decode_attn for callers that cannot allocate:
 * code under HIP graph capture, serving loops and harnesses that forbid hipMalloc.
 *
 * Same arguments, kernels and results as tgvkv_decode_attn, bit for bit, without the
 * workspace: when the token ranges are split (few (sequence, layer, KV head) units),
 * the split partials go to a static device buffer of the library, one per GPU, held
 * until the process ends.  The call allocates nothing.  The first call on a device
 * looks the buffer's address up with that device current.
 * Limit: the partials must fit in 16 MiB, i.e. tgvkv_workspace_size(p, o,
 * TGVKV_CALL_DECODE) <= 16 MiB (every shape these kernels split stays below 9 MiB);
 * above it TGVKV_E_WORKSPACE and nothing is launched.  Every element of the buffer
 * that a call reads it first writes itself, so nothing is cleared between calls.
 * Calls that overlap on one GPU (other streams or threads while one is in flight)
 * share that GPU's buffer and race: serialise them, or use tgvkv_decode_attn with a
 * workspace each.  Calls on different GPUs do not interact.
 */
tgvkv_status tgvkv_decode_attn_noalloc(const tgvkv_problem* problem, const tgvkv_opts* opts,
                                       void* kc, void* vc, const int32_t* budgets,
                                       const int64_t* seg_offsets, int32_t decode_reserve, int32_t step,
                                       const void* q, const void* k_new, const void* v_new, float* out,
                                       const int32_t* unit_order_or_null, hipStream_t stream);

/*
 * Paged cache, for serving with continuous batching.
 *
 * The retained rows of Eq. (10) and the rows decode appends (Eq. (3)-(4)) may
 * instead live in fixed-size pages of one pool shared by every sequence in
 * service, so a serving loop admits a newly evicted batch and retires finished
 * sequences without moving anyone else's cache.  A page holds page_size rows of
 * every KV head:
 *   k_pool, v_pool  bf16 [n_pages][heads_kv][page_size][head_dim]
 * and row n of (sequence b, layer l) is row n % page_size of page
 *   block_table[(b*L + l) * max_pages + n / page_size].
 * page_size is a power of two in [1, 4096] (TGVKV_E_INVAL otherwise); max_pages
 * is in [1, 4096] (TGVKV_E_UNSUPPORTED above); 1 <= n_pages <= 2^31 - 1.  A page
 * id outside [0, n_pages) (such as an unused entry's -1) is clamped into the
 * pool, so a wrong table gives wrong values but never addresses outside it.
 * Rows are bit-identical to tgvkv_compact's, and tgvkv_decode_attn_paged does
 * the same arithmetic as tgvkv_decode_attn, so the layouts give equal results.
 */

/* tgvkv_page_plan -- host-only sizes of a paged batch (no HIP call).
 * With the total_budget / decode_reserve given to tgvkv_budget:
 *   *max_pages_out  = ceil((b_max + decode_reserve) / page_size), the table width
 *                     every segment fits in, b_max the largest budget one layer can
 *                     get (min(N, B_tot); N_t + F_v + min(n_vis - F_v, V_tot) with
 *                     vision_only), at least 1;
 *   *pool_pages_out = floor((B*K + B*L*(decode_reserve + page_size - 1)) / page_size),
 *                     an upper bound on the pages tgvkv_page_table takes (K as in
 *                     tgvkv_budget).
 * TGVKV_E_UNSUPPORTED if the width exceeds 4096. */
tgvkv_status tgvkv_page_plan(const tgvkv_problem* problem, const tgvkv_opts* opts, int64_t total_budget,
                             int32_t decode_reserve, int32_t page_size, int32_t* max_pages_out,
                             int64_t* pool_pages_out);

/* tgvkv_page_table -- give every (sequence, layer) of a batch its pages.
 * Segment i = b*L + l needs n_i = ceil((budgets[i] + decode_reserve) / page_size)
 * pages; they are the next entries of free_pages in order of i:
 *   block_table[i * max_pages + j] = free_pages[P_i + j] for j < n_i, P_i = sum_{i'<i} n_i',
 *   block_table[i * max_pages + j] = -1 for n_i <= j < max_pages,
 * and *pages_used = sum_i n_i (the caller drops that many ids from its free list).
 * budgets      int32 [B][L] from tgvkv_budget (same total_budget, decode_reserve)
 * free_pages   int32 [n_free] device, distinct page ids; n_free must be at least
 *              tgvkv_page_plan's pool bound and max_pages at least its width
 *              (TGVKV_E_CAPACITY otherwise)
 * block_table  int32 [B*L][max_pages] out;  pages_used  int64 device scalar out
 * With batch == 0 nothing is launched and *pages_used is not written. */
tgvkv_status tgvkv_page_table(const tgvkv_problem* problem, const tgvkv_opts* opts, const int32_t* budgets,
                              int64_t total_budget, int32_t decode_reserve, int32_t page_size,
                              const int32_t* free_pages, int64_t n_free, int32_t* block_table, int32_t max_pages,
                              int64_t* pages_used, hipStream_t stream);

/* tgvkv_compact_paged -- tgvkv_compact into the pages of block_table: row n < b_l
 * of (b, l), KV head h goes to k_pool[page][h][n % page_size][:] with page the
 * table entry n / page_size.  Rows b_l .. are left for tgvkv_decode_attn_paged.
 * TGVKV_E_CAPACITY if max_pages is below ceil(b_max / page_size).  unit_order_or_null as
 * for tgvkv_compact. */
tgvkv_status tgvkv_compact_paged(const tgvkv_problem* problem, const tgvkv_opts* opts, const void* k, const void* v,
                                 const int32_t* idx, const int32_t* budgets, const int64_t* idx_offsets,
                                 int64_t total_budget, const int32_t* block_table, int32_t max_pages,
                                 int32_t page_size, void* k_pool, void* v_pool, int64_t n_pages,
                                 const int32_t* unit_order_or_null, hipStream_t stream);

/* tgvkv_decode_attn_paged -- one decode step of a continuous batch over the paged cache.
 * Each sequence b is at its own step steps[b] (int32 [B], device): for every layer
 * it writes k_new / v_new at row budgets[b*L+l] + steps[b] of its pages and
 * attends over rows n < budgets[b*L+l] + steps[b] + 1, as tgvkv_decode_attn does.
 * A sequence whose step is outside [0, decode_reserve) (finished, or an empty slot)
 * is skipped: its pages and its rows of out are not touched.  The batch may mix
 * sequences from different prefill batches: only batch, layers, heads and
 * head_dim of `problem` are used, and budgets / block_table rows are the
 * callers' concatenation.  A segment's table row must cover its
 * ceil((b_l + steps[b] + 1) / page_size) pages (tgvkv_page_table's do).
 * Workspace: tgvkv_workspace_size(p, o, TGVKV_CALL_DECODE).  unit_order_or_null as for
 * tgvkv_decode_attn (a permutation of this batch's [0, B*L)). */
tgvkv_status tgvkv_decode_attn_paged(const tgvkv_problem* problem, const tgvkv_opts* opts, void* k_pool,
                                     void* v_pool, int64_t n_pages, int32_t page_size, const int32_t* block_table,
                                     int32_t max_pages, const int32_t* budgets, int32_t decode_reserve,
                                     const int32_t* steps, const void* q, const void* k_new, const void* v_new,
                                     float* out, void* workspace, size_t workspace_bytes,
                                     const int32_t* unit_order_or_null, hipStream_t stream);

/* tgvkv_sizes -- host-only sizes that follow from the problem and options (no HIP call).
 * With the total_budget given to tgvkv_budget:
 *   *kept_out              K, the tokens each sequence keeps over its layers: B_tot, or
 *                          L*(N_t + F_v) + V_tot with vision_only (App. B.3).  One
 *                          sequence's tgvkv_select output holds g * K positions, and its
 *                          compacted cache K + L * decode_reserve rows per KV head;
 *   *vision_threshold_out  a layer's vision scores are needed, and tgvkv_score given
 *                          budgets computes them, only when its budget exceeds this:
 *                          |forced U T| (Eq. (10) takes text first), or |forced| with
 *                          opts.joint_rank.
 * Either output may be NULL.  TGVKV_E_INVAL for a negative total_budget,
 * TGVKV_E_CAPACITY above what tgvkv_budget accepts. */
tgvkv_status tgvkv_sizes(const tgvkv_problem* problem, const tgvkv_opts* opts, int64_t total_budget,
                         int64_t* kept_out, int32_t* vision_threshold_out);

/* Workspace bytes needed by tgvkv_score (which = TGVKV_CALL_SCORE) or
 * tgvkv_decode_attn / tgvkv_decode_attn_paged (TGVKV_CALL_DECODE); 0 for an invalid problem. */
size_t tgvkv_workspace_size(const tgvkv_problem* problem, const tgvkv_opts* opts, int32_t which);

/* Static, NUL-terminated description of a status code. */
const char* tgvkv_status_string(tgvkv_status status);

/* TGVKV_ABI_VERSION of the library. */
int32_t tgvkv_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TGVKV_H */
