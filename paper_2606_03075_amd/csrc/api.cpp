// libtgvkv C ABI: argument validation on the host, workspace layout, launches.
//
// Every entry point checks its arguments before touching the HIP runtime, so an
// invalid call returns a negative status and enqueues nothing.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>

#include "tgvkv.h"
#include "tgvkv_shape.h"

using tgvkv::RowPlan;
using tgvkv::Shape;

namespace {

constexpr int32_t kMaxLayers = 512;
constexpr int64_t kMaxTokens = int64_t(1) << 24;
constexpr int64_t kMaxTextRowsPerKvHead = 16384;  // LDS row-normaliser buffer of the text pass
constexpr int32_t kMaxGroup = 16;                  // query heads per KV head (decode registers)
constexpr int64_t kMaxBlocks = (int64_t(1) << 31) - 1;
constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

tgvkv_status make_shape(const tgvkv_problem* p, const tgvkv_opts* o, Shape* s) {
    if (p == nullptr || s == nullptr) return TGVKV_E_INVAL;
    tgvkv_opts d;
    std::memset(&d, 0, sizeof(d));
    if (o != nullptr) d = *o;
    if (p->batch < 0 || p->layers < 1 || p->heads_q < 1 || p->heads_kv < 1 || p->n_sys < 0 || p->n_vis < 0 ||
        p->n_qst < 0)
        return TGVKV_E_INVAL;
    if (p->heads_q % p->heads_kv != 0) return TGVKV_E_INVAL;
    const int64_t N = (int64_t)p->n_sys + p->n_vis + p->n_qst;
    if (N < 1) return TGVKV_E_INVAL;
    if (d.head_mode != 0 && d.head_mode != 1) return TGVKV_E_INVAL;
    if (d.n_sink < 0 || d.n_recent < 0) return TGVKV_E_INVAL;
    if (d.vision_only != 0 && d.vision_only != 1) return TGVKV_E_INVAL;
    if (d.budget_rule < 0 || d.budget_rule > 2 || d.vision_rank < 0 || d.vision_rank > 1 || d.joint_rank < 0 ||
        d.joint_rank > 1 || (d.vision_only && d.joint_rank))
        return TGVKV_E_INVAL;
    if (!std::isfinite(d.sm_scale)) return TGVKV_E_INVAL;
    if (p->head_dim != 64 && p->head_dim != 128) return TGVKV_E_UNSUPPORTED;
    if (p->layers > kMaxLayers || N > kMaxTokens) return TGVKV_E_UNSUPPORTED;
    const int64_t G = p->heads_q / p->heads_kv;
    if (G * ((int64_t)p->n_sys + p->n_qst) > kMaxTextRowsPerKvHead) return TGVKV_E_UNSUPPORTED;
    if (G > kMaxGroup) return TGVKV_E_UNSUPPORTED;
    if ((int64_t)p->batch * p->layers * p->heads_q * 8 > kMaxBlocks) return TGVKV_E_UNSUPPORTED;

    s->B = p->batch;
    s->L = p->layers;
    s->H = p->heads_q;
    s->Hkv = p->heads_kv;
    s->D = p->head_dim;
    s->G = (int32_t)G;
    s->Ns = p->n_sys;
    s->Nv = p->n_vis;
    s->Nq = p->n_qst;
    s->N = (int32_t)N;
    s->Nt = p->n_sys + p->n_qst;
    s->head_mode = d.head_mode;
    s->ngroups = d.head_mode == 0 ? 1 : p->heads_kv;
    s->n_sink = d.n_sink;
    s->n_recent = d.n_recent;
    s->vision_only = d.vision_only;
    s->budget_rule = d.budget_rule;
    s->vision_rank = d.vision_rank;
    s->joint_rank = d.joint_rank;
    s->sm_scale = d.sm_scale > 0.f ? d.sm_scale : 1.0f / std::sqrt((float)p->head_dim);
    s->scale2 = s->sm_scale * 1.4426950408889634f;
    return TGVKV_OK;
}

// |forced|: the first n_sink and the last n_recent positions.
int32_t forced_count(const Shape& s) {
    const int64_t fs = std::min<int64_t>(s.n_sink, s.N);
    const int64_t fr = std::max<int64_t>(s.N - (int64_t)s.n_recent, fs);
    return (int32_t)(fs + (s.N - fr));
}

// Forced positions that are vision tokens.
int32_t forced_vision_count(const Shape& s) {
    const int64_t fs = std::min<int64_t>(s.n_sink, s.N);
    const int64_t fr = std::max<int64_t>(s.N - (int64_t)s.n_recent, fs);
    const int64_t v0 = s.Ns, v1 = (int64_t)s.Ns + s.Nv;
    int64_t fv = 0;
    fv += std::max<int64_t>(0, std::min(fs, v1) - v0);
    fv += std::max<int64_t>(0, v1 - std::max(fr, v0));
    return (int32_t)fv;
}

// |forced U T|.
int32_t forced_or_text_count(const Shape& s) { return s.Nt + forced_vision_count(s); }

// A layer needs vision scores only when its budget exceeds this: |forced U T| with TPR
// (vision tokens compete only once all text is kept), |forced| when ranked jointly.
int32_t vision_threshold(const Shape& s) { return s.joint_rank ? forced_count(s) : forced_or_text_count(s); }

// Vision-only eviction (App. B.3): every layer keeps its text and its forced vision
// positions; the budget shares out the other vision tokens.
int32_t always_kept(const Shape& s) { return s.vision_only ? forced_or_text_count(s) : 0; }

// Largest valid total_budget per sequence, and the tokens each sequence keeps for it.
int64_t budget_capacity(const Shape& s) {
    return (int64_t)s.L * (s.vision_only ? s.Nv - forced_vision_count(s) : s.N);
}
int64_t kept_per_sequence(const Shape& s, int64_t total_budget) {
    return total_budget + (int64_t)s.L * always_kept(s);
}

struct ScoreWs {
    float* vm;
    float* colsum;
    float* vmh;
    float* part;
    size_t bytes;
};

ScoreWs score_workspace(const Shape& s, const RowPlan& rp, void* base) {
    const size_t bl = (size_t)s.B * s.L;
    size_t off = 0;
    ScoreWs w;
    char* b = static_cast<char*>(base);
    w.vm = reinterpret_cast<float*>(b ? b + off : nullptr);  // [vision splits][B*L*H][N_q] row masses
    off = align_up(off + sizeof(float) * bl * s.H * s.Nq * (size_t)tgvkv::vision_splits(s, rp));
    w.colsum = reinterpret_cast<float*>(b ? b + off : nullptr);
    off = align_up(off + sizeof(float) * bl * s.H * s.Nt);
    w.vmh = reinterpret_cast<float*>(b ? b + off : nullptr);
    off = align_up(off + sizeof(float) * bl * s.H);
    w.part = reinterpret_cast<float*>(b ? b + off : nullptr);
    off = align_up(off + sizeof(float) * bl * s.Hkv * (size_t)std::max(rp.rowgroups, 1) * s.Nv);
    w.bytes = off;
    return w;
}

size_t decode_workspace_bytes(const Shape& s) {
    const int ns = tgvkv::decode_splits(s);
    if (ns <= 1) return 0;
    return align_up(sizeof(float) * (size_t)s.B * s.L * s.H * ns * (s.D + 2));
}

// Paged cache limits: page_size and max_pages bound the LDS copy of a segment's page ids.
constexpr int32_t kMaxPageSize = 4096;
constexpr int32_t kMaxTablePages = 4096;

// log2(page_size), or -1 unless page_size is a power of two in [1, kMaxPageSize].
int32_t page_shift(int32_t page_size) {
    if (page_size < 1 || page_size > kMaxPageSize || (page_size & (page_size - 1)) != 0) return -1;
    int32_t sh = 0;
    while ((1 << sh) < page_size) ++sh;
    return sh;
}

// Largest b_l a layer can get for this total_budget (every b_l <= N and sum_l b_l = total).
int64_t max_layer_budget(const Shape& s, int64_t total_budget) {
    if (s.vision_only) return always_kept(s) + std::min<int64_t>(s.Nv - forced_vision_count(s), total_budget);
    return std::min<int64_t>(s.N, total_budget);
}

// Table width and pool pages (upper bound) of a batch: sum_i ceil((b_i + R) / P) <=
// (sum_i b_i + B*L*(R + P - 1)) / P.
void page_plan(const Shape& s, int64_t total_budget, int32_t reserve, int32_t page_size, int64_t* width,
               int64_t* pool) {
    *width = (max_layer_budget(s, total_budget) + reserve + page_size - 1) / page_size;
    *pool = ((int64_t)s.B * kept_per_sequence(s, total_budget) + (int64_t)s.B * s.L * (reserve + page_size - 1)) /
            page_size;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

tgvkv_status hip_status(hipError_t e) { return e == hipSuccess ? TGVKV_OK : TGVKV_E_HIP; }

}  // namespace

extern "C" {

int32_t tgvkv_abi_version(void) { return TGVKV_ABI_VERSION; }

const char* tgvkv_status_string(tgvkv_status st) {
    switch (st) {
        case TGVKV_OK: return "ok";
        case TGVKV_E_INVAL: return "invalid argument";
        case TGVKV_E_UNSUPPORTED: return "unsupported problem (head_dim or size limit)";
        case TGVKV_E_WORKSPACE: return "workspace missing or too small";
        case TGVKV_E_CAPACITY: return "budget or decode step exceeds the cache capacity";
        case TGVKV_E_HIP: return "HIP launch failed";
    }
    return "unknown status";
}

size_t tgvkv_workspace_size(const tgvkv_problem* problem, const tgvkv_opts* opts, int32_t which) {
    Shape s;
    if (make_shape(problem, opts, &s) != TGVKV_OK) return 0;
    if (which == TGVKV_CALL_SCORE) return score_workspace(s, tgvkv::plan_question_rows(s), nullptr).bytes;
    if (which == TGVKV_CALL_DECODE) return decode_workspace_bytes(s);
    return 0;
}

tgvkv_status tgvkv_score(const tgvkv_problem* problem, const tgvkv_opts* opts, int32_t phases, const void* q_text,
                         const void* k, float* lse, float* s_txt, float* w_txt, float* tv_mass, float* s_vis,
                         const int32_t* budgets_or_null, void* workspace, size_t workspace_bytes,
                         hipStream_t stream) {
    Shape s;
    tgvkv_status st = make_shape(problem, opts, &s);
    if (st != TGVKV_OK) return st;
    const bool lse_in = (phases & TGVKV_SCORE_LSE_IN) != 0;
    phases &= ~TGVKV_SCORE_LSE_IN;
    if (phases < 1 || phases > TGVKV_SCORE_ALL) return TGVKV_E_INVAL;
    // given normalisers: text and vision scores and the TV mass in one pass, for every layer
    if (lse_in && (phases != (TGVKV_SCORE_TEXT | TGVKV_SCORE_VISION) || budgets_or_null != nullptr))
        return TGVKV_E_INVAL;
    if (lse_in && (int64_t)s.B * s.L * s.H * ((s.Nt + 15) / 16) > kMaxBlocks) return TGVKV_E_UNSUPPORTED;
    if (s.B == 0) return TGVKV_OK;
    const bool text_rows = s.Nt > 0;
    if (q_text == nullptr && text_rows) return TGVKV_E_INVAL;
    if (k == nullptr || (lse == nullptr && text_rows)) return TGVKV_E_INVAL;
    if ((phases & TGVKV_SCORE_TEXT) && (tv_mass == nullptr || (text_rows && (s_txt == nullptr || w_txt == nullptr))))
        return TGVKV_E_INVAL;
    if ((phases & TGVKV_SCORE_VISION) && s.Nv > 0 && (s_vis == nullptr || (text_rows && w_txt == nullptr)))
        return TGVKV_E_INVAL;
    if (!aligned16(q_text) || !aligned16(k)) return TGVKV_E_INVAL;
    const RowPlan rp = tgvkv::plan_question_rows(s);
    if ((int64_t)s.B * s.L * s.Hkv * std::max(rp.rowgroups, 1) > kMaxBlocks) return TGVKV_E_UNSUPPORTED;
    const ScoreWs need = score_workspace(s, rp, nullptr);
    if (workspace == nullptr || workspace_bytes < need.bytes) return TGVKV_E_WORKSPACE;
    const ScoreWs w = score_workspace(s, rp, workspace);
    const uint16_t* q = static_cast<const uint16_t*>(q_text);
    const uint16_t* kk = static_cast<const uint16_t*>(k);
    const int32_t vthr = vision_threshold(s);

    hipError_t e = hipSuccess;
    if (lse_in) {
        e = tgvkv::launch_score_text(s, q, kk, lse, w.vm, w.colsum, w.vmh, true, stream);
        if (e == hipSuccess) e = tgvkv::launch_score_fin(s, w.colsum, w.vmh, s_txt, w_txt, tv_mass, false, stream);
        if (e == hipSuccess)
            e = tgvkv::launch_score_vision(s, rp, q, kk, lse, w_txt, nullptr, vthr, w.part, w.vm, stream);
        if (e == hipSuccess) e = tgvkv::launch_score_vis_reduce(s, rp, w.part, nullptr, vthr, s_vis, stream);
        if (e == hipSuccess) e = tgvkv::launch_score_mass(s, rp, w.vm, w.vmh, tv_mass, stream);
        return hip_status(e);
    }
    const bool both = (phases & TGVKV_SCORE_STATS) && (phases & TGVKV_SCORE_TEXT);
    if (both && tgvkv::stats_text_eligible(s, rp)) {
        e = tgvkv::launch_score_stats_text(s, rp, q, kk, lse, w.vm, w.colsum, w.vmh, stream);
        if (e == hipSuccess) e = tgvkv::launch_score_fin(s, w.colsum, w.vmh, s_txt, w_txt, tv_mass, true, stream);
    } else {
        if (phases & TGVKV_SCORE_STATS) e = tgvkv::launch_score_stats(s, rp, q, kk, lse, w.vm, stream);
        if ((phases & TGVKV_SCORE_TEXT) && e == hipSuccess) {
            e = tgvkv::launch_score_text(s, q, kk, lse, w.vm, w.colsum, w.vmh, false, stream);
            if (e == hipSuccess) e = tgvkv::launch_score_fin(s, w.colsum, w.vmh, s_txt, w_txt, tv_mass, true, stream);
        }
    }
    if ((phases & TGVKV_SCORE_VISION) && e == hipSuccess && s.Nv > 0) {
        e = tgvkv::launch_score_vision(s, rp, q, kk, lse, w_txt, budgets_or_null, vthr, w.part, nullptr, stream);
        if (e == hipSuccess) e = tgvkv::launch_score_vis_reduce(s, rp, w.part, budgets_or_null, vthr, s_vis, stream);
    }
    return hip_status(e);
}

tgvkv_status tgvkv_budget(const tgvkv_problem* problem, const tgvkv_opts* opts, const float* tv_mass,
                          int64_t total_budget, int32_t decode_reserve, int32_t* budgets, int64_t* idx_offsets,
                          int64_t* seg_offsets, int32_t* unit_order_or_null, hipStream_t stream) {
    Shape s;
    tgvkv_status st = make_shape(problem, opts, &s);
    if (st != TGVKV_OK) return st;
    if (decode_reserve < 0 || total_budget < 0) return TGVKV_E_INVAL;
    if (total_budget > budget_capacity(s)) return TGVKV_E_CAPACITY;
    if (idx_offsets == nullptr || seg_offsets == nullptr) return TGVKV_E_INVAL;
    if (s.B > 0 && (tv_mass == nullptr || budgets == nullptr)) return TGVKV_E_INVAL;
    const int64_t seg_total = (int64_t)s.B * (kept_per_sequence(s, total_budget) + (int64_t)s.L * decode_reserve);
    if (seg_total > (int64_t(1) << 40)) return TGVKV_E_UNSUPPORTED;
    if (s.B == 0) return TGVKV_OK;
    // vision-only eviction (App. B.3): the budget is shared out over the vision tokens that
    // are not forced, and every layer also keeps its text and forced vision positions
    const int32_t cap = s.vision_only ? s.Nv - forced_vision_count(s) : s.N;
    const int32_t add = always_kept(s);
    const int32_t floor_n = s.vision_only ? 0 : forced_count(s);
    return hip_status(tgvkv::launch_budget(s, tv_mass, total_budget, cap, add, decode_reserve, floor_n, budgets,
                                           idx_offsets, seg_offsets, unit_order_or_null, stream));
}

tgvkv_status tgvkv_select(const tgvkv_problem* problem, const tgvkv_opts* opts, const float* s_vis,
                          const float* s_txt, const int32_t* budgets, const int64_t* idx_offsets, int32_t* idx,
                          hipStream_t stream) {
    Shape s;
    tgvkv_status st = make_shape(problem, opts, &s);
    if (st != TGVKV_OK) return st;
    if (s.B == 0) return TGVKV_OK;
    if (budgets == nullptr || idx_offsets == nullptr || idx == nullptr) return TGVKV_E_INVAL;
    if ((s.Nv > 0 && s_vis == nullptr) || (s.Nt > 0 && s_txt == nullptr)) return TGVKV_E_INVAL;
    if ((int64_t)s.B * s.L * s.ngroups > kMaxBlocks) return TGVKV_E_UNSUPPORTED;
    return hip_status(tgvkv::launch_select(s, s_vis, s_txt, budgets, idx_offsets, idx, stream));
}

tgvkv_status tgvkv_compact(const tgvkv_problem* problem, const tgvkv_opts* opts, const void* k, const void* v,
                           const int32_t* idx, const int32_t* budgets, const int64_t* idx_offsets,
                           const int64_t* seg_offsets, int64_t total_budget, int32_t decode_reserve, void* kc,
                           void* vc, const int32_t* unit_order_or_null, hipStream_t stream) {
    Shape s;
    tgvkv_status st = make_shape(problem, opts, &s);
    if (st != TGVKV_OK) return st;
    if (decode_reserve < 0 || total_budget < 0) return TGVKV_E_INVAL;
    if (total_budget > budget_capacity(s)) return TGVKV_E_CAPACITY;
    const int64_t kept = kept_per_sequence(s, total_budget);
    if (s.B == 0 || kept == 0) return TGVKV_OK;
    if (k == nullptr || v == nullptr || idx == nullptr || budgets == nullptr || idx_offsets == nullptr ||
        seg_offsets == nullptr || kc == nullptr || vc == nullptr)
        return TGVKV_E_INVAL;
    if (!aligned16(k) || !aligned16(v) || !aligned16(kc) || !aligned16(vc)) return TGVKV_E_INVAL;
    const int64_t rows = (int64_t)s.B * kept;
    if ((int64_t)s.B * s.L * s.Hkv * 16 > kMaxBlocks) return TGVKV_E_UNSUPPORTED;
    return hip_status(tgvkv::launch_compact(s, static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), idx,
                                            budgets, idx_offsets, seg_offsets, decode_reserve, rows,
                                            unit_order_or_null, static_cast<uint16_t*>(kc),
                                            static_cast<uint16_t*>(vc), stream));
}

tgvkv_status tgvkv_decode_attn(const tgvkv_problem* problem, const tgvkv_opts* opts, void* kc, void* vc,
                               const int32_t* budgets, const int64_t* seg_offsets, int32_t decode_reserve,
                               int32_t step, const void* q, const void* k_new, const void* v_new, float* out,
                               void* workspace, size_t workspace_bytes, const int32_t* unit_order_or_null,
                               hipStream_t stream) {
    Shape s;
    tgvkv_status st = make_shape(problem, opts, &s);
    if (st != TGVKV_OK) return st;
    if (decode_reserve < 0) return TGVKV_E_INVAL;
    if (step < 0 || step >= decode_reserve) return TGVKV_E_CAPACITY;
    if (s.B == 0) return TGVKV_OK;
    if (kc == nullptr || vc == nullptr || budgets == nullptr || seg_offsets == nullptr || q == nullptr ||
        k_new == nullptr || v_new == nullptr || out == nullptr)
        return TGVKV_E_INVAL;
    if (!aligned16(kc) || !aligned16(vc) || !aligned16(q) || !aligned16(k_new) || !aligned16(v_new))
        return TGVKV_E_INVAL;
    const size_t need = decode_workspace_bytes(s);
    if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return TGVKV_E_WORKSPACE;
    return hip_status(tgvkv::launch_decode(s, static_cast<uint16_t*>(kc), static_cast<uint16_t*>(vc), budgets,
                                           seg_offsets, decode_reserve, step, static_cast<const uint16_t*>(q),
                                           static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new),
                                           out, static_cast<float*>(workspace), unit_order_or_null, stream));
}

tgvkv_status tgvkv_decode_attn_noalloc(const tgvkv_problem* problem, const tgvkv_opts* opts, void* kc, void* vc,
                                       const int32_t* budgets, const int64_t* seg_offsets, int32_t decode_reserve,
                                       int32_t step, const void* q, const void* k_new, const void* v_new, float* out,
                                       const int32_t* unit_order_or_null, hipStream_t stream) {
    Shape s;
    tgvkv_status st = make_shape(problem, opts, &s);
    if (st != TGVKV_OK) return st;
    if (decode_reserve < 0) return TGVKV_E_INVAL;
    if (step < 0 || step >= decode_reserve) return TGVKV_E_CAPACITY;
    if (s.B == 0) return TGVKV_OK;
    if (kc == nullptr || vc == nullptr || budgets == nullptr || seg_offsets == nullptr || q == nullptr ||
        k_new == nullptr || v_new == nullptr || out == nullptr)
        return TGVKV_E_INVAL;
    if (!aligned16(kc) || !aligned16(vc) || !aligned16(q) || !aligned16(k_new) || !aligned16(v_new))
        return TGVKV_E_INVAL;
    const size_t need = decode_workspace_bytes(s);
    if (need > tgvkv::kDecodeScratchBytes) return TGVKV_E_WORKSPACE;
    float* ws = nullptr;
    if (need > 0) {
        const hipError_t e = tgvkv::decode_scratch(&ws);
        if (e != hipSuccess) return TGVKV_E_HIP;
    }
    return hip_status(tgvkv::launch_decode(s, static_cast<uint16_t*>(kc), static_cast<uint16_t*>(vc), budgets,
                                           seg_offsets, decode_reserve, step, static_cast<const uint16_t*>(q),
                                           static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new),
                                           out, ws, unit_order_or_null, stream));
}

tgvkv_status tgvkv_page_plan(const tgvkv_problem* problem, const tgvkv_opts* opts, int64_t total_budget,
                             int32_t decode_reserve, int32_t page_size, int32_t* max_pages_out,
                             int64_t* pool_pages_out) {
    Shape s;
    tgvkv_status st = make_shape(problem, opts, &s);
    if (st != TGVKV_OK) return st;
    if (max_pages_out == nullptr || pool_pages_out == nullptr) return TGVKV_E_INVAL;
    if (decode_reserve < 0 || total_budget < 0 || page_shift(page_size) < 0) return TGVKV_E_INVAL;
    if (total_budget > budget_capacity(s)) return TGVKV_E_CAPACITY;
    int64_t width, pool;
    page_plan(s, total_budget, decode_reserve, page_size, &width, &pool);
    if (width > kMaxTablePages) return TGVKV_E_UNSUPPORTED;
    *max_pages_out = (int32_t)std::max<int64_t>(width, 1);
    *pool_pages_out = pool;
    return TGVKV_OK;
}

tgvkv_status tgvkv_sizes(const tgvkv_problem* problem, const tgvkv_opts* opts, int64_t total_budget,
                         int64_t* kept_out, int32_t* vision_threshold_out) {
    Shape s;
    tgvkv_status st = make_shape(problem, opts, &s);
    if (st != TGVKV_OK) return st;
    if (total_budget < 0) return TGVKV_E_INVAL;
    if (total_budget > budget_capacity(s)) return TGVKV_E_CAPACITY;
    if (kept_out != nullptr) *kept_out = kept_per_sequence(s, total_budget);
    if (vision_threshold_out != nullptr) *vision_threshold_out = vision_threshold(s);
    return TGVKV_OK;
}

tgvkv_status tgvkv_page_table(const tgvkv_problem* problem, const tgvkv_opts* opts, const int32_t* budgets,
                              int64_t total_budget, int32_t decode_reserve, int32_t page_size,
                              const int32_t* free_pages, int64_t n_free, int32_t* block_table, int32_t max_pages,
                              int64_t* pages_used, hipStream_t stream) {
    Shape s;
    tgvkv_status st = make_shape(problem, opts, &s);
    if (st != TGVKV_OK) return st;
    const int32_t sh = page_shift(page_size);
    if (decode_reserve < 0 || total_budget < 0 || sh < 0 || n_free < 0 || max_pages < 1) return TGVKV_E_INVAL;
    if (max_pages > kMaxTablePages) return TGVKV_E_UNSUPPORTED;
    if (total_budget > budget_capacity(s)) return TGVKV_E_CAPACITY;
    if (pages_used == nullptr) return TGVKV_E_INVAL;
    if (s.B > 0 && (budgets == nullptr || block_table == nullptr || (n_free > 0 && free_pages == nullptr)))
        return TGVKV_E_INVAL;
    int64_t width, pool;
    page_plan(s, total_budget, decode_reserve, page_size, &width, &pool);
    if (width > max_pages || pool > n_free) return TGVKV_E_CAPACITY;
    if (s.B == 0) return TGVKV_OK;
    return hip_status(tgvkv::launch_page_table(s, budgets, decode_reserve, sh, free_pages, n_free, block_table,
                                               max_pages, pages_used, stream));
}

tgvkv_status tgvkv_compact_paged(const tgvkv_problem* problem, const tgvkv_opts* opts, const void* k, const void* v,
                                 const int32_t* idx, const int32_t* budgets, const int64_t* idx_offsets,
                                 int64_t total_budget, const int32_t* block_table, int32_t max_pages,
                                 int32_t page_size, void* k_pool, void* v_pool, int64_t n_pages,
                                 const int32_t* unit_order_or_null, hipStream_t stream) {
    Shape s;
    tgvkv_status st = make_shape(problem, opts, &s);
    if (st != TGVKV_OK) return st;
    const int32_t sh = page_shift(page_size);
    if (total_budget < 0 || sh < 0 || max_pages < 1 || n_pages < 1) return TGVKV_E_INVAL;
    if (max_pages > kMaxTablePages || n_pages > INT32_MAX) return TGVKV_E_UNSUPPORTED;
    if (total_budget > budget_capacity(s)) return TGVKV_E_CAPACITY;
    if ((max_layer_budget(s, total_budget) + page_size - 1) / page_size > max_pages) return TGVKV_E_CAPACITY;
    const int64_t kept = kept_per_sequence(s, total_budget);
    if (s.B == 0 || kept == 0) return TGVKV_OK;
    if (k == nullptr || v == nullptr || idx == nullptr || budgets == nullptr || idx_offsets == nullptr ||
        block_table == nullptr || k_pool == nullptr || v_pool == nullptr)
        return TGVKV_E_INVAL;
    if (!aligned16(k) || !aligned16(v) || !aligned16(k_pool) || !aligned16(v_pool)) return TGVKV_E_INVAL;
    if ((int64_t)s.B * s.L * s.Hkv * 16 > kMaxBlocks) return TGVKV_E_UNSUPPORTED;
    return hip_status(tgvkv::launch_compact_paged(
        s, static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), idx, budgets, idx_offsets,
        (int64_t)s.B * kept, block_table, max_pages, sh, n_pages, unit_order_or_null, static_cast<uint16_t*>(k_pool),
        static_cast<uint16_t*>(v_pool), stream));
}

tgvkv_status tgvkv_decode_attn_paged(const tgvkv_problem* problem, const tgvkv_opts* opts, void* k_pool,
                                     void* v_pool, int64_t n_pages, int32_t page_size, const int32_t* block_table,
                                     int32_t max_pages, const int32_t* budgets, int32_t decode_reserve,
                                     const int32_t* steps, const void* q, const void* k_new, const void* v_new,
                                     float* out, void* workspace, size_t workspace_bytes,
                                     const int32_t* unit_order_or_null, hipStream_t stream) {
    Shape s;
    tgvkv_status st = make_shape(problem, opts, &s);
    if (st != TGVKV_OK) return st;
    const int32_t sh = page_shift(page_size);
    if (decode_reserve < 0 || sh < 0 || max_pages < 1 || n_pages < 1) return TGVKV_E_INVAL;
    if (max_pages > kMaxTablePages || n_pages > INT32_MAX) return TGVKV_E_UNSUPPORTED;
    if (s.B == 0) return TGVKV_OK;
    if (k_pool == nullptr || v_pool == nullptr || block_table == nullptr || budgets == nullptr || steps == nullptr ||
        q == nullptr || k_new == nullptr || v_new == nullptr || out == nullptr)
        return TGVKV_E_INVAL;
    if (!aligned16(k_pool) || !aligned16(v_pool) || !aligned16(q) || !aligned16(k_new) || !aligned16(v_new))
        return TGVKV_E_INVAL;
    const size_t need = decode_workspace_bytes(s);
    if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return TGVKV_E_WORKSPACE;
    return hip_status(tgvkv::launch_decode_paged(
        s, static_cast<uint16_t*>(k_pool), static_cast<uint16_t*>(v_pool), n_pages, block_table, max_pages, sh,
        budgets, decode_reserve, steps, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k_new),
        static_cast<const uint16_t*>(v_new), out, static_cast<float*>(workspace), unit_order_or_null, stream));
}

}  // extern "C\"
