// Problem geometry passed by value to every kernel, and the host-side launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tgvkv {

struct Shape {
    int32_t B, L, H, Hkv, D, G;
    int32_t Ns, Nv, Nq, N, Nt;
    int32_t head_mode, ngroups;
    int32_t n_sink, n_recent;
    int32_t vision_only;  // every layer keeps all text; budgets count vision tokens
    int32_t budget_rule;  // 0: TV mass, 1: uniform, 2: TT mass
    int32_t vision_rank;  // 0: TWR, 1: plain attention sum
    int32_t joint_rank;   // 1: no TPR (text and vision ranked together)
    float sm_scale;
    float scale2;  // sm_scale * log2(e): logits in base-2 units
};

// Launch plan of the question-row passes: waves split 16-row blocks into row sets
// (each up to NSLOT blocks) and, for few blocks, split each key tile into KS parts.
struct RowPlan {
    int nslot, ks, rowgroups;
};

RowPlan plan_question_rows(const Shape& s);

// Score phases.
hipError_t launch_score_stats(const Shape& s, const RowPlan& rp, const uint16_t* q_text,
                              const uint16_t* k, float* lse, float* ws_vm, hipStream_t st);
bool stats_text_eligible(const Shape& s, const RowPlan& rp);
hipError_t launch_score_stats_text(const Shape& s, const RowPlan& rp, const uint16_t* q_text, const uint16_t* k,
                                   float* lse, float* ws_vm, float* ws_colsum, float* ws_vmh, hipStream_t st);
hipError_t launch_score_text(const Shape& s, const uint16_t* q_text, const uint16_t* k, float* lse,
                             const float* ws_vm, float* ws_colsum, float* ws_vmh, bool lse_given, hipStream_t st);
hipError_t launch_score_fin(const Shape& s, const float* ws_colsum, const float* ws_vmh, float* s_txt,
                            float* w_txt, float* tv_mass, bool with_mass, hipStream_t st);
hipError_t launch_score_vision(const Shape& s, const RowPlan& rp, const uint16_t* q_text,
                               const uint16_t* k, const float* lse, const float* w_txt,
                               const int32_t* budgets, int32_t vis_threshold, float* ws_part, float* ws_vm,
                               hipStream_t st);
// Shares of the vision keys a unit's vision sweep is split over (the mass-collecting sweep
// writes one row-mass partial per share).
int vision_splits(const Shape& s, const RowPlan& rp);
hipError_t launch_score_mass(const Shape& s, const RowPlan& rp, const float* ws_vm, float* ws_vmh, float* tv_mass,
                             hipStream_t st);
hipError_t launch_score_vis_reduce(const Shape& s, const RowPlan& rp, const float* ws_part,
                                   const int32_t* budgets, int32_t vis_threshold, float* s_vis,
                                   hipStream_t st);

// Water-fills `total` over the layers with per-layer cap `cap_tokens` and floor
// n_floor, then writes b_l = add + share (add = N_t in vision-only eviction), and,
// if unit_order is given, decode's longest-first dispatch order.
hipError_t launch_budget(const Shape& s, const float* tv_mass, int64_t total, int32_t cap_tokens, int32_t add,
                         int32_t reserve, int32_t n_floor, int32_t* budgets, int64_t* idx_off, int64_t* seg_off,
                         int32_t* unit_order, hipStream_t st);
hipError_t launch_select(const Shape& s, const float* s_vis, const float* s_txt, const int32_t* budgets,
                         const int64_t* idx_off, int32_t* idx, hipStream_t st);
hipError_t launch_compact(const Shape& s, const uint16_t* k, const uint16_t* v, const int32_t* idx,
                          const int32_t* budgets, const int64_t* idx_off, const int64_t* seg_off,
                          int32_t reserve, int64_t rows_total, const int32_t* unit_order, uint16_t* kc,
                          uint16_t* vc, hipStream_t st);

// Paged cache: pages of 2^page_shift rows, [n_pages][H_kv][2^page_shift][D]; row n of
// (sequence, layer) bl lives in page block_table[bl * max_pages + (n >> page_shift)].
hipError_t launch_page_table(const Shape& s, const int32_t* budgets, int32_t reserve, int32_t page_shift,
                             const int32_t* free_pages, int64_t n_free, int32_t* block_table, int32_t max_pages,
                             int64_t* pages_used, hipStream_t st);
hipError_t launch_compact_paged(const Shape& s, const uint16_t* k, const uint16_t* v, const int32_t* idx,
                                const int32_t* budgets, const int64_t* idx_off, int64_t rows_total,
                                const int32_t* block_table, int32_t max_pages, int32_t page_shift, int64_t n_pages,
                                const int32_t* unit_order, uint16_t* k_pool, uint16_t* v_pool, hipStream_t st);

int decode_splits(const Shape& s);
// Bytes of the per-GPU static buffer that holds decode's split partials for callers that
// cannot allocate, and its device address on the current device (looked up once per device).
constexpr size_t kDecodeScratchBytes = size_t(16) << 20;
hipError_t decode_scratch(float** ptr);
hipError_t launch_decode(const Shape& s, uint16_t* kc, uint16_t* vc, const int32_t* budgets,
                         const int64_t* seg_off, int32_t reserve, int32_t step, const uint16_t* q,
                         const uint16_t* k_new, const uint16_t* v_new, float* out, float* ws_part,
                         const int32_t* unit_order, hipStream_t st);
// steps: per-sequence decode step [B]; a sequence whose step is outside [0, reserve) is skipped.
hipError_t launch_decode_paged(const Shape& s, uint16_t* k_pool, uint16_t* v_pool, int64_t n_pages,
                               const int32_t* block_table, int32_t max_pages, int32_t page_shift,
                               const int32_t* budgets, int32_t reserve, const int32_t* steps, const uint16_t* q,
                               const uint16_t* k_new, const uint16_t* v_new, float* out, float* ws_part,
                               const int32_t* unit_order, hipStream_t st);

}  // namespace tgvkv
