// Launchers behind the C ABI (one per stage).  Host code; arguments already validated.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace echo {

// num_sig == 0: plain top-B; otherwise sparse checkpoint gating first (host
// arrays sig_depth / log_tau of num_sig entries, already validated).
int32_t launch_gate(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                    int32_t R, int32_t N, int32_t budget, const int32_t* sig_depth,
                    const float* log_tau, int32_t num_sig, float* path_score, uint8_t* selected,
                    int32_t* num_selected, int32_t* trunc_depth, void* workspace, int32_t* status,
                    hipStream_t stream);
size_t gate_workspace_bytes(int32_t R, int32_t N, int32_t budget);
// The top-B gate without its last phase (gate_finish), which the fused step's
// front kernel runs.
int32_t launch_gate_select_only(const int32_t* cand_offsets, const int32_t* parent,
                                const float* logq, int32_t R, int32_t N, int32_t budget,
                                float* path_score, uint8_t* selected, int32_t* num_selected,
                                void* workspace, int32_t* status, hipStream_t stream);

// Path scores only (the first gate launch): per candidate the orderable key
// (0 = never selectable), the clamped parent as a global index (-1: child of
// the root) and the depth (capped at ECHO_MAX_DEPTH + 1), in the gate workspace.
struct GateScoreBufs {
  const uint32_t* keys;
  const int32_t* pglob;
  const uint8_t* depth;
};
int32_t launch_gate_score(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                          int32_t R, int32_t N, float* path_score, void* workspace,
                          int32_t* status, hipStream_t stream, GateScoreBufs* out);

// Alg. 1 scheduler (checkpoint table as for launch_gate; w_topk >= 1, w_max >= 0).
int32_t launch_gate_elastic(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                            int32_t R, int32_t N, int32_t budget, const int32_t* sig_depth,
                            const float* log_tau, int32_t num_sig, int32_t w_topk, int32_t w_max,
                            float* path_score, uint8_t* selected, int32_t* num_selected,
                            int32_t* trunc_depth, void* workspace, int32_t* status,
                            hipStream_t stream);
size_t gate_elastic_workspace_bytes(int32_t R, int32_t N, int32_t budget);

int32_t launch_build_tree_mask(const int32_t* cand_offsets, const int32_t* parent,
                               const int32_t* token, const uint8_t* selected,
                               const int32_t* root_token, const int32_t* prefix_len, int32_t R,
                               int32_t N, int32_t budget, int32_t* q_offsets, int32_t* slot_cand,
                               int32_t* slot_parent, int32_t* slot_token, int32_t* position_ids,
                               uint32_t* tree_mask, int32_t mask_words, int32_t* status,
                               hipStream_t stream);
size_t mask_lds_bytes(int32_t R, int32_t budget);

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k_new;
  const uint16_t* v_new;
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  const int64_t* kv_offsets;
  int64_t kv_rows;
  // paged prefix (block_table != nullptr): request r's position p lives in page
  // block_table[r * max_pages + p / page_size], row p % page_size, of
  // k_cache / v_cache seen as [num_pages][page_size][Hkv][128]; its length is
  // prefix_len[r] (kv_offsets and kv_rows are not used)
  const int32_t* block_table;
  const int32_t* prefix_len;
  int32_t page_size;
  int32_t max_pages;
  int64_t num_pages;
  const int32_t* q_offsets;
  const uint32_t* tree_mask;
  int32_t mask_words;
  int32_t R;
  int32_t max_rows;
  int32_t hq;
  int32_t hkv;
  float sm_scale;
  float* out;
  float* lse;
  void* workspace;
  int32_t* status;
  // measurement only: recorded on the launch stream right before and right
  // after the main attention kernel (both null, or both set)
  hipEvent_t ev_start;
  hipEvent_t ev_stop;
};
int32_t launch_tree_verify_attn(const AttnArgs& a, hipStream_t stream);
// The main kernel alone: the fused step's front kernel wrote the plan into the
// workspace (contiguous cache only) and its tail kernel runs the combine.
int32_t launch_tree_verify_attn_main(const AttnArgs& a, hipStream_t stream);
size_t attn_workspace_bytes(int32_t R, int32_t max_rows, int32_t hq, int32_t hkv);

int32_t launch_accept(const int32_t* q_offsets, const int32_t* slot_parent,
                      const int32_t* slot_token, const int32_t* target_token, int32_t R,
                      int32_t max_rows, int32_t max_depth, int32_t* accept_len,
                      int32_t* accept_slots, int32_t* bonus_token, int32_t* status,
                      hipStream_t stream);

int32_t launch_accept_logits(const int32_t* q_offsets, const int32_t* slot_parent,
                             const int32_t* slot_token, const uint16_t* logits, int64_t vocab,
                             int32_t R, int32_t max_rows, int32_t max_depth, int32_t* target,
                             int32_t* accept_len, int32_t* accept_slots, int32_t* bonus_token,
                             int32_t* status, hipStream_t stream);

int32_t launch_commit_kv(const int32_t* q_offsets, const int32_t* accept_len,
                         const int32_t* accept_slots, int32_t max_depth, const uint16_t* k_new,
                         const uint16_t* v_new, int32_t R, int32_t max_rows, int32_t hkv,
                         uint16_t* k_pages, uint16_t* v_pages, int64_t num_pages,
                         int32_t page_size, const int32_t* block_table, int32_t max_pages,
                         int32_t* prefix_len, int32_t* status, hipStream_t stream);

int device_cu_count();

// Fused step (front.hip): the gate's last phase, flatten & pack and the
// attention plan (contiguous cache) in one single-workgroup launch, after
// launch_gate_select_only and before launch_tree_verify_attn_main.
struct FrontLaunch {
  int32_t N, R, budget, mask_words;
  void* gate_workspace;
  uint8_t* selected;
  const int32_t* cand_offsets;
  const int32_t* parent;
  const int32_t* token;
  const int32_t* root_token;
  const int32_t* prefix_len;
  int32_t* q_offsets;
  int32_t* slot_cand;
  int32_t* slot_parent;
  int32_t* slot_token;
  int32_t* position_ids;
  uint32_t* tree_mask;
  const int64_t* kv_offsets;
  int64_t kv_rows;
  int32_t max_rows, hq, hkv;
  void* attn_workspace;
  int32_t* status;
};
size_t front_lds_bytes(int32_t R, int32_t budget);
int32_t launch_front(const FrontLaunch& f, hipStream_t stream);

// Fused step (tail.hip): the attention's combine and the greedy acceptance in
// one launch, after launch_tree_verify_attn_main; `a` as for that call.
int32_t launch_tail(const AttnArgs& a, const int32_t* slot_parent, const int32_t* slot_token,
                    const int32_t* target_token, int32_t max_depth, int32_t* accept_len,
                    int32_t* accept_slots, int32_t* bonus_token, hipStream_t stream);

}  // namespace echo
