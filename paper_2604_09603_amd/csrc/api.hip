// C ABI entry points: host-side argument checks, workspace sizing, launch.
#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>

#include "echo.h"
#include "echo_internal.h"

namespace echo {

int device_cu_count() {
  static std::mutex mu;
  static std::vector<int> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  std::lock_guard<std::mutex> lock(mu);
  if (dev >= int(cache.size())) cache.resize(dev + 1, 0);
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

}  // namespace echo

namespace {
inline bool aligned256(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 255u) == 0; }
inline hipStream_t as_stream(echo_stream_t s) { return reinterpret_cast<hipStream_t>(s); }

// The softmax takes each row's maximum of the raw logits as its reference and
// scales it afterwards, which is only valid for a positive finite scale.
inline bool scale_ok(float s) { return s > 0.0f && s <= 3.4028234663852886e38f; }

// Host-side checks and argument packing of the contiguous-cache attention:
// ECHO_OK with *a filled, or the error code.
int32_t attn_contiguous_args(const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new,
                             const uint16_t* k_cache, const uint16_t* v_cache,
                             const int64_t* kv_offsets, int64_t kv_rows, const int32_t* q_offsets,
                             const uint32_t* tree_mask, int32_t mask_words, int32_t R,
                             int32_t max_rows, int32_t num_q_heads, int32_t num_kv_heads,
                             int32_t head_dim, float sm_scale, float* out, float* lse,
                             void* workspace, size_t workspace_bytes, int32_t* status,
                             hipEvent_t ev_start, hipEvent_t ev_stop, echo::AttnArgs* a_out) {
  if (R < 1 || max_rows < 0 || num_q_heads < 1 || num_kv_heads < 1 || mask_words < 1 ||
      kv_rows < 0)
    return ECHO_ERR_INVALID_ARG;
  if (num_q_heads % num_kv_heads != 0 || !scale_ok(sm_scale)) return ECHO_ERR_INVALID_ARG;
  if (head_dim != ECHO_HEAD_DIM || R > ECHO_MAX_REQUESTS || kv_rows >= (int64_t(1) << 31))
    return ECHO_ERR_UNSUPPORTED;
  if (int64_t(max_rows) * num_q_heads >= (int64_t(1) << 26)) return ECHO_ERR_UNSUPPORTED;
  if (!q || !k_new || !v_new || !kv_offsets || !q_offsets || !tree_mask || !out || !workspace)
    return ECHO_ERR_INVALID_ARG;
  if (kv_rows > 0 && (!k_cache || !v_cache)) return ECHO_ERR_INVALID_ARG;
  if ((ev_start == nullptr) != (ev_stop == nullptr)) return ECHO_ERR_INVALID_ARG;
  if (!aligned256(workspace) ||
      workspace_bytes < echo::attn_workspace_bytes(R, max_rows, num_q_heads, num_kv_heads))
    return ECHO_ERR_WORKSPACE;
  // 16-byte vector loads of every bf16 row
  const uintptr_t mis = reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(k_new) |
                        reinterpret_cast<uintptr_t>(v_new) | reinterpret_cast<uintptr_t>(k_cache) |
                        reinterpret_cast<uintptr_t>(v_cache) | reinterpret_cast<uintptr_t>(out);
  if (mis & 15u) return ECHO_ERR_INVALID_ARG;
  echo::AttnArgs& a = *a_out;
  a = echo::AttnArgs{};
  a.q = q;
  a.k_new = k_new;
  a.v_new = v_new;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.kv_offsets = kv_offsets;
  a.kv_rows = kv_rows;
  a.q_offsets = q_offsets;
  a.tree_mask = tree_mask;
  a.mask_words = mask_words;
  a.R = R;
  a.max_rows = max_rows;
  a.hq = num_q_heads;
  a.hkv = num_kv_heads;
  a.sm_scale = sm_scale;
  a.out = out;
  a.lse = lse;
  a.workspace = workspace;
  a.status = status;
  a.ev_start = ev_start;
  a.ev_stop = ev_stop;
  return ECHO_OK;
}

int32_t attn_contiguous(const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new,
                        const uint16_t* k_cache, const uint16_t* v_cache, const int64_t* kv_offsets,
                        int64_t kv_rows, const int32_t* q_offsets, const uint32_t* tree_mask,
                        int32_t mask_words, int32_t R, int32_t max_rows, int32_t num_q_heads,
                        int32_t num_kv_heads, int32_t head_dim, float sm_scale, float* out,
                        float* lse, void* workspace, size_t workspace_bytes, int32_t* status,
                        hipEvent_t ev_start, hipEvent_t ev_stop, hipStream_t stream) {
  echo::AttnArgs a;
  const int32_t rc = attn_contiguous_args(q, k_new, v_new, k_cache, v_cache, kv_offsets, kv_rows,
                                          q_offsets, tree_mask, mask_words, R, max_rows,
                                          num_q_heads, num_kv_heads, head_dim, sm_scale, out, lse,
                                          workspace, workspace_bytes, status, ev_start, ev_stop,
                                          &a);
  if (rc != ECHO_OK || max_rows == 0) return rc;
  return echo::launch_tree_verify_attn(a, stream);
}

// The same for a paged prefix.
int32_t attn_paged(const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new,
                   const uint16_t* k_pages, const uint16_t* v_pages, int64_t num_pages,
                   int32_t page_size, const int32_t* block_table, int32_t max_pages_per_request,
                   const int32_t* prefix_len, const int32_t* q_offsets, const uint32_t* tree_mask,
                   int32_t mask_words, int32_t R, int32_t max_rows, int32_t num_q_heads,
                   int32_t num_kv_heads, int32_t head_dim, float sm_scale, float* out, float* lse,
                   void* workspace, size_t workspace_bytes, int32_t* status, hipEvent_t ev_start,
                   hipEvent_t ev_stop, hipStream_t stream) {
  if (R < 1 || max_rows < 0 || num_q_heads < 1 || num_kv_heads < 1 || mask_words < 1 ||
      num_pages < 1 || max_pages_per_request < 1)
    return ECHO_ERR_INVALID_ARG;
  if (num_q_heads % num_kv_heads != 0 || !scale_ok(sm_scale)) return ECHO_ERR_INVALID_ARG;
  // a page holds whole 32-key tiles and a power-of-two number of rows
  if (page_size < 32 || (page_size & (page_size - 1)) != 0) return ECHO_ERR_UNSUPPORTED;
  if (head_dim != ECHO_HEAD_DIM || R > ECHO_MAX_REQUESTS) return ECHO_ERR_UNSUPPORTED;
  if (num_pages * int64_t(page_size) >= (int64_t(1) << 31)) return ECHO_ERR_UNSUPPORTED;
  if (int64_t(max_pages_per_request) * page_size >= (int64_t(1) << 31)) return ECHO_ERR_UNSUPPORTED;
  if (int64_t(max_rows) * num_q_heads >= (int64_t(1) << 26)) return ECHO_ERR_UNSUPPORTED;
  if (!q || !k_new || !v_new || !k_pages || !v_pages || !block_table || !prefix_len ||
      !q_offsets || !tree_mask || !out || !workspace)
    return ECHO_ERR_INVALID_ARG;
  if ((ev_start == nullptr) != (ev_stop == nullptr)) return ECHO_ERR_INVALID_ARG;
  if (!aligned256(workspace) ||
      workspace_bytes < echo::attn_workspace_bytes(R, max_rows, num_q_heads, num_kv_heads))
    return ECHO_ERR_WORKSPACE;
  const uintptr_t mis = reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(k_new) |
                        reinterpret_cast<uintptr_t>(v_new) | reinterpret_cast<uintptr_t>(k_pages) |
                        reinterpret_cast<uintptr_t>(v_pages) | reinterpret_cast<uintptr_t>(out);
  if (mis & 15u) return ECHO_ERR_INVALID_ARG;
  if (max_rows == 0) return ECHO_OK;
  echo::AttnArgs a{};
  a.q = q;
  a.k_new = k_new;
  a.v_new = v_new;
  a.k_cache = k_pages;
  a.v_cache = v_pages;
  a.kv_offsets = nullptr;
  a.kv_rows = 0;
  a.block_table = block_table;
  a.prefix_len = prefix_len;
  a.page_size = page_size;
  a.max_pages = max_pages_per_request;
  a.num_pages = num_pages;
  a.q_offsets = q_offsets;
  a.tree_mask = tree_mask;
  a.mask_words = mask_words;
  a.R = R;
  a.max_rows = max_rows;
  a.hq = num_q_heads;
  a.hkv = num_kv_heads;
  a.sm_scale = sm_scale;
  a.out = out;
  a.lse = lse;
  a.workspace = workspace;
  a.status = status;
  a.ev_start = ev_start;
  a.ev_stop = ev_stop;
  return echo::launch_tree_verify_attn(a, stream);
}
}  // namespace

extern "C" {

size_t echo_gate_workspace_size(int32_t R, int32_t N, int32_t budget) {
  if (R < 0 || N < 0 || budget < 0) return 0;
  return echo::gate_workspace_bytes(R, N, budget);
}

int32_t echo_gate(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                  int32_t R, int32_t N, int32_t budget, float* path_score, uint8_t* selected,
                  int32_t* num_selected, void* workspace, size_t workspace_bytes, int32_t* status,
                  echo_stream_t stream) {
  if (R < 1 || N < 0 || budget < 0) return ECHO_ERR_INVALID_ARG;
  if (R > ECHO_MAX_REQUESTS || budget > ECHO_MAX_BUDGET) return ECHO_ERR_UNSUPPORTED;
  if (!cand_offsets || !num_selected || !workspace) return ECHO_ERR_INVALID_ARG;
  if (N > 0 && (!parent || !logq || !selected)) return ECHO_ERR_INVALID_ARG;
  if (!aligned256(workspace) || workspace_bytes < echo::gate_workspace_bytes(R, N, budget))
    return ECHO_ERR_WORKSPACE;
  return echo::launch_gate(cand_offsets, parent, logq, R, N, budget, nullptr, nullptr, 0,
                           path_score, selected, num_selected, nullptr, workspace, status,
                           as_stream(stream));
}

size_t echo_gate_sparse_workspace_size(int32_t R, int32_t N, int32_t budget) {
  return echo_gate_workspace_size(R, N, budget);
}

int32_t echo_gate_sparse(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                         int32_t R, int32_t N, int32_t budget, const int32_t* sig_depth,
                         const float* log_tau, int32_t num_sig, float* path_score,
                         uint8_t* selected, int32_t* num_selected, int32_t* trunc_depth,
                         void* workspace, size_t workspace_bytes, int32_t* status,
                         echo_stream_t stream) {
  if (R < 1 || N < 0 || budget < 0) return ECHO_ERR_INVALID_ARG;
  if (R > ECHO_MAX_REQUESTS || budget > ECHO_MAX_BUDGET) return ECHO_ERR_UNSUPPORTED;
  if (!cand_offsets || !num_selected || !workspace) return ECHO_ERR_INVALID_ARG;
  if (N > 0 && (!parent || !logq || !selected)) return ECHO_ERR_INVALID_ARG;
  if (num_sig < 0 || num_sig > ECHO_MAX_CHECKPOINTS) return ECHO_ERR_INVALID_ARG;
  if (num_sig > 0 && (!sig_depth || !log_tau)) return ECHO_ERR_INVALID_ARG;
  for (int k = 0; k < num_sig; ++k) {
    if (sig_depth[k] < 1 || sig_depth[k] > ECHO_MAX_DEPTH) return ECHO_ERR_INVALID_ARG;
    if (log_tau[k] != log_tau[k]) return ECHO_ERR_INVALID_ARG;  // NaN
  }
  if (!aligned256(workspace) || workspace_bytes < echo::gate_workspace_bytes(R, N, budget))
    return ECHO_ERR_WORKSPACE;
  return echo::launch_gate(cand_offsets, parent, logq, R, N, budget, sig_depth, log_tau, num_sig,
                           path_score, selected, num_selected, trunc_depth, workspace, status,
                           as_stream(stream));
}

size_t echo_gate_elastic_workspace_size(int32_t R, int32_t N, int32_t budget) {
  if (R < 0 || N < 0 || budget < 0) return 0;
  return echo::gate_elastic_workspace_bytes(R, N, budget);
}

int32_t echo_gate_elastic(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                          int32_t R, int32_t N, int32_t budget, const int32_t* sig_depth,
                          const float* log_tau, int32_t num_sig, int32_t w_topk, int32_t w_max,
                          float* path_score, uint8_t* selected, int32_t* num_selected,
                          int32_t* trunc_depth, void* workspace, size_t workspace_bytes,
                          int32_t* status, echo_stream_t stream) {
  if (R < 1 || N < 0 || budget < 0 || w_topk < 1 || w_max < 0) return ECHO_ERR_INVALID_ARG;
  if (R > ECHO_MAX_REQUESTS || budget > ECHO_MAX_BUDGET) return ECHO_ERR_UNSUPPORTED;
  if (!cand_offsets || !num_selected || !workspace) return ECHO_ERR_INVALID_ARG;
  if (N > 0 && (!parent || !logq || !selected)) return ECHO_ERR_INVALID_ARG;
  if (num_sig < 0 || num_sig > ECHO_MAX_CHECKPOINTS) return ECHO_ERR_INVALID_ARG;
  if (num_sig > 0 && (!sig_depth || !log_tau)) return ECHO_ERR_INVALID_ARG;
  for (int k = 0; k < num_sig; ++k) {
    if (sig_depth[k] < 1 || sig_depth[k] > ECHO_MAX_DEPTH) return ECHO_ERR_INVALID_ARG;
    if (log_tau[k] != log_tau[k]) return ECHO_ERR_INVALID_ARG;  // NaN
  }
  if (!aligned256(workspace) ||
      workspace_bytes < echo::gate_elastic_workspace_bytes(R, N, budget))
    return ECHO_ERR_WORKSPACE;
  return echo::launch_gate_elastic(cand_offsets, parent, logq, R, N, budget, sig_depth, log_tau,
                                   num_sig, w_topk, w_max, path_score, selected, num_selected,
                                   trunc_depth, workspace, status, as_stream(stream));
}

size_t echo_build_tree_mask_workspace_size(int32_t R, int32_t N, int32_t budget) {
  (void)R;
  (void)N;
  (void)budget;
  return 0;  // everything lives in LDS
}

int32_t echo_build_tree_mask(const int32_t* cand_offsets, const int32_t* parent,
                             const int32_t* token, const uint8_t* selected,
                             const int32_t* root_token, const int32_t* prefix_len, int32_t R,
                             int32_t N, int32_t budget, int32_t* q_offsets, int32_t* slot_cand,
                             int32_t* slot_parent, int32_t* slot_token, int32_t* position_ids,
                             uint32_t* tree_mask, int32_t mask_words, void* workspace,
                             size_t workspace_bytes, int32_t* status, echo_stream_t stream) {
  (void)workspace;
  (void)workspace_bytes;
  if (R < 1 || N < 0 || budget < 0) return ECHO_ERR_INVALID_ARG;
  if (R > ECHO_MAX_REQUESTS || budget > ECHO_MAX_BUDGET) return ECHO_ERR_UNSUPPORTED;
  if (int64_t(mask_words) * 32 < int64_t(budget) + 1) return ECHO_ERR_INVALID_ARG;
  if (!cand_offsets || !root_token || !prefix_len || !q_offsets || !slot_cand || !slot_parent ||
      !slot_token || !position_ids || !tree_mask)
    return ECHO_ERR_INVALID_ARG;
  if (N > 0 && (!parent || !token || !selected)) return ECHO_ERR_INVALID_ARG;
  if (echo::mask_lds_bytes(R, budget) > 150 * 1024) return ECHO_ERR_UNSUPPORTED;
  return echo::launch_build_tree_mask(cand_offsets, parent, token, selected, root_token,
                                      prefix_len, R, N, budget, q_offsets, slot_cand, slot_parent,
                                      slot_token, position_ids, tree_mask, mask_words, status,
                                      as_stream(stream));
}

size_t echo_tree_verify_attn_workspace_size(int32_t R, int32_t max_rows, int32_t num_q_heads,
                                            int32_t num_kv_heads, int32_t head_dim) {
  if (R < 1 || max_rows < 0 || num_q_heads < 1 || num_kv_heads < 1 || head_dim != ECHO_HEAD_DIM)
    return 0;
  return echo::attn_workspace_bytes(R, max_rows, num_q_heads, num_kv_heads);
}

int32_t echo_tree_verify_attn(const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new,
                              const uint16_t* k_cache, const uint16_t* v_cache,
                              const int64_t* kv_offsets, int64_t kv_rows,
                              const int32_t* q_offsets, const uint32_t* tree_mask,
                              int32_t mask_words, int32_t R, int32_t max_rows,
                              int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                              float sm_scale, float* out, float* lse, void* workspace,
                              size_t workspace_bytes, int32_t* status, echo_stream_t stream) {
  return attn_contiguous(q, k_new, v_new, k_cache, v_cache, kv_offsets, kv_rows, q_offsets,
                         tree_mask, mask_words, R, max_rows, num_q_heads, num_kv_heads, head_dim,
                         sm_scale, out, lse, workspace, workspace_bytes, status, nullptr, nullptr,
                         as_stream(stream));
}

int32_t echo_tree_verify_attn_timed(const uint16_t* q, const uint16_t* k_new,
                                    const uint16_t* v_new, const uint16_t* k_cache,
                                    const uint16_t* v_cache, const int64_t* kv_offsets,
                                    int64_t kv_rows, const int32_t* q_offsets,
                                    const uint32_t* tree_mask, int32_t mask_words, int32_t R,
                                    int32_t max_rows, int32_t num_q_heads, int32_t num_kv_heads,
                                    int32_t head_dim, float sm_scale, float* out, float* lse,
                                    void* workspace, size_t workspace_bytes, int32_t* status,
                                    void* ev_start, void* ev_stop, echo_stream_t stream) {
  if (ev_start == nullptr || ev_stop == nullptr) return ECHO_ERR_INVALID_ARG;
  return attn_contiguous(q, k_new, v_new, k_cache, v_cache, kv_offsets, kv_rows, q_offsets,
                         tree_mask, mask_words, R, max_rows, num_q_heads, num_kv_heads, head_dim,
                         sm_scale, out, lse, workspace, workspace_bytes, status,
                         reinterpret_cast<hipEvent_t>(ev_start),
                         reinterpret_cast<hipEvent_t>(ev_stop), as_stream(stream));
}

int32_t echo_tree_verify_attn_paged(
    const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new, const uint16_t* k_pages,
    const uint16_t* v_pages, int64_t num_pages, int32_t page_size, const int32_t* block_table,
    int32_t max_pages_per_request, const int32_t* prefix_len, const int32_t* q_offsets,
    const uint32_t* tree_mask, int32_t mask_words, int32_t R, int32_t max_rows,
    int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, float sm_scale, float* out,
    float* lse, void* workspace, size_t workspace_bytes, int32_t* status, echo_stream_t stream) {
  return attn_paged(q, k_new, v_new, k_pages, v_pages, num_pages, page_size, block_table,
                    max_pages_per_request, prefix_len, q_offsets, tree_mask, mask_words, R,
                    max_rows, num_q_heads, num_kv_heads, head_dim, sm_scale, out, lse, workspace,
                    workspace_bytes, status, nullptr, nullptr, as_stream(stream));
}

int32_t echo_tree_verify_attn_paged_timed(
    const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new, const uint16_t* k_pages,
    const uint16_t* v_pages, int64_t num_pages, int32_t page_size, const int32_t* block_table,
    int32_t max_pages_per_request, const int32_t* prefix_len, const int32_t* q_offsets,
    const uint32_t* tree_mask, int32_t mask_words, int32_t R, int32_t max_rows,
    int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, float sm_scale, float* out,
    float* lse, void* workspace, size_t workspace_bytes, int32_t* status, void* ev_start,
    void* ev_stop, echo_stream_t stream) {
  if (ev_start == nullptr || ev_stop == nullptr) return ECHO_ERR_INVALID_ARG;
  return attn_paged(q, k_new, v_new, k_pages, v_pages, num_pages, page_size, block_table,
                    max_pages_per_request, prefix_len, q_offsets, tree_mask, mask_words, R,
                    max_rows, num_q_heads, num_kv_heads, head_dim, sm_scale, out, lse, workspace,
                    workspace_bytes, status, reinterpret_cast<hipEvent_t>(ev_start),
                    reinterpret_cast<hipEvent_t>(ev_stop), as_stream(stream));
}

int32_t echo_accept(const int32_t* q_offsets, const int32_t* slot_parent,
                    const int32_t* slot_token, const int32_t* target_token, int32_t R,
                    int32_t max_rows, int32_t max_depth, int32_t* accept_len,
                    int32_t* accept_slots, int32_t* bonus_token, int32_t* status,
                    echo_stream_t stream) {
  if (R < 1 || max_rows < 0 || max_depth < 1) return ECHO_ERR_INVALID_ARG;
  if (max_depth > ECHO_MAX_DEPTH || R > ECHO_MAX_REQUESTS) return ECHO_ERR_UNSUPPORTED;
  if (!q_offsets || !accept_len || !accept_slots || !bonus_token) return ECHO_ERR_INVALID_ARG;
  if (max_rows > 0 && (!slot_parent || !slot_token || !target_token)) return ECHO_ERR_INVALID_ARG;
  return echo::launch_accept(q_offsets, slot_parent, slot_token, target_token, R, max_rows,
                             max_depth, accept_len, accept_slots, bonus_token, status,
                             as_stream(stream));
}

int32_t echo_verify_step(
    const int32_t* cand_offsets, const int32_t* parent, const float* logq, const int32_t* token,
    int32_t R, int32_t N, int32_t budget, float* path_score, uint8_t* selected,
    int32_t* num_selected, void* gate_workspace, size_t gate_workspace_bytes,
    const int32_t* root_token, const int32_t* prefix_len, int32_t* q_offsets, int32_t* slot_cand,
    int32_t* slot_parent, int32_t* slot_token, int32_t* position_ids, uint32_t* tree_mask,
    int32_t mask_words, const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new,
    const uint16_t* k_cache, const uint16_t* v_cache, const int64_t* kv_offsets, int64_t kv_rows,
    int32_t max_rows, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
    float sm_scale, float* out, float* lse, void* attn_workspace, size_t attn_workspace_bytes,
    const int32_t* target_token, int32_t max_depth, int32_t* accept_len, int32_t* accept_slots,
    int32_t* bonus_token, int32_t* status, echo_stream_t stream) {
  // every check of the four calls, before anything is launched
  if (R < 1 || N < 0 || budget < 0) return ECHO_ERR_INVALID_ARG;
  if (R > ECHO_MAX_REQUESTS || budget > ECHO_MAX_BUDGET) return ECHO_ERR_UNSUPPORTED;
  if (!cand_offsets || !num_selected || !gate_workspace) return ECHO_ERR_INVALID_ARG;
  if (N > 0 && (!parent || !logq || !selected || !token)) return ECHO_ERR_INVALID_ARG;
  if (!aligned256(gate_workspace) ||
      gate_workspace_bytes < echo::gate_workspace_bytes(R, N, budget))
    return ECHO_ERR_WORKSPACE;
  if (int64_t(mask_words) * 32 < int64_t(budget) + 1) return ECHO_ERR_INVALID_ARG;
  if (!root_token || !prefix_len || !q_offsets || !slot_cand || !slot_parent || !slot_token ||
      !position_ids || !tree_mask)
    return ECHO_ERR_INVALID_ARG;
  if (echo::mask_lds_bytes(R, budget) > 150 * 1024) return ECHO_ERR_UNSUPPORTED;
  echo::AttnArgs a;
  int32_t rc = attn_contiguous_args(q, k_new, v_new, k_cache, v_cache, kv_offsets, kv_rows,
                                    q_offsets, tree_mask, mask_words, R, max_rows, num_q_heads,
                                    num_kv_heads, head_dim, sm_scale, out, lse, attn_workspace,
                                    attn_workspace_bytes, status, nullptr, nullptr, &a);
  if (rc != ECHO_OK) return rc;
  if (max_depth < 1) return ECHO_ERR_INVALID_ARG;
  if (max_depth > ECHO_MAX_DEPTH) return ECHO_ERR_UNSUPPORTED;
  if (!accept_len || !accept_slots || !bonus_token) return ECHO_ERR_INVALID_ARG;
  if (max_rows > 0 && !target_token) return ECHO_ERR_INVALID_ARG;
  hipStream_t s = as_stream(stream);
  rc = echo::launch_gate_select_only(cand_offsets, parent, logq, R, N, budget, path_score,
                                     selected, num_selected, gate_workspace, status, s);
  if (rc != ECHO_OK) return rc;
  echo::FrontLaunch f;
  f.N = N;
  f.R = R;
  f.budget = budget;
  f.mask_words = mask_words;
  f.gate_workspace = gate_workspace;
  f.selected = selected;
  f.cand_offsets = cand_offsets;
  f.parent = parent;
  f.token = token;
  f.root_token = root_token;
  f.prefix_len = prefix_len;
  f.q_offsets = q_offsets;
  f.slot_cand = slot_cand;
  f.slot_parent = slot_parent;
  f.slot_token = slot_token;
  f.position_ids = position_ids;
  f.tree_mask = tree_mask;
  f.kv_offsets = kv_offsets;
  f.kv_rows = kv_rows;
  f.max_rows = max_rows;
  f.hq = num_q_heads;
  f.hkv = num_kv_heads;
  f.attn_workspace = attn_workspace;
  f.status = status;
  rc = echo::launch_front(f, s);
  if (rc != ECHO_OK) return rc;
  if (max_rows == 0)  // no attention rows: the acceptance alone
    return echo::launch_accept(q_offsets, slot_parent, slot_token, target_token, R, max_rows,
                               max_depth, accept_len, accept_slots, bonus_token, status, s);
  rc = echo::launch_tree_verify_attn_main(a, s);
  if (rc != ECHO_OK) return rc;
  return echo::launch_tail(a, slot_parent, slot_token, target_token, max_depth, accept_len,
                           accept_slots, bonus_token, s);
}

const char* echo_status_string(int32_t code) {
  switch (code) {
    case ECHO_OK: return "ok";
    case ECHO_ERR_INVALID_ARG: return "invalid argument";
    case ECHO_ERR_UNSUPPORTED: return "unsupported size or shape";
    case ECHO_ERR_WORKSPACE: return "workspace too small or not 256-byte aligned";
    case ECHO_ERR_HIP: return "HIP launch or runtime failure";
    default: return "unknown status";
  }
}

const char* echo_version(void) { return "echo-mi355x 0.1.0 (gfx950)"; }

}  // extern "C"

extern "C" {

int32_t echo_accept_logits(const int32_t* q_offsets, const int32_t* slot_parent,
                           const int32_t* slot_token, const uint16_t* logits, int64_t vocab,
                           int32_t R, int32_t max_rows, int32_t max_depth, int32_t* target_token,
                           int32_t* accept_len, int32_t* accept_slots, int32_t* bonus_token,
                           int32_t* status, echo_stream_t stream) {
  if (R < 1 || max_rows < 0 || vocab < 1 || vocab > 0x7FFFFFFF) return ECHO_ERR_INVALID_ARG;
  if (max_depth < 1 || max_depth > ECHO_MAX_DEPTH || R > ECHO_MAX_REQUESTS)
    return ECHO_ERR_UNSUPPORTED;
  if (!q_offsets || !accept_len || !accept_slots || !bonus_token || !target_token)
    return ECHO_ERR_INVALID_ARG;
  if (max_rows > 0 && (!slot_parent || !slot_token || !logits)) return ECHO_ERR_INVALID_ARG;
  return echo::launch_accept_logits(q_offsets, slot_parent, slot_token, logits, vocab, R,
                                    max_rows, max_depth, target_token, accept_len, accept_slots,
                                    bonus_token, status, as_stream(stream));
}

int32_t echo_commit_kv(const int32_t* q_offsets, const int32_t* accept_len,
                       const int32_t* accept_slots, int32_t max_depth, const uint16_t* k_new,
                       const uint16_t* v_new, int32_t R, int32_t max_rows, int32_t num_kv_heads,
                       uint16_t* k_pages, uint16_t* v_pages, int64_t num_pages, int32_t page_size,
                       const int32_t* block_table, int32_t max_pages_per_request,
                       int32_t* prefix_len, int32_t* status, echo_stream_t stream) {
  if (R < 1 || max_rows < 0 || num_kv_heads < 1 || num_pages < 1 || page_size < 1 ||
      max_pages_per_request < 1)
    return ECHO_ERR_INVALID_ARG;
  if (max_depth < 1 || max_depth > ECHO_MAX_DEPTH || R > ECHO_MAX_REQUESTS)
    return ECHO_ERR_UNSUPPORTED;
  if (!q_offsets || !accept_len || !accept_slots || !k_new || !v_new || !k_pages || !v_pages ||
      !block_table || !prefix_len)
    return ECHO_ERR_INVALID_ARG;
  const uintptr_t al = reinterpret_cast<uintptr_t>(k_new) | reinterpret_cast<uintptr_t>(v_new) |
                       reinterpret_cast<uintptr_t>(k_pages) | reinterpret_cast<uintptr_t>(v_pages);
  if (al & 15) return ECHO_ERR_INVALID_ARG;
  return echo::launch_commit_kv(q_offsets, accept_len, accept_slots, max_depth, k_new, v_new, R,
                                max_rows, num_kv_heads, k_pages, v_pages, num_pages, page_size,
                                block_table, max_pages_per_request, prefix_len, status,
                                as_stream(stream));
}

}  // extern "C"
