// Flatten & pack (Fig. 3, stage 3): the selected super-tree becomes per-request
// verify slots with parent slots, position ids and ancestor bitmasks.
//
// One workgroup of 1024 threads (the selection holds at most B <= 16384 nodes,
// so the whole step is latency-bound and a single CU avoids any grid-wide
// synchronisation):
//   1. ordered compaction of `selected` (128 bytes per thread per round, one
//      block scan per round) into an LDS list of global indices, ascending;
//   2. q_offsets[r] = r + #(packed candidates before request r) (binary search)
//      and the root slot of each request;
//   3. one thread per packed node writes its slot's candidate and token and
//      finds the local slot of its nearest packed ancestor (its parent, unless
//      the selection is not ancestor-closed), kept in LDS: one round of global
//      loads for all nodes;
//   4. one thread per slot walks that chain in LDS only, marking its
//      ancestors in its bitmask row.
#include "echo_device.h"
#include "echo_internal.h"
#include "mask_device.h"

namespace echo {
namespace {

template <bool kAligned>
__global__ __launch_bounds__(kMaskThreads) void mask_kernel(
    const int32_t* __restrict__ cand_offsets, const int32_t* __restrict__ parent,
    const int32_t* __restrict__ token, const uint8_t* __restrict__ selected,
    const int32_t* __restrict__ root_token, const int32_t* __restrict__ prefix_len, int R, int N,
    int budget, int32_t* __restrict__ q_offsets, int32_t* __restrict__ slot_cand,
    int32_t* __restrict__ slot_parent, int32_t* __restrict__ slot_token,
    int32_t* __restrict__ position_ids, uint32_t* __restrict__ tree_mask, int W,
    int32_t* status) {
  extern __shared__ int32_t smem[];
  const MaskTables tab = load_mask_tables(cand_offsets, root_token, prefix_len, R);
  mask_body<kAligned>(tab, parent, token, selected, R, N, budget, q_offsets, slot_cand,
                      slot_parent, slot_token, position_ids, tree_mask, W, status, smem);
}

}  // namespace

size_t mask_lds_bytes(int32_t R, int32_t budget) {
  return size_t(3 * (R + 1) + budget) * sizeof(int32_t) + size_t(budget) * sizeof(uint16_t);
}

int32_t launch_build_tree_mask(const int32_t* cand_offsets, const int32_t* parent,
                               const int32_t* token, const uint8_t* selected,
                               const int32_t* root_token, const int32_t* prefix_len, int32_t R,
                               int32_t N, int32_t budget, int32_t* q_offsets, int32_t* slot_cand,
                               int32_t* slot_parent, int32_t* slot_token, int32_t* position_ids,
                               uint32_t* tree_mask, int32_t mask_words, int32_t* status,
                               hipStream_t stream) {
  (void)hipGetLastError();  // clear errors left by unrelated runtime calls
  const size_t lds = mask_lds_bytes(R, budget);
  const bool aligned = (reinterpret_cast<uintptr_t>(selected) & 15u) == 0;
  auto kern = aligned ? mask_kernel<true> : mask_kernel<false>;
  if (lds > 64 * 1024) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                            hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess)
      return ECHO_ERR_HIP;
  }
  hipLaunchKernelGGL(kern, dim3(1), dim3(kMaskThreads), lds, stream, cand_offsets, parent, token,
                     selected, root_token, prefix_len, R, N, budget, q_offsets, slot_cand,
                     slot_parent, slot_token, position_ids, tree_mask, mask_words, status);
  return hipGetLastError() == hipSuccess ? ECHO_OK : ECHO_ERR_HIP;
}

}  // namespace echo
