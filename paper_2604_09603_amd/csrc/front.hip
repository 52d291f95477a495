// The fused step's front kernel: the last phase of the top-B gate (eq. 4),
// flatten & pack (Fig. 3, stage 3) and the attention plan, one after another
// on one workgroup.  Each of the three is one workgroup that waits for the one
// before it, so as separate launches the step pays a kernel boundary (one
// kernel's drain, the next one's launch) between each pair.
//
// The three phases share one dynamic LDS buffer: the gate's gathered
// candidates (2 x 32 KB and the select blocks' offsets) first, then the mask's
// request tables, compacted list and ancestor slots.  A barrier separates the
// phases; the selection flags and slot offsets pass through global memory,
// where the workgroup's own stores before a barrier are seen by its loads
// after it.
#include "attn_device.h"
#include "echo_device.h"
#include "echo_internal.h"
#include "gate_device.h"
#include "mask_device.h"

namespace echo {
namespace {

constexpr int kFrontThreads = 1024;
static_assert(kGateThreads == kFrontThreads && kMaskThreads == kFrontThreads,
              "the gate's last phase and the mask run on one workgroup of the same size");

// LDS of the gate's last phase: keys and indices of kSortCap candidates and the
// kGateThreads + 1 offsets of the select blocks.
constexpr size_t kFinishLds = size_t(2 * kSortCap + kGateThreads + 1) * sizeof(int32_t);

struct FrontArgs {
  // gate, last phase
  int N, nblocks;
  GateWs gws;
  uint8_t* selected;
  // flatten & pack
  const int32_t* cand_offsets;
  const int32_t* parent;
  const int32_t* token;
  const int32_t* root_token;
  const int32_t* prefix_len;
  int R, budget, W;
  int32_t* q_offsets;
  int32_t* slot_cand;
  int32_t* slot_parent;
  int32_t* slot_token;
  int32_t* position_ids;
  uint32_t* tree_mask;
  // attention plan
  KvSource kv;
  int hkv, G, max_rows, nb;
  int plan;  // 0: no rows (the attention call does nothing either)
  long long ucap;
  AttnWs aws;
  int32_t* status;
};

template <bool kAligned>
__global__ __launch_bounds__(kFrontThreads) void front_kernel(FrontArgs a) {
  extern __shared__ int32_t smem[];
  // The request tables of flatten & pack are loaded first, into registers, so
  // that their memory latency passes with that of the gate's first loads.
  const MaskTables tab = load_mask_tables(a.cand_offsets, a.root_token, a.prefix_len, a.R);
  // and the plan's KV offsets (one request per thread), which no phase before
  // it writes
  const int tid = threadIdx.x;
  const bool pre = a.plan && a.R <= kFrontThreads;
  long long k0 = 0, k1 = 0;
  if (pre && tid < a.R) {
    k0 = a.kv.kv_offsets[tid];
    k1 = a.kv.kv_offsets[tid + 1];
  }
  if (a.N > 0)  // as the gate call, which skips its last phase without candidates
    gate_finish_body(a.N, a.nblocks, a.gws, a.selected, a.status,
                     FinishLds{reinterpret_cast<uint32_t*>(smem), smem + kSortCap,
                               smem + 2 * kSortCap});
  __syncthreads();
  mask_body<kAligned>(tab, a.parent, a.token, a.selected, a.R, a.N, a.budget, a.q_offsets,
                      a.slot_cand, a.slot_parent, a.slot_token, a.position_ids, a.tree_mask, a.W,
                      a.status, smem);
  if (!a.plan) return;
  __syncthreads();
  // the slot offsets the mask phase just wrote are still in its LDS table
  const int32_t* s_qoff = smem + (a.R + 1);
  RequestIn in;
  in.q0 = tid < a.R ? s_qoff[tid] : 0;
  in.q1 = tid < a.R ? s_qoff[tid + 1] : 0;
  in.k0 = k0;
  in.k1 = k1;
  in.P = k1 - k0;
  // (the tables reuse the LDS of the phases before; every thread has read its
  // slot offsets before the plan's first barrier)
  plan_body<kFrontThreads>(a.q_offsets, a.kv, a.R, a.hkv, a.G, a.max_rows, a.nb, a.ucap, a.aws,
                           a.status, smem, pre ? &in : nullptr);
}

}  // namespace

size_t front_lds_bytes(int32_t R, int32_t budget) {
  const size_t m = mask_lds_bytes(R, budget);
  const size_t p = plan_table_words(R < kFrontThreads ? R : kFrontThreads) * sizeof(int32_t);
  const size_t f = m > kFinishLds ? m : kFinishLds;
  return f > p ? f : p;
}

int32_t launch_front(const FrontLaunch& f, hipStream_t stream) {
  (void)hipGetLastError();  // clear errors left by unrelated runtime calls
  FrontArgs a;
  a.N = f.N;
  a.nblocks = gate_blocks(f.N);
  a.gws = gate_ws_layout(f.gate_workspace, f.N, f.R);
  a.selected = f.selected;
  a.cand_offsets = f.cand_offsets;
  a.parent = f.parent;
  a.token = f.token;
  a.root_token = f.root_token;
  a.prefix_len = f.prefix_len;
  a.R = f.R;
  a.budget = f.budget;
  a.W = f.mask_words;
  a.q_offsets = f.q_offsets;
  a.slot_cand = f.slot_cand;
  a.slot_parent = f.slot_parent;
  a.slot_token = f.slot_token;
  a.position_ids = f.position_ids;
  a.tree_mask = f.tree_mask;
  a.kv.kv_offsets = f.kv_offsets;
  a.kv.kv_rows = static_cast<long long>(f.kv_rows);
  a.kv.block_table = nullptr;
  a.kv.prefix_len = nullptr;
  a.kv.page_size = 0;
  a.kv.max_pages = 0;
  a.kv.num_pages = 0;
  a.kv.page_bad = nullptr;
  a.kv.page_chunks = 0;
  a.hkv = f.hkv;
  a.G = f.hq / f.hkv;
  a.max_rows = f.max_rows;
  a.plan = f.max_rows > 0 ? 1 : 0;
  a.nb = device_cu_count();
  a.ucap = static_cast<long long>(unit_capacity(f.R, f.max_rows, f.hq, f.hkv));
  a.aws = attn_layout(f.attn_workspace, size_t(a.ucap), a.nb);
  a.status = f.status;
  const size_t lds = front_lds_bytes(f.R, f.budget);
  const bool aligned = (reinterpret_cast<uintptr_t>(f.selected) & 15u) == 0;
  auto kern = aligned ? front_kernel<true> : front_kernel<false>;
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                          hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess)
    return ECHO_ERR_HIP;
  hipLaunchKernelGGL(kern, dim3(1), dim3(kFrontThreads), lds, stream, a);
  return hipGetLastError() == hipSuccess ? ECHO_OK : ECHO_ERR_HIP;
}

}  // namespace echo
