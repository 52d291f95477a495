// The fused step's tail kernel: the attention's combine and the greedy
// acceptance in one launch.  The acceptance reads flatten & pack's slots and
// the target tokens, nothing the attention writes, so its workgroups run beside
// the combine's instead of in a launch of their own after them.  They come
// first in the grid, so that they are dispatched first.
#include "accept_device.h"
#include "attn_device.h"
#include "echo_device.h"
#include "echo_internal.h"

namespace echo {
namespace {

constexpr int kAcceptWaves = kThreads / kWave;  // requests per acceptance workgroup
// Slots per request staged in LDS (longer requests read memory).  Small, since
// the combine's workgroups reserve the same LDS.
constexpr int kTailStage = 256;

struct TailArgs {
  // combine
  int hq, hkv, G;
  AttnWs ws;
  float* out;
  float* lse;
  // acceptance: workgroups [0, nacc), request 4 b + w on wave w of workgroup b
  int nacc, R;
  const int32_t* q_offsets;
  const int32_t* slot_parent;
  const int32_t* slot_token;
  const int32_t* target_token;
  int max_rows, max_depth;
  int32_t* accept_len;
  int32_t* accept_slots;
  int32_t* bonus_token;
  int32_t* status;
};

template <int NR>
__global__ __launch_bounds__(kThreads) void tail_kernel(TailArgs a) {
  __shared__ int32_t s_stage[kAcceptWaves][3][kTailStage];
  const int b = blockIdx.x;
  if (b < a.nacc) {
    const int w = threadIdx.x / kWave;
    const int r = b * kAcceptWaves + w;
    if (r < a.R)
      accept_request(r, a.q_offsets, a.slot_parent, a.slot_token, a.target_token, a.max_rows,
                     a.max_depth, a.accept_len, a.accept_slots, a.bonus_token, a.status,
                     AcceptLds{s_stage[w][0], s_stage[w][1], s_stage[w][2], kTailStage});
    return;
  }
  combine_body<NR>(a.hq, a.hkv, a.G, a.ws, a.out, a.lse, b - a.nacc);
}

}  // namespace

int32_t launch_tail(const AttnArgs& a, const int32_t* slot_parent, const int32_t* slot_token,
                    const int32_t* target_token, int32_t max_depth, int32_t* accept_len,
                    int32_t* accept_slots, int32_t* bonus_token, hipStream_t stream) {
  (void)hipGetLastError();  // clear errors left by unrelated runtime calls
  const int nb = device_cu_count();
  TailArgs t;
  t.hq = a.hq;
  t.hkv = a.hkv;
  t.G = a.hq / a.hkv;
  t.ws = attn_layout(a.workspace, unit_capacity(a.R, a.max_rows, a.hq, a.hkv), nb);
  t.out = a.out;
  t.lse = a.lse;
  t.nacc = (a.R + kAcceptWaves - 1) / kAcceptWaves;
  t.R = a.R;
  t.q_offsets = a.q_offsets;
  t.slot_parent = slot_parent;
  t.slot_token = slot_token;
  t.target_token = target_token;
  t.max_rows = a.max_rows;
  t.max_depth = max_depth;
  t.accept_len = accept_len;
  t.accept_slots = accept_slots;
  t.bonus_token = bonus_token;
  t.status = a.status;
  const long long cache_rows = a.block_table == nullptr
                                   ? static_cast<long long>(a.kv_rows)
                                   : static_cast<long long>(a.num_pages) * a.page_size;
  if (combine_rows_per_thread(a.R, a.max_rows, a.hq, a.hkv, nb, cache_rows) == 1)
    hipLaunchKernelGGL(tail_kernel<1>, dim3(unsigned(t.nacc + nb * combine_blocks<1>())),
                       dim3(kThreads), 0, stream, t);
  else
    hipLaunchKernelGGL(tail_kernel<2>, dim3(unsigned(t.nacc + nb * combine_blocks<2>())),
                       dim3(kThreads), 0, stream, t);
  return hipGetLastError() == hipSuccess ? ECHO_OK : ECHO_ERR_HIP;
}

}  // namespace echo
