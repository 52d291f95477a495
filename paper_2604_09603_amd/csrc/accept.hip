// Greedy acceptance: one wavefront per request (see accept_request).
#include "accept_device.h"
#include "echo_device.h"
#include "echo_internal.h"

namespace echo {
namespace {

constexpr int kStage = 2048;  // slots per request staged in LDS

__global__ __launch_bounds__(kWave) void accept_kernel(
    const int32_t* __restrict__ q_offsets, const int32_t* __restrict__ slot_parent,
    const int32_t* __restrict__ slot_token, const int32_t* __restrict__ target_token,
    int max_rows, int max_depth, int32_t* __restrict__ accept_len,
    int32_t* __restrict__ accept_slots, int32_t* __restrict__ bonus_token, int32_t* status) {
  __shared__ int32_t s_par[kStage];
  __shared__ int32_t s_tok[kStage];
  __shared__ int32_t s_tgt[kStage];
  accept_request(blockIdx.x, q_offsets, slot_parent, slot_token, target_token, max_rows, max_depth,
                 accept_len, accept_slots, bonus_token, status, AcceptLds{s_par, s_tok, s_tgt, kStage});
}

}  // namespace

int32_t launch_accept(const int32_t* q_offsets, const int32_t* slot_parent,
                      const int32_t* slot_token, const int32_t* target_token, int32_t R,
                      int32_t max_rows, int32_t max_depth, int32_t* accept_len,
                      int32_t* accept_slots, int32_t* bonus_token, int32_t* status,
                      hipStream_t stream) {
  (void)hipGetLastError();  // clear errors left by unrelated runtime calls
  if (R == 0) return ECHO_OK;
  hipLaunchKernelGGL(accept_kernel, dim3(R), dim3(kWave), 0, stream, q_offsets, slot_parent,
                     slot_token, target_token, max_rows, max_depth, accept_len, accept_slots,
                     bonus_token, status);
  return hipGetLastError() == hipSuccess ? ECHO_OK : ECHO_ERR_HIP;
}

}  // namespace echo
