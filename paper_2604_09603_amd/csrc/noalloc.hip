// echo_gate_noalloc: the top-B gate of echo_gate with its workspace in a
// fixed device array of this library instead of a caller buffer, for callers
// that cannot allocate device memory.  The kernels are echo_gate's.
//
// Each device that calls it holds its own copy of the array (kernel code
// objects are loaded per device) until the process ends.  Its device address
// is looked up once per device, with that device current, and kept; the
// array's name is never handed to a kernel or a copy from host code (there it
// names a host-side stand-in, not device memory).
//
// Nothing in the array has to start at zero: every gate launch writes each
// word it later reads.  Calls on one device share the array, so calls that
// overlap on one device (two streams, two threads) race on it.
#include <mutex>

#include "echo.h"
#include "echo_internal.h"

namespace {

constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[ECHO_GATE_SCRATCH_BYTES];

std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the array on the device of `stream` (the current device
// for the null stream).  The first call on a device makes that device current
// for the lookup and restores the previous one.
int32_t scratch_on(hipStream_t stream, void** out) {
  int cur = 0;
  if (hipGetDevice(&cur) != hipSuccess) return ECHO_ERR_HIP;
  int dev = cur;
  if (stream != nullptr && hipStreamGetDevice(stream, &dev) != hipSuccess) return ECHO_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return ECHO_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_ptr[dev] == nullptr) {
    if (dev != cur && hipSetDevice(dev) != hipSuccess) return ECHO_ERR_HIP;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur && hipSetDevice(cur) != hipSuccess) return ECHO_ERR_HIP;
    if (e != hipSuccess || p == nullptr || (reinterpret_cast<uintptr_t>(p) & 255u) != 0)
      return ECHO_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ECHO_OK;
}

}  // namespace

extern "C" int32_t echo_gate_noalloc(const int32_t* cand_offsets, const int32_t* parent,
                                     const float* logq, int32_t R, int32_t N, int32_t budget,
                                     float* path_score, uint8_t* selected, int32_t* num_selected,
                                     int32_t* status, echo_stream_t stream) {
  if (R < 1 || N < 0 || budget < 0) return ECHO_ERR_INVALID_ARG;
  if (R > ECHO_MAX_REQUESTS || budget > ECHO_MAX_BUDGET) return ECHO_ERR_UNSUPPORTED;
  if (!cand_offsets || !num_selected) return ECHO_ERR_INVALID_ARG;
  if (N > 0 && (!parent || !logq || !selected)) return ECHO_ERR_INVALID_ARG;
  // the size check comes before any runtime call
  if (echo::gate_workspace_bytes(R, N, budget) > size_t(ECHO_GATE_SCRATCH_BYTES))
    return ECHO_ERR_UNSUPPORTED;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  void* ws = nullptr;
  const int32_t rc = scratch_on(s, &ws);
  if (rc != ECHO_OK) return rc;
  return echo::launch_gate(cand_offsets, parent, logq, R, N, budget, nullptr, nullptr, 0,
                           path_score, selected, num_selected, nullptr, ws, status, s);
}
