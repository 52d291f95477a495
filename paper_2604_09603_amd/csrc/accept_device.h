// Greedy acceptance (standard SD, greedy decoding) of one request by one wave,
// shared by the acceptance launch and the fused step's tail kernel: the deepest
// verify slot whose whole root path matches the target argmax.  The request's
// slot parents, tokens and targets are staged in LDS in one round of loads (up
// to `stage` slots; longer requests read memory), each lane walks the parent
// chain of its slots (strictly decreasing slot indices, so every walk ends),
// then a wave reduction picks the deepest valid slot (ties: smallest local slot).
#pragma once

#include "echo_device.h"
#include "echo_internal.h"

namespace echo {
namespace {

// Per-wave LDS staging of accept_request: `stage` entries of each array.
struct AcceptLds {
  int32_t* par;
  int32_t* tok;
  int32_t* tgt;
  int stage;
};

// Request r by the calling wave (every lane of it); the staging belongs to this
// wave alone.
__device__ __forceinline__ void accept_request(
    int r, const int32_t* __restrict__ q_offsets, const int32_t* __restrict__ slot_parent,
    const int32_t* __restrict__ slot_token, const int32_t* __restrict__ target_token,
    int max_rows, int max_depth, int32_t* __restrict__ accept_len,
    int32_t* __restrict__ accept_slots, int32_t* __restrict__ bonus_token, int32_t* status,
    const AcceptLds& lds) {
  const int lane = threadIdx.x & (kWave - 1);
  const int q0 = q_offsets[r];
  const int q1 = q_offsets[r + 1];
  int32_t* out_slots = accept_slots + size_t(r) * max_depth;
  if (q0 < 0 || q1 < q0 || q1 > max_rows) {
    if (lane == 0) status_or(status, ECHO_DATA_BAD_OFFSETS);
    for (int i = lane; i < max_depth; i += kWave) out_slots[i] = -1;
    if (lane == 0) { accept_len[r] = 0; bonus_token[r] = -1; }
    return;
  }
  const int n = q1 - q0;
  const bool staged = n <= lds.stage;
  if (staged) {
    for (int i = lane; i < n; i += kWave) {
      lds.par[i] = slot_parent[q0 + i];
      lds.tok[i] = slot_token[q0 + i];
      lds.tgt[i] = target_token[q0 + i];
    }
  }
  // the staging is read by other lanes of this wave only
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  auto par_of = [&](int x) { return staged ? lds.par[x] : slot_parent[q0 + x]; };
  auto tok_of = [&](int x) { return staged ? lds.tok[x] : slot_token[q0 + x]; };
  auto tgt_of = [&](int x) { return staged ? lds.tgt[x] : target_token[q0 + x]; };
  int bits = 0;
  // best (depth, slot) of this lane; slot 0 (the root) is always valid at depth 0
  int best_d = 0, best_s = 0;
  for (int s = 1 + lane; s < n; s += kWave) {
    const int own_p = par_of(s);
    if (own_p < 0 || own_p >= s) bits |= ECHO_DATA_BAD_SLOT_PARENT;
    bool ok = true;
    int depth = 0;
    int x = s;
    while (x > 0) {
      const int p = par_of(x);
      if (p < 0 || p >= x) { ok = false; break; }
      if (tok_of(x) != tgt_of(p)) { ok = false; break; }
      ++depth;
      x = p;
    }
    if (ok && depth <= max_depth && (depth > best_d || (depth == best_d && s < best_s))) {
      best_d = depth;
      best_s = s;
    }
  }
  // wave argmax: larger depth, then smaller slot
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const int od = __shfl_xor(best_d, off, kWave);
    const int os = __shfl_xor(best_s, off, kWave);
    if (od > best_d || (od == best_d && os < best_s)) { best_d = od; best_s = os; }
  }
  wave_status_or(status, bits);
  if (n == 0) {
    for (int i = lane; i < max_depth; i += kWave) out_slots[i] = -1;
    if (lane == 0) { accept_len[r] = 0; bonus_token[r] = -1; }
    return;
  }
  for (int i = lane; i < max_depth; i += kWave)
    if (i >= best_d) out_slots[i] = -1;
  if (lane == 0) {
    int x = best_s;
    for (int i = best_d - 1; i >= 0; --i) {
      out_slots[i] = q0 + x;
      x = par_of(x);
    }
    accept_len[r] = best_d;
    bonus_token[r] = tgt_of(best_s);
  }
}

}  // namespace
}  // namespace echo
