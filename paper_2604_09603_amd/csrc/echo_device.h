// Device-side helpers shared by the library's HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "echo.h"

namespace echo {

constexpr int kWave = 64;

// Orderable 32-bit key of a path score: larger S -> larger key, -0 == +0.
// -inf (and anything that is not finite-or-zero) maps to 0 = "not selectable".
__device__ __forceinline__ uint32_t score_key(float s) {
  if (!(s > -__builtin_inff())) return 0u;  // -inf or NaN
  uint32_t b = __float_as_uint(s);
  if (b == 0x80000000u) b = 0u;               // -0 -> +0
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ void status_or(int32_t* status, int32_t bits) {
  if (status != nullptr && bits != 0) atomicOr(status, bits);
}

// Status bits of the lanes of a wave.  Bits are rare (invalid data only), so a
// wave whose lanes have none does no more than one ballot, and a lane that has
// some sets them with its own atomic.  Safe in divergent code.
__device__ __forceinline__ void wave_status_or(int32_t* status, int32_t bits) {
  if (status == nullptr || __ballot(bits != 0) == 0ull) return;
  if (bits != 0) atomicOr(status, bits);
}

// Largest r in [0, n) with offs[r] <= x (offs non-decreasing, offs[0] <= x).
template <typename T>
__device__ __forceinline__ int upper_bound_idx(const T* offs, int n, T x) {
  int lo = 0, hi = n;  // invariant: offs[lo] <= x, answer in [lo, hi)
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (offs[mid] <= x) lo = mid; else hi = mid;
  }
  return lo;
}

}  // namespace echo

namespace echo {

// Cross-lane steps of the wave scans below, as DPP moves (GFX9): row_shr:n reads
// the lane n below in the same row of 16 lanes; row_bcast:15 and row_bcast:31
// read lane 15 of the row before, and lane 31, into the rows that the row mask
// enables.  Lanes with no source, and rows the mask leaves out, take `id`.
constexpr int kDppRowShr = 0x110;
constexpr int kDppRowBcast15 = 0x142;
constexpr int kDppRowBcast31 = 0x143;

template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint32_t dpp_move(uint32_t id, uint32_t x) {
  return uint32_t(__builtin_amdgcn_update_dpp(int(id), int(x), kCtrl, kRowMask, 0xf, false));
}

// Inclusive scan of a 32-bit value across one wave (64 lanes, all active) under
// an associative operation with identity `id`: a Hillis-Steele scan within each
// row of 16 lanes (distances 1, 2, 4, 8), then the total of row 0 (row 2) added
// to row 1 (row 3), then lane 31, the total of rows 0-1, added to rows 2 and 3.
template <typename Op>
__device__ __forceinline__ uint32_t wave_scan(uint32_t v, uint32_t id, Op op) {
  v = op(v, dpp_move<kDppRowShr + 1, 0xf>(id, v));
  v = op(v, dpp_move<kDppRowShr + 2, 0xf>(id, v));
  v = op(v, dpp_move<kDppRowShr + 4, 0xf>(id, v));
  v = op(v, dpp_move<kDppRowShr + 8, 0xf>(id, v));
  v = op(v, dpp_move<kDppRowBcast15, 0xa>(id, v));
  v = op(v, dpp_move<kDppRowBcast31, 0xc>(id, v));
  return v;
}

struct AddOp {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a + b; }
};
struct MaxOp {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a > b ? a : b; }
};

// Inclusive prefix sum across one wave (64 lanes, all active).
__device__ __forceinline__ int wave_inclusive_sum(int v) {
  return int(wave_scan(uint32_t(v), 0u, AddOp{}));
}

// Sum and maximum over the 64 lanes of a wave (all active), in every lane.
__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
  return uint32_t(__builtin_amdgcn_readlane(int(wave_scan(v, 0u, AddOp{})), kWave - 1));
}
__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
  return uint32_t(__builtin_amdgcn_readlane(int(wave_scan(v, 0u, MaxOp{})), kWave - 1));
}

// Exclusive prefix sum over a whole block of NT threads; *total receives the
// block sum.  `scratch` must hold NT/64 + 1 ints of shared memory.  Each wave
// scans its lanes, then every wave scans the wave totals for itself.  Contains
// two __syncthreads(): every thread of the block must call it, and it may be
// called again right away with the same scratch.
template <int NT>
__device__ __forceinline__ int block_exclusive_sum(int v, int* scratch, int* total) {
  constexpr int NW = NT / kWave;
  static_assert(NW <= kWave, "one lane per wave total");
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = __builtin_amdgcn_readfirstlane(int(threadIdx.x / kWave));
  const int inc = wave_inclusive_sum(v);
  if (lane == kWave - 1) scratch[wid] = inc;
  __syncthreads();
  const int t = lane < NW ? scratch[lane] : 0;
  const int tinc = wave_inclusive_sum(t);
  *total = __builtin_amdgcn_readlane(tinc, NW - 1);
  const int base = __builtin_amdgcn_readlane(tinc - t, wid);
  __syncthreads();  // the next call may write the scratch
  return base + inc - v;
}

// Two exclusive prefix sums at once (same barriers as one); *total_x and
// *total_y receive the block sums.  `scratch` holds NT/64 + 1 int2 of shared
// memory.
template <int NT>
__device__ __forceinline__ int2 block_exclusive_sum2(int2 v, int2* scratch, int* total_x,
                                                     int* total_y) {
  constexpr int NW = NT / kWave;
  static_assert(NW <= kWave, "one lane per wave total");
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = __builtin_amdgcn_readfirstlane(int(threadIdx.x / kWave));
  const int ix = wave_inclusive_sum(v.x);
  const int iy = wave_inclusive_sum(v.y);
  if (lane == kWave - 1) scratch[wid] = make_int2(ix, iy);
  __syncthreads();
  const int2 t = lane < NW ? scratch[lane] : make_int2(0, 0);
  const int tx = wave_inclusive_sum(t.x);
  const int ty = wave_inclusive_sum(t.y);
  *total_x = __builtin_amdgcn_readlane(tx, NW - 1);
  *total_y = __builtin_amdgcn_readlane(ty, NW - 1);
  const int bx = __builtin_amdgcn_readlane(tx - t.x, wid);
  const int by = __builtin_amdgcn_readlane(ty - t.y, wid);
  __syncthreads();  // the next call may write the scratch
  return make_int2(bx + ix - v.x, by + iy - v.y);
}

}  // namespace echo
