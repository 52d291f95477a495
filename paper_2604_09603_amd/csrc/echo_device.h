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

// Wave-wide OR of a per-lane int (for status bits), then one atomic per wave.
__device__ __forceinline__ void wave_status_or(int32_t* status, int32_t bits) {
  if (status == nullptr) return;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) bits |= __shfl_xor(bits, off, kWave);
  if ((threadIdx.x & (kWave - 1)) == 0 && bits != 0) atomicOr(status, bits);
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

// Inclusive prefix sum across one wave (64 lanes).
__device__ __forceinline__ int wave_inclusive_sum(int v) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    int u = __shfl_up(v, off, kWave);
    if (lane >= off) v += u;
  }
  return v;
}

// Exclusive prefix sum over a whole block of NT threads; *total receives the
// block sum.  `scratch` must hold NT/64 + 1 ints of shared memory.  Contains
// three __syncthreads(): every thread of the block must call it, and it may be
// called again right away with the same scratch.
template <int NT>
__device__ __forceinline__ int block_exclusive_sum(int v, int* scratch, int* total) {
  constexpr int NW = NT / kWave;
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = threadIdx.x / kWave;
  int inc = wave_inclusive_sum(v);
  if (lane == kWave - 1) scratch[wid] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < NW; ++w) { int t = scratch[w]; scratch[w] = run; run += t; }
    scratch[NW] = run;
  }
  __syncthreads();
  int ex = scratch[wid] + inc - v;
  *total = scratch[NW];
  __syncthreads();
  return ex;
}

// Two exclusive prefix sums at once (same barriers as one); *total_x and
// *total_y receive the block sums.  `scratch` holds NT/64 + 1 int2 of shared
// memory.
template <int NT>
__device__ __forceinline__ int2 block_exclusive_sum2(int2 v, int2* scratch, int* total_x,
                                                     int* total_y) {
  constexpr int NW = NT / kWave;
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = threadIdx.x / kWave;
  int ix = v.x, iy = v.y;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int ux = __shfl_up(ix, off, kWave);
    const int uy = __shfl_up(iy, off, kWave);
    if (lane >= off) {
      ix += ux;
      iy += uy;
    }
  }
  if (lane == kWave - 1) scratch[wid] = make_int2(ix, iy);
  __syncthreads();
  if (threadIdx.x == 0) {
    int rx = 0, ry = 0;
    for (int w = 0; w < NW; ++w) {
      const int2 t = scratch[w];
      scratch[w] = make_int2(rx, ry);
      rx += t.x;
      ry += t.y;
    }
    scratch[NW] = make_int2(rx, ry);
  }
  __syncthreads();
  const int2 base = scratch[wid];
  const int2 tot = scratch[NW];
  *total_x = tot.x;
  *total_y = tot.y;
  __syncthreads();
  return make_int2(base.x + ix - v.x, base.y + iy - v.y);
}

}  // namespace echo
