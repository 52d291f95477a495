// Flatten & pack (Fig. 3, stage 3) as a device function, shared by the mask
// launch and the fused step's front kernel.
#pragma once

#include "echo_device.h"
#include "echo_internal.h"

namespace echo {
namespace {

constexpr int kMaskThreads = 1024;
constexpr int kBytesPerThread = 128;
constexpr int kRegWords = 8;  // mask words kept in registers; the rest is updated in memory
constexpr int kRootsPerThread = (ECHO_MAX_REQUESTS + kMaskThreads) / kMaskThreads;

// First index i in [lo, hi) with a[i] >= x (hi if none).
__device__ __forceinline__ int lower_bound_lds(const int32_t* a, int lo, int hi, int32_t x) {
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if (a[mid] < x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// Selection flags of 128 consecutive candidates as a 128-bit mask (bit b: byte
// start + b is non-zero).
struct Flags {
  uint64_t lo, hi;
};

// Non-zero bytes of a 32-bit word as 4 bits (byte i -> bit i).
__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t w) {
  uint32_t y = w | (w >> 4);
  y |= y >> 2;
  y |= y >> 1;
  y &= 0x01010101u;                  // bit 0 of each byte: that byte was non-zero
  return (y * 0x02040810u) >> 25 & 0xFu;  // gather bits 0, 8, 16, 24 at 25..28
}

template <bool kAligned>
__device__ __forceinline__ Flags load_flags(const uint8_t* __restrict__ sel, int start, int N) {
  constexpr int kWords = kBytesPerThread / 4;
  uint32_t w[kWords];
  if (kAligned && start + kBytesPerThread <= N) {
    const uint4* p = reinterpret_cast<const uint4*>(sel + start);
#pragma unroll
    for (int v = 0; v < kWords / 4; ++v) {
      const uint4 q = p[v];
      w[4 * v] = q.x;
      w[4 * v + 1] = q.y;
      w[4 * v + 2] = q.z;
      w[4 * v + 3] = q.w;
    }
  } else {
    // the end of the array, or an array that is not 16-byte aligned: single
    // bytes, every load issued before the first is used (one memory round trip,
    // not one per byte).  Addresses are clamped into the array (start < N) and
    // the bytes past its end are dropped afterwards.
    uint8_t bt[kBytesPerThread];
#pragma unroll
    for (int k = 0; k < kBytesPerThread; ++k) bt[k] = sel[min(start + k, N - 1)];
#pragma unroll
    for (int v = 0; v < kWords; ++v) {
      uint32_t x = 0u;
#pragma unroll
      for (int k = 0; k < 4; ++k)
        x |= (start + 4 * v + k < N ? uint32_t(bt[4 * v + k]) : 0u) << (8 * k);
      w[v] = x;
    }
  }
  Flags f = {0ull, 0ull};
#pragma unroll
  for (int v = 0; v < kWords / 4; ++v) {
    const uint64_t nib = uint64_t(nonzero_bytes(w[4 * v])) |
                         (uint64_t(nonzero_bytes(w[4 * v + 1])) << 4) |
                         (uint64_t(nonzero_bytes(w[4 * v + 2])) << 8) |
                         (uint64_t(nonzero_bytes(w[4 * v + 3])) << 12);
    if (v < 4) f.lo |= nib << (16 * v);
    else f.hi |= nib << (16 * (v - 4));
  }
  return f;
}

// The whole flatten & pack on one workgroup of kMaskThreads; `smem` holds
// mask_lds_bytes(R, budget) bytes of LDS.
template <bool kAligned>
__device__ void mask_body(
    const int32_t* __restrict__ cand_offsets, const int32_t* __restrict__ parent,
    const int32_t* __restrict__ token, const uint8_t* __restrict__ selected,
    const int32_t* __restrict__ root_token, const int32_t* __restrict__ prefix_len, int R, int N,
    int budget, int32_t* __restrict__ q_offsets, int32_t* __restrict__ slot_cand,
    int32_t* __restrict__ slot_parent, int32_t* __restrict__ slot_token,
    int32_t* __restrict__ position_ids, uint32_t* __restrict__ tree_mask, int W,
    int32_t* status, int32_t* smem) {
  int32_t* s_offs = smem;              // R + 1
  int32_t* s_qoff = smem + (R + 1);    // R + 1
  int32_t* s_plen = smem + 2 * (R + 1);  // R + 1 (prefix lengths)
  int32_t* s_comp = smem + 3 * (R + 1);  // budget
  // local slot of each packed node's nearest packed ancestor (0: the root)
  uint16_t* s_pslot = reinterpret_cast<uint16_t*>(smem + 3 * (R + 1) + budget);
  __shared__ int s_scan[kMaskThreads / kWave + 1];
  __shared__ int s_flag;

  const int tid = threadIdx.x;
  // the first round of flags is loaded together with the CSR
  Flags f0 = tid * kBytesPerThread < N ? load_flags<kAligned>(selected, tid * kBytesPerThread, N)
                                       : Flags{0ull, 0ull};
  // root tokens of this thread's requests (r = tid + 1024 k), stored in step 2
  int32_t rtok[kRootsPerThread];
#pragma unroll
  for (int k = 0; k < kRootsPerThread; ++k) {
    const int r = tid + kMaskThreads * k;
    rtok[k] = r < R ? root_token[r] : 0;
  }
  for (int i = tid; i <= R; i += kMaskThreads) {
    s_offs[i] = cand_offsets[i];
    if (i < R) s_plen[i] = prefix_len[i];
  }
  __syncthreads();
  if (tid == 0) s_flag = (s_offs[0] != 0 || s_offs[R] != N) ? 1 : 0;
  __syncthreads();
  for (int r = tid; r < R; r += kMaskThreads)
    if (s_offs[r + 1] < s_offs[r]) s_flag = 1;
  __syncthreads();
  const bool ok = s_flag == 0;
  int bits = 0;
  if (!ok && tid == 0) bits |= ECHO_DATA_BAD_OFFSETS;

  // 1. ordered compaction of the selection
  int count = 0;  // uniform
  if (ok) {
    for (int base = 0; base < N; base += kMaskThreads * kBytesPerThread) {
      const int start = base + tid * kBytesPerThread;
      Flags f = base == 0 ? f0
                          : (start < N ? load_flags<kAligned>(selected, start, N)
                                       : Flags{0ull, 0ull});
      int tot;
      int pos = count + block_exclusive_sum<kMaskThreads>(__popcll(f.lo) + __popcll(f.hi), s_scan,
                                                          &tot);
      for (int half = 0; half < 2; ++half) {
        uint64_t m = half ? f.hi : f.lo;
        while (m) {
          const int b = __ffsll(static_cast<long long>(m)) - 1;
          m &= m - 1;
          if (pos < budget) s_comp[pos] = start + 64 * half + b;
          ++pos;
        }
      }
      count += tot;
    }
  }
  if (count > budget && tid == 0) bits |= ECHO_DATA_OVER_CAPACITY;
  const int n_inc = count < budget ? count : budget;
  __syncthreads();

  // 2. slot offsets and the root slots
#pragma unroll
  for (int k = 0; k < kRootsPerThread; ++k) {
    const int r = tid + kMaskThreads * k;
    if (r >= R) break;
    int v = r + lower_bound_lds(s_comp, 0, n_inc, s_offs[r]);
    s_qoff[r] = v;
    q_offsets[r] = v;
    slot_cand[v] = -1;
    slot_parent[v] = -1;
    slot_token[v] = rtok[k];
    position_ids[v] = s_plen[r];
  }
  if (tid == 0) {
    s_qoff[R] = R + n_inc;
    q_offsets[R] = R + n_inc;
  }
  __syncthreads();

  // 3. nearest packed ancestor of every packed node, as a local slot
  for (int i = tid; i < n_inc; i += kMaskThreads) {
    const int g = s_comp[i];
    const int r = upper_bound_idx(s_offs, R + 1, g);  // request of g
    const int lo = s_offs[r];
    const int cbase = s_qoff[r] - r;                  // list index of the request's first packed node
    const int cend = s_qoff[r + 1] - (r + 1);
    int p = parent[g];
    const int s = s_qoff[r] + 1 + (i - cbase);  // this node's slot
    slot_cand[s] = g;
    slot_token[s] = token[g];
    if (p < -1 || p >= g - lo) { bits |= ECHO_DATA_BAD_PARENT; p = -1; }
    int pslot = 0;
    bool first = true;
    while (p >= 0) {
      const int x = lo + p;
      const int idx = lower_bound_lds(s_comp, cbase, cend, x);
      if (idx < cend && s_comp[idx] == x) { pslot = idx - cbase + 1; break; }
      if (first) bits |= ECHO_DATA_NOT_CLOSED;  // attach to the nearest packed ancestor
      first = false;
      int pp = parent[x];
      if (pp < -1 || pp >= p) { bits |= ECHO_DATA_BAD_PARENT; pp = -1; }
      p = pp;
    }
    s_pslot[i] = static_cast<uint16_t>(pslot);
  }
  __syncthreads();

  // 4. one thread per slot: ancestor bits, parent slot, depth
  const int nslots = R + n_inc;
  for (int s = tid; s < nslots; s += kMaskThreads) {
    const int r = upper_bound_idx(s_qoff, R + 1, s);
    const int j = s - s_qoff[r];
    uint32_t* row = tree_mask + size_t(s) * W;
    uint32_t regs[kRegWords];
#pragma unroll
    for (int w = 0; w < kRegWords; ++w) regs[w] = 0u;
    for (int w = kRegWords; w < W; ++w) row[w] = 0u;
    regs[0] = 1u;  // the root is everyone's ancestor
    if (j > 0) {
      const int cbase = s_qoff[r] - r;
      auto set_bit = [&](int lj) {
        const int w = lj >> 5;
        const uint32_t m = 1u << (lj & 31);
        if (w < kRegWords) {
#pragma unroll
          for (int u = 0; u < kRegWords; ++u)
            if (u == w) regs[u] |= m;
        } else {
          row[w] |= m;
        }
      };
      set_bit(j);
      const int pj = s_pslot[cbase + j - 1];
      int depth = 1;
      // local slots strictly decrease along the chain, so the walk ends
      for (int x = pj; x > 0; x = s_pslot[cbase + x - 1]) {
        set_bit(x);
        ++depth;
      }
      if (depth > ECHO_MAX_DEPTH) bits |= ECHO_DATA_TOO_DEEP;
      slot_parent[s] = pj;
      position_ids[s] = s_plen[r] + depth;
    }
#pragma unroll
    for (int w = 0; w < kRegWords; ++w)
      if (w < W) row[w] = regs[w];
  }
  wave_status_or(status, bits);
}

}  // namespace
}  // namespace echo
