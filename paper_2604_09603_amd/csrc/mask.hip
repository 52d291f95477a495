// Flatten & pack (Fig. 3, stage 3): the selected super-tree becomes per-request
// verify slots with parent slots, position ids and ancestor bitmasks.
//
// One workgroup of 1024 threads (the selection holds at most B <= 16384 nodes,
// so the whole step is latency-bound and a single CU avoids any grid-wide
// synchronisation):
//   1. ordered compaction of `selected` (64 bytes per thread per round, one
//      block scan per round) into an LDS list of global indices, ascending;
//   2. q_offsets[r] = r + #(packed candidates before request r) (binary search);
//   3. one thread per slot walks its candidate's ancestor chain, marking the
//      packed ancestors (binary search in the LDS list) in its bitmask row.
#include "echo_device.h"
#include "echo_internal.h"

namespace echo {
namespace {

constexpr int kMaskThreads = 1024;
constexpr int kBytesPerThread = 64;
constexpr int kRegWords = 8;  // mask words kept in registers; the rest is updated in memory

// First index i in [lo, hi) with a[i] >= x (hi if none).
__device__ __forceinline__ int lower_bound_lds(const int32_t* a, int lo, int hi, int32_t x) {
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if (a[mid] < x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

template <bool kAligned>
__device__ __forceinline__ uint64_t load_flags(const uint8_t* __restrict__ sel, int start, int N) {
  uint64_t bits = 0;
  if (kAligned && start + kBytesPerThread <= N) {
    const uint4* p = reinterpret_cast<const uint4*>(sel + start);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      uint4 w = p[v];
      uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int b = 0; b < 4; ++b)
          if ((ws[u] >> (8 * b)) & 0xFFu) bits |= uint64_t(1) << (16 * v + 4 * u + b);
    }
  } else {
    for (int b = 0; b < kBytesPerThread; ++b) {
      int g = start + b;
      if (g < N && sel[g] != 0) bits |= uint64_t(1) << b;
    }
  }
  return bits;
}

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
  int32_t* s_offs = smem;              // R + 1
  int32_t* s_qoff = smem + (R + 1);    // R + 1
  int32_t* s_comp = smem + 2 * (R + 1);  // budget
  __shared__ int s_scan[kMaskThreads / kWave + 1];
  __shared__ int s_flag;

  const int tid = threadIdx.x;
  for (int i = tid; i <= R; i += kMaskThreads) s_offs[i] = cand_offsets[i];
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
      uint64_t f = start < N ? load_flags<kAligned>(selected, start, N) : 0ull;
      int tot;
      int pos = count + block_exclusive_sum<kMaskThreads>(__popcll(f), s_scan, &tot);
      while (f) {
        int b = __ffsll(static_cast<long long>(f)) - 1;
        f &= f - 1;
        if (pos < budget) s_comp[pos] = start + b;
        ++pos;
      }
      count += tot;
    }
  }
  if (count > budget && tid == 0) bits |= ECHO_DATA_OVER_CAPACITY;
  const int n_inc = count < budget ? count : budget;
  __syncthreads();

  // 2. slot offsets
  for (int r = tid; r < R; r += kMaskThreads) {
    int v = r + lower_bound_lds(s_comp, 0, n_inc, s_offs[r]);
    s_qoff[r] = v;
    q_offsets[r] = v;
  }
  if (tid == 0) {
    s_qoff[R] = R + n_inc;
    q_offsets[R] = R + n_inc;
  }
  __syncthreads();

  // 3. one thread per slot
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
    if (j == 0) {
      slot_cand[s] = -1;
      slot_parent[s] = -1;
      slot_token[s] = root_token[r];
      position_ids[s] = prefix_len[r];
    } else {
      const int cbase = s_qoff[r] - r;             // list index of the request's first packed node
      const int cend = s_qoff[r + 1] - (r + 1);
      const int g = s_comp[s - r - 1];
      const int lo = s_offs[r];
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
      int p = parent[g];
      if (p < -1 || p >= g - lo) { bits |= ECHO_DATA_BAD_PARENT; p = -1; }
      int pj = 0;
      int depth = 1;
      bool found_parent = false;
      while (p >= 0) {
        const int x = lo + p;
        const int idx = lower_bound_lds(s_comp, cbase, cend, x);
        if (idx < cend && s_comp[idx] == x) {
          const int lj = idx - cbase + 1;
          if (!found_parent) { pj = lj; found_parent = true; }
          set_bit(lj);
          ++depth;
        } else if (!found_parent) {
          bits |= ECHO_DATA_NOT_CLOSED;
        }
        int pp = parent[x];
        if (pp < -1 || pp >= p) { bits |= ECHO_DATA_BAD_PARENT; pp = -1; }
        p = pp;
      }
      if (depth > ECHO_MAX_DEPTH) bits |= ECHO_DATA_TOO_DEEP;
      slot_cand[s] = g;
      slot_parent[s] = pj;
      slot_token[s] = token[g];
      position_ids[s] = prefix_len[r] + depth;
    }
#pragma unroll
    for (int w = 0; w < kRegWords; ++w)
      if (w < W) row[w] = regs[w];
  }
  wave_status_or(status, bits);
}

}  // namespace

size_t mask_lds_bytes(int32_t R, int32_t budget) {
  return size_t(2 * (R + 1) + budget) * sizeof(int32_t);
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
