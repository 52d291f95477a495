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

// Non-zero bytes of a 32-bit word as 4 bits (byte i -> bit i).
__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t w) {
  uint32_t y = w | (w >> 4);
  y |= y >> 2;
  y |= y >> 1;
  y &= 0x01010101u;                  // bit 0 of each byte: that byte was non-zero
  return (y * 0x02040810u) >> 25 & 0xFu;  // gather bits 0, 8, 16, 24 at 25..28
}

// 16-bit mask of the non-zero bytes of 16 flags (bit b: byte b), keeping the n
// first (n <= 0: none).
__device__ __forceinline__ uint32_t chunk_bits(const uint32_t (&w)[4], int n) {
  const uint32_t m = nonzero_bytes(w[0]) | (nonzero_bytes(w[1]) << 4) |
                     (nonzero_bytes(w[2]) << 8) | (nonzero_bytes(w[3]) << 12);
  return n >= 16 ? m : (n <= 0 ? 0u : m & ((1u << n) - 1u));
}

// The compaction reads the flags in rounds of kMaskThreads * kBytesPerThread
// candidates.  Wave w takes the kWave * kBytesPerThread candidates from
// round + w * kWaveSpan on; its lane l reads the 16-byte chunks l, l + 64, ... of
// them, so that each load of the wave covers 1 KB of consecutive flags.  m[v]
// receives the bits of the lane's chunk v (candidates past N count as zero).
// Every load is issued before the first is used: chunks at or past N read the
// chunk holding flag N - 1 instead and are dropped afterwards.
constexpr int kChunksPerLane = kBytesPerThread / 16;
constexpr int kWaveSpan = kWave * kBytesPerThread;

template <bool kAligned>
__device__ __forceinline__ void load_round(const uint8_t* __restrict__ sel, int base, int N,
                                           uint32_t (&m)[kChunksPerLane]) {
  const int wbase = base + int(threadIdx.x / kWave) * kWaveSpan;
  if (wbase >= N) {  // the whole wave past the end: no loads
#pragma unroll
    for (int v = 0; v < kChunksPerLane; ++v) m[v] = 0u;
    return;
  }
  const int c0 = wbase + int(threadIdx.x & (kWave - 1)) * 16;
  const int last = (N - 1) & ~15;  // the chunk that holds the last flag (N > 0)
  uint32_t w[kChunksPerLane][4];
  if (kAligned) {
    // 16-byte loads, also of the chunk that holds the last flag: a 16-byte
    // aligned block never crosses a page, and the bytes past N are dropped
#pragma unroll
    for (int v = 0; v < kChunksPerLane; ++v) {
      const uint4 q = *reinterpret_cast<const uint4*>(sel + min(c0 + v * kWave * 16, last));
      w[v][0] = q.x;
      w[v][1] = q.y;
      w[v][2] = q.z;
      w[v][3] = q.w;
    }
  } else {
    // an array that is not 16-byte aligned: single bytes, addresses clamped
    // into the array
    uint8_t bt[kChunksPerLane][16];
#pragma unroll
    for (int v = 0; v < kChunksPerLane; ++v)
#pragma unroll
      for (int k = 0; k < 16; ++k) bt[v][k] = sel[min(c0 + v * kWave * 16 + k, N - 1)];
#pragma unroll
    for (int v = 0; v < kChunksPerLane; ++v)
#pragma unroll
      for (int u = 0; u < 4; ++u)
        w[v][u] = uint32_t(bt[v][4 * u]) | (uint32_t(bt[v][4 * u + 1]) << 8) |
                  (uint32_t(bt[v][4 * u + 2]) << 16) | (uint32_t(bt[v][4 * u + 3]) << 24);
  }
#pragma unroll
  for (int v = 0; v < kChunksPerLane; ++v) m[v] = chunk_bits(w[v], N - (c0 + v * kWave * 16));
}

// The request tables that flatten & pack starts from, entry r = tid + kMaskThreads k
// of each in this thread's registers: candidate offsets (r <= R), root tokens and
// prefix lengths (r < R).  The loads are issued together, before anything waits.
struct MaskTables {
  int32_t offs[kRootsPerThread];
  int32_t rtok[kRootsPerThread];
  int32_t plen[kRootsPerThread];
};

__device__ __forceinline__ MaskTables load_mask_tables(const int32_t* __restrict__ cand_offsets,
                                                       const int32_t* __restrict__ root_token,
                                                       const int32_t* __restrict__ prefix_len,
                                                       int R) {
  MaskTables t;
#pragma unroll
  for (int k = 0; k < kRootsPerThread; ++k) {
    const int r = int(threadIdx.x) + kMaskThreads * k;
    t.offs[k] = r <= R ? cand_offsets[r] : 0;
    t.rtok[k] = r < R ? root_token[r] : 0;
    t.plen[k] = r < R ? prefix_len[r] : 0;
  }
  return t;
}

// The whole flatten & pack on one workgroup of kMaskThreads, from the tables
// load_mask_tables returned; `smem` holds mask_lds_bytes(R, budget) bytes of LDS.
template <bool kAligned>
__device__ void mask_body(
    const MaskTables& tab, const int32_t* __restrict__ parent,
    const int32_t* __restrict__ token, const uint8_t* __restrict__ selected, int R, int N,
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
  uint32_t m0[kChunksPerLane] = {};
  if (N > 0) load_round<kAligned>(selected, 0, N, m0);
  // the tables into LDS; a request's root token waits in its slot-offset entry,
  // which the same thread reads before it writes the offset in step 2
#pragma unroll
  for (int k = 0; k < kRootsPerThread; ++k) {
    const int r = tid + kMaskThreads * k;
    if (r <= R) s_offs[r] = tab.offs[k];
    if (r < R) {
      s_plen[r] = tab.plen[k];
      s_qoff[r] = tab.rtok[k];
    }
  }
  if (tid == 0) s_flag = 0;
  __syncthreads();
  // the CSR: starts at 0, ends at N, never decreases (any failing thread sets the flag)
  for (int r = tid; r <= R; r += kMaskThreads)
    if ((r == 0 && s_offs[0] != 0) || (r == R && s_offs[R] != N) ||
        (r < R && s_offs[r + 1] < s_offs[r]))
      s_flag = 1;
  __syncthreads();
  const bool ok = s_flag == 0;
  int bits = 0;
  if (!ok && tid == 0) bits |= ECHO_DATA_BAD_OFFSETS;

  // 1. ordered compaction of the selection.  Within a wave the candidates run
  // chunk by chunk (chunk v of every lane, lane order, then chunk v + 1), so a
  // lane's position for chunk v is the wave's base, the wave's counts of the
  // chunks before v, and the counts of chunk v in the lanes below it.
  int count = 0;  // uniform
  if (ok) {
    const int lane = tid & (kWave - 1);
    for (int base = 0; base < N; base += kMaskThreads * kBytesPerThread) {
      uint32_t m[kChunksPerLane];
      if (base == 0) {
#pragma unroll
        for (int v = 0; v < kChunksPerLane; ++v) m[v] = m0[v];
      } else {
        load_round<kAligned>(selected, base, N, m);
      }
      // the counts of chunks 2q and 2q + 1 in the low and high halves of one word
      // (at most 64 * 16 per wave, so the halves never carry into each other)
      uint32_t inc[kChunksPerLane / 2];
      int mine = 0;
#pragma unroll
      for (int q = 0; q < kChunksPerLane / 2; ++q) {
        const uint32_t lo = uint32_t(__popc(m[2 * q])), hi = uint32_t(__popc(m[2 * q + 1]));
        mine += int(lo + hi);
        inc[q] = wave_scan(lo | (hi << 16), 0u, AddOp{});
      }
      int tot;
      const int ex = block_exclusive_sum<kMaskThreads>(mine, s_scan, &tot);
      int run = count + __builtin_amdgcn_readfirstlane(ex);  // lane 0: the waves before this one
      const int c0 = base + (tid / kWave) * kWaveSpan + lane * 16;
      // position of the lane's first selected candidate in each chunk
      int first[kChunksPerLane];
#pragma unroll
      for (int v = 0; v < kChunksPerLane; ++v) {
        const uint32_t word = inc[v / 2];
        const uint32_t all = uint32_t(__builtin_amdgcn_readlane(int(word), kWave - 1));
        const int sh = (v & 1) * 16;
        first[v] = run + int((word >> sh) & 0xFFFFu) - __popc(m[v]);
        run += int((all >> sh) & 0xFFFFu);
      }
      // one loop over all of the lane's selected candidates, in order: a wave runs
      // as many rounds as its lane with the most of them (a run of selected nodes
      // usually sits in one chunk of one lane)
      uint64_t lo = 0ull, hi = 0ull;
#pragma unroll
      for (int v = 0; v < kChunksPerLane / 2; ++v) {
        lo |= uint64_t(m[v]) << (16 * v);
        hi |= uint64_t(m[v + kChunksPerLane / 2]) << (16 * v);
      }
      int cur = -1, pos = 0;
      while (lo | hi) {
        int b;
        if (lo != 0ull) {
          b = __ffsll(static_cast<long long>(lo)) - 1;
          lo &= lo - 1ull;
        } else {
          b = 64 + __ffsll(static_cast<long long>(hi)) - 1;
          hi &= hi - 1ull;
        }
        const int v = b >> 4;
        if (v != cur) {
          cur = v;
          pos = first[0];
#pragma unroll
          for (int u = 1; u < kChunksPerLane; ++u) pos = v == u ? first[u] : pos;
        }
        if (pos < budget) s_comp[pos] = c0 + v * kWave * 16 + (b & 15);
        ++pos;
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
    const int32_t root = s_qoff[r];
    int v = r + lower_bound_lds(s_comp, 0, n_inc, s_offs[r]);
    s_qoff[r] = v;
    q_offsets[r] = v;
    slot_cand[v] = -1;
    slot_parent[v] = -1;
    slot_token[v] = root;
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
