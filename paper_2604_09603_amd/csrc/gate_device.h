// Gate state shared by the gate launches and the fused step's front kernel:
// the workspace layout, the radix selection and the last phase of the global
// top-B selection (eq. 4).
#pragma once

#include "echo_device.h"
#include "echo_internal.h"

namespace echo {
namespace {

constexpr int kGateThreads = 1024;
constexpr int kHistBins = 2048;   // top 11 bits of the key
constexpr int kHistShift = 21;
constexpr int kSortCap = 8192;    // candidates gate_finish gathers into LDS
constexpr int kWinBack = 3072;    // nodes before a score block kept in its LDS window
constexpr int kWin = kWinBack + kGateThreads;
constexpr int kDepths = ECHO_MAX_DEPTH + 1;  // per-request depth slots (0 = root, unused)
constexpr int kTabReq = 64;                  // requests per score block with an LDS max table

struct GateMeta {
  int32_t num_selected;  // m
  uint32_t bin;          // histogram bin of the m-th largest key
  uint32_t bin_need;     // how many keys of that bin are selected
  uint32_t bin_cnt;      // keys in that bin
  uint32_t thr_key;      // selected iff key > thr_key || (key == thr_key && g <= thr_g)
  int32_t thr_g;
};

struct GateWs {
  GateMeta* meta;
  uint32_t* keys;    // [N] orderable key, 0 = never selected
  int32_t* pglob;    // [N] clamped parent, global index (-1: child of the root)
  uint32_t* bhist;   // [nblocks][2048] per-block histograms
  uint32_t* ccount;  // [nblocks] candidates found by each select block
  uint2* bsum;       // [nblocks] (finite keys, highest occupied bin + 1) of each score block
  uint2* cand;       // [nblocks * 1024] (key, index) candidates, block slices
  uint32_t* lmax;    // [R][kDepths] max key per (request, depth), checkpoint depths only
  uint8_t* depth;    // [N] node depth (1 = child of the root), capped at ECHO_MAX_DEPTH + 1
};

// Checkpoint table of sparse gating: request r passes depth d iff the largest
// path score among its depth-d nodes is above lt[d] (eq. 7 in the log domain).
struct SparseArgs {
  int enabled;
  uint32_t mask;     // bit d set iff depth d is a checkpoint
  float lt[kDepths]; // ln tau of each checkpoint depth (the largest if repeated)
  int32_t* trunc_out;  // nullable [R]: first failed checkpoint, ECHO_MAX_DEPTH + 1 if none
};

__host__ __device__ inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

__host__ __device__ inline int gate_blocks(int32_t N) {
  return N > 0 ? (N + kGateThreads - 1) / kGateThreads : 1;
}

__host__ __device__ inline GateWs gate_ws_layout(void* base, int32_t N, int32_t R) {
  const size_t nb = size_t(gate_blocks(N));
  char* p = static_cast<char*>(base);
  GateWs w;
  w.meta = reinterpret_cast<GateMeta*>(p);
  p += 256;
  w.keys = reinterpret_cast<uint32_t*>(p);
  p += align_up(size_t(N) * 4, 256);
  w.pglob = reinterpret_cast<int32_t*>(p);
  p += align_up(size_t(N) * 4, 256);
  w.bhist = reinterpret_cast<uint32_t*>(p);
  p += align_up(nb * kHistBins * 4, 256);
  w.ccount = reinterpret_cast<uint32_t*>(p);
  p += align_up(nb * 4, 256);
  w.bsum = reinterpret_cast<uint2*>(p);
  p += align_up(nb * 8, 256);
  w.cand = reinterpret_cast<uint2*>(p);
  p += align_up(nb * kGateThreads * 8, 256);
  w.lmax = reinterpret_cast<uint32_t*>(p);
  p += align_up(size_t(R) * kDepths * 4, 256);
  w.depth = reinterpret_cast<uint8_t*>(p);
  return w;
}

// --------------------------------------------------------------- finish ----
// Radix selection: among the entries i < n with match(i), each carrying an
// unsigned value val(i), find the value of the need-th largest, 8 bits at a
// time from the top.  A step counts the entries whose value has the known high
// bits into a 256-bin LDS histogram and one wave finds the bin where the count
// from the top reaches need.  Once every entry matching the known bits is
// selected (need == cnt) the lower bits no longer matter and the walk stops.
struct RadixSel {
  uint32_t prefix;  // known high bits of the value (value >> shift)
  int shift;        // number of still unknown low bits
  uint32_t need;    // rank of the sought entry among those matching the prefix (1..cnt)
  uint32_t cnt;     // entries matching the prefix
};

struct RadixLds {
  uint32_t h[2][256];  // histograms, used alternately
  int d[2][2];         // (bin, count above the bin) of each step
};

// One wave: the bin of h whose cumulative count from bin 255 downwards first
// reaches need, and the count of the bins above it.
__device__ __forceinline__ void digit_search(const uint32_t* h, uint32_t need, int* out) {
  const int lane = threadIdx.x & (kWave - 1);
  uint32_t c[4];
  uint32_t sum = 0u;
#pragma unroll
  for (int j = 0; j < 4; ++j) {  // lane l holds bins 255-4l .. 252-4l, highest first
    c[j] = h[255 - 4 * lane - j];
    sum += c[j];
  }
  const uint32_t incl = wave_scan(sum, 0u, AddOp{});
  const unsigned long long hit = __ballot(incl >= need);
  const int l0 = hit != 0ull ? __builtin_ctzll(hit) : 0;
  if (lane == l0) {
    uint32_t above = incl - sum;
    int j = 0;
    for (; j < 3; ++j) {
      if (above + c[j] >= need) break;
      above += c[j];
    }
    out[0] = 255 - 4 * lane - j;
    out[1] = int(above);
  }
}

// The histograms of both buffers must be zero on entry; they are on return.
template <typename Val, typename Match>
__device__ void radix_select(RadixSel& st, int n, Val val, Match match, RadixLds& L) {
  int cur = 0;
  while (st.shift > 0 && st.need < st.cnt) {
    const int bits = st.shift >= 8 ? 8 : st.shift;
    const int nsh = st.shift - bits;
    const uint32_t pre = st.prefix, sh = uint32_t(st.shift);
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
      if (match(i)) {
        const uint32_t v = val(i);
        if ((v >> sh) == pre) atomicAdd(&L.h[cur][(v >> nsh) & ((1u << bits) - 1u)], 1u);
      }
    }
    __syncthreads();
    if (threadIdx.x < kWave) {
      digit_search(L.h[cur], st.need, L.d[cur]);
    } else {  // the other buffer was read before the barrier above
      for (int i = threadIdx.x - kWave; i < 256; i += blockDim.x - kWave) L.h[cur ^ 1][i] = 0u;
    }
    __syncthreads();
    const int d = L.d[cur][0];
    st.need -= uint32_t(L.d[cur][1]);
    st.cnt = L.h[cur][d];
    st.prefix = (pre << bits) | uint32_t(d);
    st.shift = nsh;
    cur ^= 1;
  }
  __syncthreads();  // every thread has read the last histogram
  for (int i = threadIdx.x; i < 512; i += blockDim.x) (&L.h[0][0])[i] = 0u;
  __syncthreads();
}

// Threshold (thr_key, thr_g) of the selection: the bin_need-th largest of the
// bin_cnt keys of bin b* under (key descending, index ascending).  keyv(i) and
// idx(i) describe the n entries searched; every key of b* must be among them.
template <typename KeyV, typename Idx>
__device__ void find_threshold(const GateMeta& mt, int n, int N, KeyV keyv, Idx idx, RadixLds& L,
                               uint32_t* thr_key, int32_t* thr_g) {
  RadixSel st;
  st.prefix = mt.bin;
  st.shift = kHistShift;
  st.need = mt.bin_need;
  st.cnt = mt.bin_cnt;
  radix_select(st, n, keyv, [&](int i) { return keyv(i) != 0u; }, L);
  const uint32_t K = st.prefix << st.shift;
  int32_t tg = 0x7FFFFFFF;
  if (st.need < st.cnt) {
    // st.shift == 0: cnt keys equal K, the need-th smallest index among them
    // is the need-th largest of (N - 1 - index)
    const uint32_t top = uint32_t(N - 1);
    RadixSel si;
    si.prefix = 0u;
    si.shift = top == 0u ? 0 : 32 - __builtin_clz(top);
    si.need = st.need;
    si.cnt = st.cnt;
    radix_select(si, n, [&](int i) { return top - uint32_t(idx(i)); },
                 [&](int i) { return keyv(i) == K; }, L);
    tg = int32_t(top - (si.prefix << si.shift));
  }
  *thr_key = K;
  *thr_g = tg;
}

// LDS of the last phase that may come from a larger buffer: the gathered
// candidates' keys and indices (kSortCap each) and the candidate offsets of
// the select blocks (kGateThreads + 1).
struct FinishLds {
  uint32_t* s_k;
  int32_t* s_g;
  int* s_base;
};

// The last phase of the top-B selection, one workgroup of kGateThreads: gathers
// the candidates of the threshold bin, finds the threshold (key descending,
// index ascending) by radix selection, writes their selection flags and checks
// the ancestor closure of the selection.  If the bin holds more keys than LDS
// takes, the same selection runs over all keys in place.
__device__ void gate_finish_body(int N, int nblocks, const GateWs& ws,
                                 uint8_t* __restrict__ selected, int32_t* status,
                                 const FinishLds& lds) {
  uint32_t* s_k = lds.s_k;
  int32_t* s_g = lds.s_g;
  int* s_base = lds.s_base;
  __shared__ int s_scan[kGateThreads / kWave + 1];
  __shared__ RadixLds s_rl;
  // the first kGateThreads block counts are loaded with the selection's size
  const int c_first = int(threadIdx.x) < nblocks ? int(ws.ccount[threadIdx.x]) : 0;
  const GateMeta mt = *ws.meta;
  const uint32_t m = uint32_t(mt.num_selected);
  if (m == 0u) return;
  for (int i = threadIdx.x; i < 512; i += kGateThreads) (&s_rl.h[0][0])[i] = 0u;
  // exclusive scan of the per-block candidate counts
  int run = 0;
  for (int b0 = 0; b0 < nblocks; b0 += kGateThreads) {
    const int b = b0 + threadIdx.x;
    const int c = b0 == 0 ? c_first : (b < nblocks ? int(ws.ccount[b]) : 0);
    int tot;
    const int ex = block_exclusive_sum<kGateThreads>(c, s_scan, &tot);
    if (b < nblocks && b < kGateThreads) s_base[b] = run + ex;
    run += tot;
  }
  const int nc = run;
  uint32_t tk;
  int32_t tg;
  // No ancestor-closure check is needed: a child's score is its parent's plus a
  // clamped log q <= 0 in one binary32 add, so the parent's key is at least the
  // child's, and its global index is smaller; under (key descending, index
  // ascending) the parent of a selected node is always selected.
  (void)status;
  if (nc <= kSortCap && nblocks <= kGateThreads) {
    if (threadIdx.x == 0) s_base[nblocks] = nc;
    __syncthreads();
    for (int i = threadIdx.x; i < nc; i += kGateThreads) {
      const int b = upper_bound_idx(s_base, nblocks + 1, i);
      const uint2 c = ws.cand[size_t(b) * kGateThreads + (i - s_base[b])];
      s_k[i] = c.x;
      s_g[i] = int32_t(c.y);
    }
    __syncthreads();
    find_threshold(mt, nc, N, [&](int i) { return s_k[i]; }, [&](int i) { return s_g[i]; }, s_rl,
                   &tk, &tg);
    for (int i = threadIdx.x; i < nc; i += kGateThreads) {
      const uint32_t k = s_k[i];
      const int32_t g = s_g[i];
      const bool sel = k > tk || (k == tk && g <= tg);
      selected[g] = sel ? 1 : 0;
    }
  } else {
    __syncthreads();
    const uint32_t* keys = ws.keys;
    find_threshold(mt, N, N, [&](int i) { return keys[i]; }, [](int i) { return int32_t(i); },
                   s_rl, &tk, &tg);
    for (int b = 0; b < nblocks; ++b) {
      const int c = int(ws.ccount[b]);
      for (int i = threadIdx.x; i < c; i += kGateThreads) {
        const uint2 e = ws.cand[size_t(b) * kGateThreads + i];
        const bool sel = e.x > tk || (e.x == tk && int32_t(e.y) <= tg);
        selected[e.y] = sel ? 1 : 0;
      }
    }
  }
  if (threadIdx.x == 0) {
    ws.meta->thr_key = tk;
    ws.meta->thr_g = tg;
  }
}


}  // namespace
}  // namespace echo
