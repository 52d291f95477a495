// Gate: path scores (eq. 5) and the global top-B selection under the batch
// verification cap (eq. 4).  Four launches, none of which contends on a
// global atomic (on a multi-XCD part those serialise far from the CUs):
//
//   gate_score   one thread per candidate: root->leaf binary32 fold of the path
//                score, 32-bit orderable key, and each block's 2048-bin histogram
//                of the key's top 11 bits, written to its own slice.
//   gate_bin     one block: sums the block histograms and finds the bin b* that
//                holds the m-th largest key, m = min(B, #finite), and how many
//                keys of b* are selected.
//   gate_select  one thread per candidate: keys above b* are selected, keys below
//                are not; keys inside b* go to the block's own candidate slice.
//   gate_finish  one block: gathers the candidates, sorts them in LDS by (key
//                descending, index ascending), selects the head and checks the
//                ancestor closure of the selection.  If b* holds more keys than
//                the sort takes, it falls back to radix refinement over all keys.
#include "echo_device.h"
#include "echo_internal.h"

namespace echo {
namespace {

constexpr int kGateThreads = 1024;
constexpr int kHistBins = 2048;   // top 11 bits of the key
constexpr int kHistShift = 21;
constexpr int kSortCap = 4096;    // candidates gate_finish sorts in LDS
constexpr int kGatherCap = 4096;  // keys the fallback holds in LDS

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
  uint2* cand;       // [nblocks * 1024] (key, index) candidates, block slices
};

__host__ __device__ inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

__host__ __device__ inline int gate_blocks(int32_t N) {
  return N > 0 ? (N + kGateThreads - 1) / kGateThreads : 1;
}

__host__ __device__ inline GateWs gate_ws_layout(void* base, int32_t N) {
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
  w.cand = reinterpret_cast<uint2*>(p);
  return w;
}

size_t gate_ws_bytes(int32_t N) {
  const size_t nb = size_t(gate_blocks(N));
  return 256 + 2 * align_up(size_t(N) * 4, 256) + align_up(nb * kHistBins * 4, 256) +
         align_up(nb * 4, 256) + align_up(nb * kGateThreads * 8, 256);
}

// ---------------------------------------------------------------- score ----
__global__ __launch_bounds__(kGateThreads) void gate_score_kernel(
    const int32_t* __restrict__ cand_offsets, const int32_t* __restrict__ parent,
    const float* __restrict__ logq, int R, int N, GateWs ws, float* __restrict__ path_score_out,
    int32_t* status) {
  extern __shared__ int32_t s_offs[];  // R + 1 entries
  __shared__ uint32_t s_hist[kHistBins];
  __shared__ int s_flag;

  for (int i = threadIdx.x; i <= R; i += kGateThreads) s_offs[i] = cand_offsets[i];
  for (int i = threadIdx.x; i < kHistBins; i += kGateThreads) s_hist[i] = 0u;
  if (threadIdx.x == 0) s_flag = 0;
  __syncthreads();
  // the candidate CSR must be well formed before anything is read through it
  if (threadIdx.x == 0 && (s_offs[0] != 0 || s_offs[R] != N)) s_flag = 1;
  for (int r = threadIdx.x; r < R; r += kGateThreads)
    if (s_offs[r + 1] < s_offs[r]) s_flag = 1;
  __syncthreads();
  const bool ok = s_flag == 0;

  const int g = blockIdx.x * kGateThreads + threadIdx.x;
  int bits = 0;
  if (g < N) {
    uint32_t key = 0u;
    int32_t pg = -1;
    float s = -__builtin_inff();
    if (ok) {
      const int r = upper_bound_idx(s_offs, R + 1, g);
      const int lo = s_offs[r];
      const int n = g - lo;
      int p = parent[g];
      if (p < -1 || p >= n) { bits |= ECHO_DATA_BAD_PARENT; p = -1; }
      pg = p < 0 ? -1 : lo + p;
      float own = logq[g];
      if (own != own) { bits |= ECHO_DATA_NAN_LOGQ; own = -__builtin_inff(); }
      else if (own > 0.0f) { bits |= ECHO_DATA_POS_LOGQ; own = 0.0f; }
      // collect log q along the path, leaf first: vals[0] = own, vals[i] = i-th ancestor
      float vals[ECHO_MAX_DEPTH + 1];
      vals[0] = own;
      int depth = 1;
#pragma unroll
      for (int i = 1; i <= ECHO_MAX_DEPTH; ++i) {
        vals[i] = 0.0f;
        if (p >= 0) {
          const int a = lo + p;
          float v = logq[a];
          if (v != v) v = -__builtin_inff();
          else if (v > 0.0f) v = 0.0f;
          int pp = parent[a];
          if (pp < -1 || pp >= p) pp = -1;
          vals[i] = v;
          depth = i + 1;
          p = pp;
        }
      }
      if (depth > ECHO_MAX_DEPTH) {
        bits |= ECHO_DATA_TOO_DEEP;
      } else {
        // root -> leaf: S = ((0 + lq[top]) + ...) + lq[own], one binary32 add per level
        s = 0.0f;
#pragma unroll
        for (int i = ECHO_MAX_DEPTH; i >= 0; --i)
          if (i < depth) s = s + vals[i];
      }
      key = score_key(s);
      if (key != 0u) atomicAdd(&s_hist[key >> kHistShift], 1u);
    }
    ws.keys[g] = key;
    ws.pglob[g] = pg;
    if (path_score_out != nullptr) path_score_out[g] = s;
  }
  if (!ok && blockIdx.x == 0 && threadIdx.x == 0) bits |= ECHO_DATA_BAD_OFFSETS;
  wave_status_or(status, bits);
  __syncthreads();
  uint32_t* mine = ws.bhist + size_t(blockIdx.x) * kHistBins;
  for (int i = threadIdx.x; i < kHistBins; i += kGateThreads) mine[i] = s_hist[i];
}

// ------------------------------------------------------------------ bin ----
__global__ __launch_bounds__(kGateThreads) void gate_bin_kernel(int nblocks, int budget, GateWs ws,
                                                               int32_t* __restrict__ num_selected) {
  __shared__ int s_scan[kGateThreads / kWave + 1];
  __shared__ uint32_t s_part[2][kHistBins];
  constexpr int per = kHistBins / kGateThreads;  // bins per thread, high bins first
  const int t = threadIdx.x;
  {
    // thread (half h, quad q) sums bins 4q..4q+3 over blocks h, h+2, ...; many loads in flight
    const int h = t / (kGateThreads / 2);
    const int q4 = (t % (kGateThreads / 2)) * 4;
    uint4 acc = make_uint4(0, 0, 0, 0);
#pragma unroll 8
    for (int b = h; b < nblocks; b += 2) {
      const uint4 v = *reinterpret_cast<const uint4*>(ws.bhist + size_t(b) * kHistBins + q4);
      acc.x += v.x;
      acc.y += v.y;
      acc.z += v.z;
      acc.w += v.w;
    }
    *reinterpret_cast<uint4*>(&s_part[h][q4]) = acc;
  }
  __syncthreads();
  uint32_t cnt[per];
#pragma unroll
  for (int j = 0; j < per; ++j) {
    const int b = kHistBins - per * t - 1 - j;
    cnt[j] = s_part[0][b] + s_part[1][b];
  }
  uint32_t local = 0;
#pragma unroll
  for (int j = 0; j < per; ++j) local += cnt[j];
  int finite;
  const uint32_t above0 = uint32_t(block_exclusive_sum<kGateThreads>(int(local), s_scan, &finite));
  const uint32_t m = min(uint32_t(budget), uint32_t(finite));
  if (t == 0) {
    ws.meta->num_selected = int32_t(m);
    ws.meta->bin = 0u;
    ws.meta->bin_need = 0u;
    ws.meta->bin_cnt = 0u;
    ws.meta->thr_key = 0xFFFFFFFFu;
    ws.meta->thr_g = -1;
    *num_selected = int32_t(m);
  }
  __syncthreads();
  if (m == 0u) return;
  uint32_t above = above0;
  if (above < m && above + local >= m) {
#pragma unroll
    for (int j = 0; j < per; ++j) {
      const int b = kHistBins - per * t - 1 - j;
      if (above < m && above + cnt[j] >= m) {
        ws.meta->bin = uint32_t(b);
        ws.meta->bin_cnt = cnt[j];
        ws.meta->bin_need = m - above;
      }
      above += cnt[j];
    }
  }
}

// --------------------------------------------------------------- select ----
__global__ __launch_bounds__(kGateThreads) void gate_select_kernel(int N, GateWs ws,
                                                                   uint8_t* __restrict__ selected,
                                                                   int32_t* status) {
  __shared__ uint32_t s_cnt;
  const uint32_t m = uint32_t(ws.meta->num_selected);
  const uint32_t bin = ws.meta->bin;
  const int g = blockIdx.x * kGateThreads + threadIdx.x;
  int bits = 0;
  if (threadIdx.x == 0) s_cnt = 0u;
  __syncthreads();
  if (g < N) {
    const uint32_t k = ws.keys[g];
    const uint32_t kb = k >> kHistShift;
    if (m == 0u || k == 0u || kb < bin) {
      selected[g] = 0;
    } else if (kb > bin) {
      selected[g] = 1;
      const int32_t p = ws.pglob[g];
      // a parent's key is never below its child's, so it lies in a higher bin too
      if (p >= 0 && !(ws.keys[p] >> kHistShift > bin)) bits |= ECHO_DATA_NOT_CLOSED;
    } else {
      const uint32_t slot = atomicAdd(&s_cnt, 1u);  // LDS; the order is fixed by the sort
      ws.cand[size_t(blockIdx.x) * kGateThreads + slot] = make_uint2(k, uint32_t(g));
    }
  }
  wave_status_or(status, bits);
  __syncthreads();
  if (threadIdx.x == 0) ws.ccount[blockIdx.x] = s_cnt;
}

// --------------------------------------------------------------- finish ----
// Fallback (the threshold bin holds more keys than the LDS sort takes): radix
// refinement of the threshold key over all keys, ties by index in order.
struct Refine {
  uint32_t prefix;  // known high bits of the threshold key (value >> shift)
  int shift;        // number of still unknown low bits
  uint32_t cnt;     // keys matching the known prefix
  uint32_t need;    // how many of those are selected (1..cnt)
};

template <typename Get>
__device__ void refine_step(Refine& st, int n, Get get, uint32_t* s_h256, int* s_scan) {
  const int bits = st.shift >= 8 ? 8 : st.shift;
  const int nsh = st.shift - bits;
  const uint32_t nb = 1u << bits;
  for (int i = threadIdx.x; i < 256; i += blockDim.x) s_h256[i] = 0u;
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const uint32_t k = get(i);
    if (k != 0u && (k >> st.shift) == st.prefix) atomicAdd(&s_h256[(k >> nsh) & (nb - 1)], 1u);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t above = 0;
    int d = int(nb) - 1;
    for (; d > 0; --d) {
      if (above + s_h256[d] >= st.need) break;
      above += s_h256[d];
    }
    s_scan[0] = d;
    s_scan[1] = int(above);
  }
  __syncthreads();
  const uint32_t d = uint32_t(s_scan[0]);
  st.need -= uint32_t(s_scan[1]);
  st.cnt = s_h256[d];
  st.prefix = (st.prefix << bits) | d;
  st.shift = nsh;
  __syncthreads();
}

// Index of the `need`-th key equal to key_t in ascending order of i.
template <typename Get, typename Idx>
__device__ int32_t nth_equal(uint32_t key_t, uint32_t need, int n, Get get, Idx idx, int* s_scan,
                             int* s_found) {
  if (threadIdx.x == 0) *s_found = -1;
  __syncthreads();
  uint32_t run = 0;
  for (int base = 0; base < n; base += blockDim.x) {
    const int i = base + threadIdx.x;
    const int f = (i < n && get(i) == key_t) ? 1 : 0;
    int tot;
    const int ex = block_exclusive_sum<kGateThreads>(f, s_scan, &tot);
    if (f && run + uint32_t(ex) + 1u == need) *s_found = idx(i);
    run += uint32_t(tot);
    if (run >= need) break;  // uniform: run is the same in every thread
  }
  __syncthreads();
  return *s_found;
}

__device__ void refine_threshold(const GateWs& ws, int N, uint32_t* thr_key, int32_t* thr_g,
                                 uint32_t* s_gk, int32_t* s_gi) {
  __shared__ uint32_t s_h256[256];
  __shared__ int s_scan[kGateThreads / kWave + 1];
  __shared__ int s_found;
  Refine st;
  st.prefix = ws.meta->bin;
  st.shift = kHistShift;
  st.cnt = ws.meta->bin_cnt;
  st.need = ws.meta->bin_need;
  const uint32_t* keys = ws.keys;
  auto gget = [&](int i) { return keys[i]; };
  while (st.shift > 0 && st.cnt > uint32_t(kGatherCap)) refine_step(st, N, gget, s_h256, s_scan);
  int32_t tg;
  if (st.cnt <= uint32_t(kGatherCap)) {
    // ordered gather of the remaining keys (ascending candidate index) into LDS
    const int sh = st.shift;
    const uint32_t pre = st.prefix;
    int filled = 0;
    for (int base = 0; base < N; base += kGateThreads) {
      const int g = base + threadIdx.x;
      const uint32_t k = g < N ? keys[g] : 0u;
      const int f = (k != 0u && (k >> sh) == pre) ? 1 : 0;
      int tot;
      const int ex = block_exclusive_sum<kGateThreads>(f, s_scan, &tot);
      if (f) {
        s_gk[filled + ex] = k;
        s_gi[filled + ex] = g;
      }
      filled += tot;
      if (uint32_t(filled) >= st.cnt) break;
    }
    __syncthreads();
    auto lget = [&](int i) { return s_gk[i]; };
    while (st.shift > 0) refine_step(st, filled, lget, s_h256, s_scan);
    tg = st.need == st.cnt ? 0x7FFFFFFF
                           : nth_equal(st.prefix, st.need, filled, lget,
                                       [&](int i) { return s_gi[i]; }, s_scan, &s_found);
  } else {
    tg = st.need == st.cnt ? 0x7FFFFFFF
                           : nth_equal(st.prefix, st.need, N, gget,
                                       [](int i) { return int32_t(i); }, s_scan, &s_found);
  }
  *thr_key = st.prefix;
  *thr_g = tg;
}

__device__ __forceinline__ uint64_t sort_word(uint32_t key, int32_t g) {
  // larger key first, then smaller index first
  return (uint64_t(key) << 32) | uint64_t(0xFFFFFFFFu - uint32_t(g));
}

__global__ __launch_bounds__(kGateThreads) void gate_finish_kernel(int N, int nblocks, GateWs ws,
                                                                   uint8_t* __restrict__ selected,
                                                                   int32_t* status) {
  __shared__ uint64_t s_sort[kSortCap];  // also the fallback's gather buffers
  __shared__ int s_base[kGateThreads + 1];
  __shared__ int s_scan[kGateThreads / kWave + 1];
  __shared__ uint32_t s_tk;
  __shared__ int32_t s_tg;
  const uint32_t m = uint32_t(ws.meta->num_selected);
  if (m == 0u) return;
  const uint32_t need = ws.meta->bin_need;
  // exclusive scan of the per-block candidate counts
  int run = 0;
  for (int b0 = 0; b0 < nblocks; b0 += kGateThreads) {
    const int b = b0 + threadIdx.x;
    const int c = b < nblocks ? int(ws.ccount[b]) : 0;
    int tot;
    const int ex = block_exclusive_sum<kGateThreads>(c, s_scan, &tot);
    if (b < nblocks && b < kGateThreads) s_base[b] = run + ex;
    run += tot;
  }
  const int nc = run;
  int bits = 0;
  if (nc <= kSortCap && nblocks <= kGateThreads) {
    if (threadIdx.x == 0) s_base[nblocks] = nc;
    __syncthreads();
    uint32_t n2 = 1;
    while (n2 < uint32_t(nc)) n2 <<= 1;
    for (uint32_t i = threadIdx.x; i < n2; i += kGateThreads) {
      uint64_t w = 0ull;
      if (i < uint32_t(nc)) {
        const int b = upper_bound_idx(s_base, nblocks + 1, int(i));
        const uint2 c = ws.cand[size_t(b) * kGateThreads + (int(i) - s_base[b])];
        w = sort_word(c.x, int32_t(c.y));
      }
      s_sort[i] = w;
    }
    __syncthreads();
    // bitonic sort, descending
    for (uint32_t size = 2; size <= n2; size <<= 1) {
      for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
        for (uint32_t i = threadIdx.x; i < n2; i += kGateThreads) {
          const uint32_t j = i ^ stride;
          if (j > i) {
            const uint64_t a = s_sort[i], b = s_sort[j];
            const bool desc = (i & size) == 0;
            if (desc ? (a < b) : (a > b)) {
              s_sort[i] = b;
              s_sort[j] = a;
            }
          }
        }
        __syncthreads();
      }
    }
    const uint64_t thr = s_sort[need - 1];
    if (threadIdx.x == 0) {
      ws.meta->thr_key = uint32_t(thr >> 32);
      ws.meta->thr_g = int32_t(0xFFFFFFFFu - uint32_t(thr));
    }
    for (uint32_t i = threadIdx.x; i < uint32_t(nc); i += kGateThreads) {
      const uint64_t w = s_sort[i];
      const int32_t gi = int32_t(0xFFFFFFFFu - uint32_t(w));
      const bool sel = i < need;
      selected[gi] = sel ? 1 : 0;
      if (sel) {
        const int32_t p = ws.pglob[gi];
        if (p >= 0) {
          const uint32_t kp = ws.keys[p];
          if (kp == 0u || sort_word(kp, p) < thr) bits |= ECHO_DATA_NOT_CLOSED;
        }
      }
    }
  } else {
    uint32_t tk;
    int32_t tg;
    refine_threshold(ws, N, &tk, &tg, reinterpret_cast<uint32_t*>(s_sort),
                     reinterpret_cast<int32_t*>(s_sort) + kGatherCap);
    if (threadIdx.x == 0) {
      s_tk = tk;
      s_tg = tg;
      ws.meta->thr_key = tk;
      ws.meta->thr_g = tg;
    }
    __syncthreads();
    tk = s_tk;
    tg = s_tg;
    for (int b = 0; b < nblocks; ++b) {
      const int c = int(ws.ccount[b]);
      for (int i = threadIdx.x; i < c; i += kGateThreads) {
        const uint2 e = ws.cand[size_t(b) * kGateThreads + i];
        const bool sel = e.x > tk || (e.x == tk && int32_t(e.y) <= tg);
        selected[e.y] = sel ? 1 : 0;
        if (sel) {
          const int32_t p = ws.pglob[e.y];
          if (p >= 0) {
            const uint32_t kp = ws.keys[p];
            if (kp == 0u || !(kp > tk || (kp == tk && p <= tg))) bits |= ECHO_DATA_NOT_CLOSED;
          }
        }
      }
    }
  }
  wave_status_or(status, bits);
}

}  // namespace

int32_t launch_gate(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                    int32_t R, int32_t N, int32_t budget, float* path_score, uint8_t* selected,
                    int32_t* num_selected, void* workspace, int32_t* status, hipStream_t stream) {
  (void)hipGetLastError();  // clear errors left by unrelated runtime calls
  GateWs ws = gate_ws_layout(workspace, N);
  const int blocks = gate_blocks(N);
  const size_t lds = size_t(R + 1) * sizeof(int32_t);
  hipLaunchKernelGGL(gate_score_kernel, dim3(blocks), dim3(kGateThreads), lds, stream,
                     cand_offsets, parent, logq, R, N, ws, path_score, status);
  hipLaunchKernelGGL(gate_bin_kernel, dim3(1), dim3(kGateThreads), 0, stream, blocks, budget, ws,
                     num_selected);
  if (N > 0) {
    hipLaunchKernelGGL(gate_select_kernel, dim3(blocks), dim3(kGateThreads), 0, stream, N, ws,
                       selected, status);
    hipLaunchKernelGGL(gate_finish_kernel, dim3(1), dim3(kGateThreads), 0, stream, N, blocks, ws,
                       selected, status);
  }
  return hipGetLastError() == hipSuccess ? ECHO_OK : ECHO_ERR_HIP;
}

size_t gate_workspace_bytes(int32_t R, int32_t N, int32_t budget) {
  (void)R;
  (void)budget;
  return gate_ws_bytes(N);
}

}  // namespace echo
