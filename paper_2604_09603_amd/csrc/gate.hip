// Gate: path scores (eq. 5) and the global top-B selection under the batch
// verification cap (eq. 4).  Three launches:
//
//   gate_init      zero the histogram and the counters in the workspace
//   gate_score     one thread per candidate: root->leaf binary32 fold of the
//                  path score, 32-bit orderable key, 2048-bin histogram of the
//                  key's top 11 bits (LDS, then one global atomic per bin).
//                  The last block to finish finds the B-th largest key (radix
//                  refinement, ties resolved by candidate index in order).
//   gate_finalize  one thread per candidate: selected = key above the
//                  threshold; ancestor-closure check; optional path_score.
#include "echo_device.h"
#include "echo_internal.h"

namespace echo {
namespace {

constexpr int kScoreThreads = 256;
constexpr int kHistBins = 2048;  // top 11 bits of the key
constexpr int kHistShift = 21;
constexpr int kGatherCap = 4096;  // keys the finishing block can hold in LDS

struct GateMeta {
  uint32_t blocks_done;
  uint32_t finite;     // number of selectable candidates
  uint32_t thr_key;    // selected iff key > thr_key || (key == thr_key && g <= thr_g)
  int32_t thr_g;
  int32_t num_selected;
  int32_t bad_csr;
};

struct GateWs {
  uint32_t* hist;
  GateMeta* meta;
  uint32_t* keys;
  int32_t* pglob;  // clamped parent, global index (-1: child of the root)
};

__host__ __device__ inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

__host__ __device__ inline GateWs gate_ws_layout(void* base, int32_t N) {
  char* p = static_cast<char*>(base);
  GateWs w;
  w.hist = reinterpret_cast<uint32_t*>(p);
  p += align_up(kHistBins * sizeof(uint32_t), 256);
  w.meta = reinterpret_cast<GateMeta*>(p);
  p += 256;
  w.keys = reinterpret_cast<uint32_t*>(p);
  p += align_up(size_t(N) * 4, 256);
  w.pglob = reinterpret_cast<int32_t*>(p);
  return w;
}

size_t gate_ws_bytes(int32_t N) {
  return align_up(kHistBins * 4, 256) + 256 + 2 * align_up(size_t(N) * 4, 256);
}

__global__ void gate_init_kernel(uint32_t* hist, GateMeta* meta) {
  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) hist[i] = 0u;
  if (threadIdx.x == 0) {
    meta->blocks_done = 0u;
    meta->finite = 0u;
    meta->thr_key = 0xFFFFFFFFu;
    meta->thr_g = -1;
    meta->num_selected = 0;
    meta->bad_csr = 0;
  }
}

// Validate the candidate CSR held in LDS; returns true if well formed.
__device__ bool csr_ok(const int32_t* s_offs, int R, int N, int* s_flag) {
  if (threadIdx.x == 0) *s_flag = (s_offs[0] != 0 || s_offs[R] != N) ? 1 : 0;
  __syncthreads();
  for (int r = threadIdx.x; r < R; r += blockDim.x)
    if (s_offs[r + 1] < s_offs[r]) *s_flag = 1;
  __syncthreads();
  bool ok = (*s_flag == 0);
  __syncthreads();
  return ok;
}

// ---- finishing block: k-th largest key ---------------------------------
// Radix refinement over keys matching `prefix` in the bits above `shift`.
// Keys come from global memory (all N) or from the LDS gather list.
struct Refine {
  uint32_t prefix;  // known high bits of the threshold key (value >> shift)
  int shift;        // number of still unknown low bits
  uint32_t cnt;     // keys matching the known prefix
  uint32_t need;    // how many of those are selected (1..cnt)
};

// One 8-bit (or shorter) digit step.  `get(i)` returns the i-th key, n keys.
template <typename Get>
__device__ void refine_step(Refine& st, int n, Get get, uint32_t* s_h256, int* s_scan) {
  const int bits = st.shift >= 8 ? 8 : st.shift;
  const int nsh = st.shift - bits;
  const uint32_t nb = 1u << bits;
  for (int i = threadIdx.x; i < 256; i += blockDim.x) s_h256[i] = 0u;
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    uint32_t k = get(i);
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

// Smallest index position among keys == key_t (in ascending order of i) such
// that `need` of them are at or before it; returns the global candidate index.
template <typename Get, typename Idx>
__device__ int32_t nth_equal(uint32_t key_t, uint32_t need, int n, Get get, Idx idx, int* s_scan) {
  __shared__ int s_found;
  if (threadIdx.x == 0) s_found = -1;
  __syncthreads();
  uint32_t run = 0;
  for (int base = 0; base < n; base += blockDim.x) {
    int i = base + threadIdx.x;
    int f = (i < n && get(i) == key_t) ? 1 : 0;
    int tot;
    int ex = block_exclusive_sum<kScoreThreads>(f, s_scan, &tot);
    if (f && run + uint32_t(ex) + 1u == need) s_found = idx(i);
    run += uint32_t(tot);
    if (run >= need) break;  // uniform: run is the same in every thread
  }
  __syncthreads();
  return s_found;
}

__device__ void select_threshold(const GateWs& ws, int N, int budget, int32_t* num_selected) {
  __shared__ uint32_t s_h256[256];
  __shared__ int s_scan[kScoreThreads / kWave + 1];
  __shared__ uint32_t s_gk[kGatherCap];
  __shared__ int32_t s_gi[kGatherCap];
  __shared__ uint32_t s_bin[3];

  GateMeta* meta = ws.meta;
  const uint32_t finite = meta->finite;
  const uint32_t m = min(uint32_t(budget), finite);
  if (m == 0u) {
    if (threadIdx.x == 0) {
      meta->thr_key = 0xFFFFFFFFu;
      meta->thr_g = -1;
      meta->num_selected = 0;
      *num_selected = 0;
    }
    return;
  }
  // 1. histogram bin holding the m-th largest key: suffix sums over 2048 bins.
  {
    constexpr int per = kHistBins / kScoreThreads;  // 8 bins per thread
    const int t = threadIdx.x;
    // thread t owns bins [2048 - per*(t+1), 2048 - per*t): high bins first
    uint32_t local = 0;
    for (int j = 0; j < per; ++j) local += ws.hist[kHistBins - per * t - 1 - j];
    int tot;
    int ex = block_exclusive_sum<kScoreThreads>(int(local), s_scan, &tot);
    uint32_t above = uint32_t(ex);
    if (above < m && above + local >= m) {
      for (int j = 0; j < per; ++j) {
        int b = kHistBins - per * t - 1 - j;
        uint32_t c = ws.hist[b];
        if (above + c >= m) {
          s_bin[0] = uint32_t(b);
          s_bin[1] = c;
          s_bin[2] = m - above;
          break;
        }
        above += c;
      }
    }
    __syncthreads();
  }
  Refine st;
  st.prefix = s_bin[0];
  st.shift = kHistShift;
  st.cnt = s_bin[1];
  st.need = s_bin[2];
  __syncthreads();

  const uint32_t* keys = ws.keys;
  auto gget = [&](int i) { return keys[i]; };
  // 2. refine over global memory while the candidate bin is too big to gather.
  while (st.shift > 0 && st.cnt > uint32_t(kGatherCap)) refine_step(st, N, gget, s_h256, s_scan);

  int32_t thr_g;
  if (st.cnt <= uint32_t(kGatherCap)) {
    // 3. ordered gather of the bin (ascending candidate index) into LDS.
    const int sh = st.shift;
    const uint32_t pre = st.prefix;
    int filled = 0;
    for (int base = 0; base < N; base += kScoreThreads) {
      int g = base + threadIdx.x;
      uint32_t k = g < N ? keys[g] : 0u;
      int f = (k != 0u && (k >> sh) == pre) ? 1 : 0;
      int tot;
      int ex = block_exclusive_sum<kScoreThreads>(f, s_scan, &tot);
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
    if (st.need == st.cnt) {
      thr_g = 0x7FFFFFFF;
    } else {
      thr_g = nth_equal(st.prefix, st.need, filled, lget, [&](int i) { return s_gi[i]; }, s_scan);
    }
  } else {
    // every remaining key equals the threshold: resolve ties by index in global order
    if (st.need == st.cnt) {
      thr_g = 0x7FFFFFFF;
    } else {
      thr_g = nth_equal(st.prefix, st.need, N, gget, [](int i) { return int32_t(i); }, s_scan);
    }
  }
  if (threadIdx.x == 0) {
    meta->thr_key = st.prefix;
    meta->thr_g = thr_g;
    meta->num_selected = int32_t(m);
    *num_selected = int32_t(m);
  }
}

__global__ __launch_bounds__(kScoreThreads) void gate_score_kernel(
    const int32_t* __restrict__ cand_offsets, const int32_t* __restrict__ parent,
    const float* __restrict__ logq, int R, int N, int budget, GateWs ws,
    float* __restrict__ path_score_out, int32_t* __restrict__ num_selected, int32_t* status) {
  extern __shared__ int32_t s_offs[];  // R + 1 entries
  __shared__ uint32_t s_hist[kHistBins];
  __shared__ int s_flag;
  __shared__ uint32_t s_finite;
  __shared__ bool s_last;

  for (int i = threadIdx.x; i <= R; i += blockDim.x) s_offs[i] = cand_offsets[i];
  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) s_hist[i] = 0u;
  if (threadIdx.x == 0) s_finite = 0u;
  __syncthreads();
  const bool ok = csr_ok(s_offs, R, N, &s_flag);

  const int g = blockIdx.x * kScoreThreads + threadIdx.x;
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
      if (key != 0u) {
        atomicAdd(&s_hist[key >> kHistShift], 1u);
        atomicAdd(&s_finite, 1u);
      }
    }
    ws.keys[g] = key;
    ws.pglob[g] = pg;
    if (path_score_out != nullptr) path_score_out[g] = s;
  }
  wave_status_or(status, bits);
  __syncthreads();
  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) {
    uint32_t c = s_hist[i];
    if (c) atomicAdd(&ws.hist[i], c);
  }
  if (threadIdx.x == 0) {
    if (s_finite) atomicAdd(&ws.meta->finite, s_finite);
    if (!ok && blockIdx.x == 0) {
      ws.meta->bad_csr = 1;
      status_or(status, ECHO_DATA_BAD_OFFSETS);
    }
  }
  // last block to finish selects the threshold
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t ticket = atomicAdd(&ws.meta->blocks_done, 1u);
    s_last = (ticket == gridDim.x - 1);
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  select_threshold(ws, N, budget, num_selected);
}

__global__ __launch_bounds__(256) void gate_finalize_kernel(int N, GateWs ws,
                                                            uint8_t* __restrict__ selected,
                                                            int32_t* status) {
  const uint32_t tk = ws.meta->thr_key;
  const int32_t tg = ws.meta->thr_g;
  const int g = blockIdx.x * 256 + threadIdx.x;
  int bits = 0;
  if (g < N) {
    const uint32_t k = ws.keys[g];
    const bool sel = k != 0u && (k > tk || (k == tk && g <= tg));
    selected[g] = sel ? 1 : 0;
    if (sel) {
      const int32_t p = ws.pglob[g];
      if (p >= 0) {
        const uint32_t kp = ws.keys[p];
        const bool psel = kp != 0u && (kp > tk || (kp == tk && p <= tg));
        if (!psel) bits |= ECHO_DATA_NOT_CLOSED;
      }
    }
  }
  wave_status_or(status, bits);
}

}  // namespace

int32_t launch_gate(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                    int32_t R, int32_t N, int32_t budget, float* path_score, uint8_t* selected,
                    int32_t* num_selected, void* workspace, int32_t* status, hipStream_t stream) {
  GateWs ws = gate_ws_layout(workspace, N);
  hipLaunchKernelGGL(gate_init_kernel, dim3(1), dim3(256), 0, stream, ws.hist, ws.meta);
  const int blocks = N > 0 ? (N + kScoreThreads - 1) / kScoreThreads : 1;
  const size_t lds = size_t(R + 1) * sizeof(int32_t);
  hipLaunchKernelGGL(gate_score_kernel, dim3(blocks), dim3(kScoreThreads), lds, stream,
                     cand_offsets, parent, logq, R, N, budget, ws, path_score, num_selected,
                     status);
  if (N > 0)
    hipLaunchKernelGGL(gate_finalize_kernel, dim3((N + 255) / 256), dim3(256), 0, stream, N, ws,
                       selected, status);
  return hipGetLastError() == hipSuccess ? ECHO_OK : ECHO_ERR_HIP;
}

size_t gate_workspace_bytes(int32_t R, int32_t N, int32_t budget) {
  (void)R;
  (void)budget;
  return gate_ws_bytes(N);
}

}  // namespace echo
