// Gate: path scores (eq. 5) and the global top-B selection under the batch
// verification cap (eq. 4).  Three launches, none of which contends on a
// global atomic (on a multi-XCD part those serialise far from the CUs):
//
//   gate_score   one thread per candidate: root->leaf binary32 fold of the path
//                score, 32-bit orderable key, and each block's 2048-bin histogram
//                of the key's top 11 bits, written to its own slice.
//   gate_select  one thread per candidate.  Every block first finds the bin b*
//                that holds the m-th largest key, m = min(B, #finite): from the
//                score blocks' finite counts and highest occupied bins it sums
//                their histograms downwards from the top in chunks of 64 bins
//                (usually one chunk: the selection is a small top).  Keys above
//                b* are selected, keys below are not; keys inside b* go to the
//                block's own candidate slice.
//   gate_finish  one block: gathers the candidates into LDS, finds the
//                threshold (key descending, index ascending) among them by radix
//                selection, selects the head and checks the ancestor closure of
//                the selection.  If b* holds more keys than LDS takes, the same
//                selection runs over all keys in place.
//
// Sparse checkpoint gating (eq. 6, eq. 7; Alg. 1 phase 1) adds two launches in
// front of gate_select: gate_lmax_clear zeroes the per-(request, depth) maximum
// keys, gate_score then also folds each block's checkpoint-depth keys into
// them (LDS first, one global atomicMax per block, request and depth) instead
// of building histograms, and gate_trunc finds each request's first failed
// checkpoint, zeroes the keys at or below it and builds the histograms.
#include "echo_device.h"
#include "echo_internal.h"
#include "gate_device.h"

namespace echo {
namespace {

size_t gate_ws_bytes(int32_t N, int32_t R) {
  const size_t nb = size_t(gate_blocks(N));
  return 256 + 2 * align_up(size_t(N) * 4, 256) + align_up(nb * kHistBins * 4, 256) +
         align_up(nb * 4, 256) + align_up(nb * 8, 256) + align_up(nb * kGateThreads * 8, 256) +
         align_up(size_t(R) * kDepths * 4, 256) + align_up(size_t(N), 256);
}

// Per-block histogram outputs shared by gate_score and gate_trunc: the block's
// 2048 bins and (finite keys, highest occupied bin + 1).
__device__ void write_block_hist(const uint32_t* s_hist, uint2* s_red, GateWs& ws) {
  uint32_t* mine = ws.bhist + size_t(blockIdx.x) * kHistBins;
  uint32_t fin = 0u, top = 0u;
  for (int i = threadIdx.x; i < kHistBins; i += kGateThreads) {
    const uint32_t c = s_hist[i];
    mine[i] = c;
    fin += c;
    if (c != 0u) top = max(top, uint32_t(i + 1));
  }
  fin = wave_sum(fin);
  top = wave_max(top);
  if ((threadIdx.x & (kWave - 1)) == 0) s_red[threadIdx.x / kWave] = make_uint2(fin, top);
  __syncthreads();
  if (threadIdx.x == 0) {
    uint2 acc = make_uint2(0u, 0u);
    for (int w = 0; w < kGateThreads / kWave; ++w) {
      acc.x += s_red[w].x;
      acc.y = max(acc.y, s_red[w].y);
    }
    ws.bsum[blockIdx.x] = acc;
  }
}

// ---------------------------------------------------------------- score ----
__global__ __launch_bounds__(kGateThreads) void gate_score_kernel(
    const int32_t* __restrict__ cand_offsets, const int32_t* __restrict__ parent,
    const float* __restrict__ logq, int R, int N, GateWs ws, float* __restrict__ path_score_out,
    int32_t* status, SparseArgs sp) {
  extern __shared__ int32_t s_offs[];  // R + 1 entries
  __shared__ uint32_t s_hist[kHistBins];
  __shared__ uint32_t s_lmax[kTabReq * kDepths];  // sparse gating: requests r0 .. r0 + 63
  __shared__ int s_flag;
  __shared__ int s_r0;
  // parent and log q of the block's nodes and of the kWinBack nodes before them:
  // the ancestors of most nodes lie there, so the path walks stay in LDS
  __shared__ int32_t s_par[kWin];
  __shared__ float s_lq[kWin];
  const int g0 = blockIdx.x * kGateThreads;
  const int wstart = max(0, g0 - kWinBack);
  const int wlen = min(N, g0 + kGateThreads) - wstart;

  if (wlen > 0) {  // N = 0 still launches one block, with nothing to read
    // every load of the window issued before the first is stored (one memory
    // round trip); addresses are clamped into the window
    constexpr int kWinLoads = kWin / kGateThreads;
    static_assert(kWin % kGateThreads == 0, "window tiling");
    int32_t vp[kWinLoads];
    float vl[kWinLoads];
#pragma unroll
    for (int k = 0; k < kWinLoads; ++k) {
      const int a = wstart + min(int(threadIdx.x) + k * kGateThreads, wlen - 1);
      vp[k] = parent[a];
      vl[k] = logq[a];
    }
#pragma unroll
    for (int k = 0; k < kWinLoads; ++k) {
      const int i = int(threadIdx.x) + k * kGateThreads;
      if (i < wlen) {
        s_par[i] = vp[k];
        s_lq[i] = vl[k];
      }
    }
  }
  for (int i = threadIdx.x; i <= R; i += kGateThreads) s_offs[i] = cand_offsets[i];
  for (int i = threadIdx.x; i < kHistBins; i += kGateThreads) s_hist[i] = 0u;
  if (sp.enabled)
    for (int i = threadIdx.x; i < kTabReq * kDepths; i += kGateThreads) s_lmax[i] = 0u;
  if (threadIdx.x == 0) s_flag = 0;
  __syncthreads();
  // the candidate CSR must be well formed before anything is read through it
  if (threadIdx.x == 0 && (s_offs[0] != 0 || s_offs[R] != N)) s_flag = 1;
  for (int r = threadIdx.x; r < R; r += kGateThreads)
    if (s_offs[r + 1] < s_offs[r]) s_flag = 1;
  __syncthreads();
  const bool ok = s_flag == 0;
  if (sp.enabled && threadIdx.x == 0) s_r0 = ok && g0 < N ? upper_bound_idx(s_offs, R + 1, g0) : 0;
  if (sp.enabled) __syncthreads();

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
      auto par_at = [&](int a) { return a >= wstart ? s_par[a - wstart] : parent[a]; };
      auto lq_at = [&](int a) { return a >= wstart ? s_lq[a - wstart] : logq[a]; };
      int p = par_at(g);
      if (p < -1 || p >= n) { bits |= ECHO_DATA_BAD_PARENT; p = -1; }
      pg = p < 0 ? -1 : lo + p;
      float own = lq_at(g);
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
          float v = lq_at(a);
          if (v != v) v = -__builtin_inff();
          else if (v > 0.0f) v = 0.0f;
          int pp = par_at(a);
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
      if (!sp.enabled) {
        if (key != 0u) atomicAdd(&s_hist[key >> kHistShift], 1u);
      } else if (key != 0u && ((sp.mask >> depth) & 1u)) {
        // depth <= ECHO_MAX_DEPTH here: deeper nodes have key 0
        const int rl = r - s_r0;
        if (rl < kTabReq) atomicMax(&s_lmax[rl * kDepths + depth], key);
        else atomicMax(&ws.lmax[size_t(r) * kDepths + depth], key);
      }
      if (sp.enabled) ws.depth[g] = uint8_t(min(depth, ECHO_MAX_DEPTH + 1));
    }
    ws.keys[g] = key;
    ws.pglob[g] = pg;
    if (path_score_out != nullptr) path_score_out[g] = s;
  }
  if (!ok && blockIdx.x == 0 && threadIdx.x == 0) bits |= ECHO_DATA_BAD_OFFSETS;
  wave_status_or(status, bits);
  __syncthreads();
  __shared__ uint2 s_red[kGateThreads / kWave];
  if (!sp.enabled) {
    write_block_hist(s_hist, s_red, ws);
  } else {
    // one global atomic per (request, checkpoint depth) present in the block
    for (int i = threadIdx.x; i < kTabReq * kDepths; i += kGateThreads) {
      const uint32_t v = s_lmax[i];
      const int r = s_r0 + i / kDepths;
      if (v != 0u && r < R) atomicMax(&ws.lmax[size_t(r) * kDepths + i % kDepths], v);
    }
  }
}

// --------------------------------------------------------- sparse gating ----
__global__ __launch_bounds__(kGateThreads) void gate_lmax_clear_kernel(int n, uint32_t* lmax) {
  const int i = blockIdx.x * kGateThreads + threadIdx.x;
  if (i < n) lmax[i] = 0u;
}

// First failed checkpoint of request r: the smallest checkpoint depth d whose
// maximum key does not exceed the key of ln tau_d (eq. 7; -0 == +0 and -inf
// has key 0 on both sides, so the key test is the float test S > ln tau).
__device__ __forceinline__ int first_failed(const SparseArgs& sp, const uint32_t* lmax_r) {
  uint32_t v[kDepths];  // every checkpoint's maximum is loaded before any is tested
#pragma unroll
  for (int d = 1; d <= ECHO_MAX_DEPTH; ++d) v[d] = ((sp.mask >> d) & 1u) ? lmax_r[d] : 0u;
  int t = ECHO_MAX_DEPTH + 1;
#pragma unroll
  for (int d = ECHO_MAX_DEPTH; d >= 1; --d)
    if (((sp.mask >> d) & 1u) && !(v[d] > score_key(sp.lt[d]))) t = d;
  return t;
}

// One thread per candidate: keys at or below the request's truncation depth
// become 0 (never selected); the block histogram is built from what is left.
__global__ __launch_bounds__(kGateThreads) void gate_trunc_kernel(const int32_t* __restrict__ cand_offsets,
                                                                 int R, int N, GateWs ws,
                                                                 SparseArgs sp) {
  extern __shared__ int32_t s_offs[];  // R + 1 entries
  __shared__ uint32_t s_hist[kHistBins];
  __shared__ uint8_t s_t[kGateThreads + 1];  // truncation depth of requests r0 .. r0 + 1024
  __shared__ uint2 s_red[kGateThreads / kWave];
  __shared__ int s_flag;
  const int g0 = blockIdx.x * kGateThreads;
  const int g = g0 + threadIdx.x;
  // this thread's key and depth, fetched while the offsets load
  uint32_t key = g < N ? ws.keys[g] : 0u;
  const int dep = g < N ? int(ws.depth[g]) : 0;
  for (int i = threadIdx.x; i <= R; i += kGateThreads) s_offs[i] = cand_offsets[i];
  for (int i = threadIdx.x; i < kHistBins; i += kGateThreads) s_hist[i] = 0u;
  if (threadIdx.x == 0) s_flag = 0;
  __syncthreads();
  if (threadIdx.x == 0 && (s_offs[0] != 0 || s_offs[R] != N)) s_flag = 1;
  for (int r = threadIdx.x; r < R; r += kGateThreads)
    if (s_offs[r + 1] < s_offs[r]) s_flag = 1;
  __syncthreads();
  const bool ok = s_flag == 0;
  // the requests of this block's candidates are r0 .. r1 (at most 1025 of them)
  const int r0 = ok && g0 < N ? upper_bound_idx(s_offs, R + 1, g0) : 0;
  const int r1 = ok && g0 < N ? upper_bound_idx(s_offs, R + 1, min(N, g0 + kGateThreads) - 1) : -1;
  // (r1 - r0 exceeds 1024 only with empty requests in between: those beyond the
  // table are looked up directly)
  for (int r = r0 + int(threadIdx.x); r <= min(r1, r0 + kGateThreads); r += kGateThreads)
    s_t[r - r0] = uint8_t(first_failed(sp, ws.lmax + size_t(r) * kDepths));
  // the optional per-request output, spread over the blocks
  if (sp.trunc_out != nullptr) {
    const int per = (R + int(gridDim.x) - 1) / int(gridDim.x);
    for (int r = blockIdx.x * per + threadIdx.x; r < min(R, (blockIdx.x + 1) * per);
         r += kGateThreads)
      sp.trunc_out[r] = ok ? first_failed(sp, ws.lmax + size_t(r) * kDepths) : ECHO_MAX_DEPTH + 1;
  }
  __syncthreads();
  if (ok && g < N) {
    if (key != 0u) {
      const int r = upper_bound_idx(s_offs, R + 1, g);
      const int t = r - r0 <= kGateThreads ? int(s_t[r - r0])
                                           : first_failed(sp, ws.lmax + size_t(r) * kDepths);
      if (dep >= t) {
        key = 0u;
        ws.keys[g] = 0u;
      } else {
        atomicAdd(&s_hist[key >> kHistShift], 1u);
      }
    }
  }
  __syncthreads();
  write_block_hist(s_hist, s_red, ws);
}

// ------------------------------------------------------------------ bin ----
constexpr int kChunkBins = 64;                         // bins per downward step
constexpr int kChunkGroups = kGateThreads / kChunkBins;  // blocks summed in parallel per bin

// The threshold bin, computed by every select block (the histograms are small
// and L2-resident; this saves a launch).  Block 0 records it for gate_finish.
struct BinResult {
  uint32_t m;     // min(B, #finite keys)
  uint32_t bin;   // bin holding the m-th largest key
  uint32_t need;  // keys of that bin that are selected
  uint32_t cnt;   // keys in that bin
};

__device__ BinResult find_bin(int nblocks, int budget, const GateWs& ws, bool record,
                              int32_t* num_selected) {
  __shared__ uint32_t s_part[kChunkGroups][kChunkBins];
  __shared__ uint2 s_red[kGateThreads / kWave];
  __shared__ uint32_t s_state[2];  // keys in the bins above the current chunk, found flag
  __shared__ BinResult s_res;
  const int t = threadIdx.x;
  const int lane = t & (kWave - 1);
  // 1. #finite keys and the highest occupied bin over all score blocks
  uint32_t fin = 0u, top = 0u;
  for (int b = t; b < nblocks; b += kGateThreads) {
    const uint2 v = ws.bsum[b];
    fin += v.x;
    top = max(top, v.y);
  }
  fin = wave_sum(fin);
  top = wave_max(top);
  if (lane == 0) s_red[t / kWave] = make_uint2(fin, top);
  __syncthreads();
  fin = 0u;
  top = 0u;
#pragma unroll
  for (int w = 0; w < kGateThreads / kWave; ++w) {
    fin += s_red[w].x;
    top = max(top, s_red[w].y);
  }
  const uint32_t m = min(uint32_t(budget), fin);
  if (t == 0) {
    s_res.m = m;
    s_res.bin = 0u;
    s_res.need = 0u;
    s_res.cnt = 0u;
    s_state[0] = 0u;
    s_state[1] = 0u;
  }
  __syncthreads();
  if (m != 0u) {
    // 2. from the highest occupied bin downwards, 64 bins at a time
    const int j = t % kChunkBins;    // bin offset below the chunk's top
    const int grp = t / kChunkBins;  // blocks grp, grp + 16, ...
    for (int hi = int(top) - 1; hi >= 0; hi -= kChunkBins) {
      const int bin = hi - j;
      uint32_t c = 0u;
      if (bin >= 0) {
#pragma unroll 4
        for (int b = grp; b < nblocks; b += kChunkGroups) c += ws.bhist[size_t(b) * kHistBins + bin];
      }
      s_part[grp][j] = c;
      __syncthreads();
      if (t < kWave) {  // one wave scans the chunk's 64 bins, highest first
        uint32_t cnt = 0u;
#pragma unroll
        for (int g = 0; g < kChunkGroups; ++g) cnt += s_part[g][t];
        const uint32_t incl = wave_scan(cnt, 0u, AddOp{});  // sum over bins hi .. hi - t
        const uint32_t above = s_state[0];
        const bool cross = above + incl >= m && above + incl - cnt < m;
        if (cross) {
          s_res.bin = uint32_t(hi - t);
          s_res.cnt = cnt;
          s_res.need = m - (above + incl - cnt);
          s_state[1] = 1u;
        }
        const uint32_t total = uint32_t(__builtin_amdgcn_readlane(int(incl), kWave - 1));
        if (t == 0) s_state[0] = above + total;
      }
      __syncthreads();
      if (s_state[1] != 0u) break;
      __syncthreads();  // s_part is rewritten by the next chunk
    }
  }
  const BinResult r = s_res;
  if (record && t == 0) {
    ws.meta->num_selected = int32_t(r.m);
    ws.meta->bin = r.bin;
    ws.meta->bin_need = r.need;
    ws.meta->bin_cnt = r.cnt;
    ws.meta->thr_key = 0xFFFFFFFFu;
    ws.meta->thr_g = -1;
    *num_selected = int32_t(r.m);
  }
  return r;
}

// --------------------------------------------------------------- select ----
__global__ __launch_bounds__(kGateThreads) void gate_select_kernel(int N, int nblocks, int budget,
                                                                   GateWs ws,
                                                                   uint8_t* __restrict__ selected,
                                                                   int32_t* __restrict__ num_selected,
                                                                   int32_t* status) {
  __shared__ uint32_t s_cnt;
  const int g = blockIdx.x * kGateThreads + threadIdx.x;
  // this thread's key is fetched while the bin is found
  const uint32_t k = g < N ? ws.keys[g] : 0u;
  if (threadIdx.x == 0) s_cnt = 0u;
  const BinResult br = find_bin(nblocks, budget, ws, blockIdx.x == 0, num_selected);
  const uint32_t m = br.m;
  const uint32_t bin = br.bin;
  if (g < N) {
    const uint32_t kb = k >> kHistShift;
    if (m == 0u || k == 0u || kb < bin) {
      selected[g] = 0;
    } else if (kb > bin) {
      // selected, and so is its parent: the child's score is the parent's plus a
      // clamped log q <= 0 in one binary32 add, so the parent's key (same walk,
      // same clamps) is never below the child's and lies in a higher bin too
      selected[g] = 1;
    } else {
      const uint32_t slot = atomicAdd(&s_cnt, 1u);  // LDS; the order is fixed by the finish
      ws.cand[size_t(blockIdx.x) * kGateThreads + slot] = make_uint2(k, uint32_t(g));
    }
  }
  (void)status;  // nothing above the threshold bin can be unclosed (see above)
  __syncthreads();
  if (threadIdx.x == 0) ws.ccount[blockIdx.x] = s_cnt;
}

__global__ __launch_bounds__(kGateThreads) void gate_finish_kernel(int N, int nblocks, GateWs ws,
                                                                   uint8_t* __restrict__ selected,
                                                                   int32_t* status) {
  __shared__ uint32_t s_k[kSortCap];  // gathered candidates: key
  __shared__ int32_t s_g[kSortCap];   // and index
  __shared__ int s_base[kGateThreads + 1];
  gate_finish_body(N, nblocks, ws, selected, status, FinishLds{s_k, s_g, s_base});
}

}  // namespace

namespace {

// The gate's launches; the last phase (gate_finish) only if `finish`.
int32_t launch_gate_impl(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                         int32_t R, int32_t N, int32_t budget, const int32_t* sig_depth,
                         const float* log_tau, int32_t num_sig, float* path_score,
                         uint8_t* selected, int32_t* num_selected, int32_t* trunc_depth,
                         void* workspace, int32_t* status, bool finish, hipStream_t stream) {
  (void)hipGetLastError();  // clear errors left by unrelated runtime calls
  GateWs ws = gate_ws_layout(workspace, N, R);
  const int blocks = gate_blocks(N);
  const size_t lds = size_t(R + 1) * sizeof(int32_t);
  SparseArgs sp{};
  sp.enabled = num_sig > 0 || trunc_depth != nullptr ? 1 : 0;
  sp.mask = 0u;
  for (int d = 0; d < kDepths; ++d) sp.lt[d] = -__builtin_inff();
  for (int k = 0; k < num_sig; ++k) {
    const int d = sig_depth[k];
    // a depth listed twice must pass both thresholds: keep the larger
    if (!((sp.mask >> d) & 1u) || log_tau[k] > sp.lt[d]) sp.lt[d] = log_tau[k];
    sp.mask |= 1u << d;
  }
  sp.trunc_out = trunc_depth;
  if (sp.enabled) {
    const int n = R * kDepths;
    hipLaunchKernelGGL(gate_lmax_clear_kernel, dim3((n + kGateThreads - 1) / kGateThreads),
                       dim3(kGateThreads), 0, stream, n, ws.lmax);
  }
  hipLaunchKernelGGL(gate_score_kernel, dim3(blocks), dim3(kGateThreads), lds, stream,
                     cand_offsets, parent, logq, R, N, ws, path_score, status, sp);
  if (sp.enabled)
    hipLaunchKernelGGL(gate_trunc_kernel, dim3(blocks), dim3(kGateThreads), lds, stream,
                       cand_offsets, R, N, ws, sp);
  hipLaunchKernelGGL(gate_select_kernel, dim3(blocks), dim3(kGateThreads), 0, stream, N, blocks,
                     budget, ws, selected, num_selected, status);
  if (N > 0 && finish) {
    hipLaunchKernelGGL(gate_finish_kernel, dim3(1), dim3(kGateThreads), 0, stream, N, blocks, ws,
                       selected, status);
  }
  return hipGetLastError() == hipSuccess ? ECHO_OK : ECHO_ERR_HIP;
}

}  // namespace

int32_t launch_gate(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                    int32_t R, int32_t N, int32_t budget, const int32_t* sig_depth,
                    const float* log_tau, int32_t num_sig, float* path_score, uint8_t* selected,
                    int32_t* num_selected, int32_t* trunc_depth, void* workspace, int32_t* status,
                    hipStream_t stream) {
  return launch_gate_impl(cand_offsets, parent, logq, R, N, budget, sig_depth, log_tau, num_sig,
                          path_score, selected, num_selected, trunc_depth, workspace, status, true,
                          stream);
}

int32_t launch_gate_select_only(const int32_t* cand_offsets, const int32_t* parent,
                                const float* logq, int32_t R, int32_t N, int32_t budget,
                                float* path_score, uint8_t* selected, int32_t* num_selected,
                                void* workspace, int32_t* status, hipStream_t stream) {
  return launch_gate_impl(cand_offsets, parent, logq, R, N, budget, nullptr, nullptr, 0,
                          path_score, selected, num_selected, nullptr, workspace, status, false,
                          stream);
}

int32_t launch_gate_score(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                          int32_t R, int32_t N, float* path_score, void* workspace,
                          int32_t* status, hipStream_t stream, GateScoreBufs* out) {
  GateWs ws = gate_ws_layout(workspace, N, R);
  SparseArgs sp{};
  sp.enabled = 1;  // depths written, no histograms, no checkpoint maxima (mask 0)
  sp.mask = 0u;
  for (int d = 0; d < kDepths; ++d) sp.lt[d] = -__builtin_inff();
  sp.trunc_out = nullptr;
  const size_t lds = size_t(R + 1) * sizeof(int32_t);
  hipLaunchKernelGGL(gate_score_kernel, dim3(gate_blocks(N)), dim3(kGateThreads), lds, stream,
                     cand_offsets, parent, logq, R, N, ws, path_score, status, sp);
  out->keys = ws.keys;
  out->pglob = ws.pglob;
  out->depth = ws.depth;
  return hipGetLastError() == hipSuccess ? ECHO_OK : ECHO_ERR_HIP;
}

size_t gate_workspace_bytes(int32_t R, int32_t N, int32_t budget) {
  (void)budget;
  return gate_ws_bytes(N, R);
}

}  // namespace echo
