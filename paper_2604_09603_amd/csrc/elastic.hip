// Elastic budget scheduling (Alg. 1, Section 3.3) as a selection policy over
// the drafted candidate pool.  Phase 1 walks the depths and serves the active
// requests, in request order, from the shared budget: a request passes the
// checkpoint test of its depth (eq. 7 on the largest path score among the
// depth-d candidates it can append, eq. 6) and appends its W_topk best ones,
// or fails and is truncated.  Phase 2 widens every truncated request's last
// kept depth up to W_max nodes while budget is left.
//
// Four launches.  The coupling between requests is only through the budget,
// and until the budget runs out every request receives its whole demand, so
// each request's phase-1 trajectory can be computed on its own:
//
//   gate_score        (shared with the top-B gate) keys, clamped parents, depths
//   elastic_request   one workgroup per request: its full-grant trajectory --
//                     per depth the appendable candidates (parent held), the
//                     checkpoint test, the demand min(W_topk, #appendable) and
//                     every appendable candidate's rank (key descending, index
//                     ascending); the first failed checkpoint and the phase-2
//                     demand at the depth above it
//   elastic_finish    one workgroup: walks the depths with the budget, finds the
//                     depth where the demands reach what is left and grants it
//                     in request order; otherwise grants the phase-2 demands in
//                     request order
//   elastic_select    one thread per candidate: selected iff its rank is below
//                     its request's grant at its depth (or inside the phase-2
//                     grant at the widened depth); checks ancestor closure
#include "echo_device.h"
#include "echo_internal.h"

namespace echo {
namespace {

constexpr int kElThreads = 256;                 // elastic_request: one workgroup per request
constexpr int kElCap = 4096;                    // candidates of a request staged in LDS
constexpr int kSlots = ECHO_MAX_DEPTH + 1;      // per-request depth slots (0 unused)
constexpr int kNone = ECHO_MAX_DEPTH + 1;       // "no failed checkpoint" / "no cut"
constexpr int kFinThreads = 1024;
constexpr int kSelThreads = 1024;

struct ElasticArgs {
  uint32_t mask;      // bit d set iff depth d is a checkpoint
  float lt[kSlots];   // ln tau of each checkpoint depth (the largest if repeated)
  int w_topk;         // default width appended per depth (>= 1)
  int w_max;          // width a truncated request may widen its last depth to
};

struct ElasticWs {
  int32_t* rank;  // [N] rank among its depth's appendable candidates on the trajectory, -1 none
  uint8_t* sel;   // [N] trajectory flags of requests too large for LDS
  int32_t* list;  // [N] appendable lists of requests too large for LDS
  uint64_t* word; // [N] their rank words
  int32_t* dem;   // [R][kSlots] phase-1 demand per depth on the full-grant trajectory
  int32_t* tdep;  // [R] first failed checkpoint on the trajectory, kNone if none
  int32_t* w2;    // [R] phase-2 demand
  int32_t* g1;    // [R] grant at the cut depth
  int32_t* g2;    // [R] phase-2 grant
  int32_t* meta;  // [0] cut depth (kNone: the budget outlasted phase 1)
};

__host__ __device__ inline size_t el_align(size_t x) { return (x + 255) / 256 * 256; }

__host__ inline size_t elastic_own_bytes(int32_t R, int32_t N) {
  return 256 + el_align(size_t(N) * 4) + el_align(size_t(N)) + el_align(size_t(N) * 4) +
         el_align(size_t(N) * 8) + el_align(size_t(R) * kSlots * 4) + 4 * el_align(size_t(R) * 4);
}

__host__ inline ElasticWs elastic_ws_layout(void* base, int32_t R, int32_t N) {
  char* p = static_cast<char*>(base);
  ElasticWs w;
  w.meta = reinterpret_cast<int32_t*>(p);
  p += 256;
  w.rank = reinterpret_cast<int32_t*>(p);
  p += el_align(size_t(N) * 4);
  w.sel = reinterpret_cast<uint8_t*>(p);
  p += el_align(size_t(N));
  w.list = reinterpret_cast<int32_t*>(p);
  p += el_align(size_t(N) * 4);
  w.word = reinterpret_cast<uint64_t*>(p);
  p += el_align(size_t(N) * 8);
  w.dem = reinterpret_cast<int32_t*>(p);
  p += el_align(size_t(R) * kSlots * 4);
  w.tdep = reinterpret_cast<int32_t*>(p);
  p += el_align(size_t(R) * 4);
  w.w2 = reinterpret_cast<int32_t*>(p);
  p += el_align(size_t(R) * 4);
  w.g1 = reinterpret_cast<int32_t*>(p);
  p += el_align(size_t(R) * 4);
  w.g2 = reinterpret_cast<int32_t*>(p);
  return w;
}

// ------------------------------------------------------------- request ----
struct ElasticLds {
  uint32_t key[kElCap];
  int32_t par[kElCap];       // request-local parent, -1 = the root
  uint16_t order[kElCap];    // finite candidates grouped by depth (staged requests)
  uint8_t dep[kElCap];
  uint8_t sel[kElCap];
  int32_t list[kElCap];
  uint64_t word[kElCap];     // (key, ~index) of each listed candidate: larger = better
  int off[kSlots + 1];       // start of each depth's group in `order`
  int fill[kSlots];
  int cnt[2];
  uint32_t mx[2];
  int A[kSlots];    // appendable candidates per depth
  int dem[kSlots];  // phase-1 demand per depth
};

__device__ __forceinline__ uint64_t rank_word(uint32_t key, int i) {
  return (uint64_t(key) << 32) | uint64_t(0xFFFFFFFFu - uint32_t(i));
}

// Position of this lane among the lanes of `bal` below it.
__device__ __forceinline__ int lanes_below(uint64_t bal) {
  return int(__builtin_amdgcn_mbcnt_hi(uint32_t(bal >> 32),
                                       __builtin_amdgcn_mbcnt_lo(uint32_t(bal), 0u)));
}

// counter[d] += 1 for every lane with `on` and depth d, with one LDS atomic per
// distinct depth in the wave; returns the counter's value before this lane's
// increment (lanes of one depth take consecutive values).  Every lane of the
// wave must call it.
__device__ __forceinline__ int add_by_depth(bool on, int d, int* counter) {
  uint64_t rem = __ballot(on);
  int before = 0;
  while (rem != 0ull) {  // uniform: one round per distinct depth
    const int lead = __builtin_ctzll(rem);
    const int dl = __builtin_amdgcn_readlane(d, lead);
    const uint64_t bal = __ballot(on && d == dl);
    int base = 0;
    if ((threadIdx.x & (kWave - 1)) == lead) base = atomicAdd(&counter[dl], __popcll(bal));
    base = __builtin_amdgcn_readlane(base, lead);
    if (on && d == dl) before = base + lanes_below(bal);
    rem &= ~bal;
  }
  return before;
}

// Append candidate i (key k) to a depth's appendable list when `take`, with one
// LDS atomic per wave for the list length and one for the depth's largest key
// (per-lane atomics on the same two words serialise).  Every lane of the wave
// must call it (the ballot and shuffles are wave-wide).
__device__ __forceinline__ void append_wave(bool take, int i, uint32_t k, int* cnt, uint32_t* mx,
                                            int32_t* list, uint64_t* word) {
  const uint64_t bal = __ballot(take);
  if (bal == 0ull) return;  // uniform
  const int lane = threadIdx.x & (kWave - 1);
  const int n = __popcll(bal);
  const uint32_t km = wave_max(take ? k : 0u);
  int base = 0;
  if (lane == 0) {
    base = atomicAdd(cnt, n);
    atomicMax(mx, km);
  }
  base = __builtin_amdgcn_readlane(base, 0);
  if (take) {
    const int pos = base + lanes_below(bal);
    list[pos] = i;
    word[pos] = rank_word(k, i);
  }
}

// Rank of every listed candidate among the A listed ones (key descending,
// local index ascending: the order of their words); the first `dem` are taken.
// Every lane of a wave reads the same word at a time (an LDS broadcast).
template <typename Sel>
__device__ __forceinline__ void rank_level(const int32_t* list, const uint64_t* word, int A,
                                           int dem, Sel sel, int lo, const ElasticWs& ew) {
  for (int j = threadIdx.x; j < A; j += kElThreads) {
    const uint64_t w = word[j];
    int rank = 0;
    int m = 0;
    for (; m + 4 <= A; m += 4)
      rank += int(word[m] > w) + int(word[m + 1] > w) + int(word[m + 2] > w) +
              int(word[m + 3] > w);
    for (; m < A; ++m) rank += int(word[m] > w);
    const int i = list[j];
    ew.rank[lo + i] = rank;
    if (rank < dem) sel(i);
  }
}

// Per-request results of the trajectory (thread 0): demands, first failed
// checkpoint t and the phase-2 demand at depth t - 1.
__device__ __forceinline__ void write_trajectory(int r, int t, const ElasticArgs& ea,
                                                 const ElasticWs& ew, const ElasticLds& L) {
  ew.dem[size_t(r) * kSlots] = 0;
  for (int d = 1; d <= ECHO_MAX_DEPTH; ++d) ew.dem[size_t(r) * kSlots + d] = L.dem[d];
  ew.tdep[r] = t;
  int w = 0;
  if (t >= 2 && t <= ECHO_MAX_DEPTH) {
    const int l = t - 1;
    w = max(0, min(ea.w_max - L.dem[l], L.A[l] - L.dem[l]));
  }
  ew.w2[r] = w;
}

// One depth of the trajectory after its appendable list is built: the
// checkpoint test (eq. 7 on keys: order-preserving, -0 == +0, -inf -> 0) and
// the demand.  Returns false when the walk stops (t set on a failed test).
__device__ __forceinline__ bool level_test(int d, int A, uint32_t mx, const ElasticArgs& ea,
                                           int* t) {
  if (((ea.mask >> d) & 1u) && !(mx > score_key(ea.lt[d]))) {
    *t = d;
    return false;
  }
  return A > 0;  // none appendable: the drafted tree is exhausted
}

// Trajectory of a request whose candidates fit in LDS: they are grouped by
// depth once, so each depth visits only its own candidates.
__device__ void trajectory_staged(int r, int lo, int n, const GateScoreBufs& sb,
                                  const ElasticArgs& ea, const ElasticWs& ew, ElasticLds& L) {
  const int tid = threadIdx.x;
  if (tid <= kSlots) L.off[tid] = 0;
  if (tid < kSlots) {
    L.fill[tid] = 0;
    L.A[tid] = 0;
    L.dem[tid] = 0;
  }
  if (tid < 2) {
    L.cnt[tid] = 0;
    L.mx[tid] = 0u;
  }
  __syncthreads();
  // all of this thread's candidates are fetched before any is stored, so the
  // loads overlap instead of paying the memory latency once per candidate
  constexpr int kPer = kElCap / kElThreads;
  uint32_t kk[kPer];
  int pp[kPer], dd[kPer];
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const int i = tid + q * kElThreads;
    kk[q] = i < n ? sb.keys[lo + i] : 0u;
    pp[q] = i < n ? sb.pglob[lo + i] : -1;
    dd[q] = i < n ? int(sb.depth[lo + i]) : 0;
  }
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const int i = tid + q * kElThreads;
    if (i < n) {
      L.key[i] = kk[q];
      L.par[i] = pp[q] < 0 ? -1 : pp[q] - lo;
      L.dep[i] = uint8_t(dd[q]);
      L.sel[i] = 0;
      ew.rank[lo + i] = -1;
    }
    add_by_depth(i < n && kk[q] != 0u, dd[q] + 1, L.off);  // finite keys have depth <= 16
  }
  __syncthreads();
  if (tid < kWave) {  // inclusive scan of the depth counts (18 entries) in one wave
    const int v = wave_inclusive_sum(tid <= kSlots ? L.off[tid] : 0);
    if (tid <= kSlots) L.off[tid] = v;
  }
  __syncthreads();
  for (int i0 = 0; i0 < n; i0 += kElThreads) {  // bounds uniform in the workgroup
    const int i = i0 + tid;
    const bool on = i < n && L.key[i] != 0u;
    const int d = on ? int(L.dep[i]) : 0;
    const int k = add_by_depth(on, d, L.fill);
    if (on) L.order[L.off[d] + k] = uint16_t(i);
  }
  __syncthreads();
  int t = kNone;
  int par = 0;
  for (int d = 1; d <= ECHO_MAX_DEPTH; ++d) {
    const int j1 = L.off[d + 1];
    for (int j0 = L.off[d]; j0 < j1; j0 += kElThreads) {  // bounds uniform in the workgroup
      const int j = j0 + tid;
      int i = 0;
      bool take = false;
      if (j < j1) {
        i = L.order[j];
        const int p = L.par[i];
        take = p < 0 || L.sel[p];
      }
      append_wave(take, i, take ? L.key[i] : 0u, &L.cnt[par], &L.mx[par], L.list, L.word);
    }
    __syncthreads();
    const int A = L.cnt[par];
    if (!level_test(d, A, L.mx[par], ea, &t)) break;
    const int dem = min(ea.w_topk, A);
    rank_level(L.list, L.word, A, dem, [&](int i) { L.sel[i] = 1; }, lo, ew);
    if (tid == 0) {
      L.A[d] = A;
      L.dem[d] = dem;
      L.cnt[par ^ 1] = 0;
      L.mx[par ^ 1] = 0u;
    }
    __syncthreads();
    par ^= 1;
  }
  if (tid == 0) write_trajectory(r, t, ea, ew, L);
}

// Trajectory of a request too large for LDS: flags and lists in the workspace,
// every depth scans the request's candidates.
__device__ void trajectory_global(int r, int lo, int n, const GateScoreBufs& sb,
                                  const ElasticArgs& ea, const ElasticWs& ew, ElasticLds& L) {
  const int tid = threadIdx.x;
  uint8_t* sel = ew.sel + lo;
  int32_t* list = ew.list + lo;
  uint64_t* word = ew.word + lo;
  for (int i = tid; i < n; i += kElThreads) {
    sel[i] = 0;
    ew.rank[lo + i] = -1;
  }
  if (tid < kSlots) {
    L.A[tid] = 0;
    L.dem[tid] = 0;
  }
  if (tid < 2) {
    L.cnt[tid] = 0;
    L.mx[tid] = 0u;
  }
  __syncthreads();
  int t = kNone;
  int par = 0;
  for (int d = 1; d <= ECHO_MAX_DEPTH; ++d) {
    for (int i0 = 0; i0 < n; i0 += kElThreads) {  // bounds uniform in the workgroup
      const int i = i0 + tid;
      uint32_t k = 0u;
      bool take = false;
      if (i < n && int(sb.depth[lo + i]) == d) {
        k = sb.keys[lo + i];
        const int p = sb.pglob[lo + i];
        take = k != 0u && (p < 0 || sel[p - lo]);
      }
      append_wave(take, i, k, &L.cnt[par], &L.mx[par], list, word);
    }
    __syncthreads();
    const int A = L.cnt[par];
    if (!level_test(d, A, L.mx[par], ea, &t)) break;
    const int dem = min(ea.w_topk, A);
    rank_level(list, word, A, dem, [&](int i) { sel[i] = 1; }, lo, ew);
    if (tid == 0) {
      L.A[d] = A;
      L.dem[d] = dem;
      L.cnt[par ^ 1] = 0;
      L.mx[par ^ 1] = 0u;
    }
    __syncthreads();
    par ^= 1;
  }
  if (tid == 0) write_trajectory(r, t, ea, ew, L);
}

__global__ __launch_bounds__(kElThreads) void elastic_request_kernel(
    const int32_t* __restrict__ cand_offsets, int N, GateScoreBufs sb, ElasticArgs ea,
    ElasticWs ew) {
  __shared__ ElasticLds L;
  const int r = blockIdx.x;
  int lo = cand_offsets[r], hi = cand_offsets[r + 1];
  // a malformed CSR leaves every key at 0 (nothing appendable); only keep the
  // range in bounds
  if (lo < 0 || hi > N || hi < lo) lo = hi = 0;
  const int n = hi - lo;
  if (n <= kElCap) trajectory_staged(r, lo, n, sb, ea, ew, L);
  else trajectory_global(r, lo, n, sb, ea, ew, L);
}

// -------------------------------------------------------------- finish ----
__global__ __launch_bounds__(kFinThreads) void elastic_finish_kernel(int R, int budget,
                                                                    ElasticWs ew,
                                                                    int32_t* __restrict__ num_selected,
                                                                    int32_t* __restrict__ trunc_out) {
  constexpr int NW = kFinThreads / kWave;
  __shared__ int s_tot[kFinThreads][kSlots];  // per-thread demands, summed by column
  __shared__ int s_col[kSlots];
  __shared__ int s_scan[NW + 1];
  __shared__ int s_cut, s_left;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
  // 1. total phase-1 demand per depth; the first request of each thread is
  // kept in registers for step 3
  const int tdep0 = tid < R ? ew.tdep[tid] : kNone;
  const int w20 = tid < R ? ew.w2[tid] : 0;
  int dem0[kSlots], tot[kSlots];
#pragma unroll
  for (int d = 0; d < kSlots; ++d) {
    dem0[d] = (d > 0 && tid < R) ? ew.dem[size_t(tid) * kSlots + d] : 0;
    tot[d] = dem0[d];
  }
  for (int r = tid + kFinThreads; r < R; r += kFinThreads) {
#pragma unroll
    for (int d = 1; d < kSlots; ++d) tot[d] += ew.dem[size_t(r) * kSlots + d];
  }
  // column sums through LDS: wave w adds depth w + 1 over all threads
  static_assert(kFinThreads / kWave == ECHO_MAX_DEPTH, "one wave per depth");
#pragma unroll
  for (int d = 1; d < kSlots; ++d) s_tot[tid][d] = tot[d];
  __syncthreads();
  {
    const int d = wid + 1;
    int v = 0;
#pragma unroll
    for (int k = 0; k < kFinThreads / kWave; ++k) v += s_tot[lane + kWave * k][d];
    v = int(wave_sum(uint32_t(v)));
    if (lane == 0) s_col[d] = v;
  }
  __syncthreads();
  // 2. the depth loop of phase 1 runs while budget is left; the cut is the
  // first depth whose demands reach what is left: there the budget runs out
  // (exactly, or part way), and the requests after that point are not tested
  if (tid < kWave) {
    int left = budget, cut = kNone;
#pragma unroll
    for (int d = 1; d <= ECHO_MAX_DEPTH; ++d) {
      const int Td = s_col[d];
      if (cut == kNone) {
        if (Td >= left) cut = d;
        else left -= Td;
      }
    }
    if (tid == 0) {
      s_cut = cut;
      s_left = left;
    }
  }
  __syncthreads();
  const int cut = s_cut;
  const int left = s_left;
  int run = 0;
  if (cut <= ECHO_MAX_DEPTH) {
    // requests in order take what is left at the cut depth; one is tested at
    // all (and can be truncated there) only while budget remains at its turn
    for (int r0 = 0; r0 < R; r0 += kFinThreads) {
      const int r = r0 + tid;
      int v = 0;
      if (r0 == 0) {
#pragma unroll
        for (int d = 1; d < kSlots; ++d) v = d == cut ? dem0[d] : v;
      } else if (r < R) {
        v = ew.dem[size_t(r) * kSlots + cut];
      }
      int tot_c;
      const int excl = run + block_exclusive_sum<kFinThreads>(v, s_scan, &tot_c);
      if (r < R) {
        ew.g1[r] = max(0, min(v, left - excl));
        ew.g2[r] = 0;
        if (trunc_out != nullptr) {
          const int td = r0 == 0 ? tdep0 : ew.tdep[r];
          trunc_out[r] = (td < cut || (td == cut && excl < left)) ? td : kNone;
        }
      }
      run += tot_c;
    }
    if (tid == 0) {
      ew.meta[0] = cut;
      *num_selected = budget;  // the cut depth consumes everything left
    }
  } else {
    // phase 2: truncated requests in order widen with what is left
    for (int r0 = 0; r0 < R; r0 += kFinThreads) {
      const int r = r0 + tid;
      const int v = r0 == 0 ? w20 : (r < R ? ew.w2[r] : 0);
      int tot_c;
      const int excl = run + block_exclusive_sum<kFinThreads>(v, s_scan, &tot_c);
      if (r < R) {
        ew.g1[r] = 0;
        ew.g2[r] = max(0, min(v, left - excl));
        if (trunc_out != nullptr) trunc_out[r] = r0 == 0 ? tdep0 : ew.tdep[r];
      }
      run += tot_c;
    }
    if (tid == 0) {
      ew.meta[0] = kNone;
      *num_selected = budget - (left - min(run, left));
    }
  }
}

// -------------------------------------------------------------- select ----
__global__ __launch_bounds__(kSelThreads) void elastic_select_kernel(
    const int32_t* __restrict__ cand_offsets, int R, int N, GateScoreBufs sb, ElasticWs ew,
    uint8_t* __restrict__ selected, int32_t* status) {
  extern __shared__ int32_t s_offs[];  // R + 1 entries
  for (int i = threadIdx.x; i <= R; i += kSelThreads) s_offs[i] = cand_offsets[i];
  __syncthreads();
  const int g = blockIdx.x * kSelThreads + threadIdx.x;
  const int cut = ew.meta[0];
  // the selection rule, with each round of independent loads issued together
  auto is_sel = [&](int x) -> bool {
    const uint32_t key = sb.keys[x];
    const int rk = ew.rank[x];
    const int d = int(sb.depth[x]);
    if (key == 0u || rk < 0) return false;  // also every candidate of a malformed CSR
    const int r = upper_bound_idx(s_offs, R + 1, x);
    const int dm = ew.dem[size_t(r) * kSlots + d];  // d <= 16: the key is finite
    const int a = ew.g1[r];
    const int b = ew.g2[r];
    const int td = ew.tdep[r];
    if (d < cut && rk < dm) return true;
    if (d == cut && rk < a) return true;
    return cut == kNone && d == td - 1 && rk >= dm && rk < dm + b;
  };
  int bits = 0;
  if (g < N) {
    const int p = sb.pglob[g];
    const bool s = is_sel(g);
    selected[g] = s ? 1 : 0;
    if (s && p >= 0 && !is_sel(p)) bits |= ECHO_DATA_NOT_CLOSED;
  }
  wave_status_or(status, bits);
}

}  // namespace

size_t gate_elastic_workspace_bytes(int32_t R, int32_t N, int32_t budget) {
  return el_align(gate_workspace_bytes(R, N, budget)) + elastic_own_bytes(R, N);
}

int32_t launch_gate_elastic(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                            int32_t R, int32_t N, int32_t budget, const int32_t* sig_depth,
                            const float* log_tau, int32_t num_sig, int32_t w_topk, int32_t w_max,
                            float* path_score, uint8_t* selected, int32_t* num_selected,
                            int32_t* trunc_depth, void* workspace, int32_t* status,
                            hipStream_t stream) {
  (void)hipGetLastError();  // clear errors left by unrelated runtime calls
  ElasticArgs ea{};
  ea.mask = 0u;
  for (int d = 0; d < kSlots; ++d) ea.lt[d] = -__builtin_inff();
  for (int k = 0; k < num_sig; ++k) {
    const int d = sig_depth[k];
    // a depth listed twice must pass both thresholds: keep the larger
    if (!((ea.mask >> d) & 1u) || log_tau[k] > ea.lt[d]) ea.lt[d] = log_tau[k];
    ea.mask |= 1u << d;
  }
  ea.w_topk = w_topk;
  ea.w_max = w_max;
  GateScoreBufs sb;
  if (launch_gate_score(cand_offsets, parent, logq, R, N, path_score, workspace, status, stream,
                        &sb) != ECHO_OK)
    return ECHO_ERR_HIP;
  char* own = static_cast<char*>(workspace) + el_align(gate_workspace_bytes(R, N, budget));
  const ElasticWs ew = elastic_ws_layout(own, R, N);
  hipLaunchKernelGGL(elastic_request_kernel, dim3(R), dim3(kElThreads), 0, stream, cand_offsets,
                     N, sb, ea, ew);
  hipLaunchKernelGGL(elastic_finish_kernel, dim3(1), dim3(kFinThreads), 0, stream, R, budget, ew,
                     num_selected, trunc_depth);
  if (N > 0)
    hipLaunchKernelGGL(elastic_select_kernel, dim3((N + kSelThreads - 1) / kSelThreads),
                       dim3(kSelThreads), size_t(R + 1) * sizeof(int32_t), stream, cand_offsets,
                       R, N, sb, ew, selected, status);
  return hipGetLastError() == hipSuccess ? ECHO_OK : ECHO_ERR_HIP;
}

}  // namespace echo
