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
         el_align(size_t(R) * kSlots * 4) + 4 * el_align(size_t(R) * 4);
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
  int32_t par[kElCap];  // request-local parent, -1 = the root
  uint8_t dep[kElCap];
  uint8_t sel[kElCap];
  int32_t list[kElCap];
  int cnt[2];
  uint32_t mx[2];
  int A[kSlots];    // appendable candidates per depth
  int dem[kSlots];  // phase-1 demand per depth
};

// The trajectory of request r over its n candidates g = lo + i.  kStaged: the
// candidates live in LDS; otherwise they are read from the score buffers and
// the flags and lists live in the workspace.
template <bool kStaged>
__device__ void request_trajectory(int r, int lo, int n, const GateScoreBufs& sb,
                                   const ElasticArgs& ea, const ElasticWs& ew, ElasticLds& L) {
  const int tid = threadIdx.x;
  uint8_t* SEL = kStaged ? L.sel : ew.sel + lo;
  int32_t* LIST = kStaged ? L.list : ew.list + lo;
  auto keyf = [&](int i) -> uint32_t { return kStaged ? L.key[i] : sb.keys[lo + i]; };
  auto depf = [&](int i) -> int { return kStaged ? int(L.dep[i]) : int(sb.depth[lo + i]); };
  auto parf = [&](int i) -> int {
    if (kStaged) return L.par[i];
    const int p = sb.pglob[lo + i];
    return p < 0 ? -1 : p - lo;
  };
  for (int i = tid; i < n; i += kElThreads) {
    if (kStaged) {
      L.key[i] = sb.keys[lo + i];
      const int p = sb.pglob[lo + i];
      L.par[i] = p < 0 ? -1 : p - lo;
      L.dep[i] = sb.depth[lo + i];
    }
    SEL[i] = 0;
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
    // appendable depth-d candidates: finite, parent held (or the root)
    for (int i = tid; i < n; i += kElThreads) {
      if (depf(i) != d) continue;
      const uint32_t k = keyf(i);
      if (k == 0u) continue;
      const int p = parf(i);
      if (p >= 0 && !SEL[p]) continue;
      LIST[atomicAdd(&L.cnt[par], 1)] = i;
      atomicMax(&L.mx[par], k);
    }
    __syncthreads();
    const int A = L.cnt[par];
    const uint32_t mx = L.mx[par];
    // eq. 7: the largest appendable path score strictly above ln tau (keys are
    // order-preserving, -0 == +0, -inf has key 0)
    const bool pass = !((ea.mask >> d) & 1u) || mx > score_key(ea.lt[d]);
    if (!pass) {
      t = d;
      break;
    }
    if (A == 0) break;  // drafted tree exhausted
    const int dem = min(ea.w_topk, A);
    for (int j = tid; j < A; j += kElThreads) {
      const int i = LIST[j];
      const uint32_t k = keyf(i);
      int rank = 0;
      for (int m = 0; m < A; ++m) {
        const int o = LIST[m];
        const uint32_t ko = keyf(o);
        rank += (ko > k || (ko == k && o < i)) ? 1 : 0;
      }
      ew.rank[lo + i] = rank;
      if (rank < dem) SEL[i] = 1;
    }
    if (tid == 0) {
      L.A[d] = A;
      L.dem[d] = dem;
      L.cnt[par ^ 1] = 0;
      L.mx[par ^ 1] = 0u;
    }
    __syncthreads();
    par ^= 1;
  }
  if (tid == 0) {
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
  if (n <= kElCap) request_trajectory<true>(r, lo, n, sb, ea, ew, L);
  else request_trajectory<false>(r, lo, n, sb, ea, ew, L);
}

// -------------------------------------------------------------- finish ----
__global__ __launch_bounds__(kFinThreads) void elastic_finish_kernel(int R, int budget,
                                                                    ElasticWs ew,
                                                                    int32_t* __restrict__ num_selected,
                                                                    int32_t* __restrict__ trunc_out) {
  constexpr int NW = kFinThreads / kWave;
  __shared__ int s_tot[NW][kSlots];
  __shared__ int s_scan[NW + 1];
  __shared__ int s_cut, s_left;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
  // 1. total phase-1 demand per depth
  int tot[kSlots];
#pragma unroll
  for (int d = 0; d < kSlots; ++d) tot[d] = 0;
  for (int r = tid; r < R; r += kFinThreads) {
#pragma unroll
    for (int d = 1; d < kSlots; ++d) tot[d] += ew.dem[size_t(r) * kSlots + d];
  }
#pragma unroll
  for (int d = 1; d < kSlots; ++d) {
    int v = tot[d];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
    if (lane == 0) s_tot[wid][d] = v;
  }
  __syncthreads();
  // 2. the depth loop of phase 1 runs while budget is left; the cut is the
  // first depth whose demands reach what is left: there the budget runs out
  // (exactly, or part way), and the requests after that point are not tested
  if (tid == 0) {
    int left = budget, cut = kNone;
    for (int d = 1; d <= ECHO_MAX_DEPTH; ++d) {
      int T = 0;
      for (int w = 0; w < NW; ++w) T += s_tot[w][d];
      if (T >= left) {
        cut = d;
        break;
      }
      left -= T;
    }
    s_cut = cut;
    s_left = left;
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
      const int v = r < R ? ew.dem[size_t(r) * kSlots + cut] : 0;
      int tot_c;
      const int excl = run + block_exclusive_sum<kFinThreads>(v, s_scan, &tot_c);
      if (r < R) {
        ew.g1[r] = max(0, min(v, left - excl));
        ew.g2[r] = 0;
        if (trunc_out != nullptr) {
          const int td = ew.tdep[r];
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
      const int v = r < R ? ew.w2[r] : 0;
      int tot_c;
      const int excl = run + block_exclusive_sum<kFinThreads>(v, s_scan, &tot_c);
      if (r < R) {
        ew.g1[r] = 0;
        ew.g2[r] = max(0, min(v, left - excl));
        if (trunc_out != nullptr) trunc_out[r] = ew.tdep[r];
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
  auto is_sel = [&](int x) -> bool {
    if (sb.keys[x] == 0u) return false;  // also every candidate of a malformed CSR
    const int rk = ew.rank[x];
    if (rk < 0) return false;
    const int r = upper_bound_idx(s_offs, R + 1, x);
    const int d = int(sb.depth[x]);
    const int dm = ew.dem[size_t(r) * kSlots + d];
    if (d < cut && rk < dm) return true;
    if (d == cut && rk < ew.g1[r]) return true;
    return cut == kNone && d == ew.tdep[r] - 1 && rk >= dm && rk < dm + ew.g2[r];
  };
  int bits = 0;
  if (g < N) {
    const bool s = is_sel(g);
    selected[g] = s ? 1 : 0;
    if (s) {
      const int p = sb.pglob[g];
      if (p >= 0 && !is_sel(p)) bits |= ECHO_DATA_NOT_CLOSED;
    }
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
