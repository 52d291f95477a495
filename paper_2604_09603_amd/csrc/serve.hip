// The serving step around the verification path: the greedy target token of
// every verify slot (argmax of its vocabulary logits) feeding acceptance, and
// the commit of each request's accepted path into a paged KV cache.
//
//   target_argmax   one workgroup per slot row: streams the row's bfloat16
//                   logits with 16-byte loads, eight in flight per thread
//                   (HBM-bound: Nq * V * 2 bytes), keeps per thread the first
//                   largest value in its own index order; a workgroup reduction
//                   picks the largest value, ties to the smaller token id.  Then
//                   the acceptance kernel.
//   commit_kv       one workgroup per request: copies the root slot's and the
//                   accepted slots' K and V rows into their pages, then advances
//                   the request's cached length.
#include "echo_device.h"
#include "echo_internal.h"

namespace echo {
namespace {

constexpr int kArgThreads = 512;  // two workgroups per CU: every slot row of a batch is resident
constexpr int kArgUnroll = 8;  // 16-byte loads in flight per thread
constexpr int kCommitThreads = 256;
constexpr uint32_t kNoIdx = 0xFFFFFFFFu;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// One workgroup per slot row.  Each thread keeps the first strictly largest
// value of its own elements, visited in increasing index order (a NaN never
// compares greater, so it is never kept; -0 and +0 compare equal); the
// workgroup then takes the largest value, ties to the smaller index.  A row
// in which nothing beats -inf (only -inf and NaN) is resolved by a second
// scan for its first -inf (a row of NaN only gives 0).
__global__ __launch_bounds__(kArgThreads) void target_argmax_kernel(
    const uint16_t* __restrict__ logits, long long vocab, const int32_t* __restrict__ q_offsets,
    int R, int32_t* __restrict__ target) {
  __shared__ float s_val[kArgThreads / kWave];
  __shared__ uint32_t s_idx[kArgThreads / kWave];
  __shared__ uint32_t s_first_inf;
  const int s = blockIdx.x;
  const int nq = q_offsets[R];
  if (s >= nq) return;  // uniform over the workgroup
  const uint16_t* row = logits + size_t(s) * size_t(vocab);
  const int tid = threadIdx.x;
  float best = -__builtin_inff();
  uint32_t bidx = kNoIdx;
  auto take = [&](float v, uint32_t i) {
    if (v > best) {
      best = v;
      bidx = i;
    }
  };
  // scalar head up to 16-byte alignment, 8-value body, scalar tail
  const long long head =
      min<long long>(vocab, ((16 - (reinterpret_cast<uintptr_t>(row) & 15)) & 15) / 2);
  const long long nvec = (vocab - head) / 8;
  const long long tail0 = head + nvec * 8;
  // the head precedes the body in index order: its elements are taken first
  for (long long v = tid; v < head; v += kArgThreads)
    take(__uint_as_float(uint32_t(row[v]) << 16), uint32_t(v));
  const uint4* body = reinterpret_cast<const uint4*>(row + head);
  long long c = tid;
  for (; c + (kArgUnroll - 1) * kArgThreads < nvec; c += kArgUnroll * kArgThreads) {
    uint4 x[kArgUnroll];
#pragma unroll
    for (int u = 0; u < kArgUnroll; ++u) x[u] = body[c + u * kArgThreads];
#pragma unroll
    for (int u = 0; u < kArgUnroll; ++u) {
      const uint32_t v0 = uint32_t(head + (c + u * kArgThreads) * 8);
      take(bf16_lo(x[u].x), v0 + 0);
      take(bf16_hi(x[u].x), v0 + 1);
      take(bf16_lo(x[u].y), v0 + 2);
      take(bf16_hi(x[u].y), v0 + 3);
      take(bf16_lo(x[u].z), v0 + 4);
      take(bf16_hi(x[u].z), v0 + 5);
      take(bf16_lo(x[u].w), v0 + 6);
      take(bf16_hi(x[u].w), v0 + 7);
    }
  }
  for (; c < nvec; c += kArgThreads) {
    const uint4 x = body[c];
    const uint32_t v0 = uint32_t(head + c * 8);
    take(bf16_lo(x.x), v0 + 0);
    take(bf16_hi(x.x), v0 + 1);
    take(bf16_lo(x.y), v0 + 2);
    take(bf16_hi(x.y), v0 + 3);
    take(bf16_lo(x.z), v0 + 4);
    take(bf16_hi(x.z), v0 + 5);
    take(bf16_lo(x.w), v0 + 6);
    take(bf16_hi(x.w), v0 + 7);
  }
  // the tail follows every body element in index order
  for (long long v = tail0 + tid; v < vocab; v += kArgThreads)
    take(__uint_as_float(uint32_t(row[v]) << 16), uint32_t(v));
  // workgroup: largest value, ties (and -0 == +0) to the smaller index
  auto better = [](float va, uint32_t ia, float vb, uint32_t ib) {
    if (ib == kNoIdx) return false;
    if (ia == kNoIdx) return true;
    return vb > va || (vb == va && ib < ia);
  };
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(best, off, kWave);
    const uint32_t oi = uint32_t(__shfl_xor(int(bidx), off, kWave));
    if (better(best, bidx, ov, oi)) {
      best = ov;
      bidx = oi;
    }
  }
  if ((tid & (kWave - 1)) == 0) {
    s_val[tid / kWave] = best;
    s_idx[tid / kWave] = bidx;
  }
  if (tid == 0) s_first_inf = kNoIdx;
  __syncthreads();
  float bv = s_val[0];
  uint32_t bi = s_idx[0];
  for (int w = 1; w < kArgThreads / kWave; ++w)
    if (better(bv, bi, s_val[w], s_idx[w])) {
      bv = s_val[w];
      bi = s_idx[w];
    }
  if (bi == kNoIdx) {  // nothing above -inf: the first -inf, else 0
    for (long long v = tid; v < vocab; v += kArgThreads)
      if (row[v] == 0xFF80u) atomicMin(&s_first_inf, uint32_t(v));
    __syncthreads();
    bi = s_first_inf == kNoIdx ? 0u : s_first_inf;
  }
  if (tid == 0) target[s] = int32_t(bi);
}

__global__ __launch_bounds__(kCommitThreads) void commit_kv_kernel(
    const int32_t* __restrict__ q_offsets, const int32_t* __restrict__ accept_len,
    const int32_t* __restrict__ accept_slots, int max_depth, const uint16_t* __restrict__ k_new,
    const uint16_t* __restrict__ v_new, int max_rows, int hkv, uint16_t* __restrict__ k_pages,
    uint16_t* __restrict__ v_pages, long long num_pages, int page_size,
    const int32_t* __restrict__ block_table, int max_pages, int32_t* __restrict__ prefix_len,
    int32_t* status) {
  __shared__ int s_slot[ECHO_MAX_DEPTH + 1];
  __shared__ long long s_dst[ECHO_MAX_DEPTH + 1];  // destination row (page * page_size + offset)
  __shared__ int s_bad;
  const int r = blockIdx.x;
  const int tid = threadIdx.x;
  const int q0 = q_offsets[r], q1 = q_offsets[r + 1];
  const int L = accept_len[r];
  const int P = prefix_len[r];
  bool ok = true;
  int n = 0;
  if (q1 > q0) {  // a request without slots verified nothing and commits nothing
    ok = q0 >= 0 && q1 <= max_rows && L >= 0 && L <= max_depth && P >= 0;
    n = ok ? 1 + L : 0;
  }
  if (tid == 0) s_bad = ok ? 0 : 1;
  __syncthreads();
  // thread j resolves committed row j: its slot and its place in the pages
  if (tid < n) {
    const int j = tid;
    const int s = j == 0 ? q0 : accept_slots[size_t(r) * max_depth + (j - 1)];
    const long long pos = (long long)P + j;
    const long long e = pos / page_size;
    const int page = e < max_pages ? block_table[size_t(r) * max_pages + size_t(e)] : -1;
    if (s < 0 || s >= max_rows || page < 0 || page >= num_pages) atomicOr(&s_bad, 1);
    s_slot[j] = s;
    s_dst[j] = (long long)page * page_size + (pos % page_size);
  }
  __syncthreads();
  if (s_bad) n = 0;  // nothing of the request is written
  // each row is hkv * 128 bf16 = hkv * 16 chunks of 16 bytes, for K and for V
  const int chunks = hkv * (ECHO_HEAD_DIM * 2 / 16);
  for (int i = tid; i < n * chunks; i += kCommitThreads) {
    const int j = i / chunks, c = i % chunks;
    const size_t src = size_t(s_slot[j]) * size_t(chunks) + size_t(c);
    const size_t dst = size_t(s_dst[j]) * size_t(chunks) + size_t(c);
    reinterpret_cast<uint4*>(k_pages)[dst] = reinterpret_cast<const uint4*>(k_new)[src];
    reinterpret_cast<uint4*>(v_pages)[dst] = reinterpret_cast<const uint4*>(v_new)[src];
  }
  if (tid == 0) {
    if (s_bad) status_or(status, ECHO_DATA_BAD_OFFSETS);
    else if (n > 0) prefix_len[r] = P + n;
  }
}

}  // namespace

int32_t launch_accept_logits(const int32_t* q_offsets, const int32_t* slot_parent,
                             const int32_t* slot_token, const uint16_t* logits, int64_t vocab,
                             int32_t R, int32_t max_rows, int32_t max_depth, int32_t* target,
                             int32_t* accept_len, int32_t* accept_slots, int32_t* bonus_token,
                             int32_t* status, hipStream_t stream) {
  (void)hipGetLastError();
  if (max_rows > 0)
    hipLaunchKernelGGL(target_argmax_kernel, dim3(max_rows), dim3(kArgThreads), 0, stream,
                       logits, static_cast<long long>(vocab), q_offsets, R, target);
  if (hipGetLastError() != hipSuccess) return ECHO_ERR_HIP;
  return launch_accept(q_offsets, slot_parent, slot_token, target, R, max_rows, max_depth,
                       accept_len, accept_slots, bonus_token, status, stream);
}

int32_t launch_commit_kv(const int32_t* q_offsets, const int32_t* accept_len,
                         const int32_t* accept_slots, int32_t max_depth, const uint16_t* k_new,
                         const uint16_t* v_new, int32_t R, int32_t max_rows, int32_t hkv,
                         uint16_t* k_pages, uint16_t* v_pages, int64_t num_pages,
                         int32_t page_size, const int32_t* block_table, int32_t max_pages,
                         int32_t* prefix_len, int32_t* status, hipStream_t stream) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(commit_kv_kernel, dim3(R), dim3(kCommitThreads), 0, stream, q_offsets,
                     accept_len, accept_slots, max_depth, k_new, v_new, max_rows, hkv, k_pages,
                     v_pages, static_cast<long long>(num_pages), page_size, block_table,
                     max_pages, prefix_len, status);
  return hipGetLastError() == hipSuccess ? ECHO_OK : ECHO_ERR_HIP;
}

}  // namespace echo
