// Tree-masked grouped-query verification attention (one verification forward
// over the flattened super-tree).  Three launches:
//
//   attn_plan     one workgroup: per (request, kv head) pair, split the KV
//                 prefix into chunks so that the whole batch yields about
//                 `target_items` work items; write the item list and each
//                 pair's slice of the partial-result buffer.
//   attn_main     one workgroup (4 waves) per item.  The item's KV chunk is
//                 streamed HBM -> LDS once, 64 keys at a time, and shared by
//                 every row of the pair: rows are (slot, query head in the
//                 GQA group), slot-major, in 16-row MFMA tiles spread over
//                 the waves.  S^T = K Q^T and O^T = V^T P^T on
//                 v_mfma_f32_16x16x32_bf16 with fp32 accumulation; online
//                 softmax in base 2.  The last chunk of a pair also runs the
//                 tree tail: the new keys of the request's own slots, masked
//                 by the ancestor bitmask.  Output: unnormalised partial O,
//                 running max and sum per row.
//   attn_combine  one workgroup per pair: merge the chunk partials in chunk
//                 order (deterministic) into out and lse.
#include "echo_device.h"
#include "echo_internal.h"

namespace echo {
namespace {

constexpr int kD = ECHO_HEAD_DIM;   // 128
constexpr int kThreads = 256;       // plan / combine workgroups
constexpr int kWaves = kThreads / kWave;
constexpr int kMainWaves = 4;       // main kernel: waves per workgroup
constexpr int kMT = 2;              // 16-row tiles per wave per row pass
constexpr int kTileKeys = 64;       // keys staged in LDS per step
constexpr int kRowBytes = kD * 2 + 16;  // padded LDS row (bf16), breaks bank conflicts
constexpr int kRowHalfs = kRowBytes / 2;
constexpr int kMaxParts = 16;       // chunks per pair at most
constexpr int kChunkMin = 256;      // shortest chunk (keys)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

struct Item {
  int32_t pair;    // r * Hkv + kvh
  int32_t kb, ke;  // prefix rows [kb, ke) of the KV cache (token index)
  int32_t part;    // chunk index within the pair; bit 30 set: last chunk (runs the tree tail)
};

struct PairInfo {
  int32_t part_base;  // first partial row of this pair
  int32_t nparts;     // 0: request skipped
  int32_t q0;         // first slot of the request
  int32_t nslots;
};

struct AttnWs {
  int32_t* meta;     // [0] = number of items
  Item* items;
  PairInfo* pairs;
  float* part_ml;    // [rows][2]: running max (log2 units), sum
  float* part_o;     // [rows][128]
};

__host__ __device__ inline size_t al(size_t x) { return (x + 255) / 256 * 256; }

__host__ inline size_t item_capacity(int R, int hkv, int target_items) {
  return size_t(target_items) + size_t(R) * hkv;
}

__host__ __device__ inline AttnWs attn_layout(void* base, int R, int hkv, size_t item_cap,
                                              size_t part_rows) {
  char* p = static_cast<char*>(base);
  AttnWs w;
  w.meta = reinterpret_cast<int32_t*>(p);
  p += 256;
  w.items = reinterpret_cast<Item*>(p);
  p += al(item_cap * sizeof(Item));
  w.pairs = reinterpret_cast<PairInfo*>(p);
  p += al(size_t(R) * hkv * sizeof(PairInfo));
  w.part_ml = reinterpret_cast<float*>(p);
  p += al(part_rows * 2 * sizeof(float));
  w.part_o = reinterpret_cast<float*>(p);
  return w;
}

// ---------------------------------------------------------------- plan ----
__global__ __launch_bounds__(kThreads) void attn_plan_kernel(
    const int32_t* __restrict__ q_offsets, const int64_t* __restrict__ kv_offsets,
    long long kv_rows, int R, int hkv, int G, int max_rows, int target_items, AttnWs ws,
    int32_t* status) {
  __shared__ int s_scan[kThreads / kWave + 1];
  __shared__ long long s_total;
  const int tid = threadIdx.x;
  // total prefix keys over valid requests
  long long my = 0;
  int bits = 0;
  for (int r = tid; r < R; r += kThreads) {
    const int q0 = q_offsets[r], q1 = q_offsets[r + 1];
    const long long k0 = kv_offsets[r], k1 = kv_offsets[r + 1];
    const bool ok = q0 >= 0 && q1 >= q0 && q1 <= max_rows && k0 >= 0 && k1 >= k0 && k1 <= kv_rows;
    if (!ok) bits |= ECHO_DATA_BAD_OFFSETS;
    else if (q1 > q0) my += k1 - k0;
  }
  wave_status_or(status, bits);
  if (tid == 0) s_total = 0;
  __syncthreads();
  atomicAdd(reinterpret_cast<unsigned long long*>(&s_total), static_cast<unsigned long long>(my));
  __syncthreads();
  const long long total = s_total * hkv;
  long long ch = (total + target_items - 1) / target_items;
  ch = (ch + kTileKeys - 1) / kTileKeys * kTileKeys;
  if (ch < kChunkMin) ch = kChunkMin;

  // pairs in request-major order; scan their item counts and partial rows
  int item_run = 0, row_run = 0;
  const int npairs = R * hkv;
  for (int base = 0; base < npairs; base += kThreads) {
    const int pr = base + tid;
    int nparts = 0, rows = 0, q0 = 0, nsl = 0;
    long long k0 = 0, len = 0, chr = ch;
    if (pr < npairs) {
      const int r = pr / hkv;
      q0 = q_offsets[r];
      const int q1 = q_offsets[r + 1];
      k0 = kv_offsets[r];
      const long long k1 = kv_offsets[r + 1];
      const bool ok =
          q0 >= 0 && q1 >= q0 && q1 <= max_rows && k0 >= 0 && k1 >= k0 && k1 <= kv_rows;
      if (ok && q1 > q0) {
        nsl = q1 - q0;
        rows = nsl * G;
        len = k1 - k0;
        long long np = (len + ch - 1) / ch;
        if (np < 1) np = 1;
        if (np > kMaxParts) {
          np = kMaxParts;
          chr = (len + kMaxParts - 1) / kMaxParts;
          chr = (chr + kTileKeys - 1) / kTileKeys * kTileKeys;
          np = (len + chr - 1) / chr;
        }
        nparts = int(np);
      }
    }
    int tot_items, tot_rows;
    const int ib = item_run + block_exclusive_sum<kThreads>(nparts, s_scan, &tot_items);
    const int rb = row_run + block_exclusive_sum<kThreads>(nparts * rows, s_scan, &tot_rows);
    if (pr < npairs) {
      PairInfo pi;
      pi.part_base = rb;
      pi.nparts = nparts;
      pi.q0 = q0;
      pi.nslots = nsl;
      ws.pairs[pr] = pi;
      for (int i = 0; i < nparts; ++i) {
        Item it;
        it.pair = pr;
        long long b = k0 + i * chr;
        long long e = b + chr;
        if (e > k0 + len) e = k0 + len;
        it.kb = int(b);
        it.ke = int(e);
        it.part = i | (i == nparts - 1 ? (1 << 30) : 0);
        ws.items[ib + i] = it;
      }
    }
    item_run += tot_items;
    row_run += tot_rows;
  }
  if (tid == 0) ws.meta[0] = item_run;
}

// ---------------------------------------------------------------- main ----
__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  __bf16 a = static_cast<__bf16>(lo);
  __bf16 b = static_cast<__bf16>(hi);
  return uint32_t(__builtin_bit_cast(uint16_t, a)) | (uint32_t(__builtin_bit_cast(uint16_t, b)) << 16);
}

// Stage keys [t0, t0 + kTileKeys) of one (K, V) source into LDS; rows >= tn are zero.
// src row i lives at base + i * stride (bf16 elements).
template <int NT>
__device__ __forceinline__ void stage_tile(uint16_t* s_k, uint16_t* s_v, const uint16_t* kbase,
                                           const uint16_t* vbase, size_t stride, int tn) {
  // 64 rows x 256 bytes = 1024 16-byte pieces per tensor
#pragma unroll
  for (int it = 0; it < 1024 / NT; ++it) {
    const int piece = it * NT + threadIdx.x;
    const int row = piece >> 4;
    const int col = (piece & 15) * 8;
    uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
    if (row < tn) {
      kv = *reinterpret_cast<const uint4*>(kbase + size_t(row) * stride + col);
      vv = *reinterpret_cast<const uint4*>(vbase + size_t(row) * stride + col);
    }
    *reinterpret_cast<uint4*>(s_k + row * kRowHalfs + col) = kv;
    *reinterpret_cast<uint4*>(s_v + row * kRowHalfs + col) = vv;
  }
}

struct TileState {
  floatx4 o[8];   // O^T: lane holds dims 16*dt + 4*(lane/16) + i of row lane%16
  float m;        // running max, log2 units
  float l;        // this lane's share of the running sum
};

// One 64-key LDS tile against the wave's row tiles.
// valid_keys: keys [0, valid_keys) of the tile exist.  mask_word(t, h): for the
// tree tail, the 32-bit visibility word of this lane's row for keys [32h, 32h+32)
// of the tile (all ones for the prefix).
template <int MT, bool kTail>
__device__ __forceinline__ void process_tile(const uint16_t* s_k, const uint16_t* s_v,
                                             const bf16x8 (*qf)[4], TileState* ts, int ntiles,
                                             int valid_keys, float scale2,
                                             const uint32_t (*mword)[2]) {
  const int lane = threadIdx.x & (kWave - 1);
  const int lr = lane & 15;  // row within a tile (S^T column) / key within a subtile (A row)
  const int lg = lane >> 4;  // k-group
#pragma unroll 1
  for (int h = 0; h < 2; ++h) {
    // K fragments of the two 16-key subtiles of this 32-key block
    bf16x8 kf[2][4];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const uint16_t* krow = s_k + (32 * h + 16 * st + lr) * kRowHalfs;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        kf[st][kk] = as_bf16x8(*reinterpret_cast<const uint4*>(krow + 32 * kk + 8 * lg));
    }
    bf16x8 pf[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      if (t >= ntiles) break;
      floatx4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[0][kk], qf[t][kk], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[1][kk], qf[t][kk], s1, 0, 0, 0);
      }
      // lane holds keys 32h + 4lg + i (s0) and 32h + 16 + 4lg + i (s1) of row lr
      float sv[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int k0 = 32 * h + 4 * lg + i;
        const int k1 = k0 + 16;
        bool v0 = k0 < valid_keys, v1 = k1 < valid_keys;
        if (kTail) {
          v0 = v0 && ((mword[t][h] >> (4 * lg + i)) & 1u);
          v1 = v1 && ((mword[t][h] >> (16 + 4 * lg + i)) & 1u);
        }
        sv[i] = v0 ? s0[i] * scale2 : -__builtin_inff();
        sv[4 + i] = v1 ? s1[i] * scale2 : -__builtin_inff();
      }
      float mx = sv[0];
#pragma unroll
      for (int e = 1; e < 8; ++e) mx = fmaxf(mx, sv[e]);
      mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
      mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
      const float m_new = fmaxf(ts[t].m, mx);
      const float m_use = m_new == -__builtin_inff() ? 0.0f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(ts[t].m - m_use);
      float psum = 0.0f;
      float p[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p[e] = __builtin_amdgcn_exp2f(sv[e] - m_use);
        psum += p[e];
      }
      ts[t].l = ts[t].l * alpha + psum;
      ts[t].m = m_new;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) ts[t].o[dt] *= alpha;
      uint4 pk;
      pk.x = pack_bf16x2(p[0], p[1]);
      pk.y = pack_bf16x2(p[2], p[3]);
      pk.z = pack_bf16x2(p[4], p[5]);
      pk.w = pack_bf16x2(p[6], p[7]);
      pf[t] = as_bf16x8(pk);
    }
    // O^T += V^T P^T; V^T fragment: dim 16dt + lr, keys 32h + {4lg..4lg+3, 16+4lg..16+4lg+3}
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      const uint16_t* vcol = s_v + 16 * dt + lr;
      uint16_t e[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        e[i] = vcol[(32 * h + 4 * lg + i) * kRowHalfs];
        e[4 + i] = vcol[(32 * h + 16 + 4 * lg + i) * kRowHalfs];
      }
      uint4 vv;
      vv.x = uint32_t(e[0]) | (uint32_t(e[1]) << 16);
      vv.y = uint32_t(e[2]) | (uint32_t(e[3]) << 16);
      vv.z = uint32_t(e[4]) | (uint32_t(e[5]) << 16);
      vv.w = uint32_t(e[6]) | (uint32_t(e[7]) << 16);
      const bf16x8 vf = as_bf16x8(vv);
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        if (t >= ntiles) break;
        ts[t].o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[t], ts[t].o[dt], 0, 0, 0);
      }
    }
  }
}

template <int NW, int MT>
__global__ __launch_bounds__(NW * kWave) void attn_main_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_new,
    const uint16_t* __restrict__ v_new, const uint16_t* __restrict__ k_cache,
    const uint16_t* __restrict__ v_cache, const uint32_t* __restrict__ tree_mask, int W, int hq,
    int hkv, int G, float scale2, AttnWs ws) {
  __shared__ __attribute__((aligned(16))) uint16_t s_k[kTileKeys * kRowHalfs];
  __shared__ __attribute__((aligned(16))) uint16_t s_v[kTileKeys * kRowHalfs];

  const int n_items = ws.meta[0];
  const int item_id = blockIdx.x;
  if (item_id >= n_items) return;
  const Item it = ws.items[item_id];
  const PairInfo pi = ws.pairs[it.pair];
  const int kvh = it.pair % hkv;
  const bool last = (it.part >> 30) & 1;
  const int part = it.part & ((1 << 30) - 1);
  const int rows = pi.nslots * G;
  constexpr int NT = NW * kWave;
  constexpr int kRowsPerPass = NW * MT * 16;
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = threadIdx.x / kWave;
  const int lr = lane & 15, lg = lane >> 4;
  const size_t kv_stride = size_t(hkv) * kD;

  for (int pass = 0; pass * kRowsPerPass < rows; ++pass) {
    // row tiles of this wave: pass * NW * MT + wid + NW * t
    int ntiles = 0;
    bf16x8 qf[MT][4];
    TileState ts[MT];
    uint32_t mword[MT][2];
    int row_of_lane[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const int tile = pass * NW * MT + wid + NW * t;
      const int rho = tile * 16 + lr;
      row_of_lane[t] = rho;
      if (tile * 16 < rows) ntiles = t + 1;
      uint4 z = make_uint4(0, 0, 0, 0);
      uint4 qv[4] = {z, z, z, z};
      if (rho < rows) {
        const int slot = pi.q0 + rho / G;
        const int head = kvh * G + rho % G;
        const uint16_t* qrow = q + (size_t(slot) * hq + head) * kD;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          qv[kk] = *reinterpret_cast<const uint4*>(qrow + 32 * kk + 8 * lg);
      }
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) qf[t][kk] = as_bf16x8(qv[kk]);
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) ts[t].o[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
      ts[t].m = -__builtin_inff();
      ts[t].l = 0.0f;
    }

    // prefix chunk
    for (int t0 = it.kb; t0 < it.ke; t0 += kTileKeys) {
      const int tn = min(kTileKeys, it.ke - t0);
      stage_tile<NT>(s_k, s_v, k_cache + size_t(t0) * kv_stride + kvh * kD,
                     v_cache + size_t(t0) * kv_stride + kvh * kD, kv_stride, tn);
      __syncthreads();
      if (ntiles > 0) process_tile<MT, false>(s_k, s_v, qf, ts, ntiles, tn, scale2, nullptr);
      __syncthreads();
    }
    // tree tail: the request's own slots, visible through the ancestor bitmask
    if (last) {
      for (int j0 = 0; j0 < pi.nslots; j0 += kTileKeys) {
        const int tn = min(kTileKeys, pi.nslots - j0);
        stage_tile<NT>(s_k, s_v, k_new + size_t(pi.q0 + j0) * kv_stride + kvh * kD,
                       v_new + size_t(pi.q0 + j0) * kv_stride + kvh * kD, kv_stride, tn);
#pragma unroll
        for (int t = 0; t < MT; ++t) {
          mword[t][0] = 0u;
          mword[t][1] = 0u;
          const int rho = row_of_lane[t];
          if (rho < rows) {
            const uint32_t* mrow = tree_mask + size_t(pi.q0 + rho / G) * W;
            const int w0 = j0 >> 5;
            if (w0 < W) mword[t][0] = mrow[w0];
            if (w0 + 1 < W) mword[t][1] = mrow[w0 + 1];
          }
        }
        __syncthreads();
        if (ntiles > 0) process_tile<MT, true>(s_k, s_v, qf, ts, ntiles, tn, scale2, mword);
        __syncthreads();
      }
    }
    // partial results
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      if (t >= ntiles) break;
      float l = ts[t].l;
      l += __shfl_xor(l, 16, kWave);
      l += __shfl_xor(l, 32, kWave);
      const int rho = row_of_lane[t];
      if (rho < rows) {
        const size_t prow = size_t(pi.part_base) + size_t(part) * rows + rho;
        float* po = ws.part_o + prow * kD;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt)
          *reinterpret_cast<floatx4*>(po + 16 * dt + 4 * lg) = ts[t].o[dt];
        if (lg == 0) {
          ws.part_ml[prow * 2 + 0] = ts[t].m;
          ws.part_ml[prow * 2 + 1] = l;
        }
      }
    }
  }
}

// ------------------------------------------------------------- combine ----
__global__ __launch_bounds__(kThreads) void attn_combine_kernel(int hq, int hkv, int G, AttnWs ws,
                                                                float* __restrict__ out,
                                                                float* __restrict__ lse) {
  const int pr = blockIdx.x;
  const PairInfo pi = ws.pairs[pr];
  if (pi.nparts == 0) return;
  const int kvh = pr % hkv;
  const int rows = pi.nslots * G;
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = threadIdx.x / kWave;
  for (int rho = wid; rho < rows; rho += kWaves) {
    float M = -__builtin_inff();
    for (int i = 0; i < pi.nparts; ++i) {
      const size_t prow = size_t(pi.part_base) + size_t(i) * rows + rho;
      M = fmaxf(M, ws.part_ml[prow * 2]);
    }
    const float Mu = M == -__builtin_inff() ? 0.0f : M;
    float L = 0.0f, o0 = 0.0f, o1 = 0.0f;
    for (int i = 0; i < pi.nparts; ++i) {
      const size_t prow = size_t(pi.part_base) + size_t(i) * rows + rho;
      const float w = __builtin_amdgcn_exp2f(ws.part_ml[prow * 2] - Mu);
      L += w * ws.part_ml[prow * 2 + 1];
      const float2 v = *reinterpret_cast<const float2*>(ws.part_o + prow * kD + 2 * lane);
      o0 += w * v.x;
      o1 += w * v.y;
    }
    const int slot = pi.q0 + rho / G;
    const int head = kvh * G + rho % G;
    float* orow = out + (size_t(slot) * hq + head) * kD;
    float2 res;
    if (L > 0.0f) {
      const float inv = 1.0f / L;
      res = make_float2(o0 * inv, o1 * inv);
    } else {
      res = make_float2(0.0f, 0.0f);
    }
    *reinterpret_cast<float2*>(orow + 2 * lane) = res;
    if (lse != nullptr && lane == 0)
      lse[size_t(slot) * hq + head] = L > 0.0f ? (M + log2f(L)) * kLn2 : -__builtin_inff();
  }
}

int target_items_for_device() { return 8 * device_cu_count(); }

}  // namespace

size_t attn_workspace_bytes(int32_t R, int32_t max_rows, int32_t hq, int32_t hkv) {
  const size_t icap = item_capacity(R, hkv, target_items_for_device());
  const size_t part_rows = size_t(kMaxParts) * max_rows * hq;
  return 256 + al(icap * sizeof(Item)) + al(size_t(R) * hkv * sizeof(PairInfo)) +
         al(part_rows * 2 * sizeof(float)) + al(part_rows * kD * sizeof(float));
}

int32_t launch_tree_verify_attn(const AttnArgs& a, hipStream_t stream) {
  const int target = target_items_for_device();
  const size_t icap = item_capacity(a.R, a.hkv, target);
  const size_t part_rows = size_t(kMaxParts) * a.max_rows * a.hq;
  AttnWs ws = attn_layout(a.workspace, a.R, a.hkv, icap, part_rows);
  const int G = a.hq / a.hkv;
  if (a.R == 0) return ECHO_OK;
  hipLaunchKernelGGL(attn_plan_kernel, dim3(1), dim3(kThreads), 0, stream, a.q_offsets,
                     a.kv_offsets, static_cast<long long>(a.kv_rows), a.R, a.hkv, G, a.max_rows,
                     target, ws, a.status);
  const bool prof = g_attn_ev_start != nullptr && g_attn_ev_stop != nullptr;
  if (prof && hipEventRecord(g_attn_ev_start, stream) != hipSuccess) return ECHO_ERR_HIP;
  hipLaunchKernelGGL((attn_main_kernel<kMainWaves, kMT>), dim3(unsigned(icap)),
                     dim3(kMainWaves * kWave), 0, stream, a.q,
                     a.k_new, a.v_new, a.k_cache, a.v_cache, a.tree_mask, a.mask_words, a.hq,
                     a.hkv, G, a.sm_scale * kLog2e, ws);
  if (prof && hipEventRecord(g_attn_ev_stop, stream) != hipSuccess) return ECHO_ERR_HIP;
  hipLaunchKernelGGL(attn_combine_kernel, dim3(unsigned(a.R * a.hkv)), dim3(kThreads), 0, stream,
                     a.hq, a.hkv, G, ws, a.out, a.lse);
  return hipGetLastError() == hipSuccess ? ECHO_OK : ECHO_ERR_HIP;
}

}  // namespace echo
