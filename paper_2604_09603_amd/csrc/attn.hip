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
constexpr int kMainWaves = 8;       // main kernel: waves per workgroup
constexpr int kMT = 2;              // 16-row tiles per wave per row pass
constexpr int kStages = 4;          // LDS ring depth (64-key K+V tiles)
constexpr int kCombineRows = 8;     // rows per combine workgroup
constexpr int kTileKeys = 64;       // keys staged in LDS per step
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
  int32_t* meta;     // [0] = number of items, [1] = number of combine groups
  Item* items;
  PairInfo* pairs;
  int2* cgroups;     // (pair, first row) of each combine workgroup
  float* part_ml;    // [rows][2]: running max (log2 units), sum
  float* part_o;     // [rows][128]
};

__host__ __device__ inline size_t al(size_t x) { return (x + 255) / 256 * 256; }

__host__ inline size_t item_capacity(int R, int hkv, int target_items) {
  return size_t(target_items) + size_t(R) * hkv;
}

__host__ inline size_t cgroup_capacity(int R, int max_rows, int hq, int hkv) {
  return (size_t(max_rows) * hq + kCombineRows - 1) / kCombineRows + size_t(R) * hkv;
}

__host__ __device__ inline AttnWs attn_layout(void* base, int R, int hkv, size_t item_cap,
                                              size_t cg_cap, size_t part_rows) {
  char* p = static_cast<char*>(base);
  AttnWs w;
  w.meta = reinterpret_cast<int32_t*>(p);
  p += 256;
  w.items = reinterpret_cast<Item*>(p);
  p += al(item_cap * sizeof(Item));
  w.pairs = reinterpret_cast<PairInfo*>(p);
  p += al(size_t(R) * hkv * sizeof(PairInfo));
  w.cgroups = reinterpret_cast<int2*>(p);
  p += al(cg_cap * sizeof(int2));
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

  // pairs in request-major order; scan their item counts, partial rows, combine groups
  int item_run = 0, row_run = 0, cg_run = 0;
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
    int tot_items, tot_rows, tot_cg;
    const int ncg = nparts > 0 ? (rows + kCombineRows - 1) / kCombineRows : 0;
    const int ib = item_run + block_exclusive_sum<kThreads>(nparts, s_scan, &tot_items);
    const int rb = row_run + block_exclusive_sum<kThreads>(nparts * rows, s_scan, &tot_rows);
    const int cb = cg_run + block_exclusive_sum<kThreads>(ncg, s_scan, &tot_cg);
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
      for (int c = 0; c < ncg; ++c) ws.cgroups[cb + c] = make_int2(pr, c * kCombineRows);
    }
    item_run += tot_items;
    row_run += tot_rows;
    cg_run += tot_cg;
  }
  if (tid == 0) {
    ws.meta[0] = item_run;
    ws.meta[1] = cg_run;
  }
}

// ---------------------------------------------------------------- main ----
// LDS tile layout: 64 key rows x 256 bytes per tensor, no padding.  The 16-byte
// chunk c of row r is stored at chunk position c ^ (r & 15), so that 16 rows
// read at the same logical column fall into 16 different bank groups.
typedef __attribute__((address_space(3))) void lds_void_t;
typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) shortx4 lds_shortx4_t;

constexpr int kTileBytes = kTileKeys * kD * 2;  // 16 KB per tensor
constexpr int kStageBytes = 2 * kTileBytes;     // K then V

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  __bf16 a = static_cast<__bf16>(lo);
  __bf16 b = static_cast<__bf16>(hi);
  return uint32_t(__builtin_bit_cast(uint16_t, a)) |
         (uint32_t(__builtin_bit_cast(uint16_t, b)) << 16);
}

__device__ __forceinline__ int swz(int row, int chunk) {
  return row * 256 + ((chunk ^ (row & 15)) << 4);
}

// Direct HBM -> LDS copy of one 64-key tile of K and V (each lane moves 16 bytes
// per instruction, 1 KB = 4 rows per wave instruction).  Rows >= tn re-read row
// tn-1 (in bounds); the softmax masks those keys.
template <int NW>
__device__ __forceinline__ void issue_tile(char* stage, const uint16_t* kbase,
                                           const uint16_t* vbase, size_t stride, int tn) {
  constexpr int kLoads = 32 / NW;
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = threadIdx.x / kWave;
#pragma unroll
  for (int j = 0; j < kLoads; ++j) {
    const int q = wid * kLoads + j;  // 0..31, uniform in the wave
    const int tensor = q >> 4;
    const int rg = q & 15;
    const int row = rg * 4 + (lane >> 4);
    const int c = (lane & 15) ^ (row & 15);
    const int srow = row < tn ? row : tn - 1;
    const uint16_t* src = (tensor ? vbase : kbase) + size_t(srow) * stride + c * 8;
    __builtin_amdgcn_global_load_lds(src, (lds_void_t*)(stage + tensor * kTileBytes + rg * 1024),
                                     16, 0, 0);
  }
}

template <int N>
__device__ __forceinline__ void wait_vm() {
  // gfx9 s_waitcnt encoding: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt_hi[15:14]
  constexpr int imm = (N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14);
  __builtin_amdgcn_s_waitcnt(imm);
}

struct RowTile {
  floatx4 o[8];  // O^T: lane holds dims 16*dt + 4*(lane/16) + i of row lane%16
  float m;       // running max of scaled logits (log2 units)
  float l;       // this lane's share of the running sum
};

// Per-lane LDS byte offsets of the swizzled fragment reads (lane constants; the
// subtile / key-block parts are compile-time immediates on top of these).
struct LaneOffsets {
  int k[4];  // K A-fragment of chunk 4*kk + lg, row lr of a 16-key subtile
  int v[8];  // V^T transposed read of dims 16*dt + 4*(lr&3), key 4*lg + (lr>>2) of a 16-key block
};

__device__ __forceinline__ LaneOffsets lane_offsets() {
  const int lane = threadIdx.x & (kWave - 1);
  const int lr = lane & 15, lg = lane >> 4;
  LaneOffsets o;
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) o.k[kk] = swz(lr, 4 * kk + lg);
  const int key = 4 * lg + (lr >> 2);
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) {
    const int d = 16 * dt + 4 * (lr & 3);
    o.v[dt] = swz(key, d >> 3) + ((d & 4) << 1);
  }
  return o;
}

// One 64-key tile from LDS against the wave's row tiles.
// masked: keys >= tn are invisible, and key j is visible to a row only if bit j
// (of this tile's 64) is set in its mask words.
template <int MT>
__device__ __forceinline__ void compute_tile(const char* kt, const char* vt, const bf16x8 (*qf)[4],
                                             RowTile* rt, int ntiles, bool masked, int tn,
                                             float scale2, const uint32_t (*mword)[2],
                                             const LaneOffsets& lo) {
  const int lane = threadIdx.x & (kWave - 1);
  const int lg = lane >> 4;
  // S^T = K Q^T for the 4 subtiles of 16 keys (subtile s4 = rows 16*s4.., +4096 bytes)
  floatx4 st[MT][4];
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4) {
    bf16x8 kf[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      kf[kk] = *reinterpret_cast<const bf16x8*>(kt + lo.k[kk] + 4096 * s4);
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      if (t >= ntiles) break;
      floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[kk], qf[t][kk], acc, 0, 0, 0);
      st[t][s4] = acc;
    }
  }
  // online softmax (base 2); lane holds keys 16*s4 + 4*lg + i of row lane%16
  bf16x8 pf[MT][2];
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    if (t >= ntiles) break;
    float sv[16];
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
      for (int i = 0; i < 4; ++i) sv[4 * s4 + i] = st[t][s4][i];
    if (masked) {
      // key >> 5 == s4 >> 1 because 4 * lg + i < 16
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = 16 * s4 + 4 * lg + i;
          const bool ok = key < tn && ((mword[t][s4 >> 1] >> (key & 31)) & 1u);
          sv[4 * s4 + i] = ok ? sv[4 * s4 + i] : -__builtin_inff();
        }
    }
    float mx = sv[0];
#pragma unroll
    for (int e = 1; e < 16; ++e) mx = fmaxf(mx, sv[e]);
    mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    const float mt = mx * scale2;  // -inf stays -inf
    const float m_new = fmaxf(rt[t].m, mt);
    if (__ballot(m_new > rt[t].m) != 0ull) {
      const float alpha = __builtin_amdgcn_exp2f(rt[t].m - m_new);  // 0 for -inf, 1 if unchanged
      rt[t].l *= alpha;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) rt[t].o[dt] *= alpha;
      rt[t].m = m_new;
    }
    const float neg_m = m_new == -__builtin_inff() ? 0.0f : -m_new;
    float psum = 0.0f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      sv[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[e], scale2, neg_m));
      psum += sv[e];
    }
    rt[t].l += psum;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      uint4 pk;
      pk.x = pack_bf16x2(sv[8 * h + 0], sv[8 * h + 1]);
      pk.y = pack_bf16x2(sv[8 * h + 2], sv[8 * h + 3]);
      pk.z = pack_bf16x2(sv[8 * h + 4], sv[8 * h + 5]);
      pk.w = pack_bf16x2(sv[8 * h + 6], sv[8 * h + 7]);
      pf[t][h] = as_bf16x8(pk);
    }
  }
  // O^T += V^T P^T.  V^T fragment via transposed LDS reads: input lane i of block lg
  // reads 4 dims of one key, output lane j gets dim j of 4 keys.
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      char* base = const_cast<char*>(vt) + lo.v[dt] + 8192 * h;  // keys 32h.. (+16 keys = 4096 B)
      const shortx4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4_t*)(base));
      const shortx4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4_t*)(base + 4096));
      const bf16x8 vf =
          __builtin_bit_cast(bf16x8, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        if (t >= ntiles) break;
        rt[t].o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[t][h], rt[t].o[dt], 0, 0, 0);
      }
    }
  }
}

template <int NW, int MT, int STAGES>
__global__ __launch_bounds__(NW * kWave) void attn_main_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_new,
    const uint16_t* __restrict__ v_new, const uint16_t* __restrict__ k_cache,
    const uint16_t* __restrict__ v_cache, const uint32_t* __restrict__ tree_mask, int W, int hq,
    int hkv, int G, float scale2, AttnWs ws) {
  __shared__ __attribute__((aligned(1024))) char s_ring[STAGES * kStageBytes];
  constexpr int kLoads = 32 / NW;
  constexpr int kRowsPerPass = NW * MT * 16;

  const int n_items = ws.meta[0];
  if (int(blockIdx.x) >= n_items) return;
  const Item it = ws.items[blockIdx.x];
  const PairInfo pi = ws.pairs[it.pair];
  const int kvh = it.pair % hkv;
  const bool last = (it.part >> 30) & 1;
  const int part = it.part & ((1 << 30) - 1);
  const int rows = pi.nslots * G;
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = threadIdx.x / kWave;
  const int lr = lane & 15, lg = lane >> 4;
  const size_t stride = size_t(hkv) * kD;
  const int ntk = (it.ke - it.kb + kTileKeys - 1) / kTileKeys;
  const uint16_t* kpre = k_cache + size_t(it.kb) * stride + kvh * kD;
  const uint16_t* vpre = v_cache + size_t(it.kb) * stride + kvh * kD;
  const LaneOffsets lo = lane_offsets();

  for (int pass = 0; pass * kRowsPerPass < rows; ++pass) {
    int ntiles = 0;
    bf16x8 qf[MT][4];
    RowTile rt[MT];
    int rho_t[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const int tile = pass * NW * MT + wid + NW * t;
      const int rho = tile * 16 + lr;
      rho_t[t] = rho;
      if (tile * 16 < rows) ntiles = t + 1;
      uint4 qv[4] = {make_uint4(0, 0, 0, 0), make_uint4(0, 0, 0, 0), make_uint4(0, 0, 0, 0),
                     make_uint4(0, 0, 0, 0)};
      if (rho < rows) {
        const uint16_t* qrow = q + (size_t(pi.q0 + rho / G) * hq + kvh * G + rho % G) * kD;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          qv[kk] = *reinterpret_cast<const uint4*>(qrow + 32 * kk + 8 * lg);
      }
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) qf[t][kk] = as_bf16x8(qv[kk]);
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) rt[t].o[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
      rt[t].m = -__builtin_inff();
      rt[t].l = 0.0f;
    }
    wait_vm<0>();  // Q (and earlier stores) done: vmcnt now counts tile copies only

    // The item's tiles: the prefix chunk through a STAGES-deep ring of LDS tiles,
    // then (last chunk only) the tree tail, one synchronous tile at a time.
    const int ntail = last ? (pi.nslots + kTileKeys - 1) / kTileKeys : 0;
    uint32_t mword[MT][2];
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
      if (s < ntk)
        issue_tile<NW>(s_ring + s * kStageBytes, kpre + size_t(s) * kTileKeys * stride,
                       vpre + size_t(s) * kTileKeys * stride, stride,
                       min(kTileKeys, it.ke - it.kb - s * kTileKeys));
    for (int i = 0; i < ntk + ntail; ++i) {
      const char* stg;
      int tn;
      if (i < ntk) {
        const int ahead = min(STAGES - 2, ntk - 1 - i);  // tiles issued after tile i
        if (ahead >= 2) wait_vm<2 * kLoads>();
        else if (ahead == 1) wait_vm<kLoads>();
        else wait_vm<0>();
        __syncthreads();
        const int nx = i + STAGES - 1;
        if (nx < ntk)
          issue_tile<NW>(s_ring + (nx % STAGES) * kStageBytes,
                         kpre + size_t(nx) * kTileKeys * stride,
                         vpre + size_t(nx) * kTileKeys * stride, stride,
                         min(kTileKeys, it.ke - it.kb - nx * kTileKeys));
        stg = s_ring + (i % STAGES) * kStageBytes;
        tn = min(kTileKeys, it.ke - it.kb - i * kTileKeys);
#pragma unroll
        for (int t = 0; t < MT; ++t) mword[t][0] = mword[t][1] = 0xFFFFFFFFu;
      } else {
        // tree tail: the request's own slots, visible through the ancestor bitmask
        const int j0 = (i - ntk) * kTileKeys;
        tn = min(kTileKeys, pi.nslots - j0);
        __syncthreads();  // every wave is done with the previous tile's stage
        issue_tile<NW>(s_ring, k_new + size_t(pi.q0 + j0) * stride + kvh * kD,
                       v_new + size_t(pi.q0 + j0) * stride + kvh * kD, stride, tn);
#pragma unroll
        for (int t = 0; t < MT; ++t) {
          mword[t][0] = 0u;
          mword[t][1] = 0u;
          if (rho_t[t] < rows) {
            const uint32_t* mrow = tree_mask + size_t(pi.q0 + rho_t[t] / G) * W;
            const int w0 = j0 >> 5;
            if (w0 < W) mword[t][0] = mrow[w0];
            if (w0 + 1 < W) mword[t][1] = mrow[w0 + 1];
          }
        }
        wait_vm<0>();
        __syncthreads();
        stg = s_ring;
      }
      if (ntiles > 0)
        compute_tile<MT>(stg, stg + kTileBytes, qf, rt, ntiles, tn < kTileKeys || i >= ntk, tn,
                         scale2, mword, lo);
    }
    __syncthreads();
    // partial results of this chunk
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      if (t >= ntiles) break;
      float l = rt[t].l;
      l += __shfl_xor(l, 16, kWave);
      l += __shfl_xor(l, 32, kWave);
      const int rho = rho_t[t];
      if (rho < rows) {
        const size_t prow = size_t(pi.part_base) + size_t(part) * rows + rho;
        float* po = ws.part_o + prow * kD;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt)
          *reinterpret_cast<floatx4*>(po + 16 * dt + 4 * lg) = rt[t].o[dt];
        if (lg == 0) {
          ws.part_ml[prow * 2 + 0] = rt[t].m;
          ws.part_ml[prow * 2 + 1] = l;
        }
      }
    }
  }
}

// ------------------------------------------------------------- combine ----
// One workgroup per group of 8 rows of one pair; thread = (row, 4 dims).  All
// chunk partials of a row are loaded independently, then merged in chunk order.
__global__ __launch_bounds__(kThreads) void attn_combine_kernel(int hq, int hkv, int G, AttnWs ws,
                                                                float* __restrict__ out,
                                                                float* __restrict__ lse) {
  if (int(blockIdx.x) >= ws.meta[1]) return;
  const int2 cg = ws.cgroups[blockIdx.x];
  const PairInfo pi = ws.pairs[cg.x];
  const int kvh = cg.x % hkv;
  const int rows = pi.nslots * G;
  const int rho = cg.y + (threadIdx.x >> 5);
  const int d4 = (threadIdx.x & 31) * 4;
  if (rho >= rows) return;
  float mv[kMaxParts], lv[kMaxParts];
  float M = -__builtin_inff();
#pragma unroll
  for (int i = 0; i < kMaxParts; ++i) {
    mv[i] = -__builtin_inff();
    lv[i] = 0.0f;
    if (i < pi.nparts) {
      const size_t prow = size_t(pi.part_base) + size_t(i) * rows + rho;
      const float2 ml = *reinterpret_cast<const float2*>(ws.part_ml + prow * 2);
      mv[i] = ml.x;
      lv[i] = ml.y;
      M = fmaxf(M, ml.x);
    }
  }
  const float Mu = M == -__builtin_inff() ? 0.0f : M;
  float L = 0.0f;
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < kMaxParts; ++i) {
    if (i < pi.nparts) {
      const size_t prow = size_t(pi.part_base) + size_t(i) * rows + rho;
      const float w = __builtin_amdgcn_exp2f(mv[i] - Mu);
      L += w * lv[i];
      const floatx4 v = *reinterpret_cast<const floatx4*>(ws.part_o + prow * kD + d4);
      acc += w * v;
    }
  }
  const int slot = pi.q0 + rho / G;
  const int head = kvh * G + rho % G;
  float* orow = out + (size_t(slot) * hq + head) * kD + d4;
  const float inv = L > 0.0f ? 1.0f / L : 0.0f;
  *reinterpret_cast<floatx4*>(orow) = acc * inv;
  if (lse != nullptr && d4 == 0)
    lse[size_t(slot) * hq + head] = L > 0.0f ? (M + log2f(L)) * kLn2 : -__builtin_inff();
}

int target_items_for_device() { return 8 * device_cu_count(); }

}  // namespace

size_t attn_workspace_bytes(int32_t R, int32_t max_rows, int32_t hq, int32_t hkv) {
  const size_t icap = item_capacity(R, hkv, target_items_for_device());
  const size_t cgcap = cgroup_capacity(R, max_rows, hq, hkv);
  const size_t part_rows = size_t(kMaxParts) * max_rows * hq;
  return 256 + al(icap * sizeof(Item)) + al(size_t(R) * hkv * sizeof(PairInfo)) +
         al(cgcap * sizeof(int2)) + al(part_rows * 2 * sizeof(float)) +
         al(part_rows * kD * sizeof(float));
}

int32_t launch_tree_verify_attn(const AttnArgs& a, hipStream_t stream) {
  const int target = target_items_for_device();
  const size_t icap = item_capacity(a.R, a.hkv, target);
  const size_t cgcap = cgroup_capacity(a.R, a.max_rows, a.hq, a.hkv);
  const size_t part_rows = size_t(kMaxParts) * a.max_rows * a.hq;
  AttnWs ws = attn_layout(a.workspace, a.R, a.hkv, icap, cgcap, part_rows);
  const int G = a.hq / a.hkv;
  hipLaunchKernelGGL(attn_plan_kernel, dim3(1), dim3(kThreads), 0, stream, a.q_offsets,
                     a.kv_offsets, static_cast<long long>(a.kv_rows), a.R, a.hkv, G, a.max_rows,
                     target, ws, a.status);
  const bool prof = g_attn_ev_start != nullptr && g_attn_ev_stop != nullptr;
  if (prof && hipEventRecord(g_attn_ev_start, stream) != hipSuccess) return ECHO_ERR_HIP;
  hipLaunchKernelGGL((attn_main_kernel<kMainWaves, kMT, kStages>), dim3(unsigned(icap)),
                     dim3(kMainWaves * kWave), 0, stream, a.q, a.k_new, a.v_new, a.k_cache,
                     a.v_cache, a.tree_mask, a.mask_words, a.hq, a.hkv, G, a.sm_scale * kLog2e, ws);
  if (prof && hipEventRecord(g_attn_ev_stop, stream) != hipSuccess) return ECHO_ERR_HIP;
  hipLaunchKernelGGL(attn_combine_kernel, dim3(unsigned(cgcap)), dim3(kCombineRows * 32), 0,
                     stream, a.hq, a.hkv, G, ws, a.out, a.lse);
  return hipGetLastError() == hipSuccess ? ECHO_OK : ECHO_ERR_HIP;
}

}  // namespace echo
