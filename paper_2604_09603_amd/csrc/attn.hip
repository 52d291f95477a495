// Tree-masked grouped-query verification attention (one verification forward
// over the flattened super-tree).  Three launches:
//
//   attn_plan     one workgroup.  The work is a stream of 32-key tiles: for each
//                 (request, kv head) pair and each 128-row pass over its rows
//                 (rows = verify slots x query heads of the GQA group), first
//                 the tree-tail tiles (the new keys of the request's own slots)
//                 and then the KV-prefix tiles.  The stream is cut into equal
//                 contiguous ranges, one per workgroup of the main kernel; the
//                 plan records each unit's tiles and which units are cut.
//   attn_main     persistent, two workgroups (4 waves each) per CU.  Each
//                 workgroup streams its range HBM -> LDS through a 4-stage
//                 ring of direct-to-LDS copies that runs across unit
//                 boundaries; every tile is shared by all rows of its unit.
//                 S^T = K Q^T and O^T = V^T P^T on v_mfma_f32_16x16x32_bf16
//                 (fp32 accumulation), online softmax in base 2, ancestor
//                 bitmask on tree-tail tiles.  A unit that lies inside one
//                 range is normalised and written to out/lse directly; a cut
//                 unit leaves one partial (O, max, sum) per workgroup.
//   attn_combine  one workgroup per cut unit: merges its partials in range
//                 order (deterministic) into out and lse.
#include "echo_device.h"
#include "echo_internal.h"

namespace echo {
namespace {

constexpr int kD = ECHO_HEAD_DIM;   // 128
constexpr int kThreads = 256;       // plan / combine workgroups
constexpr int kMainWaves = 4;       // main kernel: waves per workgroup (two workgroups per CU)
constexpr int kMT = 2;              // 16-row tiles per wave
constexpr int kPassRows = kMainWaves * kMT * 16;  // rows per unit (128)
constexpr int kStages = 4;          // LDS ring depth (32-key K+V tiles, 16 KB each)
constexpr int kTileKeys = 32;       // keys per tile
constexpr int kMaskWords = 4;       // tree-tail mask words preloaded per unit (128 slots)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// One unit of the tile stream: a row pass of one (request, kv head) pair.
struct Unit {
  int32_t tile_start, tile_end;  // global tile range: ntail tail tiles, then prefix tiles
  int32_t q0, nslots;            // the request's verify slots
  int32_t row0, rows;            // rows [row0, row0 + rows) of the pair (slot-major, G per slot)
  int32_t kb, P;                 // KV prefix rows [kb, kb + P)
  int32_t kvh, ntail;            // kv head; ceil(nslots / 32)
  int32_t cut, pad;              // cut: covered by more than one workgroup
};

struct Cut {
  int32_t unit, b0, b1, first_slot;  // workgroups b0..b1; partial slot of b0's segment
};

struct AttnWs {
  int32_t* meta;   // [0] = units, [1] = tiles, [2] = cut units
  Unit* units;
  int32_t* wg_unit;  // [nb] unit holding each workgroup's first tile
  Cut* cuts;
  float* part_ml;  // [2 * nb * 128][2]: running max (log2 units), sum
  float* part_o;   // [2 * nb * 128][128]
};

__host__ __device__ inline size_t al(size_t x) { return (x + 255) / 256 * 256; }

__host__ inline size_t unit_capacity(int R, int max_rows, int hq, int hkv) {
  return size_t(R) * hkv + (size_t(max_rows) * hq + kPassRows - 1) / kPassRows;
}

__host__ __device__ inline AttnWs attn_layout(void* base, size_t ucap, int nb) {
  char* p = static_cast<char*>(base);
  AttnWs w;
  w.meta = reinterpret_cast<int32_t*>(p);
  p += 256;
  w.units = reinterpret_cast<Unit*>(p);
  p += al(ucap * sizeof(Unit));
  w.wg_unit = reinterpret_cast<int32_t*>(p);
  p += al(size_t(nb) * sizeof(int32_t));
  w.cuts = reinterpret_cast<Cut*>(p);
  p += al(size_t(nb) * sizeof(Cut));
  w.part_ml = reinterpret_cast<float*>(p);
  p += al(size_t(2) * nb * kPassRows * 2 * sizeof(float));
  w.part_o = reinterpret_cast<float*>(p);
  return w;
}

__host__ inline size_t attn_ws_total(size_t ucap, int nb) {
  return 256 + al(ucap * sizeof(Unit)) + al(size_t(nb) * 4) + al(size_t(nb) * sizeof(Cut)) +
         al(size_t(2) * nb * kPassRows * 2 * 4) + al(size_t(2) * nb * kPassRows * kD * 4);
}

// First tile of workgroup b when T tiles are cut into nb equal ranges.
__device__ __forceinline__ long long range_lo(long long T, int b, int nb) { return T * b / nb; }
// Workgroup whose range holds tile t.
__device__ __forceinline__ int range_of(long long t, long long T, int nb) {
  return int(((t + 1) * nb + T - 1) / T) - 1;
}

// ---------------------------------------------------------------- plan ----
__device__ __forceinline__ bool pair_ok(const int32_t* q_offsets, const int64_t* kv_offsets,
                                        long long kv_rows, int max_rows, int r) {
  const int q0 = q_offsets[r], q1 = q_offsets[r + 1];
  const long long k0 = kv_offsets[r], k1 = kv_offsets[r + 1];
  return q0 >= 0 && q1 >= q0 && q1 <= max_rows && k0 >= 0 && k1 >= k0 && k1 <= kv_rows;
}

__global__ __launch_bounds__(kThreads) void attn_plan_kernel(
    const int32_t* __restrict__ q_offsets, const int64_t* __restrict__ kv_offsets,
    long long kv_rows, int R, int hkv, int G, int max_rows, int nb, AttnWs ws, int32_t* status) {
  __shared__ int s_scan[kThreads / kWave + 1];
  const int tid = threadIdx.x;
  const int npairs = R * hkv;
  int bits = 0;
  for (int r = tid; r < R; r += kThreads)
    if (!pair_ok(q_offsets, kv_offsets, kv_rows, max_rows, r)) bits |= ECHO_DATA_BAD_OFFSETS;
  wave_status_or(status, bits);

  // pass A: total tiles
  long long T = 0;
  for (int base = 0; base < npairs; base += kThreads) {
    const int pr = base + tid;
    int tiles = 0;
    if (pr < npairs) {
      const int r = pr / hkv;
      if (pair_ok(q_offsets, kv_offsets, kv_rows, max_rows, r)) {
        const int nsl = q_offsets[r + 1] - q_offsets[r];
        const long long P = kv_offsets[r + 1] - kv_offsets[r];
        const int passes = (nsl * G + kPassRows - 1) / kPassRows;
        tiles = passes * ((nsl + kTileKeys - 1) / kTileKeys + int((P + kTileKeys - 1) / kTileKeys));
      }
    }
    int tot;
    block_exclusive_sum<kThreads>(tiles, s_scan, &tot);
    T += tot;
  }
  // pass B: units, the cut units and each workgroup's first unit
  int unit_run = 0, tile_run = 0, cut_run = 0;
  for (int base = 0; base < npairs; base += kThreads) {
    const int pr = base + tid;
    int passes = 0, per_pass = 0, nsl = 0, q0 = 0, ntail = 0, P = 0, kb = 0;
    if (pr < npairs) {
      const int r = pr / hkv;
      if (pair_ok(q_offsets, kv_offsets, kv_rows, max_rows, r)) {
        q0 = q_offsets[r];
        nsl = q_offsets[r + 1] - q0;
        kb = int(kv_offsets[r]);
        P = int(kv_offsets[r + 1] - kv_offsets[r]);
        passes = (nsl * G + kPassRows - 1) / kPassRows;
        ntail = (nsl + kTileKeys - 1) / kTileKeys;
        per_pass = ntail + (P + kTileKeys - 1) / kTileKeys;
      }
    }
    int tot_u, tot_t;
    const int ub = unit_run + block_exclusive_sum<kThreads>(passes, s_scan, &tot_u);
    const int tb = tile_run + block_exclusive_sum<kThreads>(passes * per_pass, s_scan, &tot_t);
    // a unit is cut if two workgroup ranges share it
    int ncut = 0;
    for (int p = 0; p < passes; ++p) {
      const long long ts = tb + p * per_pass, te = ts + per_pass;
      if (range_of(ts, T, nb) != range_of(te - 1, T, nb)) ++ncut;
    }
    int tot_c;
    const int cb = cut_run + block_exclusive_sum<kThreads>(ncut, s_scan, &tot_c);
    int c = cb;
    for (int p = 0; p < passes; ++p) {
      Unit u;
      u.tile_start = tb + p * per_pass;
      u.tile_end = u.tile_start + per_pass;
      u.q0 = q0;
      u.nslots = nsl;
      u.row0 = p * kPassRows;
      u.rows = min(kPassRows, nsl * G - p * kPassRows);
      u.kb = kb;
      u.P = P;
      u.kvh = pr % hkv;
      u.ntail = ntail;
      const int b0 = range_of(u.tile_start, T, nb), b1 = range_of(u.tile_end - 1, T, nb);
      u.cut = b0 != b1;
      u.pad = 0;
      ws.units[ub + p] = u;
      if (u.cut) {
        Cut cu;
        cu.unit = ub + p;
        cu.b0 = b0;
        cu.b1 = b1;
        cu.first_slot = range_lo(T, b0, nb) < u.tile_start ? 1 : 0;
        ws.cuts[c++] = cu;
      }
      // workgroups whose range starts inside this unit
      int b = b0;
      if (range_lo(T, b, nb) < u.tile_start) ++b;
      for (; b <= b1; ++b) ws.wg_unit[b] = ub + p;
    }
    unit_run += tot_u;
    tile_run += tot_t;
    cut_run += tot_c;
  }
  if (tid == 0) {
    ws.meta[0] = unit_run;
    ws.meta[1] = int(T);
    ws.meta[2] = cut_run;
  }
}

// ---------------------------------------------------------------- main ----
// LDS tile layout: 32 key rows x 256 bytes per tensor, no padding.  The 16-byte
// chunk c of row r is stored at chunk position c ^ (r & 15), so that 16 rows
// read at the same logical column fall into 16 different bank groups.
typedef __attribute__((address_space(3))) void lds_void_t;
typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) shortx4 lds_shortx4_t;

constexpr int kTileBytes = kTileKeys * kD * 2;  // 8 KB per tensor
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

// One direct HBM -> LDS copy instruction: every lane moves 16 bytes from its
// global address to lds_base + 16 * lane.  Issued through inline assembly so
// that the compiler does not track it: its own bookkeeping would otherwise
// drain every copy in flight before each LDS read.  Completion is awaited
// explicitly (vmcnt) before a barrier in front of the reads.
__device__ __forceinline__ void dma16(const void* src, const char* lds_dst) {
  // the LDS destination is uniform in the wave; make that explicit for the SGPR operand
  const uint32_t lds = __builtin_amdgcn_readfirstlane(
      uint32_t(reinterpret_cast<uintptr_t>((const lds_void_t*)lds_dst)));
  uint32_t saved;  // M0 belongs to the compiler: restore it
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %2, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds), "v"(src)
      : "memory");
}

// Direct HBM -> LDS copy of one 32-key tile of K and V: 16 wave instructions of
// 1 KB (4 rows; each lane moves 16 bytes).  Rows >= tn re-read row tn-1 (in
// bounds); the softmax masks those keys.
template <int NW>
__device__ __forceinline__ void issue_tile(char* stage, const uint16_t* kbase,
                                           const uint16_t* vbase, size_t stride, int tn) {
  constexpr int kLoads = 16 / NW;
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = threadIdx.x / kWave;
#pragma unroll
  for (int j = 0; j < kLoads; ++j) {
    const int q = wid * kLoads + j;  // 0..15, uniform in the wave
    const int tensor = q >> 3;
    const int rg = q & 7;
    const int row = rg * 4 + (lane >> 4);
    const int c = (lane & 15) ^ (row & 15);
    const int srow = row < tn ? row : tn - 1;
    const uint16_t* src = (tensor ? vbase : kbase) + size_t(srow) * stride + c * 8;
    dma16(src, stage + tensor * kTileBytes + rg * 1024);
  }
}

template <int N>
__device__ __forceinline__ void wait_vm() {
  // gfx9 s_waitcnt encoding: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt_hi[15:14]
  constexpr int imm = (N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14);
  __builtin_amdgcn_s_waitcnt(imm);
}

// Wait until at most n * L vector-memory operations of this wave are in flight.
template <int L>
__device__ __forceinline__ void wait_vm_tiles(int n) {
  if (n >= 3) wait_vm<3 * L>();
  else if (n == 2) wait_vm<2 * L>();
  else if (n == 1) wait_vm<L>();
  else wait_vm<0>();
}

struct RowTile {
  floatx4 o[8];  // O^T: lane holds dims 16*dt + 4*(lane/16) + i of row lane%16
  float m;       // running max of scaled logits (log2 units)
  float l;       // this lane's share of the running sum
};

// Per-lane LDS byte offsets of the swizzled fragment reads (lane constants; the
// second 16-key subtile is +4096 bytes on top of these).
struct LaneOffsets {
  int k[4];  // K A-fragment: chunk 4*kk + lg of row lr
  int v[8];  // V^T transposed read: dims 16*dt + 4*(lr&3) of key 4*lg + (lr>>2)
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

// Reductions over the four lanes that hold one row (lanes l, l^16, l^32, l^48)
// with the gfx950 row/half swaps instead of LDS permutes.
__device__ __forceinline__ float row_max4(float v) {
  const uint32_t u = __float_as_uint(v);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const uint32_t w = __float_as_uint(v);
  const auto b = __builtin_amdgcn_permlane32_swap(w, w, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float row_sum4(float v) {
  const uint32_t u = __float_as_uint(v);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const uint32_t w = __float_as_uint(v);
  const auto b = __builtin_amdgcn_permlane32_swap(w, w, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// One 32-key tile from LDS against the wave's first NT row tiles.  masked: keys
// >= tn are invisible, and key j is visible to a row only if bit j of its mask
// word is set.  All LDS reads are issued up front and the independent MFMA
// chains are interleaved, so LDS and MFMA latencies overlap.
template <int NT>
__device__ __forceinline__ void compute_tile(const char* kt, const char* vt, const bf16x8 (*qf)[4],
                                             RowTile* rt, bool masked, int tn, float scale2,
                                             const uint32_t* mword, const LaneOffsets& lo) {
  const int lane = threadIdx.x & (kWave - 1);
  const int lg = lane >> 4;
  bf16x8 kf[2][4];
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      kf[s2][kk] = *reinterpret_cast<const bf16x8*>(kt + lo.k[kk] + 4096 * s2);
  // S^T = K Q^T: 2 subtiles x NT row tiles of independent accumulation chains
  floatx4 st[NT][2];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) st[t][s2] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < 4; ++kk)
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
      for (int t = 0; t < NT; ++t)
        st[t][s2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[s2][kk], qf[t][kk], st[t][s2], 0, 0, 0);
  // V^T fragments via transposed LDS reads (input lane i of block lg reads 4 dims of
  // one key, output lane j gets dim j of 4 keys); their latency hides under the softmax
  bf16x8 vf[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) {
    char* base = const_cast<char*>(vt) + lo.v[dt];
    const shortx4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4_t*)(base));
    const shortx4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4_t*)(base + 4096));
    vf[dt] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
  }
  // online softmax (base 2); lane holds keys 16*s2 + 4*lg + i of row lane%16
  bf16x8 pf[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    float sv[8];
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
      for (int i = 0; i < 4; ++i) sv[4 * s2 + i] = st[t][s2][i];
    if (masked) {
      // key >> 5 == 0: one mask word covers the tile
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = 16 * s2 + 4 * lg + i;
          const bool ok = key < tn && ((mword[t] >> key) & 1u);
          sv[4 * s2 + i] = ok ? sv[4 * s2 + i] : -__builtin_inff();
        }
    }
    float mx = fmaxf(fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3])),
                     fmaxf(fmaxf(sv[4], sv[5]), fmaxf(sv[6], sv[7])));
    mx = row_max4(mx);
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
    for (int e = 0; e < 8; ++e) {
      sv[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[e], scale2, neg_m));
      psum += sv[e];
    }
    rt[t].l += psum;
    uint4 pk;
    pk.x = pack_bf16x2(sv[0], sv[1]);
    pk.y = pack_bf16x2(sv[2], sv[3]);
    pk.z = pack_bf16x2(sv[4], sv[5]);
    pk.w = pack_bf16x2(sv[6], sv[7]);
    pf[t] = as_bf16x8(pk);
  }
  // O^T += V^T P^T
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
#pragma unroll
    for (int t = 0; t < NT; ++t)
      rt[t].o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[dt], pf[t], rt[t].o[dt], 0, 0, 0);
}

template <int NW, int MT, int STAGES>
__global__ __launch_bounds__(NW * kWave, 8 / NW) void attn_main_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_new,
    const uint16_t* __restrict__ v_new, const uint16_t* __restrict__ k_cache,
    const uint16_t* __restrict__ v_cache, const uint32_t* __restrict__ tree_mask, int W, int hq,
    int hkv, int G, float scale2, AttnWs ws, float* __restrict__ out, float* __restrict__ lse) {
  __shared__ __attribute__((aligned(1024))) char s_ring[STAGES * kStageBytes];
  constexpr int kLoads = 16 / NW;
  static_assert(STAGES >= 2 && STAGES <= 4, "ring depth");
  static_assert(NW * MT * 16 == kPassRows && MT == 2, "rows per unit");

  const int nb = gridDim.x;
  const int b = blockIdx.x;
  const long long T = ws.meta[1];
  const int lo = int(range_lo(T, b, nb));
  const int hi = int(range_lo(T, b + 1, nb));
  if (lo >= hi) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = threadIdx.x / kWave;
  const int lr = lane & 15, lg = lane >> 4;
  const size_t stride = size_t(hkv) * kD;
  const LaneOffsets lof = lane_offsets();

  // issue side of the ring: unit of the next tile to copy
  const int nunits = ws.meta[0];
  int iu = ws.wg_unit[b];
  Unit iud = ws.units[iu];
  auto issue = [&](int u) {
    while (u >= iud.tile_end && iu + 1 < nunits) iud = ws.units[++iu];
    const int lt = u - iud.tile_start;
    if (lt < 0 || u >= iud.tile_end) return;  // unreachable: units tile [0, T) contiguously
    const uint16_t *kb, *vb;
    int tn;
    if (lt < iud.ntail) {
      const size_t row = size_t(iud.q0) + size_t(lt) * kTileKeys;
      kb = k_new + row * stride + iud.kvh * kD;
      vb = v_new + row * stride + iud.kvh * kD;
      tn = min(kTileKeys, iud.nslots - lt * kTileKeys);
    } else {
      const int pt = lt - iud.ntail;
      const size_t row = size_t(iud.kb) + size_t(pt) * kTileKeys;
      kb = k_cache + row * stride + iud.kvh * kD;
      vb = v_cache + row * stride + iud.kvh * kD;
      tn = min(kTileKeys, iud.P - pt * kTileKeys);
    }
    issue_tile<NW>(s_ring + (u % STAGES) * kStageBytes, kb, vb, stride, tn);
  };

  // compute side: the unit of the current tile and the wave's rows in it
  int cu = iu;
  Unit cud = iud;
  int ntiles = 0;
  bf16x8 qf[MT][4];
  RowTile rt[MT];
  int rho_t[MT];
  uint32_t mw[MT][kMaskWords];
  int mw0 = 0;  // tail tile of mw[.][0]

  // ring prologue
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (lo + s < hi) issue(lo + s);

  for (int t = lo; t < hi; ++t) {
    wait_vm_tiles<kLoads>(min(STAGES - 2, hi - 1 - t));  // tile t has landed
    __syncthreads();  // ... for every wave, and tile t-1 is no longer read
    while (t >= cud.tile_end && cu + 1 < nunits) cud = ws.units[++cu];
    const int lt = t - cud.tile_start;
    const bool seg_start = (t == lo) || (lt == 0);
    if (t + STAGES - 1 < hi) issue(t + STAGES - 1);
    if (seg_start) {
      // Q fragments of this wave's row tiles, the tree-tail mask words, fresh state.
      // Loaded after the ring copy above and awaited with vmcnt(0): afterwards no
      // compiler-visible load is outstanding, so the steady-state tiles carry no
      // implicit wait that would drain the ring.
      ntiles = 0;
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const int tile = wid + NW * i;
        const int rho = tile * 16 + lr;  // row within the unit
        rho_t[i] = rho;
        if (tile * 16 < cud.rows) ntiles = i + 1;
        uint4 qv[4] = {make_uint4(0, 0, 0, 0), make_uint4(0, 0, 0, 0), make_uint4(0, 0, 0, 0),
                       make_uint4(0, 0, 0, 0)};
        const int ra = cud.row0 + rho;  // row within the pair
        if (rho < cud.rows) {
          const uint16_t* qrow = q + (size_t(cud.q0 + ra / G) * hq + cud.kvh * G + ra % G) * kD;
#pragma unroll
          for (int kk = 0; kk < 4; ++kk)
            qv[kk] = *reinterpret_cast<const uint4*>(qrow + 32 * kk + 8 * lg);
        }
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) qf[i][kk] = as_bf16x8(qv[kk]);
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) rt[i].o[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
        rt[i].m = -__builtin_inff();
        rt[i].l = 0.0f;
        mw0 = lt;
#pragma unroll
        for (int k = 0; k < kMaskWords; ++k) {
          const int word = lt + k;
          mw[i][k] = (rho < cud.rows && word < cud.ntail && word < W)
                         ? tree_mask[size_t(cud.q0 + ra / G) * W + word]
                         : 0u;
        }
      }
      wait_vm<0>();
    }
    // this tile: tree tail (masked by the ancestor bits) or KV prefix
    const char* stg = s_ring + (t % STAGES) * kStageBytes;
    bool masked;
    int tn;
    uint32_t word[MT];
    if (lt < cud.ntail) {
      tn = min(kTileKeys, cud.nslots - lt * kTileKeys);
      masked = true;
      const int k = lt - mw0;
      if (k < kMaskWords) {
#pragma unroll
        for (int i = 0; i < MT; ++i) {
          uint32_t w = 0u;
#pragma unroll
          for (int kk = 0; kk < kMaskWords; ++kk) w = (kk == k) ? mw[i][kk] : w;
          word[i] = w;
        }
      } else {  // requests with more than 128 verify slots: fetch the word now
#pragma unroll
        for (int i = 0; i < MT; ++i) {
          const int ra = cud.row0 + rho_t[i];
          word[i] = (rho_t[i] < cud.rows && lt < W) ? tree_mask[size_t(cud.q0 + ra / G) * W + lt]
                                                     : 0u;
        }
        wait_vm<0>();
      }
    } else {
      tn = min(kTileKeys, cud.P - (lt - cud.ntail) * kTileKeys);
      masked = tn < kTileKeys;
#pragma unroll
      for (int i = 0; i < MT; ++i) word[i] = 0xFFFFFFFFu;
    }
    if (ntiles == MT)
      compute_tile<MT>(stg, stg + kTileBytes, qf, rt, masked, tn, scale2, word, lof);
    else if (ntiles > 0)
      compute_tile<1>(stg, stg + kTileBytes, qf, rt, masked, tn, scale2, word, lof);

    if (t + 1 == hi || t + 1 == cud.tile_end) {
      // end of this workgroup's segment of the unit: final output or a partial
      const int slot = lo < cud.tile_start ? 1 : 0;
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        if (i >= ntiles) break;
        const float l = row_sum4(rt[i].l);
        const int rho = rho_t[i];
        if (rho < cud.rows) {
          if (!cud.cut) {
            const int ra = cud.row0 + rho;
            const size_t orow = size_t(cud.q0 + ra / G) * hq + cud.kvh * G + ra % G;
            const float inv = l > 0.0f ? 1.0f / l : 0.0f;
            float* po = out + orow * kD;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt)
              *reinterpret_cast<floatx4*>(po + 16 * dt + 4 * lg) = rt[i].o[dt] * inv;
            if (lse != nullptr && lg == 0)
              lse[orow] = l > 0.0f ? (rt[i].m + log2f(l)) * kLn2 : -__builtin_inff();
          } else {
            const size_t prow = (size_t(2 * b + slot)) * kPassRows + rho;
            float* po = ws.part_o + prow * kD;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt)
              *reinterpret_cast<floatx4*>(po + 16 * dt + 4 * lg) = rt[i].o[dt];
            if (lg == 0) {
              ws.part_ml[prow * 2 + 0] = rt[i].m;
              ws.part_ml[prow * 2 + 1] = l;
            }
          }
        }
      }
      wait_vm<0>();  // stores drained: later waits count tile copies only
    }
  }
}

// ------------------------------------------------------------- combine ----
// One workgroup per cut unit; thread = (row, 4 dims).  The unit's partials are
// merged in workgroup order.
__global__ __launch_bounds__(kThreads) void attn_combine_kernel(int hq, int G, AttnWs ws,
                                                                float* __restrict__ out,
                                                                float* __restrict__ lse) {
  if (int(blockIdx.x) >= ws.meta[2]) return;
  const Cut c = ws.cuts[blockIdx.x];
  const Unit u = ws.units[c.unit];
  const long long T = ws.meta[1];
  const int nb = gridDim.x;  // the main kernel's workgroup count
  // workgroups with an empty range (fewer tiles than workgroups) left no partial
  auto live = [&](int bb) { return range_lo(T, bb, nb) < range_lo(T, bb + 1, nb); };
  for (int e = threadIdx.x; e < u.rows * (kD / 4); e += kThreads) {
    const int rho = e / (kD / 4);
    const int d4 = (e % (kD / 4)) * 4;
    float M = -__builtin_inff();
    for (int bb = c.b0; bb <= c.b1; ++bb) {
      if (!live(bb)) continue;
      const size_t prow = size_t(2 * bb + (bb == c.b0 ? c.first_slot : 0)) * kPassRows + rho;
      M = fmaxf(M, ws.part_ml[prow * 2]);
    }
    const float Mu = M == -__builtin_inff() ? 0.0f : M;
    float L = 0.0f;
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int bb = c.b0; bb <= c.b1; ++bb) {
      if (!live(bb)) continue;
      const size_t prow = size_t(2 * bb + (bb == c.b0 ? c.first_slot : 0)) * kPassRows + rho;
      const float2 ml = *reinterpret_cast<const float2*>(ws.part_ml + prow * 2);
      const float w = __builtin_amdgcn_exp2f(ml.x - Mu);
      L += w * ml.y;
      acc += w * *reinterpret_cast<const floatx4*>(ws.part_o + prow * kD + d4);
    }
    const int ra = u.row0 + rho;
    const size_t orow = size_t(u.q0 + ra / G) * hq + u.kvh * G + ra % G;
    const float inv = L > 0.0f ? 1.0f / L : 0.0f;
    *reinterpret_cast<floatx4*>(out + orow * kD + d4) = acc * inv;
    if (lse != nullptr && d4 == 0) lse[orow] = L > 0.0f ? (M + log2f(L)) * kLn2 : -__builtin_inff();
  }
}

int main_workgroups() { return 2 * device_cu_count(); }

}  // namespace

size_t attn_workspace_bytes(int32_t R, int32_t max_rows, int32_t hq, int32_t hkv) {
  return attn_ws_total(unit_capacity(R, max_rows, hq, hkv), main_workgroups());
}

int32_t launch_tree_verify_attn(const AttnArgs& a, hipStream_t stream) {
  (void)hipGetLastError();  // clear errors left by unrelated runtime calls
  const int nb = main_workgroups();
  const size_t ucap = unit_capacity(a.R, a.max_rows, a.hq, a.hkv);
  AttnWs ws = attn_layout(a.workspace, ucap, nb);
  const int G = a.hq / a.hkv;
  hipLaunchKernelGGL(attn_plan_kernel, dim3(1), dim3(kThreads), 0, stream, a.q_offsets,
                     a.kv_offsets, static_cast<long long>(a.kv_rows), a.R, a.hkv, G, a.max_rows,
                     nb, ws, a.status);
  const bool prof = g_attn_ev_start != nullptr && g_attn_ev_stop != nullptr;
  if (prof && hipEventRecord(g_attn_ev_start, stream) != hipSuccess) return ECHO_ERR_HIP;
  hipLaunchKernelGGL((attn_main_kernel<kMainWaves, kMT, kStages>), dim3(unsigned(nb)),
                     dim3(kMainWaves * kWave), 0, stream, a.q, a.k_new, a.v_new, a.k_cache,
                     a.v_cache, a.tree_mask, a.mask_words, a.hq, a.hkv, G, a.sm_scale * kLog2e, ws,
                     a.out, a.lse);
  if (prof && hipEventRecord(g_attn_ev_stop, stream) != hipSuccess) return ECHO_ERR_HIP;
  hipLaunchKernelGGL(attn_combine_kernel, dim3(unsigned(nb)), dim3(kThreads), 0, stream, a.hq, G,
                     ws, a.out, a.lse);
  return hipGetLastError() == hipSuccess ? ECHO_OK : ECHO_ERR_HIP;
}

}  // namespace echo
