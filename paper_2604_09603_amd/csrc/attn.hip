// Tree-masked grouped-query verification attention (one verification forward
// over the flattened super-tree).  Three launches (a paged cache adds
// attn_pages first, which checks the block tables' page ids):
//
//   attn_plan     one workgroup.  A stream is one KV head of one request
//                 together with a pass over its rows (rows = verify slots x
//                 query heads of the GQA group, at most 64 per pass).  The
//                 streams of a request are grouped four at a time, head-major;
//                 a group is one unit of work whose tiles are the request's
//                 32-key tiles: first the tree-tail tiles (the new keys of the
//                 request's own slots), then the KV-prefix tiles.  The tiles of
//                 all units are cut into equal contiguous ranges, one per
//                 workgroup of the main kernel; the plan records each unit's
//                 tiles and which units are cut.
//   attn_main     persistent, one workgroup of four waves per CU.  Wave w runs
//                 stream w of every unit in its workgroup's range over the same
//                 tiles as its three siblings: it copies its head's slice of
//                 each tile HBM -> LDS into its own two-stage ring with
//                 direct-to-LDS loads, reads the tile into registers, refills
//                 the stage and multiplies the tile against all rows of its
//                 stream.  The four waves read the four heads of the same token
//                 rows at the same time (whole rows of the KV cache), and the
//                 passes of one head share their reads in the caches.  No
//                 barrier is needed: every wave owns its ring and its softmax
//                 state.  S^T = K Q^T and O^T = V^T P^T on
//                 v_mfma_f32_16x16x32_bf16 (fp32 accumulation), online softmax
//                 in base 2 between the products of the neighbouring 16-row
//                 tiles, ancestor bitmask on tree-tail tiles.  A unit that
//                 lies inside one range is normalised and written to out/lse; a
//                 cut unit leaves one partial (O, max, sums) per stream and
//                 workgroup.
//   attn_combine  one thread per (cut unit, stream, two rows, 4 dims): merges the
//                 partials in range order (deterministic) into out and lse.
#include <hip/hip_ext.h>

#include "attn_device.h"
#include "echo_device.h"
#include "echo_internal.h"

namespace echo {
namespace {

// Paged prefixes: workgroup (r, c) checks page ids c * 256 .. c * 256 + 255 of
// request r and records whether one is outside [0, num_pages) (every chunk is
// written, so nothing needs clearing first).
__global__ __launch_bounds__(kPageChunk) void attn_pages_kernel(KvSource kv) {
  const int r = blockIdx.x, c = blockIdx.y;
  const long long P = kv.prefix_len[r];
  const bool len_ok = P >= 0 && P <= (long long)kv.max_pages * kv.page_size;
  const long long np = len_ok ? (P + kv.page_size - 1) / kv.page_size : 0;
  const long long e = (long long)c * kPageChunk + threadIdx.x;
  int bad = 0;
  if (e < np) {
    const int pg = kv.block_table[size_t(r) * size_t(kv.max_pages) + size_t(e)];
    bad = pg < 0 || pg >= kv.num_pages;
  }
  bad = __syncthreads_or(bad);
  if (threadIdx.x == 0) const_cast<int32_t*>(kv.page_bad)[size_t(r) * kv.page_chunks + c] = bad;
}

__global__ __launch_bounds__(kThreads) void attn_plan_kernel(
    const int32_t* __restrict__ q_offsets, KvSource kv, int R, int hkv, int G, int max_rows,
    int nb, long long ucap, AttnWs ws, int32_t* status) {
  extern __shared__ int32_t plan_tables[];  // plan_table_words(min(R, kThreads))
  plan_body<kThreads>(q_offsets, kv, R, hkv, G, max_rows, nb, ucap, ws, status, plan_tables);
}

// ---------------------------------------------------------------- main ----
// LDS tile layout: 32 key rows x 256 bytes per tensor, no padding.  The 16-byte
// chunk c of row r is stored at chunk position c ^ rot(r & 15), rot swapping
// the two 2-bit halves of the row's low four bits.  Rows 16 apart share a
// pattern; within 16 consecutive rows every pattern differs, so the K fragment
// reads (16 rows, one column) fall into 16 different bank groups, and so do
// the transposed V reads of two 16-lane blocks (8 rows, 4 at a time, of 2
// consecutive chunks: the rows' low bits select the chunk's high bits and
// the next two bits its low bits).
typedef __attribute__((address_space(3))) void lds_void_t;
typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) shortx4 lds_shortx4_t;

constexpr int kTileBytes = kTileKeys * kD * 2;  // 8 KB per tensor
constexpr int kStageBytes = 2 * kTileBytes;     // K then V
constexpr int kMainLds = kWaves * kWaveStages * kStageBytes;  // 128 KB
static_assert(kMainLds <= 160 * 1024, "gfx950 LDS per workgroup");

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Round two floats to bfloat16 (to nearest even) in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2{lo, hi}, bf16x2));
}

// acc plus the two bfloat16 values packed in w (one v_dot2c_f32_bf16 against
// (1, 1); the products are exact).
__device__ __forceinline__ float add_bf16x2(uint32_t w, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w),
                                         __builtin_bit_cast(bf16x2, 0x3F803F80u), acc, false);
}

__device__ __forceinline__ int swz_pattern(int row) { return ((row & 3) << 2) | ((row >> 2) & 3); }

__device__ __forceinline__ int swz(int row, int chunk) {
  return row * 256 + ((chunk ^ swz_pattern(row)) << 4);
}

__device__ __forceinline__ uint64_t uniform64(uint64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(x));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(x >> 32));
  return (uint64_t(hi) << 32) | lo;
}

constexpr int kCopiesPerTile = 16;  // wave instructions of 1 KB (4 key rows) per K+V tile

// Per-lane source offsets of one tile copy: instruction j (per tensor) fills LDS
// rows 4j .. 4j+3; the lane fetches the source chunk that the swizzle puts at
// its LDS position.
__device__ __forceinline__ int copy_row(int j) { return j * 4 + ((threadIdx.x & (kWave - 1)) >> 4); }
__device__ __forceinline__ uint32_t copy_chunk16(int row) {
  return uint32_t(((threadIdx.x & 15) ^ swz_pattern(row)) * 16);
}

// Lane offsets of a full tile's copy.  The copies of a full tile go in four
// groups of four 1 KB loads (K rows 0-15, K rows 16-31, V rows 0-15, V rows
// 16-31), one LDS base per group; load j of a group adds 1024 j to both its
// global and its LDS address (the instruction offset applies to both), so the
// lane offset is the source offset of its chunk minus 1024 j.  Rows 16 apart
// have the same swizzle, so the second group of a tensor reuses the offsets
// from a base 16 rows further on.
struct CopyPlan {
  uint32_t off[4];
};

__device__ __forceinline__ CopyPlan copy_plan(uint32_t row_bytes) {
  CopyPlan cp;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int row = copy_row(j);
    cp.off[j] = uint32_t(row) * row_bytes + copy_chunk16(row) - 1024u * uint32_t(j);
  }
  return cp;
}

// One K+V tile into a stage with 16 direct HBM -> LDS loads: in load j every
// lane moves 16 bytes from kbase + off[j] (V: vbase + off[j]) to 1 KB block j
// (V: block 8 + j) of the stage, at lds_stage + 1024 * block + 16 * lane.  The
// bases and lds_stage are wave-uniform, the offsets per lane.  One inline
// assembly block issues them, for two reasons: the compiler does not track
// these loads (its own bookkeeping would drain every load in flight before each
// LDS read; completion is awaited explicitly with vmcnt), and M0, which holds
// the LDS address of such a load, is set once and stepped by 1 KB.  A write of
// M0 needs one wait state before an LDS load reads it (s_nop 0).  M0 belongs to
// the compiler and is restored; the steps clobber SCC.  kNT marks the loads
// non-temporal (data no other wave of the workgroup reads): streamed with that
// hint, HBM-bound batches copy 5-8% faster, while data that sibling waves read
// again must stay cached.
#define ECHO_DMA_STEP(J, B, POL) \
  "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %" #J ", %" #B POL "\n\t"
#define ECHO_DMA_TILE(POL)                                                                      \
  "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %2, %10" POL    \
  "\n\t" ECHO_DMA_STEP(3, 10, POL) ECHO_DMA_STEP(4, 10, POL) ECHO_DMA_STEP(5, 10, POL)        \
      ECHO_DMA_STEP(6, 10, POL) ECHO_DMA_STEP(7, 10, POL) ECHO_DMA_STEP(8, 10, POL)             \
          ECHO_DMA_STEP(9, 10, POL) ECHO_DMA_STEP(2, 11, POL) ECHO_DMA_STEP(3, 11, POL)         \
              ECHO_DMA_STEP(4, 11, POL) ECHO_DMA_STEP(5, 11, POL) ECHO_DMA_STEP(6, 11, POL)     \
                  ECHO_DMA_STEP(7, 11, POL) ECHO_DMA_STEP(8, 11, POL) ECHO_DMA_STEP(9, 11, POL) \
                      "s_mov_b32 m0, %0"

// A full tile: M0 is set once per group of four loads (four writes per tile
// instead of sixteen); see CopyPlan.  Operands: %1 LDS stage, %2-%5 lane
// offsets, %6/%7 K at rows 0 and 16, %8/%9 V at rows 0 and 16.
#define ECHO_DMA_GROUP(B, POL)                                                        \
  "global_load_lds_dwordx4 %2, %" #B POL "\n\tglobal_load_lds_dwordx4 %3, %" #B     \
  " offset:1024" POL "\n\tglobal_load_lds_dwordx4 %4, %" #B " offset:2048" POL      \
  "\n\tglobal_load_lds_dwordx4 %5, %" #B " offset:3072" POL "\n\t"
#define ECHO_DMA_FULL(POL)                                                            \
  "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t" ECHO_DMA_GROUP(6, POL)       \
  "s_add_u32 m0, m0, 0x1000\n\ts_nop 0\n\t" ECHO_DMA_GROUP(7, POL)                   \
  "s_add_u32 m0, m0, 0x1000\n\ts_nop 0\n\t" ECHO_DMA_GROUP(8, POL)                   \
  "s_add_u32 m0, m0, 0x1000\n\ts_nop 0\n\t" ECHO_DMA_GROUP(9, POL) "s_mov_b32 m0, %0"

template <bool kNT>
__device__ __forceinline__ void dma_tile_full(uint32_t lds_stage, uint64_t kbase, uint64_t vbase,
                                              uint32_t half_bytes, const uint32_t (&off)[4]) {
  const uint32_t lds = __builtin_amdgcn_readfirstlane(lds_stage);
  const uint64_t kb = uniform64(kbase), vb = uniform64(vbase);
  const uint64_t kb16 = kb + half_bytes, vb16 = vb + half_bytes;
  uint32_t saved;
  if (kNT) {
    asm volatile(ECHO_DMA_FULL(" nt")
                 : "=&s"(saved)
                 : "s"(lds), "v"(off[0]), "v"(off[1]), "v"(off[2]), "v"(off[3]), "s"(kb),
                   "s"(kb16), "s"(vb), "s"(vb16)
                 : "memory", "scc");
  } else {
    asm volatile(ECHO_DMA_FULL("")
                 : "=&s"(saved)
                 : "s"(lds), "v"(off[0]), "v"(off[1]), "v"(off[2]), "v"(off[3]), "s"(kb),
                   "s"(kb16), "s"(vb), "s"(vb16)
                 : "memory", "scc");
  }
}
#undef ECHO_DMA_FULL
#undef ECHO_DMA_GROUP

// A partial tile (rows clamped to the last valid one): one M0 write per load.
template <bool kNT>
__device__ __forceinline__ void dma_tile(uint32_t lds_stage, uint64_t kbase, uint64_t vbase,
                                         const uint32_t (&off)[8]) {
  const uint32_t lds = __builtin_amdgcn_readfirstlane(lds_stage);
  const uint64_t kb = uniform64(kbase), vb = uniform64(vbase);
  uint32_t saved;
  if (kNT) {
    asm volatile(ECHO_DMA_TILE(" nt")
                 : "=&s"(saved)
                 : "s"(lds), "v"(off[0]), "v"(off[1]), "v"(off[2]), "v"(off[3]), "v"(off[4]),
                   "v"(off[5]), "v"(off[6]), "v"(off[7]), "s"(kb), "s"(vb)
                 : "memory", "scc");
  } else {
    asm volatile(ECHO_DMA_TILE("")
                 : "=&s"(saved)
                 : "s"(lds), "v"(off[0]), "v"(off[1]), "v"(off[2]), "v"(off[3]), "v"(off[4]),
                   "v"(off[5]), "v"(off[6]), "v"(off[7]), "s"(kb), "s"(vb)
                 : "memory", "scc");
  }
}
#undef ECHO_DMA_TILE
#undef ECHO_DMA_STEP

// Copy one K+V tile (tn <= 32 valid key rows, rows row_bytes apart) into the
// stage at LDS address lds_stage.  Rows >= tn re-read row tn-1 (in bounds); the
// softmax masks those keys.
template <bool kNT>
__device__ __forceinline__ void issue_tile(uint32_t lds_stage, uint64_t kbase, uint64_t vbase,
                                           uint32_t row_bytes, int tn, const CopyPlan& cp) {
  if (tn == kTileKeys) {
    dma_tile_full<kNT>(lds_stage, kbase, vbase, 16u * row_bytes, cp.off);
  } else {
    uint32_t off[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int row = copy_row(j);
      const int srow = row < tn ? row : tn - 1;
      off[j] = uint32_t(srow) * row_bytes + copy_chunk16(row);
    }
    dma_tile<kNT>(lds_stage, kbase, vbase, off);
  }
}

template <int N>
__device__ __forceinline__ void wait_vm() {
  // gfx9 s_waitcnt encoding: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt_hi[15:14]
  constexpr int imm = (N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14);
  __builtin_amdgcn_s_waitcnt(imm);
}

__device__ __forceinline__ void wait_lds() {
  // lgkmcnt(0); vmcnt and expcnt left at their maxima
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
}

struct RowTile {
  floatx4 o[8];  // O^T: lane holds dims 16*dt + 4*(lane/16) + i of row lane%16
  float m;       // softmax reference max of scaled logits (log2 units)
  float l;       // this lane's share of the running sum (for the LSE)
  float lq;      // the same over the bf16-rounded probabilities (normalises O)
  float mgrow;   // m + kRescaleSlack: a tile max above it raises the reference
  float negm;    // -m (0 while m is -inf): the exponent's offset
  float thr;     // screen of the residual split: m + log2(row sum) - 5, taken
                 // when last refreshed (see compute_tile)
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

// A whole 32-key tile in registers: the K A-fragments of both 16-key subtiles
// and the V^T A-fragments of the eight 16-dim blocks.
struct TileFrags {
  bf16x8 kf[2][4];
  bf16x8 vf[8];
};

// Read a tile from its LDS stage.  V^T comes from transposed reads (input lane i
// of block lg reads 4 dims of one key, output lane j gets dim j of 4 keys).
__device__ __forceinline__ void load_tile(const char* kt, const char* vt, const LaneOffsets& lo,
                                          TileFrags& f) {
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      f.kf[s2][kk] = *reinterpret_cast<const bf16x8*>(kt + lo.k[kk] + 4096 * s2);
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) {
    char* base = const_cast<char*>(vt) + lo.v[dt];
    const shortx4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4_t*)(base));
    const shortx4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4_t*)(base + 4096));
    f.vf[dt] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
  }
}

// One 32-key tile (already in registers) against MT row tiles (all rows of the
// unit).  masked: keys >= tn are invisible, and key j is visible to a row only
// if bit j of its mask word is set.
//
// Row tile t's softmax runs between the S^T products of row tile t + 1 and the
// P V products of row tile t - 1, which do not depend on it, one product at a
// time between a few vector instructions: the matrix unit works on those
// while the vector unit computes the probabilities.  (Left to itself the
// scheduler issues the eight products of a group back to back, and a wave
// issues in order, so nothing would overlap.)  Scheduling fences
// (sched_barrier) hold that order; the arithmetic and its order per row are
// the same as with the products grouped.
template <int MT>
__device__ __forceinline__ void compute_tile(const TileFrags& f, const bf16x8 (*qf)[4],
                                             RowTile* rt, bool masked, float scale2,
                                             const uint32_t* mword) {
  const int lane = threadIdx.x & (kWave - 1);
  const int lg = lane >> 4;
  floatx4 st[MT][2];  // S^T of each row tile: two 16-key subtiles
  bf16x8 pf[MT];      // bf16 probabilities, the B operand of P V
  // product j (0..7) of row tile t's S^T = K Q^T: key subtile j & 1, dims
  // 32 (j >> 1) .. 32 (j >> 1) + 31
  auto s_step = [&](int t, int j) {
    const int s2 = j & 1, kk = j >> 1;
    st[t][s2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
        f.kf[s2][kk], qf[t][kk], kk == 0 ? floatx4{0.f, 0.f, 0.f, 0.f} : st[t][s2], 0, 0, 0);
  };
  // product dt of row tile t's O^T += V^T P^T (dims 16 dt .. 16 dt + 15)
  auto pv_step = [&](int t, int dt) {
    rt[t].o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.vf[dt], pf[t], rt[t].o[dt], 0, 0, 0);
  };
#define ECHO_FENCE() __builtin_amdgcn_sched_barrier(0)
#pragma unroll
  for (int j = 0; j < 8; ++j) s_step(0, j);
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const bool nx = t + 1 < MT;
    // lane holds keys 16*s2 + 4*lg + i of row lane%16
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
          const bool ok = (mword[t] >> key) & 1u;
          sv[4 * s2 + i] = ok ? sv[4 * s2 + i] : -__builtin_inff();
        }
    }
    // this lane's max over its 8 of the row's 32 keys, beside row tile t + 1's
    // S^T.  A lane's max exceeds a bound in some lane of a row
    // exactly when the row's max does, so the rescale test and the residual
    // screen need no reduction over the row's four lanes; the rare branches
    // that do take the row's max.
    ECHO_FENCE();
    if (nx) s_step(t + 1, 0);
    ECHO_FENCE();
    const float a01 = fmaxf(sv[0], sv[1]), a23 = fmaxf(sv[2], sv[3]);
    ECHO_FENCE();
    if (nx) s_step(t + 1, 1);
    ECHO_FENCE();
    const float a47 = fmaxf(fmaxf(sv[4], sv[5]), fmaxf(sv[6], sv[7]));
    ECHO_FENCE();
    if (nx) s_step(t + 1, 2);
    ECHO_FENCE();
    const float lmt = fmaxf(fmaxf(a01, a23), a47) * scale2;  // -inf stays -inf
    // raise the reference only when a logit would exceed it by more than the slack
    if (__ballot(lmt > rt[t].mgrow) != 0ull) {
      const float mt = row_max4(lmt);
      const bool grow = mt > rt[t].mgrow;
      const float alpha = grow ? __builtin_amdgcn_exp2f(rt[t].m - mt) : 1.0f;  // 0 from -inf
      rt[t].l *= alpha;
      rt[t].lq *= alpha;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) rt[t].o[dt] *= alpha;
      rt[t].m = grow ? mt : rt[t].m;
      rt[t].mgrow = rt[t].m + kRescaleSlack;
      rt[t].negm = rt[t].m == -__builtin_inff() ? 0.0f : -rt[t].m;
    }
    // probabilities beside row tile t - 1's P V and the rest of row tile t + 1's S^T
    const float neg_m = rt[t].negm;
    float psum = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      ECHO_FENCE();
      if (t >= 1) pv_step(t - 1, e);
      ECHO_FENCE();
      if (nx && e < 5) s_step(t + 1, 3 + e);
      ECHO_FENCE();
      sv[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[e], scale2, neg_m));
      psum += sv[e];
    }
    ECHO_FENCE();
    rt[t].l += psum;
    uint4 pk;
    pk.x = pack_bf16x2(sv[0], sv[1]);
    pk.y = pack_bf16x2(sv[2], sv[3]);
    pk.z = pack_bf16x2(sv[4], sv[5]);
    pk.w = pack_bf16x2(sv[6], sv[7]);
    // O is normalised by the sum of the same rounded probabilities that
    // multiply V, so the output is an exact convex combination of V rows with
    // the rounded weights: each weight is off by at most 2^-8 of itself and the
    // output by at most 2^-9 times the spread of the V values that carry the
    // weight.  (Dividing by the unrounded sum leaves an error of up to 2^-9 of
    // |v| even on a row whose weight sits on one key.)  The LSE keeps the
    // unrounded sum.
    rt[t].lq = add_bf16x2(pk.w, add_bf16x2(pk.z, add_bf16x2(pk.y, add_bf16x2(pk.x, rt[t].lq))));
    pf[t] = as_bf16x8(pk);
    // Where a few keys carry the row's weight, the rounding of their
    // probabilities moves the output by up to 2^-9 of the spread of their
    // values.  A key of this tile has at most 2^(mt - m) of weight; if that can
    // exceed 1/16 of the row's running sum (the sum over its four lanes, a
    // lower bound of the row's final sum), the residuals p - bf16(p), rounded
    // to bf16 too, go through a second product and into the normaliser,
    // leaving 2^-17 of relative error on these weights.  Long rows over many
    // keys take this path only on their first tiles and on outliers.
    //
    // The test is screened first: m + log2(row sum) is the log2 of the row's
    // running sum in absolute units, which only grows from tile to tile (a
    // rescale moves m and the sum together), so thr = m + log2(sum) - 5 taken
    // at any earlier tile is at most the test's threshold now, m + log2(sum)
    // - 4, and a tile max at or below it cannot pass the test.  The exact test
    // (and a refresh of thr) runs only when the screen lets a tile through.
    bool split = false;
    if (__ballot(lmt > rt[t].thr) != 0ull) {
      const float mt = row_max4(lmt);
      const float rs = row_sum4(rt[t].l);
      split = __ballot(__builtin_amdgcn_exp2f(mt - rt[t].m) > kSplitFrac * rs) != 0ull;
      rt[t].thr = rt[t].m + __builtin_amdgcn_logf(rs) - 5.0f;
    }
    if (split) {
      uint4 pl;
      const auto res = [](float p, uint32_t hi2, int half) {
        const uint32_t b = half ? (hi2 & 0xFFFF0000u) : (hi2 << 16);
        return p - __uint_as_float(b);
      };
      pl.x = pack_bf16x2(res(sv[0], pk.x, 0), res(sv[1], pk.x, 1));
      pl.y = pack_bf16x2(res(sv[2], pk.y, 0), res(sv[3], pk.y, 1));
      pl.z = pack_bf16x2(res(sv[4], pk.z, 0), res(sv[5], pk.z, 1));
      pl.w = pack_bf16x2(res(sv[6], pk.w, 0), res(sv[7], pk.w, 1));
      rt[t].lq = add_bf16x2(pl.w, add_bf16x2(pl.z, add_bf16x2(pl.y, add_bf16x2(pl.x, rt[t].lq))));
      const bf16x8 plo = as_bf16x8(pl);
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
        rt[t].o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.vf[dt], plo, rt[t].o[dt], 0, 0, 0);
    }
  }
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) pv_step(MT - 1, dt);
#undef ECHO_FENCE
}

// The wave's index in the workgroup, known to the compiler as wave-uniform (so
// that everything derived from it stays in scalar registers).
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane(int(threadIdx.x) / kWave);
}

struct MainArgs {
  const uint16_t* q;
  const uint16_t* k_new;
  const uint16_t* v_new;
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  const int32_t* block_table;  // paged prefix (else nullptr): see KvSource
  int page_shift;              // log2 of the page size (>= 5: a tile never straddles pages)
  int max_pages;
  const uint32_t* tree_mask;
  int W, hq, hkv, G;
  float scale2;
  float* out;
  float* lse;
};

// Unit descriptors are written by the plan launch and only read here: load
// them through the constant address space (scalar loads when the index is
// wave-uniform).
typedef __attribute__((address_space(4))) const int32_t const_i32_t;
__device__ __forceinline__ Unit load_unit(const Unit* units, int i) {
  static_assert(sizeof(Unit) == 12 * sizeof(int32_t), "unit layout");
  const_i32_t* p = (const_i32_t*)(units + i);
  Unit u;
  u.tile_start = p[0];
  u.tile_end = p[1];
  u.q0 = p[2];
  u.nslots = p[3];
  u.kb = p[4];
  u.P = p[5];
  u.ntail = p[6];
  u.passes = p[7];
  u.rpp = p[8];
  u.group = p[9];
  u.cut = p[10];
  u.pad = p[11];
  return u;
}

// A workgroup's start record, through the constant address space as the units.
__device__ __forceinline__ WgStart load_wg_start(const WgStart* starts, int b) {
  static_assert(sizeof(WgStart) == 16 * sizeof(int32_t), "start record layout");
  const_i32_t* p = (const_i32_t*)(starts + b);
  int32_t w[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) w[k] = p[k];
  return __builtin_bit_cast(WgStart, w);
}

// Issue side of a wave's ring: the wave's k-th tile is lo + k; its copy goes to
// stage k % 2 (nothing is copied where the wave's stream of the unit is empty).
struct Issuer {
  int iu;          // unit of the next tile to copy (wave-uniform)
  Unit ud;
  Stream sm;       // this wave's stream of that unit
  int k;           // ordinal of the next tile to copy
  uint32_t copied;  // bit s: the last copy into stage s moved data
  // the stream's KV head: at the unit's first new-key row, and at its first
  // prefix row (contiguous cache) or at row 0 of the cache (paged)
  const char *tail_k, *tail_v, *pre_k, *pre_v;
  const int32_t* bt_row;  // paged: the request's block-table row
  bool nt;                // no other wave of the unit reads this stream's head
};

// Point the issue side at unit is.ud.
__device__ __forceinline__ void issuer_unit(Issuer& is, const MainArgs& a, int wid) {
  is.sm = stream_of(is.ud, wid, a.hkv, a.G);
  // streams of a group are consecutive and head-major: a sibling of the same
  // head is the previous or the next stream of the group
  is.nt = true;
  if (is.ud.passes > 1) {
    const int passes = is.ud.passes;
    const int id = kWaves * is.ud.group + wid;
    const bool prev = wid > 0 && (id - 1) / passes == id / passes;
    const bool next =
        wid + 1 < kWaves && id + 1 < a.hkv * passes && (id + 1) / passes == id / passes;
    is.nt = !(prev || next);
  }
  const size_t row_bytes = size_t(a.hkv) * kD * 2;
  const size_t head = size_t(is.sm.kvh) * kD * 2;
  is.tail_k = reinterpret_cast<const char*>(a.k_new) + size_t(is.ud.q0) * row_bytes + head;
  is.tail_v = reinterpret_cast<const char*>(a.v_new) + size_t(is.ud.q0) * row_bytes + head;
  const size_t first = a.block_table == nullptr ? size_t(is.ud.kb) * row_bytes : 0;
  is.pre_k = reinterpret_cast<const char*>(a.k_cache) + first + head;
  is.pre_v = reinterpret_cast<const char*>(a.v_cache) + first + head;
  is.bt_row = a.block_table == nullptr ? nullptr
                                       : a.block_table + size_t(is.ud.kb) * size_t(a.max_pages);
}

__device__ __forceinline__ void issue_next(Issuer& is, const MainArgs& a, const AttnWs& ws,
                                           int nunits, int lo, int hi, int wid,
                                           uint32_t ring_lds, const CopyPlan& cp) {
  const int t = lo + is.k;
  if (t >= hi) return;
  while (t >= is.ud.tile_end && is.iu + 1 < nunits) {
    is.iu = __builtin_amdgcn_readfirstlane(is.iu + 1);
    is.ud = load_unit(ws.units, is.iu);
    issuer_unit(is, a, wid);
  }
  const int lt = t - is.ud.tile_start;
  const bool copy = is.sm.rows > 0 && lt >= 0 && t < is.ud.tile_end;
  is.copied = (is.copied & ~(1u << (is.k & 1))) | (uint32_t(copy) << (is.k & 1));
  if (copy) {
    const uint32_t row_bytes = uint32_t(a.hkv) * kD * 2;
    const uint32_t tile_bytes = kTileKeys * row_bytes;
    const char *kb, *vb;
    int tn;
    if (lt < is.ud.ntail) {
      kb = is.tail_k + size_t(lt) * tile_bytes;
      vb = is.tail_v + size_t(lt) * tile_bytes;
      tn = min(kTileKeys, is.ud.nslots - lt * kTileKeys);
    } else {
      const int pt = lt - is.ud.ntail;
      size_t off;
      if (is.bt_row == nullptr) {
        off = size_t(pt) * tile_bytes;
      } else {
        // wave-uniform index: a scalar load of the tile's page
        const int pos = pt * kTileKeys;
        const int page = ((const const_i32_t*)is.bt_row)[pos >> a.page_shift];
        off = ((size_t(page) << a.page_shift) + size_t(pos & ((1 << a.page_shift) - 1))) * row_bytes;
      }
      kb = is.pre_k + off;
      vb = is.pre_v + off;
      tn = min(kTileKeys, is.ud.P - pt * kTileKeys);
    }
    const uint32_t stage = ring_lds + uint32_t((is.k & 1) * kStageBytes);
    if (is.nt)
      issue_tile<true>(stage, reinterpret_cast<uint64_t>(kb), reinterpret_cast<uint64_t>(vb),
                       row_bytes, tn, cp);
    else
      issue_tile<false>(stage, reinterpret_cast<uint64_t>(kb), reinterpret_cast<uint64_t>(vb),
                        row_bytes, tn, cp);
  }
  ++is.k;
}

// The tree-mask word of tail tile lt for a row of slot `slot` (0 outside).
__device__ __forceinline__ uint32_t mask_word(const MainArgs& a, const Unit& ud, bool row_ok,
                                              int slot, int lt) {
  return (row_ok && lt >= 0 && lt < ud.ntail && lt < a.W)
             ? a.tree_mask[size_t(slot) * a.W + lt]
             : 0u;
}

// Dims 16 (2j) + 4 g + [0, 4) and 16 (2j + 1) + 4 g + [0, 4) of a lane's row,
// scaled and rounded to fp16: one 16-byte store (see part_dim).
__device__ __forceinline__ halfx8 pack_part(floatx4 lo4, floatx4 hi4, float sc) {
  const halfx4 a0 = __builtin_convertvector(lo4 * sc, halfx4);
  const halfx4 a1 = __builtin_convertvector(hi4 * sc, halfx4);
  return halfx8{a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
}

// The partial of a workgroup's first segment when its unit is cut and more
// segments follow: the next segment's first loads would wait for its stores,
// which drain slowly while every workgroup streams the cache (14 us at q235b),
// so it is held in registers and stored after the workgroup's last segment.
struct HeldPartial {
  uint32_t h[kMaxMT][16];  // the rows in fp16, packed as the stores write them
  floatx4 ml[kMaxMT];      // max, sum, rounded sum and scale exponent of the lane's row
  int mt, rows;            // row tiles held; rows of the stream
  size_t prow0;            // partial row of the stream's row 0
};

// The wave's stream over one unit segment [seg_lo, seg_hi), then its output
// (final, partial, or, when `held` (wave-uniform), a partial kept in `hold`).
template <int MT>
__device__ __forceinline__ void run_segment(const MainArgs& a, const AttnWs& ws, const Unit& ud,
                                            const Stream& sm, int seg_lo, int seg_hi, int lo,
                                            int hi, int nunits, int b, const char* ring,
                                            uint32_t ring_lds, Issuer& is,
                                            const CopyPlan& cp, const LaneOffsets& lof,
                                            bool held, HeldPartial& hold) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = wave_id();
  const int lr = lane & 15, lg = lane >> 4;
  const int G = a.G;

  // Q fragments of the stream's rows and the mask words of the segment's first
  // tail tiles.  Loaded and awaited with vmcnt(0): afterwards no
  // compiler-visible load is in flight, so the tile loop carries no implicit
  // wait that would drain the ring.
  const int lt0 = seg_lo - ud.tile_start;
  bf16x8 qf[MT][4];
  uint32_t mw[MT][kMaskWords];
  RowTile rt[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int rho = 16 * i + lr;
    const int ra = sm.row0 + rho;
    const bool row_ok = rho < sm.rows;
    const int slot = ud.q0 + ra / G;
    uint4 qv[4] = {make_uint4(0, 0, 0, 0), make_uint4(0, 0, 0, 0), make_uint4(0, 0, 0, 0),
                   make_uint4(0, 0, 0, 0)};
    if (row_ok) {
      const uint16_t* qrow = a.q + (size_t(slot) * a.hq + sm.kvh * G + ra % G) * kD;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        qv[kk] = *reinterpret_cast<const uint4*>(qrow + 32 * kk + 8 * lg);
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) qf[i][kk] = as_bf16x8(qv[kk]);
#pragma unroll
    for (int k = 0; k < kMaskWords; ++k) mw[i][k] = mask_word(a, ud, row_ok, slot, lt0 + k);
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) rt[i].o[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
    rt[i].m = -__builtin_inff();
    rt[i].l = 0.0f;
    rt[i].lq = 0.0f;
    rt[i].mgrow = -__builtin_inff();
    rt[i].negm = 0.0f;
    rt[i].thr = -__builtin_inff();
  }
  wait_vm<0>();

  for (int t = seg_lo; t < seg_hi; ++t) {
    const int k = t - lo;  // tile ordinal of this wave
    // tile k has landed once at most the copies of the next tile are in flight
    if (is.k > k + 1 && ((is.copied >> ((k + 1) & 1)) & 1u)) wait_vm<kCopiesPerTile>();
    else wait_vm<0>();
    const char* stg = ring + (k & 1) * kStageBytes;
    const int lt = t - ud.tile_start;
    bool masked;
    int tn;
    uint32_t word[MT];
    if (lt < ud.ntail) {
      tn = min(kTileKeys, ud.nslots - lt * kTileKeys);
      masked = true;
      if (lt - lt0 < kMaskWords) {
#pragma unroll
        for (int i = 0; i < MT; ++i) word[i] = (lt == lt0) ? mw[i][0] : mw[i][1];
      } else {  // more than 64 verify slots in the segment's tail: fetch the word now
#pragma unroll
        for (int i = 0; i < MT; ++i) {
          const int rho = 16 * i + lr;
          const int ra = sm.row0 + rho;
          word[i] = mask_word(a, ud, rho < sm.rows, ud.q0 + ra / G, lt);
        }
        wait_vm<0>();
      }
    } else {
      tn = min(kTileKeys, ud.P - (lt - ud.ntail) * kTileKeys);
      masked = tn < kTileKeys;
#pragma unroll
      for (int i = 0; i < MT; ++i) word[i] = 0xFFFFFFFFu;
    }
    // keys >= tn are invisible too: one limit per tile, in the words
    const uint32_t lim = tn >= kTileKeys ? 0xFFFFFFFFu : ((1u << tn) - 1u);
#pragma unroll
    for (int i = 0; i < MT; ++i) word[i] &= lim;
    // tile -> registers, then refill the stage at once: the ring stays full
    // while the tile is multiplied
    TileFrags f;
    load_tile(stg, stg + kTileBytes, lof, f);
    wait_lds();
    issue_next(is, a, ws, nunits, lo, hi, wid, ring_lds, cp);
    compute_tile<MT>(f, qf, rt, masked, a.scale2, word);
  }

  // ---- output of the segment ----
  const bool cut = ud.cut != 0;
  const int slot_id = lo < ud.tile_start ? 1 : 0;
  if (held) {
    hold.mt = MT;
    hold.rows = sm.rows;
    hold.prow0 = part_row(b, slot_id, wid, 0);
  }
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const float L = row_sum4(rt[i].l);
    const float Lq = row_sum4(rt[i].lq);
    const float M = rt[i].m;
    // a cut unit's partial row goes out in fp16, scaled by 2^-e so that its
    // largest magnitude lies in [2^14, 2^15): half the bytes of fp32
    int e = 0;
    if (cut) {
      float mx = 0.0f;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
#pragma unroll
        for (int c = 0; c < 4; ++c) mx = fmaxf(mx, fabsf(rt[i].o[dt][c]));
      mx = row_max4(mx);
      e = mx > 0.0f ? __builtin_amdgcn_frexp_expf(mx) - 15 : 0;
    }
    const int rho = 16 * i + lr;
    if (rho < sm.rows) {
      if (!cut) {
        const int ra = sm.row0 + rho;
        const size_t orow = size_t(ud.q0 + ra / G) * a.hq + sm.kvh * G + ra % G;
        const float inv = Lq > 0.0f ? 1.0f / Lq : 0.0f;
        float* po = a.out + orow * kD;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt)
          // written once and not read again here: stored with the non-temporal hint
          __builtin_nontemporal_store(rt[i].o[dt] * inv,
                                      reinterpret_cast<floatx4*>(po + 16 * dt + 4 * lg));
        if (a.lse != nullptr && lg == 0)
          a.lse[orow] = L > 0.0f ? (M + log2f(L)) * kLn2 : -__builtin_inff();
      } else if (!held) {
        const size_t prow = part_row(b, slot_id, wid, rho);
        const float sc = __builtin_amdgcn_ldexpf(1.0f, -e);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *reinterpret_cast<halfx8*>(ws.part_o + prow * kD + part_dim(32 * j + 4 * lg)) =
              pack_part(rt[i].o[2 * j], rt[i].o[2 * j + 1], sc);
        if (lg == 0)
          *reinterpret_cast<floatx4*>(ws.part_ml + prow * 4) = floatx4{M, L, Lq, float(e)};
      }
    }
    if (cut && held) {
      const float sc = __builtin_amdgcn_ldexpf(1.0f, -e);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const halfx8 v = pack_part(rt[i].o[2 * j], rt[i].o[2 * j + 1], sc);
        const uint4 w = __builtin_bit_cast(uint4, v);
        hold.h[i][4 * j] = w.x;
        hold.h[i][4 * j + 1] = w.y;
        hold.h[i][4 * j + 2] = w.z;
        hold.h[i][4 * j + 3] = w.w;
      }
      hold.ml[i] = floatx4{M, L, Lq, float(e)};
    }
  }
  // stores drained: the ring's waits count tile copies only (stores may
  // complete out of order with respect to the copies)
  wait_vm<0>();
}

__global__ __launch_bounds__(kWaves * kWave, 1) void attn_main_kernel(MainArgs a, AttnWs ws) {
  __shared__ __attribute__((aligned(1024))) char smem[kMainLds];
  const int b = blockIdx.x;
  // one round trip before the first copy: the range, the unit count and the
  // first unit come in one record
  const WgStart st = load_wg_start(ws.wg_start, b);
  const int lo = st.lo, hi = st.hi;
  const int wid = wave_id();
  const CopyPlan cp = copy_plan(uint32_t(a.hkv) * kD * 2);
  const LaneOffsets lof = lane_offsets();
  char* ring = smem + wid * (kWaveStages * kStageBytes);
  // the ring's LDS address (wave-uniform), for the copies
  const uint32_t ring_lds = __builtin_amdgcn_readfirstlane(
      uint32_t(reinterpret_cast<uintptr_t>((lds_void_t*)ring)));
  const int nunits = st.nunits;

  // the wave walks the units from the one holding the range's first tile; the
  // issue side runs ahead of it
  const int first_unit = st.first_unit;
  Issuer is;
  is.iu = first_unit;
  is.ud = st.u;
  issuer_unit(is, a, wid);
  // (after the set-up, so that its loads are issued with the record's)
  if (lo >= hi) return;
  is.k = 0;
  is.copied = 0u;
#pragma unroll
  for (int s = 0; s < kWaveStages; ++s) issue_next(is, a, ws, nunits, lo, hi, wid, ring_lds, cp);

  HeldPartial hp;
  hp.mt = 0;
  hp.rows = 0;
  hp.prow0 = 0;
  int u = first_unit;
  Unit ud = st.u;
  while (true) {
    const int seg_lo = max(lo, ud.tile_start);
    const int seg_hi = min(hi, ud.tile_end);
    const Stream sm = stream_of(ud, wid, a.hkv, a.G);
    const int mt = (sm.rows + 15) / 16;
    // the first segment of a cut unit that began before this range, with more
    // segments after it: its partial is held (wave-uniform)
    const bool held = ud.cut != 0 && ud.tile_start < lo && ud.tile_end < hi;
    if (mt == 0) {
      // empty stream: nothing was copied for these tiles; keep the ring moving
      for (int t = seg_lo; t < seg_hi; ++t) issue_next(is, a, ws, nunits, lo, hi, wid, ring_lds, cp);
    } else if (mt == 1) {
      run_segment<1>(a, ws, ud, sm, seg_lo, seg_hi, lo, hi, nunits, b, ring, ring_lds, is, cp, lof,
                     held, hp);
    } else if (mt == 2) {
      run_segment<2>(a, ws, ud, sm, seg_lo, seg_hi, lo, hi, nunits, b, ring, ring_lds, is, cp, lof,
                     held, hp);
    } else if (mt == 3) {
      run_segment<3>(a, ws, ud, sm, seg_lo, seg_hi, lo, hi, nunits, b, ring, ring_lds, is, cp, lof,
                     held, hp);
    } else {
      run_segment<4>(a, ws, ud, sm, seg_lo, seg_hi, lo, hi, nunits, b, ring, ring_lds, is, cp, lof,
                     held, hp);
    }
    if (seg_hi >= hi || u + 1 >= nunits) break;
    u = __builtin_amdgcn_readfirstlane(u + 1);
    ud = load_unit(ws.units, u);
  }
  // the held partial, after the last segment
  const int lane = threadIdx.x & (kWave - 1);
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int i = 0; i < kMaxMT; ++i) {
    const int rho = 16 * i + lr;
    if (i < hp.mt && rho < hp.rows) {
      const size_t prow = hp.prow0 + size_t(rho);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *reinterpret_cast<uint4*>(ws.part_o + prow * kD + part_dim(32 * j + 4 * lg)) =
            make_uint4(hp.h[i][4 * j], hp.h[i][4 * j + 1], hp.h[i][4 * j + 2], hp.h[i][4 * j + 3]);
      if (lg == 0) *reinterpret_cast<floatx4*>(ws.part_ml + prow * 4) = hp.ml[i];
    }
  }
}

// ------------------------------------------------------------- combine ----
template <int NR>
__global__ __launch_bounds__(kThreads) void attn_combine_kernel(int hq, int hkv, int G, AttnWs ws,
                                                                float* __restrict__ out,
                                                                float* __restrict__ lse) {
  combine_body<NR>(hq, hkv, G, ws, out, lse, blockIdx.x);
}

int main_workgroups() { return device_cu_count(); }

}  // namespace

size_t attn_workspace_bytes(int32_t R, int32_t max_rows, int32_t hq, int32_t hkv) {
  return attn_ws_total(unit_capacity(R, max_rows, hq, hkv), main_workgroups());
}

namespace {

// The attention's launches; the plan (and a paged cache's page check) only if
// `plan`, else the plan of the fused step's front kernel is in the workspace;
// the combine only if `combine`, else the fused step's tail kernel runs it.
int32_t launch_attn_impl(const AttnArgs& a, bool plan, bool combine, hipStream_t stream) {
  (void)hipGetLastError();  // clear errors left by unrelated runtime calls
  const int nb = main_workgroups();
  const size_t ucap = unit_capacity(a.R, a.max_rows, a.hq, a.hkv);
  AttnWs ws = attn_layout(a.workspace, ucap, nb);
  const int G = a.hq / a.hkv;
  KvSource kv;
  kv.kv_offsets = a.kv_offsets;
  kv.kv_rows = static_cast<long long>(a.kv_rows);
  kv.block_table = a.block_table;
  kv.prefix_len = a.prefix_len;
  kv.page_size = a.page_size;
  kv.max_pages = a.max_pages;
  kv.num_pages = static_cast<long long>(a.num_pages);
  kv.page_bad = nullptr;
  kv.page_chunks = 0;
  if (plan && a.block_table != nullptr) {
    // the flags borrow the start of the partials, which the main kernel only
    // writes later on the same stream
    kv.page_chunks = (a.max_pages + kPageChunk - 1) / kPageChunk;
    if (size_t(a.R) * size_t(kv.page_chunks) * 4 > part_rows(nb) * kD * sizeof(_Float16))
      return ECHO_ERR_UNSUPPORTED;
    kv.page_bad = reinterpret_cast<const int32_t*>(ws.part_o);
    hipLaunchKernelGGL(attn_pages_kernel, dim3(unsigned(a.R), unsigned(kv.page_chunks)),
                       dim3(kPageChunk), 0, stream, kv);
  }
  if (plan)
    hipLaunchKernelGGL(attn_plan_kernel, dim3(1), dim3(kThreads),
                       plan_table_words(a.R < kThreads ? a.R : kThreads) * sizeof(int32_t), stream,
                       a.q_offsets, kv, a.R, a.hkv, G, a.max_rows, nb,
                       static_cast<long long>(ucap), ws, a.status);
  MainArgs m;
  m.q = a.q;
  m.k_new = a.k_new;
  m.v_new = a.v_new;
  m.k_cache = a.k_cache;
  m.v_cache = a.v_cache;
  m.block_table = a.block_table;
  m.page_shift = 0;
  if (a.block_table != nullptr)
    while ((1 << m.page_shift) < a.page_size) ++m.page_shift;
  m.max_pages = a.max_pages;
  m.tree_mask = a.tree_mask;
  m.W = a.mask_words;
  m.hq = a.hq;
  m.hkv = a.hkv;
  m.G = G;
  m.scale2 = a.sm_scale * kLog2e;
  m.out = a.out;
  m.lse = a.lse;
  // the measurement events (timed entry points only) travel with the dispatch;
  // they still leave a few microseconds of idle time around the kernel, so a
  // step timed for throughput runs without them
  void* main_args[] = {&m, &ws};
  if (hipExtLaunchKernel(reinterpret_cast<const void*>(&attn_main_kernel), dim3(unsigned(nb)),
                         dim3(kWaves * kWave), main_args, 0, stream, a.ev_start, a.ev_stop,
                         0) != hipSuccess)
    return ECHO_ERR_HIP;
  // cut units number fewer than the main kernel's workgroups
  if (combine) {
    const long long cache_rows = a.block_table == nullptr
                                     ? static_cast<long long>(a.kv_rows)
                                     : static_cast<long long>(a.num_pages) * a.page_size;
    if (combine_rows_per_thread(a.R, a.max_rows, a.hq, a.hkv, nb, cache_rows) == 1)
      hipLaunchKernelGGL(attn_combine_kernel<1>, dim3(unsigned(nb * combine_blocks<1>())),
                         dim3(kThreads), 0, stream, a.hq, a.hkv, G, ws, a.out, a.lse);
    else
      hipLaunchKernelGGL(attn_combine_kernel<2>, dim3(unsigned(nb * combine_blocks<2>())),
                         dim3(kThreads), 0, stream, a.hq, a.hkv, G, ws, a.out, a.lse);
  }
  return hipGetLastError() == hipSuccess ? ECHO_OK : ECHO_ERR_HIP;
}

}  // namespace

int32_t launch_tree_verify_attn(const AttnArgs& a, hipStream_t stream) {
  return launch_attn_impl(a, true, true, stream);
}

int32_t launch_tree_verify_attn_main(const AttnArgs& a, hipStream_t stream) {
  return launch_attn_impl(a, false, false, stream);
}

}  // namespace echo
