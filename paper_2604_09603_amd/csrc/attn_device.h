// Verification attention, the part shared by the attention launches and the
// fused step's front kernel: constants, the workspace layout, streams and
// units, and the plan that cuts the units' tiles into one range per workgroup
// of the main kernel.
#pragma once

#include "echo_device.h"
#include "echo_internal.h"

namespace echo {
namespace {

constexpr int kD = ECHO_HEAD_DIM;   // 128
constexpr int kThreads = 256;       // plan / combine workgroups
constexpr int kWaves = 4;           // main kernel: waves (streams) per workgroup, one per CU
constexpr int kMaxMT = 4;           // 16-row tiles per stream (394 of the 512 registers a wave has)
constexpr int kPassRows = kMaxMT * 16;  // rows per stream (64)
constexpr int kWaveStages = 2;      // per-wave LDS ring depth (32-key K+V tiles)
constexpr int kTileKeys = 32;       // keys per tile
constexpr int kMaskWords = 2;       // tree-tail mask words preloaded per row and segment
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// The softmax reference max is raised only when a logit exceeds it by more than
// 2^8 (in the exponent): probabilities stay <= 256, exact after normalisation.
constexpr float kRescaleSlack = 8.0f;
// A tile whose largest probability in a row exceeds this fraction of the
// row's running sum also multiplies V by the bf16 residual p - bf16(p) (see
// compute_tile).
constexpr float kSplitFrac = 1.0f / 16.0f;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// One unit of the tile stream: a group of four streams of one request.
// Stream s = 4 * group + w runs KV head s / passes over the rows of pass
// s % passes; s >= hkv * passes is empty.
struct Unit {
  int32_t tile_start, tile_end;  // global tile range: ntail tail tiles, then prefix tiles
  int32_t q0, nslots;            // the request's verify slots
  int32_t kb, P;                 // KV prefix rows [kb, kb + P)
  int32_t ntail, passes;         // ceil(nslots / 32); row passes per KV head
  int32_t rpp, group;            // rows per pass (the last pass may have fewer); stream group
  int32_t cut, pad;              // cut: covered by more than one workgroup
};

struct Cut {
  int32_t unit, b0, b1, first_slot;  // workgroups b0..b1; partial slot of b0's segment
  Unit u;                            // the unit itself (the merge needs no second lookup)
};

// What a workgroup of the main kernel needs before its first copy, in one
// 64-byte record: its tile range [lo, hi) (lo == hi: no work), the number of
// units, the unit holding tile lo and a copy of that unit.
struct WgStart {
  int32_t lo, hi, nunits, first_unit;
  Unit u;
};

struct AttnWs {
  int32_t* meta;   // [0] units, [1] tiles, [2] cut units, [3] workgroups with work
  Unit* units;
  WgStart* wg_start;  // [nb], written for every workgroup by each plan
  Cut* cuts;
  // partials of the cut units: [2 * nb * 4 * 64][4] reference max (log2 units),
  // sum, rounded sum and the exponent e of the row's scale; [2 * nb * 4 * 64][128]
  // the row's unnormalised output times 2^-e in fp16 (e puts the row's largest
  // magnitude in [2^14, 2^15))
  float* part_ml;
  _Float16* part_o;
};

__host__ __device__ inline size_t al(size_t x) { return (x + 255) / 256 * 256; }

// Row passes of a request with fewer KV heads than a unit has waves: enough to
// give every wave of its units a stream (see request_shape).
__host__ __device__ inline int fill_passes(int hkv) { return (kWaves + hkv - 1) / hkv; }

// Units never exceed one per request plus one per four streams; a request has at
// most ceil(rows / 64) or fill_passes(hkv) passes per KV head.
__host__ inline size_t unit_capacity(int R, int max_rows, int hq, int hkv) {
  const size_t passes = size_t(R) * size_t(fill_passes(hkv)) +
                        (size_t(max_rows) * (hq / hkv) + kPassRows - 1) / kPassRows;
  return size_t(R) + (size_t(hkv) * passes + kWaves - 1) / kWaves;
}

__host__ __device__ inline size_t part_rows(int nb) {
  return size_t(2) * nb * kWaves * kPassRows;
}

__host__ __device__ inline AttnWs attn_layout(void* base, size_t ucap, int nb) {
  char* p = static_cast<char*>(base);
  AttnWs w;
  w.meta = reinterpret_cast<int32_t*>(p);
  p += 256;
  w.units = reinterpret_cast<Unit*>(p);
  p += al(ucap * sizeof(Unit));
  w.wg_start = reinterpret_cast<WgStart*>(p);
  p += al(size_t(nb) * sizeof(WgStart));
  w.cuts = reinterpret_cast<Cut*>(p);
  p += al(size_t(nb) * sizeof(Cut));
  w.part_ml = reinterpret_cast<float*>(p);
  p += al(part_rows(nb) * 4 * sizeof(float));
  w.part_o = reinterpret_cast<_Float16*>(p);
  return w;
}

__host__ inline size_t attn_ws_total(size_t ucap, int nb) {
  return 256 + al(ucap * sizeof(Unit)) + al(size_t(nb) * sizeof(WgStart)) +
         al(size_t(nb) * sizeof(Cut)) +
         al(part_rows(nb) * 4 * 4) + al(part_rows(nb) * kD * 2);
}

// Partial row of (workgroup b, slot, stream w, row rho).
__device__ __forceinline__ size_t part_row(int b, int slot, int w, int rho) {
  return (size_t(2 * b + slot) * kWaves + w) * kPassRows + rho;
}

// floor(n / d) for 0 <= n < 2^42 and 0 < d < 2^31, without a 64-bit integer
// division: the quotient through d's double reciprocal is within one of the
// floor (the product's error is below 2^-9), and one integer step corrects it.
struct DivBy {
  long long d;
  double inv;
  __device__ explicit DivBy(long long d_) : d(d_), inv(1.0 / double(d_)) {}
  __device__ __forceinline__ long long operator()(long long n) const {
    long long q = static_cast<long long>(double(n) * inv);
    if (q * d > n) --q;
    else if ((q + 1) * d <= n) ++q;
    return q;
  }
};

// First tile of workgroup b when T tiles are cut into nw equal ranges (nw <= T).
__device__ __forceinline__ long long range_lo(long long T, int b, int nw) { return T * b / nw; }
__device__ __forceinline__ long long range_lo(long long T, int b, const DivBy& by_nw) {
  return by_nw(T * b);
}
// Workgroup whose range holds tile t.
__device__ __forceinline__ int range_of(long long t, long long T, int nw, const DivBy& by_t) {
  return int(by_t((t + 1) * nw + T - 1)) - 1;
}

// The rows of stream w of a unit: KV head, first row and row count (rows == 0:
// the stream is empty).
struct Stream {
  int kvh, row0, rows;
};

__device__ __forceinline__ Stream stream_of(const Unit& u, int w, int hkv, int G) {
  Stream s = {0, 0, 0};
  const int id = kWaves * u.group + w;
  if (u.passes <= 0 || id >= hkv * u.passes) return s;
  s.kvh = id / u.passes;
  s.row0 = (id % u.passes) * u.rpp;
  s.rows = min(u.rpp, u.nslots * G - s.row0);
  return s;
}

// ---------------------------------------------------------------- plan ----
// Where the requests' KV prefixes live: rows [kv_offsets[r], kv_offsets[r+1])
// of a token-major cache, or (block_table != nullptr) prefix_len[r] positions
// read through the request's row of the block table.
struct KvSource {
  const int64_t* kv_offsets;
  long long kv_rows;
  const int32_t* block_table;
  const int32_t* prefix_len;
  int page_size;
  int max_pages;
  long long num_pages;
  const int32_t* page_bad;  // [R][page_chunks]: written by attn_pages, read by the plan
  int page_chunks;
};

constexpr int kPageChunk = 256;  // page ids checked per attn_pages workgroup

// What the plan reads of request r, loaded together: its slot range and its
// prefix (a contiguous prefix's rows [k0, k1); a paged one's length P).
struct RequestIn {
  int q0, q1;
  long long k0, k1, P;
};

__device__ __forceinline__ RequestIn load_request(const int32_t* q_offsets, const KvSource& kv,
                                                  int r) {
  RequestIn in;
  in.q0 = q_offsets[r];
  in.q1 = q_offsets[r + 1];
  if (kv.block_table == nullptr) {
    in.k0 = kv.kv_offsets[r];
    in.k1 = kv.kv_offsets[r + 1];
    in.P = in.k1 - in.k0;
  } else {
    in.k0 = 0;
    in.k1 = 0;
    in.P = kv.prefix_len[r];
  }
  return in;
}

// Slot range and prefix extent of a request are usable (for a paged prefix: its
// length fits its block-table row; the page ids are checked separately).
__device__ __forceinline__ bool request_ok(const RequestIn& in, const KvSource& kv, int max_rows) {
  if (!(in.q0 >= 0 && in.q1 >= in.q0 && in.q1 <= max_rows)) return false;
  if (kv.block_table == nullptr) return in.k0 >= 0 && in.k1 >= in.k0 && in.k1 <= kv.kv_rows;
  return in.P >= 0 && in.P <= (long long)kv.max_pages * kv.page_size;
}

struct RequestShape {
  int groups, tiles, q0, nsl, kb, P, ntail, passes, rpp;
};

// A request's rows per head split into passes of at most 64 rows, as even as
// possible; its hkv * passes streams form ceil(/4) groups over the same tiles.
// With fewer KV heads than a unit has waves (one KV head, or a tensor-parallel
// share of a few), that would leave waves idle: the rows are then split into
// fill_passes(hkv) passes (at least one row each), whose streams read the same
// head's tiles and share them in the caches.
// `ok` is request_ok of request r (evaluated once per plan).  A paged request's
// kb is its index (its block table row), a contiguous one's its first row.
__device__ __forceinline__ RequestShape request_shape(const RequestIn& in, const KvSource& kv,
                                                      bool ok, int R, int hkv, int G, int r) {
  RequestShape s = {0, 0, 0, 0, 0, 0, 0, 0, 0};
  if (r >= R || !ok) return s;
  s.q0 = in.q0;
  s.nsl = in.q1 - in.q0;
  s.kb = kv.block_table == nullptr ? int(in.k0) : r;
  s.P = int(in.P);
  const int rows = s.nsl * G;
  s.passes = (rows + kPassRows - 1) / kPassRows;
  if (s.passes == 0) return s;
  s.passes = max(s.passes, min(rows, fill_passes(hkv)));
  s.rpp = (rows + s.passes - 1) / s.passes;
  s.ntail = (s.nsl + kTileKeys - 1) / kTileKeys;
  s.groups = (hkv * s.passes + kWaves - 1) / kWaves;
  s.tiles = s.ntail + (s.P + kTileKeys - 1) / kTileKeys;
  return s;
}

// request_shape of request r, its fields loaded here (r < R).
__device__ __forceinline__ RequestShape request_shape_at(const int32_t* q_offsets,
                                                         const KvSource& kv, bool ok, int R,
                                                         int hkv, int G, int r) {
  if (r >= R || !ok) return RequestShape{0, 0, 0, 0, 0, 0, 0, 0, 0};
  return request_shape(load_request(q_offsets, kv, r), kv, ok, R, hkv, G, r);
}

// Unit g of a request of shape s whose tiles start at tile tb; b0 and b1: the
// workgroups whose ranges hold its first and its last tile.
__device__ __forceinline__ Unit make_unit(const RequestShape& s, int tb, int g, long long T, int nw,
                                          const DivBy& by_t, int& b0, int& b1) {
  Unit u;
  u.tile_start = tb + g * s.tiles;
  u.tile_end = u.tile_start + s.tiles;
  u.q0 = s.q0;
  u.nslots = s.nsl;
  u.kb = s.kb;
  u.P = s.P;
  u.ntail = s.ntail;
  u.passes = s.passes;
  u.rpp = s.rpp;
  u.group = g;
  b0 = range_of(u.tile_start, T, nw, by_t);
  b1 = range_of(u.tile_end - 1, T, nw, by_t);
  u.cut = b0 != b1;
  u.pad = 0;
  return u;
}

// LDS (32-bit words) for the plan's request tables when it runs with one
// request per thread: tile and unit bases and the shapes of R requests.
__host__ __device__ inline size_t plan_table_words(int R) {
  return size_t(2) * (R + 1) + size_t(R) * (sizeof(RequestShape) / 4);
}

// The plan on one workgroup of NT threads (see attn_plan above): the units,
// each workgroup's start record and the cut units, written to ws; meta[0..3] =
// units, tiles, cut units, workgroups with work.
// * `tables` (may be null): plan_table_words(min(R, NT)) words of LDS.  With it
//   and R <= NT, one thread per workgroup writes the start records, from the
//   request tables; without it, the thread of the request holding a range's
//   first tile writes that range's record.
// * `pre` (may be null): request threadIdx.x's fields as load_request gives
//   them, already in hand (R <= NT).
template <int NT>
__device__ void plan_body(const int32_t* __restrict__ q_offsets, const KvSource& kv, int R, int hkv,
                          int G, int max_rows, int nb, long long ucap, const AttnWs& ws,
                          int32_t* status, int32_t* tables = nullptr,
                          const RequestIn* pre = nullptr) {
  __shared__ int s_scan[NT / kWave + 1];
  __shared__ int2 s_scan2[NT / kWave + 1];
  __shared__ uint8_t s_ok[ECHO_MAX_REQUESTS + 1];
  const int tid = threadIdx.x;
  // one request per thread (R <= 256, the usual case): shapes and their scans
  // are computed once and kept for pass B; the shape is taken with the same
  // loads as the validity check
  const bool single = R <= NT;
  RequestShape s1 = {0, 0, 0, 0, 0, 0, 0, 0, 0};
  int ub1 = 0, tb1 = 0;
  int bits = 0;
  for (int r = tid; r < R; r += NT) {
    const RequestIn in = single && pre != nullptr ? *pre : load_request(q_offsets, kv, r);
    bool ok = request_ok(in, kv, max_rows);
    if (kv.block_table != nullptr)
      for (int c = 0; c < kv.page_chunks; ++c) ok = ok && kv.page_bad[size_t(r) * kv.page_chunks + c] == 0;
    s_ok[r] = ok ? 1 : 0;
    if (!ok) bits |= ECHO_DATA_BAD_OFFSETS;
    if (single) s1 = request_shape(in, kv, ok, R, hkv, G, r);
  }
  __syncthreads();
  auto ok_of = [&](int r) { return r < R && s_ok[r] != 0; };

  // pass A: total units and tiles
  long long T = 0, U = 0;
  for (int base = 0; base < R; base += NT) {
    const RequestShape s =
        single ? s1 : request_shape_at(q_offsets, kv, ok_of(base + tid), R, hkv, G, base + tid);
    int tot_u, tot_t;
    const int2 ex = block_exclusive_sum2<NT>(make_int2(s.groups, s.groups * s.tiles), s_scan2,
                                                   &tot_u, &tot_t);
    if (single) {
      s1 = s;
      ub1 = ex.x;
      tb1 = ex.y;
    }
    U += tot_u;
    T += tot_t;
  }
  // slot ranges that overlap (a non-monotone CSR) could ask for more units than
  // the workspace holds, and tile indices are 32-bit: then nothing is scheduled
  // workgroups with work: never more than tiles, so that no range is empty
  const bool fits = U <= ucap && T <= 0x7FFFFFFFll;
  const int nw = !fits ? 0 : T < nb ? int(T) : nb;
  // the workgroups without work get an empty range
  for (int b = nw + tid; b < nb; b += NT) ws.wg_start[b] = WgStart{};
  if (!fits) {
    if (tid == 0) {
      bits |= ECHO_DATA_BAD_OFFSETS;
      ws.meta[0] = 0;
      ws.meta[1] = 0;
      ws.meta[2] = 0;
      ws.meta[3] = 0;
    }
    wave_status_or(status, bits);
    return;
  }
  wave_status_or(status, bits);
  // pass B: units, the cut units and each workgroup's start record
  const DivBy by_t(T > 0 ? T : 1), by_nw(nw > 0 ? nw : 1);
  const bool by_wg = single && tables != nullptr;
  int32_t* s_tb = tables;             // R + 1: first tile of each request's units, then T
  int32_t* s_ub = tables + (R + 1);   // R: first unit of each request
  RequestShape* s_sh = reinterpret_cast<RequestShape*>(tables + 2 * (R + 1));  // R
  int unit_run = 0, tile_run = 0, cut_run = 0;
  for (int base = 0; base < R; base += NT) {
    RequestShape s;
    int ub, tb, tot_u, tot_t;
    if (single) {
      s = s1;
      ub = ub1;
      tb = tb1;
      tot_u = int(U);
      tot_t = int(T);
    } else {
      s = request_shape_at(q_offsets, kv, ok_of(base + tid), R, hkv, G, base + tid);
      const int2 ex = block_exclusive_sum2<NT>(make_int2(s.groups, s.groups * s.tiles),
                                                     s_scan2, &tot_u, &tot_t);
      ub = unit_run + ex.x;
      tb = tile_run + ex.y;
    }
    // a unit is cut if two workgroup ranges share it
    int ncut = 0;
    for (int g = 0; g < s.groups; ++g) {
      const long long ts = tb + g * s.tiles, te = ts + s.tiles;
      if (range_of(ts, T, nw, by_t) != range_of(te - 1, T, nw, by_t)) ++ncut;
    }
    int tot_c;
    const int cb = cut_run + block_exclusive_sum<NT>(ncut, s_scan, &tot_c);
    if (by_wg && tid < R) {
      s_tb[tid] = tb;
      s_ub[tid] = ub;
      s_sh[tid] = s;
    }
    if (by_wg && tid == 0) s_tb[R] = int(T);
    int c = cb;
    for (int g = 0; g < s.groups; ++g) {
      int b0, b1;
      const Unit u = make_unit(s, tb, g, T, nw, by_t, b0, b1);
      ws.units[ub + g] = u;
      if (u.cut) {
        Cut cu;
        cu.unit = ub + g;
        cu.b0 = b0;
        cu.b1 = b1;
        cu.first_slot = range_lo(T, b0, by_nw) < u.tile_start ? 1 : 0;
        cu.u = u;
        ws.cuts[c++] = cu;
      }
      if (by_wg) continue;
      // workgroups whose range starts inside this unit
      int b = b0;
      long long blo = range_lo(T, b, by_nw);
      if (blo < u.tile_start) {
        ++b;
        blo = range_lo(T, b, by_nw);
      }
      for (; b <= b1; ++b) {
        const long long bhi = range_lo(T, b + 1, by_nw);
        WgStart st;
        st.lo = int(blo);
        st.hi = int(bhi);
        st.nunits = int(U);
        st.first_unit = ub + g;
        st.u = u;
        ws.wg_start[b] = st;
        blo = bhi;
      }
    }
    unit_run += tot_u;
    tile_run += tot_t;
    cut_run += tot_c;
  }
  if (by_wg) {
    // one workgroup per thread: the request holding the range's first tile is
    // the last one whose units start at or before it (requests without tiles
    // share their successor's start)
    __syncthreads();
    for (int b = tid; b < nw; b += NT) {
      const int blo = int(range_lo(T, b, by_nw));
      const int r = upper_bound_idx(s_tb, R + 1, blo);
      const RequestShape s = s_sh[r];
      const int g = s.tiles > 0 ? (blo - s_tb[r]) / s.tiles : 0;
      int b0, b1;
      WgStart st;
      st.lo = blo;
      st.hi = int(range_lo(T, b + 1, by_nw));
      st.nunits = int(U);
      st.first_unit = s_ub[r] + g;
      st.u = make_unit(s, s_tb[r], g, T, nw, by_t, b0, b1);
      ws.wg_start[b] = st;
    }
  }
  if (tid == 0) {
    ws.meta[0] = unit_run;
    ws.meta[1] = int(T);
    ws.meta[2] = cut_run;
    ws.meta[3] = nw;
  }
}

// ------------------------------------------------------------- combine ----
// One thread per (cut unit, stream, NR rows, 4 dims): rows rho, rho + 64 / NR, ...
// of the stream; a cut's items span combine_blocks<NR>() workgroups.  The
// partials are merged in workgroup order.
template <int NR>
constexpr int combine_blocks() {
  static_assert((kWaves * (kPassRows / NR) * (kD / 4)) % kThreads == 0, "combine tiling");
  return kWaves * (kPassRows / NR) * (kD / 4) / kThreads;
}
constexpr int kFastParts = 4;  // cuts over at most this many workgroups merge in one round trip

// Rows per combine thread for a launch.  Two rows per thread load both rows'
// partials in one round trip with half the threads; one row per thread needs
// half the registers, so more waves wait at once.  The second wins when cuts
// span many workgroups (their rows merge in several batches): with U units over
// nb workgroups a cut spans about 1 + nb / U of them.  U is estimated from the
// mean slots per request (max_rows / R), as the plan shapes requests.  With
// fewer tiles than about two per workgroup (kv_rows: the cache's rows, an upper
// bound of the prefixes) most of the grid has no cut to merge, and the smaller
// grid of two rows per thread is kept.
__host__ inline int combine_rows_per_thread(int R, int max_rows, int hq, int hkv, int nb,
                                            long long kv_rows) {
  if (R <= 0 || hkv <= 0) return 2;
  const int rows = (max_rows / R) * (hq / hkv);
  int passes = (rows + kPassRows - 1) / kPassRows;
  passes = passes > 0 ? passes : 1;
  const int fill = fill_passes(hkv) < rows ? fill_passes(hkv) : rows;
  passes = passes > fill ? passes : fill;
  const long long units = (long long)R * ((hkv * passes + kWaves - 1) / kWaves);
  const long long tiles = units * ((kv_rows / R + kTileKeys - 1) / kTileKeys + 1);
  return units * 3 <= nb && tiles >= 2LL * nb ? 1 : 2;
}

typedef _Float16 halfx4 __attribute__((ext_vector_type(4)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
typedef uint32_t uint32x4 __attribute__((ext_vector_type(4)));

// Where dim d of a partial row sits: the main kernel's lane with dims
// 16 dt + 4 g + [0, 4) writes those of dt = 2j and 2j + 1 as 8 consecutive
// halves at 32 j + 8 g, so that one 16-byte store covers both.
__host__ __device__ inline int part_dim(int d) {
  const int dt = d >> 4, g = (d >> 2) & 3;
  return (dt >> 1) * 32 + g * 8 + (dt & 1) * 4 + (d & 3);
}

// Four dims of a partial row, back in the row's fp32 scale (e: its exponent).
__device__ __forceinline__ floatx4 load_part_o(const AttnWs& ws, size_t prow, int d4, float e) {
  const halfx4 h = *reinterpret_cast<const halfx4*>(ws.part_o + prow * kD + part_dim(d4));
  return __builtin_convertvector(h, floatx4) * __builtin_amdgcn_ldexpf(1.0f, int(e));
}

// acc + w * v, fused in every lane: the merges round the same way whatever the
// code around them (the combine's launch shapes give bit-identical rows).
__device__ __forceinline__ floatx4 fma4(float w, const floatx4& v, const floatx4& acc) {
  return floatx4{__builtin_fmaf(w, v[0], acc[0]), __builtin_fmaf(w, v[1], acc[1]),
                 __builtin_fmaf(w, v[2], acc[2]), __builtin_fmaf(w, v[3], acc[3])};
}

// One output row (4 dims) and its LSE from the partials of its parts: (max,
// sum, rounded sum) and O of each (parts with max -inf are absent or empty).
template <int NP>
__device__ __forceinline__ void merge_parts(const floatx4 (&ml)[NP], const floatx4 (&po)[NP],
                                            int np, float* o, float* l) {
  float M = -__builtin_inff();
#pragma unroll
  for (int i = 0; i < NP; ++i)
    if (i < np) M = fmaxf(M, ml[i][0]);
  float L = 0.0f, Lq = 0.0f;
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
  if (M != -__builtin_inff()) {
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      if (i >= np || ml[i][0] == -__builtin_inff()) continue;
      const float wgt = __builtin_amdgcn_exp2f(ml[i][0] - M);
      L = __builtin_fmaf(wgt, ml[i][1], L);
      Lq = __builtin_fmaf(wgt, ml[i][2], Lq);
      acc = fma4(wgt, po[i], acc);
    }
  }
  const float inv = Lq > 0.0f ? 1.0f / Lq : 0.0f;
  __builtin_nontemporal_store(acc * inv, reinterpret_cast<floatx4*>(o));
  if (l != nullptr) *l = L > 0.0f ? (M + log2f(L)) * kLn2 : -__builtin_inff();
}

// Workgroup `block` of the combine (kThreads threads; combine_blocks<NR>() per
// cut unit).
template <int NR>
__device__ __forceinline__ void combine_body(int hq, int hkv, int G, const AttnWs& ws,
                                             float* __restrict__ out, float* __restrict__ lse,
                                             int block) {
  constexpr int kBlocks = combine_blocks<NR>();
  const int ci = block / kBlocks;
  // the cut record (ci < nb: inside the array) is loaded with the cut count, in
  // the same round trip; a workgroup past the count only waits for it to land
  // (the empty asm uses it there, so that the loads are not moved below the test)
  static_assert(sizeof(Cut) == 4 * sizeof(uint32x4), "cut record: four 16-byte loads");
  uint32x4 raw[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) raw[k] = reinterpret_cast<const uint32x4*>(ws.cuts + ci)[k];
  if (ci >= ws.meta[2]) {
    asm volatile("" ::"v"(raw[0]), "v"(raw[1]), "v"(raw[2]), "v"(raw[3]));
    return;
  }
  const Cut c = __builtin_bit_cast(Cut, raw);
  const int e = (block % kBlocks) * kThreads + threadIdx.x;
  constexpr int kRowSpan = kPassRows / NR;
  const int w = e / (kRowSpan * (kD / 4));
  const int rho0 = (e / (kD / 4)) % kRowSpan;
  const int d4 = (e % (kD / 4)) * 4;
  const Unit& u = c.u;
  const Stream sm = stream_of(u, w, hkv, G);
  if (rho0 >= sm.rows) return;
  const int nparts = c.b1 - c.b0 + 1;
  // partial of part i: workgroup b0 + i, whose segment may sit in its second slot
  auto prow_of = [&](int i, int rho) {
    return part_row(c.b0 + i, i == 0 ? c.first_slot : 0, w, rho);
  };
  auto out_row = [&](int rho) {
    const int ra = sm.row0 + rho;
    return size_t(u.q0 + ra / G) * hq + sm.kvh * G + ra % G;
  };
  if (nparts <= kFastParts) {
    // every load of both rows issued at once: one memory round trip
    floatx4 ml[NR][kFastParts], po[NR][kFastParts];
#pragma unroll
    for (int k = 0; k < NR; ++k) {
      const int rho = rho0 + k * kRowSpan;
#pragma unroll
      for (int i = 0; i < kFastParts; ++i) {
        ml[k][i] = floatx4{-__builtin_inff(), 0.0f, 0.0f, 0.0f};
        po[k][i] = floatx4{0.f, 0.f, 0.f, 0.f};
        if (i < nparts && rho < sm.rows) {
          const size_t prow = prow_of(i, rho);
          ml[k][i] = *reinterpret_cast<const floatx4*>(ws.part_ml + prow * 4);
          po[k][i] = load_part_o(ws, prow, d4, ml[k][i][3]);
        }
      }
    }
#pragma unroll
    for (int k = 0; k < NR; ++k) {
      const int rho = rho0 + k * kRowSpan;
      if (rho >= sm.rows) continue;
      const size_t orow = out_row(rho);
      merge_parts<kFastParts>(ml[k], po[k], nparts, out + orow * kD + d4,
                              lse != nullptr && d4 == 0 ? lse + orow : nullptr);
    }
    return;
  }
  // more parts: kFastParts at a time for both rows, in order (the same arithmetic
  // as the fast path; two memory round trips per batch instead of two per part)
  float M[NR], L[NR], Lq[NR];
  floatx4 acc[NR];
#pragma unroll
  for (int k = 0; k < NR; ++k) {
    M[k] = -__builtin_inff();
    L[k] = 0.0f;
    Lq[k] = 0.0f;
    acc[k] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  for (int i0 = 0; i0 < nparts; i0 += kFastParts) {
    float mb[NR][kFastParts];
#pragma unroll
    for (int k = 0; k < NR; ++k)
#pragma unroll
      for (int j = 0; j < kFastParts; ++j) {
        const int rho = rho0 + k * kRowSpan;
        mb[k][j] = i0 + j < nparts && rho < sm.rows ? ws.part_ml[prow_of(i0 + j, rho) * 4]
                                                    : -__builtin_inff();
      }
#pragma unroll
    for (int k = 0; k < NR; ++k)
#pragma unroll
      for (int j = 0; j < kFastParts; ++j) M[k] = fmaxf(M[k], mb[k][j]);
  }
  for (int i0 = 0; i0 < nparts; i0 += kFastParts) {
    floatx4 ml[NR][kFastParts], po[NR][kFastParts];
#pragma unroll
    for (int k = 0; k < NR; ++k)
#pragma unroll
      for (int j = 0; j < kFastParts; ++j) {
        const int rho = rho0 + k * kRowSpan;
        ml[k][j] = floatx4{-__builtin_inff(), 0.0f, 0.0f, 0.0f};
        po[k][j] = floatx4{0.f, 0.f, 0.f, 0.f};
        if (i0 + j < nparts && rho < sm.rows) {
          const size_t prow = prow_of(i0 + j, rho);
          ml[k][j] = *reinterpret_cast<const floatx4*>(ws.part_ml + prow * 4);
          po[k][j] = load_part_o(ws, prow, d4, ml[k][j][3]);
        }
      }
#pragma unroll
    for (int k = 0; k < NR; ++k) {
      if (M[k] == -__builtin_inff()) continue;
#pragma unroll
      for (int j = 0; j < kFastParts; ++j) {
        if (ml[k][j][0] == -__builtin_inff()) continue;
        const float wgt = __builtin_amdgcn_exp2f(ml[k][j][0] - M[k]);
        L[k] = __builtin_fmaf(wgt, ml[k][j][1], L[k]);
        Lq[k] = __builtin_fmaf(wgt, ml[k][j][2], Lq[k]);
        acc[k] = fma4(wgt, po[k][j], acc[k]);
      }
    }
  }
#pragma unroll
  for (int k = 0; k < NR; ++k) {
    const int rho = rho0 + k * kRowSpan;
    if (rho >= sm.rows) continue;
    const size_t orow = out_row(rho);
    const float inv = Lq[k] > 0.0f ? 1.0f / Lq[k] : 0.0f;
    __builtin_nontemporal_store(acc[k] * inv, reinterpret_cast<floatx4*>(out + orow * kD + d4));
    if (lse != nullptr && d4 == 0)
      lse[orow] = L[k] > 0.0f ? (M[k] + log2f(L[k])) * kLn2 : -__builtin_inff();
  }
}

}  // namespace
}  // namespace echo
