// Query-block attention over the packed Distance-KV cache (Sec. 3.4: after
// the one-time compaction the query tokens attend to the compressed context,
// while their own K/V are appended like every new token and kept).
//
// Rows.  Segment s = (sequence b, KV head g) has R = n_q * G query rows; row
// r is token r / G of query head g * G + r % G and sees the segment's first
// seg_len + n_tail + r / G + 1 rows (the packed context, the tokens appended
// before the block, and the block causally up to its own token).
//
// Work split.  A workgroup (8 waves of 32 rows) takes one item: 256 query
// rows (a query tile) of one segment and one key range.  Each segment's
// keys are cut into max(1, round(tiles / C)) near-equal ranges of whole
// 64-key tiles, C the same for every segment, so items are about equally
// long however unequal the segments are.  A one-workgroup plan kernel counts
// the ranges and lays the items out segment by segment, range by range,
// query tile fastest; the workgroups of one hardware L2 domain (ids equal
// mod 8) take consecutive items, so the query tiles of a key range read it
// through the same L2.  With one range a workgroup writes the output; with
// several, each range writes (max, sum, unnormalised output) per row and a
// combine kernel folds the ranges in order.  When the keys are too few to
// split at all there is no plan: one workgroup per (segment, query tile).
//
// Per 64-key tile, K and V go from memory straight into LDS (16 bytes per
// lane, two buffers per matrix, a whole tile ahead); every wave then works
// on 32-key halves:
//   * S^T = K Q^T with v_mfma_f32_16x16x32_bf16: 16 K rows from LDS are the
//     A operand, the wave's two 16-row groups (registers) two B operands, so
//     lane (query n, group kg) receives the scores of keys 4kg..4kg+3 of each
//     16-key block.
//   * Online softmax per query row: max over the lane's scores, then over the
//     row's 4 lanes (permlane swaps); probabilities 2^(c s - m) stay fp32
//     until the product.  The reference max m moves only when a half's max
//     exceeds it by more than 2^8, so the accumulators are rarely rescaled.
//   * O += P V with v_mfma_f32_16x16x32_bf16 per 32 keys: the probabilities
//     are the A operand as the scores sit in the lanes (lane (query n, kg)
//     holds keys 4kg..4kg+3 of two 16-key blocks: its eight K slots), split
//     into a bf16 high part and a bf16 remainder (two products, ~16
//     significant bits kept).  The B operand needs, per lane, the same eight
//     keys of one V column; two ds_read_b64_tr_b16 transpose reads fetch them
//     (within each 16-lane group, lanes 4r..4r+3 address row r of a 4 x 16
//     block and lane i receives its column i).
// The two waves on a SIMD play ping-pong: while one issues the products of
// its half, the other runs the softmax and bf16 split of its own, so the
// matrix and the vector units of a SIMD work at once.  Attention here is a
// dense contraction (G * n_q query rows against every key), so it is MFMA
// work, unlike the one-query decode step.
//
// This file is compiled with IEEE mode off and no NaN semantics
// (-mno-amdgpu-ieee -fno-honor-nans): the maxima then need no NaN
// canonicalisation.  With finite inputs no NaN arises anywhere (masked keys
// are -inf and every -inf - x difference feeds a factor of 0 or 1); for NaN
// inputs the outputs are unspecified.

#include <hip/hip_runtime.h>

#include <type_traits>

#include "dkv_device.hpp"
#include "dkv_query.hpp"

namespace dkv {

namespace {

constexpr int kQThreads = 512;
constexpr int kRG = 2;                   // 16-row groups per wave
constexpr int kQRows = kQueryRowsPerWG;  // query rows per workgroup
static_assert(kQRows == kQThreads / kWave * 16 * kRG, "rows per workgroup");
constexpr int kQKeys = 64;               // keys per tile
constexpr float kLazy = 8.f;             // log2 headroom of the lazy running max
constexpr int kPlanThreads = 1024;

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

template <int D>
struct QCfg {
  static constexpr int kRowBytes = D * 2;
  static constexpr int kChunks = D / 32;    // 16-byte chunks of a row per lane (QK)
  static constexpr int kBlocks = D / 16;    // 16-column output blocks per lane
  static constexpr int kRowChunks = D / 8;  // 16-byte chunks per row
  static constexpr int kDma = kQKeys * kRowChunks / kWave / (kQThreads / kWave);  // loads per wave per matrix
  static constexpr int kRec = D + 2;        // floats per partial record row
  static_assert(kDma >= 1, "a tile needs one direct load per wave at least");
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t q_rsrc(const char* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<char*>(((uint64_t)hi << 32) | lo), (short)0,
                                           (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

__device__ __forceinline__ int64_t q_uniform64(int64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Two probabilities as a bf16 pair (round to nearest even) and the bf16 pair
// of what that rounding left out: a + b carries ~16 significant bits.
__device__ __forceinline__ void bf16_split(float x0, float x1, uint32_t& a, uint32_t& b) {
  const f32x2 x = {x0, x1};
  const bf16x2 h = __builtin_convertvector(x, bf16x2);
  const bf16x2 l = __builtin_convertvector(x - __builtin_convertvector(h, f32x2), bf16x2);
  a = __builtin_bit_cast(uint32_t, h);
  b = __builtin_bit_cast(uint32_t, l);
}

// Maximum over the lanes that share (lane % 16).
__device__ __forceinline__ float row4_max(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Key tiles of segment s for its last query row (the most any row sees).
// A negative length marks a segment dkv_compact could not pack: no tiles.
__device__ __forceinline__ int64_t seg_tiles(const QueryParams& p, int s) {
  const int32_t len = p.seg_len[s];
  return len < 0 ? 0 : ((int64_t)len + p.n_tail + p.n_q + kQKeys - 1) / kQKeys;
}

__device__ __forceinline__ int64_t seg_ranges(int64_t tiles, int64_t c) {
  const int64_t r = (tiles + c / 2) / c;
  return r < 1 ? 1 : r;
}

// Plan of the split: with C tiles per range (raised if the ranges would not
// fit the records the workspace holds), ranges per segment and the first
// item of every segment.
__global__ __launch_bounds__(kPlanThreads) void query_plan_kernel(QueryParams p) {
  __shared__ int64_t red[kPlanThreads / kWave + 1];
  const int tid = threadIdx.x;
  int64_t part = 0;
  for (int s = tid; s < p.nseg; s += kPlanThreads) part += seg_tiles(p, s);
  int64_t total_tiles;
  block_exclusive_scan<kPlanThreads>(part, red, &total_tiles);
  // qtiles * sum_s max(1, round(T_s / C)) <= qtiles * (total / C + nseg) <= max_items
  const int64_t room = p.max_items / p.qtiles - p.nseg;  // >= 1 (host)
  int64_t c = p.tiles_per_range;
  const int64_t cmin = (total_tiles + room - 1) / room;
  if (c < cmin) c = cmin;
  int64_t base = 0;
  for (int s0 = 0; s0 < p.nseg; s0 += kPlanThreads) {
    const int s = s0 + tid;
    const int64_t r = s < p.nseg ? seg_ranges(seg_tiles(p, s), c) : 0;
    int64_t sum;
    const int64_t ex = block_exclusive_scan<kPlanThreads>(r, red, &sum);
    if (s < p.nseg) p.plan[kQueryPlanHead + s] = (int32_t)((base + ex) * p.qtiles);
    base += sum;
  }
  if (tid == 0) {
    p.plan[kQueryPlanHead + p.nseg] = (int32_t)(base * p.qtiles);
    p.plan[0] = (int32_t)(base * p.qtiles);
    p.plan[1] = (int32_t)(c < INT32_MAX ? c : INT32_MAX);  // for inspection; no kernel reads it
  }
}

template <int D>
__global__ __launch_bounds__(kQThreads) void query_attn_kernel(QueryParams p) {
  using C = QCfg<D>;
  // two tile buffers per matrix (separate arrays: the compiler then tells the
  // direct loads into one apart from the reads of the other)
  __shared__ __align__(1024) uint16_t k0[kQKeys * D], k1[kQKeys * D];
  __shared__ __align__(1024) uint16_t v0[kQKeys * D], v1[kQKeys * D];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int n16 = lane & 15;
  const int kg = lane >> 4;

  // ---- this workgroup's item: segment, query tile, key tiles ---------------
  int item, s, qt;
  bool single;             // the segment has one range: write the output
  int64_t t_lo, t_hi;      // key tiles [t_lo, t_hi) of the range
  if (p.plan == nullptr) {
    item = blockIdx.x;
    s = item / p.qtiles;
    qt = item - s * p.qtiles;
    single = true;
    t_lo = 0;
    t_hi = seg_tiles(p, s);
  } else {
    // the grid is a multiple of 8 and at least the items, so every item
    // i = x * per + y (x < 8, y < per) has its workgroup 8y + x
    const int total = p.plan[0];
    const int per = (total + 7) / 8;  // items per L2 domain
    const int b = blockIdx.x;
    if (b / 8 >= per) return;
    item = (b % 8) * per + b / 8;
    if (item >= total) return;
    // the segment: the last s with first item <= item
    int lo = 0, hi = p.nseg;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (p.plan[kQueryPlanHead + mid] <= item) lo = mid;
      else hi = mid;
    }
    s = lo;
    const int first = p.plan[kQueryPlanHead + s];
    const int nr = (p.plan[kQueryPlanHead + s + 1] - first) / p.qtiles;
    const int r = (item - first) / p.qtiles;
    qt = item - first - r * p.qtiles;
    single = nr == 1;
    const int64_t tiles = seg_tiles(p, s);
    t_lo = (int64_t)r * tiles / nr;
    t_hi = (int64_t)(r + 1) * tiles / nr;
  }
  const int bseq = s / p.Hkv;
  const int g = s - bseq * p.Hkv;
  if (p.seg_len[s] < 0) {
    // a segment dkv_compact could not pack (one range, so this workgroup
    // owns its query tile's output): no rows to attend, zeros
    for (int i = tid; i < kQRows * D; i += kQThreads) {
      const int rq = qt * kQRows + i / D;
      if (rq >= p.rows) break;
      const int tq = rq / p.G;
      p.out[(((int64_t)bseq * p.n_q + tq) * p.Hq + (int64_t)g * p.G + (rq - tq * p.G)) * D + i % D] = 0.f;
    }
    return;
  }
  const int64_t base_len = q_uniform64((int64_t)p.seg_len[s] + p.n_tail);  // rows every query row sees
  const int64_t row0 = q_uniform64(p.seg_off[s]);

  // this lane's query rows (one per row group) in the score layout, and the keys they see
  int r[kRG], tok[kRG];
  bool row_ok[kRG];
  int64_t limit[kRG];
#pragma unroll
  for (int q = 0; q < kRG; ++q) {
    r[q] = qt * kQRows + wave * 16 * kRG + 16 * q + n16;
    row_ok[q] = r[q] < p.rows;
    tok[q] = row_ok[q] ? r[q] / p.G : 0;
    limit[q] = base_len + tok[q] + 1;
  }
  // this workgroup's keys: the range, up to what its last row sees
  // (all workgroup-uniform; readfirstlane keeps them in scalar registers)
  const int r_last = min(p.rows - 1, qt * kQRows + kQRows - 1);
  const int64_t lim_max = base_len + r_last / p.G + 1;
  const int64_t k_lo = q_uniform64(t_lo * kQKeys);
  const int64_t k_end = t_hi * kQKeys < lim_max ? t_hi * kQKeys : lim_max;
  const int64_t k_hi = q_uniform64(k_end > k_lo ? k_end : k_lo);
  int32_t cut[kRG];  // keys [k_lo, k_lo + cut) count for the row (cut <= the range length)
#pragma unroll
  for (int q = 0; q < kRG; ++q) cut[q] = (int32_t)((limit[q] < k_hi ? limit[q] : k_hi) - k_lo);
  // every row of the workgroup sees all keys below this one
  const int64_t all_see = q_uniform64(base_len + 1 < k_hi ? base_len + 1 : k_hi);

  // Scores are taken with |scale| (a negative scale negates the queries,
  // exactly); a zero scale becomes the smallest normal float, so masked keys
  // (-inf) stay at -inf after scaling.
  const bool qneg = p.scale_log2 < 0.f;
  const float cpos = fmaxf(fabsf(p.scale_log2), 1.17549435e-38f);
  // B operand of QK: query row r, dims 32u + 8kg .. +7
  u32x4 qb[kRG][C::kChunks];
#pragma unroll
  for (int q = 0; q < kRG; ++q) {
    const int hh = r[q] - tok[q] * p.G;
    const char* qrow = reinterpret_cast<const char*>(p.q) +
                       (((int64_t)bseq * p.n_q + tok[q]) * p.Hq + (int64_t)g * p.G + (row_ok[q] ? hh : 0)) *
                           C::kRowBytes;
#pragma unroll
    for (int u = 0; u < C::kChunks; ++u) {
      const u32x4 z = {0u, 0u, 0u, 0u};
      qb[q][u] = row_ok[q] ? *reinterpret_cast<const u32x4*>(qrow + 64 * u + 16 * kg) : z;
      if (qneg) qb[q][u] ^= u32x4{0x80008000u, 0x80008000u, 0x80008000u, 0x80008000u};
    }
  }

  // output accumulators as scalars: a rescale in a branch then updates them
  // in place instead of in a second set of registers
  float o[kRG][C::kBlocks][4];
  float m[kRG], l[kRG];  // reference max of query row n16 (log2 units), this lane's share of its sum
#pragma unroll
  for (int q = 0; q < kRG; ++q) {
#pragma unroll
    for (int b = 0; b < C::kBlocks; ++b) o[q][b][0] = o[q][b][1] = o[q][b][2] = o[q][b][3] = 0.f;
    m[q] = -INFINITY;
    l[q] = 0.f;
  }

  const char* kbase = reinterpret_cast<const char*>(p.k) + row0 * C::kRowBytes;
  const char* vbase = reinterpret_cast<const char*>(p.v) + row0 * C::kRowBytes;
  // LDS layouts (16-byte chunk units; chunk c of key row R is bytes 16c..16c+15):
  //   K: ((R / 16) * kRowChunks + c) * 16 + R % 16   -- 16 rows of one chunk column together
  //   V: ((R / 8) * kRowChunks / 2 + c / 2) * 16 + (R % 8) * 2 + c % 2
  //      -- 8 rows of one 32-byte column pair together
  // The score product's lanes then read 16 consecutive chunks (K) and the
  // transpose reads 32 consecutive 8-byte halves (V): no bank conflicts, and
  // every read is a per-lane base plus a constant.  One wave instruction of
  // the direct loads fills 64 consecutive chunks (lane l chunk l).
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  // byte offsets of this lane's chunk within a tile for the wave's first
  // instruction; instruction i covers the chunks 1 KiB x (waves) x i further
  // on in both layouts, in LDS and in memory alike (the layouts are made of
  // whole 16-row / 8-row blocks)
  uint32_t koff, voff;
  {
    const int qk_ = 4 * wave + (lane >> 4);  // K: (R / 16) * kRowChunks + c
    const int rk = 16 * (qk_ / C::kRowChunks) + (lane & 15);
    koff = (uint32_t)(rk * C::kRowBytes + 16 * (qk_ % C::kRowChunks));
    const int qv = 4 * wave + (lane >> 4);  // V: (R / 8) * kRowChunks / 2 + c / 2
    const int rv = 8 * (qv / (C::kRowChunks / 2)) + ((lane >> 1) & 7);
    voff = (uint32_t)(rv * C::kRowBytes + 16 * (2 * (qv % (C::kRowChunks / 2)) + (lane & 1)));
  }
  // Global -> LDS: K or V rows [kt, kt + kQKeys) of the segment into a tile
  // buffer.  Keys past k_hi (a whole tile past it included) read zeros
  // without touching memory, so the loads are issued unconditionally.
  auto issue = [&](const char* base, uint32_t off, int64_t kt, uint16_t* buf) __attribute__((always_inline)) {
    const int64_t left = k_hi - kt;
    const uint32_t nk = (uint32_t)(left <= 0 ? 0 : (left < kQKeys ? left : kQKeys));
    const __amdgpu_buffer_rsrc_t rs = q_rsrc(base + kt * C::kRowBytes, nk * C::kRowBytes);
#pragma unroll
    for (int i = 0; i < C::kDma; ++i) {
      const int mi = i * (kQThreads / kWave) + wave_u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(buf + 512 * mi), 16, off,
                                               1024 * (kQThreads / kWave) * i, 0, 0);
    }
  };

  // Scores S^T = K Q^T of half h (keys 32h .. 32h + 31) of the tile in kb:
  // lane (n16, kg) reads K row 16j + n16, chunk 4u + kg, i.e. chunk index
  // (j * kRowChunks + 4u + kg) * 16 + n16 = lane + 16 (j kRowChunks + 4u).
  // Four independent accumulation chains (two key blocks x two row groups).
  auto qk = [&](const uint16_t* kb, int h, float (&sc)[kRG][2][4]) __attribute__((always_inline)) {
    f32x4 acc[2][kRG];
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
      for (int q = 0; q < kRG; ++q) acc[jj][q] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < C::kChunks; ++u)
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int j = 2 * h + jj;
        const u32x4 a = *reinterpret_cast<const u32x4*>(&kb[8 * (lane + 16 * (j * C::kRowChunks + 4 * u))]);
#pragma unroll
        for (int q = 0; q < kRG; ++q)
          acc[jj][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                               __builtin_bit_cast(bf16x8, qb[q][u]), acc[jj][q], 0, 0, 0);
      }
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
      for (int q = 0; q < kRG; ++q)
#pragma unroll
        for (int v = 0; v < 4; ++v) sc[q][jj][v] = acc[jj][q][v];
  };

  // Online softmax of a half whose first key is kh: the raw scores become
  // the probabilities 2^(c s - m), m and l move on, alpha is each row's
  // rescale factor.  The reference max m is lazy: it moves only when a
  // half's max exceeds it by more than kLazy (log2 units), so probabilities
  // stay below 2^kLazy and the accumulators are rescaled only then.
  auto softmax = [&](auto masked, float (&sc)[kRG][2][4], int64_t kh, float (&alpha)[kRG])
                     __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < kRG; ++q) {
      // keys past a row's causal limit or past the range: only in the
      // halves that reach min over rows of that limit
      if (decltype(masked)::value && kh + 32 > all_see) {
        const int32_t lim = cut[q] - (int32_t)(kh - k_lo);  // keys [0, lim) of this half count
#pragma unroll
        for (int jj = 0; jj < 2; ++jj)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (16 * jj + 4 * kg + v >= lim) sc[q][jj][v] = -INFINITY;
      }
      float mx = sc[q][0][0];
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int v = 0; v < 4; ++v) mx = fmaxf(mx, sc[q][jj][v]);
      mx = row4_max(mx) * cpos;
      const bool grow = mx > m[q] + kLazy;
      alpha[q] = fast_exp2(grow ? m[q] - mx : 0.f);
      m[q] = grow ? mx : m[q];
      const float m_use = m[q] == -INFINITY ? 0.f : m[q];
      float ps = 0.f;
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          sc[q][jj][v] = fast_exp2(__builtin_fmaf(sc[q][jj][v], cpos, -m_use));
          ps += sc[q][jj][v];
        }
      l[q] = l[q] * alpha[q] + ps;
      // an empty operand barrier: the sum is formed here, in the vector
      // phase, instead of being sunk into a later one (which unbalances the
      // phases and keeps the probabilities alive across them)
      asm volatile("" : "+v"(l[q]));
    }
  };

  // O *= alpha per row.  Output rows of this lane are queries 4kg + v of the
  // group: their factors live in the lanes of those rows.  The wave skips
  // the rescale unless a factor differs from 1.
  auto rescale = [&](const float (&alpha)[kRG]) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < kRG; ++q) {
      if (__builtin_amdgcn_ballot_w64(alpha[q] != 1.f)) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float av = __shfl(alpha[q], 4 * kg + v, 64);
#pragma unroll
          for (int b = 0; b < C::kBlocks; ++b) o[q][b][v] *= av;
        }
      }
    }
  };

  // Probabilities of a half as the A operand of P V: K slot e of lane group
  // kg is key 4kg + e (e < 4) or 16 + 4kg + (e - 4) of the half, the lane's
  // scores of its two 16-key blocks; high part and remainder.
  auto split = [&](const float (&sc)[kRG][2][4], u32x4 (&ph)[kRG], u32x4 (&pl)[kRG]) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < kRG; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        uint32_t x, y;
        bf16_split(sc[q][e >> 1][2 * (e & 1)], sc[q][e >> 1][2 * (e & 1) + 1], x, y);
        ph[q][e] = x;
        pl[q][e] = y;
      }
  };

  // O += P V over half h of the tile whose V is in vb; each V fragment
  // serves both row groups.  Transpose-read addresses: lane 4r + q of group
  // kg reads row R = 32h + 4kg + r (and R + 16), columns 16b + 4q .. +3, i.e.
  // chunk c = 2b + q / 2, half q % 2: chunk index
  // ((4h + kg / 2) * kRowChunks / 2 + b) * 16 + (4 (kg % 2) + r) * 2 + q / 2.
  // Two V blocks at a time: the high parts of both, then the remainders, so
  // a product never waits for the one just before it.
  auto pv = [&](const uint16_t* vb, int h, const u32x4 (&ph)[kRG], const u32x4 (&pl)[kRG])
                __attribute__((always_inline)) {
    const uint16_t* vr0 = &vb[8 * ((4 * h + (kg >> 1)) * (C::kRowChunks / 2) * 16 + (4 * (kg & 1) + (n16 >> 2)) * 2 +
                                   ((n16 >> 1) & 1)) + 4 * (n16 & 1)];
#pragma unroll
    for (int b0 = 0; b0 < C::kBlocks; b0 += 2) {
      u32x4 vbo[2];
#pragma unroll
      for (int bb = 0; bb < 2; ++bb) {
        const int b = b0 + bb;
        const s16x4 t0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vr0 + 8 * 16 * b));
        const s16x4 t1 =
            __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vr0 + 8 * 16 * (2 * (C::kRowChunks / 2) + b)));
        const uint2 w0 = __builtin_bit_cast(uint2, t0);
        const uint2 w1 = __builtin_bit_cast(uint2, t1);
        vbo[bb] = u32x4{w0.x, w0.y, w1.x, w1.y};
      }
#pragma unroll
      for (int part = 0; part < 2; ++part)
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
#pragma unroll
          for (int q = 0; q < kRG; ++q) {
            const int b = b0 + bb;
            f32x4 c = {o[q][b][0], o[q][b][1], o[q][b][2], o[q][b][3]};
            c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, part ? pl[q] : ph[q]),
                                                        __builtin_bit_cast(bf16x8, vbo[bb]), c, 0, 0, 0);
            o[q][b][0] = c[0];
            o[q][b][1] = c[1];
            o[q][b][2] = c[2];
            o[q][b][3] = c[3];
          }
    }
  };

  // Ping-pong over 32-key halves.  Each wave alternates a product phase
  // (P V products of half g, then score products of half g + 1) with a
  // vector phase (softmax, rescale and bf16 split of half g + 1), and the
  // waves meet after every phase.  Waves w and w + 4 share a SIMD (waves are
  // dealt to the four SIMDs in turn); waves 0-3 (lead) run one phase ahead
  // of waves 4-7 (follow), so on every SIMD one wave issues matrix products
  // while the other does vector work, and the product wave runs at raised
  // priority.  A meeting is a bare s_barrier that nothing is scheduled
  // across: LDS reads of a phase are consumed by its own products before the
  // meeting, and tile loads are made visible by each wave's own vmcnt wait
  // before the meeting that precedes their first reader (a workgroup fence
  // here would wait for every direct load in flight, including the tile
  // just issued).
  auto meet = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_sched_barrier(0);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_sched_barrier(0);
  };
  uint16_t* const kbuf[2] = {k0, k1};
  uint16_t* const vbuf[2] = {v0, v1};
  const bool lead = __builtin_amdgcn_readfirstlane(wave < 4 ? 1 : 0) != 0;
  issue(kbase, koff, k_lo, kbuf[0]);
  issue(vbase, voff, k_lo, vbuf[0]);
  issue(kbase, koff, k_lo + kQKeys, kbuf[1]);
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  __syncthreads();
  float sc[kRG][2][4], al[kRG];
  u32x4 ph[kRG], pl[kRG];
  constexpr int kWaitOne = 0x0F70 | C::kDma;  // vmcnt(kDma): the younger of two tiles may still be in flight
  auto vphase = [&](auto masked, int64_t kh) __attribute__((always_inline)) {
    softmax(masked, sc, kh, al);
    rescale(al);
    split(sc, ph, pl);
  };
  // P V first: the probabilities are dead before the new scores are formed
  auto mphase = [&](const uint16_t* kb, int hk, const uint16_t* vb, int hv, bool do_pv) __attribute__((always_inline)) {
    __builtin_amdgcn_s_setprio(1);
    if (do_pv) pv(vb, hv, ph, pl);
    __builtin_amdgcn_sched_barrier(0);
    qk(kb, hk, sc);
    __builtin_amdgcn_s_setprio(0);
  };
  const int64_t ntile = k_hi > k_lo ? (k_hi - k_lo + kQKeys - 1) / kQKeys : 0;
  const int64_t nround = q_uniform64((ntile + 1) / 2);
  // pairs of tiles whose halves (up to 32 keys past the pair) all lie below
  // every row's limit need no masking
  const int64_t clear = all_see - k_lo - 5 * 32;
  int64_t nclear = clear >= 0 ? clear / (2 * kQKeys) + 1 : 0;
  nclear = q_uniform64(nclear < nround ? nclear : nround);
  int64_t kt = k_lo;
  // Tile t (K in kbuf[i], V in vbuf[i]) takes phases 4t + 1 .. 4t + 4.  K of
  // tile t is read in phases 4t .. 4t + 3 and V in 4t + 2 .. 4t + 5; V of
  // tile t + 1 is loaded from phase 4t + 2 on and K of tile t + 2 from
  // 4t + 4 on, each a whole tile before its first reader.  Each group runs
  // its own copy of the loop, so no phase branches on the group (a branch
  // gave the accumulators a second register set).  Both groups meet equally
  // often: every wave passes the same number of barriers.
  auto tile_pair = [&](auto masked, auto leadc) __attribute__((always_inline)) {
    constexpr bool L = decltype(leadc)::value;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      // 4t + 1: lead: vector phase of half 2t; follow: P V of half 2t - 1, scores of 2t
      if (L) vphase(masked, kt);
      else mphase(kbuf[i], 0, vbuf[1 - i], 1, i == 1 || kt != k_lo);
      __builtin_amdgcn_s_waitcnt(kWaitOne);  // V of tile t
      meet();
      // 4t + 2: lead: P V of 2t, scores of 2t + 1; follow: vector phase of 2t
      issue(vbase, voff, kt + kQKeys, vbuf[1 - i]);
      if (L) mphase(kbuf[i], 1, vbuf[i], 0, true);
      else vphase(masked, kt);
      meet();
      // 4t + 3: lead: vector phase of 2t + 1; follow: P V of 2t, scores of 2t + 1
      if (L) vphase(masked, kt + 32);
      else mphase(kbuf[i], 1, vbuf[i], 0, true);
      __builtin_amdgcn_s_waitcnt(kWaitOne);  // K of tile t + 1
      meet();
      // 4t + 4: lead: P V of 2t + 1, scores of 2t + 2; follow: vector phase of 2t + 1
      issue(kbase, koff, kt + 2 * kQKeys, kbuf[i]);
      if (L) mphase(kbuf[1 - i], 0, vbuf[i], 1, true);
      else vphase(masked, kt + 32);
      meet();
      kt += kQKeys;
    }
  };
  auto run = [&](auto leadc) __attribute__((always_inline)) {
    constexpr bool L = decltype(leadc)::value;
    if (L) mphase(kbuf[0], 0, vbuf[0], 0, false);  // scores of half 0
    meet();
    for (int64_t rd = 0; rd < nclear; ++rd) tile_pair(std::false_type{}, leadc);
    for (int64_t rd = nclear; rd < nround; ++rd) tile_pair(std::true_type{}, leadc);
    // the follow group's P V products of the last half (tiles past k_hi hold
    // zeros and all their keys are masked, so the lead's last scores are unused)
    if (!L && nround > 0) pv(vbuf[1], 1, ph, pl);
  };
  if (lead) run(std::true_type{});
  else run(std::false_type{});
  // no direct load may still be writing LDS when the workgroup ends
  __builtin_amdgcn_s_waitcnt(0x0F70);

  // ---- row totals; write the output or this range's record ------------------
  float* rec = p.rec + (int64_t)item * kQRows * C::kRec;
#pragma unroll
  for (int q = 0; q < kRG; ++q) {
    l[q] = lane_xor_sum<16>(l[q]);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int rr = wave * 16 * kRG + 16 * q + 4 * kg + v;  // row within the tile
      const int rq = qt * kQRows + rr;
      const float lq = __shfl(l[q], 4 * kg + v, 64);
      const float mq = __shfl(m[q], 4 * kg + v, 64);
      if (rq < p.rows) {
        if (single) {
          const int tq = rq / p.G;
          float* orow = p.out + (((int64_t)bseq * p.n_q + tq) * p.Hq + (int64_t)g * p.G + (rq - tq * p.G)) * D;
          const float inv = lq > 0.f ? 1.f / lq : 0.f;
#pragma unroll
          for (int b = 0; b < C::kBlocks; ++b) orow[16 * b + n16] = o[q][b][v] * inv;
        } else {
          float* rrow = rec + (int64_t)rr * C::kRec;
          if (n16 == 0) {
            rrow[0] = mq;
            rrow[1] = lq;
          }
#pragma unroll
          for (int b = 0; b < C::kBlocks; ++b) rrow[2 + 16 * b + n16] = o[q][b][v];
        }
      }
    }
  }
}

// Combine kernel: thread item (row, 4 columns) of one (segment, query tile);
// kMergeThreads items per workgroup.  Segments with one range were written
// by the attention kernel.  A thread loads the row's max, sum and 4 columns
// from eight ranges at once (one memory round trip per eight), then folds
// them in range order into
//   M = max_k m_k,  out = sum_k 2^(m_k - M) o_k / sum_k 2^(m_k - M) l_k.
constexpr int kMergeThreads = 256;
constexpr int kMergeBatch = 8;

template <int D>
__global__ __launch_bounds__(kMergeThreads) void query_merge_kernel(QueryParams p) {
  using C = QCfg<D>;
  constexpr int kItems = kQRows * (D / 4);        // items per query tile
  constexpr int kParts = kItems / kMergeThreads;  // workgroups per query tile
  const int tile = blockIdx.x / kParts;           // s * qtiles + qt
  const int it = (blockIdx.x - tile * kParts) * kMergeThreads + threadIdx.x;
  const int s = tile / p.qtiles;
  const int qt = tile - s * p.qtiles;
  const int rr = it / (D / 4);
  const int c4 = it - rr * (D / 4);
  const int rq = qt * kQRows + rr;
  if (rq >= p.rows) return;
  const int first = p.plan[kQueryPlanHead + s];
  const int nr = (p.plan[kQueryPlanHead + s + 1] - first) / p.qtiles;
  if (nr <= 1) return;
  const int bseq = s / p.Hkv;
  const int g = s - bseq * p.Hkv;
  // record of range k: item first + k * qtiles + qt
  const float* recs = p.rec + ((int64_t)first + qt) * kQRows * C::kRec + (int64_t)rr * C::kRec;
  const int64_t stride = (int64_t)p.qtiles * kQRows * C::kRec;
  float M = -INFINITY, L = 0.f;
  f32x4 A = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < nr; k0 += kMergeBatch) {
    float mk[kMergeBatch], lk[kMergeBatch];
    f32x4 ak[kMergeBatch];
#pragma unroll
    for (int k = 0; k < kMergeBatch; ++k) {
      if (k0 + k < nr) {
        const float* r = recs + (int64_t)(k0 + k) * stride;
        mk[k] = r[0];
        lk[k] = r[1];
        ak[k] = *reinterpret_cast<const f32x4*>(r + 2 + 4 * c4);
      } else {
        mk[k] = -INFINITY;
        lk[k] = 0.f;
        ak[k] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
    float Mn = M;
#pragma unroll
    for (int k = 0; k < kMergeBatch; ++k) Mn = fmaxf(Mn, mk[k]);
    const float Mu = Mn == -INFINITY ? 0.f : Mn;
    const float fo = fast_exp2(M - Mu);
    L *= fo;
    A *= fo;
#pragma unroll
    for (int k = 0; k < kMergeBatch; ++k) {
      const float f = fast_exp2(mk[k] - Mu);
      L += f * lk[k];
      A += f * ak[k];
    }
    M = Mn;
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  const int tq = rq / p.G;
  float* orow = p.out + (((int64_t)bseq * p.n_q + tq) * p.Hq + (int64_t)g * p.G + (rq - tq * p.G)) * D;
  *reinterpret_cast<f32x4*>(orow + 4 * c4) = A * inv;
}

template <int D>
hipError_t launch_d(const QueryParams& p, int64_t grid, hipStream_t stream) {
  if (p.plan != nullptr) hipLaunchKernelGGL(query_plan_kernel, dim3(1), dim3(kPlanThreads), 0, stream, p);
  hipLaunchKernelGGL((query_attn_kernel<D>), dim3((unsigned)grid), dim3(kQThreads), 0, stream, p);
  if (p.plan != nullptr) {
    const int64_t parts = (int64_t)kQRows * (D / 4) / kMergeThreads;
    hipLaunchKernelGGL((query_merge_kernel<D>), dim3((unsigned)((int64_t)p.nseg * p.qtiles * parts)),
                       dim3(kMergeThreads), 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace

QueryPlanShape query_plan_shape(int32_t nseg, int32_t rows, int32_t head_dim, int64_t rows_hint) {
  QueryPlanShape sh;
  sh.qtiles = (rows + kQRows - 1) / kQRows;
  const int64_t units = (int64_t)nseg * sh.qtiles;
  // key tiles of all segments: the hint's rows, or (unknown) a long context
  const int64_t hint = rows_hint < ((int64_t)1 << 40) ? rows_hint : ((int64_t)1 << 40);
  const int64_t tiles = hint > 0 ? (hint + kQKeys - 1) / kQKeys + nseg : (int64_t)nseg * kQueryUnknownTiles;
  sh.tiles_per_range = (sh.qtiles * tiles + kQueryTargetItems - 1) / kQueryTargetItems;
  if (sh.tiles_per_range < kQueryMinTiles) sh.tiles_per_range = kQueryMinTiles;
  if (sh.tiles_per_range > ((int64_t)1 << 30)) sh.tiles_per_range = (int64_t)1 << 30;
  // segments of fewer than two ranges' worth of keys on average: no split
  if (tiles < (int64_t)nseg * 2 * kQueryMinTiles) {
    sh.max_items = units;
    sh.plan_bytes = 0;
    sh.rec_bytes = 0;
    return sh;
  }
  // sum_s max(1, round(T_s / C)) <= tiles / C + nseg for the hinted tiles;
  // the plan kernel raises C if the real keys would need more
  // (launched as a multiple of 8 workgroups: items are dealt to the 8 L2
  // domains in runs of ceil(items / 8))
  sh.max_items = (sh.qtiles * (tiles / sh.tiles_per_range + nseg + 1) + 7) / 8 * 8;
  sh.plan_bytes = ((size_t)(kQueryPlanHead + nseg + 1) * sizeof(int32_t) + 255) / 256 * 256;
  sh.rec_bytes = (size_t)sh.max_items * kQRows * (head_dim + 2) * sizeof(float);
  return sh;
}

hipError_t launch_query_attn(const QueryParams& p, int head_dim, int64_t grid, hipStream_t stream) {
  return head_dim == 64 ? launch_d<64>(p, grid, stream) : launch_d<128>(p, grid, stream);
}

}  // namespace dkv
