// Query-block attention over the packed Distance-KV cache (Sec. 3.4: after
// the one-time compaction the query tokens attend to the compressed context,
// while their own K/V are appended like every new token and kept).
//
// Rows and work split.  Segment s = (sequence b, KV head g) has
// R = n_q * G query rows; row r is token r / G of query head g * G + r % G
// and sees the segment's first seg_len + n_tail + r / G + 1 rows (the packed
// context, the tokens appended before the block, and the block causally up
// to its own token).  A workgroup takes 128 query rows (8 waves of 16) of one
// segment and one of `nsplit` equal key ranges.  With one range it writes the
// output; with several, each range writes (max, sum, unnormalised output)
// per row and a combine kernel folds the ranges in order.
//
// Per 64-key tile (K and V staged through LDS by the whole workgroup; the
// next tile's global loads are in flight while the current one is computed):
//   * S^T = K Q^T with v_mfma_f32_16x16x32_bf16: 16 K rows from LDS are the
//     A operand, the wave's 16 query rows (registers) the B operand, so lane
//     (query n, group kg) receives the scores of keys 4kg..4kg+3 of each
//     16-key block.
//   * Online softmax per query row: max over the lane's 16 scores, then over
//     the row's 4 lanes (permlane swaps); probabilities stay fp32 until the
//     product.
//   * O += P V with v_mfma_f32_16x16x32_bf16 per 32 keys: the probabilities
//     are the A operand as the scores sit in the lanes (lane (query n, kg)
//     holds keys 4kg..4kg+3 of two 16-key blocks: its eight K slots), split
//     into a bf16 high part and a bf16 remainder (two products, ~16
//     significant bits kept).  The B operand needs, per lane, the same eight
//     keys of one V column; two ds_read_b64_tr_b16 transpose reads fetch them
//     from the row-major V tile in LDS (within each 16-lane group, lanes
//     4r..4r+3 address row r of a 4 x 16 block and lane i receives its column
//     i).
// Attention here is a dense contraction (G * n_q query rows against every
// key), so it is MFMA work, unlike the one-query decode step.

#include <hip/hip_runtime.h>

#include "dkv_device.hpp"
#include "dkv_query.hpp"

namespace dkv {

namespace {

constexpr int kQThreads = 512;
constexpr int kQRows = kQueryRowsPerWG;  // 16 query rows per wave
constexpr int kQDepth = 2;               // register stages: key tiles whose global loads are in flight
constexpr int kQKeys = 64;               // keys per tile

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

template <int D>
struct QCfg {
  static constexpr int kRowBytes = D * 2;
  static constexpr int kKStride = D + 8;   // bf16 per K row in LDS (rows 16-byte aligned)
  static constexpr int kVStride = D + 16;  // bf16 per V row in LDS (16-byte rows, stride = 32 B mod 128)
  static constexpr int kChunks = D / 32;   // 16-byte chunks of a row per lane (QK)
  static constexpr int kBlocks = D / 16;   // 16-column output blocks per lane
  static constexpr int kRowChunks = D / 8; // 16-byte chunks per row
  static constexpr int kStage = kQKeys * kRowChunks / kQThreads;  // chunks per thread per matrix
  static constexpr int kRec = D + 2;       // floats per partial record row
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

template <int D>
__global__ __launch_bounds__(kQThreads) void query_attn_kernel(QueryParams p) {
  using C = QCfg<D>;
  __shared__ __align__(16) uint16_t ks_lds[2][kQKeys * C::kKStride];
  __shared__ __align__(16) uint16_t vs_lds[2][kQKeys * C::kVStride];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int n16 = lane & 15;
  const int kg = lane >> 4;
  const int slot = blockIdx.x;  // (segment, query tile, key range), range fastest
  const int ks = slot % p.nsplit;
  const int qt = (slot / p.nsplit) % p.qtiles;
  const int s = slot / p.nsplit / p.qtiles;
  const int bseq = s / p.Hkv;
  const int g = s - bseq * p.Hkv;
  const int64_t base_len = q_uniform64((int64_t)p.seg_len[s] + p.n_tail);  // rows every query row sees
  const int64_t row0 = q_uniform64(p.seg_off[s]);

  // this lane's query row in the score layout, and the keys it sees
  const int r = qt * kQRows + wave * 16 + n16;
  const bool row_ok = r < p.rows;
  const int tok = row_ok ? r / p.G : 0;
  const int64_t limit = base_len + tok + 1;
  // this workgroup's key range
  const int r_last = min(p.rows - 1, qt * kQRows + kQRows - 1);
  const int64_t lim_max = base_len + r_last / p.G + 1;
  // (all workgroup-uniform; readfirstlane keeps them in scalar registers)
  const int64_t chunk = ((lim_max + p.nsplit - 1) / p.nsplit + kQKeys - 1) / kQKeys * kQKeys;
  const int64_t k_lo = q_uniform64((int64_t)ks * chunk);
  const int64_t k_hi = q_uniform64(k_lo + chunk < lim_max ? k_lo + chunk : lim_max);
  const int64_t cut = limit < k_hi ? limit : k_hi;  // keys [k_lo, cut) count for this row
  // every row of the workgroup sees all keys below this one
  const int64_t all_see = q_uniform64(base_len + 1 < k_hi ? base_len + 1 : k_hi);

  // B operand of QK: query row r, dims 32u + 8kg .. +7
  u32x4 qb[C::kChunks];
  {
    const int hh = r - tok * p.G;
    const char* qrow = reinterpret_cast<const char*>(p.q) +
                       (((int64_t)bseq * p.n_q + tok) * p.Hq + (int64_t)g * p.G + (row_ok ? hh : 0)) * C::kRowBytes;
#pragma unroll
    for (int u = 0; u < C::kChunks; ++u) {
      const u32x4 z = {0u, 0u, 0u, 0u};
      qb[u] = row_ok ? *reinterpret_cast<const u32x4*>(qrow + 64 * u + 16 * kg) : z;
    }
  }

  f32x4 o[C::kBlocks];
#pragma unroll
  for (int b = 0; b < C::kBlocks; ++b) o[b] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY;  // running max of query row n16 (log2 units)
  float l = 0.f;        // this lane's share of the row's sum

  const char* kbase = reinterpret_cast<const char*>(p.k) + row0 * C::kRowBytes;
  const char* vbase = reinterpret_cast<const char*>(p.v) + row0 * C::kRowBytes;
  // A ring of kQDepth register stages: while one tile is computed, the
  // global loads of the next kQDepth tiles are in flight.
  u32x4 kreg[kQDepth][C::kStage], vreg[kQDepth][C::kStage];
  // Global -> registers for the tile at key kt: chunk c of the tile is key
  // c / kRowChunks, bytes 16 * (c % kRowChunks).  Keys past k_hi (a whole
  // tile past it included) read zeros without touching memory, so the loads
  // can be issued unconditionally.
  auto load_stage = [&](u32x4 (&kreg)[C::kStage], u32x4 (&vreg)[C::kStage], int64_t kt) {
    const int64_t left = k_hi - kt;
    const uint32_t nk = (uint32_t)(left <= 0 ? 0 : (left < kQKeys ? left : kQKeys));
    const __amdgpu_buffer_rsrc_t kr = q_rsrc(kbase + kt * C::kRowBytes, nk * C::kRowBytes);
    const __amdgpu_buffer_rsrc_t vr = q_rsrc(vbase + kt * C::kRowBytes, nk * C::kRowBytes);
#pragma unroll
    for (int i = 0; i < C::kStage; ++i) {
      const int c = i * kQThreads + tid;
      const uint32_t off = (uint32_t)((c / C::kRowChunks) * C::kRowBytes + (c % C::kRowChunks) * 16);
      kreg[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(kr, off, 0, 0));
      vreg[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(vr, off, 0, 0));
    }
  };

  // ---- scores S^T[key][query] of the tile at key kt (K in LDS at kb) --------
  auto qk = [&](const uint16_t* kb, int64_t kt, float (&sc)[4][4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u < C::kChunks; ++u) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(&kb[(16 * j + n16) * C::kKStride + 32 * u + 8 * kg]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, qb[u]),
                                                      acc, 0, 0, 0);
      }
#pragma unroll
      for (int v = 0; v < 4; ++v) sc[j][v] = acc[v];
    }
  };

  // ---- softmax of the tile's scores and O += P V (V in LDS at vb) ---------
  auto softmax_pv = [&](float (&sc)[4][4], const uint16_t* vb, int64_t kt) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) sc[j][v] *= p.scale_log2;
    // keys past a row's causal limit or past the range: only in the tiles
    // that reach min over rows of that limit
    if (kt + kQKeys > all_see) {
      const int64_t lim = cut - kt;  // keys [0, lim) of this tile count for the row
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (16 * j + 4 * kg + v >= lim) sc[j][v] = -INFINITY;
    }

    // online softmax of row n16
    float mx = sc[0][0];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) mx = fmaxf(mx, sc[j][v]);
    mx = row4_max(mx);
    const float m_new = fmaxf(m, mx);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2(m - m_use);
    float ps = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        sc[j][v] = fast_exp2(sc[j][v] - m_use);
        ps += sc[j][v];
      }
    l = l * alpha + ps;
    m = m_new;
    // output rows of this lane are queries 4kg + v: their factors live in
    // the lanes of those rows.  Once the maxima settle every factor is 1 and
    // the wave skips the rescale.
    if (__builtin_amdgcn_ballot_w64(alpha != 1.f)) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float av = __shfl(alpha, 4 * kg + v, 64);
#pragma unroll
        for (int b = 0; b < C::kBlocks; ++b) o[b][v] *= av;
      }
    }

    // O += P V, 32 keys per product.  K slot e of lane group kg is key
    // 32h + 4kg + e (e < 4) or 32h + 16 + 4kg + (e - 4): the lane's scores of
    // blocks 2h and 2h + 1.
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      u32x4 ph, pl;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        uint32_t a, b;
        bf16_split(sc[2 * h + (e >> 1)][2 * (e & 1)], sc[2 * h + (e >> 1)][2 * (e & 1) + 1], a, b);
        ph[e] = a;
        pl[e] = b;
      }
      // transpose-read addresses: lane 4r + q of group kg reads row
      // 32h + 4kg + r (and the row 16 below), columns 16b + 4q .. +3
      const uint16_t* v0 = &vb[(32 * h + 4 * kg + (n16 >> 2)) * C::kVStride + 4 * (n16 & 3)];
#pragma unroll
      for (int b = 0; b < C::kBlocks; ++b) {
        const s16x4 t0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(v0 + 16 * b));
        const s16x4 t1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(v0 + 16 * C::kVStride + 16 * b));
        const uint2 w0 = __builtin_bit_cast(uint2, t0);
        const uint2 w1 = __builtin_bit_cast(uint2, t1);
        const u32x4 vbo = {w0.x, w0.y, w1.x, w1.y};
        o[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ph), __builtin_bit_cast(bf16x8, vbo),
                                                       o[b], 0, 0, 0);
        o[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, pl), __builtin_bit_cast(bf16x8, vbo),
                                                       o[b], 0, 0, 0);
      }
    }
  };

  auto store_tile = [&](const u32x4 (&kr)[C::kStage], const u32x4 (&vr)[C::kStage], uint16_t* kb, uint16_t* vb) {
#pragma unroll
    for (int c0 = 0; c0 < C::kStage; ++c0) {
      const int c = c0 * kQThreads + tid;
      const int key = c / C::kRowChunks;
      const int part = c % C::kRowChunks;
      *reinterpret_cast<u32x4*>(&kb[key * C::kKStride + part * 8]) = kr[c0];
      *reinterpret_cast<u32x4*>(&vb[key * C::kVStride + part * 8]) = vr[c0];
    }
  };

  // Software pipeline over key tiles.  Tile t sits in LDS buffer t % 2; the
  // global loads of tiles t + 1 and t + 2 are in flight in the two register
  // stages.  Iteration t stores tile t + 1 into the other buffer, issues the
  // score products of tile t + 1 and then does the softmax and P V of tile t,
  // so the matrix unit works on tile t + 1 while the vector unit works on
  // tile t.  Loads are issued in ring order (scheduling barriers keep them
  // there), so every store waits only for its own stage.  Tiles past k_hi
  // hold zeros and all their keys are masked, so they change nothing.
  load_stage(kreg[0], vreg[0], k_lo);
  __builtin_amdgcn_sched_barrier(0);
  load_stage(kreg[1], vreg[1], k_lo + kQKeys);
  __builtin_amdgcn_sched_barrier(0);
  store_tile(kreg[0], vreg[0], ks_lds[0], vs_lds[0]);
  __syncthreads();
  load_stage(kreg[0], vreg[0], k_lo + 2 * kQKeys);
  float sc[2][4][4];
  qk(ks_lds[0], k_lo, sc[0]);
  const int64_t ntile = k_hi > k_lo ? (k_hi - k_lo + kQKeys - 1) / kQKeys : 0;
  const int64_t nround = q_uniform64((ntile + 1) / 2);
  int64_t kt = k_lo;
  for (int64_t rd = 0; rd < nround; ++rd) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      __syncthreads();  // every wave is done with tile t - 1 (buffer 1 - i)
      store_tile(kreg[1 - i], vreg[1 - i], ks_lds[1 - i], vs_lds[1 - i]);
      __syncthreads();
      load_stage(kreg[1 - i], vreg[1 - i], kt + 3 * kQKeys);
      qk(ks_lds[1 - i], kt + kQKeys, sc[1 - i]);
      softmax_pv(sc[i], vs_lds[i], kt);
      kt += kQKeys;
    }
  }

  // ---- row totals; write the output or this range's record ------------------
  l = lane_xor_sum<16>(l);
  float* rec = p.rec + (int64_t)slot * kQRows * C::kRec;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int rr = wave * 16 + 4 * kg + v;  // row within the tile
    const int rq = qt * kQRows + rr;
    const float lq = __shfl(l, 4 * kg + v, 64);
    const float mq = __shfl(m, 4 * kg + v, 64);
    if (rq < p.rows) {
      if (p.nsplit == 1) {
        const int tq = rq / p.G;
        float* orow = p.out + (((int64_t)bseq * p.n_q + tq) * p.Hq + (int64_t)g * p.G + (rq - tq * p.G)) * D;
        const float inv = lq > 0.f ? 1.f / lq : 0.f;
#pragma unroll
        for (int b = 0; b < C::kBlocks; ++b) orow[16 * b + n16] = o[b][v] * inv;
      } else {
        float* rrow = rec + (int64_t)rr * C::kRec;
        if (n16 == 0) {
          rrow[0] = mq;
          rrow[1] = lq;
        }
#pragma unroll
        for (int b = 0; b < C::kBlocks; ++b) rrow[2 + 16 * b + n16] = o[b][v];
      }
    }
  }
}

// Combine kernel: thread item (row, 4 columns) of one (segment, query tile);
// kMergeThreads items per workgroup.  A thread loads the row's max and sum
// and its 4 columns from every key range at once (one memory round trip),
// then folds the ranges in order:
//   M = max_k m_k,  out = sum_k 2^(m_k - M) o_k / sum_k 2^(m_k - M) l_k.
constexpr int kMergeThreads = 256;

template <int D>
__global__ __launch_bounds__(kMergeThreads) void query_merge_kernel(QueryParams p) {
  using C = QCfg<D>;
  constexpr int kItems = kQRows * (D / 4);                 // items per query tile
  constexpr int kParts = kItems / kMergeThreads;           // workgroups per query tile
  const int tile = blockIdx.x / kParts;                    // s * qtiles + qt
  const int item = (blockIdx.x - tile * kParts) * kMergeThreads + threadIdx.x;
  const int s = tile / p.qtiles;
  const int qt = tile - s * p.qtiles;
  const int rr = item / (D / 4);
  const int c4 = item - rr * (D / 4);
  const int rq = qt * kQRows + rr;
  if (rq >= p.rows) return;
  const int bseq = s / p.Hkv;
  const int g = s - bseq * p.Hkv;
  const float* recs = p.rec + (int64_t)tile * p.nsplit * kQRows * C::kRec + (int64_t)rr * C::kRec;
  float mk[kQueryMaxSplit], lk[kQueryMaxSplit];
  f32x4 ak[kQueryMaxSplit];
#pragma unroll
  for (int k = 0; k < kQueryMaxSplit; ++k) {
    if (k < p.nsplit) {
      const float* r = recs + (int64_t)k * kQRows * C::kRec;
      mk[k] = r[0];
      lk[k] = r[1];
      ak[k] = *reinterpret_cast<const f32x4*>(r + 2 + 4 * c4);
    } else {
      mk[k] = -INFINITY;
      lk[k] = 0.f;
      ak[k] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
  float M = -INFINITY;
#pragma unroll
  for (int k = 0; k < kQueryMaxSplit; ++k) M = fmaxf(M, mk[k]);
  const float Mu = M == -INFINITY ? 0.f : M;
  float L = 0.f;
  f32x4 A = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int k = 0; k < kQueryMaxSplit; ++k) {
    const float f = fast_exp2(mk[k] - Mu);
    L += f * lk[k];
    A += f * ak[k];
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  const int tq = rq / p.G;
  float* orow = p.out + (((int64_t)bseq * p.n_q + tq) * p.Hq + (int64_t)g * p.G + (rq - tq * p.G)) * D;
  *reinterpret_cast<f32x4*>(orow + 4 * c4) = A * inv;
}

template <int D>
hipError_t launch_d(const QueryParams& p, hipStream_t stream) {
  const int64_t wgs = (int64_t)p.nseg * p.qtiles * p.nsplit;
  hipLaunchKernelGGL((query_attn_kernel<D>), dim3((unsigned)wgs), dim3(kQThreads), 0, stream, p);
  if (p.nsplit > 1) {
    const int64_t parts = (int64_t)kQRows * (D / 4) / kMergeThreads;
    hipLaunchKernelGGL((query_merge_kernel<D>), dim3((unsigned)(p.nseg * p.qtiles * parts)), dim3(kMergeThreads), 0,
                       stream, p);
  }
  return hipGetLastError();
}

}  // namespace

int32_t query_split_count(int32_t nseg, int32_t rows, int64_t rows_hint) {
  // about two workgroups per compute unit of a 256-CU part
  constexpr int64_t kTargetWG = 512;
  const int64_t qtiles = (rows + kQRows - 1) / kQRows;
  const int64_t base = (int64_t)nseg * qtiles;
  int64_t n = (kTargetWG + base - 1) / base;
  // each range keeps at least 8 key tiles
  const int64_t keys = rows_hint > 0 ? rows_hint / (nseg > 0 ? nseg : 1) : (int64_t)1 << 30;
  const int64_t by_keys = keys / (8 * kQKeys);
  if (n > by_keys) n = by_keys;
  if (n > kQueryMaxSplit) n = kQueryMaxSplit;
  return (int32_t)(n < 1 ? 1 : n);
}

size_t query_workspace_bytes(int32_t nseg, int32_t rows, int32_t head_dim, int64_t rows_hint) {
  const int32_t n = query_split_count(nseg, rows, rows_hint);
  if (n <= 1) return 0;
  const int64_t qtiles = (rows + kQRows - 1) / kQRows;
  return (size_t)nseg * qtiles * n * kQRows * (head_dim + 2) * sizeof(float);
}

hipError_t launch_query_attn(const QueryParams& p, int head_dim, hipStream_t stream) {
  return head_dim == 64 ? launch_d<64>(p, stream) : launch_d<128>(p, stream);
}

}  // namespace dkv
