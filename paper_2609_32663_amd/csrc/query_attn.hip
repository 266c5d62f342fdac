// Query-block attention over the packed Distance-KV cache (Sec. 3.4: after
// the one-time compaction the query tokens attend to the compressed context,
// while their own K/V are appended like every new token and kept).
//
// Rows and work split.  Segment s = (sequence b, KV head g) has
// R = n_q * G query rows; row r is token r / G of query head g * G + r % G
// and sees the segment's first seg_len + n_tail + r / G + 1 rows (the packed
// context, the tokens appended before the block, and the block causally up
// to its own token).  A workgroup takes 64 query rows (16 per wave) of one
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
//   * O += P V with v_mfma_f32_16x16x16_bf16: the probabilities are the A
//     operand exactly as the scores sit in the lanes, split into a bf16 high
//     part and a bf16 remainder (two products, ~16 significant bits kept);
//     the B operand (4 keys of one V column per lane) is gathered from
//     row-major LDS with 16-bit reads, free of bank conflicts with a row
//     stride of d + 4 elements.
// Attention here is a dense contraction (G * n_q query rows against every
// key), so it is MFMA work, unlike the one-query decode step.

#include <hip/hip_runtime.h>

#include "dkv_device.hpp"
#include "dkv_query.hpp"

namespace dkv {

namespace {

constexpr int kQThreads = 256;
constexpr int kQRows = kQueryRowsPerWG;  // 16 query rows per wave
constexpr int kQKeys = 64;               // keys per tile

typedef short s16x4 __attribute__((ext_vector_type(4)));

template <int D>
struct QCfg {
  static constexpr int kRowBytes = D * 2;
  static constexpr int kKStride = D + 8;   // bf16 per K row in LDS (rows 16-byte aligned)
  static constexpr int kVStride = D + 4;   // bf16 per V row in LDS (conflict-free column gathers)
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

// bf16 of x, rounded to nearest even (x finite).
__device__ __forceinline__ uint32_t bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
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
  __shared__ __align__(16) uint16_t ks_lds[kQKeys * C::kKStride];
  __shared__ __align__(16) uint16_t vs_lds[kQKeys * C::kVStride];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int n16 = lane & 15;
  const int kg = lane >> 4;
  int x = blockIdx.x;
  const int ks = x % p.nsplit;
  x /= p.nsplit;
  const int qt = x % p.qtiles;
  const int s = x / p.qtiles;
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
  const int64_t chunk = ((lim_max + p.nsplit - 1) / p.nsplit + kQKeys - 1) / kQKeys * kQKeys;
  const int64_t k_lo = (int64_t)ks * chunk;
  const int64_t k_hi = k_lo + chunk < lim_max ? k_lo + chunk : lim_max;
  const int64_t cut = limit < k_hi ? limit : k_hi;  // keys [k_lo, cut) count for this row

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
  u32x4 kreg[C::kStage], vreg[C::kStage];
  // Global -> registers for the tile at key kt: chunk c of the tile is key
  // c / kRowChunks, bytes 16 * (c % kRowChunks); keys past k_hi read zeros.
  auto load_stage = [&](int64_t kt) {
    const uint32_t nk = (uint32_t)(k_hi - kt < kQKeys ? k_hi - kt : kQKeys);
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

  if (k_lo < k_hi) load_stage(k_lo);
  for (int64_t kt = k_lo; kt < k_hi; kt += kQKeys) {
    __syncthreads();  // every wave is done with the previous tile
#pragma unroll
    for (int i = 0; i < C::kStage; ++i) {
      const int c = i * kQThreads + tid;
      const int key = c / C::kRowChunks;
      const int part = c % C::kRowChunks;
      *reinterpret_cast<u32x4*>(&ks_lds[key * C::kKStride + part * 8]) = kreg[i];
      uint2* vd = reinterpret_cast<uint2*>(&vs_lds[key * C::kVStride + part * 8]);
      vd[0] = uint2{vreg[i][0], vreg[i][1]};
      vd[1] = uint2{vreg[i][2], vreg[i][3]};
    }
    __syncthreads();
    if (kt + kQKeys < k_hi) load_stage(kt + kQKeys);

    // ---- scores S^T[key][query] of the 4 blocks of 16 keys ----------------
    float sc[4][4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u < C::kChunks; ++u) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(&ks_lds[(16 * j + n16) * C::kKStride + 32 * u + 8 * kg]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, qb[u]),
                                                      acc, 0, 0, 0);
      }
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t key = kt + 16 * j + 4 * kg + v;
        sc[j][v] = key < cut ? acc[v] * p.scale_log2 : -INFINITY;
      }
    }

    // ---- online softmax of row n16 -----------------------------------------
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
    // the lanes of those rows
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const float av = __shfl(alpha, 4 * kg + v, 64);
#pragma unroll
      for (int b = 0; b < C::kBlocks; ++b) o[b][v] *= av;
    }

    // ---- O += P V ------------------------------------------------------------
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t hi[4], lo[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        hi[v] = bf16_rne(sc[j][v]);
        lo[v] = bf16_rne(sc[j][v] - __uint_as_float(hi[v] << 16));
      }
      const s16x4 ph = {(short)hi[0], (short)hi[1], (short)hi[2], (short)hi[3]};
      const s16x4 pl = {(short)lo[0], (short)lo[1], (short)lo[2], (short)lo[3]};
      const uint16_t* vrow = &vs_lds[(16 * j + 4 * kg) * C::kVStride + n16];
#pragma unroll
      for (int b = 0; b < C::kBlocks; ++b) {
        const s16x4 vb = {(short)vrow[16 * b], (short)vrow[C::kVStride + 16 * b],
                          (short)vrow[2 * C::kVStride + 16 * b], (short)vrow[3 * C::kVStride + 16 * b]};
        o[b] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ph, vb, o[b], 0, 0, 0);
        o[b] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pl, vb, o[b], 0, 0, 0);
      }
    }
  }

  // ---- row totals; write the output or this range's record ------------------
  l = lane_xor_sum<16>(l);
  float* rec = p.rec + (int64_t)blockIdx.x * kQRows * C::kRec;
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

// Combine kernel: one workgroup per (segment, query tile); thread items are
// (row, 4 columns); the nsplit records of a row are folded in range order:
//   M = max_k m_k,  out = sum_k 2^(m_k - M) o_k / sum_k 2^(m_k - M) l_k.
template <int D>
__global__ __launch_bounds__(kQThreads) void query_merge_kernel(QueryParams p) {
  using C = QCfg<D>;
  const int s = blockIdx.x / p.qtiles;
  const int qt = blockIdx.x - s * p.qtiles;
  const int bseq = s / p.Hkv;
  const int g = s - bseq * p.Hkv;
  const float* recs = p.rec + (int64_t)blockIdx.x * p.nsplit * kQRows * C::kRec;
  for (int idx = threadIdx.x; idx < kQRows * (D / 4); idx += kQThreads) {
    const int rr = idx / (D / 4);
    const int c4 = idx - rr * (D / 4);
    const int rq = qt * kQRows + rr;
    if (rq >= p.rows) continue;
    float M = -INFINITY;
    for (int k = 0; k < p.nsplit; ++k) M = fmaxf(M, recs[((int64_t)k * kQRows + rr) * C::kRec]);
    const float Mu = M == -INFINITY ? 0.f : M;
    float L = 0.f;
    f32x4 A = {0.f, 0.f, 0.f, 0.f};
    for (int k = 0; k < p.nsplit; ++k) {
      const float* rrow = recs + ((int64_t)k * kQRows + rr) * C::kRec;
      const float f = fast_exp2(rrow[0] - Mu);
      L += f * rrow[1];
      const float* a = rrow + 2 + 4 * c4;
      A[0] += f * a[0];
      A[1] += f * a[1];
      A[2] += f * a[2];
      A[3] += f * a[3];
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    const int tq = rq / p.G;
    float* orow = p.out + (((int64_t)bseq * p.n_q + tq) * p.Hq + (int64_t)g * p.G + (rq - tq * p.G)) * D;
    *reinterpret_cast<f32x4*>(orow + 4 * c4) = A * inv;
  }
}

template <int D>
hipError_t launch_d(const QueryParams& p, hipStream_t stream) {
  const int64_t wgs = (int64_t)p.nseg * p.qtiles * p.nsplit;
  hipLaunchKernelGGL((query_attn_kernel<D>), dim3((unsigned)wgs), dim3(kQThreads), 0, stream, p);
  if (p.nsplit > 1)
    hipLaunchKernelGGL((query_merge_kernel<D>), dim3((unsigned)(p.nseg * p.qtiles)), dim3(kQThreads), 0, stream, p);
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
