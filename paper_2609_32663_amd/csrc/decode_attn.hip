// Decode attention over the packed, ragged Distance-KV cache (Sec. 3.4: the
// query attends to the compressed context plus the appended tokens; every
// query head of a GQA group attends to the group's union segment).  The same
// kernel with dense addressing is the Dense comparator of Sec. 4.3.
//
// Work split.  The rows of all segments of the call are laid end to end and
// the flat row range is cut into P equal slices, one per workgroup
// (P = min(launched workgroups, total rows)), so heads that kept 128 rows and
// heads that kept 130,000 rows cost the same per workgroup.  A slice that
// crosses segment boundaries yields one piece per segment.  Piece (w, s) of
// workgroup w in segment s writes its online-softmax state (max m, sum l and
// unnormalised accumulator per query head) to slot w + s of the workspace;
// these slots are unique and a segment's slots are contiguous.  The last
// workgroup to finish a segment (device-scope counter) merges its slots in
// slot order, so the result does not depend on arrival order, and resets the
// counter.  A segment covered by one workgroup skips the workspace.
//
// Inside a workgroup the 4 waves take 32-key tiles round-robin.  Per tile:
//   * K rows go straight from HBM into MFMA operands: lane (j, kg) of a wave
//     loads 16-byte chunks kg, kg+4, ... of key j (j = lane % 16), which is
//     exactly the B-operand layout of v_mfma_f32_16x16x32_bf16 (8 bf16 per
//     lane) or of four v_mfma_f32_16x16x4_f32 (4 fp32 per lane); the query
//     group, zero-padded to 16 rows, is the A operand.  The output holds the
//     scores of key j for heads 4*(lane/16)+v in lane j + 16*(lane/16).
//   * Scores are scaled by sm_scale*log2(e), reduced per head across the 16
//     key lanes with DPP, and folded into a running max; p = exp2(s - m)
//     stays fp32 (no bf16 rounding of probabilities) and goes to a per-wave
//     LDS tile together with the rescale factors.
//   * V rows are read fully coalesced (LPR lanes x 16 bytes per row, 64/LPR
//     rows per instruction) and accumulated on the VALU: lane (cc, rp) owns
//     16 bytes of columns of rows rp, rp + RP, ... for every head.
// The decode step is a GEMV per KV row (about G flop per byte), far below the
// MFMA ridge, so the kernel is built to keep HBM busy rather than the ALUs.

#include "dkv_device.hpp"
#include "dkv_launch.hpp"

namespace dkv {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kTK = 32;  // keys per wave tile

template <bool BF16, int D, int GP>
struct DecodeCfg {
  static constexpr int kElem = BF16 ? 2 : 4;
  static constexpr int kRowBytes = D * kElem;
  static constexpr int kChunks = kRowBytes / 64;   // 16-byte chunks per lane per key (QK)
  static constexpr int kLPR = kRowBytes / 16;      // lanes per row (PV)
  static constexpr int kCPL = 16 / kElem;          // columns per lane (PV)
  static constexpr int kRP = kWave / kLPR;         // row phases (PV)
  static constexpr int kRPT = kTK / kRP;           // V rows per lane per tile
  static constexpr int kKG = kTK / 16;             // 16-key groups per tile
  static constexpr int kRec = GP * (D + 2);        // floats per partial record
  static_assert(kTK % kRP == 0, "tile must cover whole row phases");
};

__device__ __forceinline__ f32x4 qk_mfma(const u32x4& a, const u32x4& b, f32x4 c, bool bf16) {
  if (bf16) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                    __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
#pragma unroll
  for (int e = 0; e < 4; ++e)
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[e]), __uint_as_float(b[e]), c, 0, 0, 0);
  return c;
}

template <bool BF16>
__device__ __forceinline__ void widen16(const u32x4& w, float* out) {
  if (BF16) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      out[2 * q] = bf16_lo(w[q]);
      out[2 * q + 1] = bf16_hi(w[q]);
    }
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) out[q] = __uint_as_float(w[q]);
  }
}

// Workgroup that owns flat row x when `total` rows are cut into P slices
// [floor(w*total/P), floor((w+1)*total/P)).
__device__ __forceinline__ int64_t owner_of(int64_t x, int64_t total, int64_t P) {
  const int64_t w = ((x + 1) * P - 1) / total;
  return w < P - 1 ? w : P - 1;
}

template <bool BF16, int D, int GP>
__global__ __launch_bounds__(kThreads) void decode_kernel(DecodeParams p) {
  using C = DecodeCfg<BF16, D, GP>;
  extern __shared__ __align__(16) int64_t pre[];          // [nseg + 1] row prefix
  __shared__ __align__(16) float pbuf[kWaves][kTK][GP];   // probabilities per wave tile
  __shared__ __align__(16) float abuf[kWaves][GP];        // rescale factors per wave
  __shared__ __align__(16) float wacc[kWaves][GP][D];     // per-wave accumulators
  __shared__ float wm[kWaves][GP];
  __shared__ float wl[kWaves][GP];
  __shared__ int64_t red[kWaves + 1];
  __shared__ int last_flag;

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int w = blockIdx.x;
  const int nseg = p.nseg;
  const bool dense = p.seg_len == nullptr;

  // ---- flat row prefix over the call's segments ------------------------
  {
    const int per = (nseg + kThreads - 1) / kThreads;
    const int s_lo = tid * per;
    const int s_hi = min(nseg, s_lo + per);
    int64_t sum = 0;
    for (int s = s_lo; s < s_hi; ++s) sum += dense ? p.dense_len : (int64_t)p.seg_len[s] + p.n_tail;
    int64_t total_unused;
    int64_t run = block_exclusive_scan<kThreads>(sum, red, &total_unused);
    for (int s = s_lo; s < s_hi; ++s) {
      pre[s] = run;
      run += dense ? p.dense_len : (int64_t)p.seg_len[s] + p.n_tail;
    }
    if (s_hi == nseg && s_lo <= nseg) pre[nseg] = run;
    if (nseg == 0 && tid == 0) pre[0] = 0;
  }
  __syncthreads();
  const int64_t total = pre[nseg];

  // ---- segments with no rows at all produce zeros ----------------------
  for (int s = w; s < nseg; s += p.P) {
    if (pre[s + 1] == pre[s]) {
      const int b = s / p.Hkv, g = s - (s / p.Hkv) * p.Hkv;
      float* o = p.out + ((int64_t)b * p.Hq + (int64_t)g * p.G) * D;
      for (int i = tid; i < p.G * D; i += kThreads) o[i] = 0.f;
    }
  }
  const int64_t P = total < p.P ? total : p.P;
  if (w >= P) return;
  const int64_t lo = (int64_t)w * total / P;
  const int64_t hi = (int64_t)(w + 1) * total / P;

  // first segment whose row range contains lo
  int s = 0;
  {
    int a = 0, b = nseg;  // pre[a] <= lo < pre[b]
    while (b - a > 1) {
      const int mid = (a + b) >> 1;
      if (pre[mid] <= lo) a = mid; else b = mid;
    }
    s = a;
  }

  const char* kbytes = reinterpret_cast<const char*>(p.k);
  const char* vbytes = reinterpret_cast<const char*>(p.v);
  const char* qbytes = reinterpret_cast<const char*>(p.q);
  const int j16 = lane & 15;   // key (QK) / head row (A operand) within a 16-group
  const int kg = lane >> 4;    // 16-byte chunk group (QK)
  const int cc = lane % C::kLPR;
  const int rp = lane / C::kLPR;

  for (; s < nseg && pre[s] < hi; ++s) {
    const int64_t seg_lo = pre[s], seg_hi = pre[s + 1];
    const int64_t a = (lo > seg_lo ? lo : seg_lo) - seg_lo;
    const int64_t bnd = (hi < seg_hi ? hi : seg_hi) - seg_lo;
    if (a >= bnd) continue;
    const int bseq = s / p.Hkv;
    const int g = s - bseq * p.Hkv;
    const int64_t row0 = dense ? (int64_t)s * p.dense_stride : p.seg_off[s];

    // A operand: query head j16 of the group (zero beyond G), chunks kg + 4u.
    u32x4 qa[C::kChunks];
    {
      const bool real = j16 < p.G;
      const char* qrow = qbytes + ((int64_t)bseq * p.Hq + (int64_t)g * p.G + (real ? j16 : 0)) * C::kRowBytes;
#pragma unroll
      for (int u = 0; u < C::kChunks; ++u) {
        u32x4 z = {0u, 0u, 0u, 0u};
        qa[u] = real ? *reinterpret_cast<const u32x4*>(qrow + 64 * u + 16 * kg) : z;
      }
    }

    float m_run[4], l_part[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) { m_run[v] = -INFINITY; l_part[v] = 0.f; }
    float acc[GP][C::kCPL];
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
      for (int c = 0; c < C::kCPL; ++c) acc[h][c] = 0.f;

    const int64_t ntile = (bnd - a + kTK - 1) / kTK;
    const int64_t last = bnd - 1;
    const bool head_lanes = 4 * kg < GP;

    for (int64_t t = wave; t < ntile; t += kWaves) {
      const int64_t rbase = a + t * kTK;
      u32x4 kf[C::kKG][C::kChunks];
      u32x4 vf[C::kRPT];
#pragma unroll
      for (int kk = 0; kk < C::kKG; ++kk) {
        int64_t key = rbase + 16 * kk + j16;
        key = key < last ? key : last;
        const char* src = kbytes + (row0 + key) * C::kRowBytes + 16 * kg;
#pragma unroll
        for (int u = 0; u < C::kChunks; ++u) kf[kk][u] = *reinterpret_cast<const u32x4*>(src + 64 * u);
      }
#pragma unroll
      for (int i = 0; i < C::kRPT; ++i) {
        int64_t key = rbase + C::kRP * i + rp;
        key = key < last ? key : last;
        vf[i] = *reinterpret_cast<const u32x4*>(vbytes + (row0 + key) * C::kRowBytes + 16 * cc);
      }

      // scores: lane j16 + 16*kg holds key 16*kk + j16, heads 4*kg + v
      float sc[C::kKG][4];
#pragma unroll
      for (int kk = 0; kk < C::kKG; ++kk) {
        f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int u = 0; u < C::kChunks; ++u) c = qk_mfma(qa[u], kf[kk][u], c, BF16);
        const bool valid = rbase + 16 * kk + j16 <= last;
#pragma unroll
        for (int v = 0; v < 4; ++v) sc[kk][v] = valid ? c[v] * p.scale_log2 : -INFINITY;
      }

      float alpha[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        float mt = sc[0][v];
#pragma unroll
        for (int kk = 1; kk < C::kKG; ++kk) mt = fmaxf(mt, sc[kk][v]);
        mt = row16_max(mt);
        const float m_new = fmaxf(m_run[v], mt);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        alpha[v] = fast_exp2(m_run[v] - m_use);
        float psum = 0.f;
#pragma unroll
        for (int kk = 0; kk < C::kKG; ++kk) {
          sc[kk][v] = fast_exp2(sc[kk][v] - m_use);
          psum += sc[kk][v];
        }
        l_part[v] = l_part[v] * alpha[v] + psum;
        m_run[v] = m_new;
      }

      if (head_lanes) {
#pragma unroll
        for (int kk = 0; kk < C::kKG; ++kk) {
          f32x4 pv = {sc[kk][0], sc[kk][1], sc[kk][2], sc[kk][3]};
          *reinterpret_cast<f32x4*>(&pbuf[wave][16 * kk + j16][4 * kg]) = pv;
        }
        if (j16 == 0) {
          f32x4 av = {alpha[0], alpha[1], alpha[2], alpha[3]};
          *reinterpret_cast<f32x4*>(&abuf[wave][4 * kg]) = av;
        }
      }
      wave_lds_fence();

#pragma unroll
      for (int h4 = 0; h4 < GP / 4; ++h4) {
        const f32x4 al = *reinterpret_cast<const f32x4*>(&abuf[wave][4 * h4]);
#pragma unroll
        for (int v = 0; v < 4; ++v)
#pragma unroll
          for (int c = 0; c < C::kCPL; ++c) acc[4 * h4 + v][c] *= al[v];
      }
#pragma unroll
      for (int i = 0; i < C::kRPT; ++i) {
        float vv[C::kCPL];
        widen16<BF16>(vf[i], vv);
        const int r = C::kRP * i + rp;
#pragma unroll
        for (int h4 = 0; h4 < GP / 4; ++h4) {
          const f32x4 pr = *reinterpret_cast<const f32x4*>(&pbuf[wave][r][4 * h4]);
#pragma unroll
          for (int v = 0; v < 4; ++v)
#pragma unroll
            for (int c = 0; c < C::kCPL; ++c) acc[4 * h4 + v][c] = fmaf(pr[v], vv[c], acc[4 * h4 + v][c]);
        }
      }
      wave_lds_fence();
    }

    // ---- wave state -> LDS ---------------------------------------------
#pragma unroll
    for (int v = 0; v < 4; ++v) l_part[v] = row16_sum(l_part[v]);
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
      for (int c = 0; c < C::kCPL; ++c) {
        float x = acc[h][c];
#pragma unroll
        for (int o = C::kLPR; o < kWave; o <<= 1) x += __shfl_xor(x, o, kWave);
        acc[h][c] = x;
      }
    if (rp == 0) {
#pragma unroll
      for (int h = 0; h < GP; ++h)
#pragma unroll
        for (int c = 0; c < C::kCPL; ++c) wacc[wave][h][cc * C::kCPL + c] = acc[h][c];
    }
    if (j16 == 0 && head_lanes) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        wm[wave][4 * kg + v] = m_run[v];
        wl[wave][4 * kg + v] = l_part[v];
      }
    }
    __syncthreads();

    // ---- combine the waves; write the output or a partial record ---------
    const int64_t w_first = owner_of(seg_lo, total, P);
    const int64_t w_last = owner_of(seg_hi - 1, total, P);
    const bool single = w_first == w_last;
    float* rec = p.partials + (int64_t)(w + s) * C::kRec;
    float* outp = p.out + ((int64_t)bseq * p.Hq + (int64_t)g * p.G) * D;
    for (int idx = tid; idx < p.G * D; idx += kThreads) {
      const int h = idx / D, c = idx - (idx / D) * D;
      float M = wm[0][h];
#pragma unroll
      for (int q = 1; q < kWaves; ++q) M = fmaxf(M, wm[q][h]);
      const float Mu = M == -INFINITY ? 0.f : M;
      float L = 0.f, A = 0.f;
#pragma unroll
      for (int q = 0; q < kWaves; ++q) {
        const float f = fast_exp2(wm[q][h] - Mu);
        L += f * wl[q][h];
        A += f * wacc[q][h][c];
      }
      if (single) {
        outp[idx] = L > 0.f ? A / L : 0.f;
      } else {
        rec[2 * GP + h * D + c] = A;
        if (c == 0) {
          rec[h] = M;
          rec[GP + h] = L;
        }
      }
    }
    if (!single) {
      __threadfence();
      __syncthreads();
      if (tid == 0) {
        const int prev = atomicAdd(p.counters + s, 1);
        last_flag = prev == (int)(w_last - w_first);
      }
      __syncthreads();
      if (last_flag) {
        __threadfence();
        const float* first = p.partials + (w_first + s) * C::kRec;
        const int npieces = (int)(w_last - w_first + 1);
        for (int idx = tid; idx < p.G * D; idx += kThreads) {
          const int h = idx / D, c = idx - (idx / D) * D;
          float M = -INFINITY;
          for (int k = 0; k < npieces; ++k) M = fmaxf(M, first[(int64_t)k * C::kRec + h]);
          const float Mu = M == -INFINITY ? 0.f : M;
          float L = 0.f, A = 0.f;
          for (int k = 0; k < npieces; ++k) {
            const float* r = first + (int64_t)k * C::kRec;
            const float f = fast_exp2(r[h] - Mu);
            L += f * r[GP + h];
            A += f * r[2 * GP + h * D + c];
          }
          outp[idx] = L > 0.f ? A / L : 0.f;
        }
        if (tid == 0) p.counters[s] = 0;
      }
    }
    __syncthreads();
  }
}

template <bool BF16, int D>
hipError_t launch_d(const DecodeParams& p, int GP, hipStream_t stream) {
  const size_t lds = ((size_t)p.nseg + 1) * sizeof(int64_t);
  switch (GP) {
    case 4: hipLaunchKernelGGL((decode_kernel<BF16, D, 4>), dim3(p.P), dim3(kThreads), lds, stream, p); break;
    case 8: hipLaunchKernelGGL((decode_kernel<BF16, D, 8>), dim3(p.P), dim3(kThreads), lds, stream, p); break;
    case 16: hipLaunchKernelGGL((decode_kernel<BF16, D, 16>), dim3(p.P), dim3(kThreads), lds, stream, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

int decode_group_pad(int G) { return G <= 4 ? 4 : (G <= 8 ? 8 : 16); }

size_t decode_partials_bytes(int nseg, int G, int head_dim) {
  const size_t rec = (size_t)decode_group_pad(G) * (head_dim + 2) * 4;
  return ((size_t)kDecodeMaxWG + nseg) * rec;
}

hipError_t launch_decode(const DecodeParams& p, dkv_dtype dtype, int head_dim, hipStream_t stream) {
  const int GP = decode_group_pad(p.G);
  if (dtype == DKV_BF16) {
    if (head_dim == 128) return launch_d<true, 128>(p, GP, stream);
    if (head_dim == 64) return launch_d<true, 64>(p, GP, stream);
  } else {
    if (head_dim == 128) return launch_d<false, 128>(p, GP, stream);
    if (head_dim == 64) return launch_d<false, 64>(p, GP, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace dkv
