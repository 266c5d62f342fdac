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
// these slots are unique and a segment's slots are contiguous.  A second,
// wide kernel (one workgroup per segment and query head) merges each
// segment's slots in slot order, so the result does not depend on timing.  A
// segment covered by one workgroup is written directly and skips the merge.
// Publishing the partials through the kernel boundary instead of a
// last-workgroup-merges scheme avoids device-scope fences, which on this part
// are whole-L2 write-backs and cost more than the merge itself.
//
// Inside a workgroup the 4 waves take 16-key tiles round-robin, with the next
// tile's loads in flight while the current one is computed.  Per tile:
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
//
// Paged addressing (the zero-copy variant): K and V stay in a page pool and a
// segment's rows are the page_rows slots of each of its entries (page, logical
// page, lo, hi), so the split, the ring and the combine are the same.  Tiles
// are aligned to the 16-row grid of that row space and never straddle a page;
// each tile gets its own buffer descriptor over the page rows from the tile's
// start to the end of the attended slots, so slots past an entry's end (and
// past the tokens appended so far) read zeros without touching memory, and the
// softmax masks every slot outside [lo, hi).  Each wave holds a chunk of 64
// entries in registers, one per lane, and reads a tile's entry with readlane.

#include <atomic>

#include "dkv_device.hpp"
#include "dkv_launch.hpp"

namespace dkv {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
// Keys per wave tile.  With one tile loading while the other is computed a
// wave keeps 8 KiB of bf16 d128 K/V in flight, 32 KiB per compute unit: on
// this part a stream with fewer bytes in flight per compute unit runs faster
// (32-key tiles three deep, 128 KiB per unit: 40.4 us per headline call;
// two deep, 64 KiB: 38.8; 16-key tiles two deep: 37.7; three or four deep
// or two workgroups per unit: 38.3-39.2).
constexpr int kTK = 16;

#if DKV_PHASE_STAMPS
// Phase-stamp build (a separate library, built on request; the product
// library has none of this): per call slot and workgroup, the constant
// 100 MHz clock at kernel entry [0], after the prologue [1], at wave 0's
// first tile [2], at each wave's loop end [3..6] and at the workgroup's end
// [7]; per combine workgroup, its start and end.
constexpr int kStampCalls = 64, kStampWG = kDecodeMaxWG, kStampMergeWG = 4096;
__device__ unsigned long long stamp_split[kStampCalls][kStampWG][8];
__device__ unsigned long long stamp_merge[kStampCalls][kStampMergeWG][2];
#define DKV_STAMP(...) __VA_ARGS__
#else
#define DKV_STAMP(...)
#endif

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
  // Row-phase partial accumulators each wave leaves in LDS for the fold: all
  // kRP of them, or fewer (summed across lanes first) when the partials of
  // all waves would pass 64 KiB.
  static constexpr int kRPK =
      (kWaves * kRP * GP * D * 4 <= 65536) ? kRP : (kWaves * (kRP / 2) * GP * D * 4 <= 65536 ? kRP / 2 : kRP / 4);
  static_assert(kRPK >= 1 && kWaves * kRPK * GP * D * 4 <= 65536, "fold partials must fit 64 KiB of LDS");
  static constexpr int64_t kSubRows = (1LL << 30) / kRowBytes;  // rows per buffer descriptor
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
// The quotient comes from an fp64 division (the numerator is below 2^53) and
// is corrected by one where rounding crossed an integer; a 64-bit integer
// division is a long emulated sequence.
__device__ __forceinline__ int64_t owner_of(int64_t x, int64_t total, int64_t P) {
  const int64_t num = (x + 1) * P - 1;
  int64_t w = (int64_t)((double)num / (double)total);
  if (w * total > num) --w;
  else if ((w + 1) * total <= num) ++w;
  return w < P - 1 ? w : P - 1;
}

template <int W>
__device__ __forceinline__ float group_max(float x) {
#pragma unroll
  for (int o = W / 2; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, W));
  return x;
}

template <int W>
__device__ __forceinline__ float group_sum(float x) {
#pragma unroll
  for (int o = W / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, W);
  return x;
}

// K and V registers of one wave tile.  Paged tiles also carry the range
// [lo, hi) of their kTK rows that is attended.
template <bool BF16, int D, int GP>
struct Tile {
  using C = DecodeCfg<BF16, D, GP>;
  u32x4 k[C::kKG][C::kChunks];
  u32x4 v[C::kRPT];
  int32_t lo, hi;
};

// Buffer descriptor over `bytes` bytes at `base` (raw buffer, stride 0).  A
// load whose offset lies past the range returns zeros instead of touching
// memory, which is what the ragged end of a piece relies on.
// Every argument must be wave-uniform; readfirstlane makes that explicit so
// the descriptor lives in SGPRs (otherwise each load becomes a loop).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const char* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  char* ub = reinterpret_cast<char*>(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(ub, (short)0, (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

__device__ __forceinline__ int64_t uniform64(int64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Cache policy of the K/V loads: non-temporal.  Every K/V byte is read once
// per step, so keeping it out of the caches' normal replacement is worth
// about 10-15% of streaming bandwidth on this part.
constexpr int kStreamLoad = 2;

// Loads the K and V rows [row, row + kTK) of a piece.  k_lane / v_lane are
// the lane-constant byte offsets (key j16 chunk kg, and row phase rp column
// chunk cc).  The whole offset stays in the vector offset; loads past the
// descriptor's range return zeros.
template <bool BF16, int D, int GP>
__device__ __forceinline__ void load_tile(Tile<BF16, D, GP>& t, __amdgpu_buffer_rsrc_t kr, __amdgpu_buffer_rsrc_t vr,
                                          uint32_t row, uint32_t k_lane, uint32_t v_lane) {
  using C = DecodeCfg<BF16, D, GP>;
#pragma unroll
  for (int kk = 0; kk < C::kKG; ++kk) {
    const uint32_t vo = k_lane + (row + 16 * kk) * C::kRowBytes;
#pragma unroll
    for (int u = 0; u < C::kChunks; ++u)
      t.k[kk][u] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(kr, vo + 64 * u, 0, kStreamLoad));
  }
#pragma unroll
  for (int i = 0; i < C::kRPT; ++i) {
    const uint32_t vo = v_lane + (row + C::kRP * i) * C::kRowBytes;
    t.v[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(vr, vo, 0, kStreamLoad));
  }
}

// Online-softmax state of one wave.
template <bool BF16, int D, int GP>
struct WaveState {
  using C = DecodeCfg<BF16, D, GP>;
  float m[4];                 // running max of heads 4*kg + v (uniform over the 16 key lanes)
  float l[4];                 // this lane's share of the running sum
  float acc[GP][C::kCPL];     // unnormalised output, columns cc*CPL.., rows of phase rp
};

// Packed tiles attend rows row + r < nrows of their range; paged tiles the
// rows r in [t.lo, t.hi) (row and nrows unused).
template <bool BF16, int D, int GP, bool PAGED>
__device__ __forceinline__ void compute_tile(WaveState<BF16, D, GP>& st, const Tile<BF16, D, GP>& t,
                                             const u32x4* qa, uint32_t row, uint32_t nrows, float scale_log2,
                                             float (*pb)[GP], float* ab, int j16, int kg, int rp) {
  using C = DecodeCfg<BF16, D, GP>;
  float sc[C::kKG][4];
#pragma unroll
  for (int kk = 0; kk < C::kKG; ++kk) {
    f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < C::kChunks; ++u) c = qk_mfma(qa[u], t.k[kk][u], c, BF16);
    const int r = 16 * kk + j16;
    const bool valid = PAGED ? (r >= t.lo && r < t.hi) : row + r < nrows;
#pragma unroll
    for (int v = 0; v < 4; ++v) sc[kk][v] = valid ? c[v] * scale_log2 : -INFINITY;
  }

  float alpha[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    float mt = sc[0][v];
#pragma unroll
    for (int kk = 1; kk < C::kKG; ++kk) mt = fmaxf(mt, sc[kk][v]);
    mt = row16_max(mt);
    const float m_new = fmaxf(st.m[v], mt);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    alpha[v] = fast_exp2(st.m[v] - m_use);
    float psum = 0.f;
#pragma unroll
    for (int kk = 0; kk < C::kKG; ++kk) {
      sc[kk][v] = fast_exp2(sc[kk][v] - m_use);
      psum += sc[kk][v];
    }
    st.l[v] = st.l[v] * alpha[v] + psum;
    st.m[v] = m_new;
  }

  if (4 * kg < GP) {
#pragma unroll
    for (int kk = 0; kk < C::kKG; ++kk) {
      f32x4 pv = {sc[kk][0], sc[kk][1], sc[kk][2], sc[kk][3]};
      *reinterpret_cast<f32x4*>(&pb[16 * kk + j16][4 * kg]) = pv;
    }
    if (j16 == 0) {
      f32x4 av = {alpha[0], alpha[1], alpha[2], alpha[3]};
      *reinterpret_cast<f32x4*>(&ab[4 * kg]) = av;
    }
  }
  wave_lds_fence();

  // Once the running maxima settle they rarely move, and then every factor
  // is exactly 1: the whole wave skips the rescale.
  if (__builtin_amdgcn_ballot_w64(alpha[0] != 1.f || alpha[1] != 1.f || alpha[2] != 1.f || alpha[3] != 1.f)) {
#pragma unroll
    for (int h4 = 0; h4 < GP / 4; ++h4) {
      const f32x4 al = *reinterpret_cast<const f32x4*>(&ab[4 * h4]);
#pragma unroll
      for (int v = 0; v < 4; ++v)
#pragma unroll
        for (int c = 0; c < C::kCPL; ++c) st.acc[4 * h4 + v][c] *= al[v];
    }
  }
#pragma unroll
  for (int i = 0; i < C::kRPT; ++i) {
    float vv[C::kCPL];
    widen16<BF16>(t.v[i], vv);
    const int r = C::kRP * i + rp;
#pragma unroll
    for (int h4 = 0; h4 < GP / 4; ++h4) {
      const f32x4 pr = *reinterpret_cast<const f32x4*>(&pb[r][4 * h4]);
#pragma unroll
      for (int v = 0; v < 4; ++v)
#pragma unroll
        for (int c = 0; c < C::kCPL; ++c) st.acc[4 * h4 + v][c] = fmaf(pr[v], vv[c], st.acc[4 * h4 + v][c]);
    }
  }
  wave_lds_fence();
}

// Work units of segment s in the flat split: its rows plus, when it has any,
// `seg_cost` units that stand for the fixed cost of a piece (loading the
// query, the cross-wave fold and the record).  A workgroup whose slice
// crosses a segment boundary pays that cost twice, so charging it here gives
// such a workgroup fewer rows and keeps the slowest workgroup close to the
// median.
// Paged segments have page_rows units per entry (the slots outside an
// entry's range are masked, not removed).  Row counts are multiples of 32.
template <bool PAGED>
__device__ __forceinline__ int64_t segment_rows(const DecodeParams& p, int s) {
  if (PAGED) {
    const int32_t n = p.n_entries[s];
    return (int64_t)(n < 0 ? 0 : (n > p.max_entries ? p.max_entries : n)) * p.page_rows;
  }
  if (p.seg_len == nullptr) return (int64_t)p.dense_len + p.n_new;
  // a negative length marks a segment dkv_compact could not pack: no rows
  // and no room to append
  const int32_t len = p.seg_len[s];
  return len < 0 ? 0 : (int64_t)len + p.n_tail + p.n_new;
}

// Flat prefix of work units over the call's segments: pre[s] = units of
// segments < s, pre[nseg] = total.  A non-empty segment s covers
// [pre[s], pre[s + 1]); its first seg_cost units are the fixed cost and its
// rows are the units after them.  The packed cache's segment offsets (the
// paged cache's row counts and flags) are copied to offs[] in the same pass, so the
// workgroup learns where its rows are after a single round trip to memory.
// Called by every thread of a workgroup; `red` holds kWaves + 1 int64 of LDS.
template <bool PAGED>
__device__ __forceinline__ void build_row_prefix(const DecodeParams& p, int64_t seg_cost, int64_t* pre,
                                                 int64_t* offs, int64_t* red) {
  const int tid = threadIdx.x;
  const int nseg = p.nseg;
  const int per = (nseg + kThreads - 1) / kThreads;
  const int s_lo = tid * per;
  const int s_hi = min(nseg, s_lo + per);
  int64_t sum = 0;
  for (int s = s_lo; s < s_hi; ++s) {
    if (!PAGED && p.seg_len != nullptr) offs[s] = p.seg_off[s];
    const int64_t rows = segment_rows<PAGED>(p, s);
    // paged: the row count, with bit 0 set when the segment's entry list was
    // cut at max_entries (its append-region entries may then be missing)
    if (PAGED) offs[s] = rows | (p.n_entries[s] > p.max_entries ? 1 : 0);
    const int64_t u = rows > 0 ? rows + seg_cost : 0;
    pre[s] = u;  // this thread's own slots: units now, prefix after the scan
    sum += u;
  }
  int64_t total_unused;
  int64_t run = block_exclusive_scan<kThreads>(sum, red, &total_unused);
  for (int s = s_lo; s < s_hi; ++s) {
    const int64_t u = pre[s];
    pre[s] = run;
    run += u;
  }
  if (s_hi == nseg && s_lo <= nseg) pre[nseg] = run;
  if (nseg == 0 && tid == 0) pre[0] = 0;
  __syncthreads();
}

// Register tiles per wave (pipeline depth of the K/V stream): the ring keeps
// S - 1 tiles loading, about 8 KiB per wave (bf16 d64 tiles are half that,
// fp32 d128 ones twice).
template <bool BF16, int D, int GP>
constexpr int decode_stages() {
  return (BF16 && D == 64) ? 3 : 2;
}

constexpr int kEntryChunk = kWave;  // paged entries held per wave (one per lane)

// An entry as validated when a wave loads it: one naming a page outside the
// pool or slots outside a page becomes empty.
struct PagedEntry {
  int32_t page, lpage, lo, hi;
};

// Chunk-relative bounds of a paged piece, all in rows of the segment's row
// space counted from the chunk's first entry (they fit 32 bits: a chunk
// holds at most kEntryChunk pages).
struct PagedChunk {
  int32_t r_base;  // first tile's row
  int32_t a, b;    // the piece [a, b), clamped to [-1, INT32_MAX]
  int32_t n;       // entries in the chunk
  uint32_t ntile;  // tiles of the piece in the chunk
};

// Descriptors of paged tile `t` of the current chunk: the tile's rows
// [r0, r0 + 32) lie in one page; the attended ones are [lo, hi) of the tile,
// clipped to the piece, the entry's slots and the positions below `limit`.
// The descriptors start at row lo, so rows before it get a wrapped (huge)
// offset and rows from hi on lie past the range: both read zeros without
// touching memory.  `row` is what load_tile adds to a row index to get the
// row's offset in the descriptor.  Tiles past the chunk read nothing.
template <bool BF16, int D, int GP>
__device__ __forceinline__ void paged_tile(const DecodeParams& p, const PagedEntry& ent, const PagedChunk& ck,
                                           uint32_t t, int32_t limit, __amdgpu_buffer_rsrc_t& kr,
                                           __amdgpu_buffer_rsrc_t& vr, uint32_t& row, int32_t& lo, int32_t& hi) {
  using C = DecodeCfg<BF16, D, GP>;
  const int sh = p.page_shift;  // page sizes are powers of two
  const int32_t r0 = ck.r_base + (int32_t)t * kTK;
  const int32_t e = r0 >> sh;
  const int li = e < ck.n - 1 ? e : ck.n - 1;
  const int32_t page = __builtin_amdgcn_readlane(ent.page, li);
  const int32_t lpage = __builtin_amdgcn_readlane(ent.lpage, li);
  const int32_t e_lo = __builtin_amdgcn_readlane(ent.lo, li);
  const int32_t e_hi = __builtin_amdgcn_readlane(ent.hi, li);
  const int32_t slot0 = r0 & ((1 << sh) - 1);
  int32_t l = ck.a - r0;
  if (e_lo - slot0 > l) l = e_lo - slot0;
  if (l < 0) l = 0;
  if (l > kTK) l = kTK;
  int32_t h = ck.b - r0;
  if (e_hi - slot0 < h) h = e_hi - slot0;
  if (limit - (lpage << sh) - slot0 < h) h = limit - (lpage << sh) - slot0;
  if (h > kTK) h = kTK;
  if (t >= ck.ntile || h < l) h = l;
  lo = l;
  hi = h;
  row = (uint32_t)(-l);
  const int64_t off = (((int64_t)page << sh) + slot0 + l) * C::kRowBytes;
  const uint32_t bytes = (uint32_t)(h - l) * C::kRowBytes;
  kr = make_rsrc(reinterpret_cast<const char*>(p.k) + off, bytes);
  vr = make_rsrc(reinterpret_cast<const char*>(p.v) + off, bytes);
}

template <bool BF16, int D, int GP, bool PAGED>
__global__ __launch_bounds__(kThreads) void decode_kernel(DecodeParams p) {
  using C = DecodeCfg<BF16, D, GP>;
  extern __shared__ __align__(16) int64_t pre[];          // [nseg + 1] unit prefix, then [nseg] offsets / rows
  int64_t* offs = pre + p.nseg + 1;
  __shared__ __align__(16) float pbuf[kWaves][kTK][GP];   // probabilities per wave tile
  __shared__ __align__(16) float abuf[kWaves][GP];        // rescale factors per wave
  __shared__ __align__(16) float wacc[kWaves][C::kRPK][GP][D];  // per-wave row-phase partial accumulators
  __shared__ float wm[kWaves][GP];
  __shared__ float wl[kWaves][GP];
  __shared__ int64_t red[kWaves + 1];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int w = blockIdx.x;
  const int nseg = p.nseg;
  const bool dense = !PAGED && p.seg_len == nullptr;

  // fixed cost of a piece, in rows: about as long as streaming 192 KiB of K
  // and V.  A piece restarts the ring (its first tiles wait out the load
  // queue: ~4 us under full load, per-workgroup clock stamps) and ends with
  // the cross-wave fold (~1.1 us); at ~25 KB/us per workgroup that is ~125
  // KiB, and more where a restart also empties the ring.  (Measured on
  // graph-replayed steps: 192 KiB takes 4-5% off the 70B-shaped batch at 10%
  // and 1-2% at 20% against 256 KiB; 128 KiB is within noise of 192; the
  // headline and Qwen-shaped stacks are unchanged from 128 to 384 KiB.)
  constexpr int64_t kSegCost = 196608 / (2 * C::kRowBytes);
  DKV_STAMP(const unsigned long long stamp_t0 = __builtin_amdgcn_s_memrealtime();)
  build_row_prefix<PAGED>(p, kSegCost, pre, offs, red);
  const int64_t total = uniform64(pre[nseg]);
  DKV_STAMP(unsigned long long* stamp = stamp_split[p.stamp_slot][w]; bool stamp_first = true;
            if (tid == 0) { stamp[0] = stamp_t0; stamp[1] = __builtin_amdgcn_s_memrealtime(); })

  // ---- segments with no rows at all produce zeros ----------------------
  for (int s = w; s < nseg; s += p.P) {
    if (pre[s + 1] == pre[s]) {
      const int b = s / p.Hkv, g = s - (s / p.Hkv) * p.Hkv;
      float* o = p.out + ((int64_t)b * p.Hq + (int64_t)g * p.G) * D;
      for (int i = tid; i < p.G * D; i += kThreads) o[i] = 0.f;
      if (tid == 0) {
        p.seg_meta[2 * s] = 0;
        p.seg_meta[2 * s + 1] = 0;  // nothing to combine
      }
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

  const char* qbytes = reinterpret_cast<const char*>(p.q);
  const int j16 = lane & 15;   // key (QK) / head row (A operand) within a 16-group
  const int kg = lane >> 4;    // 16-byte chunk group (QK)
  const int cc = lane % C::kLPR;
  const int rp = lane / C::kLPR;

  s = __builtin_amdgcn_readfirstlane(s);
  for (; s < nseg && pre[s] < hi; ++s) {
    // rows of segment s are the units [seg_lo, seg_hi); a workgroup whose
    // slice holds only the segment's fixed-cost units has no piece of it
    const int64_t seg_lo = uniform64(pre[s]) + kSegCost, seg_hi = uniform64(pre[s + 1]);
    const int64_t a = (lo > seg_lo ? lo : seg_lo) - seg_lo;
    const int64_t bnd = (hi < seg_hi ? hi : seg_hi) - seg_lo;
    if (a >= bnd) continue;
    const int bseq = s / p.Hkv;
    const int g = s - bseq * p.Hkv;
    const int64_t row0 = PAGED ? 0 : uniform64(dense ? (int64_t)s * p.dense_stride : offs[s]);
    const char* kbase = reinterpret_cast<const char*>(p.k) + row0 * C::kRowBytes;
    const char* vbase = reinterpret_cast<const char*>(p.v) + row0 * C::kRowBytes;

    // Tokens appended by this call are the segment's last n_new rows.  The
    // workgroup whose slice holds them writes them into the cache (they stay
    // for later steps) and is also the only one that reads them, so a
    // workgroup-scope fence and barrier order the writes before its loads.
    // (Paged segments append inside the entry loop below.)
    if (!PAGED && p.n_new > 0) {
      const int64_t base_len = seg_hi - seg_lo - p.n_new;
      const int64_t t_lo = (a > base_len ? a : base_len) - base_len;
      const int64_t t_hi = (bnd < base_len + p.n_new ? bnd : base_len + p.n_new) - base_len;
      if (t_lo < t_hi) {
        const u32x4* ks = reinterpret_cast<const u32x4*>(p.k_new) + ((int64_t)s * p.n_new) * C::kLPR;
        const u32x4* vs = reinterpret_cast<const u32x4*>(p.v_new) + ((int64_t)s * p.n_new) * C::kLPR;
        u32x4* kd = reinterpret_cast<u32x4*>(const_cast<char*>(kbase) + base_len * C::kRowBytes);
        u32x4* vd = reinterpret_cast<u32x4*>(const_cast<char*>(vbase) + base_len * C::kRowBytes);
        for (int64_t i = t_lo * C::kLPR + tid; i < t_hi * C::kLPR; i += kThreads) {
          kd[i] = ks[i];
          vd[i] = vs[i];
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __syncthreads();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
      }
    }

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

    WaveState<BF16, D, GP> st;
#pragma unroll
    for (int v = 0; v < 4; ++v) { st.m[v] = -INFINITY; st.l[v] = 0.f; }
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
      for (int c = 0; c < C::kCPL; ++c) st.acc[h][c] = 0.f;

    // Rows are addressed through buffer descriptors over at most kSubRows
    // rows at a time (32-bit offsets); the ragged end of each range reads
    // zeros and is masked out of the softmax.
    const uint32_t k_lane = (uint32_t)(j16 * C::kRowBytes + 16 * kg);
    const uint32_t v_lane = (uint32_t)(rp * C::kRowBytes + 16 * cc);
    constexpr int S = decode_stages<BF16, D, GP>();
    Tile<BF16, D, GP> tl[S];
    if constexpr (PAGED) {
      // Each wave loads the piece's entries kEntryChunk at a time, one per
      // lane; within a chunk the ring is the packed one, with descriptors
      // built per tile.
      const int64_t pr = p.page_rows;
      const int sh = p.page_shift;
      const int32_t limit = p.ctx_len + p.n_tail + p.n_new;  // checked to fit 31 bits
      const int32_t* ents = p.entries + (int64_t)s * p.max_entries * 4;
      const int64_t e_end = (bnd + pr - 1) >> sh;
      const int64_t enc = uniform64(offs[s]);
      // the append region is the last tail_entries entries, unless the list
      // was cut short
      const int64_t tail0 = (enc & 1) ? -1 : (enc >> sh) - p.tail_entries;
      for (int64_t c0 = a >> sh; c0 < e_end; c0 += kEntryChunk) {
        const int64_t c1 = c0 + kEntryChunk < e_end ? c0 + kEntryChunk : e_end;
        PagedEntry ent = {0, 0, 0, 0};
        if (lane < c1 - c0) {
          const int4 e = *reinterpret_cast<const int4*>(ents + (c0 + lane) * 4);
          // positions (logical page << shift) + slot must fit 31 bits
          const bool ok = e.x >= 0 && e.x < p.num_pages && e.y >= 0 && e.y <= (INT32_MAX >> sh) && e.z >= 0 &&
                          e.z < e.w && e.w <= pr;
          if (ok) ent = PagedEntry{e.x, e.y, e.z, e.w};
        }
        // Appended token k is position ctx_len + n_tail + k, a slot of one of
        // the append-region entries; the workgroup whose piece holds that
        // slot's row writes it, from the staged entry, before loading it.
        if (p.n_new > 0 && tail0 >= 0) {
          bool wrote = false;
          for (int k = 0; k < p.n_new; ++k) {
            const int64_t pos = (int64_t)p.ctx_len + p.n_tail + k;
            const int64_t e = tail0 + ((pos >> sh) - ((int64_t)p.ctx_len >> sh));
            const int64_t slot = pos & (pr - 1);
            const int64_t row = (e << sh) + slot;
            if (row < a || row >= bnd || e < c0 || e >= c1) continue;
            const int li = (int)(e - c0);
            if (__builtin_amdgcn_readlane(ent.lpage, li) != (pos >> sh) || slot < __builtin_amdgcn_readlane(ent.lo, li) ||
                slot >= __builtin_amdgcn_readlane(ent.hi, li))
              continue;
            const int64_t dst = (((int64_t)__builtin_amdgcn_readlane(ent.page, li) << sh) + slot) * C::kLPR;
            const int64_t src = ((int64_t)s * p.n_new + k) * C::kLPR;
            for (int i = tid; i < C::kLPR; i += kThreads) {
              reinterpret_cast<u32x4*>(const_cast<void*>(p.k))[dst + i] =
                  reinterpret_cast<const u32x4*>(p.k_new)[src + i];
              reinterpret_cast<u32x4*>(const_cast<void*>(p.v))[dst + i] =
                  reinterpret_cast<const u32x4*>(p.v_new)[src + i];
            }
            wrote = true;
          }
          if (wrote) {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            __syncthreads();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
          }
        }
        const int64_t cb = c0 << sh;
        const int64_t r_lo = a > cb ? a : cb;
        const int64_t r_hi = bnd < (c1 << sh) ? bnd : (c1 << sh);
        const int64_t k0 = r_lo / kTK;
        PagedChunk ck;
        ck.r_base = (int32_t)(k0 * kTK - cb);
        ck.a = (int32_t)(a - cb < -1 ? -1 : a - cb);
        ck.b = (int32_t)(bnd - cb > INT32_MAX ? INT32_MAX : bnd - cb);
        ck.n = (int32_t)(c1 - c0);
        ck.ntile = (uint32_t)((r_hi + kTK - 1) / kTK - k0);
        const uint32_t ntile = ck.ntile;
        uint32_t t = wave;
#pragma unroll
        for (int i = 0; i < S - 1; ++i) {
          __amdgpu_buffer_rsrc_t kr, vr;
          uint32_t rr;
          paged_tile<BF16, D, GP>(p, ent, ck, t + i * kWaves, limit, kr, vr, rr, tl[i].lo, tl[i].hi);
          load_tile(tl[i], kr, vr, rr, k_lane, v_lane);
          __builtin_amdgcn_sched_barrier(0);
        }
        const uint32_t n_round = t < ntile ? (ntile - t + S * kWaves - 1) / (S * kWaves) : 0;
        for (uint32_t r = 0; r < n_round; ++r) {
#pragma unroll
          for (int i = 0; i < S; ++i) {
            Tile<BF16, D, GP>& nx = tl[(i + S - 1) % S];
            __amdgpu_buffer_rsrc_t kr, vr;
            uint32_t rr;
            paged_tile<BF16, D, GP>(p, ent, ck, t + (S - 1) * kWaves, limit, kr, vr, rr, nx.lo, nx.hi);
            load_tile(nx, kr, vr, rr, k_lane, v_lane);
            __builtin_amdgcn_sched_barrier(0);
            if (t < ntile)
              compute_tile<BF16, D, GP, true>(st, tl[i], qa, 0, 0, p.scale_log2, pbuf[wave], abuf[wave], j16, kg,
                                              rp);
            t += kWaves;
          }
        }
      }
    }
    for (int64_t a2 = a; !PAGED && a2 < bnd; a2 += C::kSubRows) {
      const uint32_t nrows = (uint32_t)((bnd - a2) < C::kSubRows ? (bnd - a2) : C::kSubRows);
      const __amdgpu_buffer_rsrc_t kr = make_rsrc(kbase + a2 * C::kRowBytes, nrows * C::kRowBytes);
      const __amdgpu_buffer_rsrc_t vr = make_rsrc(vbase + a2 * C::kRowBytes, nrows * C::kRowBytes);
      const uint32_t ntile = (nrows + kTK - 1) / kTK;
      // A ring of S register tiles per wave: S - 1 later tiles are loading
      // while one is computed.  The ring is unrolled so each stage keeps its
      // own registers (reusing the registers of a tile still in flight makes
      // the compiler wait for it).  Prefetches are unconditional: past the
      // last tile their offsets fall outside the descriptor and read zeros
      // without touching memory, whereas a load under a branch makes the
      // compiler wait for every outstanding load.
      // Scheduling barriers keep every stage's loads ahead of its compute
      // and the prologue's tiles in ring order, so each compute waits only
      // for its own tile.
      uint32_t t = wave;
#pragma unroll
      for (int i = 0; i < S - 1; ++i) {
        load_tile(tl[i], kr, vr, (t + i * kWaves) * kTK, k_lane, v_lane);
        __builtin_amdgcn_sched_barrier(0);
      }
      // The loop runs whole rounds of S stages and has a single exit: an
      // exit after any stage makes the register allocator copy in-flight
      // tiles at the loop head, which waits for every outstanding load.
      // Stages past the last tile only issue (zero-returning) loads.
      const uint32_t n_round = t < ntile ? (ntile - t + S * kWaves - 1) / (S * kWaves) : 0;
      for (uint32_t r = 0; r < n_round; ++r) {
#pragma unroll
        for (int i = 0; i < S; ++i) {
          load_tile(tl[(i + S - 1) % S], kr, vr, (t + (S - 1) * kWaves) * kTK, k_lane, v_lane);
          __builtin_amdgcn_sched_barrier(0);
          if (t < ntile) {
            DKV_STAMP(if (stamp_first && wave == 0 && lane == 0) stamp[2] = __builtin_amdgcn_s_memrealtime();
                      stamp_first = false;)
            compute_tile<BF16, D, GP, false>(st, tl[i], qa, t * kTK, nrows, p.scale_log2, pbuf[wave], abuf[wave],
                                             j16, kg, rp);
          }
          t += kWaves;
        }
      }
    }

    DKV_STAMP(if (lane == 0) stamp[3 + wave] = __builtin_amdgcn_s_memrealtime();)
    // ---- wave state -> LDS ---------------------------------------------
    // Every lane's accumulators are partial sums over its row phase; they go
    // to LDS as they are (a cross-lane sum first only where the partials of
    // all waves would not fit), and the fold below adds them up.  (Summing
    // all row phases with lane swaps first cost ~0.5 us more per piece.)
#pragma unroll
    for (int v = 0; v < 4; ++v) st.l[v] = row16_sum(st.l[v]);
    if constexpr (C::kRPK < C::kRP) {
#pragma unroll
      for (int h = 0; h < GP; ++h)
#pragma unroll
        for (int c = 0; c < C::kCPL; ++c) st.acc[h][c] = lane_xor_sum<C::kRPK * C::kLPR>(st.acc[h][c]);
    }
    if (rp < C::kRPK) {
#pragma unroll
      for (int h = 0; h < GP; ++h)
#pragma unroll
        for (int c4 = 0; c4 < C::kCPL; c4 += 4)
          *reinterpret_cast<f32x4*>(&wacc[wave][rp][h][cc * C::kCPL + c4]) =
              f32x4{st.acc[h][c4], st.acc[h][c4 + 1], st.acc[h][c4 + 2], st.acc[h][c4 + 3]};
    }
    if (j16 == 0 && 4 * kg < GP) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        wm[wave][4 * kg + v] = st.m[v];
        wl[wave][4 * kg + v] = st.l[v];
      }
    }
    __syncthreads();

    // ---- combine the waves; write the output or a partial record ---------
    const int64_t w_first = owner_of(seg_lo, total, P);
    const int64_t w_last = owner_of(seg_hi - 1, total, P);
    const bool single = w_first == w_last;
    if (w == w_first && tid == 0) {
      // the combine kernel reads where the segment's records start and how
      // many there are (1: finished here, nothing to combine)
      p.seg_meta[2 * s] = (int32_t)(w_first + s);
      p.seg_meta[2 * s + 1] = (int32_t)(w_last - w_first + 1);
    }
    float* rec = p.partials + (int64_t)(w + s) * C::kRec;
    float* outp = p.out + ((int64_t)bseq * p.Hq + (int64_t)g * p.G) * D;
    // thread -> (head h, columns 4 c4 .. 4 c4 + 3)
    for (int idx = tid; idx < p.G * (D / 4); idx += kThreads) {
      const int h = idx / (D / 4), c = 4 * (idx - h * (D / 4));
      float M = wm[0][h];
#pragma unroll
      for (int q = 1; q < kWaves; ++q) M = fmaxf(M, wm[q][h]);
      const float Mu = M == -INFINITY ? 0.f : M;
      float L = 0.f;
      f32x4 A = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int q = 0; q < kWaves; ++q) {
        const float f = fast_exp2(wm[q][h] - Mu);
        L += f * wl[q][h];
        f32x4 part = *reinterpret_cast<const f32x4*>(&wacc[q][0][h][c]);
#pragma unroll
        for (int r = 1; r < C::kRPK; ++r) part += *reinterpret_cast<const f32x4*>(&wacc[q][r][h][c]);
        A += f * part;
      }
      if (single) {
        *reinterpret_cast<f32x4*>(outp + h * D + c) = A * (L > 0.f ? 1.f / L : 0.f);
      } else {
        *reinterpret_cast<f32x4*>(rec + 2 * GP + h * D + c) = A;
        if (c == 0) {
          rec[h] = M;
          rec[GP + h] = L;
        }
      }
    }
    __syncthreads();  // LDS is reused by the next piece
    DKV_STAMP(if (tid == 0) stamp[7] = __builtin_amdgcn_s_memrealtime();)
  }
}

// Combine kernel: one workgroup per (segment, query head).  The attention
// kernel left, per segment, the first record slot and the number of pieces
// (n <= 1: nothing to combine).  Thread (ph, cq) folds pieces
// k = ph, ph + kPhases, ... of columns 4cq..4cq+3 into its own running
// (max, sum, accumulator), loading kBatch pieces' records at once so that the
// merge costs one memory round trip per batch; the kPhases partial states are
// then folded through LDS in phase order:
//   M = max_k m_k,  out = sum_k 2^(m_k - M) acc_k / sum_k 2^(m_k - M) l_k.
// The order of combination is fixed, so the result does not depend on timing.
// The kernel boundary makes the records visible: neither kernel needs
// device-scope fences or counters.
template <int D, int GP>
__global__ __launch_bounds__(kThreads) void decode_merge_kernel(DecodeParams p) {
  constexpr int kRec = GP * (D + 2);
  constexpr int kQuads = D / 4;               // float4 column groups per head row
  constexpr int kPhases = kThreads / kQuads;  // pieces folded side by side
  constexpr int kBatch = 8;                   // pieces per thread per round trip
  __shared__ __align__(16) float xa[kThreads * 4];
  __shared__ float xm[kThreads], xl[kThreads];

  const int s = blockIdx.x / p.G;
  const int h = blockIdx.x - s * p.G;
  DKV_STAMP(const unsigned long long stamp_m0 = __builtin_amdgcn_s_memrealtime();
            unsigned long long* mstamp = stamp_merge[p.stamp_slot][blockIdx.x < kStampMergeWG ? blockIdx.x : 0];)
  const int n = p.seg_meta[2 * s + 1];
  if (n <= 1) {
    DKV_STAMP(if (threadIdx.x == 0) { mstamp[0] = stamp_m0; mstamp[1] = stamp_m0; })
    return;
  }
  const float* first = p.partials + (int64_t)p.seg_meta[2 * s] * kRec;
  const int tid = threadIdx.x;
  const int cq = tid % kQuads, ph = tid / kQuads;

  float M = -INFINITY, L = 0.f;
  f32x4 A = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = ph; k0 < n; k0 += kPhases * kBatch) {
    float m[kBatch], l[kBatch];
    f32x4 a[kBatch];
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const int k = k0 + i * kPhases;
      if (k < n) {
        const float* r = first + (int64_t)k * kRec;
        m[i] = r[h];
        l[i] = r[GP + h];
        a[i] = *reinterpret_cast<const f32x4*>(r + 2 * GP + h * D + 4 * cq);
      } else {
        m[i] = -INFINITY;
        l[i] = 0.f;
        a[i] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
    float mb = M;
#pragma unroll
    for (int i = 0; i < kBatch; ++i) mb = fmaxf(mb, m[i]);
    const float mu = mb == -INFINITY ? 0.f : mb;
    const float rs = fast_exp2(M - mu);
    L *= rs;
    A *= rs;
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const float f = fast_exp2(m[i] - mu);
      L += f * l[i];
      A += f * a[i];
    }
    M = mb;
  }
  xm[tid] = M;
  xl[tid] = L;
  *reinterpret_cast<f32x4*>(&xa[4 * tid]) = A;
  __syncthreads();
  if (tid < kQuads) {
    float Mx = -INFINITY;
    for (int q = 0; q < kPhases; ++q) Mx = fmaxf(Mx, xm[tid + q * kQuads]);
    const float mu = Mx == -INFINITY ? 0.f : Mx;
    float Lt = 0.f;
    f32x4 At = {0.f, 0.f, 0.f, 0.f};
    for (int q = 0; q < kPhases; ++q) {
      const int t = tid + q * kQuads;
      const float f = fast_exp2(xm[t] - mu);
      Lt += f * xl[t];
      At += f * *reinterpret_cast<const f32x4*>(&xa[4 * t]);
    }
    const int bseq = s / p.Hkv, g = s - bseq * p.Hkv;
    float* o = p.out + ((int64_t)bseq * p.Hq + (int64_t)g * p.G + h) * D + 4 * cq;
    *reinterpret_cast<f32x4*>(o) = At * (Lt > 0.f ? 1.f / Lt : 0.f);
  }
  DKV_STAMP(__syncthreads(); if (threadIdx.x == 0) { mstamp[0] = stamp_m0; mstamp[1] = __builtin_amdgcn_s_memrealtime(); })
}

#if DKV_PHASE_STAMPS
std::atomic<int>& stamp_slot_counter() {
  static std::atomic<int> c{0};
  return c;
}
int stamp_next_slot() { return stamp_slot_counter().fetch_add(1) % kStampCalls; }
#endif

// Split count: about one 128-row slice per workgroup, capped at one workgroup
// per compute unit (so every slice starts immediately, all finish together,
// and each unit streams one slice: two resident workgroups per unit doubled
// the bytes in flight and ran slower) and at the workspace bound.  The
// device's compute-unit count is looked up once per device and cached: the
// query costs more host time than a launch.
constexpr int kMaxDevices = 64;

inline int device_cus(int dev) {
  static std::atomic<int> cache[kMaxDevices];
  if (dev < 0 || dev >= kMaxDevices) dev = 0;
  int c = cache[dev].load(std::memory_order_relaxed);
  if (c <= 0) {
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || c <= 0) c = 256;
    cache[dev].store(c, std::memory_order_relaxed);
  }
  return c;
}

int32_t split_count(int64_t rows_hint) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) dev = 0;
  int64_t cap = device_cus(dev);
  if (cap > kDecodeMaxWG) cap = kDecodeMaxWG;
  if (rows_hint <= 0) return (int32_t)cap;
  int64_t P = (rows_hint + 127) / 128;
  return (int32_t)(P < 1 ? 1 : (P > cap ? cap : P));
}

template <bool BF16, int D, int GP>
hipError_t launch_g(DecodeParams p, int64_t rows_hint, hipStream_t stream) {
  const size_t lds = (2 * (size_t)p.nseg + 1) * sizeof(int64_t);
  DKV_STAMP(p.stamp_slot = stamp_next_slot();)
  if (p.entries != nullptr) {
    p.P = split_count(rows_hint);
    hipLaunchKernelGGL((decode_kernel<BF16, D, GP, true>), dim3(p.P), dim3(kThreads), lds, stream, p);
  } else {
    p.P = split_count(rows_hint);
    hipLaunchKernelGGL((decode_kernel<BF16, D, GP, false>), dim3(p.P), dim3(kThreads), lds, stream, p);
  }
  // Segments split over several workgroups are finished by the combine
  // kernel; when the call has a single split there is nothing to combine.
  if (p.P > 1)
    hipLaunchKernelGGL((decode_merge_kernel<D, GP>), dim3(p.nseg * p.G), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

template <bool BF16, int D>
hipError_t launch_d(const DecodeParams& p, int GP, int64_t rows_hint, hipStream_t stream) {
  switch (GP) {
    case 4: return launch_g<BF16, D, 4>(p, rows_hint, stream);
    case 8: return launch_g<BF16, D, 8>(p, rows_hint, stream);
    case 16: return launch_g<BF16, D, 16>(p, rows_hint, stream);
    default: return hipErrorInvalidValue;
  }
}

// Scratch of the allocation-free entry point (dkv_append_decode_attn_noalloc):
// the split's partial records and segment metadata, in a file-scope array
// that every GPU the library runs on holds until the process ends.  Host code
// never passes the array's name to a kernel (on the host it is a stand-in,
// not a device address); it passes the address hipGetSymbolAddress returns
// for the current device.  The records need no initial contents.
static __device__ __align__(256) unsigned char scratch[DKV_NOALLOC_SCRATCH_BYTES];

}  // namespace

#if DKV_PHASE_STAMPS
}  // namespace dkv
// Phase-stamp build only: the stamps of every call slot, and a reset of the
// slot counter (launches take slots 0, 1, ... modulo 64 from then on).
extern "C" int dkv_phase_stamps(void* split, void* merge) {
  hipError_t e = hipMemcpyFromSymbol(split, HIP_SYMBOL(dkv::stamp_split), sizeof(dkv::stamp_split));
  if (e == hipSuccess) e = hipMemcpyFromSymbol(merge, HIP_SYMBOL(dkv::stamp_merge), sizeof(dkv::stamp_merge));
  return (int)e;
}
extern "C" void dkv_phase_reset() { dkv::stamp_slot_counter().store(0); }
namespace dkv {
#endif

hipError_t decode_static_scratch(void** ptr) {
  static std::atomic<void*> addr[kMaxDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* a = addr[dev].load(std::memory_order_acquire);
  if (a == nullptr) {
    // once per device, with that device current: each GPU holds its own copy
    e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (e != hipSuccess || a == nullptr) return e != hipSuccess ? e : hipErrorInvalidSymbol;
    addr[dev].store(a, std::memory_order_release);
  }
  *ptr = a;
  return hipSuccess;
}

int decode_group_pad(int G) { return G <= 4 ? 4 : (G <= 8 ? 8 : 16); }

size_t decode_partials_bytes(int nseg, int G, int head_dim) {
  const size_t rec = (size_t)decode_group_pad(G) * (head_dim + 2) * 4;
  return ((size_t)kDecodeMaxWG + nseg) * rec;
}

size_t decode_workspace_bytes(int nseg, int G, int head_dim) {
  return decode_partials_bytes(nseg, G, head_dim) + (size_t)nseg * 2 * sizeof(int32_t);
}

hipError_t launch_decode(const DecodeParams& p, dkv_dtype dtype, int head_dim, int64_t rows_hint,
                         hipStream_t stream) {
  const int GP = decode_group_pad(p.G);
  if (dtype == DKV_BF16) {
    if (head_dim == 128) return launch_d<true, 128>(p, GP, rows_hint, stream);
    if (head_dim == 64) return launch_d<true, 64>(p, GP, rows_hint, stream);
  } else {
    if (head_dim == 128) return launch_d<false, 128>(p, GP, rows_hint, stream);
    if (head_dim == 64) return launch_d<false, 64>(p, GP, rows_hint, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace dkv
