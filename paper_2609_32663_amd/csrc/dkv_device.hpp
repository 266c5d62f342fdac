// Device-side helpers shared by the Distance-KV HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dkv {

constexpr int kWave = 64;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// bf16 halves of a 32-bit word, widened exactly to fp32.
__device__ __forceinline__ float bf16_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t x) { return __uint_as_float(x & 0xffff0000u); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ---------------------------------------------------------------------------
// DPP reductions inside each 16-lane row of a wave.  quad_perm [1,0,3,2] and
// [2,3,0,1] combine within a quad, row_half_mirror pairs the two quads of an
// 8-lane half, row_mirror pairs the two halves; afterwards every lane of the
// row holds the row's result.
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ float row16_max(float x) {
  x = fmaxf(x, dpp_mov<0xB1>(x));
  x = fmaxf(x, dpp_mov<0x4E>(x));
  x = fmaxf(x, dpp_mov<0x141>(x));
  x = fmaxf(x, dpp_mov<0x140>(x));
  return x;
}

__device__ __forceinline__ float row16_sum(float x) {
  x += dpp_mov<0xB1>(x);
  x += dpp_mov<0x4E>(x);
  x += dpp_mov<0x141>(x);
  x += dpp_mov<0x140>(x);
  return x;
}

// Sum over the lanes of a wave that share (lane % FROM), FROM in {8, 16, 32}:
// lanes i and i ^ 8 meet through a rotation by 8 inside each 16-lane row,
// i ^ 16 and i ^ 32 through the permlane swaps (each swap exchanges half of
// one copy with the other half of a second copy, so adding the two copies
// gives every lane its partner's value).  Every lane ends with the sum.
template <int FROM>
__device__ __forceinline__ float lane_xor_sum(float x) {
  static_assert(FROM == 8 || FROM == 16 || FROM == 32, "unsupported stride");
  if constexpr (FROM <= 8) x += dpp_mov<0x128>(x);  // row_ror:8
  if constexpr (FROM <= 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Keeps the compiler from moving LDS accesses of one wave across this point.
// LDS instructions of a single wave execute in issue order, so no wait is
// needed between a lane's write and another lane's later read.
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// ---------------------------------------------------------------------------
// Block-wide exclusive scan of one int64 per thread.  `tmp` holds NT/64 + 1
// int64 in LDS.  Returns the exclusive prefix; *total receives the sum.
// Must be called by every thread of the block.
// ---------------------------------------------------------------------------
template <int NT>
__device__ __forceinline__ int64_t block_exclusive_scan(int64_t v, int64_t* tmp, int64_t* total) {
  constexpr int NW = NT / kWave;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  int64_t x = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    int64_t y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  if (lane == kWave - 1) tmp[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t run = 0;
    for (int w = 0; w < NW; ++w) {
      int64_t t = tmp[w];
      tmp[w] = run;
      run += t;
    }
    tmp[NW] = run;
  }
  __syncthreads();
  const int64_t excl = x - v + tmp[wave];
  *total = tmp[NW];
  __syncthreads();
  return excl;
}

// Number of nonzero bytes in a 32-bit word.
__device__ __forceinline__ int nonzero_bytes(uint32_t x) {
  uint32_t y = ((x & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | x;
  return __popc(y & 0x80808080u);
}

// Bit e set when byte e of the 16 bytes is nonzero.
__device__ __forceinline__ uint32_t nonzero_byte_bits(u32x4 w) {
  uint32_t bits = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t x = w[q];
#pragma unroll
    for (int b = 0; b < 4; ++b) bits |= (((x >> (8 * b)) & 0xFFu) != 0u ? 1u : 0u) << (4 * q + b);
  }
  return bits;
}

// The 16 mask bytes of positions [j0, j0+16) of one mask row, zero beyond T
// (16-byte loads when every row starts 16-byte aligned, bytes otherwise).
__device__ __forceinline__ u32x4 load_mask16(const uint8_t* row, int64_t j0, int32_t T) {
  u32x4 w = {0u, 0u, 0u, 0u};
  if ((T & 15) == 0) {
    if (j0 < T) w = *reinterpret_cast<const u32x4*>(row + j0);
  } else {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int64_t j = j0 + e;
      const uint32_t b = (j < T && row[j] != 0) ? 1u : 0u;
      w[e >> 2] |= b << (8 * (e & 3));
    }
  }
  return w;
}

}  // namespace dkv
