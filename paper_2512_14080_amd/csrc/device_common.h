// Device helpers shared by the gfx950 kernels: bf16 conversion, vector types
// and wave64 reductions.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace smoe {

constexpr int kWave = 64;

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// fp32 -> bf16, round to nearest even (gfx950 v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint16_t f2bf(float x) {
  __bf16 h = (__bf16)x;
  return __builtin_bit_cast(uint16_t, h);
}
typedef float f32x2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
// two fp32 -> packed bf16 pair (one v_cvt_pk_bf16_f32, round to nearest even)
__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
  const f32x2v v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2v));
}
// logistic sigmoid with the hardware exp and reciprocal (about 1 ulp each)
__device__ __forceinline__ float fast_sigmoid(float x) { return __builtin_amdgcn_rcpf(1.f + __expf(-x)); }

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
// inclusive scan over the wave
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    int t = __shfl_up(v, o, kWave);
    if (l >= o) v += t;
  }
  return v;
}

// Wave reductions with DPP (no LDS): quad swaps, half-row and row mirrors,
// then the row broadcasts; lane 63 ends with the result, which is read back
// as a wave-uniform value.  Lanes that receive no value keep their own.
template <int CTRL, int ROW_MASK, class T>
__device__ __forceinline__ T dpp_mov(T v) {
  if constexpr (sizeof(T) == 8) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const int lo = (int)(uint32_t)u, hi = (int)(uint32_t)(u >> 32);
    const uint32_t nlo = (uint32_t)__builtin_amdgcn_update_dpp(lo, lo, CTRL, ROW_MASK, 0xf, false);
    const uint32_t nhi = (uint32_t)__builtin_amdgcn_update_dpp(hi, hi, CTRL, ROW_MASK, 0xf, false);
    return __builtin_bit_cast(T, ((uint64_t)nhi << 32) | nlo);
  } else {
    const int b = __builtin_bit_cast(int, v);
    return __builtin_bit_cast(T, __builtin_amdgcn_update_dpp(b, b, CTRL, ROW_MASK, 0xf, false));
  }
}

template <class T, class Op>
__device__ __forceinline__ T dpp_reduce(T x, Op op) {
  x = op(x, dpp_mov<0xB1, 0xf>(x));   // quad_perm [1,0,3,2]
  x = op(x, dpp_mov<0x4E, 0xf>(x));   // quad_perm [2,3,0,1]
  x = op(x, dpp_mov<0x141, 0xf>(x));  // row_half_mirror
  x = op(x, dpp_mov<0x140, 0xf>(x));  // row_mirror: every lane holds its row's value
  x = op(x, dpp_mov<0x142, 0xa>(x));  // row_bcast:15 into rows 1 and 3
  x = op(x, dpp_mov<0x143, 0xc>(x));  // row_bcast:31 into rows 2 and 3
  if constexpr (sizeof(T) == 8) {
    const uint64_t u = __builtin_bit_cast(uint64_t, x);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), 63);
    return __builtin_bit_cast(T, ((uint64_t)hi << 32) | lo);
  } else {
    return __builtin_bit_cast(T, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 63));
  }
}

// 64-bit value of lane l (wave-uniform l).  The readlane builtin works on
// 32-bit ints: given a 64-bit argument it keeps only the sign-extended low
// half, so the two halves are read separately.
__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int l = lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// Block-wide exclusive scan of one int per thread (blockDim = 256 or 1024).
template <int NT>
__device__ __forceinline__ int block_excl_scan(int v, int* total, int* lds) {
  const int wave = threadIdx.x >> 6;
  const int lane = lane_id();
  const int inc = wave_incl_scan(v);
  if (lane == 63) lds[wave] = inc;
  __syncthreads();
  if (wave == 0) {
    int s = lane < NT / 64 ? lds[lane] : 0;
    s = wave_incl_scan(s);
    if (lane < NT / 64) lds[lane] = s;
  }
  __syncthreads();
  const int base = wave ? lds[wave - 1] : 0;
  *total = lds[NT / 64 - 1];
  __syncthreads();
  return base + inc - v;
}

}  // namespace smoe
