// Wave-level helpers for gfx950 (64-lane wavefronts).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace omnimoe {

constexpr int kWave = 64;

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }

// Workgroups are dispatched to the eight XCDs round robin (workgroup b runs on XCD b % 8).
// xcd_contiguous(b, n) is a bijection on [0, n) under which each XCD works through one
// contiguous block of items, so neighbouring items share an L2 (and its partial lines).
__device__ __forceinline__ int64_t xcd_contiguous(int64_t b, int64_t n) {
  constexpr int kXcds = 8;
  const int64_t full = n - n % kXcds;
  if (b >= full) return b;
  return (b % kXcds) * (full / kXcds) + b / kXcds;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  return (1ull << lane_id()) - 1ull;
}

// Orders a wave's own LDS traffic: every lane's earlier LDS writes are visible to the
// wave's later LDS reads.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// fp32 -> bf16 bits, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Order-preserving maps of floats onto unsigned integers (larger value -> larger key);
// -0 maps like +0.
__device__ __forceinline__ uint32_t ord_f32(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u << 1) == 0u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float f32_from_ord(uint32_t o) {
  uint32_t u = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
  return __uint_as_float(u);
}
__device__ __forceinline__ uint64_t ord_f64(double f) {
  uint64_t u = (uint64_t)__double_as_longlong(f);
  if ((u << 1) == 0ull) u = 0ull;
  return (u & 0x8000000000000000ull) ? ~u : (u | 0x8000000000000000ull);
}
__device__ __forceinline__ double f64_from_ord(uint64_t o) {
  uint64_t u = (o & 0x8000000000000000ull) ? (o & 0x7FFFFFFFFFFFFFFFull) : ~o;
  return __longlong_as_double((long long)u);
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  lo = (uint32_t)__shfl_xor((int)lo, m, kWave);
  hi = (uint32_t)__shfl_xor((int)hi, m, kWave);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  lo = (uint32_t)__shfl((int)lo, src, kWave);
  hi = (uint32_t)__shfl((int)hi, src, kWave);
  return ((uint64_t)hi << 32) | lo;
}

// Sum over the wave; every lane receives the same value (each butterfly level adds the
// same two partial sums on both partners, and fp addition commutes).
__device__ __forceinline__ float wave_sum_f32(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}
__device__ __forceinline__ int wave_sum_i32(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}
// Exclusive prefix sum over lanes.
__device__ __forceinline__ int wave_excl_scan_i32(int v) {
  int x = v;
  const int l = lane_id();
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) {
    int y = __shfl_up(x, m, kWave);
    if (l >= m) x += y;
  }
  return x - v;
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2_bf16(uint32_t p, uint32_t q, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, p),
                                         __builtin_bit_cast(bf16x2, q), acc, false);
}

// fp32 dot of one 16-byte chunk pair (bf16 pairs through v_dot2_f32_bf16), the products
// added in a fixed order; the expert dot kernels and the fused selection share it, so that
// every path forms the same a[p].
template <bool BF16>
__device__ __forceinline__ float chunk_dot(const uint4& p, const uint4& q, float acc) {
  if constexpr (BF16) {
    acc = dot2_bf16(p.x, q.x, acc);
    acc = dot2_bf16(p.y, q.y, acc);
    acc = dot2_bf16(p.z, q.z, acc);
    acc = dot2_bf16(p.w, q.w, acc);
  } else {
    acc = fmaf(__uint_as_float(p.x), __uint_as_float(q.x), acc);
    acc = fmaf(__uint_as_float(p.y), __uint_as_float(q.y), acc);
    acc = fmaf(__uint_as_float(p.z), __uint_as_float(q.z), acc);
    acc = fmaf(__uint_as_float(p.w), __uint_as_float(q.w), acc);
  }
  return acc;
}

// Wave-uniform sum: DPP adds within each 16-lane row (quad swaps, then rotations by 4 and 8),
// then the four row sums read out in a fixed order. Every lane gets the same value.
__device__ __forceinline__ float wave_sum_uniform(float v) {
  int x = __float_as_int(v);
  v += __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0xB1, 0xF, 0xF, false));  // quad [1,0,3,2]
  x = __float_as_int(v);
  v += __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0x4E, 0xF, 0xF, false));  // quad [2,3,0,1]
  x = __float_as_int(v);
  v += __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0x124, 0xF, 0xF, false));  // row_ror:4
  x = __float_as_int(v);
  v += __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0x128, 0xF, 0xF, false));  // row_ror:8
  x = __float_as_int(v);
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(x, 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(x, 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(x, 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(x, 48));
  return (r0 + r1) + (r2 + r3);
}

// Integer wave sum with the same DPP pattern; every lane gets the total.
__device__ __forceinline__ int wave_sum_uniform_i32(int v) {
  v += __builtin_amdgcn_update_dpp(v, v, 0xB1, 0xF, 0xF, false);   // quad [1,0,3,2]
  v += __builtin_amdgcn_update_dpp(v, v, 0x4E, 0xF, 0xF, false);   // quad [2,3,0,1]
  v += __builtin_amdgcn_update_dpp(v, v, 0x124, 0xF, 0xF, false);  // row_ror:4
  v += __builtin_amdgcn_update_dpp(v, v, 0x128, 0xF, 0xF, false);  // row_ror:8
  return (__builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16)) +
         (__builtin_amdgcn_readlane(v, 32) + __builtin_amdgcn_readlane(v, 48));
}

__device__ __forceinline__ int readlane_i32(int v, int lane) {
  return __builtin_amdgcn_readlane(v, lane);
}
__device__ __forceinline__ float readlane_f32(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// Activation of Eq. 4 in fp32. GELU uses Phi(z) = erfc(-z / sqrt 2) / 2, which keeps full
// relative precision for negative z, where 1 + erf(z / sqrt 2) would cancel.
__device__ __forceinline__ float activation(int act, float z) {
  if (act == 1) return z / (1.0f + expf(-z));
  return 0.5f * z * erfcf(-z * 0.70710678118654752f);
}

// Its derivative: GELU (erf form) z Phi(z) -> Phi(z) + z phi(z); SiLU z s(z) ->
// s(z) (1 + z (1 - s(z))).
__device__ __forceinline__ float activation_grad(int act, float z) {
  if (act == 1) {
    const float sg = 1.0f / (1.0f + expf(-z));
    return sg * (1.0f + z * (1.0f - sg));
  }
  return 0.5f * erfcf(-z * 0.70710678118654752f) + z * expf(-0.5f * z * z) * 0.39894228040143268f;
}

}  // namespace omnimoe
