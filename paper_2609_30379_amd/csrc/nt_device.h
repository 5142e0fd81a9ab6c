// Device-side helpers for gfx950 (CDNA4, wave64): vector types, bf16/fp32
// conversion, 16-byte vector loads/stores and the bf16 matrix-core op.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nt {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// D(16x16, f32) += A(16x32, bf16) * B(32x16, bf16).  Lane l supplies A row
// l%16 and B column l%16, each with eight k values selected by l/16; the k
// order is the same for A and B, so any consistent k permutation gives the
// same product.  Lane l receives D rows 4*(l/16) + i, i = 0..3, column l%16.
__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// ---- pair-tiled operand layout -----------------------------------------------
// One channel plane of sample i (an N x N matrix, rows r, columns k) is cut
// into 16 x 32 tiles, row tiles outer, each tile stored in the lane order of a
// matrix-core fragment: element (r, k) of a tile sits at ((k/8)*16 + r%16)*8
// + k%8, so lane l of a wave reads the 8 consecutive k of tile row l%16 and
// k-group l/16 as one 16-byte piece and the whole wave reads 1 KB contiguously.
// Planes occupy round_up(N,16) x round_up(N,32) elements; nkt = round_up(N,32)/32.
__host__ __device__ __forceinline__ int32_t tiled_offset(int32_t r, int32_t k, int32_t nkt) {
  return (((r >> 4) * nkt + (k >> 5)) << 9) + ((((k & 31) >> 3) << 4) + (r & 15)) * 8 + (k & 7);
}

// ---- 16-byte vectors of a storage type, converted to/from fp32 ------------
template <typename T> struct Vec;

template <> struct Vec<float> {
  static constexpr int N = 4;
  float v[4];
  __device__ __forceinline__ void load(const float* p) {
    const float4 t = *reinterpret_cast<const float4*>(p);
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  }
  __device__ __forceinline__ void store(float* p) const {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
};

template <> struct Vec<bf16> {
  static constexpr int N = 8;
  float v[8];
  __device__ __forceinline__ void load(const bf16* p) {
    const uint4 t = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[2 * j] = __uint_as_float(w[j] << 16);
      v[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
    }
  }
  __device__ __forceinline__ void store(bf16* p) const {
    bf16x8 t;
#pragma unroll
    for (int j = 0; j < 8; ++j) t[j] = (bf16)v[j];
    *reinterpret_cast<bf16x8*>(p) = t;
  }
};

// Non-temporal 16- and 8-byte stores (streaming hint: the lines are not kept
// in the caches on the way out).
typedef uint32_t u32x4_nt __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_nt __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void store_nt(bf16* p, const bf16x8& v) {
  __builtin_nontemporal_store(__builtin_bit_cast(u32x4_nt, v), reinterpret_cast<u32x4_nt*>(p));
}
__device__ __forceinline__ void store_nt(bf16* p, const bf16x4& v) {
  __builtin_nontemporal_store(__builtin_bit_cast(u32x2_nt, v), reinterpret_cast<u32x2_nt*>(p));
}

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }

// Sum over the four lanes l, l^16, l^32, l^48 (the k-groups holding one row
// of a matrix-core fragment): two lane-row swaps, no LDS round trip.  Every
// lane adds the same two values in either order, so all four get identical
// bits.
__device__ __forceinline__ float sum_over_kgroups(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Reductions within aligned groups of `width` lanes (width a power of two <= 64).
template <int width>
__device__ __forceinline__ float group_sum(float x) {
#pragma unroll
  for (int m = width / 2; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}
template <int width>
__device__ __forceinline__ float group_max(float x) {
#pragma unroll
  for (int m = width / 2; m >= 1; m >>= 1) x = fmaxf(x, __shfl_xor(x, m, 64));
  return x;
}

}  // namespace nt
