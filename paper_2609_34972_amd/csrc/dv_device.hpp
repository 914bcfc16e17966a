// Device-side building blocks for gfx950 (CDNA4): vector types, MFMA steps,
// bf16 rounding and the LDS swizzle shared by the GEMM-shaped kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dv {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int WAVE = 64;

// Eight consecutive K-elements held by one lane for one 16-deep K step of a
// 32x32 MFMA tile: lanes 0..31 hold k = 0..7 of rows/cols 0..31, lanes 32..63
// hold k = 8..15. Any assignment of k to (lane half, slot) is valid as long as
// both operands use the same one, since the instruction sums over all of them.
template <typename T> struct Frag8;
template <> struct Frag8<bf16> { typedef bf16x8 type; };
template <> struct Frag8<float> { typedef f32x8 type; };

// acc(32x32, fp32) += A(32x16) * B(16x32)
__device__ __forceinline__ void mfma_k16(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ void mfma_k16(f32x16& acc, const f32x8& a, const f32x8& b) {
#pragma unroll
  for (int j = 0; j < 8; ++j) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[j], b[j], acc, 0, 0, 0);
}

// Row (within a 32x32 accumulator tile) of accumulator item i for this lane;
// the column is lane % 32.
__device__ __forceinline__ int acc_row(int lane, int i) {
  return (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3);
}

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }  // RNE

// XOR swizzle of 16-byte chunks inside 128-byte LDS rows. Consecutive row pairs
// share one 256-byte bank line, so the XOR key is (row / 2) mod 8: the 16 rows
// read together by a 32x32 fragment load then hit 16 distinct bank groups.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

__device__ __forceinline__ float silu(float x) { return x / (1.0f + __expf(-x)); }
__device__ __forceinline__ float gelu(float x) { return 0.5f * x * erfcf(-x * 0.70710678118654752f); }

template <typename V>
__device__ __forceinline__ V shfl_xor(V v, int mask) {
  return __shfl_xor(v, mask, WAVE);
}

}  // namespace dv
