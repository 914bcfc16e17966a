// Measurement probe: the sustained bf16 MFMA rate of the GPU on register operands.
//
// The clock of gfx950 drops under MFMA load, and the more the operand bits toggle the further
// it drops, so the rate a GEMM can reach depends on its data. The probe runs the same
// instruction as the pipelined GEMM engine (v_mfma_f32_16x16x32_bf16, 64 x 128 fragments per
// wave, 8 waves per block, 1024 blocks) with no memory traffic at all, once on random bf16
// operands and once on constant ones; the bench reports the GEMM's rate against both.
#include "probe.hpp"
#include "dv_device.hpp"

namespace dv {

__device__ __forceinline__ uint32_t probe_hash(uint32_t x) {
  x *= 2654435761u;
  x ^= x >> 13;
  x *= 0x5bd1e995u;
  x ^= x >> 15;
  return x;
}

// Two bf16 values with random signs and mantissas and exponents spread over 2^-8 .. 2^-1.
__device__ __forceinline__ uint32_t probe_bf16x2(uint32_t seed) {
  const uint32_t x = probe_hash(seed);
  const uint32_t lo = (x & 0x807fu) | ((119u + ((x >> 7) & 7u)) << 7);
  const uint32_t hi = ((x >> 16) & 0x807fu) | ((119u + ((x >> 23) & 7u)) << 7);
  return lo | (hi << 16);
}

template <bool RANDOM>
__global__ __launch_bounds__(512) void k_probe_mfma(float* __restrict__ sink, int iters) {
  constexpr int FM = 4, FN = 8;
  bf16x8 fa[FM], fb[FN];
  const uint32_t t = blockIdx.x * 512u + threadIdx.x;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    u32x4 v;
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = RANDOM ? probe_bf16x2(t * 64u + i * 4u + e) : 0x3f803f80u;
    fa[i] = __builtin_bit_cast(bf16x8, v);
  }
#pragma unroll
  for (int i = 0; i < FN; ++i) {
    u32x4 v;
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = RANDOM ? probe_bf16x2(t * 64u + 16u + i * 4u + e) : 0x3f803f80u;
    fb[i] = __builtin_bit_cast(bf16x8, v);
  }
  f32x4 acc[FM][FN];
#pragma unroll
  for (int a = 0; a < FM; ++a)
#pragma unroll
    for (int b = 0; b < FN; ++b) acc[a][b] = f32x4{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int a = 0; a < FM; ++a)
#pragma unroll
      for (int b = 0; b < FN; ++b)
        acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[b], fa[a], acc[a][b], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int a = 0; a < FM; ++a)
#pragma unroll
    for (int b = 0; b < FN; ++b) s += acc[a][b][0] + acc[a][b][1] + acc[a][b][2] + acc[a][b][3];
  if (threadIdx.x == 0) sink[blockIdx.x] = s;
}

hipError_t launch_probe_mfma(bool random, int iters, float* sink, hipStream_t s) {
  if (random)
    k_probe_mfma<true><<<kProbeBlocks, 512, 0, s>>>(sink, iters);
  else
    k_probe_mfma<false><<<kProbeBlocks, 512, 0, s>>>(sink, iters);
  return hipGetLastError();
}

}  // namespace dv
