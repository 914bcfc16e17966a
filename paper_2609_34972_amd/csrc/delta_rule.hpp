// Host-side launcher of the gated delta-rule visual write (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "build_kernels.hpp"

namespace dv {

// Workspace of the chunked delta rule: per (sequence, value head, chunk of 64 tokens) the
// products W [64][dk], Uv [64][dv], Kt [dk][64] in the call dtype and gamma_C (fp32), and per
// segment of the two-level scan the affine map (Phi, Psi) in fp32.
struct GdrWs {
  void* w_;
  void* uv_;
  void* kt_;
  float* gc;
  float* phi;  // per segment: the linear part Phi [dk][dk] of the segment's affine map
  float* psi;  // per segment: the state Psi [dk][dv] it reaches from a zero start
  int P;       // segments of the two-level scan (1: a single in-order scan)
  int cps;     // chunks per segment
  size_t bytes;
  template <typename T>
  __host__ __device__ T* w(int64_t chunk, int dk) const { return (T*)w_ + chunk * 64 * dk; }
  template <typename T>
  __host__ __device__ T* uv(int64_t chunk, int dv) const { return (T*)uv_ + chunk * 64 * dv; }
  template <typename T>
  __host__ __device__ T* kt(int64_t chunk, int dk) const { return (T*)kt_ + chunk * 64 * dk; }
};

// Layout of the workspace at base (sizes only when base is null).
GdrWs gdr_layout(void* base, int B, int Hv, int N, int dk, int dv, int dtype);

// S [B,Hv,dk,dv] fp32 <- state after writing tokens 0..N-1 (dtype 0 = fp32, 1 = bf16 for k, v).
hipError_t launch_delta_rule(const void* k, const void* v, const float* alpha, const float* beta,
                             float* S, int B, int Hk, int Hv, int N, int dk, int dv, int dtype,
                             GdrWs ws, hipStream_t s, const LaunchEvents& ev);

}  // namespace dv
