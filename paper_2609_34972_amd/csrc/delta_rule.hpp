// Host-side launcher of the gated delta-rule visual write (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "build_kernels.hpp"

namespace dv {

// Workspace of the chunked delta rule: per (sequence, value head, chunk of 64 tokens) one
// record of -W [64][dk], Kt [dk][64] and Uv^T [dv][64] in the call dtype (in the fragment order
// of the chunk kernels) and gamma_C (fp32), and per segment of the two-level scan the affine
// map (Phi, Psi) in fp32.
struct GdrWs {
  void* rec_;
  float* gc;
  float* phi;     // per segment: the linear part Phi [dk][dk] of the segment's affine map
  float* psi;     // per segment: the state Psi [dk][dv] it reaches (segment 0: from S)
  int P;          // segments of the two-level scan (1: a single in-order scan)
  int cps;        // chunks per segment
  int rec_elems;  // elements per chunk record, 64 (2 dk + dv)
  size_t bytes;
  template <typename T>
  __host__ __device__ T* rec(int64_t chunk) const { return (T*)rec_ + chunk * rec_elems; }
};

// Layout of the workspace at base (sizes only when base is null).
GdrWs gdr_layout(void* base, int B, int Hv, int N, int dk, int dv, int dtype);

// S [B,Hv,dk,dv] fp32 <- state after writing tokens 0..N-1 (dtype 0 = fp32, 1 = bf16 for k, v).
hipError_t launch_delta_rule(const void* k, const void* v, const float* alpha, const float* beta,
                             float* S, int B, int Hk, int Hv, int N, int dk, int dv, int dtype,
                             GdrWs ws, hipStream_t s, const LaunchEvents& ev);

}  // namespace dv
