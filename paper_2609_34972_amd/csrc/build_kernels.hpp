// Host-side launchers of the visual-memory build kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>

namespace dv {

// Optional hipEvent pairs recorded around kernel launches (profiling hook).
struct LaunchEvents {
  hipEvent_t down[2] = {nullptr, nullptr};
  hipEvent_t up[2] = {nullptr, nullptr};
  hipEvent_t kv[2] = {nullptr, nullptr};
  hipEvent_t attn[2] = {nullptr, nullptr};
  hipEvent_t gdr_prep[2] = {nullptr, nullptr};
  hipEvent_t gdr_scan[2] = {nullptr, nullptr};
};

inline void record(hipEvent_t e, hipStream_t s) {
  if (e) (void)hipEventRecord(e, s);
}

// Z[l] = phi(E D_l) for all layers (dtype 0 = fp32, 1 = bf16; act 0 = SiLU, 1 = GELU).
hipError_t launch_down_act(const void* E, const void* Dw, void* Z, int64_t T, int d, int L, int r,
                           int act, int dtype, hipStream_t s, const LaunchEvents& ev);

// Number of fp32 partial sums of squares per row written by the up kernel of this call, and
// the largest count over every variant (used to size the workspace).
int kv_partials(int d, int r, int dtype);
int kv_partials_max(int d);

// Backbone epilogue of the visual K/V: projection bias, per-head key RMSNorm and rotary
// embedding from a prepared table. A null member skips its step.
struct KvEpiArgs {
  const void* k_bias = nullptr;  // [L, Hkv*hd], call dtype
  const void* v_bias = nullptr;  // [L, Hkv*hd], call dtype
  const void* k_norm = nullptr;  // [L, hd], call dtype
  float k_norm_eps = 0.f;
  const float* rope = nullptr;   // [T][hd/2] (cos, sin) pairs from launch_rope_table
  bool any() const { return k_bias || v_bias || k_norm || rope; }
};

// cos/sin table of the rotary embedding for every visual token: entry (t, j) for token
// t = b*Nv + i turns by pos[b][a][i] * theta^(-2j/hd), a = position axis of frequency j
// (sections s0, s1, s2 of hd/2 frequencies). table holds T*hd/2 (cos, sin) float pairs.
hipError_t launch_rope_table(const int32_t* pos, int B, int Nv, int hd, int s0, int s1,
                             float theta, float* table, hipStream_t s);

// Layers l0..l0+nl-1: memory, RMSNorm and K/V projection. Mg holds nl*T*d
// elements of the call dtype and ssq nl*kv_partials(d)*T floats. With epi, the backbone
// epilogue is applied to the projected K/V (fused into the bf16 pipelined kernel).
hipError_t launch_project_kv(const void* E, const void* Z, const void* Uw, const void* gamma,
                             const void* Wk, const void* Wv, void* Kv, void* Vv, int B, int Nv,
                             int d, int r, int Hkv, int hd, int l0, int nl, float eps, int dtype,
                             void* Mg, float* ssq, hipStream_t s, const LaunchEvents& ev,
                             bool first_group, bool last_group, const KvEpiArgs* epi = nullptr);

// Which kernel computes M_l * gamma_l and the row sums of squares for the bf16 projection:
// 0 picks by shape (the Z-resident kernel for r = 256 once there are at least eight rounds of its
// blocks), 1 always the tiled kernel, 2 the Z-resident kernel wherever it applies (r = 256, 512).
void set_up_kernel(int mode);
bool up_z_resident(int64_t T, int d, int r, int nl);

// The fused kernel (fused_kv.hip) computes M_l, its RMSNorm and the K/V projection of 64 tokens
// in one block and needs no workspace. It covers bf16, 2 Hkv hd = 1024, r in {128, 256, 512},
// d a multiple of 64, no backbone epilogue (up_kv_fused_eligible), and the projection takes it
// only once switched on (set_up_kv_fused; off at load).
bool up_kv_fused_eligible(int d, int r, int Hkv, int hd, int dtype);
void set_up_kv_fused(bool on);
bool up_kv_fused(int d, int r, int Hkv, int hd, int dtype, bool epilogue);
hipError_t launch_up_kv_fused(const void* E, const void* Z, const void* Uw, const void* gamma,
                              const void* Wk, const void* Wv, void* Kv, void* Vv, int B, int Nv,
                              int d, int r, int Hkv, int hd, int l0, int nl, float eps,
                              hipStream_t s);

// K/V projection alone (Eq. 7) for layers l0..l0+nl-1 from a prepared workspace: Mg holds
// M_l * gamma_l for each layer of the range (call dtype) and ssq np partial sums of M_l^2 per row.
hipError_t launch_kv_only(const void* Mg, const float* ssq, const void* Wk, const void* Wv,
                          void* Kv, void* Vv, int B, int Nv, int d, int Hkv, int hd, int l0, int nl,
                          int np, float eps, int dtype, hipStream_t s, const LaunchEvents& ev);

// Workspace layout of the recurrent adapter (byte offsets, 256-aligned).
struct RecLayout {
  size_t mg, ssq, state, op, z, part, bytes;
  int np;      // RMSNorm partial sums per row
  int splits;  // split-K factor of the per-layer down projection
  int kchunk;  // reduction length of one split (a multiple of the K tile)
};
RecLayout recurrent_layout(int64_t T, int d, int L, int r, int dtype);

// Recurrent adapter (Eq. 6) for all L layers followed by the K/V projection of every layer.
hipError_t launch_recurrent(const void* E, const void* Dw, const void* Uw, const void* gamma,
                            const void* Wk, const void* Wv, void* Kv, void* Vv, int B, int Nv,
                            int d, int L, int r, int Hkv, int hd, int act, float eps, int dtype,
                            void* ws, const RecLayout& w, hipStream_t s, const LaunchEvents& ev);

}  // namespace dv
