// C ABI of the visual-memory library: argument validation, workspace layout
// and dispatch to the gfx950 kernels. Every check runs on the host before
// anything is enqueued, so a rejected call launches nothing and writes nothing.
#include "../../include/deltavision.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "attention.hpp"
#include "build_kernels.hpp"
#include "delta_rule.hpp"
#include "probe.hpp"

namespace {

thread_local char g_err[512] = "";
thread_local dv::LaunchEvents g_ev;

dv_status fail(dv_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

dv_status ok() {
  g_err[0] = '\0';
  return DV_OK;
}

// Token rows per call: the row-tile index of the GEMM kernels is a 16-bit grid
// dimension (65535 tiles of 64 rows).
constexpr int64_t kMaxTokens = 65535LL * 64;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t elem_size(int32_t dtype) { return dtype == DV_BF16 ? 2 : 4; }

dv_status check_dtype(int32_t dtype) {
  if (dtype != DV_F32 && dtype != DV_BF16)
    return fail(DV_ERR_UNSUPPORTED, "dtype %d is not DV_F32 or DV_BF16", dtype);
  return DV_OK;
}

#define DV_CHECK(expr)              \
  do {                              \
    dv_status s_ = (expr);          \
    if (s_ != DV_OK) return s_;     \
  } while (0)

dv_status need_ptr(const void* p, const char* name) {
  if (!p) return fail(DV_ERR_NULL, "%s is NULL", name);
  if (!aligned16(p)) return fail(DV_ERR_ALIGN, "%s is not 16-byte aligned", name);
  return DV_OK;
}

dv_status hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(DV_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

// DV_DEBUG set (and not "0") in the environment: every call waits for the kernels it enqueued and
// reports a failure of any of them (a memory fault, an invalid launch) as DV_ERR_HIP from that
// call, instead of from some later HIP call.
bool debug_sync() {
  const char* v = std::getenv("DV_DEBUG");
  return v && *v && std::strcmp(v, "0") != 0;
}

// Status of a call whose kernels have been enqueued on stream s (launch result e).
dv_status launched(hipError_t e, const char* what, hipStream_t s) {
  if (e != hipSuccess) return fail(DV_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  if (debug_sync()) {
    e = hipStreamSynchronize(s);
    if (e == hipSuccess) e = hipGetLastError();
    if (e != hipSuccess)
      return fail(DV_ERR_HIP, "%s: the enqueued kernels failed (DV_DEBUG): %s", what,
                  hipGetErrorString(e));
  }
  return ok();
}

// Bytes of one layer's slot in the projection workspace: the gamma-weighted
// memory in the call dtype, then the fp32 partial sums of squares.
size_t kv_ws_layer_bytes(int64_t T, int32_t d, int32_t dtype) {
  const size_t mem = (size_t)T * (size_t)d * elem_size(dtype);
  const size_t mem_al = (mem + 255) / 256 * 256;
  const size_t ssq = (size_t)dv::kv_partials_max(d) * (size_t)T * 4;
  return mem_al + (ssq + 255) / 256 * 256;
}

}  // namespace

extern "C" {

int32_t dv_abi_version(void) { return 1; }

const char* dv_status_string(int32_t status) {
  switch (status) {
    case DV_OK: return "DV_OK";
    case DV_ERR_NULL: return "DV_ERR_NULL";
    case DV_ERR_SHAPE: return "DV_ERR_SHAPE";
    case DV_ERR_UNSUPPORTED: return "DV_ERR_UNSUPPORTED";
    case DV_ERR_ALIGN: return "DV_ERR_ALIGN";
    case DV_ERR_WORKSPACE: return "DV_ERR_WORKSPACE";
    case DV_ERR_HIP: return "DV_ERR_HIP";
    case DV_ERR_INTERNAL: return "DV_ERR_INTERNAL";
    default: return "DV_UNKNOWN_STATUS";
  }
}

const char* dv_last_error(void) { return g_err; }

dv_status dv_time_kernel(int32_t kernel, void* ev_begin, void* ev_end) {
  if ((ev_begin == nullptr) != (ev_end == nullptr))
    return fail(DV_ERR_NULL, "dv_time_kernel needs both events or neither");
  hipEvent_t* slot = nullptr;
  switch (kernel) {
    case DV_KERNEL_DOWN: slot = g_ev.down; break;
    case DV_KERNEL_UP: slot = g_ev.up; break;
    case DV_KERNEL_KV: slot = g_ev.kv; break;
    case DV_KERNEL_ATTENTION: slot = g_ev.attn; break;
    case DV_KERNEL_DELTA_PREP: slot = g_ev.gdr_prep; break;
    case DV_KERNEL_DELTA_SCAN: slot = g_ev.gdr_scan; break;
    default: return fail(DV_ERR_UNSUPPORTED, "unknown kernel id %d", kernel);
  }
  slot[0] = (hipEvent_t)ev_begin;
  slot[1] = (hipEvent_t)ev_end;
  return ok();
}

dv_status dv_probe_mfma(int32_t random, int32_t iters, float* sink, void* stream) {
  DV_CHECK(need_ptr(sink, "sink"));
  if (iters < 1 || iters > (1 << 20))
    return fail(DV_ERR_SHAPE, "iters=%d must lie in [1, 2^20]", iters);
  return launched(dv::launch_probe_mfma(random != 0, iters, sink, (hipStream_t)stream),
                  "dv_probe_mfma launch", (hipStream_t)stream);
}

dv_status dv_build_visual_memory(const void* E, const void* Dw, void* Z, int64_t T, int32_t d,
                                 int32_t L, int32_t r, int32_t act, int32_t dtype, void* stream) {
  DV_CHECK(check_dtype(dtype));
  if (T <= 0 || d <= 0 || L <= 0 || r <= 0)
    return fail(DV_ERR_SHAPE, "sizes must be positive (T=%lld d=%d L=%d r=%d)", (long long)T, d, L, r);
  if (T > kMaxTokens || (int64_t)L * r > INT32_MAX)
    return fail(DV_ERR_SHAPE, "T=%lld exceeds %lld or L*r=%lld exceeds 2^31-1", (long long)T,
                (long long)kMaxTokens, (long long)L * r);
  if (d % 64 != 0) return fail(DV_ERR_UNSUPPORTED, "d=%d must be a multiple of 64", d);
  if (r % 16 != 0) return fail(DV_ERR_UNSUPPORTED, "r=%d must be a multiple of 16", r);
  if (act != DV_ACT_SILU && act != DV_ACT_GELU)
    return fail(DV_ERR_UNSUPPORTED, "act=%d is not DV_ACT_SILU or DV_ACT_GELU", act);
  DV_CHECK(need_ptr(E, "E"));
  DV_CHECK(need_ptr(Dw, "Dw"));
  DV_CHECK(need_ptr(Z, "Z"));
  return launched(dv::launch_down_act(E, Dw, Z, T, d, L, r, act, dtype == DV_BF16 ? 1 : 0,
                                      (hipStream_t)stream, g_ev),
                  "dv_build_visual_memory launch", (hipStream_t)stream);
}

size_t dv_project_visual_kv_workspace(int64_t T, int32_t d, int32_t nl, int32_t dtype) {
  if (T <= 0 || d <= 0 || nl <= 0 || (dtype != DV_F32 && dtype != DV_BF16)) return 0;
  return (size_t)nl * kv_ws_layer_bytes(T, d, dtype);
}

int32_t dv_project_visual_kv_fused(int32_t d, int32_t r, int32_t Hkv, int32_t hd, int32_t dtype) {
  if (d <= 0 || r <= 0 || Hkv <= 0 || hd <= 0 || (dtype != DV_F32 && dtype != DV_BF16)) return 0;
  return dv::up_kv_fused(d, r, Hkv, hd, dtype == DV_BF16 ? 1 : 0, false) ? 1 : 0;
}

dv_status dv_set_fused_kv(int32_t on) {
  if (on != 0 && on != 1) return fail(DV_ERR_SHAPE, "on must be 0 or 1 (got %d)", on);
  dv::set_up_kv_fused(on != 0);
  return ok();
}

dv_status dv_set_up_kernel(int32_t mode) {
  if (mode < 0 || mode > 2) return fail(DV_ERR_SHAPE, "mode must be 0, 1 or 2 (got %d)", mode);
  dv::set_up_kernel(mode);
  return ok();
}

int32_t dv_project_visual_kv_up_kernel(int64_t T, int32_t d, int32_t r, int32_t nl,
                                       int32_t dtype) {
  if (T <= 0 || d <= 0 || r <= 0 || nl <= 0 || dtype != DV_BF16) return 1;
  return dv::up_z_resident(T, d, r, nl) ? 2 : 1;
}

}  // extern "C"

namespace {

size_t rope_table_bytes(int64_t T, int32_t hd) { return ((size_t)T * (size_t)hd * 4 + 255) / 256 * 256; }

dv_status check_epilogue(const dv_kv_epilogue* epi, int32_t hd) {
  if (!epi) return DV_OK;
  if (epi->k_bias && !aligned16(epi->k_bias)) return fail(DV_ERR_ALIGN, "k_bias is not 16-byte aligned");
  if (epi->v_bias && !aligned16(epi->v_bias)) return fail(DV_ERR_ALIGN, "v_bias is not 16-byte aligned");
  if (epi->k_norm) {
    if (!aligned16(epi->k_norm)) return fail(DV_ERR_ALIGN, "k_norm is not 16-byte aligned");
    if (!(epi->k_norm_eps >= 0.f) || !std::isfinite(epi->k_norm_eps))
      return fail(DV_ERR_SHAPE, "k_norm_eps must be finite and >= 0");
  }
  if (epi->positions) {
    if ((reinterpret_cast<uintptr_t>(epi->positions) & 3u) != 0)
      return fail(DV_ERR_ALIGN, "positions is not 4-byte aligned");
    const int32_t* sc = epi->rope_sections;
    if (sc[0] < 0 || sc[1] < 0 || sc[2] < 0 || (int64_t)sc[0] + sc[1] + sc[2] != hd / 2)
      return fail(DV_ERR_SHAPE, "rope_sections {%d, %d, %d} must be >= 0 and add up to hd/2 = %d",
                  sc[0], sc[1], sc[2], hd / 2);
    if (!std::isfinite(epi->rope_theta) || !(epi->rope_theta > 0.f))
      return fail(DV_ERR_SHAPE, "rope_theta must be finite and > 0");
  }
  return DV_OK;
}

dv_status project_impl(const void* E, const void* Z, const void* Uw, const void* gamma,
                       const void* Wk, const void* Wv, void* Kv, void* Vv, int32_t B, int32_t Nv,
                       int32_t d, int32_t L, int32_t r, int32_t Hkv, int32_t hd, int32_t l0,
                       int32_t nl, float eps, const dv_kv_epilogue* epi, int32_t dtype, void* ws,
                       size_t ws_bytes, hipStream_t stream, const char* name) {
  DV_CHECK(check_dtype(dtype));
  if (B <= 0 || Nv <= 0 || d <= 0 || L <= 0 || r <= 0 || Hkv <= 0 || hd <= 0)
    return fail(DV_ERR_SHAPE, "sizes must be positive (B=%d Nv=%d d=%d L=%d r=%d Hkv=%d hd=%d)", B,
                Nv, d, L, r, Hkv, hd);
  if (l0 < 0 || nl <= 0 || l0 + nl > L)
    return fail(DV_ERR_SHAPE, "layer range [%d, %d) is not inside [0, %d)", l0, l0 + nl, L);
  const int64_t T = (int64_t)B * Nv;
  if (T > kMaxTokens || (int64_t)2 * Hkv * hd > INT32_MAX || nl > 65535)
    return fail(DV_ERR_SHAPE, "B*Nv=%lld exceeds %lld (or nl > 65535)", (long long)T,
                (long long)kMaxTokens);
  if (d % 64 != 0) return fail(DV_ERR_UNSUPPORTED, "d=%d must be a multiple of 64", d);
  if (r % 16 != 0) return fail(DV_ERR_UNSUPPORTED, "r=%d must be a multiple of 16", r);
  if (hd != 64 && hd != 128) return fail(DV_ERR_UNSUPPORTED, "hd=%d must be 64 or 128", hd);
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(DV_ERR_SHAPE, "eps must be finite and >= 0");
  DV_CHECK(check_epilogue(epi, hd));
  DV_CHECK(need_ptr(E, "E"));
  DV_CHECK(need_ptr(Z, "Z"));
  DV_CHECK(need_ptr(Uw, "Uw"));
  DV_CHECK(need_ptr(gamma, "gamma"));
  DV_CHECK(need_ptr(Wk, "Wk"));
  DV_CHECK(need_ptr(Wv, "Wv"));
  DV_CHECK(need_ptr(Kv, "Kv"));
  DV_CHECK(need_ptr(Vv, "Vv"));
  const bool rope = epi && epi->positions;
  const size_t table = rope ? rope_table_bytes(T, hd) : 0;
  const size_t per_layer = kv_ws_layer_bytes(T, d, dtype);
  if (!ws || ws_bytes < table + per_layer)
    return fail(DV_ERR_WORKSPACE, "workspace of %zu bytes is below the one-layer minimum %zu",
                ws ? ws_bytes : (size_t)0, table + per_layer);
  if (!aligned16(ws)) return fail(DV_ERR_ALIGN, "ws is not 16-byte aligned");
  dv::KvEpiArgs ea;
  if (epi) {
    ea.k_bias = epi->k_bias;
    ea.v_bias = epi->v_bias;
    ea.k_norm = epi->k_norm;
    ea.k_norm_eps = epi->k_norm_eps;
  }
  if (rope) {
    ea.rope = (const float*)ws;
    hipError_t e = dv::launch_rope_table(epi->positions, B, Nv, hd, epi->rope_sections[0],
                                         epi->rope_sections[1], epi->rope_theta, (float*)ws, stream);
    if (e != hipSuccess) return hip_status(e, name);
  }
  char* slots = (char*)ws + table;
  const int group = (int)std::min<size_t>((size_t)nl, (ws_bytes - table) / per_layer);
  const size_t mem_al = ((size_t)T * d * elem_size(dtype) + 255) / 256 * 256;
  for (int g0 = 0; g0 < nl; g0 += group) {
    const int gl = std::min(group, nl - g0);
    void* Mg = slots;
    float* ssq = (float*)(slots + (size_t)gl * mem_al);
    hipError_t e = dv::launch_project_kv(E, Z, Uw, gamma, Wk, Wv, Kv, Vv, B, Nv, d, r, Hkv, hd,
                                         l0 + g0, gl, eps, dtype == DV_BF16 ? 1 : 0, Mg, ssq,
                                         stream, g_ev, g0 == 0, g0 + gl >= nl,
                                         ea.any() ? &ea : nullptr);
    if (e != hipSuccess) return hip_status(e, name);
  }
  return launched(hipSuccess, name, stream);
}

}  // namespace

extern "C" {

dv_status dv_project_visual_kv(const void* E, const void* Z, const void* Uw, const void* gamma,
                               const void* Wk, const void* Wv, void* Kv, void* Vv, int32_t B,
                               int32_t Nv, int32_t d, int32_t L, int32_t r, int32_t Hkv,
                               int32_t hd, int32_t l0, int32_t nl, float eps, int32_t dtype,
                               void* ws, size_t ws_bytes, void* stream) {
  return project_impl(E, Z, Uw, gamma, Wk, Wv, Kv, Vv, B, Nv, d, L, r, Hkv, hd, l0, nl, eps,
                      nullptr, dtype, ws, ws_bytes, (hipStream_t)stream,
                      "dv_project_visual_kv launch");
}

size_t dv_project_visual_kv_ex_workspace(int64_t T, int32_t d, int32_t nl, int32_t hd,
                                         int32_t dtype) {
  if (T <= 0 || d <= 0 || nl <= 0 || (hd != 64 && hd != 128) ||
      (dtype != DV_F32 && dtype != DV_BF16))
    return 0;
  return rope_table_bytes(T, hd) + (size_t)nl * kv_ws_layer_bytes(T, d, dtype);
}

dv_status dv_project_visual_kv_ex(const void* E, const void* Z, const void* Uw, const void* gamma,
                                  const void* Wk, const void* Wv, void* Kv, void* Vv, int32_t B,
                                  int32_t Nv, int32_t d, int32_t L, int32_t r, int32_t Hkv,
                                  int32_t hd, int32_t l0, int32_t nl, float eps,
                                  const dv_kv_epilogue* epi, int32_t dtype, void* ws,
                                  size_t ws_bytes, void* stream) {
  return project_impl(E, Z, Uw, gamma, Wk, Wv, Kv, Vv, B, Nv, d, L, r, Hkv, hd, l0, nl, eps, epi,
                      dtype, ws, ws_bytes, (hipStream_t)stream, "dv_project_visual_kv_ex launch");
}

size_t dv_recurrent_visual_kv_workspace(int64_t T, int32_t d, int32_t L, int32_t r,
                                        int32_t dtype) {
  if (T <= 0 || d <= 0 || L <= 0 || r <= 0 || (dtype != DV_F32 && dtype != DV_BF16)) return 0;
  return dv::recurrent_layout(T, d, L, r, dtype == DV_BF16 ? 1 : 0).bytes;
}

dv_status dv_recurrent_visual_kv(const void* E, const void* Dw, const void* Uw, const void* gamma,
                                 const void* Wk, const void* Wv, void* Kv, void* Vv, int32_t B,
                                 int32_t Nv, int32_t d, int32_t L, int32_t r, int32_t Hkv,
                                 int32_t hd, int32_t act, float eps, int32_t dtype, void* ws,
                                 size_t ws_bytes, void* stream) {
  DV_CHECK(check_dtype(dtype));
  if (B <= 0 || Nv <= 0 || d <= 0 || L <= 0 || r <= 0 || Hkv <= 0 || hd <= 0)
    return fail(DV_ERR_SHAPE, "sizes must be positive (B=%d Nv=%d d=%d L=%d r=%d Hkv=%d hd=%d)", B,
                Nv, d, L, r, Hkv, hd);
  const int64_t T = (int64_t)B * Nv;
  if (T > kMaxTokens || (int64_t)2 * Hkv * hd > INT32_MAX || L > 65535)
    return fail(DV_ERR_SHAPE, "B*Nv=%lld exceeds %lld (or L > 65535)", (long long)T,
                (long long)kMaxTokens);
  if (d % 64 != 0) return fail(DV_ERR_UNSUPPORTED, "d=%d must be a multiple of 64", d);
  if (r % 16 != 0) return fail(DV_ERR_UNSUPPORTED, "r=%d must be a multiple of 16", r);
  if (hd != 64 && hd != 128) return fail(DV_ERR_UNSUPPORTED, "hd=%d must be 64 or 128", hd);
  if (act != DV_ACT_SILU && act != DV_ACT_GELU)
    return fail(DV_ERR_UNSUPPORTED, "act=%d is not DV_ACT_SILU or DV_ACT_GELU", act);
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(DV_ERR_SHAPE, "eps must be finite and >= 0");
  DV_CHECK(need_ptr(E, "E"));
  DV_CHECK(need_ptr(Dw, "Dw"));
  DV_CHECK(need_ptr(Uw, "Uw"));
  DV_CHECK(need_ptr(gamma, "gamma"));
  DV_CHECK(need_ptr(Wk, "Wk"));
  DV_CHECK(need_ptr(Wv, "Wv"));
  DV_CHECK(need_ptr(Kv, "Kv"));
  DV_CHECK(need_ptr(Vv, "Vv"));
  const dv::RecLayout w = dv::recurrent_layout(T, d, L, r, dtype == DV_BF16 ? 1 : 0);
  if (!ws || ws_bytes < w.bytes)
    return fail(DV_ERR_WORKSPACE, "workspace of %zu bytes is below the required %zu",
                ws ? ws_bytes : (size_t)0, w.bytes);
  if (!aligned16(ws)) return fail(DV_ERR_ALIGN, "ws is not 16-byte aligned");
  return launched(dv::launch_recurrent(E, Dw, Uw, gamma, Wk, Wv, Kv, Vv, B, Nv, d, L, r, Hkv,
                                       hd, act, eps, dtype == DV_BF16 ? 1 : 0, ws, w,
                                       (hipStream_t)stream, g_ev),
                  "dv_recurrent_visual_kv launch", (hipStream_t)stream);
}

// Z of the kept layers (call dtype, 256-byte aligned) followed by the projection slots.
static size_t kept_z_bytes(int64_t T, int32_t r, int32_t nkeep, int32_t dtype) {
  return ((size_t)nkeep * (size_t)T * (size_t)r * elem_size(dtype) + 255) / 256 * 256;
}

size_t dv_kept_visual_kv_workspace(int64_t T, int32_t d, int32_t r, int32_t nkeep,
                                   int32_t dtype) {
  if (T <= 0 || d <= 0 || r <= 0 || nkeep <= 0 || (dtype != DV_F32 && dtype != DV_BF16)) return 0;
  return kept_z_bytes(T, r, nkeep, dtype) + (size_t)nkeep * kv_ws_layer_bytes(T, d, dtype);
}

dv_status dv_kept_visual_kv(const void* E, const void* Dw, const void* Uw, const void* gamma,
                            const void* Wk, const void* Wv, const uint8_t* keep, void* Kv,
                            void* Vv, int32_t B, int32_t Nv, int32_t d, int32_t L, int32_t r,
                            int32_t Hkv, int32_t hd, int32_t act, float eps, int32_t dtype,
                            void* ws, size_t ws_bytes, void* stream) {
  DV_CHECK(check_dtype(dtype));
  if (B <= 0 || Nv <= 0 || d <= 0 || L <= 0 || r <= 0 || Hkv <= 0 || hd <= 0)
    return fail(DV_ERR_SHAPE, "sizes must be positive (B=%d Nv=%d d=%d L=%d r=%d Hkv=%d hd=%d)", B,
                Nv, d, L, r, Hkv, hd);
  const int64_t T = (int64_t)B * Nv;
  if (T > kMaxTokens || (int64_t)2 * Hkv * hd > INT32_MAX || L > 65535 ||
      (int64_t)L * r > INT32_MAX)
    return fail(DV_ERR_SHAPE, "B*Nv=%lld exceeds %lld (or L > 65535)", (long long)T,
                (long long)kMaxTokens);
  if (d % 64 != 0) return fail(DV_ERR_UNSUPPORTED, "d=%d must be a multiple of 64", d);
  if (r % 16 != 0) return fail(DV_ERR_UNSUPPORTED, "r=%d must be a multiple of 16", r);
  if (hd != 64 && hd != 128) return fail(DV_ERR_UNSUPPORTED, "hd=%d must be 64 or 128", hd);
  if (act != DV_ACT_SILU && act != DV_ACT_GELU)
    return fail(DV_ERR_UNSUPPORTED, "act=%d is not DV_ACT_SILU or DV_ACT_GELU", act);
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(DV_ERR_SHAPE, "eps must be finite and >= 0");
  if (!keep) return fail(DV_ERR_NULL, "keep is NULL");
  int nkeep = 0;
  for (int l = 0; l < L; ++l) nkeep += keep[l] != 0;
  if (nkeep == 0) return ok();
  DV_CHECK(need_ptr(E, "E"));
  DV_CHECK(need_ptr(Dw, "Dw"));
  DV_CHECK(need_ptr(Uw, "Uw"));
  DV_CHECK(need_ptr(gamma, "gamma"));
  DV_CHECK(need_ptr(Wk, "Wk"));
  DV_CHECK(need_ptr(Wv, "Wv"));
  DV_CHECK(need_ptr(Kv, "Kv"));
  DV_CHECK(need_ptr(Vv, "Vv"));
  const size_t zb = kept_z_bytes(T, r, nkeep, dtype);
  const size_t per_layer = kv_ws_layer_bytes(T, d, dtype);
  if (!ws || ws_bytes < zb + per_layer)
    return fail(DV_ERR_WORKSPACE, "workspace of %zu bytes is below the minimum %zu",
                ws ? ws_bytes : (size_t)0, zb + per_layer);
  if (!aligned16(ws)) return fail(DV_ERR_ALIGN, "ws is not 16-byte aligned");
  const size_t e = elem_size(dtype);
  const size_t kvw = (size_t)Hkv * hd;
  const size_t mem_al = ((size_t)T * d * e + 255) / 256 * 256;
  const int group = (int)std::min<size_t>((size_t)nkeep, (ws_bytes - zb) / per_layer);
  char* Zall = (char*)ws;
  char* pw = Zall + zb;
  const int bf = dtype == DV_BF16 ? 1 : 0;
  hipStream_t s = (hipStream_t)stream;
  // Runs of consecutive kept layers [a, b) fill cache slots [c, c + b - a). Weights are
  // addressed from layer a, Z and the caches from slot c, so each run is an ordinary
  // all-layer call on shifted base pointers.
  int c = 0;
  for (int a = 0; a < L;) {
    if (!keep[a]) { ++a; continue; }
    int b = a;
    while (b < L && keep[b]) ++b;
    const int n = b - a;
    char* Z = Zall + (size_t)c * T * r * e;
    hipError_t err = dv::launch_down_act(E, (const char*)Dw + (size_t)a * r * d * e, Z, T, d, n, r,
                                         act, bf, s, g_ev);
    if (err != hipSuccess) return hip_status(err, "dv_kept_visual_kv down launch");
    for (int g0 = 0; g0 < n; g0 += group) {
      const int gl = std::min(group, n - g0);
      const size_t la = (size_t)(a + g0), lc = (size_t)(c + g0);
      err = dv::launch_project_kv(
          E, Z + (size_t)g0 * T * r * e, (const char*)Uw + la * d * r * e,
          (const char*)gamma + la * d * e, (const char*)Wk + la * kvw * d * e,
          (const char*)Wv + la * kvw * d * e, (char*)Kv + lc * T * kvw * e,
          (char*)Vv + lc * T * kvw * e, B, Nv, d, r, Hkv, hd, 0, gl, eps, bf, pw,
          (float*)(pw + (size_t)gl * mem_al), s, g_ev, g0 == 0, g0 + gl >= n);
      if (err != hipSuccess) return hip_status(err, "dv_kept_visual_kv projection launch");
    }
    c += n;
    a = b;
  }
  return launched(hipSuccess, "dv_kept_visual_kv launch", s);
}

size_t dv_delta_rule_workspace(int32_t B, int32_t Hv, int32_t N, int32_t dk, int32_t dv,
                               int32_t dtype) {
  if (B <= 0 || Hv <= 0 || N <= 0 || (dk != 64 && dk != 128) || (dv != 64 && dv != 128) ||
      (dtype != DV_F32 && dtype != DV_BF16))
    return 0;
  return dv::gdr_layout(nullptr, B, Hv, N, dk, dv, dtype == DV_BF16 ? 1 : 0).bytes;
}

dv_status dv_delta_rule_write(const void* k, const void* v, const float* alpha, const float* beta,
                              float* S, int32_t B, int32_t Hk, int32_t Hv, int32_t N, int32_t dk,
                              int32_t dv, int32_t dtype, void* ws, size_t ws_bytes, void* stream) {
  DV_CHECK(check_dtype(dtype));
  if (B <= 0 || Hk <= 0 || Hv <= 0 || N < 0)
    return fail(DV_ERR_SHAPE, "B=%d Hk=%d Hv=%d must be positive and N=%d >= 0", B, Hk, Hv, N);
  if (Hv % Hk != 0) return fail(DV_ERR_SHAPE, "Hv=%d is not a multiple of Hk=%d", Hv, Hk);
  if (B > 65535 || Hv > 65535) return fail(DV_ERR_SHAPE, "B and Hv must be at most 65535");
  if ((dk != 64 && dk != 128) || (dv != 64 && dv != 128))
    return fail(DV_ERR_UNSUPPORTED, "dk=%d and dv=%d must be 64 or 128", dk, dv);
  DV_CHECK(need_ptr(S, "S"));
  if (N == 0) return ok();
  DV_CHECK(need_ptr(k, "k"));
  DV_CHECK(need_ptr(v, "v"));
  if (!alpha || !beta) return fail(DV_ERR_NULL, "alpha and beta must not be NULL");
  if ((reinterpret_cast<uintptr_t>(alpha) & 3u) || (reinterpret_cast<uintptr_t>(beta) & 3u))
    return fail(DV_ERR_ALIGN, "alpha and beta must be 4-byte aligned");
  const int bf = dtype == DV_BF16 ? 1 : 0;
  const size_t need = dv::gdr_layout(nullptr, B, Hv, N, dk, dv, bf).bytes;
  if (!ws || ws_bytes < need)
    return fail(DV_ERR_WORKSPACE, "workspace of %zu bytes is below the required %zu",
                ws ? ws_bytes : (size_t)0, need);
  if (!aligned16(ws)) return fail(DV_ERR_ALIGN, "ws is not 16-byte aligned");
  const dv::GdrWs w = dv::gdr_layout(ws, B, Hv, N, dk, dv, bf);
  return launched(dv::launch_delta_rule(k, v, alpha, beta, S, B, Hk, Hv, N, dk, dv, bf, w,
                                        (hipStream_t)stream, g_ev),
                  "dv_delta_rule_write launch", (hipStream_t)stream);
}

size_t dv_text_visual_attention_workspace(int32_t B, int32_t Hq, int32_t Hkv, int32_t hd,
                                          int32_t Nv, int32_t Nq, int32_t Nkt) {
  if (B <= 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0 || (hd != 64 && hd != 128) || Nv < 0 ||
      Nq <= 0 || Nkt < Nq)
    return 0;
  return dv::attention_workspace(B, Hq, Hkv, hd, Nv, Nq, Nkt);
}

}  // extern "C"

namespace {

// Validation shared by both attention entry points; nothing is enqueued here.
dv_status check_attention(const void* Q, const void* Kv, const void* Vv, const void* Kt,
                          const void* Vt, const void* O, int32_t B, int32_t Hq, int32_t Hkv,
                          int32_t hd, int32_t Nv, int32_t Nq, int32_t Nkt, int32_t q_pos0,
                          float scale, int32_t dtype) {
  DV_CHECK(check_dtype(dtype));
  if (B <= 0 || Hq <= 0 || Hkv <= 0 || hd <= 0 || Nv < 0 || Nq <= 0 || Nkt <= 0 || q_pos0 < 0)
    return fail(DV_ERR_SHAPE,
                "sizes must be positive (B=%d Hq=%d Hkv=%d hd=%d Nq=%d Nkt=%d), Nv and q_pos0 >= 0 "
                "(Nv=%d q_pos0=%d)", B, Hq, Hkv, hd, Nq, Nkt, Nv, q_pos0);
  if (Hq % Hkv != 0) return fail(DV_ERR_SHAPE, "Hq=%d is not a multiple of Hkv=%d", Hq, Hkv);
  if ((int64_t)q_pos0 + Nq > Nkt)
    return fail(DV_ERR_SHAPE, "q_pos0 + Nq = %lld exceeds the %d text keys",
                (long long)q_pos0 + Nq, Nkt);
  if ((int64_t)Nv + Nkt > INT32_MAX / 2 || (int64_t)B * Nq * Hq > INT32_MAX / 256)
    return fail(DV_ERR_SHAPE, "key count exceeds 2^30 or B*Nq*Hq exceeds 2^23");
  if ((int64_t)B * Hkv > 65535) return fail(DV_ERR_SHAPE, "B*Hkv=%lld exceeds 65535", (long long)B * Hkv);
  if (hd != 64 && hd != 128) return fail(DV_ERR_UNSUPPORTED, "hd=%d must be 64 or 128", hd);
  // The streaming kernels address one (batch, kv-head) slice of a cache through a buffer
  // resource with a 32-bit byte range and 32-bit offsets.
  if ((int64_t)Nv * hd * (int64_t)elem_size(dtype) > INT32_MAX ||
      (int64_t)Nkt * hd * (int64_t)elem_size(dtype) > INT32_MAX)
    return fail(DV_ERR_SHAPE, "a (batch, kv-head) cache slice exceeds 2^31-1 bytes (Nv=%d Nkt=%d hd=%d)",
                Nv, Nkt, hd);
  if (!std::isfinite(scale) || !(scale > 0.f))
    return fail(DV_ERR_SHAPE, "scale must be finite and > 0");
  DV_CHECK(need_ptr(Q, "Q"));
  if (Nv > 0) {
    DV_CHECK(need_ptr(Kv, "Kv"));
    DV_CHECK(need_ptr(Vv, "Vv"));
  }
  DV_CHECK(need_ptr(Kt, "Kt"));
  DV_CHECK(need_ptr(Vt, "Vt"));
  DV_CHECK(need_ptr(O, "O"));
  return DV_OK;
}

dv_status run_attention(const void* Q, const void* Kv, const void* Vv, const void* Kt,
                        const void* Vt, void* O, int32_t B, int32_t Hq, int32_t Hkv, int32_t hd,
                        int32_t Nv, int32_t Nq, int32_t Nkt, int32_t q_pos0, float scale,
                        int32_t dtype, void* ws, const dv::AttnPlan& plan, hipStream_t stream,
                        const char* name) {
  dv::AttnArgs a{};
  a.Q = Q;
  a.Kv = Kv;
  a.Vv = Vv;
  a.Kt = Kt;
  a.Vt = Vt;
  a.O = O;
  const int64_t rows = (int64_t)B * Nq * Hq;
  a.Opart = (float*)ws;
  a.MLpart = ws ? (float*)((char*)ws + (size_t)plan.splits * rows * hd * 4) : nullptr;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.hd = hd;
  a.Nv = Nv;
  a.Nq = Nq;
  a.Nkt = Nkt;
  a.q_pos0 = q_pos0;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.splits = plan.splits;
  a.keys_per_split = plan.keys_per_split;
  a.tiles_per_split = plan.tiles_per_split;
  return launched(dv::launch_attention(a, plan, dtype == DV_BF16 ? 1 : 0, stream, g_ev), name,
                  stream);
}

}  // namespace

extern "C" {

dv_status dv_text_visual_attention(const void* Q, const void* Kv, const void* Vv, const void* Kt,
                                   const void* Vt, void* O, int32_t B, int32_t Hq, int32_t Hkv,
                                   int32_t hd, int32_t Nv, int32_t Nq, int32_t Nkt,
                                   int32_t q_pos0, float scale, int32_t dtype, void* ws,
                                   size_t ws_bytes, void* stream) {
  DV_CHECK(check_attention(Q, Kv, Vv, Kt, Vt, O, B, Hq, Hkv, hd, Nv, Nq, Nkt, q_pos0, scale,
                           dtype));
  if (ws && !aligned16(ws)) return fail(DV_ERR_ALIGN, "ws is not 16-byte aligned");
  const dv::AttnPlan plan =
      dv::plan_attention(B, Hq, Hkv, hd, Nv, Nq, Nkt, q_pos0, dtype == DV_BF16 ? 1 : 0,
                         ws ? ws_bytes : 0);
  return run_attention(Q, Kv, Vv, Kt, Vt, O, B, Hq, Hkv, hd, Nv, Nq, Nkt, q_pos0, scale, dtype,
                       ws, plan, (hipStream_t)stream, "dv_text_visual_attention launch");
}

dv_status dv_text_visual_attention_noalloc(const void* Q, const void* Kv, const void* Vv,
                                           const void* Kt, const void* Vt, void* O, int32_t B,
                                           int32_t Hq, int32_t Hkv, int32_t hd, int32_t Nv,
                                           int32_t Nq, int32_t Nkt, int32_t q_pos0, float scale,
                                           int32_t dtype, void* stream) {
  DV_CHECK(check_attention(Q, Kv, Vv, Kt, Vt, O, B, Hq, Hkv, hd, Nv, Nq, Nkt, q_pos0, scale,
                           dtype));
  // The split dv_text_visual_attention takes with its recommended workspace, so both entry
  // points give the same bits; a split whose partials exceed the static scratch is refused.
  const dv::AttnPlan plan = dv::plan_attention(B, Hq, Hkv, hd, Nv, Nq, Nkt, q_pos0,
                                               dtype == DV_BF16 ? 1 : 0, (size_t)-1);
  const size_t cap = dv::attention_scratch_bytes();
  if (plan.ws_needed > cap)
    return fail(DV_ERR_WORKSPACE,
                "this call's key split needs %zu bytes of partials, more than the %zu bytes of the "
                "static scratch; call dv_text_visual_attention with a workspace instead",
                plan.ws_needed, cap);
  void* scr = nullptr;  // resolved on the first call on each device
  hipError_t e = dv::attention_scratch(&scr);
  if (e != hipSuccess) return hip_status(e, "dv_text_visual_attention_noalloc scratch lookup");
  return run_attention(Q, Kv, Vv, Kt, Vt, O, B, Hq, Hkv, hd, Nv, Nq, Nkt, q_pos0, scale, dtype,
                       plan.splits > 1 ? scr : nullptr, plan, (hipStream_t)stream, "dv_text_visual_attention_noalloc launch");
}

}  // extern "C"
