// Calls every entry point of the C ABI with arguments that fail validation, plus the workspace
// queries and the status strings, so that a host build with AddressSanitizer and
// UndefinedBehaviorSanitizer checks the validation code itself (argument checks, size arithmetic,
// error formatting). Nothing is launched: every call is rejected before any HIP work is enqueued.
// Prints "ok" on success.
#include <cstdint>
#include <cstdio>
#include <cstring>

#include "../../include/deltavision.h"

namespace {
void* const FAKE = reinterpret_cast<void*>(0x10000);
int failures = 0;

void expect(dv_status got, dv_status want, const char* what) {
  if (got != want) {
    std::fprintf(stderr, "%s: status %d, expected %d (%s)\n", what, (int)got, (int)want,
                 dv_last_error());
    ++failures;
  } else if (want != DV_OK && std::strlen(dv_last_error()) == 0) {
    std::fprintf(stderr, "%s: no error text\n", what);
    ++failures;
  }
}
}  // namespace

int main() {
  for (int s = -1; s < 10; ++s) (void)std::strlen(dv_status_string(s));
  // down projection
  expect(dv_build_visual_memory(nullptr, FAKE, FAKE, 64, 256, 4, 16, 0, DV_F32, nullptr), DV_ERR_NULL, "build null");
  expect(dv_build_visual_memory(FAKE, FAKE, FAKE, (int64_t)1 << 40, 256, 4, 16, 0, DV_F32, nullptr), DV_ERR_SHAPE, "build huge T");
  expect(dv_build_visual_memory(FAKE, FAKE, FAKE, 64, 100, 4, 16, 0, DV_F32, nullptr), DV_ERR_UNSUPPORTED, "build d");
  expect(dv_build_visual_memory(FAKE, FAKE, FAKE, 64, 256, 0x7fffffff, 0x7ff0, 0, DV_BF16, nullptr), DV_ERR_SHAPE, "build L*r overflow");
  // projection
  const size_t ws1 = dv_project_visual_kv_workspace(64, 256, 1, DV_F32);
  if (ws1 == 0 || dv_project_visual_kv_workspace(0, 256, 1, DV_F32) != 0) ++failures;
  expect(dv_project_visual_kv(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 64, 256, 4, 16, 4, 64, 0, 4,
                              1e-5f, DV_F32, FAKE, 16, nullptr), DV_ERR_WORKSPACE, "project small ws");
  expect(dv_project_visual_kv(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 64, 256, 4, 16, 4, 64, 3, 2,
                              1e-5f, DV_F32, FAKE, ws1, nullptr), DV_ERR_SHAPE, "project layer range");
  expect(dv_project_visual_kv(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 64, 256, 4, 16, 4, 96, 0, 4,
                              1e-5f, DV_F32, FAKE, ws1, nullptr), DV_ERR_UNSUPPORTED, "project hd");
  expect(dv_project_visual_kv(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0x7fffffff, 0x7fffffff, 256, 4, 16,
                              4, 64, 0, 4, 1e-5f, DV_F32, FAKE, ws1, nullptr), DV_ERR_SHAPE, "project T overflow");
  dv_kv_epilogue epi{};
  epi.positions = reinterpret_cast<const int32_t*>(FAKE);
  epi.rope_sections[0] = 31;
  epi.rope_theta = 1e4f;
  expect(dv_project_visual_kv_ex(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 64, 256, 4, 16, 4, 64, 0,
                                 4, 1e-5f, &epi, DV_F32, FAKE, (size_t)1 << 30, nullptr), DV_ERR_SHAPE,
         "epilogue sections");
  if (dv_project_visual_kv_ex_workspace(64, 256, 4, 64, DV_BF16) <= dv_project_visual_kv_workspace(64, 256, 4, DV_BF16))
    ++failures;
  // recurrent and kept
  expect(dv_recurrent_visual_kv(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 64, 256, 4, 16, 4, 64, 7,
                                1e-5f, DV_F32, FAKE, (size_t)1 << 30, nullptr), DV_ERR_UNSUPPORTED, "recurrent act");
  if (dv_recurrent_visual_kv_workspace(64, 256, 4, 16, DV_F32) == 0) ++failures;
  const uint8_t keep[4] = {1, 0, 1, 1};
  expect(dv_kept_visual_kv(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, nullptr, FAKE, FAKE, 1, 64, 256, 4, 16, 4, 64,
                           0, 1e-5f, DV_F32, FAKE, (size_t)1 << 30, nullptr), DV_ERR_NULL, "kept mask");
  expect(dv_kept_visual_kv(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, keep, FAKE, FAKE, 1, 64, 256, 4, 16, 4, 64, 0,
                           1e-5f, DV_F32, FAKE, 16, nullptr), DV_ERR_WORKSPACE, "kept ws");
  const uint8_t none[4] = {0, 0, 0, 0};
  expect(dv_kept_visual_kv(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, none, nullptr, nullptr, 1, 64, 256, 4, 16, 4,
                           64, 0, 1e-5f, DV_F32, nullptr, 0, nullptr), DV_OK, "kept nothing");
  // attention (both entry points)
  expect(dv_text_visual_attention(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 2, 8, 2, 64, 300, 9, 20, 12, 0.125f,
                                  DV_BF16, nullptr, 0, nullptr), DV_ERR_SHAPE, "attention causal range");
  expect(dv_text_visual_attention(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 2, 8, 2, 128, 0x7ffffff, 9, 20, 11, 0.125f,
                                  DV_BF16, nullptr, 0, nullptr), DV_ERR_SHAPE, "attention cache slice bytes");
  expect(dv_text_visual_attention(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 2, 8, 2, 64, 300, 9, 20, 11, -1.f,
                                  DV_BF16, nullptr, 0, nullptr), DV_ERR_SHAPE, "attention scale");
  expect(dv_text_visual_attention_noalloc(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 64, 8, 128, 4096, 128, 128, 0,
                                          0.088f, DV_F32, nullptr), DV_ERR_WORKSPACE, "noalloc beyond scratch");
  expect(dv_text_visual_attention_noalloc(FAKE, nullptr, FAKE, FAKE, FAKE, FAKE, 2, 8, 2, 64, 300, 9, 20, 11,
                                          0.125f, DV_BF16, nullptr), DV_ERR_NULL, "noalloc null");
  (void)dv_text_visual_attention_workspace(64, 32, 32, 128, 576, 1, 513);
  (void)dv_text_visual_attention_workspace(1, 28, 4, 128, 16384, 128, 128);
  if (dv_text_visual_attention_workspace(1, 7, 2, 128, 16, 4, 8) != 0) ++failures;  // Hq % Hkv
  // delta rule
  expect(dv_delta_rule_write(FAKE, FAKE, reinterpret_cast<float*>(FAKE), reinterpret_cast<float*>(FAKE),
                             reinterpret_cast<float*>(FAKE), 1, 3, 4, 10, 128, 128, DV_BF16, FAKE, 1 << 20,
                             nullptr), DV_ERR_SHAPE, "delta heads");
  expect(dv_delta_rule_write(FAKE, FAKE, reinterpret_cast<float*>(FAKE), reinterpret_cast<float*>(FAKE),
                             reinterpret_cast<float*>(FAKE), 1, 2, 4, 10, 128, 128, DV_BF16, FAKE, 16,
                             nullptr), DV_ERR_WORKSPACE, "delta ws");
  if (dv_delta_rule_workspace(1, 32, 16384, 128, 128, DV_BF16) == 0) ++failures;
  // profiling hook and probe
  expect(dv_time_kernel(99, nullptr, nullptr), DV_ERR_UNSUPPORTED, "time kernel id");
  expect(dv_time_kernel(DV_KERNEL_KV, FAKE, nullptr), DV_ERR_NULL, "time kernel events");
  expect(dv_probe_mfma(1, 0, reinterpret_cast<float*>(FAKE), nullptr), DV_ERR_SHAPE, "probe iters");
  if (failures) {
    std::fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  std::printf("ok\n");
  return 0;
}
