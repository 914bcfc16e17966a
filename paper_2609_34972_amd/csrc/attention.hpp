// Host-side interface of the text-query attention kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>

#include "build_kernels.hpp"

namespace dv {

struct AttnArgs {
  const void* Q;
  const void* Kv;
  const void* Vv;
  const void* Kt;
  const void* Vt;
  void* O;
  float* Opart;   // [splits, B*Nq*Hq, hd] unnormalised partial outputs (splits > 1)
  float* MLpart;  // [splits, B*Nq*Hq, 2]  running max (log2 domain) and sum
  int B, Hq, Hkv, hd, Nv, Nq, Nkt, q_pos0;
  float scale_log2;  // softmax scale times log2(e)
  int splits, keys_per_split;
  int tiles_per_split;  // bf16 hd-128 prefill: key tiles per split (32 keys for the key-split
                        // kernel, 64 for the streaming kernel)
};

struct AttnPlan {
  bool decode;         // one query per sequence: the bandwidth-bound kernel
  bool stream;         // bf16 hd-128 prefill: direct-to-LDS streaming kernel
  bool ksplit;         // (stream) few rows per kv-head: four waves split the keys of 32 rows
  bool pp;             // (stream) over 96 rows per kv-head: the eight-wave ping-pong kernel
  int tiles_per_split;  // (stream) key tiles per split: 32 keys each if ksplit, else 64
  int nw;              // waves per block (prefill)
  int row_blocks;      // blocks along the packed (query, head) rows (prefill)
  int splits;          // key splits merged by a log-sum-exp combine
  int keys_per_split;  // decode and the generic prefill: a multiple of their 64-key tile
  size_t ws_needed;    // bytes of partials for this plan
};

AttnPlan plan_attention(int B, int Hq, int Hkv, int hd, int Nv, int Nq, int Nkt, int q_pos0,
                        int dtype, size_t ws_bytes);
size_t attention_workspace(int B, int Hq, int Hkv, int hd, int Nv, int Nq, int Nkt);
hipError_t launch_attention(const AttnArgs& a, const AttnPlan& p, int dtype, hipStream_t s,
                            const LaunchEvents& ev);
// Address of the library's static scratch array (attention_scratch_bytes() bytes) on the
// current device; resolved once per device.
hipError_t attention_scratch(void** ptr);
size_t attention_scratch_bytes();

}  // namespace dv
