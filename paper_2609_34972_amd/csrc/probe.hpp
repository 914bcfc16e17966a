// Host-side launcher of the MFMA-rate probe (internal to the library).
#pragma once

#include <hip/hip_runtime.h>

namespace dv {

// Blocks of the probe (8 waves each); every block writes one float of the sink.
constexpr int kProbeBlocks = 1024;
// Floating-point operations of one 16x16x32 MFMA and MFMAs per wave and iteration.
constexpr double kProbeFlopPerMfma = 2.0 * 16 * 16 * 32;
constexpr int kProbeMfmaPerIter = 32;

hipError_t launch_probe_mfma(bool random, int iters, float* sink, hipStream_t s);

}  // namespace dv
