// On-device bf16 matrix-core rate (the diagnostic of mla_probe.h).
#pragma once

#include "common.h"

namespace mla {

constexpr int kProbeWaves = 4;     // waves per workgroup
constexpr int kProbeChains = 4;    // independent accumulation chains per wave

// n_wg workgroups of kProbeWaves waves, each wave kProbeChains x iters products
hipError_t launch_probe_mfma(int iters, int n_wg, float* sink, hipStream_t s);

}  // namespace mla
