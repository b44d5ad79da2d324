// Host-visible launcher of the quantizer with an HQQ-style optimised zero-point
// (internal; the public ABI is include/subspec.h).
#pragma once

#include "kernels.h"

namespace subspec {

hipError_t launch_quantize_hqq(const float* w, int bits, int group, int N, int K, uint8_t* codes,
                               uint16_t* sc, uint16_t* zr, hipStream_t st);

}  // namespace subspec
