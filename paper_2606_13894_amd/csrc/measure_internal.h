// Measurement kernels of libgefen (not part of the optimizer's arithmetic).
#pragma once
#include "gefen_internal.h"

namespace gefen {

// One pass of the step's byte mix over n elements: theta[i] += g (two lanes of each
// vector), codes[i] ^= 1. theta 16-byte, grad 16 (fp32) or 8 (bf16) byte, codes
// 4-byte aligned.
hipError_t launch_stream_mix(float* theta, const void* grad, int gdtype, uint8_t* codes,
                             int64_t n, hipStream_t stream);

}  // namespace gefen
