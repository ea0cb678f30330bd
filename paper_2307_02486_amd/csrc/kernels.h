// Launchers of the two device stages of the dilated-attention forward pass.
#pragma once

#include <hip/hip_runtime.h>

#include "plan.h"

namespace da {

// Stage 1: per pattern, gather the kept rows of every segment and run causal
// (or full) softmax attention on them, writing the normalised per-pattern
// output and its log-sum-exp to the workspace (Sec. 2.2, Eqs. 3-6).
hipError_t launch_attention(const Plan& plan, const void* q, const void* k, const void* v,
                            void* workspace, hipStream_t stream);

// Stage 2: scatter the per-pattern rows back to their sequence positions and
// mix them by their softmax denominators, writing out and lse
// (Sec. 2.2, Eqs. 7-10).
hipError_t launch_combine(const Plan& plan, const void* workspace, void* out, float* lse,
                          hipStream_t stream);

}  // namespace da
