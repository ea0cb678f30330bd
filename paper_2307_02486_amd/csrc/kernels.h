// Launchers of the device stages of the dilated-attention forward and backward passes.
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

// Backward: per-row -delta and -lse*log2(e), the per-pattern dq and dk/dv
// kernels into compact workspace rows, and their sum per row into dq, dk, dv.
hipError_t launch_backward(const Plan& plan, const BwdLayout& lay, const void* q, const void* k,
                           const void* v, const void* out, const float* lse, const void* dout, void* dq,
                           void* dk, void* dv, void* workspace, hipStream_t stream);

}  // namespace da
