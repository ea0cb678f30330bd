// Launchers of the device stages of the dilated-attention forward and backward passes.
#pragma once

#include <hip/hip_runtime.h>

#include "plan.h"

namespace da {

// A pattern as the combine step sees it: the divisions that map a sequence
// position to the pattern's segment and kept-row index, and where the
// pattern's rows sit in the workspace.
struct MixPat {
  FastDiv fw;       // division by w
  FastDiv fr;       // division by r
  int32_t nseg, lmax;
  int64_t o_off;    // byte offset of the pattern's output rows
  int64_t lse_off;  // byte offset of the pattern's (lse, scale) row records
};

inline MixPat make_mixpat(const PatternPlan& pp) {
  return MixPat{make_fastdiv(static_cast<uint32_t>(pp.w)), make_fastdiv(static_cast<uint32_t>(pp.r)),
                static_cast<int32_t>(pp.nseg), static_cast<int32_t>(pp.lmax),
                static_cast<int64_t>(pp.o_off), static_cast<int64_t>(pp.lse_off)};
}

// Stage 1: per pattern, gather the kept rows of every segment and run causal
// (or full) softmax attention on them, writing the normalised per-pattern
// output rows and their (lse, scale) records to the workspace
// (Sec. 2.2, Eqs. 3-6).
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

// xPos of a [B, N, H, D] query (sign = +1) or key (sign = -1) tensor, or its
// transpose (the backward's map), from x into y (y may equal x).
hipError_t launch_xpos(const void* x, void* y, int64_t B, int64_t N, int64_t H, int64_t D, int sign,
                       bool transpose, int64_t center, float base, float gamma, float scale_base,
                       int dtype, hipStream_t stream);

// Weight gradient dw[M][N] = sum_k dy[k][M] x[k][N] (bf16, M and N multiples
// of 128): float32 partial sums over k-chunks in workspace, then their sum.
// With db non-null, also db[M] = the column sums of dy (the bias gradient).
int64_t wgrad_splits(int64_t K, int64_t M, int64_t N, int64_t* chunk);
uint64_t wgrad_workspace(int64_t K, int64_t M, int64_t N);
hipError_t launch_wgrad(const void* dy, const void* x, void* dw, void* db, int64_t K, int64_t M, int64_t N,
                        void* workspace, hipStream_t stream);

// LayerNorm over rows of E bf16 elements (E a multiple of 8, at most 2048),
// float32 statistics; the backward's parameter gradients go through a
// float32 workspace of layernorm_bwd_workspace(rows, E) bytes.
hipError_t launch_layernorm_fwd(const void* x, const void* g, const void* b, void* y, float* mean, float* rstd,
                                int64_t rows, int64_t E, float eps, hipStream_t stream);
uint64_t layernorm_bwd_workspace(int64_t rows, int64_t E);
hipError_t launch_layernorm_bwd(const void* dy, const void* x, const void* g, const float* mean, const float* rstd,
                                void* dx, void* dg, void* db, int64_t rows, int64_t E, void* workspace,
                                hipStream_t stream);

}  // namespace da
