// Host-side plan of one dilated-attention forward call: validation, per-pattern
// geometry, work-item enumeration, workspace layout and exact work accounting.
// No HIP dependency, so it builds and runs with a plain host compiler.
#pragma once

#include <cstddef>
#include <cstdint>

#include "../../include/dilated_attn.h"

#if defined(__HIPCC__)
#define DA_HD __host__ __device__
#else
#define DA_HD
#endif

namespace da {

// Division by a divisor fixed at plan time, for numerators below 2^31:
// q = floor(n * mul / 2^shift) with shift = 31 + ceil(log2 d) and
// mul = ceil(2^shift / d) < 2^32 (Granlund and Montgomery, "Division by
// invariant integers using multiplication", 1994, Thm. 4.2 with N = 31).
struct FastDiv {
  uint32_t d;
  uint32_t mul;
  uint32_t shift;
  DA_HD uint32_t div(uint32_t n) const {
    return static_cast<uint32_t>((static_cast<uint64_t>(n) * mul) >> shift);
  }
};
FastDiv make_fastdiv(uint32_t d);

// Geometry of one pattern (w, r) after validation.  Segment g covers rows
// [g*w, min((g+1)*w, N)); head h keeps the rows at local offsets
// h mod r, h mod r + r, ... (Sec. 2.2 Eqs. 3-5, offset of Sec. 2.3).
struct PatternPlan {
  int64_t w;          // segment length, clamped to N (w > N means one segment)
  int64_t r;          // dilation rate
  int64_t nseg;       // ceil(N / w)
  int64_t lmax;       // kept rows of a full segment at offset 0: ceil(w / r)
  int64_t ntiles;     // query tiles per (b, h, segment) unit: ceil(lmax / block_m)
  int64_t units;      // B * H * nseg
  int64_t item_begin; // index of this pattern's first work item
  uint64_t o_off;     // byte offset of the per-pattern output in the workspace
                      // (fp16 rows scaled by a power of two for bf16 inputs,
                      // fp32 rows for fp32 inputs)
  uint64_t lse_off;   // byte offset of the per-row records (float lse, float
                      // scale: the row's values are the stored ones times it)
};

struct Plan {
  int64_t B, N, H, D;
  int causal;
  int dtype;
  float scale;        // softmax scale actually used
  int npat;
  int block_m;        // query rows per attention work item
  PatternPlan pat[DA_MAX_PATTERNS];
  int64_t total_items;
  int64_t launch_items;  // workgroups of the attention launch (XCD-balanced, >= total_items)
  bool offsets32;        // every key tile spans < 2^31 bytes: 32-bit buffer offsets suffice
  uint64_t workspace_bytes;
  int64_t covered_rows;
  double sparse_flops;
  double bytes_attn;
  double bytes_combine;
};

// Workspace of a backward call: per (b, h, row) -lse*log2(e) and -delta
// (float32, [B][H][N] each), then per pattern the compact float32 gradients
// of its kept rows, [units][lmax][D] for dq, dk and dv.
struct BwdLayout {
  uint64_t nl2_off;   // byte offset of -lse*log2(e)
  uint64_t nd_off;    // byte offset of -delta
  // Per pattern, the compact gradients dq, dk, dv: fp16 rows [units*lmax][D],
  // each row scaled by a power of two per chunk of kGradChunk columns, and
  // the float scales [units*lmax][chunks] (see grad_chunks).
  uint64_t dq_off[DA_MAX_PATTERNS];
  uint64_t dk_off[DA_MAX_PATTERNS];
  uint64_t dv_off[DA_MAX_PATTERNS];
  uint64_t dq_rec_off[DA_MAX_PATTERNS];
  uint64_t dk_rec_off[DA_MAX_PATTERNS];
  uint64_t dv_rec_off[DA_MAX_PATTERNS];
  uint64_t workspace_bytes;
  double flops;          // 10*D per unmasked pair
  double bytes_grad;     // algorithmic HBM bytes of the dq and dk/dv kernels
  double bytes_combine;  // algorithmic HBM bytes of the delta and sum kernels
};

// Columns of a compact gradient row that share one scale: the columns one
// backward work item accumulates.
constexpr int64_t kGradChunk = 64;
inline int64_t grad_chunks(int64_t D) { return (D + kGradChunk - 1) / kGradChunk; }

// Backward workspace and work of a validated forward plan.  DA_EUNSUPPORTED
// unless the plan is bf16 (and for tiles whose offsets need 64 bits).
int make_bwd_layout(const Plan& p, BwdLayout* out);

// Query rows per work item of the attention kernel for a dtype.
int block_m_for(int dtype);

// Number of rows a pattern keeps in a segment of `seg_len` rows at offset s.
inline int64_t kept_rows(int64_t seg_len, int64_t s, int64_t r) {
  return seg_len > s ? (seg_len - s + r - 1) / r : 0;
}

// Validate and fill a plan.  Returns DA_OK or a negative DA_E* code.
int make_plan(int64_t B, int64_t N, int64_t H, int64_t D, const da_pattern_t* patterns,
              int64_t num_patterns, int64_t causal, int64_t dtype, float softmax_scale,
              Plan* out);

}  // namespace da
