/*
 * dilated_attn.h - C ABI of the MI355X (gfx950) dilated-attention forward and
 * backward passes.
 *
 * The operator is LongNet's dilated attention (Sec. 2.2-2.3 of the paper):
 *   1. split the sequence into segments of length w_i          (Sec. 2.2, Eqs. 3-5)
 *   2. in each segment keep every r_i-th row, starting at the  (Sec. 2.3, s_j = j mod r)
 *      head's offset h mod r_i
 *   3. dense softmax attention inside each sparsified segment  (Sec. 2.2, Eq. 6)
 *   4. scatter the rows back and mix the k patterns, each      (Sec. 2.2, Eqs. 7-10)
 *      weighted by its softmax denominator
 *
 * Semantics fixed by this library where the paper is silent:
 *   - scores are scaled by softmax_scale (0 selects 1/sqrt(D));
 *   - causal != 0: inside a sparsified segment, a query sees the kept rows at
 *     or before its own position; causal == 0: it sees every kept row;
 *   - the offset is segment-local: segment g keeps rows p in
 *     [g*w, min((g+1)*w, N)) with (p - g*w) mod r == h mod r, heads from 0;
 *     a last segment shorter than w is truncated, w > N means one segment;
 *   - a pattern's weight is its unshifted softmax denominator; a pattern that
 *     does not keep a row contributes nothing there; duplicate patterns count
 *     twice; a row kept by no pattern gets out = 0 and lse = -inf.
 *
 * Layouts (row-major, contiguous, no strides):
 *   q, k, v, out : [B, N, H, D] elements of `dtype`
 *   lse          : [B, H, N] float32, natural log of the summed denominators
 *
 * Every integer is 64-bit on the ABI.  Limits: 1 <= B, 1 <= N, N + H < 2^31,
 * 1 <= H < 2^16, D in {32, 64, 128}, 1 <= num_patterns <= DA_MAX_PATTERNS,
 * 1 <= r_i <= w_i.
 */
#ifndef DILATED_ATTN_H
#define DILATED_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DA_MAX_PATTERNS 16

/* One dilated pattern (Sec. 2.2, the pairs {r_i, w_i}). */
typedef struct {
  int64_t w; /* segment length, >= 1 */
  int64_t r; /* dilation rate, 1 <= r <= w */
} da_pattern_t;

/* Element types of q, k, v and out. */
enum { DA_F32 = 0, DA_BF16 = 1 };

/* Error codes.  Every entry point returns DA_OK or one of these; on error
 * nothing is written to any caller buffer and nothing is launched. */
enum {
  DA_OK = 0,
  DA_EINVAL = -1,       /* null pointer, non-positive size, bad pattern list,
                           out aliasing an input, size beyond the limits  */
  DA_EUNSUPPORTED = -2, /* head dim or dtype the library has no kernel for */
  DA_EWORKSPACE = -3,   /* workspace smaller than dilated_attn_plan asks  */
  DA_EALIGN = -4,       /* a device pointer not 16-byte aligned           */
  DA_EHIP = -5,         /* the HIP runtime reported an error at launch    */
  DA_ETOOLARGE = -6     /* dilated_attn_fwd_noalloc: the problem needs more
                           workspace than DA_NOALLOC_MAX_BYTES              */
};

/* Sizes and work of one call, filled by dilated_attn_plan. */
typedef struct {
  uint64_t workspace_bytes; /* device memory the caller passes to fwd        */
  int64_t num_work_items;   /* attention work items (pattern, b, h, segment,
                               query tile) launched by fwd                    */
  int64_t covered_rows;     /* sum over patterns of kept (b, row, head) rows  */
  double sparse_flops;      /* 4*D per unmasked (query, key) pair, the work of
                               Sec. 2.4 counted exactly                       */
  double bytes_attn;        /* algorithmic HBM bytes of the attention stage:
                               kept q/k/v rows read once, per-pattern output
                               rows and their 8-byte records written once    */
  double bytes_combine;     /* algorithmic HBM bytes of the combine stage:
                               per-pattern output rows and records read once,
                               out and lse written once                       */
} da_plan_info_t;

/*
 * dilated_attn_plan - validate a problem and report its workspace and work.
 *
 * Host only: touches no device and may be called without a GPU.  Arguments
 * are those of dilated_attn_fwd without the buffers.  `patterns` points to
 * num_patterns host structs, read during the call only.  Returns DA_OK and
 * fills *info, or a negative error code (info untouched).
 */
int dilated_attn_plan(int64_t B, int64_t N, int64_t H, int64_t D,
                      const da_pattern_t* patterns, int64_t num_patterns,
                      int64_t causal, int64_t dtype, float softmax_scale,
                      da_plan_info_t* info);

/*
 * dilated_attn_fwd - dilated-attention forward pass (Sec. 2.2-2.3).
 *
 * q, k, v   device pointers, [B, N, H, D] of dtype, read only.
 * out       device pointer, [B, N, H, D] of dtype, written (every element).
 * lse       device pointer, [B, H, N] float32, written (every element).
 * patterns  host pointer to num_patterns (w, r) pairs, read during the call.
 * workspace device scratch of at least info.workspace_bytes from
 *           dilated_attn_plan, owned by the caller; contents on entry are
 *           ignored and on return are unspecified.
 * stream    a hipStream_t (NULL = the default stream).  Work is enqueued
 *           asynchronously; buffers must stay valid until the stream reaches
 *           this point.  Nothing is allocated and nothing synchronises.
 *
 * All device pointers must be 16-byte aligned and out must not overlap q, k
 * or v.  Returns DA_OK or a negative error code; before any launch, every
 * argument is checked and an error leaves all buffers untouched.
 *
 * Arithmetic for DA_BF16: scores q.k as exact bf16 products summed in
 * float32, times softmax_scale*log2(e) in float32; probabilities rounded to
 * bf16 for the product with v (float32 sums); each pattern's normalised rows
 * kept in the workspace as fp16 divided by a power of two per row, within
 * 2^-11 of the row's largest magnitude; the mixture in float32; out rounded
 * once to bf16.  Results are finite whenever every scaled score is finite in
 * float32 and max|v| < 2^95.  DA_F32 computes in float32 throughout.
 */
int dilated_attn_fwd(const void* q, const void* k, const void* v, void* out,
                     float* lse, int64_t B, int64_t N, int64_t H, int64_t D,
                     const da_pattern_t* patterns, int64_t num_patterns,
                     int64_t causal, int64_t dtype, float softmax_scale,
                     void* workspace, uint64_t workspace_bytes, void* stream);

/*
 * dilated_attn_fwd_noalloc - dilated_attn_fwd without a workspace argument,
 * for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation).
 *
 * The workspace is a device array owned by the library, DA_NOALLOC_MAX_BYTES
 * (128 MiB) on every device the function runs on, held until the process
 * ends; its address is looked up once per device.  Problems whose
 * dilated_attn_plan workspace_bytes exceeds DA_NOALLOC_MAX_BYTES return
 * DA_ETOOLARGE (the 8K- and 32K-token workloads of the benchmark fit; larger
 * ones need dilated_attn_fwd).  The call allocates nothing, host or device.
 * All calls on one device share its array: calls that may overlap in time on
 * one device (other streams, other threads) race and must not be made.
 * Arguments, results and other errors as for dilated_attn_fwd.
 */
#define DA_NOALLOC_MAX_BYTES (128ull << 20)
int dilated_attn_fwd_noalloc(const void* q, const void* k, const void* v, void* out,
                             float* lse, int64_t B, int64_t N, int64_t H, int64_t D,
                             const da_pattern_t* patterns, int64_t num_patterns,
                             int64_t causal, int64_t dtype, float softmax_scale,
                             void* stream);

/*
 * Backward pass: gradients of a loss with respect to q, k and v, given the
 * gradient dout of the loss with respect to out.
 *
 * The mixture of Eqs. 9-10 is one softmax over the multiset of (pattern, key)
 * pairs a query sees (Sec. 2.2, after Eq. 10), so with the combined lse of
 * the forward pass and delta = sum_d dout * out per row, each pattern's
 * contribution is the softmax-attention derivative on its sparsified
 * segments: P = exp(scale q.k - lse), dS = P (dout.v - delta),
 * dq += scale dS k, dk += scale dS q, dv += P dout; a row collects the
 * contributions of every pattern that keeps it (the paper's distributed
 * algorithm has this backward, Sec. 3.1).
 *
 * The library computes the backward for dtype DA_BF16 (D in {32, 64, 128});
 * DA_F32 returns DA_EUNSUPPORTED, and so do patterns whose dilation makes a
 * tile of 65 kept rows span 2 GiB or more (r*H*D*2*129 >= 2^31, or
 * r*4*65 >= 2^31).
 */

/*
 * dilated_attn_bwd_plan - validate a backward problem and report its
 * workspace and work.  Host only; arguments as for dilated_attn_plan.  Fills
 * *info: workspace_bytes for dilated_attn_bwd, num_work_items = the dq and
 * the dk/dv kernels' work items, covered_rows, sparse_flops = 10*D per
 * unmasked (query, key) pair (the five products of the derivative),
 * bytes_attn = algorithmic HBM bytes of the two gradient kernels and
 * bytes_combine = those of the delta and gradient-sum kernels.
 */
int dilated_attn_bwd_plan(int64_t B, int64_t N, int64_t H, int64_t D,
                          const da_pattern_t* patterns, int64_t num_patterns,
                          int64_t causal, int64_t dtype, float softmax_scale,
                          da_plan_info_t* info);

/*
 * dilated_attn_bwd - dilated-attention backward pass.
 *
 * q, k, v     device pointers, [B, N, H, D] of dtype, read only: the
 *             forward's inputs.
 * out, lse    device pointers, the forward's outputs for these inputs
 *             ([B, N, H, D] of dtype and [B, H, N] float32), read only.
 * dout        device pointer, [B, N, H, D] of dtype, read only.
 * dq, dk, dv  device pointers, [B, N, H, D] of dtype, written (every
 *             element; rows no pattern keeps get 0).
 * patterns, causal, dtype, softmax_scale: those of the forward call.
 * workspace   device scratch of at least info.workspace_bytes from
 *             dilated_attn_bwd_plan, owned by the caller; contents on entry
 *             are ignored and on return are unspecified.
 * stream      a hipStream_t (NULL = the default stream), asynchronous as for
 *             dilated_attn_fwd.
 *
 * All device pointers must be 16-byte aligned; dq, dk and dv must not overlap
 * each other or any input.  Returns DA_OK or a negative error code; every
 * argument is checked before any launch and an error leaves all buffers
 * untouched.
 */
int dilated_attn_bwd(const void* q, const void* k, const void* v, const void* out,
                     const float* lse, const void* dout, void* dq, void* dk, void* dv,
                     int64_t B, int64_t N, int64_t H, int64_t D,
                     const da_pattern_t* patterns, int64_t num_patterns,
                     int64_t causal, int64_t dtype, float softmax_scale,
                     void* workspace, uint64_t workspace_bytes, void* stream);

/*
 * dilated_attn_xpos - the xPos relative position encoding (Sun et al.,
 * "A Length-Extrapolatable Transformer", 2022), which the paper's language
 * model applies to queries and keys before its dilated attention (Sec. 4.1).
 *
 * For the row at sequence position n (0-based) of each (b, h) and each pair
 * of head-dimension elements (2i, 2i+1), i < D/2:
 *   y[2i]   = s * (x[2i] * cos(a) - x[2i+1] * sin(a))
 *   y[2i+1] = s * (x[2i] * sin(a) + x[2i+1] * cos(a))
 * with a = n * base^(-2i/D), s = zeta_i^(sign * (n - center) / scale_base)
 * and zeta_i = (2i/D + gamma) / (1 + gamma).  sign = +1 for queries and -1
 * for keys: a query at n and a key at m then meet with factors that depend
 * on n - m only (center cancels; it keeps the separate factors in range).
 * transpose = 1 applies the transpose instead (angle -a, the same s), the map
 * a backward pass multiplies the incoming gradient by.
 *
 * x, y        device pointers, [B, N, H, D] of dtype, 16-byte aligned; y may
 *             equal x (in place) but must not overlap it otherwise.
 * D           a multiple of 8, 8 <= D <= 256; B * N * H * D <= 2^34.
 * center      in [0, N).
 * base > 1, gamma > 0, scale_base > 0, all finite.  The scale exponents
 *             |n - center| / scale_base * |log2 zeta_i| must stay <= 64 for
 *             every position and pair (so that no factor leaves a 2^+-64
 *             range), else DA_EINVAL: with gamma = 0.4 and scale_base = 512
 *             about 36K positions around the center.
 * stream      a hipStream_t (NULL = the default stream); asynchronous.
 *
 * Arithmetic in float32, the angle formed and reduced in float64; y rounded
 * to dtype.  Returns DA_OK or a negative code; errors launch nothing.
 */
int dilated_attn_xpos(const void* x, void* y, int64_t B, int64_t N, int64_t H, int64_t D,
                      int64_t sign, int64_t transpose, int64_t center, float base, float gamma,
                      float scale_base, int64_t dtype, void* stream);

/*
 * dilated_attn_wgrad - weight (and bias) gradient of a linear projection of
 * the layer around the dilated attention (the Q, K, V and output projections
 * of the paper's Magneto-based language model, Sec. 4.1):
 *   dw[m][n] = sum over k < K of dy[k][m] * x[k][n],   db[m] = sum over k of dy[k][m]
 * for a projection y = x w^T + b applied to K = B * N rows, dy its incoming
 * gradient.  The long reduction over rows is split into chunks whose float32
 * partial sums go to the workspace and are then added.
 *
 * dy          device pointer, [K, M] bf16 row-major (may be NULL when K = 0).
 * x           device pointer, [K, N] bf16 row-major (may be NULL when K = 0).
 * dw          device pointer, [M, N] bf16 row-major (output, overwritten;
 *             all zeros when K = 0).
 * db          device pointer, [M] bf16 (output), or NULL for no bias gradient.
 *             dw, db and workspace must not overlap each other, dy or x.
 * K           0 <= K <= 2^30.
 * M, N        multiples of 128, at most 16384.
 * dtype       DA_BF16 (others: DA_EUNSUPPORTED).
 * workspace   device scratch of at least the bytes that
 *             dilated_attn_wgrad_workspace reports (0 when K = 0, and then
 *             workspace may be NULL), owned by the caller; contents on entry
 *             ignored, on return unspecified.
 * stream      a hipStream_t (NULL = the default stream); asynchronous.
 *
 * Products and sums in float32 (matrix cores; db on the vector units, summed
 * per 256-row slice and then over the slices), rounded to bf16 once.
 * All device pointers 16-byte aligned.  Returns DA_OK or a negative code;
 * errors launch nothing.
 */
int dilated_attn_wgrad_workspace(int64_t K, int64_t M, int64_t N, uint64_t* bytes);
int dilated_attn_wgrad(const void* dy, const void* x, void* dw, void* db, int64_t K, int64_t M,
                       int64_t N, int64_t dtype, void* workspace, uint64_t workspace_bytes,
                       void* stream);

/*
 * dilated_attn_layernorm_fwd - LayerNorm of the layer around the dilated
 * attention (the input LayerNorm and Magneto's sub-LayerNorm of the paper's
 * language model, Sec. 4.1), over rows of E elements:
 *   mean = sum(x) / E,  rstd = 1 / sqrt(sum((x - mean)^2) / E + eps),
 *   y = (x - mean) * rstd * g + b.
 *
 * x, y        device pointers, [rows, E] bf16 row-major, 16-byte aligned; y may
 *             equal x (in place) but must not overlap it otherwise.  x may be
 *             NULL when rows = 0.
 * g, b        device pointers, [E] bf16, 16-byte aligned.
 * mean, rstd  device pointers, [rows] float32 (outputs, kept for the backward).
 * rows        0 <= rows <= 2^26.
 * E           a multiple of 8, 8 <= E <= 2048.
 * eps         finite, > 0.
 * dtype       DA_BF16 (others: DA_EUNSUPPORTED).
 * stream      a hipStream_t (NULL = the default stream); asynchronous.
 *
 * Statistics and arithmetic in float32, y rounded to bf16.  Outputs must not
 * overlap each other, g, b or (mean, rstd) x.  Returns DA_OK or a negative
 * code; errors launch nothing.
 */
int dilated_attn_layernorm_fwd(const void* x, const void* g, const void* b, void* y, float* mean,
                               float* rstd, int64_t rows, int64_t E, float eps, int64_t dtype,
                               void* stream);

/*
 * dilated_attn_layernorm_bwd - gradients of dilated_attn_layernorm_fwd given
 * the incoming gradient dy and the forward's saved mean and rstd: with
 * xhat = (x - mean) * rstd and dxhat = dy * g,
 *   dx = rstd * (dxhat - mean_row(dxhat) - xhat * mean_row(dxhat * xhat)),
 *   dg = sum over rows of dy * xhat,  db = sum over rows of dy.
 *
 * dy, x       device pointers, [rows, E] bf16, 16-byte aligned.
 * g           device pointer, [E] bf16, 16-byte aligned.
 * mean, rstd  device pointers, [rows] float32 from the forward call.
 * dx          device pointer, [rows, E] bf16 (output).
 * dg, db      device pointers, [E] bf16 (outputs; zeros when rows = 0).
 * rows, E     as for the forward.
 * workspace   device scratch of at least the bytes that
 *             dilated_attn_layernorm_bwd_workspace reports, owned by the
 *             caller, 16-byte aligned; contents on entry ignored, on return
 *             unspecified.
 * stream      a hipStream_t (NULL = the default stream); asynchronous.
 *
 * Float32 arithmetic; dg and db summed per 32 rows and then over those sums
 * in a fixed order (the result does not depend on scheduling), rounded to
 * bf16 once.  Outputs and workspace must not overlap each other or any
 * input.  Returns DA_OK or a negative code; errors launch nothing.
 */
int dilated_attn_layernorm_bwd_workspace(int64_t rows, int64_t E, uint64_t* bytes);
int dilated_attn_layernorm_bwd(const void* dy, const void* x, const void* g, const float* mean,
                               const float* rstd, void* dx, void* dg, void* db, int64_t rows,
                               int64_t E, int64_t dtype, void* workspace, uint64_t workspace_bytes,
                               void* stream);

/* Human-readable text for an error code (static storage, never NULL). */
const char* dilated_attn_strerror(int code);

/*
 * Stage timing, a profiling aid (not part of the operator).
 *
 * dilated_attn_profile_begin(capacity) creates 3*capacity HIP events on the
 * current device; each of the next `capacity` dilated_attn_fwd calls records
 * one event before its first launch, one between its two launches and one
 * after the second, on the call's stream (calls beyond capacity are not
 * timed).  The two launches are the attention stage and the combine stage.
 * dilated_attn_profile_end waits for the recorded events, writes the
 * summed durations of the two stages in milliseconds and the number of timed
 * calls, and destroys the events.  capacity must be in [1, 1<<20]; any
 * pointer argument of profile_end may be NULL.  Not thread safe: one profiling
 * window per process at a time (DA_EINVAL otherwise); DA_EHIP if an event
 * call fails.
 */
int dilated_attn_profile_begin(int64_t capacity);
int dilated_attn_profile_end(double* ms_attention, double* ms_combine, int64_t* calls);

#ifdef __cplusplus
}
#endif

#endif /* DILATED_ATTN_H */
