// Stage 2 of the dilated-attention forward pass: one pass over the per-pattern
// workspace that scatters each pattern's rows back to their sequence positions
// (Sec. 2.2, Eq. 7: rows a pattern does not keep contribute nothing) and mixes
// the patterns with weights s_i / sum_j s_j, s_i = exp(lse_i) being pattern
// i's softmax denominator (Sec. 2.2, Eqs. 9-10).  It writes out [B,N,H,D] in
// the input dtype and the combined lse [B,H,N] = log(sum_i s_i) in float32.
//
// A workgroup handles a run of consecutive positions p of one (b, h): each
// lane owns four consecutive head-dim elements of one row, so a row of the
// compact per-pattern output is read with D/4 16-byte loads and consecutive
// positions of a dense pattern are consecutive in memory.  Whether pattern i
// keeps row p for head h, and at which compact index t, follows from
// g = p div w, t = (p - g w) div r and (p - g w) mod r == h mod r, with the
// divisions done by multiply-shift constants prepared on the host.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace da {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.442695040888963407f;
constexpr float kLn2 = 0.693147180559945309f;
constexpr int kThreads = 256;

struct CombPat {
  FastDiv fw;      // division by w
  FastDiv fr;      // division by r
  int32_t nseg, lmax;
  int64_t o_off;   // float offset of the pattern's output rows
  int64_t lse_off; // float offset of the pattern's lse
};

struct CombArgs {
  const float* ws;
  void* out;
  float* lse;
  int32_t N, H, npat;
  int32_t chunks;  // workgroups per (b, h)
  CombPat pat[DA_MAX_PATTERNS];
};

__device__ inline void store4(float* p, const f32x4& v) { *reinterpret_cast<f32x4*>(p) = v; }

__device__ inline void store4(unsigned short* p, const f32x4& v) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  bf16x4 b;
  b[0] = (__bf16)v[0];
  b[1] = (__bf16)v[1];
  b[2] = (__bf16)v[2];
  b[3] = (__bf16)v[3];
  *reinterpret_cast<bf16x4*>(p) = b;
}

template <int D, typename OutT>
__global__ __launch_bounds__(kThreads) void combine_fwd(CombArgs a) {
  constexpr int LPR = D / 4;             // lanes per row
  constexpr int RPB = kThreads / LPR;    // rows per workgroup
  const int tid = threadIdx.x;
  const int bh = blockIdx.x / a.chunks;
  const int p = (blockIdx.x - bh * a.chunks) * RPB + tid / LPR;
  const int d0 = (tid % LPR) * 4;
  if (p >= a.N) return;
  const int h = bh % a.H;

  float m = -INFINITY;  // running max of lse_i (natural log)
  float den = 0.0f;     // sum_i exp(lse_i - m)
  f32x4 acc = f32x4{0, 0, 0, 0};
  for (int i = 0; i < a.npat; ++i) {
    const CombPat& P = a.pat[i];
    const uint32_t g = P.fw.div(static_cast<uint32_t>(p));
    const uint32_t pos = static_cast<uint32_t>(p) - g * P.fw.d;
    const uint32_t t = P.fr.div(pos);
    const uint32_t s = static_cast<uint32_t>(h) - P.fr.div(static_cast<uint32_t>(h)) * P.fr.d;
    if (pos - t * P.fr.d != s) continue;
    const int64_t row = ((int64_t)bh * P.nseg + g) * P.lmax + t;
    const float li = a.ws[P.lse_off + row];
    const f32x4 o = *reinterpret_cast<const f32x4*>(a.ws + P.o_off + row * D + d0);
    if (li > m) {
      const float c = __builtin_amdgcn_exp2f((m - li) * kLog2e);
      den *= c;
      acc *= c;
      m = li;
    }
    const float e = __builtin_amdgcn_exp2f((li - m) * kLog2e);
    den += e;
    acc += e * o;
  }
  const int b = bh / a.H;
  OutT* out = static_cast<OutT*>(a.out) + (((int64_t)b * a.N + p) * a.H + h) * D + d0;
  float lse_v;
  if (den > 0.0f) {
    const float inv = 1.0f / den;
    store4(out, acc * inv);
    lse_v = m + __builtin_amdgcn_logf(den) * kLn2;
  } else {
    store4(out, f32x4{0, 0, 0, 0});
    lse_v = -INFINITY;
  }
  if (d0 == 0) a.lse[(int64_t)bh * a.N + p] = lse_v;
}

}  // namespace

hipError_t launch_combine(const Plan& plan, const void* workspace, void* out, float* lse,
                          hipStream_t stream) {
  CombArgs a;
  a.ws = static_cast<const float*>(workspace);
  a.out = out;
  a.lse = lse;
  a.N = static_cast<int32_t>(plan.N);
  a.H = static_cast<int32_t>(plan.H);
  a.npat = plan.npat;
  for (int i = 0; i < DA_MAX_PATTERNS; ++i) {
    CombPat& c = a.pat[i];
    if (i < plan.npat) {
      const PatternPlan& pp = plan.pat[i];
      c.fw = make_fastdiv(static_cast<uint32_t>(pp.w));
      c.fr = make_fastdiv(static_cast<uint32_t>(pp.r));
      c.nseg = static_cast<int32_t>(pp.nseg);
      c.lmax = static_cast<int32_t>(pp.lmax);
      c.o_off = static_cast<int64_t>(pp.o_off / 4);
      c.lse_off = static_cast<int64_t>(pp.lse_off / 4);
    } else {
      c = CombPat{make_fastdiv(1), make_fastdiv(1), 1, 1, 0, 0};
    }
  }
  const int rpb = kThreads / (static_cast<int>(plan.D) / 4);
  a.chunks = static_cast<int32_t>((plan.N + rpb - 1) / rpb);
  const int64_t blocks = static_cast<int64_t>(a.chunks) * plan.B * plan.H;
  if (blocks >= (int64_t{1} << 31)) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(blocks));
  const bool bf = plan.dtype == DA_BF16;
  switch (plan.D) {
    case 32:
      if (bf) hipLaunchKernelGGL((combine_fwd<32, unsigned short>), grid, dim3(kThreads), 0, stream, a);
      else hipLaunchKernelGGL((combine_fwd<32, float>), grid, dim3(kThreads), 0, stream, a);
      break;
    case 64:
      if (bf) hipLaunchKernelGGL((combine_fwd<64, unsigned short>), grid, dim3(kThreads), 0, stream, a);
      else hipLaunchKernelGGL((combine_fwd<64, float>), grid, dim3(kThreads), 0, stream, a);
      break;
    case 128:
      if (bf) hipLaunchKernelGGL((combine_fwd<128, unsigned short>), grid, dim3(kThreads), 0, stream, a);
      else hipLaunchKernelGGL((combine_fwd<128, float>), grid, dim3(kThreads), 0, stream, a);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace da
