// Stage 2 of the dilated-attention forward pass: one pass over the per-pattern
// workspace that scatters each pattern's rows back to their sequence positions
// (Sec. 2.2, Eq. 7: rows a pattern does not keep contribute nothing) and mixes
// the patterns with weights s_i / sum_j s_j, s_i = exp(lse_i) being pattern
// i's softmax denominator (Sec. 2.2, Eqs. 9-10).  It writes out [B,N,H,D] in
// the input dtype and the combined lse [B,H,N] = log(sum_i s_i) in float32.
//
// A workgroup handles a run of consecutive positions p of one (b, h); each
// lane owns eight consecutive head-dim elements of one row, so a row of a
// per-pattern output is read with D/8 16-byte (fp16) or 32-byte (fp32) loads
// and consecutive positions of a dense pattern are consecutive in memory.
// Workgroups are launched with the head innermost, so that those running at
// the same time write whole [H][D] spans of out (a position's rows of all
// heads are adjacent): 3-9 % faster than one head's positions at a time,
// whose row writes are H*D elements apart and land in as many DRAM pages.
// A per-pattern row is stored divided by a power of two (its record's
// scale), which multiplies the row's weight.
// Whether pattern i keeps row p for head h, and at which compact index t,
// follows from g = p div w, t = (p - g w) div r and (p - g w) mod r ==
// h mod r, with the divisions done by multiply-shift constants prepared on
// the host.  All loads of a row are issued before any is consumed.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace da {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr float kLog2e = 1.442695040888963407f;
constexpr float kLn2 = 0.693147180559945309f;
constexpr int kThreads = 256;

struct CombArgs {
  const char* ws;
  void* out;
  float* lse;
  int32_t N, H, npat;
  int32_t chunks;  // workgroups per (b, h); launch index = (b * chunks + chunk) * H + h
  MixPat pat[DA_MAX_PATTERNS];
};

// Eight consecutive workspace elements as loaded (converted to fp32 when used).
template <typename WsT> struct Vec8;
template <> struct Vec8<_Float16> { typedef f16x8 type; };
template <> struct Vec8<float> { typedef f32x8 type; };

// Workspace rows and records are read exactly once, but the attention
// launch just wrote them and part of them is still held in the L2 and the
// Infinity Cache: plain loads, which can hit there (nontemporal loads
// measured 9 % slower on the 32K-token workload, equal at 256K).
template <typename WsT>
__device__ inline typename Vec8<WsT>::type load8(const WsT* p) {
  typedef typename Vec8<WsT>::type V;
  return *reinterpret_cast<const V*>(p);
}

__device__ inline f32x8 to_f32(const f16x8& h) {
  f32x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = static_cast<float>(h[e]);
  return r;
}
__device__ inline f32x8 to_f32(const f32x8& v) { return v; }

// out and lse are written once and not read again by this call: nontemporal stores.
__device__ inline void store8(float* p, const f32x8& v) {
  __builtin_nontemporal_store(f32x4{v[0], v[1], v[2], v[3]}, reinterpret_cast<f32x4*>(p));
  __builtin_nontemporal_store(f32x4{v[4], v[5], v[6], v[7]}, reinterpret_cast<f32x4*>(p + 4));
}

__device__ inline void store8(unsigned short* p, const f32x8& v) {
  bf16x8 b;
#pragma unroll
  for (int e = 0; e < 8; ++e) b[e] = (__bf16)v[e];
  __builtin_nontemporal_store(b, reinterpret_cast<bf16x8*>(p));
}

// Each lane owns eight head-dim elements of kRows rows; a workgroup covers
// kRows * RPB consecutive positions (RPB = threads / lanes per row), and a
// lane's rows are RPB positions apart.  NP >= npat bounds the pattern loop at
// compile time, so that only NP sets of registers are held per row.
constexpr int kRows = 1;  // rows per lane (two measured slower: fewer waves resident)

template <int D, typename OutT, typename WsT, int NP>
__global__ __launch_bounds__(kThreads) void combine_fwd(CombArgs a) {
  constexpr int LPR = D / 8;            // lanes per row
  constexpr int RPB = kThreads / LPR;   // rows per workgroup and pass
  const int tid = __builtin_amdgcn_workitem_id_x();
  const int blk = __builtin_amdgcn_workgroup_id_x();
  const int h = blk % a.H;
  const int rest = blk / a.H;
  const int chunk = rest % a.chunks;
  const int b = rest / a.chunks;
  const int bh = b * a.H + h;
  const int p0 = chunk * (RPB * kRows) + tid / LPR;
  const int d0 = (tid % LPR) * 8;

  // Issue the loads of every pattern that keeps each of this lane's rows.
  typename Vec8<WsT>::type o[kRows][NP];
  float li[kRows][NP], sc[kRows][NP];
#pragma unroll
  for (int k = 0; k < kRows; ++k) {
    const int p = p0 + k * RPB;
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      li[k][i] = -INFINITY;
      if (i >= a.npat || p >= a.N) continue;
      const MixPat& P = a.pat[i];
      const uint32_t g = P.fw.div(static_cast<uint32_t>(p));
      const uint32_t pos = static_cast<uint32_t>(p) - g * P.fw.d;
      const uint32_t t = P.fr.div(pos);
      const uint32_t s = static_cast<uint32_t>(h) - P.fr.div(static_cast<uint32_t>(h)) * P.fr.d;
      if (pos - t * P.fr.d != s) continue;
      const int64_t row = ((int64_t)bh * P.nseg + g) * P.lmax + t;
      const f32x2 rec = reinterpret_cast<const f32x2*>(a.ws + P.lse_off)[row];
      li[k][i] = rec[0];
      sc[k][i] = rec[1];
      o[k][i] = load8(reinterpret_cast<const WsT*>(a.ws + P.o_off) + row * D + d0);
    }
  }
  // Combined log-sum-exp, then the denominator-weighted sum.
#pragma unroll
  for (int k = 0; k < kRows; ++k) {
    const int p = p0 + k * RPB;
    if (p >= a.N) continue;
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < NP; ++i) m = fmaxf(m, li[k][i]);
    OutT* out = static_cast<OutT*>(a.out) + (((int64_t)b * a.N + p) * a.H + h) * D + d0;
    float lse_v = -INFINITY;
    f32x8 acc = f32x8{0, 0, 0, 0, 0, 0, 0, 0};
    if (m != -INFINITY) {
      float den = 0.0f;
#pragma unroll
      for (int i = 0; i < NP; ++i) {
        if (li[k][i] == -INFINITY) continue;
        const float e = __builtin_amdgcn_exp2f((li[k][i] - m) * kLog2e);
        den += e;
        acc += (e * sc[k][i]) * to_f32(o[k][i]);
      }
      acc *= 1.0f / den;
      lse_v = m + __builtin_amdgcn_logf(den) * kLn2;
    }
    store8(out, acc);
    if (d0 == 0) __builtin_nontemporal_store(lse_v, a.lse + (int64_t)bh * a.N + p);
  }
}

template <int D, typename OutT, typename WsT>
void launch_one(const dim3& grid, hipStream_t stream, const CombArgs& a) {
  if (a.npat <= 4)
    hipLaunchKernelGGL((combine_fwd<D, OutT, WsT, 4>), grid, dim3(kThreads), 0, stream, a);
  else if (a.npat <= 8)
    hipLaunchKernelGGL((combine_fwd<D, OutT, WsT, 8>), grid, dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((combine_fwd<D, OutT, WsT, DA_MAX_PATTERNS>), grid, dim3(kThreads), 0, stream, a);
}

}  // namespace

hipError_t launch_combine(const Plan& plan, const void* workspace, void* out, float* lse,
                          hipStream_t stream) {
  CombArgs a;
  a.ws = static_cast<const char*>(workspace);
  a.out = out;
  a.lse = lse;
  a.N = static_cast<int32_t>(plan.N);
  a.H = static_cast<int32_t>(plan.H);
  a.npat = plan.npat;
  for (int i = 0; i < DA_MAX_PATTERNS; ++i) {
    a.pat[i] = i < plan.npat ? make_mixpat(plan.pat[i]) : MixPat{make_fastdiv(1), make_fastdiv(1), 1, 1, 0, 0};
  }
  const int rows = kThreads / (static_cast<int>(plan.D) / 8) * kRows;  // positions per workgroup
  a.chunks = static_cast<int32_t>((plan.N + rows - 1) / rows);
  const int64_t blocks = static_cast<int64_t>(a.chunks) * plan.B * plan.H;
  if (blocks >= (int64_t{1} << 31)) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(blocks));
  const bool bf = plan.dtype == DA_BF16;
  switch (plan.D) {
    case 32:
      if (bf) launch_one<32, unsigned short, _Float16>(grid, stream, a);
      else launch_one<32, float, float>(grid, stream, a);
      break;
    case 64:
      if (bf) launch_one<64, unsigned short, _Float16>(grid, stream, a);
      else launch_one<64, float, float>(grid, stream, a);
      break;
    case 128:
      if (bf) launch_one<128, unsigned short, _Float16>(grid, stream, a);
      else launch_one<128, float, float>(grid, stream, a);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace da
