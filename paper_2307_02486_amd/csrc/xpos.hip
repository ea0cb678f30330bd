// xPos relative position encoding (Sun et al. 2022), which the paper's
// language model uses together with dilated attention (Sec. 4.1), applied to
// a query or key tensor [B, N, H, D] before the attention.  Each pair of
// head-dimension elements (2i, 2i+1) of the row at position n is rotated by
// a = n * base^(-2i/D) and scaled by zeta_i^(sign (n - center) / scale_base),
// zeta_i = (2i/D + gamma) / (1 + gamma); the transpose rotates by -a with the
// same scale.  Elementwise and bound by HBM: each thread reads and writes 8
// consecutive elements (16 bytes in bf16) of one row.
#include <hip/hip_runtime.h>

#include <cmath>

#include "kernels.h"

namespace da {
namespace {

constexpr int kXposThreads = 256;
constexpr double kTwoPi = 6.283185307179586476925286766559;
constexpr double kInvTwoPi = 0.15915494309189533576888376337251;
constexpr int kMaxPairs = 128;  // D <= 256

struct XposArgs {
  const void* x;
  void* y;
  int64_t chunks;      // B * N * H * D / 8
  int32_t N, H, D, center;
  float sign;          // +1 (queries) or -1 (keys)
  float angle_sign;    // +1, or -1 for the transpose
  float inv_scale_base;
  float gamma;
  double log2_base;
};

typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ inline f32x8 load8(const float* p) { return *reinterpret_cast<const f32x8*>(p); }
__device__ inline f32x8 load8(const unsigned short* p) {
  const bf16x8 b = *reinterpret_cast<const bf16x8*>(p);
  f32x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = static_cast<float>(b[e]);
  return r;
}
__device__ inline void store8(float* p, const f32x8& v) { *reinterpret_cast<f32x8*>(p) = v; }
__device__ inline void store8(unsigned short* p, const f32x8& v) {
  bf16x8 b;
#pragma unroll
  for (int e = 0; e < 8; ++e) b[e] = (__bf16)v[e];
  *reinterpret_cast<bf16x8*>(p) = b;
}

template <typename T>
__global__ __launch_bounds__(kXposThreads) void xpos_kernel(XposArgs a) {
  // Per-pair constants, once per workgroup: theta_i = base^(-2i/D) in
  // float64 (it multiplies positions of up to tens of thousands) and
  // log2 zeta_i.
  __shared__ double theta[kMaxPairs];
  __shared__ float l2zeta[kMaxPairs];
  const int tid = __builtin_amdgcn_workitem_id_x();
  for (int i = tid; i < a.D / 2; i += kXposThreads) {
    theta[i] = exp2(-2.0 * i / a.D * a.log2_base);
    l2zeta[i] = log2f((2.0f * i / a.D + a.gamma) / (1.0f + a.gamma));
  }
  __syncthreads();
  const int64_t c = static_cast<int64_t>(__builtin_amdgcn_workgroup_id_x()) * kXposThreads + tid;
  if (c >= a.chunks) return;
  const int per_row = a.D / 8;
  const int64_t row = c / per_row;                         // (b, n, h) row
  const int i0 = static_cast<int>(c - row * per_row) * 4;  // first pair of this thread
  const int n = static_cast<int>((row / a.H) % a.N);
  const f32x8 x = load8(static_cast<const T*>(a.x) + c * 8);
  f32x8 y;
  const float rel = a.sign * static_cast<float>(n - a.center) * a.inv_scale_base;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int i = i0 + e;
    // angle n * theta_i in float64, reduced to [-pi, pi] before the float32
    // sine and cosine (n * theta_0 reaches tens of thousands of radians)
    const double ang = static_cast<double>(n) * theta[i];
    const float red = static_cast<float>(fma(-kTwoPi, rint(ang * kInvTwoPi), ang)) * a.angle_sign;
    const float sn = __sinf(red), cs = __cosf(red);
    const float s = exp2f(rel * l2zeta[i]);
    const float x0 = x[2 * e], x1 = x[2 * e + 1];
    y[2 * e] = s * (x0 * cs - x1 * sn);
    y[2 * e + 1] = s * (x0 * sn + x1 * cs);
  }
  store8(static_cast<T*>(a.y) + c * 8, y);
}

}  // namespace

hipError_t launch_xpos(const void* x, void* y, int64_t B, int64_t N, int64_t H, int64_t D, int sign,
                       bool transpose, int64_t center, float base, float gamma, float scale_base,
                       int dtype, hipStream_t stream) {
  XposArgs a;
  a.x = x;
  a.y = y;
  a.chunks = B * N * H * D / 8;
  a.N = static_cast<int32_t>(N);
  a.H = static_cast<int32_t>(H);
  a.D = static_cast<int32_t>(D);
  a.center = static_cast<int32_t>(center);
  a.sign = static_cast<float>(sign);
  a.angle_sign = transpose ? -1.0f : 1.0f;
  a.inv_scale_base = 1.0f / scale_base;
  a.gamma = gamma;
  a.log2_base = std::log2(static_cast<double>(base));
  const int64_t blocks = (a.chunks + kXposThreads - 1) / kXposThreads;
  if (blocks >= (int64_t{1} << 31)) return hipErrorInvalidValue;
  if (blocks == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(blocks));
  if (dtype == DA_BF16)
    hipLaunchKernelGGL(xpos_kernel<unsigned short>, grid, dim3(kXposThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(xpos_kernel<float>, grid, dim3(kXposThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace da
