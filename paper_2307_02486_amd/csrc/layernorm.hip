// LayerNorm of the LongNet attention layer (the input LayerNorm and Magneto's
// sub-LayerNorm around the dilated attention, Sec. 4.1), forward and
// backward, bf16 rows of E <= 2048 elements with float32 statistics.
//
// Forward: one wave per row; each lane holds J chunks of 8 elements
// (chunk c = lane + 64 j), the mean and then the variance of the deviations
// come from two wave sums, y = (x - mean) rstd g + b.
// Backward: one wave per row as well, 8 rows per wave and 32 per workgroup;
// with xhat = (x - mean) rstd recomputed from the saved statistics and
// dxhat = dy g,  dx = rstd (dxhat - mean(dxhat) - xhat mean(dxhat xhat)).
// The parameter gradients dg = sum_rows dy xhat and db = sum_rows dy are
// summed per lane over a wave's rows, over the workgroup's waves through LDS,
// and then over workgroups by two small reduction kernels, all in a fixed
// order (the result does not depend on scheduling).
#include <hip/hip_runtime.h>

#include "device_common.h"

namespace da {
namespace {

constexpr int kLnThreads = 256;
constexpr int kLnRowsPerWave = 8;
constexpr int kLnRowsPerWg = kLnRowsPerWave * kLnThreads / 64;
constexpr int kLnSlice = 32;  // workgroup partials summed per thread in the first reduction

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

__device__ inline void unpack8(const u32x4 w, float* f) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __builtin_bit_cast(float, w[i] << 16);
    f[2 * i + 1] = __builtin_bit_cast(float, w[i] & 0xffff0000u);
  }
}

__device__ inline void load8f(const u16* p, float* f) { unpack8(*reinterpret_cast<const u32x4*>(p), f); }

__device__ inline void store8bf(u16* p, const float* f) {
  u32x4 w;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = static_cast<unsigned>(__builtin_bit_cast(u16, (__bf16)f[2 * i])) |
           (static_cast<unsigned>(__builtin_bit_cast(u16, (__bf16)f[2 * i + 1])) << 16);
  *reinterpret_cast<u32x4*>(p) = w;
}

struct LnFwdArgs {
  const u16 *x, *g, *b;
  u16* y;
  float *mean, *rstd;
  int64_t rows;
  int32_t E;
  float eps;
};

template <int J>
__global__ __launch_bounds__(kLnThreads) void ln_fwd(LnFwdArgs a) {
  const int lane = __builtin_amdgcn_workitem_id_x() & 63;
  const int64_t row = static_cast<int64_t>(__builtin_amdgcn_workgroup_id_x()) * (kLnThreads / 64) +
                      (__builtin_amdgcn_workitem_id_x() >> 6);
  if (row >= a.rows) return;  // whole waves only; the kernel has no barrier
  const int nch = a.E >> 3;
  const u16* xr = a.x + row * a.E;
  float v[J][8];
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int c = lane + 64 * j;
    if (c < nch) {
      load8f(xr + 8 * c, v[j]);
#pragma unroll
      for (int e = 0; e < 8; ++e) s += v[j][e];
    }
  }
  const float inv_e = 1.0f / static_cast<float>(a.E);
  const float mean = wave_sum(s) * inv_e;
  float q = 0.0f;
#pragma unroll
  for (int j = 0; j < J; ++j)
    if (lane + 64 * j < nch)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = v[j][e] - mean;
        q += d * d;
      }
  const float rstd = 1.0f / sqrtf(wave_sum(q) * inv_e + a.eps);
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int c = lane + 64 * j;
    if (c < nch) {
      float g[8], b[8], y[8];
      load8f(a.g + 8 * c, g);
      load8f(a.b + 8 * c, b);
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = (v[j][e] - mean) * rstd * g[e] + b[e];
      store8bf(a.y + row * a.E + 8 * c, y);
    }
  }
  if (lane == 0) {
    a.mean[row] = mean;
    a.rstd[row] = rstd;
  }
}

struct LnBwdArgs {
  const u16 *dy, *x, *g;
  const float *mean, *rstd;
  u16* dx;
  float* part;  // [workgroups][2E]: dg partials, then db partials
  int64_t rows;
  int32_t E;
};

template <int J>
__global__ __launch_bounds__(kLnThreads) void ln_bwd(LnBwdArgs a) {
  extern __shared__ __attribute__((aligned(16))) float red[];  // [4 waves][2E]
  const int tid = __builtin_amdgcn_workitem_id_x();
  const int lane = tid & 63, wv = tid >> 6;
  const int nch = a.E >> 3;
  float g[J][8], pg[J][8], pb[J][8];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int c = lane + 64 * j;
#pragma unroll
    for (int e = 0; e < 8; ++e) g[j][e] = pg[j][e] = pb[j][e] = 0.0f;
    if (c < nch) load8f(a.g + 8 * c, g[j]);
  }
  const float inv_e = 1.0f / static_cast<float>(a.E);
  const int64_t r0 = static_cast<int64_t>(__builtin_amdgcn_workgroup_id_x()) * kLnRowsPerWg + wv * kLnRowsPerWave;
  const int nrow = static_cast<int>(min(static_cast<int64_t>(kLnRowsPerWave), a.rows - r0));  // may be <= 0
  // Row i + 1's x and dy are loaded (as raw bf16) while row i is processed.
  u32x4 nx[J], ndy[J];
  auto load_row = [&](int64_t row) {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int c = lane + 64 * j;
      if (c < nch) {
        nx[j] = *reinterpret_cast<const u32x4*>(a.x + row * a.E + 8 * c);
        ndy[j] = *reinterpret_cast<const u32x4*>(a.dy + row * a.E + 8 * c);
      }
    }
  };
  if (nrow > 0) load_row(r0);
  for (int i = 0; i < nrow; ++i) {
    const int64_t row = r0 + i;
    const float mean = a.mean[row], rstd = a.rstd[row];
    u32x4 xr[J], dyr[J];
#pragma unroll
    for (int j = 0; j < J; ++j) {
      xr[j] = nx[j];
      dyr[j] = ndy[j];
    }
    if (i + 1 < nrow) load_row(row + 1);
    float s1 = 0.0f, s2 = 0.0f;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      if (lane + 64 * j < nch) {
        float x[8], dy[8];
        unpack8(xr[j], x);
        unpack8(dyr[j], dy);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float xh = (x[e] - mean) * rstd, dxh = dy[e] * g[j][e];
          s1 += dxh;
          s2 += dxh * xh;
          pg[j][e] += dy[e] * xh;
          pb[j][e] += dy[e];
        }
      }
    }
    const float m1 = wave_sum(s1) * inv_e, m2 = wave_sum(s2) * inv_e;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int c = lane + 64 * j;
      if (c < nch) {
        float x[8], dy[8], dx[8];
        unpack8(xr[j], x);
        unpack8(dyr[j], dy);
#pragma unroll
        for (int e = 0; e < 8; ++e) dx[e] = rstd * (dy[e] * g[j][e] - m1 - (x[e] - mean) * rstd * m2);
        store8bf(a.dx + row * a.E + 8 * c, dx);
      }
    }
  }
  float* mine = red + wv * 2 * a.E;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int c = lane + 64 * j;
    if (c < nch) {
      *reinterpret_cast<f32x4*>(mine + 8 * c) = f32x4{pg[j][0], pg[j][1], pg[j][2], pg[j][3]};
      *reinterpret_cast<f32x4*>(mine + 8 * c + 4) = f32x4{pg[j][4], pg[j][5], pg[j][6], pg[j][7]};
      *reinterpret_cast<f32x4*>(mine + a.E + 8 * c) = f32x4{pb[j][0], pb[j][1], pb[j][2], pb[j][3]};
      *reinterpret_cast<f32x4*>(mine + a.E + 8 * c + 4) = f32x4{pb[j][4], pb[j][5], pb[j][6], pb[j][7]};
    }
  }
  __syncthreads();
  float* out = a.part + static_cast<int64_t>(__builtin_amdgcn_workgroup_id_x()) * 2 * a.E;
  for (int i = tid; i < 2 * a.E; i += kLnThreads)
    out[i] = (red[i] + red[2 * a.E + i]) + (red[4 * a.E + i] + red[6 * a.E + i]);
}

// part [nwg][W] -> part2 [ceil(nwg / kLnSlice)][W]: column sums over slices of kLnSlice rows.
__global__ __launch_bounds__(kLnThreads) void ln_reduce_slices(const float* part, float* part2, int nwg, int W) {
  const int col = __builtin_amdgcn_workgroup_id_x() * kLnThreads + __builtin_amdgcn_workitem_id_x();
  const int sl = __builtin_amdgcn_workgroup_id_y();
  if (col >= W) return;
  const int r1 = min(nwg, (sl + 1) * kLnSlice);
  float s = 0.0f;
#pragma unroll 8
  for (int r = sl * kLnSlice; r < r1; ++r) s += part[static_cast<int64_t>(r) * W + col];
  part2[static_cast<int64_t>(sl) * W + col] = s;
}

// part2 [S][2E] -> dg [E], db [E] in bf16.
__global__ __launch_bounds__(kLnThreads) void ln_reduce_final(const float* part2, u16* dg, u16* db, int S, int E) {
  const int col = __builtin_amdgcn_workgroup_id_x() * kLnThreads + __builtin_amdgcn_workitem_id_x();
  if (col >= 2 * E) return;
  float s = 0.0f;
#pragma unroll 8
  for (int r = 0; r < S; ++r) s += part2[static_cast<int64_t>(r) * 2 * E + col];
  u16* dst = col < E ? dg + col : db + (col - E);
  *dst = __builtin_bit_cast(u16, (__bf16)s);
}

}  // namespace

uint64_t layernorm_bwd_workspace(int64_t rows, int64_t E) {
  const int64_t nwg = (rows + kLnRowsPerWg - 1) / kLnRowsPerWg;
  const int64_t S = (nwg + kLnSlice - 1) / kLnSlice;
  return static_cast<uint64_t>(nwg + S) * 2 * E * 4;
}

hipError_t launch_layernorm_fwd(const void* x, const void* g, const void* b, void* y, float* mean, float* rstd,
                                int64_t rows, int64_t E, float eps, hipStream_t stream) {
  LnFwdArgs a{static_cast<const u16*>(x), static_cast<const u16*>(g), static_cast<const u16*>(b),
              static_cast<u16*>(y), mean, rstd, rows, static_cast<int32_t>(E), eps};
  if (rows == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((rows + 3) / 4));
  const int J = static_cast<int>((E / 8 + 63) / 64);
  if (J == 1) hipLaunchKernelGGL(ln_fwd<1>, grid, dim3(kLnThreads), 0, stream, a);
  else if (J == 2) hipLaunchKernelGGL(ln_fwd<2>, grid, dim3(kLnThreads), 0, stream, a);
  else hipLaunchKernelGGL(ln_fwd<4>, grid, dim3(kLnThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_layernorm_bwd(const void* dy, const void* x, const void* g, const float* mean, const float* rstd,
                                void* dx, void* dg, void* db, int64_t rows, int64_t E, void* workspace,
                                hipStream_t stream) {
  const int64_t nwg = (rows + kLnRowsPerWg - 1) / kLnRowsPerWg;
  const int64_t S = (nwg + kLnSlice - 1) / kLnSlice;
  float* part = static_cast<float*>(workspace);
  float* part2 = part + nwg * 2 * E;
  LnBwdArgs a{static_cast<const u16*>(dy), static_cast<const u16*>(x), static_cast<const u16*>(g), mean, rstd,
              static_cast<u16*>(dx), part, rows, static_cast<int32_t>(E)};
  const int J = static_cast<int>((E / 8 + 63) / 64);
  const dim3 grid(static_cast<unsigned>(nwg));
  const int W = static_cast<int>(2 * E);
  const size_t smem = static_cast<size_t>(kLnThreads / 64) * 2 * E * sizeof(float);
  if (nwg > 0) {  // no rows: only the final kernel, which then writes zeros
    if (J == 1) hipLaunchKernelGGL(ln_bwd<1>, grid, dim3(kLnThreads), smem, stream, a);
    else if (J == 2) hipLaunchKernelGGL(ln_bwd<2>, grid, dim3(kLnThreads), smem, stream, a);
    else hipLaunchKernelGGL(ln_bwd<4>, grid, dim3(kLnThreads), smem, stream, a);
    hipLaunchKernelGGL(ln_reduce_slices, dim3(static_cast<unsigned>((W + kLnThreads - 1) / kLnThreads),
                                            static_cast<unsigned>(S)),
                       dim3(kLnThreads), 0, stream, part, part2, static_cast<int>(nwg), W);
  }
  hipLaunchKernelGGL(ln_reduce_final, dim3(static_cast<unsigned>((W + kLnThreads - 1) / kLnThreads)),
                     dim3(kLnThreads), 0, stream, part2, static_cast<u16*>(dg), static_cast<u16*>(db),
                     static_cast<int>(S), static_cast<int>(E));
  return hipGetLastError();
}

}  // namespace da
