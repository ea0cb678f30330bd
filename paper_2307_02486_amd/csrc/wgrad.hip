// Weight gradient of the LongNet attention layer's projections (the layer
// around the dilated attention, Sec. 4.1): dW[m][n] = sum_k dY[k][m] X[k][n]
// for dY [K, M] and X [K, N] bf16 row-major, K = the layer's B * N rows.
// The reduction is long (tens of thousands of rows) and the output small
// (E x E), so the work is split along k: workgroup (tile, split) computes a
// 128 x 128 output tile over one k-chunk into a float32 partial, and a second
// kernel sums the partials into bf16.  Both operands go from HBM straight to
// LDS as row-major 64 x 128 tiles (double buffered) and reach the MFMA
// (v_mfma_f32_32x32x16_bf16) through transposed LDS reads, which give each
// lane eight consecutive k of one column, the operand layout both A = dY^T
// and B = X need.  Four waves, each a 64 x 64 quarter of the tile.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "device_common.h"

namespace da {
namespace {

constexpr int kWgThreads = 256;
constexpr int kTileK = 64;    // k rows per LDS tile
constexpr int kTileMN = 128;  // output tile edge
using TLw = TileLayout<kTileMN>;
constexpr int kWgLoads = kTileK * TLw::kSlots / 64 / (kWgThreads / 64);  // 16-byte loads per lane and operand

struct WgradArgs {
  const u16* dy;
  const u16* x;
  float* part;     // [splits][M][N]
  int64_t K;
  int32_t M, N, chunk, tiles_n, tiles;
  int32_t items, per_xcd;  // tiles * splits, and items per XCD (rounded up)
};

struct SmemWgrad {
  __attribute__((aligned(16))) u16 a[2][kTileK * kTileMN];
  __attribute__((aligned(16))) u16 b[2][kTileK * kTileMN];
};

__global__ __launch_bounds__(kWgThreads) void wgrad_partial(WgradArgs a) {
  __shared__ SmemWgrad sm;
  const int tid = __builtin_amdgcn_workitem_id_x();
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hi = lane >> 5;
  // Workgroup i runs on XCD i % 8.  Item (split, tile) = split * tiles + tile
  // goes to workgroup (item % per) * 8 + item / per, so that XCD x takes items
  // [x per, (x + 1) per): the tiles of one or two neighbouring k-chunks, whose
  // rows its own L2 then serves to every tile after the first fetch.
  const int blk = __builtin_amdgcn_workgroup_id_x();
  const int item = (blk & 7) * a.per_xcd + (blk >> 3);
  if (item >= a.items) return;
  const int tile = item % a.tiles, split = item / a.tiles;
  const int m0 = (tile / a.tiles_n) * kTileMN, n0 = (tile % a.tiles_n) * kTileMN;
  const int64_t k0 = static_cast<int64_t>(split) * a.chunk;
  const int64_t k1 = k0 + a.chunk < a.K ? k0 + a.chunk : a.K;
  const int ntk = static_cast<int>((k1 - k0 + kTileK - 1) / kTileK);

  // HBM -> LDS loads: load i of this wave fills 64 consecutive 16-byte slots.
  int lrow[kWgLoads], lslot[kWgLoads];
#pragma unroll
  for (int i = 0; i < kWgLoads; ++i) {
    const int s = 64 * (wv * kWgLoads + i) + lane;
    lrow[i] = s / TLw::kSlots;
    lslot[i] = (s % TLw::kSlots) ^ TLw::swz(lrow[i]);
  }
  auto load_tile = [&](int kt, int buf) {
    const int64_t r0 = k0 + static_cast<int64_t>(kt) * kTileK;
    const int valid = static_cast<int>(k1 - r0 < kTileK ? k1 - r0 : kTileK);  // rows past k1 read as 0
    const __amdgpu_buffer_rsrc_t sa = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<u16*>(a.dy + r0 * a.M + m0), 0, valid * a.M * 2, kBufferFlags);
    const __amdgpu_buffer_rsrc_t sb = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<u16*>(a.x + r0 * a.N + n0), 0, valid * a.N * 2, kBufferFlags);
    char* la = reinterpret_cast<char*>(&sm.a[buf][0]);
    char* lb = reinterpret_cast<char*>(&sm.b[buf][0]);
#pragma unroll
    for (int i = 0; i < kWgLoads; ++i) {
      const int lds_off = 1024 * (wv * kWgLoads + i);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(sa, (lds_void*)(la + lds_off), 16, lrow[i] * a.M * 2 + lslot[i] * 16,
                                               0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(sb, (lds_void*)(lb + lds_off), 16, lrow[i] * a.N * 2 + lslot[i] * 16,
                                               0, 0, 0);
    }
  };

  // Transposed-read addresses: lane's column (m or n) within its wave's 64,
  // rows 8t + 4hi + 0..3 of each 16-row k-step.
  const int wm = wv & 1, wn = wv >> 1;
  const int tr_r = (lane & 15) >> 2;
  const int tr_c = ((lane >> 4) & 1) * 16 + (lane & 3) * 4;
  int aoff[2][2], boff[2][2];
#pragma unroll
  for (int blk2 = 0; blk2 < 2; ++blk2)
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int cm = wm * 64 + blk2 * 32 + tr_c, cn = wn * 64 + blk2 * 32 + tr_c;
      aoff[blk2][t] = TLw::offset(8 * t + 4 * hi + tr_r, cm >> 3) + (cm & 7) * 2;
      boff[blk2][t] = TLw::offset(8 * t + 4 * hi + tr_r, cn >> 3) + (cn & 7) * 2;
    }

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  if (ntk > 0) load_tile(0, 0);
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  __syncthreads();
  for (int kt = 0; kt < ntk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < ntk) load_tile(kt + 1, cur ^ 1);
    const uint32_t la = lds_addr(&sm.a[cur][0]), lb = lds_addr(&sm.b[cur][0]);
    static_for<0, kTileK / 16>([&](auto KK) {
      constexpr int row = 16 * decltype(KK)::value;  // multiple of 16: the swizzle of rows 0..15
      u32x2 fa[2][2], fb[2][2];
      static_for<0, 2>([&](auto B2) {
        static_for<0, 2>([&](auto T) {
          constexpr int bb = decltype(B2)::value, t = decltype(T)::value;
          fa[bb][t] = lds_read_tr16<row * TLw::kRowBytes>(la + aoff[bb][t]);
          fb[bb][t] = lds_read_tr16<row * TLw::kRowBytes>(lb + boff[bb][t]);
        });
      });
      lds_wait<0>();
      bf16x8 av[2], bv[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        lds_bind(fa[i][0]);
        lds_bind(fa[i][1]);
        lds_bind(fb[i][0]);
        lds_bind(fb[i][1]);
        av[i] = __builtin_bit_cast(bf16x8, u32x4{fa[i][0][0], fa[i][0][1], fa[i][1][0], fa[i][1][1]});
        bv[i] = __builtin_bit_cast(bf16x8, u32x4{fb[i][0][0], fb[i][0][1], fb[i][1][0], fb[i][1][1]});
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
    });
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();
  }

  // C layout: lane holds column n = lane % 32 and rows 8 jj + 4 hi + e.
  float* part = a.part + static_cast<int64_t>(split) * a.M * a.N;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int m = m0 + wm * 64 + i * 32 + 8 * jj + 4 * hi + e;
          const int n = n0 + wn * 64 + j * 32 + (lane & 31);
          part[static_cast<int64_t>(m) * a.N + n] = acc[i][j][4 * jj + e];
        }
}

__global__ __launch_bounds__(kWgThreads) void wgrad_sum(const float* part, u16* dw, int64_t mn, int splits) {
  const int64_t i = (static_cast<int64_t>(__builtin_amdgcn_workgroup_id_x()) * kWgThreads +
                     __builtin_amdgcn_workitem_id_x()) * 4;
  if (i >= mn) return;
  f32x4 s = f32x4{0, 0, 0, 0};
  for (int p = 0; p < splits; ++p) s += *reinterpret_cast<const f32x4*>(part + p * mn + i);
  u16 o[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) o[e] = __builtin_bit_cast(u16, (__bf16)s[e]);
  *reinterpret_cast<u32x2*>(dw + i) = u32x2{o[0] | (static_cast<unsigned>(o[1]) << 16),
                                            o[2] | (static_cast<unsigned>(o[3]) << 16)};
}

// Bias gradient db[m] = sum_k dy[k][m], in two steps.  colsum_partial: the
// workgroup (column block bx, slice y) sums rows [y rs, (y + 1) rs) of 512
// columns, each lane 8 columns (one 16-byte load per row) over every fourth
// row, the four row lanes combined through LDS, into part[y][M].
__global__ __launch_bounds__(kWgThreads) void colsum_partial(const u16* dy, float* part, int64_t K, int M, int rs,
                                                             int col_blocks) {
  __shared__ __attribute__((aligned(16))) float red[4][64 * 8];
  const int tid = __builtin_amdgcn_workitem_id_x();
  const int cgl = tid & 63, rl = tid >> 6;
  const int blk = __builtin_amdgcn_workgroup_id_x();
  const int y = blk / col_blocks;
  const int cg = (blk % col_blocks) * 64 + cgl;  // group of 8 columns
  const int64_t r0 = static_cast<int64_t>(y) * rs;
  const int64_t r1 = r0 + rs < K ? r0 + rs : K;
  float s[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) s[e] = 0.0f;
  if (cg < (M >> 3)) {
#pragma unroll 8
    for (int64_t r = r0 + rl; r < r1; r += 4) {
      const u32x4 w = *reinterpret_cast<const u32x4*>(dy + r * M + 8 * cg);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        s[2 * i] += __builtin_bit_cast(float, w[i] << 16);
        s[2 * i + 1] += __builtin_bit_cast(float, w[i] & 0xffff0000u);
      }
    }
  }
  *reinterpret_cast<f32x4*>(&red[rl][8 * cgl]) = f32x4{s[0], s[1], s[2], s[3]};
  *reinterpret_cast<f32x4*>(&red[rl][8 * cgl + 4]) = f32x4{s[4], s[5], s[6], s[7]};
  __syncthreads();
  if (rl == 0 && cg < (M >> 3)) {
    float* out = part + static_cast<int64_t>(y) * M + 8 * cg;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const f32x4 v = (*reinterpret_cast<const f32x4*>(&red[0][8 * cgl + 4 * h]) +
                       *reinterpret_cast<const f32x4*>(&red[1][8 * cgl + 4 * h])) +
                      (*reinterpret_cast<const f32x4*>(&red[2][8 * cgl + 4 * h]) +
                       *reinterpret_cast<const f32x4*>(&red[3][8 * cgl + 4 * h]));
      *reinterpret_cast<f32x4*>(out + 4 * h) = v;
    }
  }
}

// colsum_final: db[c] = sum over the R slices of part[y][c], 32 columns per
// workgroup and 8 row lanes per column, combined through LDS; zeros for R = 0.
__global__ __launch_bounds__(kWgThreads) void colsum_final(const float* part, u16* db, int M, int R) {
  __shared__ float red[8][32];
  const int tid = __builtin_amdgcn_workitem_id_x();
  const int cl = tid & 31, rl = tid >> 5;
  const int c = __builtin_amdgcn_workgroup_id_x() * 32 + cl;  // M is a multiple of 32
  float s = 0.0f;
#pragma unroll 16
  for (int y = rl; y < R; y += 8) s += part[static_cast<int64_t>(y) * M + c];
  red[rl][cl] = s;
  __syncthreads();
  if (rl == 0) {
    const float t = ((red[0][cl] + red[1][cl]) + (red[2][cl] + red[3][cl])) +
                    ((red[4][cl] + red[5][cl]) + (red[6][cl] + red[7][cl]));
    db[c] = __builtin_bit_cast(u16, (__bf16)t);
  }
}

}  // namespace

// Slices of the bias-gradient column sums: 256 rows each, at most 1024.
int64_t colsum_slices(int64_t K, int64_t* rows_per_slice) {
  *rows_per_slice = 0;
  if (K <= 0) return 0;
  int64_t R = (K + 255) / 256;
  if (R > 1024) R = 1024;
  *rows_per_slice = (K + R - 1) / R;
  return (K + *rows_per_slice - 1) / *rows_per_slice;
}

uint64_t wgrad_workspace(int64_t K, int64_t M, int64_t N) {
  int64_t chunk = 0, rs = 0;
  return (static_cast<uint64_t>(wgrad_splits(K, M, N, &chunk)) * N + colsum_slices(K, &rs)) * M * 4;
}

// Splits of the reduction: at most 512 workgroups in all (two per compute
// unit, as 64 KiB of LDS per workgroup allows) unless the output alone has
// more tiles, each split a whole number of k tiles; no split for K = 0 (dW
// is then zero).
int64_t wgrad_splits(int64_t K, int64_t M, int64_t N, int64_t* chunk) {
  *chunk = 0;
  if (K <= 0) return 0;
  const int64_t tiles = (M / kTileMN) * (N / kTileMN);
  const int64_t ktiles = (K + kTileK - 1) / kTileK;
  const int64_t s = std::max<int64_t>(1, std::min<int64_t>(512 / tiles, ktiles));
  *chunk = (ktiles + s - 1) / s * kTileK;
  return (K + *chunk - 1) / *chunk;
}

hipError_t launch_wgrad(const void* dy, const void* x, void* dw, void* db, int64_t K, int64_t M, int64_t N,
                        void* workspace, hipStream_t stream) {
  int64_t chunk = 0;
  const int64_t splits = wgrad_splits(K, M, N, &chunk);
  WgradArgs a;
  a.dy = static_cast<const u16*>(dy);
  a.x = static_cast<const u16*>(x);
  a.part = static_cast<float*>(workspace);
  a.K = K;
  a.M = static_cast<int32_t>(M);
  a.N = static_cast<int32_t>(N);
  a.chunk = static_cast<int32_t>(chunk);
  a.tiles_n = static_cast<int32_t>(N / kTileMN);
  a.tiles = static_cast<int32_t>((M / kTileMN) * (N / kTileMN));
  a.items = static_cast<int32_t>(a.tiles * splits);
  a.per_xcd = (a.items + 7) / 8;
  if (splits > 0)
    hipLaunchKernelGGL(wgrad_partial, dim3(static_cast<unsigned>(8 * a.per_xcd)), dim3(kWgThreads), 0, stream, a);
  const int64_t mn = M * N;
  hipLaunchKernelGGL(wgrad_sum, dim3(static_cast<unsigned>((mn / 4 + kWgThreads - 1) / kWgThreads)),
                     dim3(kWgThreads), 0, stream, static_cast<const float*>(workspace), static_cast<u16*>(dw), mn,
                     static_cast<int>(splits));
  if (db) {
    int64_t rs = 0;
    const int64_t R = colsum_slices(K, &rs);
    float* part = static_cast<float*>(workspace) + splits * mn;
    const int col_blocks = static_cast<int>((M / 8 + 63) / 64);
    if (R > 0)
      hipLaunchKernelGGL(colsum_partial, dim3(static_cast<unsigned>(R * col_blocks)), dim3(kWgThreads), 0, stream,
                         static_cast<const u16*>(dy), part, K, static_cast<int>(M), static_cast<int>(rs), col_blocks);
    hipLaunchKernelGGL(colsum_final, dim3(static_cast<unsigned>(M / 32)), dim3(kWgThreads), 0, stream,
                       static_cast<const float*>(part), static_cast<u16*>(db), static_cast<int>(M), static_cast<int>(R));
  }
  return hipGetLastError();
}

}  // namespace da
