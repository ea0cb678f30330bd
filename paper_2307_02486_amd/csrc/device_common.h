// Device-side pieces shared by the attention kernels: vector types, the
// per-pattern records and the work-item decode, the LDS tile layout and LDS
// access helpers.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

#include "kernels.h"

namespace da {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned short u16;

constexpr float kLn2 = 0.693147180559945309f;
constexpr float kLog2e = 1.442695040888963407f;

struct PatArgs {
  int32_t w, r, nseg, lmax, ntiles, units;
  int64_t o_off;    // byte offset of this pattern's output rows in the workspace
  int64_t lse_off;  // byte offset of this pattern's (lse, scale) row records
};

// One attention work item: which segment of which pattern, and which query tile.
struct Item {
  int pi;          // pattern index
  int b, h, g;     // batch, head, segment
  int unit;        // (b*H + h)*nseg + g
  int tq;          // query tile index inside the segment
  int L;           // kept rows of this (head, segment)
  int64_t row0;    // [B,N,H] row index of kept row t = 0
  int64_t rstride; // row-index step between consecutive kept rows (r*H)
  int p0;          // sequence position of kept row t = 0
};

// Workgroups are handed to the eight XCDs round-robin (launch index mod 8),
// so launch index x is mapped to XCD c = x mod 8 and the units with index = c
// (mod 8) are given to that XCD: the query tiles of one segment run on one
// XCD and its K/V rows are fetched into that XCD's L2 once.  (A pattern whose
// unit count is not a multiple of 8 has the long query tiles of its last
// units mod 8 units dealt to the XCDs one by one instead, trading their L2
// reuse for balance.)  On each XCD the
// items come in two phases.  First, pattern by pattern (in the order of the
// records, those with the most query tiles per segment first) and unit by unit, the query tiles from the
// last (the longest under a causal mask) down to tile kShortTiles, so the
// tiles of a segment run close together in time.  Then
// the first kShortTiles query tiles of every unit, level by level from tile
// kShortTiles - 1 down to tile 0: the shortest items are dispatched last and
// fill the gaps as the longer ones drain.
constexpr int kShortTiles = 3;

// Number of units of a pattern that XCD c owns.
template <typename Pat>
__device__ inline int units_on_xcd(const Pat& P, int c) {
  return P.units > c ? (P.units - c + 7) >> 3 : 0;
}

template <typename Args>
__device__ inline bool decode_item(const Args& a, int bid, int block_m, Item& it) {
  const int c = bid & 7;
  int slot = bid >> 3;
  int pi = -1, unit = 0, tq = 0;
  // Fully unrolled: the records are read with constant offsets, in a few
  // scalar loads issued together.
#pragma unroll
  for (int p = 0; p < DA_MAX_PATTERNS; ++p) {
    if (p >= a.npat) break;
    const auto& P = a.pat[p];
    const int nlong = P.ntiles > kShortTiles ? P.ntiles - kShortTiles : 0;
    if ((P.units & 7) == 0) {
      const int n = units_on_xcd(P, c) * nlong;
      if (slot < n) {
        pi = p;
        const int j = slot / nlong;
        unit = c + 8 * j;
        tq = P.ntiles - 1 - (slot - j * nlong);
        break;
      }
      slot -= n;
    } else {
      // A unit count that is not a multiple of 8 would load the XCDs
      // unevenly: the first units8 = units - units mod 8 units go to the
      // XCDs whole as above, and the long items f = (unit - units8) * nlong +
      // (ntiles-1-tq) of the remaining ones are dealt to the XCDs one by one
      // (f = c mod 8 to XCD c), trading their L2 reuse for balance.
      const int units8 = P.units & ~7;
      const int na = (units8 >> 3) * nlong;
      if (slot < na) {
        pi = p;
        const int j = slot / nlong;
        unit = c + 8 * j;
        tq = P.ntiles - 1 - (slot - j * nlong);
        break;
      }
      const int rest = (P.units - units8) * nlong;
      const int nb = rest > c ? (rest - c + 7) >> 3 : 0;
      if (slot - na < nb) {
        pi = p;
        const int f = c + 8 * (slot - na);
        const int j = f / nlong;
        unit = units8 + j;
        tq = P.ntiles - 1 - (f - j * nlong);
        break;
      }
      slot -= na + nb;
    }
  }
#pragma unroll
  for (int t = kShortTiles - 1; t >= 0; --t) {
    if (pi >= 0) break;
#pragma unroll
    for (int p = 0; p < DA_MAX_PATTERNS; ++p) {
      if (p >= a.npat) break;
      const auto& P = a.pat[p];
      const int n = P.ntiles > t ? units_on_xcd(P, c) : 0;
      if (slot < n) {
        pi = p;
        unit = c + 8 * slot;
        tq = t;
        break;
      }
      slot -= n;
    }
  }
  if (pi < 0) return false;
  const auto& P = a.pat[pi];
  it.tq = tq;
  it.pi = pi;
  it.unit = unit;
  it.g = unit % P.nseg;
  const int bh = unit / P.nseg;
  it.h = bh % a.H;
  it.b = bh / a.H;
  const int s = it.h % P.r;
  const int seg_start = it.g * P.w;
  const int seg_len = min(P.w, a.N - seg_start);
  it.L = seg_len > s ? (seg_len - s + P.r - 1) / P.r : 0;
  it.row0 = ((int64_t)it.b * a.N + seg_start + s) * a.H + it.h;
  it.rstride = (int64_t)P.r * a.H;
  it.p0 = seg_start + s;
  return it.tq * block_m < it.L;
}

// Tiles of rows live in LDS row-major (D bf16 per row), without padding:
// a row is D/8 16-byte slots and logical slot c of row k is stored at slot
// c ^ swz(k).  LDS serves 256 bytes per cycle from 64 four-byte banks, i.e.
// sixteen 16-byte bank groups; a 16-byte read is served 16 lanes per cycle,
// an 8-byte read 32 lanes per cycle.  swz(k) makes both access patterns of
// the kernel conflict-free:
//   row fragments (ds_read_b128): 16 consecutive rows at one logical slot
//     -> 16 bank groups;
//   transposed reads (ds_read_b64_tr_b16): 4 consecutive rows (aligned) x 4
//     consecutive slots -> 16.
// Row k starts at bank group (k * D/8) mod 16, which swz(k) complements; it
// depends on bits 0-3 of k only, so rows 16 apart share it.
template <int D>
struct TileLayout {
  static constexpr int kSlots = D / 8;                     // 16-byte slots per row
  static constexpr int kRowBytes = D * 2;
  __device__ static int swz(int row) {
    if constexpr (D == 32) return (row >> 2) & 3;
    else if constexpr (D == 64) return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
    else return ((row & 3) << 2) | ((row >> 2) & 3);
  }
  __device__ static int offset(int row, int slot) {        // byte offset of a slot
    return row * kRowBytes + ((slot ^ swz(row)) << 4);
  }
};

typedef __attribute__((address_space(3))) void lds_void;

__device__ inline u32x4 load16(const u16* p) { return *reinterpret_cast<const u32x4*>(p); }

// The value held by lane l ^ 32 (the other half-wave), via v_permlane32_swap.
__device__ inline float other_half(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto sw = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const unsigned lane = __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  return __builtin_bit_cast(float, lane < 32 ? sw[1] : sw[0]);
}

// LDS byte address of a pointer into a __shared__ array.
__device__ inline uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<size_t>((const lds_void*)p));
}

// ds_read_b64_tr_b16 at a VGPR address plus a constant byte offset.  Within
// each 16-lane group, lane 4r + c supplies the address of four consecutive
// 16-bit elements of row r (c = 0..3) and receives element c of each of the
// four rows.  Issued as inline assembly: the compiler's builtin for this
// instruction makes it wait for every outstanding HBM-to-LDS load first,
// including the prefetch of the next tile, which it cannot tell apart from
// the tile being read.  The results are therefore not tracked by the
// compiler; lds_wait<N>() followed by lds_bind() on each result makes them
// usable once at most N LDS operations of this wave are still outstanding
// (LDS operations complete in order).
template <int kOff>
__device__ inline u32x2 lds_read_tr16(uint32_t addr) {
  u32x2 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(kOff) : "memory");
  return r;
}
// The counter field holds at most 15: a wave cannot have more LDS operations
// in flight, so with more than 15 younger ones issued the awaited one is done.
template <int N>
__device__ inline void lds_wait() {
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"i"(N > 15 ? 15 : N) : "memory");
}
__device__ inline void lds_bind(u32x2& r) { asm volatile("" : "+v"(r)); }

// Calls f(std::integral_constant<int, I>) for I = 0 .. N-1, so that the index
// can form a constant operand.
template <int I, int N, typename F>
__device__ inline void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// Rows stored as fp16 scaled by a power of two per row (the forward pass's
// per-pattern outputs, the backward pass's per-pattern gradients): a row x is
// stored as x * 2^-e with e chosen so that the row's largest magnitude lands
// in [2^14, 2^15), and 2^e is kept beside it.  The row keeps fp16's eleven
// significant bits relative to its largest element and bf16's exponent range.
// amax_times_inv = (largest |element| of the row) * inv, where inv is a factor
// the row is multiplied by before it is stored; returns mul = inv * 2^-e (the
// factor to apply) and stored = 2^e.
__device__ inline void row_scale(float amax_times_inv, float inv, float& mul, float& stored) {
  // biased exponent E of a = amax_times_inv: a in [2^(E-127), 2^(E-126));
  // a * 2^(141-E) is in [2^14, 2^15).  E is clamped to [15, 254] so that both
  // powers of two are normal floats (rows below 2^-111 keep fewer bits).
  int E = static_cast<int>((__builtin_bit_cast(unsigned, amax_times_inv) >> 23) & 0xff);
  E = min(max(E, 15), 254);
  mul = inv * __builtin_bit_cast(float, static_cast<unsigned>(268 - E) << 23);     // inv * 2^(141-E)
  stored = __builtin_bit_cast(float, static_cast<unsigned>(E - 14) << 23);         // 2^(E-141)
}

// Word 3 of a raw buffer resource on gfx9-family GPUs (32-bit data format,
// no swizzle); with stride 0 the size field is a byte count and reads at or
// beyond it return zero.
constexpr int kBufferFlags = 0x00020000;
// s_waitcnt immediate: vmcnt(0), expcnt and lgkmcnt left at their maxima.
constexpr int kWaitVmcnt0 = 0x0F70;

}  // namespace
}  // namespace da
