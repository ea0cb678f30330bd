// Stage 1 of the dilated-attention forward pass on gfx950: per pattern, per
// (batch, head, segment), gather the kept rows (every r-th row from the head's
// offset, Sec. 2.2 Eqs. 3-5 and Sec. 2.3) straight from HBM into registers and
// LDS, and run softmax attention on them (Sec. 2.2 Eq. 6) with an online
// softmax.  The normalised output rows and their log-sum-exp go to the
// workspace in compact per-pattern order [b][h][segment][t][D].
//
// bf16 path: one work item = 128 query rows of one sparsified segment, four
// waves of 32 rows.  Scores are computed transposed, S^T = K Q^T, with
// v_mfma_f32_32x32x16_bf16, so that every lane owns one query row: the row
// max needs one exchange between the two half-waves and the probabilities can
// feed the P V product (computed as O^T = V^T P^T) straight from registers.
// V is stored transposed in LDS, with keys permuted inside each group of 16
// so a lane's eight keys of one MFMA step are contiguous.
//
// f32 path: a plain VALU kernel (one thread per query row) used for float32
// inputs, where accuracy rather than speed is the point.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace da {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16;

constexpr float kLn2 = 0.693147180559945309f;
constexpr float kLog2e = 1.442695040888963407f;
constexpr float kNegBig = -1.0e30f;   // finite "minus infinity" for running maxima

struct PatArgs {
  int32_t w, r, nseg, lmax, ntiles, units;
  int64_t o_off;    // byte offset of this pattern's output rows in the workspace
  int64_t lse_off;  // byte offset of this pattern's lse in the workspace
};

struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  char* ws;
  int32_t B, N, H, npat, causal, total_items;
  float scale_log2;  // softmax scale times log2(e): scores go to exp2 directly
  PatArgs pat[DA_MAX_PATTERNS];
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
};

// Work items are ordered pattern by pattern; inside a pattern, unit by unit
// (segment fastest), and inside a unit the query tiles run from the last (the
// longest under a causal mask) to the first.  Workgroups are handed to the
// eight XCDs round-robin (launch index mod 8), so launch index x is mapped to
// XCD c = x mod 8 and the units with index = c (mod 8) are given to that XCD:
// the query tiles of one segment then run on one XCD, close together in time,
// and its K/V rows are fetched into that XCD's L2 once.
__device__ inline bool decode_item(const AttnArgs& a, int bid, int block_m, Item& it) {
  const int c = bid & 7;
  int slot = bid >> 3;
  int pi = 0;
  for (;; ++pi) {
    if (pi >= a.npat) return false;
    const PatArgs& P = a.pat[pi];
    const int n = (P.units > c ? (P.units - c + 7) >> 3 : 0) * P.ntiles;
    if (slot < n) break;
    slot -= n;
  }
  const PatArgs& P = a.pat[pi];
  const int j = slot / P.ntiles;
  const int unit = c + 8 * j;
  it.tq = P.ntiles - 1 - (slot - j * P.ntiles);
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
  return it.tq * block_m < it.L;
}

// ---------------------------------------------------------------------------
// bf16 MFMA kernel
// ---------------------------------------------------------------------------
#ifndef DA_BF16_WAVES
#define DA_BF16_WAVES 4
#endif
constexpr int kThreads = 64 * DA_BF16_WAVES;  // waves of 32 query rows each
constexpr int kBM = 32 * DA_BF16_WAVES;       // query rows per work item
// A row's running max is raised only when a tile's max exceeds it by more than
// this (log2 units); until then probabilities may reach 2^kRescaleSlack, which
// bf16 and the fp32 sums hold exactly as well as values below 1.
constexpr float kRescaleSlack = 8.0f;

// Keys per K/V tile for a head dim: 128 where the registers allow it.
#ifndef DA_KEY_TILE_SMALL_D
#define DA_KEY_TILE_SMALL_D 64
#endif
// 32-key blocks of S^T whose K fragments are read from LDS together, before
// their MFMAs, so LDS latency is paid once per group rather than per MFMA.
#ifndef DA_QK_GROUP
#define DA_QK_GROUP 2
#endif
template <int D> struct KeyTile { static constexpr int value = D <= 64 ? DA_KEY_TILE_SMALL_D : 64; };

// Position of key `key` inside a transposed V row: within each group of 16
// keys, keys {0-3, 8-11} come first and {4-7, 12-15} second, which is the
// order in which the upper and lower half-waves hold them after S^T.
__device__ inline int vt_pos(int key) {
  const int k16 = key & 15;
  return (key & ~15) | (((k16 >> 2) & 1) << 3) | ((k16 >> 3) << 2) | (k16 & 3);
}

template <int D, int BN>
struct SmemBf16 {
  static constexpr int KSTR = D + 8;    // row pitch (elements) of a K tile
  static constexpr int VSTR = BN + 8;   // row pitch (elements) of a V^T tile
  u16 k[2][BN * KSTR];                  // double-buffered
  u16 vt[2][D * VSTR];
};

__device__ inline u32x4 load16(const u16* p) { return *reinterpret_cast<const u32x4*>(p); }

// The value held by lane l ^ 32 (the other half-wave), via v_permlane32_swap.
__device__ inline float other_half(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto sw = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const unsigned lane = __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  return __builtin_bit_cast(float, lane < 32 ? sw[1] : sw[0]);
}

// Word 3 of a raw buffer resource on gfx9-family GPUs (32-bit data format,
// no swizzle); with stride 0 the size field is a byte count and reads at or
// beyond it return zero.
constexpr int kBufferFlags = 0x00020000;

template <int D, bool kBufferLoads>
__global__ __launch_bounds__(kThreads) void attn_fwd_bf16(AttnArgs a) {
  static_assert(D % 32 == 0, "head dim must be a multiple of 32");
  constexpr int BN = KeyTile<D>::value;
  constexpr int KC = D / 16;  // MFMA k-steps over the head dim
  constexpr int DB = D / 32;  // 32-wide blocks of the head dim in O^T
  constexpr int SB = BN / 32; // 32-key blocks of S^T per tile
  constexpr int KTASKS = BN * D / 8;                        // 16-B K chunks per tile
  constexpr int KT = (KTASKS + kThreads - 1) / kThreads;    // K chunks per thread
  constexpr int VTASKS = (BN / 2) * (D / 8);                // (key pair, 8-wide chunk) V tasks
  constexpr int VT = (VTASKS + kThreads - 1) / kThreads;    // V tasks per thread
  using Smem = SmemBf16<D, BN>;
  __shared__ __attribute__((aligned(16))) Smem sm;

  Item it;
  if (!decode_item(a, __builtin_amdgcn_workgroup_id_x(), kBM, it)) return;
  const PatArgs& P = a.pat[it.pi];
  const u16* __restrict__ qg = static_cast<const u16*>(a.q);

  const int tid = __builtin_amdgcn_workitem_id_x();
  const int lane = tid & 63;
  const int wv = tid >> 6;
  const int qr = lane & 31;   // query column of this lane in S^T / O^T
  const int hi = lane >> 5;   // half-wave
  const int L = it.L;
  const int q0 = it.tq * kBM;
  const int qend = min(q0 + kBM, L);
  const int tq_row = q0 + wv * 32 + qr;  // this lane's query (kept-row index)
  const bool q_valid = tq_row < L;
  const int64_t row_step = it.rstride * D;  // elements between consecutive kept rows

  // Q^T operand: lane holds query tq_row, head-dim slice [16c + 8hi, +8).
  bf16x8 qreg[KC];
  {
    const u16* qp = qg + (it.row0 + (int64_t)tq_row * it.rstride) * D + 8 * hi;
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      u32x4 x = q_valid ? load16(qp + 16 * c) : u32x4{0, 0, 0, 0};
      // q * scale * log2(e), rounded to bf16: the MFMA then yields scores in
      // log2 units and the exponent needs no per-score multiply.
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const unsigned bits = (x[e >> 1] >> (16 * (e & 1))) << 16;
        qreg[c][e] = (__bf16)(__builtin_bit_cast(float, bits) * a.scale_log2);
      }
    }
  }

  // Fixed per-thread roles in the tile loads:
  //  K chunk i: key (tid + 256i) / (D/8), head-dim chunk (tid + 256i) % (D/8)
  //  V task i:  keys 2kp, 2kp+1 with kp = (tid + 256i) % (BN/2), chunk (tid + 256i) / (BN/2)
  // With kBufferLoads, a tile is read through a buffer resource whose base is
  // the tile's first kept row and whose size ends at the segment's last kept
  // row: each thread keeps a fixed 32-bit offset, and rows past the end read
  // as zero without any per-load test.  Otherwise 64-bit pointers and tests.
  int kkey[KT], kdc[KT];
#pragma unroll
  for (int i = 0; i < KT; ++i) {
    const int task = min(tid + i * kThreads, KTASKS - 1);
    kkey[i] = task / (D / 8);
    kdc[i] = task % (D / 8);
  }
  int vkey[VT], vdc[VT];
#pragma unroll
  for (int i = 0; i < VT; ++i) {
    const int task = min(tid + i * kThreads, VTASKS - 1);
    vkey[i] = 2 * (task % (BN / 2));
    vdc[i] = task / (BN / 2);
  }
  const u16* kbase = static_cast<const u16*>(a.k) + it.row0 * D;
  const u16* vbase = static_cast<const u16*>(a.v) + it.row0 * D;
  const int64_t tile_step = row_step * BN;

  u32x4 rk[KT], rv0[VT], rv1[VT];
  auto load_tile = [&](int jt) {
    const int k0 = jt * BN;
    if constexpr (kBufferLoads) {
      const uint64_t row_bytes = static_cast<uint64_t>(row_step) * 2;
      const uint64_t valid = static_cast<uint64_t>(L - k0) * row_bytes;
      const int nrec = static_cast<int>(valid < 0x7fffffffull ? valid : 0x7fffffffull);
      const __amdgpu_buffer_rsrc_t rk_src = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<u16*>(kbase + tile_step * jt), 0, nrec, kBufferFlags);
      const __amdgpu_buffer_rsrc_t rv_src = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<u16*>(vbase + tile_step * jt), 0, nrec, kBufferFlags);
#pragma unroll
      for (int i = 0; i < KT; ++i)
        rk[i] = __builtin_amdgcn_raw_buffer_load_b128(
            rk_src, static_cast<int>(kkey[i] * row_bytes) + kdc[i] * 16, 0, 0);
#pragma unroll
      for (int i = 0; i < VT; ++i) {
        const int off = static_cast<int>(vkey[i] * row_bytes) + vdc[i] * 16;
        rv0[i] = __builtin_amdgcn_raw_buffer_load_b128(rv_src, off, 0, 0);
        rv1[i] = __builtin_amdgcn_raw_buffer_load_b128(rv_src, off + static_cast<int>(row_bytes), 0, 0);
      }
    } else {
      const int64_t off = tile_step * jt;
#pragma unroll
      for (int i = 0; i < KT; ++i)
        rk[i] = k0 + kkey[i] < L ? load16(kbase + off + kkey[i] * row_step + kdc[i] * 8) : u32x4{0, 0, 0, 0};
#pragma unroll
      for (int i = 0; i < VT; ++i) {
        const int t = k0 + vkey[i];
        const u16* vp = vbase + off + vkey[i] * row_step + vdc[i] * 8;
        rv0[i] = t < L ? load16(vp) : u32x4{0, 0, 0, 0};
        rv1[i] = t + 1 < L ? load16(vp + row_step) : u32x4{0, 0, 0, 0};
      }
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KT; ++i) {
      const int task = tid + i * kThreads;
      if (KTASKS % kThreads == 0 || task < KTASKS)
        *reinterpret_cast<u32x4*>(&sm.k[buf][(task / (D / 8)) * Smem::KSTR + (task % (D / 8)) * 8]) = rk[i];
    }
#pragma unroll
    for (int i = 0; i < VT; ++i) {
      const int task = tid + i * kThreads;
      if (VTASKS % kThreads == 0 || task < VTASKS) {
        u16* dst = &sm.vt[buf][(task / (BN / 2)) * 8 * Smem::VSTR + vt_pos(2 * (task % (BN / 2)))];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          // (key 2kp, key 2kp+1) of head-dim element dc*8 + e, as one 32-bit word
          const unsigned sel = (e & 1) ? 0x07060302u : 0x05040100u;
          *reinterpret_cast<unsigned*>(dst + e * Smem::VSTR) =
              __builtin_amdgcn_perm(rv1[i][e >> 1], rv0[i][e >> 1], sel);
        }
      }
    }
  };

  f32x16 acc_o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc_o[db] = f32x16{};
  float m_run = 0.0f;     // reference max of scaled scores (log2 domain), set by tile 0
  f32x16 negm = f32x16{}; // -m_run in every slot: the initial value of each S' block
  float l_run = 0.0f;     // this half-wave's share of the running denominator

  const int kv_end = a.causal ? qend : L;
  const int ntile = (kv_end + BN - 1) / BN;
  const int wq_lo = q0 + wv * 32;  // smallest query of this wave
  const int lim = a.causal ? min(tq_row, L - 1) : L - 1;  // last visible key of this lane

  load_tile(0);
  store_tile(0);
  __syncthreads();
  for (int jt = 0; jt < ntile; ++jt) {
    const int cur = jt & 1;
    const int k0 = jt * BN;
    const bool more = jt + 1 < ntile;
    if (more) load_tile(jt + 1);

    // Tiles entirely after this wave's queries are skipped (causal).
    if (!(a.causal && k0 > wq_lo + 31)) {
      // S^T = K Q^T, one 32x32 block per 32 keys; the K fragments of a group
      // of blocks are all requested from LDS before the group's MFMAs.
      f32x16 acc_s[SB];
      constexpr int QG = DA_QK_GROUP < SB ? DA_QK_GROUP : SB;
#pragma unroll
      for (int kb0 = 0; kb0 < SB; kb0 += QG) {
        u32x4 kf[QG][KC];
#pragma unroll
        for (int g = 0; g < QG; ++g)
#pragma unroll
          for (int c = 0; c < KC; ++c)
            kf[g][c] = *reinterpret_cast<const u32x4*>(
                &sm.k[cur][((kb0 + g) * 32 + qr) * Smem::KSTR + 16 * c + 8 * hi]);
        __builtin_amdgcn_sched_barrier(0);  // keep the reads ahead of the MFMAs
#pragma unroll
        for (int g = 0; g < QG; ++g) {
          acc_s[kb0 + g] = negm;  // scores start at -m: S' = q'k - m
#pragma unroll
          for (int c = 0; c < KC; ++c)
            acc_s[kb0 + g] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8, kf[g][c]), qreg[c], acc_s[kb0 + g], 0, 0, 0);
        }
      }
      // Mask keys after the query (causal) and past the segment's end.
      if ((a.causal && k0 + BN - 1 > wq_lo) || k0 + BN > L) {
        const int base = k0 + 4 * hi - lim;   // key - lim = base + offset(kb, j)
#pragma unroll
        for (int kb = 0; kb < SB; ++kb)
#pragma unroll
          for (int j = 0; j < 16; ++j)
            if (base + kb * 32 + 8 * (j >> 2) + (j & 3) > 0) acc_s[kb][j] = -INFINITY;
      }
      // Tile max of this lane's query, across both half-waves.
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < SB; ++kb)
#pragma unroll
        for (int j = 0; j < 16; j += 2) mx = fmaxf(mx, fmaxf(acc_s[kb][j], acc_s[kb][j + 1]));
      mx = fmaxf(mx, other_half(mx));  // already relative to m_run, log2 units
      // Lazy rescale: the first tile fixes the reference max; later tiles move
      // it only when some row of the wave would see probabilities above
      // 2^kRescaleSlack.
      if (jt == 0 || __any(mx > kRescaleSlack)) {
        const float delta = jt == 0 ? mx : fmaxf(mx, 0.0f);
        const float alpha = __builtin_amdgcn_exp2f(-delta);
        m_run += delta;
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int j = 0; j < 16; ++j) acc_o[db][j] *= alpha;
#pragma unroll
        for (int kb = 0; kb < SB; ++kb)
#pragma unroll
          for (int j = 0; j < 16; ++j) acc_s[kb][j] -= delta;
#pragma unroll
        for (int j = 0; j < 16; ++j) negm[j] = -m_run;
      }
      // P = exp2(S'); bf16 P feeds the PV MFMA.  The row sums are taken in
      // fp32 with plain adds (dot-product instructions would not issue while
      // other waves' MFMAs run).  The V^T fragments of a 32-key block are
      // requested before its exps.
      float lp[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kb = 0; kb < SB; ++kb) {
        u32x4 vf[2][DB];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int db = 0; db < DB; ++db)
            vf[kk][db] = *reinterpret_cast<const u32x4*>(
                &sm.vt[cur][(db * 32 + qr) * Smem::VSTR + (kb * 2 + kk) * 16 + 8 * hi]);
        __builtin_amdgcn_sched_barrier(0);  // keep the reads ahead of the exps
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          bf16x8 pb;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float pe = __builtin_amdgcn_exp2f(acc_s[kb][8 * kk + e]);
            lp[e & 3] += pe;
            pb[e] = (__bf16)pe;
          }
#pragma unroll
          for (int db = 0; db < DB; ++db)
            acc_o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vf[kk][db]),
                                                                pb, acc_o[db], 0, 0, 0);
        }
      }
      l_run += (lp[0] + lp[1]) + (lp[2] + lp[3]);
    }
    if (more) store_tile(cur ^ 1);
    __syncthreads();
  }

  // Epilogue: normalise and write this lane's row of the per-pattern output.
  const float l_tot = l_run + other_half(l_run);
  if (!q_valid) return;
  const float inv = 1.0f / l_tot;
  const int64_t wrow = (int64_t)it.unit * P.lmax + tq_row;
  _Float16* orow = reinterpret_cast<_Float16*>(a.ws + P.o_off) + wrow * D;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      f16x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = (_Float16)(acc_o[db][4 * jj + e] * inv);
      *reinterpret_cast<f16x4*>(orow + db * 32 + 8 * jj + 4 * hi) = o;
    }
  if (hi == 0)
    reinterpret_cast<float*>(a.ws + P.lse_off)[wrow] = (m_run + __builtin_amdgcn_logf(l_tot)) * kLn2;
}

// ---------------------------------------------------------------------------
// f32 VALU kernel: one thread per query row, 64 rows per work item.
// ---------------------------------------------------------------------------
constexpr int kBM32 = 64;
constexpr int kBN32 = 16;

template <int D>
__global__ __launch_bounds__(kBM32) void attn_fwd_f32(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) float ks[kBN32][D];
  __shared__ __attribute__((aligned(16))) float vs[kBN32][D];
  Item it;
  if (!decode_item(a, __builtin_amdgcn_workgroup_id_x(), kBM32, it)) return;
  const PatArgs& P = a.pat[it.pi];
  const float* __restrict__ qg = static_cast<const float*>(a.q);
  const float* __restrict__ kg = static_cast<const float*>(a.k);
  const float* __restrict__ vg = static_cast<const float*>(a.v);
  const int tid = __builtin_amdgcn_workitem_id_x();
  const int L = it.L;
  const int q0 = it.tq * kBM32;
  const int qend = min(q0 + kBM32, L);
  const int t = q0 + tid;
  const bool valid = t < L;

  float qv[D], o[D];
  {
    const float* qp = qg + (it.row0 + (int64_t)min(t, L - 1) * it.rstride) * D;
#pragma unroll
    for (int d = 0; d < D; d += 4) {
      const f32x4 x = *reinterpret_cast<const f32x4*>(qp + d);
      qv[d] = x[0]; qv[d + 1] = x[1]; qv[d + 2] = x[2]; qv[d + 3] = x[3];
      o[d] = o[d + 1] = o[d + 2] = o[d + 3] = 0.0f;
    }
  }
  float m_run = kNegBig, l_run = 0.0f;
  const int kv_end = a.causal ? qend : L;
  const int lim = a.causal ? t : L - 1;
  for (int k0 = 0; k0 < kv_end; k0 += kBN32) {
    __syncthreads();
    for (int task = tid; task < kBN32 * D / 4; task += kBM32) {
      const int key = task / (D / 4);
      const int dc = (task % (D / 4)) * 4;
      const int tk = k0 + key;
      f32x4 xk = f32x4{0, 0, 0, 0}, xv = f32x4{0, 0, 0, 0};
      if (tk < L) {
        const int64_t off = (it.row0 + (int64_t)tk * it.rstride) * D + dc;
        xk = *reinterpret_cast<const f32x4*>(kg + off);
        xv = *reinterpret_cast<const f32x4*>(vg + off);
      }
      *reinterpret_cast<f32x4*>(&ks[key][dc]) = xk;
      *reinterpret_cast<f32x4*>(&vs[key][dc]) = xv;
    }
    __syncthreads();
    float s[kBN32];
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < kBN32; ++j) {
      float acc = 0.0f;
#pragma unroll
      for (int d = 0; d < D; ++d) acc = fmaf(qv[d], ks[j][d], acc);
      s[j] = (k0 + j <= lim) ? acc : -INFINITY;
      mx = fmaxf(mx, s[j]);
    }
    const float m_new = fmaxf(m_run, mx * a.scale_log2);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    float psum = 0.0f;
#pragma unroll
    for (int j = 0; j < kBN32; ++j) {
      s[j] = __builtin_amdgcn_exp2f(fmaf(s[j], a.scale_log2, -m_new));
      psum += s[j];
    }
    l_run = fmaf(l_run, alpha, psum);
#pragma unroll
    for (int d = 0; d < D; ++d) {
      float acc = o[d] * alpha;
#pragma unroll
      for (int j = 0; j < kBN32; ++j) acc = fmaf(s[j], vs[j][d], acc);
      o[d] = acc;
    }
  }
  if (!valid) return;
  const float inv = 1.0f / l_run;
  const int64_t wrow = (int64_t)it.unit * P.lmax + t;
  float* orow = reinterpret_cast<float*>(a.ws + P.o_off) + wrow * D;
#pragma unroll
  for (int d = 0; d < D; d += 4)
    *reinterpret_cast<f32x4*>(orow + d) = f32x4{o[d] * inv, o[d + 1] * inv, o[d + 2] * inv, o[d + 3] * inv};
  reinterpret_cast<float*>(a.ws + P.lse_off)[wrow] = (m_run + __builtin_amdgcn_logf(l_run)) * kLn2;
}

}  // namespace

hipError_t launch_attention(const Plan& plan, const void* q, const void* k, const void* v,
                            void* workspace, hipStream_t stream) {
  AttnArgs a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.ws = static_cast<char*>(workspace);
  a.B = static_cast<int32_t>(plan.B);
  a.N = static_cast<int32_t>(plan.N);
  a.H = static_cast<int32_t>(plan.H);
  a.npat = plan.npat;
  a.causal = plan.causal;
  a.total_items = static_cast<int32_t>(plan.total_items);
  a.scale_log2 = plan.scale * kLog2e;
  for (int i = 0; i < DA_MAX_PATTERNS; ++i) {
    PatArgs& pa = a.pat[i];
    if (i < plan.npat) {
      const PatternPlan& pp = plan.pat[i];
      pa.w = static_cast<int32_t>(pp.w);
      pa.r = static_cast<int32_t>(pp.r);
      pa.nseg = static_cast<int32_t>(pp.nseg);
      pa.lmax = static_cast<int32_t>(pp.lmax);
      pa.ntiles = static_cast<int32_t>(pp.ntiles);
      pa.units = static_cast<int32_t>(pp.units);
      pa.o_off = static_cast<int64_t>(pp.o_off);
      pa.lse_off = static_cast<int64_t>(pp.lse_off);
    } else {
      pa = PatArgs{1, 1, 1, 1, 1, 0, 0, 0};
    }
  }
  if (plan.total_items == 0) return hipSuccess;
  // XCD 0 holds the most units of every pattern; the launch covers 8 times its slots.
  const dim3 grid(static_cast<unsigned>(plan.launch_items));
  if (plan.dtype == DA_BF16) {
    switch (plan.D) {
      case 32:
        if (plan.offsets32) hipLaunchKernelGGL((attn_fwd_bf16<32, true>), grid, dim3(kThreads), 0, stream, a);
        else hipLaunchKernelGGL((attn_fwd_bf16<32, false>), grid, dim3(kThreads), 0, stream, a);
        break;
      case 64:
        if (plan.offsets32) hipLaunchKernelGGL((attn_fwd_bf16<64, true>), grid, dim3(kThreads), 0, stream, a);
        else hipLaunchKernelGGL((attn_fwd_bf16<64, false>), grid, dim3(kThreads), 0, stream, a);
        break;
      case 128:
        if (plan.offsets32) hipLaunchKernelGGL((attn_fwd_bf16<128, true>), grid, dim3(kThreads), 0, stream, a);
        else hipLaunchKernelGGL((attn_fwd_bf16<128, false>), grid, dim3(kThreads), 0, stream, a);
        break;
      default: return hipErrorInvalidValue;
    }
  } else {
    switch (plan.D) {
      case 32: hipLaunchKernelGGL(attn_fwd_f32<32>, grid, dim3(kBM32), 0, stream, a); break;
      case 64: hipLaunchKernelGGL(attn_fwd_f32<64>, grid, dim3(kBM32), 0, stream, a); break;
      case 128: hipLaunchKernelGGL(attn_fwd_f32<128>, grid, dim3(kBM32), 0, stream, a); break;
      default: return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

}  // namespace da
