// Stage 1 of the dilated-attention forward pass on gfx950: per pattern, per
// (batch, head, segment), gather the kept rows (every r-th row from the head's
// offset, Sec. 2.2 Eqs. 3-5 and Sec. 2.3) straight from HBM into LDS, and run
// softmax attention on them (Sec. 2.2 Eq. 6) with an online softmax.  The
// normalised output rows go to the workspace in compact per-pattern order
// [b][h][segment][t][D], with one (lse, scale) record per row.
//
// bf16 path: one work item = 128 query rows of one sparsified segment, four
// waves of 32 rows.  Scores are computed transposed, S^T = K Q^T, with
// v_mfma_f32_32x32x16_bf16, so that every lane owns one query row: the row
// max needs one exchange between the two half-waves and the probabilities can
// feed the P V product (computed as O^T = V^T P^T) straight from registers.
// K and V tiles are loaded from HBM into LDS without passing through
// registers; V^T fragments come from transposed LDS reads.
//
// f32 path: a plain VALU kernel (one thread per query row) used for float32
// inputs, where accuracy rather than speed is the point.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "device_common.h"

namespace da {
namespace {

constexpr float kNegBig = -1.0e30f;   // finite "minus infinity" for running maxima

struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  char* ws;
  int32_t B, N, H, npat, causal, total_items;
  float scale_log2;  // softmax scale times log2(e), applied to the fp32 scores
  // The patterns of this launch, ordered by query tiles per unit, most first
  // (the kernels only use a pattern's index to find its record here).
  PatArgs pat[DA_MAX_PATTERNS];
};

// ---------------------------------------------------------------------------
// bf16 MFMA kernel
// ---------------------------------------------------------------------------
constexpr int kThreads = 256;  // four waves of 32 query rows each
constexpr int kBM = 128;       // query rows per work item
#ifndef DA_KEY_TILE
#define DA_KEY_TILE 64
#endif
constexpr int kBN = DA_KEY_TILE;  // keys per K/V tile
// Online softmax without a per-tile row max.  Each row's reference max m is
// the true max of its first key tile; later tiles exponentiate S - m directly
// and the row's reference is moved only afterwards, from the tile's row sums:
// a tile whose probabilities of one half-row sum to more than kSumSlack moves
// m up by log2 of the row's tile sum (so that the tile's probabilities, and
// the output accumulated so far, are rescaled to a sum of one).  Probabilities
// above 1 are held by bf16 and the fp32 sums exactly as well as those below.
// A half-row sum above kSumLimit (or not finite: a probability overflowed)
// makes the whole work item run again in the safe mode, which takes the row
// max of every tile before exponentiating (raising m when the tile max exceeds
// it by more than kRescaleSlack).
constexpr float kRescaleSlack = 8.0f;
constexpr float kSumSlack = 1024.0f;
constexpr float kSumLimit = 4294967296.0f;  // 2^32

template <int D>
struct SmemBf16 {
  __attribute__((aligned(16))) u16 k[2][kBN * D];  // double-buffered K tiles
  __attribute__((aligned(16))) u16 v[2][kBN * D];  // double-buffered V tiles
  int redo;  // set by a wave whose tile sums left the fast path's range
};

template <int D, bool kBufferLoads>
__global__ __launch_bounds__(kThreads) void attn_fwd_bf16(AttnArgs a) {
  static_assert(D % 32 == 0, "head dim must be a multiple of 32");
  constexpr int BN = kBN;
  constexpr int KC = D / 16;  // MFMA k-steps over the head dim
  constexpr int DB = D / 32;  // 32-wide blocks of the head dim in O^T
  constexpr int SB = BN / 32; // 32-key blocks of S^T per tile
  using TL = TileLayout<D>;
  // A wave's load instruction fills 64 consecutive 16-byte LDS slots.
  constexpr int kLoadsPerWave = BN * TL::kSlots / 64 / (kThreads / 64);
  static_assert(kLoadsPerWave >= 1, "tile too small for four waves");
  __shared__ SmemBf16<D> sm;

  Item it;
  if (!decode_item(a, __builtin_amdgcn_workgroup_id_x(), kBM, it)) return;
  const PatArgs& P = a.pat[it.pi];
  const u16* __restrict__ qg = static_cast<const u16*>(a.q);

  const int tid = __builtin_amdgcn_workitem_id_x();
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index (uniform)
  const int qr = lane & 31;   // query column of this lane in S^T / O^T
  const int hi = lane >> 5;   // half-wave
  const int L = it.L;
  const int q0 = it.tq * kBM;
  const int qend = min(q0 + kBM, L);
  const int tq_row = q0 + wv * 32 + qr;  // this lane's query (kept-row index)
  const bool q_valid = tq_row < L;
  const int64_t row_step = it.rstride * D;  // elements between consecutive kept rows
  const float c = a.scale_log2;             // > 0

  // Q^T operand: lane holds query tq_row, head-dim slice [16c + 8hi, +8).  The
  // loads are issued here and consumed after the first K/V tile's loads have
  // been issued, so the two latencies overlap.
  // Rows past the segment's end load its last row (unconditional loads, no
  // branches) and are zeroed before use.
  u32x4 qraw[KC];
  {
    const int qrow = min(tq_row, L - 1);
    const u16* qp = qg + (it.row0 + (int64_t)qrow * it.rstride) * D + 8 * hi;
#pragma unroll
    for (int c = 0; c < KC; ++c) qraw[c] = load16(qp + 16 * c);
  }

  // Tile loads go straight from HBM to LDS (no registers, no LDS stores).
  // Load i of this wave fills LDS slots [64 (wv*kLoadsPerWave + i), +64): lane
  // l takes slot s = 64 (wv*kLoadsPerWave + i) + l, i.e. row s / kSlots and
  // physical slot s % kSlots, and fetches the logical slot stored there.
  int lrow[kLoadsPerWave], lslot[kLoadsPerWave];
#pragma unroll
  for (int i = 0; i < kLoadsPerWave; ++i) {
    const int s = 64 * (wv * kLoadsPerWave + i) + lane;
    lrow[i] = s / TL::kSlots;
    lslot[i] = (s % TL::kSlots) ^ TL::swz(lrow[i]);
  }
  const u16* kbase = static_cast<const u16*>(a.k) + it.row0 * D;
  const u16* vbase = static_cast<const u16*>(a.v) + it.row0 * D;
  const int64_t tile_step = row_step * BN;
  auto load_tile = [&](int jt, int buf) {
    const int k0 = jt * BN;
    char* kl = reinterpret_cast<char*>(&sm.k[buf][0]);
    char* vl = reinterpret_cast<char*>(&sm.v[buf][0]);
    if constexpr (kBufferLoads) {
      // Buffer resources based at the tile's first kept row, sized to end at
      // the segment's last kept row: rows past it arrive as zeros.
      const uint64_t row_bytes = static_cast<uint64_t>(row_step) * 2;
      const uint64_t valid = static_cast<uint64_t>(L - k0) * row_bytes;
      const int nrec = static_cast<int>(valid < 0x7fffffffull ? valid : 0x7fffffffull);
      const __amdgpu_buffer_rsrc_t ksrc = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<u16*>(kbase + tile_step * jt), 0, nrec, kBufferFlags);
      const __amdgpu_buffer_rsrc_t vsrc = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<u16*>(vbase + tile_step * jt), 0, nrec, kBufferFlags);
#pragma unroll
      for (int i = 0; i < kLoadsPerWave; ++i) {
        const int off = static_cast<int>(lrow[i] * row_bytes) + lslot[i] * 16;
        const int lds_off = 1024 * (wv * kLoadsPerWave + i);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ksrc, (lds_void*)(kl + lds_off), 16, off, 0, 0, 0);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(vsrc, (lds_void*)(vl + lds_off), 16, off, 0, 0, 0);
      }
    } else {
      // 64-bit addresses; rows past the segment's end re-read its last row
      // (those keys are masked, and their probabilities are zero).
#pragma unroll
      for (int i = 0; i < kLoadsPerWave; ++i) {
        const int64_t row = min(k0 + lrow[i], L - 1);
        const int64_t off = row * row_step + lslot[i] * 8;
        const int lds_off = 1024 * (wv * kLoadsPerWave + i);
        __builtin_amdgcn_global_load_lds(kbase + off, (lds_void*)(kl + lds_off), 16, 0, 0);
        __builtin_amdgcn_global_load_lds(vbase + off, (lds_void*)(vl + lds_off), 16, 0, 0);
      }
    }
  };

  const int kv_end = a.causal ? qend : L;
  const int ntile = (kv_end + BN - 1) / BN;
  const int wq_lo = q0 + wv * 32;  // smallest query of this wave
  const int lim = a.causal ? min(tq_row, L - 1) : L - 1;  // last visible key of this lane
  // Lane roles in the transposed V reads (ds_read_b64_tr_b16): within each
  // 16-lane group, lane 4r + cb supplies the address of key row r, head-dim
  // columns 4cb..4cb+3, and receives one column across the four rows.
  const int tr_r = (lane & 15) >> 2;
  const int tr_d = ((lane >> 4) & 1) * 16 + (lane & 3) * 4;
  int vtr_off[DB][2];  // byte offset of this lane's address in key rows 0..15
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int d = db * 32 + tr_d;
      vtr_off[db][t] = TL::offset(8 * t + 4 * hi + tr_r, d >> 3) + (d & 7) * 2;
    }

  load_tile(0, 0);
  // Q enters the MFMA exactly as given (bf16): the softmax scale is applied to
  // the fp32 scores, so no second rounding of q enters them.
  bf16x8 qreg[KC];
#pragma unroll
  for (int c = 0; c < KC; ++c) {
    const u32x4 x = q_valid ? qraw[c] : u32x4{0u, 0u, 0u, 0u};
    qreg[c] = __builtin_bit_cast(bf16x8, x);
  }
  if (tid == 0) sm.redo = 0;

  f32x16 acc_o[DB];
  float m_run, l_run;  // reference max (log2 units) and this half-wave's share of the denominator
  bool safe = false;   // safe mode: a row max for every tile
  for (;;) {
#pragma unroll
  for (int db = 0; db < DB; ++db) acc_o[db] = f32x16{};
  m_run = 0.0f;
  l_run = 0.0f;
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  __syncthreads();
  for (int jt = 0; jt < ntile; ++jt) {
    const int cur = jt & 1;
    const int k0 = jt * BN;
    const bool more = jt + 1 < ntile;
    if (more) load_tile(jt + 1, cur ^ 1);
    const char* kl = reinterpret_cast<const char*>(&sm.k[cur][0]);
    const char* vl = reinterpret_cast<const char*>(&sm.v[cur][0]);

    // Tiles entirely after this wave's queries are skipped (causal).
    if (!(a.causal && k0 > wq_lo + 31)) {
      // S^T = K Q^T (unscaled fp32 scores), one 32x32 block per 32 keys; the
      // K fragments of a group of QG blocks are requested from LDS before the
      // group's MFMAs.
      constexpr int QG = (D <= 64 ? SB : 1);
      f32x16 acc_s[SB];
#pragma unroll
      for (int kb0 = 0; kb0 < SB; kb0 += QG) {
        u32x4 kf[QG][KC];
#pragma unroll
        for (int g = 0; g < QG; ++g)
#pragma unroll
          for (int c = 0; c < KC; ++c)
            kf[g][c] = *reinterpret_cast<const u32x4*>(kl + TL::offset((kb0 + g) * 32 + qr, 2 * c + hi));
        __builtin_amdgcn_sched_barrier(0);  // keep the reads ahead of the MFMAs
#pragma unroll
        for (int g = 0; g < QG; ++g) {
          acc_s[kb0 + g] = f32x16{};
#pragma unroll
          for (int c = 0; c < KC; ++c)
            acc_s[kb0 + g] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kf[g][c]),
                                                                     qreg[c], acc_s[kb0 + g], 0, 0, 0);
        }
      }
      // Mask keys after the query (causal) and past the segment's end.
      if ((a.causal && k0 + BN - 1 > wq_lo) || k0 + BN > L) {
        int base = k0 + 4 * hi - lim;   // key - lim = base + offset(kb, j)
        // Opaque to the compiler, so that the compares are made here: hoisted
        // out of the loops (for the first tile) they become 32 lane masks held
        // in scalar registers, which spill.
        asm volatile("" : "+v"(base));
#pragma unroll
        for (int kb = 0; kb < SB; ++kb)
#pragma unroll
          for (int j = 0; j < 16; ++j)
            if (base + kb * 32 + 8 * (j >> 2) + (j & 3) > 0) acc_s[kb][j] = -INFINITY;
      }
      // The first tile (and every tile in the safe mode) takes the row max of
      // this lane's query, across both half-waves.
      if (jt == 0 || safe) {
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < SB; ++kb)
#pragma unroll
          for (int j = 0; j < 16; j += 2) mx = fmaxf(mx, fmaxf(acc_s[kb][j], acc_s[kb][j + 1]));
        mx = fmaxf(mx, other_half(mx)) * c - m_run;  // log2 units, relative to m_run
        // The first tile fixes the reference max; in the safe mode later tiles
        // move it only when some row of the wave would see probabilities above
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
        }
      }
      // P = exp2(c S - m); bf16 P feeds the PV MFMA.  Row sums are taken in
      // fp32 with plain adds (dot-product instructions would not issue while
      // other waves' MFMAs run).  The A operand V^T comes from the row-major V
      // tile through transposed LDS reads: for MFMA step (kb, kk) the lane's
      // eight keys are kb*32 + 16kk + 4hi + {0..3} and the same + 8, matching
      // the keys its half-wave holds in S^T.
      const float negm = -m_run;
      float lp[4];
      const uint32_t vaddr = lds_addr(vl);
      static_for<0, SB>([&](auto KB) {
        constexpr int kb = decltype(KB)::value;
        // vf[kk][db][t]: V^T elements of head-dim block db for keys
        // kb*32 + 16kk + 8t + 4hi + {0..3} (half t of MFMA step kk's A operand).
        u32x2 vf[2][DB][2];
        static_for<0, 2>([&](auto KK) {
          static_for<0, DB>([&](auto DBI) {
            static_for<0, 2>([&](auto T) {
              constexpr int kk = decltype(KK)::value, db = decltype(DBI)::value, t = decltype(T)::value;
              constexpr int row = kb * 32 + 16 * kk;  // multiple of 16: same swizzle as rows 0..15
              vf[kk][db][t] = lds_read_tr16<row * TL::kRowBytes>(vaddr + vtr_off[db][t]);
            });
          });
        });
        static_for<0, 2>([&](auto KK) {
          constexpr int kk = decltype(KK)::value;
          bf16x8 pb;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float pe = __builtin_amdgcn_exp2f(__builtin_fmaf(acc_s[kb][8 * kk + e], c, negm));
            if (kb == 0 && kk == 0 && e < 4) lp[e] = pe;
            else lp[e & 3] += pe;
            pb[e] = (__bf16)pe;
          }
          lds_wait<(1 - kk) * 2 * DB>();  // step kk's reads done, the later step's may be pending
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            lds_bind(vf[kk][db][0]);
            lds_bind(vf[kk][db][1]);
            const u32x4 a4 = {vf[kk][db][0][0], vf[kk][db][0][1], vf[kk][db][1][0], vf[kk][db][1][1]};
            acc_o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a4), pb,
                                                                acc_o[db], 0, 0, 0);
          }
        });
      });
      const float lt = (lp[0] + lp[1]) + (lp[2] + lp[3]);
      l_run += lt;
      // Fast mode: move the reference max after the fact when this tile's
      // probabilities grew large (rare), or ask for a safe rerun when they
      // could have overflowed.
      if (!safe && __any(!(lt <= kSumSlack))) {
        if (__any(!(lt <= kSumLimit))) {
          sm.redo = 1;
        } else {
          const float lc = lt + other_half(lt);
          const float delta = lc > 1.0f ? __builtin_amdgcn_logf(lc) : 0.0f;  // log2
          const float alpha = __builtin_amdgcn_exp2f(-delta);
          m_run += delta;
          l_run *= alpha;
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int j = 0; j < 16; ++j) acc_o[db][j] *= alpha;
        }
      }
    }
    // The next tile's loads have landed in LDS and every wave is done with
    // this tile before anyone moves on.
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();
  }
  // A wave that saw a tile sum beyond kSumLimit makes the whole workgroup run
  // the item again (uniformly: the flag is read after the last barrier).
  if (safe || __builtin_amdgcn_readfirstlane(sm.redo) == 0) break;
  safe = true;
  __syncthreads();  // every wave has read the flag before the tiles are reloaded
  load_tile(0, 0);
  }

  // Epilogue: normalise this wave's 32 rows of the per-pattern output, scale
  // each row by its power of two and stage the fp16 rows in a private LDS
  // region (the tiles are no longer read: the loop ended with a barrier), so
  // that the stores write whole rows, 16 bytes per lane.  Staged 16-byte
  // chunk x of row k sits at chunk x ^ ((k >> 1) mod D/8): the 8-byte writes
  // (one row per lane) then hit at most two lanes per bank pair and the
  // 16-byte reads none.
  const float l_tot = l_run + other_half(l_run);
  const float inv = 1.0f / l_tot;
  float amax = 0.0f;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int j = 0; j < 16; ++j) amax = fmaxf(amax, fabsf(acc_o[db][j]));
  amax = fmaxf(amax, other_half(amax));
  float mul, rscale;
  row_scale(amax * inv, inv, mul, rscale);
  char* stg = reinterpret_cast<char*>(&sm.k[0][0]) + wv * 32 * TL::kRowBytes;
  auto stg_off = [&](int row, int chunk) {
    return row * TL::kRowBytes + ((chunk ^ ((row >> 1) & (TL::kSlots - 1))) << 4);
  };
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      f16x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = (_Float16)(acc_o[db][4 * jj + e] * mul);
      *reinterpret_cast<f16x4*>(stg + stg_off(qr, db * 4 + jj) + 8 * hi) = o;
    }
  const float lse_own = (m_run + __builtin_amdgcn_logf(l_tot)) * kLn2;
  // Each pass covers 64 consecutive 16-byte chunks: 1024 / (2 D) rows.
  constexpr int kPasses = 32 * TL::kRowBytes / 1024;
  if (hi == 0 && q_valid)
    reinterpret_cast<f32x2*>(a.ws + P.lse_off)[(int64_t)it.unit * P.lmax + tq_row] = f32x2{lse_own, rscale};
  _Float16* obase = reinterpret_cast<_Float16*>(a.ws + P.o_off) + ((int64_t)it.unit * P.lmax + wq_lo) * D;
#pragma unroll
  for (int i = 0; i < kPasses; ++i) {
    const int row = (i * 64 + lane) / TL::kSlots;
    const int chunk = (i * 64 + lane) % TL::kSlots;
    const u32x4 x = *reinterpret_cast<const u32x4*>(stg + stg_off(row, chunk));
    if (wq_lo + row < L) *reinterpret_cast<u32x4*>(obase + row * D + chunk * 8) = x;
  }
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
  // float32 rows need no scale: the record's scale is 1
  reinterpret_cast<f32x2*>(a.ws + P.lse_off)[wrow] = f32x2{(m_run + __builtin_amdgcn_logf(l_run)) * kLn2, 1.0f};
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
  a.causal = plan.causal;
  a.scale_log2 = plan.scale * kLog2e;
  // The patterns of the launch, most query tiles per unit first.
  int order[DA_MAX_PATTERNS];
  const int n = plan.npat;
  for (int i = 0; i < n; ++i) order[i] = i;
  std::stable_sort(order, order + n, [&](int x, int y) { return plan.pat[x].ntiles > plan.pat[y].ntiles; });
  a.npat = n;
  int64_t items = 0, launch = 0;
  for (int i = 0; i < DA_MAX_PATTERNS; ++i) {
    PatArgs& pa = a.pat[i];
    if (i < n) {
      const PatternPlan& pp = plan.pat[order[i]];
      pa.w = static_cast<int32_t>(pp.w);
      pa.r = static_cast<int32_t>(pp.r);
      pa.nseg = static_cast<int32_t>(pp.nseg);
      pa.lmax = static_cast<int32_t>(pp.lmax);
      pa.ntiles = static_cast<int32_t>(pp.ntiles);
      pa.units = static_cast<int32_t>(pp.units);
      pa.o_off = static_cast<int64_t>(pp.o_off);
      pa.lse_off = static_cast<int64_t>(pp.lse_off);
      items += pp.units * pp.ntiles;
      // XCD 0 holds the most units of every pattern; the launch covers 8 times its slots.
      launch += (pp.units + 7) / 8 * pp.ntiles * 8;
    } else {
      pa = PatArgs{1, 1, 1, 1, 1, 0, 0, 0};
    }
  }
  a.total_items = static_cast<int32_t>(items);
  if (items == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(launch));
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
