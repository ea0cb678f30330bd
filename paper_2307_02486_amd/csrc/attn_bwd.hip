// Backward of the dilated-attention forward pass on gfx950 (bf16, D = 32/64/128).
//
// The mixture of the patterns (Sec. 2.2, Eqs. 9-10) is one softmax over the
// multiset of (pattern, key) pairs a query sees (Sec. 2.2, after Eq. 10).  With
// the combined lse of the forward pass and delta = sum_d dout * out per row,
// the gradient splits into one softmax-attention derivative per pattern and
// sparsified segment (gathered rows as in the forward, Sec. 2.2 Eqs. 3-5 and
// the offsets of Sec. 2.3):
//   P = exp(scale q.k - lse),  dS = P (dout.v - delta),
//   dq += scale dS k,  dk += scale dS q,  dv += P dout.
// Scores are exact bf16 products q.k summed in fp32; the softmax scale is
// applied to the fp32 sum (P = exp2(scale log2(e) (q.k - lse / scale))), so q
// and k enter the MFMAs as given.
// Four kernels:
//   bwd_delta  per row: -delta and -lse/scale into the workspace;
//   bwd_dq     per (pattern, segment, 128-query tile): each lane owns a query;
//              over the segment's key tiles, S^T = K Q^T and (dP - delta)^T =
//              V dO^T start from -lse and -delta (no running max: lse is
//              known), and dQ^T += K^T dS^T;
//   bwd_dkdv   per (pattern, segment, 128-key tile): each lane owns a key;
//              over the query tiles that see it, S = Q K^T and dP - delta =
//              dO V^T, then dV^T += dO^T P and dK^T += Q^T dS;
//   bwd_sum    per row: the compact per-pattern gradients of every pattern
//              that keeps the row, summed and rounded to bf16.
// The compact per-pattern gradients are fp16 rows scaled by a power of two
// per row and 64-column chunk (row_scale), with the float scale beside them:
// an error of at most 2^-11 of the chunk's largest element before the sum.
// Tiles of the rows that are shared by a workgroup (K/V for dq, Q/dO for
// dk/dv) go from HBM into LDS without passing through registers; transposed
// operands come from transposed LDS reads.  Work items are mapped to XCDs as
// in the forward pass.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "device_common.h"

namespace da {
namespace {

struct BwdPat {
  int32_t w, r, nseg, lmax, ntiles, units;
  int64_t dq_off, dk_off, dv_off;           // byte offsets of the compact fp16 gradient rows
  int64_t dq_rec_off, dk_rec_off, dv_rec_off;  // and of their float scales
};

struct BwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* dout;
  const float* nl2;  // -lse / scale, [B][H][N]: the score offset before the scale
  const float* nd;   // -delta, [B][H][N]
  char* ws;
  int32_t B, N, H, npat, causal;
  float scale_log2;  // softmax scale * log2(e)
  float scale;
  BwdPat pat[DA_MAX_PATTERNS];  // by query tiles per unit, most first
};

constexpr int kThreadsB = 256;  // four waves
// Head-dim columns of dq (or dk, dv) one work item accumulates: all of them up
// to D = 64; at D = 128 each item is run twice, once per 64-column half (the
// scores and dP are recomputed, the accumulators fit in registers).
template <int D>
constexpr int kCols = D <= 64 ? D : 64;
// Scales per compact gradient row: one per item's column range.
template <int D>
constexpr int kChunks = D / kCols<D>;
// Launch index of a split work item: the two halves of an item take two
// consecutive slots of the same XCD.  Returns the item's launch index and sets
// `half`.
template <int D>
__device__ inline int split_index(int bid, int& half) {
  if constexpr (kCols<D> == D) {
    half = 0;
    return bid;
  } else {
    half = (bid >> 3) & 1;
    return ((bid >> 4) << 3) | (bid & 7);
  }
}
constexpr int kTileB = 128;     // rows (queries for dq, keys for dk/dv) per work item
constexpr int kStepB = 64;      // rows per LDS tile of the other operand

template <int D>
struct SmemTiles {
  __attribute__((aligned(16))) u16 a[2][kStepB * D];  // K (dq) or Q (dk/dv) tiles
  __attribute__((aligned(16))) u16 b[2][kStepB * D];  // V (dq) or dO (dk/dv) tiles
  __attribute__((aligned(16))) float s0[2][kStepB];   // -lse*log2(e) of the query rows (dk/dv)
  __attribute__((aligned(16))) float s1[2][kStepB];   // -delta of the query rows (dk/dv)
};

// bf16 row slice [16c + 8hi, +8) of a row, as the MFMA operand layout wants,
// optionally multiplied by `mul` and rounded back to bf16.
template <int KC>
__device__ inline void load_rowslices(const u16* row, int hi, float mul, bool zero, bf16x8 (&out)[KC]) {
  u32x4 raw[KC];
#pragma unroll
  for (int c = 0; c < KC; ++c) raw[c] = *reinterpret_cast<const u32x4*>(row + 16 * c + 8 * hi);
#pragma unroll
  for (int c = 0; c < KC; ++c)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const unsigned bits = zero ? 0u : (raw[c][e >> 1] >> (16 * (e & 1))) << 16;
      out[c][e] = (__bf16)(__builtin_bit_cast(float, bits) * mul);
    }
}

// Loads of one tile of kStepB kept rows (row stride row_step elements, base at
// the tile's first row, `valid` rows before the segment's end) straight into
// LDS: load i of wave wv fills 16-byte LDS slots [64 (wv*kLoads + i), +64).
template <int D>
struct TileLoader {
  using TL = TileLayout<D>;
  static constexpr int kLoads = kStepB * TL::kSlots / 64 / (kThreadsB / 64);
  int lrow[kLoads], lslot[kLoads];
  __device__ void init(int wv, int lane) {
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      const int s = 64 * (wv * kLoads + i) + lane;
      lrow[i] = s / TL::kSlots;
      lslot[i] = (s % TL::kSlots) ^ TL::swz(lrow[i]);
    }
  }
  __device__ void load(const u16* base, int64_t row_step, int valid, char* dst, int wv) const {
    const uint64_t row_bytes = static_cast<uint64_t>(row_step) * 2;
    const uint64_t vb = static_cast<uint64_t>(valid > 0 ? valid : 0) * row_bytes;
    const int nrec = static_cast<int>(vb < 0x7fffffffull ? vb : 0x7fffffffull);
    const __amdgpu_buffer_rsrc_t src = __builtin_amdgcn_make_buffer_rsrc(const_cast<u16*>(base), 0, nrec,
                                                                         kBufferFlags);
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      const int off = static_cast<int>(lrow[i] * row_bytes) + lslot[i] * 16;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (lds_void*)(dst + 1024 * (wv * kLoads + i)), 16, off, 0,
                                               0, 0);
    }
  }
};

// ---------------------------------------------------------------------------
// bwd_delta: -delta = -sum_d dout*out and -lse/scale, per (b, h, p).
// ---------------------------------------------------------------------------
struct DeltaArgs {
  const u16* out;
  const u16* dout;
  const float* lse;
  float* nl2;
  float* nd;
  float inv_scale;
  int32_t N, H, chunks;
};

template <int D>
__global__ __launch_bounds__(kThreadsB) void bwd_delta(DeltaArgs a) {
  constexpr int LPR = D / 8;           // lanes per row
  constexpr int RPB = kThreadsB / LPR; // rows per workgroup
  const int tid = __builtin_amdgcn_workitem_id_x();
  const int blk = __builtin_amdgcn_workgroup_id_x();
  // heads innermost, as in bwd_sum: the out and dout rows read together are adjacent
  const int h = blk % a.H;
  const int rest = blk / a.H;
  const int chunk = rest % a.chunks;
  const int b = rest / a.chunks;
  const int bh = b * a.H + h;
  const int p = chunk * RPB + tid / LPR;
  const int d0 = (tid % LPR) * 8;
  const bool ok = p < a.N;
  const int pp = ok ? p : a.N - 1;
  const int64_t off = (((int64_t)b * a.N + pp) * a.H + h) * D + d0;
  const u32x4 o = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(a.out + off));
  const u32x4 g = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(a.dout + off));
  float acc = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float x = __builtin_bit_cast(float, (o[e >> 1] >> (16 * (e & 1))) << 16);
    const float y = __builtin_bit_cast(float, (g[e >> 1] >> (16 * (e & 1))) << 16);
    acc += x * y;
  }
  // sum over the LPR lanes of the row (consecutive lanes, LPR a power of two)
#pragma unroll
  for (int m = 1; m < LPR; m <<= 1) acc += __shfl_xor(acc, m, 64);
  if (ok && d0 == 0) {
    const int64_t o2 = (int64_t)bh * a.N + p;
    a.nd[o2] = -acc;
    a.nl2[o2] = -a.lse[o2] * a.inv_scale;
  }
}

// ---------------------------------------------------------------------------
// bwd_dq: one work item = 128 query rows of one sparsified segment.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kThreadsB) void bwd_dq(BwdArgs a) {
  constexpr int BN = kStepB;
  constexpr int KC = D / 16, DB = kCols<D> / 32, SB = BN / 32;
  using TL = TileLayout<D>;
  __shared__ SmemTiles<D> sm;

  Item it;
  int half;
  const int bid = split_index<D>(__builtin_amdgcn_workgroup_id_x(), half);
  const int c0 = half * kCols<D>;  // first head-dim column this item accumulates
  if (!decode_item(a, bid, kTileB, it)) return;
  const BwdPat& P = a.pat[it.pi];
  const int tid = __builtin_amdgcn_workitem_id_x();
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qr = lane & 31, hi = lane >> 5;
  const int L = it.L;
  const int q0 = it.tq * kTileB;
  const int qend = min(q0 + kTileB, L);
  const int wq_lo = q0 + wv * 32;
  const int tq_row = wq_lo + qr;
  const bool q_valid = tq_row < L;
  const int qrow = min(tq_row, L - 1);
  const int64_t row_step = it.rstride * D;

  TileLoader<D> ld;
  ld.init(wv, lane);
  const u16* kbase = static_cast<const u16*>(a.k) + it.row0 * D;
  const u16* vbase = static_cast<const u16*>(a.v) + it.row0 * D;
  auto load_tile = [&](int jt, int buf) {
    const int64_t o = row_step * BN * jt;
    ld.load(kbase + o, row_step, L - jt * BN, reinterpret_cast<char*>(&sm.a[buf][0]), wv);
    ld.load(vbase + o, row_step, L - jt * BN, reinterpret_cast<char*>(&sm.b[buf][0]), wv);
  };
  load_tile(0, 0);

  // Q^T (times scale*log2e) and dO^T operands of this lane's query, its
  // -lse*log2e and -delta.
  const int64_t qoff = (it.row0 + (int64_t)qrow * it.rstride) * D;
  bf16x8 qreg[KC], doreg[KC];
  load_rowslices<KC>(static_cast<const u16*>(a.q) + qoff, hi, 1.0f, !q_valid, qreg);
  load_rowslices<KC>(static_cast<const u16*>(a.dout) + qoff, hi, 1.0f, !q_valid, doreg);
  const int64_t srow = ((int64_t)it.b * a.H + it.h) * a.N + it.p0 + (int64_t)qrow * P.r;
  const float nl2 = a.nl2[srow], nd = a.nd[srow];
  f32x16 vnl2, vnd;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    vnl2[j] = nl2;
    vnd[j] = nd;
  }
  f32x16 acc_dq[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc_dq[db] = f32x16{};

  const int kv_end = a.causal ? qend : L;
  const int ntile = (kv_end + BN - 1) / BN;
  const int lim = a.causal ? qrow : L - 1;  // last visible key of this lane
  const int tr_r = (lane & 15) >> 2;
  const int tr_d = ((lane >> 4) & 1) * 16 + (lane & 3) * 4;
  int vtr_off[DB][2];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int d = c0 + db * 32 + tr_d;
      vtr_off[db][t] = TL::offset(8 * t + 4 * hi + tr_r, d >> 3) + (d & 7) * 2;
    }

  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  __syncthreads();
  for (int jt = 0; jt < ntile; ++jt) {
    const int cur = jt & 1;
    const int k0 = jt * BN;
    if (jt + 1 < ntile) load_tile(jt + 1, cur ^ 1);
    const char* kl = reinterpret_cast<const char*>(&sm.a[cur][0]);
    const char* vl = reinterpret_cast<const char*>(&sm.b[cur][0]);
    if (!(a.causal && k0 > wq_lo + 31)) {
      const bool masked = (a.causal && k0 + BN - 1 > wq_lo) || k0 + BN > L;
      const uint32_t kaddr = lds_addr(kl);
      static_for<0, SB>([&](auto KB) {
        constexpr int kb = decltype(KB)::value;
        // S'^T = K Q^T - lse/scale and (dP - delta)^T = V dO^T - delta
        u32x4 kf[KC], vf[KC];
#pragma unroll
        for (int c = 0; c < KC; ++c) {
          kf[c] = *reinterpret_cast<const u32x4*>(kl + TL::offset(kb * 32 + qr, 2 * c + hi));
          vf[c] = *reinterpret_cast<const u32x4*>(vl + TL::offset(kb * 32 + qr, 2 * c + hi));
        }
        f32x16 s = vnl2, dp = vnd;
#pragma unroll
        for (int c = 0; c < KC; ++c) {
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kf[c]), qreg[c], s, 0, 0, 0);
          dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vf[c]), doreg[c], dp, 0, 0, 0);
        }
        if (masked) {
          const int base = k0 + kb * 32 + 4 * hi - lim;
#pragma unroll
          for (int j = 0; j < 16; ++j)
            if (base + 8 * (j >> 2) + (j & 3) > 0) s[j] = -INFINITY;
        }
        // dS^T = P^T (dP - delta)^T as the bf16 B operand of dQ^T += K^T dS^T
        bf16x8 dsb[2];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int e = 0; e < 8; ++e)
            dsb[kk][e] = (__bf16)(__builtin_amdgcn_exp2f(s[8 * kk + e] * a.scale_log2) * dp[8 * kk + e]);
        // K^T fragments through transposed reads (keys kb*32 + 16kk + 8t + 4hi + {0..3})
        u32x2 kt[2][DB][2];
        static_for<0, 2>([&](auto KK) {
          static_for<0, DB>([&](auto DBI) {
            static_for<0, 2>([&](auto T) {
              constexpr int kk = decltype(KK)::value, db = decltype(DBI)::value, t = decltype(T)::value;
              kt[kk][db][t] = lds_read_tr16<(kb * 32 + 16 * kk) * TL::kRowBytes>(kaddr + vtr_off[db][t]);
            });
          });
        });
        lds_wait<0>();
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            lds_bind(kt[kk][db][0]);
            lds_bind(kt[kk][db][1]);
            const u32x4 a4 = {kt[kk][db][0][0], kt[kk][db][0][1], kt[kk][db][1][0], kt[kk][db][1][1]};
            acc_dq[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a4), dsb[kk],
                                                                 acc_dq[db], 0, 0, 0);
          }
      });
    }
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();
  }

  // dq = scale * acc over this item's columns, stored scaled (both half-waves
  // hold parts of the row: the max is exchanged before any lane leaves).
  float amax = 0.0f;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int j = 0; j < 16; ++j) amax = fmaxf(amax, fabsf(acc_dq[db][j]));
  amax = fmaxf(amax, other_half(amax));
  if (!q_valid) return;
  float mul, rs;
  row_scale(amax * a.scale, a.scale, mul, rs);
  const int64_t wrow = (int64_t)it.unit * P.lmax + tq_row;
  _Float16* orow = reinterpret_cast<_Float16*>(a.ws + P.dq_off) + wrow * D;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
      *reinterpret_cast<f16x4*>(orow + c0 + db * 32 + 8 * jj + 4 * hi) =
          f16x4{(_Float16)(acc_dq[db][4 * jj] * mul), (_Float16)(acc_dq[db][4 * jj + 1] * mul),
                (_Float16)(acc_dq[db][4 * jj + 2] * mul), (_Float16)(acc_dq[db][4 * jj + 3] * mul)};
  if (hi == 0) reinterpret_cast<float*>(a.ws + P.dq_rec_off)[wrow * kChunks<D> + half] = rs;
}

// ---------------------------------------------------------------------------
// bwd_dkdv: one work item = 128 key rows of one sparsified segment.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kThreadsB) void bwd_dkdv(BwdArgs a) {
  constexpr int BQ = kStepB;
  constexpr int KC = D / 16, DB = kCols<D> / 32, QB = BQ / 32;
  using TL = TileLayout<D>;
  __shared__ SmemTiles<D> sm;

  Item it;
  int half;
  const int bid = split_index<D>(__builtin_amdgcn_workgroup_id_x(), half);
  const int c0 = half * kCols<D>;  // first head-dim column this item accumulates
  if (!decode_item(a, bid, 0, it)) return;
  const BwdPat& P = a.pat[it.pi];
  const int kt_idx = P.ntiles - 1 - it.tq;  // longest (first) key tiles first
  const int L = it.L;
  const int kt0 = kt_idx * kTileB;
  if (kt0 >= L) return;
  const int tid = __builtin_amdgcn_workitem_id_x();
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kr = lane & 31, hi = lane >> 5;
  const int kw0 = kt0 + wv * 32;  // this wave's first key
  const int tk_row = kw0 + kr;
  const bool k_valid = tk_row < L;
  const int krow = min(tk_row, L - 1);
  const int64_t row_step = it.rstride * D;

  TileLoader<D> ld;
  ld.init(wv, lane);
  const u16* qbase = static_cast<const u16*>(a.q) + it.row0 * D;
  const u16* obase = static_cast<const u16*>(a.dout) + it.row0 * D;
  const int64_t sbase = ((int64_t)it.b * a.H + it.h) * a.N + it.p0;
  // Query tiles: every tile holding a query at or after the first key (causal).
  const int qt_first = a.causal ? kt0 / BQ : 0;
  const int qt_end = (L + BQ - 1) / BQ;
  auto load_tile = [&](int qt, int buf) {
    const int64_t o = row_step * BQ * qt;
    ld.load(qbase + o, row_step, L - qt * BQ, reinterpret_cast<char*>(&sm.a[buf][0]), wv);
    ld.load(obase + o, row_step, L - qt * BQ, reinterpret_cast<char*>(&sm.b[buf][0]), wv);
    if (wv < 2) {
      // the 64 query rows' scalars: one 4-byte load per lane, rows r apart
      const float* src = (wv == 0 ? a.nl2 : a.nd) + sbase + (int64_t)qt * BQ * P.r;
      const int valid = L - qt * BQ;
      const uint64_t vb = static_cast<uint64_t>(valid > 0 ? (valid - 1) * P.r + 1 : 0) * 4;
      const int nrec = static_cast<int>(vb < 0x7fffffffull ? vb : 0x7fffffffull);
      const __amdgpu_buffer_rsrc_t rs =
          __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(src), 0, nrec, kBufferFlags);
      float* dst = wv == 0 ? &sm.s0[buf][0] : &sm.s1[buf][0];
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)dst, 4, lane * P.r * 4, 0, 0, 0);
    }
  };
  if (qt_first < qt_end) load_tile(qt_first, 0);

  // K^T and V^T operands of this lane's key (as given).
  const int64_t koff = (it.row0 + (int64_t)krow * it.rstride) * D;
  bf16x8 kreg[KC], vreg[KC];
  load_rowslices<KC>(static_cast<const u16*>(a.k) + koff, hi, 1.0f, !k_valid, kreg);
  load_rowslices<KC>(static_cast<const u16*>(a.v) + koff, hi, 1.0f, !k_valid, vreg);
  f32x16 acc_dk[DB], acc_dv[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc_dk[db] = acc_dv[db] = f32x16{};
  const int tr_r = (lane & 15) >> 2;
  const int tr_d = ((lane >> 4) & 1) * 16 + (lane & 3) * 4;
  int vtr_off[DB][2];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int d = c0 + db * 32 + tr_d;
      vtr_off[db][t] = TL::offset(8 * t + 4 * hi + tr_r, d >> 3) + (d & 7) * 2;
    }

  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  __syncthreads();
  for (int qt = qt_first; qt < qt_end; ++qt) {
    const int cur = (qt - qt_first) & 1;
    const int q0 = qt * BQ;
    if (qt + 1 < qt_end) load_tile(qt + 1, cur ^ 1);
    const char* ql = reinterpret_cast<const char*>(&sm.a[cur][0]);
    const char* ol = reinterpret_cast<const char*>(&sm.b[cur][0]);
    const float* nl2t = &sm.s0[cur][0];
    const float* ndt = &sm.s1[cur][0];
    // Tiles entirely before this wave's keys are skipped (causal).
    if (!(a.causal && q0 + BQ - 1 < kw0)) {
      const bool masked = (a.causal && q0 < kw0 + 31) || q0 + BQ > L;
      const uint32_t qaddr = lds_addr(ql), oaddr = lds_addr(ol);
      static_for<0, QB>([&](auto QBI) {
        constexpr int qb = decltype(QBI)::value;
        // C layout of S[q][key]: this lane's key, queries qb*32 + 8(j/4) + 4hi + j%4.
        f32x16 s, dp;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const f32x4 x = *reinterpret_cast<const f32x4*>(nl2t + qb * 32 + 8 * i + 4 * hi);
          const f32x4 y = *reinterpret_cast<const f32x4*>(ndt + qb * 32 + 8 * i + 4 * hi);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            s[4 * i + e] = x[e];
            dp[4 * i + e] = y[e];
          }
        }
        u32x4 qf[KC], of[KC];
#pragma unroll
        for (int c = 0; c < KC; ++c) {
          qf[c] = *reinterpret_cast<const u32x4*>(ql + TL::offset(qb * 32 + kr, 2 * c + hi));
          of[c] = *reinterpret_cast<const u32x4*>(ol + TL::offset(qb * 32 + kr, 2 * c + hi));
        }
#pragma unroll
        for (int c = 0; c < KC; ++c) {
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, qf[c]), kreg[c], s, 0, 0, 0);
          dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, of[c]), vreg[c], dp, 0, 0, 0);
        }
        if (masked) {
          // masked: queries before the key (causal) and past the segment's end
          const int qbase = q0 + qb * 32 + 4 * hi;
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int qj = qbase + 8 * (j >> 2) + (j & 3);
            if ((a.causal && qj < tk_row) || qj >= L) s[j] = -INFINITY;
          }
        }
        bf16x8 pb[2], dsb[2];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float p = __builtin_amdgcn_exp2f(s[8 * kk + e] * a.scale_log2);
            pb[kk][e] = (__bf16)p;
            dsb[kk][e] = (__bf16)(p * dp[8 * kk + e]);
          }
        // dO^T and Q^T fragments through transposed reads (queries
        // qb*32 + 16kk + 8t + 4hi + {0..3}, matching the B operands above).
        u32x2 ot[2][DB][2], qtr[2][DB][2];
        static_for<0, 2>([&](auto KK) {
          static_for<0, DB>([&](auto DBI) {
            static_for<0, 2>([&](auto T) {
              constexpr int kk = decltype(KK)::value, db = decltype(DBI)::value, t = decltype(T)::value;
              constexpr int off = (qb * 32 + 16 * kk) * TL::kRowBytes;
              ot[kk][db][t] = lds_read_tr16<off>(oaddr + vtr_off[db][t]);
              qtr[kk][db][t] = lds_read_tr16<off>(qaddr + vtr_off[db][t]);
            });
          });
        });
        lds_wait<0>();
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            lds_bind(ot[kk][db][0]);
            lds_bind(ot[kk][db][1]);
            lds_bind(qtr[kk][db][0]);
            lds_bind(qtr[kk][db][1]);
            const u32x4 ao = {ot[kk][db][0][0], ot[kk][db][0][1], ot[kk][db][1][0], ot[kk][db][1][1]};
            const u32x4 aq = {qtr[kk][db][0][0], qtr[kk][db][0][1], qtr[kk][db][1][0], qtr[kk][db][1][1]};
            acc_dv[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, ao), pb[kk],
                                                                 acc_dv[db], 0, 0, 0);
            acc_dk[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, aq), dsb[kk],
                                                                 acc_dk[db], 0, 0, 0);
          }
      });
    }
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();
  }

  // dk = scale * acc_dk and dv = acc_dv over this item's columns, stored
  // scaled (the row maxima are exchanged before any lane leaves).
  float amax_k = 0.0f, amax_v = 0.0f;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      amax_k = fmaxf(amax_k, fabsf(acc_dk[db][j]));
      amax_v = fmaxf(amax_v, fabsf(acc_dv[db][j]));
    }
  amax_k = fmaxf(amax_k, other_half(amax_k));
  amax_v = fmaxf(amax_v, other_half(amax_v));
  if (!k_valid) return;
  float mul_k, rs_k, mul_v, rs_v;
  row_scale(amax_k * a.scale, a.scale, mul_k, rs_k);
  row_scale(amax_v, 1.0f, mul_v, rs_v);
  const int64_t wrow = (int64_t)it.unit * P.lmax + tk_row;
  _Float16* krow_out = reinterpret_cast<_Float16*>(a.ws + P.dk_off) + wrow * D;
  _Float16* vrow_out = reinterpret_cast<_Float16*>(a.ws + P.dv_off) + wrow * D;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int d = c0 + db * 32 + 8 * jj + 4 * hi;
      *reinterpret_cast<f16x4*>(krow_out + d) =
          f16x4{(_Float16)(acc_dk[db][4 * jj] * mul_k), (_Float16)(acc_dk[db][4 * jj + 1] * mul_k),
                (_Float16)(acc_dk[db][4 * jj + 2] * mul_k), (_Float16)(acc_dk[db][4 * jj + 3] * mul_k)};
      *reinterpret_cast<f16x4*>(vrow_out + d) =
          f16x4{(_Float16)(acc_dv[db][4 * jj] * mul_v), (_Float16)(acc_dv[db][4 * jj + 1] * mul_v),
                (_Float16)(acc_dv[db][4 * jj + 2] * mul_v), (_Float16)(acc_dv[db][4 * jj + 3] * mul_v)};
    }
  if (hi == 0) {
    reinterpret_cast<float*>(a.ws + P.dk_rec_off)[wrow * kChunks<D> + half] = rs_k;
    reinterpret_cast<float*>(a.ws + P.dv_rec_off)[wrow * kChunks<D> + half] = rs_v;
  }
}

// ---------------------------------------------------------------------------
// bwd_sum: dq, dk, dv of each (b, p, h) = the sum over the patterns keeping p
// of their compact rows, rounded to bf16; rows kept by no pattern get 0.
// ---------------------------------------------------------------------------
struct SumPat {
  FastDiv fw, fr;
  int32_t nseg, lmax;
  int64_t dq_off, dk_off, dv_off;
  int64_t dq_rec_off, dk_rec_off, dv_rec_off;
};

struct SumArgs {
  const char* ws;
  u16* dq;
  u16* dk;
  u16* dv;
  int32_t N, H, npat, chunks;
  SumPat pat[DA_MAX_PATTERNS];
};

__device__ inline void store_bf16x8(u16* p, const f32x8& v) {
  bf16x8 b;
#pragma unroll
  for (int e = 0; e < 8; ++e) b[e] = (__bf16)v[e];
  __builtin_nontemporal_store(b, reinterpret_cast<bf16x8*>(p));
}

// Eight elements of a compact gradient row, times the row chunk's scale.
__device__ inline f32x8 load_scaled(const char* ws, int64_t off, int64_t rec_off, int64_t row, int64_t rec,
                                    int d0) {
  const f16x8 h = *reinterpret_cast<const f16x8*>(reinterpret_cast<const _Float16*>(ws + off) + row + d0);
  const float sc = reinterpret_cast<const float*>(ws + rec_off)[rec];
  f32x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = static_cast<float>(h[e]) * sc;
  return r;
}

template <int D>
__global__ __launch_bounds__(kThreadsB) void bwd_sum(SumArgs a) {
  constexpr int LPR = D / 8;
  constexpr int RPB = kThreadsB / LPR;
  const int tid = __builtin_amdgcn_workitem_id_x();
  const int blk = __builtin_amdgcn_workgroup_id_x();
  // heads innermost (launch index = (b * chunks + chunk) * H + h), as in the
  // forward combine: workgroups running together write whole [H][D] spans
  const int h = blk % a.H;
  const int rest = blk / a.H;
  const int chunk = rest % a.chunks;
  const int b = rest / a.chunks;
  const int bh = b * a.H + h;
  const int p = chunk * RPB + tid / LPR;
  const int d0 = (tid % LPR) * 8;
  if (p >= a.N) return;
  f32x8 sq = f32x8{0, 0, 0, 0, 0, 0, 0, 0}, sk = sq, sv = sq;
  for (int i = 0; i < a.npat; ++i) {
    const SumPat& P = a.pat[i];
    const uint32_t g = P.fw.div(static_cast<uint32_t>(p));
    const uint32_t pos = static_cast<uint32_t>(p) - g * P.fw.d;
    const uint32_t t = P.fr.div(pos);
    const uint32_t s = static_cast<uint32_t>(h) - P.fr.div(static_cast<uint32_t>(h)) * P.fr.d;
    if (pos - t * P.fr.d != s) continue;
    const int64_t crow = ((int64_t)bh * P.nseg + g) * P.lmax + t;
    const int64_t rec = crow * kChunks<D> + (d0 / kCols<D>);
    sq += load_scaled(a.ws, P.dq_off, P.dq_rec_off, crow * D, rec, d0);
    sk += load_scaled(a.ws, P.dk_off, P.dk_rec_off, crow * D, rec, d0);
    sv += load_scaled(a.ws, P.dv_off, P.dv_rec_off, crow * D, rec, d0);
  }
  const int64_t o = (((int64_t)b * a.N + p) * a.H + h) * D + d0;
  store_bf16x8(a.dq + o, sq);
  store_bf16x8(a.dk + o, sk);
  store_bf16x8(a.dv + o, sv);
}

}  // namespace

hipError_t launch_backward(const Plan& plan, const BwdLayout& lay, const void* q, const void* k, const void* v,
                           const void* out, const float* lse, const void* dout, void* dq, void* dk, void* dv,
                           void* workspace, hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  const int rpb = kThreadsB / (static_cast<int>(plan.D) / 8);
  const int chunks = static_cast<int>((plan.N + rpb - 1) / rpb);
  const int64_t rblocks = static_cast<int64_t>(chunks) * plan.B * plan.H;
  if (rblocks >= (int64_t{1} << 31)) return hipErrorInvalidValue;

  DeltaArgs da_;
  da_.out = static_cast<const u16*>(out);
  da_.dout = static_cast<const u16*>(dout);
  da_.lse = lse;
  da_.nl2 = reinterpret_cast<float*>(ws + lay.nl2_off);
  da_.nd = reinterpret_cast<float*>(ws + lay.nd_off);
  da_.inv_scale = 1.0f / plan.scale;
  da_.N = static_cast<int32_t>(plan.N);
  da_.H = static_cast<int32_t>(plan.H);
  da_.chunks = chunks;

  BwdArgs a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.dout = dout;
  a.nl2 = da_.nl2;
  a.nd = da_.nd;
  a.ws = ws;
  a.B = static_cast<int32_t>(plan.B);
  a.N = static_cast<int32_t>(plan.N);
  a.H = static_cast<int32_t>(plan.H);
  a.npat = plan.npat;
  a.causal = plan.causal;
  a.scale = plan.scale;
  a.scale_log2 = plan.scale * kLog2e;
  int order[DA_MAX_PATTERNS];
  for (int i = 0; i < plan.npat; ++i) order[i] = i;
  std::stable_sort(order, order + plan.npat,
                   [&](int x, int y) { return plan.pat[x].ntiles > plan.pat[y].ntiles; });
  SumArgs sa;
  sa.ws = ws;
  sa.dq = static_cast<u16*>(dq);
  sa.dk = static_cast<u16*>(dk);
  sa.dv = static_cast<u16*>(dv);
  sa.N = a.N;
  sa.H = a.H;
  sa.npat = plan.npat;
  sa.chunks = chunks;
  for (int i = 0; i < DA_MAX_PATTERNS; ++i) {
    BwdPat& bp = a.pat[i];
    SumPat& sp = sa.pat[i];
    if (i < plan.npat) {
      const int j = order[i];
      const PatternPlan& pp = plan.pat[j];
      bp = BwdPat{static_cast<int32_t>(pp.w), static_cast<int32_t>(pp.r), static_cast<int32_t>(pp.nseg),
                  static_cast<int32_t>(pp.lmax), static_cast<int32_t>(pp.ntiles), static_cast<int32_t>(pp.units),
                  static_cast<int64_t>(lay.dq_off[j]), static_cast<int64_t>(lay.dk_off[j]),
                  static_cast<int64_t>(lay.dv_off[j]), static_cast<int64_t>(lay.dq_rec_off[j]),
                  static_cast<int64_t>(lay.dk_rec_off[j]), static_cast<int64_t>(lay.dv_rec_off[j])};
      sp = SumPat{make_fastdiv(static_cast<uint32_t>(pp.w)), make_fastdiv(static_cast<uint32_t>(pp.r)),
                  static_cast<int32_t>(pp.nseg), static_cast<int32_t>(pp.lmax),
                  static_cast<int64_t>(lay.dq_off[j]), static_cast<int64_t>(lay.dk_off[j]),
                  static_cast<int64_t>(lay.dv_off[j]), static_cast<int64_t>(lay.dq_rec_off[j]),
                  static_cast<int64_t>(lay.dk_rec_off[j]), static_cast<int64_t>(lay.dv_rec_off[j])};
    } else {
      bp = BwdPat{1, 1, 1, 1, 1, 0, 0, 0, 0, 0, 0, 0};
      sp = SumPat{make_fastdiv(1), make_fastdiv(1), 1, 1, 0, 0, 0, 0, 0, 0};
    }
  }
  const dim3 rgrid(static_cast<unsigned>(rblocks));
  const dim3 igrid(static_cast<unsigned>(plan.launch_items));
  if (2 * plan.launch_items >= (int64_t{1} << 31)) return hipErrorInvalidValue;
  switch (plan.D) {
    case 32:
      hipLaunchKernelGGL(bwd_delta<32>, rgrid, dim3(kThreadsB), 0, stream, da_);
      if (plan.total_items > 0) {
        hipLaunchKernelGGL(bwd_dq<32>, igrid, dim3(kThreadsB), 0, stream, a);
        hipLaunchKernelGGL(bwd_dkdv<32>, igrid, dim3(kThreadsB), 0, stream, a);
      }
      hipLaunchKernelGGL(bwd_sum<32>, rgrid, dim3(kThreadsB), 0, stream, sa);
      break;
    case 64:
      hipLaunchKernelGGL(bwd_delta<64>, rgrid, dim3(kThreadsB), 0, stream, da_);
      if (plan.total_items > 0) {
        hipLaunchKernelGGL(bwd_dq<64>, igrid, dim3(kThreadsB), 0, stream, a);
        hipLaunchKernelGGL(bwd_dkdv<64>, igrid, dim3(kThreadsB), 0, stream, a);
      }
      hipLaunchKernelGGL(bwd_sum<64>, rgrid, dim3(kThreadsB), 0, stream, sa);
      break;
    case 128: {
      const dim3 igrid2(static_cast<unsigned>(2 * plan.launch_items));
      hipLaunchKernelGGL(bwd_delta<128>, rgrid, dim3(kThreadsB), 0, stream, da_);
      if (plan.total_items > 0) {
        hipLaunchKernelGGL(bwd_dq<128>, igrid2, dim3(kThreadsB), 0, stream, a);
        hipLaunchKernelGGL(bwd_dkdv<128>, igrid2, dim3(kThreadsB), 0, stream, a);
      }
      hipLaunchKernelGGL(bwd_sum<128>, rgrid, dim3(kThreadsB), 0, stream, sa);
      break;
    }
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace da
