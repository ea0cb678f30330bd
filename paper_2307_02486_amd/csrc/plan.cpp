// Host-side plan of a dilated-attention forward call (see plan.h).
#include "plan.h"

#include <cmath>
#include <cstring>

namespace da {

FastDiv make_fastdiv(uint32_t d) {
  FastDiv f;
  f.d = d;
  uint32_t l = 0;
  while ((uint64_t{1} << l) < d) ++l;           // l = ceil(log2 d)
  f.shift = 31 + l;
  const uint64_t num = uint64_t{1} << f.shift;  // 2^(31+l) <= 2^62
  f.mul = static_cast<uint32_t>((num + d - 1) / d);
  return f;
}

#ifndef DA_BF16_WAVES
#define DA_BF16_WAVES 4
#endif
int block_m_for(int dtype) { return dtype == DA_BF16 ? 32 * DA_BF16_WAVES : 64; }

namespace {

constexpr uint64_t kAlign = 256;

uint64_t align_up(uint64_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

}  // namespace

int make_plan(int64_t B, int64_t N, int64_t H, int64_t D, const da_pattern_t* patterns,
              int64_t num_patterns, int64_t causal, int64_t dtype, float softmax_scale,
              Plan* out) {
  if (!patterns || !out) return DA_EINVAL;
  if (B < 1 || N < 1 || H < 1 || D < 1) return DA_EINVAL;
  if (N + H >= (int64_t{1} << 31) || H >= (int64_t{1} << 16) || B >= (int64_t{1} << 31))
    return DA_EINVAL;
  if (num_patterns < 1 || num_patterns > DA_MAX_PATTERNS) return DA_EINVAL;
  if (!(softmax_scale >= 0.0f) || std::isinf(softmax_scale)) return DA_EINVAL;
  if (causal != 0 && causal != 1) return DA_EINVAL;
  for (int64_t i = 0; i < num_patterns; ++i) {
    const int64_t w = patterns[i].w, r = patterns[i].r;
    if (w < 1 || r < 1 || r > w) return DA_EINVAL;
  }
  if (dtype != DA_F32 && dtype != DA_BF16) return DA_EUNSUPPORTED;
  if (D != 32 && D != 64 && D != 128) return DA_EUNSUPPORTED;
  // every row offset ((b*N + p)*H + h) must fit in 63 bits with room to spare
  if (static_cast<double>(B) * N * H * D > 4.0e18) return DA_EINVAL;

  Plan p;
  std::memset(&p, 0, sizeof(p));
  p.B = B;
  p.N = N;
  p.H = H;
  p.D = D;
  p.causal = static_cast<int>(causal);
  p.dtype = static_cast<int>(dtype);
  p.scale = softmax_scale > 0.0f ? softmax_scale : static_cast<float>(1.0 / std::sqrt(double(D)));
  p.npat = static_cast<int>(num_patterns);
  p.block_m = block_m_for(p.dtype);
  const int64_t esize = dtype == DA_BF16 ? 2 : 4;
  // Per-pattern output rows are kept as fp16 for bf16 inputs, each row divided
  // by a power of two that brings its largest magnitude into [2^14, 2^15)
  // (fp16's eleven significant bits with bf16's exponent range), and as fp32
  // for fp32 inputs.  Each row has an 8-byte record: its lse and its scale.
  const int64_t ws_esize = dtype == DA_BF16 ? 2 : 4;
  constexpr int64_t kRecBytes = 8;

  uint64_t ws = 0;
  int64_t items = 0;
  long double pairs = 0.0L;
  int64_t covered = 0;
  for (int i = 0; i < p.npat; ++i) {
    PatternPlan& pp = p.pat[i];
    pp.w = patterns[i].w < N ? patterns[i].w : N;
    // A dilation beyond N + H keeps exactly the rows it would keep at N + H:
    // every head's offset is its own index and each segment keeps one row.
    pp.r = patterns[i].r < N + H ? patterns[i].r : N + H;
    pp.nseg = (N + pp.w - 1) / pp.w;
    pp.lmax = (pp.w + pp.r - 1) / pp.r;
    pp.ntiles = (pp.lmax + p.block_m - 1) / p.block_m;
    pp.units = B * H * pp.nseg;
    pp.item_begin = items;
    items += pp.units * pp.ntiles;
    const uint64_t rows = static_cast<uint64_t>(pp.units) * static_cast<uint64_t>(pp.lmax);
    pp.o_off = ws;
    ws = align_up(ws + rows * static_cast<uint64_t>(D) * ws_esize);
    pp.lse_off = ws;
    ws = align_up(ws + rows * kRecBytes);

    // exact kept rows and unmasked pairs: full segments, then the short tail
    const int64_t nfull = N / pp.w;
    const int64_t tail = N - nfull * pp.w;
    const int64_t nres = pp.r < H ? pp.r : H;  // offsets actually used by heads
    for (int64_t s = 0; s < nres; ++s) {
      const int64_t heads = H / pp.r + (s < H % pp.r ? 1 : 0);  // heads with h mod r == s
      const int64_t Lf = kept_rows(pp.w, s, pp.r);
      const int64_t Lt = tail > 0 ? kept_rows(tail, s, pp.r) : 0;
      covered += B * heads * (nfull * Lf + Lt);
      const long double pf = causal ? 0.5L * Lf * (Lf + 1) : (long double)Lf * Lf;
      const long double pt = causal ? 0.5L * Lt * (Lt + 1) : (long double)Lt * Lt;
      pairs += (long double)B * heads * (nfull * pf + pt);
    }
  }
  int64_t launch = 0;
  for (int i = 0; i < p.npat; ++i) launch += (p.pat[i].units + 7) / 8 * p.pat[i].ntiles;
  launch *= 8;
  if (items >= (int64_t{1} << 31) || launch >= (int64_t{1} << 31)) return DA_EINVAL;
  p.launch_items = launch;
  // A key tile of the attention kernel spans at most 128 kept rows, each r*H*D
  // elements after the previous one; 32-bit byte offsets inside a tile (plus
  // one row) must stay below 2^31.
  p.offsets32 = true;
  for (int i = 0; i < p.npat; ++i)
    if (static_cast<double>(p.pat[i].r) * H * D * esize * 129.0 >= 2147483648.0) p.offsets32 = false;
  // the combine stage launches one workgroup per 8..32 positions of each (b, h)
  if ((N + 7) / 8 * B * H >= (int64_t{1} << 31)) return DA_EINVAL;
  p.total_items = items;
  p.workspace_bytes = ws;
  p.covered_rows = covered;
  p.sparse_flops = static_cast<double>(4.0L * D * pairs);
  p.bytes_attn = static_cast<double>(covered) * (3.0 * D * esize + D * ws_esize + kRecBytes);
  p.bytes_combine = static_cast<double>(covered) * (D * ws_esize + kRecBytes) +
                    static_cast<double>(B) * N * H * (D * esize + 4.0);
  *out = p;
  return DA_OK;
}

int make_bwd_layout(const Plan& p, BwdLayout* out) {
  if (!out) return DA_EINVAL;
  if (p.dtype != DA_BF16) return DA_EUNSUPPORTED;
  // 32-bit offsets inside a tile of 64 kept rows (rows r*H*D elements apart,
  // and the rows' per-row scalars r floats apart)
  if (!p.offsets32) return DA_EUNSUPPORTED;
  for (int i = 0; i < p.npat; ++i)
    if (static_cast<double>(p.pat[i].r) * 4.0 * 65.0 >= 2147483648.0) return DA_EUNSUPPORTED;
  BwdLayout l;
  std::memset(&l, 0, sizeof(l));
  const uint64_t rows_all = static_cast<uint64_t>(p.B) * p.N * p.H;
  uint64_t ws = 0;
  l.nl2_off = ws;
  ws = align_up(ws + rows_all * 4);
  l.nd_off = ws;
  ws = align_up(ws + rows_all * 4);
  const uint64_t chunks = static_cast<uint64_t>(grad_chunks(p.D));
  for (int i = 0; i < p.npat; ++i) {
    const uint64_t rows = static_cast<uint64_t>(p.pat[i].units) * static_cast<uint64_t>(p.pat[i].lmax);
    const uint64_t bytes = rows * static_cast<uint64_t>(p.D) * 2;  // fp16 rows
    const uint64_t rec = rows * chunks * 4;                           // float scales
    l.dq_off[i] = ws;
    ws = align_up(ws + bytes);
    l.dk_off[i] = ws;
    ws = align_up(ws + bytes);
    l.dv_off[i] = ws;
    ws = align_up(ws + bytes);
    l.dq_rec_off[i] = ws;
    ws = align_up(ws + rec);
    l.dk_rec_off[i] = ws;
    ws = align_up(ws + rec);
    l.dv_rec_off[i] = ws;
    ws = align_up(ws + rec);
  }
  l.workspace_bytes = ws;
  const double D = static_cast<double>(p.D), es = 2.0, cov = static_cast<double>(p.covered_rows);
  const double grad_row = D * 2.0 + 4.0 * static_cast<double>(chunks);  // a compact row and its scales
  l.flops = 2.5 * p.sparse_flops;
  // each gradient kernel reads the kept q, k, v, dout rows once and the two
  // per-row scalars; dq writes one compact row, dk/dv two
  l.bytes_grad = cov * (2.0 * (4.0 * D * es + 8.0) + 3.0 * grad_row);
  // delta: out, dout and lse of every row read, two scalars written; sum:
  // the compact gradients read, dq, dk, dv written
  l.bytes_combine = static_cast<double>(rows_all) * (2.0 * D * es + 4.0 + 8.0 + 3.0 * D * es) +
                    cov * 3.0 * grad_row;
  *out = l;
  return DA_OK;
}

}  // namespace da
