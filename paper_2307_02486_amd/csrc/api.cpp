// C ABI of the dilated-attention forward and backward passes (declared in include/dilated_attn.h).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "kernels.h"
#include "plan.h"

namespace {

bool overlaps(const void* a, uint64_t na, const void* b, uint64_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a);
  const uintptr_t y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Profiling window of dilated_attn_profile_begin/end: three events per call.
struct ProfileWindow {
  bool active = false;
  int64_t capacity = 0;
  int64_t used = 0;
  std::vector<hipEvent_t> ev;  // [call][0..2]
};
ProfileWindow g_prof;

void destroy_events(ProfileWindow& w) {
  for (hipEvent_t e : w.ev)
    if (e) (void)hipEventDestroy(e);
  w.ev.clear();
  w.active = false;
  w.capacity = w.used = 0;
}

}  // namespace

extern "C" {

int dilated_attn_plan(int64_t B, int64_t N, int64_t H, int64_t D, const da_pattern_t* patterns,
                      int64_t num_patterns, int64_t causal, int64_t dtype, float softmax_scale,
                      da_plan_info_t* info) {
  if (!info) return DA_EINVAL;
  da::Plan p;
  const int rc = da::make_plan(B, N, H, D, patterns, num_patterns, causal, dtype, softmax_scale, &p);
  if (rc != DA_OK) return rc;
  info->workspace_bytes = p.workspace_bytes;
  info->num_work_items = p.total_items;
  info->covered_rows = p.covered_rows;
  info->sparse_flops = p.sparse_flops;
  info->bytes_attn = p.bytes_attn;
  info->bytes_combine = p.bytes_combine;
  return DA_OK;
}

int dilated_attn_fwd(const void* q, const void* k, const void* v, void* out, float* lse,
                     int64_t B, int64_t N, int64_t H, int64_t D, const da_pattern_t* patterns,
                     int64_t num_patterns, int64_t causal, int64_t dtype, float softmax_scale,
                     void* workspace, uint64_t workspace_bytes, void* stream) {
  da::Plan p;
  const int rc = da::make_plan(B, N, H, D, patterns, num_patterns, causal, dtype, softmax_scale, &p);
  if (rc != DA_OK) return rc;
  if (!q || !k || !v || !out || !lse || !workspace) return DA_EINVAL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) || !aligned16(lse) ||
      !aligned16(workspace))
    return DA_EALIGN;
  const uint64_t esize = dtype == DA_BF16 ? 2 : 4;
  const uint64_t tensor_bytes = static_cast<uint64_t>(B * N * H * D) * esize;
  const uint64_t lse_bytes = static_cast<uint64_t>(B * H * N) * 4;
  if (overlaps(out, tensor_bytes, q, tensor_bytes) || overlaps(out, tensor_bytes, k, tensor_bytes) ||
      overlaps(out, tensor_bytes, v, tensor_bytes) || overlaps(lse, lse_bytes, out, tensor_bytes) ||
      overlaps(lse, lse_bytes, q, tensor_bytes) || overlaps(lse, lse_bytes, k, tensor_bytes) ||
      overlaps(lse, lse_bytes, v, tensor_bytes))
    return DA_EINVAL;
  if (workspace_bytes < p.workspace_bytes) return DA_EWORKSPACE;
  const void* bufs[5] = {q, k, v, out, lse};
  const uint64_t sizes[5] = {tensor_bytes, tensor_bytes, tensor_bytes, tensor_bytes, lse_bytes};
  for (int i = 0; i < 5; ++i)
    if (overlaps(workspace, p.workspace_bytes, bufs[i], sizes[i])) return DA_EINVAL;

  hipStream_t s = static_cast<hipStream_t>(stream);
  hipEvent_t* ev = nullptr;
  if (g_prof.active && g_prof.used < g_prof.capacity) ev = &g_prof.ev[3 * g_prof.used++];
  if (ev && hipEventRecord(ev[0], s) != hipSuccess) return DA_EHIP;
  if (da::launch_attention(p, q, k, v, workspace, s) != hipSuccess) return DA_EHIP;
  if (ev && hipEventRecord(ev[1], s) != hipSuccess) return DA_EHIP;
  if (da::launch_combine(p, workspace, out, lse, s) != hipSuccess) return DA_EHIP;
  if (ev && hipEventRecord(ev[2], s) != hipSuccess) return DA_EHIP;
  return DA_OK;
}

int dilated_attn_bwd_plan(int64_t B, int64_t N, int64_t H, int64_t D, const da_pattern_t* patterns,
                          int64_t num_patterns, int64_t causal, int64_t dtype, float softmax_scale,
                          da_plan_info_t* info) {
  if (!info) return DA_EINVAL;
  da::Plan p;
  int rc = da::make_plan(B, N, H, D, patterns, num_patterns, causal, dtype, softmax_scale, &p);
  if (rc != DA_OK) return rc;
  da::BwdLayout l;
  rc = da::make_bwd_layout(p, &l);
  if (rc != DA_OK) return rc;
  info->workspace_bytes = l.workspace_bytes;
  info->num_work_items = 2 * p.total_items;
  info->covered_rows = p.covered_rows;
  info->sparse_flops = l.flops;
  info->bytes_attn = l.bytes_grad;
  info->bytes_combine = l.bytes_combine;
  return DA_OK;
}

int dilated_attn_bwd(const void* q, const void* k, const void* v, const void* out, const float* lse,
                     const void* dout, void* dq, void* dk, void* dv, int64_t B, int64_t N, int64_t H,
                     int64_t D, const da_pattern_t* patterns, int64_t num_patterns, int64_t causal,
                     int64_t dtype, float softmax_scale, void* workspace, uint64_t workspace_bytes,
                     void* stream) {
  da::Plan p;
  int rc = da::make_plan(B, N, H, D, patterns, num_patterns, causal, dtype, softmax_scale, &p);
  if (rc != DA_OK) return rc;
  da::BwdLayout l;
  rc = da::make_bwd_layout(p, &l);
  if (rc != DA_OK) return rc;
  const void* ins[6] = {q, k, v, out, lse, dout};
  void* outs[3] = {dq, dk, dv};
  for (const void* x : ins)
    if (!x) return DA_EINVAL;
  for (const void* x : outs)
    if (!x) return DA_EINVAL;
  if (!workspace) return DA_EINVAL;
  for (const void* x : ins)
    if (!aligned16(x)) return DA_EALIGN;
  for (const void* x : outs)
    if (!aligned16(x)) return DA_EALIGN;
  if (!aligned16(workspace)) return DA_EALIGN;
  const uint64_t tb = static_cast<uint64_t>(B * N * H * D) * 2;
  const uint64_t lb = static_cast<uint64_t>(B * H * N) * 4;
  const uint64_t in_sizes[6] = {tb, tb, tb, tb, lb, tb};
  for (int i = 0; i < 3; ++i) {
    for (int j = 0; j < 6; ++j)
      if (overlaps(outs[i], tb, ins[j], in_sizes[j])) return DA_EINVAL;
    for (int j = i + 1; j < 3; ++j)
      if (overlaps(outs[i], tb, outs[j], tb)) return DA_EINVAL;
  }
  if (workspace_bytes < l.workspace_bytes) return DA_EWORKSPACE;
  for (int j = 0; j < 6; ++j)
    if (overlaps(workspace, l.workspace_bytes, ins[j], in_sizes[j])) return DA_EINVAL;
  for (int i = 0; i < 3; ++i)
    if (overlaps(workspace, l.workspace_bytes, outs[i], tb)) return DA_EINVAL;

  hipStream_t s = static_cast<hipStream_t>(stream);
  if (da::launch_backward(p, l, q, k, v, out, lse, dout, dq, dk, dv, workspace, s) != hipSuccess)
    return DA_EHIP;
  return DA_OK;
}

int dilated_attn_xpos(const void* x, void* y, int64_t B, int64_t N, int64_t H, int64_t D,
                      int64_t sign, int64_t transpose, int64_t center, float base, float gamma,
                      float scale_base, int64_t dtype, void* stream) {
  if (!x || !y) return DA_EINVAL;
  if (B <= 0 || N <= 0 || H <= 0 || D < 8 || D > 256 || D % 8 != 0) return DA_EINVAL;
  if (dtype != DA_BF16 && dtype != DA_F32) return DA_EUNSUPPORTED;
  if ((sign != 1 && sign != -1) || (transpose != 0 && transpose != 1)) return DA_EINVAL;
  if (center < 0 || center >= N) return DA_EINVAL;
  if (!std::isfinite(base) || !(base > 1.0f) || !std::isfinite(gamma) || !(gamma > 0.0f) ||
      !std::isfinite(scale_base) || !(scale_base > 0.0f))
    return DA_EINVAL;
  // At most 2^34 elements: one thread per 8 keeps the grid within 2^32 work-items.
  if (B > (int64_t{1} << 34) / N || B * N > (int64_t{1} << 34) / H ||
      B * N * H > (int64_t{1} << 34) / D)
    return DA_EINVAL;
  // zeta_i ranges over [gamma / (1 + gamma), 1): the smallest gives the
  // largest |log2 zeta| (every zeta_i < 1 for gamma > 0 and i < D/2).
  const double l2z = std::fabs(std::log2(static_cast<double>(gamma) / (1.0 + gamma)));
  const double far = static_cast<double>(std::max(center, N - 1 - center));
  if (far / scale_base * l2z > 64.0) return DA_EINVAL;
  if (!aligned16(x) || !aligned16(y)) return DA_EALIGN;
  const uint64_t bytes = static_cast<uint64_t>(B * N * H * D) * (dtype == DA_BF16 ? 2 : 4);
  if (x != y && overlaps(x, bytes, y, bytes)) return DA_EINVAL;
  if (da::launch_xpos(x, y, B, N, H, D, static_cast<int>(sign), transpose != 0, center, base, gamma,
                      scale_base, static_cast<int>(dtype), static_cast<hipStream_t>(stream)) != hipSuccess)
    return DA_EHIP;
  return DA_OK;
}

int dilated_attn_wgrad_workspace(int64_t K, int64_t M, int64_t N, uint64_t* bytes) {
  if (!bytes) return DA_EINVAL;
  if (K < 0 || K > (int64_t{1} << 30) || M <= 0 || N <= 0 || M % 128 || N % 128 || M > 16384 || N > 16384)
    return DA_EINVAL;
  *bytes = da::wgrad_workspace(K, M, N);
  return DA_OK;
}

int dilated_attn_wgrad(const void* dy, const void* x, void* dw, void* db, int64_t K, int64_t M, int64_t N,
                       int64_t dtype, void* workspace, uint64_t workspace_bytes, void* stream) {
  uint64_t need = 0;
  if (!dw || (K > 0 && (!dy || !x))) return DA_EINVAL;
  if (dilated_attn_wgrad_workspace(K, M, N, &need) != DA_OK) return DA_EINVAL;
  if (dtype != DA_BF16) return DA_EUNSUPPORTED;
  if (need > 0 && !workspace) return DA_EINVAL;
  if (!aligned16(dy) || !aligned16(x) || !aligned16(dw) || !aligned16(db) || (need > 0 && !aligned16(workspace)))
    return DA_EALIGN;
  if (workspace_bytes < need) return DA_EWORKSPACE;
  const void* ins[2] = {dy, x};
  const uint64_t isz[2] = {static_cast<uint64_t>(K * M) * 2, static_cast<uint64_t>(K * N) * 2};
  const void* outs[3] = {dw, db, workspace};
  const uint64_t osz[3] = {static_cast<uint64_t>(M * N) * 2, db ? static_cast<uint64_t>(M) * 2 : 0, need};
  for (int i = 0; i < 3; ++i) {
    for (int j = i + 1; j < 3; ++j)
      if (overlaps(outs[i], osz[i], outs[j], osz[j])) return DA_EINVAL;
    for (int j = 0; j < 2; ++j)
      if (overlaps(outs[i], osz[i], ins[j], isz[j])) return DA_EINVAL;
  }
  if (da::launch_wgrad(dy, x, dw, db, K, M, N, workspace, static_cast<hipStream_t>(stream)) != hipSuccess)
    return DA_EHIP;
  return DA_OK;
}

int dilated_attn_layernorm_fwd(const void* x, const void* g, const void* b, void* y, float* mean, float* rstd,
                               int64_t rows, int64_t E, float eps, int64_t dtype, void* stream) {
  if (!g || !b || !y || !mean || !rstd || (rows > 0 && !x)) return DA_EINVAL;
  if (rows < 0 || rows > (int64_t{1} << 26) || E < 8 || E > 2048 || E % 8 || !std::isfinite(eps) || !(eps > 0.0f))
    return DA_EINVAL;
  if (dtype != DA_BF16) return DA_EUNSUPPORTED;
  if (!aligned16(x) || !aligned16(g) || !aligned16(b) || !aligned16(y)) return DA_EALIGN;
  const uint64_t xb = static_cast<uint64_t>(rows * E) * 2, sb = static_cast<uint64_t>(rows) * 4;
  if (x != y && overlaps(x, xb, y, xb)) return DA_EINVAL;
  const void* outs[3] = {y, mean, rstd};
  const uint64_t osz[3] = {xb, sb, sb};
  for (int i = 0; i < 3; ++i) {
    for (int j = i + 1; j < 3; ++j)
      if (overlaps(outs[i], osz[i], outs[j], osz[j])) return DA_EINVAL;
    if (overlaps(outs[i], osz[i], g, static_cast<uint64_t>(E) * 2) ||
        overlaps(outs[i], osz[i], b, static_cast<uint64_t>(E) * 2))
      return DA_EINVAL;
  }
  if (overlaps(mean, sb, x, xb) || overlaps(rstd, sb, x, xb)) return DA_EINVAL;
  if (da::launch_layernorm_fwd(x, g, b, y, mean, rstd, rows, E, eps, static_cast<hipStream_t>(stream)) !=
      hipSuccess)
    return DA_EHIP;
  return DA_OK;
}

int dilated_attn_layernorm_bwd_workspace(int64_t rows, int64_t E, uint64_t* bytes) {
  if (!bytes || rows < 0 || rows > (int64_t{1} << 26) || E < 8 || E > 2048 || E % 8) return DA_EINVAL;
  *bytes = da::layernorm_bwd_workspace(rows, E);
  return DA_OK;
}

int dilated_attn_layernorm_bwd(const void* dy, const void* x, const void* g, const float* mean, const float* rstd,
                               void* dx, void* dg, void* db, int64_t rows, int64_t E, int64_t dtype,
                               void* workspace, uint64_t workspace_bytes, void* stream) {
  uint64_t need = 0;
  if (dilated_attn_layernorm_bwd_workspace(rows, E, &need) != DA_OK) return DA_EINVAL;
  if (!g || !dg || !db || !workspace || (rows > 0 && (!dy || !x || !mean || !rstd || !dx))) return DA_EINVAL;
  if (dtype != DA_BF16) return DA_EUNSUPPORTED;
  if (!aligned16(dy) || !aligned16(x) || !aligned16(g) || !aligned16(dx) || !aligned16(workspace)) return DA_EALIGN;
  if (workspace_bytes < need) return DA_EWORKSPACE;
  const uint64_t xb = static_cast<uint64_t>(rows * E) * 2, sb = static_cast<uint64_t>(rows) * 4,
                 eb = static_cast<uint64_t>(E) * 2;
  const void* ins[5] = {dy, x, g, mean, rstd};
  const uint64_t isz[5] = {xb, xb, eb, sb, sb};
  const void* outs[4] = {dx, dg, db, workspace};
  const uint64_t osz[4] = {xb, eb, eb, need};
  for (int i = 0; i < 4; ++i) {
    for (int j = i + 1; j < 4; ++j)
      if (overlaps(outs[i], osz[i], outs[j], osz[j])) return DA_EINVAL;
    for (int j = 0; j < 5; ++j)
      if (overlaps(outs[i], osz[i], ins[j], isz[j])) return DA_EINVAL;
  }
  if (da::launch_layernorm_bwd(dy, x, g, mean, rstd, dx, dg, db, rows, E, workspace,
                               static_cast<hipStream_t>(stream)) != hipSuccess)
    return DA_EHIP;
  return DA_OK;
}

int dilated_attn_profile_begin(int64_t capacity) {
  if (g_prof.active || capacity < 1 || capacity > (int64_t{1} << 20)) return DA_EINVAL;
  g_prof.ev.assign(static_cast<size_t>(3 * capacity), nullptr);
  for (hipEvent_t& e : g_prof.ev) {
    if (hipEventCreate(&e) != hipSuccess) {
      e = nullptr;
      destroy_events(g_prof);
      return DA_EHIP;
    }
  }
  g_prof.capacity = capacity;
  g_prof.used = 0;
  g_prof.active = true;
  return DA_OK;
}

int dilated_attn_profile_end(double* ms_attention, double* ms_combine, int64_t* calls) {
  if (!g_prof.active) return DA_EINVAL;
  double ta = 0.0, tc = 0.0;
  int rc = DA_OK;
  if (g_prof.used > 0 && hipEventSynchronize(g_prof.ev[3 * g_prof.used - 1]) != hipSuccess) rc = DA_EHIP;
  for (int64_t i = 0; i < g_prof.used && rc == DA_OK; ++i) {
    float a = 0.0f, c = 0.0f;
    if (hipEventElapsedTime(&a, g_prof.ev[3 * i], g_prof.ev[3 * i + 1]) != hipSuccess ||
        hipEventElapsedTime(&c, g_prof.ev[3 * i + 1], g_prof.ev[3 * i + 2]) != hipSuccess)
      rc = DA_EHIP;
    ta += a;
    tc += c;
  }
  const int64_t n = g_prof.used;
  destroy_events(g_prof);
  if (rc != DA_OK) return rc;
  if (ms_attention) *ms_attention = ta;
  if (ms_combine) *ms_combine = tc;
  if (calls) *calls = n;
  return DA_OK;
}

const char* dilated_attn_strerror(int code) {
  switch (code) {
    case DA_OK: return "success";
    case DA_EINVAL: return "invalid argument (null pointer, size, pattern list or overlapping buffers)";
    case DA_EUNSUPPORTED: return "unsupported head dimension or dtype";
    case DA_EWORKSPACE: return "workspace smaller than dilated_attn_plan requires";
    case DA_EALIGN: return "device pointer not 16-byte aligned";
    case DA_EHIP: return "HIP runtime error at kernel launch";
    case DA_ETOOLARGE: return "problem needs more workspace than the no-alloc entry point's fixed buffer";
    default: return "unknown error code";
  }
}

}  // extern "C"
