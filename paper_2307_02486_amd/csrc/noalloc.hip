// dilated_attn_fwd_noalloc: the forward pass with its workspace in a
// library-owned device array instead of caller memory, for callers that
// cannot allocate (code under HIP graph capture, serving loops, harnesses that
// forbid allocation).  The kernels are those of dilated_attn_fwd.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "kernels.h"
#include "plan.h"

namespace {

// The workspace of every no-alloc call on a device.  In host code this name
// stands for the array but is not its device address: the address comes from
// hipGetSymbolAddress, once per device.
constexpr uint64_t kScratchBytes = DA_NOALLOC_MAX_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of `scratch` on the current device (looked up on the first
// call there), or nullptr if the runtime reports an error.
void* scratch_ptr() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    g_scratch[dev] = p;
  }
  return g_scratch[dev];
}

bool overlaps(const void* a, uint64_t na, const void* b, uint64_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a);
  const uintptr_t y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

extern "C" int dilated_attn_fwd_noalloc(const void* q, const void* k, const void* v, void* out, float* lse,
                                        int64_t B, int64_t N, int64_t H, int64_t D, const da_pattern_t* patterns,
                                        int64_t num_patterns, int64_t causal, int64_t dtype, float softmax_scale,
                                        void* stream) {
  da::Plan p;
  const int rc = da::make_plan(B, N, H, D, patterns, num_patterns, causal, dtype, softmax_scale, &p);
  if (rc != DA_OK) return rc;
  if (!q || !k || !v || !out || !lse) return DA_EINVAL;
  if (p.workspace_bytes > kScratchBytes) return DA_ETOOLARGE;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) || !aligned16(lse)) return DA_EALIGN;
  const uint64_t esize = dtype == DA_BF16 ? 2 : 4;
  const uint64_t tb = static_cast<uint64_t>(B * N * H * D) * esize;
  const uint64_t lb = static_cast<uint64_t>(B * H * N) * 4;
  if (overlaps(out, tb, q, tb) || overlaps(out, tb, k, tb) || overlaps(out, tb, v, tb) ||
      overlaps(lse, lb, out, tb) || overlaps(lse, lb, q, tb) || overlaps(lse, lb, k, tb) ||
      overlaps(lse, lb, v, tb))
    return DA_EINVAL;
  void* ws = scratch_ptr();
  if (!ws) return DA_EHIP;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (da::launch_attention(p, q, k, v, ws, s) != hipSuccess) return DA_EHIP;
  if (da::launch_combine(p, ws, out, lse, s) != hipSuccess) return DA_EHIP;
  return DA_OK;
}
