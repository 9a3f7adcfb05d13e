// attn_fwd_noalloc: the fused forward with its split workspace in a static
// device array instead of an allocation, for callers that cannot allocate
// device memory (code under stream capture, tight serving loops).
//
// The array below exists once per GPU the library runs on, for the life of
// the process.  Its host-side name is not a device address: the address is
// looked up once per device (with that device current) and only that
// address is handed to kernels.  Every call on a GPU uses the same array, so
// calls that overlap in time on one GPU (different streams, or graphs
// replayed concurrently) race on it; calls on one stream are ordered.  The
// fused kernel writes every partial row the merge reads, so nothing has to
// start at zero and no clearing is issued.
#include <mutex>

#include "internal.h"

static __device__ __align__(256) unsigned char scratch[ATTN_NOALLOC_SCRATCH_BYTES];

namespace attn {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of this device's copy of `scratch`.
int scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return ATTN_E_HIP;
  if (dev < 0 || dev >= kMaxDevices) return ATTN_E_DEVICE;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return ATTN_E_HIP;
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return ATTN_OK;
}

}  // namespace
}  // namespace attn

extern "C" int attn_fwd_noalloc(const void* Q, const void* K, const void* V, void* O, int B, int H, int L, int d,
                                float scale, int causal, int dtype, void* stream) {
  using namespace attn;
  Prepared pr;
  int rc = prepare(Q, K, V, O, B, H, L, d, scale, causal, dtype, &pr);
  if (rc != ATTN_OK) return rc;
  if (pr.ws_bytes > (size_t)ATTN_NOALLOC_SCRATCH_BYTES) return ATTN_E_SCRATCH;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (pr.ws_bytes > 0) {
    void* ws = nullptr;
    rc = scratch_address(&ws);
    if (rc != ATTN_OK) return rc;
    bind_workspace(pr.p, ws, d);
  }
  if (launch_fused(pr, s) != hipSuccess) return ATTN_E_HIP;
  if (pr.p.n_split > 1 && launch_combine(pr.p, d, dtype, s) != hipSuccess) return ATTN_E_HIP;
  return ATTN_OK;
}
