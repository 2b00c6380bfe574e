// The MoE layer forward on a scratch buffer the library holds itself, for
// callers that cannot allocate device memory (code under HIP graph capture,
// serving loops or harnesses that forbid hipMalloc).  It runs exactly the
// kernels of qd_moe_layer_forward; only the workspace differs.
//
// The scratch buffer is one file-scope device array.  On the host its name
// stands for a host-side symbol, not a device address: the device address is
// looked up once per device with hipGetSymbolAddress (with that device
// current) and only that address is handed to kernels.  Each device holds
// its own copy of the array until the process ends.  Every call on a device
// reuses that device's copy, so calls that overlap on one device (different
// streams, different host threads) race on it; calls on one stream are
// ordered and safe.  Nothing in the scratch buffer needs to start at zero:
// the layer's kernels clear what they accumulate into.
#include <mutex>

#include "common.h"

namespace {

static __device__ __align__(256) unsigned char scratch[QD_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_scratch[kMaxDevices];   // device address of `scratch` per device

// The current device's scratch address, looked up on its first use there.
qd_status scratch_address(void **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return QD_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return QD_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return QD_ERR_HIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return QD_OK;
}

}  // namespace

extern "C" size_t qd_moe_layer_noalloc_max_bytes(void) { return QD_NOALLOC_SCRATCH_BYTES; }

extern "C" qd_status qd_moe_layer_forward_noalloc(const void *x, const float *logits, int64_t T,
                                                  int64_t H, int32_t E, int32_t k, int64_t I,
                                                  int32_t Ks, int32_t Ks2, int32_t renorm,
                                                  const qd_nvfp4 *w13, const qd_nvfp4 *w2,
                                                  void *y, void *stream) {
  // the size check comes first: a batch too large for the scratch buffer is
  // refused before any device work (qd_moe_layer_workspace is 0 for invalid
  // sizes, which the forward below then rejects)
  const size_t need = qd_moe_layer_workspace(T, H, E, k, I);
  if (need > (size_t)QD_NOALLOC_SCRATCH_BYTES) return QD_ERR_WORKSPACE;
  void *ws = nullptr;
  const qd_status st = scratch_address(&ws);
  if (st) return st;
  return qd_moe_layer_forward(x, logits, T, H, E, k, I, Ks, Ks2, renorm, w13, w2, y, ws,
                              (size_t)QD_NOALLOC_SCRATCH_BYTES, stream);
}
