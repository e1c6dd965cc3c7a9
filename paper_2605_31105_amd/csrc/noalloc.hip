// grkv_compress without a caller workspace, for callers that cannot allocate
// device memory (code under stream capture, serving loops, harnesses that
// forbid hipMalloc).  The workspace is a file-scope device array of fixed size
// instead; the kernels and the launch sequence are grkv_compress's own.
//
// In host code the array's name stands for a host-side shadow, not a device
// address.  Its device address is looked up once per device, with that device
// current (hipGetSymbolAddress), and kept; only that address is handed to the
// kernels.  Every region of the workspace is written before it is read within
// a call, so nothing needs clearing between calls.  All calls on one device
// share the array: calls that overlap in time on one device (two streams, two
// host threads) race on it.
#include <mutex>

#include "grkv_internal.h"

namespace grkv {
namespace {

constexpr size_t kScratchBytes = (size_t)GRKV_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];   // device address of `scratch` on each device

// Device address of the scratch array on the current device.
int scratch_on_current_device(void** ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return GRKV_ERR_HIP;
  if (dev >= kMaxDevices) return GRKV_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return GRKV_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return GRKV_OK;
}

}  // namespace
}  // namespace grkv

extern "C" int grkv_compress_noalloc(const void* q_obs, const void* K, const void* V, int64_t n,
                                     int32_t window, int32_t budget, int32_t pool_kernel,
                                     float lambda, void* stream, const grkv_problem* prob,
                                     const grkv_options* opt, const grkv_outputs* out) {
  // argument errors and the size check come first: a call that cannot run
  // touches no device state
  if (!q_obs || !K || !V || !out || !out->idx || !out->k_out || !out->v_out)
    return GRKV_ERR_INVALID;
  grkv::Plan p;
  int st = grkv::make_plan(prob, n, window, budget, pool_kernel, lambda, opt, &p);
  if (st != GRKV_OK) return st;
  if (p.total > grkv::kScratchBytes) return GRKV_ERR_WORKSPACE;
  void* ws = nullptr;
  st = grkv::scratch_on_current_device(&ws);
  if (st != GRKV_OK) return st;
  grkv_outputs o = *out;
  o.workspace = ws;
  o.workspace_bytes = grkv::kScratchBytes;
  return grkv_compress(q_obs, K, V, n, window, budget, pool_kernel, lambda, stream, prob, opt,
                       &o);
}
