// moe_ffn_layer without a caller-supplied workspace, for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid hipMalloc).  The layer's intermediate tensors live in
// one file-scope device array, `scratch`, of MOE_NOALLOC_SCRATCH_BYTES bytes
// that each GPU the library runs on holds until the process ends.
//
// Host code never passes the array's name to a kernel or a copy: on the host
// it is a stand-in, not a device address.  The first call on a device (with
// that device current) looks the array's device address up with
// hipGetSymbolAddress and keeps it per device; every later call uses that
// address.  The call then runs moe_ffn_layer with the array as its
// workspace: the same kernels, bit-identical results, nothing allocated or
// freed.  No kernel of the layer needs its workspace cleared (every
// intermediate is fully written before it is read), so the contents left by
// the previous call are harmless.  All calls on one GPU share its array:
// calls that may overlap on one GPU (on different streams, or from several
// host threads without ordering) race on it.
#include <mutex>

#include "common.h"

namespace moe {
namespace {

static __device__ __align__(256) uint8_t scratch[MOE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of the current device's copy of `scratch` (looked up
// once per device).
moe_status_t scratch_of_current_device(void** out) {
  int dev = -1;
  const hipError_t ge = hipGetDevice(&dev);
  if (ge != hipSuccess) return fail(MOE_ERR_HIP, "moe_ffn_layer_noalloc: hipGetDevice: %s", hipGetErrorString(ge));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(MOE_ERR_HIP, "moe_ffn_layer_noalloc: device %d beyond the %d the library tracks", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(MOE_ERR_HIP, "moe_ffn_layer_noalloc: hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MOE_OK;
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" moe_status_t moe_ffn_layer_noalloc(moe_dims_t d, int32_t T, moe_regime_t regime, const uint16_t* x_bf16,
                                              const int32_t* topk_ids, const float* topk_w, const uint8_t* w_gate,
                                              const float* s_gate, const uint8_t* w_up, const float* s_up,
                                              const uint8_t* w_down, const float* s_down, uint16_t* out_bf16,
                                              int32_t* dev_status, hipStream_t stream) {
  // Argument and shape errors come from moe_ffn_layer itself: without a
  // workspace it checks every argument, returns MOE_OK for T == 0 and
  // otherwise stops at the missing workspace (MOE_ERR_WORKSPACE), all before
  // anything is enqueued.
  const moe_status_t pre = moe_ffn_layer(d, T, regime, x_bf16, topk_ids, topk_w, w_gate, s_gate, w_up, s_up, w_down,
                                         s_down, out_bf16, dev_status, nullptr, 0, stream);
  if (pre != MOE_ERR_WORKSPACE) return pre;
  const size_t need = moe_ffn_layer_workspace(d, T, regime);
  if (need > (size_t)MOE_NOALLOC_SCRATCH_BYTES)
    return fail(MOE_ERR_WORKSPACE,
                "moe_ffn_layer_noalloc: T=%d needs %zu bytes of scratch, more than the %zu this entry point holds "
                "(use moe_ffn_layer with a workspace)",
                T, need, (size_t)MOE_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  const moe_status_t st = scratch_of_current_device(&ws);
  if (st != MOE_OK) return st;
  return moe_ffn_layer(d, T, regime, x_bf16, topk_ids, topk_w, w_gate, s_gate, w_up, s_up, w_down, s_down, out_bf16,
                       dev_status, ws, (size_t)MOE_NOALLOC_SCRATCH_BYTES, stream);
}
