// sarathi_hybrid_layer_forward_noalloc: the hybrid-batch layer forward with
// its workspace (normalised rows, q/k/v, attention partials and output,
// residual stream, FFN activation, split-K partials, batch metadata) in a
// static device array instead of a caller-passed buffer, for callers that
// cannot allocate device memory.  Every kernel and the launch sequence are
// those of sarathi_hybrid_layer_forward.
//
// The array is part of this library's code object: each GPU the library runs
// on holds its own copy of NOALLOC_SCRATCH_BYTES from the first call on that
// device until the process ends.  Host code never uses the array's name as an
// address (on the host it is only a stand-in symbol): the device address is
// looked up once per device with hipGetSymbolAddress and kept here.
#include <hip/hip_runtime.h>

#include <mutex>

#include "host_error.h"
#include "runtime_internal.h"
#include "sarathi.h"

namespace {

constexpr size_t NOALLOC_SCRATCH_BYTES = SARATHI_NOALLOC_SCRATCH_BYTES;
constexpr int MAX_DEVICES = 64;

__device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

std::mutex g_mu;
void* g_ptr[MAX_DEVICES];   // device address of `scratch` on each device (null: not looked up yet)

// Device address of the scratch array on the current device, looked up on the
// first call there (with that device current).
int scratch_on_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return sarathi::fail(SARATHI_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= MAX_DEVICES) return sarathi::fail(SARATHI_EUNSUPPORTED, "device %d >= %d", dev, MAX_DEVICES);
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return sarathi::fail(SARATHI_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return SARATHI_OK;
}

}  // namespace

extern "C" int sarathi_hybrid_layer_forward_noalloc(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w,
                                                    sarathi_kv* kv, int layer, const sarathi_hybrid_batch* batch,
                                                    const void* x_in, void* x_out, void* hip_stream) {
  size_t need = 0;
  int rc = sarathi::hybrid_check_noalloc(cfg, w, kv, layer, batch, x_in, x_out, &need);
  if (rc) return rc;
  if (need > NOALLOC_SCRATCH_BYTES)
    return sarathi::fail(SARATHI_ENOSPC,
                         "batch needs %zu bytes of workspace; the static scratch of the no-allocation entry point "
                         "holds %zu",
                         need, NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  rc = scratch_on_current_device(&ws);
  if (rc) return rc;
  return sarathi_hybrid_layer_forward(cfg, w, kv, layer, batch, x_in, x_out, ws, NOALLOC_SCRATCH_BYTES, hip_stream);
}
