// mlp_train_step_static: one SGD iteration whose workspace is a scratch array inside the
// library, for callers that cannot allocate device memory.
//
// The array is a file-scope __device__ variable: every GPU the library runs on holds its
// own copy, at its own address, from the library's load until the process ends. Host code
// never passes the array's name to a kernel (on the host that name is only a stand-in);
// it looks up the device address once per device with hipGetSymbolAddress, with that
// device current, and uses that address everywhere.

#include <mutex>

#include "common.h"

namespace imbd {
namespace {

static __device__ __align__(256) unsigned char scratch[IMBD_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's scratch array (looked up on the first call per device).
int scratch_for_current_device(void **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    set_error("mlp_train_step_static: no usable current device (%d)", dev);
    return IMBD_EHIP;
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      set_error("mlp_train_step_static: hipGetSymbolAddress failed on device %d: %s", dev, hipGetErrorString(e));
      return IMBD_EHIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return IMBD_OK;
}

}  // namespace
}  // namespace imbd

using namespace imbd;

extern "C" int mlp_train_step_static(const imbd_mlp_desc *desc, imbd_layer *layers, const void *x,
                                     const int32_t *labels, float lr, float *loss, void *stream) {
  const size_t need = mlp_workspace_bytes(desc);  // 0 for an invalid description
  if (need == 0) return mlp_train_step(desc, layers, x, labels, nullptr, 0, lr, loss, stream);  // reports why
  if (need > (size_t)IMBD_STATIC_SCRATCH_BYTES) {
    set_error("mlp_train_step_static: this network needs %zu bytes of workspace, the static scratch holds %zu",
              need, (size_t)IMBD_STATIC_SCRATCH_BYTES);
    return IMBD_EWORKSPACE;
  }
  void *ws = nullptr;
  const int rc = scratch_for_current_device(&ws);
  if (rc != IMBD_OK) return rc;
  // Every region the iteration reads is written earlier in the same iteration, so the
  // previous call's contents need no clearing.
  return mlp_train_step(desc, layers, x, labels, ws, (size_t)IMBD_STATIC_SCRATCH_BYTES, lr, loss, stream);
}
