// Device scratch of hermes_kv_init_static: the workspace of contexts whose
// callers cannot allocate device memory, as one file-scope array that the
// code object's loader places on every GPU the library runs on (each GPU
// holds its own copy until the process ends).  Host code never passes the
// array's name to a kernel: its device address is looked up once per device
// with that device current, and only that address is handed out.
#include <mutex>

#include "hermes_internal.h"

namespace hermes {
namespace {

__device__ __align__(256) unsigned char scratch[kStaticWorkspaceBytes];

struct DeviceSlot {
  void *ptr = nullptr;   // device address of `scratch` on this GPU (0 until looked up)
  bool busy = false;     // a live context owns it
};

DeviceSlot g_slot[kMaxDevices];
std::mutex g_mu;

}  // namespace

int static_workspace_acquire(void **ptr, int *device) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return HERMES_EHIP;
  if (dev < 0 || dev >= kMaxDevices) return HERMES_ENOTSUP;
  std::lock_guard<std::mutex> lock(g_mu);
  DeviceSlot &s = g_slot[dev];
  if (s.busy) return HERMES_ESTATE;
  if (s.ptr == nullptr) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return HERMES_EHIP;
    s.ptr = p;
  }
  s.busy = true;
  *ptr = s.ptr;
  *device = dev;
  return HERMES_OK;
}

void static_workspace_release(int device) {
  if (device < 0 || device >= kMaxDevices) return;
  std::lock_guard<std::mutex> lock(g_mu);
  g_slot[device].busy = false;
}

}  // namespace hermes
