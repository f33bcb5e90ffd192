// Status strings and the per-device architecture check.
#include <atomic>
#include <cstring>

#include "w4a8_host.h"

extern "C" const char *w4a8_strerror(int code) {
  switch (code) {
    case W4A8_OK: return "success";
    case W4A8_ENULL: return "a required pointer is NULL";
    case W4A8_ESHAPE: return "invalid shape";
    case W4A8_ERANGE: return "k, E or a size is outside the supported range";
    case W4A8_EWORKSPACE: return "workspace too small";
    case W4A8_EALIGN: return "a base pointer is not 16-byte aligned";
    case W4A8_EHIP: return "HIP runtime error or kernel launch failure";
    case W4A8_EDEVICE: return "current device is not gfx950 (MI355X)";
    case W4A8_EALIAS: return "an output buffer aliases an input or another output";
    case W4A8_ESCRATCH:
      return "these sizes need more workspace than the fixed scratch of the no-allocation "
             "entry point holds (W4A8_NOALLOC_SCRATCH_BYTES)";
    default: return "unknown status code";
  }
}

namespace w4a8 {

namespace {
constexpr int kMaxDevices = 64;
// 0 = unknown, 1 = gfx950, 2 = other architecture
std::atomic<int> g_arch[kMaxDevices];
std::atomic<int> g_cus[kMaxDevices];   // compute units, set with g_arch
}  // namespace

int check_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return W4A8_EHIP;
  if (dev < 0 || dev >= kMaxDevices) return W4A8_EDEVICE;
  int state = g_arch[dev].load(std::memory_order_relaxed);
  if (state == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return W4A8_EHIP;
    state = (std::strncmp(prop.gcnArchName, "gfx950", 6) == 0) ? 1 : 2;
    g_cus[dev].store(prop.multiProcessorCount, std::memory_order_relaxed);
    g_arch[dev].store(state, std::memory_order_relaxed);
  }
  return state == 1 ? W4A8_OK : W4A8_EDEVICE;
}

int device_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
  return g_cus[dev].load(std::memory_order_relaxed);
}

int check_launch() {
  return hipGetLastError() == hipSuccess ? W4A8_OK : W4A8_EHIP;
}

}  // namespace w4a8
