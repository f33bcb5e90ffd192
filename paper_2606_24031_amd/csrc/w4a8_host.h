// Host-side helpers shared by the libw4a8 entry points.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/w4a8.h"

namespace w4a8 {

// W4A8_OK if the current device is gfx950, else W4A8_EDEVICE / W4A8_EHIP.
// Cached per device after the first query.
int check_device();

// W4A8_EHIP if a launch on this thread failed since the last check.
int check_launch();

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

// Compute units of the current device, known once check_device has run on
// it (0 otherwise).
int device_cus();

// Token rows per work item of the small-group (VALU) kernels; the sorted
// pair list in the workspace is padded by this many entries.
constexpr int SMALL_CHUNK = 8;

// Pre-norm residual input of a layer call: with gamma set, the layer's input
// is xn = RMSNorm(x + resid) * gamma, and x + resid goes to x_out.
struct DecodeNorm {
  const float *resid = nullptr;
  const float *gamma = nullptr;
  float *x_out = nullptr;
  float *xn = nullptr;
  float eps = 0.0f;
};

// Router in front of the single-token layer: the top-k of the token's logits
// (and the shared expert's sigmoid gate) taken inside the layer's launch;
// ids, weights and the gate value are also written out.
struct DecodeRoute {
  const float *logits = nullptr;   // [E]
  const float *gate = nullptr;     // [1] or null (shared expert weight 1)
  int32_t *ids = nullptr;          // [k]
  float *w = nullptr;              // [k]
  float *gate_w = nullptr;         // [1], written when gate is set
};

}  // namespace w4a8
