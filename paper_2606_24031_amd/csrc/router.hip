// Router top-k (paper Sec. 2.2: a sparsely gated MoE layer sends each token
// to its top-k of E routed experts; the k gate values are renormalized over
// the selection, as the Qwen3-series models do).
//
// One wave per token.  The token's logits sit in registers (E <= 512, see
// wave_topk) or in LDS (larger E: k rounds in which each lane scans its
// strided share in index order and DPP exchanges and row broadcasts keep the
// larger value, or on equal values the lower index).
#include "router_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int RT = 256;            // threads: four waves, one token each

// (av, ai) replaced by (bv, bi) when that is larger, or equal with a lower index.
__device__ __forceinline__ void take_better(float &av, int &ai, float bv, int bi) {
  // bitwise on the conditions: a branch-free select
  const bool take = (bv > av) | ((bv == av) & (bi < ai));
  av = take ? bv : av;
  ai = take ? bi : ai;
}

// Largest (value, index) over the wave, equal values by the lower index:
// DPP exchanges inside each 16-lane row (lane^1, lane^2, the half-row
// mirror, lane^8), then row broadcasts (row 0's result into row 1 and row
// 2's into row 3, then row 1's into rows 2 and 3), and lane 63 read out.
template <int CTRL, int ROWS>
__device__ __forceinline__ void dpp_better(float &v, int &i) {
  const float ov = __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, v), __builtin_bit_cast(int, v),
                                         CTRL, ROWS, 0xF, false));
  const int oi = __builtin_amdgcn_update_dpp(i, i, CTRL, ROWS, 0xF, false);
  take_better(v, i, ov, oi);
}

__device__ __forceinline__ void wave_argmax(float &v, int &i) {
  dpp_better<DPP_XOR1, 0xF>(v, i);
  dpp_better<DPP_XOR2, 0xF>(v, i);
  dpp_better<DPP_HALF_MIRROR, 0xF>(v, i);
  dpp_better<DPP_ROR8, 0xF>(v, i);
  dpp_better<DPP_ROW_BCAST15, 0xA>(v, i);   // into rows 1 and 3
  dpp_better<DPP_ROW_BCAST31, 0xC>(v, i);   // into rows 2 and 3
  v = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
  i = __builtin_amdgcn_readlane(i, 63);
}

// RV > 0: the token's logits live in registers, RV per lane (E <= 64 * RV);
// RV == 0: in LDS.
template <int RV>
__global__ __launch_bounds__(RT) void router_kernel(const float *__restrict__ logits,
                                                    int32_t *__restrict__ ids,
                                                    float *__restrict__ weights,
                                                    const float *__restrict__ gate,
                                                    float *__restrict__ gate_w, int64_t T, int E,
                                                    int k) {
  extern __shared__ float lv[];    // [RT / 64][E] (LDS form only)
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * (RT / 64) + wave;
  if (t >= T) return;              // whole waves; no workgroup barrier below
  const float *row = logits + t * E;
  float selv = 0.0f;
  int seli = 0;                    // lane j < k: the j-th selection
  float gv = 0.0f;                 // the gate logit (lane 0)
  if (RV > 0) {
    float x[RV > 0 ? RV : 1];
    // every load in flight at once (clamped addresses, masked afterwards),
    // the gate logit's too
#pragma unroll
    for (int r = 0; r < RV; r++) x[r] = row[min(lane + 64 * r, E - 1)];
    gv = gate != nullptr && lane == 0 ? gate[t] : 0.0f;
#pragma unroll
    for (int r = 0; r < RV; r++)
      if (lane + 64 * r >= E) x[r] = -INFINITY;
    wave_topk<(RV > 0 ? RV : 1)>(x, k, selv, seli);
  } else {
    float *v = lv + (size_t)wave * E;
    for (int e = lane; e < E; e += 64) v[e] = row[e];
    for (int j = 0; j < k; j++) {
      float bv = -INFINITY;
      int bi = 0x7fffffff;
      for (int e = lane; e < E; e += 64) {
        const float xv = v[e];
        if (xv > bv) { bv = xv; bi = e; }
      }
      wave_argmax(bv, bi);
      if (lane == j) { selv = bv; seli = bi; }
      if (lane == (bi & 63)) v[bi] = -INFINITY;
    }
  }
  const float wt = topk_weight(selv, k);
  if (lane < k) {
    ids[t * k + lane] = seli;
    weights[t * k + lane] = wt;
  }
  // the shared expert's sigmoid gate
  if (gate != nullptr && lane == 0) gate_w[t] = shared_gate(RV > 0 ? gv : gate[t]);
}

}  // namespace

// Validated arguments; gate and gate_w may be null (no shared-expert gate).
int router_launch(const float *logits, int32_t *ids, float *weights, const float *gate,
                  float *gate_w, int64_t T, int64_t E, int64_t k, hipStream_t s) {
  const int64_t grid = (T + RT / 64 - 1) / (RT / 64);
  if (E <= 256) {
    router_kernel<4><<<dim3((unsigned)grid), dim3(RT), 0, s>>>(logits, ids, weights, gate, gate_w,
                                                               T, (int)E, (int)k);
  } else if (E <= 512) {
    router_kernel<8><<<dim3((unsigned)grid), dim3(RT), 0, s>>>(logits, ids, weights, gate, gate_w,
                                                               T, (int)E, (int)k);
  } else {
    const size_t lds = sizeof(float) * (RT / 64) * (size_t)E;
    router_kernel<0><<<dim3((unsigned)grid), dim3(RT), lds, s>>>(logits, ids, weights, gate,
                                                                 gate_w, T, (int)E, (int)k);
  }
  return check_launch();
}

}  // namespace w4a8

using namespace w4a8;

extern "C" int moe_router_topk(const float *logits, int32_t *ids, float *weights, int64_t T,
                               int64_t E, int64_t k, void *stream) {
  if (!logits || !ids || !weights) return W4A8_ENULL;
  if (T < 0) return W4A8_ESHAPE;
  if (E < 1 || E > 4096 || k < 1 || k > 32 || k > E) return W4A8_ERANGE;
  if (T > 0 && (T >= ((int64_t)1 << 31) || T * E >= ((int64_t)1 << 40))) return W4A8_ERANGE;
  const uintptr_t m = reinterpret_cast<uintptr_t>(logits) | reinterpret_cast<uintptr_t>(ids) |
                      reinterpret_cast<uintptr_t>(weights);
  if (m & 3u) return W4A8_EALIGN;
  if (T == 0) return W4A8_OK;
  int rc = check_device();
  if (rc != W4A8_OK) return rc;
  return router_launch(logits, ids, weights, nullptr, nullptr, T, E, k, as_stream(stream));
}
