// Router top-k (paper Sec. 2.2: a sparsely gated MoE layer sends each token
// to its top-k of E routed experts; the k gate values are renormalized over
// the selection, as the Qwen3-series models do).
//
// One wave per token.  The token's logits are staged in LDS; k rounds each
// take the wave's largest remaining logit (a lane scans its strided share in
// index order, then DPP exchanges and four lane reads keep the larger value,
// or on equal values the lower index) and mark it taken.  The selection compares the fp32
// logits themselves: softmax is monotone, so this is the order of the
// probabilities without any rounding in the decision.  The weights are
// exp(l_j - l_max) over their sum across the selection (the full softmax
// denominator cancels in the renormalization), summed in a fixed butterfly.
#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int RT = 256;            // threads: four waves, one token each

// (av, ai) replaced by (bv, bi) when that is larger, or equal with a lower index.
__device__ __forceinline__ void take_better(float &av, int &ai, float bv, int bi) {
  if (bv > av || (bv == av && bi < ai)) { av = bv; ai = bi; }
}

// Largest (value, index) over the wave, equal values by the lower index, in
// every lane: DPP exchanges inside each 16-lane row (lane^1, lane^2, the
// half-row mirror, lane^8), then the four row results read out in row order.
__device__ __forceinline__ void wave_argmax(float &v, int &i) {
  take_better(v, i, dpp_f<DPP_XOR1>(v), dpp_i<DPP_XOR1>(i));
  take_better(v, i, dpp_f<DPP_XOR2>(v), dpp_i<DPP_XOR2>(i));
  take_better(v, i, dpp_f<DPP_HALF_MIRROR>(v), dpp_i<DPP_HALF_MIRROR>(i));
  take_better(v, i, dpp_f<DPP_ROR8>(v), dpp_i<DPP_ROR8>(i));
  float bv = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  int bi = __builtin_amdgcn_readlane(i, 0);
#pragma unroll
  for (int r = 1; r < 4; r++)
    take_better(bv, bi,
                __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16 * r)),
                __builtin_amdgcn_readlane(i, 16 * r));
  v = bv;
  i = bi;
}

__global__ __launch_bounds__(RT) void router_kernel(const float *__restrict__ logits,
                                                    int32_t *__restrict__ ids,
                                                    float *__restrict__ weights,
                                                    const float *__restrict__ gate,
                                                    float *__restrict__ gate_w, int64_t T, int E,
                                                    int k) {
  extern __shared__ float lv[];    // [RT / 64][E]
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * (RT / 64) + wave;
  if (t >= T) return;              // whole waves; no workgroup barrier below
  float *v = lv + (size_t)wave * E;
  const float *row = logits + t * E;
  for (int e = lane; e < E; e += 64) v[e] = row[e];
  float selv = 0.0f;
  int seli = 0;                    // lane j < k: the j-th selection
  for (int j = 0; j < k; j++) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    for (int e = lane; e < E; e += 64) {
      const float x = v[e];
      if (x > bv) { bv = x; bi = e; }
    }
    wave_argmax(bv, bi);
    if (lane == j) { selv = bv; seli = bi; }
    if (lane == (bi & 63)) v[bi] = -INFINITY;   // taken (the logits are finite)
  }
  const float lmax = __shfl(selv, 0);
  const float ex = lane < k ? expf(selv - lmax) : 0.0f;
  float s = ex;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  if (lane < k) {
    ids[t * k + lane] = seli;
    weights[t * k + lane] = ex / s;
  }
  // the shared expert's sigmoid gate
  if (gate != nullptr && lane == 0) gate_w[t] = 1.0f / (1.0f + expf(-gate[t]));
}

}  // namespace

// Validated arguments; gate and gate_w may be null (no shared-expert gate).
int router_launch(const float *logits, int32_t *ids, float *weights, const float *gate,
                  float *gate_w, int64_t T, int64_t E, int64_t k, hipStream_t s) {
  const int64_t grid = (T + RT / 64 - 1) / (RT / 64);
  const size_t lds = sizeof(float) * (RT / 64) * (size_t)E;
  router_kernel<<<dim3((unsigned)grid), dim3(RT), lds, s>>>(logits, ids, weights, gate, gate_w, T,
                                                            (int)E, (int)k);
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
