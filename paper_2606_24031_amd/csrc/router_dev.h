// Router top-k inside one wave (paper Sec. 2.2: a sparsely gated MoE layer
// sends each token to its top-k of E routed experts; the k gate values are
// renormalized over the selection, as the Qwen3-series models do).  Shared by
// the router kernel and the single-token layer kernel, so both take the same
// decisions and produce the same bits.
#ifndef W4A8_ROUTER_DEV_H
#define W4A8_ROUTER_DEV_H

#include "w4a8_dev.h"

namespace w4a8 {

// row_bcast:15 and row_bcast:31 (lane 15 of a row into the next row, lane 31
// into rows 2 and 3), applied to the rows in the row mask.
constexpr int DPP_ROW_BCAST15 = 0x142, DPP_ROW_BCAST31 = 0x143;

// v combined with its DPP-moved copy; lanes outside the row mask ROWS take
// the identity ID as the moved value.
template <int CTRL, int ROWS, int ID>
__device__ __forceinline__ int dpp_or_id(int v) {
  return __builtin_amdgcn_update_dpp(ID, v, CTRL, ROWS, 0xF, false);
}

// Order-preserving int32 key of a finite float (-0 and +0 both map to 0, so
// they compare equal, as the floats do): non-negative floats keep their bits,
// negative ones flip the magnitude bits.
__device__ __forceinline__ int order_key(float f) {
  const int b = __builtin_bit_cast(int, f + 0.0f);   // -0 + 0 = +0
  return b ^ ((b >> 31) & 0x7FFFFFFF);
}
__device__ __forceinline__ float key_value(int key) {
  return __builtin_bit_cast(float, key ^ ((key >> 31) & 0x7FFFFFFF));
}

// Largest key over the wave (all 64 lanes active), in a scalar register: max
// over each 16-lane row (lane^1, lane^2, half-row mirror, lane^8), then row 0
// into row 1 and row 2 into row 3, then row 1 into rows 2 and 3; lane 63 ends
// with the maximum.
__device__ __forceinline__ int wave_max_key(int v) {
  constexpr int LO = (int)0x80000000;
  v = max(v, dpp_or_id<DPP_XOR1, 0xF, LO>(v));
  v = max(v, dpp_or_id<DPP_XOR2, 0xF, LO>(v));
  v = max(v, dpp_or_id<DPP_HALF_MIRROR, 0xF, LO>(v));
  v = max(v, dpp_or_id<DPP_ROR8, 0xF, LO>(v));
  v = max(v, dpp_or_id<DPP_ROW_BCAST15, 0xA, LO>(v));
  v = max(v, dpp_or_id<DPP_ROW_BCAST31, 0xC, LO>(v));
  return __builtin_amdgcn_readlane(v, 63);
}

// Sum over the wave in a fixed order, in a scalar register: the same
// exchanges, each partner pair adding the same two values (so every lane of a
// row holds the identical row sum), then (r0 + r1) + (r2 + r3) in lane 63.
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<DPP_XOR1>(v);
  v += dpp_f<DPP_XOR2>(v);
  v += dpp_f<DPP_HALF_MIRROR>(v);
  v += dpp_f<DPP_ROR8>(v);
  v += __builtin_bit_cast(float, dpp_or_id<DPP_ROW_BCAST15, 0xA, 0>(__builtin_bit_cast(int, v)));
  v += __builtin_bit_cast(float, dpp_or_id<DPP_ROW_BCAST31, 0xC, 0>(__builtin_bit_cast(int, v)));
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// Top-k of one token's logits held by a wave: x[r] is the logit of expert
// lane + 64 r (-inf past E; the logits are finite).  Round j takes the
// largest remaining value and, among equal values, the lowest index (the
// first r whose ballot of key[r] == max is non-empty, then its lowest lane;
// +0 and -0 count as equal), and removes it.  The fp32 logits are compared
// themselves: softmax is monotone, so this is the order of the probabilities
// without rounding in the decision.  Lane j < k ends with the j-th selection
// (value selv, index seli).  All 64 lanes must be active.
template <int RV>
__device__ __forceinline__ void wave_topk(float (&x)[RV], int k, float &selv, int &seli) {
  const int lane = threadIdx.x & 63;
  int key[RV];
#pragma unroll
  for (int r = 0; r < RV; r++) key[r] = order_key(x[r]);
  constexpr int TAKEN = (int)0x80000000;   // below every key, -inf's included
  selv = 0.0f;
  seli = 0;
  for (int j = 0; j < k; j++) {
    int m = key[0];
#pragma unroll
    for (int r = 1; r < RV; r++) m = max(m, key[r]);
    m = wave_max_key(m);
    int e = 0;
#pragma unroll
    for (int r = RV - 1; r >= 0; r--) {
      const uint64_t b = __ballot(key[r] == m);
      if (b != 0) e = 64 * r + __ffsll((unsigned long long)b) - 1;
    }
    if (lane == j) { selv = key_value(m); seli = e; }
#pragma unroll
    for (int r = 0; r < RV; r++)
      if (e == lane + 64 * r) key[r] = TAKEN;
  }
}

// Renormalized gate value of lane j < k's selection: exp(l_j - l_0) over its
// sum across the selection (the full softmax denominator cancels), the sum
// in the fixed order of wave_sum; 0 on the other lanes.  All 64 lanes must
// be active.
__device__ __forceinline__ float topk_weight(float selv, int k) {
  const int lane = threadIdx.x & 63;
  const float lmax = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(
                                                    __builtin_bit_cast(int, selv)));
  const float ex = lane < k ? expf(selv - lmax) : 0.0f;
  return ex / wave_sum(ex);
}

// The shared expert's sigmoid gate.
__device__ __forceinline__ float shared_gate(float g) { return 1.0f / (1.0f + expf(-g)); }

}  // namespace w4a8

#endif  // W4A8_ROUTER_DEV_H
