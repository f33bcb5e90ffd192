// The routed + shared MoE layer in the paper's own block format (Sec. 2.2:
// top-k routed experts plus one always-on shared expert; Sec. 2.3: weights
// in {-7..7} with an FP32 scale per group; Sec. 3.3: activations quantized
// per group to 8 bits with an FP32 scale, integer block dots, one scaling
// per group).  Four launches:
//   1. Q8_F32 of every token's row (the quantizer of sym.hip);
//   2. gate/up: one workgroup per (pair, 32-column block of h): its 32 gate
//      and 32 up rows against the pair's token, four lanes per row, then
//      SwiGLU and Q8_F32 of the 32 values of h in the workgroup;
//   3. down: one workgroup per (pair, slab of output rows) against the
//      pair's Q8_F32(h), scaled by the pair's routing weight;
//   4. combine: per token, the routed slots in order, then the shared one.
// The activations of a workgroup sit in LDS in nibble-split form (as in the
// GEMV of this format), so the block dots are the 4-bit dot products of the
// Q4_0 path on the stored nibbles.
#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int Q4SB = W4A8_Q4_SYM_BLOCK_BYTES;   // 20
constexpr int Q8FB = W4A8_Q8_F32_BLOCK_BYTES;   // 36
constexpr int SNT = 256;
constexpr int64_t SYM_LAYER_K_MAX = 16384;      // H, I: the staged activation row fits LDS

inline size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }

struct SymLayout {
  size_t xq, h, hq, y, total;
};

SymLayout sym_layout(int64_t T, int64_t H, int64_t I, int64_t k) {
  const int64_t P = T * k + T;
  SymLayout L;
  size_t off = 0;
  L.xq = off; off += up256((size_t)T * (H / QK) * Q8FB);
  L.h = off;  off += up256(sizeof(float) * (size_t)P * I);
  L.hq = off; off += up256((size_t)P * (I / QK) * Q8FB);
  L.y = off;  off += up256(sizeof(float) * (size_t)P * H);
  L.total = off;
  return L;
}

int sym_validate(int64_t T, int64_t H, int64_t I, int64_t E, int64_t k) {
  if (T < 0 || H <= 0 || I <= 0 || E <= 0 || k <= 0 || H % 256 != 0 || I % 256 != 0)
    return W4A8_ESHAPE;
  if (H > SYM_LAYER_K_MAX || I > SYM_LAYER_K_MAX || k > 64 || E >= ((int64_t)1 << 24) ||
      T >= ((int64_t)1 << 24))
    return W4A8_ERANGE;
  const int64_t P = T * k + T;
  if (P * (I / QK) >= ((int64_t)1 << 31) || P * (H / 64) >= ((int64_t)1 << 31))
    return W4A8_ERANGE;
  return W4A8_OK;
}

struct SymArgs {
  const int32_t *ids;
  const float *topk_w;
  const uint8_t *w_gu, *w_d, *ws_gu, *ws_d;
  const uint8_t *xq;     // [T][H/32] Q8_F32
  float *h;              // [P][I]
  uint8_t *hq;           // [P][I/32] Q8_F32
  float *y;              // [P][H]: w_pair * (down product)
  int64_t T, H, I, E, k;
};

// Pair p's token and expert matrix (gate/up or down), or null when the slot
// is skipped (id outside [0, E)) or there is no shared expert.
__device__ __forceinline__ const uint8_t *pair_matrix(const SymArgs &a, int64_t p, bool gateup,
                                                      int64_t *tok) {
  const int64_t pr = a.T * a.k;
  if (p < pr) {
    *tok = p / a.k;
    const int e = a.ids[p];
    if (e < 0 || e >= a.E) return nullptr;
    const int64_t bytes = gateup ? 2 * a.I * (a.H / QK) * Q4SB : a.H * (a.I / QK) * Q4SB;
    return (gateup ? a.w_gu : a.w_d) + (int64_t)e * bytes;
  }
  *tok = p - pr;
  return gateup ? a.ws_gu : a.ws_d;
}

// One row of Q8_F32 blocks into the workgroup's nibble-split activation
// buffer (whole 8-lane groups per block).
__device__ __forceinline__ void stage_q8f32(ActBuf xb, const uint8_t *row, int nb) {
  for (int t = threadIdx.x; t < nb * 8; t += blockDim.x) {
    const int blk = t >> 3, j = t & 7;
    const uint8_t *bp = row + (int64_t)blk * Q8FB;
    const uint32_t packed = *reinterpret_cast<const uint32_t *>(bp + 4 + 4 * j);
    const uint32_t word = split_word(packed, j);
    const int lsum = sum8(low_nibble_sum(packed));
    *code_word(xb, blk, j) = word;
    if (j == 0) {
      xb.d[blk] = *reinterpret_cast<const float *>(bp);
      xb.corr[blk] = -8 * lsum;
    }
  }
}

// LPR lanes per weight row, each taking groups li, li + LPR, ... of eight
// blocks; the row's sum over its lanes.
template <int LPR>
__device__ __forceinline__ float row_dot(const uint8_t *wrow, ActBuf xb, int li, int G, bool live) {
  float acc = 0.0f;
  if (live) {
    for (int g = li; g < G; g += LPR) {
      W8S wv;
      load_w8s(wrow + (int64_t)g * (8 * Q4SB), wv);
      acc = dot8s_lds(wv, group_codes(xb, g * 8), xb.d + g * 8, xb.corr + g * 8, acc);
    }
  }
  return lane_group_sum<LPR>(acc);
}

__global__ __launch_bounds__(SNT) void sym_gateup_kernel(SymArgs a) {
  extern __shared__ __align__(16) uint8_t lds[];
  const int nbh = (int)(a.I / QK), nbx = (int)(a.H / QK), G = (int)(a.H / 256);
  const int64_t p = blockIdx.x / nbh;
  const int cb = (int)(blockIdx.x % nbh);
  int64_t tok;
  const uint8_t *W = pair_matrix(a, p, true, &tok);
  if (!W) return;                                  // uniform over the workgroup
  const ActBuf xb = act_buf(lds, nbx);
  float *vals = reinterpret_cast<float *>(lds + act_buf_bytes(nbx));   // [64]: gate, up
  // 64 rows, 4 lanes each: rows 0..31 gate columns 32cb.., rows 32..63 up
  const int r = (int)(threadIdx.x >> 2), li = (int)(threadIdx.x & 3);
  const int64_t row = r < 32 ? (int64_t)cb * 32 + r : a.I + (int64_t)cb * 32 + (r - 32);
  const int64_t rowbytes = (int64_t)nbx * Q4SB;
  stage_q8f32(xb, a.xq + tok * nbx * Q8FB, nbx);
  __syncthreads();
  const float s = row_dot<4>(W + row * rowbytes, xb, li, G, true);
  if (li == 0) vals[r] = s;
  __syncthreads();
  // SwiGLU of the 32 columns and Q8_F32 of the block: lanes 0..7, four
  // values each (same fp32 steps as the format definition)
  if (threadIdx.x < 8) {
    const int j = (int)threadIdx.x;
    float v[4];
#pragma unroll
    for (int i = 0; i < 4; i++) v[i] = silu_f32(vals[4 * j + i]) * vals[32 + 4 * j + i];
    const float amax =
        max8(fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
    const float d = amax / 127.0f;
    const float id = sym_inverse(d);
    uint32_t packed = 0;
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int q = id == 0.0f ? 0 : round_clamp(v[i] * id, 127);
      packed |= ((uint32_t)q & 0xFFu) << (8 * i);
    }
    uint8_t *blk = a.hq + (p * nbh + cb) * Q8FB;
    *reinterpret_cast<uint32_t *>(blk + 4 + 4 * j) = packed;
    if (j == 0) *reinterpret_cast<float *>(blk) = d;
    *reinterpret_cast<float4 *>(a.h + p * a.I + cb * 32 + 4 * j) = make_float4(v[0], v[1], v[2], v[3]);
  }
}

// down: SNT / LPR output rows per workgroup, against the pair's Q8_F32(h).
template <int LPR>
__global__ __launch_bounds__(SNT) void sym_down_kernel(SymArgs a, int nslab) {
  extern __shared__ __align__(16) uint8_t lds[];
  constexpr int ROWS = SNT / LPR;
  const int nbh = (int)(a.I / QK), G = (int)(a.I / 256);
  const int64_t p = blockIdx.x / nslab;
  const int slab = (int)(blockIdx.x % nslab);
  int64_t tok;
  const uint8_t *W = pair_matrix(a, p, false, &tok);
  if (!W) return;
  const ActBuf hb = act_buf(lds, nbh);
  const int r = (int)(threadIdx.x / LPR), li = (int)(threadIdx.x % LPR);
  const int64_t n = (int64_t)slab * ROWS + r;
  const bool live = n < a.H;
  stage_q8f32(hb, a.hq + p * nbh * Q8FB, nbh);
  __syncthreads();
  const int64_t rowbytes = (int64_t)nbh * Q4SB;
  const float s = row_dot<LPR>(W + (live ? n : 0) * rowbytes, hb, li, G, live);
  const int64_t pr = a.T * a.k;
  const float wt = p < pr ? a.topk_w[p] : 1.0f;
  if (live && li == 0) a.y[p * a.H + n] = wt * s;
}

// out[t] = the routed slots of token t in order (skipped ones left out),
// then the shared expert's.
__global__ __launch_bounds__(256) void sym_combine_kernel(SymArgs a, float *__restrict__ out,
                                                          int has_shared) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t h4 = a.H / 4;
  if (i >= a.T * h4) return;
  const int64_t t = i / h4, c = i % h4;
  const float4 *y4 = reinterpret_cast<const float4 *>(a.y);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int64_t j = 0; j < a.k; j++) {
    const int e = a.ids[t * a.k + j];
    if (e < 0 || e >= a.E) continue;
    const float4 v = y4[(t * a.k + j) * h4 + c];
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  if (has_shared) {
    const float4 v = y4[(a.T * a.k + t) * h4 + c];
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  reinterpret_cast<float4 *>(out)[i] = acc;
}

}  // namespace

}  // namespace w4a8

using namespace w4a8;

extern "C" size_t moe_sym_workspace_size(int64_t T, int64_t H, int64_t I, int64_t E, int64_t k) {
  if (sym_validate(T, H, I, E, k) != W4A8_OK) return 0;
  return sym_layout(T, H, I, k).total;
}

extern "C" int moe_sym_workspace_layout(int64_t T, int64_t H, int64_t I, int64_t E, int64_t k,
                                        size_t *offsets) {
  const int rc = sym_validate(T, H, I, E, k);
  if (rc != W4A8_OK) return rc;
  if (!offsets) return W4A8_ENULL;
  const SymLayout L = sym_layout(T, H, I, k);
  offsets[W4A8_SYM_WS_XQ] = L.xq;
  offsets[W4A8_SYM_WS_H] = L.h;
  offsets[W4A8_SYM_WS_HQ] = L.hq;
  return W4A8_OK;
}

extern "C" int moe_sym_forward(const float *hidden, const int32_t *topk_ids, const float *topk_w,
                               const void *w_gate_up, const void *w_down, const void *ws_gate_up,
                               const void *ws_down, float *out, int64_t T, int64_t H, int64_t I,
                               int64_t E, int64_t k, void *workspace, size_t ws_bytes,
                               void *stream) {
  int rc = sym_validate(T, H, I, E, k);
  if (rc != W4A8_OK || T == 0) return rc;
  if (!hidden || !topk_ids || !topk_w || !w_gate_up || !w_down || !out || !workspace)
    return W4A8_ENULL;
  if ((ws_gate_up == nullptr) != (ws_down == nullptr)) return W4A8_ENULL;
  if (!aligned16(hidden) || !aligned16(w_gate_up) || !aligned16(w_down) || !aligned16(out) ||
      !aligned16(workspace) || (ws_gate_up && (!aligned16(ws_gate_up) || !aligned16(ws_down))))
    return W4A8_EALIGN;
  const SymLayout L = sym_layout(T, H, I, k);
  if (ws_bytes < L.total) return W4A8_EWORKSPACE;
  if ((rc = check_device()) != W4A8_OK) return rc;
  hipStream_t s = as_stream(stream);
  uint8_t *ws = reinterpret_cast<uint8_t *>(workspace);
  if ((rc = q8_f32_quantize(hidden, ws + L.xq, T, H, stream)) != W4A8_OK) return rc;
  SymArgs a{};
  a.ids = topk_ids; a.topk_w = topk_w;
  a.w_gu = reinterpret_cast<const uint8_t *>(w_gate_up);
  a.w_d = reinterpret_cast<const uint8_t *>(w_down);
  a.ws_gu = reinterpret_cast<const uint8_t *>(ws_gate_up);
  a.ws_d = reinterpret_cast<const uint8_t *>(ws_down);
  a.xq = ws + L.xq;
  a.h = reinterpret_cast<float *>(ws + L.h);
  a.hq = ws + L.hq;
  a.y = reinterpret_cast<float *>(ws + L.y);
  a.T = T; a.H = H; a.I = I; a.E = E; a.k = k;
  const int64_t P = T * k + T;
  const size_t lds_gu = act_buf_bytes((int)(H / QK)) + 64 * sizeof(float);
  sym_gateup_kernel<<<dim3((unsigned)(P * (I / QK))), dim3(SNT), lds_gu, s>>>(a);
  if ((rc = check_launch()) != W4A8_OK) return rc;
  const size_t lds_dn = act_buf_bytes((int)(I / QK));
  if (I / 256 <= 2) {
    const int nslab = (int)((H + SNT / 2 - 1) / (SNT / 2));
    sym_down_kernel<2><<<dim3((unsigned)(P * nslab)), dim3(SNT), lds_dn, s>>>(a, nslab);
  } else {
    const int nslab = (int)((H + SNT / 4 - 1) / (SNT / 4));
    sym_down_kernel<4><<<dim3((unsigned)(P * nslab)), dim3(SNT), lds_dn, s>>>(a, nslab);
  }
  if ((rc = check_launch()) != W4A8_OK) return rc;
  const int64_t n4 = T * (H / 4);
  sym_combine_kernel<<<dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s>>>(
      a, out, ws_gate_up != nullptr);
  return check_launch();
}
