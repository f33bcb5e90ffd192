// The routed + shared MoE layer in the paper's own block format (Sec. 2.2:
// top-k routed experts plus one always-on shared expert; Sec. 2.3: weights
// in {-7..7} with an FP32 scale per group; Sec. 3.3: activations quantized
// per group to 8 bits with an FP32 scale, integer block dots, one scaling
// per group).  Two launches:
//   1. gate/up: one workgroup per (pair, 32-column block of h): Q8_F32 of the
//      pair's token row into LDS (the format's fp32 steps, as the quantizer
//      of sym.hip), its 32 gate and 32 up rows against it, four lanes per
//      row, then SwiGLU and Q8_F32 of the 32 values of h in the workgroup;
//      T more workgroups write the documented Q8_F32 copy of each row;
//   2. down and combine: one workgroup per (token, slab of output rows)
//      takes the slab's rows of every pair of the token against the pair's
//      Q8_F32(h), scales them by the pair's routing weight and sums the
//      routed slots in order, then the shared one.
// (When a token's Q8_F32(h) does not fit LDS, down per (pair, slab) and a
// separate combine launch instead.)
// The activations of a workgroup sit in LDS in nibble-split form (as in the
// GEMV of this format), so the block dots are the 4-bit dot products of the
// Q4_0 path on the stored nibbles.
#include <algorithm>

#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int Q4SB = W4A8_Q4_SYM_BLOCK_BYTES;   // 20
constexpr int Q8FB = W4A8_Q8_F32_BLOCK_BYTES;   // 36
constexpr int SNT = 256;
constexpr int64_t SYM_LAYER_K_MAX = 16384;      // H, I: the staged activation row fits LDS
constexpr size_t SYM_DC_LDS_MAX = 48 * 1024;    // LDS of the fused down + combine workgroup

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
  if (P * (I / QK) + T >= ((int64_t)1 << 31) || P * (H / 64) >= ((int64_t)1 << 31))
    return W4A8_ERANGE;
  return W4A8_OK;
}

struct SymArgs {
  const float *x;        // [T][H] hidden
  const int32_t *ids;
  const float *topk_w;
  const uint8_t *w_gu, *w_d, *ws_gu, *ws_d;
  uint8_t *xq;           // [T][H/32] Q8_F32 (written by the gate/up launch)
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

// Q8_F32 of one fp32 row of nb 32-blocks (8 lanes per block, 4 values
// each; the format's steps: amax, one division by 127, the scale's inverse,
// round half away from zero, clamp) into the nibble-split buffer, and with
// q (not null) as 36-byte blocks.  nb * 8 is a multiple of 64 (H % 256 ==
// 0), so whole 8-lane groups are active.
__device__ __forceinline__ void quantize_q8f32_row(const float *x, ActBuf xb, int nb,
                                                   uint8_t *q) {
  for (int t = threadIdx.x; t < nb * 8; t += blockDim.x) {
    const int blk = t >> 3, j = t & 7;
    const float4 x4 = reinterpret_cast<const float4 *>(x)[t];
    const float v[4] = {x4.x, x4.y, x4.z, x4.w};
    const float amax =
        max8(fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
    const float d = amax / 127.0f;
    const float id = sym_inverse(d);
    uint32_t packed = 0;
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int c = id == 0.0f ? 0 : round_clamp(v[i] * id, 127);
      packed |= ((uint32_t)c & 0xFFu) << (8 * i);
    }
    const int lsum = sum8(low_nibble_sum(packed));
    if (xb.codes) {
      *code_word(xb, blk, j) = split_word(packed, j);
      if (j == 0) {
        xb.d[blk] = d;
        xb.corr[blk] = -8 * lsum;
      }
    }
    if (q) {
      uint8_t *bp = q + (int64_t)blk * Q8FB;
      *reinterpret_cast<uint32_t *>(bp + 4 + 4 * j) = packed;
      if (j == 0) *reinterpret_cast<float *>(bp) = d;
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

// The lane's first two groups of a row (li and li + LPR, clamped to the
// row: no conditional loads into registers), issued before the activations
// are staged so that their round trip overlaps the staging.
template <int LPR>
__device__ __forceinline__ void row_pre(const uint8_t *wrow, int li, int G, W8S &p0, W8S &p1) {
  load_w8s(wrow + (int64_t)min(li, G - 1) * (8 * Q4SB), p0);
  load_w8s(wrow + (int64_t)min(li + LPR, G - 1) * (8 * Q4SB), p1);
}
// row_dot with the first two groups preloaded (the same groups in the same
// order, so the same sum).
template <int LPR>
__device__ __forceinline__ float row_dot_pre(const uint8_t *wrow, ActBuf xb, int li, int G,
                                             bool live, const W8S &p0, const W8S &p1) {
  float acc = 0.0f;
  if (live) {
    if (li < G) acc = dot8s_lds(p0, group_codes(xb, li * 8), xb.d + li * 8, xb.corr + li * 8, acc);
    const int g1 = li + LPR;
    if (g1 < G) acc = dot8s_lds(p1, group_codes(xb, g1 * 8), xb.d + g1 * 8, xb.corr + g1 * 8, acc);
    for (int g = li + 2 * LPR; g < G; g += LPR) {
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
  const int64_t P = a.T * a.k + a.T;
  if ((int64_t)blockIdx.x >= P * nbh) {
    // the documented Q8_F32 copy of token row blockIdx.x - P * nbh
    const int64_t t = (int64_t)blockIdx.x - P * nbh;
    quantize_q8f32_row(a.x + t * a.H, ActBuf{nullptr, nullptr, nullptr}, nbx,
                       a.xq + t * nbx * Q8FB);
    return;
  }
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
  W8S p0, p1;
  row_pre<4>(W + row * rowbytes, li, G, p0, p1);
  quantize_q8f32_row(a.x + tok * a.H, xb, nbx, nullptr);
  __syncthreads();
  const float s = row_dot_pre<4>(W + row * rowbytes, xb, li, G, true, p0, p1);
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

// Pair slot q of token t (q == k: the shared pair): its weight in the
// combine, or false when the slot is skipped or there is no shared expert.
__device__ __forceinline__ bool slot_live(const SymArgs &a, int64_t t, int q, int has_shared,
                                          float *wt) {
  if (q < a.k) {
    const int e = a.ids[t * a.k + q];
    *wt = a.topk_w[t * a.k + q];
    return e >= 0 && e < a.E;
  }
  *wt = 1.0f;
  return has_shared != 0;
}

// The view of pair slot q's blocks in a buffer that holds nbh blocks per
// slot (nbh a multiple of 8: whole code groups).
__device__ __forceinline__ ActBuf slot_view(ActBuf b, int q, int nbh) {
  ActBuf v;
  v.codes = b.codes + (size_t)(q * nbh / 8) * GROUP_U4;
  v.d = b.d + q * nbh;
  v.corr = b.corr + q * nbh;
  return v;
}

// Down and combine of one token: workgroup (token t, slab of R output rows).
// Every pair's Q8_F32(h) of the token is staged in LDS; unit (slot q, row r)
// takes LPR lanes (groups li, li + LPR, ... as row_dot) and leaves
// w_q * (its sum) in yv[q][r]; then out[t][n] is the sum of the routed slots
// in order and then the shared one (the combine kernel's order and fp32
// steps).
template <int LPR>
__global__ __launch_bounds__(SNT) void sym_down_combine_kernel(SymArgs a, float *__restrict__ out,
                                                               int R, int nslab,
                                                               int has_shared) {
  extern __shared__ __align__(16) uint8_t lds[];
  const int nbh = (int)(a.I / QK), G = (int)(a.I / 256);
  const int np = (int)a.k + 1;
  const int64_t t = blockIdx.x / nslab;
  const int slab = (int)(blockIdx.x % nslab);
  const ActBuf hb = act_buf(lds, np * nbh);
  float *yv = reinterpret_cast<float *>(lds + act_buf_bytes(np * nbh));   // [np][R]
  const int rpw = SNT / LPR;                  // units per pass
  const int rl = (int)(threadIdx.x / LPR), li = (int)(threadIdx.x % LPR);
  const int64_t rowbytes = (int64_t)nbh * Q4SB;
  // unit u: slot u / R, row u % R; its weight row (the matrix base when the
  // unit has none)
  auto unit = [&](int u, float &wt, bool &live) -> const uint8_t * {
    const int q = u / R, r = u - q * R;
    const int64_t n = (int64_t)slab * R + r;
    wt = 0.0f;
    live = u < np * R && n < a.H && slot_live(a, t, q, has_shared, &wt);
    const uint8_t *W = nullptr;
    if (live) {
      int64_t tok;
      W = pair_matrix(a, q < a.k ? t * a.k + q : a.T * a.k + t, false, &tok);
      live = W != nullptr;
    }
    return live ? W + n * rowbytes : a.w_d;
  };
  // the first pass's weights, issued before the staging
  float wt0;
  bool live0;
  const uint8_t *w0 = unit(rl, wt0, live0);
  W8S p0, p1;
  row_pre<LPR>(w0, li, G, p0, p1);
  for (int q = 0; q < np; q++) {
    float wt;
    if (!slot_live(a, t, q, has_shared, &wt)) continue;             // uniform
    const int64_t p = q < a.k ? t * a.k + q : a.T * a.k + t;
    stage_q8f32(slot_view(hb, q, nbh), a.hq + p * nbh * Q8FB, nbh);
  }
  __syncthreads();
  {
    const float s = row_dot_pre<LPR>(w0, slot_view(hb, live0 ? rl / R : 0, nbh), li, G, live0,
                                     p0, p1);
    if (li == 0 && rl < np * R) yv[rl] = live0 ? wt0 * s : 0.0f;
  }
  for (int u0 = rpw; u0 < np * R; u0 += rpw) {
    const int u = u0 + rl;
    float wt;
    bool live;
    const uint8_t *W = unit(u, wt, live);
    const float s = row_dot<LPR>(W, slot_view(hb, live ? u / R : 0, nbh), li, G, live);
    if (li == 0 && u < np * R) yv[u] = live ? wt * s : 0.0f;
  }
  __syncthreads();
  for (int r = threadIdx.x; r < R; r += SNT) {
    const int64_t n = (int64_t)slab * R + r;
    if (n >= a.H) continue;
    float o = 0.0f;
    for (int q = 0; q < np; q++) {
      float wt;
      if (slot_live(a, t, q, has_shared, &wt)) o += yv[q * R + r];
    }
    out[t * a.H + n] = o;
  }
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
  SymArgs a{};
  a.x = hidden;
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
  // the pairs' workgroups, then one per token row for the documented Q8_F32 copy
  sym_gateup_kernel<<<dim3((unsigned)(P * (I / QK) + T)), dim3(SNT), lds_gu, s>>>(a);
  if ((rc = check_launch()) != W4A8_OK) return rc;
  // down and combine in one launch when a token's Q8_F32(h) fits LDS
  const int np = (int)k + 1;
  const int lpr = I / 256 <= 2 ? 2 : 4;
  const int R = std::max(1, (SNT / lpr) / np);
  const int64_t nslab_dc = (H + R - 1) / R;
  const size_t lds_dc = act_buf_bytes(np * (int)(I / QK)) + sizeof(float) * (size_t)np * R;
  if (lds_dc <= SYM_DC_LDS_MAX && T * nslab_dc < ((int64_t)1 << 31)) {
    const dim3 grid((unsigned)(T * nslab_dc));
    const int hs = ws_gate_up != nullptr;
    if (lpr == 2)
      sym_down_combine_kernel<2><<<grid, dim3(SNT), lds_dc, s>>>(a, out, R, (int)nslab_dc, hs);
    else
      sym_down_combine_kernel<4><<<grid, dim3(SNT), lds_dc, s>>>(a, out, R, (int)nslab_dc, hs);
    return check_launch();
  }
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
