// The paper's own block format (Sec. 2.3: each weight an integer in {-7..7}
// with one FP32 scale per group, packed two per byte; Sec. 3.3: activations
// quantized per group to 8 bits with an FP32 scale, every 4-bit weight held
// as the unsigned value in {1..15}): quantizers and the matrix-vector product.
//
// Q4_SYM block (20 bytes): fp32 scale, then 16 payload bytes in the Q4_0
// nibble order.  Eight blocks are 160 bytes, 16-byte aligned when K % 256 == 0,
// and every scale and payload dword sits on a dword boundary, so a lane's
// group of eight blocks needs no byte realignment.  Q8_F32 block (36 bytes):
// fp32 scale, then 32 int8 codes.  The stored nibble minus 8 is the weight
// code, so the integer block dot is the one of the Q4_0 path: 4-bit dot
// products of the payload as loaded against the activation block in
// nibble-split form, staged once per workgroup in LDS.
#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int Q4SB = W4A8_Q4_SYM_BLOCK_BYTES;   // 20
constexpr int Q8FB = W4A8_Q8_F32_BLOCK_BYTES;   // 36
constexpr int SYM_K_MAX = 32768;                // the LDS staging holds the whole vector

// Eight lanes per block, lane j holding elements 4j..4j+3: amax over the 8
// lanes, one division, one reciprocal, one multiply per element.
__device__ __forceinline__ void load4(const float *__restrict__ src, int64_t blk, int j, bool live,
                                      float v[4]) {
  v[0] = v[1] = v[2] = v[3] = 0.0f;
  if (live) {
    const float4 t = reinterpret_cast<const float4 *>(src + blk * QK)[j];
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  }
}
__device__ __forceinline__ float amax8(const float v[4]) {
  return max8(fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
}

__global__ __launch_bounds__(256) void q4_sym_kernel(const float *__restrict__ w,
                                                     uint8_t *__restrict__ wq, int64_t nblocks) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t blk = tid >> 3;
  const int j = (int)(tid & 7);
  const bool live = blk < nblocks;
  float v[4];
  load4(w, blk, j, live, v);
  const float d = amax8(v) / 7.0f;
  const float id = sym_inverse(d);
  uint32_t nib = 0;   // four stored nibbles q + 8, element i in byte i
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const int q = id == 0.0f ? 0 : round_clamp(v[i] * id, 7);
    nib |= (uint32_t)(q + 8) << (8 * i);
  }
  const uint32_t hi = __shfl_xor(nib, 4, 8);    // lanes 4..7 hold elements 16..31
  if (live && j < 4) {
    uint8_t *b = wq + blk * Q4SB;
    *reinterpret_cast<uint32_t *>(b + 4 + 4 * j) = nib | (hi << 4);
    if (j == 0) *reinterpret_cast<float *>(b) = d;
  }
}

__global__ __launch_bounds__(256) void q8_f32_kernel(const float *__restrict__ x,
                                                     uint8_t *__restrict__ xq, int64_t nblocks) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t blk = tid >> 3;
  const int j = (int)(tid & 7);
  const bool live = blk < nblocks;
  float v[4];
  load4(x, blk, j, live, v);
  const float d = amax8(v) / 127.0f;
  const float id = sym_inverse(d);
  uint32_t packed = 0;
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const int q = id == 0.0f ? 0 : round_clamp(v[i] * id, 127);
    packed |= ((uint32_t)q & 0xFFu) << (8 * i);
  }
  if (live) {
    uint8_t *b = xq + blk * Q8FB;
    *reinterpret_cast<uint32_t *>(b + 4 + 4 * j) = packed;
    if (j == 0) *reinterpret_cast<float *>(b) = d;
  }
}

// LPR lanes share a row (one 160-byte group of eight blocks per lane at a
// time); the activation vector is staged once per workgroup in nibble-split
// form after the lane's first weight group has been issued.
template <int LPR>
__global__ __launch_bounds__(256) void gemv_sym_kernel(const uint8_t *__restrict__ w,
                                                       const uint8_t *__restrict__ xq,
                                                       float *__restrict__ y, int64_t N, int G) {
  extern __shared__ __align__(16) uint8_t lds[];
  constexpr int RPW = 64 / LPR;
  const int nb = G * 8;
  const ActBuf xb = act_buf(lds, nb);
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const int64_t row = wave * RPW + lane / LPR;
  const int li = lane % LPR;
  const bool live = row < N && li < G;
  const int64_t rowbytes = (int64_t)nb * Q4SB;
  const uint8_t *wrow = w + (live ? row : 0) * rowbytes;
  W8S wv;
  load_w8s(wrow + (int64_t)(live ? li : 0) * (8 * Q4SB), wv);
  for (int t = threadIdx.x; t < nb * 8; t += blockDim.x) {   // whole 8-lane groups
    const int blk = t >> 3, j = t & 7;
    const uint8_t *bp = xq + (int64_t)blk * Q8FB;
    const uint32_t packed = *reinterpret_cast<const uint32_t *>(bp + 4 + 4 * j);
    const uint32_t word = split_word(packed, j);
    const int lsum = sum8(low_nibble_sum(packed));
    *code_word(xb, blk, j) = word;
    if (j == 0) {
      xb.d[blk] = *reinterpret_cast<const float *>(bp);
      xb.corr[blk] = -8 * lsum;
    }
  }
  __syncthreads();
  float acc = 0.0f;
  if (live) {
    acc = dot8s_lds(wv, group_codes(xb, li * 8), xb.d + li * 8, xb.corr + li * 8, acc);
    for (int g = li + LPR; g < G; g += LPR) {
      load_w8s(wrow + (int64_t)g * (8 * Q4SB), wv);
      acc = dot8s_lds(wv, group_codes(xb, g * 8), xb.d + g * 8, xb.corr + g * 8, acc);
    }
  }
  acc = lane_group_sum<LPR>(acc);
  if (row < N && li == 0) y[row] = acc;
}

template <int LPR>
void launch_gemv_sym(const uint8_t *w, const uint8_t *xq, float *y, int64_t N, int G,
                     hipStream_t s) {
  constexpr int RPW = 64 / LPR;
  const int64_t waves = (N + RPW - 1) / RPW;
  const int64_t grid = (waves + 3) / 4;
  gemv_sym_kernel<LPR><<<dim3((unsigned)grid), dim3(256), act_buf_bytes(G * 8), s>>>(w, xq, y,
                                                                                    N, G);
}

int quant_sym_args(const void *in, const void *out, int64_t rows, int64_t K) {
  if (!in || !out) return W4A8_ENULL;
  if (rows < 0 || K <= 0 || K % QK != 0) return W4A8_ESHAPE;
  if (rows > 0 && rows * (K / QK) >= ((int64_t)1 << 36)) return W4A8_ERANGE;
  if (!aligned16(in) || !aligned16(out)) return W4A8_EALIGN;
  return W4A8_OK;
}

}  // namespace

}  // namespace w4a8

using namespace w4a8;

extern "C" int q4_sym_quantize(const float *w, void *wq, int64_t rows, int64_t K, void *stream) {
  int rc = quant_sym_args(w, wq, rows, K);
  if (rc != W4A8_OK || rows == 0) return rc;
  if ((rc = check_device()) != W4A8_OK) return rc;
  const int64_t nblocks = rows * (K / QK);
  q4_sym_kernel<<<dim3((unsigned)((nblocks * 8 + 255) / 256)), dim3(256), 0, as_stream(stream)>>>(
      w, reinterpret_cast<uint8_t *>(wq), nblocks);
  return check_launch();
}

extern "C" int q8_f32_quantize(const float *x, void *xq, int64_t rows, int64_t K, void *stream) {
  int rc = quant_sym_args(x, xq, rows, K);
  if (rc != W4A8_OK || rows == 0) return rc;
  if ((rc = check_device()) != W4A8_OK) return rc;
  const int64_t nblocks = rows * (K / QK);
  q8_f32_kernel<<<dim3((unsigned)((nblocks * 8 + 255) / 256)), dim3(256), 0, as_stream(stream)>>>(
      x, reinterpret_cast<uint8_t *>(xq), nblocks);
  return check_launch();
}

extern "C" int q4sym_q8f32_gemv(const void *w, const void *xq, float *y, int64_t N, int64_t K,
                                void *stream) {
  if (!w || !xq || !y) return W4A8_ENULL;
  if (N <= 0 || K <= 0 || K % 256 != 0) return W4A8_ESHAPE;
  if (K > SYM_K_MAX || N >= ((int64_t)1 << 36)) return W4A8_ERANGE;
  if (!aligned16(w) || !aligned16(xq) || !aligned16(y)) return W4A8_EALIGN;
  int rc = check_device();
  if (rc != W4A8_OK) return rc;
  const uint8_t *wb = reinterpret_cast<const uint8_t *>(w);
  const uint8_t *xb = reinterpret_cast<const uint8_t *>(xq);
  const hipStream_t s = as_stream(stream);
  const int G = (int)(K / 256);
  int lpr = 1;
  while (lpr * 2 <= G && lpr < 64) lpr *= 2;
  switch (lpr) {
    case 1: launch_gemv_sym<1>(wb, xb, y, N, G, s); break;
    case 2: launch_gemv_sym<2>(wb, xb, y, N, G, s); break;
    case 4: launch_gemv_sym<4>(wb, xb, y, N, G, s); break;
    case 8: launch_gemv_sym<8>(wb, xb, y, N, G, s); break;
    case 16: launch_gemv_sym<16>(wb, xb, y, N, G, s); break;
    case 32: launch_gemv_sym<32>(wb, xb, y, N, G, s); break;
    default: launch_gemv_sym<64>(wb, xb, y, N, G, s); break;
  }
  return check_launch();
}
