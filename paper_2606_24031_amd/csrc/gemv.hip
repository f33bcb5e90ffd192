// W4A8 matrix-vector product (paper Sec. 3.3: 4-bit weight codes times 8-bit
// activation codes as integer multiply-adds, one scaling per 32-block).
//
// HBM-bound streaming kernel.  A lane owns one "group" of eight consecutive
// Q4_0 blocks of a row (144 bytes, 16-byte aligned because K % 256 == 0),
// loads it with nine 16-byte loads, unpacks the nibbles in registers and takes
// the eight int32 block dots with v_dot4_i32_i8 against the Q8_0 activation
// group held in registers.  LPR lanes share a row (LPR = groups per row, up to
// 64) and reduce with cross-lane shuffles; a wave covers 64/LPR rows.
#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

template <int LPR>
__global__ __launch_bounds__(256) void gemv_kernel(const uint8_t *__restrict__ w,
                                                   const uint8_t *__restrict__ xq,
                                                   float *__restrict__ y, int64_t N, int G,
                                                   int64_t rowbytes) {
  constexpr int RPW = 64 / LPR;  // rows per wave
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const int64_t row = wave * RPW + lane / LPR;
  const int li = lane % LPR;
  float acc = 0.0f;
  if (row < N) {
    for (int g = li; g < G; g += LPR) {
      W8 wv;
      load_w8(w + row * rowbytes + (int64_t)g * (8 * Q4B), wv);
      Act8 a;
      load_act8(xq + (int64_t)g * (8 * Q8B), a);
      acc = dot8(wv, a, acc);
    }
  }
  acc = lane_group_sum<LPR>(acc);
  if (row < N && li == 0) y[row] = acc;
}

// The same product with the activation staged once per workgroup in LDS,
// in nibble-split form (8 lanes per Q8_0 block convert the 34-byte block),
// so a lane's block dots read it from LDS with 4-bit dot products against
// its weight group as loaded (dot8_lds), instead of each lane loading and
// unpacking its 272 bytes of Q8_0 blocks.  The first weight group is issued
// before the staging.
template <int LPR>
__global__ __launch_bounds__(256) void gemv_lds_kernel(const uint8_t *__restrict__ w,
                                                       const uint8_t *__restrict__ xq,
                                                       float *__restrict__ y, int64_t N, int G,
                                                       int64_t rowbytes) {
  extern __shared__ __align__(16) uint8_t lds[];
  constexpr int RPW = 64 / LPR;
  const int nb = G * 8;
  const ActBuf xb = act_buf(lds, nb);
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const int64_t row = wave * RPW + lane / LPR;
  const int li = lane % LPR;
  const bool live = row < N && li < G;
  const uint8_t *wrow = w + (live ? row : 0) * rowbytes;
  W8 wv;
  load_w8(wrow + (int64_t)(live ? li : 0) * (8 * Q4B), wv);
  for (int t = threadIdx.x; t < nb * 8; t += blockDim.x) {   // whole 8-lane groups
    const int blk = t >> 3, j = t & 7;
    const uint16_t *bp = reinterpret_cast<const uint16_t *>(xq + (int64_t)blk * Q8B);
    const uint32_t packed = (uint32_t)bp[1 + 2 * j] | ((uint32_t)bp[2 + 2 * j] << 16);
    const uint32_t word = split_word(packed, j);
    const int lsum = sum8(low_nibble_sum(packed));
    *code_word(xb, blk, j) = word;
    if (j == 0) {
      xb.d[blk] = f16_bits_to_f32(bp[0]);
      xb.corr[blk] = -8 * lsum;
    }
  }
  __syncthreads();
  float acc = 0.0f;
  if (live) {
    acc = dot8_lds(wv, group_codes(xb, li * 8), xb.d + li * 8, xb.corr + li * 8, acc);
    for (int g = li + LPR; g < G; g += LPR) {
      load_w8(wrow + (int64_t)g * (8 * Q4B), wv);
      acc = dot8_lds(wv, group_codes(xb, g * 8), xb.d + g * 8, xb.corr + g * 8, acc);
    }
  }
  acc = lane_group_sum<LPR>(acc);
  if (row < N && li == 0) y[row] = acc;
}

constexpr size_t GEMV_LDS_MAX = 48 * 1024;

template <int LPR>
static void launch_gemv(const uint8_t *w, const uint8_t *xq, float *y, int64_t N, int G,
                        hipStream_t s) {
  constexpr int RPW = 64 / LPR;
  const int64_t waves = (N + RPW - 1) / RPW;
  const int64_t grid = (waves + 3) / 4;
  const size_t lds = act_buf_bytes(G * 8);
  if (lds <= GEMV_LDS_MAX)
    gemv_lds_kernel<LPR><<<dim3((unsigned)grid), dim3(256), lds, s>>>(w, xq, y, N, G,
                                                                      (int64_t)G * 8 * Q4B);
  else
    gemv_kernel<LPR><<<dim3((unsigned)grid), dim3(256), 0, s>>>(w, xq, y, N, G,
                                                                 (int64_t)G * 8 * Q4B);
}

int gemv_dispatch(const uint8_t *w, const uint8_t *xq, float *y, int64_t N, int64_t K,
                  hipStream_t s) {
  const int G = (int)(K / 256);
  int lpr = 1;
  while (lpr * 2 <= G && lpr < 64) lpr *= 2;
  switch (lpr) {
    case 1: launch_gemv<1>(w, xq, y, N, G, s); break;
    case 2: launch_gemv<2>(w, xq, y, N, G, s); break;
    case 4: launch_gemv<4>(w, xq, y, N, G, s); break;
    case 8: launch_gemv<8>(w, xq, y, N, G, s); break;
    case 16: launch_gemv<16>(w, xq, y, N, G, s); break;
    case 32: launch_gemv<32>(w, xq, y, N, G, s); break;
    default: launch_gemv<64>(w, xq, y, N, G, s); break;
  }
  return check_launch();
}

}  // namespace w4a8

using namespace w4a8;

extern "C" int q4q8_gemv(const void *w, const void *xq, float *y, int64_t N, int64_t K,
                         void *stream) {
  if (!w || !xq || !y) return W4A8_ENULL;
  if (N <= 0 || K <= 0 || K % 256 != 0) return W4A8_ESHAPE;
  if (K / 256 >= ((int64_t)1 << 24) || N >= ((int64_t)1 << 36)) return W4A8_ERANGE;
  if (!aligned16(w) || !aligned16(xq) || !aligned16(y)) return W4A8_EALIGN;
  int rc = check_device();
  if (rc != W4A8_OK) return rc;
  return gemv_dispatch(reinterpret_cast<const uint8_t *>(w),
                       reinterpret_cast<const uint8_t *>(xq), y, N, K, as_stream(stream));
}
