// Q8_0 activation and Q4_0 weight quantizers (paper Sec. 3.3: activations
// quantized per group to 8 bits with a scale; Sec. 2.3: group-wise symmetric
// 4-bit weights, two per byte, one scale per group), plus the workspace fill.
//
// Eight lanes own one 32-element block, four elements each, so a wave reads
// 1 KB of fp32 input per instruction fully coalesced.  The 34- and 18-byte
// output blocks are only 2-byte aligned, so they are written with 16-bit
// stores.
#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

// 8 lanes per block (q8_0_lane).
__global__ __launch_bounds__(256) void q8_0_kernel(const float *__restrict__ x,
                                                   uint8_t *__restrict__ xq, int64_t nblocks) {
  q8_0_lane(x, xq, nullptr, nullptr, nullptr, nblocks, 1,
            (int64_t)blockIdx.x * blockDim.x + threadIdx.x);
}

__global__ __launch_bounds__(256) void q4_0_kernel(const float *__restrict__ w,
                                                   uint8_t *__restrict__ wq, int64_t nblocks) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t blk = tid >> 3;
  const int j = (int)(tid & 7);
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  const bool live = blk < nblocks;
  if (live) {
    const float4 t = reinterpret_cast<const float4 *>(w + blk * QK)[j];
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  }
  // signed element of largest magnitude, first index on ties
  float amax = 0.0f, m = 0.0f;
  int idx = 4 * j;
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const float a = fabsf(v[i]);
    if (a > amax) { amax = a; m = v[i]; idx = 4 * j + i; }
  }
#pragma unroll
  for (int o = 4; o > 0; o >>= 1) {
    const float a2 = __shfl_xor(amax, o, 8);
    const float m2 = __shfl_xor(m, o, 8);
    const int i2 = __shfl_xor(idx, o, 8);
    if (a2 > amax || (a2 == amax && i2 < idx)) { amax = a2; m = m2; idx = i2; }
  }
  const float d32 = m / -8.0f;
  const uint32_t d16 = f32_to_f16_bits(d32);
  const float df = f16_bits_to_f32(d16);
  const float id = (df != 0.0f) ? 1.0f / df : 0.0f;
  uint32_t codes = 0;  // four 4-bit codes, element i in byte i
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const float p = v[i] * id;      // one fp32 multiply (no contraction)
    const float s = p + 8.5f;       // one fp32 add
    int q = (int)floorf(s);
    q = q > 15 ? 15 : (q < 0 ? 0 : q);
    codes |= (uint32_t)q << (8 * i);
  }
  const uint32_t hi = __shfl_xor(codes, 4, 8);  // lanes 4..7 hold elements 16..31
  if (live && j < 4) {
    const uint32_t bytes = codes | (hi << 4);
    uint16_t *p = reinterpret_cast<uint16_t *>(wq + blk * Q4B + 2 + 4 * j);
    p[0] = (uint16_t)(bytes & 0xFFFFu);
    p[1] = (uint16_t)(bytes >> 16);
    if (j == 0) *reinterpret_cast<uint16_t *>(wq + blk * Q4B) = (uint16_t)d16;
  }
}

__global__ __launch_bounds__(256) void fill_zero_kernel(uint4 *__restrict__ p, int64_t n16,
                                                        uint8_t *__restrict__ tail, int ntail) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n16) p[i] = make_uint4(0u, 0u, 0u, 0u);
  if (i < ntail) tail[i] = 0;
}

int launch_fill_zero(void *ptr, size_t bytes, hipStream_t s) {
  const int64_t n16 = (int64_t)(bytes / 16);
  const int ntail = (int)(bytes % 16);
  const int64_t n = n16 > ntail ? n16 : ntail;
  if (n == 0) return W4A8_OK;
  const int64_t grid = (n + 255) / 256;
  fill_zero_kernel<<<dim3((unsigned)grid), dim3(256), 0, s>>>(
      reinterpret_cast<uint4 *>(ptr), n16, reinterpret_cast<uint8_t *>(ptr) + n16 * 16, ntail);
  return check_launch();
}

int launch_q8_0(const float *x, uint8_t *xq, int64_t nblocks, hipStream_t s) {
  if (nblocks == 0) return W4A8_OK;
  const int64_t grid = (nblocks * 8 + 255) / 256;
  q8_0_kernel<<<dim3((unsigned)grid), dim3(256), 0, s>>>(x, xq, nblocks);
  return check_launch();
}

}  // namespace w4a8

using namespace w4a8;

static int quant_args(const void *in, const void *out, int64_t rows, int64_t K) {
  if (!in || !out) return W4A8_ENULL;
  if (rows < 0 || K <= 0 || K % QK != 0) return W4A8_ESHAPE;
  if (rows > 0 && rows * (K / QK) >= ((int64_t)1 << 36)) return W4A8_ERANGE;
  if (!aligned16(in) || !aligned16(out)) return W4A8_EALIGN;
  return W4A8_OK;
}

extern "C" int q8_0_quantize(const float *x, void *xq, int64_t rows, int64_t K, void *stream) {
  int rc = quant_args(x, xq, rows, K);
  if (rc != W4A8_OK) return rc;
  if (rows == 0) return W4A8_OK;
  if ((rc = check_device()) != W4A8_OK) return rc;
  return launch_q8_0(x, reinterpret_cast<uint8_t *>(xq), rows * (K / QK), as_stream(stream));
}

extern "C" int q4_0_quantize(const float *w, void *wq, int64_t rows, int64_t K, void *stream) {
  int rc = quant_args(w, wq, rows, K);
  if (rc != W4A8_OK) return rc;
  if (rows == 0) return W4A8_OK;
  if ((rc = check_device()) != W4A8_OK) return rc;
  const int64_t nblocks = rows * (K / QK);
  const int64_t grid = (nblocks * 8 + 255) / 256;
  q4_0_kernel<<<dim3((unsigned)grid), dim3(256), 0, as_stream(stream)>>>(
      w, reinterpret_cast<uint8_t *>(wq), nblocks);
  return check_launch();
}
