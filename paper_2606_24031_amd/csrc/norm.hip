// Residual add and RMSNorm between chained MoE layers: the pre-norm chaining
// of the Qwen3-series model family (Sec. 2.2); the paper does not spell the
// norm out, so it is the standard RMSNorm.
//
// One workgroup per row: x_out = x + y in one fp32 add per element, the sum
// of squares in a fixed order (per thread in index order, then a fixed
// butterfly per wave and the waves in order), then
// xn = x_out * (1 / sqrt(sum / H + eps)) * gamma.  16-byte accesses.
#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int NT = 256;

// x_out may alias x (in-place residual add): no restrict on x, y, xo.
__global__ __launch_bounds__(NT) void rmsnorm_kernel(const float4 *x, const float4 *y,
                                                     const float4 *__restrict__ gamma, float4 *xo,
                                                     float4 *__restrict__ xn, int64_t H4, float eps) {
  __shared__ float wsum[NT / 64];
  const int64_t row = blockIdx.x;
  const float4 *xr = x + row * H4;
  float4 *vo = xo + row * H4;
  float ss = 0.0f;
  for (int64_t i = threadIdx.x; i < H4; i += NT) {
    float4 v = xr[i];
    if (y) {
      const float4 d = y[row * H4 + i];
      v.x += d.x; v.y += d.y; v.z += d.z; v.w += d.w;
    }
    vo[i] = v;
    ss = fmaf(v.x, v.x, ss);
    ss = fmaf(v.y, v.y, ss);
    ss = fmaf(v.z, v.z, ss);
    ss = fmaf(v.w, v.w, ss);
  }
  if (!xn) return;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.0f;
#pragma unroll
  for (int w = 0; w < NT / 64; w++) tot += wsum[w];
  const float r = 1.0f / sqrtf(tot / (float)(H4 * 4) + eps);
  for (int64_t i = threadIdx.x; i < H4; i += NT) {
    const float4 v = vo[i], g = gamma[i];
    xn[row * H4 + i] = make_float4(v.x * r * g.x, v.y * r * g.y, v.z * r * g.z, v.w * r * g.w);
  }
}

}  // namespace

int launch_rmsnorm(const float *x, const float *y, const float *gamma, float *x_out, float *xn,
                   int64_t T, int64_t H, float eps, hipStream_t s) {
  rmsnorm_kernel<<<dim3((unsigned)T), dim3(NT), 0, s>>>(
      reinterpret_cast<const float4 *>(x), reinterpret_cast<const float4 *>(y),
      reinterpret_cast<const float4 *>(gamma), reinterpret_cast<float4 *>(x_out),
      reinterpret_cast<float4 *>(xn), H / 4, eps);
  return check_launch();
}

}  // namespace w4a8

extern "C" int rmsnorm_residual(const float *x, const float *y, const float *gamma, float *x_out,
                                float *xn, int64_t T, int64_t H, float eps, void *stream) {
  using namespace w4a8;
  if (!x || !x_out || (xn && !gamma)) return W4A8_ENULL;
  if (T < 0 || H <= 0 || H % 4 != 0 || !(eps >= 0.0f)) return W4A8_ESHAPE;
  if (T >= ((int64_t)1 << 31)) return W4A8_ERANGE;
  if (!aligned16(x) || !aligned16(y) || !aligned16(gamma) || !aligned16(x_out) || !aligned16(xn))
    return W4A8_EALIGN;
  if (T == 0) return W4A8_OK;
  if (int rc = check_device(); rc != W4A8_OK) return rc;
  return launch_rmsnorm(x, y, gamma, x_out, xn, T, H, eps, as_stream(stream));
}
