// Dense W4A8 matrix product for M > 1 activation rows (the dense per-layer
// projections and the output projection, which take about three quarters of
// the paper's decode time, Sec. 5.2, and the prefill products of Sec. 3.2):
// y[m][n] = sum_b d_w[n,b] * d_x[m,b] * s[m,n,b], s the exact int32 block
// dot of Sec. 3.3.  The rows of Q8_0 activations are first copied into the
// aligned form the int8 MFMA tiles read (32 codes on a 32-byte boundary, the
// scale as fp32 beside), then one launch of the tile kernel of mfma.hip in
// its dense mode.  One row goes to the GEMV.
#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

int mfma_dense(const uint8_t *w, const uint32_t *act, const float *actd, float *y, int64_t M,
               int64_t N, int64_t K, hipStream_t s);

namespace {

inline size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }

// Q8_0 blocks -> aligned codes and fp32 scales, 8 lanes per block (lane j
// moves codes 4j..4j+3, two 16-bit loads: the 34-byte blocks are only 2-byte
// aligned).
__global__ __launch_bounds__(256) void align_q8_0_kernel(const uint8_t *__restrict__ xq,
                                                         uint32_t *__restrict__ act,
                                                         float *__restrict__ actd,
                                                         int64_t nblocks) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t blk = t >> 3;
  const int j = (int)(t & 7);
  if (blk >= nblocks) return;
  const uint16_t *p = reinterpret_cast<const uint16_t *>(xq + blk * Q8B + 2 + 4 * j);
  act[blk * 8 + j] = (uint32_t)p[0] | ((uint32_t)p[1] << 16);
  if (j == 0) actd[blk] = f16_bits_to_f32(*reinterpret_cast<const uint16_t *>(xq + blk * Q8B));
}

int gemm_shape(int64_t M, int64_t N, int64_t K) {
  if (M < 0 || N <= 0 || K <= 0 || K % 256 != 0) return W4A8_ESHAPE;
  if (M >= ((int64_t)1 << 31) || N >= ((int64_t)1 << 31) || K > (1 << 20) ||
      M * N >= ((int64_t)1 << 40) || M * K >= ((int64_t)1 << 40))
    return W4A8_ERANGE;
  return W4A8_OK;
}

}  // namespace

}  // namespace w4a8

using namespace w4a8;

extern "C" size_t q4q8_gemm_workspace_size(int64_t M, int64_t K) {
  if (gemm_shape(M, 1, K) != W4A8_OK) return 0;
  return up256((size_t)M * K) + up256(sizeof(float) * (size_t)M * (K / 32));
}

extern "C" int q4q8_gemm(const void *w, const void *xq, float *y, int64_t M, int64_t N, int64_t K,
                         void *workspace, size_t ws_bytes, void *stream) {
  int rc = gemm_shape(M, N, K);
  if (rc != W4A8_OK) return rc;
  if (M == 0) return W4A8_OK;
  if (!w || !xq || !y) return W4A8_ENULL;
  if (!aligned16(w) || !aligned16(xq) || !aligned16(y)) return W4A8_EALIGN;
  if (M == 1) return q4q8_gemv(w, xq, y, N, K, stream);
  if (!workspace) return W4A8_ENULL;
  if (!aligned16(workspace)) return W4A8_EALIGN;
  if (ws_bytes < q4q8_gemm_workspace_size(M, K)) return W4A8_EWORKSPACE;
  if ((rc = check_device()) != W4A8_OK) return rc;
  hipStream_t s = as_stream(stream);
  uint8_t *ws = reinterpret_cast<uint8_t *>(workspace);
  uint32_t *act = reinterpret_cast<uint32_t *>(ws);
  float *actd = reinterpret_cast<float *>(ws + up256((size_t)M * K));
  const int64_t nblocks = M * (K / 32);
  align_q8_0_kernel<<<dim3((unsigned)((nblocks * 8 + 255) / 256)), dim3(256), 0, s>>>(
      reinterpret_cast<const uint8_t *>(xq), act, actd, nblocks);
  if ((rc = check_launch()) != W4A8_OK) return rc;
  return mfma_dense(reinterpret_cast<const uint8_t *>(w), act, actd, y, M, N, K, s);
}
