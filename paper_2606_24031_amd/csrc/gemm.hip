// Dense W4A8 matrix product for M > 1 activation rows (the dense per-layer
// projections and the output projection, which take about three quarters of
// the paper's decode time, Sec. 5.2, and the prefill products of Sec. 3.2):
// y[m][n] = sum_b d_w[n,b] * d_x[m,b] * s[m,n,b], s the exact int32 block
// dot of Sec. 3.3.  The rows of Q8_0 activations are first copied into the
// aligned form the int8 MFMA tiles read (32 codes on a 32-byte boundary, the
// scale as fp32 beside), then one launch of the tile kernel of mfma.hip in
// its dense mode.  One row goes to the GEMV; a few rows (see dense_small) to
// the VALU kernel of the small expert groups, in nibble-split form.
#include <algorithm>

#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

int mfma_dense(const uint8_t *w, const uint32_t *act, const float *actd, float *y, int64_t M,
               int64_t N, int64_t K, hipStream_t s);
bool small_supported(int64_t H, int64_t I);
int small_dense(const uint8_t *w, const uint8_t *act, const int32_t *meta, const int32_t *perm,
                const int4 *chunks, float *y, int64_t M, int64_t N, int64_t K, hipStream_t s);

// Up to 128 rows (K <= 2048) run on the small-group VALU kernel: its
// workgroups keep every weight load in flight at once, where the matrix-core
// tiles of a handful of rows stream the weights one group of eight blocks at
// a time over few workgroups (32 and 64 rows over 2048 x 2048: 14.7 and 14.7
// us against 14.6-15.3 and 22.7 on the tiles; 128 rows 20.7 against 23.1).
// Each chunk of 8 rows reads the whole weight matrix, so only while the
// weights times the chunks stay small (the re-reads then come from the
// caches): the output projection of 151936 x 2048 (175 MB) took 224 us
// against 60 at 32 rows and 66 against 43 at 8 rows.
constexpr int64_t DENSE_SMALL_M = 128;
constexpr int64_t DENSE_SMALL_REREAD = (int64_t)64 << 20;   // bytes of weights x chunks
inline bool dense_small_ws(int64_t M, int64_t K) {           // the workspace may need it
  return M <= DENSE_SMALL_M && small_supported(K, 256);
}
inline bool dense_small(int64_t M, int64_t N, int64_t K) {
  if (!dense_small_ws(M, K)) return false;
  const int64_t chunks = (M + SMALL_CHUNK - 1) / SMALL_CHUNK;
  return N * (K / 32) * Q4B * chunks <= DENSE_SMALL_REREAD;
}

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

// Q8_0 rows -> the small-group kernel's nibble-split rows (8 lanes per
// block, lane j the codes 4j..4j+3), plus the identity permutation (padded by
// a chunk), the chunk records and their count, by the first workgroup.
__global__ __launch_bounds__(256) void split_q8_0_kernel(const uint8_t *__restrict__ xq,
                                                         uint8_t *__restrict__ xs,
                                                         int32_t *__restrict__ meta,
                                                         int32_t *__restrict__ perm,
                                                         int4 *__restrict__ chunks, int64_t M,
                                                         int64_t nbrow) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t blk = t >> 3;
  const int j = (int)(t & 7);
  const bool live = blk < M * nbrow;          // whole 8-lane groups agree
  if (blockIdx.x == 0) {
    const int nch = (int)((M + SMALL_CHUNK - 1) / SMALL_CHUNK);
    for (int i = threadIdx.x; i < M + SMALL_CHUNK; i += blockDim.x) perm[i] = i;
    for (int c = threadIdx.x; c < nch; c += blockDim.x)
      chunks[c] = make_int4(0, c * SMALL_CHUNK, (int)min((int64_t)SMALL_CHUNK, M - c * SMALL_CHUNK), 0);
    if (threadIdx.x == 0) meta[3] = nch;        // META_NSMALL
  }
  uint32_t packed = 0, d16 = 0;
  if (live) {
    const uint16_t *p = reinterpret_cast<const uint16_t *>(xq + blk * Q8B + 2 + 4 * j);
    packed = (uint32_t)p[0] | ((uint32_t)p[1] << 16);
    d16 = *reinterpret_cast<const uint16_t *>(xq + blk * Q8B);
  }
  const uint32_t word = split_word(packed, j);
  const int lsum = sum8(low_nibble_sum(packed));
  if (live) {
    const int64_t r = blk / nbrow;
    SplitBlk *sb = split_blk(xs, r, nbrow, blk - r * nbrow);
    sb->w[j] = word;
    if (j == 0) {
      sb->d = f16_bits_to_f32(d16);
      sb->corr = -8 * lsum;
    }
  }
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

// Workspace: the aligned codes and scales of the matrix-core path, or, for a
// few rows, the nibble-split rows, meta words, permutation and chunk records
// of the VALU path (the larger of the two).
namespace w4a8 {
namespace {
struct DenseSmallLayout {
  size_t meta, perm, chunks, xs, total;
};
DenseSmallLayout dense_small_layout(int64_t M, int64_t K) {
  DenseSmallLayout L;
  size_t off = 0;
  L.meta = off;   off += 256;
  L.perm = off;   off += up256(sizeof(int32_t) * (size_t)(M + SMALL_CHUNK));
  L.chunks = off; off += up256(sizeof(int4) * (size_t)((M + SMALL_CHUNK - 1) / SMALL_CHUNK));
  L.xs = off;     off += up256((size_t)M * split_row_bytes(K / 32));
  L.total = off;
  return L;
}
}  // namespace
}  // namespace w4a8

extern "C" size_t q4q8_gemm_workspace_size(int64_t M, int64_t K) {
  if (gemm_shape(M, 1, K) != W4A8_OK) return 0;
  // (at least the VALU path's size for min(M, DENSE_SMALL_M) rows, so the
  // size never shrinks as M grows: a workspace sized for some M serves every
  // smaller M)
  const size_t tiles = up256((size_t)M * K) + up256(sizeof(float) * (size_t)M * (K / 32));
  const int64_t ms = std::min(M, DENSE_SMALL_M);
  return dense_small_ws(ms, K) ? std::max(tiles, dense_small_layout(ms, K).total) : tiles;
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
  if (dense_small(M, N, K)) {
    const DenseSmallLayout L = dense_small_layout(M, K);
    const int64_t nb = M * (K / 32);
    split_q8_0_kernel<<<dim3((unsigned)((nb * 8 + 255) / 256)), dim3(256), 0, s>>>(
        reinterpret_cast<const uint8_t *>(xq), ws + L.xs, reinterpret_cast<int32_t *>(ws + L.meta),
        reinterpret_cast<int32_t *>(ws + L.perm), reinterpret_cast<int4 *>(ws + L.chunks), M,
        K / 32);
    if ((rc = check_launch()) != W4A8_OK) return rc;
    return small_dense(reinterpret_cast<const uint8_t *>(w), ws + L.xs,
                       reinterpret_cast<const int32_t *>(ws + L.meta),
                       reinterpret_cast<const int32_t *>(ws + L.perm),
                       reinterpret_cast<const int4 *>(ws + L.chunks), y, M, N, K, s);
  }
  uint32_t *act = reinterpret_cast<uint32_t *>(ws);
  float *actd = reinterpret_cast<float *>(ws + up256((size_t)M * K));
  const int64_t nblocks = M * (K / 32);
  align_q8_0_kernel<<<dim3((unsigned)((nblocks * 8 + 255) / 256)), dim3(256), 0, s>>>(
      reinterpret_cast<const uint8_t *>(xq), act, actd, nblocks);
  if ((rc = check_launch()) != W4A8_OK) return rc;
  return mfma_dense(reinterpret_cast<const uint8_t *>(w), act, actd, y, M, N, K, s);
}
