// Grouped W4A8 products for expert groups of few token rows, on the VALU
// (paper Sec. 3.2: the token-expert pairs grouped by expert; Sec. 3.3: 4-bit
// weight codes times 8-bit activation codes, one scaling per 32 elements).
//
// The grouped MFMA kernels pad each group to tiles of 16, 32 or 64 rows and
// stream a tile's weights one group of eight blocks at a time, so the
// groups of a batch of up to 128 tokens (a few rows each: the routed experts
// of the batch) would spend most of that work on padding and wait on each
// group's load.  Here those groups are cut into chunks of at most
// SMALL_CHUNK token rows, and a workgroup takes one chunk and a slab of
// weight rows.  Each weight row is read by LPR consecutive lanes, one
// 144-byte group of eight blocks each (LPR = K/256 rounded up to a power of
// two), so a wave reads 64/LPR whole rows, consecutive in memory; the lane's
// weights stay in registers and feed the 4-bit dot products once per token
// row of the chunk, and the LPR partial sums of a row meet through DPP.  The
// chunk's activation rows (nibble-split, padded per group of eight blocks,
// see split_blk) are loaded straight into LDS behind the weights, so the
// token loop waits on nothing but LDS; the lanes of a wave read LPR different
// groups of one row, in distinct banks thanks to the padding.  A workgroup's
// life is mostly the wait for its loads: the chunk's description is one
// record, so the weight loads are issued after a single scalar round trip.
//
// gate/up: HC = 256/LPR columns of h: their HC gate rows and HC up rows; per
//   token SwiGLU, then Q8_0 of each 32-wide block, written as the 34-byte
//   block, as fp32 h, and in nibble-split form for the down kernel.
// down:    512/LPR rows of the down projection; y[pair][n] = w_pair * sum.
#include <algorithm>

#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int SNT = 512;           // threads: 8 waves
constexpr int SW = SNT / 64;
constexpr int SC = SMALL_CHUNK;    // token rows per chunk
constexpr int GMAX = 8;            // eight-block groups per row (K <= 2048)
constexpr int PPG = SPLIT_GROUP_BYTES / 16;   // 16-byte pieces per padded group
constexpr int WGR_MAX = SNT;       // weight rows per workgroup (LPR = 1)

typedef __attribute__((address_space(4))) const int32_t CInt;

struct SmallArgs {
  const uint8_t *w, *ws;      // routed experts [E][N][K/32] Q4_0 / shared [N][K/32]
  const uint8_t *act;         // nibble-split activations, rows of K/32 blocks (split_blk)
  const int32_t *meta, *perm;
  const int4 *chunks;         // {expert, first sorted position, rows, group}
  const float *topk_w;
  const float *shared_w;      // down: the shared expert's weight per token, or null (1)
  float *h;                   // gate/up: fp32 h [P][I]
  uint8_t *hq;                // gate/up: Q8_0(h) [P][I/32]
  uint8_t *hs;                // gate/up: nibble-split Q8_0(h), rows of I/32 blocks
  float *y;                   // down: w * y [P][H]
  int64_t T, k, E, N, K, I;
  int lpr;                    // lanes per weight row (a power of two >= K/256)
  int nslab;                  // workgroups per chunk
};

struct SmallLds {
  uint4 act[SC][GMAX * PPG];       // the chunk's activation rows
  float part[SC][WGR_MAX];         // gate/up: row sums, then h in the gate half
  int pair[SC];
};

// Activation row of pair p (its token for gate/up), in a scalar register.
__device__ __forceinline__ int pair_row(const SmallArgs &a, int p, bool by_token) {
  int r = p;
  if (by_token) {
    const int tk = (int)(a.T * a.k);
    r = p < tk ? p / (int)a.k : p - tk;
  }
  return __builtin_amdgcn_readfirstlane(r);
}

// Sum over the LPR lanes of a row (consecutive, LPR a power of two <= 8),
// left in every one of them.
__device__ __forceinline__ float row_sum(float v, int lpr) {
  if (lpr >= 2) v += dpp_f<DPP_XOR1>(v);
  if (lpr >= 4) v += dpp_f<DPP_XOR2>(v);
  if (lpr >= 8) v += dpp_f<DPP_HALF_MIRROR>(v);
  return v;
}

// One work item (a workgroup): chunk item / nslab, slab item % nslab.
template <bool GATEUP>
__device__ __forceinline__ void small_item(const SmallArgs &a, SmallLds &L, int item) {
  const int c = item / a.nslab, slab = item % a.nslab;
  CInt *cp = (CInt *)a.chunks + 4 * c;
  const int expert = cp[0], pos = cp[1], rows = cp[2];
  // the wave index, known to the compiler as wave-uniform
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int lpr = a.lpr, rpw = 64 / lpr;                   // rows per wave
  const int wgr = SW * rpw, hc = wgr / 2;                  // rows per workgroup, h columns
  const int R = wave * rpw + lane / lpr, li = lane % lpr;  // workgroup row, group
  const int G = (int)(a.K / 256);
  const int nblk = (int)(a.K / 32);
  const bool live_g = li < G;

  // this lane's 144-byte group li of its weight row
  int64_t row;
  if (GATEUP)
    row = R < hc ? (int64_t)slab * hc + R : a.I + (int64_t)slab * hc + (R - hc);
  else
    row = (int64_t)slab * wgr + R;
  const bool live = live_g && row < a.N;
  const int64_t rowbytes = (int64_t)nblk * Q4B;
  const uint8_t *W = (expert < a.E ? a.w + (int64_t)expert * a.N * rowbytes : a.ws) +
                     (live ? row : 0) * rowbytes + (int64_t)(live ? li : 0) * (8 * Q4B);
  W8 w;
  load_w8(W, w);

  // the chunk's pairs with one scalar read (the permutation is padded by a
  // chunk), then every activation row straight into LDS (global_load_lds:
  // lane l's 16 bytes land 16*l past the wave's LDS address), 64 pieces per
  // wave load, behind the weights and before anything waits
  int prs[SC];
#pragma unroll
  for (int m = 0; m < SC; m++) prs[m] = ((CInt *)a.perm)[pos + m];
  const int per_row = G * PPG;
  const int nch = (per_row + 63) / 64;                     // wave loads per row
  const int64_t srow = (int64_t)split_row_bytes(nblk);
  for (int j = wave; j < rows * nch; j += SW) {
    const int m = j / nch, ch = j - m * nch;
    int pm = prs[0];
#pragma unroll
    for (int mm = 1; mm < SC; mm++) pm = m == mm ? prs[mm] : pm;
    const uint4 *row_src =
        reinterpret_cast<const uint4 *>(a.act + (int64_t)pair_row(a, pm, GATEUP) * srow);
    const int piece = ch * 64 + lane;
    if (piece < per_row)
      __builtin_amdgcn_global_load_lds(
          (const void __attribute__((address_space(1))) *)(row_src + piece),
          (void __attribute__((address_space(3))) *)(&L.act[m][ch * 64]), 16, 0, 0);
  }
  if (threadIdx.x == 0) {
#pragma unroll
    for (int m = 0; m < SC; m++) L.pair[m] = prs[m];
  }
  __builtin_amdgcn_s_waitcnt(0);   // the LDS-direct loads (and the weights) have landed
  __syncthreads();
  // per token row: the 8 block dots of this lane's group, then the row's sum
  // over its lpr lanes
  float acc[SC];
#pragma unroll
  for (int m = 0; m < SC; m++) acc[m] = 0.0f;
#pragma unroll
  for (int m = 0; m < SC; m++) {
    if (m < rows) {
      if (live_g) {
        const uint4 *ar = &L.act[m][li * PPG];
#pragma unroll
        for (int kk = 0; kk < 8; kk++) {
          const uint4 hi = ar[3 * kk], lo = ar[3 * kk + 1];
          const uint2 dc = *reinterpret_cast<const uint2 *>(&ar[3 * kk + 2]);
          const int s = blockdot_split(w, kk, hi, lo, (int)dc.y);
          acc[m] = fmaf((float)s, w8_scale(w, kk) * __builtin_bit_cast(float, dc.x), acc[m]);
        }
      }
      acc[m] = row_sum(acc[m], lpr);
    }
  }

  if (GATEUP) {
    if (li == 0) {
#pragma unroll
      for (int m = 0; m < SC; m++)
        if (m < rows) L.part[m][R] = acc[m];
    }
    __syncthreads();
    const int hcol0 = slab * hc;
    for (int t = threadIdx.x; t < rows * hc; t += SNT) {
      const int m = t / hc, cc = t - m * hc;
      const float hval = silu_f32(L.part[m][cc]) * L.part[m][hc + cc];
      L.part[m][cc] = hval;
      a.h[(int64_t)L.pair[m] * a.I + hcol0 + cc] = hval;
    }
    __syncthreads();
    // Q8_0 of each row's 32-wide blocks: 8 lanes per block, whole 8-lane groups
    const int bpr = hc / 32;                               // h blocks per row
    const int nbh = (int)(a.I / 32);
    for (int t = threadIdx.x; t < rows * bpr * 8; t += SNT) {
      const int m = t / (bpr * 8), rem = t - m * (bpr * 8), bi = rem >> 3, jj = rem & 7;
      const float *hv = &L.part[m][32 * bi + 4 * jj];
      const float v[4] = {hv[0], hv[1], hv[2], hv[3]};
      uint32_t d16;
      const uint32_t packed = q8_0_block8(v, d16);
      const uint32_t word = split_word(packed, jj);
      const int lsum = sum8(low_nibble_sum(packed));
      const int p = L.pair[m];
      const int b = slab * bpr + bi;
      store_q8_0_block8(a.hq + ((int64_t)p * nbh + b) * Q8B, jj, packed, d16);
      SplitBlk *hsb = split_blk(a.hs, p, nbh, b);
      hsb->w[jj] = word;
      if (jj == 0) {
        hsb->d = f16_bits_to_f32(d16);
        hsb->corr = -8 * lsum;
      }
    }
  } else {
    if (li == 0 && row < a.N) {
      const int64_t pr = a.T * a.k;
#pragma unroll
      for (int m = 0; m < SC; m++) {
        if (m < rows) {
          const int p = L.pair[m];
          const float wt = p < pr ? a.topk_w[p] : (a.shared_w ? a.shared_w[p - pr] : 1.0f);
          a.y[(int64_t)p * a.N + row] = wt * acc[m];
        }
      }
    }
  }
}

template <bool GATEUP>
__global__ __launch_bounds__(SNT) __attribute__((amdgpu_waves_per_eu(4))) void small_kernel(SmallArgs a) {
  __shared__ SmallLds L;
  const int nchunk = ((CInt *)a.meta)[3];   // META_NSMALL
  if ((int)blockIdx.x < nchunk * a.nslab) small_item<GATEUP>(a, L, blockIdx.x);
}

// Lanes per weight row: K/256 groups rounded up to a power of two.
int small_lpr(int64_t K) {
  int lpr = 1;
  while (lpr < K / 256) lpr *= 2;
  return lpr;
}

}  // namespace

// Shapes the kernels cover: a row's activations fit their LDS rows (H, I <=
// 2048).
bool small_supported(int64_t H, int64_t I) {
  return H <= 256 * GMAX && I <= 256 * GMAX && H % 256 == 0 && I % 256 == 0;
}

// Upper bound on the chunks of a call: one per group, plus one more per
// SMALL_CHUNK rows.
int64_t small_max_chunks(int64_t T, int64_t E, int64_t k, int has_shared) {
  return std::min<int64_t>(E, T * k) + has_shared + (T * k + T) / SC + 1;
}

int small_gateup(const uint8_t *w_gu, const uint8_t *ws_gu, const uint8_t *xs,
                 const int32_t *meta, const int32_t *perm, const int4 *chunks, float *h,
                 uint8_t *hq, uint8_t *hs, int64_t maxchunks, int64_t T, int64_t H, int64_t I,
                 int64_t E, int64_t k, hipStream_t s) {
  SmallArgs a{};
  a.w = w_gu; a.ws = ws_gu; a.act = xs;
  a.meta = meta; a.perm = perm; a.chunks = chunks;
  a.h = h; a.hq = hq; a.hs = hs;
  a.T = T; a.k = k; a.E = E; a.N = 2 * I; a.K = H; a.I = I;
  a.lpr = small_lpr(H);
  a.nslab = (int)(I / (256 / a.lpr));          // h columns per workgroup: 256 / lpr
  small_kernel<true><<<dim3((unsigned)(maxchunks * a.nslab)), dim3(SNT), 0, s>>>(a);
  return check_launch();
}

int small_down(const uint8_t *w_d, const uint8_t *ws_d, const uint8_t *hs, const int32_t *meta,
               const int32_t *perm, const int4 *chunks, const float *topk_w,
               const float *shared_w, float *y, int64_t maxchunks, int64_t T, int64_t H,
               int64_t I, int64_t E, int64_t k, hipStream_t s) {
  SmallArgs a{};
  a.w = w_d; a.ws = ws_d; a.act = hs;
  a.meta = meta; a.perm = perm; a.chunks = chunks;
  a.topk_w = topk_w; a.shared_w = shared_w; a.y = y;
  a.T = T; a.k = k; a.E = E; a.N = H; a.K = I; a.I = I;
  a.lpr = small_lpr(I);
  const int64_t wgr = SW * (64 / a.lpr);         // down rows per workgroup
  a.nslab = (int)((H + wgr - 1) / wgr);
  small_kernel<false><<<dim3((unsigned)(maxchunks * a.nslab)), dim3(SNT), 0, s>>>(a);
  return check_launch();
}

// Dense product of a few activation rows (q4q8_gemm, M <= 128) on the down
// kernel: the rows are the "pairs" 0..M-1 of chunks of SMALL_CHUNK rows
// against one weight matrix (ws), each scaled by 1; act holds the rows in
// nibble-split form, perm the identity (padded by a chunk), chunks their
// records and meta[3] their count (written by the caller's conversion launch).
int small_dense(const uint8_t *w, const uint8_t *act, const int32_t *meta, const int32_t *perm,
                const int4 *chunks, float *y, int64_t M, int64_t N, int64_t K, hipStream_t s) {
  SmallArgs a{};
  a.w = nullptr; a.ws = w; a.act = act;
  a.meta = meta; a.perm = perm; a.chunks = chunks;
  a.y = y;
  a.T = 0; a.k = 0; a.E = 0; a.N = N; a.K = K; a.I = K;
  a.lpr = small_lpr(K);
  const int64_t wgr = SW * (64 / a.lpr);         // output rows per workgroup
  a.nslab = (int)((N + wgr - 1) / wgr);
  const int64_t nchunks = (M + SC - 1) / SC;
  if (nchunks * a.nslab >= ((int64_t)1 << 31)) return W4A8_ERANGE;
  small_kernel<false><<<dim3((unsigned)(nchunks * a.nslab)), dim3(SNT), 0, s>>>(a);
  return check_launch();
}

}  // namespace w4a8
