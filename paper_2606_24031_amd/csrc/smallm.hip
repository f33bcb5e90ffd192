// Grouped W4A8 products for expert groups of few token rows, on the VALU
// (paper Sec. 3.2: the token-expert pairs grouped by expert; Sec. 3.3: 4-bit
// weight codes times 8-bit activation codes, one scaling per 32 elements).
//
// The grouped MFMA kernels pad each group to 32-row tiles, so a group of a
// few rows -- the routed experts of a batch of a few dozen tokens, or the
// sparsely routed experts of a prefill -- would spend most of that work on
// padding.  Here the small groups are cut into chunks of at most
// SMALL_CHUNK token rows, and a workgroup takes one chunk and 64 weight rows
// per row set: lane = weight row, wave = (row set, eight-block group of K).
// The lane's 144 bytes of weights stay in registers and feed the 4-bit dot
// products once per token row of the chunk.  All lanes of a wave multiply
// the same activation block: the chunk's activation rows (nibble-split, see
// split_word) are loaded together with the weights and parked in LDS, so the
// token loop waits on nothing but LDS.  The waves of a row set add their
// partial sums through LDS (over the activation staging) in a fixed order, so
// results do not depend on scheduling.  A workgroup's life is mostly the wait
// for its loads: the chunk's description is one record, so the weight loads
// are issued after a single scalar round trip.
//
// gate/up: the 32 gate and the 32 matching up rows of one 32-wide block of
//   h; per token SwiGLU, then Q8_0 of the block, written as the 34-byte
//   block, as fp32 h, and in nibble-split form for the down kernel.
// down:    64 * nrs rows of the down projection; y[pair][n] = w_pair * sum.
#include <algorithm>

#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int SNT = 512;           // threads: 8 waves
constexpr int SW = SNT / 64;
constexpr int SC = SMALL_CHUNK;    // token rows per chunk
constexpr int KB_MAX = 64;         // blocks of K per row (K <= 2048)
constexpr int PPB = sizeof(SplitBlk) / 16;   // 16-byte pieces per split block

typedef __attribute__((address_space(4))) const int32_t CInt;
// 16-byte pieces as a native vector (a copy of HIP's uint4 struct becomes a
// memcpy, which keeps arrays of them out of registers)
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

struct SmallArgs {
  const uint8_t *w, *ws;      // routed experts [E][N][K/32] Q4_0 / shared [N][K/32]
  const SplitBlk *act;        // nibble-split activations [row][K/32]
  const int32_t *meta, *perm;
  const int4 *chunks;         // {expert, first sorted position, rows, group}
  const float *topk_w;
  const float *shared_w;      // down: the shared expert's weight per token, or null (1)
  float *h;                   // gate/up: fp32 h [P][I]
  uint8_t *hq;                // gate/up: Q8_0(h) [P][I/32]
  SplitBlk *hs;               // gate/up: nibble-split Q8_0(h) [P][I/32]
  float *y;                   // down: w * y [P][H]
  int64_t T, k, E, N, K, I;
  int nrs;                    // row sets (64 rows each) per workgroup
  int nslab;                  // workgroups per chunk
};

struct SmallLds {
  union {
    uint4 act[SC][KB_MAX * PPB];   // the chunk's activation rows
    float part[SW][SC][64];        // then: partial row sums of each wave
  };
  float hv[SC][33];                // gate/up: the h block of each token row
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

// One work item (a workgroup): chunk item / nslab, slab item % nslab.
template <bool GATEUP>
__device__ __forceinline__ void small_item(const SmallArgs &a, SmallLds &L, int nchunk, int item) {
  const int c = item / a.nslab, slab = item % a.nslab;
  (void)nchunk;
  CInt *cp = (CInt *)a.chunks + 4 * c;
  const int expert = cp[0], pos = cp[1], rows = cp[2];
  // the wave index, known to the compiler as wave-uniform
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int nrs = a.nrs, rs = wave % nrs, gg = wave / nrs;
  const int G = (int)(a.K / 256);
  const int nblk = (int)(a.K / 32);
  const bool live = gg < G;

  // this lane's 144-byte group gg of its weight row
  int64_t row;
  if (GATEUP)
    row = lane < 32 ? (int64_t)slab * 32 + lane : a.I + (int64_t)slab * 32 + (lane - 32);
  else
    row = (int64_t)slab * (64 * nrs) + rs * 64 + lane;
  const int64_t rowbytes = (int64_t)nblk * Q4B;
  const uint8_t *W = (expert < a.E ? a.w + (int64_t)expert * a.N * rowbytes : a.ws) +
                     row * rowbytes + (int64_t)(live ? gg : 0) * (8 * Q4B);
  W8 w;
  load_w8(W, w);

  // the chunk's pairs with one scalar read (the permutation is padded by a
  // chunk), then every activation row straight into LDS (global_load_lds:
  // lane l's 16 bytes land 16*l past the wave's LDS address), 64 pieces per
  // wave load, behind the weights and before anything waits
  int prs[SC];
#pragma unroll
  for (int m = 0; m < SC; m++) prs[m] = ((CInt *)a.perm)[pos + m];
  const int per_row = nblk * PPB;
  const int nch = (per_row + 63) / 64;                     // wave loads per row
  for (int j = wave; j < rows * nch; j += SW) {
    const int m = j / nch, ch = j - m * nch;
    int pm = prs[0];
#pragma unroll
    for (int mm = 1; mm < SC; mm++) pm = m == mm ? prs[mm] : pm;
    const SplitBlk *row_src = a.act + (int64_t)pair_row(a, pm, GATEUP) * nblk;
    const int piece = ch * 64 + lane;
    if (piece < per_row)
      __builtin_amdgcn_global_load_lds(
          (const void __attribute__((address_space(1))) *)(reinterpret_cast<const uint4 *>(row_src) + piece),
          (void __attribute__((address_space(3))) *)(&L.act[m][ch * 64]), 16, 0, 0);
  }
  if (threadIdx.x == 0) {
#pragma unroll
    for (int m = 0; m < SC; m++) L.pair[m] = prs[m];
  }
  __builtin_amdgcn_s_waitcnt(0);   // the LDS-direct loads (and the weights) have landed
  __syncthreads();
  // per token row: the 8 block dots of this lane's group (payload views of
  // the weights taken at use: registers are the scarce resource here)
  float acc[SC];
#pragma unroll
  for (int m = 0; m < SC; m++) acc[m] = 0.0f;
  if (live) {
#pragma unroll
    for (int m = 0; m < SC; m++) {
      if (m < rows) {
        const uint4 *ar = &L.act[m][gg * 8 * PPB];
#pragma unroll
        for (int kk = 0; kk < 8; kk++) {
          const uint4 hi = ar[PPB * kk], lo = ar[PPB * kk + 1];
          const uint2 dc = *reinterpret_cast<const uint2 *>(&ar[PPB * kk + 2]);
          const uint32_t h4[4] = {hi.x, hi.y, hi.z, hi.w};
          const uint32_t l4[4] = {lo.x, lo.y, lo.z, lo.w};
          int sa = 0;
          uint32_t sb = dc.y;
#pragma unroll
          for (int cc = 0; cc < 4; cc++) {
            const uint32_t nb = w8_nib(w, kk, cc);
            sa = __builtin_amdgcn_sdot8((int)(nb ^ 0x88888888u), (int)h4[cc], sa, false);
            sb = __builtin_amdgcn_udot8(nb, l4[cc], sb, false);
          }
          const int s = (int)(((uint32_t)sa << 4) + sb);
          acc[m] = fmaf((float)s, w8_scale(w, kk) * __builtin_bit_cast(float, dc.x), acc[m]);
        }
      }
    }
  }
  __syncthreads();                       // every wave is done with the activations
  float *mypart = &L.part[wave][0][0];
#pragma unroll
  for (int m = 0; m < SC; m++)
    if (m < rows) mypart[m * 64 + lane] = acc[m];
  __syncthreads();

  if (GATEUP) {
    const int hcol0 = slab * 32;
    if ((int)threadIdx.x < rows * 32) {
      const int m = threadIdx.x >> 5, cc = threadIdx.x & 31;
      float g = 0.0f, u = 0.0f;
      for (int wv = 0; wv < SW; wv++) {
        g += L.part[wv][m][cc];
        u += L.part[wv][m][32 + cc];
      }
      const float hval = silu_f32(g) * u;
      L.hv[m][cc] = hval;
      a.h[(int64_t)L.pair[m] * a.I + hcol0 + cc] = hval;
    }
    __syncthreads();
    // Q8_0 of each row's 32-wide block: 8 lanes per row, whole 8-lane groups
    if ((int)threadIdx.x < rows * 8) {
      const int m = threadIdx.x >> 3, jj = threadIdx.x & 7;
      const float v[4] = {L.hv[m][4 * jj], L.hv[m][4 * jj + 1], L.hv[m][4 * jj + 2],
                          L.hv[m][4 * jj + 3]};
      uint32_t d16;
      const uint32_t packed = q8_0_block8(v, d16);
      const uint32_t word = split_word(packed, jj);
      const int lsum = sum8(low_nibble_sum(packed));
      const int64_t blk = (int64_t)L.pair[m] * (a.I / 32) + slab;
      store_q8_0_block8(a.hq + blk * Q8B, jj, packed, d16);
      SplitBlk *hsb = a.hs + blk;
      hsb->w[jj] = word;
      if (jj == 0) {
        hsb->d = f16_bits_to_f32(d16);
        hsb->corr = -8 * lsum;
      }
    }
  } else {
    const int R = 64 * nrs;
    for (int idx = threadIdx.x; idx < rows * R; idx += SNT) {
      const int m = idx / R, r = idx - m * R;
      const int rset = r >> 6, rl = r & 63;
      float v = 0.0f;
      for (int wv = rset; wv < SW; wv += nrs) v += L.part[wv][m][rl];
      const int p = L.pair[m];
      const int64_t pr = a.T * a.k;
      const float wt = p < pr ? a.topk_w[p] : (a.shared_w ? a.shared_w[p - pr] : 1.0f);
      a.y[(int64_t)p * a.N + (int64_t)slab * R + r] = wt * v;
    }
  }
}

template <bool GATEUP>
__global__ __launch_bounds__(SNT) __attribute__((amdgpu_waves_per_eu(4))) void small_kernel(SmallArgs a) {
  __shared__ SmallLds L;
  const int nchunk = ((CInt *)a.meta)[3];   // META_NSMALL
  if ((int)blockIdx.x < nchunk * a.nslab) small_item<GATEUP>(a, L, nchunk, blockIdx.x);
}

}  // namespace

// Row sets per down workgroup: as many as leave each wave one eight-block
// group of K (I/256 groups), while the slab still divides H.
int small_down_rowsets(int64_t H, int64_t I) {
  const int64_t G = I / 256;
  int nrs = (G < SW && SW % G == 0) ? (int)(SW / G) : 1;
  while (nrs > 1 && H % (64 * nrs) != 0) nrs /= 2;
  return nrs;
}

// Shapes the kernels cover: every wave holds at most one eight-block group
// of its row and a row's activations fit their LDS rows (H, I <= 2048).
bool small_supported(int64_t H, int64_t I) {
  return H <= 32 * KB_MAX && I <= 32 * KB_MAX && H % 256 == 0 && I % 256 == 0;
}

// Upper bound on the chunks of a call: one per group, plus one more per
// SMALL_CHUNK rows.
int64_t small_max_chunks(int64_t T, int64_t E, int64_t k, int has_shared) {
  return std::min<int64_t>(E, T * k) + has_shared + (T * k + T) / SC + 1;
}

int small_gateup(const uint8_t *w_gu, const uint8_t *ws_gu, const SplitBlk *xs,
                 const int32_t *meta, const int32_t *perm, const int4 *chunks, float *h,
                 uint8_t *hq, SplitBlk *hs, int64_t maxchunks, int64_t T, int64_t H, int64_t I,
                 int64_t E, int64_t k, hipStream_t s) {
  SmallArgs a{};
  a.w = w_gu; a.ws = ws_gu; a.act = xs;
  a.meta = meta; a.perm = perm; a.chunks = chunks;
  a.h = h; a.hq = hq; a.hs = hs;
  a.T = T; a.k = k; a.E = E; a.N = 2 * I; a.K = H; a.I = I;
  a.nrs = 1; a.nslab = (int)(I / 32);
  small_kernel<true><<<dim3((unsigned)(maxchunks * a.nslab)), dim3(SNT), 0, s>>>(a);
  return check_launch();
}

int small_down(const uint8_t *w_d, const uint8_t *ws_d, const SplitBlk *hs, const int32_t *meta,
               const int32_t *perm, const int4 *chunks, const float *topk_w,
               const float *shared_w, float *y, int64_t maxchunks, int64_t T, int64_t H,
               int64_t I, int64_t E, int64_t k, hipStream_t s) {
  SmallArgs a{};
  a.w = w_d; a.ws = ws_d; a.act = hs;
  a.meta = meta; a.perm = perm; a.chunks = chunks;
  a.topk_w = topk_w; a.shared_w = shared_w; a.y = y;
  a.T = T; a.k = k; a.E = E; a.N = H; a.K = I; a.I = I;
  a.nrs = small_down_rowsets(H, I);
  a.nslab = (int)(H / (64 * a.nrs));
  small_kernel<false><<<dim3((unsigned)(maxchunks * a.nslab)), dim3(SNT), 0, s>>>(a);
  return check_launch();
}

}  // namespace w4a8
