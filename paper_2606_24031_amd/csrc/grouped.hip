// Grouped W4A8 GEMMs over the routed token-expert pairs of a layer on int8
// MFMA (paper Sec. 3.2: one grouped launch over all routed pairs; Sec. 3.3:
// integer products of 4-bit weight codes with 8-bit activation codes, one
// scaling per 32-element group).
//
// Tile: 32 token rows by 256 weight rows; each of the four waves owns 64
// weight rows as two 32x32 output tiles.  One Q-block is exactly one
// v_mfma_i32_32x32x32_i8 (K = 32), so every block's int32 dot stays separate
// until it is scaled:
//   * the MFMA accumulator input is the constant 0x4B400000, so the int32
//     result read as a float is exactly 1.5*2^23 + s (|s| < 2^22);
//   * t = fma(f, d_w, -1.5*2^23*d_w) = s*d_w rounded once, and
//     acc = fma(t, d_x, acc): two VALU ops per (row, column, block), no
//     int-to-float conversion.
// Lane l of an MFMA holds token row l%32 of the A operand and weight row
// l%32 of the B operand, with the block's codes 16*(l/32)..+15 in both; the
// low nibbles of a Q4_0 block are its elements 0..15 and the high nibbles
// 16..31, so the staged weight row of a block is [16 low codes][16 high
// codes], each as int8 (q - 8).  Output element e of lane l is token row
// 8*(e/4) + 4*(l/32) + e%4, weight row l%32.
//
// Staging: each thread owns one weight row and keeps its 144-byte group of
// eight blocks (16-byte aligned) in registers; the group is decoded into LDS
// four blocks at a time.  Activation rows are gathered through the expert
// permutation, one 34-byte block per thread.  LDS rows are 144 bytes apart,
// so the 16-byte reads of 16 lanes fall in distinct banks.  About 50 KB of
// LDS and at most 168 registers let three workgroups share a compute unit.
//
// Gate/up tiles pair 32 gate rows with the 32 matching up rows in each wave,
// so SwiGLU needs no data movement; Q8_0 of each 32-wide h block goes through
// a small LDS transpose, one row per lane.  Down tiles write w * y per pair
// for the fixed-order combine.
#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int GT = 256;            // threads: four waves
constexpr int BM = 32;             // token rows per tile
constexpr int BN = 256;            // weight rows per tile (one per thread)
constexpr int KC = 4;              // Q-blocks per K chunk
constexpr int ROWB = KC * 32 + 16; // LDS bytes per staged code row (padded)
constexpr int BIAS = 0x4B400000;   // float 1.5 * 2^23
constexpr float BIASF = 12582912.0f;

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));

struct LdsTile {
  uint8_t wc[BN * ROWB];           // weight codes [n][block][32]
  float2 wd[KC * BN];              // {d_w, -1.5*2^23*d_w} [block][n]
  uint8_t ac[BM * ROWB];           // activation codes [m][block][32]
  float ad[KC * BM];               // d_x [block][m]
};
constexpr int HT_STRIDE = 33;      // floats per row of the h transpose
static_assert(4 * 32 * HT_STRIDE * 4 <= BN * ROWB, "h transpose fits in the weight staging");

struct GemmArgs {
  const uint8_t *w, *ws;           // routed experts [E][N][K/32] / shared [N][K/32]
  const uint8_t *act;              // Q8_0 rows, [row][K/32] blocks
  const int32_t *meta, *perm;
  const int4 *groups;
  const int2 *tiles;
  const float *topk_w;
  float *h;                        // gate/up: fp32 h [P][I]
  uint8_t *hq;                     // gate/up: Q8_0(h) [P][I/32]
  float *y;                        // down: w * y [P][H]
  int64_t T, k, E, N, K, I;
  int act_by_pair;                 // activation row = pair (down) or its token (gate/up)
};

__device__ __forceinline__ int64_t pair_token(const GemmArgs &a, int p) {
  return p < a.T * a.k ? p / a.k : p - a.T * a.k;
}

// Global weight row of LDS row r (= thread) for column slice `slice`.
// Gate/up: wave w = r / 64 holds gate rows (r % 64 < 32) and up rows of the
// 32 h columns slice*128 + 32w + (r % 32).
template <bool GATEUP>
__device__ __forceinline__ int64_t weight_row(const GemmArgs &a, int slice, int r) {
  if (GATEUP) {
    const int64_t col = (int64_t)slice * 128 + 32 * (r >> 6) + (r & 31);
    return (r & 32) ? a.I + col : col;
  }
  return (int64_t)slice * BN + r;
}

__device__ __forceinline__ uint32_t signed_codes(uint32_t x) {
  // bytes 0..15 -> (value - 8) as int8: +0x78 per byte (no carries), flip bit 7
  return (x + 0x78787878u) ^ 0x80808080u;
}

// The thread's activation block for the current 8-block group: 9 dwords
// around the 34-byte block (4-byte aligned), decoded at store time.
struct ABlock {
  uint32_t D[9];
  bool live;
};

__device__ __forceinline__ void load_group(const GemmArgs &a, const uint8_t *wrow,
                                           const int *rowact, int grp, W8 &w, ABlock &ab) {
  load_w8(wrow + (int64_t)grp * (8 * Q4B), w);
  const int m = threadIdx.x >> 3, b = threadIdx.x & 7;
  const int ra = rowact[m];
  ab.live = ra >= 0;
  if (ab.live) {
    const int64_t rowbytes = (a.K / 32) * Q8B;
    // block 8*grp + b starts at byte 34*(8*grp + b): 4-byte aligned for even
    // b, two bytes past a 4-byte boundary for odd b
    const int64_t off = (int64_t)ra * rowbytes + ((int64_t)grp * 8 + b) * Q8B - ((b & 1) ? 2 : 0);
    const uint32_t *src = reinterpret_cast<const uint32_t *>(a.act + off);
#pragma unroll
    for (int i = 0; i < 9; i++) ab.D[i] = src[i];
  }
}

// Decode blocks 4*half .. 4*half+3 of the thread's weight group into its LDS
// row, and, for the threads holding one of those activation blocks, the
// activation codes and scale.
__device__ __forceinline__ void store_half(LdsTile &L, const W8 &w, const ABlock &ab, int half) {
  const int n = threadIdx.x;
#pragma unroll
  for (int kk = 0; kk < KC; kk++) {
    const int k = 4 * half + kk;
    uint32_t lo[4], hi[4];
#pragma unroll
    for (int c = 0; c < 4; c++) {
      const uint32_t nb = w8_nib(w, k, c);
      lo[c] = signed_codes(nb & 0x0F0F0F0Fu);
      hi[c] = signed_codes((nb >> 4) & 0x0F0F0F0Fu);
    }
    uint4 *dst = reinterpret_cast<uint4 *>(L.wc + n * ROWB + kk * 32);
    dst[0] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
    dst[1] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
    const float dw = w8_scale(w, k);
    L.wd[kk * BN + n] = make_float2(dw, -BIASF * dw);
  }
  const int m = threadIdx.x >> 3, b = threadIdx.x & 7;
  if ((b >> 2) == half) {
    const int kk = b & 3;
    uint32_t q[8];
    float d;
    if ((b & 1) == 0) {           // scale in bytes 0..1, codes from byte 2
      d = f16_bits_to_f32(ab.D[0]);
#pragma unroll
      for (int c = 0; c < 8; c++) q[c] = align2(ab.D[c + 1], ab.D[c]);
    } else {                      // two bytes before the block, codes aligned
      d = f16_bits_to_f32(ab.D[0] >> 16);
#pragma unroll
      for (int c = 0; c < 8; c++) q[c] = ab.D[c + 1];
    }
    uint4 *dst = reinterpret_cast<uint4 *>(L.ac + m * ROWB + kk * 32);
    dst[0] = ab.live ? make_uint4(q[0], q[1], q[2], q[3]) : make_uint4(0u, 0u, 0u, 0u);
    dst[1] = ab.live ? make_uint4(q[4], q[5], q[6], q[7]) : make_uint4(0u, 0u, 0u, 0u);
    L.ad[kk * BM + m] = ab.live ? d : 0.0f;
  }
}

// One K chunk of MFMAs for this wave's two 32x32 output tiles; acc[j][e] is
// (token row 8*(e/4) + 4*(lane/32) + e%4, weight row 64*wave + 32j + lane%32).
__device__ __forceinline__ void chunk_mfma(const LdsTile &L, int wave, const v16i &c0,
                                           float acc[2][16]) {
  const int lane = threadIdx.x & 63;
  const int r32 = lane & 31, hh = lane >> 5;
  // one block at a time: unrolling the blocks would hold four blocks'
  // operands and MFMA results at once and spill
#pragma unroll 1
  for (int kk = 0; kk < KC; kk++) {
    const v4i av = *reinterpret_cast<const v4i *>(L.ac + r32 * ROWB + kk * 32 + 16 * hh);
    float dx[16];
#pragma unroll
    for (int q = 0; q < 4; q++) {
      const float4 v = *reinterpret_cast<const float4 *>(L.ad + kk * BM + 8 * q + 4 * hh);
      dx[4 * q + 0] = v.x; dx[4 * q + 1] = v.y; dx[4 * q + 2] = v.z; dx[4 * q + 3] = v.w;
    }
#pragma unroll
    for (int j = 0; j < 2; j++) {
      const int n = 64 * wave + 32 * j + r32;
      const v4i bv = *reinterpret_cast<const v4i *>(L.wc + n * ROWB + kk * 32 + 16 * hh);
      const float2 wd = L.wd[kk * BN + n];
      // the whole int32 result vector reinterpreted at once (an element-wise
      // bit cast of a vector's elements has been folded to element 0)
      const v16f f =
          __builtin_bit_cast(v16f, __builtin_amdgcn_mfma_i32_32x32x32_i8(av, bv, c0, 0, 0, 0));
#pragma unroll
      for (int e = 0; e < 16; e++) {
        const float t = fmaf(f[e], wd.x, wd.y);
        acc[j][e] = fmaf(t, dx[e], acc[j][e]);
      }
    }
  }
}

// Q8_0 code of v for the reciprocal id of the stored scale (the same fp32
// steps as the format definition).
__device__ __forceinline__ uint32_t q8_code(float v, float id) {
  int q = (int)roundf(v * id);
  q = q > 127 ? 127 : (q < -127 ? -127 : q);
  return (uint32_t)q & 0xFFu;
}

template <bool GATEUP>
__global__ __launch_bounds__(GT, 3) void grouped_kernel(GemmArgs a) {
  __shared__ LdsTile L;
  __shared__ int rowact[BM];       // activation row of each tile row (-1: padding)
  __shared__ int rowpair[BM];      // pair of each tile row (-1: padding)
  const int nslices = (int)(GATEUP ? a.I / 128 : a.N / BN);
  const int tile = blockIdx.x / nslices, slice = blockIdx.x % nslices;
  if (tile >= a.meta[2]) return;                     // META_NTILES
  const int2 td = a.tiles[tile];
  const int4 gd = a.groups[td.x];
  const int mc = min(BM, gd.z - td.y);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (tid < BM) {
    int p = -1, r = -1;
    if (tid < mc) {
      p = a.perm[gd.y + td.y + tid];
      r = a.act_by_pair ? p : (int)pair_token(a, p);
    }
    rowpair[tid] = p;
    rowact[tid] = r;
  }
  __syncthreads();
  const int64_t wexpert = (int64_t)a.N * (a.K / 32) * Q4B;
  const uint8_t *W = gd.x < a.E ? a.w + (int64_t)gd.x * wexpert : a.ws;
  const uint8_t *wrow = W + weight_row<GATEUP>(a, slice, tid) * ((a.K / 32) * Q4B);
  const int ngroups = (int)(a.K / 256);

  float acc[2][16];
#pragma unroll
  for (int j = 0; j < 2; j++)
#pragma unroll
    for (int e = 0; e < 16; e++) acc[j][e] = 0.0f;

  v16i c0;                                           // accumulator input of every MFMA
#pragma unroll
  for (int e = 0; e < 16; e++) c0[e] = BIAS;
  W8 w;
  ABlock ab;
  load_group(a, wrow, rowact, 0, w, ab);
  for (int g = 0; g < ngroups; g++) {
#pragma unroll
    for (int half = 0; half < 2; half++) {
      __syncthreads();                               // previous chunk's MFMAs done
      store_half(L, w, ab, half);
      __syncthreads();
      if (half == 1 && g + 1 < ngroups) load_group(a, wrow, rowact, g + 1, w, ab);
      chunk_mfma(L, wave, c0, acc);
    }
  }

  const int r32 = lane & 31, hh = lane >> 5;
  if (GATEUP) {
    // lane holds gate (j = 0) and up (j = 1) of h column slice*128 + 32*wave
    // + r32 for token rows 8*(e/4) + 4*hh + e%4; transpose through LDS so
    // that one lane holds a row's 32-wide h block
    __syncthreads();
    float *ht = reinterpret_cast<float *>(L.wc) + wave * 32 * HT_STRIDE;
#pragma unroll
    for (int e = 0; e < 16; e++) {
      const int m = 8 * (e >> 2) + 4 * hh + (e & 3);
      ht[m * HT_STRIDE + r32] = silu_f32(acc[0][e]) * acc[1][e];
    }
    __syncthreads();
    if (lane < BM) {
      const int m = lane;
      const int p = rowpair[m];
      if (p >= 0) {
        const float *hr = ht + m * HT_STRIDE;
        float amax = 0.0f;
        for (int c = 0; c < 32; c++) amax = fmaxf(amax, fabsf(hr[c]));
        const float d32 = amax / 127.0f;
        const uint32_t d16 = f32_to_f16_bits(d32);
        const float df = f16_bits_to_f32(d16);
        const float id = df != 0.0f ? 1.0f / df : 0.0f;
        const int64_t hcol = (int64_t)slice * 128 + 32 * wave;
        uint16_t *dst =
            reinterpret_cast<uint16_t *>(a.hq + ((int64_t)p * (a.I / 32) + hcol / 32) * Q8B);
        dst[0] = (uint16_t)d16;
        for (int c = 0; c < 32; c += 2) {
          const uint32_t q0 = df != 0.0f ? q8_code(hr[c], id) : 0u;
          const uint32_t q1 = df != 0.0f ? q8_code(hr[c + 1], id) : 0u;
          dst[1 + c / 2] = (uint16_t)(q0 | (q1 << 8));
        }
        float4 *hout = reinterpret_cast<float4 *>(a.h + (int64_t)p * a.I + hcol);
        for (int c = 0; c < 32; c += 4)
          hout[c / 4] = make_float4(hr[c], hr[c + 1], hr[c + 2], hr[c + 3]);
      }
    }
  } else {
#pragma unroll
    for (int e = 0; e < 16; e++) {
      const int m = 8 * (e >> 2) + 4 * hh + (e & 3);
      const int p = rowpair[m];
      if (p < 0) continue;
      const float wt = p < a.T * a.k ? a.topk_w[p] : 1.0f;
#pragma unroll
      for (int j = 0; j < 2; j++)
        a.y[(int64_t)p * a.N + (int64_t)slice * BN + 64 * wave + 32 * j + r32] = wt * acc[j][e];
    }
  }
}

}  // namespace

int grouped_tile_rows() { return BM; }

int grouped_gateup(const uint8_t *w_gu, const uint8_t *ws_gu, const uint8_t *xq,
                   const int32_t *meta, const int32_t *perm, const int4 *groups, const int2 *tiles,
                   float *h, uint8_t *hq, int64_t maxtiles, int64_t T, int64_t H, int64_t I,
                   int64_t E, int64_t k, hipStream_t s) {
  GemmArgs a{};
  a.w = w_gu; a.ws = ws_gu; a.act = xq;
  a.meta = meta; a.perm = perm; a.groups = groups; a.tiles = tiles;
  a.h = h; a.hq = hq;
  a.T = T; a.k = k; a.E = E; a.N = 2 * I; a.K = H; a.I = I;
  a.act_by_pair = 0;
  const unsigned grid = (unsigned)(maxtiles * (I / 128));
  grouped_kernel<true><<<dim3(grid), dim3(GT), 0, s>>>(a);
  return check_launch();
}

int grouped_down(const uint8_t *w_d, const uint8_t *ws_d, const uint8_t *hq, const int32_t *meta,
                 const int32_t *perm, const int4 *groups, const int2 *tiles, const float *topk_w,
                 float *y, int64_t maxtiles, int64_t T, int64_t H, int64_t I, int64_t E,
                 int64_t k, hipStream_t s) {
  GemmArgs a{};
  a.w = w_d; a.ws = ws_d; a.act = hq;
  a.meta = meta; a.perm = perm; a.groups = groups; a.tiles = tiles;
  a.topk_w = topk_w; a.y = y;
  a.T = T; a.k = k; a.E = E; a.N = H; a.K = I; a.I = I;
  a.act_by_pair = 1;
  const unsigned grid = (unsigned)(maxtiles * (H / BN));
  grouped_kernel<false><<<dim3(grid), dim3(GT), 0, s>>>(a);
  return check_launch();
}

}  // namespace w4a8
