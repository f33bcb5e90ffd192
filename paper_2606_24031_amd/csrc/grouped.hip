// Grouped W4A8 GEMMs over the routed token-expert pairs of a layer on int8
// MFMA (paper Sec. 3.2: one grouped launch over all routed pairs; Sec. 3.3:
// integer products of 4-bit weight codes with 8-bit activation codes, one
// scaling per 32-element group).
//
// Tile: 64 token rows (four waves x one 16-row MFMA tile) by 64 weight rows
// (four 16-column MFMA tiles), K in chunks of eight Q-blocks.  One Q-block is
// exactly one v_mfma_i32_16x16x32_i8, so every block's int32 dot stays
// separate until it is scaled:
//   * the MFMA accumulator input is the constant 0x4B400000, so the int32
//     result read as a float is exactly 1.5*2^23 + s (|s| < 2^22);
//   * t = fma(f, d_w, -1.5*2^23*d_w) = s*d_w rounded once, and
//     acc = fma(t, d_x, acc): two VALU ops per (row, column, block), no
//     int-to-float conversion.
// Weights are staged in LDS as signed int8 codes (q - 8) with d_w and
// -1.5*2^23*d_w precomputed; activation rows are gathered through the expert
// permutation and staged as codes with their scale.  Row strides carry 8
// bytes of padding (264-byte rows, 8-byte aligned) so the 16 lanes of one
// 64-bit LDS read hit distinct banks.
// The next chunk's global loads are issued before the current chunk's MFMAs.
//
// Gate/up tiles pair 32 gate rows with the 32 matching up rows, so SwiGLU and
// Q8_0 of the 32-wide h block happen in registers; down tiles write w * y per
// pair for the fixed-order combine.
#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int GT = 256;            // threads: four waves
constexpr int BM = 64;             // token rows per tile
constexpr int BN = 64;             // weight rows per tile
constexpr int KC = 8;              // Q-blocks per K chunk
constexpr int ROWB = KC * 32 + 8;  // LDS bytes per staged code row (padded)
constexpr int BIAS = 0x4B400000;   // float 1.5 * 2^23
constexpr float BIASF = 12582912.0f;

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

struct LdsTile {
  uint8_t wc[BN * ROWB];           // weight codes [n][block][32]
  float2 wd[KC * BN];              // {d_w, -1.5*2^23*d_w} [block][n]
  uint8_t ac[BM * ROWB];           // activation codes [m][block][32]
  float ad[KC * BM];               // d_x [block][m]
};

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

// Staged rows of one K chunk held in registers between the global loads and
// the LDS writes: threads 0..63 hold one weight row group (9 x 16 bytes),
// threads 64..127 one activation row group (17 x 16 bytes).  One raw array
// with constant indices for both roles keeps it all in registers.
struct Stage {
  uint4 raw[17];
  int n;                            // 16-byte pieces loaded (0: padding row or idle thread)
};

template <bool GATEUP>
__device__ __forceinline__ int64_t weight_row(const GemmArgs &a, int slice, int r) {
  if (GATEUP) return r < 32 ? (int64_t)slice * 32 + r : a.I + (int64_t)slice * 32 + (r - 32);
  return (int64_t)slice * BN + r;
}

template <bool GATEUP>
__device__ __forceinline__ void stage_load(const GemmArgs &a, const uint8_t *W, int slice,
                                           const int *rowact, int chunk, Stage &st) {
  const int tid = threadIdx.x;
  const int64_t gbytes_w = (a.K / 256) * (8 * Q4B), gbytes_x = (a.K / 256) * (8 * Q8B);
  const uint4 *src = nullptr;
  st.n = 0;
  if (tid < BN) {
    src = reinterpret_cast<const uint4 *>(W + weight_row<GATEUP>(a, slice, tid) * gbytes_w +
                                          (int64_t)chunk * (8 * Q4B));
    st.n = 9;
  } else if (tid < BN + BM && rowact[tid - BN] >= 0) {
    src = reinterpret_cast<const uint4 *>(a.act + (int64_t)rowact[tid - BN] * gbytes_x +
                                          (int64_t)chunk * (8 * Q8B));
    st.n = 17;
  }
#pragma unroll
  for (int i = 0; i < 17; i++)
    if (i < st.n) st.raw[i] = src[i];
}

__device__ __forceinline__ uint32_t signed_codes(uint32_t x) {
  // bytes 0..15 -> (value - 8) as int8: +0x78 per byte (no carries), flip bit 7
  return (x + 0x78787878u) ^ 0x80808080u;
}

__device__ __forceinline__ void stage_store(LdsTile &L, const Stage &st) {
  const int tid = threadIdx.x;
  uint32_t D[68];
#pragma unroll
  for (int i = 0; i < 17; i++) {
    D[4 * i + 0] = st.raw[i].x; D[4 * i + 1] = st.raw[i].y;
    D[4 * i + 2] = st.raw[i].z; D[4 * i + 3] = st.raw[i].w;
  }
  if (tid < BN) {
    const int n = tid;
    W8 w;
#pragma unroll
    for (int i = 0; i < 36; i++) w.D[i] = D[i];
#pragma unroll
    for (int k = 0; k < KC; k++) {
      uint32_t lo[4], hi[4];
#pragma unroll
      for (int c = 0; c < 4; c++) {
        const uint32_t nb = w8_nib(w, k, c);
        lo[c] = signed_codes(nb & 0x0F0F0F0Fu);
        hi[c] = signed_codes((nb >> 4) & 0x0F0F0F0Fu);
      }
      uint2 *dst = reinterpret_cast<uint2 *>(L.wc + n * ROWB + k * 32);  // rows 8-byte aligned
      dst[0] = make_uint2(lo[0], lo[1]);
      dst[1] = make_uint2(lo[2], lo[3]);
      dst[2] = make_uint2(hi[0], hi[1]);
      dst[3] = make_uint2(hi[2], hi[3]);
      const float dw = w8_scale(w, k);
      L.wd[k * BN + n] = make_float2(dw, -BIASF * dw);
    }
  } else if (tid < BN + BM) {
    const int m = tid - BN;
    const bool live = st.n != 0;
#pragma unroll
    for (int k = 0; k < KC; k++) {
      // block k of the 272-byte group: even blocks start on a dword, their
      // codes two bytes on; odd blocks the other way round
      const int i = k >> 1;
      uint32_t q[8];
      float d;
      if ((k & 1) == 0) {
        d = f16_bits_to_f32(D[17 * i]);
#pragma unroll
        for (int c = 0; c < 8; c++) q[c] = align2(D[17 * i + c + 1], D[17 * i + c]);
      } else {
        d = f16_bits_to_f32(D[17 * i + 8] >> 16);
#pragma unroll
        for (int c = 0; c < 8; c++) q[c] = D[17 * i + 9 + c];
      }
      uint2 *dst = reinterpret_cast<uint2 *>(L.ac + m * ROWB + k * 32);  // rows 8-byte aligned
#pragma unroll
      for (int c = 0; c < 4; c++) dst[c] = live ? make_uint2(q[2 * c], q[2 * c + 1]) : make_uint2(0u, 0u);
      L.ad[k * BM + m] = live ? d : 0.0f;
    }
  }
}

// One K chunk of MFMAs for this wave's 16-row tile against the four column
// tiles; acc[j][i] is (row 4*(lane/16)+i, column 16j + lane%16).
__device__ __forceinline__ void chunk_mfma(const LdsTile &L, int wave, float acc[4][4]) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, g = lane >> 4;
  const v4i c0 = {BIAS, BIAS, BIAS, BIAS};
#pragma unroll
  for (int k = 0; k < KC; k++) {
    const long av = *reinterpret_cast<const long *>(L.ac + (wave * 16 + r16) * ROWB + k * 32 + 8 * g);
    const float4 dx = *reinterpret_cast<const float4 *>(L.ad + k * BM + wave * 16 + 4 * g);
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const long bv = *reinterpret_cast<const long *>(L.wc + (j * 16 + r16) * ROWB + k * 32 + 8 * g);
      const float2 wd = L.wd[k * BN + j * 16 + r16];
      // the whole int32 result vector reinterpreted at once (an element-wise
      // bit cast of the vector's elements was folded to element 0)
      const v4f f = __builtin_bit_cast(v4f, __builtin_amdgcn_mfma_i32_16x16x32_i8(av, bv, c0, 0, 0, 0));
      const float dxv[4] = {dx.x, dx.y, dx.z, dx.w};
#pragma unroll
      for (int i = 0; i < 4; i++) {
        const float t = fmaf(f[i], wd.x, wd.y);
        acc[j][i] = fmaf(t, dxv[i], acc[j][i]);
      }
    }
  }
}

__device__ __forceinline__ float silu_f32(float g) { return g / (1.0f + expf(-g)); }

template <bool GATEUP>
__global__ __launch_bounds__(GT, 2) void grouped_kernel(GemmArgs a) {
  __shared__ LdsTile L;
  __shared__ int rowact[BM];       // activation row of each tile row (-1: padding)
  __shared__ int rowpair[BM];      // pair of each tile row (-1: padding)
  const int nslices = (int)(GATEUP ? a.I / 32 : a.N / BN);
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
  const int nchunks = (int)(a.K / 256);
  const bool active = wave * 16 < mc;                // this wave has rows

  float acc[4][4];
#pragma unroll
  for (int j = 0; j < 4; j++)
#pragma unroll
    for (int i = 0; i < 4; i++) acc[j][i] = 0.0f;

  Stage st;
  stage_load<GATEUP>(a, W, slice, rowact, 0, st);
  for (int c = 0; c < nchunks; c++) {
    __syncthreads();                                 // previous chunk's MFMAs done
    stage_store(L, st);
    __syncthreads();
    if (c + 1 < nchunks) stage_load<GATEUP>(a, W, slice, rowact, c + 1, st);
    if (active) chunk_mfma(L, wave, acc);
  }

  const int r16 = lane & 15, g = lane >> 4;
  if (GATEUP) {
    // lane holds gate (j = 0, 1) and up (j = 2, 3) of h columns 16jj + r16
    // for rows 4g + i of this wave's tile
    __syncthreads();
    uint8_t *hq_lds = L.ac;                          // [64 rows][34 bytes]
    float hv[2][4];
#pragma unroll
    for (int jj = 0; jj < 2; jj++)
#pragma unroll
      for (int i = 0; i < 4; i++) hv[jj][i] = silu_f32(acc[jj][i]) * acc[jj + 2][i];
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int m = wave * 16 + 4 * g + i;
      // Q8_0 of the 32 h values of row m: 16 lanes (r16) x 2 columns each
      float amax = fmaxf(fabsf(hv[0][i]), fabsf(hv[1][i]));
#pragma unroll
      for (int o = 8; o > 0; o >>= 1) amax = fmaxf(amax, __shfl_xor(amax, o, 16));
      const float d32 = amax / 127.0f;
      const uint32_t d16 = f32_to_f16_bits(d32);
      const float df = f16_bits_to_f32(d16);
      const float id = df != 0.0f ? 1.0f / df : 0.0f;
#pragma unroll
      for (int jj = 0; jj < 2; jj++) {
        int q = 0;
        if (df != 0.0f) {
          q = (int)roundf(hv[jj][i] * id);
          q = q > 127 ? 127 : (q < -127 ? -127 : q);
        }
        hq_lds[m * Q8B + 2 + 16 * jj + r16] = (uint8_t)(int8_t)q;
      }
      if (r16 == 0) *reinterpret_cast<uint16_t *>(hq_lds + m * Q8B) = (uint16_t)d16;
      const int p = rowpair[m];
      if (active && p >= 0) {
#pragma unroll
        for (int jj = 0; jj < 2; jj++)
          a.h[(int64_t)p * a.I + (int64_t)slice * 32 + 16 * jj + r16] = hv[jj][i];
      }
    }
    __syncthreads();
    // copy the 64 rows' blocks out: 17 16-bit words per 34-byte block
    for (int idx = tid; idx < BM * 17; idx += GT) {
      const int m = idx / 17, w = idx % 17;
      const int p = rowpair[m];
      if (p < 0) continue;
      uint16_t *dst = reinterpret_cast<uint16_t *>(a.hq + ((int64_t)p * (a.I / 32) + slice) * Q8B);
      dst[w] = reinterpret_cast<const uint16_t *>(hq_lds + m * Q8B)[w];
    }
  } else {
    if (!active) return;
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int m = wave * 16 + 4 * g + i;
      const int p = rowpair[m];
      if (p < 0) continue;
      const float wt = p < a.T * a.k ? a.topk_w[p] : 1.0f;
#pragma unroll
      for (int j = 0; j < 4; j++)
        a.y[(int64_t)p * a.N + (int64_t)slice * BN + 16 * j + r16] = wt * acc[j][i];
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
  const unsigned grid = (unsigned)(maxtiles * (I / 32));
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
