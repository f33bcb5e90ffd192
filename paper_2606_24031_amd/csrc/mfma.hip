// Grouped W4A8 GEMMs on int8 MFMA for expert groups of more than a few token
// rows (paper Sec. 3.2: the token-expert pairs grouped by expert, one launch
// over all groups; Sec. 3.3: 4-bit weight codes times 8-bit activation codes,
// one scaling per 32 elements).
//
// Workgroup tile: up to 64 token rows of one group by 128 weight rows (one
// slice).  Each of the four waves owns 32 weight rows and both 32-row halves
// of the tokens (the second half is compiled out for tiles of at most 32
// rows), so one weight operand feeds two v_mfma_i32_32x32x32_i8 per Q-block.
//   * Weights: lanes l and l + 32 own the same weight row; they stream its
//     144-byte groups of 8 blocks one group ahead, lane l the first 72 bytes
//     (blocks 0..3), lane l + 32 the last 72 (blocks 4..7).  Each lane splits
//     its block j into low- and high-nibble codes, each as the int8 16*(q-8)
//     (the nibble q ^ 8 in the high half of its byte), and one swap between
//     the wave halves (v_permlane32_swap) leaves in lanes 0..31 the low and in
//     lanes 32..63 the high codes of block j in one register and of block
//     j + 4 in the other: the A operands of both blocks.
//   * Activations: the tile's aligned Q8_0 codes for 8 blocks go to LDS by
//     direct loads (global_load_lds), the 16-byte chunks of a row XOR-swizzled
//     by the row so the rows a half-wave reads sit in distinct banks.  With
//     K <= 512 all of K stays resident and the workgroup runs several weight
//     slices with no barrier; otherwise the next 8 blocks are staged while the
//     current 8 are used, one barrier per 8 blocks.
//   * Products: the weights are the A operand and the token rows the B
//     operand, so element e of an MFMA in lane l is weight row
//     8*(e/4) + 4*(l/32) + e%4 of the wave's 32 and token row l%32 of the
//     half: a lane holds one token's sums for 16 weight rows.
//   * Scaling: the accumulator input is 0x4B400000, so the int32 result read
//     as a float is exactly 1.5*2^23 + 16 s (|16 s| < 2^22); with dx the
//     token's activation scale divided by 16 (exact), t = fma(f, dx,
//     -1.5*2^23*dx) = s dx rounded once and acc = fma(t, d_w, acc).  The
//     per-lane factor is the activation scale; the per-element factor is
//     the weight-row scale, which both token halves share: each wave puts
//     its rows' scales of the current 8 blocks in a small LDS table and
//     reads 16 of them per block (broadcast reads, one set for both halves).
// Gate/up waves hold 16 gate rows and the 16 matching up rows, so element e
// and e + 8 of a lane are the gate and up sums of one column and SwiGLU
// needs no lane exchange; Q8_0 of each 32-wide h block goes through LDS.
// Down tiles write w * y per pair, four consecutive columns per store.
#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int MNT = 256;           // threads: four waves
constexpr int MT = 64;             // token rows per tile
constexpr int WROWS = 128;         // weight rows per slice (32 per wave)
constexpr int SPW_MAX = 4;         // slices per workgroup when the codes are resident
constexpr int BIAS = 0x4B400000;   // float 1.5 * 2^23
constexpr float BIASF = 12582912.0f;

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef uint32_t v2u __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(4))) const int32_t CInt;

struct MArgs {
  const uint8_t *w, *ws;           // routed experts [E][N][K/32] Q4_0 / shared [N][K/32]
  const uint32_t *act;             // aligned Q8_0 codes [row][K/32][8 dwords]
  const float *actd;               // their scales [row][K/32]
  const int32_t *meta, *perm;
  const int4 *tiles;               // {expert, first sorted position, rows, -}
  const float *topk_w;
  const float *shared_w;           // down: the shared expert's weight per token, or null (1)
  float *h;                        // gate/up: fp32 h [P][I]
  uint8_t *hq;                     // gate/up: Q8_0(h) [P][I/32]
  uint32_t *ha;                    // gate/up: aligned codes of Q8_0(h) [P][I/32][8]
  float *hd;                       // gate/up: their scales [P][I/32]
  float *y;                        // down: w * y [P][H]
  int64_t T, k, E, N, K, I;
  int64_t M;                       // dense product (M > 0): M activation rows in implicit
                                   // tiles of tr rows, one weight matrix (ws), no route
  int tr;                          // dense product: rows per tile
  int spw;                         // slices per workgroup
};

// Weight of pair p in the combine: its routing weight, or for the shared
// pair of token t = p - T*k the shared expert's weight (1 without a gate).
__device__ __forceinline__ float pair_weight(const MArgs &a, int p) {
  const int64_t pr = a.T * a.k;
  return p < pr ? a.topk_w[p] : (a.shared_w ? a.shared_w[p - pr] : 1.0f);
}

constexpr int DWS = 36;             // row stride of a wave's weight-scale table

struct MLds {
  union {
    uint4 a[2][MT * 16];           // codes of 8 blocks, [buffer][row][chunk ^ row%16]
    float hv[MT][68];              // gate/up epilogue: h of the tile, [row][64 columns]
  };
  float2 dx[2][8][MT];             // activation scales of 8 blocks divided by 16, and
                                   // their products with -1.5*2^23: [buffer][block][row]
  float dw[4][8][DWS];             // weight-row scales of the current group, [wave][block][row]
  int arow[MT];                    // activation row of each tile row
  int pair[MT];                    // pair of each tile row (-1: padding)
  float pw[MT];                    // down: combine weight of the row's pair
};

// Half of a weight row's group of 8 blocks (72 bytes): blocks 0..3 in lanes
// 0..31, blocks 4..7 in lanes 32..63.
struct HW {
  uint32_t D[18];
};

__device__ __forceinline__ void load_hw(const uint8_t *p, HW &w) {
  const v2u *v = reinterpret_cast<const v2u *>(p);
#pragma unroll
  for (int i = 0; i < 9; i++) {
    const v2u t = v[i];
    w.D[2 * i] = t.x;
    w.D[2 * i + 1] = t.y;
  }
}

// Payload dword c of the half's block j (bytes 18j + 2 + 4c ..), and the
// dword holding its fp16 scale (low half for even j, high half for odd j).
__device__ __forceinline__ uint32_t hw_nib(const HW &w, int j, int c) {
  const int i = j >> 1;
  return (j & 1) == 0 ? align2(w.D[9 * i + c + 1], w.D[9 * i + c]) : w.D[9 * i + 5 + c];
}
__device__ __forceinline__ uint32_t hw_sdw(const HW &w, int j) {
  return (j & 1) == 0 ? w.D[9 * (j >> 1)] : w.D[9 * (j >> 1) + 4];
}

// Weight operands and scale dwords of blocks j and j + 4 of the group.
__device__ __forceinline__ void pair_ops(const HW &w, int j, v4i &b0, v4i &b1, uint32_t &s0,
                                         uint32_t &s1) {
#pragma unroll
  for (int c = 0; c < 4; c++) {
    // q ^ 8 read as a signed 4-bit number is q - 8; placed in the high half
    // of a byte it is the int8 16 * (q - 8).  nib << 4 for the low nibbles
    // comes from one funnel shift of the two dwords the payload straddles
    // (the bits shifted in land in the masked low half of each byte)
    const int i = j >> 1;
    const uint32_t nib = hw_nib(w, j, c);
    const uint32_t sh = (j & 1) == 0 ? __builtin_amdgcn_alignbit(w.D[9 * i + c + 1], w.D[9 * i + c], 12)
                                     : nib << 4;
    const v2u r = __builtin_amdgcn_permlane32_swap((sh ^ 0x80808080u) & 0xF0F0F0F0u,
                                                   (nib ^ 0x88888888u) & 0xF0F0F0F0u, false, false);
    b0[c] = (int)r.x;
    b1[c] = (int)r.y;
  }
  const uint32_t sd = hw_sdw(w, j);
  const v2u r = __builtin_amdgcn_permlane32_swap(sd, sd, false, false);
  s0 = r.x;
  s1 = r.y;
}

// Direct load of 16 bytes per lane into LDS at dst + 16 * lane.  Written as
// an instruction the compiler does not model: through the builtin it cannot
// tell a copy into one staging buffer from reads of the other, and waits for
// every outstanding load (the prefetched weights with it) before reading
// LDS.  The copies are ordered by the explicit wait and barrier at the top
// of the group that reads them.
// M0 is named as clobbered; nothing else in these kernels keeps a value in it.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_dma16(const uint32_t *src, const void *dst) {
  const uint32_t m0 =
      (uint32_t)(uintptr_t)(const void __attribute__((address_space(3))) *)dst;
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(m0)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// Copy the tile's codes of blocks 8g..8g+7 into buffer buf: wave w < nwv
// moves rows 16w..16w+15 (the tile's rows rounded up to 16, 32 or 64), four rows per
// instruction; lane l writes chunk position l%16 of row r0 + l/16, which holds
// chunk (l%16) ^ (row % 16) of the row's 256 bytes.
__device__ __forceinline__ void stage_codes(const MArgs &a, MLds &L, int g, int buf, int nwv,
                                            int wave, int lane, int nblk) {
  if (wave >= nwv) return;
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const int r0 = wave * 16 + i * 4;
    const int r = r0 + (lane >> 4);
    const int c = (lane & 15) ^ (r & 15);
    const uint32_t *src = a.act + ((int64_t)L.arow[r] * nblk + 8 * g) * 8 + c * 4;
    lds_dma16(src, &L.a[buf][r0 * 16]);
  }
}

// A operand of block kk for tile row `row`: its codes 16*hh..+15 of the
// block, from the swizzled staging buffer.
__device__ __forceinline__ v4i aop(const uint4 *abuf, int row, int kk, int hh) {
  const uint4 u = abuf[row * 16 + ((2 * kk + hh) ^ (row & 15))];
  return v4i{(int)u.x, (int)u.y, (int)u.z, (int)u.w};
}

// Integer product with the bias accumulator input, read as floats (the whole
// vector at once: an element-wise bit cast has been folded to element 0).
__device__ __forceinline__ v16f mm(v4i a, v4i b, v16i c) {
  return __builtin_bit_cast(v16f, __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0));
}

// acc[e] += s_e * dx * dw[e] for elements 4q..4q+3: f holds the biased int32
// results of one block for this lane's token (dx its activation scale
// divided by 16, nbx = -1.5*2^23 * dx) and 16 weight rows; t = fma(f, dx,
// nbx) = 16 s dx / 16 rounded once, then one fma with each row's weight
// scale (dw4: rows 8q + 4hh .. +3).
__device__ __forceinline__ void scale4(float acc[16], const v16f &f, int q, float dx, float nbx,
                                       float4 dw4) {
  acc[4 * q + 0] = fmaf(fmaf(f[4 * q + 0], dx, nbx), dw4.x, acc[4 * q + 0]);
  acc[4 * q + 1] = fmaf(fmaf(f[4 * q + 1], dx, nbx), dw4.y, acc[4 * q + 1]);
  acc[4 * q + 2] = fmaf(fmaf(f[4 * q + 2], dx, nbx), dw4.z, acc[4 * q + 2]);
  acc[4 * q + 3] = fmaf(fmaf(f[4 * q + 3], dx, nbx), dw4.w, acc[4 * q + 3]);
}

// A token's activation scale of one block (divided by 16) with its product
// with -1.5*2^23, staged once per tile and group instead of formed per block.
__device__ __forceinline__ float2 scale_pair(float dx) { return make_float2(dx, -BIASF * dx); }

// One block: the weight operand b (32 weight rows) against both token
// halves; dw points at the block's 32 weight-row scales of this wave, dxb
// at the block's 64 activation scales.  The scales of four weight rows are
// read once for both halves.
// The operands of one block read from LDS: the token codes of both halves,
// the weight-row scales (four rows per float4) and the activation scales.
// AHEAD: the scales too are read with the codes (else at their use, for the
// short kernel's register budget).
struct BlockIn {
  v4i a0, a1;
  float4 dw[4];
  float2 dx0, dx1;
  const float *dwp;
  const float2 *dxp;
};
template <bool TWO, bool AHEAD>
__device__ __forceinline__ BlockIn block_in(const uint4 *abuf, const float *dw, const float2 *dxb,
                                            int kk, int r32, int hh) {
  BlockIn o;
  o.a0 = aop(abuf, r32, kk, hh);
  o.a1 = TWO ? aop(abuf, 32 + r32, kk, hh) : v4i{0, 0, 0, 0};
  o.dwp = dw + 4 * hh;
  o.dxp = dxb;
  if (AHEAD) {
#pragma unroll
    for (int q = 0; q < 4; q++) o.dw[q] = *reinterpret_cast<const float4 *>(dw + 8 * q + 4 * hh);
    o.dx0 = dxb[r32];
    o.dx1 = TWO ? dxb[32 + r32] : make_float2(0.0f, 0.0f);
  }
  return o;
}
template <bool TWO, bool AHEAD>
__device__ __forceinline__ void block(float acc0[16], float acc1[16], const BlockIn &in, v4i b,
                                      v16i c0, int r32) {
  const v16f f0 = mm(b, in.a0, c0);
  v16f f1;
  if (TWO) f1 = mm(b, in.a1, c0);
  const float2 dx0 = AHEAD ? in.dx0 : in.dxp[r32];
  const float2 dx1 = AHEAD ? in.dx1 : (TWO ? in.dxp[32 + r32] : make_float2(0.0f, 0.0f));
#pragma unroll
  for (int q = 0; q < 4; q++) {
    const float4 dw4 = AHEAD ? in.dw[q] : *reinterpret_cast<const float4 *>(in.dwp + 8 * q);
    scale4(acc0, f0, q, dx0.x, dx0.y, dw4);
    if (TWO) scale4(acc1, f1, q, dx1.x, dx1.y, dw4);
  }
}

// Tiles of at most 16 rows run v_mfma_i32_16x16x32_i8 instead (half the
// padding of a 32-row half): per block and wave two products, weight rows
// 0..15 and 16..31 of the wave as the A operand, the tile's 16 token rows as
// the B operand.  Lane l of a product holds token l%16 and weight rows
// 4*(l/16)..+3 of the product's 16, so a lane takes eight sums of one token:
// e < 4 of rows 4*(l/16) + e, e >= 4 of rows 16 + 4*(l/16) + e - 4.
typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4f mm16(long a, long b, v4i c) {
  return __builtin_bit_cast(v4f, __builtin_amdgcn_mfma_i32_16x16x32_i8(a, b, c, 0, 0, 0));
}

// The A operands of both products of one block from its 32x32x32 A operand
// b (lane l < 32: codes 0..15 of wave row l; lane l + 32: codes 16..31 of
// the same row).  A 16x16x32 product wants in lane l codes 8*(l/16)..+7 of
// row l%16 (of its 16 rows): each 16-lane row of the wave keeps the half it
// needs for one product and trades the other half with its neighbouring
// row, one v_permlane16_swap per dword (odd rows of the first operand
// against even rows of the second).
__device__ __forceinline__ void split16(v4i b, long &m0, long &m1) {
  const v2u s0 = __builtin_amdgcn_permlane16_swap((uint32_t)b[0], (uint32_t)b[2], false, false);
  const v2u s1 = __builtin_amdgcn_permlane16_swap((uint32_t)b[1], (uint32_t)b[3], false, false);
  m0 = __builtin_bit_cast(long, v2u{s0.x, s1.x});
  m1 = __builtin_bit_cast(long, v2u{s0.y, s1.y});
}

// B operand of block kk for token row t: codes 8c..8c+7 of the block, c =
// lane / 16, from the swizzled staging buffer.
__device__ __forceinline__ long aop16(const uint4 *abuf, int t, int kk, int c) {
  const v2u *p = reinterpret_cast<const v2u *>(abuf + t * 16 + ((2 * kk + (c >> 1)) ^ (t & 15)));
  return __builtin_bit_cast(long, p[c & 1]);
}

struct BlockIn16 {
  long a;
  float4 dw0, dw1;
  float2 dx;
};
__device__ __forceinline__ BlockIn16 block_in16(const uint4 *abuf, const float *dw,
                                                const float2 *dxb, int kk, int t, int c) {
  BlockIn16 o;
  o.a = aop16(abuf, t, kk, c);
  o.dw0 = *reinterpret_cast<const float4 *>(dw + 4 * c);
  o.dw1 = *reinterpret_cast<const float4 *>(dw + 16 + 4 * c);
  o.dx = dxb[t];
  return o;
}
// One block of a 16-row tile: acc[e] += s_e * dx * dw[e] as in scale4.
__device__ __forceinline__ void block16(float acc[16], const BlockIn16 &in, v4i b, v4i c4) {
  long m0, m1;
  split16(b, m0, m1);
  const v4f f0 = mm16(m0, in.a, c4);
  const v4f f1 = mm16(m1, in.a, c4);
  const float dx = in.dx.x, nbx = in.dx.y;
  acc[0] = fmaf(fmaf(f0[0], dx, nbx), in.dw0.x, acc[0]);
  acc[1] = fmaf(fmaf(f0[1], dx, nbx), in.dw0.y, acc[1]);
  acc[2] = fmaf(fmaf(f0[2], dx, nbx), in.dw0.z, acc[2]);
  acc[3] = fmaf(fmaf(f0[3], dx, nbx), in.dw0.w, acc[3]);
  acc[4] = fmaf(fmaf(f1[0], dx, nbx), in.dw1.x, acc[4]);
  acc[5] = fmaf(fmaf(f1[1], dx, nbx), in.dw1.y, acc[5]);
  acc[6] = fmaf(fmaf(f1[2], dx, nbx), in.dw1.z, acc[6]);
  acc[7] = fmaf(fmaf(f1[3], dx, nbx), in.dw1.w, acc[7]);
}

// One tile: rows token rows (1..64) of expert's group from sorted position
// pos (or of the dense rows from pos), against weight slices s0 .. s0 + ns
// - 1 (ns > 1 only for resident codes and the down projection).  TWO: the
// tile holds more than 32 rows (a compile-time branch: a run-time one inside
// the block loop makes the compiler keep every block's second product until
// the loop's end).
template <bool GATEUP, bool TWO, bool RES, bool SK, bool H16 = false>
__device__ __forceinline__ void mfma_tile(const MArgs &a, MLds &L, int expert, int pos, int rows,
                                          int s0, int ns) {
  static_assert(!(TWO && H16), "a 16-row tile has one half");
  constexpr int NWV = TWO ? 4 : (H16 ? 1 : 2);   // waves that stage the codes
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int r32 = lane & 31, hh = lane >> 5;
  const int nblk = (int)(a.K / 32), G = (int)(a.K / 256);
  constexpr bool resident = RES;                  // G <= 2: every group staged once

  if (tid < MT) {
    int p = -1, r = -1;
    if (tid < rows) {
      p = a.M ? pos + tid : a.perm[pos + tid];
      r = GATEUP ? (p < a.T * a.k ? p / (int)a.k : p - (int)(a.T * a.k)) : p;
    }
    L.pair[tid] = p;
    L.arow[tid] = r;
    if (!GATEUP) L.pw[tid] = p >= 0 ? pair_weight(a, p) : 0.0f;
  }
  __syncthreads();
  if (tid < MT && L.arow[tid] < 0) L.arow[tid] = L.arow[0];   // padding rows read a valid row
  __syncthreads();
  // activation scales: thread t moves row t%64, blocks t/64 and t/64 + 4 of
  // each group, divided by 16 (zero for padding rows)
  const int dm = tid & (MT - 1), dj = tid >> 6;
  const float dlive = L.pair[dm] >= 0 ? 0.0625f : 0.0f;
  const float *dsrc = a.actd + (int64_t)L.arow[dm] * nblk + dj;
  float dx0 = 0.0f, dx1 = 0.0f;
  if (resident) {
    for (int g = 0; g < G; g++) {
      stage_codes(a, L, g, g, NWV, wave, lane, nblk);
      L.dx[g][dj][dm] = scale_pair(dlive * dsrc[8 * g]);
      L.dx[g][dj + 4][dm] = scale_pair(dlive * dsrc[8 * g + 4]);
    }
  } else {
    stage_codes(a, L, 0, 0, NWV, wave, lane, nblk);
    dx0 = dsrc[0];
    dx1 = dsrc[4];
  }

  // this lane's half of its weight row in slice s, and the step to the
  // next group of 8 blocks
  const int64_t rowbytes = (int64_t)nblk * Q4B;
  const uint8_t *Wx = (expert < a.E ? a.w + (int64_t)expert * a.N * rowbytes : a.ws) + 72 * hh;
  auto wrow = [&](int s) -> const uint8_t * {
    int64_t grow;
    if (GATEUP) {
      const int64_t col = (int64_t)s * 64 + 16 * wave + (r32 & 15);
      grow = r32 < 16 ? col : a.I + col;
    } else {
      // a last slice past N (dense products) reads row N - 1 and stores nothing
      grow = min((int64_t)s * WROWS + 32 * wave + r32, a.N - 1);
    }
    return Wx + grow * rowbytes;
  };
  // this wave's weight-row scales of the current group: [block][row], rows
  // padded to 36 so the two wave halves write distinct banks
  float *const Lw = &L.dw[wave][0][0];

  float acc0[16], acc1[16];
#pragma unroll
  for (int e = 0; e < 16; e++) { acc0[e] = 0.0f; acc1[e] = 0.0f; }
  v16i c0;
#pragma unroll
  for (int e = 0; e < 16; e++) c0[e] = BIAS;

  const int J = ns * G;
  // group j with its weights in w; loads group j + 1 into wn (the last group
  // reloads itself: no conditional loads into a register array)
  auto step = [&](int j, const HW &w, HW &wn) {
    const int sj = j / G, g = j - sj * G;
    if (!resident) {
      // buffer g&1 was last read in group g - 2, before the previous barrier
      L.dx[g & 1][dj][dm] = scale_pair(dlive * dx0);
      L.dx[g & 1][dj + 4][dm] = scale_pair(dlive * dx1);
    }
    if (!resident || j == 0) {
      __builtin_amdgcn_s_waitcnt(0);              // codes, scales and weights have landed
      __syncthreads();                            // ... for every wave
    }
    // next group's codes, then its weights.  The codes go first: the
    // compiler cannot tell the direct loads into the other buffer from the
    // reads of this one and waits for them before this group's products,
    // so only loads issued after them stay in flight across the group.
    if (!resident && g + 1 < G) {
      stage_codes(a, L, g + 1, (g + 1) & 1, NWV, wave, lane, nblk);
      dx0 = dsrc[8 * (g + 1)];
      dx1 = dsrc[8 * (g + 1) + 4];
    }
    const int jn = j + 1 < J ? j + 1 : j;
    const int sn = jn / G;
    load_hw(wrow(s0 + sn) + (int64_t)(jn - sn * G) * (8 * Q4B), wn);
    // this group's weight-row scales to the wave's table: blocks 4hh..4hh+3
    // of row r32 (the wave's earlier reads of the table were issued before
    // these writes, and LDS runs one wave's accesses in order)
#pragma unroll
    for (int jj = 0; jj < 4; jj++) {
      const uint32_t sd = hw_sdw(w, jj);
      Lw[(4 * hh + jj) * DWS + r32] = f16_bits_to_f32((jj & 1) ? sd >> 16 : sd);
    }
    __builtin_amdgcn_wave_barrier();
    const int buf = resident ? g : (g & 1);
    const float2(*dxb)[MT] = L.dx[buf];
    const uint4 *abuf = L.a[buf];
    // each block's LDS operands are read one block ahead of its products
    // (order 0, 4, 1, 5, 2, 6, 3, 7)
    if constexpr (H16) {
      const int t16 = lane & 15, c16 = lane >> 4;
      const v4i c4 = v4i{BIAS, BIAS, BIAS, BIAS};
      BlockIn16 nx = block_in16(abuf, Lw, dxb[0], 0, t16, c16);
#pragma unroll
      for (int jj = 0; jj < 4; jj++) {
        v4i b0, b1;
        uint32_t sd0, sd1;
        pair_ops(w, jj, b0, b1, sd0, sd1);
        BlockIn16 cur = nx;
        nx = block_in16(abuf, Lw + (jj + 4) * DWS, dxb[jj + 4], jj + 4, t16, c16);
        block16(acc0, cur, b0, c4);
        cur = nx;
        if (jj + 1 < 4) nx = block_in16(abuf, Lw + (jj + 1) * DWS, dxb[jj + 1], jj + 1, t16, c16);
        block16(acc0, cur, b1, c4);
      }
    } else {
      BlockIn nx = block_in<TWO, !SK>(abuf, Lw, dxb[0], 0, r32, hh);
#pragma unroll
      for (int jj = 0; jj < 4; jj++) {
        v4i b0, b1;
        uint32_t sd0, sd1;
        pair_ops(w, jj, b0, b1, sd0, sd1);
        BlockIn cur = nx;
        nx = block_in<TWO, !SK>(abuf, Lw + (jj + 4) * DWS, dxb[jj + 4], jj + 4, r32, hh);
        block<TWO, !SK>(acc0, acc1, cur, b0, c0, r32);
        cur = nx;
        if (jj + 1 < 4)
          nx = block_in<TWO, !SK>(abuf, Lw + (jj + 1) * DWS, dxb[jj + 1], jj + 1, r32, hh);
        block<TWO, !SK>(acc0, acc1, cur, b1, c0, r32);
      }
    }
    if (g + 1 < G) return;

    const int slice = s0 + sj;
    if (GATEUP) {
      __syncthreads();                            // the code buffers become the h tile
      // element e < 8 holds the gate sum and e + 8 the up sum of column
      // 16*wave + 8*(e/4) + 4*hh + e%4 for this lane's token (16-row tiles:
      // e < 4 gate and e + 4 up of column 16*wave + 4*(lane/16) + e of
      // token lane%16)
      if constexpr (H16) {
        const float *acc = acc0;
        *reinterpret_cast<float4 *>(&L.hv[lane & 15][16 * wave + 4 * (lane >> 4)]) =
            make_float4(silu_f32(acc[0]) * acc[4], silu_f32(acc[1]) * acc[5],
                        silu_f32(acc[2]) * acc[6], silu_f32(acc[3]) * acc[7]);
      } else {
#pragma unroll
      for (int half = 0; half < (TWO ? 2 : 1); half++) {
        const float *acc = half ? acc1 : acc0;
        float *hrow = &L.hv[32 * half + r32][16 * wave + 4 * hh];
#pragma unroll
        for (int q = 0; q < 2; q++)
          *reinterpret_cast<float4 *>(hrow + 8 * q) =
              make_float4(silu_f32(acc[4 * q + 0]) * acc[4 * q + 8],
                          silu_f32(acc[4 * q + 1]) * acc[4 * q + 9],
                          silu_f32(acc[4 * q + 2]) * acc[4 * q + 10],
                          silu_f32(acc[4 * q + 3]) * acc[4 * q + 11]);
      }
      }
      __syncthreads();
      // Q8_0 of each row's two 32-wide blocks: 8 lanes per block
      const int nbh = (int)(a.I / 32);
#pragma unroll
      for (int pass = 0; pass < 4; pass++) {
        const int idx = pass * MNT + tid;
        const int rb = idx >> 3, jq = idx & 7, m = rb >> 1, cb = rb & 1;
        const int p = L.pair[m];
        if (p >= 0) {                             // whole 8-lane groups agree
          const float4 hv4 = *reinterpret_cast<const float4 *>(&L.hv[m][32 * cb + 4 * jq]);
          const float v[4] = {hv4.x, hv4.y, hv4.z, hv4.w};
          uint32_t d16;
          const uint32_t packed = q8_0_block8(v, d16);
          const int bi = 2 * slice + cb;
          const int64_t blk = (int64_t)p * nbh + bi;
          store_q8_0_block8(a.hq + blk * Q8B, jq, packed, d16);
          a.ha[blk * 8 + jq] = packed;
          if (jq == 0) a.hd[blk] = f16_bits_to_f32(d16);
          *reinterpret_cast<float4 *>(a.h + (int64_t)p * a.I + 32 * bi + 4 * jq) = hv4;
        }
      }
    } else {
      // element 4q + i: output column slice*128 + 32*wave + 8q + 4hh + i
      // (16-row tiles: element 4q + i of token lane%16, column slice*128 +
      // 32*wave + 16q + 4*(lane/16) + i)
      const bool vec = (a.N & 3) == 0;
      if constexpr (H16) {
        const int m = lane & 15;
        const int p = L.pair[m];
        const float pw = L.pw[m];
        if (p >= 0) {
          float *yrow = a.y + (int64_t)p * a.N;
          const int64_t nb = (int64_t)slice * WROWS + 32 * wave + 4 * (lane >> 4);
#pragma unroll
          for (int q = 0; q < 2; q++) {
            const int64_t n = nb + 16 * q;
            if (vec && n + 3 < a.N) {
              *reinterpret_cast<float4 *>(yrow + n) =
                  make_float4(pw * acc0[4 * q], pw * acc0[4 * q + 1], pw * acc0[4 * q + 2],
                              pw * acc0[4 * q + 3]);
            } else {
#pragma unroll
              for (int i = 0; i < 4; i++)
                if (n + i < a.N) yrow[n + i] = pw * acc0[4 * q + i];
            }
          }
        }
      }
      const int64_t n0 = (int64_t)slice * WROWS + 32 * wave + 4 * hh;
#pragma unroll
      for (int half = 0; half < (H16 ? 0 : (TWO ? 2 : 1)); half++) {
        const float *acc = half ? acc1 : acc0;
        const int m = 32 * half + r32;
        const int p = L.pair[m];
        const float pw = L.pw[m];
        if (p < 0) continue;
        float *yrow = a.y + (int64_t)p * a.N;
#pragma unroll
        for (int q = 0; q < 4; q++) {
          const int64_t n = n0 + 8 * q;
          if (vec && n + 3 < a.N) {
            *reinterpret_cast<float4 *>(yrow + n) =
                make_float4(pw * acc[4 * q], pw * acc[4 * q + 1], pw * acc[4 * q + 2],
                            pw * acc[4 * q + 3]);
          } else {
#pragma unroll
            for (int i = 0; i < 4; i++)
              if (n + i < a.N) yrow[n + i] = pw * acc[4 * q + i];
          }
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 16; e++) { acc0[e] = 0.0f; acc1[e] = 0.0f; }
  };

  HW wa, wb;
  load_hw(wrow(s0), wa);
  for (int j = 0; j < J; j += 2) {
    step(j, wa, wb);
    if (j + 1 < J) step(j + 1, wb, wa);
  }
}

template <bool GATEUP, bool SHORT>
__device__ __forceinline__ void mfma_body(const MArgs &a, MLds &L) {
  // Work items are (tile, chunk), chunk = a run of spw slices.  Workgroup b
  // runs on XCD b % 8 and is the (b / 8)-th item there.  Each XCD takes an
  // even share of the long tiles (more than 32 rows), then an even share of
  // the short ones, each share a contiguous run of tiles (neighbouring tiles
  // of one expert share its weights in that XCD's L2), and all chunks of a
  // tile in a row (they share the tile's codes).
  const int nsl = (int)(GATEUP ? a.I / 64 : (a.N + WROWS - 1) / WROWS);
  const int nch = (nsl + a.spw - 1) / a.spw;
  const int x = blockIdx.x & 7, q = blockIdx.x >> 3;
  int expert, pos, rows, s0;
  if (a.M) {
    // Dense products: the items in chunk-major order (all 64-row tiles of
    // the activations for one chunk of weight rows in a row), XCD x taking
    // the x-th of 8 even contiguous runs: the tiles of one chunk share its
    // weights in that XCD's L2, and every XCD streams its own part of the
    // weights, so a handful of tiles still spreads over all 8.
    const int ntl = (int)((a.M + a.tr - 1) / a.tr);
    const int tot = nch * ntl;
    const int i0 = x * tot / 8, nx = (x + 1) * tot / 8 - i0;
    if (q >= nx) return;
    const int c = (i0 + q) / ntl, tile = (i0 + q) - c * ntl;
    s0 = c * a.spw;
    expert = 0;                  // E = 0: the weights are ws
    pos = tile * a.tr;
    rows = (int)min((int64_t)a.tr, a.M - pos);
  } else {
    const int ch = q % nch, qt = q / nch;
    const int ntiles = ((CInt *)a.meta)[2], nlong = ((CInt *)a.meta)[4];   // META_NTILES, META_NLONG
    const int l0 = x * nlong / 8, nl = (x + 1) * nlong / 8 - l0;
    const int nshort = ntiles - nlong;
    const int s0t = nlong + x * nshort / 8, ns_ = nlong + (x + 1) * nshort / 8 - s0t;
    if (qt >= nl + ns_) return;
    const int tile = qt < nl ? l0 + qt : s0t + (qt - nl);
    s0 = ch * a.spw;
    CInt *tp = (CInt *)a.tiles + 4 * tile;
    expert = tp[0]; pos = tp[1]; rows = tp[2];
  }
  const int ns = min(a.spw, nsl - s0);
  if (a.K <= 512) {
    if (!SHORT && rows > 32)
      mfma_tile<GATEUP, true, true, SHORT>(a, L, expert, pos, rows, s0, ns);
    else if (rows > 16)
      mfma_tile<GATEUP, false, true, SHORT>(a, L, expert, pos, rows, s0, ns);
    else
      mfma_tile<GATEUP, false, true, SHORT, true>(a, L, expert, pos, rows, s0, ns);
  } else {
    if (!SHORT && rows > 32)
      mfma_tile<GATEUP, true, false, SHORT>(a, L, expert, pos, rows, s0, ns);
    else if (rows > 16)
      mfma_tile<GATEUP, false, false, SHORT>(a, L, expert, pos, rows, s0, ns);
    else
      mfma_tile<GATEUP, false, false, SHORT, true>(a, L, expert, pos, rows, s0, ns);
  }
}

// Tiles of up to 64 rows: two waves per SIMD (the 64-row tile's two sets of
// sums and products need about 200 registers a lane; at three waves the
// compiler spills inside the block loop).
template <bool GATEUP>
__global__ __launch_bounds__(MNT) __attribute__((amdgpu_waves_per_eu(2))) void mfma_kernel(MArgs a) {
  __shared__ MLds L;
  mfma_body<GATEUP, false>(a, L);
}

// Dense products of at most 32 rows (every tile short): one set of sums,
// three waves per SIMD to keep more weight bytes in flight.
__global__ __launch_bounds__(MNT) __attribute__((amdgpu_waves_per_eu(3))) void mfma_short_kernel(MArgs a) {
  __shared__ MLds L;
  mfma_body<false, true>(a, L);
}

}  // namespace

int mfma_tile_rows() { return MT; }

int mfma_gateup(const uint8_t *w_gu, const uint8_t *ws_gu, const uint32_t *xa, const float *xd,
                const int32_t *meta, const int32_t *perm, const int4 *tiles, float *h,
                uint8_t *hq, uint32_t *ha, float *hd, int64_t maxtiles, int64_t T, int64_t H,
                int64_t I, int64_t E, int64_t k, hipStream_t s) {
  MArgs a{};
  a.w = w_gu; a.ws = ws_gu; a.act = xa; a.actd = xd;
  a.meta = meta; a.perm = perm; a.tiles = tiles;
  a.h = h; a.hq = hq; a.ha = ha; a.hd = hd;
  a.T = T; a.k = k; a.E = E; a.N = 2 * I; a.K = H; a.I = I;
  a.spw = 1;                       // the h tile reuses the code buffers
  // an XCD takes at most ceil(long/8) + ceil(short/8) <= ceil(maxtiles/8) + 1 tiles
  mfma_kernel<true><<<dim3((unsigned)(8 * ((maxtiles + 7) / 8 + 1) * (I / 64))), dim3(MNT), 0, s>>>(a);
  return check_launch();
}

int mfma_down(const uint8_t *w_d, const uint8_t *ws_d, const uint32_t *ha, const float *hd,
              const int32_t *meta, const int32_t *perm, const int4 *tiles, const float *topk_w,
              const float *shared_w, float *y, int64_t maxtiles, int64_t T, int64_t H, int64_t I,
              int64_t E, int64_t k, bool few, hipStream_t s) {
  MArgs a{};
  a.w = w_d; a.ws = ws_d; a.act = ha; a.actd = hd;
  a.meta = meta; a.perm = perm; a.tiles = tiles;
  a.topk_w = topk_w; a.shared_w = shared_w; a.y = y;
  a.T = T; a.k = k; a.E = E; a.N = H; a.K = I; a.I = I;
  const int64_t nsl = H / WROWS;
  // few tiles: one slice per workgroup, so the slices spread over more
  // compute units
  a.spw = I <= 512 && !few ? (int)std::min<int64_t>(SPW_MAX, nsl) : 1;
  const int64_t nch = (nsl + a.spw - 1) / a.spw;
  mfma_kernel<false><<<dim3((unsigned)(8 * ((maxtiles + 7) / 8 + 1) * nch)), dim3(MNT), 0, s>>>(a);
  return check_launch();
}

// Dense product y[m][n] = sum_b d_w[n,b] d_x[m,b] s[m,n,b] of M activation
// rows (aligned codes and fp32 scales) with one weight matrix [N][K/32].
int mfma_dense(const uint8_t *w, const uint32_t *act, const float *actd, float *y, int64_t M,
               int64_t N, int64_t K, hipStream_t s) {
  MArgs a{};
  a.w = nullptr; a.ws = w; a.act = act; a.actd = actd; a.y = y;
  a.T = 0; a.k = 0; a.E = 0; a.N = N; a.K = K; a.I = K; a.M = M;
  const int64_t nsl = (N + WROWS - 1) / WROWS;
  a.tr = MT;
  a.spw = K <= 512 ? (int)std::min<int64_t>(SPW_MAX, nsl) : 1;
  const int64_t nch = (nsl + a.spw - 1) / a.spw;
  const int64_t ntiles = (M + a.tr - 1) / a.tr;
  const int64_t grid = 8 * ((nch * ntiles + 7) / 8);    // an XCD takes at most ceil(items/8)
  if (grid >= ((int64_t)1 << 31)) return W4A8_ERANGE;
  if (M <= MT / 2)
    mfma_short_kernel<<<dim3((unsigned)grid), dim3(MNT), 0, s>>>(a);
  else
    mfma_kernel<false><<<dim3((unsigned)grid), dim3(MNT), 0, s>>>(a);
  return check_launch();
}

}  // namespace w4a8
