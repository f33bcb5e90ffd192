// Internal device helpers shared by the gfx950 kernels of libw4a8.
//
// Register-level decoding of the two block formats.  A lane that owns eight
// consecutive blocks of a row holds 144 bytes of Q4_0 (36 dwords, 16-byte
// aligned when the row length is a multiple of 256) or 272 bytes of Q8_0 (68
// dwords).  Blocks at even positions start on a dword boundary and their
// payload is two bytes off; odd blocks are the other way round, so each
// payload dword is one v_alignbyte away from the raw loads.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/w4a8.h"

namespace w4a8 {

constexpr int QK = 32;
constexpr int Q4B = W4A8_Q4_0_BLOCK_BYTES;  // 18
constexpr int Q8B = W4A8_Q8_0_BLOCK_BYTES;  // 34

__device__ __forceinline__ float f16_bits_to_f32(uint32_t bits) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(bits & 0xFFFFu));
}

__device__ __forceinline__ uint32_t f32_to_f16_bits(float f) {
  // v_cvt_f16_f32: round to nearest even (default mode), fp16 denormals kept.
  // The empty asm pins f as an fp32 register value: otherwise the compiler
  // may fuse the producing multiply into v_fma_mix with a +0 addend, which
  // turns a -0 scale into +0.
  asm volatile("" : "+v"(f));
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)f);
}

__device__ __forceinline__ uint32_t align2(uint32_t hi, uint32_t lo) {
  // bytes 2,3 of lo followed by bytes 0,1 of hi
  return __builtin_amdgcn_alignbyte(hi, lo, 2);
}

__device__ __forceinline__ int sdot4(int a, int b, int c) {
  return __builtin_amdgcn_sdot4(a, b, c, false);
}

// Eight Q8_0 blocks in registers: codes q[k][c] hold elements 4c..4c+3 of
// block k; corr[k] = -8 * sum of the 32 codes (folds the Q4_0 offset of 8
// into the integer dot); d[k] the block scale.
struct Act8 {
  int q[8][8];
  int corr[8];
  float d[8];
};

// p: 272 bytes (8 blocks), 16-byte aligned.
__device__ __forceinline__ void load_act8(const uint8_t *__restrict__ p, Act8 &a) {
  uint32_t D[68];
  const uint4 *v = reinterpret_cast<const uint4 *>(p);
#pragma unroll
  for (int i = 0; i < 17; i++) {
    uint4 t = v[i];
    D[4 * i + 0] = t.x; D[4 * i + 1] = t.y; D[4 * i + 2] = t.z; D[4 * i + 3] = t.w;
  }
#pragma unroll
  for (int k = 0; k < 8; k++) {
    const int i = k >> 1;
    if ((k & 1) == 0) {
      const int base = 17 * i;
      a.d[k] = f16_bits_to_f32(D[base]);
#pragma unroll
      for (int c = 0; c < 8; c++) a.q[k][c] = (int)align2(D[base + c + 1], D[base + c]);
    } else {
      const int base = 17 * i + 8;
      a.d[k] = f16_bits_to_f32(D[base] >> 16);
#pragma unroll
      for (int c = 0; c < 8; c++) a.q[k][c] = (int)D[base + 1 + c];
    }
    int s = 0;
#pragma unroll
    for (int c = 0; c < 8; c++) s = sdot4(a.q[k][c], 0x01010101, s);
    a.corr[k] = -8 * s;
  }
}

// Eight Q4_0 blocks of one row (144 bytes) in 36 raw dwords.
struct W8 {
  uint32_t D[36];
};

__device__ __forceinline__ void load_w8(const uint8_t *__restrict__ p, W8 &w) {
  const uint4 *v = reinterpret_cast<const uint4 *>(p);
#pragma unroll
  for (int i = 0; i < 9; i++) {
    uint4 t = v[i];
    w.D[4 * i + 0] = t.x; w.D[4 * i + 1] = t.y; w.D[4 * i + 2] = t.z; w.D[4 * i + 3] = t.w;
  }
}

// Scale and the four payload dwords (nibble bytes 4c..4c+3) of block k.
__device__ __forceinline__ float w8_scale(const W8 &w, int k) {
  const int i = k >> 1;
  return (k & 1) == 0 ? f16_bits_to_f32(w.D[9 * i]) : f16_bits_to_f32(w.D[9 * i + 4] >> 16);
}
__device__ __forceinline__ uint32_t w8_nib(const W8 &w, int k, int c) {
  const int i = k >> 1;
  return (k & 1) == 0 ? align2(w.D[9 * i + c + 1], w.D[9 * i + c]) : w.D[9 * i + 5 + c];
}

// Exact int32 block dot s = sum (q_w - 8) * q_a of block k.
__device__ __forceinline__ int blockdot(const W8 &w, const Act8 &a, int k) {
  int s = a.corr[k];
#pragma unroll
  for (int c = 0; c < 4; c++) {
    const uint32_t n = w8_nib(w, k, c);
    s = sdot4((int)(n & 0x0F0F0F0Fu), a.q[k][c], s);
    s = sdot4((int)((n >> 4) & 0x0F0F0F0Fu), a.q[k][4 + c], s);
  }
  return s;
}

// acc + sum over the eight blocks of d_w * d_a * s, in fp32.
__device__ __forceinline__ float dot8(const W8 &w, const Act8 &a, float acc) {
#pragma unroll
  for (int k = 0; k < 8; k++) {
    const int s = blockdot(w, a, k);
    acc = fmaf((float)s, w8_scale(w, k) * a.d[k], acc);
  }
  return acc;
}

// Cross-lane moves through DPP (a VALU operand modifier, no LDS round trip).
// quad_perm [1,0,3,2] and [2,3,0,1] exchange with lane^1 and lane^2;
// row_half_mirror maps lane i of each 8-lane half-row to lane 7-i, which
// pairs every lane of one quad with a lane of the other; row_ror:8 within a
// 16-lane row gives lane^8.
constexpr int DPP_XOR1 = 0xB1, DPP_XOR2 = 0x4E, DPP_HALF_MIRROR = 0x141, DPP_ROR8 = 0x128;

template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, dpp_i<CTRL>(__builtin_bit_cast(int, v)));
}

// Reductions over each group of 8 consecutive lanes (all 8 must be active);
// every lane of a group ends with the same value (fp32 addition is
// commutative, so the mirrored partners compute identical sums).
__device__ __forceinline__ float sum8(float v) {
  v += dpp_f<DPP_XOR1>(v);
  v += dpp_f<DPP_XOR2>(v);
  v += dpp_f<DPP_HALF_MIRROR>(v);
  return v;
}
__device__ __forceinline__ int sum8(int v) {
  v += dpp_i<DPP_XOR1>(v);
  v += dpp_i<DPP_XOR2>(v);
  v += dpp_i<DPP_HALF_MIRROR>(v);
  return v;
}
__device__ __forceinline__ float max8(float v) {
  v = fmaxf(v, dpp_f<DPP_XOR1>(v));
  v = fmaxf(v, dpp_f<DPP_XOR2>(v));
  v = fmaxf(v, dpp_f<DPP_HALF_MIRROR>(v));
  return v;
}

// Lane i of each 8-lane group receives lane i ^ 4's value: row_ror:12 (lane
// i reads lane i + 4 of its 16-lane row) into DPP banks 0 and 2, row_ror:4
// (lane i - 4) into banks 1 and 3.
constexpr int DPP_ROR4 = 0x124, DPP_ROR12 = 0x12C;
__device__ __forceinline__ uint32_t xchg4(uint32_t v) {
  const int t = __builtin_amdgcn_update_dpp(0, (int)v, DPP_ROR12, 0xF, 0x5, false);
  return (uint32_t)__builtin_amdgcn_update_dpp(t, (int)v, DPP_ROR4, 0xF, 0xA, false);
}

// Nibble-split form of a Q8_0 block, for the 4-bit dot products.  A code x
// in [-127, 127] is 16 * (x >> 4) + (x & 15): a signed nibble in [-8, 7] and
// an unsigned nibble in [0, 15].  Dwords 0..3 of the block hold the signed
// parts, dwords 4..7 the unsigned parts, each in the nibble order of the
// Q4_0 payload dword with the same index c: nibbles 2i and 2i+1 belong to
// elements 4c+i and 4c+i+16.  Lane j of an 8-lane group holding the codes of
// elements 4j..4j+3 (one byte each, `packed`) returns dword j of the form;
// all 8 lanes must be active.
__device__ __forceinline__ uint32_t split_word(uint32_t packed, int j) {
  const uint32_t other = xchg4(packed);
  return j < 4 ? (other & 0xF0F0F0F0u) | ((packed >> 4) & 0x0F0F0F0Fu)
               : ((packed << 4) & 0xF0F0F0F0u) | (other & 0x0F0F0F0Fu);
}
// Sum of the unsigned nibbles of the lane's four codes (0..60).
__device__ __forceinline__ int low_nibble_sum(uint32_t packed) {
  return sdot4((int)(packed & 0x0F0F0F0Fu), 0x01010101, 0);
}

// A nibble-split Q8_0 block in global memory: the 8 dwords of split_word,
// the fp32 scale and -8 * (sum of the unsigned nibbles), padded to 48 bytes
// so that blocks copy and read as 16-byte pieces.
struct SplitBlk {
  uint32_t w[8];
  float d;
  int corr;
  int pad[2];
};
static_assert(sizeof(SplitBlk) == 48, "split block layout");

// Rows of SplitBlk in global memory (the small-group kernels' activations):
// every group of 8 blocks takes 8 records (384 bytes) and 16 bytes of
// padding, so that in an LDS copy of a row the lanes reading different
// groups hit different banks.  nblk (blocks per row) is a multiple of 8.
constexpr int SPLIT_GROUP_BYTES = 400;
__host__ __device__ constexpr size_t split_row_bytes(int64_t nblk) {
  return (size_t)(nblk / 8) * SPLIT_GROUP_BYTES;
}
__device__ __forceinline__ SplitBlk *split_blk(uint8_t *base, int64_t row, int64_t nblk,
                                               int64_t blk) {
  return reinterpret_cast<SplitBlk *>(base + row * (int64_t)split_row_bytes(nblk) +
                                      (blk >> 3) * SPLIT_GROUP_BYTES + (blk & 7) * 48);
}

// SiLU(g) = g / (1 + e^-g) with the hardware base-2 exponential and
// reciprocal (each within about one ulp).
__device__ __forceinline__ float silu_f32(float g) {
  return g * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(g * -1.44269504f));
}

// Exact block dot s = sum (q_w - 8) * x over a block in nibble-split form:
// q_w - 8 is the signed nibble q_w ^ 8, so
//   s = 16 * sum (q_w ^ 8) * hi + sum q_w * lo - 8 * sum lo,
// two 8-wide 4-bit dot products per payload dword and no unpacking of the
// weights; corr = -8 * sum lo.
// n: the block's four payload dwords (stored nibbles q_w).
__device__ __forceinline__ int blockdot_nib(const uint32_t n[4], uint4 hi, uint4 lo, int corr) {
  const uint32_t h[4] = {hi.x, hi.y, hi.z, hi.w};
  const uint32_t l[4] = {lo.x, lo.y, lo.z, lo.w};
  int sa = 0;
  uint32_t sb = (uint32_t)corr;
#pragma unroll
  for (int c = 0; c < 4; c++) {
    sa = __builtin_amdgcn_sdot8((int)(n[c] ^ 0x88888888u), (int)h[c], sa, false);
    sb = __builtin_amdgcn_udot8(n[c], l[c], sb, false);
  }
  return (int)(((uint32_t)sa << 4) + sb);
}
// The same for block k of a Q4_0 group.
__device__ __forceinline__ int blockdot_split(const W8 &w, int k, uint4 hi, uint4 lo, int corr) {
  const uint32_t n[4] = {w8_nib(w, k, 0), w8_nib(w, k, 1), w8_nib(w, k, 2), w8_nib(w, k, 3)};
  return blockdot_nib(n, hi, lo, corr);
}

// Activation blocks staged in LDS in nibble-split form: block i at codes[2i]
// (signed parts) and codes[2i+1] (unsigned parts), its fp32 scale d[i] and
// corr[i] = -8 * (sum of its unsigned parts).  acc + sum over the eight
// blocks of d_w * d_a * s, in fp32; one block's activations live at a time.
__device__ __forceinline__ float dot8_lds(const W8 &w, const uint4 *__restrict__ codes,
                                          const float *__restrict__ d,
                                          const int *__restrict__ corr, float acc) {
#pragma unroll
  for (int k = 0; k < 8; k++) {
    const int s = blockdot_split(w, k, codes[2 * k], codes[2 * k + 1], corr[k]);
    acc = fmaf((float)s, w8_scale(w, k) * d[k], acc);
  }
  return acc;
}

// Sum over groups of `width` consecutive lanes (width a power of two <= 64).
template <int WIDTH>
__device__ __forceinline__ float lane_group_sum(float v) {
#pragma unroll
  for (int o = WIDTH / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, WIDTH);
  return v;
}

// Q8_0 of one 32-value block held by 8 consecutive lanes, 4 values each
// (lane j of the 8 holds elements 4j..4j+3).  Returns the four codes packed
// in a dword and, through d16, the block's fp16 scale bits.  All 8 lanes of
// the group must be active.  Same fp32 steps
// as the format definition: amax, one division by 127, fp16 RNE, one
// reciprocal of the stored scale, one multiply per element, round half away.
__device__ __forceinline__ uint32_t q8_0_block8(const float v[4], uint32_t &d16) {
  const float amax =
      max8(fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
  const float d32 = amax / 127.0f;
  d16 = f32_to_f16_bits(d32);
  const float df = f16_bits_to_f32(d16);
  uint32_t packed = 0;
  if (df != 0.0f) {
    const float id = 1.0f / df;
#pragma unroll
    for (int i = 0; i < 4; i++) {
      int q = (int)roundf(v[i] * id);
      q = q > 127 ? 127 : (q < -127 ? -127 : q);
      packed |= ((uint32_t)q & 0xFFu) << (8 * i);
    }
  }
  return packed;
}

// Store a Q8_0 block produced by 8 lanes: lane j writes codes 4j..4j+3 at
// byte 2 + 4j (two 16-bit stores, the block is only 2-byte aligned) and lane
// 0 the scale.
__device__ __forceinline__ void store_q8_0_block8(uint8_t *blk, int j, uint32_t packed, uint32_t d16) {
  uint16_t *p = reinterpret_cast<uint16_t *>(blk + 2 + 4 * j);
  p[0] = (uint16_t)(packed & 0xFFFFu);
  p[1] = (uint16_t)(packed >> 16);
  if (j == 0) *reinterpret_cast<uint16_t *>(blk) = (uint16_t)d16;
}

// Q8_0 of one 32-element block of x by 8 lanes (thread tid: block tid / 8,
// elements 4 (tid % 8) .. + 3): the 34-byte block, and when the pointers are
// set its nibble-split form (xs, rows of nbrow blocks, see split_blk) and its
// 32 codes on a 32-byte boundary with the fp32 scale (xa, xd).  Lanes past
// nblocks take part in the exchanges and store nothing.  q8_0_lane_vals
// takes the lane's four values already in registers (elements 4j..4j+3 of
// block blk; live: the block exists); q8_0_lane loads them from x.
__device__ __forceinline__ void q8_0_lane_vals(const float v[4], uint8_t *__restrict__ xq,
                                               uint8_t *__restrict__ xs, uint32_t *__restrict__ xa,
                                               float *__restrict__ xd, int64_t nbrow, int64_t blk,
                                               int j, bool live) {
  uint32_t d16;
  const uint32_t packed = q8_0_block8(v, d16);
  if (live) store_q8_0_block8(xq + blk * Q8B, j, packed, d16);
  if (xs) {
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
  if (xa && live) {
    xa[blk * 8 + j] = packed;
    if (j == 0) xd[blk] = f16_bits_to_f32(d16);
  }
}

__device__ __forceinline__ void q8_0_lane(const float *__restrict__ x, uint8_t *__restrict__ xq,
                                          uint8_t *__restrict__ xs, uint32_t *__restrict__ xa,
                                          float *__restrict__ xd, int64_t nblocks, int64_t nbrow,
                                          int64_t tid) {
  const int64_t blk = tid >> 3;
  const int j = (int)(tid & 7);
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  const bool live = blk < nblocks;
  if (live) {
    const float4 t = reinterpret_cast<const float4 *>(x + blk * QK)[j];
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  }
  q8_0_lane_vals(v, xq, xs, xa, xd, nbrow, blk, j, live);
}

// LDS staging of activation blocks (see dot8_lds): each block's nibble-split
// form as 8 dwords, groups of 8 blocks 272 bytes apart (16 bytes of padding
// per group), then scale [n] fp32 and correction [n] int32, carved from one
// dynamic LDS buffer.  The lanes of a wave read up to 8 different groups at
// once; without the padding those addresses would be 256 bytes apart and all
// fall in the same LDS banks.
constexpr int GROUP_U4 = 17;   // uint4 per 8-block group: 16 of codes + 1 of padding
struct ActBuf {
  uint4 *codes;
  float *d;
  int *corr;
};

__host__ __device__ constexpr size_t act_codes_bytes(int nblocks) {
  return (size_t)((nblocks + 7) / 8) * GROUP_U4 * 16;
}
__device__ __forceinline__ ActBuf act_buf(uint8_t *base, int nblocks) {
  ActBuf b;
  b.codes = reinterpret_cast<uint4 *>(base);
  b.d = reinterpret_cast<float *>(base + act_codes_bytes(nblocks));
  b.corr = reinterpret_cast<int *>(base + act_codes_bytes(nblocks) + (size_t)nblocks * 4);
  return b;
}
__host__ __device__ constexpr size_t act_buf_bytes(int nblocks) {
  return (act_codes_bytes(nblocks) + (size_t)nblocks * 8 + 15) / 16 * 16;
}
// dword j (0..7) of block blk's nibble-split form
__device__ __forceinline__ uint32_t *code_word(ActBuf b, int blk, int j) {
  return reinterpret_cast<uint32_t *>(b.codes + (blk >> 3) * GROUP_U4) + (blk & 7) * 8 + j;
}
// the codes of the 8-block group starting at block blk0 (a multiple of 8)
__device__ __forceinline__ const uint4 *group_codes(ActBuf b, int blk0) {
  return b.codes + (blk0 >> 3) * GROUP_U4;
}

// Reciprocal of a block scale, or 0 when the block's codes are all zero (a
// zero scale, or one whose reciprocal overflows fp32).
__device__ __forceinline__ float sym_inverse(float d) {
  if (d == 0.0f) return 0.0f;
  const float id = 1.0f / d;                    // correctly rounded division
  return __builtin_isinf(id) ? 0.0f : id;
}

__device__ __forceinline__ int round_clamp(float v, int lim) {
  const int q = (int)roundf(v);                 // half away from zero
  return q > lim ? lim : (q < -lim ? -lim : q);
}

// Eight Q4_SYM blocks of one row (160 bytes) in 40 raw dwords: block k's
// scale in dword 5k, its payload in dwords 5k+1 .. 5k+4.
struct W8S {
  uint32_t D[40];
};

__device__ __forceinline__ void load_w8s(const uint8_t *__restrict__ p, W8S &w) {
  const uint4 *v = reinterpret_cast<const uint4 *>(p);
#pragma unroll
  for (int i = 0; i < 10; i++) {
    const uint4 t = v[i];
    w.D[4 * i + 0] = t.x; w.D[4 * i + 1] = t.y; w.D[4 * i + 2] = t.z; w.D[4 * i + 3] = t.w;
  }
}

__device__ __forceinline__ float dot8s_lds(const W8S &w, const uint4 *__restrict__ codes,
                                           const float *__restrict__ d,
                                           const int *__restrict__ corr, float acc) {
#pragma unroll
  for (int k = 0; k < 8; k++) {
    const uint32_t n[4] = {w.D[5 * k + 1], w.D[5 * k + 2], w.D[5 * k + 3], w.D[5 * k + 4]};
    const int s = blockdot_nib(n, codes[2 * k], codes[2 * k + 1], corr[k]);
    acc = fmaf((float)s, __builtin_bit_cast(float, w.D[5 * k]) * d[k], acc);
  }
  return acc;
}


}  // namespace w4a8
