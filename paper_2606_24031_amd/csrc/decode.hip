// Single-token MoE layer in one kernel launch (decode, T = 1).
//
// At M = 1 the layer streams (k + 1) experts' weights (8 routed + 1 shared,
// 15.9 MB for the Qwen3-family shape) and does almost no arithmetic, so its
// cost is HBM latency plus the chain of hand-offs between the gate/up and the
// down projection; an extra kernel boundary alone costs about 1.6 us.
// Everything therefore runs in one grid of about one workgroup per compute
// unit, of two kinds (the routed top-k experts and the always-on shared
// expert of Sec. 2.2; the W4A8 product of Sec. 3.3):
//
//   gate/up items (pair q, 32-column block b of h): issue the 64 gate/up row
//     loads (one 144-byte eight-block group per lane for H = 2048), quantize
//     x to Q8_0 into LDS, take the W4A8 dots, reduce each row over its 8
//     lanes with DPP (gate row and up row of one h column sit in the same
//     wave), h = SiLU(g) * u, and publish Q8_0 of the 32 h values (one block).
//   The block dots run on the 4-bit dot products: activations are staged
//   in a nibble-split form (see split_word) so that the Q4_0 payload dwords
//   feed the dots as loaded, with no unpacking of the weight nibbles.
//   down slabs (rb down rows, all pairs): first load into their XCD's L2 a
//     share of the gate/up rows that the items on that XCD read last (see
//     prefetch_gateup), then issue the down weight loads of every pair,
//     collect every pair's Q8_0(h), take the dots and write
//     out[n] = sum_q w_q y_q[n] (slots in order, then the shared expert) --
//     the combine never leaves the workgroup.  The slabs fill the compute
//     units the gate/up items leave free.
//
// Hand-off: each published word is 64 bits, the payload in the low half and
// the call's tag in the high half (per block: the fp16 scale and the sum of
// the unsigned nibbles, then the 8 dwords of the nibble-split codes), written with agent-scope (sc1) stores;
// each block's words sit alone in one 128-byte line, so no line is written
// from two XCDs.  A slab polls all the words until every one carries this
// call's tag: one poll round trip and the store's visibility cost about
// 0.5 us each across XCDs, so the words are read in a single pass rather
// than a flag first and the data after.  The tag is one more than the call
// counter kept in the hand-off region; every workgroup arrives at a
// two-level counter once it has read the tag, and the last arrival advances
// the call counter and clears the arrival counters.
//
// The wait is bounded: after `spin_rounds` poll rounds (each a load round
// trip, about 0.5-1 us) a slab computes every block itself (the same code, so the same
// bytes, also published with the same tag) straight into its own staging, so
// progress never depends on the order in which the hardware starts
// workgroups.
//
// With the router in front (router logits instead of ids and weights), every
// workgroup first takes the token's top-k itself in one wave (wave_topk, the
// router kernel's own code, so the same decisions and bits) into LDS; the
// first workgroup also writes the ids, weights and gate value out.  The
// selection costs a few hundred ns on each workgroup's path to its weight
// loads, less than a launch of its own and the gap behind it.
#include <algorithm>
#include <atomic>
#include <cstdlib>

#include "router_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int NT = 512;          // threads per workgroup: 8 waves
constexpr int NSUB = 8;          // first-level arrival counters
constexpr int XW = 9;            // hand-off words per h block: scale and nibble sum, 8 code words
constexpr int XSTRIDE = 16;      // 64-bit words between blocks: each block alone in a 128-byte line
constexpr int XFER_HDR = 64;     // uint32 words ahead of the hand-off words: the call counter

// Arrival counters (uint32, zero between calls), each alone in its own
// 256-byte line: same-line atomics serialize in the memory system.
constexpr int SYNC_STRIDE = 64;
constexpr int SYNC_SUB = 0, SYNC_TOP = NSUB, SYNC_SLOTS = NSUB + 1;
__device__ __forceinline__ uint32_t *sync_word(uint32_t *sync, int slot) {
  return sync + slot * SYNC_STRIDE;
}

struct DecodeArgs {
  const float *x;          // [H]
  const int32_t *ids;      // [k]
  const float *topk_w;     // [k]
  const float *shared_w;   // the shared expert's weight [1], or null (1)
  const uint8_t *w_gu, *w_d, *ws_gu, *ws_d;
  float *out;              // [H]
  uint32_t *sync;          // arrival counters
  uint32_t *calls;         // call counter (tag of this call = *calls + 1)
  uint64_t *xfer;          // Q8_0(h) hand-off: [(k+1) * I/32][XSTRIDE] tagged words (XW used)
  // pre-norm residual input (gamma != nullptr): the layer's input is
  // xn = RMSNorm(x + resid) * gamma instead of x; workgroup 0 writes
  // x_out = x + resid and the documented copy xn
  const float *resid;      // [H] or nullptr
  const float *gamma;      // [H] or nullptr (no norm)
  float *x_out, *xn;       // [H]
  float eps;
  uint8_t *xq;             // documented copy of Q8_0(x)   [H/32 blocks]
  float *h;                // documented copy of h          [(k+1)][I]
  uint8_t *hq;             // documented copy of Q8_0(h)    [(k+1)][I/32 blocks]
  // router in front (logits != nullptr): ids, topk_w and shared_w are
  // taken in the launch (see route_in_wg) and written out by workgroup 0
  const float *logits;     // [E] or nullptr
  const float *gate;       // the shared expert's gate logit [1], or nullptr
  int32_t *route_ids;      // [k]
  float *route_w;          // [k]
  float *route_gate;       // [1]
  int H, I, E, k;
  int rb;                  // down rows per slab
  int spin_rounds;         // poll rounds before a slab computes h itself
  int prefetch;            // down slabs first load the late gate/up rows (L2)
};

__device__ __forceinline__ bool pair_valid(const DecodeArgs &a, int q, int &expert) {
  if (q < a.k) {
    expert = a.ids[q];
    return expert >= 0 && expert < a.E;
  }
  expert = a.E;
  return a.ws_gu != nullptr;
}

__device__ __forceinline__ uint32_t counter_add(uint32_t *p, uint32_t v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_agent(const uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(uint32_t *p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// agent-coherent (sc1) 64-bit store and load of tagged hand-off words
__device__ __forceinline__ void st_agent64(uint64_t *p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_agent64(const uint64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ const uint8_t *expert_gu(const DecodeArgs &a, int e) {
  return e < a.E ? a.w_gu + (int64_t)e * (2 * a.I) * (a.H / 256) * (8 * Q4B) : a.ws_gu;
}
__device__ __forceinline__ const uint8_t *expert_d(const DecodeArgs &a, int e) {
  return e < a.E ? a.w_d + (int64_t)e * a.H * (a.I / 256) * (8 * Q4B) : a.ws_d;
}

// Element 4t..4t+3 of the layer's input: x, or x + resid in norm mode.
__device__ __forceinline__ float4 input4(const DecodeArgs &a, int t) {
  float4 v = reinterpret_cast<const float4 *>(a.x)[t];
  if (a.resid) {
    const float4 d = reinterpret_cast<const float4 *>(a.resid)[t];
    v.x += d.x; v.y += d.y; v.z += d.z; v.w += d.w;
  }
  return v;
}

// The lane's first float4 of x, of resid and of gamma (norm mode), loaded
// ahead of the weight loads: the first chunk of the input then needs no load
// issued after them (loads retire in order, so waiting for one issued after
// the weights would wait for the weights too).
struct XFirst {
  float4 x, r, g;
};
__device__ __forceinline__ XFirst issue_x_first(const DecodeArgs &a) {
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
  XFirst f{z, z, z};
  if ((int)threadIdx.x < a.H / 4) {
    f.x = reinterpret_cast<const float4 *>(a.x)[threadIdx.x];
    if (a.resid) f.r = reinterpret_cast<const float4 *>(a.resid)[threadIdx.x];
    if (a.gamma) f.g = reinterpret_cast<const float4 *>(a.gamma)[threadIdx.x];
  }
  return f;
}
__device__ __forceinline__ float4 x_first(const DecodeArgs &a, const XFirst &f) {
  float4 v = f.x;
  if (a.resid) {
    v.x += f.r.x; v.y += f.r.y; v.z += f.r.z; v.w += f.r.w;
  }
  return v;
}

// Q8_0 of the layer's input (x, or RMSNorm(x + resid) * gamma) into the LDS
// staging; with `first_wg` also the 34-byte blocks to xq and, in norm mode,
// x + resid to x_out and the normalized row to xn.  8 lanes per block, 4
// values per lane.  `xf` holds the lane's first float4 of the inputs, loaded
// by the caller ahead of the weight loads; for H <= 4 * NT nothing else is
// loaded.  Every thread must call it.
__device__ __forceinline__ void quantize_chunk(const DecodeArgs &a, ActBuf xb, bool first_wg,
                                               int t, float4 f, float4 g, float r) {
  const bool live = t < a.H / 4;  // H / 4 % 8 == 0: whole 8-lane groups agree
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  if (live) {
    if (a.gamma) {
      if (first_wg) reinterpret_cast<float4 *>(a.x_out)[t] = f;
      f = make_float4(f.x * r * g.x, f.y * r * g.y, f.z * r * g.z, f.w * r * g.w);
      if (first_wg) reinterpret_cast<float4 *>(a.xn)[t] = f;
    }
    v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
  }
  uint32_t d16;
  const uint32_t packed = q8_0_block8(v, d16);
  const uint32_t word = split_word(packed, t & 7);
  const int lsum = sum8(low_nibble_sum(packed));
  if (live) {
    const int blk = t >> 3, j = t & 7;
    *code_word(xb, blk, j) = word;
    if (j == 0) {
      xb.d[blk] = f16_bits_to_f32(d16);
      xb.corr[blk] = -8 * lsum;
    }
    if (first_wg) store_q8_0_block8(a.xq + blk * Q8B, j, packed, d16);
  }
}
__device__ void quantize_x_to_lds(const DecodeArgs &a, ActBuf xb, bool first_wg,
                                  const XFirst &xf) {
  __shared__ float wss[NT / 64];
  const int tasks = a.H / 4;
  const float4 first = x_first(a, xf);
  float r = 1.0f;
  if (a.gamma) {
    // sum of squares in a fixed order: per thread in index order, a
    // butterfly per wave, the waves in order
    float ss = 0.0f;
    if ((int)threadIdx.x < tasks) {
      ss = fmaf(first.x, first.x, ss);
      ss = fmaf(first.y, first.y, ss);
      ss = fmaf(first.z, first.z, ss);
      ss = fmaf(first.w, first.w, ss);
    }
    for (int t = threadIdx.x + NT; t < tasks; t += NT) {
      const float4 v = input4(a, t);
      ss = fmaf(v.x, v.x, ss);
      ss = fmaf(v.y, v.y, ss);
      ss = fmaf(v.z, v.z, ss);
      ss = fmaf(v.w, v.w, ss);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
    if ((threadIdx.x & 63) == 0) wss[threadIdx.x >> 6] = ss;
    __syncthreads();
    float tot = 0.0f;
#pragma unroll
    for (int w = 0; w < NT / 64; w++) tot += wss[w];
    r = 1.0f / sqrtf(tot / (float)a.H + a.eps);
  }
  // the first chunk from registers, outside the loop: at the loop's head the
  // compiler waits for every load in flight, the weights included
  quantize_chunk(a, xb, first_wg, threadIdx.x, first, xf.g, r);
  for (int t0 = NT; t0 < tasks; t0 += NT) {
    const int t = t0 + threadIdx.x;
    float4 f = make_float4(0.f, 0.f, 0.f, 0.f), g = f;
    if (t < tasks) {
      f = input4(a, t);
      if (a.gamma) g = reinterpret_cast<const float4 *>(a.gamma)[t];
    }
    quantize_chunk(a, xb, first_wg, t, f, g, r);
  }
}

// Lane roles in an A item: wave w owns h columns 4w..4w+3 of the block; in a
// wave, lanes 16c..16c+7 hold the gate row of column 4w+c and lanes
// 16c+8..16c+15 its up row; lane g of the 8 takes the eight-block groups
// g, g+8, ... of that row (H/256 groups per row).
struct ARole {
  int hcol;     // column of h within the block, 0..31
  bool up;      // this lane's row is the up row
  int gg;       // first group of the lane
};
__device__ __forceinline__ ARole a_role() {
  ARole r;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  r.hcol = wave * 4 + (lane >> 4);
  r.up = (lane >> 3) & 1;
  r.gg = lane & 7;
  return r;
}
__device__ __forceinline__ const uint8_t *a_row(const DecodeArgs &a, int e, int b, const ARole &r) {
  const int64_t row = r.up ? a.I + b * 32 + r.hcol : b * 32 + r.hcol;
  return expert_gu(a, e) + row * ((int64_t)(a.H / 256) * 8 * Q4B);
}

// Gate/up for h block b of pair q with expert e.  xb must hold Q8_0(x); with
// PRE the lane's first group is already loaded in `w0`.  Publishes the Q8_0
// block of the 32 h values to the hand-off words with `tag`, and, for
// inspection, h and the 34-byte block to the documented workspace regions;
// with `stage` also into that LDS staging (block q * I/32 + b).  Uses hv[32]
// in LDS; every thread of the workgroup must call it.
template <bool PRE>
__device__ void gateup_block(const DecodeArgs &a, int q, int e, int b, ActBuf xb, const W8 &w0,
                             float *hv, uint32_t tag, const ActBuf *stage) {
  const int G = a.H / 256;
  const ARole r = a_role();
  const uint8_t *W = a_row(a, e, b, r);
  float acc = 0.0f;
  int g = r.gg;
  if (PRE) {
    if (g < G) acc = dot8_lds(w0, group_codes(xb, g * 8), xb.d + g * 8, xb.corr + g * 8, acc);
    g += 8;
  }
  for (; g < G; g += 8) {
    W8 w;
    load_w8(W + (int64_t)g * (8 * Q4B), w);
    acc = dot8_lds(w, group_codes(xb, g * 8), xb.d + g * 8, xb.corr + g * 8, acc);
  }
  const float s = sum8(acc);               // row sum, in every lane of the 8
  const float other = dpp_f<DPP_ROR8>(s);  // the up row's sum, seen from a gate lane
  if (!r.up && r.gg == 0) {
    const float h = silu_f32(s) * other;
    hv[r.hcol] = h;
    a.h[(int64_t)q * a.I + b * 32 + r.hcol] = h;
  }
  __syncthreads();
  if (threadIdx.x < 8) {                   // Q8_0 of the 32-value block, 8 lanes
    const int j = threadIdx.x;
    const float v[4] = {hv[4 * j], hv[4 * j + 1], hv[4 * j + 2], hv[4 * j + 3]};
    uint32_t d16;
    const uint32_t packed = q8_0_block8(v, d16);
    const uint32_t word = split_word(packed, j);
    const int lsum = sum8(low_nibble_sum(packed));              // 0..480
    uint64_t *xf = a.xfer + (int64_t)(q * (a.I / 32) + b) * XSTRIDE;
    const uint64_t hi = (uint64_t)tag << 32;
    st_agent64(xf + 1 + j, hi | word);
    if (j == 0) st_agent64(xf, hi | d16 | ((uint32_t)lsum << 16));
    store_q8_0_block8(a.hq + ((int64_t)q * (a.I / 32) + b) * Q8B, j, packed, d16);
    if (stage != nullptr) {
      const int blk = q * (a.I / 32) + b;
      *code_word(*stage, blk, j) = word;
      if (j == 0) {
        stage->d[blk] = f16_bits_to_f32(d16);
        stage->corr[blk] = -8 * lsum;
      }
    }
  }
}

// Every workgroup arrives once; the last arrival of the launch advances the
// call counter to `tag` and clears the arrival counters.  Each workgroup has
// read the call counter before it arrives.
__device__ void arrive(const DecodeArgs &a, uint32_t tag) {
  if (threadIdx.x != 0) return;
  const int nblocks = (int)gridDim.x;
  const int s = blockIdx.x % NSUB;
  const uint32_t sub_total = (uint32_t)((nblocks - s + NSUB - 1) / NSUB);
  const uint32_t old = counter_add(sync_word(a.sync, SYNC_SUB + s), 1u);
  if (old + 1u != sub_total) return;
  const uint32_t nsubs = (uint32_t)(nblocks < NSUB ? nblocks : NSUB);
  const uint32_t top = counter_add(sync_word(a.sync, SYNC_TOP), 1u);
  if (top + 1u != nsubs) return;
  for (int i = 0; i < SYNC_SLOTS; i++) st_agent(sync_word(a.sync, i), 0u);
  st_agent(a.calls, tag);
}

// Stage word w of block blk of the hand-off.
__device__ __forceinline__ void stage_word(ActBuf hb, int blk, int w, uint32_t v) {
  if (w == 0) {
    hb.d[blk] = f16_bits_to_f32(v);
    hb.corr[blk] = -8 * (int)(v >> 16);
  } else {
    *code_word(hb, blk, w - 1) = v;
  }
}

// Collect hand-off words [0, cnt) of the valid pairs into the staging (word
// i is word i % XW of block i / XW); lane takes the words
// threadIdx.x + j * NT, j < NWMAX.  Every wave polls its own words, one
// round of loads in flight (two in flight were slower: the doubled poll
// traffic), with no barrier between rounds; a wave that passes the round bound
// sets notdone[0].  One barrier at the end; returns false (uniformly) when
// some wave passed the bound.  notdone[0] must be zero on entry.
constexpr int NWMAX = 8;
__device__ bool collect(const DecodeArgs &a, ActBuf hb, uint32_t tag, int cnt, uint64_t vmask,
                        int *notdone) {
  const int nb_h = a.I / 32;
  uint32_t pending = 0;
  int blk[NWMAX], w[NWMAX];
#pragma unroll
  for (int j = 0; j < NWMAX; j++) {
    const int i = (int)threadIdx.x + j * NT;
    blk[j] = i / XW;
    w[j] = i - blk[j] * XW;
    if (i < cnt && ((vmask >> (blk[j] / nb_h)) & 1)) pending |= 1u << j;
  }
  auto issue = [&](uint64_t (&v)[NWMAX]) {
#pragma unroll
    for (int j = 0; j < NWMAX; j++)
      v[j] = ((pending >> j) & 1) ? ld_agent64(a.xfer + (int64_t)blk[j] * XSTRIDE + w[j]) : 0;
  };
  auto take = [&](const uint64_t (&v)[NWMAX]) {
#pragma unroll
    for (int j = 0; j < NWMAX; j++) {
      if (((pending >> j) & 1) && (uint32_t)(v[j] >> 32) == tag) {
        stage_word(hb, blk[j], w[j], (uint32_t)v[j]);
        pending &= ~(1u << j);
      }
    }
    return __ballot(pending != 0) == 0;         // this wave has all its words
  };
  uint64_t va[NWMAX];
  for (int it = 0;; it++) {
    issue(va);
    if (take(va)) break;
    if (it + 1 > a.spin_rounds) { if ((threadIdx.x & 63) == 0) notdone[0] = 1; break; }
  }
  __syncthreads();
  return notdone[0] == 0;
}

// The router's inputs, loaded by wave 0 at the start of the launch (RV
// logits per lane, E <= 64 * RV, clamped addresses masked afterwards, and
// the gate logit) so that they are first in the wave's load queue.
template <int RV>
__device__ __forceinline__ void route_issue(const DecodeArgs &a, float (&x)[RV], float &g) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int r = 0; r < RV; r++) x[r] = a.logits[min(lane + 64 * r, a.E - 1)];
  // a vector load (an index the compiler cannot see through): a scalar load
  // would be waited for before the loads issued after it
  int zero = 0;
  asm volatile("" : "+v"(zero));
  g = a.gate ? a.gate[zero] : 0.0f;
}

// The token's top-k in wave 0 into the LDS arrays rid[k] and rw[k + 1] (the
// shared expert's weight last), which then stand in for the ids and
// weights; workgroup 0 also writes them out.  Every thread must call it.
template <int RV>
__device__ void route_finish(DecodeArgs &a, float (&x)[RV], float g, int32_t *rid, float *rw) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
#pragma unroll
    for (int r = 0; r < RV; r++)
      if (lane + 64 * r >= a.E) x[r] = -INFINITY;
    float selv;
    int seli;
    wave_topk<RV>(x, a.k, selv, seli);
    const float wt = topk_weight(selv, a.k);
    const float gw = a.gate ? shared_gate(g) : 1.0f;
    if (lane < a.k) {
      rid[lane] = seli;
      rw[lane] = wt;
    }
    if (lane == 0) rw[a.k] = gw;
    if (blockIdx.x == 0) {
      if (lane < a.k) {
        a.route_ids[lane] = seli;
        a.route_w[lane] = wt;
      }
      if (lane == 0 && a.gate) a.route_gate[0] = gw;
    }
  }
  __syncthreads();
  a.ids = rid;
  a.topk_w = rw;
  a.shared_w = rw + a.k;
}

// A down slab's eight weight blocks decoded while it waits for h: each
// block's payload dwords as stored (the unsigned nibbles q) and with every
// nibble xor 8 (the signed nibbles q - 8), and its fp32 scale.  After the
// wait only the 4-bit dot products and one scaling per block remain.
struct W8Dec {
  uint32_t n[8][4], x[8][4];
  float d[8];
};
__device__ __forceinline__ void decode_w8(const W8 &w, W8Dec &o) {
#pragma unroll
  for (int k = 0; k < 8; k++) {
#pragma unroll
    for (int c = 0; c < 4; c++) {
      o.n[k][c] = w8_nib(w, k, c);
      o.x[k][c] = o.n[k][c] ^ 0x88888888u;
      // materialized here, ahead of the wait, not next to their use after it
      asm volatile("" : "+v"(o.n[k][c]), "+v"(o.x[k][c]));
    }
    o.d[k] = w8_scale(w, k);
    asm volatile("" : "+v"(o.d[k]));
  }
}
// acc + sum over the eight blocks of d_w * d_h * s against activations
// staged in LDS (see dot8_lds), on decoded weights.
__device__ __forceinline__ float dot8_dec(const W8Dec &w, const uint4 *__restrict__ codes,
                                          const float *__restrict__ d,
                                          const int *__restrict__ corr, float acc) {
#pragma unroll
  for (int k = 0; k < 8; k++) {
    const uint4 hi = codes[2 * k], lo = codes[2 * k + 1];
    const uint32_t h4[4] = {hi.x, hi.y, hi.z, hi.w}, l4[4] = {lo.x, lo.y, lo.z, lo.w};
    int sa = 0;
    uint32_t sb = (uint32_t)corr[k];
#pragma unroll
    for (int c = 0; c < 4; c++) {
      sa = __builtin_amdgcn_sdot8((int)w.x[k][c], (int)h4[c], sa, false);
      sb = __builtin_amdgcn_udot8(w.n[k][c], l4[c], sb, false);
    }
    const int s = (int)(((uint32_t)sa << 4) + sb);
    acc = fmaf((float)s, w.d[k] * d[k], acc);
  }
  return acc;
}

// L2 prefetch by the down slabs.  A compute unit keeps only about 36 KB of
// loads in flight, so a gate/up item (72 KB of weights for H = 2048) streams
// in two rounds: waves 4..7 (h columns 16..31 of the block) can issue their
// loads only once those of waves 0..3 have returned.  The down slabs need
// their own weights only after every h block is in, so each first loads a
// share of those late rows of the gate/up items on its own XCD (workgroup w
// runs on XCD w % 8, and the compute units of one XCD share its L2): the
// items' second round then hits in L2.  The late rows of an item form two
// chunks of 16 consecutive rows (gate rows, then up rows); the C chunks on
// XCD x go to its S slabs in even runs of whole chunks, at most PF_CH chunks
// and PF_U 16-byte loads per lane and chunk.  Returns the values loaded (to
// be waited for and dropped by the caller) in pf; false (uniformly) when the
// slab has no chunk.
constexpr int PF_CH = 3, PF_U = 3;
__device__ __forceinline__ bool prefetch_gateup(const DecodeArgs &a, int wg, int nbh, int nb_h,
                                                uint64_t vmask, int ev,
                                                uint4 (&pf)[PF_CH][PF_U]) {
  const int x = wg & 7;
  const int nitems = nbh > x ? (nbh - x + 7) / 8 : 0;
  const int first = nbh + ((x - nbh % 8) + 8) % 8;           // first slab on XCD x
  const int nslabs = (int)gridDim.x > first ? ((int)gridDim.x - first + 7) / 8 : 0;
  if (nitems == 0 || nslabs == 0) return false;
  const int slab = (wg - first) / 8;
  const int c0 = 2 * nitems * slab / nslabs, c1 = 2 * nitems * (slab + 1) / nslabs;
  if (c1 <= c0) return false;
  const int64_t rowbytes = (int64_t)(a.H / 32) * Q4B;
  const int cu = (int)rowbytes;                               // 16-byte units per chunk
#pragma unroll
  for (int j = 0; j < PF_CH; j++) {
    // chunk c0 + j (the last chunk again past c1), wave-uniform
    const int c = min(c0 + j, c1 - 1);
    const int item = x + 8 * (c >> 1);
    const int q = item / nb_h, b = item - q * nb_h;
    const int e = __builtin_amdgcn_readlane(ev, q);
    const bool live = (vmask >> q) & 1;
    const uint8_t *base = live ? expert_gu(a, e) + (((c & 1) ? a.I : 0) + b * 32 + 16) * rowbytes
                               : reinterpret_cast<const uint8_t *>(a.x);
    const int span = live ? cu : 1;
#pragma unroll
    for (int i = 0; i < PF_U; i++) {
      const int u = min((int)threadIdx.x + i * NT, span - 1);
      pf[j][i] = reinterpret_cast<const uint4 *>(base)[u];
    }
  }
  return true;
}

// LDS: Q8_0(x) staging, then Q8_0(h) staging of every pair, then the
// weighted per-pair sums [rb][k+1 padded to 4] and, when I > 512, the down
// partials (NT floats).
__host__ __device__ constexpr size_t lds_x_bytes(int H) { return act_buf_bytes(H / 32); }
__host__ __device__ constexpr size_t lds_bytes(int H, int I, int k, int rb) {
  return lds_x_bytes(H) + act_buf_bytes((k + 1) * (I / 32)) +
         sizeof(float) * ((size_t)rb * ((k + 1 + 3) & ~3) + (size_t)NT);
}

// RV > 0: the router in front, RV logits per lane (see route_in_wg).
template <int RV>
__global__ __launch_bounds__(NT) void decode_kernel(DecodeArgs a) {
  extern __shared__ __align__(16) uint8_t lds[];
  __shared__ float hv[32];
  __shared__ float wq[64];
  __shared__ int notdone[3];
  __shared__ int32_t rid[64];
  __shared__ float rw[64];
  const int npairs = a.k + 1;
  const int nb_h = a.I / 32;                  // gate/up items per pair
  const int nbh = npairs * nb_h;              // h blocks of every pair
  const int wg = blockIdx.x;
  const ActBuf xb = act_buf(lds, a.H / 32);
  // the router's inputs first, then a gate/up item's x, all in flight
  // before anything waits
  constexpr int RVX = RV > 0 ? RV : 1;
  float lx[RVX];
  float lg = 0.0f;
  if (RV > 0 && threadIdx.x < 64) route_issue<RVX>(a, lx, lg);
  const float4 z4 = make_float4(0.f, 0.f, 0.f, 0.f);
  XFirst xf{z4, z4, z4};
  uint32_t calls = 0;
  if (wg < nbh) {
    xf = issue_x_first(a);
    calls = ld_agent(a.calls);   // in flight with x and the expert id
  }
  if (RV > 0) route_finish<RVX>(a, lx, lg, rid, rw);

  if (wg < nbh) {
    // --------------------------------------------------- gate/up item
    const int q = wg / nb_h, b = wg - q * nb_h;
    // x and the expert id land before the weights are issued: on every path
    // the later uses of x then wait for nothing in flight behind them
    // (the call tag too: a load issued after the weights would be waited for
    // together with them, since loads retire in order)
    int e;
    const bool valid = pair_valid(a, q, e);
    const uint32_t tag = calls + 1u;
    asm volatile("" ::"v"(xf.x.x), "v"(xf.x.y), "v"(xf.x.z), "v"(xf.x.w), "v"(xf.r.x),
                 "v"(xf.r.y), "v"(xf.r.z), "v"(xf.r.w), "v"(xf.g.x), "v"(xf.g.y), "v"(xf.g.z),
                 "v"(xf.g.w), "v"(e), "v"(tag));
    W8 w0;
    const ARole r = a_role();
    if (valid && r.gg < a.H / 256) load_w8(a_row(a, e, b, r) + (int64_t)r.gg * (8 * Q4B), w0);
    if (valid || wg == 0) {
      quantize_x_to_lds(a, xb, wg == 0, xf);
      __syncthreads();
    }
    if (valid) gateup_block<true>(a, q, e, b, xb, w0, hv, tag, nullptr);
    arrive(a, tag);
    return;
  }

  // ------------------------------------------------------ down slab
  const int rb = a.rb;
  const int GI = a.I / 256;
  const int units = npairs * rb * GI;
  // unit u = (q * rb + r) * GI + g: one 144-byte group per lane; a wave then
  // reads the Q8_0(h) groups of one or two pairs only, so its LDS reads of
  // them are mostly broadcasts
  const int uq = threadIdx.x / (rb * GI), ur = (threadIdx.x / GI) % rb, ug = threadIdx.x % GI;
  const int64_t row0 = (int64_t)(wg - nbh) * rb;
  const int64_t un = row0 + ur;
  // the units' experts, every pair's validity (lane q of each wave reads
  // slot q) and the routing weights land before the weight loads are issued
  int ue = 0;
  const bool ulive = (int)threadIdx.x < units && un < a.H && pair_valid(a, uq, ue);
  int ev = 0;
  const int lq = threadIdx.x & 63;
  const bool lane_valid = lq < npairs && pair_valid(a, lq, ev);
  const float wl = (int)threadIdx.x < a.k ? a.topk_w[threadIdx.x]
                                           : (a.shared_w ? a.shared_w[0] : 1.0f);
  asm volatile("" ::"v"(ue), "v"((int)ulive), "v"((int)lane_valid), "v"(wl));
  const uint64_t vmask = __ballot(lane_valid);    // wave-uniform
  if (a.prefetch) {
    uint4 pf[PF_CH][PF_U];
    if (prefetch_gateup(a, wg, nbh, nb_h, vmask, ev, pf)) {
      // the values are dropped (an empty asm that takes them keeps the
      // loads); waiting for them here also holds the slab's own weight
      // loads back until the gate/up rows are in
      uint32_t sink = 0;
#pragma unroll
      for (int j = 0; j < PF_CH; j++)
#pragma unroll
        for (int i = 0; i < PF_U; i++) sink ^= pf[j][i].x ^ pf[j][i].y ^ pf[j][i].z ^ pf[j][i].w;
      asm volatile("" ::"v"(sink));
    }
  }
  W8 wpre;
  if (ulive)
    load_w8(expert_d(a, ue) + un * ((int64_t)GI * 8 * Q4B) + (int64_t)ug * (8 * Q4B), wpre);
  if ((int)threadIdx.x < npairs) wq[threadIdx.x] = wl;
  const uint32_t tag = ld_agent(a.calls) + 1u;
  // a workgroup may arrive as soon as it has read the tag; here the atomic's
  // return (which waits for this wave's weight loads) also keeps the first
  // poll off the memory system while the gate/up weights stream
  arrive(a, tag);

  const ActBuf hb = act_buf(lds + lds_x_bytes(a.H), nbh);
  float *part = reinterpret_cast<float *>(lds + lds_x_bytes(a.H) + act_buf_bytes(nbh));
  if (threadIdx.x < 3) notdone[threadIdx.x] = 0;
  W8Dec wd;
  if (ulive) decode_w8(wpre, wd);
  __syncthreads();
  const bool ok = collect(a, hb, tag, XW * nbh, vmask, notdone);
  if (!ok) {
    // fallback: compute every pair's Q8_0(h) here (same code, same bytes)
    quantize_x_to_lds(a, xb, false, issue_x_first(a));
    __syncthreads();
    for (int q = 0; q < npairs; q++) {
      if (!((vmask >> q) & 1)) continue;
      int e;
      pair_valid(a, q, e);
      for (int b = 0; b < nb_h; b++) {
        gateup_block<false>(a, q, e, b, xb, W8{}, hv, tag, &hb);
        __syncthreads();
      }
    }
  }
  float acc = 0.0f;
  if (ulive) {
    const int blk0 = uq * nb_h + ug * 8;
    acc = dot8_dec(wd, group_codes(hb, blk0), hb.d + blk0, hb.corr + blk0, 0.0f);
  }
  // weighted y_q[n] = w_q * (sum over g in order), stored transposed
  // yw[r][q] with the pair count padded to a multiple of 4 (pads and skipped
  // slots are 0).  For GI <= 2 the g sum stays in registers: the two groups
  // of a row are adjacent lanes.
  const int npad = (npairs + 3) & ~3;
  float *yw = part;
  if (GI <= 2) {
    const float y = GI == 2 ? acc + dpp_f<DPP_XOR1>(acc) : acc;
    const bool valid_q = (int)threadIdx.x < units && ((vmask >> uq) & 1);
    if (ug == 0 && (int)threadIdx.x < units) yw[ur * npad + uq] = valid_q ? wq[uq] * y : 0.0f;
    if ((int)threadIdx.x < (npad - npairs) * rb)       // the pads
      yw[((int)threadIdx.x % rb) * npad + npairs + (int)threadIdx.x / rb] = 0.0f;
  } else {
    float *pt = part + rb * npad;
    if ((int)threadIdx.x < units) pt[threadIdx.x] = acc;
    __syncthreads();
    for (int t = threadIdx.x; t < npad * rb; t += NT) {
      const int q = t / rb, rr = t - q * rb;
      float v = 0.0f;
      if (q < npairs && ((vmask >> q) & 1)) {
        float y = 0.0f;
        for (int g = 0; g < GI; g++) y += pt[t * GI + g];
        v = wq[q] * y;
      }
      yw[rr * npad + q] = v;
    }
  }
  __syncthreads();
  // out[n] = sum over the slots in order, then the shared expert
  for (int rr = threadIdx.x; rr < rb; rr += NT) {
    const int64_t n = row0 + rr;
    if (n >= a.H) continue;
    const float4 *yrow = reinterpret_cast<const float4 *>(yw + rr * npad);
    float o = 0.0f;
    for (int q4 = 0; q4 < npad / 4; q4++) {
      const float4 v = yrow[q4];
      o += v.x;
      o += v.y;
      o += v.z;
      o += v.w;
    }
    a.out[n] = o;
  }
}

// Workgroups and down rows per slab: one gate/up item per h block, then the
// down slabs, enough of them to fill the remaining compute units but with
// few enough rows that a slab's units fit the workgroup.  The gate/up items
// never wait, so no slab waits for a workgroup that cannot start.
void decode_grid(int64_t H, int64_t I, int64_t k, int ncu, int &grid, int &rb) {
  const int64_t nbh = (k + 1) * (I / 32);
  const int64_t rb_max = NT / ((k + 1) * (I / 256));
  int64_t nb = (H + rb_max - 1) / rb_max;   // fewest slabs
  if (nb < ncu - nbh) nb = ncu - nbh;
  rb = (int)((H + nb - 1) / nb);
  nb = (H + rb - 1) / rb;
  grid = (int)(nbh + nb);
}

}  // namespace

size_t decode_sync_words(int64_t) { return (size_t)SYNC_SLOTS * SYNC_STRIDE; }

// Largest number of h blocks a single-token call hands off (decode_supported
// bounds (k + 1) * I/32 by it).
constexpr int XBLK_MAX = NWMAX * NT / XW;

// Hand-off region for T = 1, in uint32 words: the call counter's line, then
// one 128-byte line (XSTRIDE 64-bit words, XW used) per h block, sized for
// the largest supported (I, k).  Its size does not depend on the call's
// shape, so no region of any other call's layout ever overlaps it: every
// word in it was last written by a single-token call, with that call's tag,
// which is below the current tag (the counter only grows; it would take 2^32
// calls for a tag to come back).
size_t decode_xfer_words() { return (size_t)XFER_HDR + (size_t)XBLK_MAX * XSTRIDE * 2; }

// Bound on the poll rounds of the hand-off wait: W4A8_DECODE_SPIN_ROUNDS if
// set when the library first needs it, else 2000 (about 1-2 ms);
// w4a8_decode_wait_bound changes it.
std::atomic<int> g_spin_rounds{-1};

int spin_rounds() {
  int v = g_spin_rounds.load(std::memory_order_relaxed);
  if (v >= 0) return v;
  int d = 2000;
  if (const char *env = std::getenv("W4A8_DECODE_SPIN_ROUNDS")) d = std::max(0, std::atoi(env));
  int expected = -1;
  g_spin_rounds.compare_exchange_strong(expected, d, std::memory_order_relaxed);
  return g_spin_rounds.load(std::memory_order_relaxed);
}

// L2 prefetch by the down slabs: off when W4A8_DECODE_PREFETCH is 0.
int prefetch_on() {
  static const int on = [] {
    const char *env = std::getenv("W4A8_DECODE_PREFETCH");
    return env == nullptr || std::atoi(env) != 0 ? 1 : 0;
  }();
  return on;
}

// Router in front of the launch: the logits of E experts fit wave 0's
// registers.
bool decode_routes(int64_t E, int64_t k) { return E <= 512 && k <= 32 && k <= E; }

bool decode_supported(int64_t H, int64_t I, int64_t k) {
  // Gate/up items: 8 waves x 4 h columns = one 32-column block.  Down slabs
  // hold every pair of one down row at one unit per lane; a lane collects at
  // most NWMAX hand-off words per pass; LDS holds the staged Q8_0(x), the
  // staged Q8_0(h) of every pair and the partials.
  if (H < 256 || I < 256 || k < 1 || H > 16384 || k + 1 > 64 || (k + 1) * (I / 256) > NT)
    return false;
  const int64_t nbh = (k + 1) * (I / 32);
  const int rb = (int)(NT / ((k + 1) * (I / 256)));   // the largest slab
  return nbh <= XBLK_MAX && lds_bytes((int)H, (int)I, (int)k, rb) <= 48 * 1024;
}

int decode_forward(const float *x, const DecodeNorm &norm, const DecodeRoute *route,
                   const int32_t *ids,
                   const float *topk_w, const float *shared_w, const uint8_t *w_gu,
                   const uint8_t *w_d,
                   const uint8_t *ws_gu, const uint8_t *ws_d, float *out, int64_t H, int64_t I,
                   int64_t E, int64_t k, uint32_t *sync, uint32_t *xfer, uint8_t *xq, float *h,
                   uint8_t *hq, hipStream_t s) {
  const int ncu = device_cus();
  if (ncu <= 0) return W4A8_EHIP;
  DecodeArgs a;
  a.x = x; a.ids = ids; a.topk_w = topk_w; a.shared_w = shared_w;
  a.w_gu = w_gu; a.w_d = w_d; a.ws_gu = ws_gu; a.ws_d = ws_d;
  a.out = out;
  a.sync = sync;
  a.calls = xfer;
  a.xfer = reinterpret_cast<uint64_t *>(xfer + XFER_HDR);
  a.resid = norm.resid; a.gamma = norm.gamma; a.x_out = norm.x_out; a.xn = norm.xn;
  a.eps = norm.eps;
  a.xq = xq; a.h = h; a.hq = hq;
  a.logits = nullptr; a.gate = nullptr;
  a.route_ids = nullptr; a.route_w = nullptr; a.route_gate = nullptr;
  if (route != nullptr) {
    if (!decode_routes(E, k)) return W4A8_ERANGE;
    a.logits = route->logits; a.gate = route->gate;
    a.route_ids = route->ids; a.route_w = route->w; a.route_gate = route->gate_w;
  }
  a.H = (int)H; a.I = (int)I; a.E = (int)E; a.k = (int)k;
  int grid = 0;
  decode_grid(H, I, k, ncu, grid, a.rb);
  a.spin_rounds = spin_rounds();
  a.prefetch = prefetch_on();
  const size_t lds = lds_bytes((int)H, (int)I, (int)k, a.rb);
  if (route == nullptr)
    decode_kernel<0><<<dim3((unsigned)grid), dim3(NT), lds, s>>>(a);
  else if (E <= 256)
    decode_kernel<4><<<dim3((unsigned)grid), dim3(NT), lds, s>>>(a);
  else
    decode_kernel<8><<<dim3((unsigned)grid), dim3(NT), lds, s>>>(a);
  return check_launch();
}

}  // namespace w4a8

extern "C" int w4a8_decode_wait_bound(int64_t rounds) {
  const int prev = w4a8::spin_rounds();
  if (rounds >= 0) w4a8::g_spin_rounds.store((int)std::min<int64_t>(rounds, 1 << 30),
                                             std::memory_order_relaxed);
  return prev;
}
