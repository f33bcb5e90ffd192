// Single-token MoE layer in one kernel launch (decode, T = 1).
//
// At M = 1 the layer streams (k + 1) experts' weights (8 routed + 1 shared,
// 15.9 MB for the Qwen3-family shape) and does almost no arithmetic, so its
// cost is HBM latency plus the chain of hand-offs between the gate/up and the
// down projection; an extra kernel boundary alone costs about 1.6 us.
// Everything therefore runs in one grid of two kinds of workgroups (the routed
// top-k experts and the always-on shared expert of Sec. 2.2; the W4A8 product
// of Sec. 3.3):
//
//   A items (pair q, 32-column block b of h): issue the 64 gate/up row loads
//     (one 144-byte eight-block group per lane for H = 2048), quantize x to
//     Q8_0 into LDS, take the W4A8 dots, reduce each row over its 8 lanes
//     with DPP (gate row and up row of one h column sit in the same wave),
//     h = SiLU(g) * u, and publish Q8_0 of the 32 h values (one block).
//   B items (slab of RB down rows, all pairs): issue the down weight loads of
//     every pair first, collect every pair's Q8_0(h) blocks, take the dots and
//     write out[n] = sum_q w_q y_q[n] (slots in order, then the shared
//     expert) -- the combine never leaves the workgroup.
//
// Hand-off: each published word is 64 bits, the payload in the low half and
// the call's tag in the high half, written with agent-scope (sc1) stores.  A
// B item polls the words themselves until every one carries this call's tag,
// so there is no counter, no store acknowledgement wait and no second read.
// The tag is one more than the call counter kept in the hand-off region; the
// last workgroup of the launch to arrive at a two-level counter advances the
// call counter and clears the arrival counters, after every workgroup has
// read it.
//
// The wait is bounded: after `spin_limit` ticks of the 100 MHz real-time
// counter a B item computes every block itself (the same code, so the same
// bytes, also published with the same tag) straight into its own staging, so
// progress never depends on the order in which the hardware starts
// workgroups.
#include <cstdlib>

#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int NT = 512;          // threads per workgroup: 8 waves
constexpr int NSUB = 8;          // first-level arrival counters
constexpr int XW = 9;            // hand-off words per h block: scale and code sum, 8 code words
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
  const uint8_t *w_gu, *w_d, *ws_gu, *ws_d;
  float *out;              // [H]
  uint32_t *sync;          // arrival counters
  uint32_t *calls;         // call counter (tag of this call = *calls + 1)
  uint64_t *xfer;          // Q8_0(h) hand-off: [(k+1)][I/32][XW] tagged words
  uint8_t *xq;             // documented copy of Q8_0(x)   [H/32 blocks]
  float *h;                // documented copy of h          [(k+1)][I]
  uint8_t *hq;             // documented copy of Q8_0(h)    [(k+1)][I/32 blocks]
  int H, I, E, k;
  int rb;                  // down rows per B item
  int n_b;                 // B items
  int64_t spin_limit;      // real-time ticks before a B item computes h itself
};

__device__ __forceinline__ bool pair_valid(const DecodeArgs &a, int q, int &expert) {
  if (q < a.k) {
    expert = a.ids[q];
    return expert >= 0 && expert < a.E;
  }
  expert = a.E;
  return a.ws_gu != nullptr;
}

__device__ __forceinline__ float silu_f32(float g) { return g / (1.0f + expf(-g)); }

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

// LDS staging of activation blocks (see dot8_lds): codes [n][8] dwords,
// scale [n] fp32, correction [n] int32, carved from one dynamic LDS buffer.
struct ActBuf {
  uint4 *codes;
  float *d;
  int *corr;
};

__device__ __forceinline__ ActBuf act_buf(uint8_t *base, int nblocks) {
  ActBuf b;
  b.codes = reinterpret_cast<uint4 *>(base);
  b.d = reinterpret_cast<float *>(base + (size_t)nblocks * 32);
  b.corr = reinterpret_cast<int *>(base + (size_t)nblocks * 36);
  return b;
}
__host__ __device__ constexpr size_t act_buf_bytes(int nblocks) {
  return ((size_t)nblocks * 40 + 15) / 16 * 16;
}

// B item LDS after the staged Q8_0(h): NT dot partials, then the weighted
// per-pair sums [rb][npairs padded to 4].
__host__ __device__ constexpr size_t b_part_bytes(int npairs, int rb) {
  return sizeof(float) * ((size_t)NT + (size_t)((npairs + 3) & ~3) * rb);
}

// Q8_0 of x (fp32 [H], global) into the LDS staging; with `xq_out` also the
// 34-byte blocks to global memory.  8 lanes per block, 4 values per lane.
// `first` is the lane's first float4 of x, loaded by the caller ahead of the
// weight loads.
__device__ void quantize_x_to_lds(const DecodeArgs &a, ActBuf xb, uint8_t *xq_out,
                                  float4 first) {
  const int tasks = a.H / 4;
  for (int t0 = 0; t0 < tasks; t0 += NT) {
    const int t = t0 + threadIdx.x;
    const bool live = t < tasks;  // tasks % 8 == 0: whole 8-lane groups agree
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (live) {
      const float4 f = t0 == 0 ? first : reinterpret_cast<const float4 *>(a.x)[t];
      v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
    }
    uint32_t d16;
    const uint32_t packed = q8_0_block8(v, d16);
    const int sum = sum8(sdot4((int)packed, 0x01010101, 0));
    if (live) {
      const int blk = t >> 3, j = t & 7;
      reinterpret_cast<uint32_t *>(xb.codes)[blk * 8 + j] = packed;
      if (j == 0) {
        xb.d[blk] = f16_bits_to_f32(d16);
        xb.corr[blk] = -8 * sum;
      }
      if (xq_out) store_q8_0_block8(xq_out + blk * Q8B, j, packed, d16);
    }
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
    if (g < G) acc = dot8_lds(w0, xb.codes + g * 16, xb.d + g * 8, xb.corr + g * 8, acc);
    g += 8;
  }
  for (; g < G; g += 8) {
    W8 w;
    load_w8(W + (int64_t)g * (8 * Q4B), w);
    acc = dot8_lds(w, xb.codes + g * 16, xb.d + g * 8, xb.corr + g * 8, acc);
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
    const int csum = sum8(sdot4((int)packed, 0x01010101, 0));   // |csum| <= 4064
    uint64_t *xf = a.xfer + ((int64_t)q * (a.I / 32) + b) * XW;
    const uint64_t hi = (uint64_t)tag << 32;
    st_agent64(xf + 1 + j, hi | packed);
    if (j == 0) st_agent64(xf, hi | d16 | ((uint32_t)csum << 16));
    store_q8_0_block8(a.hq + ((int64_t)q * (a.I / 32) + b) * Q8B, j, packed, d16);
    if (stage != nullptr) {
      const int blk = q * (a.I / 32) + b;
      reinterpret_cast<uint32_t *>(stage->codes)[blk * 8 + j] = packed;
      if (j == 0) {
        stage->d[blk] = f16_bits_to_f32(d16);
        stage->corr[blk] = -8 * csum;
      }
    }
  }
}

__device__ __forceinline__ float4 load_x_first(const DecodeArgs &a) {
  return threadIdx.x < a.H / 4 ? reinterpret_cast<const float4 *>(a.x)[threadIdx.x]
                               : make_float4(0.f, 0.f, 0.f, 0.f);
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

// One staged hand-off word i of the B item's LDS staging.
__device__ __forceinline__ void stage_word(ActBuf hb, int i, uint32_t v) {
  const int blk = i / XW, w = i - blk * XW;
  if (w == 0) {
    hb.d[blk] = f16_bits_to_f32(v);
    hb.corr[blk] = -8 * (int)(int16_t)(v >> 16);
  } else {
    reinterpret_cast<uint32_t *>(hb.codes)[blk * 8 + (w - 1)] = v;
  }
}

// Collect every valid pair's tagged Q8_0(h) words into the LDS staging.
// Returns false (uniformly) when the wait bound passed first.  Bit j of
// `pending` marks the lane's word i = threadIdx.x + j * NT as still to be
// collected (j < NWMAX).  Two rounds of loads are in flight: the next round
// is issued before the current one is examined, which halves the time
// between a word becoming visible and a load that returns it.
constexpr int NWMAX = 8;
__device__ bool collect_h(const DecodeArgs &a, ActBuf hb, uint32_t tag, uint32_t pending,
                          int *tflag) {
  const uint64_t t0 = wall_clock64();
  const uint64_t *src = a.xfer + threadIdx.x;
  uint64_t cur[NWMAX], nxt[NWMAX];
#pragma unroll
  for (int j = 0; j < NWMAX; j++) cur[j] = ((pending >> j) & 1) ? ld_agent64(src + j * NT) : 0;
  for (int it = 0;; it++) {
#pragma unroll
    for (int j = 0; j < NWMAX; j++) nxt[j] = ((pending >> j) & 1) ? ld_agent64(src + j * NT) : 0;
#pragma unroll
    for (int j = 0; j < NWMAX; j++) {
      if (((pending >> j) & 1) && (uint32_t)(cur[j] >> 32) == tag) {
        stage_word(hb, threadIdx.x + j * NT, (uint32_t)cur[j]);
        pending &= ~(1u << j);
      }
    }
    if (threadIdx.x == 0) tflag[it & 1] = (int64_t)(wall_clock64() - t0) > a.spin_limit;
    if (__syncthreads_and(pending == 0)) return true;
    // thread 0 wrote tflag[it & 1] before the barrier and next writes that
    // slot two barriers later, after every wave has read it
    if (tflag[it & 1]) return false;
#pragma unroll
    for (int j = 0; j < NWMAX; j++) cur[j] = nxt[j];
  }
}

__global__ __launch_bounds__(NT) void decode_kernel(DecodeArgs a) {
  extern __shared__ __align__(16) uint8_t lds[];
  __shared__ float hv[32];
  __shared__ float wq[64];
  __shared__ int tflag[2];
  const int npairs = a.k + 1;
  const int nb_h = a.I / 32;                  // A items per pair
  const int na_total = npairs * nb_h;
  const int item = blockIdx.x;
  const int nbx = a.H / 32;                   // blocks of Q8_0(x)

  if (item < na_total) {
    // ------------------------------------------------------------ A item
    const int q = item / nb_h, b = item % nb_h;
    // x and the expert id land before the weights are issued: on every path
    // the later uses of x then wait for nothing in flight behind them
    const float4 x0 = load_x_first(a);
    int e;
    const bool valid = pair_valid(a, q, e);
    asm volatile("" ::"v"(x0.x), "v"(x0.y), "v"(x0.z), "v"(x0.w), "v"(e));
    W8 w0;
    const ARole r = a_role();
    if (valid && r.gg < a.H / 256) load_w8(a_row(a, e, b, r) + (int64_t)r.gg * (8 * Q4B), w0);
    const uint32_t tag = ld_agent(a.calls) + 1u;
    const ActBuf xb = act_buf(lds, nbx);
    if (valid || item == 0) {
      quantize_x_to_lds(a, xb, item == 0 ? a.xq : nullptr, x0);
      __syncthreads();
    }
    if (valid) gateup_block<true>(a, q, e, b, xb, w0, hv, tag, nullptr);
    arrive(a, tag);
    return;
  }

  // -------------------------------------------------------------- B item
  const int slab = item - na_total;
  const int rb = a.rb;
  const int GI = a.I / 256;
  const int64_t rowbytes = (int64_t)GI * 8 * Q4B;
  const int units = npairs * rb * GI;
  // unit u = (q * rb + r) * GI + g; one unit per lane (units <= NT)
  const int uq = threadIdx.x / (rb * GI), ur = (threadIdx.x / GI) % rb, ug = threadIdx.x % GI;
  const int64_t un = (int64_t)slab * rb + ur;
  int ue = 0;
  const bool ulive = threadIdx.x < units && pair_valid(a, uq, ue) && un < a.H;
  // validity of every pair (lane q of each wave reads slot q) and the routing
  // weights, all landed before the weight loads are issued
  int ev;
  const int lq = threadIdx.x & 63;
  const bool lane_valid = lq < npairs && pair_valid(a, lq, ev);
  const float wl = (int)threadIdx.x < a.k ? a.topk_w[threadIdx.x] : 1.0f;
  asm volatile("" ::"v"(ue), "v"((int)ulive), "v"((int)lane_valid), "v"(wl));
  W8 wpre;
  if (ulive) load_w8(expert_d(a, ue) + un * rowbytes + (int64_t)ug * (8 * Q4B), wpre);
  const uint64_t vmask = __ballot(lane_valid);    // wave-uniform
  if (threadIdx.x < npairs) wq[threadIdx.x] = wl;
  const uint32_t tag = ld_agent(a.calls) + 1u;

  const int nbh_all = npairs * nb_h;
  const int nwords = nbh_all * XW;
  const ActBuf hb = act_buf(lds, nbh_all);
  float *part = reinterpret_cast<float *>(lds + act_buf_bytes(nbh_all));
  uint32_t pending = 0;
#pragma unroll
  for (int j = 0; j < NWMAX; j++) {
    const int i = threadIdx.x + j * NT;
    if (i < nwords && ((vmask >> (i / (XW * nb_h))) & 1)) pending |= 1u << j;
  }
  if (!collect_h(a, hb, tag, pending, tflag)) {
    // fallback: compute every pair's Q8_0(h) here (same code, same bytes)
    const ActBuf xb = act_buf(lds + act_buf_bytes(nbh_all) + b_part_bytes(npairs, rb), nbx);
    quantize_x_to_lds(a, xb, nullptr, load_x_first(a));
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
  if (threadIdx.x < units) {
    float acc = 0.0f;
    if (ulive) {
      const int blk0 = uq * nb_h + ug * 8;
      acc = dot8_lds(wpre, hb.codes + blk0 * 2, hb.d + blk0, hb.corr + blk0, 0.0f);
    }
    part[threadIdx.x] = acc;
  }
  __syncthreads();
  // y_q[n] = sum over g (in order), weighted; stored transposed [r][q] with
  // the pair count padded to a multiple of 4 (pads and skipped slots are 0)
  const int npad = (npairs + 3) & ~3;
  float *yw = part + NT;
  for (int t = threadIdx.x; t < npad * rb; t += NT) {
    const int q = t / rb, r = t - q * rb;
    float v = 0.0f;
    if (q < npairs && ((vmask >> q) & 1)) {
      float y = 0.0f;
      for (int g = 0; g < GI; g++) y += part[t * GI + g];
      v = wq[q] * y;
    }
    yw[r * npad + q] = v;
  }
  __syncthreads();
  // out[n] = sum over the slots in order, then the shared expert
  for (int r = threadIdx.x; r < rb; r += NT) {
    const int64_t n = (int64_t)slab * rb + r;
    if (n >= a.H) continue;
    const float4 *row = reinterpret_cast<const float4 *>(yw + r * npad);
    float o = 0.0f;
    for (int q4 = 0; q4 < npad / 4; q4++) {
      const float4 v = row[q4];
      o += v.x;
      o += v.y;
      o += v.z;
      o += v.w;
    }
    a.out[n] = o;
  }
  arrive(a, tag);
}

}  // namespace

size_t decode_sync_words(int64_t) { return (size_t)SYNC_SLOTS * SYNC_STRIDE; }

// Hand-off region for T = 1, in uint32 words: the call counter's line, then
// XW 64-bit words per h block.
size_t decode_xfer_words(int64_t I, int64_t k) {
  return (size_t)XFER_HDR + (size_t)(k + 1) * (I / 32) * XW * 2;
}

bool decode_supported(int64_t H, int64_t I, int64_t k) {
  // A items: 8 waves x 4 h columns = one 32-column block.  B items hold
  // every pair of one down row at one unit per lane, and at most NWMAX
  // hand-off words per lane; LDS holds the staged Q8_0(x) (A) or the staged
  // Q8_0(h) of every pair, the partials and, for the fallback, Q8_0(x) (B).
  if (H < 256 || I < 256 || k < 1 || H > 16384 || k + 1 > 64 || (k + 1) * (I / 256) > NT)
    return false;
  const int64_t nbh_all = (k + 1) * (I / 32);
  const size_t lda = act_buf_bytes((int)(H / 32));
  const int rb = (int)(NT / ((k + 1) * (I / 256)));
  const size_t ldb = act_buf_bytes((int)nbh_all) + b_part_bytes((int)(k + 1), rb) + lda;
  return nbh_all * XW <= NWMAX * NT && lda <= 48 * 1024 && ldb <= 48 * 1024;
}

int decode_forward(const float *x, const int32_t *ids, const float *topk_w, const uint8_t *w_gu,
                   const uint8_t *w_d, const uint8_t *ws_gu, const uint8_t *ws_d, float *out,
                   int64_t H, int64_t I, int64_t E, int64_t k, uint32_t *sync, uint32_t *xfer,
                   uint8_t *xq, float *h, uint8_t *hq, hipStream_t s) {
  DecodeArgs a;
  a.x = x; a.ids = ids; a.topk_w = topk_w;
  a.w_gu = w_gu; a.w_d = w_d; a.ws_gu = ws_gu; a.ws_d = ws_d;
  a.out = out;
  a.sync = sync;
  a.calls = xfer;
  a.xfer = reinterpret_cast<uint64_t *>(xfer + XFER_HDR);
  a.xq = xq; a.h = h; a.hq = hq;
  a.H = (int)H; a.I = (int)I; a.E = (int)E; a.k = (int)k;
  const int npairs = (int)k + 1;
  const int GI = (int)(I / 256);
  a.rb = NT / (npairs * GI);                     // >= 1 by decode_supported
  a.n_b = (int)((H + a.rb - 1) / a.rb);
  // default wait bound: 1 ms of the 100 MHz real-time counter
  a.spin_limit = 100000;
  if (const char *env = std::getenv("W4A8_DECODE_SPIN_TICKS")) a.spin_limit = std::atoll(env);
  const unsigned grid = (unsigned)(npairs * (I / 32) + a.n_b);
  const size_t lda = act_buf_bytes((int)(H / 32));
  const size_t ldb = act_buf_bytes(npairs * (int)(I / 32)) + b_part_bytes(npairs, a.rb) + lda;
  const size_t lds = lda > ldb ? lda : ldb;
  decode_kernel<<<dim3(grid), dim3(NT), lds, s>>>(a);
  return check_launch();
}

}  // namespace w4a8
