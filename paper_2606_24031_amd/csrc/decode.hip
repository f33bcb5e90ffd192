// Single-token MoE layer in one kernel launch (decode, T = 1).
//
// At M = 1 the layer streams (k + 1) experts' weights (8 routed + 1 shared,
// 15.9 MB for the Qwen3-family shape) and does almost no arithmetic, so its
// cost is HBM latency plus the chain of hand-offs between the gate/up and the
// down projection; an extra kernel boundary alone costs about a third of the
// layer.  Everything therefore runs in one grid of two kinds of workgroups
// (the routed top-k experts and the always-on shared expert of Sec. 2.2; the
// W4A8 product of Sec. 3.3):
//
//   A items (pair q, 32-column block b of h): issue the 64 gate/up row loads
//     (one 144-byte eight-block group per lane for H = 2048),
//     quantize x to Q8_0 into LDS, take the W4A8 dots, h = SiLU(g) * u, and
//     publish Q8_0 of the 32 h values (exactly one block); count it in the
//     pair's counter.
//   B items (slab of RB down rows, all pairs): issue the down weight loads of
//     every pair first, wait until every pair's h blocks are published, read
//     them, take the dots and write out[n] = sum_q w_q y_q[n] (slots in
//     order, then the shared expert) -- the combine never leaves the
//     workgroup.
//
// The wait is bounded: after `spin_limit` ticks of the 100 MHz real-time
// counter a B item computes the missing Q8_0(h) blocks itself (the same code,
// so the same bytes), so progress never depends on the order in which the
// hardware starts workgroups.  Hand-off data crosses XCDs through agent-
// coherent (sc1) stores and loads: a writer waits until its stores are
// acknowledged (vmcnt 0) before the workgroup barrier and the counter add; a
// reader polls the counter and then reads with sc1 loads, so no whole-L2
// writeback or invalidate is needed.  Every workgroup finally arrives at a
// two-level counter (one word per XCD slot, then one top word); the last
// arrival of the launch clears every counter, so the sync words are zero
// again when the call completes.
#include <cstdlib>

#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int NT = 512;    // threads per workgroup
constexpr int NSUB = 8;    // first-level arrival counters

// Sync words (uint32, zero between calls), each alone in its own 256-byte
// line: same-line atomics and polls serialize in the memory system, which
// costs microseconds at this scale.  Slots: pair counters [64], arrival
// counters [NSUB], top arrival counter [1].
constexpr int SYNC_STRIDE = 64;   // words between sync slots (256 bytes)
constexpr int SYNC_PAIR = 0, SYNC_SUB = 64, SYNC_TOP = 64 + NSUB, SYNC_SLOTS = 64 + NSUB + 1;
__device__ __forceinline__ uint32_t *sync_word(uint32_t *sync, int slot) {
  return sync + slot * SYNC_STRIDE;
}

struct DecodeArgs {
  const float *x;          // [H]
  const int32_t *ids;      // [k]
  const float *topk_w;     // [k]
  const uint8_t *w_gu, *w_d, *ws_gu, *ws_d;
  float *out;              // [H]
  uint32_t *sync;
  uint32_t *xfer;          // Q8_0(h) hand-off: [(k+1)][I/32][9 words]: scale, 8 code words
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
__device__ __forceinline__ uint32_t counter_load(const uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// agent-coherent (sc1) store and load of hand-off words
__device__ __forceinline__ void st_agent(uint32_t *p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_agent(const uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// wait until this wave's stores are acknowledged (s_waitcnt vmcnt(0))
__device__ __forceinline__ void wait_stores() { __builtin_amdgcn_s_waitcnt(0x0F70); }

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

// Q8_0 of x (fp32 [H], global) into the LDS staging; with `xq_out` also the
// 34-byte blocks to global memory.  8 lanes per block, 4 values per lane.
// `first` is the lane's first float4 of x, loaded by the caller ahead of the
// weight loads (a wave's loads return in order, so x is then not stuck
// behind the weights).
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
    int sum = sdot4((int)packed, 0x01010101, 0);
#pragma unroll
    for (int o = 4; o > 0; o >>= 1) sum += __shfl_xor(sum, o, 8);
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

// Gate/up for h block b of pair q with expert e: 64 rows (32 gate + 32 up) of
// G = H/256 eight-block groups each, unit u = row * G + g over the NT lanes.
// Publishes Q8_0 of the 32 h values to the hand-off buffer (sc1) and, for
// inspection, h and the 34-byte block to the documented workspace regions.
// xb must hold Q8_0(x); `w0` is the lane's first unit, already loaded.
// Uses part[64 * G] and hv[32] in LDS.
__device__ void gateup_block(const DecodeArgs &a, int q, int e, int b, ActBuf xb, const W8 &w0,
                             float *part, float *hv) {
  const int G = a.H / 256;
  const int units = 64 * G;
  const uint8_t *W = expert_gu(a, e);
  const int64_t rowbytes = (int64_t)G * 8 * Q4B;
  for (int u = threadIdx.x, j = 0; u < units; u += NT, j++) {
    const int row = u / G, g = u % G;
    const uint4 *codes = xb.codes + g * 16;
    const float *dd = xb.d + g * 8;
    const int *cc = xb.corr + g * 8;
    float acc;
    if (j == 0) {
      acc = dot8_lds(w0, codes, dd, cc, 0.0f);
    } else {
      const int64_t r = row < 32 ? b * 32 + row : a.I + b * 32 + (row - 32);
      W8 w;
      load_w8(W + r * rowbytes + (int64_t)g * (8 * Q4B), w);
      acc = dot8_lds(w, codes, dd, cc, 0.0f);
    }
    part[u] = acc;
  }
  __syncthreads();
  if (threadIdx.x < 64) {               // row sums in fixed group order
    float s = 0.0f;
    for (int g = 0; g < G; g++) s += part[threadIdx.x * G + g];
    part[threadIdx.x * G] = s;
  }
  __syncthreads();
  if (threadIdx.x < 32) {
    const float gsum = part[threadIdx.x * G], usum = part[(32 + threadIdx.x) * G];
    const float h = silu_f32(gsum) * usum;
    hv[threadIdx.x] = h;
    a.h[(int64_t)q * a.I + b * 32 + threadIdx.x] = h;
  }
  __syncthreads();
  if (threadIdx.x < 8) {                // Q8_0 of the 32-value block, 8 lanes
    const int j = threadIdx.x;
    const float v[4] = {hv[4 * j], hv[4 * j + 1], hv[4 * j + 2], hv[4 * j + 3]};
    uint32_t d16;
    const uint32_t packed = q8_0_block8(v, d16);
    uint32_t *xf = a.xfer + ((int64_t)q * (a.I / 32) + b) * 9;
    st_agent(xf + 1 + j, packed);
    if (j == 0) st_agent(xf, d16);
    store_q8_0_block8(a.hq + ((int64_t)q * (a.I / 32) + b) * Q8B, j, packed, d16);
  }
}

__device__ __forceinline__ void load_gateup_unit(const DecodeArgs &a, int e, int b, W8 &w0) {
  const int G = a.H / 256;
  const int u = threadIdx.x;
  if (u < 64 * G) {
    const int64_t rowbytes = (int64_t)G * 8 * Q4B;
    const int row = u / G, g = u % G;
    const int64_t r = row < 32 ? b * 32 + row : a.I + b * 32 + (row - 32);
    load_w8(expert_gu(a, e) + r * rowbytes + (int64_t)g * (8 * Q4B), w0);
  }
}

__device__ __forceinline__ float4 load_x_first(const DecodeArgs &a) {
  return threadIdx.x < a.H / 4 ? reinterpret_cast<const float4 *>(a.x)[threadIdx.x]
                               : make_float4(0.f, 0.f, 0.f, 0.f);
}

// Last arrival of the launch clears every sync word.
__device__ void arrive(const DecodeArgs &a) {
  if (threadIdx.x != 0) return;
  const int nblocks = (int)gridDim.x;
  const int s = blockIdx.x % NSUB;
  const uint32_t sub_total = (uint32_t)((nblocks - s + NSUB - 1) / NSUB);
  const uint32_t old = counter_add(sync_word(a.sync, SYNC_SUB + s), 1u);
  if (old + 1u != sub_total) return;
  const uint32_t nsubs = (uint32_t)(nblocks < NSUB ? nblocks : NSUB);
  const uint32_t top = counter_add(sync_word(a.sync, SYNC_TOP), 1u);
  if (top + 1u != nsubs) return;
  for (int i = 0; i < SYNC_SLOTS; i++)
    __hip_atomic_store(sync_word(a.sync, i), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(NT) void decode_kernel(DecodeArgs a) {
  extern __shared__ __align__(16) uint8_t lds[];
  __shared__ float hv[32];
  __shared__ int flag;
  const int npairs = a.k + 1;
  const int nb_h = a.I / 32;                  // A items per pair
  const int na_total = npairs * nb_h;
  const int item = blockIdx.x;
  const int nbx = a.H / 32;                   // blocks of Q8_0(x)

  if (item < na_total) {
    // ------------------------------------------------------------ A item
    const int q = item / nb_h, b = item % nb_h;
    // x and the expert id together, both landed before the weights are
    // issued (a wave's loads return in order)
    const float4 x0 = load_x_first(a);
    int e;
    const bool valid = pair_valid(a, q, e);
    asm volatile("" ::"v"(x0.x), "v"(x0.y), "v"(x0.z), "v"(x0.w), "s"(e));
    W8 w0;
    if (valid) load_gateup_unit(a, e, b, w0);
    const ActBuf xb = act_buf(lds, nbx);
    float *part = reinterpret_cast<float *>(lds + act_buf_bytes(nbx));
    if (valid || item == 0) {
      quantize_x_to_lds(a, xb, item == 0 ? a.xq : nullptr, x0);
      __syncthreads();
    }
    if (valid) {
      gateup_block(a, q, e, b, xb, w0, part, hv);
      wait_stores();
      __syncthreads();
      if (threadIdx.x == 0) counter_add(sync_word(a.sync, SYNC_PAIR + q), 1u);
    }
    arrive(a);
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
  int ue = 0, ev = 0;
  const bool ulive = threadIdx.x < units && pair_valid(a, uq, ue) && un < a.H;
  // lane q polls pair q below; its validity is read now, before the weight
  // loads, so the poll does not wait behind them
  const bool mine = threadIdx.x < npairs && pair_valid(a, threadIdx.x, ev);
  asm volatile("" ::"v"(ue), "v"((int)mine));
  W8 wpre;
  if (ulive) load_w8(expert_d(a, ue) + un * rowbytes + (int64_t)ug * (8 * Q4B), wpre);

  // wait until every valid pair has all nb_h blocks of Q8_0(h) (bounded):
  // lane q polls pair q, all pairs at once (a coherent poll costs ~0.3 us
  // under load, so polling them one after another would add up)
  {
    const uint64_t t0 = wall_clock64();
    for (;;) {
      const int ready = !mine || counter_load(sync_word(a.sync, SYNC_PAIR + threadIdx.x)) >=
                                     (uint32_t)nb_h;
      if (__syncthreads_and(ready)) { if (threadIdx.x == 0) flag = 1; break; }
      if (threadIdx.x == 0) flag = (int64_t)(wall_clock64() - t0) > a.spin_limit ? 0 : 2;
      __syncthreads();
      if (flag == 0) break;
      __builtin_amdgcn_s_sleep(2);
      __syncthreads();   // everyone has read flag before thread 0 rewrites it
    }
  }
  __syncthreads();
  if (!flag) {
    // fallback: produce every pair's Q8_0(h) here (same code, same bytes)
    const ActBuf xb = act_buf(lds, nbx);
    float *gpart = reinterpret_cast<float *>(lds + act_buf_bytes(nbx));
    quantize_x_to_lds(a, xb, nullptr, load_x_first(a));
    __syncthreads();
    for (int q = 0; q < npairs; q++) {
      int e;
      if (!pair_valid(a, q, e)) continue;
      for (int b = 0; b < nb_h; b++) {
        W8 w0;
        load_gateup_unit(a, e, b, w0);
        gateup_block(a, q, e, b, xb, w0, gpart, hv);
        __syncthreads();
      }
    }
    wait_stores();
    __syncthreads();
  }
  // Q8_0(h) of every valid pair: hand-off words -> LDS staging
  const int nbh_all = npairs * nb_h;
  const ActBuf hb = act_buf(lds, nbh_all);
  float *part = reinterpret_cast<float *>(lds + act_buf_bytes(nbh_all));
  for (int i = threadIdx.x; i < nbh_all * 9; i += NT) {
    const int blk = i / 9, w = i % 9;
    int e;
    if (!pair_valid(a, blk / nb_h, e)) continue;
    const uint32_t v = ld_agent(a.xfer + i);
    if (w == 0)
      hb.d[blk] = f16_bits_to_f32(v);
    else
      reinterpret_cast<uint32_t *>(hb.codes)[blk * 8 + (w - 1)] = v;
  }
  __syncthreads();
  for (int blk = threadIdx.x; blk < nbh_all; blk += NT) {
    int e;
    if (!pair_valid(a, blk / nb_h, e)) continue;
    const uint32_t *c = reinterpret_cast<const uint32_t *>(hb.codes) + blk * 8;
    int s = 0;
#pragma unroll
    for (int i = 0; i < 8; i++) s = sdot4((int)c[i], 0x01010101, s);
    hb.corr[blk] = -8 * s;
  }
  __syncthreads();
  if (threadIdx.x < units) {
    float acc = 0.0f;
    if (ulive) {
      const int blk0 = uq * nb_h + ug * 8;
      if (flag) {
        acc = dot8_lds(wpre, hb.codes + blk0 * 2, hb.d + blk0, hb.corr + blk0, 0.0f);
      } else {
        W8 w;
        load_w8(expert_d(a, ue) + un * rowbytes + (int64_t)ug * (8 * Q4B), w);
        acc = dot8_lds(w, hb.codes + blk0 * 2, hb.d + blk0, hb.corr + blk0, 0.0f);
      }
    }
    part[threadIdx.x] = acc;
  }
  __syncthreads();
  for (int r = threadIdx.x; r < rb; r += NT) {
    const int64_t n = (int64_t)slab * rb + r;
    if (n >= a.H) continue;
    float o = 0.0f;
    for (int q = 0; q < npairs; q++) {
      int e;
      if (!pair_valid(a, q, e)) continue;
      float y = 0.0f;
      for (int g = 0; g < GI; g++) y += part[(q * rb + r) * GI + g];
      o += (q < a.k ? a.topk_w[q] : 1.0f) * y;
    }
    a.out[n] = o;
  }
  arrive(a);
}

}  // namespace

size_t decode_sync_words(int64_t) { return (size_t)SYNC_SLOTS * SYNC_STRIDE; }

// Hand-off buffer words for T = 1.
size_t decode_xfer_words(int64_t I, int64_t k) { return (size_t)(k + 1) * (I / 32) * 9; }

bool decode_supported(int64_t H, int64_t I, int64_t k) {
  // B items hold every pair of one down row at one unit per lane; LDS holds
  // the staged Q8_0(x) plus 64 * H/256 partials (A) or the staged Q8_0(h) of
  // every pair plus NT partials (B).
  const size_t lda = act_buf_bytes((int)(H / 32)) + sizeof(float) * 64 * (H / 256);
  const size_t ldb = act_buf_bytes((int)((k + 1) * (I / 32))) + sizeof(float) * NT;
  return H <= 16384 && (k + 1) <= 64 && (k + 1) * (I / 256) <= NT && lda <= 48 * 1024 &&
         ldb <= 48 * 1024;
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
  a.xfer = xfer;
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
  const size_t lda = act_buf_bytes((int)(H / 32)) + sizeof(float) * 64 * (H / 256);
  const size_t ldb = act_buf_bytes(npairs * (int)(I / 32)) + sizeof(float) * NT;
  const size_t lds = lda > ldb ? lda : ldb;
  decode_kernel<<<dim3(grid), dim3(NT), lds, s>>>(a);
  return check_launch();
}

}  // namespace w4a8
