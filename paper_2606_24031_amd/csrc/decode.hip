// Single-token MoE layer in one kernel launch (decode, T = 1).
//
// At M = 1 the layer streams (k + 1) experts' weights (8 routed + 1 shared,
// 15.9 MB for the Qwen3-family shape) and does almost no arithmetic, so the
// cost is the latency of a few passes over HBM; an extra kernel boundary
// costs about as much as a quarter of the whole layer.  Everything therefore
// runs in one grid of two kinds of workgroups (the routed top-k experts and
// the always-on shared expert of Sec. 2.2; the W4A8 product of Sec. 3.3):
//
//   A items (pair q, 128/LPR h columns): issue the gate and up weight loads,
//     quantize x to Q8_0 into LDS, take the W4A8 dots, h = SiLU(g) * u,
//     store h, then count the slab done in a per-pair counter.
//   B items (pair q, 256/LPR down rows): issue the down weight loads first,
//     then wait for the pair's counter, quantize h to Q8_0 into LDS, take the
//     dots, store w_q * y; the last of the pairs to finish a row slab adds
//     the slab up in slot order (then the shared pair) and writes out.
//
// The wait is bounded: after `spin_limit` ticks of the 100 MHz real-time
// counter a B item computes the pair's h itself (the same code, so the same
// bytes), so progress never depends on the order in which the hardware starts
// workgroups.  Hand-off data (h, the per-pair y) crosses XCDs through
// agent-coherent (sc1) stores and loads: a writer waits until its stores are
// acknowledged (vmcnt 0) before the workgroup barrier and the counter add, a
// reader polls the counter and then reads with sc1 loads, so no whole-L2
// writeback or invalidate is needed.  Counters return to zero when the call
// completes: every
// arrival adds to a per-pair word (A items +1, B items +0x10000) and the
// arrival that completes the total clears it; the per-slab combine counter is
// cleared by its last arrival.
#include <cstdlib>

#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int NT = 256;  // threads per workgroup

struct DecodeArgs {
  const float *x;          // [H]
  const int32_t *ids;      // [k]
  const float *topk_w;     // [k]
  const uint8_t *w_gu, *w_d, *ws_gu, *ws_d;
  float *out;              // [H]
  uint32_t *pair_cnt;      // [k + 1]
  uint32_t *slab_cnt;      // [H / RB]
  uint8_t *xq;             // workspace copy of Q8_0(x)  [H/32 blocks]
  float *h;                // [(k + 1)][I]
  uint8_t *hq;             // [(k + 1)][I/32 blocks]
  float *y;                // [(k + 1)][H]
  int H, I, E, k;
  int n_a;                 // A items per pair
  int n_b;                 // B items per pair
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
__device__ __forceinline__ void counter_clear(uint32_t *p) {
  __hip_atomic_store(p, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// agent-coherent (sc1) store and load of hand-off data
__device__ __forceinline__ void st_agent(float *p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_agent(const float *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// wait until this wave's stores are acknowledged (s_waitcnt vmcnt(0))
__device__ __forceinline__ void wait_stores() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Q8_0 of n contiguous fp32 values (n % 32 == 0) from global memory into LDS,
// 8 lanes per block.  COHERENT: read with agent-coherent loads (data another
// workgroup wrote during this launch).
template <bool COHERENT>
__device__ void quantize_to_lds(const float *__restrict__ src, uint8_t *lds, int n) {
  const int tasks = n / 4;  // 8 lanes x 4 values per block
  for (int t0 = 0; t0 < tasks; t0 += NT) {
    const int t = t0 + threadIdx.x;
    const bool live = t < tasks;   // tasks % 8 == 0: whole 8-lane groups agree
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (live) {
      if (COHERENT) {
#pragma unroll
        for (int i = 0; i < 4; i++) v[i] = ld_agent(src + 4 * t + i);
      } else {
        const float4 f = reinterpret_cast<const float4 *>(src)[t];
        v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
      }
    }
    uint32_t d16;
    const uint32_t packed = q8_0_block8(v, d16);
    if (live) store_q8_0_block8(lds + (t >> 3) * Q8B, t & 7, packed, d16);
  }
}

// Gate/up W4A8 dots for h columns [c0, c0 + HC) of one expert, HC = 128/LPR:
// lane (row rr = tid / LPR, K-groups li, li + LPR, ...), rows 0..HC-1 gate,
// HC..2HC-1 up.  `wpre` holds the lane's first weight group, already loaded.
// Returns through shrow[2*HC] (LDS).
template <int LPR>
__device__ void gateup_rows(const DecodeArgs &a, const uint8_t *W, int c0, const uint8_t *xq_lds,
                            const W8 &wpre, float *shrow) {
  constexpr int HC = 128 / LPR;
  const int rr = threadIdx.x / LPR, li = threadIdx.x % LPR;
  const int G = a.H / 256;
  const int64_t rowbytes = (int64_t)G * 8 * Q4B;
  const int64_t row = rr < HC ? c0 + rr : a.I + c0 + (rr - HC);
  float acc = 0.0f;
  if (li < G) {
    Act8 x;
    load_act8(xq_lds + li * (8 * Q8B), x);
    acc = dot8(wpre, x, acc);
  }
  for (int g = li + LPR; g < G; g += LPR) {
    W8 w;
    load_w8(W + row * rowbytes + (int64_t)g * (8 * Q4B), w);
    Act8 x;
    load_act8(xq_lds + g * (8 * Q8B), x);
    acc = dot8(w, x, acc);
  }
  acc = lane_group_sum<LPR>(acc);
  if (li == 0) shrow[rr] = acc;
}

template <int LPR>
__device__ __forceinline__ void load_gateup_pre(const DecodeArgs &a, const uint8_t *W, int c0,
                                                W8 &w) {
  constexpr int HC = 128 / LPR;
  const int rr = threadIdx.x / LPR, li = threadIdx.x % LPR;
  const int G = a.H / 256;
  const int64_t rowbytes = (int64_t)G * 8 * Q4B;
  const int64_t row = rr < HC ? c0 + rr : a.I + c0 + (rr - HC);
  if (li < G) load_w8(W + row * rowbytes + (int64_t)li * (8 * Q4B), w);
}

// h = SiLU(gate) * up for the HC columns in shrow, stored to the workspace.
template <int LPR>
__device__ __forceinline__ void store_h(const DecodeArgs &a, int q, int c0, const float *shrow) {
  constexpr int HC = 128 / LPR;
  if (threadIdx.x < HC) {
    const float hv = silu_f32(shrow[threadIdx.x]) * shrow[HC + threadIdx.x];
    st_agent(a.h + (int64_t)q * a.I + c0 + threadIdx.x, hv);
  }
}

template <int LPRA, int LPRB>
__global__ __launch_bounds__(NT) void decode_kernel(DecodeArgs a) {
  extern __shared__ __align__(16) uint8_t lds[];
  constexpr int HC = 128 / LPRA;   // h columns per A item
  constexpr int RB = 256 / LPRB;   // down rows per B item
  __shared__ float shrow[2 * HC];
  __shared__ int flag;
  const int npairs = a.k + 1;
  const int item = blockIdx.x;
  const int na_total = npairs * a.n_a;

  if (item < na_total) {
    // ------------------------------------------------------------ A item
    const int q = item / a.n_a, slab = item % a.n_a;
    int e;
    if (!pair_valid(a, q, e)) {
      if (item == 0) {                              // workspace copy of Q8_0(x)
        quantize_to_lds<false>(a.x, lds, a.H);
        __syncthreads();
        for (int i = threadIdx.x; i < (a.H / 32) * Q8B / 2; i += NT)
          reinterpret_cast<uint16_t *>(a.xq)[i] = reinterpret_cast<const uint16_t *>(lds)[i];
      }
      return;
    }
    const uint8_t *W = (e < a.E) ? a.w_gu + (int64_t)e * (2 * a.I) * (a.H / 256) * (8 * Q4B) : a.ws_gu;
    const int c0 = slab * HC;
    W8 wpre;
    load_gateup_pre<LPRA>(a, W, c0, wpre);          // weight loads in flight first
    uint8_t *xq_lds = lds;
    quantize_to_lds<false>(a.x, xq_lds, a.H);
    __syncthreads();
    if (item == 0)                                  // workspace copy of Q8_0(x)
      for (int i = threadIdx.x; i < (a.H / 32) * Q8B / 2; i += NT)
        reinterpret_cast<uint16_t *>(a.xq)[i] = reinterpret_cast<const uint16_t *>(xq_lds)[i];
    gateup_rows<LPRA>(a, W, c0, xq_lds, wpre, shrow);
    __syncthreads();
    store_h<LPRA>(a, q, c0, shrow);
    wait_stores();
    __syncthreads();
    if (threadIdx.x == 0) {
      const uint32_t total = (uint32_t)a.n_a + ((uint32_t)a.n_b << 16);
      const uint32_t old = counter_add(&a.pair_cnt[q], 1u);
      if (old + 1u == total) counter_clear(&a.pair_cnt[q]);
    }
    return;
  }

  // -------------------------------------------------------------- B item
  const int bi = item - na_total;
  const int q = bi / a.n_b, slab = bi % a.n_b;
  int nvalid = 0;
  for (int j = 0; j < npairs; j++) {
    int ej;
    nvalid += pair_valid(a, j, ej) ? 1 : 0;
  }
  int e;
  if (!pair_valid(a, q, e)) {
    if (nvalid == 0 && q == 0)                      // nothing routed: out = 0
      for (int n = threadIdx.x; n < RB; n += NT) a.out[slab * RB + n] = 0.0f;
    return;
  }
  const int GI = a.I / 256;
  const int64_t rowbytes = (int64_t)GI * 8 * Q4B;
  const uint8_t *Wd = (e < a.E) ? a.w_d + (int64_t)e * a.H * rowbytes : a.ws_d;
  const int r = threadIdx.x / LPRB, li = threadIdx.x % LPRB;
  const int64_t n = (int64_t)slab * RB + r;
  W8 wpre;
  if (li < GI) load_w8(Wd + n * rowbytes + (int64_t)li * (8 * Q4B), wpre);   // in flight first

  // wait for the pair's h (bounded)
  if (threadIdx.x == 0) {
    const uint64_t t0 = wall_clock64();
    int ok = 0;
    for (;;) {
      const uint32_t v = counter_load(&a.pair_cnt[q]);
      if ((v & 0xFFFFu) >= (uint32_t)a.n_a) { ok = 1; break; }
      if ((int64_t)(wall_clock64() - t0) > a.spin_limit) break;
      __builtin_amdgcn_s_sleep(2);
    }
    flag = ok;
  }
  __syncthreads();
  if (!flag) {
    // fallback: compute every h slab of this pair here (same code, same bytes)
    const uint8_t *W = (e < a.E) ? a.w_gu + (int64_t)e * (2 * a.I) * (a.H / 256) * (8 * Q4B) : a.ws_gu;
    uint8_t *xq_lds = lds;
    quantize_to_lds<false>(a.x, xq_lds, a.H);
    __syncthreads();
    for (int s = 0; s < a.n_a; s++) {
      W8 w;
      load_gateup_pre<LPRA>(a, W, s * HC, w);
      gateup_rows<LPRA>(a, W, s * HC, xq_lds, w, shrow);
      __syncthreads();
      store_h<LPRA>(a, q, s * HC, shrow);
      __syncthreads();
    }
    wait_stores();
    __syncthreads();
  }

  // Q8_0(h) of the pair into LDS; the first slab also stores it to the workspace
  uint8_t *hq_lds = lds;
  quantize_to_lds<true>(a.h + (int64_t)q * a.I, hq_lds, a.I);
  __syncthreads();
  if (slab == 0)
    for (int i = threadIdx.x; i < (a.I / 32) * Q8B / 2; i += NT)
      reinterpret_cast<uint16_t *>(a.hq + (int64_t)q * (a.I / 32) * Q8B)[i] =
          reinterpret_cast<const uint16_t *>(hq_lds)[i];

  float acc = 0.0f;
  if (li < GI) {
    Act8 x;
    load_act8(hq_lds + li * (8 * Q8B), x);
    acc = dot8(wpre, x, acc);
  }
  for (int g = li + LPRB; g < GI; g += LPRB) {
    W8 w;
    load_w8(Wd + n * rowbytes + (int64_t)g * (8 * Q4B), w);
    Act8 x;
    load_act8(hq_lds + g * (8 * Q8B), x);
    acc = dot8(w, x, acc);
  }
  acc = lane_group_sum<LPRB>(acc);
  const float wq = (q < a.k) ? a.topk_w[q] : 1.0f;
  if (li == 0) st_agent(a.y + (int64_t)q * a.H + n, wq * acc);
  wait_stores();
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t total = (uint32_t)a.n_a + ((uint32_t)a.n_b << 16);
    const uint32_t old = counter_add(&a.pair_cnt[q], 0x10000u);
    if (old + 0x10000u == total) counter_clear(&a.pair_cnt[q]);
    const uint32_t prev = counter_add(&a.slab_cnt[slab], 1u);
    flag = (prev + 1u == (uint32_t)nvalid) ? 1 : 0;
    if (flag) counter_clear(&a.slab_cnt[slab]);
  }
  __syncthreads();
  if (!flag) return;
  // last pair to finish this slab: out = sum over slots in order, then shared
  for (int i = threadIdx.x; i < RB; i += NT) {
    float s = 0.0f;
    for (int j = 0; j < npairs; j++) {
      int ej;
      if (pair_valid(a, j, ej)) s += ld_agent(a.y + (int64_t)j * a.H + (int64_t)slab * RB + i);
    }
    a.out[(int64_t)slab * RB + i] = s;
  }
}

int pow2_le(int g, int cap) {
  int l = 1;
  while (l * 2 <= g && l < cap) l *= 2;
  return l;
}

template <int A, int B>
void launch(const DecodeArgs &a, unsigned grid, size_t lds, hipStream_t s) {
  decode_kernel<A, B><<<dim3(grid), dim3(NT), lds, s>>>(a);
}

}  // namespace

// Workspace words used by the decode kernel (inside the zero-filled sync
// region): pair counters [k + 1], slab counters [H / 32 max].
size_t decode_sync_words(int64_t H) { return 64 + (size_t)(H / 32); }

int decode_forward(const float *x, const int32_t *ids, const float *topk_w, const uint8_t *w_gu,
                   const uint8_t *w_d, const uint8_t *ws_gu, const uint8_t *ws_d, float *out,
                   int64_t H, int64_t I, int64_t E, int64_t k, uint32_t *sync, uint8_t *xq,
                   float *h, uint8_t *hq, float *y, hipStream_t s) {
  DecodeArgs a;
  a.x = x; a.ids = ids; a.topk_w = topk_w;
  a.w_gu = w_gu; a.w_d = w_d; a.ws_gu = ws_gu; a.ws_d = ws_d;
  a.out = out;
  a.pair_cnt = sync;
  a.slab_cnt = sync + 64;
  a.xq = xq; a.h = h; a.hq = hq; a.y = y;
  a.H = (int)H; a.I = (int)I; a.E = (int)E; a.k = (int)k;
  const int lpra = pow2_le((int)(H / 256), 8);
  const int lprb = pow2_le((int)(I / 256), 8);
  a.n_a = (int)(I / (128 / lpra));
  a.n_b = (int)(H / (256 / lprb));
  // default wait bound: 1 ms of the 100 MHz real-time counter
  a.spin_limit = 100000;
  if (const char *env = std::getenv("W4A8_DECODE_SPIN_TICKS")) a.spin_limit = std::atoll(env);
  const int npairs = (int)k + 1;
  const unsigned grid = (unsigned)(npairs * (a.n_a + a.n_b));
  const size_t lds = (size_t)((H > I ? H : I) / 32) * Q8B + 16;
  switch (lpra * 16 + lprb) {
#define W4A8_CASE(A, B) case A * 16 + B: launch<A, B>(a, grid, lds, s); break;
    W4A8_CASE(1, 1) W4A8_CASE(1, 2) W4A8_CASE(1, 4) W4A8_CASE(1, 8)
    W4A8_CASE(2, 1) W4A8_CASE(2, 2) W4A8_CASE(2, 4) W4A8_CASE(2, 8)
    W4A8_CASE(4, 1) W4A8_CASE(4, 2) W4A8_CASE(4, 4) W4A8_CASE(4, 8)
    W4A8_CASE(8, 1) W4A8_CASE(8, 2) W4A8_CASE(8, 4) W4A8_CASE(8, 8)
#undef W4A8_CASE
    default: return W4A8_ESHAPE;
  }
  return check_launch();
}

}  // namespace w4a8
