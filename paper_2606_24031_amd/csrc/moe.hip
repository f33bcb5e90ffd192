// Routed + shared MoE feed-forward layer in W4A8 (paper Sec. 2.2: top-k routed
// experts plus one always-on shared expert; Sec. 3.2: one grouped launch over
// all routed token-expert pairs instead of one launch per expert; Sec. 3.3:
// 4-bit x 8-bit integer products).
//
// Stages (all on the caller's stream):
//   1. Q8_0 of the hidden rows                          -> workspace xq
//   2. route: stable counting sort of the T*k pairs by expert (plus the T
//      shared pairs), the list of non-empty expert groups and of row tiles
//   3. gate/up: per (row tile, 32 h columns) the gate and up rows of the
//      expert against the tile's token rows, SwiGLU, Q8_0 of the 32-wide h
//      block                                           -> workspace h, hq
//   4. down: per (row tile, output row slab) the down rows against Q8_0(h),
//      scaled by the routing weight                    -> workspace y
//   5. combine: out[t] = sum over slots in slot order, then the shared pair
//      (fixed order, so the result does not depend on scheduling)
#include <algorithm>

#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

int launch_fill_zero(void *ptr, size_t bytes, hipStream_t s);
int launch_q8_0(const float *x, uint8_t *xq, int64_t nblocks, hipStream_t s);
size_t decode_sync_words(int64_t H);
size_t decode_xfer_words(int64_t I, int64_t k);
bool decode_supported(int64_t H, int64_t I, int64_t k);
int decode_forward(const float *x, const int32_t *ids, const float *topk_w, const uint8_t *w_gu,
                   const uint8_t *w_d, const uint8_t *ws_gu, const uint8_t *ws_d, float *out,
                   int64_t H, int64_t I, int64_t E, int64_t k, uint32_t *sync, uint32_t *xfer,
                   uint8_t *xq, float *h, uint8_t *hq, hipStream_t s);

namespace {

constexpr int MC = 4;           // token rows per tile
constexpr int ROUTE_T = 1024;   // threads of the route kernel
constexpr int LDS_INTS = 16000; // int32 cells of dynamic LDS for the route kernel (< 64 KB)

inline size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }

struct Layout {
  size_t meta, sync, xfer, perm, count, rank, groups, tiles, xq, h, hq, y, total;
  int64_t maxtiles;
};

// Region sizes depend only on (T, H, I, E, k).
Layout make_layout(int64_t T, int64_t H, int64_t I, int64_t E, int64_t k) {
  Layout L;
  const int64_t P = T * k + T;
  L.maxtiles = (T * k + MC - 1) / MC + std::min<int64_t>(E, T * k) + (T + MC - 1) / MC + 1;
  size_t off = 0;
  L.meta = off;   off += 256;
  L.sync = off;   off += up256(sizeof(uint32_t) * decode_sync_words(H));
  L.xfer = off;   off += up256(sizeof(uint32_t) * decode_xfer_words(I, k));
  L.perm = off;   off += up256(sizeof(int32_t) * P);
  L.count = off;  off += up256(sizeof(int32_t) * E);
  L.rank = off;   off += up256(sizeof(int32_t) * (T * k + 1));
  L.groups = off; off += up256(sizeof(int4) * (E + 1));
  L.tiles = off;  off += up256(sizeof(int2) * L.maxtiles);
  L.xq = off;     off += up256((size_t)T * (H / QK) * Q8B);
  L.h = off;      off += up256(sizeof(float) * (size_t)P * I);
  L.hq = off;     off += up256((size_t)P * (I / QK) * Q8B);
  L.y = off;      off += up256(sizeof(float) * (size_t)P * H);
  L.total = off;
  return L;
}

// Meta words (int32) at the start of the workspace.
enum { META_NROUTED = 0, META_NGROUPS = 1, META_NTILES = 2 };

int validate(int64_t T, int64_t H, int64_t I, int64_t E, int64_t k) {
  if (T < 0 || H <= 0 || I <= 0 || H % 256 != 0 || I % 256 != 0) return W4A8_ESHAPE;
  if (k < 1 || k > 32 || E < 1 || E > 4096) return W4A8_ERANGE;
  if (T * (k + 1) >= ((int64_t)1 << 31) || H > (1 << 20) || I > (1 << 20)) return W4A8_ERANGE;
  return W4A8_OK;
}

// ------------------------------------------------------------------ route
// Exclusive scan of a[0..n) in LDS by all ROUTE_T threads; returns the total.
__device__ int block_exscan(int *a, int n, int *wtot) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int per = (n + ROUTE_T - 1) / ROUTE_T;
  const int lo = min(tid * per, n), hi = min(lo + per, n);
  int s = 0;
  for (int i = lo; i < hi; i++) s += a[i];
  int x = s;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wtot[wave] = x;
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int w = 0; w < ROUTE_T / 64; w++) { const int v = wtot[w]; wtot[w] = run; run += v; }
    wtot[ROUTE_T / 64] = run;
  }
  __syncthreads();
  int base = wtot[wave] + x - s;
  for (int i = lo; i < hi; i++) { const int v = a[i]; a[i] = base; base += v; }
  const int total = wtot[ROUTE_T / 64];
  __syncthreads();
  return total;
}

struct RouteArgs {
  const int32_t *ids;
  int32_t *meta, *perm, *count, *rank;
  int4 *groups;  // {expert (E = shared), first sorted position, rows, first tile}
  int2 *tiles;   // {group, first row within the group}
  int T, k, E, has_shared, seg, nseg, ebits;
};

// One workgroup.  Pairs are cut into segments of `seg` (a multiple of 64);
// wave w owns segments w, w+16, ...  For every pair, its rank among the
// earlier pairs of the same expert inside its segment comes from wave ballots
// (lanes agreeing on every bit of the expert id); the per-(expert, segment)
// counts, laid out expert-major, are then scanned once, which yields at the
// same time each expert's offset and each segment's base inside it.  The
// resulting order is stable in pair index.
__global__ __launch_bounds__(ROUTE_T) void route_kernel(RouteArgs a) {
  extern __shared__ int hist[];  // [E][nseg]
  __shared__ int wtot[ROUTE_T / 64 + 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Pr = a.T * a.k;
  const int L = a.E * a.nseg;
  for (int i = tid; i < L; i += ROUTE_T) hist[i] = 0;
  __syncthreads();

  for (int s = wave; s < a.nseg; s += ROUTE_T / 64) {
    const int end = min((s + 1) * a.seg, Pr);
    for (int base = s * a.seg; base < end; base += 64) {
      const int p = base + lane;
      int e = -1;
      if (p < end) {
        e = a.ids[p];
        if (e < 0 || e >= a.E) e = -1;
      }
      const uint64_t valid = __ballot(e >= 0);
      uint64_t peers = valid;
      for (int bit = 0; bit < a.ebits; bit++) {
        const int mine = (e >> bit) & 1;
        const uint64_t b = __ballot(mine);
        peers &= mine ? b : ~b;
      }
      if (e >= 0) {
        const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
        const int idx = e * a.nseg + s;
        const int before = hist[idx];
        a.rank[p] = before + __popcll(peers & lt);
        if ((peers & lt) == 0) hist[idx] = before + __popcll(peers);
      }
    }
  }
  __syncthreads();
  const int nrouted = block_exscan(hist, L, wtot);

  for (int p = tid; p < Pr; p += ROUTE_T) {
    const int e = a.ids[p];
    if (e < 0 || e >= a.E) continue;
    a.perm[hist[e * a.nseg + p / a.seg] + a.rank[p]] = p;
  }
  if (a.has_shared)
    for (int t = tid; t < a.T; t += ROUTE_T) a.perm[nrouted + t] = Pr + t;
  __syncthreads();

  // counts, then the compacted list of non-empty groups (expert order) with
  // their tile ranges; the shared expert is the last group.
  int *gflag = hist + L;  // E + 1 entries after the histogram
  int *gtile = gflag + a.E + 1;
  for (int e = tid; e < a.E; e += ROUTE_T) {
    const int start = hist[e * a.nseg];
    const int stop = (e + 1 < a.E) ? hist[(e + 1) * a.nseg] : nrouted;
    a.count[e] = stop - start;
    gflag[e] = stop > start ? 1 : 0;
    gtile[e] = (stop - start + MC - 1) / MC;
  }
  if (tid == 0) {
    gflag[a.E] = (a.has_shared && a.T > 0) ? 1 : 0;
    gtile[a.E] = a.has_shared ? (a.T + MC - 1) / MC : 0;
  }
  __syncthreads();
  const int ngroups = block_exscan(gflag, a.E + 1, wtot);
  const int ntiles = block_exscan(gtile, a.E + 1, wtot);
  for (int e = tid; e <= a.E; e += ROUTE_T) {
    const int start = (e < a.E) ? hist[e * a.nseg] : nrouted;
    const int rows = (e < a.E) ? a.count[e] : (a.has_shared ? a.T : 0);
    if (rows == 0) continue;
    const int gi = gflag[e], t0 = gtile[e];
    a.groups[gi] = make_int4(e, start, rows, t0);
    for (int m0 = 0, t = t0; m0 < rows; m0 += MC, t++) a.tiles[t] = make_int2(gi, m0);
  }
  if (tid == 0) {
    a.meta[META_NROUTED] = nrouted;
    a.meta[META_NGROUPS] = ngroups;
    a.meta[META_NTILES] = ntiles;
  }
}

// ------------------------------------------------------------------ expert MLP
struct MlpArgs {
  const uint8_t *w_gu, *w_d, *ws_gu, *ws_d;
  const float *topk_w;
  const int32_t *meta, *perm;
  const int4 *groups;
  const int2 *tiles;
  const uint8_t *xq;
  float *h;
  uint8_t *hq;
  float *y;
  int64_t T, H, I, E, k;
};

__device__ __forceinline__ float silu_f32(float g) { return g / (1.0f + expf(-g)); }

// Gate/up for one (tile, 32-column h slab).  Thread (r, li): h column
// slab*32 + r, K-groups li, li+LPR, ...  Each lane holds its gate and up row
// group (2 x 144 bytes) and streams the tile's activation groups.
template <int LPR>
__global__ __launch_bounds__(32 * LPR) void gateup_kernel(MlpArgs a) {
  const int nslab = (int)(a.I / 32);
  const int tile = blockIdx.x / nslab, slab = blockIdx.x % nslab;
  if (tile >= a.meta[META_NTILES]) return;
  const int2 td = a.tiles[tile];
  const int4 gd = a.groups[td.x];
  const int mc = min(MC, gd.z - td.y);
  const int r = threadIdx.x / LPR, li = threadIdx.x % LPR;
  const int G = (int)(a.H / 256);
  const int64_t rowbytes = (int64_t)G * 8 * Q4B;
  const uint8_t *W = (gd.x < a.E) ? a.w_gu + (int64_t)gd.x * (2 * a.I) * rowbytes : a.ws_gu;
  const int64_t col = (int64_t)slab * 32 + r;
  const uint8_t *wg_row = W + col * rowbytes;
  const uint8_t *wu_row = W + (a.I + col) * rowbytes;

  int pair[MC];
  const uint8_t *act[MC];
  const int64_t xrow = (int64_t)G * 8 * Q8B;
#pragma unroll
  for (int m = 0; m < MC; m++) {
    const int p = a.perm[gd.y + td.y + min(m, mc - 1)];
    pair[m] = p;
    const int64_t t = (p < a.T * a.k) ? p / a.k : p - a.T * a.k;
    act[m] = a.xq + t * xrow;
  }
  float accg[MC], accu[MC];
#pragma unroll
  for (int m = 0; m < MC; m++) accg[m] = accu[m] = 0.0f;
  for (int g = li; g < G; g += LPR) {
    W8 wg, wu;
    load_w8(wg_row + (int64_t)g * (8 * Q4B), wg);
    load_w8(wu_row + (int64_t)g * (8 * Q4B), wu);
#pragma unroll
    for (int m = 0; m < MC; m++) {
      if (m < mc) {
        Act8 x;
        load_act8(act[m] + (int64_t)g * (8 * Q8B), x);
        accg[m] = dot8(wg, x, accg[m]);
        accu[m] = dot8(wu, x, accu[m]);
      }
    }
  }
  __shared__ float sh[MC][32];
#pragma unroll
  for (int m = 0; m < MC; m++) {
    const float gsum = lane_group_sum<LPR>(accg[m]);
    const float usum = lane_group_sum<LPR>(accu[m]);
    if (li == 0 && m < mc) {
      const float hv = silu_f32(gsum) * usum;
      sh[m][r] = hv;
      a.h[(int64_t)pair[m] * a.I + col] = hv;
    }
  }
  __syncthreads();
  // Q8_0 of the 32-wide h block of each token: 8 lanes per token.
  const int tid = threadIdx.x;
  if (tid < 8 * MC) {
    const int m = tid >> 3, j = tid & 7;
    if (m < mc) {
      float v[4] = {sh[m][4 * j], sh[m][4 * j + 1], sh[m][4 * j + 2], sh[m][4 * j + 3]};
      uint32_t d16;
      const uint32_t packed = q8_0_block8(v, d16);
      uint8_t *blk = a.hq + ((int64_t)pair[m] * (a.I / QK) + slab) * Q8B;
      store_q8_0_block8(blk, j, packed, d16);
    }
  }
}

// Down projection for one (tile, slab of 256/LPR output rows), scaled by the
// routing weight of each pair (1 for the shared expert).
template <int LPR>
__global__ __launch_bounds__(256) void down_kernel(MlpArgs a) {
  constexpr int RPB = 256 / LPR;
  const int nslab = (int)(a.H / RPB);
  const int tile = blockIdx.x / nslab, slab = blockIdx.x % nslab;
  if (tile >= a.meta[META_NTILES]) return;
  const int2 td = a.tiles[tile];
  const int4 gd = a.groups[td.x];
  const int mc = min(MC, gd.z - td.y);
  const int r = threadIdx.x / LPR, li = threadIdx.x % LPR;
  const int G = (int)(a.I / 256);
  const int64_t rowbytes = (int64_t)G * 8 * Q4B;
  const uint8_t *W = (gd.x < a.E) ? a.w_d + (int64_t)gd.x * a.H * rowbytes : a.ws_d;
  const int64_t n = (int64_t)slab * RPB + r;
  const uint8_t *wrow = W + n * rowbytes;

  int pair[MC];
  float wt[MC];
  const int64_t hrow = (int64_t)G * 8 * Q8B;
#pragma unroll
  for (int m = 0; m < MC; m++) {
    const int p = a.perm[gd.y + td.y + min(m, mc - 1)];
    pair[m] = p;
    wt[m] = (p < a.T * a.k) ? a.topk_w[p] : 1.0f;
  }
  float acc[MC];
#pragma unroll
  for (int m = 0; m < MC; m++) acc[m] = 0.0f;
  for (int g = li; g < G; g += LPR) {
    W8 w;
    load_w8(wrow + (int64_t)g * (8 * Q4B), w);
#pragma unroll
    for (int m = 0; m < MC; m++) {
      if (m < mc) {
        Act8 x;
        load_act8(a.hq + (int64_t)pair[m] * hrow + (int64_t)g * (8 * Q8B), x);
        acc[m] = dot8(w, x, acc[m]);
      }
    }
  }
#pragma unroll
  for (int m = 0; m < MC; m++) {
    const float v = lane_group_sum<LPR>(acc[m]);
    if (li == 0 && m < mc) a.y[(int64_t)pair[m] * a.H + n] = wt[m] * v;
  }
}

// out[t] = sum_j y[t*k + j] (slots in order, skipped slots left out) + y[T*k + t].
__global__ __launch_bounds__(256) void combine_kernel(const float *__restrict__ y,
                                                      const int32_t *__restrict__ ids,
                                                      float *__restrict__ out, int64_t T,
                                                      int64_t H, int k, int E, int has_shared) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t h4 = H / 4;
  if (i >= T * h4) return;
  const int64_t t = i / h4, c = i % h4;
  const float4 *y4 = reinterpret_cast<const float4 *>(y);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int j = 0; j < k; j++) {
    const int e = ids[t * k + j];
    if (e < 0 || e >= E) continue;
    const float4 v = y4[(t * k + j) * h4 + c];
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  if (has_shared) {
    const float4 v = y4[(T * k + t) * h4 + c];
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  reinterpret_cast<float4 *>(out)[i] = acc;
}

int pow2_floor_le(int g, int cap) {
  int l = 1;
  while (l * 2 <= g && l < cap) l *= 2;
  return l;
}

}  // namespace

int moe_forward_impl(const float *hidden, const int32_t *ids, const float *topk_w,
                     const uint8_t *w_gu, const uint8_t *w_d, const uint8_t *ws_gu,
                     const uint8_t *ws_d, float *out, int64_t T, int64_t H, int64_t I,
                     int64_t E, int64_t k, uint8_t *ws, size_t ws_bytes, hipStream_t s) {
  const Layout L = make_layout(T, H, I, E, k);
  const int has_shared = ws_gu != nullptr;
  int rc;

  // One token: the whole layer in a single launch (see decode.hip).
  if (T == 1 && decode_supported(H, I, k))
    return decode_forward(hidden, ids, topk_w, w_gu, w_d, ws_gu, ws_d, out, H, I, E, k,
                          reinterpret_cast<uint32_t *>(ws + L.sync),
                          reinterpret_cast<uint32_t *>(ws + L.xfer), ws + L.xq,
                          reinterpret_cast<float *>(ws + L.h), ws + L.hq, s);

  if ((rc = launch_q8_0(hidden, ws + L.xq, T * (H / QK), s)) != W4A8_OK) return rc;

  RouteArgs ra;
  ra.ids = ids;
  ra.meta = reinterpret_cast<int32_t *>(ws + L.meta);
  ra.perm = reinterpret_cast<int32_t *>(ws + L.perm);
  ra.count = reinterpret_cast<int32_t *>(ws + L.count);
  ra.rank = reinterpret_cast<int32_t *>(ws + L.rank);
  ra.groups = reinterpret_cast<int4 *>(ws + L.groups);
  ra.tiles = reinterpret_cast<int2 *>(ws + L.tiles);
  ra.T = (int)T; ra.k = (int)k; ra.E = (int)E; ra.has_shared = has_shared;
  const int64_t Pr = T * k;
  // smallest segment (multiple of 64 pairs) whose histogram fits in LDS
  int64_t seg = 64, nseg = std::max<int64_t>(1, (Pr + 63) / 64);
  while (E * nseg + 2 * (E + 1) > LDS_INTS) {
    seg += 64;
    nseg = std::max<int64_t>(1, (Pr + seg - 1) / seg);
  }
  ra.seg = (int)seg;
  ra.nseg = (int)nseg;
  ra.ebits = 0;
  while ((1 << ra.ebits) < E) ra.ebits++;
  const size_t lds = sizeof(int) * ((size_t)E * ra.nseg + 2 * (E + 1));
  route_kernel<<<dim3(1), dim3(ROUTE_T), lds, s>>>(ra);
  if ((rc = check_launch()) != W4A8_OK) return rc;

  MlpArgs ma;
  ma.w_gu = w_gu; ma.w_d = w_d; ma.ws_gu = ws_gu; ma.ws_d = ws_d;
  ma.topk_w = topk_w;
  ma.meta = ra.meta; ma.perm = ra.perm; ma.groups = ra.groups; ma.tiles = ra.tiles;
  ma.xq = ws + L.xq;
  ma.h = reinterpret_cast<float *>(ws + L.h);
  ma.hq = ws + L.hq;
  ma.y = reinterpret_cast<float *>(ws + L.y);
  ma.T = T; ma.H = H; ma.I = I; ma.E = E; ma.k = k;

  const int lpr_h = pow2_floor_le((int)(H / 256), 8);
  const unsigned grid_gu = (unsigned)(L.maxtiles * (I / 32));
  switch (lpr_h) {
    case 1: gateup_kernel<1><<<grid_gu, 32, 0, s>>>(ma); break;
    case 2: gateup_kernel<2><<<grid_gu, 64, 0, s>>>(ma); break;
    case 4: gateup_kernel<4><<<grid_gu, 128, 0, s>>>(ma); break;
    default: gateup_kernel<8><<<grid_gu, 256, 0, s>>>(ma); break;
  }
  if ((rc = check_launch()) != W4A8_OK) return rc;

  const int lpr_i = pow2_floor_le((int)(I / 256), 8);
  const unsigned grid_d = (unsigned)(L.maxtiles * (H / (256 / lpr_i)));
  switch (lpr_i) {
    case 1: down_kernel<1><<<grid_d, 256, 0, s>>>(ma); break;
    case 2: down_kernel<2><<<grid_d, 256, 0, s>>>(ma); break;
    case 4: down_kernel<4><<<grid_d, 256, 0, s>>>(ma); break;
    default: down_kernel<8><<<grid_d, 256, 0, s>>>(ma); break;
  }
  if ((rc = check_launch()) != W4A8_OK) return rc;

  const int64_t n4 = T * (H / 4);
  combine_kernel<<<dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s>>>(
      ma.y, ids, out, T, H, (int)k, (int)E, has_shared);
  return check_launch();
}

}  // namespace w4a8

using namespace w4a8;

extern "C" size_t moe_w4a8_workspace_size(int64_t T, int64_t H, int64_t I, int64_t E,
                                          int64_t k) {
  if (validate(T, H, I, E, k) != W4A8_OK) return 0;
  return make_layout(T, H, I, E, k).total;
}

extern "C" int moe_w4a8_workspace_layout(int64_t T, int64_t H, int64_t I, int64_t E,
                                         int64_t k, size_t *offsets) {
  if (!offsets) return W4A8_ENULL;
  const int rc = validate(T, H, I, E, k);
  if (rc != W4A8_OK) return rc;
  const Layout L = make_layout(T, H, I, E, k);
  offsets[W4A8_WS_XQ] = L.xq;
  offsets[W4A8_WS_H] = L.h;
  offsets[W4A8_WS_HQ] = L.hq;
  offsets[W4A8_WS_PERM] = L.perm;
  offsets[W4A8_WS_COUNT] = L.count;
  offsets[W4A8_WS_SYNC] = L.sync;
  offsets[W4A8_WS_SYNC_END] = L.xfer;
  return W4A8_OK;
}

extern "C" int moe_w4a8_workspace_init(void *workspace, size_t ws_bytes, void *stream) {
  if (!workspace) return W4A8_ENULL;
  if (!aligned16(workspace)) return W4A8_EALIGN;
  const int rc = check_device();
  if (rc != W4A8_OK) return rc;
  return launch_fill_zero(workspace, ws_bytes, as_stream(stream));
}

extern "C" int moe_w4a8_forward(const float *hidden, const int32_t *topk_ids,
                                const float *topk_w, const void *w_gate_up, const void *w_down,
                                const void *ws_gate_up, const void *ws_down, float *out,
                                int64_t T, int64_t H, int64_t I, int64_t E, int64_t k,
                                void *workspace, size_t ws_bytes, void *stream) {
  int rc = validate(T, H, I, E, k);
  if (rc != W4A8_OK) return rc;
  if (T == 0) return W4A8_OK;
  if (!hidden || !topk_ids || !topk_w || !w_gate_up || !w_down || !out || !workspace)
    return W4A8_ENULL;
  if ((ws_gate_up == nullptr) != (ws_down == nullptr)) return W4A8_ENULL;
  const void *ptrs[] = {hidden, topk_ids, topk_w, w_gate_up, w_down, out, workspace};
  for (const void *p : ptrs)
    if (!aligned16(p)) return W4A8_EALIGN;
  if (ws_gate_up && (!aligned16(ws_gate_up) || !aligned16(ws_down))) return W4A8_EALIGN;
  if (ws_bytes < make_layout(T, H, I, E, k).total) return W4A8_EWORKSPACE;
  if ((rc = check_device()) != W4A8_OK) return rc;
  return moe_forward_impl(hidden, topk_ids, topk_w,
                          reinterpret_cast<const uint8_t *>(w_gate_up),
                          reinterpret_cast<const uint8_t *>(w_down),
                          reinterpret_cast<const uint8_t *>(ws_gate_up),
                          reinterpret_cast<const uint8_t *>(ws_down), out, T, H, I, E, k,
                          reinterpret_cast<uint8_t *>(workspace), ws_bytes, as_stream(stream));
}
