// Routed + shared MoE feed-forward layer in W4A8 (paper Sec. 2.2: top-k routed
// experts plus one always-on shared expert; Sec. 3.2: one grouped launch over
// all routed token-expert pairs instead of one launch per expert; Sec. 3.3:
// 4-bit x 8-bit integer products).
//
// Stages (all on the caller's stream):
//   1. Q8_0 of the hidden rows                          -> workspace xq
//      (plus the copies the grouped kernels read: nibble-split, aligned)
//   2. route: stable counting sort of the T*k pairs by expert (plus the T
//      shared pairs), the list of non-empty expert groups, the chunks of the
//      small groups and the row tiles of the others (one workgroup, in the
//      same launch as stage 1)
//   3. gate/up: per (row tile, 64 h columns) the gate and up rows of the
//      expert against the tile's token rows, SwiGLU, Q8_0 of the 32-wide h
//      blocks (mfma.hip)                               -> workspace h, hq
//      (a batch of at most 128 tokens: the VALU kernels of smallm.hip
//      instead, which take the activations in nibble-split form)
//   4. down: per (row tile, 128 output rows) the down rows against Q8_0(h),
//      scaled by the routing weight                    -> workspace y
//   5. combine: out[t] = sum over slots in slot order, then the shared pair
//      (fixed order, so the result does not depend on scheduling)
#include <algorithm>
#include <mutex>

#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

int launch_fill_zero(void *ptr, size_t bytes, hipStream_t s);
bool small_supported(int64_t H, int64_t I);
int64_t small_max_chunks(int64_t T, int64_t E, int64_t k, int has_shared);
int small_gateup(const uint8_t *w_gu, const uint8_t *ws_gu, const uint8_t *xs,
                 const int32_t *meta, const int32_t *perm, const int4 *chunks, float *h,
                 uint8_t *hq, uint8_t *hs, int64_t maxchunks, int64_t T, int64_t H, int64_t I,
                 int64_t E, int64_t k, hipStream_t s);
int small_down(const uint8_t *w_d, const uint8_t *ws_d, const uint8_t *hs, const int32_t *meta,
               const int32_t *perm, const int4 *chunks, const float *topk_w,
               const float *shared_w, float *y, int64_t maxchunks, int64_t T, int64_t H,
               int64_t I, int64_t E, int64_t k, hipStream_t s);
int mfma_tile_rows();
int mfma_gateup(const uint8_t *w_gu, const uint8_t *ws_gu, const uint32_t *xa, const float *xd,
                const int32_t *meta, const int32_t *perm, const int4 *tiles, float *h,
                uint8_t *hq, uint32_t *ha, float *hd, int64_t maxtiles, int64_t T, int64_t H,
                int64_t I, int64_t E, int64_t k, hipStream_t s);
int mfma_down(const uint8_t *w_d, const uint8_t *ws_d, const uint32_t *ha, const float *hd,
              const int32_t *meta, const int32_t *perm, const int4 *tiles, const float *topk_w,
              const float *shared_w, float *y, int64_t maxtiles, int64_t T, int64_t H, int64_t I,
              int64_t E, int64_t k, bool few, hipStream_t s);
size_t decode_sync_words(int64_t H);
size_t decode_xfer_words();
bool decode_supported(int64_t H, int64_t I, int64_t k);
bool decode_routes(int64_t E, int64_t k);
int decode_forward(const float *x, const DecodeNorm &norm, const DecodeRoute *route,
                   const int32_t *ids,
                   const float *topk_w, const float *shared_w, const uint8_t *w_gu,
                   const uint8_t *w_d,
                   const uint8_t *ws_gu, const uint8_t *ws_d, float *out, int64_t H, int64_t I,
                   int64_t E, int64_t k, uint32_t *sync, uint32_t *xfer, uint8_t *xq, float *h,
                   uint8_t *hq, hipStream_t s);
int launch_rmsnorm(const float *x, const float *y, const float *gamma, float *x_out, float *xn,
                   int64_t T, int64_t H, float eps, hipStream_t s);
int router_launch(const float *logits, int32_t *ids, float *weights, const float *gate,
                  float *gate_w, int64_t T, int64_t E, int64_t k, hipStream_t s);

namespace {

constexpr int MC = 64;          // token rows per tile of the grouped MFMA kernels
constexpr int MC_FEW = 32;      // ... when 64-row tiles would leave compute units idle
constexpr int ROUTE_T = 1024;   // threads of the route kernel
constexpr int LDS_INTS = 16000; // int32 cells of dynamic LDS for the route kernel (< 64 KB)

inline size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }

constexpr int SLICE = ROUTE_T;   // pairs per slice of the split route
constexpr int RCH = 16;          // pairs a route thread keeps in registers

// The route splits into slices of ROUTE_T pairs ranked beside the
// quantization when a slice's per-chunk counts fit in LDS (16 x E ints); a
// single slice finishes the route in its own workgroup, several in a
// finishing launch of one workgroup per slice plus one for the lists.
inline bool split_route(int64_t E) { return E <= 1024; }

struct Layout {
  size_t meta, sync, xfer, perm, count, rank, hist, groups, tiles, chunks, xq, h, hq, y, xn, xs, hs,
      xa, xd, ha, hd, sw, total;
  int64_t maxtiles, maxchunks;
};

// Largest group that takes the VALU path (small_gateup / small_down, in
// chunks of SMALL_CHUNK rows): every group of a batch of up to 128 tokens,
// whose few-row groups are bound by weight streaming, where the VALU
// kernels keep every weight load of a workgroup in flight at once (64
// tokens: 104 us per layer against 127 on the tiles; 128 tokens: 137
// against 148; 256 tokens: 213 against 157).  Above that every group goes
// to the MFMA tiles, whose 16-row tiles pad a few-row group less than
// separate VALU launches for those groups cost (947 tokens: 207 us per
// layer against 214-218 with groups of up to 8 rows on the VALU kernels).
constexpr int64_t SMALL_T_MAX = 128;
inline int small_rows(int64_t T) { return T <= SMALL_T_MAX ? (int)SMALL_T_MAX : 0; }

// Region sizes depend only on (T, H, I, E, k).
Layout make_layout(int64_t T, int64_t H, int64_t I, int64_t E, int64_t k) {
  Layout L;
  const int64_t P = T * k + T;
  L.maxtiles = (T * k + MC_FEW - 1) / MC_FEW + std::min<int64_t>(E, T * k) + (T + MC_FEW - 1) / MC_FEW + 1;
  size_t off = 0;
  L.meta = off;   off += 256;
  L.sync = off;   off += up256(sizeof(uint32_t) * decode_sync_words(H));
  L.xfer = off;   off += up256(sizeof(uint32_t) * decode_xfer_words());
  L.perm = off;   off += up256(sizeof(int32_t) * (P + SMALL_CHUNK));
  L.count = off;  off += up256(sizeof(int32_t) * E);
  L.rank = off;   off += up256(sizeof(int32_t) * (T * k + 1));
  L.hist = off;   off += up256(sizeof(int32_t) * (size_t)E * ((T * k + SLICE - 1) / SLICE));
  L.groups = off; off += up256(sizeof(int4) * (E + 1));
  L.tiles = off;  off += up256(sizeof(int4) * L.maxtiles);
  L.maxchunks = small_max_chunks(T, E, k, 1);
  L.chunks = off; off += up256(sizeof(int4) * L.maxchunks);
  L.xq = off;     off += up256((size_t)T * (H / QK) * Q8B);
  L.h = off;      off += up256(sizeof(float) * (size_t)P * I);
  L.hq = off;     off += up256((size_t)P * (I / QK) * Q8B);
  L.y = off;      off += up256(sizeof(float) * (size_t)P * H);
  L.xn = off;     off += up256(sizeof(float) * (size_t)T * H);
  L.xs = off;     off += up256((size_t)T * split_row_bytes(H / QK));
  L.hs = off;     off += up256((size_t)P * split_row_bytes(I / QK));
  L.xa = off;     off += up256((size_t)T * H);          // aligned Q8_0 codes of x
  L.xd = off;     off += up256(sizeof(float) * (size_t)T * (H / QK));
  L.ha = off;     off += up256((size_t)P * I);          // aligned Q8_0 codes of h
  L.hd = off;     off += up256(sizeof(float) * (size_t)P * (I / QK));
  L.sw = off;     off += up256(sizeof(float) * (size_t)T);   // shared expert's gate weights
  L.total = off;
  return L;
}

// Meta words (int32) at the start of the workspace.
enum { META_NROUTED = 0, META_NGROUPS = 1, META_NTILES = 2, META_NSMALL = 3, META_NLONG = 4 };

int validate(int64_t T, int64_t H, int64_t I, int64_t E, int64_t k) {
  if (T < 0 || H <= 0 || I <= 0 || H % 256 != 0 || I % 256 != 0) return W4A8_ESHAPE;
  if (k < 1 || k > 32 || E < 1 || E > 4096) return W4A8_ERANGE;
  if (T * (k + 1) >= ((int64_t)1 << 31) || H > (1 << 20) || I > (1 << 20)) return W4A8_ERANGE;
  return W4A8_OK;
}

// ------------------------------------------------------------------ route
// Inclusive prefix sum over each 16-lane row (ROW16) or over the whole wave,
// all lanes active, on DPP: the row_shr 1, 2, 3 partials of the original
// values, then row_shr 4 and 8 (into the lanes of banks 1-3 and 2-3), then
// row 0's total into row 1 and row 2's into row 3, then row 1's into rows 2
// and 3.  Integer sums, so exact in any order.
template <int CTRL, int ROWS, int BANKS, bool BOUND>
__device__ __forceinline__ int dpp_or0(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, ROWS, BANKS, BOUND);
}
template <bool ROW16>
__device__ __forceinline__ int scan_incl(int v) {
  int s = v + dpp_or0<0x111, 0xF, 0xF, true>(v);   // row_shr:1
  s += dpp_or0<0x112, 0xF, 0xF, true>(v);            // row_shr:2
  s += dpp_or0<0x113, 0xF, 0xF, true>(v);            // row_shr:3
  s += dpp_or0<0x114, 0xF, 0xE, true>(s);            // row_shr:4, banks 1-3
  s += dpp_or0<0x118, 0xF, 0xC, true>(s);            // row_shr:8, banks 2-3
  if (!ROW16) {
    s += dpp_or0<0x142, 0xA, 0xF, false>(s);         // row_bcast:15 into rows 1, 3
    s += dpp_or0<0x143, 0xC, 0xF, false>(s);         // row_bcast:31 into rows 2, 3
  }
  return s;
}

// Exclusive scans of NA arrays a[j][0..n) in LDS at once by all ROUTE_T
// threads; tot[j] receives the total of array j.
template <int NA>
__device__ void block_exscan(int *const (&a)[NA], int n, int (*wtot)[ROUTE_T / 64 + 1],
                             int (&tot)[NA]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int per = (n + ROUTE_T - 1) / ROUTE_T;
  const int lo = min(tid * per, n), hi = min(lo + per, n);
  int s[NA], x[NA];
#pragma unroll
  for (int j = 0; j < NA; j++) {
    s[j] = 0;
    for (int i = lo; i < hi; i++) s[j] += a[j][i];
    x[j] = scan_incl<false>(s[j]);
  }
  if (lane == 63)
#pragma unroll
    for (int j = 0; j < NA; j++) wtot[j][wave] = x[j];
  __syncthreads();
  // the wave totals: exclusive scan in the first NA rows of 16 lanes, one
  // array per row (whole rows stay active)
  constexpr int NW = ROUTE_T / 64;
  static_assert(NW == 16 && NA <= 4, "one 16-lane row per array");
  if (tid < 64) {
    const int j = tid / NW, w = tid - j * NW;
    const int v = j < NA ? wtot[j][w] : 0;
    const int c = scan_incl<true>(v);
    if (j < NA) {
      wtot[j][w] = c - v;
      if (w == NW - 1) wtot[j][NW] = c;
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < NA; j++) {
    int base = wtot[j][wave] + x[j] - s[j];
    for (int i = lo; i < hi; i++) { const int v = a[j][i]; a[j][i] = base; base += v; }
    tot[j] = wtot[j][ROUTE_T / 64];
  }
  __syncthreads();
}


struct RouteArgs {
  const int32_t *ids;
  int32_t *meta, *perm, *count, *rank;
  int4 *groups;     // {expert (E = shared), first sorted position, rows, first tile}
  int4 *tiles;      // groups of more than ms rows, cut into tiles of mc rows:
                    // {expert, first sorted position, rows, group}
  int4 *chunks;     // groups of at most ms rows, cut into chunks of SMALL_CHUNK
                    // rows: {expert, first sorted position, rows, group}, in
                    // reverse group order
  int *hist_g;      // split route: per-(slice, expert) counts, slice-major [nseg][E]
  int T, k, E, has_shared, seg, nseg, ebits, ms;
  int mc;           // token rows per MFMA tile (MC, or MC_FEW for few tiles)
  int tpe;          // split route: threads per expert summing the slices' counts
  int stage;        // REG path: the permutation goes through LDS (it fits)
};

// Rank of this lane's pair among the earlier pairs of the same expert in its
// 64-pair chunk (lanes agreeing on every bit of the expert id), plus the
// pairs of that expert in the segment's earlier chunks (hist[e][s], advanced
// by the chunk's first lane of each expert).  e < 0: no pair.
__device__ __forceinline__ int chunk_rank(int e, int s, int *hist, const RouteArgs &a,
                                          int lane) {
  uint64_t peers = __ballot(e >= 0);
  for (int bit = 0; bit < a.ebits; bit++) {
    const int mine = (e >> bit) & 1;
    const uint64_t b = __ballot(mine);
    peers &= mine ? b : ~b;
  }
  int r = 0;
  if (e >= 0) {
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int idx = e * a.nseg + s;
    const int before = hist[idx];
    r = before + __popcll(peers & lt);
    if ((peers & lt) == 0) hist[idx] = before + __popcll(peers);
  }
  return r;
}

__device__ void build_lists(const RouteArgs &a, const int *rows_l, int *start_l, int *gi_l,
                            int *t0_l);

// Split route, first part, in the quantizing launch: slice s of ROUTE_T
// pairs, one 64-pair chunk per wave.  Each pair's rank among the earlier
// pairs of its slice with the same expert: its rank in its chunk (wave
// ballots) plus that expert's count in the slice's earlier chunks (a scan
// over the 16 chunks per expert, in LDS); the slice's count of each expert
// goes to the slice-major histogram hist_g[s][e], the ranks to `rank`.
// WHOLE: the slice is every pair (at most ROUTE_T), so the same workgroup
// finishes the route: the counts are the groups' rows, the lists come from
// them, and each pair's sorted position is its group's start plus its rank.
template <bool WHOLE>
__device__ void slice_ranks(const RouteArgs &a, int s) {
  extern __shared__ int cnt[];   // [16 chunks][E], later (WHOLE) the lists' 4 x (E + 1)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Pr = a.T * a.k;
  for (int i = tid; i < 16 * a.E; i += ROUTE_T) cnt[i] = 0;
  const int p = s * SLICE + tid;
  int e = -1;
  if (p < Pr) {
    e = a.ids[p];
    if (e < 0 || e >= a.E) e = -1;
  }
  __syncthreads();
  uint64_t peers = __ballot(e >= 0);
  for (int bit = 0; bit < a.ebits; bit++) {
    const int mine = (e >> bit) & 1;
    const uint64_t b = __ballot(mine);
    peers &= mine ? b : ~b;
  }
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int r = __popcll(peers & lt);
  if (e >= 0 && r == 0) cnt[wave * a.E + e] = __popcll(peers);   // the expert's first lane
  __syncthreads();
  int own = 0;    // WHOLE: the count of expert tid (E <= ROUTE_T)
  for (int ee = tid; ee < a.E; ee += ROUTE_T) {
    int run = 0;
#pragma unroll
    for (int w = 0; w < 16; w++) {
      const int c = cnt[w * a.E + ee];
      cnt[w * a.E + ee] = run;
      run += c;
    }
    if (WHOLE)
      own = run;
    else
      a.hist_g[s * a.E + ee] = run;
  }
  __syncthreads();
  const int rk = e >= 0 ? cnt[wave * a.E + e] + r : 0;
  if (!WHOLE) {
    if (e >= 0) a.rank[p] = rk;
    return;
  }
  __syncthreads();
  const int n = a.E + 1;
  int *rows_l = cnt, *start_l = cnt + n, *gi_l = cnt + 2 * n, *t0_l = cnt + 3 * n;
  if (tid < a.E) rows_l[tid] = own;
  if (tid == 0) rows_l[a.E] = a.has_shared ? a.T : 0;
  __syncthreads();
  build_lists(a, rows_l, start_l, gi_l, t0_l);
  if (e >= 0) a.perm[start_l[e] + rk] = p;
  if (a.has_shared && tid < a.T) a.perm[start_l[a.E] + tid] = Pr + tid;
}

// Experts per route thread: e = tid + j * ROUTE_T, j < EPT, covers E + 1 <=
// EPT * ROUTE_T groups (the shared expert is group E) for E <= 4096.
constexpr int EPT = 5;

// The group lists.  gst[j], grw[j]: first sorted position and rows of group
// e = tid + j * ROUTE_T (e <= E; the shared expert is group E, the last).
// Writes the compacted list of non-empty groups (expert order); a group of at
// most ms rows goes to the small-group list, a larger one gets its MFMA row
// tiles: those of more than mc/2 rows (full cost) first, in expert order, then
// the tiles of at most mc/2 rows (half cost), so each XCD can take an even
// share of both kinds, the longer work first.  The small-chunk and short-tile
// counts share one scanned word (low and high 16 bits: each total is at most
// E + 1).  cnt3: 3 x (E + 1) ints of LDS.  Every thread of the workgroup
// calls it.
__device__ void group_lists(const RouteArgs &a, const int (&gst)[EPT], const int (&grw)[EPT],
                            int *cnt3, int (*wtot)[ROUTE_T / 64 + 1], int nrouted) {
  const int tid = threadIdx.x;
  int *gflag = cnt3, *gtile = cnt3 + a.E + 1, *gsmall = gtile + a.E + 1;
#pragma unroll
  for (int j = 0; j < EPT; j++) {
    const int e = tid + j * ROUTE_T, rows = grw[j];
    if (e > a.E) break;
    gflag[e] = rows > 0 ? 1 : 0;
    const int rem = rows % a.mc;
    const bool tiled = rows > a.ms;
    gsmall[e] = ((rows > 0 && !tiled) ? (rows + SMALL_CHUNK - 1) / SMALL_CHUNK : 0) |
                ((tiled && rem > 0 && rem <= a.mc / 2) ? 1 << 16 : 0);
    gtile[e] = tiled ? rows / a.mc + (rem > a.mc / 2 ? 1 : 0) : 0;
  }
  __syncthreads();
  int tot[3];
  {
    int *const arr[3] = {gflag, gtile, gsmall};
    block_exscan<3>(arr, a.E + 1, wtot, tot);
  }
  const int ngroups = tot[0], nlong = tot[1], nsmall = tot[2] & 0xFFFF;
  const int ntiles = nlong + (tot[2] >> 16);
#pragma unroll
  for (int j = 0; j < EPT; j++) {
    const int e = tid + j * ROUTE_T, start_e = gst[j], rows = grw[j];
    if (e > a.E) break;
    if (rows == 0) continue;
    const int gi = gflag[e], t0 = gtile[e];
    a.groups[gi] = make_int4(e, start_e, rows, t0);
    if (rows <= a.ms) {
      // back to front: the shared expert (the largest group) comes first
      for (int m0 = 0, c = gsmall[e] & 0xFFFF; m0 < rows; m0 += SMALL_CHUNK, c++)
        a.chunks[nsmall - 1 - c] = make_int4(e, start_e + m0, min(SMALL_CHUNK, rows - m0), gi);
    } else {
      for (int m0 = 0, t = t0; m0 < rows; m0 += a.mc) {
        const int r = min(a.mc, rows - m0);
        a.tiles[r > a.mc / 2 ? t++ : nlong + (gsmall[e] >> 16)] = make_int4(e, start_e + m0, r, gi);
      }
    }
  }
  if (tid == 0) {
    a.meta[META_NROUTED] = nrouted;
    a.meta[META_NGROUPS] = ngroups;
    a.meta[META_NTILES] = ntiles;
    a.meta[META_NSMALL] = nsmall;
    a.meta[META_NLONG] = nlong;
  }
}

// The route in one workgroup, for expert counts above the split route's
// (E > 1024).  Pairs are cut into segments of `seg` (a multiple of 64);
// wave w owns segments w, w+16, ...  For every pair, its rank among the
// earlier pairs of the same expert inside its segment comes from wave ballots;
// the per-(expert, segment) counts, laid out expert-major, are then scanned
// once, which yields at the same time each expert's offset and each segment's
// base inside it.  The resulting order is stable in pair index.  MODE 1: every
// wave's chunks fit in RCH registers, so the ids are loaded in one batch and
// the ranks stay in registers until the scatter; MODE 0: the ranks go through
// the workspace.
template <int MODE>
__device__ __forceinline__ void route_body(const RouteArgs &a) {
  constexpr bool REG = MODE == 1;
  extern __shared__ int hist[];  // [E][nseg], later the group counters
  __shared__ int wtot[3][ROUTE_T / 64 + 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Pr = a.T * a.k;
  const int L = a.E * a.nseg;
  const int cps = a.seg >> 6;    // chunks per segment
  // register slot i (MODE 1): chunk i of this wave, segment wave + 16 (i /
  // cps), its chunk i % cps
  auto pair_of = [&](int i) {
    const int j = i / cps;
    return (wave + 16 * j) * a.seg + 64 * (i - j * cps) + lane;
  };
  auto seg_of = [&](int i) { return wave + 16 * (i / cps); };
  int er[RCH], rr[RCH];
  for (int i = tid; i < L; i += ROUTE_T) hist[i] = 0;

  if (REG) {
#pragma unroll
    for (int i = 0; i < RCH; i++) {
      const int j = i / cps, sg = wave + 16 * j;
      const int p = sg * a.seg + 64 * (i - j * cps) + lane;
      const bool live = sg < a.nseg && p < Pr;
      const int e = a.ids[live ? p : 0];
      er[i] = (live && e >= 0 && e < a.E) ? e : -1;
    }
  }
  __syncthreads();

  if (REG) {
#pragma unroll
    for (int i = 0; i < RCH; i++) {
      const int sg = wave + 16 * (i / cps);
      rr[i] = sg < a.nseg ? chunk_rank(er[i], sg, hist, a, lane) : 0;
    }
  } else {
    for (int sg = wave; sg < a.nseg; sg += ROUTE_T / 64) {
      const int end = (int)min((int64_t)(sg + 1) * a.seg, (int64_t)Pr);
      for (int base = sg * a.seg; base < end; base += 64) {
        const int p = base + lane;
        int e = -1;
        if (p < end) {
          e = a.ids[p];
          if (e < 0 || e >= a.E) e = -1;
        }
        const int r = chunk_rank(e, sg, hist, a, lane);
        if (e >= 0) a.rank[p] = r;
      }
    }
  }
  __syncthreads();
  int nrouted;
  {
    int *const arr[1] = {hist};
    int tot[1];
    block_exscan<1>(arr, L, wtot, tot);
    nrouted = tot[0];
  }

  // sorted position of each register-held pair; written straight to the
  // workspace, or (stage) through LDS so that the permutation leaves in
  // coalesced stores
  int dst[RCH];
  if (REG) {
#pragma unroll
    for (int i = 0; i < RCH; i++) {
      const int p = pair_of(i);
      dst[i] = er[i] >= 0 ? hist[er[i] * a.nseg + seg_of(i)] + rr[i] : -1;
      if (!a.stage && dst[i] >= 0) a.perm[dst[i]] = p;
    }
  } else {
    for (int p = tid; p < Pr; p += ROUTE_T) {
      const int e = a.ids[p];
      if (e < 0 || e >= a.E) continue;
      a.perm[hist[e * a.nseg + p / a.seg] + a.rank[p]] = p;
    }
  }
  if (a.has_shared && !a.stage)
    for (int t = tid; t < a.T; t += ROUTE_T) a.perm[nrouted + t] = Pr + t;

  // Each thread keeps the start and size of its groups in registers, and
  // the histogram's space then holds the three group counters.
  int gst[EPT], grw[EPT];
#pragma unroll
  for (int j = 0; j < EPT; j++) {
    const int e = tid + j * ROUTE_T;
    gst[j] = nrouted;
    grw[j] = 0;
    if (e < a.E) {
      gst[j] = hist[e * a.nseg];
      grw[j] = ((e + 1 < a.E) ? hist[(e + 1) * a.nseg] : nrouted) - gst[j];
      a.count[e] = grw[j];
    } else if (e == a.E) {
      grw[j] = a.has_shared ? a.T : 0;
    }
  }
  __syncthreads();
  if (REG && a.stage) {
#pragma unroll
    for (int i = 0; i < RCH; i++)
      if (dst[i] >= 0) hist[dst[i]] = pair_of(i);
    if (a.has_shared)
      for (int t = tid; t < a.T; t += ROUTE_T) hist[nrouted + t] = Pr + t;
    __syncthreads();
    const int ptot = nrouted + (a.has_shared ? a.T : 0);
    for (int i = tid; i < ptot; i += ROUTE_T) a.perm[i] = hist[i];
  }
  group_lists(a, gst, grw, hist + (a.stage ? Pr + a.T : 0), wtot, nrouted);
}

// Split route, second part: expert e's count over all slices (tot[e]) and
// over the slices before s (pre[e], if pre is not null), from the slice-major
// histogram; tpe consecutive threads per expert (a power of two dividing 64)
// each sum every tpe-th slice, eight loads in flight at a time, and combine
// with butterfly exchanges.  tot[E] = the shared expert's rows.  `between`
// runs once the first eight loads are issued (a loop head would wait for
// every load in flight, the caller's own included).  Every thread of the
// workgroup calls it.
template <typename F>
__device__ void expert_sums(const RouteArgs &a, int s, int *tot, int *pre, F between) {
  const int tid = threadIdx.x;
  const int e = tid / a.tpe, sub = tid & (a.tpe - 1);
  const int ec = e < a.E ? e : 0;     // threads past the experts read expert 0 and drop it
  int t = 0, b = 0;
  auto round = [&](int sg0, int (&v)[8]) {
#pragma unroll
    for (int i = 0; i < 8; i++) v[i] = a.hist_g[min(sg0 + i * a.tpe, a.nseg - 1) * a.E + ec];
  };
  auto add = [&](int sg0, const int (&v)[8]) {
#pragma unroll
    for (int i = 0; i < 8; i++) {
      const int sg = sg0 + i * a.tpe;
      const int x = sg < a.nseg ? v[i] : 0;
      t += x;
      b += sg < s ? x : 0;
    }
  };
  int v[8];
  round(sub, v);
  between();
  add(sub, v);
  for (int sg0 = sub + 8 * a.tpe; sg0 < a.nseg; sg0 += 8 * a.tpe) {
    round(sg0, v);
    add(sg0, v);
  }
  if (e >= a.E) t = b = 0;
  for (int o = 1; o < a.tpe; o <<= 1) {
    t += __shfl_xor(t, o);
    b += __shfl_xor(b, o);
  }
  if (e < a.E && sub == 0) {
    tot[e] = t;
    if (pre) pre[e] = b;
  }
  if (tid == 0) tot[a.E] = a.has_shared ? a.T : 0;
}

// Exclusive scan of n ints of LDS in place by one whole wave: lane l sums its
// contiguous run of ceil(n / 64) entries, the runs' sums are scanned across
// the wave, and each lane rewrites its run.  Returns the total (every lane).
__device__ int wave_exscan(int *v, int n) {
  const int lane = threadIdx.x & 63;
  const int per = (n + 63) / 64;
  const int lo = min(lane * per, n), hi = min(lo + per, n);
  int sum = 0;
  for (int i = lo; i < hi; i++) sum += v[i];
  const int incl = scan_incl<false>(sum);
  int base = incl - sum;
  for (int i = lo; i < hi; i++) { const int x = v[i]; v[i] = base; base += x; }
  return __shfl(incl, 63);
}

// The group lists from the groups' rows rows_l[0..E] (LDS; the shared expert
// is group E, the last), in the layout group_lists describes: wave 0 sums, per
// lane, a contiguous run of groups' rows, list entries, full tiles, small
// chunks and short tiles, scans the runs across the wave, and writes each
// group's first sorted position (start_l), list index (gi_l) and first full
// tile (t0_l) to LDS and its count, group, chunk and short-tile records; then
// every thread writes full tiles, each finding its group by binary search over
// t0_l.  Every thread of the workgroup calls it; start_l is valid on return.
__device__ void build_lists(const RouteArgs &a, const int *rows_l, int *start_l, int *gi_l,
                            int *t0_l) {
  __shared__ int nlong_s;
  const int tid = threadIdx.x;
  const int n = a.E + 1;
  if (tid < 64) {
    // lane l: groups [l * per, (l + 1) * per), the per-group quantities of
    // group_lists summed over the run, scanned across the wave, then each
    // group's records written from its bases
    const int lane = tid, per = (n + 63) / 64;
    const int lo = min(lane * per, n), hi = min(lo + per, n);
    int c[5] = {0, 0, 0, 0, 0};   // rows, groups, full tiles, small chunks, short tiles
    for (int g = lo; g < hi; g++) {
      const int rows = rows_l[g], rem = rows % a.mc;
      const bool tiled = rows > a.ms;
      c[0] += rows;
      c[1] += rows > 0 ? 1 : 0;
      c[2] += tiled ? rows / a.mc + (rem > a.mc / 2 ? 1 : 0) : 0;
      c[3] += (rows > 0 && !tiled) ? (rows + SMALL_CHUNK - 1) / SMALL_CHUNK : 0;
      c[4] += (tiled && rem > 0 && rem <= a.mc / 2) ? 1 : 0;
    }
    int base[5], tot5[5];
#pragma unroll
    for (int j = 0; j < 5; j++) {
      const int incl = scan_incl<false>(c[j]);
      base[j] = incl - c[j];
      tot5[j] = __shfl(incl, 63);
    }
    const int nlong = tot5[2], nsmall = tot5[3];
    for (int g = lo; g < hi; g++) {
      const int rows = rows_l[g], rem = rows % a.mc;
      const bool tiled = rows > a.ms;
      const int start = base[0], gi = base[1], t0 = base[2];
      start_l[g] = start;
      gi_l[g] = gi;
      t0_l[g] = t0;
      if (g < a.E) a.count[g] = rows;
      if (rows > 0) {
        a.groups[gi] = make_int4(g, start, rows, t0);
        if (!tiled) {
          // back to front: the shared group (the largest) comes first
          for (int m0 = 0, ch = base[3]; m0 < rows; m0 += SMALL_CHUNK, ch++)
            a.chunks[nsmall - 1 - ch] = make_int4(g, start + m0, min(SMALL_CHUNK, rows - m0), gi);
        } else if (rem > 0 && rem <= a.mc / 2) {
          a.tiles[nlong + base[4]] = make_int4(g, start + rows - rem, rem, gi);
        }
      }
      base[0] += rows;
      base[1] += rows > 0 ? 1 : 0;
      base[2] += tiled ? rows / a.mc + (rem > a.mc / 2 ? 1 : 0) : 0;
      base[3] += (rows > 0 && !tiled) ? (rows + SMALL_CHUNK - 1) / SMALL_CHUNK : 0;
      base[4] += (tiled && rem > 0 && rem <= a.mc / 2) ? 1 : 0;
    }
    if (lane == 0) {
      nlong_s = nlong;
      a.meta[META_NROUTED] = tot5[0] - (a.has_shared ? a.T : 0);
      a.meta[META_NGROUPS] = tot5[1];
      a.meta[META_NTILES] = nlong + tot5[4];
      a.meta[META_NSMALL] = nsmall;
      a.meta[META_NLONG] = nlong;
    }
  }
  __syncthreads();
  // full tiles, one per thread: tile ti belongs to the last group whose
  // first full tile is at most ti (binary search over the scanned counts)
  const int nlong = nlong_s;
  for (int ti = tid; ti < nlong; ti += ROUTE_T) {
    int lo = 0, hi = a.E;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (t0_l[mid] <= ti) lo = mid; else hi = mid - 1;
    }
    const int m0 = (ti - t0_l[lo]) * a.mc;
    a.tiles[ti] = make_int4(lo, start_l[lo] + m0, min(a.mc, rows_l[lo] - m0), gi_l[lo]);
  }
}

// Split route, second part, one workgroup per slice plus one: workgroup s <
// nseg writes the sorted positions of slice s's pairs (the expert's offset,
// plus its count in the earlier slices, plus the pair's rank in its slice;
// stable in pair index) and of the shared expert's rows s * SLICE ..; the
// last workgroup writes the counts, the group, tile and chunk lists and the
// meta words (the list layout of group_lists).
__global__ __launch_bounds__(ROUTE_T) void route_finish_kernel(RouteArgs a) {
  extern __shared__ int sm[];     // 4 x (E + 1) ints
  const int tid = threadIdx.x;
  const int s = blockIdx.x;
  const int n = a.E + 1;
  if (s < a.nseg) {
    const int Pr = a.T * a.k;
    const int p = s * SLICE + tid;
    // loaded from a clamped index beside the counts (a pair past the end
    // or with a skipped slot is dropped below)
    const int pc = min(p, Pr - 1);
    int e0, r;
    int *tot = sm, *pre = sm + n;
    expert_sums(a, s, tot, pre, [&] {
      e0 = a.ids[pc];
      r = a.rank[pc];
    });
    const int e = (p < Pr && e0 >= 0 && e0 < a.E) ? e0 : -1;
    __syncthreads();
    if (tid < 64) wave_exscan(tot, n);
    __syncthreads();
    if (e >= 0) a.perm[tot[e] + pre[e] + r] = p;
    if (a.has_shared && p < a.T) a.perm[tot[a.E] + p] = Pr + p;
    return;
  }
  int *rows_l = sm, *start_l = sm + n, *gi_l = sm + 2 * n, *t0_l = sm + 3 * n;
  expert_sums(a, -1, rows_l, nullptr, [] {});
  __syncthreads();
  build_lists(a, rows_l, start_l, gi_l, t0_l);
}

struct Q8Args {
  const float *x;
  uint8_t *xq;
  uint8_t *xs;      // nibble-split copy (small-group kernels, split_blk rows), or null
  uint32_t *xa;     // aligned codes and fp32 scales (MFMA kernels), or null
  float *xd;
  int64_t nblocks, nbrow;   // blocks in all, per row
  // pre-norm residual step folded in (norm_rows > 0): x_out = x + resid,
  // xn = RMSNorm(x_out) * gamma, and the Q8_0 forms are those of xn
  const float *resid;       // or null (no residual add)
  const float *gamma;
  float *x_out, *xn;
  float eps;
  int norm_rows;            // whole rows per quantizing workgroup, or 0
};

// The quantizing workgroup wg with the residual step folded in: rows
// wg * norm_rows .. + norm_rows - 1, H/4 threads per row (a multiple of 64),
// each thread the four elements 4c..4c+3 of its row: x_out = x + resid (one
// fp32 add per element), the sum of squares in a fixed order (the lane's four
// in index order, a butterfly over the wave, the row's waves in order), then
// xn = x_out * (1 / sqrt(sum / H + eps)) * gamma, written out and quantized
// in registers.  Every thread of the workgroup must call it.
__device__ void norm_q8_rows(const Q8Args &q, int64_t wg) {
  __shared__ float wsum[ROUTE_T / 64];
  const int h4 = (int)(q.nbrow * 8);
  const int t = (int)threadIdx.x;
  const int rl = t / h4, c = t - rl * h4;
  const int64_t T = q.nblocks / q.nbrow;
  const int64_t row = wg * q.norm_rows + rl;
  const bool live = rl < q.norm_rows && row < T;
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  if (live) {
    v = reinterpret_cast<const float4 *>(q.x)[row * h4 + c];
    if (q.resid) {
      const float4 d = reinterpret_cast<const float4 *>(q.resid)[row * h4 + c];
      v.x += d.x; v.y += d.y; v.z += d.z; v.w += d.w;
    }
    reinterpret_cast<float4 *>(q.x_out)[row * h4 + c] = v;
  }
  float ss = 0.0f;
  ss = fmaf(v.x, v.x, ss);
  ss = fmaf(v.y, v.y, ss);
  ss = fmaf(v.z, v.z, ss);
  ss = fmaf(v.w, v.w, ss);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  if ((t & 63) == 0) wsum[t >> 6] = ss;
  __syncthreads();
  const int w0 = (rl * h4) >> 6, nw = h4 >> 6;
  float tot = 0.0f;
  for (int w = 0; w < nw && live; w++) tot += wsum[w0 + w];
  const float r = 1.0f / sqrtf(tot / (float)(h4 * 4) + q.eps);
  float xn[4] = {0.f, 0.f, 0.f, 0.f};
  if (live) {
    const float4 g = reinterpret_cast<const float4 *>(q.gamma)[c];
    xn[0] = v.x * r * g.x; xn[1] = v.y * r * g.y; xn[2] = v.z * r * g.z; xn[3] = v.w * r * g.w;
    reinterpret_cast<float4 *>(q.xn)[row * h4 + c] = make_float4(xn[0], xn[1], xn[2], xn[3]);
  }
  q8_0_lane_vals(xn, q.xq, q.xs, q.xa, q.xd, q.nbrow, row * q.nbrow + (c >> 3), c & 7, live);
}

// Stages 1 and 2 in one launch (they are independent): the first `nroute`
// workgroups route -- the whole route in workgroup 0 (MODE 0, 1; MODE 3, one
// slice of at most ROUTE_T pairs), or the ranks of one slice each (MODE 2,
// finished by route_finish) -- the others quantize the hidden rows, ROUTE_T /
// 8 blocks each.
template <int MODE>
__global__ __launch_bounds__(ROUTE_T) void prep_kernel(RouteArgs a, Q8Args q, int nroute) {
  if ((int)blockIdx.x < nroute) {
    if (MODE >= 2)
      slice_ranks<MODE == 3>(a, blockIdx.x);
    else
      route_body<MODE>(a);
    return;
  }
  if (q.norm_rows)
    norm_q8_rows(q, (int64_t)(blockIdx.x - nroute));
  else
    q8_0_lane(q.x, q.xq, q.xs, q.xa, q.xd, q.nblocks, q.nbrow,
              (int64_t)(blockIdx.x - nroute) * ROUTE_T + threadIdx.x);
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
  // every load of a group of 8 slots in flight before any is waited for (a
  // skipped slot's row is read and left out), the shared expert's first
  const float4 vs = has_shared ? y4[(T * k + t) * h4 + c] : make_float4(0.f, 0.f, 0.f, 0.f);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int j0 = 0; j0 < k; j0 += 8) {
    int e[8];
    float4 v[8];
#pragma unroll
    for (int jj = 0; jj < 8; jj++) {
      const int j = min(j0 + jj, k - 1);
      e[jj] = ids[t * k + j];
      v[jj] = y4[(t * k + j) * h4 + c];
    }
#pragma unroll
    for (int jj = 0; jj < 8; jj++) {
      if (j0 + jj < k && e[jj] >= 0 && e[jj] < E) {
        acc.x += v[jj].x; acc.y += v[jj].y; acc.z += v[jj].z; acc.w += v[jj].w;
      }
    }
  }
  if (has_shared) {
    acc.x += vs.x; acc.y += vs.y; acc.z += vs.z; acc.w += vs.w;
  }
  reinterpret_cast<float4 *>(out)[i] = acc;
}

}  // namespace

int moe_forward_impl(const float *hidden, DecodeNorm norm, const int32_t *ids,
                     const float *topk_w, const float *shared_w, const uint8_t *w_gu,
                     const uint8_t *w_d,
                     const uint8_t *ws_gu, const uint8_t *ws_d, float *out, int64_t T, int64_t H,
                     int64_t I, int64_t E, int64_t k, uint8_t *ws, size_t ws_bytes,
                     hipStream_t s) {
  const Layout L = make_layout(T, H, I, E, k);
  const int has_shared = ws_gu != nullptr;
  int rc;
  if (norm.gamma) norm.xn = reinterpret_cast<float *>(ws + L.xn);

  // One token: the whole layer in a single launch, the residual RMSNorm
  // included (see decode.hip).
  if (T == 1 && decode_supported(H, I, k))
    return decode_forward(hidden, norm, nullptr, ids, topk_w, shared_w, w_gu, w_d, ws_gu, ws_d, out, H, I,
                          E, k,
                          reinterpret_cast<uint32_t *>(ws + L.sync),
                          reinterpret_cast<uint32_t *>(ws + L.xfer), ws + L.xq,
                          reinterpret_cast<float *>(ws + L.h), ws + L.hq, s);

  // the pre-norm residual step: inside the quantizing workgroups of the
  // prep launch when a row fits one of them, else a launch of its own
  const bool fold_norm = norm.gamma && H / 4 <= ROUTE_T;
  if (norm.gamma && !fold_norm) {
    if ((rc = launch_rmsnorm(hidden, norm.resid, norm.gamma, norm.x_out, norm.xn, T, H, norm.eps,
                             s)) != W4A8_OK)
      return rc;
    hidden = norm.xn;
  }
  const int ms = small_supported(H, I) ? small_rows(T) : 0;
  // with ms >= T every group (at most T rows) is small: no MFMA tiles
  const bool tiles = ms < T;
  uint8_t *xs = ws + L.xs;
  uint8_t *hs = ws + L.hs;
  uint32_t *xa = reinterpret_cast<uint32_t *>(ws + L.xa);
  uint32_t *ha = reinterpret_cast<uint32_t *>(ws + L.ha);
  float *xd = reinterpret_cast<float *>(ws + L.xd);
  float *hd = reinterpret_cast<float *>(ws + L.hd);
  Q8Args qa;
  qa.x = hidden;
  qa.xq = ws + L.xq;
  qa.xs = ms > 0 ? xs : nullptr;
  qa.xa = tiles ? xa : nullptr;
  qa.xd = xd;
  qa.nblocks = T * (H / QK);
  qa.nbrow = H / QK;
  qa.resid = norm.resid;
  qa.gamma = norm.gamma;
  qa.x_out = norm.x_out;
  qa.xn = norm.xn;
  qa.eps = norm.eps;
  qa.norm_rows = fold_norm ? (int)(ROUTE_T / (H / 4)) : 0;

  RouteArgs ra;
  ra.ids = ids;
  ra.meta = reinterpret_cast<int32_t *>(ws + L.meta);
  ra.perm = reinterpret_cast<int32_t *>(ws + L.perm);
  ra.count = reinterpret_cast<int32_t *>(ws + L.count);
  ra.rank = reinterpret_cast<int32_t *>(ws + L.rank);
  ra.groups = reinterpret_cast<int4 *>(ws + L.groups);
  ra.tiles = reinterpret_cast<int4 *>(ws + L.tiles);
  ra.chunks = reinterpret_cast<int4 *>(ws + L.chunks);
  ra.hist_g = reinterpret_cast<int32_t *>(ws + L.hist);
  ra.T = (int)T; ra.k = (int)k; ra.E = (int)E; ra.has_shared = has_shared; ra.ms = ms;
  // 64-row tiles, unless the pairs fill so few of them that most compute
  // units would get no gate/up workgroup (one expert over a prompt, a short
  // prompt's shared group): then 32-row tiles, and one down slice per
  // workgroup
  const int64_t est64 = (std::max<int64_t>((T * k + MC - 1) / MC, std::min<int64_t>(E, T * k)) +
                         (has_shared ? (T + MC - 1) / MC : 0)) * (I / 64);
  ra.mc = est64 < 2 * std::max(1, device_cus()) ? MC_FEW : MC;
  // launch bound on the tiles at this tile size (the workspace's tile list
  // is sized for MC_FEW)
  const int64_t gtiles =
      (T * k + ra.mc - 1) / ra.mc + std::min<int64_t>(E, T * k) + (T + ra.mc - 1) / ra.mc + 1;
  const int64_t Pr = T * k;
  ra.tpe = 1;
  ra.ebits = 0;
  while ((1 << ra.ebits) < E) ra.ebits++;
  const unsigned nq = qa.norm_rows ? (unsigned)((T + qa.norm_rows - 1) / qa.norm_rows)
                                   : (unsigned)((qa.nblocks * 8 + ROUTE_T - 1) / ROUTE_T);
  const int64_t nslice = (Pr + SLICE - 1) / SLICE;
  if (split_route(E)) {
    // slices of ROUTE_T pairs ranked beside the quantization; a single slice
    // finishes the route in the same workgroup, several in one more launch
    // (one workgroup per slice for the permutation, one for the lists)
    ra.seg = SLICE;
    ra.nseg = (int)nslice;
    ra.stage = 0;
    int e2 = 1;
    while (e2 < E) e2 *= 2;
    ra.tpe = (int)std::max<int64_t>(1, std::min<int64_t>(64, ROUTE_T / e2));
    const size_t lds1 = sizeof(int) * 16 * (size_t)E;
    if (nslice == 1) {
      prep_kernel<3><<<dim3(1 + nq), dim3(ROUTE_T), lds1, s>>>(ra, qa, 1);
    } else {
      prep_kernel<2><<<dim3((unsigned)nslice + nq), dim3(ROUTE_T), lds1, s>>>(ra, qa, (int)nslice);
      if ((rc = check_launch()) != W4A8_OK) return rc;
      route_finish_kernel<<<dim3((unsigned)nslice + 1), dim3(ROUTE_T),
                            sizeof(int) * 4 * (size_t)(E + 1), s>>>(ra);
    }
  } else {
    // smallest segment (multiple of 64 pairs) whose histogram fits in LDS
    const int64_t nseg_max = std::max<int64_t>(1, LDS_INTS / E);
    const int64_t seg = std::max<int64_t>(64, ((Pr + nseg_max - 1) / nseg_max + 63) / 64 * 64);
    const int64_t nseg = std::max<int64_t>(1, (Pr + seg - 1) / seg);
    ra.seg = (int)seg;
    ra.nseg = (int)nseg;
    // every wave's chunks fit the register arrays: at most RCH per wave
    const bool reg = (ra.nseg + 15) / 16 * (seg / 64) <= RCH;
    ra.stage = reg && Pr + T + 3 * (E + 1) <= LDS_INTS;
    const size_t lds = sizeof(int) * std::max<size_t>((size_t)E * ra.nseg,
                                                      (ra.stage ? Pr + T : 0) + 3 * (E + 1));
    if (reg)
      prep_kernel<1><<<dim3(1 + nq), dim3(ROUTE_T), lds, s>>>(ra, qa, 1);
    else
      prep_kernel<0><<<dim3(1 + nq), dim3(ROUTE_T), lds, s>>>(ra, qa, 1);
  }
  if ((rc = check_launch()) != W4A8_OK) return rc;

  uint8_t *hq = ws + L.hq;
  float *h = reinterpret_cast<float *>(ws + L.h);
  float *y = reinterpret_cast<float *>(ws + L.y);
  // launch bound on the small chunks (every group small when there are any)
  const int64_t maxchunks = small_max_chunks(T, E, k, has_shared);
  if (ms > 0 && (rc = small_gateup(w_gu, ws_gu, xs, ra.meta, ra.perm, ra.chunks, h, hq, hs,
                                   maxchunks, T, H, I, E, k, s)) != W4A8_OK)
    return rc;
  if (tiles && (rc = mfma_gateup(w_gu, ws_gu, xa, xd, ra.meta, ra.perm, ra.tiles, h, hq, ha, hd,
                                 gtiles, T, H, I, E, k, s)) != W4A8_OK)
    return rc;
  if (ms > 0 && (rc = small_down(w_d, ws_d, hs, ra.meta, ra.perm, ra.chunks, topk_w, shared_w, y,
                                 maxchunks, T, H, I, E, k, s)) != W4A8_OK)
    return rc;
  if (tiles && (rc = mfma_down(w_d, ws_d, ha, hd, ra.meta, ra.perm, ra.tiles, topk_w, shared_w,
                               y, gtiles, T, H, I, E, k, ra.mc == MC_FEW, s)) != W4A8_OK)
    return rc;

  const int64_t n4 = T * (H / 4);
  combine_kernel<<<dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s>>>(
      y, ids, out, T, H, (int)k, (int)E, has_shared);
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
  offsets[W4A8_WS_XN] = L.xn;
  return W4A8_OK;
}

extern "C" int moe_w4a8_workspace_init(void *workspace, size_t ws_bytes, void *stream) {
  if (!workspace) return W4A8_ENULL;
  if (!aligned16(workspace)) return W4A8_EALIGN;
  const int rc = check_device();
  if (rc != W4A8_OK) return rc;
  return launch_fill_zero(workspace, ws_bytes, as_stream(stream));
}

namespace w4a8 {
namespace {

// Arguments of a layer call other than the workspace.
int layer_core_args(const float *hidden, const int32_t *topk_ids, const float *topk_w,
                    const void *w_gate_up, const void *w_down, const void *ws_gate_up,
                    const void *ws_down, const float *out) {
  if (!hidden || !topk_ids || !topk_w || !w_gate_up || !w_down || !out) return W4A8_ENULL;
  if ((ws_gate_up == nullptr) != (ws_down == nullptr)) return W4A8_ENULL;
  const void *ptrs[] = {hidden, topk_ids, topk_w, w_gate_up, w_down, out};
  for (const void *p : ptrs)
    if (!aligned16(p)) return W4A8_EALIGN;
  if (ws_gate_up && (!aligned16(ws_gate_up) || !aligned16(ws_down))) return W4A8_EALIGN;
  // the single-token kernel reads the input row after other workgroups have
  // begun writing the output: no in-place calls
  if (static_cast<const void *>(out) == static_cast<const void *>(hidden)) return W4A8_EALIAS;
  return W4A8_OK;
}

int moe_args(const float *hidden, const int32_t *topk_ids, const float *topk_w,
             const void *w_gate_up, const void *w_down, const void *ws_gate_up,
             const void *ws_down, const float *out, int64_t T, int64_t H, int64_t I, int64_t E,
             int64_t k, const void *workspace, size_t ws_bytes) {
  int rc = validate(T, H, I, E, k);
  if (rc != W4A8_OK) return rc;
  if (T == 0) return W4A8_OK;
  if (!workspace) return W4A8_ENULL;
  if ((rc = layer_core_args(hidden, topk_ids, topk_w, w_gate_up, w_down, ws_gate_up, ws_down,
                            out)) != W4A8_OK)
    return rc;
  if (!aligned16(workspace)) return W4A8_EALIGN;
  if (ws_bytes < make_layout(T, H, I, E, k).total) return W4A8_EWORKSPACE;
  return W4A8_OK;
}

// moe_w4a8_layer's arguments (see include/w4a8.h).
int layer_args(const float *x, const float *y_prev, const float *gamma, float eps,
               const float *x_out, const int32_t *topk_ids, const float *topk_w,
               const void *w_gate_up, const void *w_down, const void *ws_gate_up,
               const void *ws_down, const float *out, int64_t T, int64_t H, int64_t I, int64_t E,
               int64_t k, const void *workspace, size_t ws_bytes) {
  int rc = moe_args(x, topk_ids, topk_w, w_gate_up, w_down, ws_gate_up, ws_down, out, T, H, I, E,
                    k, workspace, ws_bytes);
  if (rc != W4A8_OK || T == 0) return rc;
  if (!gamma || !x_out) return W4A8_ENULL;
  if (!(eps >= 0.0f)) return W4A8_ESHAPE;
  if (!aligned16(y_prev) || !aligned16(gamma) || !aligned16(x_out)) return W4A8_EALIGN;
  if (x_out == x || x_out == out || out == x || (y_prev && (x_out == y_prev || out == y_prev)))
    return W4A8_EALIAS;
  return W4A8_OK;
}

}  // namespace
}  // namespace w4a8

extern "C" int moe_w4a8_forward(const float *hidden, const int32_t *topk_ids,
                                const float *topk_w, const void *w_gate_up, const void *w_down,
                                const void *ws_gate_up, const void *ws_down, float *out,
                                int64_t T, int64_t H, int64_t I, int64_t E, int64_t k,
                                void *workspace, size_t ws_bytes, void *stream) {
  int rc = moe_args(hidden, topk_ids, topk_w, w_gate_up, w_down, ws_gate_up, ws_down, out, T, H,
                    I, E, k, workspace, ws_bytes);
  if (rc != W4A8_OK || T == 0) return rc;
  if ((rc = check_device()) != W4A8_OK) return rc;
  return moe_forward_impl(hidden, DecodeNorm{}, topk_ids, topk_w, nullptr,
                          reinterpret_cast<const uint8_t *>(w_gate_up),
                          reinterpret_cast<const uint8_t *>(w_down),
                          reinterpret_cast<const uint8_t *>(ws_gate_up),
                          reinterpret_cast<const uint8_t *>(ws_down), out, T, H, I, E, k,
                          reinterpret_cast<uint8_t *>(workspace), ws_bytes, as_stream(stream));
}

extern "C" int moe_w4a8_layer(const float *x, const float *y_prev, const float *gamma, float eps,
                              float *x_out, const int32_t *topk_ids, const float *topk_w,
                              const void *w_gate_up, const void *w_down, const void *ws_gate_up,
                              const void *ws_down, float *out, int64_t T, int64_t H, int64_t I,
                              int64_t E, int64_t k, void *workspace, size_t ws_bytes,
                              void *stream) {
  int rc = layer_args(x, y_prev, gamma, eps, x_out, topk_ids, topk_w, w_gate_up, w_down,
                      ws_gate_up, ws_down, out, T, H, I, E, k, workspace, ws_bytes);
  if (rc != W4A8_OK || T == 0) return rc;
  if ((rc = check_device()) != W4A8_OK) return rc;
  DecodeNorm norm;
  norm.resid = y_prev;
  norm.gamma = gamma;
  norm.x_out = x_out;
  norm.eps = eps;
  return moe_forward_impl(x, norm, topk_ids, topk_w, nullptr,
                          reinterpret_cast<const uint8_t *>(w_gate_up),
                          reinterpret_cast<const uint8_t *>(w_down),
                          reinterpret_cast<const uint8_t *>(ws_gate_up),
                          reinterpret_cast<const uint8_t *>(ws_down), out, T, H, I, E, k,
                          reinterpret_cast<uint8_t *>(workspace), ws_bytes, as_stream(stream));
}

extern "C" int moe_w4a8_layer_routed(const float *x, const float *y_prev, const float *gamma,
                                     float eps, float *x_out, const float *router_logits,
                                     const float *shared_gate, const void *w_gate_up,
                                     const void *w_down, const void *ws_gate_up,
                                     const void *ws_down, float *out, int32_t *topk_ids,
                                     float *topk_w, int64_t T, int64_t H, int64_t I, int64_t E,
                                     int64_t k, void *workspace, size_t ws_bytes, void *stream) {
  int rc = layer_args(x, y_prev, gamma, eps, x_out, topk_ids, topk_w, w_gate_up, w_down,
                      ws_gate_up, ws_down, out, T, H, I, E, k, workspace, ws_bytes);
  if (rc != W4A8_OK || T == 0) return rc;
  if (k > E) return W4A8_ERANGE;
  if (!router_logits || (shared_gate && !ws_gate_up)) return W4A8_ENULL;
  if ((reinterpret_cast<uintptr_t>(router_logits) | reinterpret_cast<uintptr_t>(shared_gate)) & 3u)
    return W4A8_EALIGN;
  if ((rc = check_device()) != W4A8_OK) return rc;
  const Layout L = make_layout(T, H, I, E, k);
  uint8_t *ws = reinterpret_cast<uint8_t *>(workspace);
  float *sw = shared_gate ? reinterpret_cast<float *>(ws + L.sw) : nullptr;
  hipStream_t s = as_stream(stream);
  if (T == 1 && decode_supported(H, I, k) && decode_routes(E, k)) {
    // one launch: the routing runs inside the single-token layer kernel
    DecodeNorm norm;
    norm.resid = y_prev;
    norm.gamma = gamma;
    norm.x_out = x_out;
    norm.eps = eps;
    if (gamma) norm.xn = reinterpret_cast<float *>(ws + L.xn);
    DecodeRoute route;
    route.logits = router_logits;
    route.gate = shared_gate;
    route.ids = topk_ids;
    route.w = topk_w;
    route.gate_w = sw;
    return decode_forward(x, norm, &route, nullptr, nullptr, nullptr,
                          reinterpret_cast<const uint8_t *>(w_gate_up),
                          reinterpret_cast<const uint8_t *>(w_down),
                          reinterpret_cast<const uint8_t *>(ws_gate_up),
                          reinterpret_cast<const uint8_t *>(ws_down), out, H, I, E, k,
                          reinterpret_cast<uint32_t *>(ws + L.sync),
                          reinterpret_cast<uint32_t *>(ws + L.xfer), ws + L.xq,
                          reinterpret_cast<float *>(ws + L.h), ws + L.hq, s);
  }
  if ((rc = router_launch(router_logits, topk_ids, topk_w, shared_gate, sw, T, E, k, s)) !=
      W4A8_OK)
    return rc;
  DecodeNorm norm;
  norm.resid = y_prev;
  norm.gamma = gamma;
  norm.x_out = x_out;
  norm.eps = eps;
  return moe_forward_impl(x, norm, topk_ids, topk_w, sw,
                          reinterpret_cast<const uint8_t *>(w_gate_up),
                          reinterpret_cast<const uint8_t *>(w_down),
                          reinterpret_cast<const uint8_t *>(ws_gate_up),
                          reinterpret_cast<const uint8_t *>(ws_down), out, T, H, I, E, k, ws,
                          ws_bytes, s);
}

// ------------------------------------------------------------ no allocation
// moe_w4a8_forward for callers that cannot allocate (code under graph
// capture, tight serving loops): the workspace is a fixed array in device
// memory, one per GPU, that the library owns for the life of the process.
namespace w4a8 {
namespace {

static __device__ __align__(256) uint8_t scratch[W4A8_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxScratchDevices];   // device address of `scratch`, per device

// The device address of this device's scratch array, looked up once per
// device with the device current (in host code the array's name is only a
// host-side stand-in).  The array is zero when the code object is loaded; the
// first call on a device also clears it on the caller's stream (unless that
// stream is being captured), before its own kernels.
int scratch_for_device(hipStream_t s, uint8_t **out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return W4A8_EHIP;
  if (dev < 0 || dev >= kMaxScratchDevices) return W4A8_EDEVICE;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_ptr[dev] == nullptr) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return W4A8_EHIP;
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cs) != hipSuccess) return W4A8_EHIP;
    if (cs == hipStreamCaptureStatusNone) {
      const int rc = launch_fill_zero(p, W4A8_NOALLOC_SCRATCH_BYTES, s);
      if (rc != W4A8_OK) return rc;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = reinterpret_cast<uint8_t *>(g_scratch_ptr[dev]);
  return W4A8_OK;
}

}  // namespace
}  // namespace w4a8

extern "C" int moe_w4a8_forward_noalloc(const float *hidden, const int32_t *topk_ids,
                                        const float *topk_w, const void *w_gate_up,
                                        const void *w_down, const void *ws_gate_up,
                                        const void *ws_down, float *out, int64_t T, int64_t H,
                                        int64_t I, int64_t E, int64_t k, void *stream) {
  int rc = validate(T, H, I, E, k);
  if (rc != W4A8_OK || T == 0) return rc;
  if ((rc = layer_core_args(hidden, topk_ids, topk_w, w_gate_up, w_down, ws_gate_up, ws_down,
                            out)) != W4A8_OK)
    return rc;
  const size_t need = make_layout(T, H, I, E, k).total;
  if (need > W4A8_NOALLOC_SCRATCH_BYTES) return W4A8_ESCRATCH;
  if ((rc = check_device()) != W4A8_OK) return rc;
  hipStream_t s = as_stream(stream);
  uint8_t *ws = nullptr;
  if ((rc = scratch_for_device(s, &ws)) != W4A8_OK) return rc;
  return moe_forward_impl(hidden, DecodeNorm{}, topk_ids, topk_w, nullptr,
                          reinterpret_cast<const uint8_t *>(w_gate_up),
                          reinterpret_cast<const uint8_t *>(w_down),
                          reinterpret_cast<const uint8_t *>(ws_gate_up),
                          reinterpret_cast<const uint8_t *>(ws_down), out, T, H, I, E, k, ws, need,
                          s);
}
