// The gated-delta-net (GDN) recurrence of the model's linear-attention layers
// (Sec. 2.2: a state S in R^{dk x dv} per value head, updated token by token;
// the update is the gated delta rule of the work the paper cites)
//   S_t = a_t (I - b_t k_t k_t^T) S_{t-1} + b_t k_t v_t^T,   o_t = S_t^T q_t,
// a_t = exp(g_t), as a chunked scan: the paper names a chunked / parallel scan
// as the lever its token-by-token kernel lacked (Sec. 5.5).
//
// Within a chunk of C = 32 tokens, with L_i the sum of g over the chunk up to
// token i, the delta-rule corrections u_i = b_i (v_i - a_i S_{i-1}^T k_i)
// solve a unit lower-triangular system, and everything else is products:
//   (I + A) U = diag(b) (V - diag(e^L) K S),  A_ij = b_i e^{L_i - L_j} k_i.k_j (j < i)
//   O = diag(e^L) Q S + P U,                  P_ij = e^{L_i - L_j} q_i.k_j  (j <= i)
//   S <- e^{L_C} S + K^T diag(e^{L_C - L}) U.
// Up to 8 tokens (decode) one launch steps through the recurrence as
// written (gdn_step).  Longer sequences take two launches:
//   gdn_prep: per (head, chunk), in parallel: L, the dot products k.k and q.k,
//     A and P, T' = (I + A)^{-1} diag(b) by forward substitution (each
//     column of the inverse depends only on itself: one lane per column) and
//     P T';
//   gdn_scan: per (head, 8 columns of the value dimension) -- the columns of
//     S evolve independently -- the chunks in order.  The workgroup's slice
//     of S (DK x 8) stays in the accumulators of 16 x 16 x 4 fp32 matrix
//     products and is copied column-major to LDS at each chunk; per chunk:
//     X = K S and Y = Q S on those products (one wave per 16-token tile of K
//     or of Q), W = V - e^L X, then per (token, column) thread U = T' W and
//     O = e^L Y + (P T') W (P T' from gdn_prep), and the state update
//     S <- e^{L_C} S + K^T (e^{L_C - L} U) on the products again.  All
//     column slices of a head run on one XCD, so the head's inputs are
//     fetched into that XCD's L2 once.
// All arithmetic in fp32.
#include "w4a8_dev.h"
#include "w4a8_host.h"

namespace w4a8 {

namespace {

constexpr int GC = 32;      // tokens per chunk
constexpr int GNT = 256;    // threads per workgroup
constexpr int DVS = 8;      // value columns per scan workgroup
constexpr int MAT = GC * GC;
constexpr int GDN_STEP_T = 8;   // up to this many tokens: the step kernel, no chunks

inline size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }

typedef float v4f __attribute__((ext_vector_type(4)));

struct GdnArgs {
  const float *q, *k, *v, *g, *beta, *s0;
  float *out, *s_out;
  float *tw, *pw, *lw;      // workspace: T' and P T' [NH][nch][C][C], L [NH][nch][C]
  int64_t T, NH, DV;
  int nch;
};

// Rows t0 .. t0 + 31 of head h of a [T][NH][D] tensor into LDS rows of
// stride D + 4 (zero past T).
template <int D>
__device__ __forceinline__ void load_rows(float (*dst)[D + 4], const float *src, int64_t t0,
                                          int64_t T, int64_t NH, int64_t h) {
  constexpr int D4 = D / 4;
  for (int idx = threadIdx.x; idx < GC * D4; idx += GNT) {
    const int i = idx / D4, c4 = idx - i * D4;
    const int64_t t = t0 + i;
    float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
    if (t < T) x = reinterpret_cast<const float4 *>(src)[(t * NH + h) * D4 + c4];
    *reinterpret_cast<float4 *>(&dst[i][4 * c4]) = x;
  }
}

// One chunk's inputs of a scan workgroup, loaded into registers while the
// previous chunk is computed: rows of K and Q (KF float4 per thread), the
// 32 x 8 slice of V, T' and P T' (4 values each) and L.
template <int DK>
struct ChunkRegs {
  static constexpr int KF = GC * DK / 4 / GNT;
  float4 k[KF], q[KF];
  float v[GC * DVS / GNT], tp[MAT / GNT], p[MAT / GNT], l;
};

template <int DK>
__device__ __forceinline__ void chunk_load(const GdnArgs &a, int64_t h, int cb, int ch,
                                           ChunkRegs<DK> &r) {
  constexpr int D4 = DK / 4;
  const int tid = threadIdx.x;
  const int64_t t0 = (int64_t)ch * GC;
#pragma unroll
  for (int u = 0; u < ChunkRegs<DK>::KF; u++) {
    const int idx = tid + u * GNT, i = idx / D4, c4 = idx - i * D4;
    const int64_t t = t0 + i;
    r.k[u] = r.q[u] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (t < a.T) {
      r.k[u] = reinterpret_cast<const float4 *>(a.k)[(t * a.NH + h) * D4 + c4];
      r.q[u] = reinterpret_cast<const float4 *>(a.q)[(t * a.NH + h) * D4 + c4];
    }
  }
#pragma unroll
  for (int u = 0; u < GC * DVS / GNT; u++) {
    const int idx = tid + u * GNT, i = idx / DVS, cc = idx - i * DVS;
    const int64_t t = t0 + i;
    r.v[u] = t < a.T ? a.v[(t * a.NH + h) * a.DV + cb + cc] : 0.0f;
  }
  const int64_t mat = (h * a.nch + ch) * MAT;
#pragma unroll
  for (int u = 0; u < MAT / GNT; u++) {
    r.tp[u] = a.tw[mat + tid + u * GNT];
    r.p[u] = a.pw[mat + tid + u * GNT];
  }
  r.l = tid < GC ? a.lw[(h * a.nch + ch) * GC + tid] : 0.0f;
}

template <int DK>
__global__ __launch_bounds__(GNT) void gdn_prep_kernel(GdnArgs a) {
  __shared__ __align__(16) float Ks[GC][DK + 4];
  __shared__ __align__(16) float Qs[GC][DK + 4];
  __shared__ float Am[GC][GC + 1], Pm[GC][GC + 1];
  __shared__ float Lc[GC], Bc[GC];
  const int tid = threadIdx.x;
  const int64_t h = blockIdx.x % a.NH;
  const int ch = (int)(blockIdx.x / a.NH);
  const int64_t t0 = (int64_t)ch * GC;
  load_rows<DK>(Ks, a.k, t0, a.T, a.NH, h);
  load_rows<DK>(Qs, a.q, t0, a.T, a.NH, h);
  if (tid < GC) {
    const int64_t t = t0 + tid;
    Lc[tid] = t < a.T ? a.g[t * a.NH + h] : 0.0f;      // g, summed below
    Bc[tid] = t < a.T ? a.beta[t * a.NH + h] : 0.0f;
  }
  __syncthreads();
  if (tid == 0) {                                      // inclusive sums, in token order
    float acc = 0.0f;
    for (int i = 0; i < GC; i++) {
      acc += Lc[i];
      Lc[i] = acc;
    }
  }
  __syncthreads();
  // k_i.k_j and q_i.k_j for i = tid / 8, j = 4 (tid % 8) .. + 3
  const int i = tid >> 3, j4 = (tid & 7) * 4;
  float kk[4] = {0.f, 0.f, 0.f, 0.f}, qk[4] = {0.f, 0.f, 0.f, 0.f};
  for (int c = 0; c < DK; c += 4) {
    const float4 ki = *reinterpret_cast<const float4 *>(&Ks[i][c]);
    const float4 qi = *reinterpret_cast<const float4 *>(&Qs[i][c]);
#pragma unroll
    for (int jj = 0; jj < 4; jj++) {
      const float4 kj = *reinterpret_cast<const float4 *>(&Ks[j4 + jj][c]);
      kk[jj] = fmaf(ki.x, kj.x, fmaf(ki.y, kj.y, fmaf(ki.z, kj.z, fmaf(ki.w, kj.w, kk[jj]))));
      qk[jj] = fmaf(qi.x, kj.x, fmaf(qi.y, kj.y, fmaf(qi.z, kj.z, fmaf(qi.w, kj.w, qk[jj]))));
    }
  }
  const int64_t mat = ((int64_t)h * a.nch + ch) * MAT;
#pragma unroll
  for (int jj = 0; jj < 4; jj++) {
    const int j = j4 + jj;
    const float d = j <= i ? expf(Lc[i] - Lc[j]) : 0.0f;
    Am[i][j] = j < i ? Bc[i] * d * kk[jj] : 0.0f;
    Pm[i][j] = d * qk[jj];
  }
  if (tid < GC) a.lw[((int64_t)h * a.nch + ch) * GC + tid] = Lc[tid];
  __syncthreads();
  // column j of (I + A)^{-1}: m_ij = -sum_{l=j}^{i-1} A_il m_lj (i > j), m_jj = 1
  // (rows above j are zero, so the sum may start at l = 0; both loops are
  // unrolled so the column stays in registers)
  if (tid < GC) {
    const int j = tid;
    float m[GC];
#pragma unroll
    for (int r = 0; r < GC; r++) {
      float acc = r == j ? 1.0f : 0.0f;
#pragma unroll
      for (int l = 0; l < r; l++) acc = fmaf(-Am[r][l], m[l], acc);
      m[r] = r >= j ? acc : 0.0f;
    }
    const float bj = Bc[j];
#pragma unroll
    for (int r = 0; r < GC; r++) {
      m[r] *= bj;
      a.tw[mat + r * GC + j] = m[r];
    }
    // column j of P T' (both lower triangular): the scan forms the output's
    // second term P U = (P T') W from W directly
#pragma unroll
    for (int r = 0; r < GC; r++) {
      float acc = 0.0f;
#pragma unroll
      for (int l = 0; l <= r; l++) acc = fmaf(Pm[r][l], m[l], acc);
      a.pw[mat + r * GC + j] = acc;
    }
  }
}

template <int DK>
__global__ __launch_bounds__(GNT) void gdn_scan_kernel(GdnArgs a) {
  constexpr int DKP = DK + 4;            // LDS row stride (rows of 8 threads hit distinct banks)
  static_assert(DK % 64 == 0 && GC * DVS == GNT && GC == 32 && DVS <= 16, "roles of the scan");
  // K in two buffers: the next chunk's rows are written while the state
  // update still reads this chunk's
  __shared__ __align__(16) float Ks[2][GC][DKP], Qs[GC][DKP];
  __shared__ __align__(16) float St[DVS][DKP];       // the slice of S, column-major
  // rows of T' and P T', and the columns of W and of e^{L_C - L} U, padded
  // to 36 floats: 16-byte reads, and the 8 rows a wave reads at once fall
  // in distinct banks
  constexpr int MP = GC + 4;
  __shared__ __align__(16) float Tp[GC][MP], PT[GC][MP];
  __shared__ __align__(16) float Wt[DVS][MP], Ugt[DVS][MP], Yt[DVS][MP];
  __shared__ float Vs[GC][DVS + 1];
  __shared__ float Lc[GC], eLs[GC];
  const int tid = threadIdx.x;
  const int nsl = (int)(a.DV / DVS);
  // workgroup b runs on XCD b % 8: with NH a multiple of 8, all column
  // slices of head h run on XCD h % 8, so each head's K, Q, T' and P come
  // from HBM once and are shared in that XCD's L2
  int64_t h;
  int sl;
  if (a.NH % 8 == 0) {
    const int x = blockIdx.x % 8, slot = blockIdx.x / 8;
    h = x + 8 * (slot / nsl);
    sl = slot % nsl;
  } else {
    h = blockIdx.x / nsl;
    sl = blockIdx.x % nsl;
  }
  const int cb = sl * DVS;
  // state: the slice S (DK x 8) as TPW 16 x 16 product tiles per wave
  // (columns 8..15 zero padding): lane l of wave w holds rows
  // 16 (TPW w + t) + 4 (l / 16) + e, e = 0..3, of column l % 16
  constexpr int TPW = DK / 64;
  const int wave = tid >> 6, lane = tid & 63, n = lane & 15, gq = lane >> 4;
  v4f S[TPW];
#pragma unroll
  for (int t = 0; t < TPW; t++) {
#pragma unroll
    for (int e = 0; e < 4; e++) {
      const int row = 16 * (TPW * wave + t) + 4 * gq + e;
      S[t][e] = a.s0 && n < DVS ? a.s0[(h * DK + row) * a.DV + cb + n] : 0.0f;
    }
  }
  // token role: token oi of the chunk, column oc (its value v_{oi,oc} is
  // element tid of the chunk's V slice)
  const int oi = tid / DVS, oc = tid % DVS;

  // chunk ch's inputs in nx, loaded two chunks ahead: once its values are
  // in LDS, nx takes chunk ch + 2
  auto chunk_step = [&](int ch, ChunkRegs<DK> &nx) {
    const int64_t t0 = (int64_t)ch * GC;
    float(*const Kb)[DKP] = Ks[ch & 1];
    {
      constexpr int D4 = DK / 4;
#pragma unroll
      for (int u = 0; u < ChunkRegs<DK>::KF; u++) {
        const int idx = tid + u * GNT, i = idx / D4, c4 = idx - i * D4;
        *reinterpret_cast<float4 *>(&Kb[i][4 * c4]) = nx.k[u];
        *reinterpret_cast<float4 *>(&Qs[i][4 * c4]) = nx.q[u];
      }
#pragma unroll
      for (int u = 0; u < MAT / GNT; u++) {
        const int idx = tid + u * GNT;
        Tp[idx >> 5][idx & 31] = nx.tp[u];
        PT[idx >> 5][idx & 31] = nx.p[u];
      }
      if (tid < GC) {
        Lc[tid] = nx.l;
        eLs[tid] = expf(nx.l);
      }
      Vs[oi][oc] = nx.v[0];
      if (n < DVS) {
#pragma unroll
        for (int t = 0; t < TPW; t++)
          *reinterpret_cast<float4 *>(&St[n][16 * (TPW * wave + t) + 4 * gq]) =
              make_float4(S[t][0], S[t][1], S[t][2], S[t][3]);
      }
    }
    __syncthreads();
    // the next chunk's inputs stream in while this one is computed
    if (ch + 2 < a.nch) chunk_load<DK>(a, h, cb, ch + 2, nx);

    // X = K S (waves 0, 1: tokens 0..15, 16..31) and Y = Q S (waves 2, 3)
    // on fp32 matrix products of 16 x 16 x 4 (value columns 8..15 of the
    // product are zero padding); lane group g = lane / 16 feeds the four k
    // of each step, taken as 4 consecutive rows per 4 steps so each operand
    // is one 16-byte LDS read per 4 products.  Then W = V - e^L X and e^L Y
    // into LDS by column.
    {
      const float(*A)[DKP] = wave < 2 ? Kb : Qs;
      const int arow = 16 * (wave & 1) + n;
      v4f acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
      for (int kb = 0; kb < DK; kb += 16) {
        const float4 av = *reinterpret_cast<const float4 *>(&A[arow][kb + 4 * gq]);
        const float4 bv = n < DVS ? *reinterpret_cast<const float4 *>(&St[n][kb + 4 * gq])
                                  : make_float4(0.f, 0.f, 0.f, 0.f);
        acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(av.x, bv.x, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(av.y, bv.y, acc1, 0, 0, 0);
        acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(av.z, bv.z, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(av.w, bv.w, acc1, 0, 0, 0);
      }
      if (n < DVS) {
#pragma unroll
        for (int e = 0; e < 4; e++) {
          const int tk = 16 * (wave & 1) + 4 * gq + e;
          const float d = acc0[e] + acc1[e];
          if (wave < 2) Wt[n][tk] = Vs[tk][n] - eLs[tk] * d;
          else Yt[n][tk] = eLs[tk] * d;
        }
      }
    }
    __syncthreads();
    // U = T' W (T' lower triangular) and e^{L_C - L_i} U for the state;
    // O = e^L Y + P U = e^L Y + (P T') W
    const float eC = expf(Lc[GC - 1]);
    {
      float u = 0.0f, o = Yt[oc][oi];
#pragma unroll
      for (int j = 0; j < GC; j += 4) {      // zero above the diagonal
        const float4 w = *reinterpret_cast<const float4 *>(&Wt[oc][j]);
        const float4 t = *reinterpret_cast<const float4 *>(&Tp[oi][j]);
        const float4 pt = *reinterpret_cast<const float4 *>(&PT[oi][j]);
        u = fmaf(t.w, w.w, fmaf(t.z, w.z, fmaf(t.y, w.y, fmaf(t.x, w.x, u))));
        o = fmaf(pt.w, w.w, fmaf(pt.z, w.z, fmaf(pt.y, w.y, fmaf(pt.x, w.x, o))));
      }
      Ugt[oc][oi] = expf(Lc[GC - 1] - Lc[oi]) * u;
      const int64_t t = t0 + oi;
      if (t < a.T) a.out[(t * a.NH + h) * a.DV + cb + oc] = o;
    }
    __syncthreads();
    // S <- e^{L_C} S + K^T Ug on the same products: A = K^T (this lane's
    // row of the tile, four tokens per four products), B = Ug by column
    // (this chunk's K stays in its buffer while the next chunk's inputs go to
    // the other one)
    {
#pragma unroll
      for (int t = 0; t < TPW; t++) S[t] *= eC;
#pragma unroll
      for (int kb = 0; kb < GC; kb += 16) {
        const float4 bv = n < DVS ? *reinterpret_cast<const float4 *>(&Ugt[n][kb + 4 * gq])
                                  : make_float4(0.f, 0.f, 0.f, 0.f);
        const float b4[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
        for (int t = 0; t < TPW; t++) {
          const int row = 16 * (TPW * wave + t) + n;
#pragma unroll
          for (int u = 0; u < 4; u++)
            S[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(Kb[kb + 4 * gq + u][row], b4[u], S[t], 0, 0, 0);
        }
      }
    }
  };
  ChunkRegs<DK> na, nb;
  if (a.nch > 0) chunk_load<DK>(a, h, cb, 0, na);
  if (a.nch > 1) chunk_load<DK>(a, h, cb, 1, nb);
  for (int ch = 0; ch < a.nch; ch += 2) {
    chunk_step(ch, na);
    if (ch + 1 < a.nch) chunk_step(ch + 1, nb);
  }
  if (a.s_out && n < DVS) {
#pragma unroll
    for (int t = 0; t < TPW; t++)
#pragma unroll
      for (int e = 0; e < 4; e++)
        a.s_out[(h * DK + 16 * (TPW * wave + t) + 4 * gq + e) * a.DV + cb + n] = S[t][e];
  }
}

// A few tokens (decode) step by step, the recurrence as written: per token,
// d = k^T S and o = S^T q reduced over the rows (8 neighbouring lanes by DPP,
// the four waves through LDS), S <- a (S - b k d^T) + b k v^T in between.
// Same thread layout as the scan (8 value columns per workgroup, DK/32 rows
// per thread).
template <int DK>
__global__ __launch_bounds__(GNT) void gdn_step_kernel(GdnArgs a) {
  constexpr int RPT = DK / (GNT / DVS);
  __shared__ float red[2][GNT / 64][DVS];
  const int tid = threadIdx.x;
  const int nsl = (int)(a.DV / DVS);
  const int64_t h = blockIdx.x / nsl;
  const int cb = (int)(blockIdx.x % nsl) * DVS;
  const int wave = tid >> 6, part = tid & 7;
  const int c = (tid >> 3) & (DVS - 1), r0 = (8 * wave + part) * RPT;
  float S[RPT];
#pragma unroll
  for (int m = 0; m < RPT; m++)
    S[m] = a.s0 ? a.s0[(h * DK + r0 + m) * a.DV + cb + c] : 0.0f;
  for (int64_t t = 0; t < a.T; t++) {
    const int64_t tk = (t * a.NH + h) * DK + r0;
    float kr[RPT], qr[RPT];
#pragma unroll
    for (int m = 0; m < RPT; m += 2) {
      const float2 k2 = *reinterpret_cast<const float2 *>(a.k + tk + m);
      const float2 q2 = *reinterpret_cast<const float2 *>(a.q + tk + m);
      kr[m] = k2.x; kr[m + 1] = k2.y;
      qr[m] = q2.x; qr[m + 1] = q2.y;
    }
    const float vc = a.v[(t * a.NH + h) * a.DV + cb + c];
    const float al = expf(a.g[t * a.NH + h]), be = a.beta[t * a.NH + h];
    float dp = 0.0f;
#pragma unroll
    for (int m = 0; m < RPT; m++) dp = fmaf(kr[m], S[m], dp);
    dp = sum8(dp);
    if (part == 0) red[0][wave][c] = dp;
    __syncthreads();
    float d = 0.0f;
#pragma unroll
    for (int w = 0; w < GNT / 64; w++) d += red[0][w][c];
    float op = 0.0f;
#pragma unroll
    for (int m = 0; m < RPT; m++) {
      S[m] = al * (S[m] - be * kr[m] * d) + be * kr[m] * vc;
      op = fmaf(qr[m], S[m], op);
    }
    op = sum8(op);
    if (part == 0) red[1][wave][c] = op;
    __syncthreads();
    if (tid < DVS) {
      float o = 0.0f;
#pragma unroll
      for (int w = 0; w < GNT / 64; w++) o += red[1][w][tid];
      a.out[(t * a.NH + h) * a.DV + cb + tid] = o;
    }
    __syncthreads();                       // red is rewritten for the next token
  }
  if (a.s_out) {
#pragma unroll
    for (int m = 0; m < RPT; m++) a.s_out[(h * DK + r0 + m) * a.DV + cb + c] = S[m];
  }
}

int gdn_validate(int64_t T, int64_t NH, int64_t DK, int64_t DV) {
  if (T < 0 || NH <= 0 || DV <= 0 || DV % DVS != 0 || (DK != 64 && DK != 128)) return W4A8_ESHAPE;
  if (T >= ((int64_t)1 << 31) || NH >= (1 << 16) || DV > 4096) return W4A8_ERANGE;
  const int64_t nch = (T + GC - 1) / GC;
  if (nch * NH >= ((int64_t)1 << 31) || T * NH * (DK > DV ? DK : DV) >= ((int64_t)1 << 40))
    return W4A8_ERANGE;
  return W4A8_OK;
}

}  // namespace

}  // namespace w4a8

using namespace w4a8;

extern "C" size_t gdn_workspace_size(int64_t T, int64_t NH, int64_t DK, int64_t DV) {
  if (gdn_validate(T, NH, DK, DV) != W4A8_OK) return 0;
  const int64_t nch = (T + GC - 1) / GC;
  return 2 * up256(sizeof(float) * (size_t)(NH * nch) * MAT) +
         up256(sizeof(float) * (size_t)(NH * nch) * GC) + 256;
}

extern "C" int gdn_chunked_scan(const float *q, const float *k, const float *v, const float *g,
                                const float *beta, const float *s0, float *out, float *s_out,
                                int64_t T, int64_t NH, int64_t DK, int64_t DV, void *workspace,
                                size_t ws_bytes, void *stream) {
  int rc = gdn_validate(T, NH, DK, DV);
  if (rc != W4A8_OK) return rc;
  if (T == 0 && !s_out) return W4A8_OK;
  if (!q || !k || !v || !g || !beta || !out || !workspace) return W4A8_ENULL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) || !aligned16(s0) ||
      !aligned16(s_out) || !aligned16(workspace) || (reinterpret_cast<uintptr_t>(g) & 3) ||
      (reinterpret_cast<uintptr_t>(beta) & 3))
    return W4A8_EALIGN;
  if (ws_bytes < gdn_workspace_size(T, NH, DK, DV)) return W4A8_EWORKSPACE;
  if ((rc = check_device()) != W4A8_OK) return rc;
  hipStream_t s = as_stream(stream);
  const int64_t nch = (T + GC - 1) / GC;
  uint8_t *ws = reinterpret_cast<uint8_t *>(workspace);
  GdnArgs a{};
  a.q = q; a.k = k; a.v = v; a.g = g; a.beta = beta; a.s0 = s0;
  a.out = out; a.s_out = s_out;
  a.tw = reinterpret_cast<float *>(ws);
  a.pw = reinterpret_cast<float *>(ws + up256(sizeof(float) * (size_t)(NH * nch) * MAT));
  a.lw = reinterpret_cast<float *>(ws + 2 * up256(sizeof(float) * (size_t)(NH * nch) * MAT));
  a.T = T; a.NH = NH; a.DV = DV; a.nch = (int)nch;
  const unsigned nwg = (unsigned)(NH * (DV / DVS));
  if (T <= GDN_STEP_T) {                      // a few tokens: the recurrence step by step
    if (DK == 128)
      gdn_step_kernel<128><<<dim3(nwg), dim3(GNT), 0, s>>>(a);
    else
      gdn_step_kernel<64><<<dim3(nwg), dim3(GNT), 0, s>>>(a);
    return check_launch();
  }
  if (nch > 0) {
    if (DK == 128)
      gdn_prep_kernel<128><<<dim3((unsigned)(NH * nch)), dim3(GNT), 0, s>>>(a);
    else
      gdn_prep_kernel<64><<<dim3((unsigned)(NH * nch)), dim3(GNT), 0, s>>>(a);
    if ((rc = check_launch()) != W4A8_OK) return rc;
  }
  if (DK == 128)
    gdn_scan_kernel<128><<<dim3(nwg), dim3(GNT), 0, s>>>(a);
  else
    gdn_scan_kernel<64><<<dim3(nwg), dim3(GNT), 0, s>>>(a);
  return check_launch();
}
