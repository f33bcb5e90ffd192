/*
 * w4a8.h -- C ABI of libw4a8.so: Q4_0-weight x Q8_0-activation (W4A8) matrix
 * products over routed Mixture-of-Experts experts, for AMD Instinct MI355X
 * (gfx950).
 *
 * The method: 4-bit group-wise weights paired with 8-bit per-group
 * activations so that the inner product runs as integer multiply-adds, then
 * one scaling per group (paper Sec. 2.3 "Weight quantization", Sec. 3.3 "CPU
 * decode: W4A8"), applied to a sparse MoE feed-forward layer with top-k routed
 * experts and one always-on shared expert (Sec. 2.2 "The model"), where all
 * routed token-expert pairs of a layer are processed by one grouped launch
 * rather than one launch per expert (Sec. 3.2 "GPU prefill").
 *
 * Formats (fixed by this ABI):
 *   Q4_0 block, 18 bytes, 32 weights: fp16 scale d (little endian), then 16
 *     bytes; byte j holds code q_j in its low nibble and q_{j+16} in its high
 *     nibble; weight value = (q - 8) * d, q in 0..15.  Quantizer: d =
 *     fp16(m / -8) where m is the signed weight of largest magnitude (first
 *     index on ties), q = clamp(floor(w * (1/d) + 8.5), 0, 15) with 1/d taken
 *     as 0 when d == 0.
 *   Q8_0 block, 34 bytes, 32 activations: fp16 scale d, then 32 int8 codes;
 *     d = fp16(amax / 127), q = clamp(round_half_away(x * (1/d)), -127, 127),
 *     q = 0 when d == 0.  Every step is one IEEE binary32 operation, fp16
 *     rounding is to nearest even with subnormals kept.
 *   A matrix of N rows by K columns is N rows of K/32 consecutive blocks.
 *
 * Conventions for every entry point:
 *   - All data pointers are DEVICE pointers owned by the caller; the library
 *     never allocates, frees or keeps them after the call returns.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     Work is enqueued asynchronously; a return of W4A8_OK means the
 *     arguments were valid and the kernels were launched.
 *   - Every base pointer must be 16-byte aligned (W4A8_EALIGN otherwise).
 *   - Shapes are validated on the host before anything is launched; on an
 *     error nothing is enqueued and no output is touched.
 *   - Calls are thread-safe and re-entrant: the library keeps no state other
 *     than a per-device "is gfx950" check, the device's compute-unit count,
 *     the wait bound of w4a8_decode_wait_bound and, per device, the scratch
 *     array of moe_w4a8_forward_noalloc.  Concurrent calls must not share
 *     output or workspace buffers.
 */
#ifndef W4A8_H
#define W4A8_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define W4A8_OK          0
#define W4A8_ENULL      -1  /* a required pointer is NULL                        */
#define W4A8_ESHAPE     -2  /* bad shape (see each entry point)                  */
#define W4A8_ERANGE     -3  /* k, E or a size outside the supported range        */
#define W4A8_EWORKSPACE -4  /* workspace smaller than moe_w4a8_workspace_size()  */
#define W4A8_EALIGN     -5  /* a base pointer is not 16-byte aligned             */
#define W4A8_EHIP       -6  /* a HIP runtime call or kernel launch failed        */
#define W4A8_EDEVICE    -7  /* the current device is not gfx950                  */
#define W4A8_EALIAS     -8  /* an output shares its base address with an operand */
#define W4A8_ESCRATCH   -9  /* sizes beyond the fixed scratch of the no-allocation
                               entry point (W4A8_NOALLOC_SCRATCH_BYTES)           */

#define W4A8_Q4_0_BLOCK_BYTES 18
#define W4A8_Q8_0_BLOCK_BYTES 34
#define W4A8_Q4_SYM_BLOCK_BYTES 20
#define W4A8_Q8_F32_BLOCK_BYTES 36
#define W4A8_BLOCK 32

/* Static, NUL-terminated description of a status code (never NULL). */
const char *w4a8_strerror(int code);

/*
 * Q8_0 quantization of activations (Sec. 3.3: "quantized per group to 8-bit").
 *   x   [rows][K] fp32, row-major.
 *   xq  [rows][K/32] Q8_0 blocks (rows * K/32 * 34 bytes).
 * K % 32 != 0, rows < 0 or K <= 0 -> W4A8_ESHAPE.  rows == 0 is a no-op.
 * Result is bit-identical to the format definition above.
 */
int q8_0_quantize(const float *x, void *xq, int64_t rows, int64_t K, void *stream);

/*
 * Q4_0 quantization of weights (Sec. 2.3: group-wise symmetric 4-bit, two
 * values per byte, one scale per group).  Used to prepare expert tensors.
 *   w   [rows][K] fp32.   wq  [rows][K/32] Q4_0 blocks.
 * K % 32 != 0, rows < 0 or K <= 0 -> W4A8_ESHAPE.  Bit-identical to the
 * format definition above.
 */
int q4_0_quantize(const float *w, void *wq, int64_t rows, int64_t K, void *stream);

/*
 * W4A8 matrix-vector product, the decode kernel (Sec. 3.3, integer
 * multiply-add of 4-bit weights with 8-bit activations):
 *   y[n] = sum_b d_w[n,b] * d_x[b] * s[n,b],  s[n,b] = sum_i (q_w - 8) * q_x
 * with s exact in int32 and the scaled sum in fp32.
 *   w   [N][K/32] Q4_0 blocks;  xq [K/32] Q8_0 blocks;  y [N] fp32 (written).
 * K % 256 != 0 (every row then starts 16-byte aligned), N <= 0 or K <= 0
 * -> W4A8_ESHAPE.
 */
int q4q8_gemv(const void *w, const void *xq, float *y, int64_t N, int64_t K, void *stream);

/*
 * W4A8 matrix product of M activation rows with one weight matrix (the dense
 * per-layer projections and the output projection, about three quarters of
 * the paper's decode time, Sec. 5.2; the prefill products, Sec. 3.2), with the
 * block dot of Sec. 3.3:
 *   y[m][n] = sum_b d_w[n,b] * d_x[m,b] * s[m,n,b],  s exact in int32,
 *   the scaled sum in fp32.
 *   w   [N][K/32] Q4_0 blocks;  xq [M][K/32] Q8_0 blocks;  y [M][N] fp32,
 *   row-major (written).  M == 1 is q4q8_gemv (the workspace is not used);
 *   M > 1 needs workspace >= q4q8_gemm_workspace_size(M, K) bytes (the
 *   activations re-laid for the int8 matrix cores, or, for up to 128 rows
 *   over a small weight matrix, in nibble-split form with their chunk list
 *   for the VALU kernel; no initialisation).  Two launches per call.
 * K % 256 != 0, M < 0, N <= 0 or K <= 0 -> W4A8_ESHAPE; M, N >= 2^31,
 * K > 2^20, M * N >= 2^40 or M * K >= 2^40 -> W4A8_ERANGE.  M == 0 is a no-op.
 * q4q8_gemm_workspace_size returns 0 for invalid sizes.
 */
size_t q4q8_gemm_workspace_size(int64_t M, int64_t K);
int q4q8_gemm(const void *w, const void *xq, float *y, int64_t M, int64_t N, int64_t K,
              void *workspace, size_t ws_bytes, void *stream);

/*
 * The paper's own block format (Sec. 2.3 "Weight quantization": each weight
 * an integer in {-7..7} with one FP32 scale per group, two per byte;
 * Sec. 3.3: activations quantized per group to 8 bits with an FP32 scale,
 * every 4-bit weight held as the unsigned value in {1..15}).  32 per group:
 *   Q4_SYM block, 20 bytes: fp32 scale d (little endian), then 16 bytes in
 *     the Q4_0 nibble order (byte j: element j low, element j+16 high), each
 *     nibble q + 8 with q in -7..7; weight value = q * d.  Quantizer:
 *     d = amax / 7, q = clamp(round_half_away(w * (1/d)), -7, 7).
 *   Q8_F32 block, 36 bytes: fp32 scale d, then 32 int8 codes; d = amax / 127,
 *     q = clamp(round_half_away(x * (1/d)), -127, 127).
 *   In both, every step is one IEEE binary32 operation, and a zero scale, or
 *   one whose reciprocal overflows fp32 (below 2^-128), gives zero codes.
 * Quantizers: w or x [rows][K] fp32 -> [rows][K/32] blocks.  K % 32 != 0,
 * rows < 0 or K <= 0 -> W4A8_ESHAPE; rows == 0 is a no-op.  Bit-identical to
 * the definitions above.
 */
int q4_sym_quantize(const float *w, void *wq, int64_t rows, int64_t K, void *stream);
int q8_f32_quantize(const float *x, void *xq, int64_t rows, int64_t K, void *stream);

/*
 * Matrix-vector product in the paper's format (Sec. 3.3):
 *   y[n] = sum_b d_w[n,b] * d_x[b] * s[n,b],  s[n,b] = sum_i q_w * q_x
 * with s exact in int32 and the scaled sum in fp32.
 *   w  [N][K/32] Q4_SYM blocks;  xq [K/32] Q8_F32 blocks;  y [N] fp32.
 * K % 256 != 0, N <= 0 or K <= 0 -> W4A8_ESHAPE; K > 32768 -> W4A8_ERANGE
 * (the activation vector is staged whole in LDS).
 */
int q4sym_q8f32_gemv(const void *w, const void *xq, float *y, int64_t N, int64_t K,
                     void *stream);

/*
 * The routed + shared MoE layer in the paper's own format (Sec. 2.2: top-k
 * routed experts and one always-on shared expert; Sec. 2.3: Q4_SYM weights;
 * Sec. 3.3: Q8_F32 activations, integer block dots scaled once per group):
 *   for each token t, slot j with e = topk_ids[t][j] in [0, E):
 *     xq = Q8_F32(hidden[t]);  g|u = W_gu[e] xq;  h = SiLU(g) * u (fp32);
 *     hq = Q8_F32(h);  out[t] += topk_w[t][j] * (W_d[e] hq)
 *   and the shared expert the same way with weight 1.  Products as in
 *   q4sym_q8f32_gemv, SiLU and the sums in fp32.
 *   hidden [T][H] fp32, topk_ids [T][k] int32 (an id outside [0, E) skips the
 *   slot), topk_w [T][k] fp32; w_gate_up [E][2I][H/32] Q4_SYM blocks (the I
 *   gate rows, then the I up rows), w_down [E][H][I/32]; ws_gate_up [2I][H/32]
 *   and ws_down [H][I/32] the shared expert (both NULL: none); out [T][H]
 *   fp32 (may be hidden itself: hidden is read only by the first launch).
 * Two launches on the stream (gate/up with the quantization of hidden; down
 * with the combine), or three when a token's Q8_F32(h) of all k + 1 pairs
 * exceeds 48 KiB (down, then the combine on its own).  The
 * workspace (>= moe_sym_workspace_size bytes, no initialisation) holds, at
 * the offsets moe_sym_workspace_layout writes to offsets[0..2]:
 *   W4A8_SYM_WS_XQ  Q8_F32(hidden), [T][H/32] blocks;
 *   W4A8_SYM_WS_H   fp32 h, [P][I], P = T*k + T pairs (pair t*k + j, shared
 *                   pair T*k + t; rows of skipped pairs are not written);
 *   W4A8_SYM_WS_HQ  Q8_F32(h), [P][I/32] blocks.
 * Errors: H or I not a multiple of 256, T < 0, E, k <= 0 -> W4A8_ESHAPE;
 * H or I > 16384, k > 64, E or T >= 2^24, or more than 2^31 work items ->
 * W4A8_ERANGE; a required pointer NULL, or only one of the shared pair ->
 * W4A8_ENULL; base pointers not 16-byte aligned -> W4A8_EALIGN; workspace too
 * small -> W4A8_EWORKSPACE.  T == 0 is a no-op.  moe_sym_workspace_size
 * returns 0 for invalid sizes.
 */
#define W4A8_SYM_WS_XQ 0
#define W4A8_SYM_WS_H  1
#define W4A8_SYM_WS_HQ 2
size_t moe_sym_workspace_size(int64_t T, int64_t H, int64_t I, int64_t E, int64_t k);
int moe_sym_workspace_layout(int64_t T, int64_t H, int64_t I, int64_t E, int64_t k,
                             size_t *offsets);
int moe_sym_forward(const float *hidden, const int32_t *topk_ids, const float *topk_w,
                    const void *w_gate_up, const void *w_down, const void *ws_gate_up,
                    const void *ws_down, float *out, int64_t T, int64_t H, int64_t I,
                    int64_t E, int64_t k, void *workspace, size_t ws_bytes, void *stream);

/*
 * The gated-delta-net recurrence of the model's linear-attention layers
 * (Sec. 2.2: a state S in R^{dk x dv} per value head, updated token by token;
 * Sec. 5.5: a chunked / parallel scan as the lever for prefill), with the
 * update the gated delta rule of the work the paper cites, per head h and
 * token t (fp32):
 *   S_t = exp(g_t) (I - beta_t k_t k_t^T) S_{t-1} + beta_t k_t v_t^T
 *   o_t = S_t^T q_t
 * computed as a chunked scan (chunks of 32 tokens: per-chunk triangular
 * solve and products in parallel, the chunks in order per head and group of
 * 8 value columns); up to 8 tokens (decode) step by step in one launch.  The layer's projections, short convolutions, q/k
 * normalization and output gate are the caller's.
 *   q, k [T][NH][DK], v and out [T][NH][DV], g (log decay, <= 0 in the
 *   model) and beta [T][NH], all fp32; s0 [NH][DK][DV] the state before the
 *   first token (NULL: zero); s_out [NH][DK][DV] the state after the last
 *   (NULL: not written; may equal s0).  workspace >= gdn_workspace_size
 *   bytes, no initialisation.
 * Errors: DK not 64 or 128, DV not a positive multiple of 8, NH <= 0 or
 * T < 0 -> W4A8_ESHAPE; T >= 2^31, NH >= 2^16, DV > 4096 or too many
 * chunks -> W4A8_ERANGE; q, k, v, g, beta, out or workspace NULL ->
 * W4A8_ENULL (T == 0 without s_out is a no-op); q, k, v, out, s0, s_out or
 * the workspace not 16-byte aligned, g or beta not 4-byte aligned ->
 * W4A8_EALIGN; workspace too small -> W4A8_EWORKSPACE.
 * gdn_workspace_size returns 0 for invalid sizes.
 */
size_t gdn_workspace_size(int64_t T, int64_t NH, int64_t DK, int64_t DV);
int gdn_chunked_scan(const float *q, const float *k, const float *v, const float *g,
                     const float *beta, const float *s0, float *out, float *s_out, int64_t T,
                     int64_t NH, int64_t DK, int64_t DV, void *workspace, size_t ws_bytes,
                     void *stream);

/*
 * Bytes of device workspace moe_w4a8_forward needs for these sizes, or 0 if
 * the sizes are invalid.  The workspace must be zero-filled once before its
 * first use (moe_w4a8_workspace_init does that); the library leaves its
 * synchronisation words zero again when each call completes, so it can be
 * reused by later calls of any sizes whose moe_w4a8_workspace_size is at most
 * ws_bytes.  The single-token hand-off region has the same offset and size
 * for every shape, and no other region of any call overlaps it.  Calls that
 * overlap in time must not share a workspace.
 */
size_t moe_w4a8_workspace_size(int64_t T, int64_t H, int64_t I, int64_t E, int64_t k);

/* Zero-fill a workspace on `stream` with a kernel (no hipMemset node, so it
 * may be captured into a graph). */
int moe_w4a8_workspace_init(void *workspace, size_t ws_bytes, void *stream);

/*
 * Byte offsets of the documented workspace regions for these sizes, written
 * to offsets[0..W4A8_WS_NFIELDS-1] (see W4A8_WS_*).  Returns W4A8_OK or
 * W4A8_ESHAPE/W4A8_ERANGE.  The regions are valid after a forward call
 * completes and until the next call using the same workspace:
 *   W4A8_WS_XQ    Q8_0(hidden), [T][H/32] blocks.
 *   W4A8_WS_H     fp32 h = SiLU(gate) * up, [P][I], P = T*k + T pairs.
 *   W4A8_WS_HQ    Q8_0(h), [P][I/32] blocks.
 *   W4A8_WS_PERM  int32 [T*k + T]: pairs sorted by expert (stable in pair
 *                 index), routed pairs first, then the T shared pairs (not
 *                 written when T == 1: the single-token kernel needs no sort).
 *   W4A8_WS_COUNT int32 [E]: routed pairs per expert (not written when T == 1).
 *   W4A8_WS_SYNC  start of the synchronisation words, which end at
 *                 W4A8_WS_SYNC_END: zero before and after every call.
 *   W4A8_WS_XN    fp32 RMSNorm(x + y_prev) * gamma, [T][H] (moe_w4a8_layer
 *                 only).
 * Pair numbering: routed slot j of token t is pair t*k + j; the shared expert
 * of token t is pair T*k + t.  Rows of skipped slots are not written.
 */
#define W4A8_WS_XQ     0
#define W4A8_WS_H      1
#define W4A8_WS_HQ     2
#define W4A8_WS_PERM   3
#define W4A8_WS_COUNT  4
#define W4A8_WS_SYNC   5
#define W4A8_WS_SYNC_END 6
#define W4A8_WS_XN     7
#define W4A8_WS_NFIELDS 8
int moe_w4a8_workspace_layout(int64_t T, int64_t H, int64_t I, int64_t E, int64_t k,
                              size_t *offsets);

/*
 * Router top-k (Sec. 2.2: the sparsely gated MoE layer sends each token to
 * its top-k of E routed experts; the k gate values are the softmax
 * probabilities renormalized over the selection, as the Qwen3-series models
 * of Sec. 2.2 do).  Per token t of logits [T][E] fp32 (finite values):
 *   ids[t][0..k)   the k largest logits in descending order, equal logits
 *                  in increasing expert index.  Softmax is monotone, so this
 *                  is the order of the probabilities; it is decided on the
 *                  fp32 logits themselves, with no rounding in between.
 *   weights[t][j]  exp(l_j - l_max) / sum over the selection of
 *                  exp(l_i - l_max): the softmax over E restricted to the
 *                  selection and renormalized (its full denominator
 *                  cancels).  fp32, within a few ulps of the exact value.
 *   ids [T][k] int32 and weights [T][k] fp32 are overwritten; they feed
 *   moe_w4a8_forward / moe_w4a8_layer directly.
 * NULL pointer -> W4A8_ENULL; a pointer not 4-byte aligned -> W4A8_EALIGN;
 * T < 0 -> W4A8_ESHAPE; E < 1, E > 4096, k < 1, k > 32, k > E or
 * T >= 2^31 -> W4A8_ERANGE.  T == 0 is a no-op.
 */
int moe_router_topk(const float *logits, int32_t *ids, float *weights, int64_t T, int64_t E,
                    int64_t k, void *stream);

/*
 * One routed + shared MoE feed-forward layer in W4A8 (Sec. 2.2: top-k routed
 * experts plus an always-on shared expert; Sec. 3.2: one grouped pass over
 * all routed token-expert pairs; Sec. 3.3: W4A8 integer products):
 *
 *   xq_t        = Q8_0(hidden[t])
 *   for each slot j with e = topk_ids[t][j] in [0, E), and the shared expert:
 *     gu        = W4A8(w_gate_up[e], xq_t)              2I values, fp32
 *     h         = SiLU(gu[0:I]) * gu[I:2I]              fp32
 *     y         = W4A8(w_down[e], Q8_0(h))              H values, fp32
 *   out[t]      = sum_j topk_w[t][j] * y_j + y_shared
 *
 *   hidden     [T][H] fp32.
 *   topk_ids   [T][k] int32.  An id outside [0, E) (e.g. -1) skips the slot;
 *              a repeated id contributes once per slot.
 *   topk_w     [T][k] fp32 routing weights (used as given).
 *   w_gate_up  [E][2I][H/32] Q4_0 blocks: rows 0..I-1 gate, I..2I-1 up.
 *   w_down     [E][H][I/32] Q4_0 blocks.
 *   ws_gate_up, ws_down: the shared expert, shapes [2I][H/32] and [H][I/32];
 *              both NULL = no shared expert (one NULL alone -> W4A8_ENULL).
 *   out        [T][H] fp32, overwritten.
 *   workspace  ws_bytes >= moe_w4a8_workspace_size(T,H,I,E,k), zero-filled
 *              before its first use.
 * Shapes: H % 256, I % 256 != 0, T < 0 -> W4A8_ESHAPE; k < 1, k > 32, E < 1,
 * E > 4096 or T*(k+1) >= 2^31 -> W4A8_ERANGE.  T == 0 is a no-op.  out equal
 * to hidden -> W4A8_EALIAS (no in-place calls).
 * Results: Q8_0 stages bit-exact with the format definition for the fp32
 * values they receive; float outputs within fp32 rounding of the exact sums.
 */
int moe_w4a8_forward(const float *hidden, const int32_t *topk_ids, const float *topk_w,
                     const void *w_gate_up, const void *w_down,
                     const void *ws_gate_up, const void *ws_down,
                     float *out, int64_t T, int64_t H, int64_t I, int64_t E, int64_t k,
                     void *workspace, size_t ws_bytes, void *stream);

/*
 * One pre-norm residual MoE step of a chained stack (the layer input is the
 * RMSNorm of the residual stream, as in the Qwen3-series model family of
 * Sec. 2.2; the paper does not spell the norm out, so it is the standard
 * RMSNorm, see rmsnorm_residual):
 *   x_out = x + y_prev              one binary32 addition per element
 *                                   (x_out = x when y_prev is NULL)
 *   xn    = RMSNorm(x_out) * gamma  kept in the workspace region W4A8_WS_XN
 *   out   = moe_w4a8_forward's layer applied to xn
 * Arguments as for moe_w4a8_forward, plus x [T][H], y_prev [T][H] or NULL,
 * gamma [H], eps >= 0, x_out [T][H]; x_out and out must not alias x,
 * y_prev or each other (equal base addresses -> W4A8_EALIAS).  At T = 1 the
 * norm runs inside the single decode launch (every workgroup normalizes the
 * row it quantizes); at T > 1 inside the quantizing workgroups of the first
 * launch when H <= 4096 (a launch of its own for wider rows).  gamma or x_out
 * NULL -> W4A8_ENULL; eps < 0 -> W4A8_ESHAPE; other errors as for
 * moe_w4a8_forward.
 */
int moe_w4a8_layer(const float *x, const float *y_prev, const float *gamma, float eps,
                   float *x_out, const int32_t *topk_ids, const float *topk_w,
                   const void *w_gate_up, const void *w_down,
                   const void *ws_gate_up, const void *ws_down,
                   float *out, int64_t T, int64_t H, int64_t I, int64_t E, int64_t k,
                   void *workspace, size_t ws_bytes, void *stream);

/*
 * moe_w4a8_layer with the router in front (the sparsely gated layer of
 * Sec. 2.2 from its router logits on): moe_router_topk(router_logits) writes
 * topk_ids [T][k] and topk_w [T][k] (caller buffers, kept as outputs), then
 * the layer runs on them.  shared_gate [T] fp32 (or NULL): the shared
 * expert's output of token t is scaled by sigmoid(shared_gate[t]), computed
 * in fp32 (1 / (1 + exp(-g))); NULL keeps it always on with weight 1.
 *   router_logits [T][E] fp32, finite; k > E -> W4A8_ERANGE.
 *   router_logits or shared_gate not 4-byte aligned -> W4A8_EALIGN;
 *   router_logits NULL, or shared_gate without a shared expert -> W4A8_ENULL.
 * Other arguments and errors as for moe_w4a8_layer.  At T = 1 (E <= 512) the
 * routing runs inside the single launch of the layer.
 */
int moe_w4a8_layer_routed(const float *x, const float *y_prev, const float *gamma, float eps,
                          float *x_out, const float *router_logits, const float *shared_gate,
                          const void *w_gate_up, const void *w_down,
                          const void *ws_gate_up, const void *ws_down,
                          float *out, int32_t *topk_ids, float *topk_w,
                          int64_t T, int64_t H, int64_t I, int64_t E, int64_t k,
                          void *workspace, size_t ws_bytes, void *stream);

/*
 * Residual add and RMSNorm between chained MoE layers (the pre-norm chaining
 * of the Qwen3-series model family, Sec. 2.2; the paper does not spell the
 * norm out, so it is the standard RMSNorm).  Per row t of [T][H] fp32:
 *   x_out = x + y          one binary32 addition (x_out = x when y is NULL)
 *   xn    = x_out * (1 / sqrt(mean(x_out^2) + eps)) * gamma
 * The sum of squares is taken in a fixed order (the result does not depend on
 * scheduling).  x_out may alias x; xn must not alias x, y or x_out.  xn NULL
 * skips the norm (then gamma may be NULL).
 *   gamma [H] fp32.  H % 4 != 0, H <= 0, T < 0 or eps < 0 -> W4A8_ESHAPE;
 *   T >= 2^31 -> W4A8_ERANGE.  T == 0 is a no-op.
 */
int rmsnorm_residual(const float *x, const float *y, const float *gamma, float *x_out,
                     float *xn, int64_t T, int64_t H, float eps, void *stream);

/*
 * Bound on the poll rounds of the single-token kernel's wait for the h blocks
 * of other workgroups (each round one load round trip, about 0.5-1 us); past
 * it a workgroup computes the blocks itself (same code, same bytes), so
 * progress never depends on the order in which workgroups start.  Process
 * wide: rounds >= 0 sets it, rounds < 0 leaves it; returns the previous
 * value.  Default 2000, or W4A8_DECODE_SPIN_ROUNDS when set in the
 * environment at the library's first use.  (W4A8_DECODE_PREFETCH=0 there
 * turns off the kernel's L2 prefetch of gate/up rows by the down workgroups:
 * a timing aid, the results are the same.)
 */
int w4a8_decode_wait_bound(int64_t rounds);

/*
 * moe_w4a8_forward for callers that cannot allocate device memory or pass a
 * workspace: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Same arguments and results as moe_w4a8_forward
 * without the workspace, which is instead a fixed array of
 * W4A8_NOALLOC_SCRATCH_BYTES in device memory, one per GPU, held by the
 * library until the process ends (8 MiB: at the paper's layer shape, H =
 * 2048, I = 512, E = 256, k = 8, up to T = 66 tokens).  Sizes whose
 * moe_w4a8_workspace_size exceeds it -> W4A8_ESCRATCH.  The call allocates
 * nothing (no hipMalloc, no library allocation).  All calls on one GPU share
 * that GPU's array: calls that overlap in time on one GPU (other streams,
 * other threads) race and give undefined results.
 */
#define W4A8_NOALLOC_SCRATCH_BYTES ((size_t)8 << 20)
int moe_w4a8_forward_noalloc(const float *hidden, const int32_t *topk_ids, const float *topk_w,
                             const void *w_gate_up, const void *w_down,
                             const void *ws_gate_up, const void *ws_down,
                             float *out, int64_t T, int64_t H, int64_t I, int64_t E, int64_t k,
                             void *stream);

#ifdef __cplusplus
}
#endif

#endif /* W4A8_H */
