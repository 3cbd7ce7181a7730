/*
 * w8a8.h -- C ABI of the MI355X (gfx950) W8A8 SmoothQuant library.
 *
 * The operations follow arxiv 2608.28003 ("layer bit-width allocation ... under
 * a quality-degradation constraint", Gemma-3-1B):
 *   Sec. 3  eq. si, what-ffn    symmetric per-output-channel int8 weights, b = 8
 *   Sec. 4  eq. delta-attn      SmoothQuant migration factor, alpha = 0.5
 *   Sec. 6  eq. delta-lmhead, xhat-lmhead, what-lmhead   smoothing x/delta, W*delta
 *           eq. stx, xint8      dynamic per-token activation quantisation
 *           eq. gemm-final      y = s_t * s_i * sum_j q_x q_w
 *   Sec. 3  eq. ffn55, ffn1010, ffnall26   which FFN layers run in INT8
 *
 * Conventions for every entry point
 *   - Tensor pointers are DEVICE pointers allocated by the caller; the library
 *     allocates nothing, keeps no pointer after returning and holds no state
 *     beyond a cache of device properties.  Work is enqueued on `stream`
 *     (a hipStream_t; NULL is the default stream) and is asynchronous: results
 *     are ready after the caller synchronises that stream.
 *   - All matrices are row-major unless stated otherwise.  bf16 tensors are
 *     16-bit bfloat16 bit patterns.
 *   - Arguments are validated on the host before any HIP call:
 *       W8A8_EINVAL       NULL pointer, a size < 1, a pointer not 16-byte aligned
 *       W8A8_EUNSUPPORTED a dtype the call does not take, K > 133144 (the int32
 *                         accumulator bound K * 127^2 <= 2^31 - 1), or a shape
 *                         constraint stated at the call
 *       W8A8_EWORKSPACE   ws_bytes below the size the *_workspace_bytes query returns
 *       W8A8_EHIP         a HIP launch error (text in w8a8_last_error())
 *   - Numerical readings (the paper leaves them implicit): round() is round-half-
 *     to-even; codes are clamped to [-127, 127]; an all-zero row has scale 0 and
 *     codes 0; a smoothed value, its scale and the ratio that is rounded are IEEE
 *     binary32 with one rounding per operation; the dequantised value is
 *     (float(acc) * s_t) * s_i in binary32; bf16 outputs round to nearest even.
 *   - No exception crosses the ABI.  Non-finite inputs are outside the contract.
 *
 * Packed int8 layout ("fragment layout", used for weights and for quantised
 * activations).  A logical R x K int8 matrix is stored as Rp = ceil(R/16)*16 rows
 * by Kp = ceil(K/64)*64 columns, zero padded, cut into 16 x 64 fragments of
 * 1024 bytes.  Fragment (rb, kb) starts at byte (rb * Kp/64 + kb) * 1024; inside
 * it, lane l = 0..63 owns bytes [16 l, 16 l + 16), which hold row rb*16 + (l % 16),
 * columns kb*64 + (l / 16)*16 + 0..15.  One wavefront load of 16 bytes per lane
 * therefore reads one whole fragment, and a 16-row block is one contiguous run
 * of Kp*16 bytes.
 *
 * Packed bf16 layout: the same with 16 x 32 fragments of bf16 (1024 bytes):
 * Kp = ceil(K/32)*32; lane l holds row rb*16 + (l % 16), columns
 * kb*32 + (l / 16)*8 + 0..7.
 */
#ifndef W8A8_H
#define W8A8_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef void* w8a8_stream_t; /* a hipStream_t */

typedef enum {
    W8A8_OK = 0,
    W8A8_EINVAL = 1,
    W8A8_EUNSUPPORTED = 2,
    W8A8_EHIP = 3,
    W8A8_EWORKSPACE = 4,
    W8A8_ETIMEOUT = 5   /* w8a8_ffn_stack_status only: a persistent launch gave up */
} w8a8_status;

typedef enum { W8A8_F32 = 0, W8A8_BF16 = 1 } w8a8_dtype;

#define W8A8_MAX_K 133144
#define W8A8_HEAD_DIM 256   /* attention head width (Sec. 2, Tab. 2) */

/* One INT8 linear layer y = x W^T (Sec. 6): packed codes of W_hat = W diag(delta)
   (n x k, fragment layout), their per-output-channel scales s_w[n], and the
   smoothing factors delta[k] the activations are divided by (NULL: none). */
typedef struct {
    int64_t n, k;
    const void* wq;
    const float* s_w;
    const float* delta;
} w8a8_linear_desc;

/* One INT8 gated FFN block (Sec. 3): gate and up are d -> f and share the input
   and its smoothing delta_gu[d]; down is f -> d with its own delta_down[f]. */
typedef struct {
    int64_t d, f;
    const void* wq_gate; const float* s_gate;   /* f x d packed, [f] */
    const void* wq_up;   const float* s_up;     /* f x d packed, [f] */
    const float* delta_gu;                      /* [d] or NULL */
    const void* wq_down; const float* s_down;   /* d x f packed, [d] */
    const float* delta_down;                    /* [f] or NULL */
} w8a8_ffn_desc;

/* One bf16 gated FFN block (the layers a precision map keeps in bf16):
   weights in the packed bf16 layout. */
typedef struct {
    int64_t d, f;
    const void* wp_gate;  /* f x d */
    const void* wp_up;    /* f x d */
    const void* wp_down;  /* d x f */
} w8a8_bf16_ffn_desc;

/* A stack of FFN blocks with RMSNorm glue and an lm_head (used with a
   precision map).  int8_ffn[l] is read for layers the map sets to INT8,
   bf16_ffn[l] for the others; both arrays live in HOST memory. */
typedef struct {
    int64_t n_layers, d, f, vocab;
    const w8a8_ffn_desc* int8_ffn;
    const w8a8_bf16_ffn_desc* bf16_ffn;
    w8a8_linear_desc lm_head_int8;   /* n = vocab, k = d */
    const void* lm_head_bf16;        /* vocab x d, packed bf16 layout */
} w8a8_stack_desc;

/* ---------------------------------------------------------------- sizes */

/* Bytes of the packed int8 layout for a logical n x k matrix. */
size_t w8a8_packed_bytes(int64_t n, int64_t k);
/* Bytes of the packed bf16 layout for a logical n x k matrix. */
size_t w8a8_packed_bf16_bytes(int64_t n, int64_t k);
/* Workspace the calls below need (bytes, 256-byte aligned sub-buffers). */
size_t w8a8_linear_workspace_bytes(int64_t m, int64_t n, int64_t k);
size_t w8a8_ffn_workspace_bytes(int64_t m, int64_t d, int64_t f);
size_t w8a8_bf16_ffn_workspace_bytes(int64_t m, int64_t d, int64_t f);
size_t w8a8_lm_head_workspace_bytes(int64_t m, int64_t n, int64_t k);
size_t w8a8_bf16_linear_workspace_bytes(int64_t m, int64_t n, int64_t k);
size_t w8a8_stack_workspace_bytes(int64_t m, int64_t d, int64_t f, int64_t vocab);

/* ---------------------------------------------------------------- a1: calibration */

/* Running column maximum (Sec. 4 eq. delta-attn, Sec. 6 eq. delta-lmhead):
   amax[j] <- max(amax[j], max_t |x[t][j]|) over the rows x[rows][k].  Applied to
   calibration activations it gives max_t |X_tj|; applied to each weight matrix
   that consumes an input (gate and up for the FFN input) it gives max_i |W_ij|.
   x: f32 or bf16; amax: device float[k], read and written (start from zeros). */
w8a8_status w8a8_col_absmax(const void* x, w8a8_dtype x_dtype, int64_t rows, int64_t k,
                            float* amax, w8a8_stream_t stream);

/* SmoothQuant factor from the weights (Sec. 4 eq. delta-attn, Sec. 6 eq.
   delta-lmhead): delta[j] = a_j^alpha / w_j^(1 - alpha), where
   a_j = max(act_amax[j], 1e-5) is the calibration activation statistic (from
   w8a8_col_absmax over the calibration tokens) and w_j = max(max_i |W_ij|, 1e-5)
   runs over the stacked rows of EVERY matrix that consumes this input (gate and
   up for the FFN input; Wq, Wk and Wv for the attention input; the lm_head
   alone for its input).  Evaluated in binary64 and rounded once to float
   (square roots at alpha = 0.5).
   w: HOST array of n_w DEVICE pointers, matrix i row-major n_rows[i] x k of
   w_dtype (f32 or bf16); n_rows: HOST int64_t[n_w]; act_amax, delta: device
   float[k] (delta is written; it also serves as the scratch of the weight
   maximum, so it must not alias act_amax).  EUNSUPPORTED if alpha is outside
   [0, 1] or w_dtype is neither f32 nor bf16. */
w8a8_status w8a8_smooth_calibrate(const float* act_amax, const void* const* w,
                                  const int64_t* n_rows, int n_w, w8a8_dtype w_dtype, int64_t k,
                                  float alpha, float* delta, w8a8_stream_t stream);

/* The same factor from both statistics already gathered:
   delta[j] = max(act_amax[j], 1e-5)^alpha / max(w_amax[j], 1e-5)^(1 - alpha),
   with w_amax the running w8a8_col_absmax over every consumer's rows.  All three
   arrays are device float[k]; delta may alias w_amax.  EUNSUPPORTED if alpha is
   outside [0, 1]. */
w8a8_status w8a8_smooth_delta(const float* act_amax, const float* w_amax, int64_t k,
                              float alpha, float* delta, w8a8_stream_t stream);

/* ---------------------------------------------------------------- a2: weights */

/* Offline weight quantisation (Sec. 3 eq. si, what-ffn; Sec. 6 eq. what-lmhead):
   W_hat = W diag(delta) (delta NULL: W), s_w[i] = max_j |W_hat_ij| / 127,
   q_ij = clamp(rne(W_hat_ij / s_w[i]), -127, 127).
   w: n x k, f32 or bf16.  wq: w8a8_packed_bytes(n, k) bytes, fragment layout
   (padding written as zeros).  s_w: float[n]. */
w8a8_status w8a8_quantize_weights(const void* w, w8a8_dtype w_dtype, int64_t n, int64_t k,
                                  const float* delta, void* wq, float* s_w,
                                  w8a8_stream_t stream);

/* Copy the packed int8 layout back to a row-major int8 n x k matrix (checks). */
w8a8_status w8a8_unpack_weights(const void* wq, int64_t n, int64_t k, int8_t* q,
                                w8a8_stream_t stream);

/* Repack a bf16 n x k weight into the packed bf16 layout
   (w8a8_packed_bf16_bytes(n, k) bytes) for the bf16 path.  k % 8 == 0. */
w8a8_status w8a8_pack_bf16(const void* w, int64_t n, int64_t k, void* wp,
                           w8a8_stream_t stream);

/* ---------------------------------------------------------------- a3: activations */

/* Dynamic per-token quantisation (Sec. 6 eq. xhat-lmhead, stx, xint8):
   x_hat = x / delta (delta NULL: x), s_x[t] = max_j |x_hat_tj| / 127,
   q = clamp(rne(x_hat / s_x[t]), -127, 127).
   x: m x k, f32 or bf16.  qx: w8a8_packed_bytes(m, k) bytes in the fragment
   layout (zero padded).  s_x: float[m]. */
w8a8_status w8a8_quantize_act(const void* x, w8a8_dtype x_dtype, int64_t m, int64_t k,
                              const float* delta, void* qx, float* s_x,
                              w8a8_stream_t stream);

/* ---------------------------------------------------------------- a4, a5: INT8 GEMM */

/* The integer product of eq. gemm-final: acc[t][i] = sum_j qx[t][j] * wq[i][j]
   in int32, exact.  qx: packed m x k codes, wq: packed n x k codes, acc: int32
   m x n row-major.  Uses the same GEMM kernels as w8a8_linear with an identity
   epilogue.  ws: w8a8_linear_workspace_bytes(m, n, k) bytes. */
w8a8_status w8a8_gemm_i8_i32(const void* qx, int64_t m, const void* wq, int64_t n,
                             int64_t k, int32_t* acc, void* ws, size_t ws_bytes,
                             w8a8_stream_t stream);

/* W8A8 linear layer (Sec. 6): quantise x per token after x / delta, INT8 GEMM,
   dequantise y = (float(acc) * s_x[t]) * s_w[i] to y_dtype (f32 or bf16).
   x: m x k (f32 or bf16), y: m x n.  ws: w8a8_linear_workspace_bytes(m, n, k). */
w8a8_status w8a8_linear(const w8a8_linear_desc* desc, const void* x, w8a8_dtype x_dtype,
                        int64_t m, void* y, w8a8_dtype y_dtype, void* ws, size_t ws_bytes,
                        w8a8_stream_t stream);

/* ---------------------------------------------------------------- a6: FFN */

/* Gate/up stage of the INT8 FFN with the gated activation fused in its epilogue:
   g = dequant(qx . gate), u = dequant(qx . up) (binary32, never stored),
   h = bf16(gelu_tanh(g) * u), gelu_tanh(g) = 0.5 g (1 + tanh(sqrt(2/pi)(g + 0.044715 g^3))).
   qx: packed m x d codes, s_x: float[m], h: bf16 m x f row-major. */
w8a8_status w8a8_ffn_gate_up(const w8a8_ffn_desc* desc, const void* qx, const float* s_x,
                             int64_t m, void* h, w8a8_stream_t stream);

/* The stage between the FFN projections (Sec. 3, between Tab. 1 fused_fc and
   proj) from dequantised sums given in memory: h = bf16(gelu_tanh(g) * u) with
   the binary32 arithmetic of the gate/up epilogue above, then h / delta per
   token quantised as w8a8_quantize_act does (the requantisation of the down
   projection's input).  g, u: binary32 m x n row-major (n % 16 == 0); delta:
   float[n] or NULL; q: w8a8_packed_bytes(m, n) bytes, fragment layout (zero
   padded); s: float[m]; h: bf16 m x n row-major, written when not NULL (the
   stage's intermediate, for checks).  The production FFN computes the same h
   inside its gate/up GEMM and never stores g or u. */
w8a8_status w8a8_geglu_requant(const float* g, const float* u, int64_t m, int64_t n,
                               const float* delta, void* q, float* s, void* h,
                               w8a8_stream_t stream);

/* Whole INT8 FFN block (Sec. 3, Tab. 1 fused_fc + proj): quantise x / delta_gu,
   gate/up + GeGLU (above), requantise h / delta_down per token, down INT8 GEMM,
   dequantise to bf16.  x, y: bf16 m x d.  ws: w8a8_ffn_workspace_bytes(m, d, f). */
w8a8_status w8a8_ffn(const w8a8_ffn_desc* desc, const void* x, int64_t m, void* y,
                     void* ws, size_t ws_bytes, w8a8_stream_t stream);

/* For callers that cannot allocate (code under graph capture, tight serving
   loops, harnesses that forbid hipMalloc): w8a8_ffn without a workspace
   argument.  The intermediates live in a fixed device array inside the
   library, W8A8_FFN_NOALLOC_SCRATCH_BYTES (32 MiB) on every GPU it runs on,
   held until the process ends; the call itself allocates nothing.  Shapes
   whose w8a8_ffn_workspace_bytes(m, d, f) exceed it fail with EWORKSPACE
   (at d = 1152, f = 6912: m up to about 1000).  Every call on one GPU uses
   the same array: calls that overlap in time on one GPU (other streams,
   other threads) race and must be serialised by the caller.  The stream must
   belong to the current device.  Results equal w8a8_ffn's. */
#define W8A8_FFN_NOALLOC_SCRATCH_BYTES (32u << 20)
w8a8_status w8a8_ffn_noalloc(const w8a8_ffn_desc* desc, const void* x, int64_t m, void* y,
                             w8a8_stream_t stream);

/* ---------------------------------------------------------------- a7: lm_head */

/* INT8 lm_head (Sec. 6, eq. gemm-final, all 262144 rows in one launch): logits
   bf16 m x n from x bf16 m x k.  Tuned for m <= 64.
   ws: w8a8_lm_head_workspace_bytes(m, n, k). */
w8a8_status w8a8_lm_head(const w8a8_linear_desc* desc, const void* x, int64_t m,
                         void* logits, void* ws, size_t ws_bytes, w8a8_stream_t stream);

/* ---------------------------------------------------------------- FP8 variant */

/* FP8 in place of INT8 (Sec. 4, the list of further speed-ups; Sec. 8): the same
   SmoothQuant linear, FFN and lm_head with OCP FP8 E4M3 codes (1 sign, 4 exponent
   bits with bias 7, 3 mantissa bits, no infinities, largest finite 448) instead of
   int8.  The scales use the same symmetric reading with 448 in place of 127:
   s = max_j |v_j| / 448 (0 for an all-zero row) and code = E4M3(fl32(v / s)),
   rounded to nearest, ties to the even code; an all-zero row gives codes 0.
   Products of two E4M3 codes are exact in binary32 and the matrix cores sum them
   in binary32, so the sums differ from exact ones by rounding only.
   Codes use the packed int8 fragment layout byte for byte (one code per byte),
   so w8a8_packed_bytes sizes them and the descriptors above carry them unchanged.
   Every GEMM on this path needs its reduction length K to be a multiple of 128
   (EUNSUPPORTED otherwise): the FP8 matrix instruction reduces 128 codes at a
   time and the path does not pad K inside a 64-column fragment. */

size_t w8a8_fp8_linear_workspace_bytes(int64_t m, int64_t n, int64_t k);
size_t w8a8_fp8_ffn_workspace_bytes(int64_t m, int64_t d, int64_t f);

/* Offline FP8 weight quantisation: W_hat = W diag(delta) (delta NULL: W),
   s_w[i] = max_j |W_hat_ij| / 448, codes E4M3(W_hat_ij / s_w[i]).
   w: n x k, f32 or bf16; wq: w8a8_packed_bytes(n, k) bytes; s_w: float[n]. */
w8a8_status w8a8_fp8_quantize_weights(const void* w, w8a8_dtype w_dtype, int64_t n,
                                      int64_t k, const float* delta, void* wq, float* s_w,
                                      w8a8_stream_t stream);

/* Dynamic per-token FP8 quantisation of x / delta: s_x[t] = max_j |x_hat_tj| / 448,
   codes E4M3(x_hat / s_x[t]).  x: m x k, f32 or bf16; qx: w8a8_packed_bytes(m, k). */
w8a8_status w8a8_fp8_quantize_act(const void* x, w8a8_dtype x_dtype, int64_t m, int64_t k,
                                  const float* delta, void* qx, float* s_x,
                                  w8a8_stream_t stream);

/* Binary32 sums acc[t][i] = sum_j e(qx[t][j]) e(wq[i][j]) of decoded codes, the FP8
   analogue of w8a8_gemm_i8_i32 (identity epilogue, split-K partials added in
   binary32).  acc: float m x n row-major.  ws: w8a8_fp8_linear_workspace_bytes. */
w8a8_status w8a8_fp8_gemm_f32(const void* qx, int64_t m, const void* wq, int64_t n,
                              int64_t k, float* acc, void* ws, size_t ws_bytes,
                              w8a8_stream_t stream);

/* FP8 linear layer: as w8a8_linear with E4M3 codes; y = (acc * s_x[t]) * s_w[i].
   ws: w8a8_fp8_linear_workspace_bytes(m, n, k). */
w8a8_status w8a8_fp8_linear(const w8a8_linear_desc* desc, const void* x, w8a8_dtype x_dtype,
                            int64_t m, void* y, w8a8_dtype y_dtype, void* ws,
                            size_t ws_bytes, w8a8_stream_t stream);

/* Gate/up stage of the FP8 FFN with the gated activation fused in the epilogue
   (as w8a8_ffn_gate_up).  qx: E4M3 codes of m x d, packed; d % 128 == 0. */
w8a8_status w8a8_fp8_ffn_gate_up(const w8a8_ffn_desc* desc, const void* qx, const float* s_x,
                                 int64_t m, void* h, w8a8_stream_t stream);

/* Whole FP8 FFN block (as w8a8_ffn); d % 128 == 0 and f % 128 == 0.
   ws: w8a8_fp8_ffn_workspace_bytes(m, d, f). */
w8a8_status w8a8_fp8_ffn(const w8a8_ffn_desc* desc, const void* x, int64_t m, void* y,
                         void* ws, size_t ws_bytes, w8a8_stream_t stream);

/* FP8 lm_head: bf16 logits m x n from bf16 x m x k; k % 128 == 0.
   ws: w8a8_fp8_linear_workspace_bytes(m, n, k). */
w8a8_status w8a8_fp8_lm_head(const w8a8_linear_desc* desc, const void* x, int64_t m,
                             void* logits, void* ws, size_t ws_bytes, w8a8_stream_t stream);

/* ---------------------------------------------------------------- bf16 path */

/* bf16 projection y = bf16(x W^T), fp32 accumulation.  x: bf16 m x k
   (k % 32 == 0), wp: packed bf16 n x k, y: bf16 m x n.
   ws: w8a8_bf16_linear_workspace_bytes(m, n, k) bytes (may be 0, then ws may be NULL). */
w8a8_status w8a8_bf16_linear(const void* x, int64_t m, const void* wp, int64_t n,
                             int64_t k, void* y, void* ws, size_t ws_bytes,
                             w8a8_stream_t stream);

/* Gate/up stage of the bf16 FFN: h = bf16(gelu_tanh(g) * u), g and u the fp32
   accumulators of x W_gate^T and x W_up^T.  x: bf16 m x d, h: bf16 m x f.  Used
   for the bf16 layers and to gather the calibration statistic of the down
   projection's input (Sec. 6, eq. delta-lmhead applied to that input). */
w8a8_status w8a8_bf16_ffn_gate_up(const w8a8_bf16_ffn_desc* desc, const void* x, int64_t m,
                                  void* h, w8a8_stream_t stream);

/* bf16 FFN block: h = bf16(gelu_tanh(g) * u) with g, u the fp32 accumulators,
   y = bf16(h W_down^T).  ws: w8a8_bf16_ffn_workspace_bytes(m, d, f). */
w8a8_status w8a8_bf16_ffn(const w8a8_bf16_ffn_desc* desc, const void* x, int64_t m,
                          void* y, void* ws, size_t ws_bytes, w8a8_stream_t stream);

/* ---------------------------------------------------------------- a8, a9: stack */

/* RMSNorm with unit gain: y = bf16(x / sqrt(mean_j x_j^2 + 1e-6)), bf16 m x d;
   d % 8 == 0 and d <= 8192 (EUNSUPPORTED otherwise). */
w8a8_status w8a8_rmsnorm(const void* x, int64_t m, int64_t d, void* y,
                         w8a8_stream_t stream);

/* Post-FFN norm and residual: x_out = bf16(x + bf16(RMSNorm(f))), bf16 m x d.
   x_out may alias x. */
w8a8_status w8a8_rmsnorm_residual(const void* x, const void* f, int64_t m, int64_t d,
                                  void* x_out, w8a8_stream_t stream);

/* FFN layer subsets of Sec. 3 eq. ffn55 / ffn1010 / ffnall26 as a host array:
   prec[l] = 1 when layer l runs in INT8.  name: "bf16", "5+5", "10+10", "all26".
   Returns the number of INT8 layers, or -1 for an unknown name or n_layers < 26
   (the subsets index a 26-layer model). */
int w8a8_precision_map(const char* name, uint8_t* prec, int n_layers);

/* The FFN stack under a precision map (host prec[n_layers], 0 = bf16, 1 = INT8):
   for each layer x <- bf16(x + bf16(RMSNorm(FFN_l(bf16(RMSNorm(x)))))) (both norm
   outputs are bf16 activations, the residual sum is rounded again), FFN_l INT8 or
   bf16 by prec[l]; then the final RMSNorm (rounded to bf16) and the lm_head, INT8
   if lm_head_int8 != 0.
   x: bf16 m x d (not modified), logits: bf16 m x vocab.
   ws: w8a8_stack_workspace_bytes(m, d, f, vocab); calls that share a workspace
   must not overlap in time (the workspace holds the intermediates).
   At m == 1 every run of consecutive INT8 layers (up to 32 per launch) runs in
   one persistent launch with one workgroup per compute unit and device-wide
   barriers in device memory (Sec. 5, decode at batch 1); the results are
   identical to the per-layer launches.  It relies on all its workgroups being
   resident at once: the library checks that one fits per compute unit, and
   a barrier that is not reached within about a second (for instance because
   other work keeps compute units busy that long) ends the launch, leaves NaN
   in the token stream (so the logits, bf16 or INT8 lm_head, are NaN) and
   records the failure in the workspace, where w8a8_ffn_stack_status finds it.
   The call itself returns before the launch runs and cannot report it. */
w8a8_status w8a8_ffn_stack(const w8a8_stack_desc* desc, const uint8_t* prec,
                           int lm_head_int8, const void* x, int64_t m, void* logits,
                           void* ws, size_t ws_bytes, w8a8_stream_t stream);

/* Outcome of the last w8a8_ffn_stack / w8a8_ffn_stack_trace call enqueued on
   the workspace ws (every such call clears the record first): synchronises
   `stream`, then returns W8A8_OK, or W8A8_ETIMEOUT when a device-wide wait of
   the persistent decode kernel gave up in that call (its token stream and
   logits are then NaN).  ws, ws_bytes: the workspace that call used. */
w8a8_status w8a8_ffn_stack_status(const void* ws, size_t ws_bytes, w8a8_stream_t stream);

/* ---------------------------------------------------------------- sensitivity and map selection */

/* Signal-to-quantisation-noise ratio (Sec. 3 eq. sqnr-ffn; Sec. 5 eq. sqnr-block,
   the same ratio over a block's output): out[0] = sum ref^2, out[1] =
   sum (ref - test)^2, out[2] = 10 log10(out[0] / out[1]) in dB, all binary64
   (+inf when the two agree exactly, -inf for an all-zero ref, NaN for both).
   ref, test: n elements, f32 or bf16 (dtype); out: DEVICE double[3].
   Deterministic: fixed grid and fixed-order reductions.
   ws: w8a8_sqnr_workspace_bytes(n) bytes. */
size_t w8a8_sqnr_workspace_bytes(int64_t n);
w8a8_status w8a8_sqnr(const void* ref, const void* test, w8a8_dtype dtype, int64_t n,
                      double* out, void* ws, size_t ws_bytes, w8a8_stream_t stream);

/* w8a8_ffn_stack that also records the token stream after every layer:
   hidden = n_layers consecutive bf16 m x d matrices (hidden[l] after layer l).
   logits may be NULL (no lm_head; lm_head_int8 is then ignored).
   ws: w8a8_stack_workspace_bytes(m, d, f, vocab). */
w8a8_status w8a8_ffn_stack_trace(const w8a8_stack_desc* desc, const uint8_t* prec,
                                 int lm_head_int8, const void* x, int64_t m, void* logits,
                                 void* hidden, void* ws, size_t ws_bytes,
                                 w8a8_stream_t stream);

/* Layer sensitivity of the FFN stack (Sec. 3: SA-PTQ sensitivity by SQNR;
   Sec. 5 / Sec. 7: block-output SQNR).  Needs both forms of every layer in
   desc (int8_ffn and bf16_ffn).  With x (bf16 m x d, DEVICE) as input:
     isolated_db[l]   = SQNR of layer l's INT8 FFN block output against its bf16
                        FFN block output, both on layer l's input in the all-bf16
                        stack (RMSNorm of it);
     propagated_db[l] = SQNR of the token stream after layer l of the stack under
                        prec (HOST uint8[n_layers]) against the all-bf16 stack.
   Either output (HOST float[n_layers]) may be NULL (prec may then be NULL too).
   Synchronous: returns after the stream has finished.
   ws: w8a8_stack_sensitivity_workspace_bytes(m, d, f, vocab, n_layers). */
size_t w8a8_stack_sensitivity_workspace_bytes(int64_t m, int64_t d, int64_t f, int64_t vocab,
                                              int64_t n_layers);
w8a8_status w8a8_stack_sensitivity(const w8a8_stack_desc* desc, const uint8_t* prec,
                                   const void* x, int64_t m, float* isolated_db,
                                   float* propagated_db, void* ws, size_t ws_bytes,
                                   w8a8_stream_t stream);

/* Order of layers by isolated SQNR, most robust first (descending dB; NaN
   last; ties by layer index).  order: HOST int[n_layers].  Host-only; returns
   0, or -1 for NULL arguments or n_layers < 1. */
int w8a8_rank_layers(const float* isolated_db, int n_layers, int* order);

/* Automatic precision map (Sec. 2: the fastest configuration within a quality
   budget; Sec. 3: the most robust layers are quantised first).  Layers are
   visited in w8a8_rank_layers order of their isolated SQNR; each is set to INT8
   and kept there if the token stream after the last layer still has at least
   budget_db SQNR against the all-bf16 stack on x, else set back to bf16.
   prec: HOST uint8[n_layers] out; final_db (HOST float[1], may be NULL): the
   SQNR of the chosen map (+inf if no layer is INT8).  Every INT8 layer of this
   shape is faster than its bf16 form at prefill sizes, so more INT8 layers
   within the budget is faster.  Synchronous.
   ws: w8a8_stack_sensitivity_workspace_bytes(m, d, f, vocab, n_layers). */
w8a8_status w8a8_select_precision_map(const w8a8_stack_desc* desc, const void* x, int64_t m,
                                      float budget_db, uint8_t* prec, float* final_db,
                                      void* ws, size_t ws_bytes, w8a8_stream_t stream);

/* ---------------------------------------------------------------- f4: key/value cache, attention decode */

/* Sec. 4 lists an INT8 key/value cache among the further speed-ups, and Sec. 2
   gives the attention layout: four query heads share one key/value head of
   256 (grouped-query attention).  The cache of one layer is t_max rows of 256:
   either INT8 codes (row-major, 256 B a row) with one binary32 scale per row,
   or bf16 rows (512 B).  A row is quantised by the per-token rule of eq. stx /
   xint8 without smoothing: s = max_d |k_d| / 127, codes rne(k / s) clamped to
   [-127, 127] (an all-zero row stores s = 0 and zero codes), the same rule and
   results as w8a8_quantize_act with delta = NULL.  The caller owns the cache
   and every buffer below; the library keeps no state. */

/* Rows of 256 bf16 values (row r at kv + r * ld elements, ld >= 256 and a
   multiple of 8; e.g. the key part of a fused QKV projection output) ->
   codes[rows][256] and scales[rows] (kv and codes 16-byte aligned, scales
   4-byte aligned, so row slices of a cache can be filled).  EINVAL for NULL
   or unaligned pointers, rows < 1 or a bad ld. */
w8a8_status w8a8_kv_quantize(const void* kv, int64_t rows, int64_t ld, int8_t* codes,
                             float* scales, w8a8_stream_t stream);

/* Workspace of one attention decode call on a cache of t_max rows (any pos and
   window); 0 when one workgroup covers the rows. */
size_t w8a8_attn_decode_workspace_bytes(int64_t t_max);

/* One decode step of attention (Sec. 2 layout, Sec. 4 INT8 cache): qkv is the
   current token's projection output in bf16, [n_heads x 256 query | 256 key |
   256 value] (the fused QKV projection's row).  The key and value are
   quantised as above and stored at row pos of the cache, then every query
   head attends rows t0 .. pos, t0 = max(0, pos + 1 - window) (window = the
   context for the global layers, the sliding window for the others):
     out[h] = sum_t softmax_t(q_h . k_t / 16) v_t,   k_t = s_t * code (INT8 cache),
   scores and sums in binary32, out (n_heads x 256, bf16, the O projection's
   input) rounded once.  n_heads in {1, 2, 4, 8}; 0 <= pos < t_max; rows
   t0 .. pos - 1 must hold earlier tokens.  ws: w8a8_attn_decode_workspace_bytes
   (t_max) bytes (may be NULL when that is 0).  EUNSUPPORTED for other head
   counts, EINVAL for a bad pos, window or pointer, EWORKSPACE if ws is short.
   Two calls on one cache must be ordered (the second may read the first's
   row). */
w8a8_status w8a8_attn_decode(const void* qkv, int n_heads, int64_t pos, int64_t window,
                             int8_t* k_codes, float* k_scales, int8_t* v_codes, float* v_scales,
                             int64_t t_max, void* out, void* ws, size_t ws_bytes,
                             w8a8_stream_t stream);

/* The same step on a bf16 cache (k_rows, v_rows: bf16 [t_max][256]): the
   baseline the INT8 cache is measured against. */
w8a8_status w8a8_attn_decode_bf16(const void* qkv, int n_heads, int64_t pos, int64_t window,
                                  void* k_rows, void* v_rows, int64_t t_max, void* out, void* ws,
                                  size_t ws_bytes, w8a8_stream_t stream);

/* ---------------------------------------------------------------- planner overrides */

/* The GEMM planner picks tile shapes, K splits, streaming plans and the decode
   fusions by shape alone; the library never reads the environment.  For
   experiments and for the tests that check every plan gives the same results,
   these process-wide overrides replace a choice: "GLU_TILE", "GEMM_TILE",
   "GEMM_SPLITS", "DOWN_TILE", "DOWN_SPLITS", "DOWN_WK", "WIDE_NW", "WIDE_WGS",
   "STREAM_WK", "STREAM_SPLITS", "GROUP_M", "ROTATE", "NO_QLOAD",
   "NO_FUSED_GLUE", "NO_PERSISTENT", "DEC_SPIN_LIMIT", "XCD_M", "NT_OUT",
   "ATTN_WGS", "QROWS_R", "NO_STREAM", "NT_GLU", "NT_DOWN".
   Returns 0, or -1 for an unknown name.  Not for production use: an override applies to every later
   call in the process, and changing one while another thread calls the library
   races with it. */
int w8a8_set_plan_override(const char* name, int value);
void w8a8_clear_plan_overrides(void);

/* ---------------------------------------------------------------- errors */

/* Text of a status (any int: values outside w8a8_status give "unknown status"). */
const char* w8a8_status_str(int status);
/* Detail of the last error on the calling thread ("" if none). */
const char* w8a8_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* W8A8_H */
