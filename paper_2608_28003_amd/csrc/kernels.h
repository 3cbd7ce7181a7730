// Host-side launch functions of the gfx950 kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace w8a8 {

constexpr int kFragK8 = 64;   // int8 columns per 1 KiB fragment
constexpr int kFragK16 = 32;  // bf16 columns per 1 KiB fragment

enum Epi { EPI_I32 = 0, EPI_F32 = 1, EPI_BF16 = 2, EPI_GLU = 3 };

// Arguments of one GEMM launch C = A B^T.
struct GemmParams {
  const void* A;          // int8 path: packed codes (fragment layout); bf16 path: row-major bf16
  const void* B;          // packed weights (gate weights for the gated epilogue)
  const void* B2;         // packed up weights (gated epilogue only)
  int64_t lda;            // bf16 path: row stride of A in elements
  int M, N;               // logical rows of A and of B (output columns)
  int rb_a, rb_b;         // 16-row blocks stored in A and B
  int kb_count;           // fragment columns (Kp / 64 for int8, Kp / 32 for bf16)
  int kchunk;             // fragment columns per K split
  int splits;             // number of K splits (1: no split)
  const float* s_a;       // int8 path: per-token scales [M]
  const float* s_b;       // int8 path: per-channel scales [N] (gate)
  const float* s_b2;      // int8 path: per-channel scales [N] (up)
  void* out;              // int32 / f32 / bf16 output
  int64_t ldo;            // row stride of out in elements
  void* part;             // K-split partial sums: splits x M x N (int32 or f32)
  // Quantise-on-load (streaming kernel, int8 path, at most 16 rows): when
  // a_x is set, A is not read; every workgroup smooths and quantises the bf16
  // rows a_x itself (per-row absmax over all a_k columns, then its own K
  // range into LDS) and uses the resulting per-row scales in its epilogue.
  const uint16_t* a_x = nullptr;
  const float* a_delta = nullptr;  // may be null (no smoothing)
  int64_t a_ld = 0;                // row stride of a_x in elements
  int a_k = 0;                     // logical columns of a_x
  float* a_s_out = nullptr;        // optional: the per-row scales, written once
  // Fused layer glue (streaming kernel, int8, one token row, a_x null): the
  // row is the previous layer's output,  y = bf16(dequant(sum of g_splits
  // int32 partial sums)) or bf16(sum of fp32 partials),  x = bf16(g_x_in +
  // bf16(RMSNorm(y)))  (x = g_x_in without partials), written by workgroup 0
  // to g_x_out (and g_x_copy), then  a = bf16(RMSNorm(x))  is smoothed by
  // a_delta and quantised as with a_x (a_k = the row length).  The arithmetic
  // and reduction order are those of the glue kernel.
  const uint16_t* g_x_in = nullptr;
  uint16_t* g_x_out = nullptr;
  uint16_t* g_x_copy = nullptr;
  const void* g_part = nullptr;
  int g_splits = 0;
  int g_part_f32 = 0;
  const float* g_st = nullptr;     // int32 partials: token scale [1]
  const float* g_si = nullptr;     //                 column scales [a_k]
  // Tiled kernel walk order: tiles in bands of group_m M tiles (0: one band
  // of all M tiles); rotate: start each workgroup's K walk at a different step.
  int group_m = 0;
  int rotate = 1;
  // xcd_m: one-dimensional grid of m_tiles x n_tiles x splits workgroups,
  // M tiles dealt to the 8 XCDs (M tile mt on XCD mt % 8, with all its N tiles
  // and K splits), for products whose A panel outweighs B (set only when
  // m_tiles % 8 == 0).  nt_out: output stores marked non-temporal (outputs
  // far larger than the L2, e.g. the logits, so they do not evict the operands).
  int xcd_m = 0;
  int nt_out = 0;
};

// Operand / accumulator types of the GEMM kernels (the launchers take an int;
// false / true passed for the first two keep their meaning).
enum DType {
  DT_I8 = 0,    // int8 codes, int32 sums, two-scale dequant
  DT_BF16 = 1,  // row-major bf16 A, packed bf16 B, fp32 sums, no scales
  DT_F8 = 2,    // OCP E4M3 codes (packed like int8), fp32 sums, two-scale dequant
};

// tile shapes selectable at run time
enum TileCfg {
  TILE_128x128 = 0,     // 4 waves of 64 x 64
  TILE_128x64 = 1,      // 4 waves of 64 x 32
  TILE_64x64 = 2,       // 4 waves of 32 x 32
  TILE_256x128 = 3,     // 8 waves of 128 x 32
  TILE_GLU_128x32 = 4,  // gated: 4 waves of 32 x (32 gate + 32 up)
  TILE_GLU_64x64 = 5,   // gated: 4 waves of 32 x (32 + 32)
  TILE_GLU_128x64 = 6,  // gated: 4 waves of 64 x (32 + 32)
  TILE_256x256 = 7,     // 8 waves of 128 x 64
  TILE_GLU_256x128 = 8, // gated: 8 waves of 128 x (32 + 32)
  TILE_GLU_128x32_K2 = 9,  // as TILE_GLU_128x32 with two fragment columns per stage
  TILE_64x64_K2 = 10,      // as TILE_64x64, two fragment columns per stage
  TILE_128x128_K2 = 11,    // as TILE_128x128, two fragment columns per stage
  TILE_GLU_64x64_K2 = 12,  // as TILE_GLU_64x64, two fragment columns per stage
  TILE_GLU_256x64 = 13,    // gated: 4 waves of 128 x (32 + 32), 72 KiB LDS (2 per CU)
  TILE_GLU_256x64_K2_W8 = 14,  // gated: 8 waves of 64 x (32 + 32), two fragment columns
                               // per stage, 144 KiB LDS (1 per CU); FP8-capable
  TILE_GLU_128x32_K3 = 15,     // as TILE_GLU_128x32, three fragment columns per stage,
                               // four stages (1 per CU)
  TILE_64x64_K3 = 16,          // 8 waves of 32 x 16, three fragment columns per stage,
                               // four stages, 96 KiB of LDS (1 per CU)
  TILE_256x128_W4 = 17,        // 4 waves of 128 x 64, three stages, 72 KiB of LDS
                               // (2 per CU)
};

hipError_t launch_col_absmax(const void* x, bool bf16, int64_t rows, int64_t k, float* amax,
                             hipStream_t st);
// p[0 .. n) = v (a kernel, not a memset: callers may capture it in a graph)
hipError_t launch_fill_f32(float* p, int64_t n, float v, hipStream_t st);
hipError_t launch_smooth_delta(const float* a, const float* w, int64_t k, double alpha,
                               float* delta, hipStream_t st);
// rows per workgroup of the many-row bf16 quantiser: dflt unless overridden
int quant_rows_per_workgroup(int dflt);
hipError_t launch_quant_rows(const void* x, bool bf16, bool mul, int64_t rows, int64_t k,
                             const float* delta, int8_t* qpacked, float* s, hipStream_t st,
                             bool f8 = false);
// h = bf16(gelu_tanh(g) * u) of binary32 m x n rows g, u (h written if set),
// then the per-row quantisation of h / delta as launch_quant_rows.
hipError_t launch_geglu_requant(const float* g, const float* u, int64_t m, int64_t n,
                                const float* delta, int8_t* qpacked, float* s, uint16_t* h,
                                hipStream_t st);
hipError_t launch_unpack(const void* qp, int64_t n, int64_t k, int8_t* q, hipStream_t st);
hipError_t launch_pack_bf16(const void* w, int64_t n, int64_t k, void* wp, hipStream_t st);

// tiled MFMA GEMM (any M); `tile` picks the block shape
hipError_t launch_gemm_tile(int dt, int epi, int tile, const GemmParams& p, hipStream_t st);
// streaming MFMA GEMM for M <= 128: weights streamed from HBM, A staged in
// LDS; nw waves per workgroup, wk of them splitting one column block's K range
// Largest M * K / 16 a streaming workgroup of nw waves can quantise on load.
inline int64_t qload_capacity(int nw) { return (int64_t)64 * nw; }
// Fused layer glue: K splits of the previous layer it can add (loaded up front).
constexpr int kGlueMaxSplits = 4;
hipError_t launch_gemm_stream(int dt, int epi, int mb, int nw, int wk, const GemmParams& p,
                              int nb_per_block, hipStream_t st);
size_t gemm_stream_lds_bytes(int mb, int kchunk, int wk, bool glu);
// sum of K-split partials (in split order) followed by the epilogue
hipError_t launch_splitk_reduce(int dt, int epi, const GemmParams& p, hipStream_t st);

hipError_t launch_rmsnorm(const uint16_t* x, const uint16_t* f, int64_t m, int64_t d,
                          uint16_t* y, hipStream_t st);

// Row glue between FFN blocks of the stack (one launch per layer boundary):
// FFN output from split-K partial sums -> post-norm residual update of the
// token stream -> pre-norm of the next consumer, as bf16 and/or INT8 codes.
struct GlueParams {
  int64_t m = 0, d = 0;
  int64_t rows_pad = 0, kp = 0;        // packed code shape (q only)
  const uint16_t* x_in = nullptr;      // token stream in, bf16 m x d
  uint16_t* x_out = nullptr;           // token stream out (may alias x_in)
  const void* part = nullptr;          // splits x m x d partial sums, or null
  int splits = 1;
  bool part_f32 = false;               // fp32 partials (bf16 layer) or int32 (INT8 layer)
  const float* s_t = nullptr;          // int32 partials: per-token scale
  const float* s_i = nullptr;          //                 per-column scale
  uint16_t* a = nullptr;               // pre-norm output, bf16 m x d (optional)
  const float* delta = nullptr;        // smoothing of the INT8 consumer (may be null)
  int8_t* q = nullptr;                 // packed codes of the pre-norm output (optional)
  float* s = nullptr;                  // their per-row scales
  uint16_t* x_copy = nullptr;          // second copy of the token stream out (optional)
};
hipError_t launch_glue(const GlueParams& g, hipStream_t st);

// Persistent decode kernel (one token, a run of consecutive INT8 FFN blocks of
// the stack in one launch; one workgroup per CU, grid-wide barriers between
// the gate/up and down phases of every layer).
constexpr int kDecMaxLayers = 32;  // layers per launch
constexpr int kDecMaxFrags = 10;   // weight fragments a wave holds per phase
constexpr int kDecMaxPanel = 64;   // activation fragments staged in LDS
constexpr int kDecGroups = 4;      // barrier arrival groups (one counter each)
struct DecCtl {                    // 256-byte lines
  unsigned top[64];                // group completions (word 0)     } cleared before
  unsigned grp[kDecGroups][64];    // arrivals per group (word 0)    } every launch
  unsigned err[64];                // word 0 nonzero: a wait of this launch gave up
  unsigned fail[64];               // word 0 nonzero: a wait gave up in some launch since
                                   // the last launch_dec_status_clear (the run's outputs
                                   // are NaN); read by w8a8_ffn_stack_status
};
struct DecLayer {
  const void* wg;      // packed gate weights (f x d)
  const void* wu;      // packed up weights
  const float* sg;     // their per-channel scales [f]
  const float* su;
  const float* dgu;    // smoothing of the gate/up input [d] (may be null)
  const void* wd;      // packed down weights (d x f)
  const float* sd;     // their per-channel scales [d]
  const float* dd;     // smoothing of the down input [f] (may be null)
};
// Per-layer exchange buffers of the persistent kernel (all inside `scratch`,
// layer j at j * layer_bytes): the token stream x (bf16 [d]), the down
// projection's partial sums (int32, plane z, column block c at
// (z * ncd + c) * 32), the token scale of the down input (float) and the FFN
// intermediate h (bf16, 16-column item i at i * 64).  Every 128-byte line is
// written by one workgroup and read only after the barrier that follows.
struct DecLayout {
  size_t part, sh, h, layer_bytes;
};
DecLayout decode_layout(int64_t d, int64_t f, int splits);
struct DecParams {
  DecLayer L[kDecMaxLayers];
  int n_layers = 0;
  int l0 = 0;                      // stack index of L[0]
  int d = 0, f = 0;
  // the first layer's glue input: the token stream, and the previous layer's
  // K-split partial sums in planes of d (none: part_in null, splits_in 0)
  const uint16_t* x_in = nullptr;
  const void* part_in = nullptr;
  int splits_in = 0;
  int part_f32_in = 0;
  const float* st_in = nullptr;    // int32 partials: token scale [1]
  const float* si_in = nullptr;    //                 column scales [d]
  // the run's results for the launches that follow: the token stream after
  // the next-to-last layer, the last layer's partial sums (planes of d) and
  // the token scale of its down input
  uint16_t* x_out = nullptr;
  int32_t* part = nullptr;
  float* sh = nullptr;
  uint16_t* hidden = nullptr;      // optional: token stream after stack layer i at hidden + i d
  char* scratch = nullptr;         // n_layers x layout.layer_bytes
  DecLayout layout{};
  int splits = 0;                  // = decode_splits(d, f, grid)
  DecCtl* ctl = nullptr;
  int spin_limit = 1 << 20;        // polls per barrier before giving up
};
// Workgroups of the persistent kernel on `device` (one per CU), or 0 when a
// workgroup per CU cannot be resident.
int decode_grid(int device);
// K splits of the down projection for this shape and grid, or 0 when the
// shape does not fit the kernel.
int decode_splits(int64_t d, int64_t f, int grid);
hipError_t launch_decode_ffn(const DecParams& P, int grid, hipStream_t st);
// Clears ctl->fail (start of every stack call).
hipError_t launch_dec_status_clear(DecCtl* ctl, hipStream_t st);

// SQNR of test against ref over n elements (bf16 or f32): part holds
// 2 * sqnr_groups(n) doubles of scratch, out receives {sum ref^2,
// sum (ref - test)^2, 10 log10 of their ratio}.
constexpr int kSqnrMaxGroups = 1024;
int sqnr_groups(int64_t n);
hipError_t launch_sqnr(const void* ref, const void* test, bool bf16, int64_t n, double* part,
                       double* out, hipStream_t st);

// ------------------------------------------------------------------ attention decode (attn.hip)

// One token's query heads against a key/value cache of rows of 256 (INT8
// codes with per-row scales, or bf16), the new row appended at pos.
struct AttnParams {
  const uint16_t* qkv = nullptr;  // [n_heads x 256 query | 256 key | 256 value] bf16
  void* k = nullptr;              // cache rows: int8 [t_max][256] or bf16 [t_max][256]
  void* v = nullptr;
  float* sk = nullptr;            // INT8 cache: per-row scales
  float* sv = nullptr;
  int64_t pos = 0;                // row of the new token
  int64_t t0 = 0;                 // first attended row (pos + 1 - window, at least 0)
  int rows_per_wg = 0;            // set by the launcher
  int n_wg = 0;
  float* part = nullptr;          // workspace: per-workgroup partial results
  uint16_t* out = nullptr;        // n_heads x 256 bf16
};
// rows of 256 bf16 (stride ld elements) -> row-major INT8 codes and row scales
hipError_t launch_kv_quant(const uint16_t* src, int64_t rows, int64_t ld, int8_t* codes,
                           float* scales, hipStream_t st);
// target: workgroups to split the rows over (at most kAttnWgTarget)
constexpr int kAttnWgTarget = 1024;
hipError_t launch_attn_decode(AttnParams p, int nh, bool i8, int target, hipStream_t st);
size_t attn_ws_bytes(int64_t rows, int target);  // workspace of one launch over `rows` rows
size_t attn_ws_bytes_max(int64_t t_max);  // ... of any launch over at most t_max rows

}  // namespace w8a8
