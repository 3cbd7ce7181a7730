// Host side of the C ABI declared in include/w8a8.h: argument validation (done
// before any HIP call), the GEMM planner, workspace carving and the pipelines
// (linear, FFN block, lm_head, bf16 path, precision-map stack).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <climits>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>
#include <cmath>

#include "../../include/w8a8.h"
#include "kernels.h"

using namespace w8a8;

namespace {

thread_local std::string g_last_error;

w8a8_status fail(w8a8_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

w8a8_status hip_check(hipError_t e, const char* what) {
  if (e == hipSuccess) return W8A8_OK;
  return fail(W8A8_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }
inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

hipStream_t S(w8a8_stream_t s) { return reinterpret_cast<hipStream_t>(s); }

// ------------------------------------------------------------------ planner

struct Plan {
  int dt = DT_I8;       // operand type the plan was made for
  bool stream = false;  // streaming kernel (M <= 128) or tiled kernel
  int tile = TILE_128x128;
  int mb = 1;           // streaming: 16-row blocks of A
  int nw = 1, wk = 1;   // streaming: waves per workgroup, waves splitting K
  int splits = 1;
  int kchunk = 0;
  int nbpb = 1;         // streaming: column blocks per workgroup
  bool xcd_m = false;   // tiled: M tiles dealt to XCDs (A outweighs B)
  bool nt_out = false;  // tiled: non-temporal output stores (very wide outputs)
};

void tile_shape(int tile, int* bm, int* bn);
int plan_override(const char* name, int dflt);

// Walk order and store policy of a tiled plan: when A (m x k) outweighs the
// weights (n x k) and the M tiles split evenly over the 8 XCDs, each XCD
// takes whole rows of tiles so its L2 holds its rows of A once (the down
// projection at M = 2048 re-fetched its 14 MB A panel for every column tile
// spread over the XCDs: 135 MB per launch); outputs of 64K columns and more
// (the lm_head's logits) are stored non-temporally, so they do not evict A
// (the override NT_OUT sets the store policy of every tiled plan).
void plan_order(Plan& p, int64_t m, int64_t n) {
  if (p.stream) return;
  int bm = 0, bn = 0;
  tile_shape(p.tile, &bm, &bn);
  p.xcd_m = m > n && ceil_div(m, bm) % 8 == 0 && plan_override("XCD_M", 1) != 0;
  const int nt = plan_override("NT_OUT", -1);
  p.nt_out = nt >= 0 ? nt != 0 : n >= 65536;
}

// Planner overrides (w8a8_set_plan_override): experiments and the tests that
// check that every plan gives the same results set them explicitly; the
// library never reads the environment.  Unset entries hold kUnset.
constexpr int kUnset = INT32_MIN;
const char* const kOverrideNames[] = {
    "GLU_TILE", "GEMM_TILE", "GEMM_SPLITS", "DOWN_TILE", "DOWN_SPLITS", "DOWN_WK",
    "WIDE_NW", "WIDE_WGS", "STREAM_WK", "STREAM_SPLITS", "GROUP_M", "ROTATE",
    "NO_QLOAD", "NO_FUSED_GLUE", "NO_PERSISTENT", "DEC_SPIN_LIMIT", "XCD_M", "NT_OUT",
    "ATTN_WGS", "QROWS_R", "NO_STREAM", "NT_GLU", "NT_DOWN"};
constexpr int kNumOverrides = (int)(sizeof(kOverrideNames) / sizeof(kOverrideNames[0]));
std::atomic<int> g_override[kNumOverrides];
struct OverrideInit {
  OverrideInit() {
    for (auto& o : g_override) o.store(kUnset);
  }
} g_override_init;

int override_index(const char* name) {
  for (int i = 0; i < kNumOverrides; ++i)
    if (std::strcmp(name, kOverrideNames[i]) == 0) return i;
  return -1;
}

// The override named `name` (one of kOverrideNames), else dflt.
int plan_override(const char* name, int dflt) {
  const int i = override_index(name);
  const int v = i < 0 ? kUnset : g_override[i].load(std::memory_order_relaxed);
  return v == kUnset ? dflt : v;
}

void tile_shape(int tile, int* bm, int* bn) {
  switch (tile) {
    case TILE_128x128: *bm = 128; *bn = 128; break;
    case TILE_128x64: *bm = 128; *bn = 64; break;
    case TILE_64x64: *bm = 64; *bn = 64; break;
    case TILE_256x128: *bm = 256; *bn = 128; break;
    case TILE_GLU_128x32: *bm = 128; *bn = 32; break;
    case TILE_GLU_64x64: *bm = 64; *bn = 64; break;
    case TILE_GLU_128x64: *bm = 128; *bn = 64; break;
    case TILE_256x256: *bm = 256; *bn = 256; break;
    case TILE_GLU_256x128: *bm = 256; *bn = 128; break;
    case TILE_GLU_128x32_K2: *bm = 128; *bn = 32; break;
    case TILE_64x64_K2: *bm = 64; *bn = 64; break;
    case TILE_128x128_K2: *bm = 128; *bn = 128; break;
    case TILE_GLU_64x64_K2: *bm = 64; *bn = 64; break;
    case TILE_GLU_256x64: *bm = 256; *bn = 64; break;
    case TILE_GLU_256x64_K2_W8: *bm = 256; *bn = 64; break;
    case TILE_GLU_128x32_K3: *bm = 128; *bn = 32; break;
    case TILE_64x64_K3: *bm = 64; *bn = 64; break;
    case TILE_256x128_W4: *bm = 256; *bn = 128; break;
    default: *bm = 128; *bn = 128;
  }
}

int64_t tiles_of(int tile, int64_t m, int64_t n) {
  int bm, bn;
  tile_shape(tile, &bm, &bn);
  return ceil_div(m, bm) * ceil_div(n, bn);
}

// Streaming plan for M <= 128, or false if the A panel cannot fit in LDS.
bool plan_stream(Plan& p, int64_t m, int64_t n, int64_t kb, bool glu, bool f8) {
  const int64_t kstep = f8 ? 2 : 1;  // FP8: K chunks of whole 128-deep MFMA steps
  const int64_t nbc = ceil_div(n, 16);
  const int64_t lds_kb = 158;  // dynamic LDS per workgroup, KiB (one fragment = 1 KiB); the
                               // kernel's static LDS (scales, reduction scratch) takes the rest
  p.mb = m <= 16 ? 1 : (m <= 32 ? 2 : (m <= 64 ? 4 : 8));
  auto lds = [&](int64_t kchunk, int wk) { return p.mb * kchunk + (wk - 1) * (glu ? 2 : 1) * p.mb; };
  if (glu) {  // gate/up pair: no K split across workgroups (the epilogue needs full sums)
    for (int wk : {4, 2, 1}) {
      if (wk == 4 && p.mb > 4) continue;  // 4-wave K split spills at MB = 8
      if (lds(kb, wk) <= lds_kb) {
        p.nw = p.wk = wk;
        p.splits = 1;
        p.kchunk = (int)kb;
        p.nbpb = 1;
        return true;
      }
    }
    return false;
  }
  if (nbc >= 1024) {  // wide output (lm_head): every wave owns its column blocks
    if (p.mb * kb > 144) return false;
    p.wk = 1;
    p.nw = plan_override("WIDE_NW", 4);
    p.splits = 1;
    p.kchunk = (int)kb;
    // measured on the lm_head (V = 262144): 32 rows 82.7 -> 78.2 us with
    // 2048 workgroups instead of 512; one row block: 1024 and 2048 alike
    const int64_t wgs = plan_override("WIDE_WGS", p.mb == 1 ? 1024 : 2048);
    p.nbpb = p.nw == 1 ? (int)std::max<int64_t>(1, ceil_div(nbc, wgs))
                       : (int)round_up(std::max<int64_t>(4, ceil_div(nbc, wgs)), 4);
    return true;
  }
  // narrow output, long K (down projection): waves of a workgroup split one
  // column block's K range; pick the split with the most work per wave among
  // those that keep >= 768 waves busy
  bool found = false;
  int64_t best_pw = -1, best_waves = -1;
  const int force_wk = plan_override("STREAM_WK", 0);
  const int64_t min_splits = plan_override("STREAM_SPLITS", 1);
  for (int wk : {16, 4, 2}) {
    if (wk == 16 && p.mb > 1) continue;  // 16-wave workgroups only for MB = 1
    if (force_wk && wk != force_wk) continue;
    int64_t max_kc = (lds_kb - (wk - 1) * p.mb) / p.mb;
    if (max_kc < wk) continue;
    int64_t splits = std::max(min_splits, ceil_div(kb, max_kc / kstep * kstep));
    int64_t kchunk = round_up(ceil_div(kb, splits), kstep);
    splits = ceil_div(kb, kchunk);
    int64_t pw = ceil_div(kchunk, wk), waves = nbc * splits * wk;
    // splits that leave a wave fewer than 4 fragments lose to the cross-wave
    // reduction they add (measured: QKV 1152 -> 1536 at M = 1, 16 waves
    // 6.85 us, 4 waves 5.33 us)
    const bool fed = pw >= 4, best_fed = best_pw >= 4;
    bool better;
    if (!found) better = true;
    else if (fed != best_fed) better = fed;
    else if ((waves >= 768) != (best_waves >= 768)) better = waves >= 768;
    else if (waves >= 768) better = pw > best_pw;
    else better = waves > best_waves;
    if (better) {
      found = true;
      best_pw = pw;
      best_waves = waves;
      p.nw = p.wk = wk;
      p.splits = (int)splits;
      p.kchunk = (int)kchunk;
      p.nbpb = 1;
    }
  }
  return found;
}

// Deterministic in (m, n, k, path); the workspace queries use the same plan.
// Planner overrides for the tiled path: GEMM_TILE / GEMM_SPLITS (plain
// epilogues) and GLU_TILE (gated epilogue).
Plan plan_gemm(int64_t m, int64_t n, int64_t k, int dt, bool glu) {
  Plan p;
  p.dt = dt;
  const bool f8 = dt == DT_F8;
  const int64_t kb = dt == DT_BF16 ? ceil_div(k, kFragK16) : ceil_div(k, kFragK8);
  // The streaming kernel wins while the weights dominate the traffic, up to
  // 32 rows; the tiled kernel reuses operands better beyond that (measured on
  // the lm_head at 64 rows: 95.8 us streaming with 4 row blocks in LDS,
  // 84.2 us on two-column 64 x 64 tiles).
  if (m <= 32 && !plan_override("NO_STREAM", 0) && plan_stream(p, m, n, kb, glu, f8)) {
    p.stream = true;
    return p;
  }
  p = Plan();
  p.dt = dt;
  if (f8) {  // FP8 stages hold whole 128-deep MFMA steps: two-column tiles only
    if (glu)  // measured: the 8-wave 256 x 64 tile from M = 512 (216 tiles) on
      p.tile = m <= 128 ? TILE_GLU_128x32_K2
                        : (tiles_of(TILE_GLU_256x64_K2_W8, m, n) >= 128 ? TILE_GLU_256x64_K2_W8
                                                                       : TILE_GLU_64x64_K2);
    else
      p.tile = tiles_of(TILE_128x128_K2, m, n) >= 256 ? TILE_128x128_K2 : TILE_64x64_K2;
    const int want = glu ? plan_override("GLU_TILE", p.tile) : plan_override("GEMM_TILE", p.tile);
    if (glu ? (want == TILE_GLU_128x32_K2 || want == TILE_GLU_64x64_K2 ||
               want == TILE_GLU_256x64_K2_W8)
            : (want == TILE_64x64_K2 || want == TILE_128x128_K2))
      p.tile = want;
    const int64_t tiles = tiles_of(p.tile, m, n);
    int64_t splits = 1;
    if (!glu && tiles < 200)
      splits = std::min<int64_t>(ceil_div(256, tiles), std::max<int64_t>(1, kb / 8));
    splits = plan_override("GEMM_SPLITS", (int)splits);
    if (glu || splits < 1) splits = 1;
    p.kchunk = (int)round_up(ceil_div(kb, splits), 2);
    p.splits = (int)ceil_div(kb, p.kchunk);
    plan_order(p, m, n);
    if (glu && plan_override("NT_OUT", -1) < 0)  // as the int8 gated plans below
      p.nt_out = plan_override("NT_GLU", m * n * 2 >= (2 << 20) ? 1 : 0) != 0;
    return p;
  }
  // int8 and bf16 choices from sweeps of the FFN shapes (d = 1152, f = 6912)
  // and the lm_head (N = 262144) at M = 64 ... 2048
  const bool i8 = dt == DT_I8;
  const bool long_k = i8 && !glu && k >= 4096 && n <= 4096;  // down-projection-like
  // bf16 (FFN shapes d = 1152, f = 6912; the FFN block, gate/up then down):
  // the 8-wave 256 x 128 gated tile from ~200 tiles (M = 2048 242 -> 208 us,
  // M = 1024 134 -> 119 us), the 128 x 64 gated tile from 200 tiles (M = 256
  // 54.4 -> 50.0 us); the long-K down projection on 256 x 128 or 128 x 128
  // tiles with three K splits from 64 tiles (M = 2048 242 -> 178 us, M = 1024
  // 134 -> 103 us), as the int8 stack's down projection
  const bool long_k16 = dt == DT_BF16 && !glu && k >= 4096 && n <= 4096;
  int dflt_splits = 0;
  if (glu) {
    if (m <= 128)  // int8: three fragment columns a stage (M = 128: 9.95 -> 9.01 us)
      p.tile = i8 ? TILE_GLU_128x32_K3 : TILE_GLU_128x32_K2;
    else if (!i8 && tiles_of(TILE_GLU_256x128, m, n) >= 200)
      p.tile = TILE_GLU_256x128;
    else if (tiles_of(TILE_GLU_256x64, m, n) >= (i8 ? 384 : 512))  // two resident per CU
      p.tile = TILE_GLU_256x64;
    else if (i8)
      p.tile = tiles_of(TILE_GLU_128x64, m, n) >= 400 ? TILE_GLU_128x64 : TILE_GLU_64x64_K2;
    else
      p.tile = tiles_of(TILE_GLU_128x64, m, n) >= 200 ? TILE_GLU_128x64 : TILE_GLU_64x64;
  } else if (long_k16 && tiles_of(TILE_256x128, m, n) >= 64) {
    p.tile = TILE_256x128;
    dflt_splits = 3;
  } else if (long_k16 && tiles_of(TILE_128x128, m, n) >= 64) {
    p.tile = TILE_128x128;
    dflt_splits = 3;
  } else if (long_k) {
    // with K split until ~512 workgroups are in flight (the split rule below);
    // when the whole grid fits one workgroup per CU (the FFN down projection
    // up to M = 128: 216 workgroups) 8 waves and stages of three fragment
    // columns (26-layer stack at M = 128: 892 -> 844 us with 4 waves, 0.836 ->
    // 0.825 ms with 8)
    const int64_t t64 = tiles_of(TILE_64x64, m, n);
    const int64_t sp = std::min<int64_t>(std::min<int64_t>(ceil_div(512, t64), 6),
                                         std::max<int64_t>(1, kb / 8));
    p.tile = t64 * sp <= 256 ? TILE_64x64_K3 : TILE_64x64_K2;
  } else {
    // measured on the lm_head (N = 262144): 256 x 256 from M = 256 (133.7 vs
    // 162.4 us at M = 256, 888 vs 924 us at M = 2048), 128 x 128 below; from
    // M = 512 and ~400 tiles the 4-wave 256 x 128 tile, two per CU (lm_head
    // M = 2048 856 -> 827 us, M = 512 242 -> 237 us; N = 13824 at M = 1024
    // 47.5 -> 40.9 us; N = 6912 at M = 2048 50.4 -> 42.9 us; with fewer tiles
    // it loses: N = 6912 at M = 1024 36.9 vs 33.2 us)
    if (i8 && m >= 512 && tiles_of(TILE_256x128_W4, m, n) >= 400)
      p.tile = TILE_256x128_W4;
    else if (m >= 256 && tiles_of(TILE_256x256, m, n) >= 512)  // bf16 lm_head: M = 2048
      p.tile = TILE_256x256;  // 1904 -> 1419 us, M = 512 491 -> 362 us (torch 1422 / 308)
    else if (i8 && m <= 64 && kb % 2 == 0 && tiles_of(TILE_64x64, m, n) >= 1024)
      p.tile = TILE_64x64_K2;  // very wide outputs at up to 64 rows (lm_head)
    else if (tiles_of(TILE_128x128, m, n) >= 256)
      p.tile = TILE_128x128;
    else if (tiles_of(TILE_128x64, m, n) >= 256)
      p.tile = TILE_128x64;
    else  // measured on the attention projections at M = 64 ... 256: the
          // two-column stage is faster when K allows it
      p.tile = (i8 && kb % 2 == 0) ? TILE_64x64_K2 : TILE_64x64;
  }
  p.tile = glu ? plan_override("GLU_TILE", p.tile) : plan_override("GEMM_TILE", p.tile);
  const int64_t tiles = tiles_of(p.tile, m, n);
  int splits = 1;
  if (dflt_splits > 0)
    splits = dflt_splits;
  else if (long_k)
    splits = (int)std::min<int64_t>(std::min<int64_t>(ceil_div(512, tiles), 6),
                                    std::max<int64_t>(1, kb / 8));
  else if (!glu && tiles < 200)  // int8: at least 16 fragments per split (a split of a
                                 // 1152-deep K costs more than the parallelism it adds)
    splits = (int)std::min<int64_t>(ceil_div(256, tiles), std::max<int64_t>(1, kb / (i8 ? 16 : 4)));
  splits = plan_override("GEMM_SPLITS", splits);
  if (glu || splits < 1) splits = 1;
  p.kchunk = (int)ceil_div(kb, splits);
  p.splits = (int)ceil_div(kb, p.kchunk);
  plan_order(p, m, n);
  // the gated output h streams past the caches too, so its operand panels stay
  // in L2 (f = 6912: gate/up at M = 2048 44.6 -> 42.6 us, M = 1024 24.5 ->
  // 23.0 us, M = 512 16.6 -> 16.0 us; M = 128 unchanged)
  if (glu && plan_override("NT_OUT", -1) < 0)
    p.nt_out = plan_override("NT_GLU", m * n * 2 >= (2 << 20) ? 1 : 0) != 0;
  return p;
}

size_t plan_ws_bytes(const Plan& p, int64_t m, int64_t n) {
  if (p.splits <= 1) return 0;
  return align256((size_t)p.splits * m * n * 4);
}

// Run one GEMM with a plan.  A: packed codes (int8) or row-major bf16;
// B (and B2 for the gated epilogue): packed weights.  A K-split plan writes
// partial sums to gemm_ws and a second launch reduces them into `out`.
// Quantise-on-load source of a GEMM's A operand (bf16 rows), see GemmParams.
struct QLoad {
  const uint16_t* x = nullptr;
  const float* delta = nullptr;
  float* s_out = nullptr;  // where to leave the per-row scales (optional)
  // fused layer glue instead of x (one token row): see GemmParams::g_*
  const uint16_t* g_x_in = nullptr;
  uint16_t* g_x_out = nullptr;
  uint16_t* g_x_copy = nullptr;
  const void* g_part = nullptr;
  int g_splits = 0;
  bool g_part_f32 = false;
  const float* g_st = nullptr;
  const float* g_si = nullptr;
};

// Streaming int8 / E4M3 plans over at most 16 rows quantise their bf16 input
// themselves; every other plan reads codes produced by quant_rows_kernel.
bool plan_qloads(const Plan& pl, int64_t m, int64_t k) {
  if (plan_override("NO_QLOAD", 0) || (pl.dt != DT_I8 && pl.dt != DT_F8)) return false;
  return pl.stream && pl.mb == 1 && m * (k / 16) <= qload_capacity(pl.nw);
}

w8a8_status run_gemm(const Plan& pl, int dt, int epi, const void* A, int64_t lda, int64_t m,
                     const void* B, const void* B2, int64_t n, int64_t k, const float* s_a,
                     const float* s_b, const float* s_b2, void* out, int64_t ldo, void* gemm_ws,
                     hipStream_t st, QLoad ql = QLoad()) {
  GemmParams p{};
  p.a_x = ql.x;
  p.a_delta = ql.delta;
  p.a_ld = k;
  p.a_k = (int)k;
  p.a_s_out = ql.s_out;
  p.g_x_in = ql.g_x_in;
  p.g_x_out = ql.g_x_out;
  p.g_x_copy = ql.g_x_copy;
  p.g_part = ql.g_part;
  p.g_splits = ql.g_splits;
  p.g_part_f32 = ql.g_part_f32 ? 1 : 0;
  p.g_st = ql.g_st;
  p.g_si = ql.g_si;
  p.A = A;
  p.B = B;
  p.B2 = B2;
  p.lda = lda;
  p.M = (int)m;
  p.N = (int)n;
  p.rb_a = (int)ceil_div(m, 16);
  p.rb_b = (int)ceil_div(n, 16);
  p.kb_count = (int)(dt == DT_BF16 ? ceil_div(k, kFragK16) : ceil_div(k, kFragK8));
  p.kchunk = pl.kchunk;
  p.splits = pl.splits;
  p.s_a = s_a;
  if (ql.x || ql.g_x_in) {
    // quantise-on-load: the token scales exist only inside the GEMM, which
    // leaves them at s_out; a split-K reduction dequantises from there
    if (pl.splits > 1 && !ql.s_out)
      return fail(W8A8_EINVAL, "internal: quantise-on-load with split-K needs a scale buffer");
    p.s_a = ql.s_out;
  }
  p.s_b = s_b;
  p.s_b2 = s_b2;
  p.out = out;
  p.ldo = ldo;
  p.part = pl.splits > 1 ? gemm_ws : nullptr;
  p.group_m = plan_override("GROUP_M", 0);
  p.rotate = plan_override("ROTATE", 1);
  p.xcd_m = pl.xcd_m ? 1 : 0;
  p.nt_out = pl.nt_out ? 1 : 0;
  hipError_t e = pl.stream ? launch_gemm_stream(dt, epi, pl.mb, pl.nw, pl.wk, p, pl.nbpb, st)
                           : launch_gemm_tile(dt, epi, pl.tile, p, st);
  w8a8_status s = hip_check(e, pl.stream ? "gemm_stream" : "gemm_tile");
  if (s != W8A8_OK || pl.splits <= 1) return s;
  return hip_check(launch_splitk_reduce(dt, epi, p, st), "splitk_reduce");
}

// The same GEMM without any reduction or dequantisation: raw sums (int32 for
// INT8 operands, fp32 for bf16 and FP8) in the plan's split-K layout
// part[split][m][n] (one split: a plain m x n matrix), for a consumer that
// reduces them itself.
w8a8_status run_gemm_raw(const Plan& pl, int dt, const void* A, int64_t lda, int64_t m,
                         const void* B, int64_t n, int64_t k, void* part, hipStream_t st,
                         QLoad ql = QLoad()) {
  GemmParams p{};
  p.a_x = ql.x;
  p.a_delta = ql.delta;
  p.a_ld = k;
  p.a_k = (int)k;
  p.a_s_out = ql.s_out;
  p.g_x_in = ql.g_x_in;
  p.g_x_out = ql.g_x_out;
  p.g_x_copy = ql.g_x_copy;
  p.g_part = ql.g_part;
  p.g_splits = ql.g_splits;
  p.g_part_f32 = ql.g_part_f32 ? 1 : 0;
  p.g_st = ql.g_st;
  p.g_si = ql.g_si;
  p.A = A;
  p.B = B;
  p.lda = lda;
  p.M = (int)m;
  p.N = (int)n;
  p.rb_a = (int)ceil_div(m, 16);
  p.rb_b = (int)ceil_div(n, 16);
  p.kb_count = (int)(dt == DT_BF16 ? ceil_div(k, kFragK16) : ceil_div(k, kFragK8));
  p.kchunk = pl.kchunk;
  p.splits = pl.splits;
  p.out = part;
  p.ldo = n;
  p.part = pl.splits > 1 ? part : nullptr;
  p.group_m = plan_override("GROUP_M", 0);
  p.rotate = plan_override("ROTATE", 1);
  p.xcd_m = pl.xcd_m ? 1 : 0;
  p.nt_out = pl.nt_out ? 1 : 0;
  const int epi = dt == DT_BF16 ? EPI_F32 : EPI_I32;  // raw sums (fp32 for float types)
  hipError_t e = pl.stream ? launch_gemm_stream(dt, epi, pl.mb, pl.nw, pl.wk, p, pl.nbpb, st)
                           : launch_gemm_tile(dt, epi, pl.tile, p, st);
  return hip_check(e, pl.stream ? "gemm_stream" : "gemm_tile");
}

// ------------------------------------------------------------------ validation

#define REQUIRE(cond, code, msg) \
  do {                           \
    if (!(cond)) return fail(code, msg); \
  } while (0)

w8a8_status check_ptr(const void* p, const char* name) {
  if (!p) return fail(W8A8_EINVAL, std::string(name) + " is NULL");
  if (!aligned16(p)) return fail(W8A8_EINVAL, std::string(name) + " is not 16-byte aligned");
  return W8A8_OK;
}

#define CHECK_PTR(p)                                \
  do {                                              \
    w8a8_status _s = check_ptr((p), #p);            \
    if (_s != W8A8_OK) return _s;                   \
  } while (0)

w8a8_status check_k(int64_t k) {
  REQUIRE(k >= 1, W8A8_EINVAL, "k < 1");
  REQUIRE(k % 16 == 0, W8A8_EUNSUPPORTED, "k must be a multiple of 16");
  REQUIRE(k <= W8A8_MAX_K, W8A8_EUNSUPPORTED, "k > 133144 would overflow the int32 accumulator");
  return W8A8_OK;
}

#define CHECK(expr)                      \
  do {                                   \
    w8a8_status _s = (expr);             \
    if (_s != W8A8_OK) return _s;        \
  } while (0)

w8a8_status check_desc(const w8a8_linear_desc* d) {
  REQUIRE(d, W8A8_EINVAL, "desc is NULL");
  REQUIRE(d->n >= 1, W8A8_EINVAL, "desc->n < 1");
  CHECK(check_k(d->k));
  CHECK(check_ptr(d->wq, "desc->wq"));
  CHECK(check_ptr(d->s_w, "desc->s_w"));
  if (d->delta) CHECK(check_ptr(d->delta, "desc->delta"));
  REQUIRE(d->n <= (int64_t)1 << 30, W8A8_EUNSUPPORTED, "n too large");
  return W8A8_OK;
}

// ------------------------------------------------------------------ workspace layouts

struct LinearWs {
  size_t qx, sx, gemm, total;
};
LinearWs linear_ws(int64_t m, int64_t n, int64_t k, int dt = DT_I8) {
  LinearWs w;
  Plan pl = plan_gemm(m, n, k, dt, false);
  w.qx = 0;
  w.sx = align256(w8a8_packed_bytes(m, k));
  w.gemm = w.sx + align256((size_t)m * 4);
  w.total = w.gemm + plan_ws_bytes(pl, m, n);
  return w;
}

struct FfnWs {
  size_t qx, sx, h, qh, sh, gemm, total;
};
FfnWs ffn_ws(int64_t m, int64_t d, int64_t f, int dt = DT_I8) {
  FfnWs w;
  Plan pd = plan_gemm(m, d, f, dt, false);
  w.qx = 0;
  w.sx = align256(w8a8_packed_bytes(m, d));
  w.h = w.sx + align256((size_t)m * 4);
  w.qh = w.h + align256((size_t)m * f * 2);
  w.sh = w.qh + align256(w8a8_packed_bytes(m, f));
  w.gemm = w.sh + align256((size_t)m * 4);
  w.total = w.gemm + plan_ws_bytes(pd, m, d);
  return w;
}

struct Bf16FfnWs {
  size_t h, gemm_gu, gemm_dn, total;
};
Bf16FfnWs bf16_ffn_ws(int64_t m, int64_t d, int64_t f) {
  Bf16FfnWs w;
  Plan pd = plan_gemm(m, d, f, DT_BF16, false);
  w.h = 0;
  w.gemm_dn = align256((size_t)m * f * 2);
  w.total = w.gemm_dn + plan_ws_bytes(pd, m, d);
  w.gemm_gu = 0;
  return w;
}

size_t bf16_linear_ws(int64_t m, int64_t n, int64_t k) {
  return plan_ws_bytes(plan_gemm(m, n, k, DT_BF16, false), m, n);
}

// Stack workspace: token stream, next-consumer input (bf16 and codes), FFN
// intermediates, the down projection's raw partial sums, the lm_head's GEMM
// workspace.
// INT8 down projection inside the stack: its split-K sums are reduced by the
// glue launch, so the plan may split K more freely than a standalone call.
// Planner overrides: DOWN_TILE, DOWN_SPLITS.
Plan stack_down_plan(int64_t m, int64_t d, int64_t f) {
  Plan p = plan_gemm(m, d, f, DT_I8, false);
  if (p.stream) {
    // The glue adds split-K partial sums at no extra launch, so at decode
    // sizes the long-K down projection is spread over twice as many
    // workgroups as its d / 16 column blocks: one CU streams only ~25 GB/s,
    // and 72 busy CUs would cap the projection near 1.8 TB/s (measured best:
    // 2 splits of 16 waves; 4 splits leave too little work per wave).
    const int64_t kb = ceil_div(f, kFragK8), nbc = ceil_div(d, 16);
    const int splits = plan_override("DOWN_SPLITS", (int)std::min<int64_t>(
                                                       std::max<int64_t>(1, kb / 16), ceil_div(144, nbc)));
    const int wk = plan_override("DOWN_WK", p.wk);
    if (splits > p.splits && (wk == 16 || wk == 4 || wk == 2) && !(wk == 16 && p.mb > 1)) {
      Plan q = p;
      q.nw = q.wk = wk;
      q.kchunk = (int)ceil_div(kb, splits);
      q.splits = (int)ceil_div(kb, q.kchunk);
      if (q.mb * q.kchunk + (wk - 1) * q.mb <= 158) return q;  // dynamic LDS, KiB
    }
    return p;
  }
  // Large M: bigger tiles with the K range cut in three (the glue adds the
  // partial sums), measured on the 26-layer stack (all26 + lm_head): M = 2048
  // 4.41 -> 4.12 ms with 256 x 128 tiles, M = 1024 2.49 -> 2.45 ms with
  // 128 x 128; from M = 512 down the plan above stays best.
  int dflt_splits = p.splits;
  if (tiles_of(TILE_256x128, m, d) >= 64) {
    p.tile = TILE_256x128;
    dflt_splits = 3;
  } else if (tiles_of(TILE_128x128, m, d) >= 64) {
    p.tile = TILE_128x128;
    dflt_splits = 3;
  }
  p.tile = plan_override("DOWN_TILE", p.tile);
  const int64_t kb = ceil_div(f, kFragK8);
  const int splits = std::max(1, plan_override("DOWN_SPLITS", dflt_splits));
  p.kchunk = (int)ceil_div(kb, splits);
  p.splits = (int)ceil_div(kb, p.kchunk);
  plan_order(p, m, d);
  // the int32 sums go straight to the next glue through memory: stored
  // non-temporally they leave the operand panels in L2 (26-layer stack
  // 1.43 -> 1.40 ms at M = 512, 2.149 -> 2.115 ms at 1024, 3.49 -> 3.46 ms at
  // 2048)
  if (plan_override("NT_OUT", -1) < 0)
    p.nt_out = plan_override("NT_DOWN", (int64_t)p.splits * m * d * 4 >= (2 << 20) ? 1 : 0) != 0;
  return p;
}

struct StackWs {
  size_t x, x2, a, q, s, h, qh, sh, part, lm, ctl, dec, total;
};
StackWs stack_ws(int64_t m, int64_t d, int64_t f, int64_t vocab) {
  StackWs w;
  const Plan p8 = stack_down_plan(m, d, f), p16 = plan_gemm(m, d, f, DT_BF16, false);
  // at one token the persistent decode kernel may write up to kGlueMaxSplits planes
  const int planes = std::max({p8.splits, p16.splits, m == 1 ? kGlueMaxSplits : 1});
  const size_t part = (size_t)planes * m * d * 4;
  const size_t lm = std::max(plan_ws_bytes(plan_gemm(m, vocab, d, DT_I8, false), m, vocab),
                             bf16_linear_ws(m, vocab, d));
  // the persistent decode kernel's barrier counters and status first: the
  // status query finds them at the start of the workspace
  w.ctl = 0;
  w.x = align256(sizeof(DecCtl));
  w.x2 = w.x + align256((size_t)m * d * 2);  // the token stream alternates between x and x2
  w.a = w.x2 + align256((size_t)m * d * 2);
  w.q = w.a + align256((size_t)m * d * 2);
  w.s = w.q + align256(w8a8_packed_bytes(m, d));
  w.h = w.s + align256((size_t)m * 4);
  w.qh = w.h + align256((size_t)m * f * 2);
  w.sh = w.qh + align256(w8a8_packed_bytes(m, f));
  w.part = w.sh + align256((size_t)m * 4);
  w.lm = w.part + align256(part);
  // the persistent decode kernel's per-layer buffers
  w.dec = w.lm + align256(lm);
  const size_t dec = m == 1 ? (size_t)kDecMaxLayers * decode_layout(d, f, kGlueMaxSplits).layer_bytes : 0;
  w.total = w.dec + align256(dec);
  return w;
}

// ------------------------------------------------------------------ pipelines

w8a8_status quant_act_impl(const void* x, bool bf16, int64_t m, int64_t k, const float* delta,
                           void* qx, float* sx, hipStream_t st, int dt = DT_I8) {
  return hip_check(launch_quant_rows(x, bf16, false, m, k, delta, (int8_t*)qx, sx, st,
                                     dt == DT_F8),
                   "quant_rows");
}

w8a8_status linear_impl(const w8a8_linear_desc* d, const void* x, bool x_bf16, int64_t m, void* y,
                        int epi, void* ws, hipStream_t st, int dt = DT_I8) {
  LinearWs w = linear_ws(m, d->n, d->k, dt);
  char* base = (char*)ws;
  Plan pl = plan_gemm(m, d->n, d->k, dt, false);
  if (x_bf16 && plan_qloads(pl, m, d->k))  // one launch: the GEMM quantises x itself
    return run_gemm(pl, dt, epi, nullptr, 0, m, d->wq, nullptr, d->n, d->k, nullptr, d->s_w,
                    nullptr, y, d->n, base + w.gemm, st,
                    QLoad{(const uint16_t*)x, d->delta, (float*)(base + w.sx)});
  CHECK(quant_act_impl(x, x_bf16, m, d->k, d->delta, base + w.qx, (float*)(base + w.sx), st, dt));
  return run_gemm(pl, dt, epi, base + w.qx, 0, m, d->wq, nullptr, d->n, d->k,
                  (const float*)(base + w.sx), d->s_w, nullptr, y, d->n, base + w.gemm, st);
}

w8a8_status ffn_impl(const w8a8_ffn_desc* d, const void* x, int64_t m, void* y, void* ws,
                     hipStream_t st, int dt = DT_I8) {
  FfnWs w = ffn_ws(m, d->d, d->f, dt);
  char* base = (char*)ws;
  Plan pg = plan_gemm(m, d->f, d->d, dt, true);
  if (plan_qloads(pg, m, d->d)) {
    CHECK(run_gemm(pg, dt, EPI_GLU, nullptr, 0, m, d->wq_gate, d->wq_up, d->f, d->d, nullptr,
                   d->s_gate, d->s_up, base + w.h, d->f, nullptr, st,
                   QLoad{(const uint16_t*)x, d->delta_gu, (float*)(base + w.sx)}));
  } else {
    CHECK(quant_act_impl(x, true, m, d->d, d->delta_gu, base + w.qx, (float*)(base + w.sx), st,
                         dt));
    CHECK(run_gemm(pg, dt, EPI_GLU, base + w.qx, 0, m, d->wq_gate, d->wq_up, d->f, d->d,
                   (const float*)(base + w.sx), d->s_gate, d->s_up, base + w.h, d->f, nullptr,
                   st));
  }
  Plan pd = plan_gemm(m, d->d, d->f, dt, false);
  if (plan_qloads(pd, m, d->f))
    return run_gemm(pd, dt, EPI_BF16, nullptr, 0, m, d->wq_down, nullptr, d->d, d->f, nullptr,
                    d->s_down, nullptr, y, d->d, base + w.gemm, st,
                    QLoad{(const uint16_t*)(base + w.h), d->delta_down, (float*)(base + w.sh)});
  CHECK(quant_act_impl(base + w.h, true, m, d->f, d->delta_down, base + w.qh,
                       (float*)(base + w.sh), st, dt));
  return run_gemm(pd, dt, EPI_BF16, base + w.qh, 0, m, d->wq_down, nullptr, d->d, d->f,
                  (const float*)(base + w.sh), d->s_down, nullptr, y, d->d, base + w.gemm, st);
}

w8a8_status bf16_linear_impl(const void* x, int64_t m, const void* wp, int64_t n, int64_t k,
                             void* y, void* ws, hipStream_t st) {
  Plan pl = plan_gemm(m, n, k, DT_BF16, false);
  return run_gemm(pl, DT_BF16, EPI_BF16, x, k, m, wp, nullptr, n, k, nullptr, nullptr, nullptr, y, n,
                  ws, st);
}

w8a8_status bf16_ffn_impl(const w8a8_bf16_ffn_desc* d, const void* x, int64_t m, void* y,
                          void* ws, hipStream_t st) {
  Bf16FfnWs w = bf16_ffn_ws(m, d->d, d->f);
  char* base = (char*)ws;
  Plan pg = plan_gemm(m, d->f, d->d, DT_BF16, true);
  CHECK(run_gemm(pg, DT_BF16, EPI_GLU, x, d->d, m, d->wp_gate, d->wp_up, d->f, d->d, nullptr, nullptr,
                 nullptr, base + w.h, d->f, nullptr, st));
  Plan pd = plan_gemm(m, d->d, d->f, DT_BF16, false);
  return run_gemm(pd, DT_BF16, EPI_BF16, base + w.h, d->f, m, d->wp_down, nullptr, d->d, d->f,
                  nullptr, nullptr, nullptr, y, d->d, base + w.gemm_dn, st);
}

}  // namespace

// ====================================================================== C ABI

extern "C" {

size_t w8a8_packed_bytes(int64_t n, int64_t k) {
  if (n < 1 || k < 1) return 0;
  return (size_t)round_up(n, 16) * (size_t)round_up(k, 64);
}

size_t w8a8_packed_bf16_bytes(int64_t n, int64_t k) {
  if (n < 1 || k < 1) return 0;
  return (size_t)round_up(n, 16) * (size_t)round_up(k, 32) * 2;
}

size_t w8a8_linear_workspace_bytes(int64_t m, int64_t n, int64_t k) {
  if (m < 1 || n < 1 || k < 1) return 0;
  return linear_ws(m, n, k).total;
}

size_t w8a8_ffn_workspace_bytes(int64_t m, int64_t d, int64_t f) {
  if (m < 1 || d < 1 || f < 1) return 0;
  return ffn_ws(m, d, f).total;
}

size_t w8a8_bf16_ffn_workspace_bytes(int64_t m, int64_t d, int64_t f) {
  if (m < 1 || d < 1 || f < 1) return 0;
  return bf16_ffn_ws(m, d, f).total;
}

size_t w8a8_bf16_linear_workspace_bytes(int64_t m, int64_t n, int64_t k) {
  if (m < 1 || n < 1 || k < 1) return 0;
  return bf16_linear_ws(m, n, k);
}

size_t w8a8_lm_head_workspace_bytes(int64_t m, int64_t n, int64_t k) {
  return w8a8_linear_workspace_bytes(m, n, k);
}

size_t w8a8_stack_workspace_bytes(int64_t m, int64_t d, int64_t f, int64_t vocab) {
  if (m < 1 || d < 1 || f < 1 || vocab < 1) return 0;
  return stack_ws(m, d, f, vocab).total;
}

const char* w8a8_status_str(int s) {
  switch (s) {
    case W8A8_OK: return "ok";
    case W8A8_EINVAL: return "invalid argument";
    case W8A8_EUNSUPPORTED: return "unsupported shape or dtype";
    case W8A8_EHIP: return "HIP error";
    case W8A8_EWORKSPACE: return "workspace too small";
    case W8A8_ETIMEOUT: return "a device-wide wait of the persistent decode kernel gave up";
  }
  return "unknown status";
}

const char* w8a8_last_error(void) { return g_last_error.c_str(); }

int w8a8_set_plan_override(const char* name, int value) {
  if (!name) return -1;
  const int i = override_index(name);
  if (i < 0 || value == kUnset) return -1;
  g_override[i].store(value);
  return 0;
}

void w8a8_clear_plan_overrides(void) {
  for (auto& o : g_override) o.store(kUnset);
}

// ---------------------------------------------------------------- a1

w8a8_status w8a8_col_absmax(const void* x, w8a8_dtype xt, int64_t rows, int64_t k, float* amax,
                            w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(x);
  CHECK_PTR(amax);
  REQUIRE(rows >= 1 && k >= 1, W8A8_EINVAL, "rows or k < 1");
  REQUIRE(xt == W8A8_F32 || xt == W8A8_BF16, W8A8_EUNSUPPORTED, "x dtype");
  return hip_check(launch_col_absmax(x, xt == W8A8_BF16, rows, k, amax, S(stream)), "col_absmax");
}

w8a8_status w8a8_smooth_delta(const float* act_amax, const float* w_amax, int64_t k,
                              float alpha, float* delta, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(act_amax);
  CHECK_PTR(w_amax);
  CHECK_PTR(delta);
  REQUIRE(k >= 1, W8A8_EINVAL, "k < 1");
  REQUIRE(alpha >= 0.0f && alpha <= 1.0f, W8A8_EUNSUPPORTED, "alpha outside [0, 1]");
  return hip_check(launch_smooth_delta(act_amax, w_amax, k, (double)alpha, delta, S(stream)),
                   "smooth_delta");
}

w8a8_status w8a8_smooth_calibrate(const float* act_amax, const void* const* w,
                                  const int64_t* n_rows, int n_w, w8a8_dtype w_dtype, int64_t k,
                                  float alpha, float* delta, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(act_amax);
  CHECK_PTR(delta);
  REQUIRE(w != nullptr && n_rows != nullptr, W8A8_EINVAL, "w or n_rows is NULL");
  REQUIRE(n_w >= 1, W8A8_EINVAL, "n_w < 1");
  REQUIRE(k >= 1, W8A8_EINVAL, "k < 1");
  REQUIRE(w_dtype == W8A8_F32 || w_dtype == W8A8_BF16, W8A8_EUNSUPPORTED, "w dtype");
  REQUIRE(alpha >= 0.0f && alpha <= 1.0f, W8A8_EUNSUPPORTED, "alpha outside [0, 1]");
  for (int i = 0; i < n_w; ++i) {
    CHECK(check_ptr(w[i], "w[i]"));
    REQUIRE(n_rows[i] >= 1, W8A8_EINVAL, "n_rows[i] < 1");
  }
  // delta holds the running weight maximum max_i |W_ij| over the stacked rows
  // of every consumer, then the factor itself (elementwise, in place)
  hipStream_t st = S(stream);
  CHECK(hip_check(launch_fill_f32(delta, k, 0.0f, st), "fill"));
  for (int i = 0; i < n_w; ++i)
    CHECK(hip_check(launch_col_absmax(w[i], w_dtype == W8A8_BF16, n_rows[i], k, delta, st),
                    "col_absmax"));
  return hip_check(launch_smooth_delta(act_amax, delta, k, (double)alpha, delta, st),
                   "smooth_delta");
}

// ---------------------------------------------------------------- a2

w8a8_status w8a8_quantize_weights(const void* w, w8a8_dtype wt, int64_t n, int64_t k,
                                  const float* delta, void* wq, float* s_w, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(w);
  CHECK_PTR(wq);
  CHECK_PTR(s_w);
  if (delta) CHECK_PTR(delta);
  REQUIRE(n >= 1, W8A8_EINVAL, "n < 1");
  CHECK(check_k(k));
  REQUIRE(wt == W8A8_F32 || wt == W8A8_BF16, W8A8_EUNSUPPORTED, "w dtype");
  return hip_check(launch_quant_rows(w, wt == W8A8_BF16, true, n, k, delta, (int8_t*)wq, s_w,
                                     S(stream)),
                   "quant_rows");
}

w8a8_status w8a8_unpack_weights(const void* wq, int64_t n, int64_t k, int8_t* q,
                                w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(wq);
  REQUIRE(q, W8A8_EINVAL, "q is NULL");
  REQUIRE(n >= 1, W8A8_EINVAL, "n < 1");
  CHECK(check_k(k));
  return hip_check(launch_unpack(wq, n, k, q, S(stream)), "unpack");
}

w8a8_status w8a8_pack_bf16(const void* w, int64_t n, int64_t k, void* wp, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(w);
  CHECK_PTR(wp);
  REQUIRE(n >= 1 && k >= 1, W8A8_EINVAL, "n or k < 1");
  REQUIRE(k % 32 == 0, W8A8_EUNSUPPORTED, "k must be a multiple of 32 on the bf16 path");
  return hip_check(launch_pack_bf16(w, n, k, wp, S(stream)), "pack_bf16");
}

// ---------------------------------------------------------------- a3

w8a8_status w8a8_quantize_act(const void* x, w8a8_dtype xt, int64_t m, int64_t k,
                              const float* delta, void* qx, float* s_x, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(x);
  CHECK_PTR(qx);
  CHECK_PTR(s_x);
  if (delta) CHECK_PTR(delta);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  CHECK(check_k(k));
  REQUIRE(xt == W8A8_F32 || xt == W8A8_BF16, W8A8_EUNSUPPORTED, "x dtype");
  return quant_act_impl(x, xt == W8A8_BF16, m, k, delta, qx, s_x, S(stream));
}

// ---------------------------------------------------------------- a4 / a5

w8a8_status w8a8_gemm_i8_i32(const void* qx, int64_t m, const void* wq, int64_t n, int64_t k,
                             int32_t* acc, void* ws, size_t ws_bytes, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(qx);
  CHECK_PTR(wq);
  CHECK_PTR(acc);
  REQUIRE(m >= 1 && n >= 1, W8A8_EINVAL, "m or n < 1");
  CHECK(check_k(k));
  Plan pl = plan_gemm(m, n, k, DT_I8, false);
  size_t need = plan_ws_bytes(pl, m, n);
  if (need) {
    CHECK_PTR(ws);
    REQUIRE(ws_bytes >= need, W8A8_EWORKSPACE, "workspace too small");
  }
  return run_gemm(pl, DT_I8, EPI_I32, qx, 0, m, wq, nullptr, n, k, nullptr, nullptr, nullptr, acc,
                  n, ws, S(stream));
}

w8a8_status w8a8_linear(const w8a8_linear_desc* desc, const void* x, w8a8_dtype xt, int64_t m,
                        void* y, w8a8_dtype yt, void* ws, size_t ws_bytes, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_desc(desc));
  CHECK_PTR(x);
  CHECK_PTR(y);
  CHECK_PTR(ws);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  REQUIRE(xt == W8A8_F32 || xt == W8A8_BF16, W8A8_EUNSUPPORTED, "x dtype");
  REQUIRE(yt == W8A8_F32 || yt == W8A8_BF16, W8A8_EUNSUPPORTED, "y dtype");
  REQUIRE(ws_bytes >= w8a8_linear_workspace_bytes(m, desc->n, desc->k), W8A8_EWORKSPACE,
          "workspace too small");
  return linear_impl(desc, x, xt == W8A8_BF16, m, y, yt == W8A8_BF16 ? EPI_BF16 : EPI_F32, ws,
                     S(stream));
}

// ---------------------------------------------------------------- a6

static w8a8_status check_ffn_desc(const w8a8_ffn_desc* d) {
  REQUIRE(d, W8A8_EINVAL, "desc is NULL");
  REQUIRE(d->d >= 1 && d->f >= 1, W8A8_EINVAL, "d or f < 1");
  CHECK(check_k(d->d));
  CHECK(check_k(d->f));
  CHECK(check_ptr(d->wq_gate, "desc->wq_gate"));
  CHECK(check_ptr(d->s_gate, "desc->s_gate"));
  CHECK(check_ptr(d->wq_up, "desc->wq_up"));
  CHECK(check_ptr(d->s_up, "desc->s_up"));
  CHECK(check_ptr(d->wq_down, "desc->wq_down"));
  CHECK(check_ptr(d->s_down, "desc->s_down"));
  if (d->delta_gu) CHECK(check_ptr(d->delta_gu, "desc->delta_gu"));
  if (d->delta_down) CHECK(check_ptr(d->delta_down, "desc->delta_down"));
  return W8A8_OK;
}

w8a8_status w8a8_ffn_gate_up(const w8a8_ffn_desc* desc, const void* qx, const float* s_x,
                             int64_t m, void* h, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_ffn_desc(desc));
  CHECK_PTR(qx);
  CHECK_PTR(s_x);
  CHECK_PTR(h);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  Plan pg = plan_gemm(m, desc->f, desc->d, DT_I8, true);
  return run_gemm(pg, DT_I8, EPI_GLU, qx, 0, m, desc->wq_gate, desc->wq_up, desc->f, desc->d, s_x,
                  desc->s_gate, desc->s_up, h, desc->f, nullptr, S(stream));
}

w8a8_status w8a8_geglu_requant(const float* g, const float* u, int64_t m, int64_t n,
                               const float* delta, void* q, float* s, void* h,
                               w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(g);
  CHECK_PTR(u);
  CHECK_PTR(q);
  CHECK_PTR(s);
  if (delta) CHECK_PTR(delta);
  if (h) CHECK_PTR(h);
  REQUIRE(m >= 1 && n >= 1, W8A8_EINVAL, "m or n < 1");
  REQUIRE(n % 16 == 0, W8A8_EUNSUPPORTED, "n must be a multiple of 16");
  CHECK(check_k(n));
  REQUIRE(m <= INT32_MAX, W8A8_EUNSUPPORTED, "m too large");
  return hip_check(launch_geglu_requant(g, u, m, n, delta, (int8_t*)q, s, (uint16_t*)h,
                                        S(stream)),
                   "geglu_requant");
}

// ------------------------------------------------------------------ no-allocation FFN

namespace {

// Scratch memory of w8a8_ffn_noalloc: one copy of this array on every GPU the
// library runs on, resident until the process ends.  In host code the name
// is only a host-side stand-in (passing it to a kernel compiles and then
// faults); the device address of each GPU's copy comes from
// hipGetSymbolAddress, taken once per device with that device current, and
// only that address is ever handed to kernels.
__device__ __align__(256) char scratch[W8A8_FFN_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
struct ScratchSlot {
  std::once_flag once;
  void* ptr = nullptr;
  hipError_t err = hipSuccess;
};
ScratchSlot g_scratch[kMaxDevices];

// Device address of the current device's scratch array (looked up on the
// first call on that device).
w8a8_status current_scratch(void** out) {
  int dev = 0;
  CHECK(hip_check(hipGetDevice(&dev), "hipGetDevice"));
  REQUIRE(dev >= 0 && dev < kMaxDevices, W8A8_EUNSUPPORTED, "device index above 63");
  ScratchSlot& slot = g_scratch[dev];
  std::call_once(slot.once, [&slot] {
    slot.err = hipGetSymbolAddress(&slot.ptr, HIP_SYMBOL(scratch));
  });
  CHECK(hip_check(slot.err, "hipGetSymbolAddress(scratch)"));
  REQUIRE(slot.ptr != nullptr, W8A8_EHIP, "no device address for the scratch array");
  *out = slot.ptr;
  return W8A8_OK;
}

}  // namespace

w8a8_status w8a8_ffn_noalloc(const w8a8_ffn_desc* desc, const void* x, int64_t m, void* y,
                             w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_ffn_desc(desc));
  CHECK_PTR(x);
  CHECK_PTR(y);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  const size_t need = w8a8_ffn_workspace_bytes(m, desc->d, desc->f);
  REQUIRE(need <= (size_t)W8A8_FFN_NOALLOC_SCRATCH_BYTES, W8A8_EWORKSPACE,
          "this m x d x f needs " + std::to_string(need) +
              " bytes of scratch; the no-allocation FFN holds " +
              std::to_string((size_t)W8A8_FFN_NOALLOC_SCRATCH_BYTES));
  void* ws = nullptr;
  CHECK(current_scratch(&ws));
  return ffn_impl(desc, x, m, y, ws, S(stream));
}

w8a8_status w8a8_ffn(const w8a8_ffn_desc* desc, const void* x, int64_t m, void* y, void* ws,
                     size_t ws_bytes, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_ffn_desc(desc));
  CHECK_PTR(x);
  CHECK_PTR(y);
  CHECK_PTR(ws);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  REQUIRE(ws_bytes >= w8a8_ffn_workspace_bytes(m, desc->d, desc->f), W8A8_EWORKSPACE,
          "workspace too small");
  return ffn_impl(desc, x, m, y, ws, S(stream));
}

// ---------------------------------------------------------------- a7

w8a8_status w8a8_lm_head(const w8a8_linear_desc* desc, const void* x, int64_t m, void* logits,
                         void* ws, size_t ws_bytes, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_desc(desc));
  CHECK_PTR(x);
  CHECK_PTR(logits);
  CHECK_PTR(ws);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  REQUIRE(ws_bytes >= w8a8_lm_head_workspace_bytes(m, desc->n, desc->k), W8A8_EWORKSPACE,
          "workspace too small");
  return linear_impl(desc, x, true, m, logits, EPI_BF16, ws, S(stream));
}

// ---------------------------------------------------------------- FP8 variant

static w8a8_status check_k_f8(int64_t k) {
  CHECK(check_k(k));
  REQUIRE(k % 128 == 0, W8A8_EUNSUPPORTED, "k must be a multiple of 128 on the FP8 path");
  return W8A8_OK;
}

size_t w8a8_fp8_linear_workspace_bytes(int64_t m, int64_t n, int64_t k) {
  if (m < 1 || n < 1 || k < 1) return 0;
  return linear_ws(m, n, k, DT_F8).total;
}

size_t w8a8_fp8_ffn_workspace_bytes(int64_t m, int64_t d, int64_t f) {
  if (m < 1 || d < 1 || f < 1) return 0;
  return ffn_ws(m, d, f, DT_F8).total;
}

w8a8_status w8a8_fp8_quantize_weights(const void* w, w8a8_dtype wt, int64_t n, int64_t k,
                                      const float* delta, void* wq, float* s_w,
                                      w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(w);
  CHECK_PTR(wq);
  CHECK_PTR(s_w);
  if (delta) CHECK_PTR(delta);
  REQUIRE(n >= 1, W8A8_EINVAL, "n < 1");
  CHECK(check_k(k));
  REQUIRE(wt == W8A8_F32 || wt == W8A8_BF16, W8A8_EUNSUPPORTED, "w dtype");
  return hip_check(launch_quant_rows(w, wt == W8A8_BF16, true, n, k, delta, (int8_t*)wq, s_w,
                                     S(stream), true),
                   "quant_rows");
}

w8a8_status w8a8_fp8_quantize_act(const void* x, w8a8_dtype xt, int64_t m, int64_t k,
                                  const float* delta, void* qx, float* s_x, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(x);
  CHECK_PTR(qx);
  CHECK_PTR(s_x);
  if (delta) CHECK_PTR(delta);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  CHECK(check_k(k));
  REQUIRE(xt == W8A8_F32 || xt == W8A8_BF16, W8A8_EUNSUPPORTED, "x dtype");
  return quant_act_impl(x, xt == W8A8_BF16, m, k, delta, qx, s_x, S(stream), DT_F8);
}

w8a8_status w8a8_fp8_gemm_f32(const void* qx, int64_t m, const void* wq, int64_t n, int64_t k,
                              float* acc, void* ws, size_t ws_bytes, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(qx);
  CHECK_PTR(wq);
  CHECK_PTR(acc);
  REQUIRE(m >= 1 && n >= 1, W8A8_EINVAL, "m or n < 1");
  CHECK(check_k_f8(k));
  Plan pl = plan_gemm(m, n, k, DT_F8, false);
  size_t need = plan_ws_bytes(pl, m, n);
  if (need) {
    CHECK_PTR(ws);
    REQUIRE(ws_bytes >= need, W8A8_EWORKSPACE, "workspace too small");
  }
  return run_gemm(pl, DT_F8, EPI_I32, qx, 0, m, wq, nullptr, n, k, nullptr, nullptr, nullptr, acc,
                  n, ws, S(stream));
}

w8a8_status w8a8_fp8_linear(const w8a8_linear_desc* desc, const void* x, w8a8_dtype xt,
                            int64_t m, void* y, w8a8_dtype yt, void* ws, size_t ws_bytes,
                            w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_desc(desc));
  CHECK(check_k_f8(desc->k));
  CHECK_PTR(x);
  CHECK_PTR(y);
  CHECK_PTR(ws);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  REQUIRE(xt == W8A8_F32 || xt == W8A8_BF16, W8A8_EUNSUPPORTED, "x dtype");
  REQUIRE(yt == W8A8_F32 || yt == W8A8_BF16, W8A8_EUNSUPPORTED, "y dtype");
  REQUIRE(ws_bytes >= w8a8_fp8_linear_workspace_bytes(m, desc->n, desc->k), W8A8_EWORKSPACE,
          "workspace too small");
  return linear_impl(desc, x, xt == W8A8_BF16, m, y, yt == W8A8_BF16 ? EPI_BF16 : EPI_F32, ws,
                     S(stream), DT_F8);
}

w8a8_status w8a8_fp8_ffn_gate_up(const w8a8_ffn_desc* desc, const void* qx, const float* s_x,
                                 int64_t m, void* h, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_ffn_desc(desc));
  CHECK(check_k_f8(desc->d));
  CHECK_PTR(qx);
  CHECK_PTR(s_x);
  CHECK_PTR(h);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  Plan pg = plan_gemm(m, desc->f, desc->d, DT_F8, true);
  return run_gemm(pg, DT_F8, EPI_GLU, qx, 0, m, desc->wq_gate, desc->wq_up, desc->f, desc->d, s_x,
                  desc->s_gate, desc->s_up, h, desc->f, nullptr, S(stream));
}

w8a8_status w8a8_fp8_ffn(const w8a8_ffn_desc* desc, const void* x, int64_t m, void* y, void* ws,
                         size_t ws_bytes, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_ffn_desc(desc));
  CHECK(check_k_f8(desc->d));
  CHECK(check_k_f8(desc->f));
  CHECK_PTR(x);
  CHECK_PTR(y);
  CHECK_PTR(ws);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  REQUIRE(ws_bytes >= w8a8_fp8_ffn_workspace_bytes(m, desc->d, desc->f), W8A8_EWORKSPACE,
          "workspace too small");
  return ffn_impl(desc, x, m, y, ws, S(stream), DT_F8);
}

w8a8_status w8a8_fp8_lm_head(const w8a8_linear_desc* desc, const void* x, int64_t m,
                             void* logits, void* ws, size_t ws_bytes, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_desc(desc));
  CHECK(check_k_f8(desc->k));
  CHECK_PTR(x);
  CHECK_PTR(logits);
  CHECK_PTR(ws);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  REQUIRE(ws_bytes >= w8a8_fp8_linear_workspace_bytes(m, desc->n, desc->k), W8A8_EWORKSPACE,
          "workspace too small");
  return linear_impl(desc, x, true, m, logits, EPI_BF16, ws, S(stream), DT_F8);
}

// ---------------------------------------------------------------- bf16 path

w8a8_status w8a8_bf16_linear(const void* x, int64_t m, const void* wp, int64_t n, int64_t k,
                             void* y, void* ws, size_t ws_bytes, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(x);
  CHECK_PTR(wp);
  CHECK_PTR(y);
  REQUIRE(m >= 1 && n >= 1 && k >= 1, W8A8_EINVAL, "m, n or k < 1");
  REQUIRE(k % 32 == 0, W8A8_EUNSUPPORTED, "k must be a multiple of 32 on the bf16 path");
  size_t need = bf16_linear_ws(m, n, k);
  if (need) {
    CHECK_PTR(ws);
    REQUIRE(ws_bytes >= need, W8A8_EWORKSPACE, "workspace too small");
  }
  return bf16_linear_impl(x, m, wp, n, k, y, ws, S(stream));
}

static w8a8_status check_bf16_ffn_desc(const w8a8_bf16_ffn_desc* d) {
  REQUIRE(d, W8A8_EINVAL, "desc is NULL");
  REQUIRE(d->d >= 1 && d->f >= 1, W8A8_EINVAL, "d or f < 1");
  REQUIRE(d->d % 32 == 0 && d->f % 32 == 0, W8A8_EUNSUPPORTED,
          "d and f must be multiples of 32 on the bf16 path");
  CHECK(check_ptr(d->wp_gate, "desc->wp_gate"));
  CHECK(check_ptr(d->wp_up, "desc->wp_up"));
  CHECK(check_ptr(d->wp_down, "desc->wp_down"));
  return W8A8_OK;
}

w8a8_status w8a8_bf16_ffn_gate_up(const w8a8_bf16_ffn_desc* desc, const void* x, int64_t m,
                                  void* h, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_bf16_ffn_desc(desc));
  CHECK_PTR(x);
  CHECK_PTR(h);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  Plan pg = plan_gemm(m, desc->f, desc->d, DT_BF16, true);
  return run_gemm(pg, DT_BF16, EPI_GLU, x, desc->d, m, desc->wp_gate, desc->wp_up, desc->f, desc->d,
                  nullptr, nullptr, nullptr, h, desc->f, nullptr, S(stream));
}

w8a8_status w8a8_bf16_ffn(const w8a8_bf16_ffn_desc* desc, const void* x, int64_t m, void* y,
                          void* ws, size_t ws_bytes, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_bf16_ffn_desc(desc));
  CHECK_PTR(x);
  CHECK_PTR(y);
  CHECK_PTR(ws);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  REQUIRE(ws_bytes >= w8a8_bf16_ffn_workspace_bytes(m, desc->d, desc->f), W8A8_EWORKSPACE,
          "workspace too small");
  return bf16_ffn_impl(desc, x, m, y, ws, S(stream));
}

// ---------------------------------------------------------------- a8 / a9

static w8a8_status check_norm_d(int64_t d) {
  REQUIRE(d >= 1, W8A8_EINVAL, "d < 1");
  REQUIRE(d % 8 == 0 && d <= 8192, W8A8_EUNSUPPORTED, "RMSNorm needs d % 8 == 0 and d <= 8192");
  return W8A8_OK;
}

w8a8_status w8a8_rmsnorm(const void* x, int64_t m, int64_t d, void* y, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(x);
  CHECK_PTR(y);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  CHECK(check_norm_d(d));
  return hip_check(launch_rmsnorm(nullptr, (const uint16_t*)x, m, d, (uint16_t*)y, S(stream)),
                   "rmsnorm");
}

w8a8_status w8a8_rmsnorm_residual(const void* x, const void* f, int64_t m, int64_t d, void* x_out,
                                  w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(x);
  CHECK_PTR(f);
  CHECK_PTR(x_out);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  CHECK(check_norm_d(d));
  return hip_check(launch_rmsnorm((const uint16_t*)x, (const uint16_t*)f, m, d,
                                  (uint16_t*)x_out, S(stream)),
                   "rmsnorm_residual");
}

int w8a8_precision_map(const char* name, uint8_t* prec, int n_layers) {
  if (!name || !prec || n_layers < 26) return -1;
  int lo1 = 0, hi1 = -1, lo2 = 0, hi2 = -1;
  if (std::strcmp(name, "bf16") == 0) {
  } else if (std::strcmp(name, "5+5") == 0) {
    lo1 = 0; hi1 = 4; lo2 = 21; hi2 = 25;      // eq. ffn55
  } else if (std::strcmp(name, "10+10") == 0) {
    lo1 = 0; hi1 = 9; lo2 = 16; hi2 = 25;      // eq. ffn1010
  } else if (std::strcmp(name, "all26") == 0) {
    lo1 = 0; hi1 = 25;                         // eq. ffnall26
  } else {
    return -1;
  }
  int count = 0;
  for (int l = 0; l < n_layers; ++l) {
    bool q = (l >= lo1 && l <= hi1) || (l >= lo2 && l <= hi2);
    prec[l] = q ? 1 : 0;
    count += q;
  }
  return count;
}

}  // extern "C"

namespace {

// Validation shared by the stack entry points (host memory prec[n_layers]).
w8a8_status check_stack(const w8a8_stack_desc* desc, const uint8_t* prec, int lm_head_int8,
                        bool need_lm_head) {
  REQUIRE(desc, W8A8_EINVAL, "desc is NULL");
  REQUIRE(prec, W8A8_EINVAL, "prec is NULL");
  REQUIRE(desc->n_layers >= 1 && desc->d >= 1 && desc->f >= 1 && desc->vocab >= 1, W8A8_EINVAL,
          "stack sizes < 1");
  const int64_t d = desc->d, f = desc->f;
  CHECK(check_norm_d(d));
  for (int64_t l = 0; l < desc->n_layers; ++l) {
    if (prec[l]) {
      REQUIRE(desc->int8_ffn, W8A8_EINVAL, "int8_ffn is NULL");
      CHECK(check_ffn_desc(&desc->int8_ffn[l]));
      REQUIRE(desc->int8_ffn[l].d == d && desc->int8_ffn[l].f == f, W8A8_EINVAL, "layer shape");
    } else {
      REQUIRE(desc->bf16_ffn, W8A8_EINVAL, "bf16_ffn is NULL");
      CHECK(check_bf16_ffn_desc(&desc->bf16_ffn[l]));
      REQUIRE(desc->bf16_ffn[l].d == d && desc->bf16_ffn[l].f == f, W8A8_EINVAL, "layer shape");
    }
  }
  if (!need_lm_head) return W8A8_OK;
  if (lm_head_int8) {
    CHECK(check_desc(&desc->lm_head_int8));
    REQUIRE(desc->lm_head_int8.n == desc->vocab && desc->lm_head_int8.k == d, W8A8_EINVAL,
            "lm_head shape");
  } else {
    CHECK_PTR(desc->lm_head_bf16);
    REQUIRE(d % 32 == 0, W8A8_EUNSUPPORTED, "d must be a multiple of 32 on the bf16 path");
  }
  return W8A8_OK;
}

// The stack over validated arguments.  logits NULL: no lm_head (the final
// glue still runs).  hidden non-NULL: the token stream after every layer,
// hidden[l] = bf16 m x d, n_layers of them back to back.
w8a8_status stack_run(const w8a8_stack_desc* desc, const uint8_t* prec, int lm_head_int8,
                      const void* x, int64_t m, void* logits, uint16_t* hidden, void* ws,
                      hipStream_t st) {
  const int64_t d = desc->d, f = desc->f;
  char* base = (char*)ws;
  const StackWs w = stack_ws(m, d, f, desc->vocab);
  uint16_t* xbuf[2] = {(uint16_t*)(base + w.x), (uint16_t*)(base + w.x2)};
  const uint16_t* xin = (const uint16_t*)x;  // the latest token stream
  int nxt = 0;                               // the buffer the next update writes
  uint16_t* a = (uint16_t*)(base + w.a);
  int8_t* q = (int8_t*)(base + w.q);
  float* s = (float*)(base + w.s);
  uint16_t* h = (uint16_t*)(base + w.h);
  int8_t* qh = (int8_t*)(base + w.qh);
  float* sh = (float*)(base + w.sh);
  void* part = base + w.part;
  const Plan p8 = stack_down_plan(m, d, f), p16 = plan_gemm(m, d, f, DT_BF16, false);
  const Plan pg8 = plan_gemm(m, f, d, DT_I8, true), pg16 = plan_gemm(m, f, d, DT_BF16, true);
  // every call starts with a clear failure word (w8a8_ffn_stack_status)
  CHECK(hip_check(launch_dec_status_clear((DecCtl*)(base + w.ctl), st), "status clear"));

  // At one token, runs of consecutive INT8 layers go to the persistent decode
  // kernel (one launch per run of up to kDecMaxLayers layers) when the device
  // holds one of its workgroups per CU and the shape fits it.
  int dec_grid = 0, dec_splits = 0;
  if (m == 1 && !plan_override("NO_PERSISTENT", 0)) {
    int dev = 0;
    CHECK(hip_check(hipGetDevice(&dev), "hipGetDevice"));
    dec_grid = decode_grid(dev);
    dec_splits = decode_splits(d, f, dec_grid);
  }
  // K-split planes of each layer's down projection output
  std::vector<int> out_splits(desc->n_layers, 0);
  auto splits_of = [&](int64_t l) { return out_splits[l]; };

  // Glue launch l (0..n_layers): FFN output of layer l-1 into the token
  // stream (none for l = 0, which copies x in), then the pre-norm input of
  // layer l (or of the lm_head for l = n_layers), as codes for an INT8
  // consumer and as bf16 for a bf16 one.
  auto glue = [&](int64_t l) -> w8a8_status {
    GlueParams g;
    g.m = m;
    g.d = d;
    g.rows_pad = round_up(m, 16);
    g.kp = round_up(d, 64);
    g.x_in = xin;
    g.x_out = xbuf[nxt];
    if (hidden && l > 0) g.x_copy = hidden + (l - 1) * m * d;
    if (l > 0) {
      const bool i8 = prec[l - 1] != 0;
      g.part = part;
      g.splits = splits_of(l - 1);
      g.part_f32 = !i8;
      if (i8) {
        g.s_t = sh;
        g.s_i = desc->int8_ffn[l - 1].s_down;
      }
    }
    const bool next_i8 = l < desc->n_layers ? prec[l] != 0 : lm_head_int8 != 0;
    if (next_i8) {
      g.q = q;
      g.s = s;
      g.delta = l < desc->n_layers ? desc->int8_ffn[l].delta_gu : desc->lm_head_int8.delta;
    } else {
      g.a = a;
    }
    CHECK(hip_check(launch_glue(g, st), "glue"));
    xin = xbuf[nxt];
    nxt ^= 1;
    return W8A8_OK;
  };

  // At one token the glue in front of an INT8 layer runs inside that layer's
  // gate/up GEMM (every workgroup computes it for the row while its weights
  // arrive; workgroup 0 writes the token stream), one launch and one memory
  // round trip less per layer.
  const bool fuse_ok = m == 1 && !plan_override("NO_FUSED_GLUE", 0) && pg8.stream &&
                       pg8.mb == 1 && d % 8 == 0 && d / 8 <= 64 * pg8.nw;
  auto fused = [&](int64_t l) {
    if (!fuse_ok || !prec[l]) return false;
    return l == 0 || splits_of(l - 1) <= kGlueMaxSplits;
  };

  for (int64_t l = 0; l < desc->n_layers; ++l) {
    if (dec_splits && prec[l]) {
      int64_t l1 = l;
      while (l1 < desc->n_layers && prec[l1] && l1 - l < kDecMaxLayers) ++l1;
      DecParams P;
      P.n_layers = (int)(l1 - l);
      P.l0 = (int)l;
      P.d = (int)d;
      P.f = (int)f;
      for (int64_t j = l; j < l1; ++j) {
        const w8a8_ffn_desc* L = &desc->int8_ffn[j];
        P.L[j - l] = DecLayer{L->wq_gate, L->wq_up, L->s_gate, L->s_up,
                              L->delta_gu, L->wq_down, L->s_down, L->delta_down};
      }
      P.x_in = xin;
      if (l > 0) {
        const bool i8 = prec[l - 1] != 0;
        P.part_in = part;
        P.splits_in = splits_of(l - 1);
        P.part_f32_in = !i8;
        if (i8) {
          P.st_in = sh;
          P.si_in = desc->int8_ffn[l - 1].s_down;
        }
      }
      P.x_out = xbuf[nxt];
      P.part = (int32_t*)part;
      P.sh = sh;
      P.hidden = hidden;
      P.scratch = base + w.dec;
      P.layout = decode_layout(d, f, dec_splits);
      P.splits = dec_splits;
      P.ctl = (DecCtl*)(base + w.ctl);
      P.spin_limit = plan_override("DEC_SPIN_LIMIT", P.spin_limit);  // failure-path tests
      CHECK(hip_check(launch_decode_ffn(P, dec_grid, st), "decode_ffn"));
      xin = xbuf[nxt];  // the token stream after layer l1 - 2
      nxt ^= 1;
      for (int64_t j = l; j < l1; ++j) out_splits[j] = dec_splits;
      l = l1 - 1;
      continue;
    }
    out_splits[l] = prec[l] ? p8.splits : p16.splits;
    if (fused(l)) {
      const w8a8_ffn_desc* L = &desc->int8_ffn[l];
      QLoad ql;
      ql.delta = L->delta_gu;
      ql.g_x_in = xin;
      ql.g_x_out = xbuf[nxt];
      if (l > 0) {
        const bool i8 = prec[l - 1] != 0;
        ql.g_x_copy = hidden ? hidden + (l - 1) * m * d : nullptr;
        ql.g_part = part;
        ql.g_splits = splits_of(l - 1);
        ql.g_part_f32 = !i8;
        if (i8) {
          ql.g_st = sh;
          ql.g_si = desc->int8_ffn[l - 1].s_down;
        }
      }
      CHECK(run_gemm(pg8, DT_I8, EPI_GLU, nullptr, 0, m, L->wq_gate, L->wq_up, f, d, nullptr,
                     L->s_gate, L->s_up, h, f, nullptr, st, ql));
      xin = xbuf[nxt];
      nxt ^= 1;
    } else {
      CHECK(glue(l));
    }
    if (prec[l]) {
      const w8a8_ffn_desc* L = &desc->int8_ffn[l];
      if (!fused(l))
        CHECK(run_gemm(pg8, DT_I8, EPI_GLU, q, 0, m, L->wq_gate, L->wq_up, f, d, s, L->s_gate,
                       L->s_up, h, f, nullptr, st));
      if (plan_qloads(p8, m, f)) {
        CHECK(run_gemm_raw(p8, DT_I8, nullptr, 0, m, L->wq_down, d, f, part, st,
                           QLoad{h, L->delta_down, sh}));
      } else {
        CHECK(quant_act_impl(h, true, m, f, L->delta_down, qh, sh, st));
        CHECK(run_gemm_raw(p8, DT_I8, qh, 0, m, L->wq_down, d, f, part, st));
      }
    } else {
      const w8a8_bf16_ffn_desc* L = &desc->bf16_ffn[l];
      CHECK(run_gemm(pg16, DT_BF16, EPI_GLU, a, d, m, L->wp_gate, L->wp_up, f, d, nullptr, nullptr,
                     nullptr, h, f, nullptr, st));
      CHECK(run_gemm_raw(p16, DT_BF16, h, f, m, L->wp_down, d, f, part, st));
    }
  }
  const int64_t V = desc->vocab, nl = desc->n_layers;
  if (logits && lm_head_int8) {
    // At one token the final glue (the last layer's residual update, the
    // final RMSNorm and its quantisation) runs inside the INT8 lm_head's
    // streaming GEMM, as the layer glue does inside a gate/up GEMM: every
    // workgroup computes it for the row while its first weights arrive.
    const Plan pl = plan_gemm(m, V, d, DT_I8, false);
    const bool fuse_lm = m == 1 && !plan_override("NO_FUSED_GLUE", 0) && pl.stream &&
                         pl.mb == 1 && pl.splits == 1 && d % 8 == 0 && d / 8 <= 64 * pl.nw &&
                         (nl == 0 || splits_of(nl - 1) <= kGlueMaxSplits);
    if (fuse_lm) {
      QLoad ql;
      ql.delta = desc->lm_head_int8.delta;
      ql.g_x_in = xin;
      ql.g_x_out = xbuf[nxt];
      if (nl > 0) {
        const bool i8 = prec[nl - 1] != 0;
        ql.g_x_copy = hidden ? hidden + (nl - 1) * m * d : nullptr;
        ql.g_part = part;
        ql.g_splits = splits_of(nl - 1);
        ql.g_part_f32 = !i8;
        if (i8) {
          ql.g_st = sh;
          ql.g_si = desc->int8_ffn[nl - 1].s_down;
        }
      }
      return run_gemm(pl, DT_I8, EPI_BF16, nullptr, 0, m, desc->lm_head_int8.wq, nullptr, V, d,
                      nullptr, desc->lm_head_int8.s_w, nullptr, logits, V, base + w.lm, st, ql);
    }
  }
  CHECK(glue(nl));
  if (!logits) return W8A8_OK;
  if (lm_head_int8) {
    const Plan pl = plan_gemm(m, V, d, DT_I8, false);
    return run_gemm(pl, DT_I8, EPI_BF16, q, 0, m, desc->lm_head_int8.wq, nullptr, V, d, s,
                    desc->lm_head_int8.s_w, nullptr, logits, V, base + w.lm, st);
  }
  return bf16_linear_impl(a, m, desc->lm_head_bf16, V, d, logits, base + w.lm, st);
}

// Workspace of the sensitivity / selection calls: the stack's, two traces of
// the token stream, the FFN stage buffers, SQNR scratch and results.
struct SensWs {
  size_t stack, ref, quant, a, yb, y8, ffn, part, res, total;
};
SensWs sens_ws(int64_t m, int64_t d, int64_t f, int64_t vocab, int64_t n_layers) {
  SensWs w;
  const size_t trace = align256((size_t)n_layers * m * d * 2), act = align256((size_t)m * d * 2);
  w.stack = 0;
  w.ref = align256(w8a8_stack_workspace_bytes(m, d, f, vocab));
  w.quant = w.ref + trace;
  w.a = w.quant + trace;
  w.yb = w.a + act;
  w.y8 = w.yb + act;
  w.ffn = w.y8 + act;
  w.part = w.ffn + align256(std::max(w8a8_ffn_workspace_bytes(m, d, f),
                                     w8a8_bf16_ffn_workspace_bytes(m, d, f)));
  w.res = w.part + align256((size_t)2 * kSqnrMaxGroups * sizeof(double));
  w.total = w.res + align256((size_t)(2 * n_layers + 1) * 3 * sizeof(double));
  return w;
}

// SQNR results (3 doubles each) into res[slot]
w8a8_status sqnr_into(const void* ref, const void* test, int64_t n, char* base, const SensWs& w,
                      int64_t slot, hipStream_t st) {
  return hip_check(launch_sqnr(ref, test, true, n, (double*)(base + w.part),
                               (double*)(base + w.res) + 3 * slot, st),
                   "sqnr");
}

w8a8_status read_results(char* base, const SensWs& w, int64_t count, double* host,
                         hipStream_t st) {
  CHECK(hip_check(hipMemcpyAsync(host, base + w.res, (size_t)count * 3 * sizeof(double),
                                 hipMemcpyDeviceToHost, st),
                  "copy results"));
  return hip_check(hipStreamSynchronize(st), "synchronize");
}

// Reference trace (all layers bf16) and the isolated SQNR of every layer's
// FFN block on its reference input (results slots 0 .. n-1).
w8a8_status isolated_sensitivity(const w8a8_stack_desc* desc, const void* x, int64_t m, char* base,
                                 const SensWs& w, hipStream_t st) {
  const int64_t n = desc->n_layers, d = desc->d, f = desc->f;
  std::vector<uint8_t> bf(n, 0);
  uint16_t* ref = (uint16_t*)(base + w.ref);
  CHECK(stack_run(desc, bf.data(), 0, x, m, nullptr, ref, base + w.stack, st));
  const size_t ffn_bytes = std::max(w8a8_ffn_workspace_bytes(m, d, f),
                                    w8a8_bf16_ffn_workspace_bytes(m, d, f));
  for (int64_t l = 0; l < n; ++l) {
    const void* in = l == 0 ? x : (const void*)(ref + (l - 1) * m * d);
    CHECK(hip_check(launch_rmsnorm(nullptr, (const uint16_t*)in, m, d, (uint16_t*)(base + w.a), st),
                    "rmsnorm"));
    CHECK(w8a8_bf16_ffn(&desc->bf16_ffn[l], base + w.a, m, base + w.yb, base + w.ffn, ffn_bytes,
                        st));
    CHECK(w8a8_ffn(&desc->int8_ffn[l], base + w.a, m, base + w.y8, base + w.ffn, ffn_bytes, st));
    CHECK(sqnr_into(base + w.yb, base + w.y8, m * d, base, w, l, st));
  }
  return W8A8_OK;
}

}  // namespace

extern "C" {

w8a8_status w8a8_ffn_stack(const w8a8_stack_desc* desc, const uint8_t* prec, int lm_head_int8,
                           const void* x, int64_t m, void* logits, void* ws, size_t ws_bytes,
                           w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_stack(desc, prec, lm_head_int8, true));
  CHECK_PTR(x);
  CHECK_PTR(logits);
  CHECK_PTR(ws);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  REQUIRE(ws_bytes >= w8a8_stack_workspace_bytes(m, desc->d, desc->f, desc->vocab),
          W8A8_EWORKSPACE, "workspace too small");
  return stack_run(desc, prec, lm_head_int8, x, m, logits, nullptr, ws, S(stream));
}

w8a8_status w8a8_ffn_stack_status(const void* ws, size_t ws_bytes, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(ws);
  REQUIRE(ws_bytes >= sizeof(DecCtl), W8A8_EWORKSPACE, "workspace smaller than its status block");
  unsigned word = 0;
  const DecCtl* ctl = (const DecCtl*)ws;  // at the start of the stack workspace
  CHECK(hip_check(hipStreamSynchronize(S(stream)), "hipStreamSynchronize"));
  CHECK(hip_check(hipMemcpy(&word, &ctl->fail[0], sizeof(word), hipMemcpyDeviceToHost),
                  "hipMemcpy"));
  if (word != 0)
    return fail(W8A8_ETIMEOUT, "the persistent decode kernel gave up waiting at a grid barrier; "
                               "that call's token stream and logits are NaN");
  return W8A8_OK;
}

w8a8_status w8a8_ffn_stack_trace(const w8a8_stack_desc* desc, const uint8_t* prec,
                                 int lm_head_int8, const void* x, int64_t m, void* logits,
                                 void* hidden, void* ws, size_t ws_bytes, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_stack(desc, prec, lm_head_int8, logits != nullptr));
  CHECK_PTR(x);
  if (logits) CHECK_PTR(logits);
  CHECK_PTR(hidden);
  CHECK_PTR(ws);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  REQUIRE(ws_bytes >= w8a8_stack_workspace_bytes(m, desc->d, desc->f, desc->vocab),
          W8A8_EWORKSPACE, "workspace too small");
  return stack_run(desc, prec, lm_head_int8, x, m, logits, (uint16_t*)hidden, ws, S(stream));
}

size_t w8a8_sqnr_workspace_bytes(int64_t n) {
  if (n < 1) return 0;
  return (size_t)2 * sqnr_groups(n) * sizeof(double);
}

w8a8_status w8a8_sqnr(const void* ref, const void* test, w8a8_dtype dtype, int64_t n, double* out,
                      void* ws, size_t ws_bytes, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(ref);
  CHECK_PTR(test);
  CHECK_PTR(out);
  CHECK_PTR(ws);
  REQUIRE(n >= 1, W8A8_EINVAL, "n < 1");
  REQUIRE(dtype == W8A8_F32 || dtype == W8A8_BF16, W8A8_EUNSUPPORTED, "dtype");
  REQUIRE(ws_bytes >= w8a8_sqnr_workspace_bytes(n), W8A8_EWORKSPACE, "workspace too small");
  return hip_check(launch_sqnr(ref, test, dtype == W8A8_BF16, n, (double*)ws, out, S(stream)),
                   "sqnr");
}

size_t w8a8_stack_sensitivity_workspace_bytes(int64_t m, int64_t d, int64_t f, int64_t vocab,
                                              int64_t n_layers) {
  if (m < 1 || d < 1 || f < 1 || vocab < 1 || n_layers < 1) return 0;
  return sens_ws(m, d, f, vocab, n_layers).total;
}

static w8a8_status check_sens(const w8a8_stack_desc* desc, const void* x, int64_t m, void* ws,
                              size_t ws_bytes) {
  REQUIRE(desc, W8A8_EINVAL, "desc is NULL");
  std::vector<uint8_t> all(desc->n_layers > 0 ? desc->n_layers : 1, 1), none(all.size(), 0);
  CHECK(check_stack(desc, all.data(), 0, false));   // every layer needs both forms
  CHECK(check_stack(desc, none.data(), 0, false));
  CHECK_PTR(x);
  CHECK_PTR(ws);
  REQUIRE(m >= 1, W8A8_EINVAL, "m < 1");
  REQUIRE(ws_bytes >= w8a8_stack_sensitivity_workspace_bytes(m, desc->d, desc->f, desc->vocab,
                                                             desc->n_layers),
          W8A8_EWORKSPACE, "workspace too small");
  return W8A8_OK;
}

w8a8_status w8a8_stack_sensitivity(const w8a8_stack_desc* desc, const uint8_t* prec,
                                   const void* x, int64_t m, float* isolated_db,
                                   float* propagated_db, void* ws, size_t ws_bytes,
                                   w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_sens(desc, x, m, ws, ws_bytes));
  REQUIRE(prec || !propagated_db, W8A8_EINVAL, "prec is NULL");
  const int64_t n = desc->n_layers, d = desc->d;
  hipStream_t st = S(stream);
  char* base = (char*)ws;
  const SensWs w = sens_ws(m, d, desc->f, desc->vocab, n);
  CHECK(isolated_sensitivity(desc, x, m, base, w, st));  // also leaves the reference trace
  if (propagated_db) {
    uint16_t* ref = (uint16_t*)(base + w.ref);
    uint16_t* quant = (uint16_t*)(base + w.quant);
    CHECK(stack_run(desc, prec, 0, x, m, nullptr, quant, base + w.stack, st));
    for (int64_t l = 0; l < n; ++l)
      CHECK(sqnr_into(ref + l * m * d, quant + l * m * d, m * d, base, w, n + l, st));
  }
  std::vector<double> res((size_t)(2 * n) * 3);
  CHECK(read_results(base, w, propagated_db ? 2 * n : n, res.data(), st));
  for (int64_t l = 0; l < n; ++l) {
    if (isolated_db) isolated_db[l] = (float)res[3 * l + 2];
    if (propagated_db) propagated_db[l] = (float)res[3 * (n + l) + 2];
  }
  return W8A8_OK;
}

w8a8_status w8a8_select_precision_map(const w8a8_stack_desc* desc, const void* x, int64_t m,
                                      float budget_db, uint8_t* prec, float* final_db, void* ws,
                                      size_t ws_bytes, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK(check_sens(desc, x, m, ws, ws_bytes));
  REQUIRE(prec, W8A8_EINVAL, "prec is NULL");
  const int64_t n = desc->n_layers, d = desc->d;
  hipStream_t st = S(stream);
  char* base = (char*)ws;
  const SensWs w = sens_ws(m, d, desc->f, desc->vocab, n);
  CHECK(isolated_sensitivity(desc, x, m, base, w, st));
  std::vector<double> res((size_t)(2 * n + 1) * 3);
  CHECK(read_results(base, w, n, res.data(), st));
  std::vector<float> iso(n);
  for (int64_t l = 0; l < n; ++l) iso[l] = (float)res[3 * l + 2];
  std::vector<int> order(n);
  w8a8_rank_layers(iso.data(), (int)n, order.data());
  // most robust layers first; a layer stays INT8 while the last layer's
  // output keeps at least budget_db against the all-bf16 stack
  uint16_t* ref_last = (uint16_t*)(base + w.ref) + (n - 1) * m * d;
  uint16_t* quant = (uint16_t*)(base + w.quant);
  for (int64_t l = 0; l < n; ++l) prec[l] = 0;
  double best = INFINITY;
  for (int64_t i = 0; i < n; ++i) {
    const int l = order[i];
    prec[l] = 1;
    CHECK(stack_run(desc, prec, 0, x, m, nullptr, quant, base + w.stack, st));
    CHECK(sqnr_into(ref_last, quant + (n - 1) * m * d, m * d, base, w, 2 * n, st));
    std::vector<double> r(3);
    CHECK(hip_check(hipMemcpyAsync(r.data(), (double*)(base + w.res) + 3 * (2 * n), 3 * sizeof(double),
                                   hipMemcpyDeviceToHost, st),
                    "copy result"));
    CHECK(hip_check(hipStreamSynchronize(st), "synchronize"));
    if (r[2] >= (double)budget_db)
      best = r[2];
    else
      prec[l] = 0;
  }
  if (final_db) final_db[0] = (float)best;
  return W8A8_OK;
}

int w8a8_rank_layers(const float* isolated_db, int n_layers, int* order) {
  if (!isolated_db || !order || n_layers < 1) return -1;
  for (int i = 0; i < n_layers; ++i) order[i] = i;
  // descending SQNR (most robust first), NaN last, ties by layer index
  auto key = [&](int i) { return std::isnan(isolated_db[i]) ? -INFINITY : isolated_db[i]; };
  std::stable_sort(order, order + n_layers, [&](int a, int b) { return key(a) > key(b); });
  return 0;
}

// ---------------------------------------------------------------- f4: key/value cache and attention decode

size_t w8a8_attn_decode_workspace_bytes(int64_t t_max) {
  return t_max >= 1 ? attn_ws_bytes_max(t_max) : 0;
}

w8a8_status w8a8_kv_quantize(const void* kv, int64_t rows, int64_t ld, int8_t* codes,
                             float* scales, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(kv);
  CHECK_PTR(codes);
  // one binary32 store per row: a slice of a scale array need only be 4-byte aligned
  REQUIRE(scales && ((uintptr_t)scales & 3) == 0, W8A8_EINVAL, "scales is NULL or not 4-byte aligned");
  REQUIRE(rows >= 1, W8A8_EINVAL, "rows < 1");
  REQUIRE(ld >= W8A8_HEAD_DIM && ld % 8 == 0, W8A8_EINVAL, "ld must be >= 256 and a multiple of 8");
  return hip_check(launch_kv_quant((const uint16_t*)kv, rows, ld, codes, scales, S(stream)),
                   "kv_quant");
}

namespace {
// workgroups the rows of a decode attention are split over (measured at 4
// heads: 131072 rows 43.6 us with 256, 33.2 us with 512; 32768 rows equal)
int attn_wg_target() { return plan_override("ATTN_WGS", 512); }

w8a8_status attn_common(const void* qkv, int n_heads, int64_t pos, int64_t window, int64_t t_max,
                        void* out, void* ws, size_t ws_bytes, AttnParams* p) {
  CHECK_PTR(qkv);
  CHECK_PTR(out);
  REQUIRE(n_heads == 1 || n_heads == 2 || n_heads == 4 || n_heads == 8, W8A8_EUNSUPPORTED,
          "n_heads must be 1, 2, 4 or 8");
  REQUIRE(t_max >= 1 && pos >= 0 && pos < t_max, W8A8_EINVAL, "pos outside [0, t_max)");
  REQUIRE(window >= 1, W8A8_EINVAL, "window < 1");
  p->qkv = (const uint16_t*)qkv;
  p->out = (uint16_t*)out;
  p->pos = pos;
  p->t0 = std::max<int64_t>(0, pos + 1 - window);
  const size_t need = attn_ws_bytes(pos + 1 - p->t0, attn_wg_target());
  if (need) {
    CHECK_PTR(ws);
    REQUIRE(ws_bytes >= need, W8A8_EWORKSPACE, "workspace too small");
  }
  p->part = (float*)ws;
  return W8A8_OK;
}
}  // namespace

w8a8_status w8a8_attn_decode(const void* qkv, int n_heads, int64_t pos, int64_t window,
                             int8_t* k_codes, float* k_scales, int8_t* v_codes, float* v_scales,
                             int64_t t_max, void* out, void* ws, size_t ws_bytes,
                             w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(k_codes);
  CHECK_PTR(v_codes);
  CHECK_PTR(k_scales);
  CHECK_PTR(v_scales);
  AttnParams p;
  CHECK(attn_common(qkv, n_heads, pos, window, t_max, out, ws, ws_bytes, &p));
  p.k = k_codes;
  p.v = v_codes;
  p.sk = k_scales;
  p.sv = v_scales;
  return hip_check(launch_attn_decode(p, n_heads, true, attn_wg_target(), S(stream)), "attn_decode");
}

w8a8_status w8a8_attn_decode_bf16(const void* qkv, int n_heads, int64_t pos, int64_t window,
                                  void* k_rows, void* v_rows, int64_t t_max, void* out, void* ws,
                                  size_t ws_bytes, w8a8_stream_t stream) {
  g_last_error.clear();
  CHECK_PTR(k_rows);
  CHECK_PTR(v_rows);
  AttnParams p;
  CHECK(attn_common(qkv, n_heads, pos, window, t_max, out, ws, ws_bytes, &p));
  p.k = k_rows;
  p.v = v_rows;
  return hip_check(launch_attn_decode(p, n_heads, false, attn_wg_target(), S(stream)),
                   "attn_decode_bf16");
}

}  // extern "C"

// rows per workgroup of the many-row bf16 quantiser (declared in kernels.h)
int w8a8::quant_rows_per_workgroup(int dflt) { return plan_override("QROWS_R", dflt); }
