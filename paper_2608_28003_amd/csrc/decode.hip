// Persistent decode kernel: a run of consecutive INT8 FFN blocks of the stack
// (Sec. 5, the per-layer precision map) for one token in a single launch.
//
// At one token every GEMM of the block is a matrix-vector product whose
// weights stream from HBM once; with one launch per GEMM the step is bound by
// launch and first-load latency, not by bandwidth.  Here one workgroup per CU
// stays resident for the whole run and the layers' phases are separated by
// grid-wide barriers:
//
//   phase G (layer l): the layer glue for the row (previous layer's down sums
//     -> dequant -> post-norm residual update of the token stream -> pre-norm
//     -> smoothing by delta_gu -> per-token codes), then the gate/up
//     products of this workgroup's 16-column items and the GeGLU epilogue,
//     h = bf16(gelu_tanh(g) * u), written to global memory with the item's
//     absmax of h / delta_down;
//   phase D (layer l): per-token quantisation of h (smoothed by delta_down,
//     scale over the whole row: the maximum of the item maxima) for this
//     workgroup's K range, then the down products of its (column block,
//     K split) item, written as int32 partial sums that the next layer's
//     glue adds.
//
// Every weight fragment a workgroup needs in a phase is loaded into registers
// before the barrier that opens the phase, so the weight stream overlaps the
// synchronisation.  The arithmetic is that of the per-launch path (the glue
// and quantise-on-load helpers are shared, int32 sums are exact in any order,
// the epilogues use the same binary32 expressions), so the results are
// bit-identical to it.
//
// Barriers: every workgroup adds one to its group's arrival counter (4
// groups, one 256-byte line each); the last arrival of a group adds one to a
// top counter, which the waiting workgroups poll.  Every wait is bounded:
// past the spin limit, or when another workgroup has given up, a workgroup
// sets the error word and returns, so the grid always drains; workgroup 0
// then fills the run's outputs with NaN (the token stream and the token
// scale), so that every value computed from them downstream is NaN.  The
// host launches the kernel only when every workgroup fits on the device at
// once.
//
// Data passed between workgroups goes through per-layer buffers that no one
// reads before the barrier that publishes them, each 128-byte line written
// by one workgroup with a device-scope store that goes through to memory.
// Readers then use ordinary loads: a line cannot sit stale in any cache, and
// the 32 workgroups of an XCD share one fetch of it through their L2.  (A
// device-scope release / acquire pair per barrier -- an L2 write-back and
// invalidation -- cost tens of microseconds per barrier; device-scope loads
// for the broadcast data sent every workgroup's request to memory.)
#include "device.h"
#include "kernels.h"
#include "rowquant.h"

namespace w8a8 {

namespace {

constexpr int kDecNW = 8;  // waves per workgroup
constexpr int kDecThreads = 64 * kDecNW;

__global__ void dec_clear_kernel(DecCtl* ctl) {
  if (threadIdx.x < kDecGroups) ctl->grp[threadIdx.x][0] = 0u;
  if (threadIdx.x == 0) {
    ctl->top[0] = 0u;
    ctl->err[0] = 0u;
  }
}

__global__ void dec_status_clear_kernel(DecCtl* ctl) {
  if (threadIdx.x == 0) ctl->fail[0] = 0u;
}

// Arrival at barrier k (1, 2, ...): every wave waits until its own stores are
// complete, then one thread adds one to the group counter; the group's last
// arrival (the counter reaching k times the group size) adds one to the top.
__device__ __forceinline__ void grid_arrive(DecCtl* ctl, unsigned k) {
  __builtin_amdgcn_s_waitcnt(0);  // vmcnt, expcnt and lgkmcnt all zero
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned g = blockIdx.x % kDecGroups;
    const unsigned size = (gridDim.x - g + kDecGroups - 1) / kDecGroups;
    const unsigned old =
        __hip_atomic_fetch_add(&ctl->grp[g][0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old + 1 == k * size)
      __hip_atomic_fetch_add(&ctl->top[0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Wait for barrier k; false if this workgroup gave up (spin limit reached or
// the error word set by another workgroup).
__device__ __forceinline__ bool grid_wait(DecCtl* ctl, unsigned k, int spin_limit) {
  __shared__ int s_ok;
  if (threadIdx.x == 0) {
    const unsigned groups = min((unsigned)kDecGroups, gridDim.x);
    int ok = 1;
    for (int it = 0;; ++it) {
      if (__hip_atomic_load(&ctl->top[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >=
          k * groups)
        break;
      if (it >= spin_limit ||
          __hip_atomic_load(&ctl->err[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u) {
        __hip_atomic_store(&ctl->err[0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&ctl->fail[0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    s_ok = ok;
  }
  __syncthreads();
  return s_ok != 0;
}

// After a failed wait workgroup 0 fills the run's outputs with NaN (the other
// workgroups return without writing them).
__device__ __forceinline__ void poison(const DecParams& P) {
  if (blockIdx.x != 0) return;
  for (int c = threadIdx.x; c < P.d; c += kDecThreads) P.x_out[c] = 0x7fc0u;
  if (threadIdx.x == 0) P.sh[0] = __builtin_nanf("");
}

// Columns of a row one thread handles in the spread quantisation below
// (column c = t + 512 i): rows of up to 2560 values.
constexpr int kDecCols = 5;

// Byte of the LDS panel that holds the code of column c of row 0.
__device__ __forceinline__ int panel_byte(int c) {
  return ((c / kFragK8) * 64 + 16 * ((c % kFragK8) / 16)) * 16 + (c % 16);
}

// The layer glue of one token row.  The token-stream update and both
// RMSNorm sums run on the threads that own 8 consecutive columns, in the order
// of glue_panel (and of the glue kernel); the smoothing division, the absmax
// and the codes then run over all threads of the workgroup, one column each
// per step, with the same binary32 operations, so the codes and the scale are
// identical while each thread does a third of the divisions.
__device__ __forceinline__ void dec_glue(const GemmParams& p, const GlueRegs& R,
                                         const float (&dk)[kDecCols], v4i* lds_a, float* xs,
                                         float* s_row) {
  __shared__ float red_x[kDecNW], red_q[kDecNW];
  const int t = threadIdx.x, d = p.a_k;
  const bool own = t < d / 8;
  float xv[8];
  glue_stream<kDecNW, true>(p, R, xv);
  float ss = 0.0f;
  if (own) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      ss += xv[e] * xv[e];
      xs[t * 8 + e] = xv[e];
    }
  }
  ss = block_sum_in(ss, red_x);  // its barrier also publishes xs
  const float inv = 1.0f / sqrtf(ss / (float)d + 1e-6f);
  float a[kDecCols];
  float amax = 0.0f;
#pragma unroll
  for (int i = 0; i < kDecCols; ++i) {
    const int c = t + kDecThreads * i;
    a[i] = 0.0f;
    if (c < d) {
      a[i] = bf16_bits_to_float(float_to_bf16_bits(xs[c] * inv));
      if (p.a_delta) a[i] = a[i] / dk[i];
      amax = fmaxf(amax, fabsf(a[i]));
    }
  }
  amax = block_max_in(amax, red_q);
  const float sr = amax / 127.0f;
  if (t == 0) s_row[0] = sr;
  const float sinv = 1.0f / sr;
  const bool fast = isfinite(sinv);
  int8_t* bytes = reinterpret_cast<int8_t*>(lds_a);
#pragma unroll
  for (int i = 0; i < kDecCols; ++i) {
    const int c = t + kDecThreads * i;
    if (c < d) bytes[panel_byte(c)] = sr != 0.0f ? code_of(a[i], sr, sinv, fast) : (int8_t)0;
  }
}

// Per-token quantisation of the FFN intermediate h for the down phase: the
// scale comes from the whole row, max |h / delta| / 127, the codes only for
// the fragment columns [kb0, kb0 + kc).  The gate/up epilogue has left, with
// every 16-column item of h, the absmax of its smoothed values (the same
// binary32 quotients); thread t < f / 16 brings item t's values and absmax
// (hv, pmax), the workgroup maximum of the item maxima is the row's, and the
// codes of the K range are formed one column per thread from the staged h
// and the smoothing factors dk (column kb0 * 64 + t + 512 i), with
// quantize_panel's binary32 operations, so the codes and the scale are
// identical to it.
__device__ __forceinline__ void dec_quant(uint4 h0, uint4 h1, float pmax,
                                          const float (&dk)[kDecCols], bool has_delta, int f,
                                          int kb0, int kc, v4i* lds_a, uint16_t* hs, float* s_row,
                                          float* s_out) {
  __shared__ float red_m[kDecNW];
  const int t = threadIdx.x;
  const bool item = t < f / 16;
  const int i0 = kb0 * (kFragK8 / 16), i1 = (kb0 + kc) * (kFragK8 / 16);
  if (item && t >= i0 && t < i1) {
    uint4* dst = reinterpret_cast<uint4*>(hs + (t - i0) * 16);
    dst[0] = h0;
    dst[1] = h1;
  }
  const float amax = block_max_in(item ? pmax : 0.0f, red_m);  // its barrier also publishes hs
  const float sr = amax / 127.0f;
  if (t == 0) {
    s_row[0] = sr;
    if (s_out && blockIdx.x == 0) st_f32<true>(s_out, sr);
  }
  const float sinv = 1.0f / sr;
  const bool fast = isfinite(sinv);
  int8_t* bytes = reinterpret_cast<int8_t*>(lds_a);
#pragma unroll
  for (int i = 0; i < kDecCols; ++i) {
    const int c = t + kDecThreads * i;
    if (c < kc * kFragK8) {
      float v = bf16_bits_to_float(hs[c]);
      if (has_delta) v = v / dk[i];
      bytes[panel_byte(c)] = sr != 0.0f ? code_of(v, sr, sinv, fast) : (int8_t)0;
    }
  }
}

__global__ __launch_bounds__(kDecThreads) void decode_ffn_kernel(DecParams P) {
  __shared__ v4i lds_a[kDecMaxPanel * 64];
  __shared__ v4i red[kDecNW * 64];
  __shared__ float s_row[16];
  __shared__ float xs[kDecMaxPanel * kFragK8];  // glue: the token stream; down: h of the K range
  const int lane = lane_id(), wave = threadIdx.x >> 6;
  const int G = gridDim.x, b = blockIdx.x;
  const int d = P.d, f = P.f;
  const int kbd = d / kFragK8, kbf = f / kFragK8;

  // gate/up items (16 h columns, gate and up fragments over all of K):
  // b, b + G, ...; the waves of the workgroup are dealt to its items, Q per
  // item, wave q of an item taking operand q & 1 (0 gate, 1 up) and the K
  // fragments q / 2, q / 2 + Q / 2, ...
  const int ng = f / 16;
  const int n_gi = b < ng ? min(4, (ng - b + G - 1) / G) : 0;
  const int Q = n_gi ? (kDecNW / n_gi) & ~1 : 2;
  const int g_local = wave / Q, q = wave % Q;
  const bool g_wave = g_local < n_gi;
  const int g_item = b + g_local * G;
  const int g_k0 = q >> 1, g_ks = Q >> 1;
  const int g_cnt = g_wave && g_k0 < kbd ? (kbd - g_k0 + g_ks - 1) / g_ks : 0;
  const int g_col = min(g_item, ng - 1) * 16 + (lane & 15);

  // down item: column block b % ncd, K split b / ncd (kcd fragments each);
  // wave w takes the split's fragments w, w + 8, ...
  const int ncd = d / 16;
  const int kcd = kbf / P.splits;
  const bool d_item = b < ncd * P.splits;
  const int d_c = b % ncd, d_z = b / ncd;
  const int d_k0 = d_z * kcd;
  const int d_cnt = d_item && wave < kcd ? (kcd - wave + kDecNW - 1) / kDecNW : 0;

  v4i w[kDecMaxFrags];
  float sg = 0.0f, su = 0.0f, sdd = 1.0f;
  GlueRegs gr;
  // smoothing factors of the columns t + 512 i of the phase's row: the glue's
  // (delta_gu) in phase G, the K range's (delta_down) in phase D
  float dk[kDecCols];

  auto load_g = [&](const DecLayer& L) {
    const void* src = (q & 1) ? L.wu : L.wg;
#pragma unroll
    for (int j = 0; j < kDecMaxFrags; ++j)
      if (j < g_cnt) w[j] = load_frag_packed(src, g_item, g_k0 + j * g_ks, kbd, lane);
    sg = L.sg[g_col];
    su = L.su[g_col];
    if (L.dd) sdd = L.dd[g_col];  // smoothing of the epilogue's h column (down input)
    const float* dsrc = L.dgu ? L.dgu : reinterpret_cast<const float*>(L.wg);  // >= 4 d bytes
#pragma unroll
    for (int i = 0; i < kDecCols; ++i) dk[i] = dsrc[min((int)threadIdx.x + kDecThreads * i, d - 1)];
  };
  // the down weights and the smoothing factors of the K range (read-only:
  // loaded ahead of the barrier)
  const int qg = min((int)threadIdx.x, f / 16 - 1);  // this thread's item of h
  auto load_d = [&](const DecLayer& L) {
#pragma unroll
    for (int j = 0; j < kDecMaxFrags; ++j)
      if (j < d_cnt) w[j] = load_frag_packed(L.wd, d_c, d_k0 + wave + j * kDecNW, kbf, lane);
    const float* dsrc = L.dd ? L.dd + d_k0 * kFragK8 : L.sd;
    const int lim = L.dd ? kcd * kFragK8 : d;
#pragma unroll
    for (int i = 0; i < kDecCols; ++i) dk[i] = dsrc[min((int)threadIdx.x + kDecThreads * i, lim - 1)];
  };

  // layer j's exchange buffers
  auto xbuf = [&](int jj) { return reinterpret_cast<uint16_t*>(P.scratch + (size_t)jj * P.layout.layer_bytes); };
  auto pbuf = [&](int jj) {
    return reinterpret_cast<int32_t*>(P.scratch + (size_t)jj * P.layout.layer_bytes + P.layout.part);
  };
  auto sbuf = [&](int jj) {
    return reinterpret_cast<float*>(P.scratch + (size_t)jj * P.layout.layer_bytes + P.layout.sh);
  };
  auto hbuf = [&](int jj) {
    return reinterpret_cast<uint16_t*>(P.scratch + (size_t)jj * P.layout.layer_bytes + P.layout.h);
  };
  const int last = P.n_layers - 1;

  unsigned k = 0;  // the last barrier this workgroup arrived at
  if (n_gi) load_g(P.L[0]);
  for (int j = 0; j < P.n_layers; ++j) {
    const DecLayer& L = P.L[j];
    const int l = P.l0 + j;  // index of this layer in the stack
    // ---------------- phase G
    if (j > 0 && !grid_wait(P.ctl, k, P.spin_limit)) return poison(P);
    if (n_gi) {
      GemmParams p{};
      p.M = 1;
      p.B = L.wg;
      p.a_k = d;
      p.a_delta = L.dgu;
      p.g_x_out = j == last ? P.x_out : xbuf(j);
      p.g_x_copy = (P.hidden && l > 0) ? P.hidden + (int64_t)(l - 1) * d : nullptr;
      if (j == 0) {  // the launch's input (written by earlier launches)
        p.g_x_in = P.x_in;
        p.g_part = P.part_in;
        p.g_splits = P.splits_in;
        p.g_part_f32 = P.part_f32_in;
        p.g_st = P.st_in;
        p.g_si = P.si_in;
        glue_fetch(p, gr);
      } else {
        p.g_x_in = xbuf(j - 1);
        p.g_part = pbuf(j - 1);
        p.g_splits = P.splits;
        p.g_part_f32 = 0;
        p.g_st = sbuf(j - 1);
        p.g_si = P.L[j - 1].sd;
        glue_fetch<32>(p, gr, ncd);
      }
      dec_glue(p, gr, dk, lds_a, xs, s_row);
      __syncthreads();
      v4i acc = {0, 0, 0, 0};
#pragma unroll
      for (int i = 0; i < kDecMaxFrags; ++i)
        if (i < g_cnt) acc = mma_i8(lds_a[(g_k0 + i * g_ks) * 64 + lane], w[i], acc);
      red[wave * 64 + lane] = acc;
      __syncthreads();
      // GeGLU epilogue of each item by its first wave (row 0: lanes 0..15)
      if (g_wave && q == 0 && lane < 16) {
        int gs = 0, us = 0;
        for (int r = 0; r < Q; ++r) {
          const int v = red[(wave + r) * 64 + lane][0];
          if (r & 1)
            us += v;
          else
            gs += v;
        }
        const float gv = ((float)gs * s_row[0]) * sg;
        const float uv = ((float)us * s_row[0]) * su;
        const uint32_t hb = float_to_bf16_bits(gelu_tanh(gv) * uv);
        const uint32_t hn = __shfl_down(hb, 1, 16);  // the odd neighbour's column
        if (!(lane & 1))
          __hip_atomic_store(reinterpret_cast<uint32_t*>(hbuf(j) + g_item * 64 + lane),
                             hb | (hn << 16), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        // absmax of the item's smoothed values (the down input's quotients),
        // over lanes 0..15, stored after the values in the item's line
        float hm = bf16_bits_to_float(hb);
        if (L.dd) hm = hm / sdd;
        hm = fabsf(hm);
        hm = fmaxf(hm, lane_xor<8>(hm));
        hm = fmaxf(hm, lane_xor<4>(hm));
        hm = fmaxf(hm, lane_xor<2>(hm));
        hm = fmaxf(hm, lane_xor<1>(hm));
        if (lane == 0)
          __hip_atomic_store(reinterpret_cast<uint32_t*>(hbuf(j) + g_item * 64 + 16),
                             __float_as_uint(hm), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    grid_arrive(P.ctl, ++k);
    if (d_item) load_d(L);
    // ---------------- phase D
    if (!grid_wait(P.ctl, k, P.spin_limit)) return poison(P);
    if (d_item) {
      const uint16_t* xr = hbuf(j) + qg * 64;
      const uint4 h0 = *reinterpret_cast<const uint4*>(xr);
      const uint4 h1 = *reinterpret_cast<const uint4*>(xr + 8);
      const float pmax = *reinterpret_cast<const float*>(xr + 16);
      dec_quant(h0, h1, pmax, dk, L.dd != nullptr, f, d_k0, kcd, lds_a,
                reinterpret_cast<uint16_t*>(xs), s_row, j == last ? P.sh : sbuf(j));
      __syncthreads();
      v4i acc = {0, 0, 0, 0};
#pragma unroll
      for (int i = 0; i < kDecMaxFrags; ++i)
        if (i < d_cnt) acc = mma_i8(lds_a[(wave + i * kDecNW) * 64 + lane], w[i], acc);
      red[wave * 64 + lane] = acc;
      __syncthreads();
      if (wave == 0 && lane < 16) {
        int sum = 0;
        for (int r = 0; r < kDecNW; ++r) sum += red[r * 64 + lane][0];
        int32_t* dst = j == last ? P.part + (int64_t)d_z * d + d_c * 16 + lane
                                 : pbuf(j) + (d_z * ncd + d_c) * 32 + lane;
        __hip_atomic_store(dst, sum, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    grid_arrive(P.ctl, ++k);
    if (j < last && n_gi) load_g(P.L[j + 1]);
  }
  // Workgroup 0 waits for every workgroup's last arrival: a workgroup that
  // gave up returns without arriving, so this wait fails too and the outputs
  // are poisoned after every other workgroup has stopped writing.
  if (b == 0 && !grid_wait(P.ctl, k, P.spin_limit)) poison(P);
}

}  // namespace

int decode_grid(int device) {
  static int cached[64];
  static bool known[64];
  if (device < 0 || device >= 64) return 0;
  if (known[device]) return cached[device];
  int cus = 0, occ = 0;
  int g = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) == hipSuccess &&
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, decode_ffn_kernel, kDecThreads, 0) ==
          hipSuccess &&
      occ >= 1)
    g = cus;
  cached[device] = g;
  known[device] = true;
  return g;
}

int decode_splits(int64_t d, int64_t f, int grid) {
  if (grid < 1 || d % kFragK8 || f % kFragK8) return 0;
  const int64_t kbd = d / kFragK8, kbf = f / kFragK8, ng = f / 16, ncd = d / 16;
  if (d > (int64_t)kDecCols * kDecThreads || ng > kDecThreads || kbd > kDecMaxPanel) return 0;
  // gate/up: at most 4 items per workgroup, fragments per wave within the
  // register budget
  const int64_t n_gi = (ng + grid - 1) / grid;
  if (n_gi > 4) return 0;
  const int64_t Q = (kDecNW / n_gi) & ~1;
  if ((kbd + Q / 2 - 1) / (Q / 2) > kDecMaxFrags) return 0;
  // down: the most K splits (up to what the glue adds) that still give every
  // item its own workgroup and divide K evenly
  for (int s = kGlueMaxSplits; s >= 1; --s) {
    if (ncd * s > grid || kbf % s) continue;
    const int64_t kcd = kbf / s;
    if (kcd > kDecMaxPanel || kcd * kFragK8 > kDecCols * kDecThreads ||
        (kcd + kDecNW - 1) / kDecNW > kDecMaxFrags)
      continue;
    return s;
  }
  return 0;
}

DecLayout decode_layout(int64_t d, int64_t f, int splits) {
  auto a256 = [](size_t v) { return (v + 255) / 256 * 256; };
  DecLayout L;
  L.part = a256((size_t)d * 2);
  L.sh = L.part + a256((size_t)splits * (d / 16) * 128);
  L.h = L.sh + 256;
  L.layer_bytes = L.h + a256((size_t)(f / 16) * 128);
  return L;
}

hipError_t launch_decode_ffn(const DecParams& P, int grid, hipStream_t st) {
  const DecLayout want = decode_layout(P.d, P.f, P.splits);
  if (P.n_layers < 1 || P.n_layers > kDecMaxLayers || grid < 1 || !P.ctl || !P.scratch ||
      !P.part || !P.sh || !P.x_out || !P.x_in || P.splits != decode_splits(P.d, P.f, grid) ||
      P.layout.layer_bytes != want.layer_bytes || P.layout.part != want.part ||
      P.layout.sh != want.sh || P.layout.h != want.h || P.splits_in < 0 ||
      P.splits_in > kGlueMaxSplits || (P.splits_in > 0 && !P.part_in))
    return hipErrorInvalidValue;
  for (int j = 0; j < P.n_layers; ++j) {
    const DecLayer& L = P.L[j];
    if (!L.wg || !L.wu || !L.sg || !L.su || !L.wd || !L.sd) return hipErrorInvalidValue;
  }
  dec_clear_kernel<<<1, 64, 0, st>>>(P.ctl);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  decode_ffn_kernel<<<grid, kDecThreads, 0, st>>>(P);
  return hipGetLastError();
}

hipError_t launch_dec_status_clear(DecCtl* ctl, hipStream_t st) {
  dec_status_clear_kernel<<<1, 64, 0, st>>>(ctl);
  return hipGetLastError();
}

}  // namespace w8a8
