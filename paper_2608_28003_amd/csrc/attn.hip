// One-token attention over a key/value cache, with the cache held as INT8
// codes and per-row scales or as bf16 rows (Sec. 4 names the INT8 key/value
// cache among the further speed-ups; Sec. 2: four query heads share one
// key/value head of 256, grouped-query attention).
//
// The cache of one layer is a row-major array of t_max rows of 256: INT8
// codes (256 B a row) with one binary32 scale per row, or bf16 (512 B a row).
// A decode step appends the current token's key and value at row pos and
// attends rows t0 .. pos with every query head.  The work is split over the
// rows: each workgroup walks its range in passes of 64 rows with a running
// maximum and sum per head (the softmax is formed exactly as one pass would
// form it, up to binary32 rounding), and a second launch merges the
// workgroups' partial results.  The workgroup whose range holds row pos
// quantises (or copies) the new key and value, stores them in the cache and
// uses them from LDS, so no other workgroup reads the row being written.
#include <algorithm>

#include "device.h"
#include "kernels.h"

namespace w8a8 {

namespace {

constexpr int kHd = 256;       // head dimension
constexpr int kPass = 64;      // cached rows per pass of a workgroup (16 per wave)
constexpr int kMaxHeads = 8;
// q in LDS with 4 floats of padding after every 64: the four lanes of a row
// read 64 apart, and the padding puts their 16-byte reads in distinct banks
constexpr int kQStride = kHd + 16;

__device__ __forceinline__ int qidx(int d) { return d + ((d >> 6) << 2); }

// Codes of one 256-wide row held 4 per lane by one wave: the per-token rule
// (s = max |x| / 127, codes rne(x / s) clamped to +-127, zero row -> s = 0).
__device__ __forceinline__ uint32_t quant_row4(const float (&v)[4], float* s_out) {
  float a = fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3])));
  const float amax = wave_max(a);
  const float s = amax / 127.0f;
  uint32_t packed = 0;
  if (s != 0.0f) {
    const float inv = 1.0f / s;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      packed |= (uint32_t)(uint8_t)code_of(v[e], s, inv, true) << (8 * e);
  }
  *s_out = s;
  return packed;
}

__device__ __forceinline__ void load_bf16x4(const uint16_t* p, float (&v)[4]) {
  const uint2 raw = *reinterpret_cast<const uint2*>(p);
  v[0] = bf16_bits_to_float(raw.x & 0xffffu);
  v[1] = bf16_bits_to_float(raw.x >> 16);
  v[2] = bf16_bits_to_float(raw.y & 0xffffu);
  v[3] = bf16_bits_to_float(raw.y >> 16);
}

__device__ __forceinline__ float byte_f(uint32_t w, int e) {
  return (float)(int8_t)(uint8_t)(w >> (8 * e));
}

}  // namespace

// One wave per row of 256 bf16 values (stride ld elements): INT8 codes
// (row-major, 256 a row) and the row's scale.
__global__ __launch_bounds__(256) void kv_quant_kernel(const uint16_t* __restrict__ src,
                                                       int64_t rows, int64_t ld,
                                                       int8_t* __restrict__ codes,
                                                       float* __restrict__ scales) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;  // whole wave
  const int l = lane_id();
  float v[4];
  load_bf16x4(src + r * ld + 4 * l, v);
  float s;
  const uint32_t packed = quant_row4(v, &s);
  *reinterpret_cast<uint32_t*>(codes + r * kHd + 4 * l) = packed;
  if (l == 0) scales[r] = s;
}

// Partial results of one workgroup: per head the running maximum m and sum l
// of exp(score - m), and the unnormalised output o (256 values).
constexpr int kPartFloats = 2 * kMaxHeads + kMaxHeads * kHd;

template <bool I8, int NH>
__global__ __launch_bounds__(256) void attn_decode_kernel(AttnParams p) {
  __shared__ float qs[NH][kQStride];
  __shared__ float sc[NH][kPass];     // scores, then weights p (x the row's value scale)
  __shared__ float corr[NH];          // rescale of the running sums for this pass
  __shared__ float run_m[NH], run_l[NH];
  __shared__ float ored[4][NH][kHd];  // the four waves' partial outputs
  __shared__ uint32_t knew[kHd / 2], vnew[kHd / 2];  // the new row (codes or bf16 bits)
  __shared__ float knew_s, vnew_s;

  const int tid = threadIdx.x, w = tid >> 6, l = lane_id();
  const int64_t r_begin = p.t0 + (int64_t)blockIdx.x * p.rows_per_wg;
  const int64_t r_end = min(r_begin + p.rows_per_wg, p.pos + 1);  // exclusive

  const int jr = l >> 2, qd = l & 3;  // score phase: row 16w + jr, dimensions 64 qd ..
  // The keys, values and (INT8) their scales of a pass are loaded one pass
  // ahead: pass i + 1's loads are issued before pass i's arithmetic and
  // barriers; the first pass's before the staging of the query and the new
  // row, unless that pass holds the new row.
  struct PassRegs {
    uint4 kc[I8 ? 4 : 8];          // key row 16 w + jr, dimensions 64 qd .. 64 qd + 63
    uint32_t vv[16][I8 ? 1 : 2];   // value rows 16 w .. 16 w + 15, dimensions 4 l .. 4 l + 3
    float ks, vs;                  // INT8: scale of key row 16 w + jr, of value row l (the
                                   // new row's come from LDS where they are used)
  };
  // loads of a pass; the new row (pos) comes from LDS, where its codes are
  // staged behind the first barrier
  auto load_pass = [&](int64_t r0, PassRegs& R) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int64_t row = r0 + 16 * w + i;
      if (row == p.pos) {
        R.vv[i][0] = I8 ? vnew[l] : vnew[2 * l];
        if constexpr (!I8) R.vv[i][1] = vnew[2 * l + 1];
      } else if (row < r_end && row != p.pos) {
        if constexpr (I8) {
          R.vv[i][0] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const int8_t*>(p.v) +
                                                         row * kHd + 4 * l);
        } else {
          const uint2 raw = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(p.v) +
                                                           row * kHd + 4 * l);
          R.vv[i][0] = raw.x;
          R.vv[i][1] = raw.y;
        }
      } else {
        R.vv[i][0] = 0;
        if constexpr (!I8) R.vv[i][1] = 0;
      }
    }
    constexpr int NK = I8 ? 4 : 8;  // 16-byte words of 64 dimensions
    const int64_t row = r0 + 16 * w + jr;
    if (row == p.pos) {
#pragma unroll
      for (int c = 0; c < NK; ++c)
        R.kc[c] = make_uint4(knew[4 * NK * qd + 4 * c], knew[4 * NK * qd + 4 * c + 1],
                             knew[4 * NK * qd + 4 * c + 2], knew[4 * NK * qd + 4 * c + 3]);
    } else if (row < r_end && row != p.pos) {
      const uint4* src = reinterpret_cast<const uint4*>(
          reinterpret_cast<const int8_t*>(p.k) + (row * kHd + 64 * qd) * (I8 ? 1 : 2));
#pragma unroll
      for (int c = 0; c < NK; ++c) R.kc[c] = src[c];
    } else {
#pragma unroll
      for (int c = 0; c < NK; ++c) R.kc[c] = make_uint4(0, 0, 0, 0);
    }
    R.ks = 0.0f;
    R.vs = 0.0f;
    if constexpr (I8) {
      if (row < r_end && row != p.pos) R.ks = p.sk[row];
      const int64_t rv = r0 + l;
      if (rv < r_end && rv != p.pos) R.vs = p.sv[rv];
    }
  };
  PassRegs cur, nxt;
  // the first pass's loads ahead of the staging when they need nothing staged
  const bool early = r_begin < r_end && !(p.pos >= r_begin && p.pos < r_begin + kPass);
  if (early) load_pass(r_begin, cur);
  for (int i = tid; i < NH * kHd; i += 256) qs[i / kHd][qidx(i % kHd)] = bf16_bits_to_float(p.qkv[i]);
  if (tid < NH) {
    run_m[tid] = -INFINITY;
    run_l[tid] = 0.0f;
  }
  const bool has_new = r_end == p.pos + 1;
  if (has_new && w < 2) {  // wave 0: the key, wave 1: the value
    const uint16_t* src = p.qkv + NH * kHd + w * kHd + 4 * l;
    if constexpr (I8) {
      float v[4], s;
      load_bf16x4(src, v);
      const uint32_t packed = quant_row4(v, &s);
      int8_t* dst = reinterpret_cast<int8_t*>(w == 0 ? p.k : p.v) + p.pos * kHd;
      *reinterpret_cast<uint32_t*>(dst + 4 * l) = packed;
      (w == 0 ? knew : vnew)[l] = packed;
      if (l == 0) {
        (w == 0 ? p.sk : p.sv)[p.pos] = s;
        if (w == 0) knew_s = s; else vnew_s = s;
      }
    } else {
      const uint2 raw = *reinterpret_cast<const uint2*>(src);
      uint16_t* dst = reinterpret_cast<uint16_t*>(w == 0 ? p.k : p.v) + p.pos * kHd;
      *reinterpret_cast<uint2*>(dst + 4 * l) = raw;
      (w == 0 ? knew : vnew)[2 * l] = raw.x;
      (w == 0 ? knew : vnew)[2 * l + 1] = raw.y;
    }
  }
  __syncthreads();
  if (r_begin < r_end && !early) load_pass(r_begin, cur);

  // per lane: 4 output dimensions (4l .. 4l + 3) of every head, summed over
  // the rows this wave handles
  float o[NH][4];
#pragma unroll
  for (int h = 0; h < NH; ++h)
#pragma unroll
    for (int e = 0; e < 4; ++e) o[h][e] = 0.0f;

  for (int64_t r0 = r_begin; r0 < r_end; r0 += kPass) {
    if (r0 + kPass < r_end) load_pass(r0 + kPass, nxt);
    // ---- scores: four lanes per row, 64 dimensions each
    {
      const int64_t row = r0 + 16 * w + jr;
      const bool valid = row < r_end;
      float acc[NH];
#pragma unroll
      for (int h = 0; h < NH; ++h) acc[h] = 0.0f;
      if constexpr (I8) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const uint32_t wd[4] = {cur.kc[c].x, cur.kc[c].y, cur.kc[c].z, cur.kc[c].w};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int d0 = 64 * qd + 16 * c + 4 * i;
#pragma unroll
            for (int h = 0; h < NH; ++h) {
              const float4 qv = *reinterpret_cast<const float4*>(&qs[h][qidx(d0)]);
              // q (bf16) times an integer code below 128 is exact in binary32
              acc[h] = __builtin_fmaf(qv.x, byte_f(wd[i], 0), acc[h]);
              acc[h] = __builtin_fmaf(qv.y, byte_f(wd[i], 1), acc[h]);
              acc[h] = __builtin_fmaf(qv.z, byte_f(wd[i], 2), acc[h]);
              acc[h] = __builtin_fmaf(qv.w, byte_f(wd[i], 3), acc[h]);
            }
          }
        }
      } else {
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          const uint32_t wd[4] = {cur.kc[c].x, cur.kc[c].y, cur.kc[c].z, cur.kc[c].w};
#pragma unroll
          for (int i = 0; i < 4; i += 2) {
            const int d0 = 64 * qd + 8 * c + 2 * i;
#pragma unroll
            for (int h = 0; h < NH; ++h) {
              const float4 qv = *reinterpret_cast<const float4*>(&qs[h][qidx(d0)]);
              // a product of two bf16 values is exact in binary32
              acc[h] = __builtin_fmaf(qv.x, bf16_bits_to_float(wd[i] & 0xffffu), acc[h]);
              acc[h] = __builtin_fmaf(qv.y, bf16_bits_to_float(wd[i] >> 16), acc[h]);
              acc[h] = __builtin_fmaf(qv.z, bf16_bits_to_float(wd[i + 1] & 0xffffu), acc[h]);
              acc[h] = __builtin_fmaf(qv.w, bf16_bits_to_float(wd[i + 1] >> 16), acc[h]);
            }
          }
        }
      }
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        acc[h] += lane_xor<1>(acc[h]);
        acc[h] += lane_xor<2>(acc[h]);
      }
      if (qd == 0) {
        float ks = 1.0f;
        if constexpr (I8) ks = valid ? (row == p.pos ? knew_s : cur.ks) : 0.0f;
#pragma unroll
        for (int h = 0; h < NH; ++h)
          sc[h][16 * w + jr] = valid ? (acc[h] * ks) * 0.0625f : -INFINITY;
      }
    }
    __syncthreads();
    // ---- running softmax: wave w takes heads w, w + 4
#pragma unroll
    for (int h = w; h < NH; h += 4) {
      const float s = sc[h][l];
      const float m_old = run_m[h];
      const float m_new = fmaxf(m_old, wave_max(s));
      const float e = expf(s - m_new);  // 0 for rows past the end (score -inf)
      const float sum = wave_sum(e);
      float wgt = e;
      if constexpr (I8) {
        const int64_t row = r0 + l;
        wgt = row < r_end ? e * (row == p.pos ? vnew_s : cur.vs) : 0.0f;
      }
      sc[h][l] = wgt;
      if (l == 0) {
        const float c = expf(m_old - m_new);  // 0 on the first pass
        corr[h] = c;
        run_l[h] = run_l[h] * c + sum;
        run_m[h] = m_new;
      }
    }
    __syncthreads();
    // ---- weighted values: this wave's 16 rows into its 4 dimensions per lane
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      const float c = corr[h];
#pragma unroll
      for (int e = 0; e < 4; ++e) o[h][e] *= c;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float vf[4];
      if constexpr (I8) {
#pragma unroll
        for (int e = 0; e < 4; ++e) vf[e] = byte_f(cur.vv[i][0], e);
      } else {
        vf[0] = bf16_bits_to_float(cur.vv[i][0] & 0xffffu);
        vf[1] = bf16_bits_to_float(cur.vv[i][0] >> 16);
        vf[2] = bf16_bits_to_float(cur.vv[i][1] & 0xffffu);
        vf[3] = bf16_bits_to_float(cur.vv[i][1] >> 16);
      }
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        const float wt = sc[h][16 * w + i];
#pragma unroll
        for (int e = 0; e < 4; ++e) o[h][e] = __builtin_fmaf(wt, vf[e], o[h][e]);
      }
    }
    __syncthreads();  // sc and corr are rewritten by the next pass
    cur = nxt;
  }

  // ---- the four waves' sums, then the result or this workgroup's partial
#pragma unroll
  for (int h = 0; h < NH; ++h)
#pragma unroll
    for (int e = 0; e < 4; ++e) ored[w][h][4 * l + e] = o[h][e];
  __syncthreads();
  for (int i = tid; i < NH * kHd; i += 256) {
    const int h = i / kHd, d = i % kHd;
    const float od = ((ored[0][h][d] + ored[1][h][d]) + ored[2][h][d]) + ored[3][h][d];
    if (p.n_wg == 1) {
      p.out[i] = float_to_bf16_bits(od / run_l[h]);
    } else {
      float* part = p.part + (int64_t)blockIdx.x * kPartFloats;
      part[2 * kMaxHeads + h * kHd + d] = od;
      if (d == 0) {
        part[h] = run_m[h];
        part[kMaxHeads + h] = run_l[h];
      }
    }
  }
}

// Merge of the workgroups' partial results.  Four workgroups per head, each
// over 64 output dimensions with 16 waves: the maximum over the chunks, then
// every chunk's factor exp(m_c - M) and the denominator, then each thread
// sums the chunks c = wave, wave + 16, ... of one dimension (16 loads in
// flight per dimension instead of one chain over all chunks).
__global__ __launch_bounds__(1024) void attn_merge_kernel(AttnParams p) {
  __shared__ float fc[kAttnWgTarget];  // exp(m_c - M)
  __shared__ float red[16][64];
  __shared__ float wred[16];
  const int h = blockIdx.x >> 2, d = (blockIdx.x & 3) * 64 + (threadIdx.x & 63);
  const int tid = threadIdx.x, g = tid >> 6, n = p.n_wg;
  float m = -INFINITY;
  for (int c = tid; c < n; c += 1024) m = fmaxf(m, p.part[(int64_t)c * kPartFloats + h]);
  m = wave_max(m);
  if ((tid & 63) == 0) wred[g] = m;
  __syncthreads();
  m = wred[0];
  for (int i = 1; i < 16; ++i) m = fmaxf(m, wred[i]);
  __syncthreads();
  float den = 0.0f;
  for (int c = tid; c < n; c += 1024) {
    const float* part = p.part + (int64_t)c * kPartFloats;
    const float f = expf(part[h] - m);
    fc[c] = f;
    den += part[kMaxHeads + h] * f;
  }
  den = wave_sum(den);
  if ((tid & 63) == 0) wred[g] = den;
  __syncthreads();
  den = 0.0f;
  for (int i = 0; i < 16; ++i) den += wred[i];
  float num = 0.0f;
  const float* col = p.part + 2 * kMaxHeads + h * kHd + d;
#pragma unroll 4
  for (int c = g; c < n; c += 16) num += col[(int64_t)c * kPartFloats] * fc[c];
  red[g][tid & 63] = num;
  __syncthreads();
  if (g == 0) {
    float t = 0.0f;
    for (int i = 0; i < 16; ++i) t += red[i][tid & 63];
    p.out[h * kHd + d] = float_to_bf16_bits(t / den);
  }
}

hipError_t launch_kv_quant(const uint16_t* src, int64_t rows, int64_t ld, int8_t* codes,
                           float* scales, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  kv_quant_kernel<<<dim3((unsigned)((rows + 3) / 4)), 256, 0, st>>>(src, rows, ld, codes, scales);
  return hipGetLastError();
}

// Rows per workgroup: whole passes of 64, at most kAttnWgTarget workgroups
// (about one per CU: more would only add partial results to merge).
void attn_plan(int64_t rows, int target, int* rows_per_wg, int* n_wg) {
  target = std::max(1, std::min(target, kAttnWgTarget));
  const int64_t passes = (rows + kPass - 1) / kPass;
  const int64_t per = (passes + target - 1) / target;  // passes per workgroup
  *rows_per_wg = (int)(per * kPass);
  *n_wg = (int)((passes + per - 1) / per);
}

size_t attn_ws_bytes(int64_t rows, int target) {
  int rpw = 0, n = 0;
  attn_plan(rows, target, &rpw, &n);
  return n > 1 ? (size_t)n * kPartFloats * sizeof(float) : 0;
}

// Enough for every row count up to t_max: a launch uses min(passes,
// kAttnWgTarget) workgroups or fewer, and more rows never mean fewer passes.
size_t attn_ws_bytes_max(int64_t t_max) {
  const int64_t passes = (t_max + kPass - 1) / kPass;
  const int64_t n = std::min<int64_t>(passes, kAttnWgTarget);
  return n > 1 ? (size_t)n * kPartFloats * sizeof(float) : 0;
}

// Merge of at most 16 * CPT partial results: every partial's maximum, sum
// and output dimension loaded at once (one memory round trip), then the
// maximum over the chunks, each thread's factors exp(m_c - M) for its chunks
// c = wave, wave + 16, ..., and the sums over the 16 waves in wave order.
template <int CPT>
__global__ __launch_bounds__(1024) void attn_merge_few_kernel(AttnParams p) {
  __shared__ float wmax[16], wden[16];
  __shared__ float red[16][64];
  const int h = blockIdx.x >> 2, d = (blockIdx.x & 3) * 64 + (threadIdx.x & 63);
  const int tid = threadIdx.x, g = tid >> 6, lane = tid & 63, n = p.n_wg;
  float mc[CPT], lc[CPT], oc[CPT];
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    const int c = g + 16 * j;
    mc[j] = -INFINITY;
    lc[j] = 0.0f;
    oc[j] = 0.0f;
    if (c < n) {
      const float* part = p.part + (int64_t)c * kPartFloats;
      mc[j] = part[h];
      lc[j] = part[kMaxHeads + h];
      oc[j] = part[2 * kMaxHeads + h * kHd + d];
    }
  }
  float m = mc[0];
#pragma unroll
  for (int j = 1; j < CPT; ++j) m = fmaxf(m, mc[j]);
  if (lane == 0) wmax[g] = m;  // the same in every lane of the wave
  __syncthreads();
  m = wmax[0];
  for (int i = 1; i < 16; ++i) m = fmaxf(m, wmax[i]);
  float den = 0.0f, num = 0.0f;
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    if (g + 16 * j < n) {
      const float f = expf(mc[j] - m);
      den += lc[j] * f;
      num += oc[j] * f;
    }
  }
  if (lane == 0) wden[g] = den;
  red[g][lane] = num;
  __syncthreads();
  if (g == 0) {
    float t = 0.0f, dn = 0.0f;
    for (int i = 0; i < 16; ++i) {
      t += red[i][lane];
      dn += wden[i];
    }
    p.out[h * kHd + d] = float_to_bf16_bits(t / dn);
  }
}

template <bool I8>
static hipError_t attn_launch(const AttnParams& p, int nh, hipStream_t st) {
  const dim3 grid((unsigned)p.n_wg);
  switch (nh) {
    case 1: attn_decode_kernel<I8, 1><<<grid, 256, 0, st>>>(p); break;
    case 2: attn_decode_kernel<I8, 2><<<grid, 256, 0, st>>>(p); break;
    case 4: attn_decode_kernel<I8, 4><<<grid, 256, 0, st>>>(p); break;
    case 8: attn_decode_kernel<I8, 8><<<grid, 256, 0, st>>>(p); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.n_wg == 1) return e;
  if (p.n_wg <= 64)  // up to 4096 rows: one round trip for every partial
    attn_merge_few_kernel<4><<<dim3((unsigned)(4 * nh)), 1024, 0, st>>>(p);
  else
    attn_merge_kernel<<<dim3((unsigned)(4 * nh)), 1024, 0, st>>>(p);
  return hipGetLastError();
}

hipError_t launch_attn_decode(AttnParams p, int nh, bool i8, int target, hipStream_t st) {
  attn_plan(p.pos + 1 - p.t0, target, &p.rows_per_wg, &p.n_wg);
  return i8 ? attn_launch<true>(p, nh, st) : attn_launch<false>(p, nh, st);
}

}  // namespace w8a8
