// Row-level device helpers of the decode paths: quantise-on-load of a few bf16
// rows and the fused layer glue for one token row.  Shared by the streaming
// GEMM kernel and the persistent decode kernel; both run exactly these
// binary32 operations, so their codes and scales agree bit for bit with
// quant_rows_kernel and glue_kernel.
#pragma once

#include "device.h"
#include "kernels.h"

namespace w8a8 {

// Stores of data that other workgroups of the same launch read after a grid
// barrier (COH = true, the persistent decode kernel): relaxed device-scope
// atomic stores, which write through the per-XCD L2, so no L2 write-back is
// needed before the barrier.  COH = false: plain stores (the consumer is a
// later launch).
template <bool COH>
__device__ __forceinline__ void st16(void* p, uint4 v) {
  if constexpr (COH) {
    uint64_t* q = reinterpret_cast<uint64_t*>(p);
    __hip_atomic_store(q, (uint64_t)v.x | ((uint64_t)v.y << 32), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(q + 1, (uint64_t)v.z | ((uint64_t)v.w << 32), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  } else {
    *reinterpret_cast<uint4*>(p) = v;
  }
}
template <bool COH>
__device__ __forceinline__ void st_f32(float* p, float v) {
  if constexpr (COH)
    __hip_atomic_store(reinterpret_cast<uint32_t*>(p), __float_as_uint(v), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  else
    *p = v;
}

// Quantise-on-load of at most 16 bf16 rows for one streaming workgroup:
// x_hat = x / delta, per-row scale s = max|x_hat| / 127 over the whole row,
// codes as quant_rows_kernel computes them (same binary32 operations), for the
// workgroup's fragment columns [kb0, kb0 + kc) into LDS (rows >= M and columns
// >= a_k are zero codes).  Each thread loads whole 16-column groups once (at
// most MAXG of them, which the host guarantees: M * a_k / 16 <= MAXG * 64 * NW)
// and keeps the smoothed values in registers between the absmax and the
// rounding.  One group per thread: with more, the redundant per-workgroup
// divisions cost more than the separate quantisation launch they replace.  The caller's barrier publishes lds_a and s_row.
template <int NW>
constexpr int qload_max_groups() { return 1; }

// The bf16 activations and smoothing factors of this thread's groups, loaded
// before the workgroup's first weight batch: loads return in issue order, so
// the quantisation below then runs while the weights are still in flight.
// The loads are issued by every thread without branching (threads past the
// last group repeat a valid group; without quantise-on-load they read the
// first bytes of B and are ignored), which lets the compiler wait for exactly
// these loads rather than for every load outstanding.
template <int NW>
struct QloadRegs {
  uint4 x[qload_max_groups<NW>()][2];
  float4 d[qload_max_groups<NW>()][4];
};

template <int NW>
__device__ __forceinline__ void quantize_fetch(const GemmParams& p, bool qload, QloadRegs<NW>& R) {
  constexpr int NT = NW * 64;
  const int tid = threadIdx.x;
  const int rows = qload ? min(p.M, 16) : 1;
  const int G = qload ? p.a_k / 16 : 1;
  const uint16_t* xbase = qload ? p.a_x : reinterpret_cast<const uint16_t*>(p.B);
  const float* dbase = (qload && p.a_delta) ? p.a_delta : reinterpret_cast<const float*>(p.B);
  const int64_t ld = qload ? p.a_ld : 0;
  const int cmul = qload ? 16 : 0;
#pragma unroll
  for (int i = 0; i < qload_max_groups<NW>(); ++i) {
    const int gi = min(tid + i * NT, rows * G - 1);
    const int r = gi / G, c0 = (gi % G) * cmul;
    const uint16_t* xr = xbase + (int64_t)r * ld + c0;
    R.x[i][0] = *reinterpret_cast<const uint4*>(xr);
    R.x[i][1] = *reinterpret_cast<const uint4*>(xr + 8);
    const float4* dp = reinterpret_cast<const float4*>(dbase + ((qload && p.a_delta) ? c0 : 0));
#pragma unroll
    for (int q = 0; q < 4; ++q) R.d[i][q] = dp[q];
  }
}

// F8: E4M3 codes (scale amax / 448, the quantiser's conversion) instead of int8
template <int NW, bool F8>
__device__ __forceinline__ void quantize_panel(const GemmParams& p, int kb0, int kc, v4i* lds_a,
                                               float* s_row, const QloadRegs<NW>& R) {
  constexpr float QMAX = F8 ? 448.0f : 127.0f;
  constexpr int NT = NW * 64;
  constexpr int MAXG = qload_max_groups<NW>();
  __shared__ unsigned int amax_bits[16];
  const int tid = threadIdx.x;
  const int rows = min(p.M, 16);
  const int G = p.a_k / 16;  // 16-column groups per row
  float v[MAXG][16];
  float mx[MAXG];
#pragma unroll
  for (int i = 0; i < MAXG; ++i) {
    const int gi = tid + i * NT;
    mx[i] = 0.0f;
    if (gi < rows * G) {
      const uint32_t w[8] = {R.x[i][0].x, R.x[i][0].y, R.x[i][0].z, R.x[i][0].w,
                             R.x[i][1].x, R.x[i][1].y, R.x[i][1].z, R.x[i][1].w};
#pragma unroll
      for (int e = 0; e < 16; ++e)
        v[i][e] = bf16_bits_to_float((e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xffffu));
      if (p.a_delta) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 d4 = R.d[i][q];
          v[i][4 * q + 0] = v[i][4 * q + 0] / d4.x;
          v[i][4 * q + 1] = v[i][4 * q + 1] / d4.y;
          v[i][4 * q + 2] = v[i][4 * q + 2] / d4.z;
          v[i][4 * q + 3] = v[i][4 * q + 3] / d4.w;
        }
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) mx[i] = fmaxf(mx[i], fabsf(v[i][e]));
    }
  }
  // zero codes everywhere first (padding rows and columns stay zero)
  for (int idx = tid; idx < kc * 64; idx += NT) lds_a[idx] = v4i{0, 0, 0, 0};
  if (tid < 16) amax_bits[tid] = 0u;
  __syncthreads();
  // non-negative binary32 values order like their bit patterns: the maximum
  // does not depend on the order of the atomic updates
#pragma unroll
  for (int i = 0; i < MAXG; ++i) {
    const int gi = tid + i * NT;
    if (gi < rows * G) atomicMax(&amax_bits[gi / G], __float_as_uint(mx[i]));
  }
  __syncthreads();
  if (tid < rows) {
    const float s = __uint_as_float(amax_bits[tid]) / QMAX;
    s_row[tid] = s;
    if (p.a_s_out && blockIdx.x == 0 && blockIdx.y == 0) p.a_s_out[tid] = s;
  }
#pragma unroll
  for (int i = 0; i < MAXG; ++i) {
    const int gi = tid + i * NT;
    if (gi >= rows * G) continue;
    const int r = gi / G, g = gi % G;
    const int f = g / 4 - kb0;
    if (f < 0 || f >= kc) continue;
    const float sr = __uint_as_float(amax_bits[r]) / QMAX;
    if (sr == 0.0f) continue;
    int32_t packed[4] = {0, 0, 0, 0};
    if constexpr (F8) {  // the same binary32 steps as quant_rows_kernel's E4M3 mode
#pragma unroll
      for (int e = 0; e < 16; e += 2) {
        const float q0 = fminf(fmaxf(v[i][e] / sr, -448.0f), 448.0f);
        const float q1 = fminf(fmaxf(v[i][e + 1] / sr, -448.0f), 448.0f);
        packed[e >> 2] |= (int32_t)(e4m3_pack2(q0, q1) << (8 * (e & 3)));
      }
    } else {
      const float inv = 1.0f / sr;
      const bool fast = isfinite(inv);
#pragma unroll
      for (int e = 0; e < 16; ++e)
        packed[e >> 2] |= ((int32_t)code_of(v[i][e], sr, inv, fast) & 0xff) << (8 * (e & 3));
    }
    lds_a[f * 64 + r + 16 * (g & 3)] = v4i{packed[0], packed[1], packed[2], packed[3]};
  }
}

// Fused layer glue for one token row (see GemmParams): thread t owns the row's
// columns [8t, 8t + 8), as in the glue kernel, so every sum and reduction runs
// in the glue kernel's order and the codes and scale come out identical.  All
// operands are loaded without branches before the first weight batch (threads
// past the row, absent partial sums or scales read valid bytes of B instead).
struct GlueRegs {
  uint4 x;
  int4 part[kGlueMaxSplits][2];  // int32 sums, or the bits of fp32 sums
  float4 si0, si1, d0, d1;
  float st;
};

// PAD = 0: partial sums in planes of M x a_k; PAD > 0: plane z holds column
// block c (16 columns) at (z * ncd + c) * PAD elements.
template <int PAD = 0>
__device__ __forceinline__ void glue_fetch(const GemmParams& p, GlueRegs& R, int ncd = 0) {
  const int d = p.a_k;
  const int c0 = min((int)threadIdx.x, d / 8 - 1) * 8;
  const bool has_part = p.g_part != nullptr;
  const bool scaled = has_part && !p.g_part_f32;
  const int4* dummy = reinterpret_cast<const int4*>(p.B);  // >= 4 KiB of packed weights
  R.x = *reinterpret_cast<const uint4*>(p.g_x_in + c0);
  const int32_t* pp = has_part ? reinterpret_cast<const int32_t*>(p.g_part) +
                                   (PAD ? (c0 / 16) * PAD + c0 % 16 : c0)
                             : reinterpret_cast<const int32_t*>(dummy);
  const int64_t plane = has_part ? (PAD ? (int64_t)ncd * PAD : (int64_t)p.M * d) : 0;
  // planes past g_splits read one fixed 32-byte block (the same address in
  // every lane, one request per wave) rather than a second copy of the row
#pragma unroll
  for (int z = 0; z < kGlueMaxSplits; ++z) {
    const int32_t* src = z < p.g_splits ? pp + z * plane : reinterpret_cast<const int32_t*>(dummy);
    R.part[z][0] = *reinterpret_cast<const int4*>(src);
    R.part[z][1] = *reinterpret_cast<const int4*>(src + 4);
  }
  const float* si = scaled ? p.g_si + c0 : reinterpret_cast<const float*>(dummy);
  R.si0 = *reinterpret_cast<const float4*>(si);
  R.si1 = *reinterpret_cast<const float4*>(si + 4);
  R.st = *(scaled ? p.g_st : reinterpret_cast<const float*>(dummy));
  const float* dl = p.a_delta ? p.a_delta + c0 : reinterpret_cast<const float*>(dummy);
  R.d0 = *reinterpret_cast<const float4*>(dl);
  R.d1 = *reinterpret_cast<const float4*>(dl + 4);
}

// The first half of the layer glue: xv = this thread's 8 columns [8t, 8t + 8)
// of the updated token stream (post-norm of the previous layer's output added
// to g_x_in), written by workgroup 0 to g_x_out and g_x_copy.  Threads past the
// row hold unused values and add 0 to the row sum.
template <int NW, bool COH = false>
__device__ __forceinline__ void glue_stream(const GemmParams& p, const GlueRegs& R, float (&xv)[8]) {
  __shared__ float red_y[NW];
  const int t = threadIdx.x;
  const int d = p.a_k;
  const bool own = t < d / 8;
  const int c0 = t * 8;
  {
    const uint32_t w[4] = {R.x.x, R.x.y, R.x.z, R.x.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      xv[2 * j] = bf16_bits_to_float(w[j] & 0xffffu);
      xv[2 * j + 1] = bf16_bits_to_float(w[j] >> 16);
    }
  }
  if (p.g_part) {  // uniform: post-norm of the previous layer's output, residual add
    float y[8];
    if (p.g_part_f32) {
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int z = 0; z < kGlueMaxSplits; ++z)
        if (z < p.g_splits) {
          const int4 a0 = R.part[z][0], a1 = R.part[z][1];
          acc[0] += __int_as_float(a0.x); acc[1] += __int_as_float(a0.y);
          acc[2] += __int_as_float(a0.z); acc[3] += __int_as_float(a0.w);
          acc[4] += __int_as_float(a1.x); acc[5] += __int_as_float(a1.y);
          acc[6] += __int_as_float(a1.z); acc[7] += __int_as_float(a1.w);
        }
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = bf16_bits_to_float(float_to_bf16_bits(acc[e]));
    } else {
      int32_t acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
      for (int z = 0; z < kGlueMaxSplits; ++z)
        if (z < p.g_splits) {
          const int4 a0 = R.part[z][0], a1 = R.part[z][1];
          acc[0] += a0.x; acc[1] += a0.y; acc[2] += a0.z; acc[3] += a0.w;
          acc[4] += a1.x; acc[5] += a1.y; acc[6] += a1.z; acc[7] += a1.w;
        }
      const float si[8] = {R.si0.x, R.si0.y, R.si0.z, R.si0.w, R.si1.x, R.si1.y, R.si1.z, R.si1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e)
        y[e] = bf16_bits_to_float(float_to_bf16_bits(((float)acc[e] * R.st) * si[e]));
    }
    float ss = 0.0f;
    if (own) {
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += y[e] * y[e];
    }
    ss = block_sum_in(ss, red_y);
    const float inv = 1.0f / sqrtf(ss / (float)d + 1e-6f);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float b = bf16_bits_to_float(float_to_bf16_bits(y[e] * inv));
      xv[e] = bf16_bits_to_float(float_to_bf16_bits(xv[e] + b));
    }
  }
  if (own && blockIdx.x == 0 && blockIdx.y == 0) {  // the token stream, written once
    uint4 o;
    o.x = (uint32_t)float_to_bf16_bits(xv[0]) | ((uint32_t)float_to_bf16_bits(xv[1]) << 16);
    o.y = (uint32_t)float_to_bf16_bits(xv[2]) | ((uint32_t)float_to_bf16_bits(xv[3]) << 16);
    o.z = (uint32_t)float_to_bf16_bits(xv[4]) | ((uint32_t)float_to_bf16_bits(xv[5]) << 16);
    o.w = (uint32_t)float_to_bf16_bits(xv[6]) | ((uint32_t)float_to_bf16_bits(xv[7]) << 16);
    if (p.g_x_out) st16<COH>(p.g_x_out + c0, o);
    if (p.g_x_copy) *reinterpret_cast<uint4*>(p.g_x_copy + c0) = o;
  }
}

template <int NW>
__device__ __forceinline__ void glue_panel(const GemmParams& p, int kb0, int kc, v4i* lds_a,
                                           float* s_row, const GlueRegs& R) {
  constexpr int NT = NW * 64;
  __shared__ float red_x[NW], red_q[NW];
  const int t = threadIdx.x;
  const int d = p.a_k;
  const bool own = t < d / 8;
  const int c0 = t * 8;
  for (int idx = t; idx < kc * 64; idx += NT) lds_a[idx] = v4i{0, 0, 0, 0};  // padding stays 0
  float xv[8];
  glue_stream<NW, false>(p, R, xv);
  float ss = 0.0f;
  if (own) {
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += xv[e] * xv[e];
  }
  ss = block_sum_in(ss, red_x);
  const float inv = 1.0f / sqrtf(ss / (float)d + 1e-6f);
  float a[8];
  float amax = 0.0f;
  const float dl[8] = {R.d0.x, R.d0.y, R.d0.z, R.d0.w, R.d1.x, R.d1.y, R.d1.z, R.d1.w};
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = bf16_bits_to_float(float_to_bf16_bits(xv[e] * inv));
    if (p.a_delta) a[e] = a[e] / dl[e];
    if (own) amax = fmaxf(amax, fabsf(a[e]));
  }
  amax = block_max_in(amax, red_q);
  const float sr = ss == ss ? amax / 127.0f : ss;  // a NaN in the row: NaN scale
  if (t == 0) {
    s_row[0] = sr;
    if (p.a_s_out && blockIdx.x == 0 && blockIdx.y == 0) p.a_s_out[0] = sr;
  }
  const int f = c0 / kFragK8 - kb0;  // this thread's fragment column in the panel
  if (own && sr != 0.0f && f >= 0 && f < kc) {
    const float sinv = 1.0f / sr;
    const bool fast = isfinite(sinv);
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lo |= ((uint32_t)code_of(a[e], sr, sinv, fast) & 0xffu) << (8 * e);
      hi |= ((uint32_t)code_of(a[e + 4], sr, sinv, fast) & 0xffu) << (8 * e);
    }
    // row 0 of the fragment: lane 16 * ((c0 % 64) / 16), bytes c0 % 16 .. + 7
    uint2* dst = reinterpret_cast<uint2*>(&lds_a[f * 64 + 16 * ((c0 % kFragK8) / 16)]) + (c0 % 16) / 8;
    *dst = make_uint2(lo, hi);
  }
}

}  // namespace w8a8
