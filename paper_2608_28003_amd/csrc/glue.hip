// Stack glue between FFN blocks (Gemma-style sandwich norms, unit gain):
//   RMSNorm(v) = v / sqrt(mean(v^2) + 1e-6), output bf16, and the fused
//   post-norm residual x_out = bf16(x + bf16(RMSNorm(f))).
// One workgroup per row; each thread owns an 8-element (16-byte) chunk kept in
// registers; the sum of squares is a binary32 butterfly + LDS reduction.
#include <algorithm>

#include "device.h"
#include "kernels.h"

namespace w8a8 {

__device__ __forceinline__ float block_sum(float v) {
  __shared__ float red[16];
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if (lane_id() == 0) red[w] = v;
  __syncthreads();
  float s = 0.0f;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) s += red[i];
  return s;
}

// x and y may alias (in-place residual update): each element is read and then
// written by the same thread.  d % 8 == 0 and d <= 8 * 1024.
__global__ __launch_bounds__(1024) void rmsnorm_kernel(const uint16_t* x,
                                                       const uint16_t* __restrict__ f, int64_t m,
                                                       int64_t d, uint16_t* y) {
  const int64_t r = blockIdx.x;
  const int t = threadIdx.x;
  const int64_t chunks = d / 8;
  float v[8];
  float ss = 0.0f;
  if (t < chunks) {
    uint4 raw = *reinterpret_cast<const uint4*>(f + r * d + t * 8);
    uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[2 * j] = bf16_bits_to_float(w[j] & 0xffffu);
      v[2 * j + 1] = bf16_bits_to_float(w[j] >> 16);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += v[e] * v[e];
  }
  ss = block_sum(ss);
  const float inv = 1.0f / sqrtf(ss / (float)d + 1e-6f);
  if (t >= chunks) return;
  uint16_t b[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) b[e] = float_to_bf16_bits(v[e] * inv);
  if (x) {
    uint4 raw = *reinterpret_cast<const uint4*>(x + r * d + t * 8);
    uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float s0 = bf16_bits_to_float(w[j] & 0xffffu) + bf16_bits_to_float(b[2 * j]);
      float s1 = bf16_bits_to_float(w[j] >> 16) + bf16_bits_to_float(b[2 * j + 1]);
      b[2 * j] = float_to_bf16_bits(s0);
      b[2 * j + 1] = float_to_bf16_bits(s1);
    }
  }
  uint4 o;
  o.x = (uint32_t)b[0] | ((uint32_t)b[1] << 16);
  o.y = (uint32_t)b[2] | ((uint32_t)b[3] << 16);
  o.z = (uint32_t)b[4] | ((uint32_t)b[5] << 16);
  o.w = (uint32_t)b[6] | ((uint32_t)b[7] << 16);
  *reinterpret_cast<uint4*>(y + r * d + t * 8) = o;
}

// ------------------------------------------------------------------ fused row glue

// One row r per workgroup, thread t owns columns [8t, 8t + 8).  Steps, each
// optional and in this order (the arithmetic of every step is the one of the
// standalone kernels: split-K reduction + dequant epilogue, rmsnorm_kernel,
// quant_rows_kernel):
//   1. y = FFN output from split-K partial sums (int32 with two scales, or
//      fp32), rounded to bf16;  x_out = bf16(x_in + bf16(RMSNorm(y)));
//      without partial sums x_out = x_in.
//   2. a = bf16(RMSNorm(x_out)), written as bf16 and/or
//   3. smoothed by delta and quantised per row into the fragment layout
//      (codes q, scale s); rows in [m, rows_pad) and columns in [d, kp) of
//      the packed output are zero.
// NT: the workgroup size it is compiled for (the row's threads rounded up to
// whole waves); at 1152 columns 192 threads, whose registers then hold every
// partial sum without spilling.
// MAXZ: split-K partial sums held in registers (more splits stream from
// memory); 4 for the stack's plans keeps the kernel at ~80 registers, so
// every row of a 2048-token batch is resident at once.
template <int NT, int MAXZ>
__global__ __launch_bounds__(NT) void glue_kernel(GlueParams g) {
  __shared__ float red_y[16], red_x[16], red_q[16];
  const int64_t r = blockIdx.x;
  const int t = threadIdx.x;
  const int64_t d = g.d;
  const int64_t chunks = d / 8;
  const int64_t kb_count = g.kp / kFragK8;
  auto store_codes8 = [&](int64_t c, uint2 v) {  // 8 codes of columns [8c, 8c + 8)
    const int64_t col = c * 8;
    const int64_t off = frag_offset(r >> 4, col / kFragK8, kb_count) +
                        (int64_t)((r & 15) + 16 * ((col % kFragK8) / 16)) * 16 + (col % 16);
    *reinterpret_cast<uint2*>(g.q + off) = v;
  };
  if (r >= g.m) {  // padding row of the packed codes
    for (int64_t c = t; c < g.kp / 8; c += blockDim.x) store_codes8(c, make_uint2(0, 0));
    return;
  }
  const bool own = t < chunks;
  const int64_t col0 = (int64_t)t * 8;
  // every global operand of the row is requested up front, so the launch pays
  // one memory round trip before its three workgroup reductions
  float xv[8];
  uint4 xraw = make_uint4(0, 0, 0, 0);
  float4 d0 = make_float4(1.f, 1.f, 1.f, 1.f), d1 = d0;
  float4 si0 = make_float4(0.f, 0.f, 0.f, 0.f), si1 = si0;
  float st = 0.0f;
  int4 pr[MAXZ][2];  // int32 partial sums, or the bits of fp32 ones
  const int64_t plane = g.m * d;
  if (own) {
    xraw = *reinterpret_cast<const uint4*>(g.x_in + r * d + col0);
    if (g.q && g.delta) {
      d0 = *reinterpret_cast<const float4*>(g.delta + col0);
      d1 = *reinterpret_cast<const float4*>(g.delta + col0 + 4);
    }
    if (g.part) {
      const int32_t* pp = reinterpret_cast<const int32_t*>(g.part) + r * d + col0;
#pragma unroll
      for (int z = 0; z < MAXZ; ++z)
        if (z < g.splits) {
          pr[z][0] = *reinterpret_cast<const int4*>(pp + z * plane);
          pr[z][1] = *reinterpret_cast<const int4*>(pp + z * plane + 4);
        }
      if (!g.part_f32) {
        st = g.s_t[r];
        si0 = *reinterpret_cast<const float4*>(g.s_i + col0);
        si1 = *reinterpret_cast<const float4*>(g.s_i + col0 + 4);
      }
    }
    uint32_t w[4] = {xraw.x, xraw.y, xraw.z, xraw.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      xv[2 * j] = bf16_bits_to_float(w[j] & 0xffffu);
      xv[2 * j + 1] = bf16_bits_to_float(w[j] >> 16);
    }
  }
  if (g.part) {
    float y[8];
    float ss = 0.0f;
    if (own) {
      if (g.part_f32) {
        const float* pp = reinterpret_cast<const float*>(g.part) + r * d + col0;
        float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int z = 0; z < MAXZ; ++z)
          if (z < g.splits) {
            const int4 a0 = pr[z][0], a1 = pr[z][1];
            acc[0] += __int_as_float(a0.x); acc[1] += __int_as_float(a0.y);
            acc[2] += __int_as_float(a0.z); acc[3] += __int_as_float(a0.w);
            acc[4] += __int_as_float(a1.x); acc[5] += __int_as_float(a1.y);
            acc[6] += __int_as_float(a1.z); acc[7] += __int_as_float(a1.w);
          }
        for (int z = MAXZ; z < g.splits; ++z) {
          float4 a0 = *reinterpret_cast<const float4*>(pp + z * plane);
          float4 a1 = *reinterpret_cast<const float4*>(pp + z * plane + 4);
          acc[0] += a0.x; acc[1] += a0.y; acc[2] += a0.z; acc[3] += a0.w;
          acc[4] += a1.x; acc[5] += a1.y; acc[6] += a1.z; acc[7] += a1.w;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = bf16_bits_to_float(float_to_bf16_bits(acc[e]));
      } else {
        const int32_t* pp = reinterpret_cast<const int32_t*>(g.part) + r * d + col0;
        int32_t acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
        for (int z = 0; z < MAXZ; ++z)
          if (z < g.splits) {
            acc[0] += pr[z][0].x; acc[1] += pr[z][0].y; acc[2] += pr[z][0].z; acc[3] += pr[z][0].w;
            acc[4] += pr[z][1].x; acc[5] += pr[z][1].y; acc[6] += pr[z][1].z; acc[7] += pr[z][1].w;
          }
        for (int z = MAXZ; z < g.splits; ++z) {
          int4 a0 = *reinterpret_cast<const int4*>(pp + z * plane);
          int4 a1 = *reinterpret_cast<const int4*>(pp + z * plane + 4);
          acc[0] += a0.x; acc[1] += a0.y; acc[2] += a0.z; acc[3] += a0.w;
          acc[4] += a1.x; acc[5] += a1.y; acc[6] += a1.z; acc[7] += a1.w;
        }
        const float si[8] = {si0.x, si0.y, si0.z, si0.w, si1.x, si1.y, si1.z, si1.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          float v = ((float)acc[e] * st) * si[e];
          y[e] = bf16_bits_to_float(float_to_bf16_bits(v));
        }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += y[e] * y[e];
    }
    ss = block_sum_in(ss, red_y);
    const float inv = 1.0f / sqrtf(ss / (float)d + 1e-6f);
    if (own) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float b = bf16_bits_to_float(float_to_bf16_bits(y[e] * inv));
        xv[e] = bf16_bits_to_float(float_to_bf16_bits(xv[e] + b));
      }
    }
  }
  const bool write_out = g.x_out && (g.part || g.x_out != g.x_in);
  if (own && (write_out || g.x_copy)) {
    uint4 o;
    o.x = (uint32_t)float_to_bf16_bits(xv[0]) | ((uint32_t)float_to_bf16_bits(xv[1]) << 16);
    o.y = (uint32_t)float_to_bf16_bits(xv[2]) | ((uint32_t)float_to_bf16_bits(xv[3]) << 16);
    o.z = (uint32_t)float_to_bf16_bits(xv[4]) | ((uint32_t)float_to_bf16_bits(xv[5]) << 16);
    o.w = (uint32_t)float_to_bf16_bits(xv[6]) | ((uint32_t)float_to_bf16_bits(xv[7]) << 16);
    if (write_out) *reinterpret_cast<uint4*>(g.x_out + r * d + col0) = o;
    if (g.x_copy) *reinterpret_cast<uint4*>(g.x_copy + r * d + col0) = o;
  }
  if (!g.a && !g.q) return;  // uniform over the workgroup
  float ss = 0.0f;
  if (own) {
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += xv[e] * xv[e];
  }
  ss = block_sum_in(ss, red_x);
  const float inv = 1.0f / sqrtf(ss / (float)d + 1e-6f);
  float a[8];
  if (own) {
#pragma unroll
    for (int e = 0; e < 8; ++e) a[e] = bf16_bits_to_float(float_to_bf16_bits(xv[e] * inv));
    if (g.a) {
      uint4 o;
      o.x = (uint32_t)float_to_bf16_bits(a[0]) | ((uint32_t)float_to_bf16_bits(a[1]) << 16);
      o.y = (uint32_t)float_to_bf16_bits(a[2]) | ((uint32_t)float_to_bf16_bits(a[3]) << 16);
      o.z = (uint32_t)float_to_bf16_bits(a[4]) | ((uint32_t)float_to_bf16_bits(a[5]) << 16);
      o.w = (uint32_t)float_to_bf16_bits(a[6]) | ((uint32_t)float_to_bf16_bits(a[7]) << 16);
      *reinterpret_cast<uint4*>(g.a + r * d + col0) = o;
    }
  }
  if (!g.q) return;
  float amax = 0.0f;
  if (own) {
    const float dl[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (g.delta) a[e] = a[e] / dl[e];
      amax = fmaxf(amax, fabsf(a[e]));
    }
  }
  amax = block_max_in(amax, red_q);
  // a NaN in the row (a failed persistent decode run poisons the token
  // stream) reaches the norm's sum of squares; the max above would skip it,
  // so the scale takes the NaN and everything dequantised from it is NaN
  const float sr = ss == ss ? amax / 127.0f : ss;
  if (t == 0) g.s[r] = sr;
  const float sinv = 1.0f / sr;
  const bool fast = isfinite(sinv);
  for (int64_t c = t; c < g.kp / 8; c += blockDim.x) {
    uint32_t lo = 0, hi = 0;
    if (c == t && own && sr != 0.0f) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lo |= ((uint32_t)code_of(a[e], sr, sinv, fast) & 0xffu) << (8 * e);
        hi |= ((uint32_t)code_of(a[e + 4], sr, sinv, fast) & 0xffu) << (8 * e);
      }
    }
    store_codes8(c, make_uint2(lo, hi));
  }
}

hipError_t launch_glue(const GlueParams& g, hipStream_t st) {
  const int64_t rows = g.q ? g.rows_pad : g.m;
  const int64_t per_row = std::max(g.d / 8, g.q ? g.kp / 8 : 0);
  const int64_t threads = std::min<int64_t>((per_row + 63) / 64 * 64, 1024);
  const bool few = !g.part || g.splits <= 4;
  if (threads <= 256) {
    if (few)
      glue_kernel<256, 4><<<(unsigned)rows, (unsigned)threads, 0, st>>>(g);
    else
      glue_kernel<256, 8><<<(unsigned)rows, (unsigned)threads, 0, st>>>(g);
  } else {
    if (few)
      glue_kernel<1024, 4><<<(unsigned)rows, (unsigned)threads, 0, st>>>(g);
    else
      glue_kernel<1024, 8><<<(unsigned)rows, (unsigned)threads, 0, st>>>(g);
  }
  return hipGetLastError();
}

hipError_t launch_rmsnorm(const uint16_t* x, const uint16_t* f, int64_t m, int64_t d,
                          uint16_t* y, hipStream_t st) {
  int64_t threads = (d / 8 + 63) / 64 * 64;
  rmsnorm_kernel<<<(unsigned)m, (unsigned)threads, 0, st>>>(x, f, m, d, y);
  return hipGetLastError();
}

}  // namespace w8a8
