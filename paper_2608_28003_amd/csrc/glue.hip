// Stack glue between FFN blocks (Gemma-style sandwich norms, unit gain):
//   RMSNorm(v) = v / sqrt(mean(v^2) + 1e-6), output bf16, and the fused
//   post-norm residual x_out = bf16(x + bf16(RMSNorm(f))).
// One workgroup per row; each thread owns an 8-element (16-byte) chunk kept in
// registers; the sum of squares is a binary32 butterfly + LDS reduction.
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

hipError_t launch_rmsnorm(const uint16_t* x, const uint16_t* f, int64_t m, int64_t d,
                          uint16_t* y, hipStream_t st) {
  int64_t threads = (d / 8 + 63) / 64 * 64;
  rmsnorm_kernel<<<(unsigned)m, (unsigned)threads, 0, st>>>(x, f, m, d, y);
  return hipGetLastError();
}

}  // namespace w8a8
