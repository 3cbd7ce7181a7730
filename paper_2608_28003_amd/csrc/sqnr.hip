// Signal-to-quantisation-noise ratio of a quantised output against its
// reference (eq. sqnr-ffn for one layer's output, eq. sqnr-block for a block
// or stack output; both are the same ratio of sums of squares):
//   S = sum ref^2,  N = sum (ref - test)^2,  SQNR = 10 log10(S / N) dB.
// Two launches with a fixed grid and fixed-order tree reductions in binary64,
// so the result does not depend on scheduling.
#include <hip/hip_runtime.h>

#include "device.h"
#include "kernels.h"

namespace w8a8 {

namespace {

constexpr int kSqnrThreads = 256;

template <typename T>
__device__ __forceinline__ double elem(const T* p, int64_t i);
template <>
__device__ __forceinline__ double elem<uint16_t>(const uint16_t* p, int64_t i) {
  return (double)bf16_bits_to_float(p[i]);
}
template <>
__device__ __forceinline__ double elem<float>(const float* p, int64_t i) {
  return (double)p[i];
}

// fixed-order tree sum of one value per thread over the workgroup
__device__ __forceinline__ void block_sum2(double& a, double& b, double* red) {
  const int t = threadIdx.x;
  red[t] = a;
  red[kSqnrThreads + t] = b;
  __syncthreads();
  for (int s = kSqnrThreads / 2; s > 0; s >>= 1) {
    if (t < s) {
      red[t] += red[t + s];
      red[kSqnrThreads + t] += red[kSqnrThreads + t + s];
    }
    __syncthreads();
  }
  a = red[0];
  b = red[kSqnrThreads];
}

// workgroup g sums elements [g * chunk, min(n, (g + 1) * chunk)); thread t
// takes every kSqnrThreads-th element from its offset, in increasing order
template <typename T>
__global__ __launch_bounds__(kSqnrThreads) void sqnr_partial_kernel(const T* __restrict__ ref,
                                                                    const T* __restrict__ test,
                                                                    int64_t n, int64_t chunk,
                                                                    double* __restrict__ part) {
  __shared__ double red[2 * kSqnrThreads];
  const int64_t lo = (int64_t)blockIdx.x * chunk;
  const int64_t hi = min(n, lo + chunk);
  double s = 0.0, e = 0.0;
  for (int64_t i = lo + threadIdx.x; i < hi; i += kSqnrThreads) {
    const double r = elem<T>(ref, i);
    const double d = r - elem<T>(test, i);
    s += r * r;
    e += d * d;
  }
  block_sum2(s, e, red);
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = s;
    part[2 * blockIdx.x + 1] = e;
  }
}

__global__ __launch_bounds__(kSqnrThreads) void sqnr_final_kernel(const double* __restrict__ part,
                                                                  int groups,
                                                                  double* __restrict__ out) {
  __shared__ double red[2 * kSqnrThreads];
  double s = 0.0, e = 0.0;
  for (int g = threadIdx.x; g < groups; g += kSqnrThreads) {
    s += part[2 * g];
    e += part[2 * g + 1];
  }
  block_sum2(s, e, red);
  if (threadIdx.x == 0) {
    out[0] = s;
    out[1] = e;
    out[2] = 10.0 * log10(s / e);  // +inf for e = 0, -inf for s = 0, NaN for both
  }
}

}  // namespace

int sqnr_groups(int64_t n) {
  const int64_t per = (int64_t)kSqnrThreads * 16;  // >= 16 elements per thread
  int64_t g = (n + per - 1) / per;
  if (g > kSqnrMaxGroups) g = kSqnrMaxGroups;
  return (int)(g < 1 ? 1 : g);
}

hipError_t launch_sqnr(const void* ref, const void* test, bool bf16, int64_t n, double* part,
                       double* out, hipStream_t st) {
  const int groups = sqnr_groups(n);
  const int64_t chunk = (n + groups - 1) / groups;
  if (bf16)
    sqnr_partial_kernel<uint16_t><<<groups, kSqnrThreads, 0, st>>>(
        (const uint16_t*)ref, (const uint16_t*)test, n, chunk, part);
  else
    sqnr_partial_kernel<float><<<groups, kSqnrThreads, 0, st>>>((const float*)ref,
                                                                 (const float*)test, n, chunk, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  sqnr_final_kernel<<<1, kSqnrThreads, 0, st>>>(part, groups, out);
  return hipGetLastError();
}

}  // namespace w8a8
