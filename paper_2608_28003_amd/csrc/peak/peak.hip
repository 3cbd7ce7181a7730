// Measured ceilings of the device, for the benchmark's roofline columns: the
// rate of the INT8 matrix instruction the GEMMs use (v_mfma_i32_16x16x64_i8)
// with operands held in registers, and the HBM read rate of a plain streaming
// kernel.  Not part of the W8A8 path: the benchmark loads this library on its
// own (libw8a8_peak.so) and divides the path's figures by these.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../../include/w8a8_peak.h"

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));

constexpr int kChains = 8;  // independent accumulators per wave

// Every wave runs kChains independent chains of `iters` MFMAs; the operands
// never change, so nothing but the matrix cores is exercised.  The sums are
// folded into one word that is stored only if it takes a value the inputs
// cannot produce, which keeps the loop from being removed.
__global__ __launch_bounds__(256) void mfma_i8_loop_kernel(int iters, int* sink) {
  const int l = (int)threadIdx.x;
  const v4i a = {l, 3 * l + 1, 5 * l + 2, 7 * l + 3};
  const v4i b = {11 * l + 4, 13 * l + 5, 17 * l + 6, 19 * l + 7};
  v4i c[kChains];
#pragma unroll
  for (int i = 0; i < kChains; ++i) c[i] = v4i{i, 0, 0, 0};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < kChains; ++i) c[i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c[i], 0, 0, 0);
  }
  int s = 0;
#pragma unroll
  for (int i = 0; i < kChains; ++i) s ^= c[i].x ^ c[i].y ^ c[i].z ^ c[i].w;
  if (s == 0x7fffffff) sink[blockIdx.x] = s;
}

// Grid-stride read of n16 16-byte words, four loads in flight per thread.
__global__ __launch_bounds__(256) void read_stream_kernel(const v4u* __restrict__ p, int64_t n16,
                                                          unsigned* sink) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  v4u acc = {0u, 0u, 0u, 0u};
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const v4u v0 = __builtin_nontemporal_load(p + i);
    const v4u v1 = __builtin_nontemporal_load(p + i + stride);
    const v4u v2 = __builtin_nontemporal_load(p + i + 2 * stride);
    const v4u v3 = __builtin_nontemporal_load(p + i + 3 * stride);
    acc ^= v0 ^ v1 ^ v2 ^ v3;
  }
  for (; i < n16; i += stride) acc ^= __builtin_nontemporal_load(p + i);
  const unsigned s = acc.x ^ acc.y ^ acc.z ^ acc.w;
  if (s == 0x9e3779b9u) sink[0] = s;
}

// The lm_head's memory traffic without its arithmetic: runs of 64 weight rows
// (64 x k bytes, contiguous) are read with 16-byte loads, all of a thread's
// loads in flight at once, and after each run the run's 64 columns of `rows`
// bf16 output rows are written as 128-byte row segments.  Workgroups take
// runs grid-stride.  k is a multiple of 64 and at most 64 * kRwMaxLoads.
constexpr int kRwMaxLoads = 24;
__global__ __launch_bounds__(256) void read_write_kernel(const v4u* __restrict__ w, int64_t n,
                                                         int k, v4u* __restrict__ out, int rows,
                                                         unsigned* sink) {
  const int t = (int)threadIdx.x;
  const int per_t = k / 64;                  // 16-byte loads per thread and run
  const int64_t run_words = (int64_t)k * 4;  // 64 rows of k bytes, in 16-byte words
  const int64_t runs = n / 64;
  const int64_t ld_row = n / 8;              // output row stride in 16-byte words
  v4u acc = {0u, 0u, 0u, 0u};
  for (int64_t r = blockIdx.x; r < runs; r += gridDim.x) {
    const v4u* src = w + r * run_words;
    v4u v[kRwMaxLoads];
#pragma unroll
    for (int u = 0; u < kRwMaxLoads; ++u)
      if (u < per_t) v[u] = __builtin_nontemporal_load(src + u * 256 + t);
#pragma unroll
    for (int u = 0; u < kRwMaxLoads; ++u)
      if (u < per_t) acc ^= v[u];
    for (int i = t; i < rows * 8; i += 256) {
      const int row = i >> 3, ch = i & 7;
      const v4u val = {acc.x, (unsigned)row, (unsigned)ch, (unsigned)r};
      __builtin_nontemporal_store(val, out + row * ld_row + r * 8 + ch);
    }
  }
  const unsigned s = acc.x ^ acc.y ^ acc.z ^ acc.w;
  if (s == 0x9e3779b9u) sink[0] = s;
}

}  // namespace

extern "C" {

int w8a8_peak_mfma_i8(int blocks, int iters, int* sink, void* stream) {
  if (blocks < 1 || iters < 1 || !sink) return 1;
  mfma_i8_loop_kernel<<<blocks, 256, 0, reinterpret_cast<hipStream_t>(stream)>>>(iters, sink);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

double w8a8_peak_mfma_i8_ops(int blocks, int iters) {
  return (double)blocks * 4 * kChains * (double)iters * (2.0 * 16 * 16 * 64);
}

int w8a8_peak_read(const void* buf, size_t bytes, int blocks, unsigned* sink, void* stream) {
  if (!buf || bytes < 16 || blocks < 1 || !sink || (reinterpret_cast<uintptr_t>(buf) & 15))
    return 1;
  read_stream_kernel<<<blocks, 256, 0, reinterpret_cast<hipStream_t>(stream)>>>(
      reinterpret_cast<const v4u*>(buf), (int64_t)(bytes / 16), sink);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

int w8a8_peak_read_write(const void* w, int64_t n, int k, void* out, int rows, int blocks,
                         unsigned* sink, void* stream) {
  if (!w || !out || !sink || n < 64 || n % 64 || k < 64 || k % 64 || k > 64 * kRwMaxLoads ||
      rows < 0 || blocks < 1 || (reinterpret_cast<uintptr_t>(w) & 15) ||
      (reinterpret_cast<uintptr_t>(out) & 15))
    return 1;
  read_write_kernel<<<blocks, 256, 0, reinterpret_cast<hipStream_t>(stream)>>>(
      reinterpret_cast<const v4u*>(w), n, k, reinterpret_cast<v4u*>(out), rows, sink);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

}  // extern "C"
