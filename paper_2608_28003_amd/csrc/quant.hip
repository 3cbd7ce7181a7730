// Calibration, smoothing and symmetric int8 quantisation kernels (gfx950).
//
//   col_absmax      running max_t |X_tj|, the statistic of Sec. 4 eq. delta-attn
//   smooth_delta    delta_j = a_j^alpha / w_j^(1-alpha)          (eq. delta-lmhead)
//   quant_rows      per-row symmetric int8 codes of x / delta (eq. xhat-lmhead,
//                   stx, xint8) or W * delta (eq. what-lmhead, si, what-ffn),
//                   written straight into the packed fragment layout the GEMMs read
//   unpack          packed layout -> row-major int8 (checks only)
//   pack_bf16       row-major bf16 -> packed bf16 layout (bf16 path weights)
//
// Quantisation runs one workgroup per row: each thread owns a 16-column (or,
// for few rows, 8-column) chunk held in registers, a butterfly + LDS max gives
// the row absmax, and each chunk becomes one 16-byte (8-byte) store into its
// fragment slot.  All arithmetic is IEEE binary32 (correctly rounded division,
// v_rndne_f32 for round-half-to-even, no contraction).
#include "device.h"
#include "kernels.h"

namespace w8a8 {

// ------------------------------------------------------------------ loads

template <typename T>
__device__ __forceinline__ void load16(const T* p, float (&v)[16]);

template <>
__device__ __forceinline__ void load16<float>(const float* p, float (&v)[16]) {
  const float4* q = reinterpret_cast<const float4*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float4 t = q[i];
    v[4 * i + 0] = t.x; v[4 * i + 1] = t.y; v[4 * i + 2] = t.z; v[4 * i + 3] = t.w;
  }
}

template <>
__device__ __forceinline__ void load16<uint16_t>(const uint16_t* p, float (&v)[16]) {
  const uint4* q = reinterpret_cast<const uint4*>(p);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    uint4 t = q[i];
    uint32_t w[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[8 * i + 2 * j + 0] = bf16_bits_to_float(w[j] & 0xffffu);
      v[8 * i + 2 * j + 1] = bf16_bits_to_float(w[j] >> 16);
    }
  }
}

template <typename T>
__device__ __forceinline__ void load8(const T* p, float (&v)[8]);

template <>
__device__ __forceinline__ void load8<float>(const float* p, float (&v)[8]) {
  const float4* q = reinterpret_cast<const float4*>(p);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    float4 t = q[i];
    v[4 * i + 0] = t.x; v[4 * i + 1] = t.y; v[4 * i + 2] = t.z; v[4 * i + 3] = t.w;
  }
}

template <>
__device__ __forceinline__ void load8<uint16_t>(const uint16_t* p, float (&v)[8]) {
  const uint4 t = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[2 * j + 0] = bf16_bits_to_float(w[j] & 0xffffu);
    v[2 * j + 1] = bf16_bits_to_float(w[j] >> 16);
  }
}

template <typename T, int CW>
__device__ __forceinline__ void load_chunk(const T* p, float (&v)[CW]) {
  if constexpr (CW == 16)
    load16<T>(p, v);
  else
    load8<T>(p, v);
}

// ------------------------------------------------------------------ a1

template <typename T>
__global__ __launch_bounds__(256) void col_absmax_kernel(const T* __restrict__ x, int64_t rows,
                                                         int64_t k, int rows_per_block,
                                                         float* __restrict__ amax) {
  int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j >= k) return;
  int64_t r0 = (int64_t)blockIdx.y * rows_per_block;
  int64_t r1 = r0 + rows_per_block < rows ? r0 + rows_per_block : rows;
  float m = 0.0f;
  for (int64_t r = r0; r < r1; ++r) {
    float v;
    if constexpr (sizeof(T) == 2)
      v = bf16_bits_to_float(x[r * k + j]);
    else
      v = x[r * k + j];
    m = fmaxf(m, fabsf(v));
  }
  // non-negative binary32 values order like their unsigned bit patterns
  atomicMax(reinterpret_cast<unsigned int*>(amax) + j, __float_as_uint(m));
}

__global__ void smooth_delta_kernel(const float* __restrict__ a, const float* __restrict__ w,
                                    int64_t k, double alpha, float* __restrict__ delta) {
  int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= k) return;
  const double eps = 1e-5;
  double aj = (double)a[j], wj = (double)w[j];
  if (aj < eps) aj = eps;
  if (wj < eps) wj = eps;
  double d = (alpha == 0.5) ? sqrt(aj) / sqrt(wj) : pow(aj, alpha) / pow(wj, 1.0 - alpha);
  delta[j] = (float)d;
}

// ------------------------------------------------------------------ a2 / a3

// Workgroup-wide maximum (blockDim.x a multiple of 64, at most 1024).
__device__ __forceinline__ float block_max(float v) {
  __shared__ float red[16];
  v = wave_max(v);
  const int w = threadIdx.x >> 6;
  if (lane_id() == 0) red[w] = v;
  __syncthreads();
  float m = red[0];
  for (int i = 1; i < (int)(blockDim.x >> 6); ++i) m = fmaxf(m, red[i]);
  return m;
}

// Chunk c of CW (16 or 8) consecutive columns of row xr, smoothed.  GLU: the
// row's values are the gated activation h = bf16(gelu_tanh(g) * u) of the
// binary32 rows g (xr) and u (ur) -- the arithmetic of the gate/up GEMM's
// epilogue on sums given in memory -- and h is also stored to hr (if set).
template <typename T, bool MUL, int CW, bool GLU = false>
__device__ __forceinline__ void smooth_chunk(const T* __restrict__ xr,
                                             const float* __restrict__ delta, int64_t c,
                                             float (&v)[CW], const float* __restrict__ ur = nullptr,
                                             uint16_t* __restrict__ hr = nullptr) {
  if constexpr (GLU) {
    static_assert(sizeof(T) == 4, "g and u are binary32");
    float g[CW], u[CW];
    load_chunk<float, CW>(reinterpret_cast<const float*>(xr) + c * CW, g);
    load_chunk<float, CW>(ur + c * CW, u);
    uint32_t hb[CW / 2];
#pragma unroll
    for (int e = 0; e < CW; e += 2) {
      const uint16_t b0 = float_to_bf16_bits(gelu_tanh(g[e]) * u[e]);
      const uint16_t b1 = float_to_bf16_bits(gelu_tanh(g[e + 1]) * u[e + 1]);
      v[e] = bf16_bits_to_float(b0);
      v[e + 1] = bf16_bits_to_float(b1);
      hb[e / 2] = (uint32_t)b0 | ((uint32_t)b1 << 16);
    }
    if (hr) {
#pragma unroll
      for (int i = 0; i < CW / 8; ++i)
        reinterpret_cast<uint4*>(hr + c * CW)[i] =
            make_uint4(hb[4 * i], hb[4 * i + 1], hb[4 * i + 2], hb[4 * i + 3]);
    }
  } else {
    load_chunk<T, CW>(xr + c * CW, v);
  }
  if (delta) {
    float d[CW];
    load_chunk<float, CW>(delta + c * CW, d);
#pragma unroll
    for (int e = 0; e < CW; ++e) v[e] = MUL ? v[e] * d[e] : v[e] / d[e];
  }
}

// The codes of chunk c (CW columns) of row r into their fragment slot: a
// 16-column chunk is one 16-byte row segment, an 8-column chunk half of one.
template <int CW>
__device__ __forceinline__ void store_codes(int8_t* __restrict__ q, int64_t r, int64_t c,
                                            int64_t kb_count, const int32_t (&packed)[CW / 4]) {
  const int64_t c16 = c / (16 / CW);
  const int64_t kb = c16 >> 2;
  const int g = (int)(c16 & 3);
  const int64_t off = frag_offset(r >> 4, kb, kb_count) + (int64_t)((r & 15) + 16 * g) * 16;
  if constexpr (CW == 16)
    *reinterpret_cast<int4*>(q + off) = make_int4(packed[0], packed[1], packed[2], packed[3]);
  else
    *reinterpret_cast<int2*>(q + off + 8 * (c & 1)) = make_int2(packed[0], packed[1]);
}

// One workgroup per row r of a rows x k matrix (k % 16 == 0); thread t owns the
// CW-column chunk t (and t + blockDim, ... for very long rows), keeping its
// smoothed values in registers between the absmax and the rounding pass.
// CW = 16, or 8 for few rows, where halving each thread's serial divisions
// shortens the one dependent chain a launch has.
// Rows in [rows, rows_pad) and columns in [k, kp) of the packed output are
// written as zeros.  MUL: v = x * delta (weights); else v = x / delta.
// F8: OCP E4M3 codes instead of int8, s = amax / 448 and code = E4M3(v / s)
// (binary32 quotient rounded to the nearest E4M3 value, ties to even).
// GLU: the rows are the gated activation of the binary32 rows x (g) and u (see
// smooth_chunk), written to h_out (if set) as bf16 m x k.
template <typename T, bool MUL, bool F8, int CW, bool GLU = false>
__global__ __launch_bounds__(1024) void quant_rows_kernel(const T* __restrict__ x, int64_t rows,
                                                          int64_t k, const float* __restrict__ delta,
                                                          int64_t rows_pad, int64_t kp,
                                                          int8_t* __restrict__ q,
                                                          float* __restrict__ s,
                                                          const float* __restrict__ u = nullptr,
                                                          uint16_t* __restrict__ h_out = nullptr) {
  static_assert(CW == 16 || CW == 8, "chunk width");
  const int64_t r = blockIdx.x;
  const int t = threadIdx.x;
  const int nt = blockDim.x;
  const int64_t kb_count = kp / kFragK8;
  const int64_t chunks_pad = kp / CW;
  const int64_t chunks = k / CW;
  int32_t zeros[CW / 4];
#pragma unroll
  for (int i = 0; i < CW / 4; ++i) zeros[i] = 0;

  if (r >= rows) {  // padding row: zeros
    for (int64_t c = t; c < chunks_pad; c += nt) store_codes<CW>(q, r, c, kb_count, zeros);
    return;
  }

  const T* xr = x + r * k;
  const float* ur = GLU ? u + r * k : nullptr;
  uint16_t* hr = GLU && h_out ? h_out + r * k : nullptr;
  float v[CW];
  float amax = 0.0f;
  if (t < chunks) {
    smooth_chunk<T, MUL, CW, GLU>(xr, delta, t, v, ur, hr);
#pragma unroll
    for (int e = 0; e < CW; ++e) amax = fmaxf(amax, fabsf(v[e]));
  }
  for (int64_t c = t + nt; c < chunks; c += nt) {  // rows longer than CW * blockDim
    float w[CW];
    smooth_chunk<T, MUL, CW, GLU>(xr, delta, c, w, ur, hr);
#pragma unroll
    for (int e = 0; e < CW; ++e) amax = fmaxf(amax, fabsf(w[e]));
  }
  amax = block_max(amax);
  const float sr = amax / (F8 ? 448.0f : 127.0f);
  if (t == 0) s[r] = sr;
  const float inv = 1.0f / sr;
  const bool fast = isfinite(inv);

  for (int64_t c = t; c < chunks_pad; c += nt) {
    int32_t packed[CW / 4];
#pragma unroll
    for (int i = 0; i < CW / 4; ++i) packed[i] = 0;
    if (c < chunks && sr != 0.0f) {
      float w[CW];
      if (c == t) {
#pragma unroll
        for (int e = 0; e < CW; ++e) w[e] = v[e];
      } else {
        smooth_chunk<T, MUL, CW, GLU>(xr, delta, c, w, ur, nullptr);
      }
      if constexpr (F8) {
#pragma unroll
        for (int e = 0; e < CW; e += 2) {
          // the conversion gives NaN past the largest code; the quotient only
          // exceeds 448 when the scale itself lost precision (amax near the
          // binary32 subnormal range), and the nearest code is then 448
          const float q0 = fminf(fmaxf(w[e] / sr, -448.0f), 448.0f);
          const float q1 = fminf(fmaxf(w[e + 1] / sr, -448.0f), 448.0f);
          const uint32_t pair = e4m3_pack2(q0, q1);
          packed[e >> 2] |= (int32_t)(pair << (8 * (e & 3)));
        }
      } else {
#pragma unroll
        for (int e = 0; e < CW; ++e) {
          int32_t iv = (int32_t)code_of(w[e], sr, inv, fast) & 0xff;
          packed[e >> 2] |= iv << (8 * (e & 3));
        }
      }
    }
    store_codes<CW>(q, r, c, kb_count, packed);
  }
}

// ------------------------------------------------------------------ many rows of bf16

// Correctly rounded binary32 quotient a / b for binary32 a and a reciprocal
// rb = RN64(1 / b) formed once: RN32(RN64(a * rb)).  The exact quotient of two
// binary32 numbers is never a binary32 rounding midpoint and lies more than
// 2^-49 (relative) away from every midpoint of the normal range (write a = A 2^x,
// b = B 2^y, a midpoint (2K + 1) 2^(z - 1) with A, B, K < 2^24: a - midpoint * b
// is a nonzero multiple of 2^(z - 1 + y)); the two binary64 roundings err by at
// most 2^-52, so the final rounding lands on the same binary32 value as a / b
// rounded once.  Quotients below the normal range (|result| < 2^-126, a != 0)
// are not covered; callers take the IEEE division for them.
__device__ __forceinline__ float div_via_f64(float a, double rb) {
  return (float)((double)a * rb);
}

// Per-token quantisation of R rows of a bf16 matrix per workgroup (the large-M
// activation and requantisation path): thread t owns the 16-column chunk t of
// each row, the smoothing factors' reciprocals are formed once per workgroup,
// all R rows' loads are in flight together, and one block reduction gives
// the R row maxima.  Same results as quant_rows_kernel (x / delta and v / s
// correctly rounded, see div_via_f64; the maximum does not depend on order).
//
// Quotients x / delta below the normal range are the one case div_via_f64
// does not cover, and they are settled per row, not per element: if the row's
// maximum is at least 2^-118, such an element is not the maximum (its value is
// below 2^-126 on either route) and its code is 0 on either route (|v / s| <=
// 127 * 2^-126 / 2^-118 < 1/2); a row below 2^-118 is redone with IEEE
// divisions.
template <int R>
__global__ __launch_bounds__(1024) void quant_rows_bf16_kernel(
    const uint16_t* __restrict__ x, int64_t rows, int64_t k, const float* __restrict__ delta,
    int64_t rows_pad, int64_t kp, int8_t* __restrict__ q, float* __restrict__ s) {
  __shared__ float red[R][16];
  __shared__ float red_ieee[16];
  const int t = threadIdx.x;
  const int nw = blockDim.x >> 6;
  const int64_t r0 = (int64_t)blockIdx.x * R;
  const int64_t kb_count = kp / kFragK8;
  const int64_t chunks = k / 16, chunks_pad = kp / 16;
  const bool own = t < chunks;

  double rd[16];
  if (own && delta) {
    float d[16];
    load16<float>(delta + (int64_t)t * 16, d);
#pragma unroll
    for (int e = 0; e < 16; ++e) rd[e] = 1.0 / (double)d[e];
  }
  uint4 raw[R][2];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    if (own && r0 + i < rows) {
      const uint4* p = reinterpret_cast<const uint4*>(x + (r0 + i) * k + (int64_t)t * 16);
      raw[i][0] = p[0];
      raw[i][1] = p[1];
    } else {
      raw[i][0] = raw[i][1] = make_uint4(0u, 0u, 0u, 0u);
    }
  }
  float v[R][16];
  float mx[R];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const uint32_t w[8] = {raw[i][0].x, raw[i][0].y, raw[i][0].z, raw[i][0].w,
                           raw[i][1].x, raw[i][1].y, raw[i][1].z, raw[i][1].w};
    float m = 0.0f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float xv = bf16_bits_to_float((e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xffffu));
      v[i][e] = delta ? div_via_f64(xv, rd[e]) : xv;
      m = fmaxf(m, fabsf(v[i][e]));
    }
    mx[i] = wave_max(m);
  }
  if ((t & 63) == 0) {
#pragma unroll
    for (int i = 0; i < R; ++i) red[i][t >> 6] = mx[i];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < R; ++i) {
    float m = red[i][0];
    for (int w = 1; w < nw; ++w) m = fmaxf(m, red[i][w]);
    mx[i] = m;
  }
  // rows below 2^-118 (every thread holds the same maximum: a uniform branch)
#pragma unroll
  for (int i = 0; i < R; ++i) {
    if (!delta || r0 + i >= rows || !(mx[i] < 0x1p-118f)) continue;
    float m = 0.0f;
    if (own) {  // the row is read again (the registers holding it are free by now)
      float d[16];
      load16<float>(delta + (int64_t)t * 16, d);
      const uint4* p = reinterpret_cast<const uint4*>(x + (r0 + i) * k + (int64_t)t * 16);
      const uint4 w0 = p[0], w1 = p[1];
      const uint32_t w[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        v[i][e] = bf16_bits_to_float((e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xffffu)) / d[e];
        m = fmaxf(m, fabsf(v[i][e]));
      }
    }
    m = wave_max(m);
    __syncthreads();  // an earlier row's maxima have been read
    if ((t & 63) == 0) red_ieee[t >> 6] = m;
    __syncthreads();
    m = red_ieee[0];
    for (int w = 1; w < nw; ++w) m = fmaxf(m, red_ieee[w]);
    mx[i] = m;
  }
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int64_t r = r0 + i;
    if (r >= rows_pad) break;
    int32_t packed[4] = {0, 0, 0, 0};
    if (r < rows) {
      const float sr = mx[i] / 127.0f;
      if (t == 0) s[r] = sr;
      if (own && sr != 0.0f) {
        const double rs = 1.0 / (double)sr;
        uint32_t b[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          // |v / s| <= 127 (1 + 2^-23) except for a subnormal scale; clamping
          // before rounding gives the codes of rounding first, as in code_of.
          // c + 1.5 * 2^23 rounds c to an integer, ties to even (the offset is
          // even), and its low byte is that integer in two's complement.
          const float c = fminf(fmaxf(div_via_f64(v[i][e], rs), -127.0f), 127.0f);
          b[e] = __float_as_uint(c + 12582912.0f);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
          packed[j] = (int32_t)((b[4 * j] & 0xffu) | ((b[4 * j + 1] & 0xffu) << 8) |
                                ((b[4 * j + 2] & 0xffu) << 16) | (b[4 * j + 3] << 24));
      }
    }
    // blockDim covers chunks_pad: one chunk per thread (padding columns and
    // padding rows get zero codes)
    if (t < chunks_pad) store_codes<16>(q, r, t, kb_count, packed);
  }
}

// packed int8 -> row-major int8 (n x k)
__global__ void unpack_kernel(const int8_t* __restrict__ qp, int64_t n, int64_t k, int64_t kp,
                              int8_t* __restrict__ q) {
  int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n * k) return;
  int64_t r = idx / k, c = idx % k;
  int64_t kb = c / kFragK8;
  int g = (int)((c % kFragK8) / 16);
  int e = (int)(c % 16);
  int64_t off = frag_offset(r >> 4, kb, kp / kFragK8) + (int64_t)((r & 15) + 16 * g) * 16 + e;
  q[idx] = qp[off];
}

// row-major bf16 (n x k, k % 8 == 0) -> packed bf16 layout; one thread per
// 8-element (16-byte) chunk of the padded matrix.
__global__ void pack_bf16_kernel(const uint16_t* __restrict__ w, int64_t n, int64_t k,
                                 int64_t n_pad, int64_t kp, uint16_t* __restrict__ wp) {
  int64_t chunk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t chunks_row = kp / 8;
  if (chunk >= n_pad * chunks_row) return;
  int64_t r = chunk / chunks_row, c = chunk % chunks_row;
  uint4 val = make_uint4(0, 0, 0, 0);
  if (r < n && c * 8 < k) val = *reinterpret_cast<const uint4*>(w + r * k + c * 8);
  int64_t kb = c >> 2;
  int g = (int)(c & 3);
  int64_t off = frag_offset(r >> 4, kb, kp / kFragK16) + (int64_t)((r & 15) + 16 * g) * 16;
  *reinterpret_cast<uint4*>(reinterpret_cast<int8_t*>(wp) + off) = val;
}

// ------------------------------------------------------------------ launchers

hipError_t launch_col_absmax(const void* x, bool bf16, int64_t rows, int64_t k, float* amax,
                             hipStream_t st) {
  const int rpb = 64;
  dim3 grid((unsigned)((k + 255) / 256), (unsigned)((rows + rpb - 1) / rpb));
  if (bf16)
    col_absmax_kernel<uint16_t><<<grid, 256, 0, st>>>((const uint16_t*)x, rows, k, rpb, amax);
  else
    col_absmax_kernel<float><<<grid, 256, 0, st>>>((const float*)x, rows, k, rpb, amax);
  return hipGetLastError();
}

__global__ void fill_f32_kernel(float* __restrict__ p, int64_t n, float v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

hipError_t launch_fill_f32(float* p, int64_t n, float v, hipStream_t st) {
  fill_f32_kernel<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(p, n, v);
  return hipGetLastError();
}

hipError_t launch_smooth_delta(const float* a, const float* w, int64_t k, double alpha,
                               float* delta, hipStream_t st) {
  smooth_delta_kernel<<<(unsigned)((k + 255) / 256), 256, 0, st>>>(a, w, k, alpha, delta);
  return hipGetLastError();
}

template <bool F8, int CW>
static void quant_rows_launch(const void* x, bool bf16, bool mul, int64_t rows, int64_t k,
                              const float* delta, int64_t rows_pad, int64_t kp, int8_t* qpacked,
                              float* s, dim3 grid, dim3 block, hipStream_t st) {
  if (bf16) {
    if (mul)
      quant_rows_kernel<uint16_t, true, F8, CW><<<grid, block, 0, st>>>(
          (const uint16_t*)x, rows, k, delta, rows_pad, kp, qpacked, s);
    else
      quant_rows_kernel<uint16_t, false, F8, CW><<<grid, block, 0, st>>>(
          (const uint16_t*)x, rows, k, delta, rows_pad, kp, qpacked, s);
  } else {
    if (mul)
      quant_rows_kernel<float, true, F8, CW><<<grid, block, 0, st>>>(
          (const float*)x, rows, k, delta, rows_pad, kp, qpacked, s);
    else
      quant_rows_kernel<float, false, F8, CW><<<grid, block, 0, st>>>(
          (const float*)x, rows, k, delta, rows_pad, kp, qpacked, s);
  }
}

hipError_t launch_quant_rows(const void* x, bool bf16, bool mul, int64_t rows, int64_t k,
                             const float* delta, int8_t* qpacked, float* s, hipStream_t st,
                             bool f8) {
  const int64_t rows_pad = (rows + 15) / 16 * 16;
  const int64_t kp = (k + kFragK8 - 1) / kFragK8 * kFragK8;
  // 8-column chunks while the rows leave CUs idle (one workgroup per row) and a
  // row still fits one workgroup
  const bool narrow = rows_pad <= 256 && kp / 8 <= 1024;
  if (bf16 && !mul && !f8 && !narrow && kp / 16 <= 1024) {
    // many bf16 rows (activations): several rows per workgroup
    const int64_t threads = (kp / 16 + 63) / 64 * 64;
    // rows per workgroup, measured at k = 6912 (requantisation of h): 4 from
    // 2048 rows (17.9 against 19.8 us with 2), 2 below (512 rows: 8.3 against
    // 11.2 us; 1024 rows: 11.7 against 12.5 us); at k = 1152, 2048 rows: 7.4
    // against 10.0 us
    const int r = quant_rows_per_workgroup(rows_pad >= 2048 && kp >= 4096 ? 4 : 2);
#define W8A8_QROWS(R)                                                                      \
  quant_rows_bf16_kernel<R><<<(unsigned)((rows_pad + R - 1) / R), (unsigned)threads, 0, st>>>( \
      (const uint16_t*)x, rows, k, delta, rows_pad, kp, qpacked, s)
    if (r == 1) W8A8_QROWS(1);
    else if (r == 2) W8A8_QROWS(2);
    else if (r == 8) W8A8_QROWS(8);
    else W8A8_QROWS(4);
#undef W8A8_QROWS
    return hipGetLastError();
  }
  int64_t threads = (kp / (narrow ? 8 : 16) + 63) / 64 * 64;
  if (threads > 1024) threads = 1024;
  dim3 grid((unsigned)rows_pad), block((unsigned)threads);
  if (f8) {
    if (narrow)
      quant_rows_launch<true, 8>(x, bf16, mul, rows, k, delta, rows_pad, kp, qpacked, s, grid,
                                 block, st);
    else
      quant_rows_launch<true, 16>(x, bf16, mul, rows, k, delta, rows_pad, kp, qpacked, s, grid,
                                  block, st);
  } else {
    if (narrow)
      quant_rows_launch<false, 8>(x, bf16, mul, rows, k, delta, rows_pad, kp, qpacked, s, grid,
                                  block, st);
    else
      quant_rows_launch<false, 16>(x, bf16, mul, rows, k, delta, rows_pad, kp, qpacked, s, grid,
                                   block, st);
  }
  return hipGetLastError();
}

hipError_t launch_geglu_requant(const float* g, const float* u, int64_t m, int64_t n,
                                const float* delta, int8_t* qpacked, float* s, uint16_t* h,
                                hipStream_t st) {
  const int64_t rows_pad = (m + 15) / 16 * 16;
  const int64_t kp = (n + kFragK8 - 1) / kFragK8 * kFragK8;
  const bool narrow = rows_pad <= 256 && kp / 8 <= 1024;  // as launch_quant_rows
  int64_t threads = (kp / (narrow ? 8 : 16) + 63) / 64 * 64;
  if (threads > 1024) threads = 1024;
  dim3 grid((unsigned)rows_pad), block((unsigned)threads);
  if (narrow)
    quant_rows_kernel<float, false, false, 8, true><<<grid, block, 0, st>>>(
        g, m, n, delta, rows_pad, kp, qpacked, s, u, h);
  else
    quant_rows_kernel<float, false, false, 16, true><<<grid, block, 0, st>>>(
        g, m, n, delta, rows_pad, kp, qpacked, s, u, h);
  return hipGetLastError();
}

hipError_t launch_unpack(const void* qp, int64_t n, int64_t k, int8_t* q, hipStream_t st) {
  const int64_t kp = (k + kFragK8 - 1) / kFragK8 * kFragK8;
  int64_t total = n * k;
  unpack_kernel<<<(unsigned)((total + 255) / 256), 256, 0, st>>>((const int8_t*)qp, n, k, kp, q);
  return hipGetLastError();
}

hipError_t launch_pack_bf16(const void* w, int64_t n, int64_t k, void* wp, hipStream_t st) {
  const int64_t n_pad = (n + 15) / 16 * 16;
  const int64_t kp = (k + kFragK16 - 1) / kFragK16 * kFragK16;
  int64_t total = n_pad * (kp / 8);
  pack_bf16_kernel<<<(unsigned)((total + 255) / 256), 256, 0, st>>>(
      (const uint16_t*)w, n, k, n_pad, kp, (uint16_t*)wp);
  return hipGetLastError();
}

}  // namespace w8a8
