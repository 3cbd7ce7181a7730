// Device-side helpers shared by the gfx950 kernels of the W8A8 library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace w8a8 {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

constexpr int kWave = 64;        // CDNA wavefront
constexpr int kFragBytes = 1024; // one 16 x 64 int8 (or 16 x 32 bf16) fragment

__device__ __forceinline__ float bf16_bits_to_float(uint32_t b) {
  return __uint_as_float(b << 16);
}

// binary32 -> bf16, round to nearest even; NaN stays a quiet NaN.
// binary32 -> bfloat16, round to nearest even (one v_cvt_pk_bf16_f32 on gfx950)
__device__ __forceinline__ uint16_t float_to_bf16_bits(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// v[l ^ m] for the butterfly masks m = 32, 16, 8, 4, 2, 1: lane permutations
// without an LDS round trip where the hardware has one (DPP within a row of
// 16 lanes, a swizzle across 32, a permute across 64).  A permutation moves
// values exactly, so the reductions below add the same pairs in the same
// order as a butterfly of __shfl_xor and give the same bits.
template <int M>
__device__ __forceinline__ float lane_xor(float v) {
  const int b = __float_as_int(v);
  int r;
  if constexpr (M == 1) {
    r = __builtin_amdgcn_update_dpp(0, b, 0xB1, 0xF, 0xF, true);  // quad_perm [1, 0, 3, 2]
  } else if constexpr (M == 2) {
    r = __builtin_amdgcn_update_dpp(0, b, 0x4E, 0xF, 0xF, true);  // quad_perm [2, 3, 0, 1]
  } else if constexpr (M == 4) {
    // mirror within 8 lanes (l ^ 7), then reverse each quad (^ 3)
    const int h = __builtin_amdgcn_update_dpp(0, b, 0x141, 0xF, 0xF, true);
    r = __builtin_amdgcn_update_dpp(0, h, 0x1B, 0xF, 0xF, true);
  } else if constexpr (M == 8) {
    r = __builtin_amdgcn_update_dpp(0, b, 0x128, 0xF, 0xF, true);  // rotate a row of 16 by 8
  } else if constexpr (M == 16) {
    r = __builtin_amdgcn_ds_swizzle(b, 0x401F);  // bitmask swizzle: lane ^ 16 within 32
  } else {
    static_assert(M == 32, "butterfly masks 1 ... 32");
    r = __builtin_amdgcn_ds_bpermute((int)((threadIdx.x & (kWave - 1)) ^ 32) << 2, b);
  }
  return __int_as_float(r);
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, lane_xor<32>(v));
  v = fmaxf(v, lane_xor<16>(v));
  v = fmaxf(v, lane_xor<8>(v));
  v = fmaxf(v, lane_xor<4>(v));
  v = fmaxf(v, lane_xor<2>(v));
  return fmaxf(v, lane_xor<1>(v));
}

__device__ __forceinline__ float wave_sum(float v) {
  v += lane_xor<32>(v);
  v += lane_xor<16>(v);
  v += lane_xor<8>(v);
  v += lane_xor<4>(v);
  v += lane_xor<2>(v);
  return v + lane_xor<1>(v);
}

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }

// Byte offset of fragment (rb, kb) in a packed matrix with kb_count fragment columns.
__device__ __forceinline__ int64_t frag_offset(int64_t rb, int64_t kb, int64_t kb_count) {
  return (rb * kb_count + kb) * (int64_t)kFragBytes;
}

// Weight fragments stream through once: non-temporal loads keep them from
// displacing reused data in the caches (measured: +15 % on the decode lm_head).
__device__ __forceinline__ v4i load_frag_packed(const void* base, int64_t rb, int64_t kb,
                                                int64_t kb_count, int lane) {
  const int8_t* p = reinterpret_cast<const int8_t*>(base) + frag_offset(rb, kb, kb_count) + lane * 16;
  return __builtin_nontemporal_load(reinterpret_cast<const v4i*>(p));
}

// 16x16x64 int8 MFMA: C[i][j] += sum_k A[i][k] B[j][k]; lane l supplies row
// (l % 16) of A and of B with the same 16 k values, so any fixed assignment of
// k to (lane group, byte) used by both operands gives the same sum.  The
// accumulator element r of lane l is C[4 (l / 16) + r][l % 16].
__device__ __forceinline__ v4i mma_i8(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ v4f mma_bf16(v4i a, v4i b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a),
                                                 __builtin_bit_cast(v8bf, b), c, 0, 0, 0);
}

// FP8 E4M3 x E4M3 -> fp32, K = 128: the two 16 x 64 fragments of each operand
// are concatenated per lane (fragment 0's 16 bytes, then fragment 1's).  Any
// assignment of K positions to lanes works as long as A and B use the same one.
typedef int v8i __attribute__((ext_vector_type(8)));
__device__ __forceinline__ v4f mma_f8(v4i a0, v4i a1, v4i b0, v4i b1, v4f c) {
  const v8i a = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
  const v8i b = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
  // formats 0 / 0: both operands OCP E4M3; no block scales
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// binary32 pair -> two E4M3 codes (round to nearest even), low 16 bits
__device__ __forceinline__ uint32_t e4m3_pack2(float lo, float hi) {
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(lo, hi, 0, false) & 0xffffu;
}

// GELU with the tanh form, binary32 operations in a fixed order (the library
// is compiled without floating-point contraction).
__device__ __forceinline__ float gelu_tanh(float x) {
  // 0.5 x (1 + tanh(z)) equals x / (1 + 2^a) with a = -2 z log2(e): no
  // cancellation for z < 0, one exp2 and one reciprocal, no branch.
  // z = sqrt(2/pi) (x + 0.044715 x^3); kE = -2 sqrt(2/pi) log2(e).
  // For a above 126 the reciprocal leaves the normal binary32 range and the
  // result (below 2^-126 |x| in magnitude) may come out as zero.
  const float k3 = 0.044715f;
  const float kE = -2.3022082f;
  float x2 = x * x;
  float inner = x + (k3 * x2) * x;
  float a = inner * kE;
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(a));
}

// Workgroup reductions over the per-thread values of one row; each call site
// passes its own LDS array, so consecutive reductions need no extra barrier.
// The sum adds the per-wave sums in wave order, so waves whose threads all
// contribute 0 (a larger workgroup over the same row) leave it unchanged.
__device__ __forceinline__ float block_sum_in(float v, float* red) {
  v = wave_sum(v);
  if (lane_id() == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float s = 0.0f;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) s += red[i];
  return s;
}

__device__ __forceinline__ float block_max_in(float v, float* red) {
  v = wave_max(v);
  if (lane_id() == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float m = red[0];
  for (int i = 1; i < (int)(blockDim.x >> 6); ++i) m = fmaxf(m, red[i]);
  return m;
}

// q = rne(v / s) clamped to [-127, 127], with v / s the correctly rounded
// binary32 quotient.  Fast path: v * inv with inv = 1/s differs from v / s by at
// most 2.3e-5 for |v / s| <= 127.5 (two roundings of 2^-24 each plus the one of
// the quotient), so whenever v * inv is more than 2^-10 away from a half-integer
// both round to the same integer; otherwise (or when inv is not finite) the
// exact quotient is formed.
__device__ __forceinline__ int8_t code_of(float v, float s, float inv, bool fast) {
  float c;
  if (fast) {
    float q = v * inv;
    float fr = fabsf(q - truncf(q));
    if (fabsf(fr - 0.5f) > 0.0009765625f)
      c = rintf(q);
    else
      c = rintf(v / s);
  } else {
    c = rintf(v / s);
  }
  c = fminf(fmaxf(c, -127.0f), 127.0f);
  return (int8_t)(int)c;
}

}  // namespace w8a8
