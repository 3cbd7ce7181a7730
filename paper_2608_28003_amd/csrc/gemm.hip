// MFMA GEMM kernels for gfx950: C[M x N] = A[M x K] B[N x K]^T.
//
// int8 path (eq. gemm-final): A and B are int8 codes in the packed fragment
// layout, products run on v_mfma_i32_16x16x64_i8 into exact int32 sums, and the
// epilogue applies the two scales, y = (float(acc) * s_t) * s_i.
// bf16 path (the layers a precision map keeps in bf16): A is row-major bf16,
// B packed bf16, products on v_mfma_f32_16x16x32_bf16 with fp32 sums.
//
// Every operand fragment is 1024 contiguous bytes in lane order, so one
// 16-byte load per lane moves a whole fragment, global_load_lds_dwordx4 can
// drop it straight into LDS, and every LDS read is a linear ds_read_b128.
//
// Epilogues: raw int32 (checks), dequantised f32 / bf16, the gated FFN
// activation h = bf16(gelu_tanh(g) * u) computed from the gate and up
// accumulators of the same output element (both weights are streamed by the
// same workgroup, so g and u never leave registers), or K-split partial sums.
//
// K splits write plain partial sums; a separate kernel adds them in split
// order and runs the epilogue.  The kernel boundary makes the partials
// visible, so no device-scope fence (an L2 write-back + invalidate per XCD on
// this chip) is ever issued, and the result does not depend on timing.
#include "device.h"
#include "kernels.h"

namespace w8a8 {

// ------------------------------------------------------------------ helpers

__device__ __forceinline__ v4i load_frag_packed(const void* base, int64_t rb, int64_t kb,
                                                int64_t kb_count, int lane) {
  const int8_t* p = reinterpret_cast<const int8_t*>(base) + frag_offset(rb, kb, kb_count) + lane * 16;
  return *reinterpret_cast<const v4i*>(p);
}

// bf16 A operand read straight from a row-major matrix: lane l takes row
// (l % 16) of the fragment and the 8 columns (l / 16) * 8 .. +7 of its 32.
__device__ __forceinline__ v4i load_frag_rowmajor_bf16(const void* base, int64_t row,
                                                       int64_t kb, int64_t lda, int lane) {
  const uint16_t* p = reinterpret_cast<const uint16_t*>(base) + row * lda + kb * kFragK16 +
                      (lane >> 4) * 8;
  return *reinterpret_cast<const v4i*>(p);
}

template <bool BF16>
struct Acc;
template <>
struct Acc<false> {
  typedef v4i T;
  static __device__ __forceinline__ T zero() { return v4i{0, 0, 0, 0}; }
  static __device__ __forceinline__ T mma(v4i a, v4i b, T c) { return mma_i8(a, b, c); }
};
template <>
struct Acc<true> {
  typedef v4f T;
  static __device__ __forceinline__ T zero() { return v4f{0.f, 0.f, 0.f, 0.f}; }
  static __device__ __forceinline__ T mma(v4i a, v4i b, T c) { return mma_bf16(a, b, c); }
};

// Dequantised / converted value of one accumulator element.
template <bool BF16>
__device__ __forceinline__ float acc_value(float a_or_i, const GemmParams& p, int row, int col,
                                           const float* s_b) {
  if constexpr (BF16) {
    return a_or_i;
  } else {
    float t = a_or_i * p.s_a[row];
    return t * s_b[col];
  }
}

// Store one output element for the non-gated epilogues.
template <bool BF16, int EPI>
__device__ __forceinline__ void store_elem(const GemmParams& p, int row, int col, int32_t iacc,
                                           float facc) {
  if constexpr (EPI == EPI_I32) {
    reinterpret_cast<int32_t*>(p.out)[(int64_t)row * p.ldo + col] = iacc;
  } else {
    float raw = BF16 ? facc : (float)iacc;
    float y = acc_value<BF16>(raw, p, row, col, p.s_b);
    if constexpr (EPI == EPI_F32)
      reinterpret_cast<float*>(p.out)[(int64_t)row * p.ldo + col] = y;
    else
      reinterpret_cast<uint16_t*>(p.out)[(int64_t)row * p.ldo + col] = float_to_bf16_bits(y);
  }
}

template <bool BF16>
__device__ __forceinline__ void store_glu(const GemmParams& p, int row, int col, float g_raw,
                                          float u_raw) {
  float g = acc_value<BF16>(g_raw, p, row, col, p.s_b);
  float u = acc_value<BF16>(u_raw, p, row, col, p.s_b2);
  float h = gelu_tanh(g) * u;
  reinterpret_cast<uint16_t*>(p.out)[(int64_t)row * p.ldo + col] = float_to_bf16_bits(h);
}

template <bool BF16>
__device__ __forceinline__ void write_partial(const GemmParams& p, int z, int row, int col,
                                              int32_t iacc, float facc) {
  const int64_t idx = (int64_t)z * p.M * p.N + (int64_t)row * p.N + col;
  if constexpr (BF16)
    reinterpret_cast<float*>(p.part)[idx] = facc;
  else
    reinterpret_cast<int32_t*>(p.part)[idx] = iacc;
}

// Asynchronous copy of one 16-byte piece per lane from global memory to LDS
// (global_load_lds_dwordx4): lane l writes lds_base + 16 l.
__device__ __forceinline__ void to_lds_async(const void* gsrc_lane, v4i* lds_base) {
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)gsrc_lane,
                                   (__attribute__((address_space(3))) void*)lds_base, 16, 0, 0);
}

// Wait until at most N vector-memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Barrier without the implied memory fence of __syncthreads(): the LDS-DMA
// waits are explicit (wait_vmcnt), so the compiler must not add vmcnt(0).
__device__ __forceinline__ void lds_barrier() {
  // lgkmcnt(0) with vmcnt and expcnt at their maxima (no wait on them)
  __builtin_amdgcn_s_waitcnt(0xF | (7 << 4) | (0 << 8) | (3 << 14));
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

template <int PF, int S>
__device__ __forceinline__ void wait_stage(int remaining_after) {
  // stages issued after the one we need: min(S - 2, remaining_after)
  if (remaining_after >= S - 2) {
    wait_vmcnt<PF * (S - 2)>();
  } else if constexpr (S >= 4) {
    if (remaining_after == 1) wait_vmcnt<PF>(); else wait_vmcnt<0>();
  } else {
    wait_vmcnt<0>();
  }
}

// ------------------------------------------------------------------ tiled kernel

// BM x BN output tile per workgroup of 4 waves arranged WAVES_M x (4 / WAVES_M).
// The K loop runs over an S-stage LDS ring: each stage holds BM/16 A and
// BN/16 (x2 gated) B fragments, filled by LDS-DMA loads issued S-1 steps ahead,
// so S-2 stages of HBM/L2 traffic stay in flight while the MFMAs of the
// current stage run.  One barrier per K step.
template <bool BF16, int BM, int BN, int WAVES_M, int EPI, int S>
__global__ __launch_bounds__(256) void gemm_tile_kernel(GemmParams p) {
  constexpr bool GLU = (EPI == EPI_GLU);
  constexpr int WAVES_N = 4 / WAVES_M;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int NA = BM / 16;
  constexpr int NB = (BN / 16) * (GLU ? 2 : 1);
  constexpr int NF = NA + NB;
  static_assert(NF % 4 == 0, "fragments per stage must split over 4 waves");
  constexpr int PF = NF / 4;  // fragments each wave fetches per stage
  typedef typename Acc<BF16>::T AccT;

  __shared__ v4i lds[S][NF * 64];

  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;

  const int m_tiles = (p.M + BM - 1) / BM;
  const int mt = blockIdx.x % m_tiles;
  const int nt = blockIdx.x / m_tiles;
  const int z = blockIdx.y;
  const int kb0 = z * p.kchunk;
  const int kb1 = min(p.kb_count, kb0 + p.kchunk);
  const int nk = kb1 - kb0;

  // per-wave source pointers of its PF fragments at kb = 0
  const int8_t* src[PF];
  int64_t src_step[PF];
#pragma unroll
  for (int i = 0; i < PF; ++i) {
    const int f = wave + 4 * i;
    if (f < NA) {
      int rb = min(mt * (BM / 16) + f, p.rb_a - 1);
      if constexpr (BF16) {
        int64_t row = min((int64_t)rb * 16 + (lane & 15), (int64_t)p.M - 1);
        src[i] = reinterpret_cast<const int8_t*>(reinterpret_cast<const uint16_t*>(p.A) +
                                                 row * p.lda + (lane >> 4) * 8);
        src_step[i] = kFragK16 * 2;
      } else {
        src[i] = reinterpret_cast<const int8_t*>(p.A) + frag_offset(rb, 0, p.kb_count) + lane * 16;
        src_step[i] = kFragBytes;
      }
    } else {
      int fb = f - NA;
      const void* base = p.B;
      if (GLU && fb >= BN / 16) {
        base = p.B2;
        fb -= BN / 16;
      }
      int nb = min(nt * (BN / 16) + fb, p.rb_b - 1);
      src[i] = reinterpret_cast<const int8_t*>(base) + frag_offset(nb, 0, p.kb_count) + lane * 16;
      src_step[i] = kFragBytes;
    }
  }
  auto issue = [&](int j) {  // stage j (relative to kb0) into slot j % S
    const int kb = kb0 + j;
#pragma unroll
    for (int i = 0; i < PF; ++i)
      to_lds_async(src[i] + (int64_t)kb * src_step[i], &lds[j % S][(wave + 4 * i) * 64]);
  };

  AccT acc[TM][TN];
  AccT accu[GLU ? TM : 1][GLU ? TN : 1];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      acc[i][j] = Acc<BF16>::zero();
      if constexpr (GLU) accu[i][j] = Acc<BF16>::zero();
    }

#pragma unroll
  for (int j = 0; j < S - 1; ++j)
    if (j < nk) issue(j);
  for (int j = 0; j < nk; ++j) {
    wait_stage<PF, S>(nk - 1 - j);
    lds_barrier();
    if (j + S - 1 < nk) issue(j + S - 1);
    const v4i* St = lds[j % S];
    v4i a[TM], b[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) a[i] = St[(wm * TM + i) * 64 + lane];
#pragma unroll
    for (int t = 0; t < TN; ++t) b[t] = St[(NA + wn * TN + t) * 64 + lane];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int t = 0; t < TN; ++t) acc[i][t] = Acc<BF16>::mma(a[i], b[t], acc[i][t]);
    if constexpr (GLU) {
      v4i bu[TN];
#pragma unroll
      for (int t = 0; t < TN; ++t) bu[t] = St[(NA + BN / 16 + wn * TN + t) * 64 + lane];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int t = 0; t < TN; ++t) accu[i][t] = Acc<BF16>::mma(a[i], bu[t], accu[i][t]);
    }
  }

  // ---------------- epilogue
  const int row0 = mt * BM + wm * WM + (lane >> 4) * 4;
  const int col0 = nt * BN + wn * WN + (lane & 15);
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int t = 0; t < TN; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = row0 + i * 16 + r, col = col0 + t * 16;
        if (row >= p.M || col >= p.N) continue;
        if constexpr (GLU) {
          store_glu<BF16>(p, row, col, (float)acc[i][t][r], (float)accu[i][t][r]);
        } else if (p.splits > 1) {
          write_partial<BF16>(p, z, row, col, BF16 ? 0 : (int32_t)acc[i][t][r], (float)acc[i][t][r]);
        } else {
          store_elem<BF16, EPI>(p, row, col, BF16 ? 0 : (int32_t)acc[i][t][r], (float)acc[i][t][r]);
        }
      }
}

// ------------------------------------------------------------------ skinny kernel

// M <= 16 * MB rows (MB <= 4).  The workgroup stages the A fragments of its K
// range (MB x KC fragments) in LDS with LDS-DMA loads; each wave then walks its
// own output column blocks of 16, streaming the weight fragments of a block
// (one contiguous run) from HBM in batches of KU fragments, double buffered in
// registers: the loads of batch i+1 are in flight while the MFMAs (MB per
// fragment) and, at the end of a block, the epilogue of batch i run.  For
// MB == 1 a workgroup is a single wave, so the work spreads over every CU.
// K splits (a grid dimension) write partial sums.
template <bool BF16, int MB, int KC, int EPI>
__global__ __launch_bounds__(MB == 1 ? 64 : 256) void gemm_skinny_kernel(GemmParams p,
                                                                        int nb_per_block) {
  constexpr bool GLU = (EPI == EPI_GLU);
  constexpr int KU = 9;  // weight fragments per batch and operand
  constexpr int KG = GLU ? KU : 1;
  constexpr int NW = MB == 1 ? 1 : 4;
  typedef typename Acc<BF16>::T AccT;
  __shared__ v4i lds_a[MB * KC * 64];

  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int z = blockIdx.y;
  const int kb0 = z * p.kchunk;
  const int kb1 = min(p.kb_count, kb0 + p.kchunk);
  const int kc = kb1 - kb0;  // <= KC
  const int nb_begin = blockIdx.x * nb_per_block;
  const int nb_end = min(p.rb_b, nb_begin + nb_per_block);
  const int my_first = nb_begin + wave;
  const int my_count = my_first < nb_end ? (nb_end - my_first + NW - 1) / NW : 0;
  const int bpn = (kc + KU - 1) / KU;  // batches per column block
  const int total = my_count * bpn;

  for (int f = wave; f < MB * kc; f += NW) {
    const int mb = f / kc, kk = f % kc;
    const int8_t* src;
    if constexpr (BF16) {
      int64_t row = min((int64_t)mb * 16 + (lane & 15), (int64_t)p.M - 1);
      src = reinterpret_cast<const int8_t*>(reinterpret_cast<const uint16_t*>(p.A) + row * p.lda +
                                            (int64_t)(kb0 + kk) * kFragK16 + (lane >> 4) * 8);
    } else {
      src = reinterpret_cast<const int8_t*>(p.A) +
            frag_offset(min(mb, p.rb_a - 1), kb0 + kk, p.kb_count) + lane * 16;
    }
    to_lds_async(src, &lds_a[(mb * KC + kk) * 64]);
  }

  v4i b0[KU], b1[KU], u0[KG], u1[KG];
  auto load_batch = [&](int idx, v4i (&b)[KU], v4i (&bu)[KG]) {
    const int nb = my_first + NW * (idx / bpn);
    const int k0 = (idx % bpn) * KU;
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      if (k0 + u < kc) {
        b[u] = load_frag_packed(p.B, nb, kb0 + k0 + u, p.kb_count, lane);
        if constexpr (GLU) bu[u] = load_frag_packed(p.B2, nb, kb0 + k0 + u, p.kb_count, lane);
      }
    }
  };
  if (total > 0) load_batch(0, b0, u0);  // first weights go out with the A fragments
  wait_vmcnt<0>();
  lds_barrier();

  AccT acc[MB], accu[GLU ? MB : 1];
  auto compute = [&](int idx, const v4i (&b)[KU], const v4i (&bu)[KG]) {
    const int nb = my_first + NW * (idx / bpn);
    const int bi = idx % bpn;
    const int k0 = bi * KU;
    if (bi == 0) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        acc[mb] = Acc<BF16>::zero();
        if constexpr (GLU) accu[mb] = Acc<BF16>::zero();
      }
    }
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      if (k0 + u < kc) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const v4i a = lds_a[(mb * KC + k0 + u) * 64 + lane];
          acc[mb] = Acc<BF16>::mma(a, b[u], acc[mb]);
          if constexpr (GLU) accu[mb] = Acc<BF16>::mma(a, bu[u], accu[mb]);
        }
      }
    }
    if (bi != bpn - 1) return;

    // ---- epilogue of column block nb
    const int col = nb * 16 + (lane & 15);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = mb * 16 + (lane >> 4) * 4 + r;
        if (row >= p.M || col >= p.N) continue;
        if constexpr (GLU) {
          store_glu<BF16>(p, row, col, (float)acc[mb][r], (float)accu[mb][r]);
        } else if (p.splits > 1) {
          write_partial<BF16>(p, z, row, col, BF16 ? 0 : (int32_t)acc[mb][r], (float)acc[mb][r]);
        } else {
          store_elem<BF16, EPI>(p, row, col, BF16 ? 0 : (int32_t)acc[mb][r], (float)acc[mb][r]);
        }
      }
  };

  for (int idx = 0; idx < total; idx += 2) {
    if (idx + 1 < total) load_batch(idx + 1, b1, u1);
    compute(idx, b0, u0);
    if (idx + 1 < total) {
      if (idx + 2 < total) load_batch(idx + 2, b0, u0);
      compute(idx + 1, b1, u1);
    }
  }
}

// ------------------------------------------------------------------ K-split reduction

// out = epilogue(sum over z of part[z]) for 4 consecutive columns per thread,
// the splits added in order (int32 exactly; fp32 in a fixed order).
template <bool BF16, int EPI>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmParams p) {
  const int64_t n4 = (p.N + 3) / 4;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)p.M * n4) return;
  const int row = (int)(idx / n4);
  const int col0 = (int)(idx % n4) * 4;
  const int64_t plane = (int64_t)p.M * p.N;
  const int ncol = min(4, p.N - col0);
  int32_t isum[4] = {0, 0, 0, 0};
  float fsum[4] = {0.f, 0.f, 0.f, 0.f};
  for (int zz = 0; zz < p.splits; ++zz) {
    const int64_t base = zz * plane + (int64_t)row * p.N + col0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if (c < ncol) {
        if constexpr (BF16)
          fsum[c] += reinterpret_cast<const float*>(p.part)[base + c];
        else
          isum[c] += reinterpret_cast<const int32_t*>(p.part)[base + c];
      }
    }
  }
#pragma unroll
  for (int c = 0; c < 4; ++c)
    if (c < ncol) store_elem<BF16, EPI>(p, row, col0 + c, isum[c], fsum[c]);
}

// ------------------------------------------------------------------ dispatch

template <bool BF16, int EPI>
static hipError_t tile_dispatch(int tile, const GemmParams& p, hipStream_t st) {
  auto grid_for = [&](int bm, int bn) {
    int mt = (p.M + bm - 1) / bm;
    int nt = (p.N + bn - 1) / bn;
    return dim3((unsigned)(mt * nt), (unsigned)p.splits);
  };
  if constexpr (EPI == EPI_GLU) {
    switch (tile) {
      case TILE_GLU_128x32:
        gemm_tile_kernel<BF16, 128, 32, 4, EPI, 6><<<grid_for(128, 32), 256, 0, st>>>(p);
        break;
      case TILE_GLU_64x64:
        gemm_tile_kernel<BF16, 64, 64, 2, EPI, 6><<<grid_for(64, 64), 256, 0, st>>>(p);
        break;
      case TILE_GLU_128x64:
        gemm_tile_kernel<BF16, 128, 64, 2, EPI, 4><<<grid_for(128, 64), 256, 0, st>>>(p);
        break;
      default:
        return hipErrorInvalidValue;
    }
  } else {
    switch (tile) {
      case TILE_128x128:
        gemm_tile_kernel<BF16, 128, 128, 2, EPI, 4><<<grid_for(128, 128), 256, 0, st>>>(p);
        break;
      case TILE_128x64:
        gemm_tile_kernel<BF16, 128, 64, 2, EPI, 6><<<grid_for(128, 64), 256, 0, st>>>(p);
        break;
      case TILE_64x64:
        gemm_tile_kernel<BF16, 64, 64, 2, EPI, 6><<<grid_for(64, 64), 256, 0, st>>>(p);
        break;
      case TILE_256x128:
        gemm_tile_kernel<BF16, 256, 128, 2, EPI, 3><<<grid_for(256, 128), 256, 0, st>>>(p);
        break;
      default:
        return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

hipError_t launch_gemm_tile(bool bf16, int epi, int tile, const GemmParams& p, hipStream_t st) {
  if (bf16) {
    switch (epi) {
      case EPI_F32: return tile_dispatch<true, EPI_F32>(tile, p, st);
      case EPI_BF16: return tile_dispatch<true, EPI_BF16>(tile, p, st);
      case EPI_GLU: return tile_dispatch<true, EPI_GLU>(tile, p, st);
      default: return hipErrorInvalidValue;
    }
  }
  switch (epi) {
    case EPI_I32: return tile_dispatch<false, EPI_I32>(tile, p, st);
    case EPI_F32: return tile_dispatch<false, EPI_F32>(tile, p, st);
    case EPI_BF16: return tile_dispatch<false, EPI_BF16>(tile, p, st);
    case EPI_GLU: return tile_dispatch<false, EPI_GLU>(tile, p, st);
    default: return hipErrorInvalidValue;
  }
}

template <bool BF16, int EPI, int KC>
static hipError_t skinny_mb(int mb, const GemmParams& p, int nbpb, hipStream_t st) {
  dim3 grid((unsigned)((p.rb_b + nbpb - 1) / nbpb), (unsigned)p.splits);
  switch (mb) {
    case 1: gemm_skinny_kernel<BF16, 1, KC, EPI><<<grid, 64, 0, st>>>(p, nbpb); break;
    case 2: gemm_skinny_kernel<BF16, 2, KC, EPI><<<grid, 256, 0, st>>>(p, nbpb); break;
    case 4: gemm_skinny_kernel<BF16, 4, KC, EPI><<<grid, 256, 0, st>>>(p, nbpb); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <bool BF16, int EPI>
static hipError_t skinny_kc(int mb, int kc, const GemmParams& p, int nbpb, hipStream_t st) {
  switch (kc) {
    case 9: return skinny_mb<BF16, EPI, 9>(mb, p, nbpb, st);
    case 18: return skinny_mb<BF16, EPI, 18>(mb, p, nbpb, st);
    case 36: return skinny_mb<BF16, EPI, 36>(mb, p, nbpb, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm_skinny(bool bf16, int epi, int mb, int kc, const GemmParams& p,
                              int nb_per_block, hipStream_t st) {
  if (bf16) {
    switch (epi) {
      case EPI_F32: return skinny_kc<true, EPI_F32>(mb, kc, p, nb_per_block, st);
      case EPI_BF16: return skinny_kc<true, EPI_BF16>(mb, kc, p, nb_per_block, st);
      case EPI_GLU: return skinny_kc<true, EPI_GLU>(mb, kc, p, nb_per_block, st);
      default: return hipErrorInvalidValue;
    }
  }
  switch (epi) {
    case EPI_I32: return skinny_kc<false, EPI_I32>(mb, kc, p, nb_per_block, st);
    case EPI_F32: return skinny_kc<false, EPI_F32>(mb, kc, p, nb_per_block, st);
    case EPI_BF16: return skinny_kc<false, EPI_BF16>(mb, kc, p, nb_per_block, st);
    case EPI_GLU: return skinny_kc<false, EPI_GLU>(mb, kc, p, nb_per_block, st);
    default: return hipErrorInvalidValue;
  }
}

template <bool BF16>
static hipError_t reduce_epi(int epi, const GemmParams& p, hipStream_t st) {
  const int64_t n4 = (p.N + 3) / 4;
  const unsigned blocks = (unsigned)((p.M * n4 + 255) / 256);
  switch (epi) {
    case EPI_I32:
      if constexpr (BF16) return hipErrorInvalidValue;
      else splitk_reduce_kernel<false, EPI_I32><<<blocks, 256, 0, st>>>(p);
      break;
    case EPI_F32: splitk_reduce_kernel<BF16, EPI_F32><<<blocks, 256, 0, st>>>(p); break;
    case EPI_BF16: splitk_reduce_kernel<BF16, EPI_BF16><<<blocks, 256, 0, st>>>(p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_splitk_reduce(bool bf16, int epi, const GemmParams& p, hipStream_t st) {
  return bf16 ? reduce_epi<true>(epi, p, st) : reduce_epi<false>(epi, p, st);
}

}  // namespace w8a8
