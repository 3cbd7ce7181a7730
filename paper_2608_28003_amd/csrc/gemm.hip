// MFMA GEMM kernels for gfx950: C[M x N] = A[M x K] B[N x K]^T.
//
// int8 path (eq. gemm-final): A and B are int8 codes in the packed fragment
// layout, products run on v_mfma_i32_16x16x64_i8 into exact int32 sums, and the
// epilogue applies the two scales, y = (float(acc) * s_t) * s_i.
// bf16 path (the layers a precision map keeps in bf16): A is row-major bf16,
// B packed bf16, products on v_mfma_f32_16x16x32_bf16 with fp32 sums.
// FP8 path (E4M3 codes, packed like int8): one v_mfma_f32_16x16x128_f8f6f4
// takes two consecutive 16 x 64 fragments of A and of B (the same lane-to-K
// assignment on both sides, so the pair covers 128 K values) into fp32 sums;
// scales as on the int8 path.
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
#include "rowquant.h"

namespace w8a8 {

// ------------------------------------------------------------------ helpers

// bf16 A operand read straight from a row-major matrix: lane l takes row
// (l % 16) of the fragment and the 8 columns (l / 16) * 8 .. +7 of its 32.
__device__ __forceinline__ v4i load_frag_rowmajor_bf16(const void* base, int64_t row,
                                                       int64_t kb, int64_t lda, int lane) {
  const uint16_t* p = reinterpret_cast<const uint16_t*>(base) + row * lda + kb * kFragK16 +
                      (lane >> 4) * 8;
  return *reinterpret_cast<const v4i*>(p);
}

template <int DT>
struct Acc;
template <>
struct Acc<DT_I8> {
  typedef v4i T;
  static __device__ __forceinline__ T zero() { return v4i{0, 0, 0, 0}; }
  static __device__ __forceinline__ T mma(v4i a, v4i b, T c) { return mma_i8(a, b, c); }
};
template <>
struct Acc<DT_BF16> {
  typedef v4f T;
  static __device__ __forceinline__ T zero() { return v4f{0.f, 0.f, 0.f, 0.f}; }
  static __device__ __forceinline__ T mma(v4i a, v4i b, T c) { return mma_bf16(a, b, c); }
};
template <>
struct Acc<DT_F8> {
  typedef v4f T;
  static __device__ __forceinline__ T zero() { return v4f{0.f, 0.f, 0.f, 0.f}; }
  // two consecutive 16 x 64 fragments of A and B: K = 128
  static __device__ __forceinline__ T mma2(v4i a0, v4i a1, v4i b0, v4i b1, T c) {
    return mma_f8(a0, a1, b0, b1, c);
  }
};

// fragments consumed by one MFMA of a type
template <int DT>
constexpr int frags_per_mma() { return DT == DT_F8 ? 2 : 1; }

// Dequantised / converted value of one accumulator element.
template <int DT>
__device__ __forceinline__ float acc_value(float a_or_i, const GemmParams& p, int row, int col,
                                           const float* s_b) {
  if constexpr (DT == DT_BF16) {
    return a_or_i;
  } else {
    float t = a_or_i * p.s_a[row];
    return t * s_b[col];
  }
}

// Store one output element for the non-gated epilogues.
template <int DT, int EPI>
__device__ __forceinline__ void store_elem(const GemmParams& p, int row, int col, int32_t iacc,
                                           float facc) {
  if constexpr (EPI == EPI_I32) {  // raw sums: int32, or fp32 for float types
    if constexpr (DT != DT_I8)
      reinterpret_cast<float*>(p.out)[(int64_t)row * p.ldo + col] = facc;
    else
      reinterpret_cast<int32_t*>(p.out)[(int64_t)row * p.ldo + col] = iacc;
  } else {
    float raw = DT != DT_I8 ? facc : (float)iacc;
    float y = acc_value<DT>(raw, p, row, col, p.s_b);
    if constexpr (EPI == EPI_F32)
      reinterpret_cast<float*>(p.out)[(int64_t)row * p.ldo + col] = y;
    else
      reinterpret_cast<uint16_t*>(p.out)[(int64_t)row * p.ldo + col] = float_to_bf16_bits(y);
  }
}

template <int DT>
__device__ __forceinline__ void store_glu(const GemmParams& p, int row, int col, float g_raw,
                                          float u_raw) {
  float g = acc_value<DT>(g_raw, p, row, col, p.s_b);
  float u = acc_value<DT>(u_raw, p, row, col, p.s_b2);
  float h = gelu_tanh(g) * u;
  reinterpret_cast<uint16_t*>(p.out)[(int64_t)row * p.ldo + col] = float_to_bf16_bits(h);
}

template <int DT>
__device__ __forceinline__ void write_partial(const GemmParams& p, int z, int row, int col,
                                              int32_t iacc, float facc) {
  const int64_t idx = (int64_t)z * p.M * p.N + (int64_t)row * p.N + col;
  if constexpr (DT != DT_I8)
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

// Wait until at most PF * min(n, N) of this wave's loads are outstanding.
template <int PF, int N>
__device__ __forceinline__ void wait_outstanding(int n) {
  if constexpr (N <= 0) {
    wait_vmcnt<0>();
  } else {
    if (n >= N)
      wait_vmcnt<PF * N>();
    else
      wait_outstanding<PF, N - 1>(n);
  }
}

// ------------------------------------------------------------------ tiled kernel

// BM x BN output tile per workgroup of NW waves arranged WAVES_M x (NW / WAVES_M).
// The K loop runs over an S-stage LDS ring: each stage holds BM/16 A and
// BN/16 (x2 gated) B fragments, filled by LDS-DMA loads issued S-1 steps ahead,
// so S-2 stages of HBM/L2 traffic stay in flight while the MFMAs of the
// current stage run.  One barrier per K step.
//
// Workgroups are dealt to the 8 XCDs round-robin by ID; the tile order gives
// every XCD a contiguous range of tiles (M tile fastest), so the A and B
// panels a range touches stay in that XCD's L2.
// MINB: workgroups per CU the register budget is sized for (2: two co-resident
// workgroups; 1: one, with twice the registers per wave)
template <int DT, int BM, int BN, int WAVES_M, int NW, int EPI, int S, int KS, int MINB = 2>
__global__ __launch_bounds__(64 * NW, MINB) void gemm_tile_kernel(GemmParams p) {
  constexpr bool GLU = (EPI == EPI_GLU);
  constexpr bool BF16 = (DT == DT_BF16);  // row-major bf16 A, unscaled fp32 sums
  constexpr bool FACC = (DT != DT_I8);    // fp32 accumulators and partial sums
  constexpr int KP = frags_per_mma<DT>();
  static_assert(KS % KP == 0, "a stage must hold whole MFMA K steps");
  constexpr int WAVES_N = NW / WAVES_M;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int NA = BM / 16;
  constexpr int NB = (BN / 16) * (GLU ? 2 : 1);
  constexpr int NF = NA + NB;
  static_assert(NF % NW == 0, "fragments per stage must split over the waves");
  constexpr int PF = NF / NW;  // fragment rows each wave fetches per stage (KS fragments each)
  typedef typename Acc<DT>::T AccT;

  __shared__ v4i lds[S][NF * KS * 64];

  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;

  const int m_tiles = (p.M + BM - 1) / BM;
  const int n_tiles = (p.N + BN - 1) / BN;
  const int n_total = m_tiles * n_tiles;
  const int per_xcd = (n_total + 7) / 8;
  int mt, nt, z;
  if (p.xcd_m) {
    // workgroup ids are dealt to the XCDs round-robin: XCD x = id % 8 takes
    // the M tiles x, x + 8, ... with every N tile and K split of each, so an
    // XCD's L2 holds its own rows of A once
    const int x = (int)(blockIdx.x % 8), j = (int)(blockIdx.x / 8);
    const int per = n_tiles * p.splits;
    mt = x + 8 * (j / per);
    nt = (j % per) % n_tiles;
    z = (j % per) / n_tiles;
    if (mt >= m_tiles) return;  // whole workgroup, before any barrier
  } else {
    const int t = (int)(blockIdx.x % 8) * per_xcd + (int)(blockIdx.x / 8);
    if (t >= n_total) return;  // whole workgroup, before any barrier
    if (p.group_m > 0 && p.group_m < m_tiles) {  // bands of group_m M tiles, N within a band
      const int band_tiles = p.group_m * n_tiles;
      const int band = t / band_tiles, in_band = t % band_tiles;
      const int gm = min(p.group_m, m_tiles - band * p.group_m);
      mt = band * p.group_m + in_band % gm;
      nt = in_band / gm;
    } else {
      mt = t % m_tiles;
      nt = t / m_tiles;
    }
    z = blockIdx.y;
  }
  const int kb0 = z * p.kchunk;
  const int kb1 = min(p.kb_count, kb0 + p.kchunk);
  const int nk = kb1 - kb0;

  // per-wave source pointers of its PF fragments at kb = 0
  const int8_t* src[PF];
  int64_t src_step[PF];
#pragma unroll
  for (int i = 0; i < PF; ++i) {
    const int f = wave + NW * i;
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
  // Each workgroup walks its K range from a different starting point, so the
  // operand panels shared by many workgroups (A by every N tile, B by every
  // M tile) are not all requested from the same L2 lines at the same time.
  // A stage holds KS consecutive fragment columns; a ragged last stage loads
  // its last valid column again (uniform load counts) and skips its products.
  const int nsteps = (nk + KS - 1) / KS;
  const int rot = (nsteps > 0 && p.rotate) ? (int)((blockIdx.x * 5u) % (unsigned)nsteps) : 0;
  auto stage_of = [&](int j) {
    int jj = j + rot;
    if (jj >= nsteps) jj -= nsteps;
    return jj;
  };
  auto issue = [&](int j) {  // stage j (relative to kb0) into slot j % S
    const int kb = kb0 + stage_of(j) * KS;
#pragma unroll
    for (int i = 0; i < PF; ++i)
#pragma unroll
      for (int k = 0; k < KS; ++k)
        to_lds_async(src[i] + (int64_t)min(kb + k, kb1 - 1) * src_step[i],
                     &lds[j % S][((wave + NW * i) * KS + k) * 64]);
  };

  AccT acc[TM][TN];
  AccT accu[GLU ? TM : 1][GLU ? TN : 1];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      acc[i][j] = Acc<DT>::zero();
      if constexpr (GLU) accu[i][j] = Acc<DT>::zero();
    }

  // Fragments of one stage held in registers: the LDS reads of stage j+1 are
  // issued right after the barrier and complete while the MFMAs of stage j
  // (already in registers) run.
  struct Frags {
    v4i a[KS][TM];
    v4i b[KS][TN];
    v4i bu[KS][GLU ? TN : 1];
  };
  auto read_frags = [&](int j, Frags& F) {
    const v4i* St = lds[j % S];
#pragma unroll
    for (int k = 0; k < KS; ++k) {
#pragma unroll
      for (int i = 0; i < TM; ++i) F.a[k][i] = St[((wm * TM + i) * KS + k) * 64 + lane];
#pragma unroll
      for (int t = 0; t < TN; ++t) F.b[k][t] = St[((NA + wn * TN + t) * KS + k) * 64 + lane];
      if constexpr (GLU) {
#pragma unroll
        for (int t = 0; t < TN; ++t)
          F.bu[k][t] = St[((NA + BN / 16 + wn * TN + t) * KS + k) * 64 + lane];
      }
    }
  };
  auto mma_frags = [&](const Frags& F, int j) {
    const int nv = min(KS, nk - stage_of(j) * KS);  // valid fragment columns of stage j
#pragma unroll
    for (int k = 0; k < KS; k += KP) {
      if (k > 0 && k >= nv) break;
      if constexpr (DT == DT_F8) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int t = 0; t < TN; ++t)
            acc[i][t] = Acc<DT>::mma2(F.a[k][i], F.a[k + 1][i], F.b[k][t], F.b[k + 1][t], acc[i][t]);
        if constexpr (GLU) {
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int t = 0; t < TN; ++t)
              accu[i][t] = Acc<DT>::mma2(F.a[k][i], F.a[k + 1][i], F.bu[k][t], F.bu[k + 1][t],
                                         accu[i][t]);
        }
      } else {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int t = 0; t < TN; ++t) acc[i][t] = Acc<DT>::mma(F.a[k][i], F.b[k][t], acc[i][t]);
        if constexpr (GLU) {
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int t = 0; t < TN; ++t)
              accu[i][t] = Acc<DT>::mma(F.a[k][i], F.bu[k][t], accu[i][t]);
        }
      }
    }
  };

  int issued = -1;  // last stage handed to the LDS-DMA
#pragma unroll
  for (int j = 0; j < S - 1; ++j)
    if (j < nsteps) {
      issue(j);
      issued = j;
    }
  Frags F0, F1;
  if (nsteps > 0) {
    wait_outstanding<PF * KS, S - 2>(issued);
    lds_barrier();
    read_frags(0, F0);
  }
  // One step: stage j+1 must have landed (own loads, then the barrier for the
  // other waves'); the slot of stage j-1 is free (its fragments were read one
  // step earlier), so stage j+S-1 goes into it.
  auto step = [&](int j, Frags& Fc, Frags& Fn) {
    if (j + 1 < nsteps) wait_outstanding<PF * KS, S - 2>(issued - (j + 1));
    lds_barrier();
    if (j + S - 1 < nsteps) {
      issue(j + S - 1);
      issued = j + S - 1;
    }
    if (j + 1 < nsteps) read_frags(j + 1, Fn);
    mma_frags(Fc, j);
  };
  for (int j = 0; j < nsteps; j += 2) {
    step(j, F0, F1);
    if (j + 1 < nsteps) step(j + 1, F1, F0);
  }

  // ---------------- epilogue
  // Scales are read once into registers; each wave then stages one 16-row
  // block of its output at a time in a private LDS area (the K-loop ring is
  // free by now) and writes it back as 16-byte row segments.
  lds_barrier();
  const int row_w = mt * BM + wm * WM;  // first row of this wave
  const int col_w = nt * BN + wn * WN;  // first column of this wave
  const int row0 = row_w + (lane >> 4) * 4;
  const int col0 = col_w + (lane & 15);
  float sa[TM][4], sb[TN], sb2[GLU ? TN : 1];
  if constexpr (!BF16) {
    if (EPI != EPI_I32 && !(EPI != EPI_GLU && p.splits > 1)) {
      // indexes clamped into range: rows and columns past the edge are
      // computed but never stored
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) sa[i][r] = p.s_a[min(row0 + i * 16 + r, p.M - 1)];
#pragma unroll
      for (int t = 0; t < TN; ++t) {
        const int col = min(col0 + t * 16, p.N - 1);
        sb[t] = p.s_b[col];
        if constexpr (GLU) sb2[t] = p.s_b2[col];
      }
    }
  }
  // output element type and destination of this launch
  const bool partial = (EPI != EPI_GLU) && p.splits > 1;
  constexpr int OB = (EPI == EPI_GLU || EPI == EPI_BF16) ? 2 : 4;  // bytes per element
  const int esz = partial ? 4 : OB;
  char* dst = partial ? reinterpret_cast<char*>(p.part) + (int64_t)z * p.M * p.N * 4
                      : reinterpret_cast<char*>(p.out);
  const int64_t ld = partial ? p.N : p.ldo;
  static_assert(NW * 16 * WN * 4 <= S * NF * KS * 64 * 16, "epilogue staging must fit in the ring");
  char* stage = reinterpret_cast<char*>(&lds[0][0]) + wave * (16 * WN * 4);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int t = 0; t < TN; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int rr = (lane >> 4) * 4 + r;           // row within the 16-row block
        const int cc = t * 16 + (lane & 15);          // column within the wave's WN
        char* slot = stage + (rr * WN + cc) * esz;
        if constexpr (GLU) {
          float g, u;
          if constexpr (BF16) {
            g = (float)acc[i][t][r];
            u = (float)accu[i][t][r];
          } else {
            g = ((float)acc[i][t][r] * sa[i][r]) * sb[t];
            u = ((float)accu[i][t][r] * sa[i][r]) * sb2[t];
          }
          *reinterpret_cast<uint16_t*>(slot) = float_to_bf16_bits(gelu_tanh(g) * u);
        } else if (partial || EPI == EPI_I32) {  // raw sums: int32, or fp32 for float types
          if constexpr (FACC)
            *reinterpret_cast<float*>(slot) = (float)acc[i][t][r];
          else
            *reinterpret_cast<int32_t*>(slot) = (int32_t)acc[i][t][r];
        } else {
          float y;
          if constexpr (BF16)
            y = (float)acc[i][t][r];
          else
            y = ((float)acc[i][t][r] * sa[i][r]) * sb[t];
          if constexpr (EPI == EPI_F32)
            *reinterpret_cast<float*>(slot) = y;
          else
            *reinterpret_cast<uint16_t*>(slot) = float_to_bf16_bits(y);
        }
      }
    // this wave's own LDS writes are complete before its reads (in-order LDS)
    const int row_bytes = WN * esz;
    const int chunks = 16 * row_bytes / 16;
    for (int c = lane; c < chunks; c += 64) {
      const int rr = c / (row_bytes / 16);
      const int cb = (c % (row_bytes / 16)) * 16;     // byte offset within the row
      const int row = row_w + i * 16 + rr;
      const int col = col_w + cb / esz;
      if (row >= p.M) continue;
      const char* srcp = stage + rr * row_bytes + cb;
      char* gp = dst + ((int64_t)row * ld + col) * esz;
      const int n_in = min(16 / esz, p.N - col);
      if (n_in == 16 / esz && ((reinterpret_cast<uintptr_t>(gp) & 15) == 0)) {
        if (p.nt_out)  // output far larger than the caches: stream it past them
          __builtin_nontemporal_store(*reinterpret_cast<const v4i*>(srcp), reinterpret_cast<v4i*>(gp));
        else
          *reinterpret_cast<uint4*>(gp) = *reinterpret_cast<const uint4*>(srcp);
      } else {
        for (int e = 0; e < n_in; ++e)
          for (int bb = 0; bb < esz; ++bb) gp[e * esz + bb] = srcp[e * esz + bb];
      }
    }
  }
}

// ------------------------------------------------------------------ streaming kernel

// Skinny GEMM, M <= 16 * MB rows (MB <= 8), for decode and small prefill
// batches where the weights dominate the traffic.  The workgroup has NW waves.
// With WK == 1 every wave walks its own output column blocks of 16 (the wide
// lm_head); with WK == NW all waves share one column block and split its K
// range, reducing through LDS (long-K, narrow-N projections such as the FFN
// down projection, or the gated gate/up pair).  A wave stages the A fragments
// of its own K slice in LDS once (LDS-DMA), then streams the weight fragments
// of a column block -- one contiguous run -- from HBM in batches of KU,
// double buffered in registers, so the loads of batch i+1 are in flight while
// the MFMAs (MB per fragment) and the epilogue of batch i run.  Cross-workgroup
// K splits (a grid dimension) write partial sums for the reduction kernel.
template <int DT, int MB, int EPI, int NW, int WK, int QL>
__global__ __launch_bounds__(64 * NW) void gemm_stream_kernel(GemmParams p, int nb_per_block) {
  static_assert(WK == 1 || WK == NW, "either every wave owns its column blocks or all share one");
  static_assert(!QL || ((DT == DT_I8 || DT == DT_F8) && MB == 1),
                "quantise-on-load: int8 or E4M3 codes, one row block");
  static_assert(QL != 2 || DT == DT_I8, "fused layer glue: int8 codes");
  constexpr bool GLU = (EPI == EPI_GLU);
  constexpr bool BF16 = (DT == DT_BF16);
  constexpr bool FACC = (DT != DT_I8);
  constexpr int KP = frags_per_mma<DT>();
  constexpr int KU = KP == 2 ? 8 : 9;  // weight fragments per batch and operand (whole MFMA steps)
  constexpr int KG = GLU ? KU : 1;
  constexpr int NC = GLU ? 2 : 1;
  constexpr int GROUPS = NW / WK;
  typedef typename Acc<DT>::T AccT;
  extern __shared__ v4i lds_dyn[];

  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int grp = wave / WK, wk = wave % WK;
  const int z = blockIdx.y;
  const int kb0 = z * p.kchunk;
  const int kc = min(p.kb_count, kb0 + p.kchunk) - kb0;
  v4i* lds_a = lds_dyn;                                       // MB x kchunk fragments
  AccT* red = reinterpret_cast<AccT*>(lds_dyn + (int64_t)MB * p.kchunk * 64);  // (WK-1) x NC x MB

  // this wave's K slice [ks0, ks1) of the workgroup's range
  const int kpw = ((kc + WK - 1) / WK + KP - 1) / KP * KP;  // whole MFMA K steps per wave
  const int ks0 = min(kc, wk * kpw), ks1 = min(kc, ks0 + kpw);
  const int my_k = ks1 - ks0;
  const int bpn = (kpw + KU - 1) / KU;  // batches per column block (uniform over the waves)

  const int nb_begin = blockIdx.x * nb_per_block;
  const int nb_end = min(p.rb_b, nb_begin + nb_per_block);
  const int my_first = nb_begin + grp;
  const int my_count = my_first < nb_end ? (nb_end - my_first + GROUPS - 1) / GROUPS : 0;
  const int total = my_count * bpn;

  // stage the A fragments: with WK > 1 each wave its own K slice (read only
  // by itself); with WK == 1 the waves share the whole panel
  auto a_src = [&](int mb, int kk) -> const int8_t* {
    if constexpr (BF16) {
      int64_t row = min((int64_t)mb * 16 + (lane & 15), (int64_t)p.M - 1);
      return reinterpret_cast<const int8_t*>(reinterpret_cast<const uint16_t*>(p.A) + row * p.lda +
                                             (int64_t)(kb0 + kk) * kFragK16 + (lane >> 4) * 8);
    } else {
      return reinterpret_cast<const int8_t*>(p.A) +
             frag_offset(min(mb, p.rb_a - 1), kb0 + kk, p.kb_count) + lane * 16;
    }
  };
  // QL 1: the workgroup quantises its bf16 rows itself (p.a_x); QL 2: it runs
  // the layer glue for its one token row first (p.g_*).  Separate
  // instantiations, so that a quantising kernel has no staging loop whose
  // outstanding loads the compiler would have to wait for before quantising.
  constexpr bool QLOAD_OK = QL != 0;
  constexpr bool qload = QL != 0;
  if constexpr (!QL) {
    if constexpr (WK > 1) {
      for (int f = 0; f < MB * my_k; ++f) {
        const int mb = f / my_k, kk = ks0 + f % my_k;
        to_lds_async(a_src(mb, kk), &lds_a[(mb * p.kchunk + kk) * 64]);
      }
    } else {
      for (int f = wave; f < MB * kc; f += NW) {
        const int mb = f / kc, kk = f % kc;
        to_lds_async(a_src(mb, kk), &lds_a[(mb * p.kchunk + kk) * 64]);
      }
    }
  }

  // Scales live in registers: the token scales of this lane's rows loaded
  // before the weights, the channel scales of a column block together with
  // its first weight batch, so neither adds a memory round trip after the
  // weights have arrived.
  const bool scaled = !BF16 && (GLU || ((EPI == EPI_F32 || EPI == EPI_BF16) && p.splits == 1));
  float sa_r[MB][4];
  float sb_c = 0.0f, sb2_c = 0.0f;
  float sbn[2] = {0.0f, 0.0f}, sbn2[2] = {0.0f, 0.0f};  // per weight buffer
  if constexpr (!QL) {  // branch-free (reads B's first bytes where the values are unused)
    const bool from_sa = scaled;
    const float* sa_src = from_sa ? p.s_a : reinterpret_cast<const float*>(p.B);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        sa_r[mb][r] = sa_src[from_sa ? min(mb * 16 + (lane >> 4) * 4 + r, p.M - 1) : 0];
  }
  auto load_scales = [&](int nb, float& sbx, float& sbx2) {
    const int col = min(nb * 16 + (lane & 15), p.N - 1);
    sbx = p.s_b[col];
    if constexpr (GLU) sbx2 = p.s_b2[col];
  };

  v4i b0[KU], b1[KU], u0[KG], u1[KG];
  auto load_batch = [&](int idx, v4i (&b)[KU], v4i (&bu)[KG], float& sbx, float& sbx2) {
    const int nb = my_first + GROUPS * (idx / bpn);
    const int k0 = (idx % bpn) * KU;
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      if (k0 + u < my_k) {
        b[u] = load_frag_packed(p.B, nb, kb0 + ks0 + k0 + u, p.kb_count, lane);
        if constexpr (GLU) bu[u] = load_frag_packed(p.B2, nb, kb0 + ks0 + k0 + u, p.kb_count, lane);
      }
    }
    if (scaled && k0 == 0) load_scales(nb, sbx, sbx2);
  };
  // The first batch issues all KU loads per operand, indexes clamped into
  // this wave's slice (or, for a wave without work, into the workgroup's
  // range): a fixed number of loads follows the activation loads of
  // quantise-on-load, so the wait before quantising covers those alone.
  auto load_first = [&](v4i (&b)[KU], v4i (&bu)[KG], float& sbx, float& sbx2) {
    const int nb = min(my_first, p.rb_b - 1);
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      const int kf = kb0 + min(ks0 + min(u, max(my_k - 1, 0)), kc - 1);
      b[u] = load_frag_packed(p.B, nb, kf, p.kb_count, lane);
      if constexpr (GLU) bu[u] = load_frag_packed(p.B2, nb, kf, p.kb_count, lane);
    }
    if (scaled) load_scales(nb, sbx, sbx2);
  };
  QloadRegs<NW> qr;
  GlueRegs gr;
  if constexpr (QL == 1) quantize_fetch<NW>(p, true, qr);  // ahead of the weights
  if constexpr (QL == 2) glue_fetch(p, gr);

  __builtin_amdgcn_sched_barrier(0);
  load_first(b0, u0, sbn[0], sbn2[0]);  // first weights go out with the A fragments
  __shared__ float s_row[16];           // quantise-on-load: per-row scales
  if constexpr (QL == 1) quantize_panel<NW, DT == DT_F8>(p, kb0, kc, lds_a, s_row, qr);
  if constexpr (QL == 2) glue_panel<NW>(p, kb0, kc, lds_a, s_row, gr);  // both overlap the weights
  wait_vmcnt<0>();
  if ((WK == 1 && NW > 1) || qload) lds_barrier();  // the shared panel is read by every wave
  if (scaled && qload) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) sa_r[mb][r] = s_row[min(mb * 16 + (lane >> 4) * 4 + r, p.M - 1)];
  }

  AccT acc[MB], accu[GLU ? MB : 1];
  auto epilogue = [&](int nb) {
    const int col = nb * 16 + (lane & 15);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = mb * 16 + (lane >> 4) * 4 + r;
        if (row >= p.M || col >= p.N) continue;
        const int64_t o = (int64_t)row * p.ldo + col;
        if constexpr (GLU) {
          float gv, uv;
          if constexpr (BF16) {
            gv = (float)acc[mb][r];
            uv = (float)accu[mb][r];
          } else {
            gv = ((float)acc[mb][r] * sa_r[mb][r]) * sb_c;
            uv = ((float)accu[mb][r] * sa_r[mb][r]) * sb2_c;
          }
          reinterpret_cast<uint16_t*>(p.out)[o] = float_to_bf16_bits(gelu_tanh(gv) * uv);
        } else if (p.splits > 1) {
          write_partial<DT>(p, z, row, col, FACC ? 0 : (int32_t)acc[mb][r], (float)acc[mb][r]);
        } else if constexpr (EPI == EPI_I32) {  // raw sums: int32, or fp32 for float types
          if constexpr (FACC)
            reinterpret_cast<float*>(p.out)[o] = (float)acc[mb][r];
          else
            reinterpret_cast<int32_t*>(p.out)[o] = (int32_t)acc[mb][r];
        } else {
          float y;
          if constexpr (BF16)
            y = (float)acc[mb][r];
          else
            y = ((float)acc[mb][r] * sa_r[mb][r]) * sb_c;
          if constexpr (EPI == EPI_F32)
            reinterpret_cast<float*>(p.out)[o] = y;
          else
            reinterpret_cast<uint16_t*>(p.out)[o] = float_to_bf16_bits(y);
        }
      }
  };
  auto compute = [&](int idx, const v4i (&b)[KU], const v4i (&bu)[KG], float sbx, float sbx2) {
    const int nb = my_first + GROUPS * (idx / bpn);
    const int bi = idx % bpn;
    const int k0 = bi * KU;
    if (bi == 0) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        acc[mb] = Acc<DT>::zero();
        if constexpr (GLU) accu[mb] = Acc<DT>::zero();
      }
      sb_c = sbx;
      sb2_c = sbx2;
    }
#pragma unroll
    for (int u = 0; u < KU; u += KP) {
      if (k0 + u < my_k) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const v4i a = lds_a[(mb * p.kchunk + ks0 + k0 + u) * 64 + lane];
          if constexpr (DT == DT_F8) {
            const v4i a1 = lds_a[(mb * p.kchunk + ks0 + k0 + u + 1) * 64 + lane];
            acc[mb] = Acc<DT>::mma2(a, a1, b[u], b[u + 1], acc[mb]);
            if constexpr (GLU) accu[mb] = Acc<DT>::mma2(a, a1, bu[u], bu[u + 1], accu[mb]);
          } else {
            acc[mb] = Acc<DT>::mma(a, b[u], acc[mb]);
            if constexpr (GLU) accu[mb] = Acc<DT>::mma(a, bu[u], accu[mb]);
          }
        }
      }
    }
    if (bi != bpn - 1) return;
    if constexpr (WK == 1) {
      epilogue(nb);
    } else {
      // in-workgroup K reduction: waves 1..WK-1 hand their sums to wave 0,
      // which adds them in wave order and runs the epilogue
      if (wk > 0) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          red[(((wk - 1) * NC + 0) * MB + mb) * 64 + lane] = acc[mb];
          if constexpr (GLU) red[(((wk - 1) * NC + 1) * MB + mb) * 64 + lane] = accu[mb];
        }
      }
      lds_barrier();
      if (wk == 0) {
        for (int w = 1; w < WK; ++w) {
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) {
            acc[mb] += red[(((w - 1) * NC + 0) * MB + mb) * 64 + lane];
            if constexpr (GLU) accu[mb] += red[(((w - 1) * NC + 1) * MB + mb) * 64 + lane];
          }
        }
        epilogue(nb);
      }
      lds_barrier();
    }
  };

  for (int idx = 0; idx < total; idx += 2) {
    if (idx + 1 < total) load_batch(idx + 1, b1, u1, sbn[1], sbn2[1]);
    compute(idx, b0, u0, sbn[0], sbn2[0]);
    if (idx + 1 < total) {
      if (idx + 2 < total) load_batch(idx + 2, b0, u0, sbn[0], sbn2[0]);
      compute(idx + 1, b1, u1, sbn[1], sbn2[1]);
    }
  }
}

// ------------------------------------------------------------------ K-split reduction

// out = epilogue(sum over z of part[z]) for 4 consecutive columns per thread,
// the splits added in order (int32 exactly; fp32 in a fixed order).
template <int DT, int EPI>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmParams p) {
  constexpr bool FACC = (DT != DT_I8);
  const int64_t n4 = (p.N + 3) / 4;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)p.M * n4) return;
  const int row = (int)(idx / n4);
  const int col0 = (int)(idx % n4) * 4;
  const int64_t plane = (int64_t)p.M * p.N;
  const int ncol = min(4, p.N - col0);
  int32_t isum[4] = {0, 0, 0, 0};
  float fsum[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
  for (int zz = 0; zz < p.splits; ++zz) {
    const int64_t base = zz * plane + (int64_t)row * p.N + col0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if (c < ncol) {
        if constexpr (FACC)
          fsum[c] += reinterpret_cast<const float*>(p.part)[base + c];
        else
          isum[c] += reinterpret_cast<const int32_t*>(p.part)[base + c];
      }
    }
  }
#pragma unroll
  for (int c = 0; c < 4; ++c)
    if (c < ncol) store_elem<DT, EPI>(p, row, col0 + c, isum[c], fsum[c]);
}

// ------------------------------------------------------------------ dispatch

// Launch of one tile configuration: one workgroup per tile, 8 x ceil(tiles /
// 8) dealt to the XCDs round-robin with a y dimension of K splits, or the
// one-dimensional XCD-by-M grid (8 x ceil(M tiles / 8) x N tiles x splits).
template <int DT, int BM, int BN, int WAVES_M, int NW, int EPI, int S, int KS, int MINB = 2>
static hipError_t launch_tile(const GemmParams& p, hipStream_t st) {
  const int mt = (p.M + BM - 1) / BM;
  const int nt = (p.N + BN - 1) / BN;
  const int per_xcd = (mt * nt + 7) / 8;
  dim3 grid((unsigned)(8 * per_xcd), (unsigned)p.splits);
  if (p.xcd_m) {
    grid = dim3((unsigned)((mt + 7) / 8 * 8 * nt * p.splits), 1u);
  }
  gemm_tile_kernel<DT, BM, BN, WAVES_M, NW, EPI, S, KS, MINB><<<grid, 64 * NW, 0, st>>>(p);
  return hipGetLastError();
}

// Tile shapes per type: FP8 needs stages of whole 128-deep MFMA steps, so only
// the shapes with two fragment columns per stage exist for it.
template <int DT, int EPI>
static hipError_t tile_dispatch(int tile, const GemmParams& p, hipStream_t st) {
  constexpr bool K1 = DT != DT_F8;  // single-fragment stages available
  if constexpr (EPI == EPI_GLU) {
    switch (tile) {
      case TILE_GLU_128x32_K2:
        return launch_tile<DT, 128, 32, 4, 4, EPI, 6, 2>(p, st);
      case TILE_GLU_64x64_K2:
        return launch_tile<DT, 64, 64, 2, 4, EPI, 3, 2>(p, st);
      case TILE_GLU_256x64_K2_W8:  // 144 KiB of LDS: one workgroup per CU
        return launch_tile<DT, 256, 64, 4, 8, EPI, 3, 2, 1>(p, st);
      default:
        break;
    }
    if constexpr (K1) {
      switch (tile) {
        case TILE_GLU_128x32:
          return launch_tile<DT, 128, 32, 4, 4, EPI, 12, 1>(p, st);
        case TILE_GLU_64x64:
          return launch_tile<DT, 64, 64, 2, 4, EPI, 6, 1>(p, st);
        case TILE_GLU_128x64:
          return launch_tile<DT, 128, 64, 2, 4, EPI, 5, 1>(p, st);
        case TILE_GLU_256x128:
          return launch_tile<DT, 256, 128, 2, 8, EPI, 5, 1>(p, st);
        case TILE_GLU_256x64:
          return launch_tile<DT, 256, 64, 2, 4, EPI, 3, 1>(p, st);
        case TILE_GLU_128x32_K3:  // 144 KiB of LDS: one workgroup per CU
          return launch_tile<DT, 128, 32, 4, 4, EPI, 4, 3, 1>(p, st);
        default:
          break;
      }
    }
  } else {
    switch (tile) {
      case TILE_64x64_K2:
        return launch_tile<DT, 64, 64, 2, 4, EPI, 3, 2>(p, st);
      case TILE_128x128_K2:
        return launch_tile<DT, 128, 128, 2, 4, EPI, 3, 2>(p, st);
      default:
        break;
    }
    if constexpr (K1) {
      switch (tile) {
        case TILE_128x128:
          return launch_tile<DT, 128, 128, 2, 4, EPI, 5, 1>(p, st);
        case TILE_128x64:
          return launch_tile<DT, 128, 64, 2, 4, EPI, 6, 1>(p, st);
        case TILE_64x64:
          return launch_tile<DT, 64, 64, 2, 4, EPI, 6, 1>(p, st);
        case TILE_256x128:
          return launch_tile<DT, 256, 128, 2, 8, EPI, 5, 1>(p, st);
        case TILE_256x256:
          return launch_tile<DT, 256, 256, 2, 8, EPI, 5, 1>(p, st);
        case TILE_64x64_K3:  // 96 KiB of LDS: one workgroup per CU
          return launch_tile<DT, 64, 64, 2, 8, EPI, 4, 3, 1>(p, st);
        case TILE_256x128_W4:  // 72 KiB of LDS: two workgroups per CU
          return launch_tile<DT, 256, 128, 2, 4, EPI, 3, 1>(p, st);
        default:
          break;
      }
    }
  }
  return hipErrorInvalidValue;
}

template <int DT>
static hipError_t tile_epi(int epi, int tile, const GemmParams& p, hipStream_t st) {
  switch (epi) {
    case EPI_I32: return tile_dispatch<DT, EPI_I32>(tile, p, st);
    case EPI_F32: return tile_dispatch<DT, EPI_F32>(tile, p, st);
    case EPI_BF16: return tile_dispatch<DT, EPI_BF16>(tile, p, st);
    case EPI_GLU: return tile_dispatch<DT, EPI_GLU>(tile, p, st);
    default: return hipErrorInvalidValue;
  }
}

// Host-side check, before any launch, that every buffer the kernel will read
// or write is present and that the K split is consistent: a missing scale or
// partial-sum buffer becomes an error return instead of a device access.
//   kind 0: tiled kernel, 1: streaming kernel with nw waves, 2: split-K reduction
static bool gemm_params_ok(int dt, int epi, const GemmParams& p, int kind, int nw = 1) {
  const bool glu = epi == EPI_GLU;
  if (p.M < 1 || p.N < 1 || p.kb_count < 1 || p.kchunk < 1 || p.splits < 1) return false;
  if ((int64_t)p.kchunk * (p.splits - 1) >= p.kb_count) return false;  // no empty split
  if ((int64_t)p.kchunk * p.splits < p.kb_count) return false;         // K fully covered
  if (glu && p.splits != 1) return false;  // the gated epilogue needs whole sums
  const bool glue = kind == 1 && dt == DT_I8 && p.g_x_in != nullptr;
  const bool qload = (kind == 1 && (dt == DT_I8 || dt == DT_F8) && p.a_x != nullptr) || glue;
  if ((kind != 1 || dt != DT_I8) && p.g_x_in) return false;  // fused glue: int8 streaming only
  if (kind == 0 && p.a_x) return false;  // the tiled kernel reads codes only
  if (glue) {
    if (p.a_x || p.M != 1 || p.a_k < 8 || p.a_k % 8 || p.a_k / 8 > 64 * nw) return false;
    if (p.g_part && (p.g_splits < 1 || p.g_splits > kGlueMaxSplits)) return false;
    if (p.g_part && !p.g_part_f32 && (!p.g_st || !p.g_si)) return false;
  }
  if (qload && (p.M > 16 || p.a_k < 16 || (int64_t)p.M * (p.a_k / 16) > (int64_t)64 * nw))
    return false;
  if (kind == 2) {
    if (!p.part || !p.out) return false;
  } else {
    if (!p.B || (glu && !p.B2) || (!p.A && !qload)) return false;
    if (p.splits > 1 ? !p.part : !p.out) return false;
  }
  // dequantising epilogues (int8 / E4M3 operands) read both scale vectors
  const bool dequant = dt != DT_BF16 && epi != EPI_I32 && (kind == 2 || p.splits == 1);
  if (dequant) {
    if (!p.s_b || (glu && !p.s_b2)) return false;
    if (!p.s_a && !qload) return false;  // quantise-on-load keeps its scales in LDS
  }
  return true;
}

hipError_t launch_gemm_tile(int dt, int epi, int tile, const GemmParams& p, hipStream_t st) {
  if (!gemm_params_ok(dt, epi, p, 0)) return hipErrorInvalidValue;
  switch (dt) {
    case DT_I8: return tile_epi<DT_I8>(epi, tile, p, st);
    case DT_BF16: return tile_epi<DT_BF16>(epi, tile, p, st);
    case DT_F8: return tile_epi<DT_F8>(epi, tile, p, st);
    default: return hipErrorInvalidValue;
  }
}

// dynamic LDS of a streaming launch: A panel + reduction scratch
static size_t stream_lds_bytes(int mb, int kchunk, int wk, bool glu) {
  return (size_t)mb * kchunk * kFragBytes + (size_t)(wk - 1) * (glu ? 2 : 1) * mb * kFragBytes;
}

template <int DT, int MB, int EPI, int NW, int WK, int QL>
static hipError_t stream_launch_ql(const GemmParams& p, int nbpb, hipStream_t st) {
  auto kern = gemm_stream_kernel<DT, MB, EPI, NW, WK, QL>;
  static size_t static_lds = 0;  // benign race: every caller computes the same values
  static bool attr_set = false;
  if (!attr_set) {
    hipFuncAttributes fa;
    hipError_t e = hipFuncGetAttributes(&fa, reinterpret_cast<const void*>(kern));
    if (e != hipSuccess) return e;
    static_lds = fa.sharedSizeBytes;
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                            hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)(160 * 1024 - static_lds));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const size_t lds = stream_lds_bytes(MB, p.kchunk, WK, EPI == EPI_GLU);
  if (lds + static_lds > 160 * 1024) return hipErrorInvalidValue;
  dim3 grid((unsigned)((p.rb_b + nbpb - 1) / nbpb), (unsigned)p.splits);
  kern<<<grid, 64 * NW, lds, st>>>(p, nbpb);
  return hipGetLastError();
}

template <int DT, int MB, int EPI, int NW, int WK>
static hipError_t stream_launch(const GemmParams& p, int nbpb, hipStream_t st) {
  if constexpr (DT == DT_I8 && MB == 1) {
    if (p.g_x_in) return stream_launch_ql<DT, MB, EPI, NW, WK, 2>(p, nbpb, st);
  }
  if constexpr ((DT == DT_I8 || DT == DT_F8) && MB == 1) {
    if (p.a_x) return stream_launch_ql<DT, MB, EPI, NW, WK, 1>(p, nbpb, st);
  }
  return stream_launch_ql<DT, MB, EPI, NW, WK, 0>(p, nbpb, st);
}

// Instantiated wave layouts: 16-wave workgroups only for MB == 1 (at 16 waves a
// wave has 128 registers, too few for larger MB), 4 waves sharing K only where
// the accumulators still fit without spilling.
template <int DT, int MB, int EPI>
static hipError_t stream_waves(int nw, int wk, const GemmParams& p, int nbpb, hipStream_t st) {
  if (nw == 1 && wk == 1) return stream_launch<DT, MB, EPI, 1, 1>(p, nbpb, st);
  if (nw == 4 && wk == 1) return stream_launch<DT, MB, EPI, 4, 1>(p, nbpb, st);
  if (nw == 2 && wk == 2) return stream_launch<DT, MB, EPI, 2, 2>(p, nbpb, st);
  if constexpr (MB <= 4 || EPI != EPI_GLU) {
    if (nw == 4 && wk == 4) return stream_launch<DT, MB, EPI, 4, 4>(p, nbpb, st);
  }
  if constexpr (MB == 1 && EPI != EPI_GLU) {  // the gated 16-wave variant would spill
    if (nw == 16 && wk == 16) return stream_launch<DT, MB, EPI, 16, 16>(p, nbpb, st);
  }
  return hipErrorInvalidValue;
}

template <int DT, int EPI>
static hipError_t stream_mb(int mb, int nw, int wk, const GemmParams& p, int nbpb, hipStream_t st) {
  switch (mb) {
    case 1: return stream_waves<DT, 1, EPI>(nw, wk, p, nbpb, st);
    case 2: return stream_waves<DT, 2, EPI>(nw, wk, p, nbpb, st);
    case 4: return stream_waves<DT, 4, EPI>(nw, wk, p, nbpb, st);
    case 8:
      if constexpr (DT != DT_F8) return stream_waves<DT, 8, EPI>(nw, wk, p, nbpb, st);
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

template <int DT>
static hipError_t stream_epi(int epi, int mb, int nw, int wk, const GemmParams& p, int nbpb,
                             hipStream_t st) {
  switch (epi) {
    case EPI_I32:
      if constexpr (DT == DT_BF16) return hipErrorInvalidValue;
      return stream_mb<DT, EPI_I32>(mb, nw, wk, p, nbpb, st);
    case EPI_F32: return stream_mb<DT, EPI_F32>(mb, nw, wk, p, nbpb, st);
    case EPI_BF16: return stream_mb<DT, EPI_BF16>(mb, nw, wk, p, nbpb, st);
    case EPI_GLU: return stream_mb<DT, EPI_GLU>(mb, nw, wk, p, nbpb, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm_stream(int dt, int epi, int mb, int nw, int wk, const GemmParams& p,
                              int nb_per_block, hipStream_t st) {
  if (!gemm_params_ok(dt, epi, p, 1, nw)) return hipErrorInvalidValue;
  if (p.M > 16 * mb || nb_per_block < 1) return hipErrorInvalidValue;
  switch (dt) {
    case DT_I8: return stream_epi<DT_I8>(epi, mb, nw, wk, p, nb_per_block, st);
    case DT_BF16: return stream_epi<DT_BF16>(epi, mb, nw, wk, p, nb_per_block, st);
    case DT_F8: return stream_epi<DT_F8>(epi, mb, nw, wk, p, nb_per_block, st);
    default: return hipErrorInvalidValue;
  }
}

size_t gemm_stream_lds_bytes(int mb, int kchunk, int wk, bool glu) {
  return stream_lds_bytes(mb, kchunk, wk, glu);
}

template <int DT>
static hipError_t reduce_epi(int epi, const GemmParams& p, hipStream_t st) {
  const int64_t n4 = (p.N + 3) / 4;
  const unsigned blocks = (unsigned)((p.M * n4 + 255) / 256);
  switch (epi) {
    case EPI_I32:
      if constexpr (DT == DT_BF16) return hipErrorInvalidValue;
      else splitk_reduce_kernel<DT, EPI_I32><<<blocks, 256, 0, st>>>(p);
      break;
    case EPI_F32: splitk_reduce_kernel<DT, EPI_F32><<<blocks, 256, 0, st>>>(p); break;
    case EPI_BF16: splitk_reduce_kernel<DT, EPI_BF16><<<blocks, 256, 0, st>>>(p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_splitk_reduce(int dt, int epi, const GemmParams& p, hipStream_t st) {
  if (!gemm_params_ok(dt, epi, p, 2)) return hipErrorInvalidValue;
  switch (dt) {
    case DT_I8: return reduce_epi<DT_I8>(epi, p, st);
    case DT_BF16: return reduce_epi<DT_BF16>(epi, p, st);
    case DT_F8: return reduce_epi<DT_F8>(epi, p, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace w8a8
