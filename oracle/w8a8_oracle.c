/*
 * CPU oracle for the W8A8 SmoothQuant path of arxiv 2608.28003 (Gemma-3-1B
 * layer-wise INT8/bf16 allocation).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow reference that the
 * GPU library is checked against.  Only the test-suite, the smoke check and
 * the CPU-baseline leg of the benchmark may load it; the product library never
 * links, includes or calls it, and it shares no code with the HIP sources.
 *
 * Every function is a direct loop over the definition it cites: no blocking,
 * no fusion, no reordering of the arithmetic the definition states.  OpenMP
 * only distributes independent output rows.
 *
 * Precision (readings of a paper that does not fix it):
 *   - values that decide an integer code (smoothed inputs, scales, the ratio
 *     that is rounded) are formed in IEEE binary32, one rounding per
 *     operation, no contraction -- the precision the GPU kernels decide them in;
 *   - integer products are summed exactly (int64, then range-checked to int32);
 *   - the dequantised value y = s_t * s_i * acc is formed in binary32 with the
 *     token scale applied first (its result feeds the codes of the next
 *     projection inside the FFN);
 *   - tanh inside GELU is libm's binary64 tanh rounded once to binary32;
 *   - the bf16 reference path (layers the precision map keeps in bf16) and the
 *     RMSNorm glue are evaluated in binary64 and rounded once.
 *
 * Build: gcc -O3 -std=c11 -fPIC -shared -fopenmp -ffp-contract=off
 *        -fno-fast-math   (contraction would fuse a*b+c and change results)
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define ORC_MODE_DIV 0 /* activations: x_hat = x / delta   (eq. xhat-lmhead) */
#define ORC_MODE_MUL 1 /* weights:     W_hat = W * delta   (eq. what-lmhead) */

/* ------------------------------------------------------------------ */
/* Number formats                                                       */
/* ------------------------------------------------------------------ */

/* bf16 -> fp32 is exact: the bf16 pattern is the top half of the fp32 one. */
void orc_bf16_to_f32(const uint16_t* src, int64_t n, float* dst) {
    for (int64_t i = 0; i < n; ++i) {
        uint32_t u = ((uint32_t)src[i]) << 16;
        memcpy(&dst[i], &u, 4);
    }
}

/* fp32 -> bf16, round to nearest, ties to even (IEEE default rounding). */
static uint16_t f32_to_bf16_rne(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return 0x7fc0; /* NaN */
    uint32_t keep = u >> 16;
    uint32_t rest = u & 0xffffu;
    if (rest > 0x8000u || (rest == 0x8000u && (keep & 1u))) keep += 1u;
    return (uint16_t)keep;
}

void orc_f32_to_bf16(const float* src, int64_t n, uint16_t* dst) {
    for (int64_t i = 0; i < n; ++i) dst[i] = f32_to_bf16_rne(src[i]);
}

/* binary64 -> bf16 rounded once (not through binary32, which would round
   twice): scale |v| onto the grid of 8 significant bits (the bf16 spacing,
   never finer than the subnormal step 2^-133), round half to even there and
   scale back; the result has at most 8 significant bits, so it converts to
   binary32 exactly (or overflows to inf, as round-to-nearest requires). */
static uint16_t f64_to_bf16_rne(double v) {
    if (v != v) return 0x7fc0;
    if (v == 0.0) return signbit(v) ? 0x8000 : 0x0000;
    int e;
    (void)frexp(v, &e);  /* |v| in [2^(e-1), 2^e) */
    int q = e - 8;       /* spacing of 8 significant bits */
    if (q < -133) q = -133;
    double r = rint(ldexp(v, -q));
    float f = (float)ldexp(r, q);
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
}

void orc_f64_to_bf16(const double* src, int64_t n, uint16_t* dst) {
    for (int64_t i = 0; i < n; ++i) dst[i] = f64_to_bf16_rne(src[i]);
}

/* round half to even, in binary32 (the default IEEE rounding mode) */
static float rne_f32(float r) { return rintf(r); }

/* ------------------------------------------------------------------ */
/* a1  Calibration (eq. delta-attn, eq. delta-lmhead)                   */
/* ------------------------------------------------------------------ */

/* Running column maximum of |X[t][j]| over rows t: the activation statistic
   max_t |X_tj| gathered over calibration tokens, and, applied to a weight
   matrix, max_i |W_ij| over its output rows.  amax is read and updated. */
void orc_col_absmax(const float* x, int64_t rows, int64_t k, float* amax) {
    for (int64_t j = 0; j < k; ++j) {
        float m = amax[j];
        for (int64_t t = 0; t < rows; ++t) {
            float v = fabsf(x[t * k + j]);
            if (v > m) m = v;
        }
        amax[j] = m;
    }
}

/* delta_j = (max_t |X_tj|)^alpha / (max_i |W_ij|)^(1-alpha), both maxima
   floored at eps so a dead channel yields a finite factor.  Evaluated in
   binary64 and rounded once; at alpha = 1/2 the powers are square roots. */
void orc_smooth_delta(const float* act_amax, const float* w_amax, int64_t k,
                      double alpha, double eps, float* delta) {
    for (int64_t j = 0; j < k; ++j) {
        double a = (double)act_amax[j], w = (double)w_amax[j];
        if (a < eps) a = eps;
        if (w < eps) w = eps;
        double d;
        if (alpha == 0.5)
            d = sqrt(a) / sqrt(w);
        else
            d = pow(a, alpha) / pow(w, 1.0 - alpha);
        delta[j] = (float)d;
    }
}

/* ------------------------------------------------------------------ */
/* a2/a3  Symmetric per-row int8 quantisation                           */
/*   eq. si / what-ffn (per output channel of W_hat = W diag(delta))    */
/*   eq. stx / xint8   (per token of x_hat = x / delta)                 */
/* ------------------------------------------------------------------ */

/* For each row r:  v_j = x_rj / delta_j (DIV) or x_rj * delta_j (MUL), or x_rj
   when delta is NULL;  amax = max_j |v_j|;  s_r = amax / 127;
   q_rj = clamp(rne(v_j / s_r), -127, 127);  an all-zero row gives s = 0, q = 0.
   If vhat is not NULL the smoothed binary32 values v are also stored. */
void orc_quant_rows(const float* x, int64_t rows, int64_t k, const float* delta,
                    int mode, int8_t* q, float* s, float* vhat) {
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r) {
        const float* xr = x + r * k;
        float amax = 0.0f;
        for (int64_t j = 0; j < k; ++j) {
            float v = xr[j];
            if (delta) v = (mode == ORC_MODE_DIV) ? v / delta[j] : v * delta[j];
            if (vhat) vhat[r * k + j] = v;
            float a = fabsf(v);
            if (a > amax) amax = a;
        }
        float sr = amax / 127.0f;
        s[r] = sr;
        for (int64_t j = 0; j < k; ++j) {
            float v = xr[j];
            if (delta) v = (mode == ORC_MODE_DIV) ? v / delta[j] : v * delta[j];
            int8_t code = 0;
            if (sr != 0.0f) {
                float c = rne_f32(v / sr);
                if (c > 127.0f) c = 127.0f;
                if (c < -127.0f) c = -127.0f;
                code = (int8_t)c;
            }
            q[r * k + j] = code;
        }
    }
}

/* ------------------------------------------------------------------ */
/* a4  INT8 x INT8 -> INT32 product (the sum of eq. gemm-final)         */
/* ------------------------------------------------------------------ */

/* acc[t][i] = sum_j a[t][j] * b[i][j], summed exactly.  Every product is at
   most 128^2 = 2^14 in magnitude, so for k <= 2^17 - 1 no partial sum leaves
   the int32 range and the sum runs in int32 (exact, and a loop the compiler
   vectorises); longer rows sum in int64.  Returns the number of sums outside
   the int32 range (0 for every K <= 133144 with codes in [-127, 127]). */
int64_t orc_gemm_i32(const int8_t* a, const int8_t* b, int64_t m, int64_t n,
                     int64_t k, int32_t* acc) {
    int64_t overflow = 0;
    const int narrow = k < (1 << 17);
#pragma omp parallel for schedule(static) reduction(+ : overflow)
    for (int64_t t = 0; t < m; ++t) {
        const int8_t* ar = a + t * k;
        for (int64_t i = 0; i < n; ++i) {
            const int8_t* br = b + i * k;
            if (narrow) {
                int32_t sum = 0;
                for (int64_t j = 0; j < k; ++j) sum += (int32_t)ar[j] * (int32_t)br[j];
                acc[t * n + i] = sum;
            } else {
                int64_t sum = 0;
                for (int64_t j = 0; j < k; ++j) sum += (int64_t)ar[j] * (int64_t)br[j];
                if (sum > INT32_MAX || sum < INT32_MIN) overflow += 1;
                acc[t * n + i] = (int32_t)sum;
            }
        }
    }
    return overflow;
}

/* ------------------------------------------------------------------ */
/* a5  Dequantisation (eq. gemm-final)                                  */
/* ------------------------------------------------------------------ */

/* y[t][i] = (float(acc[t][i]) * s_t) * s_i, binary32, token scale first. */
void orc_dequant(const int32_t* acc, const float* s_tok, const float* s_ch,
                 int64_t m, int64_t n, float* y) {
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < m; ++t)
        for (int64_t i = 0; i < n; ++i) {
            float a = (float)acc[t * n + i];
            float p = a * s_tok[t];
            y[t * n + i] = p * s_ch[i];
        }
}

/* ------------------------------------------------------------------ */
/* a6  GeGLU with the tanh form of GELU (gate branch), times up         */
/* ------------------------------------------------------------------ */

/* gelu(g) = 0.5 g (1 + tanh(z)),  z = sqrt(2/pi) (g + 0.044715 g^3);  h = gelu(g) u.
   Binary64 throughout; the caller rounds h once to bf16 (the FFN intermediate
   format).  The factor 1 + tanh(z) is taken as 2 / (1 + exp(-2z)), the same
   number: written as 1 + tanh(z) it cancels for negative z and keeps no
   correct digit below z of about -18 in binary64. */
void orc_geglu_f64(const double* g, const double* u, int64_t n, double* h) {
    const double c = 0.79788456080286535588;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double x = g[i];
        double z = c * (x + 0.044715 * x * x * x);
        double one_plus_tanh = 2.0 / (1.0 + exp(-2.0 * z));
        double ge = 0.5 * x * one_plus_tanh;
        h[i] = ge * u[i];
    }
}

/* ------------------------------------------------------------------ */
/* FP8 variant (Sec. 4, the listed move from INT8 to FP8 codes)         */
/* ------------------------------------------------------------------ */

/* OCP FP8 E4M3 ("fn"): 1 sign, 4 exponent (bias 7), 3 mantissa bits.
   Exponent field 0 holds the subnormals m/8 * 2^-6; field 1..15 the normals
   (1 + m/8) * 2^(e-7), except field 15 with mantissa 7, which is NaN.  The
   largest finite magnitude is 1.75 * 2^8 = 448; there is no infinity. */
double orc_e4m3_decode(uint8_t c) {
    int sgn = c >> 7, e = (c >> 3) & 15, m = c & 7;
    double v;
    if (e == 15 && m == 7) return NAN;
    if (e == 0) v = ldexp((double)m / 8.0, -6);
    else v = ldexp(1.0 + (double)m / 8.0, e - 7);
    return sgn ? -v : v;
}

/* Nearest E4M3 value to a binary32 x, ties to the even code (even mantissa),
   magnitudes beyond 448 saturate to 448 (the quantiser below never produces
   them beyond rounding).  Chosen by comparing x with the exact midpoints of
   consecutive codes, which are all representable in binary64. */
uint8_t orc_e4m3_encode(float x) {
    uint8_t sgn = (x < 0.0f || (x == 0.0f && signbit(x))) ? 0x80 : 0x00;
    double a = fabs((double)x);
    if (isnan(x)) return 0x7f;
    if (a >= 448.0) return sgn | 0x7e;
    /* codes 0..126 ascend in value: find the first whose value reaches a */
    int lo = 0;
    while (lo < 126 && orc_e4m3_decode((uint8_t)(lo + 1)) <= a) ++lo;
    /* a lies in [value(lo), value(lo + 1)) */
    if (lo == 126) return sgn | 126;
    double v0 = orc_e4m3_decode((uint8_t)lo), v1 = orc_e4m3_decode((uint8_t)(lo + 1));
    double mid = 0.5 * (v0 + v1);
    int code;
    if (a < mid) code = lo;
    else if (a > mid) code = lo + 1;
    else code = (lo & 1) ? lo + 1 : lo; /* tie: even mantissa = even code */
    return sgn | (uint8_t)code;
}

void orc_e4m3_encode_n(const float* x, int64_t n, uint8_t* out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = orc_e4m3_encode(x[i]);
}

/* Row quantisation with E4M3 codes: as orc_quant_rows, with the scale
   s = amax / 448 and code = E4M3(fl32(v / s)); a zero row gets s = 0, codes 0. */
void orc_quant_rows_fp8(const float* x, int64_t rows, int64_t k, const float* delta,
                        int mode, uint8_t* q, float* s) {
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r) {
        const float* xr = x + r * k;
        float amax = 0.0f;
        for (int64_t j = 0; j < k; ++j) {
            float v = xr[j];
            if (delta) v = (mode == ORC_MODE_DIV) ? v / delta[j] : v * delta[j];
            float a = fabsf(v);
            if (a > amax) amax = a;
        }
        float sr = amax / 448.0f;
        s[r] = sr;
        for (int64_t j = 0; j < k; ++j) {
            float v = xr[j];
            if (delta) v = (mode == ORC_MODE_DIV) ? v / delta[j] : v * delta[j];
            q[r * k + j] = sr != 0.0f ? orc_e4m3_encode(v / sr) : 0;
        }
    }
}

/* acc[t][i] = sum_j dec(a[t][j]) dec(b[i][j]) in binary64 (every product is
   exact; the sum is exact up to binary64 rounding). */
void orc_gemm_fp8(const uint8_t* a, const uint8_t* b, int64_t m, int64_t n, int64_t k,
                  double* acc) {
    double table[256];
    for (int c = 0; c < 256; ++c) table[c] = orc_e4m3_decode((uint8_t)c);
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < m; ++t)
        for (int64_t i = 0; i < n; ++i) {
            double sum = 0.0;
            for (int64_t j = 0; j < k; ++j) sum += table[a[t * k + j]] * table[b[i * k + j]];
            acc[t * n + i] = sum;
        }
}

/* Dequantisation of FP8 sums: y = fl32(fl32(fl32(acc) * s_t) * s_i), the
   binary32 order of the INT8 path with the sum rounded to binary32 first (the
   matrix cores accumulate in binary32). */
void orc_dequant_fp8(const double* acc, const float* s_tok, const float* s_ch, int64_t m,
                     int64_t n, float* y) {
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < m; ++t)
        for (int64_t i = 0; i < n; ++i) {
            float a = (float)acc[t * n + i];
            float p = a * s_tok[t];
            y[t * n + i] = p * s_ch[i];
        }
}

/* ------------------------------------------------------------------ */
/* bf16 reference path and stack glue (binary64)                       */
/* ------------------------------------------------------------------ */

/* y[t][i] = sum_j x[t][j] * w[i][j] in binary64 (x, w given exactly as
   binary32 values widened from bf16). */
void orc_linear_f64(const float* x, const float* w, int64_t m, int64_t n,
                    int64_t k, double* y) {
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < m; ++t)
        for (int64_t i = 0; i < n; ++i) {
            double sum = 0.0;
            for (int64_t j = 0; j < k; ++j)
                sum += (double)x[t * k + j] * (double)w[i * k + j];
            y[t * n + i] = sum;
        }
}

/* RMSNorm with unit gain: y = x / sqrt(mean_j x_j^2 + eps), binary64. */
void orc_rmsnorm_f64(const float* x, int64_t m, int64_t d, double eps, double* y) {
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < m; ++t) {
        double ss = 0.0;
        for (int64_t j = 0; j < d; ++j) ss += (double)x[t * d + j] * (double)x[t * d + j];
        double inv = 1.0 / sqrt(ss / (double)d + eps);
        for (int64_t j = 0; j < d; ++j) y[t * d + j] = (double)x[t * d + j] * inv;
    }
}

/* ------------------------------------------------------------------ */
/* f4  One-token attention over a key/value cache (Sec. 4 lists an     */
/* INT8 key/value cache among the further speed-ups; Sec. 2 gives the   */
/* grouped-query layout: several query heads share one key/value head)  */
/* ------------------------------------------------------------------ */

/* q is h x dh (the query heads of one token), k and v are t x dh (the rows of
   the one shared key/value head), all binary64.  For every head i:
     score_t = scale * sum_d q[i][d] * k[t][d]
     p_t     = exp(score_t - max_u score_u) / sum_u exp(score_u - max_u score_u)
     out[i][d] = sum_t p_t * v[t][d]
   Subtracting the maximum leaves p unchanged and keeps every exp finite. */
void orc_attn_decode_f64(const double* q, int64_t h, int64_t dh, const double* k,
                         const double* v, int64_t t, double scale, double* out) {
    for (int64_t i = 0; i < h; ++i) {
        const double* qi = q + i * dh;
        double* oi = out + i * dh;
        double mx = -INFINITY;
        for (int64_t u = 0; u < t; ++u) {
            double sc = 0.0;
            for (int64_t d = 0; d < dh; ++d) sc += qi[d] * k[u * dh + d];
            sc *= scale;
            if (sc > mx) mx = sc;
        }
        double den = 0.0;
        for (int64_t d = 0; d < dh; ++d) oi[d] = 0.0;
        for (int64_t u = 0; u < t; ++u) {
            double sc = 0.0;
            for (int64_t d = 0; d < dh; ++d) sc += qi[d] * k[u * dh + d];
            sc *= scale;
            double p = exp(sc - mx);
            den += p;
            for (int64_t d = 0; d < dh; ++d) oi[d] += p * v[u * dh + d];
        }
        for (int64_t d = 0; d < dh; ++d) oi[d] /= den;
    }
}
