/* CPU oracle for the schedule-parameterised contractions.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the tests, the smoke check and the benchmark's CPU
 * baseline use it.  It shares no source with the HIP path.
 *
 * What it computes.  A schedule (tiling, vector width, unrolling, staging,
 * fusion, operand layout) is a semantics-preserving transformation of the
 * operator (Sec. 2, Eq. 1: every transformation maps a program to an
 * equivalent program).  So every schedule must reach the operator's plain
 * mathematical definition up to rounding order, and the oracle is that
 * definition written out as loop nests:
 *   - inputs are decoded exactly from the fp32 / bf16 bit patterns the GPU
 *     receives;
 *   - every sum and every nonlinearity is evaluated in fp64;
 *   - the only roundings are the stated storage points: fp32 output for the
 *     fp32 GEMM, bf16 (round to nearest even) for bf16 outputs, and the
 *     bf16 hidden activation H of the gated MLP and of each MoE expert.
 * The operator shapes are the layers the paper evaluates (Sec. 4.1: Llama-3
 * attention, DeepSeek-R1 MoE, FLUX convolution, Llama-4 MLP) and the fp32
 * contraction of the MoE example module in App. A.
 *
 * Each function evaluates a caller-chosen subset of independent outputs
 * (rows, tokens, query rows or pixels) so that full-size problems can be
 * checked on samples.  OpenMP parallelises over that subset only.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double bf16_val(uint16_t b) {
    uint32_t u = ((uint32_t)b) << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

/* Round an fp64 value to the nearest bf16 (8 significant bits, 8-bit
 * exponent, subnormals down to 2^-133), ties to even, overflow to inf. */
uint16_t orc_bf16_from_f64(double x) {
    if (isnan(x)) return 0x7FC0;
    if (isinf(x)) return x > 0 ? 0x7F80 : 0xFF80;
    if (x == 0.0) return signbit(x) ? 0x8000 : 0x0000;
    int ex;
    frexp(x, &ex);            /* |x| = m * 2^ex, m in [0.5, 1) */
    int e = ex - 8;           /* spacing of bf16 values near x */
    if (e < -133) e = -133;   /* subnormal spacing */
    double q = rint(ldexp(x, -e));   /* default mode: nearest, ties to even */
    double r = ldexp(q, e);
    if (fabs(r) >= 0x1p128) return x > 0 ? 0x7F80 : 0xFF80;
    float f = (float)r;       /* exact: r is a bf16 value */
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
}

void orc_bf16_round(const double *x, uint16_t *out, int64_t n) {
    for (int64_t i = 0; i < n; ++i) out[i] = orc_bf16_from_f64(x[i]);
}

/* SiLU(x) = x * sigmoid(x) = x / (1 + e^-x). */
double orc_silu(double x) { return x / (1.0 + exp(-x)); }

static int64_t pick(const int64_t *sel, int64_t i) { return sel ? sel[i] : i; }

/* fp32 GEMM: C = A B with A [M][K], B [K][N] row-major fp32; row r of the
 * output block is row sel[r] of the product, rounded once to fp32. */
void orc_gemm_f32(const float *A, const float *B, float *C, double *C64, int64_t M, int64_t N,
                  int64_t K, const int64_t *sel, int64_t nsel) {
    if (!sel) nsel = M;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < nsel; ++r) {
        int64_t m = pick(sel, r);
        for (int64_t n = 0; n < N; ++n) {
            double s = 0.0;
            for (int64_t k = 0; k < K; ++k) s += (double)A[m * K + k] * (double)B[k * N + n];
            C[r * N + n] = (float)s;
            if (C64) C64[r * N + n] = s;
        }
    }
}

/* Scaled dot-product attention for one query row.
 * Q, K, V are [B][H][S][D] bf16.  For query i of head (b, h):
 *   s_j = (q_i . k_j) / sqrt(D) for the visible keys (all j, or j <= i when
 *   causal, the top-left aligned mask), p = softmax(s), o_i = sum_j p_j v_j.
 * sel lists flat query indices (b*H + h)*S + i; O is [nsel][D] bf16. */
void orc_attention_bf16(const uint16_t *Q, const uint16_t *Kt, const uint16_t *V, uint16_t *O,
                        double *O64, int64_t B, int64_t H, int64_t S, int64_t D, int causal,
                        const int64_t *sel, int64_t nsel) {
    if (!sel) nsel = B * H * S;
    double scale = 1.0 / sqrt((double)D);
#pragma omp parallel
    {
        double *s = (double *)malloc(sizeof(double) * (size_t)S);
        double *o = (double *)malloc(sizeof(double) * (size_t)D);
#pragma omp for schedule(dynamic, 4)
        for (int64_t r = 0; r < nsel; ++r) {
            int64_t flat = pick(sel, r);
            int64_t bh = flat / S, i = flat % S;
            const uint16_t *q = Q + (bh * S + i) * D;
            const uint16_t *kb = Kt + bh * S * D;
            const uint16_t *vb = V + bh * S * D;
            int64_t nvis = causal ? i + 1 : S;
            double mx = -INFINITY;
            for (int64_t j = 0; j < nvis; ++j) {
                double dot = 0.0;
                for (int64_t d = 0; d < D; ++d) dot += bf16_val(q[d]) * bf16_val(kb[j * D + d]);
                s[j] = dot * scale;
                if (s[j] > mx) mx = s[j];
            }
            double l = 0.0;
            for (int64_t j = 0; j < nvis; ++j) {
                s[j] = exp(s[j] - mx);
                l += s[j];
            }
            for (int64_t d = 0; d < D; ++d) o[d] = 0.0;
            for (int64_t j = 0; j < nvis; ++j) {
                double p = s[j] / l;
                for (int64_t d = 0; d < D; ++d) o[d] += p * bf16_val(vb[j * D + d]);
            }
            for (int64_t d = 0; d < D; ++d) {
                O[r * D + d] = orc_bf16_from_f64(o[d]);
                if (O64) O64[r * D + d] = o[d];
            }
        }
        free(s);
        free(o);
    }
}

/* Gated MLP for one token x (length Hd):
 *   h = bf16( SiLU(x Wg) * (x Wu) )   (length I, stored as bf16)
 *   out = bf16( h Wd )                 (length Hd)
 * Wg, Wu are [Hd][I], Wd is [I][Hd], all bf16.  Hmid (optional) receives h. */
static void mlp_token(const uint16_t *x, const uint16_t *Wg, const uint16_t *Wu,
                      const uint16_t *Wd, int64_t Hd, int64_t I, double *g, double *u,
                      double *hv, uint16_t *hbits, double *out) {
    for (int64_t n = 0; n < I; ++n) { g[n] = 0.0; u[n] = 0.0; }
    for (int64_t k = 0; k < Hd; ++k) {
        double xk = bf16_val(x[k]);
        for (int64_t n = 0; n < I; ++n) {
            g[n] += xk * bf16_val(Wg[k * I + n]);
            u[n] += xk * bf16_val(Wu[k * I + n]);
        }
    }
    for (int64_t n = 0; n < I; ++n) {
        hbits[n] = orc_bf16_from_f64(orc_silu(g[n]) * u[n]);
        hv[n] = bf16_val(hbits[n]);
    }
    for (int64_t d = 0; d < Hd; ++d) out[d] = 0.0;
    for (int64_t n = 0; n < I; ++n) {
        for (int64_t d = 0; d < Hd; ++d) out[d] += hv[n] * bf16_val(Wd[n * Hd + d]);
    }
}

void orc_gated_mlp_bf16(const uint16_t *X, const uint16_t *Wg, const uint16_t *Wu,
                        const uint16_t *Wd, uint16_t *Out, double *Out64, uint16_t *Hmid,
                        int64_t T, int64_t Hd, int64_t I, const int64_t *sel, int64_t nsel) {
    if (!sel) nsel = T;
#pragma omp parallel
    {
        double *g = (double *)malloc(sizeof(double) * (size_t)I);
        double *u = (double *)malloc(sizeof(double) * (size_t)I);
        double *hv = (double *)malloc(sizeof(double) * (size_t)I);
        uint16_t *hb = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)I);
        double *o = (double *)malloc(sizeof(double) * (size_t)Hd);
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < nsel; ++r) {
            int64_t t = pick(sel, r);
            mlp_token(X + t * Hd, Wg, Wu, Wd, Hd, I, g, u, hv, hb, o);
            for (int64_t d = 0; d < Hd; ++d) {
                Out[r * Hd + d] = orc_bf16_from_f64(o[d]);
                if (Out64) Out64[r * Hd + d] = o[d];
            }
            if (Hmid) memcpy(Hmid + r * I, hb, sizeof(uint16_t) * (size_t)I);
        }
        free(g); free(u); free(hv); free(hb); free(o);
    }
}

/* Routed mixture of gated-MLP experts for one token t:
 *   out_t = bf16( sum_{s < topk} w[t][s] * ( h_s Wd[e_s] ) ),
 *   h_s = bf16( SiLU(x_t Wg[e_s]) * (x_t Wu[e_s]) ),  e_s = ids[t][s].
 * Wg, Wu are [E][Hd][I], Wd is [E][I][Hd] (bf16); ids int32 and w fp32 are
 * [T][topk].  The per-expert result is kept in fp64 before the weighted sum. */
void orc_moe_bf16(const uint16_t *X, const int32_t *ids, const float *w, const uint16_t *Wg,
                  const uint16_t *Wu, const uint16_t *Wd, uint16_t *Out, double *Out64,
                  int64_t T, int64_t Hd, int64_t E, int64_t I, int64_t topk,
                  const int64_t *sel, int64_t nsel) {
    (void)E;
    if (!sel) nsel = T;
#pragma omp parallel
    {
        double *g = (double *)malloc(sizeof(double) * (size_t)I);
        double *u = (double *)malloc(sizeof(double) * (size_t)I);
        double *hv = (double *)malloc(sizeof(double) * (size_t)I);
        uint16_t *hb = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)I);
        double *y = (double *)malloc(sizeof(double) * (size_t)Hd);
        double *acc = (double *)malloc(sizeof(double) * (size_t)Hd);
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < nsel; ++r) {
            int64_t t = pick(sel, r);
            for (int64_t d = 0; d < Hd; ++d) acc[d] = 0.0;
            for (int64_t s = 0; s < topk; ++s) {
                int64_t e = ids[t * topk + s];
                double ws = (double)w[t * topk + s];
                mlp_token(X + t * Hd, Wg + e * Hd * I, Wu + e * Hd * I, Wd + e * I * Hd, Hd, I,
                          g, u, hv, hb, y);
                for (int64_t d = 0; d < Hd; ++d) acc[d] += ws * y[d];
            }
            for (int64_t d = 0; d < Hd; ++d) {
                Out[r * Hd + d] = orc_bf16_from_f64(acc[d]);
                if (Out64) Out64[r * Hd + d] = acc[d];
            }
        }
        free(g); free(u); free(hv); free(hb); free(y); free(acc);
    }
}

/* 2-D convolution, stride 1, zero padding `pad`, NHWC activations and
 * [K][R][S][C] filters (bf16), fp32 bias:
 *   pre[n,p,q,o] = bias[o] + sum_{r,s,c} x[n, p+r-pad, q+s-pad, c] * w[o,r,s,c]
 * with x = 0 outside the image; y = bf16(SiLU(pre)) when act = 1, else
 * bf16(pre).  Output spatial size is (H + 2 pad - R + 1) x (W + 2 pad - S + 1).
 * sel lists flat output pixels (n*P + p)*Q + q; y is [nsel][K]. */
void orc_conv2d_bf16(const uint16_t *x, const uint16_t *w, const float *bias, uint16_t *y,
                     double *y64, int64_t N, int64_t H, int64_t W, int64_t C, int64_t K,
                     int64_t R, int64_t S, int64_t pad, int act, const int64_t *sel,
                     int64_t nsel) {
    int64_t P = H + 2 * pad - R + 1, Q = W + 2 * pad - S + 1;
    if (!sel) nsel = N * P * Q;
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t r0 = 0; r0 < nsel; ++r0) {
        int64_t flat = pick(sel, r0);
        int64_t n = flat / (P * Q), p = (flat / Q) % P, q = flat % Q;
        for (int64_t o = 0; o < K; ++o) {
            double s = bias ? (double)bias[o] : 0.0;
            for (int64_t r = 0; r < R; ++r) {
                int64_t ih = p + r - pad;
                if (ih < 0 || ih >= H) continue;
                for (int64_t t = 0; t < S; ++t) {
                    int64_t iw = q + t - pad;
                    if (iw < 0 || iw >= W) continue;
                    const uint16_t *xp = x + ((n * H + ih) * W + iw) * C;
                    const uint16_t *wp = w + ((o * R + r) * S + t) * C;
                    for (int64_t c = 0; c < C; ++c) s += bf16_val(xp[c]) * bf16_val(wp[c]);
                }
            }
            double v = act ? orc_silu(s) : s;
            y[r0 * K + o] = orc_bf16_from_f64(v);
            if (y64) y64[r0 * K + o] = v;
        }
    }
}

int orc_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
