/*
 * TEST INFRASTRUCTURE ONLY -- plain, slow CPU oracle for the TwinQuant
 * dual-component W4A4 linear layer.  Only the test-suite, the smoke check
 * and the benchmark's CPU-baseline leg may load this library; the product
 * path never does.  It shares no source with the HIP library.
 *
 * What it computes (paper: "TwinQuant: Learnable Subspace Decomposition for
 * 4-Bit LLM Quantization"):
 *
 *   Y = Q(X) [ Q(U') Q(V') + Q(R') ]                     (Sec. 4.1, Eq. 4/6)
 *
 * with the activation X [M,K], the residual R' stored as W_res [N,K]
 * (PyTorch Linear convention, Y = X W_res^T), and the low-rank factors
 * U' = L1 [K,r], V' = L2 [r,N].  Q is the symmetric 4-bit quantizer of
 * Sec. 2, Eq. (1) (q_max = 2^(4-1) - 1 = 7) applied group-wise with one
 * scale per contiguous group (Sec. 5.1, implementation details).  The
 * low-rank branch runs in two integer stages with the intermediate H
 * re-quantized on the fly (Sec. 4.3, "on-the-fly scaling with a single
 * epilogue"); both branches are merged once at the end.
 *
 * Steps, in the order the paper describes them:
 *   O1  quantize X per token and K-group                  (Eq. 1)
 *   O2  quantize W_res per output row along K, L1 per rank column along K,
 *       L2 per output column along r                      (Eq. 1, Sec. 5.1)
 *   O3  residual: per group an exact integer dot product, scaled by
 *       s_x * s_w and accumulated over groups             (Eq. 2)
 *   O4  stage 1: H = sum_g (s_x * s_L1) * A_g             (Sec. 4.3)
 *   O5  re-quantize H per token and r-group; the scale s_H stays fp32
 *   O6  stage 2: Y_lr = sum_h (s_H * s_L2) * B_h          (Sec. 4.3)
 *   O7  Y = Y_res + Y_lr, rounded once to fp16 (or bf16)  (Sec. 4.3)
 *
 * Readings where the paper is silent (each is listed in the design notes):
 *   - round() is round-half-to-even; codes are clamped to [-7, 7].
 *   - stored scales are fp16: s = fp16_rne(fp32(max|v|) / 7); an all-zero
 *     group has scale 0 and codes 0.
 *   - groups run along each product's reduction axis; the r-axis group is
 *     min(G, r).
 *   - the low-rank branch consumes the same Q(X) codes as the residual.
 *   - H is accumulated in fp32 in ascending group order with one fused
 *     multiply-add per group; s_H = fp32(max|H|) / 7 in fp32.  Because H
 *     decides integer codes, the oracle takes that decision in the
 *     kernel's precision (fp32, this order).
 *   - Y_res and Y_lr are accumulated the same way (ascending group, fma);
 *     the fp64 result Y64 is the same sum without intermediate rounding.
 *
 * Build: gcc -O2 -std=c99 -fopenmp -ffp-contract=off -fPIC -shared
 * (no -ffast-math: every float operation must be IEEE single precision).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ */
/* IEEE binary16 / bfloat16 encode and decode, written from the format  */
/* definitions (1 sign bit, 5 exponent bits with bias 15, 10 fraction   */
/* bits; bfloat16: 8 exponent bits with bias 127, 7 fraction bits).     */
/* ------------------------------------------------------------------ */

double tqo_f16_to_f64(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int f = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);              /* subnormal: f * 2^-24 */
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + f), e - 25);  /* (1 + f/1024) * 2^(e-15) */
    return sign ? -v : v;
}

/* Round a double to the nearest binary16 value, ties to even. */
uint16_t tqo_f64_to_f16(double x)
{
    uint16_t sign = 0;
    if (x != x) return 0x7e00;
    if (signbit(x)) { sign = 0x8000; x = -x; }
    if (x == 0.0) return sign;
    int e2;
    frexp(x, &e2);                 /* x = m * 2^e2, m in [0.5, 1) */
    int exp_unb = e2 - 1;          /* x = 1.xxx * 2^exp_unb */
    int ulp_exp = exp_unb - 10;    /* spacing of binary16 values at x */
    if (ulp_exp < -24) ulp_exp = -24;   /* subnormal range: spacing 2^-24 */
    double q = nearbyint(ldexp(x, -ulp_exp));   /* ties to even (default mode) */
    double v = ldexp(q, ulp_exp);
    if (v > 65504.0) return sign | 0x7c00;   /* overflow -> inf */
    if (v < ldexp(1.0, -14)) {
        /* subnormal (or rounded up to the smallest normal) */
        int f = (int)ldexp(v, 24);     /* v = f * 2^-24, f < 1024 */
        return sign | (uint16_t)f;
    }
    int e;
    double m = frexp(v, &e);       /* v = m * 2^e */
    int biased = e - 1 + 15;
    int frac = (int)ldexp(m * 2.0 - 1.0, 10);
    return sign | (uint16_t)(biased << 10) | (uint16_t)frac;
}

/* Round a float to the nearest bfloat16 value, ties to even. */
uint16_t tqo_f32_to_bf16(float x)
{
    double d = x;
    uint16_t sign = 0;
    if (x != x) return 0x7fc0;
    if (signbit(d)) { sign = 0x8000; d = -d; }
    if (d == 0.0) return sign;
    if (isinf(d)) return sign | 0x7f80;
    int e2;
    frexp(d, &e2);
    int ulp_exp = (e2 - 1) - 7;
    if (ulp_exp < -133) ulp_exp = -133;          /* bf16 subnormal spacing */
    double q = nearbyint(ldexp(d, -ulp_exp));
    double v = ldexp(q, ulp_exp);
    if (v >= ldexp(1.0, 128)) return sign | 0x7f80;
    /* v is exactly representable in float and in bf16: take the top half */
    float vf = (float)v;
    uint32_t bits;
    memcpy(&bits, &vf, 4);
    return sign | (uint16_t)((bits >> 16) & 0x7fff);
}

/* ------------------------------------------------------------------ */
/* Symmetric 4-bit quantizer of one group (Sec. 2, Eq. 1, q_max = 7).   */
/* v[i * stride], i < len, are binary16 bit patterns.                   */
/* ------------------------------------------------------------------ */
static void q4_group(const uint16_t *v, int64_t stride, int len,
                     int8_t *q, int64_t qstride, uint16_t *scale)
{
    double amax = 0.0;
    for (int i = 0; i < len; i++) {
        double a = fabs(tqo_f16_to_f64(v[i * stride]));
        if (a > amax) amax = a;
    }
    /* s = max|v| / q_max, computed in fp32 then stored as fp16 */
    float s32 = (float)amax / 7.0f;
    uint16_t s16 = tqo_f64_to_f16((double)s32);
    *scale = s16;
    float s = (float)tqo_f16_to_f64(s16);
    for (int i = 0; i < len; i++) {
        int code = 0;
        if (s != 0.0f) {
            float r = (float)tqo_f16_to_f64(v[i * stride]) / s;
            double rr = nearbyint((double)r);      /* round half to even */
            if (rr > 7.0) rr = 7.0;
            if (rr < -7.0) rr = -7.0;
            code = (int)rr;
        }
        q[i * qstride] = (int8_t)code;
    }
}

/*
 * Quantize n_vec vectors of length len, group size `group` along each
 * vector.  Element i of vector j sits at v[j * vec_stride + i * elem_stride];
 * its code goes to the same offset in q; the scale of group g of vector j
 * goes to s[j * (len / group) + g].  Returns 0, or -1 on bad arguments.
 */
int tqo_quantize(const uint16_t *v, int64_t n_vec, int64_t len,
                 int64_t vec_stride, int64_t elem_stride, int group,
                 int8_t *q, uint16_t *s)
{
    if (group <= 0 || len % group != 0 || n_vec < 0) return -1;
    int64_t ng = len / group;
    #pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < n_vec; j++)
        for (int64_t g = 0; g < ng; g++) {
            int64_t off = j * vec_stride + g * group * elem_stride;
            q4_group(v + off, elem_stride, group, q + off, elem_stride, &s[j * ng + g]);
        }
    return 0;
}

/* malloc that never returns NULL for an empty request */
static void *xalloc(size_t n) { return malloc(n ? n : 1); }

/* ------------------------------------------------------------------ */
/* The layer (steps O1-O7) for a chosen subset of tokens and outputs.   */
/* ------------------------------------------------------------------ */
/*
 * Inputs (binary16 bit patterns, row-major):
 *   X [M,K], W_res [N,K], L1 [K,r], L2 [r,N]; r may be 0 (L1, L2 unused).
 * rows[nr] / cols[nc] select the tokens and output channels to compute
 * (NULL selects all, in order).  Outputs, all row-major over the selection:
 *   H [nr, r] fp32, sH [nr, r/Gr] fp32, qH [nr, r] int8,
 *   Y32 [nr, nc] fp32, Y64 [nr, nc] fp64, Y16 [nr, nc] fp16 bits,
 *   Ybf [nr, nc] bf16 bits.   Any output pointer may be NULL.
 * Returns 0, or a negative value on bad arguments / allocation failure.
 */
int tqo_layer(int M, int N, int K, int r, int G,
              const uint16_t *X, const uint16_t *Wres,
              const uint16_t *L1, const uint16_t *L2,
              const int32_t *rows, int nr, const int32_t *cols, int nc,
              float *H, float *sH, int8_t *qH,
              float *Y32, double *Y64, uint16_t *Y16, uint16_t *Ybf)
{
    if (M < 0 || N <= 0 || K <= 0 || r < 0 || G <= 0 || K % G != 0) return -1;
    int Gr = r > 0 ? (r < G ? r : G) : 1;
    if (r > 0 && r % Gr != 0) return -1;
    if (rows == NULL) nr = M;
    if (cols == NULL) nc = N;
    const int KG = K / G, RG = r > 0 ? r / Gr : 0;

    int8_t *qx = xalloc((size_t)nr * K);
    uint16_t *sx = xalloc((size_t)nr * KG * 2);
    int8_t *qw = xalloc((size_t)nc * K);
    uint16_t *sw = xalloc((size_t)nc * KG * 2);
    int8_t *ql1 = r ? xalloc((size_t)K * r) : NULL;
    uint16_t *sl1 = r ? xalloc((size_t)KG * r * 2) : NULL;
    int8_t *ql2 = r ? xalloc((size_t)r * nc) : NULL;
    uint16_t *sl2 = r ? xalloc((size_t)RG * nc * 2) : NULL;
    float *h = r ? xalloc((size_t)nr * r * 4) : NULL;
    float *sh = r ? xalloc((size_t)nr * RG * 4) : NULL;
    int8_t *qh = r ? xalloc((size_t)nr * r) : NULL;
    int rc = 0;
    if (!qx || !sx || !qw || !sw || (r && (!ql1 || !sl1 || !ql2 || !sl2 || !h || !sh || !qh))) {
        rc = -2;
        goto done;
    }

    /* O1: activation codes, per token along K */
    for (int i = 0; i < nr; i++) {
        int m = rows ? rows[i] : i;
        if (m < 0 || m >= M) { rc = -1; goto done; }
        tqo_quantize(X + (int64_t)m * K, 1, K, K, 1, G, qx + (int64_t)i * K, sx + (int64_t)i * KG);
    }
    /* O2: weight codes */
    for (int c = 0; c < nc; c++) {
        int n = cols ? cols[c] : c;
        if (n < 0 || n >= N) { rc = -1; goto done; }
        tqo_quantize(Wres + (int64_t)n * K, 1, K, K, 1, G, qw + (int64_t)c * K, sw + (int64_t)c * KG);
    }
    if (r) {
        /* L1 [K, r]: vector j is column j, elements along K (stride r) */
        tqo_quantize(L1, r, K, 1, r, G, ql1, sl1);   /* codes in [K, r]; scales [r, KG] */
        /* L2 [r, N]: vector n is column n, elements along r (stride N);
           gather the selected columns into a [r, nc] copy first */
        uint16_t *l2sel = xalloc((size_t)r * nc * 2);
        if (!l2sel) { rc = -2; goto done; }
        for (int j = 0; j < r; j++)
            for (int c = 0; c < nc; c++) {
                int n = cols ? cols[c] : c;
                l2sel[(int64_t)j * nc + c] = L2[(int64_t)j * N + n];
            }
        tqo_quantize(l2sel, nc, r, 1, nc, Gr, ql2, sl2);   /* scales [nc, RG] */
        free(l2sel);

        /* O4: stage 1, H[m, j] = sum over groups, ascending, of
           fma(A_g, s_x * s_L1, h) with A_g the exact integer dot product */
        #pragma omp parallel for schedule(static)
        for (int i = 0; i < nr; i++)
            for (int j = 0; j < r; j++) {
                float acc = 0.0f;
                for (int g = 0; g < KG; g++) {
                    int32_t a = 0;
                    for (int k = g * G; k < (g + 1) * G; k++)
                        a += (int32_t)qx[(int64_t)i * K + k] * (int32_t)ql1[(int64_t)k * r + j];
                    float sxf = (float)tqo_f16_to_f64(sx[(int64_t)i * KG + g]);
                    float slf = (float)tqo_f16_to_f64(sl1[(int64_t)j * KG + g]);
                    acc = fmaf((float)a, sxf * slf, acc);
                }
                h[(int64_t)i * r + j] = acc;
            }
        /* O5: re-quantize H per token and r-group; s_H stays fp32 */
        for (int i = 0; i < nr; i++)
            for (int hg = 0; hg < RG; hg++) {
                float amax = 0.0f;
                for (int j = hg * Gr; j < (hg + 1) * Gr; j++) {
                    float a = fabsf(h[(int64_t)i * r + j]);
                    if (a > amax) amax = a;
                }
                float s = amax / 7.0f;
                sh[(int64_t)i * RG + hg] = s;
                for (int j = hg * Gr; j < (hg + 1) * Gr; j++) {
                    int code = 0;
                    if (s != 0.0f) {
                        float t = h[(int64_t)i * r + j] / s;
                        double rr = nearbyint((double)t);
                        if (rr > 7.0) rr = 7.0;
                        if (rr < -7.0) rr = -7.0;
                        code = (int)rr;
                    }
                    qh[(int64_t)i * r + j] = (int8_t)code;
                }
            }
    }

    /* O3, O6, O7 */
    #pragma omp parallel for schedule(static)
    for (int i = 0; i < nr; i++)
        for (int c = 0; c < nc; c++) {
            float yres = 0.0f, ylr = 0.0f;
            double y64 = 0.0;
            for (int g = 0; g < KG; g++) {
                int32_t acc = 0;
                for (int k = g * G; k < (g + 1) * G; k++)
                    acc += (int32_t)qx[(int64_t)i * K + k] * (int32_t)qw[(int64_t)c * K + k];
                float sxf = (float)tqo_f16_to_f64(sx[(int64_t)i * KG + g]);
                float swf = (float)tqo_f16_to_f64(sw[(int64_t)c * KG + g]);
                yres = fmaf((float)acc, sxf * swf, yres);
                y64 += (double)acc * (double)sxf * (double)swf;
            }
            for (int hg = 0; hg < RG; hg++) {
                int32_t acc = 0;
                for (int j = hg * Gr; j < (hg + 1) * Gr; j++)
                    acc += (int32_t)qh[(int64_t)i * r + j] * (int32_t)ql2[(int64_t)j * nc + c];
                float shf = sh[(int64_t)i * RG + hg];
                float s2f = (float)tqo_f16_to_f64(sl2[(int64_t)c * RG + hg]);
                ylr = fmaf((float)acc, shf * s2f, ylr);
                y64 += (double)acc * (double)shf * (double)s2f;
            }
            float y = yres + ylr;
            int64_t o = (int64_t)i * nc + c;
            if (Y32) Y32[o] = y;
            if (Y64) Y64[o] = y64;
            if (Y16) Y16[o] = tqo_f64_to_f16((double)y);
            if (Ybf) Ybf[o] = tqo_f32_to_bf16(y);
        }

    if (r) {
        if (H) memcpy(H, h, (size_t)nr * r * 4);
        if (sH) memcpy(sH, sh, (size_t)nr * RG * 4);
        if (qH) memcpy(qH, qh, (size_t)nr * r);
    }
done:
    free(qx); free(sx); free(qw); free(sw);
    free(ql1); free(sl1); free(ql2); free(sl2);
    free(h); free(sh); free(qh);
    return rc;
}
