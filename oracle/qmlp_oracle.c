/*
 * qmlp_oracle.c -- plain, slow, fp64 CPU oracle for the W4/W2-GateUp decode MLP.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file; only the test-suite, the smoke check and the benchmark's
 * CPU-baseline leg do.  It shares no code, header, table or helper with the
 * HIP library: everything below is written from the paper and from the
 * format definition (row-major codes, LSB-first packing, interleaved
 * fp16 scale/zero metadata), with plain loops and no blocking or fusion.
 *
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared (no FMA contraction, no
 * fast-math, IEEE fp64 throughout).
 *
 * What the paper fixes and what it leaves open:
 *   - Sec. 3.3 / Sec. 4.1: gate and up projections are quantized to INT2 and
 *     all other linear layers (down included) to INT4, group-wise along the
 *     input dimension.  The paper names bits and group sizes only; the
 *     quantizer itself (round-to-nearest, asymmetric min-max, integer zero
 *     point, fp16 scale and zero) is this library's reading.
 *   - Sec. 3.1, Eq. (1): a LoRA-augmented linear adds alpha * B A X to W X.
 *   - Sec. 4.2 / Sec. 7 step 5: adapters stay a separate module at inference
 *     (not merged into the 2-bit grid).
 *   - Sec. 5: the MLP is one fused gate-activation-down operator whose
 *     intermediate never leaves the chip, so h is not part of the result and
 *     is kept unrounded here.
 *   - Sec. 6.3: quantize-dequantize (QDQ) semantics: the layer computes with
 *     the dequantized weight s * (q - z).
 *   - The paper does not name the activation; SiLU(v) = v / (1 + exp(-v)).
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ */
/* Floating-point conversions (IEEE binary16 / bfloat16 <-> binary64). */
/* ------------------------------------------------------------------ */

/* binary16 bits -> double (exact). */
double orc_f16_to_f64(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1F;
    int m = h & 0x3FF;
    double v;
    if (e == 0x1F)
        v = m ? NAN : INFINITY;
    else if (e == 0)
        v = ldexp((double)m, -24);              /* subnormal: m * 2^-24 */
    else
        v = ldexp((double)(1024 + m), e - 25);  /* (1024+m) * 2^(e-15-10) */
    return sign ? -v : v;
}

/* bfloat16 bits -> double (exact): the upper half of a binary32. */
double orc_bf16_to_f64(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

/*
 * double -> binary16 bits, one rounding, round-to-nearest-even.
 * Written arithmetically: find the binary16 quantum at the value's
 * magnitude, divide by it (exact: a power of two), round the quotient with
 * rint() (default mode = nearest-even), rebuild the encoding.  Never goes
 * through binary32, which would round twice.
 */
uint16_t orc_f64_to_f16(double v)
{
    uint16_t sign = signbit(v) ? 0x8000 : 0;
    double a = fabs(v);
    if (isnan(v))
        return 0x7E00;
    if (isinf(a))
        return sign | 0x7C00;
    if (a == 0.0)
        return sign;
    int e2;
    frexp(a, &e2);                  /* a = f * 2^e2, f in [0.5, 1) */
    int lead = e2 - 1;              /* exponent of the leading bit */
    int qexp = lead >= -14 ? lead - 10 : -24;   /* quantum = 2^qexp */
    double n = rint(ldexp(a, -qexp));            /* integer multiple of quantum */
    double r = ldexp(n, qexp);
    if (r >= 65536.0)
        return sign | 0x7C00;       /* rounds past the largest finite value */
    if (r < ldexp(1.0, -14))
        return sign | (uint16_t)n;  /* subnormal (n <= 1023) or exactly 2^-14 */
    /* normal: r = (1 + frac) * 2^E with E in [-14, 15] */
    int E;
    double fr = frexp(r, &E);       /* fr in [0.5,1): r = fr*2^E */
    E -= 1;
    int mant = (int)(ldexp(fr, 11) - 1024.0);    /* 10-bit fraction */
    return sign | (uint16_t)((E + 15) << 10) | (uint16_t)mant;
}

/* ------------------------------------------------------------------ */
/* Group-wise round-to-nearest min-max quantizer (Sec. 3.3, Sec. 4.1).  */
/* ------------------------------------------------------------------ */

/*
 * Quantize W [n][k] (row-major fp32) to b-bit codes with one (scale, zero)
 * per group of g consecutive inputs of a row.  For each group:
 *   lo = min(0, min w), hi = max(0, max w)        (0 kept on the grid)
 *   s  = (hi - lo) / (2^b - 1)                    (fp64)
 *   s16 = RNE_fp16(s); s16 == 0 -> 1.0            (degenerate range)
 *   z  = clamp(rint(-lo / s16), 0, qmax)          (integer zero point)
 *   q  = clamp(rint(w / s16) + z, 0, qmax)
 * A group holding a non-finite weight, or whose scale overflows binary16,
 * is invalid: its codes are 0, its scale is the binary16 NaN 0x7E00 and its
 * zero 0.  Returns the number of invalid groups.
 * codes: uint8 [n][k]; scale, zero: binary16 bits [n][k/g].
 */
long orc_quantize(const float *W, long n, long k, long g, int bits,
                  uint8_t *codes, uint16_t *scale, uint16_t *zero)
{
    const int qmax = (1 << bits) - 1;
    const long ng = k / g;
    long bad = 0;
    for (long row = 0; row < n; ++row) {
        for (long j = 0; j < ng; ++j) {
            const float *w = W + row * k + j * g;
            uint8_t *q = codes + row * k + j * g;
            int finite = 1;
            double lo = 0.0, hi = 0.0;
            for (long i = 0; i < g; ++i) {
                double v = (double)w[i];
                if (!isfinite(v))
                    finite = 0;
                else {
                    if (v < lo) lo = v;
                    if (v > hi) hi = v;
                }
            }
            double s = (hi - lo) / (double)qmax;
            uint16_t s16 = orc_f64_to_f16(s);
            if (s16 == 0)
                s16 = 0x3C00;       /* 1.0 */
            if (!finite || s16 == 0x7C00) {
                for (long i = 0; i < g; ++i) q[i] = 0;
                scale[row * ng + j] = 0x7E00;
                zero[row * ng + j] = 0;
                ++bad;
                continue;
            }
            double sd = orc_f16_to_f64(s16);
            double zf = rint(-lo / sd);
            if (zf < 0) zf = 0;
            if (zf > qmax) zf = qmax;
            int z = (int)zf;
            for (long i = 0; i < g; ++i) {
                double t = rint((double)w[i] / sd) + (double)z;
                if (t < 0) t = 0;
                if (t > qmax) t = qmax;
                q[i] = (uint8_t)t;
            }
            scale[row * ng + j] = s16;
            zero[row * ng + j] = orc_f64_to_f16((double)z);
        }
    }
    return bad;
}

/* ------------------------------------------------------------------ */
/* Storage format.                                                      */
/* ------------------------------------------------------------------ */

/*
 * Packed codes: row-major; each row is a run of little-endian 32-bit words,
 * code i of a row sits at bits [b*(i mod 32/b), +b) of word i / (32/b).
 *
 * 3 bits (the W3 variant of Appendix B; the paper fixes no layout): a row is
 * k*3/32 words, first a plane holding the low two bits of every code in the
 * 2-bit layout (k/16 words), then a plane holding the high bit of every code,
 * code i at bit (i mod 32) of word i/32 of that plane (k/32 words).
 */
static void pack3(const uint8_t *codes, long n, long k, uint32_t *words)
{
    const long wpr = k * 3 / 32;
    for (long row = 0; row < n; ++row) {
        uint32_t *lo = words + row * wpr, *hi = lo + k / 16;
        for (long wd = 0; wd < wpr; ++wd)
            lo[wd] = 0;
        for (long i = 0; i < k; ++i) {
            uint32_t c = codes[row * k + i];
            lo[i / 16] += (c % 4) * (uint32_t)(1u << (2 * (i % 16)));
            hi[i / 32] += (c / 4) * (uint32_t)(1u << (i % 32));
        }
    }
}

static void unpack3(const uint32_t *words, long n, long k, uint8_t *codes)
{
    const long wpr = k * 3 / 32;
    for (long row = 0; row < n; ++row) {
        const uint32_t *lo = words + row * wpr, *hi = lo + k / 16;
        for (long i = 0; i < k; ++i) {
            uint32_t l = (lo[i / 16] / (1u << (2 * (i % 16)))) % 4;
            uint32_t h = (hi[i / 32] / (1u << (i % 32))) % 2;
            codes[row * k + i] = (uint8_t)(l + 4 * h);
        }
    }
}

void orc_pack(const uint8_t *codes, long n, long k, int bits, uint32_t *words)
{
    if (bits == 3) {
        pack3(codes, n, k, words);
        return;
    }
    const long per = 32 / bits;
    const long wpr = k / per;       /* words per row */
    for (long row = 0; row < n; ++row)
        for (long wd = 0; wd < wpr; ++wd) {
            uint32_t acc = 0;
            for (long i = 0; i < per; ++i) {
                uint32_t c = codes[row * k + wd * per + i];
                acc += c * (uint32_t)(1u << (bits * i));
            }
            words[row * wpr + wd] = acc;
        }
}

void orc_unpack(const uint32_t *words, long n, long k, int bits, uint8_t *codes)
{
    if (bits == 3) {
        unpack3(words, n, k, codes);
        return;
    }
    const long per = 32 / bits;
    const long wpr = k / per;
    const uint32_t mask = (1u << bits) - 1;
    for (long row = 0; row < n; ++row)
        for (long i = 0; i < k; ++i) {
            uint32_t wv = words[row * wpr + i / per];
            codes[row * k + i] = (uint8_t)((wv / (1u << (bits * (i % per)))) & mask);
        }
}

/* Metadata: per (row, group) two binary16 values, scale then zero. */
void orc_meta_interleave(const uint16_t *scale, const uint16_t *zero,
                         long count, uint16_t *meta)
{
    for (long i = 0; i < count; ++i) {
        meta[2 * i] = scale[i];
        meta[2 * i + 1] = zero[i];
    }
}

/* ------------------------------------------------------------------ */
/* Dequantization (QDQ, Sec. 6.3).                                      */
/* ------------------------------------------------------------------ */

/* w_hat = s16 * (q - z), exact in fp64. */
void orc_dequant(const uint8_t *codes, const uint16_t *scale, const uint16_t *zero,
                 long n, long k, long g, double *w)
{
    const long ng = k / g;
    for (long row = 0; row < n; ++row)
        for (long i = 0; i < k; ++i) {
            double s = orc_f16_to_f64(scale[row * ng + i / g]);
            double z = orc_f16_to_f64(zero[row * ng + i / g]);
            w[row * k + i] = s * ((double)codes[row * k + i] - z);
        }
}

/* The binary16 image of the dequantized weight: one RNE rounding of the
 * exact value; q == z gives +0. */
void orc_dequant_f16(const uint8_t *codes, const uint16_t *scale, const uint16_t *zero,
                     long n, long k, long g, uint16_t *w16)
{
    const long ng = k / g;
    for (long row = 0; row < n; ++row)
        for (long i = 0; i < k; ++i) {
            double s = orc_f16_to_f64(scale[row * ng + i / g]);
            double z = orc_f16_to_f64(zero[row * ng + i / g]);
            double v = s * ((double)codes[row * k + i] - z);
            w16[row * k + i] = orc_f64_to_f16(v + 0.0);   /* -0 -> +0 */
        }
}

/* ------------------------------------------------------------------ */
/* The MLP forward (Sec. 3.1 Eq. (1); Sec. 3.3; Sec. 4.2; Sec. 5).       */
/* ------------------------------------------------------------------ */

static double act_to_f64(uint16_t v, int bf16)
{
    return bf16 ? orc_bf16_to_f64(v) : orc_f16_to_f64(v);
}

/*
 * One quantized linear with an unmerged low-rank correction, Eq. (1):
 *   out[m][o] = sum_i w_hat[o][i] x[m][i] + lora_scale * sum_c Bm[o][c] t[m][c]
 *   t[m][c]   = sum_i Am[c][i] x[m][i]
 * W given by codes/scale/zero [nout][kin]; Am [rank][kin], Bm [nout][rank]
 * in the activation type; x [M][kin] in the activation type (given as f64).
 * rank == 0 drops the correction.
 */
static int lora_linear(const uint8_t *codes, const uint16_t *scale, const uint16_t *zero,
                       long nout, long kin, long g,
                       const uint16_t *Am, const uint16_t *Bm, long rank, double lora_scale,
                       int bf16, const double *x, long M, double *out)
{
    double *t = malloc(sizeof(double) * (size_t)(M * (rank > 0 ? rank : 1)));
    double *wrow = malloc(sizeof(double) * (size_t)kin);
    if (!t || !wrow) {
        free(t); free(wrow);
        return -1;
    }
    /* t = A x (the rank-r projection), Eq. (1) read right to left */
    for (long m = 0; m < M; ++m)
        for (long c = 0; c < rank; ++c) {
            double acc = 0.0;
            for (long i = 0; i < kin; ++i)
                acc += act_to_f64(Am[c * kin + i], bf16) * x[m * kin + i];
            t[m * rank + c] = acc;
        }
    for (long o = 0; o < nout; ++o) {
        /* dequantized row o: s * (q - z) */
        orc_dequant(codes + o * kin, scale + o * (kin / g), zero + o * (kin / g),
                    1, kin, g, wrow);
        for (long m = 0; m < M; ++m) {
            double acc = 0.0;
            for (long i = 0; i < kin; ++i)
                acc += wrow[i] * x[m * kin + i];
            double lr = 0.0;
            for (long c = 0; c < rank; ++c)
                lr += act_to_f64(Bm[o * rank + c], bf16) * t[m * rank + c];
            out[m * nout + o] = acc + lora_scale * lr;
        }
    }
    free(t); free(wrow);
    return 0;
}

/* LoRA-A projection alone: t[m][c] = sum_i A[c][i] x[m][i]. */
void orc_lora_a(const uint16_t *A, const uint16_t *x, long M, long d, long rank,
                int bf16, double *t)
{
    for (long m = 0; m < M; ++m)
        for (long c = 0; c < rank; ++c) {
            double acc = 0.0;
            for (long i = 0; i < d; ++i)
                acc += act_to_f64(A[c * d + i], bf16) * act_to_f64(x[m * d + i], bf16);
            t[m * rank + c] = acc;
        }
}

/*
 * Gate/up half of the block:
 *   G = W2gate x + s_L B_g A_g x,  U = W2up x + s_L B_u A_u x,
 *   h = SiLU(G) * U = G / (1 + exp(-G)) * U.
 * Codes/scale/zero of gate and up are [f][d]; x is [M][d] activation bits;
 * h, G, U are [M][f] in fp64 (never rounded).  G and U may be NULL.
 * Returns 0, or -1 on allocation failure.
 */
int orc_gateup(long M, long d, long f, long g,
               const uint8_t *cg, const uint16_t *sg, const uint16_t *zg,
               const uint8_t *cu, const uint16_t *su, const uint16_t *zu,
               const uint16_t *Ag, const uint16_t *Bg,
               const uint16_t *Au, const uint16_t *Bu,
               long rank, double lora_scale, int bf16,
               const uint16_t *x, double *h, double *G, double *U)
{
    double *xd = malloc(sizeof(double) * (size_t)(M * d));
    double *gv = malloc(sizeof(double) * (size_t)(M * f));
    double *uv = malloc(sizeof(double) * (size_t)(M * f));
    if (!xd || !gv || !uv) {
        free(xd); free(gv); free(uv);
        return -1;
    }
    for (long i = 0; i < M * d; ++i)
        xd[i] = act_to_f64(x[i], bf16);
    if (lora_linear(cg, sg, zg, f, d, g, Ag, Bg, rank, lora_scale, bf16, xd, M, gv) ||
        lora_linear(cu, su, zu, f, d, g, Au, Bu, rank, lora_scale, bf16, xd, M, uv)) {
        free(xd); free(gv); free(uv);
        return -1;
    }
    for (long i = 0; i < M * f; ++i) {
        double a = gv[i];
        h[i] = a / (1.0 + exp(-a)) * uv[i];
        if (G) G[i] = a;
        if (U) U[i] = uv[i];
    }
    free(xd); free(gv); free(uv);
    return 0;
}

/*
 * Down projection on an fp64 intermediate: y[m][o] = sum_n w_hat[o][n] h[m][n].
 * Codes/scale/zero [d][f].
 */
int orc_down(long M, long d, long f, long g,
             const uint8_t *cd, const uint16_t *sd, const uint16_t *zd,
             const double *h, double *y)
{
    return lora_linear(cd, sd, zd, d, f, g, NULL, NULL, 0, 0.0, 0, h, M, y);
}

/*
 * Down projection on an intermediate given in the activation type (bits):
 * checks a down-only kernel on exactly the h it was handed.
 */
int orc_down_act(long M, long d, long f, long g,
                 const uint8_t *cd, const uint16_t *sd, const uint16_t *zd,
                 const uint16_t *h_bits, int bf16, double *y)
{
    double *hd = malloc(sizeof(double) * (size_t)(M * f));
    if (!hd)
        return -1;
    for (long i = 0; i < M * f; ++i)
        hd[i] = act_to_f64(h_bits[i], bf16);
    int rc = orc_down(M, d, f, g, cd, sd, zd, hd, y);
    free(hd);
    return rc;
}

/*
 * Whole block: y = W4down( SiLU(G) * U ), with the intermediate kept in
 * fp64 (Sec. 5: it stays on-chip, so it is not part of the result).
 * h may be NULL; if given it receives the fp64 intermediate [M][f].
 */
int orc_forward(long M, long d, long f, long g_gu, long g_dn,
                const uint8_t *cg, const uint16_t *sg, const uint16_t *zg,
                const uint8_t *cu, const uint16_t *su, const uint16_t *zu,
                const uint8_t *cd, const uint16_t *sd, const uint16_t *zd,
                const uint16_t *Ag, const uint16_t *Bg,
                const uint16_t *Au, const uint16_t *Bu,
                long rank, double lora_scale, int bf16,
                const uint16_t *x, double *y, double *h_out)
{
    double *h = malloc(sizeof(double) * (size_t)(M * f));
    if (!h)
        return -1;
    int rc = orc_gateup(M, d, f, g_gu, cg, sg, zg, cu, su, zu, Ag, Bg, Au, Bu,
                        rank, lora_scale, bf16, x, h, NULL, NULL);
    if (rc == 0)
        rc = orc_down(M, d, f, g_dn, cd, sd, zd, h, y);
    if (rc == 0) {
        if (h_out)
            memcpy(h_out, h, sizeof(double) * (size_t)(M * f));
    }
    free(h);
    return rc;
}

/* ------------------------------------------------------------------ */
/* The decoder context of a stack of blocks.                          */
/* ------------------------------------------------------------------ */

/*
 * Sec. 3.3: every layer of the model carries one gated MLP; in a decoder
 * its input is the normalized residual stream and its output is added back
 * to the stream.  A stack of blocks is modelled with the attention blocks
 * left out:
 *   u = RMSNorm(x) = x / sqrt(mean_i(x_i^2) + eps)     (unit gain, per token)
 *   x_next = x + y,  y = block(u)
 * Both results are rounded once to binary16.  (A learned norm gain folds
 * into the input columns of the block's gate, up and LoRA-A weights before
 * quantization, so the run-time norm has unit gain.)
 */
void orc_rmsnorm_f16(const uint16_t *x, long M, long d, double eps, uint16_t *u)
{
    for (long m = 0; m < M; ++m) {
        double ss = 0.0;
        for (long i = 0; i < d; ++i) {
            double v = orc_f16_to_f64(x[m * d + i]);
            ss += v * v;
        }
        double inv = 1.0 / sqrt(ss / (double)d + eps);
        for (long i = 0; i < d; ++i)
            u[m * d + i] = orc_f64_to_f16(orc_f16_to_f64(x[m * d + i]) * inv);
    }
}

/* x + y of binary16 values, the exact sum rounded once to binary16. */
void orc_residual_f16(const uint16_t *x, const uint16_t *y, long n, uint16_t *out)
{
    for (long i = 0; i < n; ++i)
        out[i] = orc_f64_to_f16(orc_f16_to_f64(x[i]) + orc_f16_to_f64(y[i]));
}
