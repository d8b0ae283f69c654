/*
 * amsim_oracle.c -- plain, slow CPU oracle for the approximate-multiplier hot path of
 * ApproxTrain (arXiv 2209.04161).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library calls, links or includes this
 * file; only the test-suite, the smoke check and the benchmark's CPU-baseline leg use it.
 * It shares no code, header or table with the HIP path.
 *
 * What it computes, and where the paper defines it:
 *   - Functional multiplier models (the "approx_mul" C function a designer supplies, Sec. "AM
 *     Simulation"): Mitchell's logarithmic multiplier (the paper's MIT16, cited, defined here
 *     from Mitchell's log2(1+x) ~= x approximation) and the exact multiplier of operands
 *     truncated to M mantissa bits (bfloat16 truncation when M = 7, Sec. "Experiment Setup",
 *     Datatype paragraph: conversion between (1,8,m) formats is bit truncation).
 *     Both are evaluated in double precision from their mathematical definitions.
 *   - orc_mul: the approximate product as AMSim defines it (Algorithm 2): sign XOR, exponent
 *     sum, zero when either operand has a zero exponent field or the un-normalised exponent
 *     is <= 0, infinity when it is >= 255, otherwise the model's product.  The model is
 *     called directly on the operands; no lookup table is involved.
 *   - orc_lut: the mantissa-product table of Algorithm 1, built by calling the model.
 *   - GEMM and 2-D convolution (forward, backward-data, backward-weight) written as their
 *     direct summation definitions (Sec. "AMCONV2D" / "AMDENSE": every multiply of the
 *     layer is replaced by the approximate product), accumulated in double from -0.0 in
 *     plain loop order, with the per-output sum of |products| returned beside each result.
 *
 * Readings of the paper taken where it is silent or garbled (the same list is kept with the
 * design notes):
 *   R1 Algorithm 1's loops run over [0, 2^M) (a table of 2^(2M) entries).
 *   R2 The M table-index bits are the top M bits of the 23-bit mantissa field.
 *   R3 Zero / denormal operands give a zero product carrying the XOR sign (denormals are read
 *      as zero, as Algorithm 2's exponent-field test does).
 *   R4 Overflow gives infinity carrying the XOR sign; the zero test on the un-normalised
 *      exponent happens before the carry is added, as Algorithm 2 orders it; a carry that
 *      lifts the exponent to 255 gives infinity.
 *   R5 NaN operands give NaN; infinity times a zero/denormal operand gives NaN; infinity
 *      times any other operand gives a signed infinity (IEEE 754 behaviour; Algorithm 2
 *      does not treat these inputs).
 *   R6 The first operand of every product supplies the table's high index: forward
 *      amul(x, w), backward-data amul(dy, w), backward-weight amul(x, dy), GEMM amul(A, B).
 *
 *   R11 Padding and dilation zeros are operands: Algorithm 3 and 4 build their column matrices
 *       (IM2COL with the zero border; the error padded and dilated by the strides for the
 *       preceding-layer gradient) and multiply every element, zeros included, so every tap of the
 *       kernel window contributes amul(+0, weight) where the column matrix holds a zero -- a
 *       signed zero for a finite weight, NaN for an Inf or NaN one.
 *   R16 A (1, e, m) format with e < 8: orc_cast maps each operand into its range (see there), and
 *       Algorithm 2 runs with the format's bias and top exponent field (orc_mul_fmt).
 *   R17 The native multiply: IEEE FP32 products with denormals read and written as zero
 *       (orc_mul_native).
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fPIC -shared (no fast-math).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum {
    ORC_MODEL_MITCHELL = 0,    /* Mitchell logarithmic multiplier on M-bit truncated operands */
    ORC_MODEL_EXACT_TRUNC = 1, /* exact product of M-bit truncated operands (bfloat16 at M=7) */
    ORC_MODEL_ASYM = 2         /* test model: A truncated to M bits, B to M-1 bits, exact product */
};

/* |x| = 2^e * (1 + f), f in [0, 1), for a finite normal float x. */
static void orc_split(float x, int *e, double *f)
{
    int ex;
    double m = frexp(fabs((double)x), &ex); /* m in [0.5, 1) */
    *e = ex - 1;
    *f = 2.0 * m - 1.0;
}

/* Keep the leading `bits` bits of the fraction f in [0,1) (truncation toward zero). */
static double orc_trunc_frac(double f, int bits)
{
    double scale = ldexp(1.0, bits);
    return floor(f * scale) / scale;
}

/* Mitchell's logarithm: log2(2^e * (1 + f)) ~= e + f. */
static double orc_mitchell_log(int e, double f) { return (double)e + f; }

/* Mitchell's antilogarithm: 2^L ~= 2^floor(L) * (1 + (L - floor(L))). */
static double orc_mitchell_antilog(double L)
{
    double c = floor(L);
    return ldexp(1.0 + (L - c), (int)c);
}

/*
 * The functional models, for positive finite normal operands.  Returns the magnitude of the
 * product in double (exact: every result has at most 24 significant bits when M <= 11).
 */
static double orc_model_mag(int model, int m_bits, float a, float b)
{
    int ea, eb;
    double fa, fb;
    orc_split(a, &ea, &fa);
    orc_split(b, &eb, &fb);
    switch (model) {
    case ORC_MODEL_MITCHELL: {
        double x = orc_trunc_frac(fa, m_bits);
        double y = orc_trunc_frac(fb, m_bits);
        return orc_mitchell_antilog(orc_mitchell_log(ea, x) + orc_mitchell_log(eb, y));
    }
    case ORC_MODEL_EXACT_TRUNC: {
        double x = orc_trunc_frac(fa, m_bits);
        double y = orc_trunc_frac(fb, m_bits);
        return ldexp((1.0 + x) * (1.0 + y), ea + eb);
    }
    case ORC_MODEL_ASYM: {
        double x = orc_trunc_frac(fa, m_bits);
        double y = orc_trunc_frac(fb, m_bits - 1);
        return ldexp((1.0 + x) * (1.0 + y), ea + eb);
    }
    default:
        return NAN;
    }
}

/* The model as a designer's C function would expose it: float in, float out (R4 overflow). */
float orc_model(int model, int m_bits, float a, float b)
{
    double mag = orc_model_mag(model, m_bits, fabsf(a), fabsf(b));
    float r = (mag >= ldexp(1.0, 128)) ? INFINITY : (float)mag;
    return (signbit(a) != signbit(b)) ? -r : r;
}

static int orc_is_zero_field(float x) /* exponent field == 0: zero or denormal (R3) */
{
    int c = fpclassify(x);
    return c == FP_ZERO || c == FP_SUBNORMAL;
}

/* Biased exponent field of a finite normal float. */
static int orc_biased_exp(float x) { return ilogbf(x) + 127; }

/* Approximate product with AMSim's special-value policy (Algorithm 2 with readings R3-R5). */
float orc_mul(int model, int m_bits, float a, float b)
{
    int neg = signbit(a) != signbit(b);
    if (isnan(a) || isnan(b))
        return NAN;
    int za = orc_is_zero_field(a), zb = orc_is_zero_field(b);
    int ia = isinf(a) != 0, ib = isinf(b) != 0;
    if ((ia && zb) || (za && ib))
        return NAN;
    if (ia || ib)
        return neg ? -INFINITY : INFINITY;
    if (za || zb)
        return neg ? -0.0f : 0.0f;
    int un_normalized_exp = orc_biased_exp(a) + orc_biased_exp(b) - 127;
    if (un_normalized_exp <= 0)
        return neg ? -0.0f : 0.0f;
    if (un_normalized_exp >= 255)
        return neg ? -INFINITY : INFINITY;
    return orc_model(model, m_bits, a, b);
}

/* ---------------------------------------------------------------- other multipliers ------ */

/*
 * The native FP32 multiply (the paper's runs "with native multiply"): the IEEE product rounded to
 * nearest-even, with denormal operands read as zero and a denormal result flushed to a signed
 * zero, as the GPU's FP32 arithmetic does with denormals off.  (double)a * (double)b is exact for
 * float operands, so one rounding to float gives the IEEE result; values from the largest float
 * plus half an ulp on round to infinity.
 */
float orc_mul_native(float a, float b)
{
    if (orc_is_zero_field(a))
        a = signbit(a) ? -0.0f : 0.0f;
    if (orc_is_zero_field(b))
        b = signbit(b) ? -0.0f : 0.0f;
    double d = (double)a * (double)b;
    if (isnan(d))
        return NAN;
    if (fabs(d) >= 0x1.ffffffp127)
        return (d < 0) ? -INFINITY : INFINITY;
    float r = (float)d;
    if (r != 0.0f && fabsf(r) < 0x1p-126f)
        r = signbit(r) ? -0.0f : 0.0f;
    return r;
}

/*
 * The exponent-casting function of a (1, e, m) format (Sec. "AMSim": e can range up to 8 given a
 * casting function), reading taken here: bias beta = 2^(e-1) - 1, normal unbiased exponents
 * 1 - beta .. beta (the top field reserved for Inf/NaN, as in FP32); a finite value above that
 * range becomes a signed Inf, or with `sat` the largest finite value (2 - 2^-m) * 2^beta; a value
 * below it (the format's denormals included) a signed zero; NaN, Inf and in-range values stay as
 * they are (their mantissa is read through its top m bits by the multiplier).
 */
float orc_cast(int e_bits, int sat, int m_bits, float x)
{
    if (isnan(x) || isinf(x))
        return x;
    int neg = signbit(x) != 0;
    if (orc_is_zero_field(x))
        return neg ? -0.0f : 0.0f;
    int beta = (1 << (e_bits - 1)) - 1;
    int u = ilogbf(x);
    if (u > beta) {
        float big = sat ? (float)ldexp(2.0 - ldexp(1.0, -m_bits), beta) : INFINITY;
        return neg ? -big : big;
    }
    if (u < 1 - beta)
        return neg ? -0.0f : 0.0f;
    return x;
}

/*
 * Algorithm 2 for a (1, e, m) multiplier: both operands cast to the format, then the zero and
 * infinity rules in the format's constants -- with Ea', Eb' the operands' e-bit exponent fields
 * (unbiased exponent + beta), the un-normalised exponent Ea' + Eb' - beta <= 0 gives a signed zero
 * (before the carry, as Algorithm 2 orders it), >= 2^e - 1 a signed infinity, and so does a carry
 * that lifts it to 2^e - 1; otherwise the model's product, an FP32 value.  e = 8 is Algorithm 2
 * itself (orc_mul).
 */
float orc_mul_fmt(int model, int m_bits, int e_bits, int sat, float a, float b)
{
    if (e_bits == 8)
        return orc_mul(model, m_bits, a, b);
    float ca = orc_cast(e_bits, sat, m_bits, a), cb = orc_cast(e_bits, sat, m_bits, b);
    int neg = signbit(ca) != signbit(cb);
    if (isnan(ca) || isnan(cb))
        return NAN;
    int za = orc_is_zero_field(ca), zb = orc_is_zero_field(cb);
    int ia = isinf(ca) != 0, ib = isinf(cb) != 0;
    if ((ia && zb) || (za && ib))
        return NAN;
    if (ia || ib)
        return neg ? -INFINITY : INFINITY;
    if (za || zb)
        return neg ? -0.0f : 0.0f;
    int beta = (1 << (e_bits - 1)) - 1, top = (1 << e_bits) - 1;
    int ua = ilogbf(ca), ub = ilogbf(cb);
    int un_normalized_exp = (ua + beta) + (ub + beta) - beta;
    if (un_normalized_exp <= 0)
        return neg ? -0.0f : 0.0f;
    if (un_normalized_exp >= top)
        return neg ? -INFINITY : INFINITY;
    float c = orc_model(model, m_bits, ca, cb);
    int carry = ilogbf(c) - (ua + ub);
    if (un_normalized_exp + carry >= top)
        return neg ? -INFINITY : INFINITY;
    return c;
}

/* The multiplier of one call: the table's model through Algorithm 2 in a (1, e, m) format, or the
 * native multiply. */
typedef struct {
    int model, m_bits, e_bits, sat, native;
} orc_opts;

static float orc_product(const orc_opts *o, float a, float b)
{
    if (o->native)
        return orc_mul_native(a, b);
    return orc_mul_fmt(o->model, o->m_bits, o->e_bits, o->sat, a, b);
}

void orc_mul_array(int model, int m_bits, int64_t n, const float *a, const float *b, float *c)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        c[i] = orc_mul(model, m_bits, a[i], b[i]);
}

void orc_mul_ex_array(const orc_opts *o, int64_t n, const float *a, const float *b, float *c)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        c[i] = orc_product(o, a[i], b[i]);
}

void orc_cast_array(int e_bits, int sat, int m_bits, int64_t n, const float *x, float *y)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        y[i] = orc_cast(e_bits, sat, m_bits, x[i]);
}

/*
 * Algorithm 1: the mantissa-product table.  A and B get sign 0 and exponent field 127
 * (any legal choice, R1/R2), mantissa fields k and j placed in the top M bits; the carry is
 * set when the model's exponent exceeds the un-normalised exponent.  Returns 0, or -1 when
 * the model's exponent is neither the un-normalised exponent nor one more (the table cannot
 * represent such a model).
 */
int orc_lut(int model, int m_bits, uint32_t *out)
{
    uint32_t n = 1u << m_bits;
    for (uint32_t k = 0; k < n; ++k) {
        for (uint32_t j = 0; j < n; ++j) {
            /* A = 1.k (binary), B = 1.j, as values */
            float A = (float)(1.0 + ldexp((double)k, -m_bits));
            float B = (float)(1.0 + ldexp((double)j, -m_bits));
            float C = orc_model(model, m_bits, A, B);
            int un_normalized_exp = 127 + 127 - 127;
            int exp_c = orc_biased_exp(C);
            uint32_t carry;
            if (exp_c == un_normalized_exp)
                carry = 0;
            else if (exp_c == un_normalized_exp + 1)
                carry = 1;
            else
                return -1;
            /* mantissa field of C: fraction bits of C / 2^(exp_c - 127), 23 bits */
            double frac = ldexp((double)C, -(exp_c - 127)) - 1.0;
            uint32_t mant = (uint32_t)ldexp(frac, 23);
            out[k * n + j] = (carry << 23) | mant;
        }
    }
    return 0;
}

/* ---------------------------------------------------------------- GEMM ------------------- */

/* C = op(A) * op(B), row-major, product amul(A_ik, B_kj) (R6). */
static float orc_gemm_one(const orc_opts *o, int transa, int transb, int64_t K, const float *A,
                          int64_t lda, const float *B, int64_t ldb, int64_t i, int64_t j, double *sabs)
{
    double acc = -0.0, s = 0.0;
    for (int64_t k = 0; k < K; ++k) {
        float a = transa ? A[k * lda + i] : A[i * lda + k];
        float b = transb ? B[j * ldb + k] : B[k * ldb + j];
        float p = orc_product(o, a, b);
        acc += (double)p;
        s += fabs((double)p);
    }
    *sabs = s;
    return (float)acc;
}

/*
 * If idx is NULL, computes all M*N outputs into C[i*N + j]; otherwise computes the outputs at
 * the flat indices idx[t] = i*N + j into C[t].  S receives the matching sums of |products|.
 */
void orc_gemm_ex(const orc_opts *o, int transa, int transb, int64_t M, int64_t N, int64_t K, const float *A,
                 int64_t lda, const float *B, int64_t ldb, const int64_t *idx, int64_t nidx, float *C, double *S)
{
    int64_t total = idx ? nidx : M * N;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < total; ++t) {
        int64_t flat = idx ? idx[t] : t;
        int64_t i = flat / N, j = flat % N;
        C[t] = orc_gemm_one(o, transa, transb, K, A, lda, B, ldb, i, j, &S[t]);
    }
}

void orc_gemm(int model, int m_bits, int transa, int transb, int64_t M, int64_t N, int64_t K, const float *A,
              int64_t lda, const float *B, int64_t ldb, const int64_t *idx, int64_t nidx, float *C, double *S)
{
    orc_opts o = {model, m_bits, 8, 0, 0};
    orc_gemm_ex(&o, transa, transb, M, N, K, A, lda, B, ldb, idx, nidx, C, S);
}

/* ---------------------------------------------------------------- convolution ----------- */

/* NHWC activations, HWIO weights, explicit four-sided zero padding, no dilation/groups. */
typedef struct {
    int n, h, w, c_in, c_out, kh, kw, stride_h, stride_w, pad_top, pad_bottom, pad_left, pad_right;
} orc_conv;

static int64_t orc_out_h(const orc_conv *p) { return (p->h + p->pad_top + p->pad_bottom - p->kh) / p->stride_h + 1; }
static int64_t orc_out_w(const orc_conv *p) { return (p->w + p->pad_left + p->pad_right - p->kw) / p->stride_w + 1; }

/* y[n,oh,ow,co] = sum_{kh,kw,ci} amul(xpad[n, oh*S+kh-Pt, ow*S+kw-Pl, ci], w[kh,kw,ci,co]), xpad = x with
 * its zero border (R11) */
static float orc_fwd_one(const orc_opts *o, const orc_conv *p, const float *x, const float *w, int64_t flat,
                         double *sabs)
{
    int64_t OH = orc_out_h(p), OW = orc_out_w(p);
    int64_t co = flat % p->c_out;
    int64_t ow = (flat / p->c_out) % OW;
    int64_t oh = (flat / p->c_out / OW) % OH;
    int64_t n = flat / p->c_out / OW / OH;
    double acc = -0.0, s = 0.0;
    for (int64_t kh = 0; kh < p->kh; ++kh) {
        for (int64_t kw = 0; kw < p->kw; ++kw) {
            int64_t ih = oh * p->stride_h + kh - p->pad_top;
            int64_t iw = ow * p->stride_w + kw - p->pad_left;
            int inside = ih >= 0 && ih < p->h && iw >= 0 && iw < p->w;
            for (int64_t ci = 0; ci < p->c_in; ++ci) {
                /* a padded tap multiplies the zero the column matrix holds there (R11) */
                float a = inside ? x[((n * p->h + ih) * p->w + iw) * p->c_in + ci] : 0.0f;
                float b = w[((kh * p->kw + kw) * p->c_in + ci) * p->c_out + co];
                float q = orc_product(o, a, b);
                acc += (double)q;
                s += fabs((double)q);
            }
        }
    }
    *sabs = s;
    return (float)acc;
}

/* dx[n,h,w,ci] = sum over every (kh,kw,co) of amul(E[n, h+Pt-kh, w+Pl-kw, co], w[kh,kw,ci,co]), E the
 * error dilated by the strides and zero-padded (Algorithm 4's PaddedDilatedErrors, R11):
 * E[n,p,q,co] = dy[n,p/Sh,q/Sw,co] where p, q are multiples of the strides and p/Sh < OH, q/Sw < OW
 * (the output positions that read (h,w) in the forward pass), +0 elsewhere. */
static float orc_bwd_data_one(const orc_opts *o, const orc_conv *p, const float *dy, const float *w,
                              int64_t flat, double *sabs)
{
    int64_t OH = orc_out_h(p), OW = orc_out_w(p);
    int64_t ci = flat % p->c_in;
    int64_t iw = (flat / p->c_in) % p->w;
    int64_t ih = (flat / p->c_in / p->w) % p->h;
    int64_t n = flat / p->c_in / p->w / p->h;
    double acc = -0.0, s = 0.0;
    for (int64_t kh = 0; kh < p->kh; ++kh) {
        for (int64_t kw = 0; kw < p->kw; ++kw) {
            int64_t ph = ih + p->pad_top - kh, pw = iw + p->pad_left - kw;
            int64_t oh = ph >= 0 ? ph / p->stride_h : -1, ow = pw >= 0 ? pw / p->stride_w : -1;
            int real = ph >= 0 && pw >= 0 && ph % p->stride_h == 0 && pw % p->stride_w == 0 && oh < OH && ow < OW;
            for (int64_t co = 0; co < p->c_out; ++co) {
                float a = real ? dy[((n * OH + oh) * OW + ow) * p->c_out + co] : 0.0f;
                float b = w[((kh * p->kw + kw) * p->c_in + ci) * p->c_out + co];
                float q = orc_product(o, a, b);
                acc += (double)q;
                s += fabs((double)q);
            }
        }
    }
    *sabs = s;
    return (float)acc;
}

/* dw[kh,kw,ci,co] = sum over every (n,oh,ow) of amul(xpad[n, oh*S+kh-Pt, ow*S+kw-Pl, ci], dy[n,oh,ow,co]),
 * xpad = x with its zero border (R11) */
static float orc_bwd_weight_one(const orc_opts *o, const orc_conv *p, const float *x, const float *dy,
                                int64_t flat, double *sabs)
{
    int64_t OH = orc_out_h(p), OW = orc_out_w(p);
    int64_t co = flat % p->c_out;
    int64_t ci = (flat / p->c_out) % p->c_in;
    int64_t kw = (flat / p->c_out / p->c_in) % p->kw;
    int64_t kh = flat / p->c_out / p->c_in / p->kw;
    double acc = -0.0, s = 0.0;
    for (int64_t n = 0; n < p->n; ++n) {
        for (int64_t oh = 0; oh < OH; ++oh) {
            for (int64_t ow = 0; ow < OW; ++ow) {
                int64_t ih = oh * p->stride_h + kh - p->pad_top;
                int64_t iw = ow * p->stride_w + kw - p->pad_left;
                int inside = ih >= 0 && ih < p->h && iw >= 0 && iw < p->w;
                float a = inside ? x[((n * p->h + ih) * p->w + iw) * p->c_in + ci] : 0.0f;
                float b = dy[((n * OH + oh) * OW + ow) * p->c_out + co];
                float q = orc_product(o, a, b);
                acc += (double)q;
                s += fabs((double)q);
            }
        }
    }
    *sabs = s;
    return (float)acc;
}

/* pass: 0 forward (in0 = x, in1 = w, out = y), 1 backward-data (in0 = dy, in1 = w, out = dx),
 * 2 backward-weight (in0 = x, in1 = dy, out = dw).  idx/nidx select output elements by flat
 * index as in orc_gemm; NULL computes the whole output tensor. */
int orc_conv2d_ex(const orc_opts *o, int pass, const orc_conv *p, const float *in0, const float *in1,
                  const int64_t *idx, int64_t nidx, float *out, double *S)
{
    int64_t OH = orc_out_h(p), OW = orc_out_w(p);
    int64_t total;
    if (pass == 0)
        total = (int64_t)p->n * OH * OW * p->c_out;
    else if (pass == 1)
        total = (int64_t)p->n * p->h * p->w * p->c_in;
    else if (pass == 2)
        total = (int64_t)p->kh * p->kw * p->c_in * p->c_out;
    else
        return -1;
    if (idx)
        total = nidx;
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t t = 0; t < total; ++t) {
        int64_t flat = idx ? idx[t] : t;
        if (pass == 0)
            out[t] = orc_fwd_one(o, p, in0, in1, flat, &S[t]);
        else if (pass == 1)
            out[t] = orc_bwd_data_one(o, p, in0, in1, flat, &S[t]);
        else
            out[t] = orc_bwd_weight_one(o, p, in0, in1, flat, &S[t]);
    }
    return 0;
}

int orc_conv2d(int model, int m_bits, int pass, const orc_conv *p, const float *in0, const float *in1,
               const int64_t *idx, int64_t nidx, float *out, double *S)
{
    orc_opts o = {model, m_bits, 8, 0, 0};
    return orc_conv2d_ex(&o, pass, p, in0, in1, idx, nidx, out, S);
}

int orc_num_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
