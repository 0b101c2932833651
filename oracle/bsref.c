/*
 * bsref.c -- CPU oracle for low-precision bitserial operators.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the tests, the smoke check and the
 * benchmark's CPU-baseline leg, never by the product path.  Plain loops, int64
 * accumulation, no blocking or reordering.  Shares nothing with the GPU code.
 *
 * Build: gcc -O2 -std=c11 -fopenmp -fPIC -shared -ffp-contract=off
 *        -fno-fast-math bsref.c -o libbsref.so -lm
 * (-ffp-contract=off and the absence of fast-math keep the quantizer's single
 * binary32 multiply exact; x86-64 evaluates float arithmetic in SSE binary32.)
 */
#include "bsref.h"

#include <math.h>
#include <stddef.h>
#include <limits.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int bsref_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

int bsref_set_threads(int n)
{
    if (n < 1)
        return BSREF_EINVAL;
#ifdef _OPENMP
    omp_set_num_threads(n);
#endif
    return BSREF_OK;
}

static int64_t words_for(int64_t k) { return (k + 31) / 32; }

/* ------------------------------------------------------------------------ */
/* Quantization (Sec. 3.1).  See bsref.h for the reading of the formula.      */
/* ------------------------------------------------------------------------ */
int bsref_quantize(const float *x, uint8_t *q, int64_t n, float scale,
                   int bits, int enc)
{
    if (!x || !q || n < 0 || bits < 1 || bits > 8)
        return BSREF_EINVAL;
    if (!isfinite(scale) || !(scale > 0.0f))
        return BSREF_EINVAL;
    if (enc != BSREF_UNIPOLAR && enc != BSREF_BIPOLAR && enc != BSREF_SIGNED)
        return BSREF_EINVAL;
    if (enc == BSREF_BIPOLAR && bits != 1)
        return BSREF_EINVAL;
    if (enc == BSREF_SIGNED && bits < 2)
        return BSREF_EINVAL;

    const int qmax = (1 << bits) - 1;
    const int smin = -(1 << (bits - 1)), smax = (1 << (bits - 1)) - 1;
    for (int64_t i = 0; i < n; ++i) {
        if (enc == BSREF_BIPOLAR) {
            /* sign of the datum: +1 (bit 1) for x >= 0, -1 (bit 0) otherwise */
            q[i] = (x[i] >= 0.0f) ? 1 : 0;
            continue;
        }
        float product = x[i] * scale;   /* one binary32 multiply */
        float r = rintf(product);       /* ties to even (default mode) */
        if (enc == BSREF_SIGNED) {
            int v;
            if (r != r)                 /* NaN */
                v = 0;
            else if (r <= (float)smin)  /* saturate both ends */
                v = smin;
            else if (r >= (float)smax)
                v = smax;
            else
                v = (int)r;
            q[i] = (uint8_t)((unsigned)v & (unsigned)qmax);  /* two's complement */
            continue;
        }
        uint8_t v;
        if (!(r > 0.0f))                /* negative, zero or NaN */
            v = 0;
        else if (r >= (float)qmax)      /* saturate at the top code */
            v = (uint8_t)qmax;
        else
            v = (uint8_t)r;
        q[i] = v;
    }
    return BSREF_OK;
}

/* ------------------------------------------------------------------------ */
/* Bit packing (Sec. 2.2 and Sec. 3.1): split each element into bit-planes    */
/* and pack each plane's bits along the reduction axis into uint32 words,     */
/* element 32t+u at bit u of word t.  Layout [rows][bits][words] (MBK').      */
/* ------------------------------------------------------------------------ */
int bsref_pack(const uint8_t *q, uint32_t *packed, int64_t rows, int64_t k,
               int bits)
{
    if (!q || !packed || rows < 0 || k < 1 || bits < 1 || bits > 8)
        return BSREF_EINVAL;
    const int64_t kw = words_for(k);
    for (int64_t r = 0; r < rows; ++r) {
        for (int b = 0; b < bits; ++b) {
            for (int64_t t = 0; t < kw; ++t) {
                uint32_t word = 0;
                for (int u = 0; u < 32; ++u) {
                    int64_t e = 32 * t + u;
                    if (e < k) {
                        uint32_t bit = ((uint32_t)q[r * k + e] >> b) & 1u;
                        word |= bit << u;
                    }
                }
                packed[(r * bits + b) * kw + t] = word;
            }
        }
    }
    return BSREF_OK;
}

int bsref_pack_ex(const uint8_t *q, uint32_t *packed, int64_t outer,
                  int64_t k, int64_t inner, int bits, int layout)
{
    if (!q || !packed || outer < 0 || inner < 1 || k < 1 || bits < 1 ||
        bits > 8)
        return BSREF_EINVAL;
    if (layout != BSREF_LAYOUT_MBK && layout != BSREF_LAYOUT_MKB &&
        layout != BSREF_LAYOUT_BMK)
        return BSREF_EINVAL;
    const int64_t kw = words_for(k);
    const int64_t rows = outer * inner;
    for (int64_t o = 0; o < outer; ++o) {
        for (int64_t i = 0; i < inner; ++i) {
            const int64_t r = o * inner + i;
            for (int b = 0; b < bits; ++b) {
                for (int64_t t = 0; t < kw; ++t) {
                    uint32_t word = 0;
                    for (int u = 0; u < 32; ++u) {
                        int64_t e = 32 * t + u;
                        if (e < k) {
                            uint8_t v = q[(o * k + e) * inner + i];
                            word |= (((uint32_t)v >> b) & 1u) << u;
                        }
                    }
                    int64_t at;
                    if (layout == BSREF_LAYOUT_MBK)
                        at = (r * bits + b) * kw + t;
                    else if (layout == BSREF_LAYOUT_MKB)
                        at = (r * kw + t) * bits + b;
                    else
                        at = ((int64_t)b * rows + r) * kw + t;
                    packed[at] = word;
                }
            }
        }
    }
    return BSREF_OK;
}

/* ------------------------------------------------------------------------ */
/* Decoding of packed elements back to integer values.                        */
/* ------------------------------------------------------------------------ */

/* bit of channel c in plane `plane` of a [planes][kw] packed vector */
static int plane_bit(const uint32_t *vec, int64_t kw, int plane, int64_t c)
{
    return (int)((vec[plane * kw + c / 32] >> (c % 32)) & 1u);
}

/* integer value of element c of a [bits][kw] packed vector:
 *   unipolar  sum_j 2^j b_j
 *   bipolar   sum_j 2^j (2 b_j - 1)       (Sec. 2.2: bit 1 -> +1, 0 -> -1)
 *   signed    two's complement: the top plane weighs -2^(bits-1)
 *             (Sec. 2.2: binary dot products weighted by their sign) */
static int64_t code_value(const uint32_t *vec, int64_t kw, int bits, int enc,
                          int64_t c)
{
    int64_t v = 0;
    for (int j = 0; j < bits; ++j) {
        int64_t bit = plane_bit(vec, kw, j, c);
        int64_t level;
        if (enc == BSREF_BIPOLAR)
            level = 2 * bit - 1;
        else if (enc == BSREF_SIGNED && j == bits - 1)
            level = -bit;
        else
            level = bit;
        v += level * ((int64_t)1 << j);
    }
    return v;
}

static int valid_enc(int enc, int bits)
{
    if (enc == BSREF_UNIPOLAR || enc == BSREF_BIPOLAR)
        return 1;
    return enc == BSREF_SIGNED && bits >= 2;
}

/* ------------------------------------------------------------------------ */
/* Conv2d (Sec. 3.2): integer convolution of the decoded values.              */
/* ------------------------------------------------------------------------ */
int bsref_conv2d_out_shape(const bsref_conv2d_params *p, int32_t *oh,
                           int32_t *ow)
{
    if (!p || !oh || !ow)
        return BSREF_EINVAL;
    if (p->stride_h < 1 || p->stride_w < 1 || p->kh < 1 || p->kw < 1 ||
        p->pad_h < 0 || p->pad_w < 0)
        return BSREF_EINVAL;
    int64_t eh = (int64_t)p->h + 2 * (int64_t)p->pad_h - p->kh;
    int64_t ew = (int64_t)p->w + 2 * (int64_t)p->pad_w - p->kw;
    if (eh < 0 || ew < 0)
        return BSREF_EINVAL;
    *oh = (int32_t)(eh / p->stride_h + 1);
    *ow = (int32_t)(ew / p->stride_w + 1);
    return BSREF_OK;
}

static int check_conv(const bsref_conv2d_params *p, int32_t *oh, int32_t *ow)
{
    if (!p)
        return BSREF_EINVAL;
    if (p->n < 1 || p->h < 1 || p->w < 1 || p->c < 1 || p->oc < 1)
        return BSREF_EINVAL;
    if (p->abits < 1 || p->abits > 8 || p->wbits < 1 || p->wbits > 8)
        return BSREF_EINVAL;
    if (!valid_enc(p->aenc, p->abits) || !valid_enc(p->wenc, p->wbits))
        return BSREF_EINVAL;
    return bsref_conv2d_out_shape(p, oh, ow);
}

/* one output element, the definition written out */
static int64_t conv_point(const bsref_conv2d_params *p, const uint32_t *act,
                          const uint32_t *wts, int64_t nn, int64_t y,
                          int64_t x, int64_t o)
{
    const int64_t cw = words_for(p->c);
    int64_t sum = 0;
    for (int64_t r = 0; r < p->kh; ++r) {
        int64_t ih = y * p->stride_h - p->pad_h + r;
        if (ih < 0 || ih >= p->h)
            continue;                       /* zero padding */
        for (int64_t s = 0; s < p->kw; ++s) {
            int64_t iw = x * p->stride_w - p->pad_w + s;
            if (iw < 0 || iw >= p->w)
                continue;                   /* zero padding */
            const uint32_t *avec =
                act + ((nn * p->h + ih) * p->w + iw) * p->abits * cw;
            const uint32_t *wvec =
                wts + ((o * p->kh + r) * p->kw + s) * p->wbits * cw;
            for (int64_t c = 0; c < p->c; ++c)
                sum += code_value(avec, cw, p->abits, p->aenc, c) *
                       code_value(wvec, cw, p->wbits, p->wenc, c);
        }
    }
    return sum;
}

int bsref_conv2d(const bsref_conv2d_params *p, const uint32_t *act,
                 const uint32_t *wts, int32_t *out)
{
    int32_t oh, ow;
    if (!act || !wts || !out)
        return BSREF_EINVAL;
    int rc = check_conv(p, &oh, &ow);
    if (rc)
        return rc;
    int bad = 0;
    const int64_t rows = (int64_t)p->n * oh;
#pragma omp parallel for schedule(dynamic) reduction(| : bad)
    for (int64_t row = 0; row < rows; ++row) {
        int64_t nn = row / oh, y = row % oh;
        for (int64_t x = 0; x < ow; ++x) {
            for (int64_t o = 0; o < p->oc; ++o) {
                int64_t v = conv_point(p, act, wts, nn, y, x, o);
                if (v > INT32_MAX || v < INT32_MIN)
                    bad = 1;
                out[((nn * oh + y) * ow + x) * p->oc + o] = (int32_t)v;
            }
        }
    }
    return bad ? BSREF_ERANGE : BSREF_OK;
}

int bsref_conv2d_at(const bsref_conv2d_params *p, const uint32_t *act,
                    const uint32_t *wts, const int64_t *idx, int64_t count,
                    int32_t *vals)
{
    int32_t oh, ow;
    if (!act || !wts || !idx || !vals || count < 0)
        return BSREF_EINVAL;
    int rc = check_conv(p, &oh, &ow);
    if (rc)
        return rc;
    const int64_t total = (int64_t)p->n * oh * ow * p->oc;
    for (int64_t i = 0; i < count; ++i)
        if (idx[i] < 0 || idx[i] >= total)
            return BSREF_EINVAL;
    int bad = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : bad)
    for (int64_t i = 0; i < count; ++i) {
        int64_t f = idx[i];
        int64_t o = f % p->oc;
        f /= p->oc;
        int64_t x = f % ow;
        f /= ow;
        int64_t y = f % oh;
        int64_t nn = f / oh;
        int64_t v = conv_point(p, act, wts, nn, y, x, o);
        if (v > INT32_MAX || v < INT32_MIN)
            bad = 1;
        vals[i] = (int32_t)v;
    }
    return bad ? BSREF_ERANGE : BSREF_OK;
}

/* ------------------------------------------------------------------------ */
/* Dense (Sec. 3.2, Sec. 6.2.1): out[m][n] = sum_k a(m,k) w(n,k).             */
/* ------------------------------------------------------------------------ */
int bsref_dense_ex(int64_t m, int64_t n, int64_t k, int abits, int aenc,
                   int wbits, int wenc, const uint32_t *a, const uint32_t *w,
                   int32_t *out)
{
    if (!a || !w || !out || m < 1 || n < 1 || k < 1)
        return BSREF_EINVAL;
    if (abits < 1 || abits > 8 || wbits < 1 || wbits > 8)
        return BSREF_EINVAL;
    if (!valid_enc(aenc, abits) || !valid_enc(wenc, wbits))
        return BSREF_EINVAL;
    const int64_t kw = words_for(k);
    int bad = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : bad)
    for (int64_t i = 0; i < m; ++i) {
        const uint32_t *avec = a + i * abits * kw;
        for (int64_t j = 0; j < n; ++j) {
            const uint32_t *wvec = w + j * wbits * kw;
            int64_t sum = 0;
            for (int64_t c = 0; c < k; ++c)
                sum += code_value(avec, kw, abits, aenc, c) *
                       code_value(wvec, kw, wbits, wenc, c);
            if (sum > INT32_MAX || sum < INT32_MIN)
                bad = 1;
            out[i * n + j] = (int32_t)sum;
        }
    }
    return bad ? BSREF_ERANGE : BSREF_OK;
}

int bsref_dense(int64_t m, int64_t n, int64_t k, int abits, int wbits,
                int wenc, const uint32_t *a, const uint32_t *w, int32_t *out)
{
    return bsref_dense_ex(m, n, k, abits, BSREF_UNIPOLAR, wbits, wenc, a, w,
                          out);
}
