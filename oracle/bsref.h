/*
 * bsref.h -- CPU oracle for low-precision bitserial operators.
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, slow, obviously correct host
 * implementation of what the GPU library computes.  Only the tests, the smoke
 * check and the benchmark's CPU-baseline leg may load it; the product path
 * never does.  It shares no source, header, table or helper with the GPU
 * library: every definition below is written out from the paper
 * ("Automating Generation of Low Precision Deep Learning Operators",
 * Cowan, Moreau, Chen, Ceze) and the readings listed in the design notes.
 *
 * All pointers are HOST pointers owned by the caller.  Every function returns
 * 0 on success and a nonzero code on an invalid argument, in which case it
 * has written nothing.
 */
#ifndef BSREF_H
#define BSREF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BSREF_OK 0
#define BSREF_EINVAL 1
#define BSREF_ERANGE 3

#define BSREF_UNIPOLAR 0
#define BSREF_BIPOLAR 1
#define BSREF_SIGNED 2

/* Packed layouts (Sec. 3.1, bitpacking operator): where the bit axis B sits
 * relative to the row axis M and the packed reduction axis K'. */
#define BSREF_LAYOUT_MBK 0   /* [rows][bits][words] */
#define BSREF_LAYOUT_MKB 1   /* [rows][words][bits] */
#define BSREF_LAYOUT_BMK 2   /* [bits][rows][words] */

/* Quantization of float data to k bits (Sec. 3.1; contribution list, Sec. 1).
 * The paper names the operator but prints no formula.  Reading used here:
 *   unipolar: q = clamp(round_half_even(fl32(x * scale)), 0, 2^bits - 1),
 *             NaN -> 0, +inf -> 2^bits - 1, -inf -> 0, denormals kept;
 *   bipolar (bits == 1 only): q = 1 if x >= 0 (so -0.0 -> 1) else 0, NaN -> 0;
 *             bit 1 encodes +1 and bit 0 encodes -1 (Sec. 2.2, bipolar format);
 *   signed (bits >= 2): v = clamp(round_half_even(fl32(x * scale)),
 *             -2^(bits-1), 2^(bits-1) - 1), NaN -> 0, stored as the low `bits`
 *             bits of v in two's complement (Sec. 2.2, signed data).
 * x: [n] float32, q: [n] uint8.  scale must be finite and > 0. */
int bsref_quantize(const float *x, uint8_t *q, int64_t n, float scale,
                   int bits, int enc);

/* Bit packing (Sec. 2.2 "bitpacked"; Sec. 3.1 bitpacking operator, layout MBK').
 * q: [rows][k] uint8 -> packed: [rows][bits][ceil(k/32)] uint32 where bit u of
 * word t of plane b is bit b of q[r][32t+u]; bits past k are 0; bits of q at or
 * above `bits` are ignored. */
int bsref_pack(const uint8_t *q, uint32_t *packed, int64_t rows, int64_t k,
               int bits);

/* General bit packing (Sec. 3.1): the input is viewed as [outer][k][inner]
 * with the reduction axis k at stride `inner` (inner = 1 is bsref_pack's
 * [rows][k]; NCHW activations are outer = n, k = c, inner = h*w, and OIHW
 * filters outer = oc, k = c, inner = kh*kw).  Row r = o*inner + i of the packed
 * tensor holds the k elements q[o][.][i]; the bit axis sits where `layout`
 * says (BSREF_LAYOUT_*).  Word and bit order as in bsref_pack. */
int bsref_pack_ex(const uint8_t *q, uint32_t *packed, int64_t outer,
                  int64_t k, int64_t inner, int bits, int layout);

/* Bitserial 2-D convolution, NHWC activations, OHWI filters (Sec. 3.2).
 * The bitserial form (Eq. 1, Eq. 2) reaches exactly the integer convolution of
 * the quantized values, so this oracle computes that convolution as written:
 * decode each packed element to its integer value and sum products.  The same
 * decoding applies to activations (aenc) and weights (wenc), with b_j the bit
 * of plane j and B the bit-width:
 *   unipolar  v = sum_j 2^j b_j
 *   bipolar   v = sum_j 2^j (2 b_j - 1)        (B = 1: bit 1 -> +1, 0 -> -1)
 *   signed    v = sum_{j<B-1} 2^j b_j - 2^(B-1) b_{B-1}   (B >= 2)
 *   out[n][oh][ow][o] = sum over in-range taps (kh,kw) and channels c of a*w;
 * taps that fall in the padding contribute nothing (zero padding of the value
 * tensor, also for bipolar activations).
 * act: [n][h][w][abits][ceil(c/32)], wts: [oc][kh][kw][wbits][ceil(c/32)],
 * out: [n][oh][ow][oc] int32 with oh = (h + 2 pad_h - kh) / stride_h + 1. */
typedef struct {
    int32_t n, h, w, c;
    int32_t oc, kh, kw;
    int32_t stride_h, stride_w, pad_h, pad_w;
    int32_t abits, wbits;
    int32_t aenc, wenc;
} bsref_conv2d_params;

int bsref_conv2d_out_shape(const bsref_conv2d_params *p, int32_t *oh,
                           int32_t *ow);
int bsref_conv2d(const bsref_conv2d_params *p, const uint32_t *act,
                 const uint32_t *wts, int32_t *out);
/* Same definition, evaluated only at the flat output indices idx[0..count)
 * (index into [n][oh][ow][oc]); vals[i] receives the output at idx[i]. */
int bsref_conv2d_at(const bsref_conv2d_params *p, const uint32_t *act,
                    const uint32_t *wts, const int64_t *idx, int64_t count,
                    int32_t *vals);

/* Bitserial dense / matrix multiply (Sec. 3.2; evaluated in Sec. 6.2.1):
 * out[m][n] = sum_k a(m,k) * w(n,k) with the value decoding above.
 * a: [m][abits][ceil(k/32)], w: [n][wbits][ceil(k/32)], out: [m][n] int32. */
int bsref_dense(int64_t m, int64_t n, int64_t k, int abits, int wbits,
                int wenc, const uint32_t *a, const uint32_t *w, int32_t *out);
/* The same with an activation encoding as well. */
int bsref_dense_ex(int64_t m, int64_t n, int64_t k, int abits, int aenc,
                   int wbits, int wenc, const uint32_t *a, const uint32_t *w,
                   int32_t *out);

/* Number of host threads the oracle's parallel loops use. */
int bsref_threads(void);

/* Sets that number for later calls on the calling thread (n >= 1; the
 * results do not depend on it).  Returns BSREF_EINVAL for n < 1. */
int bsref_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif /* BSREF_H */
