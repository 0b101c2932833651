/*
 * int8_mfma.h -- C ABI of libint8mfma.so: an int8 matrix-core convolution for
 * AMD MI355X (gfx950), kept as a labelled COMPARISON BASELINE.  It is not the
 * bitserial method: it multiplies the integer codes themselves on the MFMA
 * units, the GPU counterpart of the paper's 8- and 16-bit integer baselines
 * (Sec. 6.2.1 and 6.2.2 compare bitserial operators against quantized
 * integer ones).  Nothing in libbitserial.so calls it.
 *
 * Conventions: device pointers owned by the caller, 16-byte aligned; the call
 * is asynchronous on `stream` (a hipStream_t, NULL = null stream); arguments
 * are validated on the host before anything is enqueued, and an invalid call
 * enqueues nothing.  Results are exact int32 sums (the caller keeps them
 * within int32: at most 127 * 128 * kh * kw * c in magnitude).
 */
#ifndef INT8_MFMA_H
#define INT8_MFMA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    I8MFMA_OK = 0,
    I8MFMA_ERR_INVALID_ARG = 1,   /* NULL/misaligned pointer, bad size */
    I8MFMA_ERR_UNSUPPORTED = 2,   /* a shape this kernel does not cover */
    I8MFMA_ERR_HIP = 4            /* the HIP runtime refused the launch */
};

typedef struct {
    int32_t n, h, w, c;        /* NHWC input */
    int32_t oc, kh, kw;        /* OHWI filters */
    int32_t stride, pad;       /* both axes */
} i8mfma_conv_params;

/* Direct (implicit-GEMM) convolution of int8 NHWC activations with int8
 * OHWI filters, zero padding, int32 NHWC output:
 *   out[n][y][x][o] = sum over in-range taps (r, s) and channels c of
 *                     act[n][y*stride - pad + r][x*stride - pad + s][c] *
 *                     wts[o][r][s][c]
 * act: [n][h][w][c] int8, wts: [oc][kh][kw][c] int8, out: [n][oh][ow][oc]
 * int32 with oh = (h + 2 pad - kh) / stride + 1 (ow likewise), every
 * element written.  Each wave computes 32 output pixels x 64 output channels
 * with v_mfma_i32_16x16x64_i8 (one 64-channel slice of one tap per
 * instruction); the filters are staged once per persistent workgroup in LDS.
 * Covers kh == kw, c a multiple of 64, oc a multiple of 64, oc*kh*kw*c
 * <= 64 KiB of filters, tensors below 2 GiB; I8MFMA_ERR_UNSUPPORTED
 * otherwise.  I8MFMA_ERR_INVALID_ARG for NULL or misaligned pointers,
 * non-positive sizes, stride < 1, pad < 0, or oh, ow < 1. */
int i8mfma_conv2d(const i8mfma_conv_params *p, const int8_t *act,
                  const int8_t *wts, int32_t *out, void *stream);

/* Detail of the last error on the calling thread ("" if none). */
const char *i8mfma_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* INT8_MFMA_H */
